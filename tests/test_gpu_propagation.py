"""Propagation study on the GPU (paper Sec. 3, Table 2): the unprotected
layer (same kernels, checks off) with one fault in Q, K, V, AS or CL -
INF, NaN, or a near-INF value made by flipping the exponent MSB of the
stored element - and the pattern of the errors it leaves in the
downstream matrices. Each pattern is checked against the paper's Table 2
(golden fixture) and against the oracle run with the same fault; the
error type where it follows from IEEE arithmetic alone (as in the
oracle's own Table 2 test)."""
import os

import numpy as np
import pytest
import torch

import workloads as W
from oracle import OracleParams, forward

GOLDEN = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden")
TN = 1e10


def _table2():
    rows = []
    with open(os.path.join(GOLDEN, "table2_propagation.txt")) as fh:
        for line in fh:
            line = line.strip()
            if line and not line.startswith("#"):
                rows.append(tuple(line.split()))
    return rows


def pattern(bad):
    """1R / 1C / 2D / 0D of a boolean error map of one matrix (Sec. 2.2)."""
    r, c = np.nonzero(bad)
    if len(r) == 0:
        return "-"
    if len(set(r)) == 1:
        return "1R" if len(set(c)) > 1 else "0D"
    if len(set(c)) == 1:
        return "1C"
    return "2D"


def type_class(vals):
    nan, inf = np.isnan(vals), np.isinf(vals)
    near = np.isfinite(vals) & (np.abs(vals) >= TN)
    if int(nan.any()) + int(inf.any()) + int(near.any()) > 1:
        return "M"
    if nan.all():
        return "nan"
    if inf.all():
        return "inf*" if (vals > 0).any() and (vals < 0).any() else "inf"
    return "near"


def error_map(mat, ref, near_inf_injection):
    bad = ~np.isfinite(mat) | (np.abs(np.nan_to_num(mat)) >= TN)
    if near_inf_injection:
        bad |= np.isfinite(mat) & (np.abs(mat - ref) > 1e-3 * (1 + np.abs(ref)))
    return bad


@pytest.mark.gpu
def test_table2_propagation_patterns_on_gpu():
    from paper_2410_11720_amd import abft
    sh = W.make_shape(1, 64, 128, 2, dtype="f32", block_rows=64)
    inp = W.make_inputs(sh, 8)
    cfg = abft.LayerConfig(sh.batch, sh.seq, sh.hidden, sh.heads, dtype="f32", block_rows=64,
                           protect=False)
    layer = abft.ProtectedAttention(cfg)
    X, Wqkv, Wo = (torch.from_numpy(np.ascontiguousarray(inp[k], dtype=np.float32)).to("cuda")
                   for k in ("X", "Wqkv", "Wo"))

    def gpu_run(faults=()):
        O = layer.forward(X, Wqkv, Wo, abft.faults_to_device(list(faults)))
        torch.cuda.synchronize()
        t = {k: layer.tensor(k).cpu().numpy().astype(np.float64) for k in ("QKV", "AS", "AP", "CL")}
        t["O"] = O.cpu().numpy().astype(np.float64)
        return t

    p = OracleParams(heads=2, dtype="f32", block_rows=64, protect=False)
    base_g = gpu_run()
    base_o = forward(inp["X"], inp["Wqkv"], inp["Wo"], p)
    H, d, h, i = 128, 64, 1, 17

    def source(t, fi, j):
        return {"Q": t["QKV"][0, i, h * d + j], "K": t["QKV"][0, i, H + h * d + j],
                "V": t["QKV"][0, i, 2 * H + h * d + j], "AS": t["AS"][0, h, i, j],
                "CL": t["CL"][0, i, h * d + j]}[fi]

    checked = 0
    for (etype, fi, down, want, ptype) in _table2():
        # a positive element below 1, so that the exponent flip makes a
        # positive near-INF value (a negative one in AS would only drop out
        # of the softmax row); the same element in both runs
        j = next(j for j in range(3, d) if 0.05 < source(base_g, fi, j) < 0.9
                 and 0.05 < source(base_o, fi, j) < 0.9)
        if etype == "nINF":
            fault = W.Fault(fi, 0, h, i, j, 0.0, mode="flip")
        else:
            fault = W.Fault(fi, 0, h, i, j, np.inf if etype == "INF" else np.nan)
        print(f"[case] {etype} {fi} -> {down}", flush=True)
        g = gpu_run([fault])
        o = forward(inp["X"], inp["Wqkv"], inp["Wo"], p, [fault])
        pick = {"AS": lambda t: t["AS"][0, h], "AP": lambda t: t["AP"][0, h],
                "CL": lambda t: t["CL"][0], "O": lambda t: t["O"][0]}[down]
        nflip = etype == "nINF"
        bad_g = error_map(pick(g), pick(base_g), nflip)
        bad_o = error_map(pick(o), pick(base_o), nflip)
        assert pattern(bad_g) == want, (etype, fi, down, pattern(bad_g))
        assert pattern(bad_o) == want, (etype, fi, down, "oracle", pattern(bad_o))
        if not (fi == "V" or nflip):
            got = type_class(pick(g)[bad_g])
            assert got == type_class(pick(o)[bad_o]), (etype, fi, down)
            assert got == ptype or (ptype == "inf" and got == "inf*"), (etype, fi, down, got)
        checked += 1
    assert checked == 42


@pytest.mark.gpu
def test_exponent_flip_fault_matches_oracle_value():
    """The flip injector writes the same stored value on both sides, in a
    bf16 GEMM output (Q) and an fp32 weight gradient (dWQ)."""
    from paper_2410_11720_amd import abft
    sh = W.make_shape(1, 128, 128, 2, dtype="bf16")
    inp = W.make_inputs(sh, 5)
    cfg = abft.LayerConfig(sh.batch, sh.seq, sh.hidden, sh.heads, protect=False)
    layer = abft.ProtectedAttention(cfg)
    X, Wqkv, Wo, dO = (torch.from_numpy(np.ascontiguousarray(inp[k], dtype=np.float32))
                       .to("cuda").to(torch.bfloat16) for k in ("X", "Wqkv", "Wo", "dO"))
    layer.forward(X, Wqkv, Wo)
    _, dW0, _ = layer.backward(dO, X, Wqkv, Wo)
    torch.cuda.synchronize()
    q0 = layer.tensor("QKV").float().cpu().numpy()
    dW0 = dW0.cpu().numpy()
    # backward alone first (the forward's Q fault would change every dW)
    layer.forward(X, Wqkv, Wo)
    _, dW1, _ = layer.backward(dO, X, Wqkv, Wo, abft.faults_to_device(
        [W.Fault("dWQ", 0, 0, 5, 9, 0.0, mode="flip")]))
    torch.cuda.synchronize()
    dW1 = dW1.cpu().numpy()
    layer.forward(X, Wqkv, Wo, abft.faults_to_device([W.Fault("Q", 0, 1, 33, 7, 0.0, mode="flip")]))
    torch.cuda.synchronize()
    q1 = layer.tensor("QKV").float().cpu().numpy()
    from oracle.numerics import flip_exponent_msb
    assert q1[0, 33, 64 + 7] == np.float32(flip_exponent_msb(float(q0[0, 33, 64 + 7]), "bf16"))
    assert dW1[5, 9] == np.float32(flip_exponent_msb(float(dW0[5, 9]), "f32"))
    assert np.argwhere(q1 != q0).tolist() == [[0, 33, 71]]
    assert np.argwhere(dW1 != dW0).tolist() == [[5, 9]]
