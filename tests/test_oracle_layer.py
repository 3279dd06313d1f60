"""Pins of the oracle's protected attention layer.

Pins: torch CPU autograd in float64 (an independent implementation of the
same layer, Sec. 2.1 Eq. 1-2), central finite differences of the oracle's
own forward, closed-form invariants of softmax and its backward, the
paper's Table 2 propagation patterns (golden fixture), zero false
positives with a recorded margin, exact restoration of injected faults
(Sec. 5.2: every injected error detected and corrected to its original
value), and the 1-D handling of Sec. 4.3 in the paper-literal mode.
"""
import os

import numpy as np
import pytest
import torch

import workloads as W
from oracle import OracleParams, forward, backward, pattern_of_events
from oracle.eec import col_checksums
from oracle.numerics import round_to

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def _torch_layer(X, Wqkv, Wo, dO, heads, causal, scale=None):
    X = torch.tensor(X, dtype=torch.float64, requires_grad=True)
    Wqkv = torch.tensor(Wqkv, dtype=torch.float64, requires_grad=True)
    Wo = torch.tensor(Wo, dtype=torch.float64, requires_grad=True)
    B, S, H = X.shape
    d = H // heads
    qkv = X @ Wqkv
    q, k, v = qkv.split(H, dim=-1)
    sh = lambda t: t.reshape(B, S, heads, d).transpose(1, 2)
    q, k, v = sh(q), sh(k), sh(v)
    s = (q @ k.transpose(-1, -2)) * (scale if scale else 1.0 / np.sqrt(d))
    if causal:
        s = s.masked_fill(~torch.ones(S, S, dtype=torch.bool).tril(), float("-inf"))
    p = torch.softmax(s, dim=-1)
    cl = (p @ v).transpose(1, 2).reshape(B, S, H)
    o = cl @ Wo
    (o * torch.tensor(dO, dtype=torch.float64)).sum().backward()
    return o.detach().numpy(), X.grad.numpy(), Wqkv.grad.numpy(), Wo.grad.numpy()


@pytest.mark.parametrize("causal", [False, True])
def test_matches_torch_autograd_in_float64(causal):
    sh = W.make_shape(2, 64, 48, 3, causal=causal, dtype="f32", block_rows=16)
    inp = W.make_inputs(sh, 11)
    p = OracleParams(heads=3, causal=causal, dtype="f64", block_rows=16)
    f = forward(inp["X"], inp["Wqkv"], inp["Wo"], p)
    b = backward(f, inp["dO"], p)
    o, dx, dwqkv, dwo = _torch_layer(inp["X"], inp["Wqkv"], inp["Wo"], inp["dO"], 3, causal)
    for ours, ref in ((f["O"], o), (b["dX"], dx), (b["dWqkv"], dwqkv), (b["dWo"], dwo)):
        assert np.allclose(ours, ref, rtol=1e-10, atol=1e-12)
    assert f["events"] == [] and b["events"] == []


def test_backward_matches_central_differences():
    sh = W.make_shape(1, 8, 8, 2, causal=True, dtype="f32", block_rows=4, w_std=0.5)
    inp = W.make_inputs(sh, 3)
    p = OracleParams(heads=2, causal=True, dtype="f64", block_rows=4)
    X, Wqkv, Wo, dO = (inp[k].astype(np.float64) for k in ("X", "Wqkv", "Wo", "dO"))
    b = backward(forward(X, Wqkv, Wo, p), dO, p)
    loss = lambda X_, Wq_, Wo_: float((forward(X_, Wq_, Wo_, p)["O"] * dO).sum())
    h = 1e-6
    rng = np.random.default_rng(0)
    for name, arr, grad in (("X", X, b["dX"]), ("Wqkv", Wqkv, b["dWqkv"]), ("Wo", Wo, b["dWo"])):
        for _ in range(6):
            idx = tuple(int(rng.integers(n)) for n in arr.shape)
            up, dn = arr.copy(), arr.copy()
            up[idx] += h
            dn[idx] -= h
            args = {"X": (X, Wqkv, Wo), "Wqkv": (X, Wqkv, Wo), "Wo": (X, Wqkv, Wo)}[name]
            a_up = [up if a is arr else a for a in args]
            a_dn = [dn if a is arr else a for a in args]
            fd = (loss(*a_up) - loss(*a_dn)) / (2 * h)
            assert abs(fd - grad[idx]) < 1e-6 * max(1.0, abs(fd)), (name, idx)


@pytest.fixture(scope="module")
def bf16_run():
    sh = W.make_shape(2, 256, 128, 2, causal=True, dtype="bf16")
    inp = W.make_inputs(sh, 21)
    p = OracleParams(heads=2, causal=True, dtype="bf16", block_rows=128)
    f = forward(inp["X"], inp["Wqkv"], inp["Wo"], p)
    b = backward(f, inp["dO"], p)
    return sh, inp, p, f, b


def test_softmax_invariants(bf16_run):
    sh, inp, p, f, b = bf16_run
    AP, dAS = f["AP"], b["dAS"]
    S = sh.seq
    upper = ~np.tril(np.ones((S, S), dtype=bool))
    assert np.all(AP[..., upper] == 0.0) and np.all(dAS[..., upper] == 0.0)
    # rows of AP sum to one up to storage rounding of each entry
    assert np.max(np.abs(AP.sum(-1) - 1.0)) <= 2.0 ** -8 * 1.01
    # Without storage rounding, rows of AP sum to one and rows of dAS to zero
    # (sum_j AP_j (dAP_j - D) = D (1 - sum_j AP_j)); so does the sum over keys
    # of dK: sum_j dK_j = sum_i (sum_j dAS_ij) Q_i.
    p64 = OracleParams(heads=2, causal=True, dtype="f64", block_rows=128)
    f64 = forward(inp["X"], inp["Wqkv"], inp["Wo"], p64)
    b64 = backward(f64, inp["dO"], p64)
    assert np.max(np.abs(f64["AP"].sum(-1) - 1.0)) < 1e-14
    assert np.all(np.abs(b64["dAS"].sum(-1)) <= 1e-14 * np.abs(b64["dAS"]).sum(-1) + 1e-300)
    dK = b64["dQKV"][..., sh.hidden:2 * sh.hidden]
    assert np.max(np.abs(dK.sum(axis=1))) < 1e-12 * np.abs(dK).sum(axis=1).max()


def _max_margin(f, b, p, sh):
    """max |delta1| / E over every checksum vector of QKV, O and dX."""
    e_rel = p.e_rel_value()
    worst = 0.0
    dXc = b["dQKVc"] @ f["Wqkv"].T
    for C, Cc in ((f["QKV"], f["QKVc"]), (f["O"], f["Oc"]), (b["dX"], dXc)):
        r = col_checksums(C, p.block_rows)
        n, rows, cols = C.shape
        absum = np.abs(C.reshape(n, rows // p.block_rows, p.block_rows, cols)).sum(2)
        worst = max(worst, float(np.max(np.abs(Cc[:, :, 0] - r[:, :, 0]) / (e_rel * absum))))
    return worst


@pytest.mark.parametrize("seed", range(8))
def test_zero_false_positives_bf16(seed):
    sh = W.make_shape(2, 256, 128, 2, causal=bool(seed % 2), dtype="bf16")
    inp = W.make_inputs(sh, 100 + seed)
    p = OracleParams(heads=2, causal=sh.causal, dtype="bf16")
    f = forward(inp["X"], inp["Wqkv"], inp["Wo"], p)
    b = backward(f, inp["dO"], p)
    assert f["events"] == [] and b["events"] == []
    # fault-free differences stay at least 4x inside the detection bound
    assert _max_margin(f, b, p, sh) <= 1.0 / 4


def test_zero_false_positives_fp32_config_shape():
    sh = W.C1
    inp = W.make_inputs(sh, W.data_seed("c1"))
    p = OracleParams(heads=1, dtype="f32", block_rows=128)
    f = forward(inp["X"], inp["Wqkv"], inp["Wo"], p)
    b = backward(f, inp["dO"], p)
    assert f["events"] == [] and b["events"] == []
    assert _max_margin(f, b, p, sh) <= 1.0 / 64


KINDS = {"inf": "INF", "-inf": "INF", "nan": "NAN", "+1e10": "NEAR_INF",
         "-1e10": "NEAR_INF", "1e30": "NEAR_INF", "1e6": "NUMERIC"}


@pytest.mark.parametrize("causal", [False, True])
def test_every_op_every_kind_is_restored_exactly(bf16_run, causal):
    sh = W.make_shape(2, 256, 128, 2, causal=causal, dtype="bf16")
    inp = W.make_inputs(sh, 31)
    p = OracleParams(heads=2, causal=causal, dtype="bf16")
    f0 = forward(inp["X"], inp["Wqkv"], inp["Wo"], p)
    b0 = backward(f0, inp["dO"], p)
    seed = 500 + int(causal)
    for op in W.ALL_OPS:
        for kind in KINDS:
            seed += 1
            faults = W.draw_faults(sh, seed, 1, [op], [kind])
            f = forward(inp["X"], inp["Wqkv"], inp["Wo"], p, faults)
            b = backward(f, inp["dO"], p, faults)
            evs = f["events"] + b["events"]
            fl = faults[0]
            assert [e[:5] for e in evs] == [(fl.op, fl.b, fl.h, fl.row, fl.col)], (op, kind, evs)
            assert evs[0][5] == KINDS[kind] and evs[0][6] == "RECOMPUTE"
            assert pattern_of_events(evs) == ["0D"]
            for k in ("O", "QKV", "AP", "CL"):
                assert np.array_equal(f[k], f0[k], equal_nan=False), (op, kind, k)
            for k in ("dX", "dWqkv", "dWo"):
                assert np.array_equal(b[k], b0[k]), (op, kind, k)


def test_multi_fault_step_across_fwd_and_bwd():
    sh = W.make_shape(2, 256, 128, 2, causal=True, dtype="bf16")
    inp = W.make_inputs(sh, 41)
    p = OracleParams(heads=2, causal=True, dtype="bf16")
    f0 = forward(inp["X"], inp["Wqkv"], inp["Wo"], p)
    b0 = backward(f0, inp["dO"], p)
    faults = W.draw_faults(sh, 77, 16, W.ALL_OPS, ["inf", "nan", "1e6", "1e10", "1e30"])
    f = forward(inp["X"], inp["Wqkv"], inp["Wo"], p, faults)
    b = backward(f, inp["dO"], p, faults)
    got = sorted(e[:5] for e in f["events"] + b["events"])
    assert got == sorted((x.op, x.b, x.h, x.row, x.col) for x in faults)
    assert np.array_equal(f["O"], f0["O"]) and np.array_equal(b["dX"], b0["dX"])
    assert np.array_equal(b["dWqkv"], b0["dWqkv"]) and np.array_equal(b["dWo"], b0["dWo"])


def test_two_faults_in_one_column_vector_of_as_go_to_the_row_pass():
    sh = W.make_shape(1, 128, 64, 1, dtype="bf16")
    inp = W.make_inputs(sh, 5)
    p = OracleParams(heads=1, dtype="bf16")
    f0 = forward(inp["X"], inp["Wqkv"], inp["Wo"], p)
    faults = [W.Fault("AS", 0, 0, 10, 7, np.inf), W.Fault("AS", 0, 0, 90, 7, np.nan)]
    f = forward(inp["X"], inp["Wqkv"], inp["Wo"], p, faults)
    assert sorted(e[:5] for e in f["events"]) == [("AS", 0, 0, 10, 7), ("AS", 0, 0, 90, 7)]
    assert np.array_equal(f["O"], f0["O"])
    # a 2x2 block of faults is beyond 1-D: reported, never silently passed
    faults = [W.Fault("AS", 0, 0, r, c, np.inf) for r in (3, 50) for c in (4, 60)]
    f = forward(inp["X"], inp["Wqkv"], inp["Wo"], p, faults)
    assert {e[6] for e in f["events"]} == {"UNCORRECTABLE"}
    assert set(pattern_of_events(f["events"])) == {"2D"}


def _load_table2():
    rows = []
    with open(os.path.join(GOLDEN, "table2_propagation.txt")) as fh:
        for line in fh:
            line = line.strip()
            if line and not line.startswith("#"):
                rows.append(tuple(line.split()))
    return rows


def _pattern(bad):
    """1R / 1C / 2D of a boolean [S, cols] error map (Sec. 2.2)."""
    r, c = np.nonzero(bad)
    if len(r) == 0:
        return "-"
    if len(set(r)) == 1:
        return "1R" if len(set(c)) > 1 else "0D"
    if len(set(c)) == 1:
        return "1C"
    return "2D"


def _type_class(vals, tn):
    nan = np.isnan(vals)
    inf = np.isinf(vals)
    near = np.isfinite(vals) & (np.abs(vals) >= tn)
    classes = int(nan.any()) + int(inf.any()) + int(near.any())
    if classes > 1:
        return "M"
    if nan.all():
        return "nan"
    if inf.all():
        return "inf*" if (vals > 0).any() and (vals < 0).any() else "inf"
    return "near"


def _msb_flip_f32(x):
    """Flip the most significant exponent bit (bit 30) of a float32."""
    u = np.array([x], dtype=np.float32).view(np.uint32)
    return float((u ^ np.uint32(1 << 30)).view(np.float32)[0])


def test_table2_propagation_patterns_unprotected():
    """Unprotected forward (no checksums): one fault in Q, K, V, AS or CL and
    the pattern of the errors it leaves downstream (paper Table 2). Patterns
    are checked for every entry; the error type is checked where the
    paper's entry follows from IEEE arithmetic alone. The type of the V row
    (paper: mixture) and of near-INF injections depend on the magnitudes the
    trained models produced, which random-init layers do not reproduce, so
    those types are not checked (their patterns are)."""
    sh = W.make_shape(1, 64, 64, 2, dtype="f32", block_rows=64)
    inp = W.make_inputs(sh, 8)
    p = OracleParams(heads=2, dtype="f32", block_rows=64, protect=False)
    base = forward(inp["X"], inp["Wqkv"], inp["Wo"], p)
    tn = 1e10
    i, j, h = 17, 5, 1            # row (token), head-local column, head
    checked = 0
    for (etype, fi, down, pattern, ptype) in _load_table2():
        if etype == "nINF":
            col = h * 32 + j if fi in ("Q", "K", "V", "CL") else j
            src = {"Q": base["QKV"][0, i, h * 32 + j], "K": base["QKV"][0, i, 64 + h * 32 + j],
                   "V": base["QKV"][0, i, 128 + h * 32 + j], "AS": base["AS"][0, h, i, j],
                   "CL": base["CL"][0, i, h * 32 + j]}[fi]
            val = _msb_flip_f32(src)
        else:
            val = np.inf if etype == "INF" else np.nan
        fault = W.Fault(fi, 0, h, i, j, val)
        f = forward(inp["X"], inp["Wqkv"], inp["Wo"], p, [fault])
        mat = {"AS": f["AS"][0, h], "AP": f["AP"][0, h], "CL": f["CL"][0], "O": f["O"][0]}[down]
        ref = {"AS": base["AS"][0, h], "AP": base["AP"][0, h], "CL": base["CL"][0], "O": base["O"][0]}[down]
        bad = ~np.isfinite(mat) | (np.abs(np.nan_to_num(mat)) >= tn)
        bad |= np.isfinite(mat) & (np.abs(mat - ref) > 1e-3 * (1 + np.abs(ref))) & (etype == "nINF")
        assert _pattern(bad) == pattern, (etype, fi, down)
        extreme = ~np.isfinite(mat) | (np.abs(np.nan_to_num(mat)) >= tn)
        type_checked = not (fi == "V" or etype == "nINF")
        if type_checked:
            got = _type_class(mat[extreme], tn)
            want = ptype
            if want == "inf":           # one sign in the paper's run; either sign here
                assert got in ("inf", "inf*"), (etype, fi, down, got)
            else:
                assert got == want, (etype, fi, down, got, want)
        checked += 1
    assert checked == 42


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_flip_fault_equals_writing_the_flipped_stored_value(dtype):
    """Mode "flip" writes the stored value with its exponent MSB flipped:
    the same run as mode "set" with that value computed by hand from the
    IEEE bit layout (bit 30 of the f32 word; bf16 is its upper half)."""
    sh = W.make_shape(1, 64, 64, 2, dtype=dtype, block_rows=64)
    inp = W.make_inputs(sh, 4)
    p = OracleParams(heads=2, dtype=dtype, block_rows=64, protect=False)
    base = forward(inp["X"], inp["Wqkv"], inp["Wo"], p)
    stored = base["CL"][0, 9, 32 + 3]
    word = np.array([stored], dtype=np.float32).view(np.uint32)[0]
    flipped = float(np.array([word ^ 0x40000000], dtype=np.uint32).view(np.float32)[0])
    a = forward(inp["X"], inp["Wqkv"], inp["Wo"], p, [W.Fault("CL", 0, 1, 9, 3, 0.0, mode="flip")])
    b = forward(inp["X"], inp["Wqkv"], inp["Wo"], p, [W.Fault("CL", 0, 1, 9, 3, flipped)])
    assert a["CL"][0, 9, 35] == flipped
    assert np.array_equal(a["O"], b["O"], equal_nan=True)


def test_paper_literal_mode_corrects_1d_patterns_in_as_and_cl():
    """Root check off: Q/K/V errors reach AS and CL as 1-D patterns and are
    corrected there from checksums (Sec. 4.3, Sec. 4.4)."""
    sh = W.make_shape(1, 128, 64, 2, dtype="bf16")
    inp = W.make_inputs(sh, 13)
    p = OracleParams(heads=2, dtype="f64", root_check=False)
    X, Wq, Wo = (round_to(inp[k], "bf16") for k in ("X", "Wqkv", "Wo"))
    f0 = forward(X, Wq, Wo, p)
    for op, where, pat in (("Q", "AS", "1R"), ("K", "AS", "1C"), ("V", "CL", "1C")):
        f = forward(X, Wq, Wo, p, [W.Fault(op, 0, 1, 40, 9, np.inf)])
        evs = f["events"]
        assert evs and {e[0] for e in evs} == {where}
        assert set(pattern_of_events(evs)) == {pat}
        assert {e[6] for e in evs} == {"RECONSTRUCT"}
        assert np.allclose(f["O"], f0["O"], rtol=1e-9, atol=1e-12), op


def test_disabled_section_leaves_faults_in_place():
    sh = W.make_shape(1, 128, 64, 1, dtype="bf16")
    inp = W.make_inputs(sh, 17)
    p = OracleParams(heads=1, dtype="bf16", sections=("CL", "O", "BWD"))
    f = forward(inp["X"], inp["Wqkv"], inp["Wo"], p, [W.Fault("AS", 0, 0, 9, 3, np.inf)])
    # not caught at AS; the NaN row it leaves in AP reaches CL, whose check
    # cannot repair it from the corrupted AP and reports it uncorrectable
    assert not any(e[0] == "AS" for e in f["events"])
    assert any(e[0] == "CL" and e[6] == "UNCORRECTABLE" for e in f["events"])
    assert np.isnan(f["O"][0, 9]).all()
    f = forward(inp["X"], inp["Wqkv"], inp["Wo"], p, [W.Fault("CL", 0, 0, 9, 3, np.inf)])
    assert [e[:5] for e in f["events"]] == [("CL", 0, 0, 9, 3)]


def test_masked_products_equal_dense_products_on_finite_inputs():
    """Masked products leave out exact zeros only, so on finite inputs
    they equal the dense products."""
    from oracle.layer import (masked_rows_product, masked_cols_product,
                              masked_block_rows_product, masked_block_cols_product)
    rng = np.random.default_rng(4)
    S, R, n = 320, 64, 5
    P = np.tril(rng.standard_normal((2, S, S)))
    M = rng.standard_normal((2, S, n))
    assert np.allclose(masked_rows_product(P, M, True), P @ M, rtol=1e-12, atol=1e-12)
    assert np.allclose(masked_cols_product(P, M, True), P.swapaxes(-1, -2) @ M,
                       rtol=1e-12, atol=1e-12)
    Pc = col_checksums(P, R)
    assert np.allclose(masked_block_rows_product(Pc, M, R, True), Pc @ M[:, None],
                       rtol=1e-12, atol=1e-9)
    from oracle.eec import row_checksums
    Pr = row_checksums(P, R)
    dense = (Pr.reshape(2, S, -1).swapaxes(-1, -2) @ M).reshape(2, S // R, 2, n)
    assert np.allclose(masked_block_cols_product(Pr, M, R, True), dense, rtol=1e-12, atol=1e-9)


def test_masked_products_match_brute_force_sums_with_nonfinite_operands():
    """Eq. 1 under a causal mask: query i sums over keys j <= i only, key j
    over queries i >= j. Pinned against plain Python sums over the allowed
    pairs, with INF and NaN in the unmasked factor: a masked zero never
    meets them, so rows before an INF key stay finite."""
    from oracle.layer import (masked_rows_product, masked_cols_product,
                              masked_block_rows_product, masked_block_cols_product)
    from oracle.eec import row_checksums
    rng = np.random.default_rng(5)
    S, R, n = 12, 4, 3
    P = np.tril(rng.integers(-3, 4, (S, S)).astype(np.float64))
    M = rng.integers(-3, 4, (S, n)).astype(np.float64)
    M[7, 1] = np.inf
    M[3, 2] = np.nan

    def add(terms):
        acc = 0.0
        for t in terms:
            acc = acc + t
        return acc

    rows = np.array([[add(P[i, j] * M[j, c] for j in range(i + 1)) for c in range(n)]
                     for i in range(S)])
    cols = np.array([[add(P[i, j] * M[i, c] for i in range(j, S)) for c in range(n)]
                     for j in range(S)])
    with np.errstate(invalid="ignore"):
        assert np.array_equal(masked_rows_product(P, M, True), rows, equal_nan=True)
        assert np.array_equal(masked_cols_product(P, M, True), cols, equal_nan=True)
    # query rows before the INF key are finite (no 0 * INF), later ones not
    got = masked_rows_product(P, M, True)
    assert np.all(np.isfinite(got[:7, 1]))
    assert all(not np.isfinite(got[i, 1]) for i in range(7, S) if P[i, 7] != 0)
    # checksum rows of query blocks take the keys up to the block's last
    # query; of key blocks the queries from the block's first key
    Pc = col_checksums(P, R)
    want = np.array([[[add(Pc[qb, w, j] * M[j, c] for j in range((qb + 1) * R))
                       for c in range(n)] for w in range(2)] for qb in range(S // R)])
    with np.errstate(invalid="ignore"):
        assert np.array_equal(masked_block_rows_product(Pc, M, R, True), want, equal_nan=True)
    Pr = row_checksums(P, R)
    want = np.array([[[add(Pr[i, kb, w] * M[i, c] for i in range(kb * R, S))
                       for c in range(n)] for w in range(2)] for kb in range(S // R)])
    with np.errstate(invalid="ignore"):
        assert np.array_equal(masked_block_cols_product(Pr, M, R, True), want, equal_nan=True)
