"""Parity of the HIP path (through the C ABI) with the CPU oracle.

Bar: detection events (op, b, h, row, col, kind, action) identical as
multisets; outputs and saved tensors within |gpu - oracle| <= rtol *
max(|oracle|, rms(oracle)) with rtol = 1e-2 for bf16 storage and 1e-4 for
fp32 storage (the tolerance the target states for corrected outputs).
"""
import numpy as np
import pytest
import torch

import workloads as W
from oracle import OracleParams, forward, backward
from oracle.eec import col_checksums, row_checksums, Verifier
from oracle.numerics import stored_threshold

pytestmark = pytest.mark.gpu

RTOL = {"bf16": 1e-2, "f32": 1e-4}


def _abft():
    from paper_2410_11720_amd import abft
    return abft


def dev(a, tdt):
    return torch.from_numpy(np.ascontiguousarray(a, dtype=np.float32)).to("cuda").to(tdt)


def host(t):
    return t.float().cpu().numpy().astype(np.float64)


def assert_close(gpu, ref, rtol, name, mask=None):
    gpu, ref = np.asarray(gpu, dtype=np.float64), np.asarray(ref, dtype=np.float64)
    assert gpu.shape == ref.shape, name
    if mask is not None:
        gpu, ref = gpu[mask], ref[mask]
    nf = ~np.isfinite(ref)
    if nf.any():  # faults the configuration leaves in place must match exactly
        assert np.array_equal(gpu[nf], ref[nf], equal_nan=True), f"{name}: non-finite mismatch"
        gpu, ref = gpu[~nf], ref[~nf]
    assert np.isfinite(gpu).all(), f"{name}: {np.count_nonzero(~np.isfinite(gpu))} non-finite"
    scale = np.maximum(np.abs(ref), np.sqrt(np.mean(ref ** 2)) + 1e-300)
    rel = np.abs(gpu - ref) / scale
    assert rel.max() <= rtol, f"{name}: max rel err {rel.max():.3g} ({np.count_nonzero(rel > rtol)} > {rtol})"


def run_pair(shape, faults=(), *, root_check=True, sections=15, do_bwd=True, seed=None,
             check=True):
    """Run the GPU layer and the oracle on the same seeded inputs."""
    abft = _abft()
    seed = 1 if seed is None else seed
    print(f"[case] {shape.name} causal={shape.causal} R={shape.block_rows} "
          f"faults={len(faults)} root={root_check} sections={sections}", flush=True)
    inp = W.make_inputs(shape, seed)
    cfg = abft.LayerConfig(shape.batch, shape.seq, shape.hidden, shape.heads, dtype=shape.dtype,
                           causal=shape.causal, block_rows=shape.block_rows,
                           sections=sections, root_check=root_check)
    tdt = cfg.torch_dtype
    X, Wqkv, Wo, dO = (dev(inp[k], tdt) for k in ("X", "Wqkv", "Wo", "dO"))
    layer = abft.ProtectedAttention(cfg)
    # a NaN sentinel in the probability buffer: positions the forward does
    # not write keep it, and any read of them would spread it
    layer.tensor("AP").fill_(float("nan"))
    fdev = abft.faults_to_device(faults)
    O = layer.forward(X, Wqkv, Wo, fdev)
    torch.cuda.synchronize()
    g = dict(O=host(O), rep_f=abft.read_report(layer.report))
    QKV, AP, CL = layer.saved()
    g.update(QKV=host(QKV), AP=host(AP), CL=host(CL))
    if do_bwd:
        dX, dWqkv, dWo = layer.backward(dO, X, Wqkv, Wo, fdev)
        torch.cuda.synchronize()
        g.update(dX=host(dX), dWqkv=host(dWqkv), dWo=host(dWo),
                 rep_b=abft.read_report(layer.report_bwd))
    secs = tuple(n for n, bit in (("AS", 1), ("CL", 2), ("O", 4), ("BWD", 8)) if sections & bit)
    p = OracleParams(heads=shape.heads, causal=shape.causal, dtype=shape.dtype,
                     block_rows=shape.block_rows, root_check=root_check, sections=secs)
    o = forward(inp["X"], inp["Wqkv"], inp["Wo"], p, faults)
    ob = backward(o, inp["dO"], p, faults) if do_bwd else None
    if check:
        compare(shape, g, o, ob)
    return g, o, ob


def ap_tolerance(shape, o):
    """AP's bar. Both sides round AS to bf16 from fp32 (GPU) and fp64
    (oracle) accumulations; where the exact score lies next to a rounding
    boundary they keep adjacent values, at most one bf16 step (2^-7
    relative) apart, and exp turns that into a relative change of AP of up
    to scale * 2^-7 |AS|; AP's own rounding adds up to 2^-8 on each side.
    The bar is rtol + scale * max|AS| * 2^-7 over the allowed pairs
    (fp32 storage: rtol)."""
    rtol = RTOL[shape.dtype]
    if shape.dtype != "bf16":
        return rtol
    S = shape.seq
    tri = np.tril(np.ones((S, S), dtype=bool)) if shape.causal else np.ones((S, S), dtype=bool)
    as_max = float(np.max(np.abs(o["AS"][..., tri])))
    return rtol + o["scale"] * as_max * 2.0 ** -7


def compare(shape, g, o, ob, events=True):
    rtol = RTOL[shape.dtype]
    if events:
        assert g["rep_f"]["overflow"] == 0
        assert sorted(g["rep_f"]["events"]) == sorted(o["events"]), "forward events"
    S = shape.seq
    tri = np.tril(np.ones((S, S), dtype=bool)) if shape.causal else np.ones((S, S), dtype=bool)
    assert_close(g["O"], o["O"], rtol, "O")
    assert_close(g["QKV"], o["QKV"], rtol, "QKV")
    assert_close(g["CL"], o["CL"], rtol, "CL")
    assert_close(g["AP"], o["AP"], ap_tolerance(shape, o), "AP",
                 mask=np.broadcast_to(tri, g["AP"].shape))
    if shape.causal:
        # masked probabilities: exact zeros where written, the sentinel elsewhere
        up = g["AP"][np.broadcast_to(~tri, g["AP"].shape)]
        assert np.all((up == 0.0) | np.isnan(up))
    if ob is not None:
        if events:
            assert g["rep_b"]["overflow"] == 0
            assert sorted(g["rep_b"]["events"]) == sorted(ob["events"]), "backward events"
        assert_close(g["dX"], ob["dX"], rtol, "dX")
        assert_close(g["dWqkv"], ob["dWqkv"], rtol, "dWqkv")
        assert_close(g["dWo"], ob["dWo"], rtol, "dWo")


# ---- fp32 single-head config (fwd only in the workload; bwd checked too) ----

def test_c1_fp32_fault_free():
    g, o, ob = run_pair(W.C1, seed=W.data_seed("c1"))
    assert g["rep_f"]["events"] == [] and g["rep_b"]["events"] == []


def test_c1_fp32_config_faults():
    rng = np.random.default_rng(W.fault_seed("c1", 0))
    S, d = W.C1.seq, W.C1.head_dim
    faults = [W.Fault("Q", 0, 0, int(rng.integers(S)), int(rng.integers(d)), np.inf),
              W.Fault("AS", 0, 0, int(rng.integers(S)), int(rng.integers(S)), np.nan),
              W.Fault("CL", 0, 0, int(rng.integers(S)), int(rng.integers(d)), 1e10)]
    g, o, ob = run_pair(W.C1, faults, seed=W.data_seed("c1"))
    got = sorted(e[:5] for e in g["rep_f"]["events"])
    assert got == sorted(f.as_tuple()[:5] for f in faults)


# ---- bf16 shapes spanning several tiles and ragged tile edges ----

SHAPES = [
    W.make_shape(2, 256, 128, 2, causal=False),
    W.make_shape(2, 256, 128, 2, causal=True),
    W.make_shape(3, 128, 256, 2, causal=True),               # d = 128, T = 384 (ragged 256-row tiles)
    W.make_shape(1, 384, 256, 4, causal=True, block_rows=64),  # R = 64, seq not a power of two
    W.make_shape(2, 192, 128, 2, causal=True, block_rows=64),  # seq 192: ragged score tiles
    W.make_shape(1, 256, 64, 1, causal=False, block_rows=32),
    W.make_shape(1, 320, 64, 1, causal=True, block_rows=32),   # R = 32 causal, seq 320: blocks past it
    W.make_shape(4, 512, 128, 2, causal=True),                 # long K: split-K weight gradients
]


@pytest.mark.parametrize("shape", SHAPES, ids=lambda s: f"{s.name}-c{int(s.causal)}-R{s.block_rows}")
def test_bf16_fault_free(shape):
    g, o, ob = run_pair(shape)
    assert g["rep_f"]["events"] == [] and g["rep_b"]["events"] == []


KINDS = ["inf", "-inf", "nan", "+1e10", "-1e10", "1e30", "1e6"]


@pytest.mark.parametrize("causal", [False, True])
@pytest.mark.parametrize("kind", KINDS)
def test_bf16_every_op_every_kind(causal, kind):
    """One fault of the given kind in every one of the 16 protected
    outputs in the same step: every (op, kind) pair is detected, located at
    its position, classified and corrected, as by the oracle."""
    shape = W.make_shape(2, 256, 128, 2, causal=causal)
    seed = 900 + 50 * int(causal) + 7 * KINDS.index(kind)
    faults = [W.draw_faults(shape, seed + i, 1, [op], [kind])[0] for i, op in enumerate(W.ALL_OPS)]
    g, o, ob = run_pair(shape, faults)
    got = sorted(e[:5] for e in g["rep_f"]["events"] + g["rep_b"]["events"])
    assert got == sorted(f.as_tuple()[:5] for f in faults)


def test_bf16_multi_fault_step():
    shape = W.make_shape(2, 256, 128, 2, causal=True)
    faults = W.draw_faults(shape, 4242, 16, W.ALL_OPS, ["inf", "nan", "1e6", "1e10", "1e30"])
    g, o, ob = run_pair(shape, faults)
    got = sorted(e[:5] for e in g["rep_f"]["events"] + g["rep_b"]["events"])
    assert got == sorted(f.as_tuple()[:5] for f in faults)


def test_bf16_split_k_weight_gradients_with_faults():
    shape = W.make_shape(4, 512, 128, 2, causal=True)
    faults = W.draw_faults(shape, 321, 4, ["dWQ", "dWK", "dWV", "dWO"], ["inf", "nan", "1e10", "1e6"])
    g, o, ob = run_pair(shape, faults)
    got = sorted(e[:5] for e in g["rep_b"]["events"])
    assert got == sorted(f.as_tuple()[:5] for f in faults)


def test_bf16_row_pass_and_uncorrectable_block():
    shape = W.make_shape(1, 128, 64, 1)
    faults = [W.Fault("AS", 0, 0, 10, 7, np.inf), W.Fault("AS", 0, 0, 90, 7, np.nan)]
    run_pair(shape, faults, do_bwd=False)
    faults = [W.Fault("AS", 0, 0, r, c, np.inf) for r in (3, 50) for c in (4, 60)]
    g, o, ob = run_pair(shape, faults, do_bwd=False, check=False)
    assert sorted(g["rep_f"]["events"]) == sorted(o["events"])
    assert {e[6] for e in g["rep_f"]["events"]} == {"UNCORRECTABLE"}


def masked_zero_meets(shape, fault):
    """Outputs where a causally masked zero of a masked product meets the
    faulty element: a fault in row j0 of V (column c) meets the masked
    zeros AP[i, j0] of every query i < j0 in CL[i, c]. A tiled product may
    form such terms (0 * INF = NaN) that the masked product of Eq. 1 leaves
    out; nothing else may differ."""
    if not shape.causal or fault.op != "V":
        return set()
    return {("CL", fault.b, fault.h, i, fault.col) for i in range(fault.row)}


@pytest.mark.parametrize("op", ["Q", "K", "V"])
def test_paper_literal_mode_1d_patterns(op):
    """Root check off: a Q/K/V error reaches AS or CL as a 1-D pattern and
    is corrected there from checksums (Sec. 4.3). The GPU reports every
    event the oracle does; extra events are allowed only at outputs where
    a masked zero met the faulty element, and there the value rebuilt from
    the row checksum is within the reconstruction bound of the fault-free
    value."""
    from collections import Counter
    shape = W.make_shape(2, 256, 128, 2, causal=True)
    fault = W.Fault(op, 1, 1, 200, 9, np.inf)
    g, o, ob = run_pair(shape, [fault], root_check=False, do_bwd=False, check=False)
    assert g["rep_f"]["overflow"] == 0
    gev, oev = Counter(g["rep_f"]["events"]), Counter(o["events"])
    assert not (oev - gev), "an oracle event is missing on the GPU"
    assert len(o["events"]) > 1
    extra = list((gev - oev).elements())
    allowed = masked_zero_meets(shape, fault)
    assert all(e[:5] in allowed and e[5] == "NAN" and e[6] == "RECONSTRUCT" for e in extra), extra
    if op == "V":
        assert extra, "a tiled context product meets masked zeros"
    d = shape.head_dim
    CLg = g["CL"].copy()
    for (_, b, h, i, c, _, _) in extra:
        # c1 - sum of the other stored elements: each carries at most one
        # bf16 rounding (2^-8 relative) of the exact value, the rebuilt
        # element one more
        row = o["CL"][b, i, h * d:(h + 1) * d]
        bound = 2.0 ** -8 * (np.abs(row).sum() + abs(row[c])) + 1e-6
        assert abs(CLg[b, i, h * d + c] - row[c]) <= bound
        CLg[b, i, h * d + c] = row[c]
    compare(shape, dict(g, CL=CLg), o, None, events=False)


def bf16_step(v):
    """Spacing of bf16 values at |v| (one unit in the last place)."""
    v = np.maximum(np.abs(np.asarray(v, dtype=np.float64)), 2.0 ** -126)
    return 2.0 ** (np.floor(np.log2(v)) - 7)


@pytest.mark.parametrize("causal", [False, True])
def test_softmax_stage_within_one_bf16_step(causal):
    """The softmax alone, on identical scores: the oracle's stored AS is
    written into the GPU's score buffer and only the softmax stage runs.
    AP is within one bf16 step of the oracle's softmax of the same AS;
    AP^c and AP^r are fp32 sums of the stored AP, and within the sums of
    one-step differences of the oracle's checksums."""
    abft = _abft()
    shape = W.make_shape(2, 1024, 128, 2, causal=causal)
    inp = W.make_inputs(shape, 31)
    cfg = abft.LayerConfig(shape.batch, shape.seq, shape.hidden, shape.heads, causal=causal)
    X, Wqkv, Wo = (dev(inp[k], torch.bfloat16) for k in ("X", "Wqkv", "Wo"))
    layer = abft.ProtectedAttention(cfg)
    print(f"[case] softmax stage causal={causal}", flush=True)
    O = layer.forward(X, Wqkv, Wo)
    p = OracleParams(heads=2, causal=causal)
    o = forward(inp["X"], inp["Wqkv"], inp["Wo"], p)
    layer.tensor("AS").copy_(dev(o["AS"], torch.bfloat16))
    layer.tensor("AP").fill_(float("nan"))
    abft.attn_abft_forward_stages(cfg, X, Wqkv, Wo, O, layer.workspace, None, 0, layer.report,
                                  abft.FWD_STAGES["softmax"])
    torch.cuda.synchronize()
    AP, APc, APr = (host(layer.tensor(k)) for k in ("AP", "APc", "APr"))
    S, R = shape.seq, shape.block_rows
    nq = S // R
    tri = np.tril(np.ones((S, S), dtype=bool)) if causal else np.ones((S, S), dtype=bool)
    allowed = np.broadcast_to(tri, AP.shape)
    diff = np.abs(AP - o["AP"])[allowed]
    assert np.isfinite(AP[allowed]).all()
    assert np.all(diff <= bf16_step(o["AP"][allowed])), diff.max()
    # the column checksum of query block qb covers keys up to its last query,
    # the row checksum of query i the key blocks up to its own
    colv = (np.arange(S)[None, :] < (np.arange(nq)[:, None] + 1) * R) if causal else \
        np.ones((nq, S), dtype=bool)
    rowv = (np.arange(nq)[None, :] <= (np.arange(S)[:, None] // R)) if causal else \
        np.ones((S, nq), dtype=bool)
    APz = np.where(allowed, AP, 0.0)
    steps = np.where(allowed, bf16_step(o["AP"]), 0.0)
    w = np.arange(1, R + 1, dtype=np.float64)
    for name, got, own, ref, slack, valid in (
            ("APc", APc, col_checksums(APz, R), o["APc"], col_checksums(steps, R), colv[:, None, :]),
            ("APr", APr, row_checksums(APz, R), o["APr"], row_checksums(steps, R), rowv[:, :, None])):
        v = np.broadcast_to(valid, got.shape)
        # fp32 sums of at most R stored values (weights up to R)
        assert np.all(np.abs(got - own)[v] <= 2.0 ** -20 * R * np.abs(own)[v] + 1e-30), name
        assert np.all(np.abs(got - ref)[v] <= slack[v] + 2.0 ** -20 * R * np.abs(ref)[v]), name


def test_disabled_section_matches_oracle():
    shape = W.make_shape(1, 128, 64, 1)
    faults = [W.Fault("AS", 0, 0, 9, 3, np.inf)]
    g, o, ob = run_pair(shape, faults, sections=2 | 4 | 8, do_bwd=False, check=False)
    assert sorted(g["rep_f"]["events"]) == sorted(o["events"])
    assert np.isnan(g["O"][0, 9]).all()


def test_unprotected_matches_fault_free_outputs():
    abft = _abft()
    shape = W.make_shape(2, 256, 128, 2, causal=True)
    g, o, ob = run_pair(shape)
    inp = W.make_inputs(shape, 1)
    cfg = abft.LayerConfig(shape.batch, shape.seq, shape.hidden, shape.heads, causal=True,
                           protect=False)
    X, Wqkv, Wo, dO = (dev(inp[k], torch.bfloat16) for k in ("X", "Wqkv", "Wo", "dO"))
    layer = abft.ProtectedAttention(cfg)
    O = layer.forward(X, Wqkv, Wo)
    dX, dWqkv, dWo = layer.backward(dO, X, Wqkv, Wo)
    torch.cuda.synchronize()
    assert np.array_equal(host(O), g["O"]) and np.array_equal(host(dX), g["dX"])
    assert np.array_equal(host(dWqkv), g["dWqkv"])


@pytest.mark.gpu
def test_scheduled_section_masks_change_no_output_bit():
    """Steps run with the per-step masks of the adaptive frequencies
    (attn_abft_sections_for_step) give bit-identical outputs to full
    protection on a fault-free layer, and a masked-off section lets its
    fault through while a checked one corrects it."""
    abft = _abft()
    shape = W.make_shape(2, 256, 128, 2, causal=True)
    g, o, ob = run_pair(shape)
    inp = W.make_inputs(shape, 1)
    X, Wqkv, Wo, dO = (dev(inp[k], torch.bfloat16) for k in ("X", "Wqkv", "Wo", "dO"))
    cfg = abft.LayerConfig(shape.batch, shape.seq, shape.hidden, shape.heads, causal=True)
    layer = abft.ProtectedAttention(cfg)
    freqs = [0.5, 0.25, 1 / 3, 0.75]
    for step in range(6):
        mask = abft.attn_abft_sections_for_step(freqs, step)
        print(f"[case] step {step} sections {mask}", flush=True)
        layer.cfg.sections = mask
        O = layer.forward(X, Wqkv, Wo)
        dX, dWqkv, dWo = layer.backward(dO, X, Wqkv, Wo)
        torch.cuda.synchronize()
        assert np.array_equal(host(O), g["O"]) and np.array_equal(host(dX), g["dX"])
        assert np.array_equal(host(dWqkv), g["dWqkv"]) and np.array_equal(host(dWo), g["dWo"])
    fault = abft.faults_to_device([W.Fault("AS", 1, 0, 40, 7, np.inf)])
    for mask, caught in ((abft.SEC_CL | abft.SEC_O | abft.SEC_BWD, False), (abft.SEC_ALL, True)):
        layer.cfg.sections = mask
        O = layer.forward(X, Wqkv, Wo, fault)
        torch.cuda.synchronize()
        rep = abft.read_report(layer.report)
        assert (rep["n_corrected"] == 1) == caught
        assert np.array_equal(host(O), g["O"]) == caught


# ---- standalone entry points ----

@pytest.mark.parametrize("dtype", ["bf16", "f32"])
def test_encode_checksums_matches_oracle(dtype):
    abft = _abft()
    rng = np.random.default_rng(3)
    batch, rows, cols, ld = 3, 256, 192, 200
    a = W.to_storage(rng.standard_normal((batch, rows, ld)).astype(np.float32), dtype)
    tdt = torch.float32 if dtype == "f32" else torch.bfloat16
    A = dev(a, tdt)
    cc = torch.empty((batch, rows // 64, 2, cols), dtype=torch.float32, device="cuda")
    rc = torch.empty((batch, rows, cols // 32, 2), dtype=torch.float32, device="cuda")
    print(f"[case] encode {dtype}", flush=True)
    abft.encode_checksums(A, abft.FP32 if dtype == "f32" else abft.BF16, batch, rows, cols, ld,
                          rows * ld, 64, 32, cc, rc)
    torch.cuda.synchronize()
    ref_c = col_checksums(a[..., :cols].astype(np.float64), 64)
    ref_r = row_checksums(a[..., :cols].astype(np.float64), 32)
    assert np.allclose(host(cc), ref_c, rtol=1e-5, atol=1e-3)
    assert np.allclose(host(rc), ref_r, rtol=1e-5, atol=1e-3)
    # block widths beyond one wave take the generic path
    rc2 = torch.empty((batch, rows, 1, 2), dtype=torch.float32, device="cuda")
    abft.encode_checksums(A, abft.FP32 if dtype == "f32" else abft.BF16, batch, rows, cols, ld,
                          rows * ld, 64, 192, None, rc2)
    torch.cuda.synchronize()
    assert np.allclose(host(rc2), row_checksums(a[..., :cols].astype(np.float64), 192),
                       rtol=1e-5, atol=1e-3)


@pytest.mark.gpu
@pytest.mark.parametrize("dtype", ["bf16", "f32"])
@pytest.mark.parametrize("ld,cb", [(264, 64), (264, 128), (257, 64)])
def test_encode_checksums_slabs_and_unaligned(dtype, ld, cb):
    """Wide row-checksum blocks (16-chunk slabs), and an unaligned leading
    dimension (scalar column path plus the per-row fallback)."""
    abft = _abft()
    rng = np.random.default_rng(ld + cb)
    batch, rows, cols = 2, 384, 256
    a = W.to_storage(rng.standard_normal((batch, rows, ld)).astype(np.float32), dtype)
    tdt = torch.float32 if dtype == "f32" else torch.bfloat16
    A = dev(a, tdt)
    cc = torch.empty((batch, rows // 128, 2, cols), dtype=torch.float32, device="cuda")
    rc = torch.empty((batch, rows, cols // cb, 2), dtype=torch.float32, device="cuda")
    print(f"[case] encode {dtype} ld={ld} cb={cb}", flush=True)
    abft.encode_checksums(A, abft.FP32 if dtype == "f32" else abft.BF16, batch, rows, cols, ld,
                          rows * ld, 128, cb, cc, rc)
    torch.cuda.synchronize()
    ref = a[..., :cols].astype(np.float64)
    assert np.allclose(host(cc), col_checksums(ref, 128), rtol=1e-5, atol=1e-3)
    assert np.allclose(host(rc), row_checksums(ref, cb), rtol=1e-5, atol=1e-3)


@pytest.mark.parametrize("two_sided", [False, True])
def test_verify_and_correct_matches_oracle(two_sided):
    abft = _abft()
    rng = np.random.default_rng(11)
    batch, rows, cols, Rb, Cb = 2, 256, 128, 128, 64
    M = W.to_storage(rng.standard_normal((batch, rows, cols)).astype(np.float32), "bf16")
    M = M.astype(np.float64)
    Cc = col_checksums(M, Rb)
    Cr = row_checksums(M, Cb)
    bad = M.copy()
    for (b, r, c, v) in [(0, 3, 5, np.inf), (0, 200, 77, np.nan), (1, 100, 1, 1e10),
                         (1, 10, 100, 3e3), (1, 130, 60, -1e6)]:
        bad[b, r, c] = float(W.to_storage(np.float32([v]), "bf16")[0]) if np.isfinite(v) else v
    C = dev(bad, torch.bfloat16)
    cc = dev(Cc, torch.float32)
    rc = dev(Cr, torch.float32) if two_sided else None
    rep = abft.new_report(256)
    print(f"[case] verify two_sided={two_sided}", flush=True)
    abft.verify_and_correct(C, abft.BF16, batch, rows, cols, cols, rows * cols, Rb, Cb, cc, rc,
                            1e10, 1e5, 0.0, abft.OP_ID["AS"], rep)
    torch.cuda.synchronize()
    got = abft.read_report(rep)
    ver = Verifier("bf16", 2.0 ** -4, stored_threshold(1e10, "bf16"), 1e5)
    ref = bad.copy()
    evs, unc = ver.run(ref, Cc.copy(), Rb, Cr=Cr.copy() if two_sided else None,
                       Cb=Cb if two_sided else None)
    assert unc == []
    want = sorted(("AS", k, 0, i, j, kind, act) for (k, i, j, kind, act) in evs)
    assert sorted(got["events"]) == want
    assert_close(host(C), ref, 1e-2, "corrected")


def test_determinism_bitwise():
    shape = W.make_shape(2, 256, 256, 4, causal=True)
    faults = W.draw_faults(shape, 99, 4, W.ALL_OPS, ["inf", "nan", "1e10"])
    g1, _, _ = run_pair(shape, faults, check=False)
    g2, _, _ = run_pair(shape, faults, check=False)
    for k in ("O", "dX", "dWqkv", "dWo", "QKV", "CL"):
        assert np.array_equal(g1[k], g2[k], equal_nan=True), k
    assert sorted(g1["rep_f"]["events"]) == sorted(g2["rep_f"]["events"])
    assert sorted(g1["rep_b"]["events"]) == sorted(g2["rep_b"]["events"])


# ---- full-size workloads ----

def test_c2_full_size_single_fault():
    faults = W.draw_faults(W.C2, W.fault_seed("c2", 0), 1,
                           ["Q", "K", "V", "AS", "CL", "O", "dX", "dWQ", "dWK", "dWV", "dWO"],
                           ["inf", "nan", "+1e10", "-1e10"])
    run_pair(W.C2, faults, seed=W.data_seed("c2"))


def test_c3_full_size_multi_fault():
    faults = W.draw_faults(W.C3, W.fault_seed("c3", 0), 4, W.ALL_OPS,
                           ["inf", "nan", "+1e10", "-1e10"])
    run_pair(W.C3, faults, seed=W.data_seed("c3"))
