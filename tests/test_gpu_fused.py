"""Parity of the fused attention forward (ABFT_FLAG_FUSED, through the C
ABI) with the fused-attention oracle and with the materialised layer
oracle on the same seeded inputs.

Bar: detection events identical to the fused oracle's as multisets; O and
CL within |gpu - oracle| <= 1e-2 * max(|oracle|, rms(oracle)) of both
oracles (bf16 storage; the fused forms round P to bf16, from exponentials
taken in fp32 here and fp64 there, relative to a running maximum that
depends on how the keys are grouped; the materialised form rounds AS and
AP instead). A context element fixed from its row checksum is within the
reconstruction bound of the fault-free value.
"""
import dataclasses

import numpy as np
import pytest
import torch

import workloads as W
from oracle import OracleParams, forward
from oracle.fused import fused_attention, fused_forward
from oracle.layer import _Run, project

pytestmark = pytest.mark.gpu
RTOL = 1e-2


def _abft():
    from paper_2410_11720_amd import abft
    return abft


def dev(a):
    return torch.from_numpy(np.ascontiguousarray(a, dtype=np.float32)).to("cuda").to(torch.bfloat16)


def host(t):
    return t.float().cpu().numpy().astype(np.float64)


def assert_close(gpu, ref, name):
    nf = ~np.isfinite(ref)
    assert not nf.any() and np.isfinite(gpu).all(), name
    scale = np.maximum(np.abs(ref), np.sqrt(np.mean(ref ** 2)) + 1e-300)
    rel = np.abs(gpu - ref) / scale
    assert rel.max() <= RTOL, f"{name}: max rel err {rel.max():.3g}"


def run_fused(shape, faults=(), root_check=True, seed=1):
    abft = _abft()
    print(f"[case] fused {shape.name} causal={shape.causal} R={shape.block_rows} "
          f"faults={len(faults)} root={root_check}", flush=True)
    inp = W.make_inputs(shape, seed)
    cfg = abft.LayerConfig(shape.batch, shape.seq, shape.hidden, shape.heads,
                           causal=shape.causal, block_rows=shape.block_rows,
                           root_check=root_check, fused=True)
    layer = abft.ProtectedAttention(cfg)
    X, Wqkv, Wo = (dev(inp[k]) for k in ("X", "Wqkv", "Wo"))
    O = layer.forward(X, Wqkv, Wo, abft.faults_to_device(list(faults)))
    torch.cuda.synchronize()
    g = dict(O=host(O), CL=host(layer.tensor("CL")), rep=abft.read_report(layer.report))
    p = OracleParams(heads=shape.heads, causal=shape.causal, block_rows=shape.block_rows,
                     root_check=root_check)
    o = fused_forward(inp["X"], inp["Wqkv"], inp["Wo"], p, list(faults))
    # the materialised layer, fault-free: what a corrected run must give
    o["mat"] = forward(inp["X"], inp["Wqkv"], inp["Wo"], p)
    return g, o


U = 2.0 ** -8   # bf16 unit roundoff


def rounding_bounds(m, shape, materialised):
    """Element bounds on |fused GPU - reference| for CL, O and dW^O, from
    where the forms round (computed from the materialised oracle m's AP,
    AS, V, CL, O, W^O, dO):
      fused vs fused (two groupings of the keys): each side rounds every
        unnormalised P once (relative u, against its own running maximum),
        then CL: |dCL_ic| <= 2u sum_j AP_ij |V_jc| + 2u |CL_ic|;
      fused vs materialised: the materialised form also stores AS (moving
        each probability by up to scale |AS_ij| u relative through exp,
        and the row's normaliser by at most the row's largest such move)
        and stores AP (u): 3u + 2 scale max_j |AS_ij| u in place of 2u.
    O = CL W^O adds the rounding of O on both sides: |dO| <= |dCL| |W^O| +
    2u |O|; dW^O = CL^T dO (fp32): |d dW^O| <= |dCL|^T |dO| (+ fp32)."""
    B, S, H, nh, d = shape.batch, shape.seq, shape.hidden, shape.heads, shape.head_dim
    tri = np.tril(np.ones((S, S), dtype=bool)) if shape.causal else np.ones((S, S), dtype=bool)
    bcl = np.zeros((B, S, H))
    for b in range(B):
        for h in range(nh):
            AP, AS = m["AP"][b, h], m["AS"][b, h]
            V = m["QKV"][b, :, 2 * H + h * d:2 * H + (h + 1) * d]
            if materialised:
                amax = np.where(tri, np.abs(AS), 0.0).max(axis=1, keepdims=True)
                k = 3 + 2 * m["scale"] * amax
            else:
                k = 2.0
            bcl[b, :, h * d:(h + 1) * d] = U * k * (AP @ np.abs(V))
    bcl += 2 * U * np.abs(m["CL"])
    bo = bcl @ np.abs(m["Wo"]) + 2 * U * np.abs(m["O"])
    return bcl, bo


def assert_within(got, ref, bound, name):
    assert np.isfinite(got).all(), name
    over = np.abs(got - ref) - bound
    assert over.max() <= 0.0, f"{name}: {np.count_nonzero(over > 0)} elements over the bound"


def fix_rebuilt(g, ref_cl, shape, rebuilt):
    """Elements fixed from a row checksum (rebuilt: (b, h, i, c)) against
    the reconstruction bound (each other element of the row carries at most
    one bf16 rounding, 2^-8 relative); returns CL with them set to ref."""
    d = shape.head_dim
    CL = g["CL"].copy()
    for (b, h, i, c) in rebuilt:
        row = ref_cl[b, i, h * d:(h + 1) * d]
        assert abs(CL[b, i, h * d + c] - row[c]) <= U * (np.abs(row).sum() + abs(row[c]))
        CL[b, i, h * d + c] = row[c]
    return CL


def check_outputs(g, o, shape, rebuilt=()):
    """CL and O against the fused oracle and against the fault-free
    materialised oracle, each within its rounding bounds."""
    m = o["mat"]
    for ref, materialised in ((o, False), (m, True)):
        bcl, bo = rounding_bounds(m, shape, materialised)
        CL = fix_rebuilt(g, ref["CL"], shape, rebuilt)
        tag = "materialised" if materialised else "fused oracle"
        assert_within(CL, ref["CL"], bcl, f"CL vs {tag}")
        assert_within(g["O"], ref["O"], bo, f"O vs {tag}")


SHAPES = [W.make_shape(1, 256, 128, 2, causal=c, block_rows=r, name=f"d64c{int(c)}r{r}")
          for c in (False, True) for r in (128, 32)] + \
         [W.make_shape(1, 256, 256, 2, causal=c, block_rows=64, name=f"d128c{int(c)}")
          for c in (False, True)]


@pytest.mark.parametrize("shape", SHAPES, ids=lambda s: s.name)
def test_fused_fault_free(shape):
    g, o = run_fused(shape)
    assert g["rep"]["events"] == [] and o["events"] == []
    check_outputs(g, o, shape)


@pytest.mark.parametrize("causal", [False, True])
def test_fused_score_faults(causal):
    shape = W.make_shape(2, 256, 128, 2, causal=causal, block_rows=64, name="faults")
    faults = [W.Fault("AS", 0, 0, 5, 3, np.inf), W.Fault("AS", 0, 1, 130, 129, np.nan),
              W.Fault("AS", 1, 0, 200, 70, 3e10), W.Fault("AS", 1, 1, 255, 250, 55.0),
              W.Fault("AS", 0, 1, 77, 12, 0.0, mode="flip"),
              # past the diagonal of a diagonal tile (masked under the causal mask)
              W.Fault("AS", 1, 0, 140, 180, np.inf)]
    g, o = run_fused(shape, faults)
    assert g["rep"]["overflow"] == 0
    assert sorted(g["rep"]["events"]) == sorted(o["events"])
    assert len(o["events"]) == 6
    check_outputs(g, o, shape)


def test_fused_context_faults():
    shape = W.make_shape(1, 256, 128, 2, causal=True, block_rows=128, name="clfaults")
    faults = [W.Fault("CL", 0, 0, 99, 17, np.inf), W.Fault("CL", 0, 1, 3, 63, np.nan),
              W.Fault("CL", 0, 0, 250, 0, 1e12), W.Fault("CL", 0, 1, 128, 40, 40.0),
              W.Fault("CL", 0, 0, 17, 5, 0.0, mode="flip")]
    g, o = run_fused(shape, faults)
    assert sorted(g["rep"]["events"]) == sorted(o["events"])
    assert len(o["events"]) == 5
    check_outputs(g, o, shape, [(f.b, f.h, f.row, f.col) for f in faults])


def test_fused_key_fault_without_root_check():
    """Root check off: the fused form still verifies K at the projection
    (its backward's key pass checks score columns, which cannot see a K
    error); the near-INF element is fixed there from K's checksums and the
    scores see nothing."""
    shape = W.make_shape(1, 256, 128, 2, causal=False, block_rows=128, name="kfault")
    faults = [W.Fault("K", 0, 0, 77, 5, 1e10)]
    g, o = run_fused(shape, faults, root_check=False)
    assert sorted(g["rep"]["events"]) == sorted(o["events"])
    assert [(e[0], e[3], e[4], e[6]) for e in o["events"]] == [("K", 77, 5, "RECONSTRUCT")]
    check_outputs(g, o, shape)


def test_fused_query_fault_without_root_check():
    """Root check off: the fused score check has rows only, which cannot
    see a Q error (a score row moves with its checksums), so the fused form
    verifies Q at the projection in every mode; without the root check the
    element is fixed from Q's checksums, and CL and O stay within their
    rounding bounds of the fused oracle and of the fault-free materialised
    run."""
    shape = W.make_shape(1, 256, 128, 2, causal=True, block_rows=128, name="qfault")
    faults = [W.Fault("Q", 0, 1, 200, 3, 1e8)]
    g, o = run_fused(shape, faults, root_check=False)
    want = [("Q", 0, 1, 200, 3, "RECONSTRUCT")]
    assert [(e[0], e[1], e[2], e[3], e[4], e[6]) for e in o["events"]] == want
    assert [(e[0], e[1], e[2], e[3], e[4], e[6]) for e in g["rep"]["events"]] == want
    check_outputs(g, o, shape)


def test_fused_gpt2_shape_sampled_heads():
    """The benchmark shape (B8 S1024 H768, 12 heads of 64, causal, R 128):
    no events on the GPU, and two sampled heads equal the oracle's."""
    abft = _abft()
    shape = W.CONFIGS["c3"]
    inp = W.make_inputs(shape, W.data_seed("c3"))
    cfg = abft.LayerConfig(shape.batch, shape.seq, shape.hidden, shape.heads, causal=True,
                           block_rows=shape.block_rows, fused=True)
    layer = abft.ProtectedAttention(cfg)
    print("[case] fused c3", flush=True)
    X, Wqkv, Wo = (dev(inp[k]) for k in ("X", "Wqkv", "Wo"))
    layer.forward(X, Wqkv, Wo)
    torch.cuda.synchronize()
    rep = abft.read_report(layer.report)
    assert rep["events"] == [] and rep["n_uncorrectable"] == 0
    CL = host(layer.tensor("CL"))
    p = OracleParams(heads=shape.heads, causal=True, block_rows=shape.block_rows)
    run = _Run(p, ())
    pr = project(run, inp["X"], inp["Wqkv"], p)
    only = {(0, 0), (7, 11), (3, 5), (5, 2), (1, 9), (6, 7), (2, 1), (4, 10)}
    CLo, _ = fused_attention(run, pr, p, only=only)
    d = shape.hidden // shape.heads
    from oracle.heads import head_reference
    S = shape.seq
    tri = np.tril(np.ones((S, S), dtype=bool))
    for (b, h) in sorted(only):
        ref = head_reference(inp["X"], inp["Wqkv"], inp["Wo"], None, p, h, [b], backward=False)
        AP, AS, V, CLm = ref["AP"][0], ref["AS"][0], ref["V"][0], ref["CL"][0]
        spread = AP @ np.abs(V)
        got = CL[b, :, h * d:(h + 1) * d]
        # the bounds of rounding_bounds, per head
        assert_within(got, CLo[b, :, h * d:(h + 1) * d], 2 * U * spread + 2 * U * np.abs(CLm),
                      f"CL[{b},{h}] vs fused oracle")
        amax = np.where(tri, np.abs(AS), 0.0).max(axis=1, keepdims=True)
        k = 3 + 2 * pr["scale"] * amax
        assert_within(got, CLm, U * k * spread + 2 * U * np.abs(CLm), f"CL[{b},{h}] vs materialised")
    assert run.events == []


def test_fused_rejects_unsupported_shapes():
    abft = _abft()
    with pytest.raises(abft.AbftError):
        abft.ProtectedAttention(abft.LayerConfig(1, 192, 128, 2, block_rows=64, fused=True))
    with pytest.raises(abft.AbftError):
        abft.ProtectedAttention(abft.LayerConfig(1, 256, 128, 2, dtype="f32", fused=True))


def run_fused_training(shape, faults=(), seed=1):
    """Fused forward, then the backward with the fused core (scores
    recomputed from the softmax statistics), against the fused oracle's
    forward and backward."""
    abft = _abft()
    print(f"[case] fused fwd+bwd {shape.name} causal={shape.causal} R={shape.block_rows} "
          f"faults={len(faults)}", flush=True)
    inp = W.make_inputs(shape, seed)
    cfg = abft.LayerConfig(shape.batch, shape.seq, shape.hidden, shape.heads,
                           causal=shape.causal, block_rows=shape.block_rows, fused=True)
    layer = abft.ProtectedAttention(cfg)
    X, Wqkv, Wo, dO = (dev(inp[k]) for k in ("X", "Wqkv", "Wo", "dO"))
    fdev = abft.faults_to_device(list(faults))
    O = layer.forward(X, Wqkv, Wo, fdev)
    dX, dWqkv, dWo = layer.backward(dO, X, Wqkv, Wo, fdev)
    torch.cuda.synchronize()
    g = dict(O=host(O), dQKV=host(layer.tensor("dQKV")), dX=host(dX), dWqkv=host(dWqkv),
             dWo=host(dWo), rep_f=abft.read_report(layer.report),
             rep_b=abft.read_report(layer.report_bwd))
    from oracle import backward
    from oracle.fused import fused_training_backward
    p = OracleParams(heads=shape.heads, causal=shape.causal, block_rows=shape.block_rows)
    o = fused_forward(inp["X"], inp["Wqkv"], inp["Wo"], p, list(faults))
    ob = fused_training_backward(o, inp["dO"], p, list(faults))
    # the materialised layer, fault-free
    m = forward(inp["X"], inp["Wqkv"], inp["Wo"], p)
    o["mat"], o["mat_bwd"], o["dO"] = m, backward(m, inp["dO"], p), inp["dO"]
    return g, o, ob


@pytest.mark.parametrize("causal", [False, True])
@pytest.mark.parametrize("R,H", [(128, 128), (64, 128), (128, 256)], ids=["d64r128", "d64r64", "d128"])
def test_fused_forward_backward(causal, R, H):
    shape = W.make_shape(2, 256, H, 2, causal=causal, block_rows=R, name="train")
    g, o, ob = run_fused_training(shape)
    assert g["rep_f"]["events"] == [] and g["rep_b"]["events"] == []
    assert o["events"] == [] and ob["events"] == []
    check_training_outputs(g, o, ob, shape)


def test_fused_workspace_holds_no_scores():
    """The fused form keeps no score-shaped tensor: its workspace is
    smaller than the materialised one by more than the four S x S tensors'
    worth and the score tensors are not addressable."""
    abft = _abft()
    kw = dict(causal=True, block_rows=128)
    fz = abft.LayerConfig(2, 512, 256, 4, fused=True, **kw)
    mat = abft.LayerConfig(2, 512, 256, 4, **kw)
    ss = 2 * 4 * 512 * 512 * 2
    assert abft.attn_abft_workspace_bytes(fz) + 3 * ss < abft.attn_abft_workspace_bytes(mat)
    layer = abft.ProtectedAttention(fz)
    for name in ("AS", "AP", "APc", "APr", "dAS"):
        with pytest.raises(abft.AbftError):
            layer.tensor(name)


def check_training_outputs(g, o, ob, shape):
    """dX and dW^QKV take AP recomputed from the softmax statistics, which
    do not depend on how the keys were grouped: within 1e-2 of the fused
    oracle's backward. O and dW^O take CL: within the rounding bounds of
    the fused oracle's. Against the materialised layer (no fused step on
    the CPU side) the two forms round at different points (AS and AP
    stored, or P rounded unnormalised; dP stored or not): O within its
    bound, the gradients within 1e-2 in relative norm."""
    m = o["mat"]
    bcl, bo = rounding_bounds(m, shape, False)
    dO = o["dO"].reshape(-1, shape.hidden).astype(np.float64)
    bwo = bcl.reshape(-1, shape.hidden).T @ np.abs(dO)
    assert_close(g["dX"], ob["dX"], "dX")
    assert_close(g["dWqkv"], ob["dWqkv"], "dWqkv")
    assert_within(g["O"], o["O"], bo, "O vs fused oracle")
    assert_within(g["dWo"], ob["dWo"], bwo + 2.0 ** -20 * np.abs(ob["dWo"]), "dWo vs fused oracle")
    _, bo_m = rounding_bounds(m, shape, True)
    assert_within(g["O"], m["O"], bo_m, "O vs materialised")
    for k in ("dX", "dWqkv", "dWo"):
        ref = o["mat_bwd"][k]
        nrel = np.linalg.norm(g[k] - ref) / np.linalg.norm(ref)
        assert nrel <= RTOL, f"{k} vs materialised: relative norm {nrel:.3g}"


@pytest.mark.parametrize("R,H", [(128, 128), (64, 128), (128, 256)], ids=["d64r128", "d64r64", "d128"])
def test_fused_backward_faults(R, H):
    """Faults in the scores (the forward's and both backward passes'
    recomputations see them), dP, dV, dK, dQ and dX: each located where
    injected and corrected, events identical to the fused oracle's (at
    head dim 128 the key pass runs in two parts; the event count is the
    same)."""
    shape = W.make_shape(1, 256, H, 2, causal=True, block_rows=R, name="trainf")
    faults = [W.Fault("AS", 0, 1, 200, 3, np.inf), W.Fault("dV", 0, 0, 17, 9, np.nan),
              W.Fault("dQ", 0, 1, 130, 60, 1e10), W.Fault("dX", 0, 0, 77, 100, np.inf),
              W.Fault("dAP", 0, 0, 250, 249, -1e10), W.Fault("dQ", 0, 0, 31, 5, 40.0),
              W.Fault("dAP", 0, 1, 100, 7, 0.0, mode="flip"), W.Fault("dK", 0, 1, 66, 40, -np.inf),
              W.Fault("dK", 0, 0, 255, 0, 30.0)]
    g, o, ob = run_fused_training(shape, faults)
    assert g["rep_f"]["overflow"] == 0 and g["rep_b"]["overflow"] == 0
    assert sorted(g["rep_f"]["events"]) == sorted(o["events"])
    assert sorted(g["rep_b"]["events"]) == sorted(ob["events"])
    # score and dP faults reach both passes of the fused backward
    twice = sum(f.op in ("AS", "dAP") for f in faults)
    assert len(o["events"]) == 1 and len(ob["events"]) == len(faults) + twice
    check_training_outputs(g, o, ob, shape)


def sampled_core(inp, shape, p, only, faults=()):
    """The fused oracle on the sampled (batch, head) pairs only: the
    projection of the whole layer, the fused attention of the pairs (CL and
    the softmax statistics), dCL = dO W^O^T, then the fused backward core
    on a one-head context per pair (faults of the score and gradient ops
    of a pair moved to its (0, 0)). Returns per pair dQ, dK, dV and the
    core's events, and the forward's events."""
    from oracle.eec import col_checksums
    from oracle.fused import fused_backward_core
    run = _Run(p, list(faults))
    pr = project(run, inp["X"], inp["Wqkv"], p, verify_always=True)
    st = {}
    CL, _ = fused_attention(run, pr, p, only=set(only), stats=st)
    B, S, H, nh, d, R, nq = (pr[k] for k in ("B", "S", "H", "nh", "d", "R", "nq"))
    dO = np.asarray(inp["dO"], dtype=np.float64)
    Wo = np.asarray(inp["Wo"], dtype=np.float64)
    dCL = run.rnd(dO @ Wo.T)
    dCLc = col_checksums(dO, R) @ Wo.T

    def heads_of(M):
        return M.reshape(B, S, nh, d).transpose(0, 2, 1, 3)

    def heads_of_c(Mc):
        return Mc.reshape(B, nq, 2, nh, d).transpose(0, 3, 1, 2, 4)

    Vch = heads_of_c(pr["QKVc"][..., 2 * H:])
    out = {}
    for (b, h) in only:
        sl = (slice(b, b + 1), slice(h, h + 1))
        ctx = dict(B=1, S=S, H=d, nh=1, d=d, R=R, nq=nq, scale=pr["scale"],
                   Qh=pr["Qh"][sl], Kh=pr["Kh"][sl], Vh=pr["Vh"][sl], dCLh=heads_of(dCL)[sl],
                   CLh=heads_of(CL)[sl], Qch=pr["Qch"][sl], Kch=pr["Kch"][sl], Vch=Vch[sl],
                   dCLch=heads_of_c(dCLc)[sl], m=st["m"][sl], l=st["l"][sl])
        mine = [dataclasses.replace(f, b=0, h=0) for f in faults
                if (f.b, f.h) == (b, h) and f.op in ("AS", "dAP", "dQ", "dK", "dV")]
        crun = _Run(p, mine)
        c = fused_backward_core(crun, ctx, p)
        out[(b, h)] = dict(dQ=c["dQ"][0, 0], dK=c["dK"][0, 0], dV=c["dV"][0, 0],
                           events=[(e[0], b, h) + tuple(e[3:]) for e in crun.events])
    return out, run.events


@pytest.mark.parametrize("with_faults", [False, True])
def test_fused_gpt2_training_sampled_heads(with_faults):
    """The benchmark's workload and launch configuration (B8 S1024 H768,
    12 heads of 64, causal, R 128, the fused forward and backward): the
    gradients dQ, dK, dV of sampled heads against the fused oracle's core
    for those heads, within 1e-2 in relative norm (reading 18: cascaded
    roundings), and, with faults in the sampled heads' scores, dP and
    gradients, events identical to the oracle's (a score or dP fault in the
    forward and both backward passes)."""
    abft = _abft()
    shape = W.CONFIGS["c3"]
    inp = W.make_inputs(shape, W.data_seed("c3"))
    only = [(0, 0), (7, 11), (3, 5)]
    faults = [W.Fault("AS", 3, 5, 700, 131, np.inf), W.Fault("dAP", 7, 11, 1000, 3, -1e10),
              W.Fault("dQ", 0, 0, 513, 60, np.nan), W.Fault("dK", 3, 5, 64, 7, 1e10),
              W.Fault("dV", 7, 11, 1023, 63, np.inf)] if with_faults else []
    print(f"[case] fused c3 training sampled heads faults={len(faults)}", flush=True)
    cfg = abft.LayerConfig(shape.batch, shape.seq, shape.hidden, shape.heads, causal=True,
                           block_rows=shape.block_rows, fused=True)
    layer = abft.ProtectedAttention(cfg)
    X, Wqkv, Wo, dO = (dev(inp[k]) for k in ("X", "Wqkv", "Wo", "dO"))
    fdev = abft.faults_to_device(faults)
    layer.forward(X, Wqkv, Wo, fdev)
    layer.backward(dO, X, Wqkv, Wo, fdev)
    torch.cuda.synchronize()
    rep_f, rep_b = abft.read_report(layer.report), abft.read_report(layer.report_bwd)
    dQKV = host(layer.tensor("dQKV"))
    p = OracleParams(heads=shape.heads, causal=True, block_rows=shape.block_rows)
    ref, fwd_events = sampled_core(inp, shape, p, only, faults)
    H, d = shape.hidden, shape.head_dim
    assert rep_f["n_uncorrectable"] == 0 and rep_b["n_uncorrectable"] == 0
    assert sorted(rep_f["events"]) == sorted(fwd_events)
    assert sorted(rep_b["events"]) == sorted(e for r in ref.values() for e in r["events"])
    for (b, h), r in ref.items():
        for i, k in enumerate(("dQ", "dK", "dV")):
            got = dQKV[b, :, i * H + h * d:i * H + (h + 1) * d]
            assert np.isfinite(got).all(), (b, h, k)
            nrel = np.linalg.norm(got - r[k]) / np.linalg.norm(r[k])
            assert nrel <= RTOL, f"{k}[{b},{h}]: relative norm {nrel:.3g}"
