"""Pins of the fused-attention oracle (oracle/fused.py) against facts that
do not come from it: the materialised-attention oracle (itself pinned in
test_oracle_layer.py) in the fp32 storage mode, closed forms of softmax
attention, and the restoration of a fault-free run by the row checks."""
import numpy as np
import pytest

import workloads as W
from oracle import OracleParams, forward
from oracle.eec import col_checksums, row_checksums
from oracle.fused import fused_attention, fused_forward
from oracle.layer import _Run


def _inputs(S=256, H=128, nh=2, seed=3, dtype="bf16"):
    sh = W.make_shape(1, S, H, nh, dtype=dtype)
    return W.make_inputs(sh, seed)


@pytest.mark.parametrize("causal", [False, True])
@pytest.mark.parametrize("R", [128, 64])
def test_matches_materialised_attention_in_fp32(causal, R):
    """With fp32 storage the two forms differ only by where fp32 rounding
    is applied (AS and AP stored vs P rounded per key block)."""
    inp = _inputs(dtype="f32")
    p = OracleParams(heads=2, dtype="f32", causal=causal, block_rows=R)
    a = forward(inp["X"], inp["Wqkv"], inp["Wo"], p)
    f = fused_forward(inp["X"], inp["Wqkv"], inp["Wo"], p)
    scale = np.abs(a["CL"]).max()
    assert np.abs(a["CL"] - f["CL"]).max() <= 1e-6 * scale
    assert np.abs(a["O"] - f["O"]).max() <= 1e-6 * np.abs(a["O"]).max()
    assert a["events"] == [] and f["events"] == []
    # CL^c is encoded from CL, so it equals the column sums of the result
    assert np.allclose(f["CLc"], col_checksums(f["CL"], R), rtol=0, atol=0)


def _direct(Q, K, V, causal, R=128, faults=(), root_check=True, dtype="f64"):
    """fused_attention on hand-made Q, K, V of one head ([S, d] each), with
    the checksums the projection would propagate computed from them."""
    S, d = Q.shape
    p = OracleParams(heads=1, dtype=dtype, causal=causal, block_rows=R, root_check=root_check)
    run = _Run(p, faults)
    nq = S // R
    Kc = col_checksums(K, R)                                   # [nq, 2, d]
    Vr = row_checksums(V, d)                                   # [S, 1, 2]
    pr = dict(B=1, S=S, H=d, nh=1, d=d, R=R, nq=nq, scale=1.0 / np.sqrt(d),
              Qh=Q[None, None], Kh=K[None, None], Vh=V[None, None],
              Kch=Kc[None, None], Vr=Vr[None])
    CL, CLc = fused_attention(run, pr, p)
    return CL, run.events


@pytest.mark.parametrize("causal", [False, True])
def test_zero_queries_give_the_mean_of_the_allowed_values(causal):
    """Q = 0 makes every score equal: each query averages V over the keys
    it may see (all keys, or keys 0..i under the causal mask)."""
    rng = np.random.default_rng(0)
    S, d = 256, 64
    V = rng.standard_normal((S, d))
    CL, ev = _direct(np.zeros((S, d)), rng.standard_normal((S, d)), V, causal)
    want = np.cumsum(V, axis=0) / np.arange(1, S + 1)[:, None] if causal else \
        np.broadcast_to(V.mean(axis=0), (S, d))
    assert np.allclose(CL, want, rtol=1e-12, atol=1e-12)
    assert ev == []


def test_constant_values_pass_through_and_one_hot_scores_select():
    """Rows of softmax sum to one (V constant -> CL constant), and a query
    whose score with one key dominates every other by far returns that key's
    value row."""
    rng = np.random.default_rng(1)
    S, d = 128, 64
    Q, K = rng.standard_normal((S, d)), rng.standard_normal((S, d))
    CL, _ = _direct(Q, K, np.full((S, d), 2.5), False)
    assert np.allclose(CL, 2.5, rtol=1e-13)
    K2 = np.zeros((S, d))
    K2[37, 0] = 1.0
    Q2 = np.zeros((S, d))
    Q2[:, 0] = 8.0 * 60.0       # scale 1/8: key 37 scores 60 above the others
    V = rng.standard_normal((S, d))
    CL2, _ = _direct(Q2, K2, V, False)
    assert np.allclose(CL2, np.broadcast_to(V[37], (S, d)), rtol=1e-20, atol=1e-20 + 1e-24)


def _fault_case(kind):
    return {"INF": np.inf, "NaN": np.nan, "near": 3e10, "numeric": 55.0}[kind]


@pytest.mark.parametrize("kind", ["INF", "NaN", "near", "numeric", "flip"])
@pytest.mark.parametrize("causal", [False, True])
def test_score_fault_is_recomputed_and_the_run_restored(kind, causal):
    inp = _inputs()
    p = OracleParams(heads=2, dtype="bf16", causal=causal, block_rows=64)
    f0 = fused_forward(inp["X"], inp["Wqkv"], inp["Wo"], p)
    # a masked position of a diagonal tile under the mask, else a plain one
    r, c = (150, 170) if causal else (150, 20)
    fault = W.Fault("AS", 0, 1, r, c, 0.0, mode="flip") if kind == "flip" else \
        W.Fault("AS", 0, 1, r, c, _fault_case(kind))
    f = fused_forward(inp["X"], inp["Wqkv"], inp["Wo"], p, [fault])
    assert [(e[0], e[1], e[2], e[3], e[4], e[6]) for e in f["events"]] == \
        [("AS", 0, 1, r, c, "RECOMPUTE")]
    assert np.array_equal(f["CL"], f0["CL"]) and np.array_equal(f["O"], f0["O"])


def test_key_fault_without_root_check():
    """Root check off. On the attention core alone (K unverified) a K error
    corrupts one score column in every query that sees the key (1C), which
    each row vector locates and fixes from the checksums (K^c came from the
    clean projection). The fused form verifies K at the projection in every
    mode (its backward's key pass checks score columns, which cannot see a
    K error), so there the element is fixed from K's checksums and the
    scores see nothing."""
    from oracle.fused import fused_attention
    from oracle.layer import _Run, project
    inp = _inputs()
    p = OracleParams(heads=2, dtype="bf16", causal=False, block_rows=128, root_check=False)
    f0 = fused_forward(inp["X"], inp["Wqkv"], inp["Wo"], p)
    fault = [W.Fault("K", 0, 0, 77, 5, 1e6)]
    run = _Run(p, fault)
    pr = project(run, inp["X"], inp["Wqkv"], p)               # K not verified
    CL, _ = fused_attention(run, pr, p)
    ev = [e for e in run.events if e[0] == "AS"]
    assert len(ev) == 256 and {e[4] for e in ev} == {77} and {e[3] for e in ev} == set(range(256))
    assert all(e[6] in ("DELTA", "RECONSTRUCT") for e in ev)
    assert np.abs(CL - f0["CL"]).max() <= 2.0 ** -6 * np.abs(f0["CL"]).max()
    f = fused_forward(inp["X"], inp["Wqkv"], inp["Wo"], p, fault)
    assert [(e[0], e[3], e[4]) for e in f["events"]] == [("K", 77, 5)]
    assert np.abs(f["CL"] - f0["CL"]).max() <= 2.0 ** -6 * np.abs(f0["CL"]).max()


def test_query_fault_is_caught_at_the_projection():
    """A Q error corrupts a whole score row (1R) together with that row's
    propagated checksums AS^r = Q (K^c)^T, so the row checks cannot see it
    (shown on the attention core alone, Q unverified); the fused form
    therefore verifies Q at the projection in every mode: with the root
    check on it is recomputed and the run equals the fault-free one, with
    it off it is fixed from the checksums and CL stays within rounding."""
    from oracle.fused import fused_attention
    from oracle.layer import _Run, project
    inp = _inputs()
    fault = [W.Fault("Q", 0, 1, 200, 3, 1e8)]
    p_off = OracleParams(heads=2, dtype="bf16", causal=True, block_rows=128, root_check=False)
    f0 = fused_forward(inp["X"], inp["Wqkv"], inp["Wo"], p_off)
    run = _Run(p_off, fault)
    pr = project(run, inp["X"], inp["Wqkv"], p_off)          # Q not verified
    CL, _ = fused_attention(run, pr, p_off)
    assert run.events == []
    assert not np.array_equal(CL[0, 200, 64:], f0["CL"][0, 200, 64:])
    f = fused_forward(inp["X"], inp["Wqkv"], inp["Wo"], p_off, fault)
    assert [(e[0], e[3], e[4], e[6]) for e in f["events"]] == [("Q", 200, 3, "RECONSTRUCT")]
    assert np.abs(f["CL"] - f0["CL"]).max() <= 2.0 ** -6 * np.abs(f0["CL"]).max()
    p_on = OracleParams(heads=2, dtype="bf16", causal=True, block_rows=128)
    g = fused_forward(inp["X"], inp["Wqkv"], inp["Wo"], p_on, fault)
    assert [(e[0], e[3], e[4], e[6]) for e in g["events"]] == [("Q", 200, 3, "RECOMPUTE")]
    assert np.array_equal(g["CL"], f0["CL"])


@pytest.mark.parametrize("val,action", [(np.inf, "RECONSTRUCT"), (np.nan, "RECONSTRUCT"),
                                        (1e12, "RECONSTRUCT"), (40.0, "DELTA")])
def test_context_fault_is_fixed_from_the_row_checksum(val, action):
    inp = _inputs()
    p = OracleParams(heads=2, dtype="bf16", causal=True, block_rows=128)
    f0 = fused_forward(inp["X"], inp["Wqkv"], inp["Wo"], p)
    f = fused_forward(inp["X"], inp["Wqkv"], inp["Wo"], p, [W.Fault("CL", 0, 0, 99, 17, val)])
    assert [(e[0], e[3], e[4], e[6]) for e in f["events"]] == [("CL", 99, 17, action)]
    # the fixed element is within bf16 rounding of its row's magnitude
    row = f0["CL"][0, 99, :64]
    assert abs(f["CL"][0, 99, 17] - f0["CL"][0, 99, 17]) <= 2.0 ** -7 * np.abs(row).sum()


@pytest.mark.parametrize("causal", [False, True])
def test_key_block_size_changes_rounding_only(causal):
    """The online softmax visits keys one checksum block at a time; in the
    unrounded (f64) mode the block size leaves the result unchanged up to
    fp64 rounding, and a sequence that is not a multiple of 128 works."""
    inp = _inputs(S=192, dtype="f32")
    outs = []
    for R in (32, 64):
        p = OracleParams(heads=2, dtype="f64", causal=causal, block_rows=R)
        f = fused_forward(inp["X"], inp["Wqkv"], inp["Wo"], p)
        assert f["events"] == []
        outs.append(f["CL"])
    assert np.abs(outs[0] - outs[1]).max() <= 1e-12 * np.abs(outs[0]).max()


@pytest.mark.parametrize("causal", [False, True])
def test_regenerated_probabilities_feed_the_backward(causal):
    """The softmax statistics of the fused forward regenerate AP (and AP^r),
    and with CL^r they let the layer's backward run after a fused forward:
    in fp32 storage the gradients equal those after the materialised
    forward."""
    from oracle import backward
    inp = _inputs(dtype="f32")
    p = OracleParams(heads=2, dtype="f32", causal=causal, block_rows=128)
    a = forward(inp["X"], inp["Wqkv"], inp["Wo"], p)
    f = fused_forward(inp["X"], inp["Wqkv"], inp["Wo"], p)
    assert np.abs(a["AP"] - f["AP"]).max() <= 1e-6
    assert np.abs(a["CLr"] - f["CLr"]).max() <= 1e-5 * np.abs(a["CLr"]).max()
    # every regenerated row is a probability distribution over its keys
    S = 256
    assert np.allclose(f["AP"].sum(axis=-1), 1.0, atol=1e-5)
    if causal:
        assert np.all(f["AP"][..., np.triu(np.ones((S, S), dtype=bool), 1)] == 0.0)
    ba, bf = backward(a, inp["dO"], p), backward(f, inp["dO"], p)
    for k in ("dX", "dWqkv", "dWo"):
        assert np.abs(ba[k] - bf[k]).max() <= 1e-5 * np.abs(ba[k]).max(), k
    assert ba["events"] == [] and bf["events"] == []


@pytest.mark.parametrize("causal", [False, True])
@pytest.mark.parametrize("R", [128, 64])
def test_fused_backward_equals_the_materialised_backward_unrounded(causal, R):
    """In the unrounded mode the fused backward core (scores recomputed
    from the softmax statistics, the row term D = dCL . CL) gives the
    materialised backward's gradients: sum_j P_ij dP_ij = dCL_i . CL_i."""
    from oracle import backward
    from oracle.fused import fused_training_backward
    inp = _inputs(dtype="f32")
    p = OracleParams(heads=2, dtype="f64", causal=causal, block_rows=R)
    m = forward(inp["X"], inp["Wqkv"], inp["Wo"], p)
    mb = backward(m, inp["dO"], p)
    f = fused_forward(inp["X"], inp["Wqkv"], inp["Wo"], p)
    fb = fused_training_backward(f, inp["dO"], p)
    for k in ("dX", "dWqkv", "dWo", "dQKV"):
        assert np.abs(fb[k] - mb[k]).max() <= 1e-12 * np.abs(mb[k]).max(), k
    assert fb["events"] == [] and mb["events"] == []


@pytest.mark.parametrize("seed", [1, 2, 3])
def test_fused_backward_no_false_positives(seed):
    from oracle.fused import fused_training_backward
    inp = _inputs(seed=seed)
    for causal in (False, True):
        p = OracleParams(heads=2, causal=causal, block_rows=64)
        f = fused_forward(inp["X"], inp["Wqkv"], inp["Wo"], p)
        assert fused_training_backward(f, inp["dO"], p)["events"] == []


@pytest.mark.parametrize("op,val,action", [("AS", np.inf, "RECOMPUTE"), ("AS", np.nan, "RECOMPUTE"),
                                           ("dAP", 1e10, "RECOMPUTE"), ("dAP", -np.inf, "RECOMPUTE"),
                                           ("dQ", np.nan, "RECONSTRUCT"), ("dQ", 40.0, "DELTA"),
                                           ("dK", np.inf, "RECONSTRUCT"), ("dV", -30.0, "DELTA")])
def test_fused_backward_faults_are_located_and_fixed(op, val, action):
    """A score fault and a dP fault reach both passes of the fused backward
    and are located in each (by a column in the key pass, by a row in the
    query pass) and recomputed: the gradients stay within a bf16 step of
    the fault-free ones at that element. A fault in dQ, dK or dV is fixed
    from its row checksum within the bf16 reconstruction bound."""
    from oracle.fused import fused_training_backward
    inp = _inputs()
    p = OracleParams(heads=2, dtype="bf16", causal=True, block_rows=64)
    f0 = fused_forward(inp["X"], inp["Wqkv"], inp["Wo"], p)
    b0 = fused_training_backward(f0, inp["dO"], p)
    fault = W.Fault(op, 0, 1, 150, 70 if op in ("AS", "dAP") else 17, val)
    f = fused_forward(inp["X"], inp["Wqkv"], inp["Wo"], p)
    b = fused_training_backward(f, inp["dO"], p, [fault])
    n = 2 if op in ("AS", "dAP") else 1
    assert [(e[0], e[1], e[2], e[3], e[4], e[6]) for e in b["events"]] == \
        [(op, 0, 1, 150, fault.col, action)] * n
    if op in ("dQ", "dK", "dV"):
        c0 = {"dQ": 0, "dK": 128, "dV": 256}[op] + 64
        row = b0["dQKV"][0, 150, c0:c0 + 64]
        assert abs(b["dQKV"][0, 150, c0 + 17] - row[17]) <= 2.0 ** -8 * (np.abs(row).sum() + abs(row[17]))
    else:
        for k in ("dX", "dWqkv", "dWo"):
            ref = b0[k]
            scale = np.maximum(np.abs(ref), np.sqrt(np.mean(ref ** 2)))
            assert np.max(np.abs(b[k] - ref) / scale) <= 1e-2, k


@pytest.mark.parametrize("op", ["AS", "dAP"])
def test_fused_backward_without_root_check_fixes_from_both_sides(op):
    """Root check off: a score or dP fault is fixed from the checksums in
    each pass, from the column checksums (Q^c K^T, dCL^c V^T) in the key
    pass and from the row checksums (Q (K^c)^T, dCL (V^c)^T) in the query
    pass; the gradients stay within 1e-2 of the fault-free ones."""
    from oracle.fused import fused_training_backward
    inp = _inputs()
    p = OracleParams(heads=2, dtype="bf16", causal=True, block_rows=64, root_check=False)
    f0 = fused_forward(inp["X"], inp["Wqkv"], inp["Wo"], p)
    b0 = fused_training_backward(f0, inp["dO"], p)
    fault = W.Fault(op, 0, 0, 200, 131, 1e12)
    b = fused_training_backward(f0, inp["dO"], p, [fault])
    assert [(e[0], e[3], e[4], e[6]) for e in b["events"]] == [(op, 200, 131, "RECONSTRUCT")] * 2
    for k in ("dX", "dWqkv", "dWo"):
        ref = b0[k]
        scale = np.maximum(np.abs(ref), np.sqrt(np.mean(ref ** 2)))
        assert np.max(np.abs(b[k] - ref) / scale) <= 1e-2, k


def test_key_pass_column_check_sees_a_dcl_row_error():
    """The key pass checks dP = dCL V^T by columns against dCL^c V^T, with
    dCL^c propagated from dO^c W^O^T rather than taken from the stored dCL:
    an error in a dCL row that escaped dCL's own check (here simulated by
    corrupting the operand) makes a 1R pattern in dP that every column
    vector of its block sees, and the fix from the column checksums
    restores the products of the clean operand."""
    from oracle.fused import _checked_scores_cols
    from oracle.layer import _Run
    rng = np.random.default_rng(5)
    S, d, R = 128, 64, 64
    A, Bm = rng.standard_normal((S, d)), rng.standard_normal((S, d))
    Ac = np.stack([np.stack([A[q * R:(q + 1) * R].sum(0),
                             (np.arange(1, R + 1)[:, None] * A[q * R:(q + 1) * R]).sum(0)])
                   for q in range(S // R)])
    p = OracleParams(heads=1, dtype="bf16", causal=False, block_rows=R)
    A2 = A.copy()
    A2[70, 5] += 1e6
    run = _Run(p, [])
    s = _checked_scores_cols(run, p, "dAP", 0, 0, A2, Bm, Ac, 1e10, False)
    assert sorted((e[3], e[4]) for e in run.events) == [(70, j) for j in range(S)]
    assert {e[6] for e in run.events} <= {"DELTA", "RECONSTRUCT"}
    ref = A @ Bm.T
    assert np.abs(s - ref).max() <= 1e-6 * np.abs(ref).max()
