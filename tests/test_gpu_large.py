"""The two large decoder workloads at full size on the GPU (through the C
ABI): B4 S2048 H4096 (32 heads of 128) and B1 S4096 H5120 (40 heads of
128), causal, bf16.

The whole-layer oracle is too slow on the CPU at these sizes; the
head-restricted oracle (oracle/heads.py) gives every tensor of a sampled
head, and its blocks of the weight gradients. Two kinds of check:

* Stage by stage, at full size: the oracle's stored inputs of a sampled
  head are written into the GPU's workspace, one stage of the chain runs,
  and its output for that head must be within one bf16 step of the
  oracle's output of the same stage plus the bound of an fp32 sum
  (|fp32 sum - exact| <= n 2^-24 sum|terms|; the two sides round nearby
  sums, so the stored values differ by at most one step of the larger
  plus that bound). The softmax backward adds the effect of its fp32 row
  sum on the difference dAP - rowdot.
* Chained, fault-free: every tensor of the sampled heads against the
  oracle's chain. Both sides round every stored tensor to bf16, from fp32
  sums here and fp64 sums there; where they keep adjacent values (one
  step apart) the difference passes on through exp and the cancellation
  in dAP - rowdot, so elements can move by a few steps. These are checked
  in relative norm (<= 1e-2); the projections (one rounding) elementwise,
  the weight-gradient blocks in relative norm. O and dX, which mix every
  head, are checked elementwise against an fp32 product of the GPU's own
  operands (one bf16 step plus the fp32 bound).
Fault runs (Sec. 5.2) are checked by properties that hold at any size:
the event set equals the injected list (position and class of the stored
value, corrected by recomputation with the root check on), and every
output is within 1e-2 of the fault-free run.
"""
import numpy as np
import pytest
import torch

import workloads as W
from oracle import OracleParams
from oracle.heads import head_reference
from oracle.layer import masked_cols_product, masked_rows_product, softmax_backward, softmax_forward
from oracle.numerics import classify, round_to, stored_threshold

pytestmark = pytest.mark.gpu
RTOL = 1e-2
WEIGHT_OPS = ("dWO", "dWQ", "dWK", "dWV")
EPS32 = 2.0 ** -24


def _abft():
    from paper_2410_11720_amd import abft
    return abft


def dev(a):
    return torch.from_numpy(np.ascontiguousarray(a, dtype=np.float32)).to("cuda").to(torch.bfloat16)


def host(t):
    return t.float().cpu().numpy().astype(np.float64)


def step(v):
    """bf16 spacing at |v| (numpy or torch)."""
    if isinstance(v, torch.Tensor):
        a = torch.clamp(v.abs(), min=2.0 ** -126)
        return torch.exp2(torch.floor(torch.log2(a)) - 7)
    a = np.maximum(np.abs(v), 2.0 ** -126)
    return 2.0 ** (np.floor(np.log2(a)) - 7)


def rel_err(gpu, ref):
    """max |gpu - ref| / max(|ref|, rms(ref)) (torch tensors)."""
    a, b = gpu.float(), ref.float()
    if not torch.isfinite(a).all():
        return float("inf")
    scale = torch.clamp(b.abs(), min=float(b.pow(2).mean().sqrt()) + 1e-30)
    return float(((a - b).abs() / scale).max())


def norm_err(gpu, ref):
    a, b = np.asarray(gpu, dtype=np.float64), np.asarray(ref, dtype=np.float64)
    assert np.isfinite(a).all()
    return float(np.linalg.norm(a - b) / np.linalg.norm(b))


def assert_stage(gpu, ref, acc, name):
    """|gpu - ref| <= one bf16 step at the larger + the fp32 bound acc."""
    gpu = np.asarray(gpu, dtype=np.float64)
    assert np.isfinite(gpu).all(), name
    over = np.abs(gpu - ref) - (step(np.maximum(np.abs(gpu), np.abs(ref))) + acc)
    assert over.max() <= 0.0, f"{name}: {np.count_nonzero(over > 0)} elements over the bound"


def expected_event(f, shape):
    """(op, b, h, row, col, kind, action) the library must report for an
    injected fault: its position, the class of the value as stored (fp32
    for weight gradients, else the storage dtype), corrected by
    recomputation from the checked operands."""
    dt = "f32" if f.op in WEIGHT_OPS else shape.dtype
    stored = float(round_to(np.array([f.value]), dt)[0])
    kind = classify(stored, stored_threshold(1e10, dt))
    return (f.op, f.b, f.h, f.row, f.col, kind, "RECOMPUTE")


class Layer:
    """One full-size protected layer with its inputs on the GPU."""

    def __init__(self, shape, seed):
        abft = _abft()
        self.abft, self.shape = abft, shape
        self.inp = W.make_inputs(shape, seed)
        self.cfg = abft.LayerConfig(shape.batch, shape.seq, shape.hidden, shape.heads,
                                    causal=shape.causal, block_rows=shape.block_rows)
        self.X, self.Wqkv, self.Wo, self.dO = (dev(self.inp[k]) for k in ("X", "Wqkv", "Wo", "dO"))
        self.layer = abft.ProtectedAttention(self.cfg)
        self.p = OracleParams(heads=shape.heads, causal=shape.causal, block_rows=shape.block_rows)
        self.refs = {}

    def step(self, faults=()):
        abft, L = self.abft, self.layer
        fdev = abft.faults_to_device(list(faults))
        O = L.forward(self.X, self.Wqkv, self.Wo, fdev)
        dX, dWqkv, dWo = L.backward(self.dO, self.X, self.Wqkv, self.Wo, fdev)
        torch.cuda.synchronize()
        ev = abft.read_report(L.report)["events"] + abft.read_report(L.report_bwd)["events"]
        return dict(O=O, dX=dX, dWqkv=dWqkv, dWo=dWo), ev

    def ref(self, h):
        """The head-restricted oracle for head h over every batch element."""
        if h not in self.refs:
            print(f"[case] {self.shape.name} oracle head {h}", flush=True)
            self.refs[h] = head_reference(self.inp["X"], self.inp["Wqkv"], self.inp["Wo"],
                                          self.inp["dO"], self.p, h, list(range(self.shape.batch)))
        return self.refs[h]


def check_chained(lay, heads):
    """Fault-free run against the oracle's chain for the given heads."""
    shape, L = lay.shape, lay.layer
    print(f"[case] {shape.name} fault-free run", flush=True)
    out, ev = lay.step()
    assert ev == []
    H, d, S = shape.hidden, shape.head_dim, shape.seq
    tri = np.tril(np.ones((S, S), dtype=bool)) if shape.causal else np.ones((S, S), dtype=bool)
    QKV, CL, dQKV, dCL, AP = (L.tensor(k) for k in ("QKV", "CL", "dQKV", "dCL", "AP"))
    Wa = np.abs(lay.inp["Wqkv"]).astype(np.float64)
    Woa = np.abs(lay.inp["Wo"]).astype(np.float64)
    for h in heads:
        ref = lay.ref(h)
        cs = slice(h * d, (h + 1) * d)
        for b in range(shape.batch):
            # one rounding of a sum over the hidden dimension (elementwise)
            x = np.abs(lay.inp["X"][b]).astype(np.float64)
            g = np.abs(lay.inp["dO"][b]).astype(np.float64)
            for i, name in enumerate("QKV"):
                acc = H * EPS32 * (x @ Wa[:, i * H + h * d:i * H + (h + 1) * d])
                assert_stage(host(QKV[b, :, i * H:(i + 1) * H][:, cs]), ref[name][b], acc,
                             f"{name}[{b},{h}]")
            acc = H * EPS32 * (g @ Woa[cs, :].T)
            assert_stage(host(dCL[b, :, cs]), ref["dCL"][b], acc, f"dCL[{b},{h}]")
            # the rest of the chain, in relative norm
            for name, gt, r in (("AP", host(AP[b, h])[tri], ref["AP"][b][tri]),
                                ("CL", host(CL[b, :, cs]), ref["CL"][b]),
                                ("dQ", host(dQKV[b, :, cs]), ref["dQ"][b]),
                                ("dK", host(dQKV[b, :, H:][:, cs]), ref["dK"][b]),
                                ("dV", host(dQKV[b, :, 2 * H:][:, cs]), ref["dV"][b])):
                e = norm_err(gt, r)
                assert e <= RTOL, f"{name}[{b},{h}] relative norm {e:.3g}"
        for name, gt, r in (("dWQ", out["dWqkv"][:, cs], ref["dWQ"]),
                            ("dWK", out["dWqkv"][:, H:][:, cs], ref["dWK"]),
                            ("dWV", out["dWqkv"][:, 2 * H:][:, cs], ref["dWV"]),
                            ("dWO", out["dWo"][cs, :], ref["dWO"])):
            e = norm_err(host(gt), r)
            assert e <= RTOL, f"{name} head {h} relative norm {e:.3g}"
    # O and dX mix every head: one rounding of a sum over their operands
    for name, A, B, C in (("O", CL.reshape(-1, H), lay.Wo, out["O"]),
                          ("dX", dQKV.reshape(-1, 3 * H), lay.Wqkv.T, out["dX"])):
        A32, B32 = A.float(), B.float()
        refm = A32 @ B32
        acc = 2 * A.shape[1] * EPS32 * (A32.abs() @ B32.abs())
        got = C.float().reshape(refm.shape)
        bound = step(torch.maximum(refm.abs(), got.abs())) + acc
        over = (got - refm).abs() - bound
        assert float(over.max()) <= 0.0, f"{name}: {int((over > 0).sum())} elements over"
    return {k: v.clone() for k, v in out.items()}


def check_stages(lay, h, b):
    """Each stage of the chain alone, for head h of batch element b, on
    the oracle's stored inputs written into the workspace."""
    abft, L, shape = lay.abft, lay.layer, lay.shape
    ref = lay.ref(h)
    H, d, S = shape.hidden, shape.head_dim, shape.seq
    cs = slice(h * d, (h + 1) * d)
    scale = 1.0 / np.sqrt(d)
    rnd = lambda a: round_to(a, "bf16")
    causal = shape.causal
    tri = np.tril(np.ones((S, S), dtype=bool)) if causal else np.ones((S, S), dtype=bool)
    Q, K, V = ref["Q"][b], ref["K"][b], ref["V"][b]
    AP, dCL, dAP, dAS = ref["AP"][b], ref["dCL"][b], ref["dAP"][b], ref["dAS"][b]
    QKV, CLt, dCLt, dQKV = (L.tensor(k) for k in ("QKV", "CL", "dCL", "dQKV"))
    O = torch.empty_like(lay.X)
    dX = torch.empty_like(lay.X)
    dW = torch.empty((H, 3 * H), dtype=torch.float32, device="cuda")
    dWo = torch.empty((H, H), dtype=torch.float32, device="cuda")

    def fwd(stage):
        abft.attn_abft_forward_stages(lay.cfg, lay.X, lay.Wqkv, lay.Wo, O, L.workspace, None, 0,
                                      L.report, abft.FWD_STAGES[stage])
        torch.cuda.synchronize()
        assert abft.read_report(L.report)["events"] == [], stage

    def bwd(stage):
        abft.attn_abft_backward_stages(lay.cfg, lay.dO, lay.X, lay.Wqkv, lay.Wo, L.workspace, dX,
                                       dW, dWo, None, 0, L.report_bwd, abft.BWD_STAGES[stage])
        torch.cuda.synchronize()
        assert abft.read_report(L.report_bwd)["events"] == [], stage

    print(f"[case] {shape.name} stages of head ({b},{h})", flush=True)
    lay.step()                              # every buffer holds a whole step
    QKV[b, :, cs].copy_(dev(Q))
    QKV[b, :, H:][:, cs].copy_(dev(K))
    QKV[b, :, 2 * H:][:, cs].copy_(dev(V))
    fwd("score")
    assert_stage(host(L.tensor("AS")[b, h])[tri], rnd(Q @ K.T)[tri],
                 (d * EPS32 * (np.abs(Q) @ np.abs(K).T))[tri], "score")
    L.tensor("AS")[b, h].copy_(dev(ref["AS"][b]))
    fwd("softmax")
    # fp32 exponentials and the fp32 row sum: a relative error of at most
    # (S + 8) 2^-24 before the rounding
    AP_ref = softmax_forward(ref["AS"][b], scale, causal, rnd)
    assert_stage(host(L.tensor("AP")[b, h])[tri], AP_ref[tri], (S + 8) * EPS32 * AP_ref[tri],
                 "softmax")
    L.tensor("AP")[b, h].copy_(dev(AP))
    fwd("context")
    assert_stage(host(CLt[b, :, cs]), rnd(masked_rows_product(AP, V, causal)),
                 S * EPS32 * (AP @ np.abs(V)), "context")
    # backward stages, each on the oracle's inputs of that stage
    dCLt[b, :, cs].copy_(dev(dCL))
    bwd("dAP")
    assert_stage(host(L.tensor("AS")[b, h])[tri], rnd(dCL @ V.T)[tri],
                 (d * EPS32 * (np.abs(dCL) @ np.abs(V).T))[tri], "dAP")
    bwd("dV")
    assert_stage(host(dQKV[b, :, 2 * H:][:, cs]), rnd(masked_cols_product(AP, dCL, causal)),
                 S * EPS32 * (AP.T @ np.abs(dCL)), "dV")
    L.tensor("AS")[b, h].copy_(dev(dAP))
    bwd("softmax_bwd")
    rowsum = np.where(tri, AP * np.abs(dAP), 0.0).sum(axis=1, keepdims=True)
    assert_stage(host(L.tensor("dAS")[b, h])[tri],
                 softmax_backward(AP, dAP, scale, causal, rnd)[tri],
                 (scale * AP * (S * EPS32 * rowsum + EPS32 * np.abs(dAP)))[tri], "softmax_bwd")
    L.tensor("dAS")[b, h].copy_(dev(dAS))
    bwd("dQ")
    assert_stage(host(dQKV[b, :, cs]), rnd(masked_rows_product(dAS, K, causal)),
                 S * EPS32 * (np.abs(dAS) @ np.abs(K)), "dQ")
    bwd("dK")
    assert_stage(host(dQKV[b, :, H:][:, cs]), rnd(masked_cols_product(dAS, Q, causal)),
                 S * EPS32 * (np.abs(dAS).T @ np.abs(Q)), "dK")


def check_fault_run(lay, ref_out, faults):
    """Events equal the injected list; outputs within the bar of the
    fault-free run."""
    print(f"[case] {lay.shape.name} faults {[f.as_tuple() for f in faults]}", flush=True)
    out, ev = lay.step(faults)
    want = sorted(expected_event(f, lay.shape) for f in faults)
    assert sorted(ev) == want
    for k in ("O", "dX", "dWqkv", "dWo"):
        e = rel_err(out[k], ref_out[k])
        assert e <= RTOL, f"{k} after faults: rel err {e:.3g}"


@pytest.fixture(scope="module")
def c4():
    lay = Layer(W.C4, W.data_seed("c4"))
    ref_out = check_chained(lay, [0, 31])
    return lay, ref_out


def test_c4_fault_free_sampled_heads(c4):
    """Runs in the fixture: heads 0 and 31 of every batch element."""
    lay, ref_out = c4
    assert set(ref_out) == {"O", "dX", "dWqkv", "dWo"}


@pytest.mark.parametrize("op", ["AS", "Q", "dWQ"])
def test_c4_single_faults(c4, op):
    """A single INF, NaN or near-INF (+-1e10) fault in the scores, the
    X W^Q output or dW^Q (one run each)."""
    lay, ref_out = c4
    base = 4000 + 10 * ("AS", "Q", "dWQ").index(op)
    for i, kind in enumerate(("inf", "nan", "+1e10" if op != "Q" else "-1e10")):
        faults = W.draw_faults(lay.shape, W.fault_seed("c4", base + i), 1, [op], [kind])
        check_fault_run(lay, ref_out, faults)


def test_c4_stages_sampled_heads(c4):
    lay, _ = c4
    check_stages(lay, 0, 2)
    check_stages(lay, 31, 0)


@pytest.fixture(scope="module")
def c5():
    lay = Layer(W.C5, W.data_seed("c5"))
    ref_out = check_chained(lay, [0, 39])
    return lay, ref_out


def test_c5_fault_free_sampled_heads(c5):
    """Runs in the fixture (also the count-0 point of the sweep)."""
    lay, ref_out = c5
    assert set(ref_out) == {"O", "dX", "dWqkv", "dWo"}


@pytest.mark.parametrize("count", [1, 4, 16])
@pytest.mark.parametrize("mag", ["1e6", "1e10", "1e30"])
def test_c5_fault_sweep(c5, count, mag):
    """The stress sweep: count faults (distinct rows and columns of each
    output) across all 16 protected GEMM outputs, magnitude mag with a
    random sign."""
    lay, ref_out = c5
    seed = W.fault_seed("c5", 100 * count + {"1e6": 6, "1e10": 10, "1e30": 30}[mag])
    faults = W.draw_faults(lay.shape, seed, count, W.ALL_OPS, ["+" + mag, "-" + mag])
    check_fault_run(lay, ref_out, faults)


def test_c5_stages_sampled_heads(c5):
    lay, _ = c5
    check_stages(lay, 39, 0)
