"""The report's lifetime across calls (the C ABI's report semantics): a call
without ABFT_FLAG_REPORT_APPEND starts from a cleared report (the layer
clears its counters inside its first launch, the checksum encode, when it
encodes; otherwise with a launch of its own), with the flag events
accumulate. Checked for the forward and the backward, for a protected
layer, a layer whose checksum encode is off (no sections), and an
unprotected one."""
import numpy as np
import pytest
import torch

import workloads as W

pytestmark = pytest.mark.gpu


def _abft():
    from paper_2410_11720_amd import abft
    return abft


def _setup(sections=15, protect=True):
    abft = _abft()
    shape = W.make_shape(1, 256, 128, 2, causal=True)
    inp = W.make_inputs(shape, 77)
    X, Wqkv, Wo, dO = (torch.from_numpy(inp[k]).to("cuda").to(torch.bfloat16)
                       for k in ("X", "Wqkv", "Wo", "dO"))
    cfg = abft.LayerConfig(shape.batch, shape.seq, shape.hidden, shape.heads, causal=True,
                           sections=sections, protect=protect)
    lay = abft.ProtectedAttention(cfg)
    return abft, cfg, lay, (X, Wqkv, Wo, dO)


def _fwd(abft, cfg, lay, t, faults, append):
    X, Wqkv, Wo, _ = t
    O = torch.empty_like(X)
    f, n = faults
    abft.attn_abft_forward(cfg, X, Wqkv, Wo, O, lay.workspace, f, n, lay.report, append=append)
    torch.cuda.synchronize()
    return abft.read_report(lay.report)


def _bwd(abft, cfg, lay, t, faults, append):
    X, Wqkv, Wo, dO = t
    dX = torch.empty_like(X)
    dWqkv = torch.empty((X.shape[-1], 3 * X.shape[-1]), dtype=torch.float32, device="cuda")
    dWo = torch.empty((X.shape[-1], X.shape[-1]), dtype=torch.float32, device="cuda")
    f, n = faults
    abft.attn_abft_backward(cfg, dO, X, Wqkv, Wo, lay.workspace, dX, dWqkv, dWo, f, n,
                            lay.report_bwd, append=append)
    torch.cuda.synchronize()
    return abft.read_report(lay.report_bwd)


def test_forward_report_cleared_per_call_and_appended_on_request():
    abft, cfg, lay, t = _setup()
    one = abft.faults_to_device([W.Fault("AS", 0, 1, 200, 30, np.inf)])
    assert _fwd(abft, cfg, lay, t, one, False)["n_events"] == 1
    assert _fwd(abft, cfg, lay, t, one, True)["n_events"] == 2
    rep = _fwd(abft, cfg, lay, t, (None, 0), False)
    assert rep["n_events"] == 0 and rep["n_corrected"] == 0 and rep["events"] == []
    assert _fwd(abft, cfg, lay, t, one, False)["n_events"] == 1


def test_backward_report_cleared_per_call_and_appended_on_request():
    abft, cfg, lay, t = _setup()
    _fwd(abft, cfg, lay, t, (None, 0), False)
    one = abft.faults_to_device([W.Fault("dX", 0, 0, 100, 5, np.nan)])
    assert _bwd(abft, cfg, lay, t, one, False)["n_events"] == 1
    assert _bwd(abft, cfg, lay, t, one, True)["n_events"] == 2
    assert _bwd(abft, cfg, lay, t, (None, 0), False)["n_events"] == 0


@pytest.mark.parametrize("sections,protect", [(0, True), (15, False)])
def test_report_cleared_without_an_encode(sections, protect):
    """No checksum encode runs (no section enabled, or unprotected): the
    report is still cleared by a non-appending call."""
    abft, cfg, lay, t = _setup(sections, protect)
    cfg_p = abft.LayerConfig(cfg.batch, cfg.seq, cfg.hidden, cfg.heads, causal=True)
    lay_p = abft.ProtectedAttention(cfg_p)
    one = abft.faults_to_device([W.Fault("AS", 0, 1, 200, 30, np.inf)])
    # events recorded by a protected call into this layer's report
    X, Wqkv, Wo, _ = t
    O = torch.empty_like(X)
    abft.attn_abft_forward(cfg_p, X, Wqkv, Wo, O, lay_p.workspace, one[0], one[1], lay.report)
    torch.cuda.synchronize()
    assert abft.read_report(lay.report)["n_events"] == 1
    assert _fwd(abft, cfg, lay, t, (None, 0), False)["n_events"] == 0
