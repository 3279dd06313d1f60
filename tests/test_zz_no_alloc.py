"""The allocation-free forward (attn_abft_forward_noalloc) against the
forward it is a variant of (attn_abft_forward with ABFT_FLAG_FUSED),
through the C ABI: the same kernels on the same inputs, so O and the
event set must be identical, on two calls in a row (the second with a
smaller layer, on what the first left in the library's buffer)."""
import ctypes

import numpy as np
import pytest
import torch

import workloads as W


def _abft():
    from paper_2410_11720_amd import abft
    return abft


def dev(a):
    return torch.from_numpy(np.ascontiguousarray(a, dtype=np.float32)).to("cuda").to(torch.bfloat16)


def test_oversize_and_unfused_configs_are_rejected_before_any_launch():
    """Host-side checks only (no GPU needed): a layer that does not fit the
    64 MiB buffer, and a config without ABFT_FLAG_FUSED."""
    abft = _abft()
    fake = ctypes.c_void_p(256)   # never dereferenced: the call returns first
    for cfg, want in ((abft.LayerConfig(4, 2048, 4096, 32, causal=True, fused=True), -4),
                      (abft.LayerConfig(1, 256, 128, 2, causal=True, fused=False), -2)):
        c = cfg.to_c()
        got = abft._lib.attn_abft_forward_noalloc(ctypes.byref(c), fake, fake, fake, fake, None,
                                                  0, fake, None)
        assert got == want


@pytest.mark.gpu
def test_noalloc_forward_equals_the_fused_forward_twice():
    abft = _abft()
    cases = [(W.make_shape(8, 1024, 768, 12, causal=True, name="gpt2"), 11,
              [W.Fault("AS", 3, 7, 900, 12, np.inf), W.Fault("CL", 6, 2, 77, 40, np.nan)]),
             (W.make_shape(2, 256, 128, 2, causal=True, name="small"), 12,
              [W.Fault("AS", 1, 0, 200, 3, 1e10)])]
    for shape, seed, faults in cases:
        print(f"[case] noalloc {shape.name}", flush=True)
        inp = W.make_inputs(shape, seed)
        cfg = abft.LayerConfig(shape.batch, shape.seq, shape.hidden, shape.heads,
                               causal=shape.causal, fused=True)
        X, Wqkv, Wo = (dev(inp[k]) for k in ("X", "Wqkv", "Wo"))
        fdev, n = abft.faults_to_device(faults)
        layer = abft.ProtectedAttention(cfg)
        O_ref = layer.forward(X, Wqkv, Wo, (fdev, n))
        O = torch.empty_like(O_ref)
        rep = abft.new_report(256)
        abft.attn_abft_forward_noalloc(cfg, X, Wqkv, Wo, O, fdev, n, rep)
        torch.cuda.synchronize()
        assert torch.equal(O, O_ref)
        got, want = abft.read_report(rep), abft.read_report(layer.report)
        assert sorted(got["events"]) == sorted(want["events"])
        assert len(got["events"]) == len(faults) and got["n_uncorrectable"] == 0
        del layer
