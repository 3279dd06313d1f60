"""Pin of the head-restricted oracle (oracle/heads.py) against the whole
layer oracle (itself pinned in test_oracle_layer.py): every tensor of the
chosen heads equals the layer's, and the weight-gradient blocks equal the
layer's blocks when every batch element is included."""
import numpy as np
import pytest

import workloads as W
from oracle import OracleParams, backward, forward
from oracle.heads import head_reference


def _agree(a, b, dtype, name):
    a, b = np.asarray(a), np.asarray(b)
    assert a.shape == b.shape, name
    if dtype == "f64":
        assert np.allclose(a, b, rtol=1e-10, atol=1e-12), name
    else:
        # same definitions, same rounding points: values are equal except
        # where fp64 sums in another order land on either side of a
        # rounding boundary (one storage step, rarely)
        step = 2.0 ** -7 if dtype == "bf16" else 2.0 ** -23
        diff = np.abs(a - b)
        assert np.all(diff <= step * np.abs(b) + 1e-30), name
        assert np.count_nonzero(diff) <= max(2, a.size // 1000), name


@pytest.mark.parametrize("dtype", ["f64", "bf16"])
@pytest.mark.parametrize("causal", [False, True])
def test_heads_equal_the_layer(causal, dtype):
    sh = W.make_shape(2, 96, 128, 2, causal=causal, block_rows=32, dtype="f32")
    inp = W.make_inputs(sh, 21)
    p = OracleParams(heads=2, causal=causal, dtype=dtype, block_rows=32)
    f = forward(inp["X"], inp["Wqkv"], inp["Wo"], p)
    g = backward(f, inp["dO"], p)
    H, d, S = 128, 64, 96
    for h in range(2):
        ref = head_reference(inp["X"], inp["Wqkv"], inp["Wo"], inp["dO"], p, h, [0, 1])
        for b in range(2):
            cs = slice(h * d, (h + 1) * d)
            _agree(ref["Q"][b], f["QKV"][b, :, cs], dtype, "Q")
            _agree(ref["K"][b], f["QKV"][b, :, H:][:, cs], dtype, "K")
            _agree(ref["V"][b], f["QKV"][b, :, 2 * H:][:, cs], dtype, "V")
            _agree(ref["AS"][b], f["AS"][b, h], dtype, "AS")
            _agree(ref["AP"][b], f["AP"][b, h], dtype, "AP")
            _agree(ref["CL"][b], f["CL"][b, :, cs], dtype, "CL")
            _agree(ref["dCL"][b], g["dCL"][b, :, cs], dtype, "dCL")
            _agree(ref["dAP"][b], g["dAP"][b, h], dtype, "dAP")
            _agree(ref["dAS"][b], g["dAS"][b, h], dtype, "dAS")
            _agree(ref["dQ"][b], g["dQKV"][b, :, cs], dtype, "dQ")
            _agree(ref["dK"][b], g["dQKV"][b, :, H:][:, cs], dtype, "dK")
            _agree(ref["dV"][b], g["dQKV"][b, :, 2 * H:][:, cs], dtype, "dV")
        wd = "f64" if dtype == "f64" else "f32"
        _agree(ref["dWQ"], g["dWqkv"][:, cs], wd, "dWQ")
        _agree(ref["dWK"], g["dWqkv"][:, H:][:, cs], wd, "dWK")
        _agree(ref["dWV"], g["dWqkv"][:, 2 * H:][:, cs], wd, "dWV")
        _agree(ref["dWO"], g["dWo"][cs, :], wd, "dWO")


def test_heads_forward_only_and_batch_subset():
    sh = W.make_shape(3, 64, 128, 2, causal=True, block_rows=32, dtype="f32")
    inp = W.make_inputs(sh, 22)
    p = OracleParams(heads=2, causal=True, dtype="f64", block_rows=32)
    f = forward(inp["X"], inp["Wqkv"], inp["Wo"], p)
    ref = head_reference(inp["X"], inp["Wqkv"], inp["Wo"], None, p, 1, [2], backward=False)
    assert set(ref) >= {"Q", "CL"} and "dWQ" not in ref
    assert np.allclose(ref["CL"][0], f["CL"][2, :, 64:], rtol=1e-10, atol=1e-12)
    # rows of a causal probability matrix sum to one over keys 0..i
    assert np.allclose(ref["AP"][0].sum(axis=-1), 1.0)
    assert np.all(ref["AP"][0][np.triu(np.ones((64, 64), dtype=bool), 1)] == 0.0)
