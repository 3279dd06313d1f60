"""The attention layer restricted to chosen heads (oracle; test
infrastructure).

Fault-free reference values of the layer (Sec. 2.1 Eq. 1-2 and its
backward) for a subset of (batch, head) pairs, for layers too large to run
whole on the CPU. Every value is computed by the same definitions and
rounded at the same points as `layer.forward` / `layer.backward`; a head's
values depend only on its own columns of W^Q, W^K, W^V (and rows of W^O in
the backward), its batch element's X and dO, so the restriction is exact:
  Q_h = X W^Q_h, K_h = X W^K_h, V_h = X W^V_h            (storage-rounded)
  AS = Q_h K_h^T, AP = softmax(scale AS, mask), CL_h = AP V_h
  dCL_h = dO (W^O_h)^T, dAP = dCL_h V_h^T, dV_h = AP^T dCL_h,
  dAS = softmax backward, dQ_h = dAS K_h, dK_h = dAS^T Q_h
with the masked products of `layer` (query i over keys j <= i). The weight
gradients' blocks of a head sum over every token of the batch elements
given: dW^{Q,K,V}_h = X^T d{Q,K,V}_h (columns of the head) and
dW^O rows of the head = CL_h^T dO; they equal the layer's blocks when all
batch elements are included. No checksums, faults or verification.
"""
from __future__ import annotations

import numpy as np

from .layer import (OracleParams, _w_dtype, masked_cols_product, masked_rows_product,
                    softmax_backward, softmax_forward)
from .numerics import round_to


def head_reference(X, Wqkv, Wo, dO, p: OracleParams, head: int, batches, backward=True):
    """Reference tensors of head `head` for each batch element in
    `batches` (dict of lists, one entry per batch element, in that order)
    and the head's weight-gradient blocks summed over those elements."""
    rnd = lambda a: round_to(a, p.dtype)
    rndw = lambda a: round_to(a, _w_dtype(p.dtype))
    H = X.shape[-1]
    nh = p.heads
    d = H // nh
    scale = p.scale if p.scale is not None else 1.0 / np.sqrt(d)
    cols = lambda i: slice(i * H + head * d, i * H + (head + 1) * d)
    Wq, Wk, Wv = (np.asarray(Wqkv[:, cols(i)], dtype=np.float64) for i in range(3))
    Woh = np.asarray(Wo[head * d:(head + 1) * d, :], dtype=np.float64)  # [d, H]
    out = {k: [] for k in ("Q", "K", "V", "AS", "AP", "CL", "dCL", "dAP", "dV", "dAS",
                           "dQ", "dK")}
    dWq = dWk = dWv = dWo = 0.0
    for b in batches:
        x = np.asarray(X[b], dtype=np.float64)                     # [S, H]
        Q, K, V = rnd(x @ Wq), rnd(x @ Wk), rnd(x @ Wv)
        AS = rnd(Q @ K.T)
        AP = softmax_forward(AS, scale, p.causal, rnd)
        CL = rnd(masked_rows_product(AP, V, p.causal))
        for k, v in (("Q", Q), ("K", K), ("V", V), ("AS", AS), ("AP", AP), ("CL", CL)):
            out[k].append(v)
        if not backward:
            continue
        g = np.asarray(dO[b], dtype=np.float64)                    # [S, H]
        dCL = rnd(g @ Woh.T)
        dAP = rnd(dCL @ V.T)
        dV = rnd(masked_cols_product(AP, dCL, p.causal))
        dAS = softmax_backward(AP, dAP, scale, p.causal, rnd)
        dQ = rnd(masked_rows_product(dAS, K, p.causal))
        dK = rnd(masked_cols_product(dAS, Q, p.causal))
        for k, v in (("dCL", dCL), ("dAP", dAP), ("dV", dV), ("dAS", dAS), ("dQ", dQ),
                     ("dK", dK)):
            out[k].append(v)
        dWq = dWq + x.T @ dQ
        dWk = dWk + x.T @ dK
        dWv = dWv + x.T @ dV
        dWo = dWo + CL.T @ g
    if backward:
        out.update(dWQ=rndw(dWq), dWK=rndw(dWk), dWV=rndw(dWv), dWO=rndw(dWo))
    return out
