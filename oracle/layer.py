"""The protected multi-head attention layer, forward and backward (oracle;
test infrastructure).

Forward (Sec. 2.1 Eq. 1-2, execution flow of Fig. 1; protection sections
and checksum passing of Sec. 4.4, Fig. 5):
  S_AS = {X W^Q, X W^K, Q K^T}: X is encoded with column checksums per
         R-token block; Q^c, K^c ride through X W; AS carries AS^c = Q^c K^T
         (column side) and AS^r = Q (K^c)^T (row side).
  S_CL = {X W^V, AP V}: W^V is encoded with row checksums per head so that
         V^r = X W^V r; AP is encoded with column checksums after softmax;
         CL carries CL^c = AP^c V and CL^r = AP V^r.
  S_O  = {CL W^O}: O^c = CL^c W^O.
Root check (a reading, on by default): Q, K and V are verified against
Q^c, K^c, V^c right after the projection and corrected there, so that the
backward chain, which reuses them, sees clean operands; with it off the
forward is the paper's literal scheme, where Q/K/V errors surface as 1-D
patterns in AS and CL and are corrected there from checksums only.

Backward (an extension; the paper protects the forward GEMMs only): every
backward GEMM output C = A B carries C^c = A^c B with A^c propagated from
earlier checksums (dO^c, CL^r, dCL^c, AP^r, dAS^c, dAS^r, X^r) and gets a
column pass. The softmax and its backward are unprotected, like the
forward softmax; their outputs are re-encoded.

Layouts: X [B,S,H]; Wqkv [H,3H] (Q|K|V column blocks); Wo [H,H];
head h owns columns [h d, (h+1) d). Scores are stored unscaled and before
the causal mask; softmax applies the scale and masks by selection, so
masked probabilities are exactly zero. Under a causal mask the checksums
cover only the block-lower-triangular region at the checksum-block
granularity (key block <= query block), the part a tiled score GEMM
computes.

Masked products (a reading; the paper uses dense products): a product
over keys with a causally masked factor (AP V, dAS K, and over queries
AP^T dCL, dAS^T Q) is the sum over the pairs the mask allows, as Eq. 1
defines attention under a causal mask: query i takes keys j <= i and key
j takes queries i >= j; a checksum row of an R-query block takes the keys
up to the block's last query, a checksum row of an R-key block the
queries from the block's first key. The terms left out are exact zeros,
so this equals the dense product whenever the other factor is finite; a
dense product would also multiply an INF or NaN by a masked zero
(0 * INF = NaN), which this definition never does.
"""
from __future__ import annotations

import dataclasses
from collections import defaultdict

import numpy as np

from .numerics import flip_exponent_msb, round_to, stored_threshold
from .eec import col_checksums, row_checksums, Verifier

SECTIONS = ("AS", "CL", "O", "BWD")


def masked_rows_product(P, M, causal):
    """C_i = sum over keys j <= i of P_ij M_j (all keys if not causal).
    P [..., S, S], M [..., S, n]."""
    if not causal:
        return P @ M
    S = P.shape[-1]
    out = np.empty(P.shape[:-1] + M.shape[-1:])
    with np.errstate(invalid="ignore", over="ignore"):
        for i in range(S):
            out[..., i:i + 1, :] = P[..., i:i + 1, :i + 1] @ M[..., :i + 1, :]
    return out


def masked_cols_product(P, M, causal):
    """C_j = sum over queries i >= j of P_ij M_i (dense P^T M if not
    causal)."""
    if not causal:
        return P.swapaxes(-1, -2) @ M
    S = P.shape[-1]
    out = np.empty(P.shape[:-2] + (S, M.shape[-1]))
    with np.errstate(invalid="ignore", over="ignore"):
        for j in range(S):
            out[..., j:j + 1, :] = P[..., j:, j:j + 1].swapaxes(-1, -2) @ M[..., j:, :]
    return out


def masked_block_rows_product(Pc, M, R, causal):
    """Checksum rows of a rows-product: Pc [..., nq, 2, S] are checksum rows
    over R-query blocks; block qb takes the keys up to its last query,
    j < (qb + 1) R."""
    if not causal:
        return Pc @ M[..., None, :, :]
    nq = Pc.shape[-3]
    out = np.empty(Pc.shape[:-1] + M.shape[-1:])
    with np.errstate(invalid="ignore", over="ignore"):
        for qb in range(nq):
            e = (qb + 1) * R
            out[..., qb, :, :] = Pc[..., qb, :, :e] @ M[..., :e, :]
    return out


def masked_block_cols_product(Pr, M, R, causal):
    """Checksum rows of a cols-product: Pr [..., S, nq, 2] are row checksums
    over R-key blocks; block kb takes the queries from its first key,
    i >= kb R."""
    nq = Pr.shape[-2]
    out = np.empty(Pr.shape[:-3] + (nq, 2, M.shape[-1]))
    with np.errstate(invalid="ignore", over="ignore"):
        for kb in range(nq):
            s0 = kb * R if causal else 0
            out[..., kb, :, :] = Pr[..., s0:, kb, :].swapaxes(-1, -2) @ M[..., s0:, :]
    return out


def _allowed(S, causal):
    """Pairs (query i, key j) the mask lets through: j <= i, or all."""
    return np.tril(np.ones((S, S), dtype=bool)) if causal else np.ones((S, S), dtype=bool)


def softmax_forward(AS, scale, causal, rnd):
    """AP = softmax over keys of scale * AS (Eq. 1), masked keys selected
    to -INF so their probabilities are exact zeros; the row maximum is
    subtracted first; the result is rounded by rnd (to storage)."""
    mask = _allowed(AS.shape[-1], causal)
    with np.errstate(invalid="ignore", over="ignore"):
        Z = np.where(mask, scale * AS, -np.inf)
        m = Z.max(axis=-1, keepdims=True)
        Ez = np.where(mask, np.exp(Z - m), 0.0)
        return rnd(Ez / Ez.sum(axis=-1, keepdims=True))


def softmax_backward(AP, dAP, scale, causal, rnd):
    """dAS = scale * AP * (dAP - sum_j AP_ij dAP_ij) on the allowed pairs,
    exact zeros on masked ones (the softmax Jacobian applied to dAP, with
    the scale of the forward's argument); rounded by rnd."""
    mask = _allowed(AP.shape[-1], causal)
    with np.errstate(invalid="ignore", over="ignore"):
        Dr = np.where(mask, dAP * AP, 0.0).sum(axis=-1, keepdims=True)
        return rnd(np.where(mask, scale * AP * (dAP - Dr), 0.0))


@dataclasses.dataclass
class OracleParams:
    heads: int
    causal: bool = False
    dtype: str = "bf16"            # storage dtype of activations: bf16 | f32 | f64
    block_rows: int = 128          # checksum block R along token axes
    scale: float | None = None     # softmax scale; 1/sqrt(head_dim) when None
    t_near_inf: float = 1e10       # Sec. 4.2
    t_correct: float = 1e5         # Sec. 4.2
    e_rel: float | None = None     # detection bound factor; see default_e_rel
    root_check: bool = True
    protect: bool = True
    sections: tuple = SECTIONS     # protection sections enabled this step

    def e_rel_value(self):
        return default_e_rel(self.dtype) if self.e_rel is None else self.e_rel


def default_e_rel(dtype: str) -> float:
    """E = e_rel * sum|v| (Sec. 2.3 leaves E open). Storage rounding of the
    output moves its checksum by at most u * sum|v| (unit roundoff u = 2^-8
    for bf16, 2^-24 for f32); rounding of stored upstream operands (CL
    before W^O, dQ/dK/dV before dX) reaches a propagated checksum through
    the next GEMM and is not bounded by sum|v|: on nearly constant output
    columns it was measured at up to 0.23 * 2^-5 * sum|v| on random-init
    layers. e_rel = 16u (bf16) and 2^11 u (f32) keep every fault-free vector
    well inside E while any single value >= 1e6 stays far outside."""
    return {"bf16": 2.0 ** -4, "f32": 2.0 ** -13, "f64": 2.0 ** -40}[dtype]


def _w_dtype(dtype):
    """Weight gradients are stored in fp32 (fp64 in the unrounded mode)."""
    return "f64" if dtype == "f64" else "f32"


def pattern_of_events(events):
    """Propagation pattern (Sec. 2.2) of each event, from the set of
    elements corrected in the same output: an element sharing its row with
    another correction is 1R, sharing its column is 1C, else 0D;
    uncorrectable vectors are 2D. Returns a list parallel to events."""
    rows, cols = defaultdict(int), defaultdict(int)
    for (op, b, h, r, c, kind, action) in events:
        if action != "UNCORRECTABLE":
            rows[(op, b, h, r)] += 1
            cols[(op, b, h, c)] += 1
    out = []
    for (op, b, h, r, c, kind, action) in events:
        if action == "UNCORRECTABLE":
            out.append("2D")
        elif rows[(op, b, h, r)] > 1:
            out.append("1R")
        elif cols[(op, b, h, c)] > 1:
            out.append("1C")
        else:
            out.append("0D")
    return out


class _Run:
    """Shared state of one oracle call: parameters, faults and events."""

    def __init__(self, p: OracleParams, faults):
        self.p = p
        self.rnd = lambda a: round_to(a, p.dtype)
        self.rndw = lambda a: round_to(a, _w_dtype(p.dtype))
        self.faults = defaultdict(list)
        for f in faults:
            t = f.as_tuple() if hasattr(f, "as_tuple") else tuple(f)
            self.faults[t[0]].append(t[1:])
        self.events = []
        tn = stored_threshold(p.t_near_inf, p.dtype)
        self.ver = Verifier(p.dtype, p.e_rel_value(), tn, p.t_correct)
        self.ver_w = Verifier(_w_dtype(p.dtype), p.e_rel_value(),
                              stored_threshold(p.t_near_inf, _w_dtype(p.dtype)),
                              p.t_correct)

    def inject(self, op, M, place, wdtype=False):
        """Apply op's faults to M (already rounded to storage): mode "set"
        writes the fault value rounded to storage, mode "flip" flips the
        exponent MSB of the stored value. place(b, h, r, c) -> index tuple
        into M."""
        rnd = self.rndw if wdtype else self.rnd
        dt = _w_dtype(self.p.dtype) if wdtype else self.p.dtype
        for t in self.faults.get(op, ()):
            b, h, r, c, val = t[:5]
            idx = place(b, h, r, c)
            if len(t) > 5 and t[5] == "flip":
                M[idx] = flip_exponent_msb(float(M[idx]), dt)
            else:
                M[idx] = rnd(np.array([val]))[0]

    def on(self, section):
        return self.p.protect and section in self.p.sections

    def verify(self, C3, Cc, R, name_of, *, Cr=None, Cb=None, col_valid=None,
               row_valid=None, recompute=None, weights=False):
        """Run the verification procedure on C3 [n, rows, cols] (a view whose
        writes land in the caller's tensor) and record events."""
        ver = self.ver_w if weights else self.ver
        if not self.p.root_check:
            recompute = None
        evs, unc = ver.run(C3, Cc, R, Cr=Cr, Cb=Cb, col_valid=col_valid,
                           row_valid=row_valid, recompute=recompute)
        for (k, i, j, kind, action) in evs:
            op, b, h, r, c = name_of(int(k), int(i), int(j))
            self.events.append((op, int(b), int(h), int(r), int(c), kind, action))
        for u in unc:
            if u[0] == "col":
                _, k, blk, j = u
                op, b, h, r, c = name_of(k, blk * R, j)
            else:
                _, k, i, cb = u
                op, b, h, r, c = name_of(k, i, cb * Cb)
            self.events.append((op, int(b), int(h), int(r), int(c), "-", "UNCORRECTABLE"))


def _row_dot(prow, mcol, i, S, causal):
    """One element of a rows-product: query i over keys j <= i."""
    e = i + 1 if causal else S
    return prow[:e] @ mcol[:e]


def _col_dot(pcol, mcol, j, causal):
    """One element of a cols-product: key j over queries i >= j."""
    s0 = j if causal else 0
    return pcol[s0:] @ mcol[s0:]


def _causal_valid(n, S, R):
    """Which checksum vectors of a causal score-shaped output are computed:
    column vectors (query block qb, key j) with j // R <= qb and row vectors
    (query i, key block kb) with kb <= i // R."""
    qb = np.arange(S // R)[:, None]
    j = np.arange(S)[None, :]
    colv = np.broadcast_to((j // R) <= qb, (n, S // R, S))
    i = np.arange(S)[:, None]
    kb = np.arange(S // R)[None, :]
    rowv = np.broadcast_to(kb <= (i // R), (n, S, S // R))
    return colv, rowv


def project(run, X, Wqkv, p: OracleParams, verify_always=False):
    """Encoding and the protected QKV projection (Sec. 4.4 S_AS / S_CL
    members X W^Q, X W^K, X W^V), with the root check. `verify_always`
    checks Q, K and V at the projection with the root check off too (a
    score check with one side cannot see an error of the operand on that
    side, Sec. 4.3's 1R and 1C patterns); the fix is then from the
    checksums. Returns the projection outputs, their checksums and the
    layer's dimensions."""
    X = np.asarray(X, dtype=np.float64)
    Wqkv = np.asarray(Wqkv, dtype=np.float64)
    B, S, H = X.shape
    nh = p.heads
    d = H // nh
    R = p.block_rows
    nq = S // R
    if H != nh * d or S % R:
        raise ValueError("hidden must equal heads*head_dim and R must divide seq")
    scale = p.scale if p.scale is not None else 1.0 / np.sqrt(d)
    rnd = run.rnd

    # encode (Sec. 4.4: X column checksums; W^V row checksums per head)
    Xc = col_checksums(X, R)                                   # [B,nq,2,H]
    Xr = row_checksums(X, d)                                   # [B,S,nh,2]
    WVr = row_checksums(Wqkv[:, 2 * H:], d).reshape(H, 2 * nh)  # [H,2nh]

    # projections Q|K|V = X Wqkv, checksums ride along
    QKV = rnd(X @ Wqkv)                                        # [B,S,3H]
    QKVc = Xc @ Wqkv                                           # [B,nq,2,3H]
    Vr = (X @ WVr).reshape(B, S, nh, 2)                        # [B,S,nh,2]
    for i, op in enumerate(("Q", "K", "V")):
        run.inject(op, QKV, lambda b, h, r, c, i=i: (b, r, i * H + h * d + c))
    if p.protect and (p.root_check or verify_always):
        colmask = np.zeros(3 * H, dtype=bool)
        if "AS" in p.sections:
            colmask[:2 * H] = True
        if "CL" in p.sections:
            colmask[2 * H:] = True
        if colmask.any():
            run.verify(QKV, QKVc, R,
                       lambda k, i, j: ("QKV"[j // H], k, (j % H) // d, i, j % d),
                       col_valid=np.broadcast_to(colmask, (B, nq, 3 * H)),
                       recompute=lambda k, i, j: X[k, i] @ Wqkv[:, j])


    def heads_of(M):        # [B,S,H] -> [B,nh,S,d]
        return M.reshape(B, S, nh, d).transpose(0, 2, 1, 3)

    def heads_of_c(Mc):     # [B,nq,2,H] -> [B,nh,nq,2,d]
        return Mc.reshape(B, nq, 2, nh, d).transpose(0, 3, 1, 2, 4)

    Qh, Kh, Vh = (heads_of(QKV[..., i * H:(i + 1) * H]) for i in range(3))
    Qch, Kch = heads_of_c(QKVc[..., :H]), heads_of_c(QKVc[..., H:2 * H])
    return dict(X=X, Wqkv=Wqkv, B=B, S=S, H=H, nh=nh, d=d, R=R, nq=nq, scale=scale,
                Xc=Xc, Xr=Xr, QKV=QKV, QKVc=QKVc, Vr=Vr, Qh=Qh, Kh=Kh, Vh=Vh,
                Qch=Qch, Kch=Kch)


def output_projection(run, CL, CLc_full, Wo, p: OracleParams):
    """O = CL W^O with O^c = CL^c W^O and its column pass (Sec. 4.4 S_O)."""
    rnd = run.rnd
    O = rnd(CL @ Wo)
    Oc = CLc_full @ Wo
    run.inject("O", O, lambda b, h, r, c: (b, r, c))
    if run.on("O"):
        run.verify(O, Oc, p.block_rows, lambda k, i, j: ("O", k, 0, i, j),
                   recompute=lambda k, i, j: CL[k, i] @ Wo[:, j])
    return O, Oc


def forward(X, Wqkv, Wo, p: OracleParams, faults=()):
    """Protected forward of one attention layer. Inputs hold storage-dtype
    values. Returns a dict with O, the saved tensors, propagated checksums
    the backward reuses, and the event list."""
    run = _Run(p, faults)
    pr = project(run, X, Wqkv, p)
    X, Wqkv = pr["X"], pr["Wqkv"]
    B, S, H, nh, d, R, nq, scale = (pr[k] for k in ("B", "S", "H", "nh", "d", "R", "nq", "scale"))
    Xc, Xr, QKV, QKVc, Vr = (pr[k] for k in ("Xc", "Xr", "QKV", "QKVc", "Vr"))
    Qh, Kh, Vh, Qch, Kch = (pr[k] for k in ("Qh", "Kh", "Vh", "Qch", "Kch"))
    Wo = np.asarray(Wo, dtype=np.float64)
    rnd = run.rnd

    # score GEMM AS = Q K^T (unscaled, before the mask), two-sided checksums
    AS = rnd(Qh @ Kh.swapaxes(-1, -2))                         # [B,nh,S,S]
    ASc = Qch @ Kh.swapaxes(-1, -2)[:, :, None]                # [B,nh,nq,2,S]
    ASr = (Qh @ Kch.reshape(B, nh, 2 * nq, d).swapaxes(-1, -2)).reshape(B, nh, S, nq, 2)
    run.inject("AS", AS, lambda b, h, r, c: (b, h, r, c))
    if run.on("AS"):
        colv, rowv = _causal_valid(B * nh, S, R) if p.causal else (None, None)
        run.verify(AS.reshape(B * nh, S, S), ASc.reshape(B * nh, nq, 2, S), R,
                   lambda k, i, j: ("AS", k // nh, k % nh, i, j),
                   Cr=ASr.reshape(B * nh, S, nq, 2), Cb=R,
                   col_valid=colv, row_valid=rowv,
                   recompute=lambda k, i, j: Qh[k // nh, k % nh, i] @ Kh[k // nh, k % nh, j])

    # softmax with the causal mask applied by selection (unprotected)
    AP = softmax_forward(AS, scale, p.causal, rnd)             # [B,nh,S,S]
    APc = col_checksums(AP, R)                                 # [B,nh,nq,2,S]
    APr = row_checksums(AP, R)                                 # [B,nh,S,nq,2]

    # context GEMM CL = AP V, two-sided checksums (row side via V^r)
    cz = p.causal
    CLh = rnd(masked_rows_product(AP, Vh, cz))                 # [B,nh,S,d]
    CLc = masked_block_rows_product(APc, Vh, R, cz)            # [B,nh,nq,2,d]
    CLr = np.ascontiguousarray(
        masked_rows_product(AP, Vr.transpose(0, 2, 1, 3), cz)[:, :, :, None, :])  # [B,nh,S,1,2]
    run.inject("CL", CLh, lambda b, h, r, c: (b, h, r, c))
    if run.on("CL"):
        CLh3 = CLh.reshape(B * nh, S, d)
        run.verify(CLh3, CLc.reshape(B * nh, nq, 2, d), R,
                   lambda k, i, j: ("CL", k // nh, k % nh, i, j),
                   Cr=CLr.reshape(B * nh, S, 1, 2), Cb=d,
                   recompute=lambda k, i, j: _row_dot(AP[k // nh, k % nh, i],
                                                      Vh[k // nh, k % nh, :, j], i, S, cz))
    CL = CLh.transpose(0, 2, 1, 3).reshape(B, S, H)
    CLc_full = CLc.transpose(0, 2, 3, 1, 4).reshape(B, nq, 2, H)
    CLr_full = CLr[:, :, :, 0, :].transpose(0, 2, 1, 3)        # [B,S,nh,2]

    # output projection O = CL Wo, column checksums O^c = CL^c Wo
    O, Oc = output_projection(run, CL, CLc_full, Wo, p)

    return dict(O=O, QKV=QKV, AS=AS, AP=AP, CL=CL, X=X, Wqkv=Wqkv, Wo=Wo,
                Xc=Xc, Xr=Xr, QKVc=QKVc, Vr=Vr, APc=APc, APr=APr,
                CLc=CLc_full, CLr=CLr_full, Oc=Oc, scale=scale,
                events=run.events, params=p)


def backward(fwd: dict, dO, p: OracleParams, faults=(), core=None):
    """Protected backward chain (extension). Returns dX, dWqkv, dWo, the
    intermediate gradients and the event list. core, if given, replaces
    the steps from dCL to dQ, dK and dV (dAP, the softmax backward and the
    three products): core(run, ctx, p) with ctx holding the per-head
    operands returns dQ, dK, dV and their column checksums dQ^c, dK^c,
    dV^c."""
    run = _Run(p, faults)
    rnd, rndw = run.rnd, run.rndw
    X, Wqkv, Wo = fwd["X"], fwd["Wqkv"], fwd["Wo"]
    QKV, AP, CL = fwd["QKV"], fwd["AP"], fwd["CL"]
    dO = np.asarray(dO, dtype=np.float64)
    B, S, H = X.shape
    nh = p.heads
    d = H // nh
    R = p.block_rows
    nq = S // R
    T = B * S
    scale = fwd["scale"]
    on = run.on("BWD")

    def heads_of(M):
        return M.reshape(B, S, nh, d).transpose(0, 2, 1, 3)

    def heads_of_c(Mc):
        return Mc.reshape(B, nq, 2, nh, d).transpose(0, 3, 1, 2, 4)

    Qh, Kh, Vh = (heads_of(QKV[..., i * H:(i + 1) * H]) for i in range(3))
    dOc = col_checksums(dO, R)                                 # [B,nq,2,H]

    # dCL = dO Wo^T
    dCL = rnd(dO @ Wo.T)
    dCLc = dOc @ Wo.T
    run.inject("dCL", dCL, lambda b, h, r, c: (b, r, h * d + c))
    if on:
        run.verify(dCL, dCLc, R, lambda k, i, j: ("dCL", k, j // d, i, j % d),
                   recompute=lambda k, i, j: dO[k, i] @ Wo[j, :])

    # dWo = CL^T dO; column checksums over head blocks of rows from CL^r
    CLf, dOf = CL.reshape(T, H), dO.reshape(T, H)
    dWo = rndw(CLf.T @ dOf)                                    # [H,H]
    dWoc = (fwd["CLr"].reshape(T, 2 * nh).T @ dOf).reshape(1, nh, 2, H)
    run.inject("dWO", dWo, lambda b, h, r, c: (r, c), wdtype=True)
    if on:
        run.verify(dWo[None], dWoc, d, lambda k, i, j: ("dWO", 0, 0, i, j),
                   recompute=lambda k, i, j: CLf[:, i] @ dOf[:, j], weights=True)

    dCLh = heads_of(dCL)
    cz = p.causal
    if core is None:
        APr = fwd["APr"]
        # dAP = dCL_h V_h^T
        dAP = rnd(dCLh @ Vh.swapaxes(-1, -2))                      # [B,nh,S,S]
        dAPc = heads_of_c(dCLc) @ Vh.swapaxes(-1, -2)[:, :, None]  # [B,nh,nq,2,S]
        run.inject("dAP", dAP, lambda b, h, r, c: (b, h, r, c))
        if on:
            colv = _causal_valid(B * nh, S, R)[0] if p.causal else None
            run.verify(dAP.reshape(B * nh, S, S), dAPc.reshape(B * nh, nq, 2, S), R,
                       lambda k, i, j: ("dAP", k // nh, k % nh, i, j), col_valid=colv,
                       recompute=lambda k, i, j: dCLh[k // nh, k % nh, i] @ Vh[k // nh, k % nh, j])

        # softmax backward (unprotected), masked entries selected to zero
        dAS = softmax_backward(AP, dAP, scale, p.causal, rnd)
        dASc = col_checksums(dAS, R)                               # [B,nh,nq,2,S]
        dASr = row_checksums(dAS, R)                               # [B,nh,S,nq,2]

        # dQ = dAS K_h
        dQh = rnd(masked_rows_product(dAS, Kh, cz))
        dQc = masked_block_rows_product(dASc, Kh, R, cz)           # [B,nh,nq,2,d]
        run.inject("dQ", dQh, lambda b, h, r, c: (b, h, r, c))
        if on:
            run.verify(dQh.reshape(B * nh, S, d), dQc.reshape(B * nh, nq, 2, d), R,
                       lambda k, i, j: ("dQ", k // nh, k % nh, i, j),
                       recompute=lambda k, i, j: _row_dot(dAS[k // nh, k % nh, i],
                                                          Kh[k // nh, k % nh, :, j], i, S, cz))
    else:
        ctx = dict(B=B, S=S, H=H, nh=nh, d=d, R=R, nq=nq, scale=scale, Qh=Qh, Kh=Kh, Vh=Vh,
                   dCLh=dCLh, CLh=heads_of(CL), Qch=heads_of_c(fwd["QKVc"][..., :H]),
                   Kch=heads_of_c(fwd["QKVc"][..., H:2 * H]),
                   Vch=heads_of_c(fwd["QKVc"][..., 2 * H:]), dCLch=heads_of_c(dCLc),
                   m=fwd["m"], l=fwd["l"])
        c = core(run, ctx, p)
        dQh, dKh, dVh, dQc, dKc, dVc = (c[k] for k in ("dQ", "dK", "dV", "dQc", "dKc", "dVc"))
        dAP = dAS = None

    if core is None:
        dVh, dVc, dKh, dKc = _materialised_dv_dk(run, AP, APr, dAS, dASr, dCLh, Qh, p, R, on)
    return _weight_and_input_grads(run, fwd, p, dQh, dKh, dVh, dQc, dKc, dVc, dWo, dCL, dAP,
                                   dAS, B, S, H, nh, d, nq, T)


def _materialised_dv_dk(run, AP, APr, dAS, dASr, dCLh, Qh, p, R, on):
    """dV = AP^T dCL and dK = dAS^T Q with their propagated column
    checksums over key blocks (from AP^r and dAS^r), checked."""
    rnd, cz = run.rnd, p.causal
    B, nh, S = AP.shape[:3]
    d, nq = dCLh.shape[3], S // R
    # dV = AP^T dCL_h; column checksums over key blocks from AP^r
    dVh = rnd(masked_cols_product(AP, dCLh, cz))               # [B,nh,S,d]
    dVc = masked_block_cols_product(APr, dCLh, R, cz)          # [B,nh,nq,2,d]
    run.inject("dV", dVh, lambda b, h, r, c: (b, h, r, c))
    if on:
        run.verify(dVh.reshape(B * nh, S, d), dVc.reshape(B * nh, nq, 2, d), R,
                   lambda k, i, j: ("dV", k // nh, k % nh, i, j),
                   recompute=lambda k, i, j: _col_dot(AP[k // nh, k % nh, :, i],
                                                      dCLh[k // nh, k % nh, :, j], i, cz))

    # dK = dAS^T Q_h; column checksums over key blocks from dAS^r
    dKh = rnd(masked_cols_product(dAS, Qh, cz))
    dKc = masked_block_cols_product(dASr, Qh, R, cz)           # [B,nh,nq,2,d]
    run.inject("dK", dKh, lambda b, h, r, c: (b, h, r, c))
    if on:
        run.verify(dKh.reshape(B * nh, S, d), dKc.reshape(B * nh, nq, 2, d), R,
                   lambda k, i, j: ("dK", k // nh, k % nh, i, j),
                   recompute=lambda k, i, j: _col_dot(dAS[k // nh, k % nh, :, i],
                                                      Qh[k // nh, k % nh, :, j], i, cz))
    return dVh, dVc, dKh, dKc


def _weight_and_input_grads(run, fwd, p, dQh, dKh, dVh, dQc, dKc, dVc, dWo, dCL, dAP, dAS,
                            B, S, H, nh, d, nq, T):
    """dWqkv and dX from the three head gradients, checked; the backward's
    result dictionary."""
    rnd, rndw, on = run.rnd, run.rndw, run.on("BWD")
    R = p.block_rows
    X, Wqkv = fwd["X"], fwd["Wqkv"]

    def merge(Mh):          # [B,nh,S,d] -> [B,S,H]
        return Mh.transpose(0, 2, 1, 3).reshape(B, S, H)

    def merge_c(Mc):        # [B,nh,nq,2,d] -> [B,nq,2,H]
        return Mc.transpose(0, 2, 3, 1, 4).reshape(B, nq, 2, H)

    dQKV = np.concatenate([merge(dQh), merge(dKh), merge(dVh)], axis=-1)      # [B,S,3H]
    dQKVc = np.concatenate([merge_c(dQc), merge_c(dKc), merge_c(dVc)], axis=-1)

    # dWqkv = X^T dQKV; column checksums over head blocks of rows from X^r
    Xf, dQKVf = X.reshape(T, H), dQKV.reshape(T, 3 * H)
    dW = rndw(Xf.T @ dQKVf)                                    # [H,3H]
    dWc = (fwd["Xr"].reshape(T, 2 * nh).T @ dQKVf).reshape(1, nh, 2, 3 * H)
    for i, op in enumerate(("dWQ", "dWK", "dWV")):
        run.inject(op, dW, lambda b, h, r, c, i=i: (r, i * H + c), wdtype=True)
    if on:
        run.verify(dW[None], dWc, d,
                   lambda k, i, j: (("dWQ", "dWK", "dWV")[j // H], 0, 0, i, j % H),
                   recompute=lambda k, i, j: Xf[:, i] @ dQKVf[:, j], weights=True)

    # dX = dQKV Wqkv^T; column checksums dX^c = dQKV^c Wqkv^T
    dX = rnd(dQKV @ Wqkv.T)
    dXc = dQKVc @ Wqkv.T
    run.inject("dX", dX, lambda b, h, r, c: (b, r, c))
    if on:
        run.verify(dX, dXc, R, lambda k, i, j: ("dX", k, 0, i, j),
                   recompute=lambda k, i, j: dQKV[k, i] @ Wqkv[j, :])

    return dict(dX=dX, dWqkv=dW, dWo=dWo, dCL=dCL, dAP=dAP, dAS=dAS,
                dQKV=dQKV, dQKVc=dQKVc, events=run.events)
