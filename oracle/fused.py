"""Fused protected attention, forward (oracle; test infrastructure).

The score, softmax and context steps of the layer (Sec. 2.1 Eq. 1-2) with
the S_AS and S_CL protections of Sec. 4.4, computed per query tile without
storing the score matrix AS or the probabilities AP: an online-softmax
(flash-style) form, which is an extension; the paper materialises both.
The projection before and the output projection after are the layer's
(`layer.project`, `layer.output_projection`).

Per (batch, head), all queries at once, the keys visited a block at a
time, in increasing order (the online softmax of Milakov and Gimelshein
takes its key blocks in any size; by default one checksum block of R keys,
the unit of the row check of Sec. 4.4). Under a causal mask a query takes
the keys of the R-key blocks up to its own (the block-lower-triangular
region at R granularity that the materialised form checks too):
  1. S = Q K_kb^T, not rounded (it is never stored); AS faults are
     applied to S ("set" writes the value, "flip" flips the exponent MSB of
     S as an fp32 value).
  2. Row check of S (Sec. 4.4 AS^r = Q (K^c)^T, one vector per query and
     R-key block; EEC of Sec. 4.2): a located element is recomputed from Q
     and K (root check on: the operands are clean) or fixed from the
     checksums (root check off). The column side (AS^c) is not checked
     here: a 1R pattern in AS (a Q error, Sec. 4.3) changes a score row
     together with its checksums and is invisible to the rows, and the
     backward's key pass checks columns only, which cannot see a K or V
     error; so Q, K and V are verified at the projection in every mode
     (with the root check off they are fixed from their checksums there),
     and the score checks see the 0D pattern that remains.
  3. Online softmax: m' = max(m, max_j scale S_ij) over unmasked keys,
     p = exp(scale S - m') (masked: 0), alpha = exp(m - m'),
     l = alpha l + sum_j p, P = storage-rounded p,
     A = alpha A + P V_j, A^r = alpha A^r + P V^r_j.
  4. After the last key block: CL = rounded A / l; CL faults are applied;
     CL^r = A^r / l is the propagated row checksum of CL (V^r = X W^V r,
     Sec. 4.4; the rescaling multiplies A and A^r alike). Row check of CL
     (one vector per query over the head's d columns); a located element
     is fixed from the checksum (DELTA / RECONSTRUCT, Sec. 4.2).
  5. CL^c, needed by the output projection, is encoded from the verified
     CL (column checksums per R-query block).
For the backward, the softmax statistics of every query (the final max m
and sum l of step 3) are kept; the fused backward core recomputes the
scores from them (`fused_backward_core`), and CL^r = A^r / l is the
propagated row checksum of CL the backward's dW^O check takes. For
comparisons with the materialised forward, AP is also formed from Q, K
and the statistics: AP = storage-rounded exp(scale Q K^T - m) / l on the
unmasked pairs (0 on masked ones), with its row checksums AP^r.

Rounding: S and the accumulators are kept unrounded (fp64 here, fp32 on
the GPU); P is rounded to the storage dtype (it feeds the P V product);
CL is rounded when stored. The near-INF threshold compares against S as
an fp32 value and against CL as stored.
"""
from __future__ import annotations

import numpy as np

from .eec import col_checksums, eec_locate, fix_by_checksum, row_checksums
from .layer import (OracleParams, _Run, backward, masked_cols_product, masked_rows_product,
                    output_projection, project)
from .numerics import classify, flip_exponent_msb, round_to, stored_threshold



def _check_rows(v2, c1, c2, e_rel, tn, recompute, tc, store=lambda x: x):
    """EEC over the rows of v2 [n, len] with checksums c1, c2 [n]. Fixes v2
    in place, a corrected value passing through `store` (the rounding of
    the place it is kept in). Returns [(row, index, kind, action)] of
    corrected elements and [row] of vectors still inconsistent."""
    events, unc = [], []
    for i in range(v2.shape[0]):
        res = eec_locate(v2[i], c1[i], c2[i], e_rel, tn)
        if res.status == "clean":
            continue
        if res.status == "located":
            j = res.index
            old = float(v2[i, j])
            if recompute is not None:
                new, action = recompute(i, j), "RECOMPUTE"
            else:
                new, action = fix_by_checksum(v2[i], j, c1[i], res.d1, tc)
            v2[i, j] = store(new)
            events.append((i, j, classify(old, tn), action))
        if eec_locate(v2[i], c1[i], c2[i], e_rel, tn).status != "clean":
            unc.append(i)
    return events, unc


def fused_attention(run: _Run, pr: dict, p: OracleParams, only=None, stats=None,
                    key_block=None):
    """Steps 1-5 for every (batch, head), or for the (batch, head) pairs in
    `only` (the others' CL stays zero). Returns CL [B,S,H] and CL^c
    [B,nq,2,H]; events go to run.events. With a dict `stats`, also stores
    there the final max m and sum l of every query ([B,nh,S], natural
    units) and CL^r = A^r / l ([B,S,nh,2]). key_block: keys per step of the
    online softmax (a multiple of R dividing S; default R)."""
    B, S, H, nh, d, R, nq, scale = (pr[k] for k in ("B", "S", "H", "nh", "d", "R", "nq", "scale"))
    KB = R if key_block is None else key_block
    if KB % R or S % KB:
        raise ValueError("the key block must be a multiple of R that divides seq")
    Qh, Kh, Vh, Kch, Vr = pr["Qh"], pr["Kh"], pr["Vh"], pr["Kch"], pr["Vr"]
    e_rel = p.e_rel_value()
    tn_s = stored_threshold(p.t_near_inf, "f32")
    tn_cl = stored_threshold(p.t_near_inf, p.dtype)
    check_as, check_cl = run.on("AS"), run.on("CL")
    recompute_ok = p.root_check
    faults_as = run.faults.get("AS", ())
    faults_cl = run.faults.get("CL", ())
    CLh = np.zeros((B, nh, S, d))
    M_all, L_all = np.zeros((B, nh, S)), np.zeros((B, nh, S))
    CLr_all = np.zeros((B, S, nh, 2))
    queries = np.arange(S)
    for b in range(B):
        for h in range(nh):
            if only is not None and (b, h) not in only:
                continue
            Q, K, V = Qh[b, h], Kh[b, h], Vh[b, h]
            Kc = Kch[b, h]                      # [nq, 2, d]
            vr = Vr[b, :, h, :]                 # [S, 2]
            m = np.full(S, -np.inf)
            l = np.zeros(S)
            A = np.zeros((S, d))
            Ar = np.zeros((S, 2))
            for k0 in range(0, S, KB):
                # queries that see keys from k0 on: all, or those from the
                # R-block of k0 on (the block-lower-triangular region)
                q0 = k0 if p.causal else 0
                rows = queries[q0:]
                s = Q[q0:] @ K[k0:k0 + KB].T                             # 1.
                for (fb, fh, fr, fc, val, *mode) in faults_as:
                    if fb == b and fh == h and fr >= q0 and k0 <= fc < k0 + KB and \
                            (not p.causal or fc // R <= fr // R):
                        i, j = fr - q0, fc - k0
                        if mode and mode[0] == "flip":
                            s[i, j] = flip_exponent_msb(float(round_to(s[i, j], "f32")), "f32")
                        else:
                            s[i, j] = round_to(np.array([val]), "f32")[0]
                if check_as:                                            # 2.
                    for kb in range(k0 // R, (k0 + KB) // R):
                        # the (query, R-key block) vectors of the region
                        r0 = kb * R - q0 if p.causal else 0
                        seg = s[r0:, kb * R - k0:(kb + 1) * R - k0]
                        cs = Q[q0 + r0:] @ Kc[kb].T                     # [rows, 2]
                        rec = ((lambda i, j, r0=r0, kb=kb: Q[q0 + r0 + i] @ K[kb * R + j])
                               if recompute_ok else None)
                        evs, unc = _check_rows(seg, cs[:, 0], cs[:, 1], e_rel, tn_s, rec,
                                               p.t_correct,
                                               store=lambda x: float(round_to(np.array([x]), "f32")[0]))
                        s[r0:, kb * R - k0:(kb + 1) * R - k0] = seg
                        for (i, j, kind, action) in evs:
                            run.events.append(("AS", b, h, q0 + r0 + i, kb * R + j, kind, action))
                        for i in unc:
                            run.events.append(("AS", b, h, q0 + r0 + i, kb * R, "-",
                                               "UNCORRECTABLE"))
                keys = np.arange(k0, k0 + KB)                           # 3.
                allowed = (keys[None, :] <= rows[:, None]) if p.causal else np.ones(s.shape, bool)
                mq = m[q0:]
                with np.errstate(invalid="ignore", over="ignore"):
                    z = np.where(allowed, scale * s, -np.inf)
                    m_new = np.maximum(mq, z.max(axis=1))
                    pz = np.where(allowed, np.exp(z - m_new[:, None]), 0.0)
                    alpha = np.where(np.isfinite(mq), np.exp(mq - m_new), 0.0)
                l[q0:] = alpha * l[q0:] + pz.sum(axis=1)
                P = run.rnd(pz)
                A[q0:] = alpha[:, None] * A[q0:] + P @ V[k0:k0 + KB]
                Ar[q0:] = alpha[:, None] * Ar[q0:] + P @ vr[k0:k0 + KB]
                m[q0:] = m_new
            CLt = run.rnd(A / l[:, None])                               # 4.
            CLr = Ar / l[:, None]
            M_all[b, h], L_all[b, h] = m, l
            CLr_all[b, :, h] = CLr
            for (fb, fh, fr, fc, val, *mode) in faults_cl:
                if fb == b and fh == h:
                    if mode and mode[0] == "flip":
                        CLt[fr, fc] = flip_exponent_msb(float(CLt[fr, fc]), p.dtype)
                    else:
                        CLt[fr, fc] = run.rnd(np.array([val]))[0]
            if check_cl:
                evs, unc = _check_rows(CLt, CLr[:, 0], CLr[:, 1], e_rel, tn_cl, None,
                                       p.t_correct,
                                       store=lambda x: float(run.rnd(np.array([x]))[0]))
                for (i, j, kind, action) in evs:
                    run.events.append(("CL", b, h, i, j, kind, action))
                for i in unc:
                    run.events.append(("CL", b, h, i, 0, "-", "UNCORRECTABLE"))
            CLh[b, h] = CLt
    CL = CLh.transpose(0, 2, 1, 3).reshape(B, S, H)
    CLc = col_checksums(CL, R)                                          # 5.
    if stats is not None:
        stats.update(m=M_all, l=L_all, CLr=CLr_all)
    return CL, CLc


def regenerate_ap(run: _Run, pr: dict, p: OracleParams, m, l):
    """AP = rounded exp(scale Q K^T - m) / l on the unmasked pairs (0 on
    masked ones) and its row checksums per R-key block."""
    Qh, Kh, scale, S, R = pr["Qh"], pr["Kh"], pr["scale"], pr["S"], pr["R"]
    allowed = np.tril(np.ones((S, S), dtype=bool)) if p.causal else np.ones((S, S), dtype=bool)
    with np.errstate(over="ignore", invalid="ignore"):
        Z = scale * (Qh @ Kh.swapaxes(-1, -2))
        AP = run.rnd(np.where(allowed, np.exp(Z - m[..., None]) / l[..., None], 0.0))
    return AP, row_checksums(AP, R)


def fused_forward(X, Wqkv, Wo, p: OracleParams, faults=(), key_block=None):
    """Protected forward of one attention layer with the fused attention
    core. Returns O, CL, its checksums, the projection outputs and the
    event list."""
    run = _Run(p, faults)
    pr = project(run, X, Wqkv, p, verify_always=True)
    st = {}
    CL, CLc = fused_attention(run, pr, p, stats=st, key_block=key_block)
    Wo = np.asarray(Wo, dtype=np.float64)
    O, Oc = output_projection(run, CL, CLc, Wo, p)
    AP, APr = regenerate_ap(run, pr, p, st["m"], st["l"])
    # the dict carries what the layer's backward takes from a forward
    return dict(O=O, CL=CL, CLc=CLc, Oc=Oc, QKV=pr["QKV"], QKVc=pr["QKVc"], Vr=pr["Vr"],
                X=pr["X"], Wqkv=pr["Wqkv"], Wo=Wo, Xc=pr["Xc"], Xr=pr["Xr"], AP=AP, APr=APr,
                CLr=st["CLr"], m=st["m"], l=st["l"], scale=pr["scale"], events=run.events,
                params=p)


def _checked_scores(run, p, op, b, h, A, Bm, Bc, tn, recompute_ok):
    """S = A Bm^T (fp64, not rounded) over the block-lower-triangular
    region at R granularity (all of it without the mask), the faults of op
    applied to the fp32 value, and the row check of every (row, R-column
    block) vector against A (Bc_kb)^T (Sec. 4.4's AS^r form; EEC of
    Sec. 4.2): a located element is recomputed from A and Bm (root check
    on) or fixed from the checksums. Columns of a block past the region
    stay exact products (they are masked later)."""
    S, R = A.shape[0], p.block_rows
    s = A @ Bm.T
    for (fb, fh, fr, fc, val, *mode) in run.faults.get(op, ()):
        if fb == b and fh == h and (not p.causal or fc // R <= fr // R):
            if mode and mode[0] == "flip":
                s[fr, fc] = flip_exponent_msb(float(round_to(s[fr, fc], "f32")), "f32")
            else:
                s[fr, fc] = round_to(np.array([val]), "f32")[0]
    if not run.on("BWD"):   # checks of the backward's recomputation
        return s
    for kb in range(S // R):
        r0 = kb * R if p.causal else 0
        seg = s[r0:, kb * R:(kb + 1) * R]
        cs = A[r0:] @ Bc[kb].T                                     # [rows, 2]
        rec = (lambda i, j, r0=r0, kb=kb: A[r0 + i] @ Bm[kb * R + j]) if recompute_ok else None
        evs, unc = _check_rows(seg, cs[:, 0], cs[:, 1], p.e_rel_value(), tn, rec, p.t_correct,
                               store=lambda x: float(round_to(np.array([x]), "f32")[0]))
        s[r0:, kb * R:(kb + 1) * R] = seg
        for (i, j, kind, action) in evs:
            run.events.append((op, b, h, r0 + i, kb * R + j, kind, action))
        for i in unc:
            run.events.append((op, b, h, r0 + i, kb * R, "-", "UNCORRECTABLE"))
    return s


def _checked_scores_cols(run, p, op, b, h, A, Bm, Ac, tn, recompute_ok):
    """S = A Bm^T (fp64, not rounded), the faults of op applied to the fp32
    value, and the column check of every (R-row block, column) vector
    against (Ac_qb) Bm^T (Sec. 4.4's AS^c form; Ac the column checksums of
    A per R-row block; EEC of Sec. 4.2) over the block-lower-triangular
    region at R granularity (all of it without the mask): a located
    element is recomputed from A and Bm (root check on) or fixed from the
    checksums."""
    S, R = A.shape[0], p.block_rows
    s = A @ Bm.T
    for (fb, fh, fr, fc, val, *mode) in run.faults.get(op, ()):
        if fb == b and fh == h and (not p.causal or fc // R <= fr // R):
            if mode and mode[0] == "flip":
                s[fr, fc] = flip_exponent_msb(float(round_to(s[fr, fc], "f32")), "f32")
            else:
                s[fr, fc] = round_to(np.array([val]), "f32")[0]
    if not run.on("BWD"):
        return s
    for qb in range(S // R):
        c_end = (qb + 1) * R if p.causal else S
        seg = s[qb * R:(qb + 1) * R, :c_end].T.copy()              # one vector per column
        cs = Ac[qb] @ Bm[:c_end].T                                 # [2, columns]
        rec = (lambda j, i, qb=qb: A[qb * R + i] @ Bm[j]) if recompute_ok else None
        evs, unc = _check_rows(seg, cs[0], cs[1], p.e_rel_value(), tn, rec, p.t_correct,
                               store=lambda x: float(round_to(np.array([x]), "f32")[0]))
        s[qb * R:(qb + 1) * R, :c_end] = seg.T
        for (j, i, kind, action) in evs:
            run.events.append((op, b, h, qb * R + i, j, kind, action))
        for j in unc:
            run.events.append((op, b, h, qb * R, j, "-", "UNCORRECTABLE"))
    return s


def _checked_output(run, p, op, b, h, M, cs, tn):
    """The faults of op applied to the stored output M [rows, d] of one
    head, then each row checked against its checksums cs [rows, 2]
    (unweighted, and weighted 1..d over the head's dims); a located element
    is fixed from the checksum (DELTA / RECONSTRUCT, Sec. 4.2)."""
    rnd = run.rnd
    for (fb, fh, fr, fc, val, *mode) in run.faults.get(op, ()):
        if fb == b and fh == h:
            M[fr, fc] = (flip_exponent_msb(float(M[fr, fc]), p.dtype)
                         if mode and mode[0] == "flip" else rnd(np.array([val]))[0])
    if run.on("BWD"):
        evs, unc = _check_rows(M, cs[:, 0], cs[:, 1], p.e_rel_value(), tn, None, p.t_correct,
                               store=lambda x: float(rnd(np.array([x]))[0]))
        for (i, j, kind, action) in evs:
            run.events.append((op, b, h, i, j, kind, action))
        for i in unc:
            run.events.append((op, b, h, i, 0, "-", "UNCORRECTABLE"))
    return M


def fused_backward_core(run, ctx, p):
    """The fused backward of the attention core (an extension: the
    backward without storing the scores, with Sec. 4.4's checks carried
    over), per (batch, head), from the forward's softmax statistics m, l,
    in two passes that each recompute the scores.
    Key pass (dK and dV, a key's gradients summed over the queries):
      1. S = Q K^T, AS faults applied, every (R-query block, key) column
         checked against (Q^c) K^T (Q^c propagated from X^c W^Q);
      2. P = exp(scale S - m) / l rounded to storage (0 on masked pairs);
      3. dP = dCL V^T (not rounded), dAP faults applied, columns checked
         against (dCL^c) V^T (dCL^c propagated from dO^c W^O^T);
      4. D = sum over the head's dims of dCL * CL (the softmax backward's
         row term: sum_j P_ij dP_ij = dCL_i . CL_i);
      5. dS = scale P (dP - D) rounded (0 on masked pairs);
      6. dV = P^T dCL rounded, dV faults applied, each row checked against
         P^T dCL^r, dCL^r the row checksums of the stored dCL over the
         head's dims (weights 1..d); dK = dS^T Q rounded, dK faults, rows
         checked against dS^T Q^r (Q^r likewise from the stored Q); a
         located element is fixed from the checksum (DELTA / RECONSTRUCT).
    Query pass (dQ, a query's gradient summed over the keys):
      7. S recomputed, AS faults applied, every (query, R-key block) row
         checked against Q (K^c)^T; P as in 2;
      8. dP recomputed, dAP faults applied, rows checked against
         dCL (V^c)^T; D and dS as in 4-5;
      9. dQ = dS K rounded, dQ faults applied, rows checked against dS K^r.
    A fault of AS or dAP thus reaches both passes and is located in each.
    S and dP are compared with the near-INF threshold as fp32 values, the
    gradients as stored. dQ^c, dK^c and dV^c, the column checksums per
    R-row block that dX's check takes, are encoded from the verified
    gradients."""
    B, S, nh, d, R, nq, scale = (ctx[k] for k in ("B", "S", "nh", "d", "R", "nq", "scale"))
    rnd = run.rnd
    tn_s = stored_threshold(p.t_near_inf, "f32")
    tn = stored_threshold(p.t_near_inf, p.dtype)
    allowed = np.tril(np.ones((S, S), dtype=bool)) if p.causal else np.ones((S, S), dtype=bool)
    out = {k: np.zeros((B, nh, S, d)) for k in ("dQ", "dK", "dV")}

    def probs(s, b, h):
        with np.errstate(over="ignore", invalid="ignore"):
            return rnd(np.where(allowed, np.exp(scale * s - ctx["m"][b, h][:, None])
                                / ctx["l"][b, h][:, None], 0.0))

    def grads(P, dP, D):
        with np.errstate(over="ignore", invalid="ignore"):
            return rnd(np.where(allowed, scale * P * (dP - D[:, None]), 0.0))

    for b in range(B):
        for h in range(nh):
            Q, K, V = ctx["Qh"][b, h], ctx["Kh"][b, h], ctx["Vh"][b, h]
            dCL, CL = ctx["dCLh"][b, h], ctx["CLh"][b, h]
            D = (dCL * CL).sum(axis=1)
            # key pass
            s = _checked_scores_cols(run, p, "AS", b, h, Q, K, ctx["Qch"][b, h], tn_s,
                                     p.root_check)
            P = probs(s, b, h)
            dP = _checked_scores_cols(run, p, "dAP", b, h, dCL, V, ctx["dCLch"][b, h], tn_s,
                                      p.root_check)
            dS = grads(P, dP, D)
            dCLr = row_checksums(dCL, d)[:, 0, :]                      # [S, 2]
            Qr = row_checksums(Q, d)[:, 0, :]
            out["dV"][b, h] = _checked_output(run, p, "dV", b, h,
                                              rnd(masked_cols_product(P, dCL, p.causal)),
                                              masked_cols_product(P, dCLr, p.causal), tn)
            out["dK"][b, h] = _checked_output(run, p, "dK", b, h,
                                              rnd(masked_cols_product(dS, Q, p.causal)),
                                              masked_cols_product(dS, Qr, p.causal), tn)
            # query pass
            s = _checked_scores(run, p, "AS", b, h, Q, K, ctx["Kch"][b, h], tn_s, p.root_check)
            P = probs(s, b, h)
            dP = _checked_scores(run, p, "dAP", b, h, dCL, V, ctx["Vch"][b, h], tn_s,
                                 p.root_check)
            dS = grads(P, dP, D)
            Kr = row_checksums(K, d)[:, 0, :]
            out["dQ"][b, h] = _checked_output(run, p, "dQ", b, h,
                                              rnd(masked_rows_product(dS, K, p.causal)),
                                              masked_rows_product(dS, Kr, p.causal), tn)
    return dict(dQ=out["dQ"], dK=out["dK"], dV=out["dV"], dQc=col_checksums(out["dQ"], R),
                dKc=col_checksums(out["dK"], R), dVc=col_checksums(out["dV"], R))


def fused_training_backward(fwd: dict, dO, p: OracleParams, faults=()):
    """The layer's protected backward after a fused forward, with the
    fused backward core in place of the steps from dCL to dQ, dK and dV."""
    return backward(fwd, dO, p, faults, core=fused_backward_core)
