"""Fused protected attention, forward (oracle; test infrastructure).

The score, softmax and context steps of the layer (Sec. 2.1 Eq. 1-2) with
the S_AS and S_CL protections of Sec. 4.4, computed per query tile without
storing the score matrix AS or the probabilities AP: an online-softmax
(flash-style) form, which is an extension; the paper materialises both.
The projection before and the output projection after are the layer's
(`layer.project`, `layer.output_projection`).

Per (batch, head), query tile of TQ = 128 queries and key tile of TK = 128
keys, key tiles in increasing order (causal: key tiles up to the diagonal):
  1. S = Q_t K_j^T, not rounded (it is never stored); AS faults are
     applied to S ("set" writes the value, "flip" flips the exponent MSB of
     S as an fp32 value).
  2. Row check of S (Sec. 4.4 AS^r = Q (K^c)^T, one vector per query and
     R-key block; EEC of Sec. 4.2): a located element is recomputed from Q
     and K (root check on: the operands are clean) or fixed from the
     checksums (root check off). The column side (AS^c) is not checked
     here: with the root check a 1R pattern in AS (a Q error, Sec. 4.3)
     cannot arise, and 0D and 1C patterns are located by the rows.
  3. Online softmax: m' = max(m, max_j scale S_ij) over unmasked keys,
     p = exp(scale S - m') (masked: 0), alpha = exp(m - m'),
     l = alpha l + sum_j p, P = storage-rounded p,
     A = alpha A + P V_j, A^r = alpha A^r + P V^r_j.
  4. After the last key tile: CL = rounded A / l; CL faults are applied;
     CL^r = A^r / l is the propagated row checksum of CL (V^r = X W^V r,
     Sec. 4.4; the rescaling multiplies A and A^r alike). Row check of CL
     (one vector per query over the head's d columns); a located element
     is fixed from the checksum (DELTA / RECONSTRUCT, Sec. 4.2).
  5. CL^c, needed by the output projection, is encoded from the verified
     CL (column checksums per R-query block).
For the backward (the materialised chain of the layer), the softmax
statistics of every query (the final max m and sum l of step 3) are kept,
and AP is regenerated from Q, K and them: AP = storage-rounded
exp(scale Q K^T - m) / l on the unmasked pairs (0 on masked ones), with its
row checksums AP^r encoded from the stored values; CL^r = A^r / l is the
propagated row checksum of CL the backward's dW^O check takes.

Rounding: S and the accumulators are kept unrounded (fp64 here, fp32 on
the GPU); P is rounded to the storage dtype (it feeds the P V product);
CL is rounded when stored. The near-INF threshold compares against S as
an fp32 value and against CL as stored.
"""
from __future__ import annotations

import numpy as np

from .eec import col_checksums, eec_locate, fix_by_checksum, row_checksums
from .layer import OracleParams, _Run, project, output_projection
from .numerics import classify, flip_exponent_msb, round_to, stored_threshold

TQ = 128
TK = 128


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


def fused_attention(run: _Run, pr: dict, p: OracleParams, only=None, stats=None):
    """Steps 1-5 for every (batch, head), or for the (batch, head) pairs in
    `only` (the others' CL stays zero). Returns CL [B,S,H] and CL^c
    [B,nq,2,H]; events go to run.events. With a dict `stats`, also stores
    there the final max m and sum l of every query ([B,nh,S], natural
    units) and CL^r = A^r / l ([B,S,nh,2])."""
    B, S, H, nh, d, R, nq, scale = (pr[k] for k in ("B", "S", "H", "nh", "d", "R", "nq", "scale"))
    Qh, Kh, Vh, Kch, Vr = pr["Qh"], pr["Kh"], pr["Vh"], pr["Kch"], pr["Vr"]
    if S % TQ or R > TK or TK % R:
        raise ValueError("the fused form takes seq in whole 128-row tiles and R dividing 128")
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
    for b in range(B):
        for h in range(nh):
            if only is not None and (b, h) not in only:
                continue
            Q, K, V = Qh[b, h], Kh[b, h], Vh[b, h]
            Kc = Kch[b, h]                      # [nq, 2, d]
            vr = Vr[b, :, h, :]                 # [S, 2]
            for qt in range(S // TQ):
                q0 = qt * TQ
                rows = np.arange(q0, q0 + TQ)
                m = np.full(TQ, -np.inf)
                l = np.zeros(TQ)
                A = np.zeros((TQ, d))
                Ar = np.zeros((TQ, 2))
                last = qt if p.causal else S // TK - 1
                for kt in range(last + 1):
                    k0 = kt * TK
                    s = Q[q0:q0 + TQ] @ K[k0:k0 + TK].T                # 1.
                    for (fb, fh, fr, fc, val, *mode) in faults_as:
                        if fb == b and fh == h and q0 <= fr < q0 + TQ and k0 <= fc < k0 + TK:
                            i, j = fr - q0, fc - k0
                            if mode and mode[0] == "flip":
                                s[i, j] = flip_exponent_msb(float(round_to(s[i, j], "f32")), "f32")
                            else:
                                s[i, j] = round_to(np.array([val]), "f32")[0]
                    if check_as:                                        # 2.
                        for kb in range(TK // R):
                            blk = (k0 + kb * R) // R
                            cs = Q[q0:q0 + TQ] @ Kc[blk].T             # [TQ, 2]
                            seg = s[:, kb * R:(kb + 1) * R]
                            rec = ((lambda i, j, kb=kb: Q[q0 + i] @ K[k0 + kb * R + j])
                                   if recompute_ok else None)
                            evs, unc = _check_rows(seg, cs[:, 0], cs[:, 1], e_rel, tn_s, rec,
                                                   p.t_correct,
                                                   store=lambda x: float(round_to(np.array([x]), "f32")[0]))
                            s[:, kb * R:(kb + 1) * R] = seg
                            for (i, j, kind, action) in evs:
                                run.events.append(("AS", b, h, q0 + i, k0 + kb * R + j, kind, action))
                            for i in unc:
                                run.events.append(("AS", b, h, q0 + i, k0 + kb * R, "-", "UNCORRECTABLE"))
                    keys = np.arange(k0, k0 + TK)                       # 3.
                    allowed = (keys[None, :] <= rows[:, None]) if p.causal else np.ones((TQ, TK), bool)
                    with np.errstate(invalid="ignore", over="ignore"):
                        z = np.where(allowed, scale * s, -np.inf)
                        m_new = np.maximum(m, z.max(axis=1))
                        pz = np.where(allowed, np.exp(z - m_new[:, None]), 0.0)
                        alpha = np.where(np.isfinite(m), np.exp(m - m_new), 0.0)
                    l = alpha * l + pz.sum(axis=1)
                    P = run.rnd(pz)
                    A = alpha[:, None] * A + P @ V[k0:k0 + TK]
                    Ar = alpha[:, None] * Ar + P @ vr[k0:k0 + TK]
                    m = m_new
                CLt = run.rnd(A / l[:, None])                           # 4.
                CLr = Ar / l[:, None]
                M_all[b, h, q0:q0 + TQ], L_all[b, h, q0:q0 + TQ] = m, l
                CLr_all[b, q0:q0 + TQ, h] = CLr
                for (fb, fh, fr, fc, val, *mode) in faults_cl:
                    if fb == b and fh == h and q0 <= fr < q0 + TQ:
                        i = fr - q0
                        if mode and mode[0] == "flip":
                            CLt[i, fc] = flip_exponent_msb(float(CLt[i, fc]), p.dtype)
                        else:
                            CLt[i, fc] = run.rnd(np.array([val]))[0]
                if check_cl:
                    evs, unc = _check_rows(CLt, CLr[:, 0], CLr[:, 1], e_rel, tn_cl, None,
                                           p.t_correct,
                                           store=lambda x: float(run.rnd(np.array([x]))[0]))
                    for (i, j, kind, action) in evs:
                        run.events.append(("CL", b, h, q0 + i, j, kind, action))
                    for i in unc:
                        run.events.append(("CL", b, h, q0 + i, 0, "-", "UNCORRECTABLE"))
                CLh[b, h, q0:q0 + TQ] = CLt
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


def fused_forward(X, Wqkv, Wo, p: OracleParams, faults=()):
    """Protected forward of one attention layer with the fused attention
    core. Returns O, CL, its checksums, the projection outputs and the
    event list."""
    run = _Run(p, faults)
    pr = project(run, X, Wqkv, p)
    st = {}
    CL, CLc = fused_attention(run, pr, p, stats=st)
    Wo = np.asarray(Wo, dtype=np.float64)
    O, Oc = output_projection(run, CL, CLc, Wo, p)
    AP, APr = regenerate_ap(run, pr, p, st["m"], st["l"])
    # the dict carries what the layer's backward takes from a forward
    return dict(O=O, CL=CL, CLc=CLc, Oc=Oc, QKV=pr["QKV"], QKVc=pr["QKVc"], Vr=pr["Vr"],
                X=pr["X"], Wqkv=pr["Wqkv"], Wo=Wo, Xc=pr["Xc"], Xr=pr["Xr"], AP=AP, APr=APr,
                CLr=st["CLr"], m=st["m"], l=st["l"], scale=pr["scale"], events=run.events,
                params=p)
