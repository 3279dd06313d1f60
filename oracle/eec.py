"""Checksum encoding and EEC-ABFT (oracle; test infrastructure).

Checksums (Sec. 2.3): for a vector v of length n the unweighted checksum is
sum_k v_k and the weighted one sum_k k * v_k with 1-based weights k = 1..n.
A column checksum of a matrix M over an R-row block holds both sums of each
column inside the block; a row checksum over a C-column block holds both
sums of each row inside the block. The checksum block is a parameter (the
paper encodes whole per-(batch, head) matrices; R = rows is that case).

EEC-ABFT (Sec. 4.2, Fig. 3) on one vector v with propagated checksums c1, c2:
  d1 = c1 - sum v, d2 = c2 - sum k v.  Detection: d1 non-finite or |d1| > E.
  Case 1 (d1 finite): count near-INF elements; one -> that element (its
         position must agree with round(d2/d1) when d2 is finite); none ->
         classic ratio location round(d2/d1).
  Case 2 (d1 = +-INF): candidates are INF or near-INF elements.
  Case 3 (d1 = NaN): candidates are NaN, INF or near-INF elements.
  Case 4: two or more candidates -> the error has propagated along this
         vector; no correction here (handled by the other side, Sec. 4.3).
Mixed-type rule (Sec. 4.3): the candidate set of Cases 2 and 3 counts every
class a transition could have produced.

Correction by checksum (Sec. 4.2): |d1| <= T_correct -> v_i += d1 (DELTA);
otherwise v_i = c1 - sum_{k != i} v_k (RECONSTRUCT), which avoids the
absorption of small neighbours into a large d1.
"""
from __future__ import annotations

import dataclasses
from collections import defaultdict

import numpy as np

from .numerics import round_to, classify

E_FLOOR = 1e-30


def col_checksums(M: np.ndarray, R: int) -> np.ndarray:
    """[..., rows, cols] -> [..., rows/R, 2, cols]: unweighted and weighted
    (weights 1..R) sums of every column inside each R-row block."""
    *lead, rows, cols = M.shape
    if rows % R:
        raise ValueError("rows must be a multiple of the checksum block")
    Mb = M.reshape(*lead, rows // R, R, cols)
    w = np.arange(1, R + 1, dtype=np.float64)
    with np.errstate(invalid="ignore", over="ignore"):
        c1 = Mb.sum(axis=-2)
        c2 = np.tensordot(Mb, w, axes=([-2], [0]))
    return np.stack([c1, c2], axis=-2)


def row_checksums(M: np.ndarray, C: int) -> np.ndarray:
    """[..., rows, cols] -> [..., rows, cols/C, 2]: unweighted and weighted
    sums of every row inside each C-column block."""
    *lead, rows, cols = M.shape
    if cols % C:
        raise ValueError("cols must be a multiple of the checksum block")
    Mb = M.reshape(*lead, rows, cols // C, C)
    w = np.arange(1, C + 1, dtype=np.float64)
    with np.errstate(invalid="ignore", over="ignore"):
        c1 = Mb.sum(axis=-1)
        c2 = Mb @ w
    return np.stack([c1, c2], axis=-1)


@dataclasses.dataclass
class EECResult:
    status: str          # "clean" | "located" | "propagated"
    index: int = -1      # 0-based position inside the vector when located
    case: int = 0        # 1..4 as in Sec. 4.2 (0 when clean)
    d1: float = 0.0
    d2: float = 0.0


def detection_bound(v: np.ndarray, e_rel: float) -> float:
    """Roundoff bound E (Sec. 2.3 leaves its value open): e_rel times the sum
    of magnitudes of the finite elements, plus a tiny floor."""
    fin = np.isfinite(v)
    return e_rel * float(np.abs(v[fin]).sum()) + E_FLOOR


def eec_locate(v: np.ndarray, c1: float, c2: float, e_rel: float,
               t_near_inf: float) -> EECResult:
    """EEC-ABFT detection and location on one vector (Sec. 4.2 Cases 1-4,
    Sec. 4.3 mixed types). `t_near_inf` is the threshold as stored."""
    v = np.asarray(v, dtype=np.float64)
    n = v.shape[0]
    w = np.arange(1, n + 1, dtype=np.float64)
    with np.errstate(invalid="ignore", over="ignore"):
        d1 = c1 - v.sum()
        d2 = c2 - (w * v).sum()
    E = detection_bound(v, e_rel)
    if np.isfinite(d1) and abs(d1) <= E:
        return EECResult("clean", d1=d1, d2=d2)
    fin = np.isfinite(v)
    near = fin & (np.abs(np.where(fin, v, 0.0)) >= t_near_inf)
    if np.isfinite(d1):
        cand, case = near, 1
    elif np.isinf(d1):
        cand, case = np.isinf(v) | near, 2
    else:
        cand, case = ~fin | near, 3
    idx = np.flatnonzero(cand)
    if idx.size >= 2:
        return EECResult("propagated", case=4, d1=d1, d2=d2)
    if case == 1:
        if idx.size == 1:
            i = int(idx[0])
            if np.isfinite(d2):
                q = d2 / d1
                if not abs(q - (i + 1)) < 0.25:
                    return EECResult("propagated", case=4, d1=d1, d2=d2)
            return EECResult("located", index=i, case=1, d1=d1, d2=d2)
        if not np.isfinite(d2):
            return EECResult("propagated", case=4, d1=d1, d2=d2)
        q = d2 / d1
        i = int(np.rint(q))
        if 1 <= i <= n and abs(q - i) < 0.25:
            return EECResult("located", index=i - 1, case=1, d1=d1, d2=d2)
        return EECResult("propagated", case=4, d1=d1, d2=d2)
    if idx.size == 1:
        return EECResult("located", index=int(idx[0]), case=case, d1=d1, d2=d2)
    # A non-finite difference with no extreme element means the checksum
    # itself is corrupted; nothing in the vector can be blamed.
    return EECResult("propagated", case=4, d1=d1, d2=d2)


def fix_by_checksum(v: np.ndarray, i: int, c1: float, d1: float,
                    t_correct: float):
    """Correct element i from the checksum only (Sec. 4.2 correction, with
    the T_correct switch). Returns (new value before storage rounding,
    action)."""
    if np.isfinite(d1) and abs(d1) <= t_correct:
        return float(v[i] + d1), "DELTA"
    others = np.delete(np.asarray(v, dtype=np.float64), i)
    return float(c1 - others.sum()), "RECONSTRUCT"


class Verifier:
    """The verification procedure applied to one protected GEMM output.

    C has shape [n, rows, cols] (n flattens batch and head). Cc holds the
    propagated column checksums [n, rows/R, 2, cols]; Cr, when the output is
    protected on both sides (AS and CL, Sec. 4.4), holds the propagated row
    checksums [n, rows, cols/Cb, 2].

    Procedure (Sec. 4.3, nondeterministic patterns):
      1. column pass: EEC on every flagged column vector; correct located
         elements; a propagated vector is left for the row pass;
      2. (two-sided only) recompute the row checksum of every row vector in
         which step 1 corrected two or more elements (a 1R propagation, whose
         row checksum came from the same corrupted operand row); row pass;
         recompute the column checksum of every column vector in which the
         row pass corrected two or more elements (1C: the paper's
         re-computation of the corrupted column checksums). A single (0D)
         correction leaves the other side's checksum alone, so the second
         pass re-checks it;
      3. final check of every vector on both sides: whatever is still
         flagged is reported UNCORRECTABLE (2-D, Sec. 4.3 limits EEC to 1-D).

    Correction: with `recompute` given (operands known clean), a located
    element is recomputed from its operands (action RECOMPUTE); otherwise
    the checksum formulas of Sec. 4.2 are used (DELTA / RECONSTRUCT).
    """

    def __init__(self, dtype: str, e_rel: float, t_near_inf_stored: float,
                 t_correct: float):
        self.dtype = dtype
        self.e_rel = e_rel
        self.tn = t_near_inf_stored
        self.tc = t_correct

    # -- vectorised detection over all vectors of one side ---------------
    def _flag_cols(self, C, Cc, R, valid):
        n, rows, cols = C.shape
        Cb = C.reshape(n, rows // R, R, cols)
        with np.errstate(invalid="ignore", over="ignore"):
            r1 = Cb.sum(axis=2)
            d1 = Cc[:, :, 0, :] - r1
        absum = np.where(np.isfinite(Cb), np.abs(np.nan_to_num(Cb)), 0.0).sum(axis=2)
        E = self.e_rel * absum + E_FLOOR
        flag = ~(np.isfinite(d1) & (np.abs(np.nan_to_num(d1)) <= E))
        if valid is not None:
            flag &= valid
        return flag

    def _flag_rows(self, C, Cr, Cb_, valid):
        n, rows, cols = C.shape
        Mb = C.reshape(n, rows, cols // Cb_, Cb_)
        with np.errstate(invalid="ignore", over="ignore"):
            r1 = Mb.sum(axis=3)
            d1 = Cr[:, :, :, 0] - r1
        absum = np.where(np.isfinite(Mb), np.abs(np.nan_to_num(Mb)), 0.0).sum(axis=3)
        E = self.e_rel * absum + E_FLOOR
        flag = ~(np.isfinite(d1) & (np.abs(np.nan_to_num(d1)) <= E))
        if valid is not None:
            flag &= valid
        return flag

    def _correct(self, C, v, k, i, j, res, recompute, events, where):
        old = float(C[k, i, j])
        if recompute is not None:
            new, action = recompute(k, i, j), "RECOMPUTE"
        else:
            new, action = fix_by_checksum(v, res.index, *where, self.tc)
        C[k, i, j] = round_to(np.array([new]), self.dtype)[0]
        events.append((k, i, j, classify(old, self.tn), action))

    def run(self, C, Cc, R, *, Cr=None, Cb=None, col_valid=None,
            row_valid=None, recompute=None):
        """Verify and correct C in place. Returns (events, uncorrectable)
        where events are (k, row, col, kind, action) of corrected elements
        and uncorrectable lists ("col", k, block, col) / ("row", k, row,
        block) vectors left inconsistent."""
        events = []
        n, rows, cols = C.shape
        col_fixed = set()
        # 1. column pass
        for k, blk, j in zip(*np.nonzero(self._flag_cols(C, Cc, R, col_valid))):
            v = C[k, blk * R:(blk + 1) * R, j].copy()
            res = eec_locate(v, Cc[k, blk, 0, j], Cc[k, blk, 1, j], self.e_rel, self.tn)
            if res.status == "located":
                i = blk * R + res.index
                self._correct(C, v, k, i, j, res, recompute, events,
                              (Cc[k, blk, 0, j], res.d1))
                col_fixed.add((k, i, j))
        if Cr is not None:
            # 2a. refresh the row checksums of 1R-corrected row vectors
            per_row = defaultdict(int)
            for (k, i, j) in col_fixed:
                per_row[(k, i, j // Cb)] += 1
            for (k, i, cb), cnt in per_row.items():
                if cnt >= 2:
                    seg = C[k, i, cb * Cb:(cb + 1) * Cb]
                    Cr[k, i, cb] = row_checksums(seg[None, :], Cb)[0, 0]
            # 2b. row pass
            row_fixed = set()
            for k, i, cb in zip(*np.nonzero(self._flag_rows(C, Cr, Cb, row_valid))):
                v = C[k, i, cb * Cb:(cb + 1) * Cb].copy()
                res = eec_locate(v, Cr[k, i, cb, 0], Cr[k, i, cb, 1], self.e_rel, self.tn)
                if res.status == "located":
                    j = cb * Cb + res.index
                    self._correct(C, v, k, i, j, res, recompute, events,
                                  (Cr[k, i, cb, 0], res.d1))
                    row_fixed.add((k, i, j))
            # 2c. refresh the column checksums of 1C-corrected column vectors
            per_col = defaultdict(int)
            for (k, i, j) in row_fixed:
                per_col[(k, i // R, j)] += 1
            for (k, blk, j), cnt in per_col.items():
                if cnt >= 2:
                    seg = C[k, blk * R:(blk + 1) * R, j]
                    Cc[k, blk, :, j] = col_checksums(seg[:, None], R)[0, :, 0]
        # 3. final check
        unc = [("col", int(k), int(b), int(j)) for k, b, j in
               zip(*np.nonzero(self._flag_cols(C, Cc, R, col_valid)))]
        if Cr is not None:
            unc += [("row", int(k), int(i), int(cb)) for k, i, cb in
                    zip(*np.nonzero(self._flag_rows(C, Cr, Cb, row_valid)))]
        return events, unc
