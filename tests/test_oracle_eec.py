"""Pins of the oracle's checksums and EEC-ABFT.

Pins: brute-force integer arithmetic (the checksum identities of Sec. 2.3
hold exactly on small-integer matrices), the classic location rule
delta2/delta1 = i (Sec. 2.3), hand-built vectors for every EEC case of
Sec. 4.2 with the paper's constants, the absorption hazard that motivates
T_correct (Sec. 4.2), the failure of classic ABFT on INF (Sec. 2.3), and
the 1R / 1C / 2D handling of Sec. 4.3 on integer matrices.
"""
import numpy as np
import pytest

from oracle.eec import (col_checksums, row_checksums, eec_locate,
                        fix_by_checksum, Verifier)

TN = 9999220736.0   # bf16(1e10)
E_REL = 2.0 ** -5


def _int_mats(seed, m, k, n):
    rng = np.random.default_rng(seed)
    A = rng.integers(-4, 5, (m, k))
    B = rng.integers(-4, 5, (k, n))
    return A, B


def _brute_col(M, R):
    rows, cols = len(M), len(M[0])
    out = [[[0, 0] for _ in range(cols)] for _ in range(rows // R)]
    for blk in range(rows // R):
        for j in range(cols):
            for t in range(R):
                out[blk][j][0] += int(M[blk * R + t][j])
                out[blk][j][1] += (t + 1) * int(M[blk * R + t][j])
    return out


def test_col_checksums_brute_force():
    A, _ = _int_mats(1, 12, 5, 3)
    got = col_checksums(A.astype(np.float64), 4)
    ref = _brute_col(A.tolist(), 4)
    for blk in range(3):
        for j in range(5):
            assert got[blk, 0, j] == ref[blk][j][0]
            assert got[blk, 1, j] == ref[blk][j][1]


def test_row_checksums_brute_force():
    A, _ = _int_mats(2, 3, 12, 1)
    got = row_checksums(A.astype(np.float64), 6)
    for i in range(3):
        for cb in range(2):
            seg = [int(x) for x in A[i, cb * 6:(cb + 1) * 6]]
            assert got[i, cb, 0] == sum(seg)
            assert got[i, cb, 1] == sum((t + 1) * x for t, x in enumerate(seg))


def test_checksum_identities_exact_on_integers():
    # e^T (A B) = (e^T A) B and (A B) e = A (B e), unweighted and weighted,
    # per block: exact because every quantity is a small integer.
    A, B = _int_mats(3, 16, 7, 12)
    A = A.astype(np.float64)
    B = B.astype(np.float64)
    C = A @ B
    assert np.array_equal(col_checksums(C, 4), col_checksums(A, 4) @ B)
    Br = row_checksums(B, 6).reshape(7, 4)       # [k, blocks*2]
    assert np.array_equal(row_checksums(C, 6).reshape(16, 4), A @ Br)


def test_classic_location_is_exact_on_integers():
    A, B = _int_mats(4, 8, 6, 5)
    C = (A @ B).astype(np.float64)
    Cc = col_checksums(C, 8)
    for i in range(8):
        bad = C.copy()
        bad[i, 3] += 37.0
        res = eec_locate(bad[:, 3], Cc[0, 0, 3], Cc[0, 1, 3], E_REL, TN)
        assert res.status == "located" and res.index == i and res.case == 1
        assert res.d2 / res.d1 == i + 1
        new, action = fix_by_checksum(bad[:, 3], i, Cc[0, 0, 3], res.d1, 1e5)
        assert action == "DELTA" and new == C[i, 3]


def _vec(n=64, seed=0):
    return np.random.default_rng(seed).standard_normal(n)


def _chk(v):
    w = np.arange(1, len(v) + 1)
    return float(v.sum()), float((w * v).sum())


@pytest.mark.parametrize("value,case", [
    (np.inf, 2), (-np.inf, 2), (np.nan, 3), (1e10, 1), (-1e10, 1),
    (TN, 1), (1e30, 1), (1e6, 1), (-3e5, 1)])
def test_eec_single_extreme_located(value, case):
    v = _vec()
    c1, c2 = _chk(v)
    for i in (0, 17, 63):
        bad = v.copy()
        bad[i] = value
        res = eec_locate(bad, c1, c2, E_REL, TN)
        assert res.status == "located", (value, i, res)
        assert res.index == i and res.case == case


def test_eec_clean_vector_and_rounding_noise_are_clean():
    v = _vec()
    c1, c2 = _chk(v)
    assert eec_locate(v, c1, c2, E_REL, TN).status == "clean"
    # storage rounding to 8 significant bits stays below E
    from oracle.numerics import round_to
    assert eec_locate(round_to(v, "bf16"), c1, c2, E_REL, TN).status == "clean"


@pytest.mark.parametrize("vals", [
    (np.inf, -np.inf), (np.inf, np.inf), (np.nan, 1.0e10), (1e10, 2e10),
    (np.inf, 1e10), (np.nan, np.nan), (1e30, 1e30)])
def test_eec_two_extremes_is_case4(vals):
    v = _vec()
    c1, c2 = _chk(v)
    bad = v.copy()
    bad[3], bad[40] = vals
    res = eec_locate(bad, c1, c2, E_REL, TN)
    assert res.status == "propagated" and res.case == 4


def test_eec_weighted_difference_overflow_uses_the_extreme_element():
    # Only float64 can hold such values; d1 stays finite while the weighted
    # difference overflows, so the element must be found by its magnitude.
    v = _vec(128)
    c1, c2 = _chk(v)
    bad = v.copy()
    bad[100] = 1e307
    res = eec_locate(bad, c1, c2, E_REL, TN)
    assert np.isfinite(res.d1) and np.isinf(res.d2)
    assert res.status == "located" and res.index == 100 and res.case == 1


def test_eec_nonfinite_checksum_without_extreme_element_is_not_blamed_on_data():
    v = _vec()
    _, c2 = _chk(v)
    res = eec_locate(v, np.inf, c2, E_REL, TN)
    assert res.status == "propagated"


def test_classic_abft_fails_on_inf_but_eec_locates():
    v = _vec()
    c1, c2 = _chk(v)
    bad = v.copy()
    bad[9] = np.inf
    w = np.arange(1, 65)
    with np.errstate(invalid="ignore"):
        d1 = c1 - bad.sum()
        d2 = c2 - (w * bad).sum()
        classic = d2 / d1
    assert np.isnan(classic)          # INF/INF: the classic index is undefined
    res = eec_locate(bad, c1, c2, E_REL, TN)
    assert res.status == "located" and res.index == 9


def test_absorption_hazard_and_t_correct():
    # Small neighbours vanish next to a 1e30 error: delta-addition cannot
    # restore the true value, reconstruction from the checksum can.
    v = np.linspace(0.001, 0.064, 64)
    c1, c2 = _chk(v)
    bad = v.copy()
    bad[20] = 1e30
    res = eec_locate(bad, c1, c2, E_REL, TN)
    assert res.status == "located" and res.index == 20
    by_delta, _ = fix_by_checksum(bad, 20, c1, res.d1, t_correct=1e300)
    by_rule, action = fix_by_checksum(bad, 20, c1, res.d1, t_correct=1e5)
    assert action == "RECONSTRUCT"
    assert abs(by_delta - v[20]) > 1e-3
    assert abs(by_rule - v[20]) < 1e-12


def _verifier(dtype="f64"):
    return Verifier(dtype, 2.0 ** -40, 1e10, 1e5)


def _int_product(seed=5):
    rng = np.random.default_rng(seed)
    A = rng.integers(-3, 4, (8, 5)).astype(np.float64)
    B = rng.integers(-3, 4, (5, 8)).astype(np.float64)
    return A, B


def test_verifier_1R_from_row_operand_is_corrected_by_columns():
    A, B = _int_product()
    Ac, Br = col_checksums(A, 8), row_checksums(B, 8)
    C_true = A @ B
    Abad = A.copy()
    Abad[2, 1] = np.inf                         # 1R in C, row checksum corrupted too
    with np.errstate(invalid="ignore"):
        C = Abad @ B
        Cr = (Abad @ Br.reshape(5, 2)).reshape(8, 1, 2)
    Cc = Ac @ B
    evs, unc = _verifier().run(C[None], Cc[None], 8, Cr=Cr[None], Cb=8)
    assert unc == []
    # INF * 0 is NaN, so every element of row 2 is corrupted
    assert {(i, j) for (_, i, j, _, _) in evs} == {(2, j) for j in range(8)}
    assert np.array_equal(C, C_true)


def test_verifier_1C_from_column_operand_needs_the_row_pass():
    A, B = _int_product(6)
    Ac, Br = col_checksums(A, 8), row_checksums(B, 8)
    C_true = A @ B
    Bbad = B.copy()
    Bbad[3, 5] = np.inf                         # 1C in C, column checksum corrupted
    with np.errstate(invalid="ignore"):
        C = A @ Bbad
        Cc = Ac @ Bbad
    Cr = (A @ Br.reshape(5, 2)).reshape(8, 1, 2)
    evs, unc = _verifier().run(C[None], Cc[None], 8, Cr=Cr[None], Cb=8)
    assert unc == []
    assert {(i, j) for (_, i, j, _, _) in evs} == {(i, 5) for i in range(8)}
    assert np.array_equal(C, C_true)
    # the column checksum of the repaired column was recomputed
    assert np.array_equal(Cc[0, :, 5], col_checksums(C_true, 8)[0, :, 5])


def test_verifier_moderate_1C_false_negative_then_row_pass():
    A, B = _int_product(7)
    Ac, Br = col_checksums(A, 8), row_checksums(B, 8)
    C_true = A @ B
    Bbad = B.copy()
    Bbad[0, 2] += 50.0                          # moderate, column stays consistent
    C = A @ Bbad
    Cc = Ac @ Bbad
    Cr = (A @ Br.reshape(5, 2)).reshape(8, 1, 2)
    evs, unc = _verifier().run(C[None], Cc[None], 8, Cr=Cr[None], Cb=8)
    assert unc == []
    assert np.array_equal(C, C_true)


def test_verifier_l_shape_is_fully_corrected_and_2x2_block_is_uncorrectable():
    A, B = _int_product(8)
    C_true = A @ B
    Cc = col_checksums(C_true, 8)
    Cr = row_checksums(C_true, 8)
    C = C_true.copy()
    C[1, 1], C[1, 6], C[5, 1] = np.inf, np.nan, 1e12
    evs, unc = _verifier().run(C[None], Cc[None].copy(), 8, Cr=Cr[None].copy(), Cb=8)
    assert unc == [] and len(evs) == 3 and np.array_equal(C, C_true)
    C = C_true.copy()
    C[1, 1], C[1, 6], C[5, 1], C[5, 6] = np.inf, np.nan, 1e12, -np.inf
    evs, unc = _verifier().run(C[None], Cc[None].copy(), 8, Cr=Cr[None].copy(), Cb=8)
    assert evs == []
    assert sorted(unc) == sorted([("col", 0, 0, 1), ("col", 0, 0, 6),
                                  ("row", 0, 1, 0), ("row", 0, 5, 0)])


def test_verifier_recompute_restores_exactly():
    A, B = _int_product(9)
    C_true = A @ B
    Cc = col_checksums(C_true, 4)
    C = C_true.copy()
    C[6, 2] = -np.inf
    evs, unc = _verifier().run(C[None], Cc[None], 4,
                               recompute=lambda k, i, j: A[i] @ B[:, j])
    assert unc == [] and evs == [(0, 6, 2, "INF", "RECOMPUTE")]
    assert np.array_equal(C, C_true)
