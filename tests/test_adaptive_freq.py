"""Parity of the library's adaptive-frequency calls (host code behind the C
ABI: attn_abft_unsafe_probability, attn_abft_optimize_frequencies,
attn_abft_sections_for_step) with the oracle of Sec. 4.5 / Algorithm 1.
No GPU is needed: these calls touch no device memory."""
import math

import pytest

from oracle import freq as F


def _abft():
    from paper_2410_11720_amd import abft
    return abft


def to_abi(secs):
    return [(s.cost, [(op.flops, tuple(op.p[e] for e in F.TYPES)) for op in s.ops]) for s in secs]


def lam3(L):
    return [L[e] for e in F.TYPES]


CASES = [
    # (shape, model, costs, lambda per type, target as a fraction of the range)
    ((8, 1024, 768, 12, True), "GPT-2", (100.0, 60.0, 25.0), (1e-21, 1e-21, 1e-21), 0.35),
    ((8, 1024, 768, 12, True), "GPT-2", (100.0, 60.0, 25.0), (15e-25, 15e-25, 15e-25), 0.35),
    ((8, 512, 768, 12, False), "Bert", (40.0, 90.0, 10.0), (2e-21, 5e-22, 3e-21), 0.8),
    ((4, 2048, 4096, 32, True), "Neo", (900.0, 400.0, 120.0), (3e-22, 3e-22, 3e-22), 0.1),
    ((1, 4096, 5120, 40, True), "Roberta", (700.0, 700.0, 100.0), (1e-22, 4e-22, 2e-22), 0.5),
]


@pytest.mark.parametrize("shape,model,costs,lam,frac", CASES)
def test_optimizer_matches_oracle(shape, model, costs, lam, frac):
    abft = _abft()
    secs = F.layer_sections(*shape, model, {"AS": costs[0], "CL": costs[1], "O": costs[2]})
    L = dict(zip(F.TYPES, lam))
    u0, u1 = F.unsafe_att(secs, L, [0] * 3), F.unsafe_att(secs, L, [1] * 3)
    for target in (u1 + frac * (u0 - u1), 1e-11, u1 * 0.5, u0 * 2):
        want = F.optimize(secs, L, target)
        got = abft.attn_abft_optimize_frequencies(to_abi(secs), lam3(L), target)
        assert len(got) == 3
        for a, b in zip(got, want):
            assert math.isclose(a, b, rel_tol=1e-12, abs_tol=1e-15), (target, got, want)


@pytest.mark.parametrize("shape,model,costs,lam,frac", CASES)
def test_failure_probability_matches_oracle(shape, model, costs, lam, frac):
    abft = _abft()
    secs = F.layer_sections(*shape, model, {"AS": costs[0], "CL": costs[1], "O": costs[2]})
    L = dict(zip(F.TYPES, lam))
    for fr in ([0, 0, 0], [1, 1, 1], [0.25, 0.5, 0.75], [1, 0, 0.3]):
        want = F.unsafe_att(secs, L, fr)
        got = abft.attn_abft_unsafe_probability(to_abi(secs), lam3(L), fr)
        assert math.isclose(got, want, rel_tol=1e-12, abs_tol=1e-300)


def test_four_sections_including_a_backward_section():
    """The backward (an extension) as a fourth section whose unhandled
    errors are all taken as fatal."""
    abft = _abft()
    secs = F.layer_sections(8, 1024, 768, 12, True, "GPT-2", {"AS": 90.0, "CL": 50.0, "O": 30.0})
    bwd = F.Section("BWD", [F.Op("bwd", 2.0 * 5.8e10, {e: 1.0 for e in F.TYPES})], 250.0)
    secs.append(bwd)
    L = {e: 2e-21 for e in F.TYPES}
    u0, u1 = F.unsafe_att(secs, L, [0] * 4), F.unsafe_att(secs, L, [1] * 4)
    target = u1 + 0.4 * (u0 - u1)
    want = F.optimize(secs, L, target)
    got = abft.attn_abft_optimize_frequencies(to_abi(secs), lam3(L), target)
    assert all(math.isclose(a, b, rel_tol=1e-12, abs_tol=1e-15) for a, b in zip(got, want))


@pytest.mark.parametrize("freqs", [(0, 0, 0, 0), (1, 1, 1, 1), (0.5, 0.25, 1 / 3, 0.9),
                                   (0.01, 0.999, 0.125, 0.0)])
def test_step_masks_match_oracle_schedule(freqs):
    abft = _abft()
    bits = (abft.SEC_AS, abft.SEC_CL, abft.SEC_O, abft.SEC_BWD)
    for k in range(400):
        want = sum(b for b, f in zip(bits, freqs) if F.schedule(f, k))
        assert abft.attn_abft_sections_for_step(list(freqs), k) == want, (k, freqs)


def test_invalid_arguments_are_rejected():
    abft = _abft()
    good = [(10.0, [(1e9, (0.5, 0.5, 0.5))])]
    with pytest.raises(abft.AbftError):
        abft.attn_abft_optimize_frequencies([(10.0, [(1e9, (1.5, 0.5, 0.5))])], [1e-20] * 3, 1e-11)
    with pytest.raises(abft.AbftError):
        abft.attn_abft_optimize_frequencies(good, [-1e-20, 0, 0], 1e-11)
    with pytest.raises(abft.AbftError):
        abft.attn_abft_optimize_frequencies([], [1e-20] * 3, 1e-11)
    with pytest.raises(abft.AbftError):
        abft.attn_abft_unsafe_probability(good, [1e-20] * 3, [1.2])
    assert abft.attn_abft_sections_for_step([0.5] * 4, -1) == 0


@pytest.mark.parametrize("free", [0, 1, 2])
def test_free_section_matches_oracle_and_meets_the_target(free):
    abft = _abft()
    costs = [100.0, 60.0, 25.0]
    costs[free] = 0.0
    secs = F.layer_sections(8, 1024, 768, 12, True, "GPT-2",
                            {"AS": costs[0], "CL": costs[1], "O": costs[2]})
    L = {e: 1e-21 for e in F.TYPES}
    u0, u1 = F.unsafe_att(secs, L, [0] * 3), F.unsafe_att(secs, L, [1] * 3)
    for target in (u1 + 0.3 * (u0 - u1), u1 + 0.9 * (u0 - u1), u0 * 2):
        got = abft.attn_abft_optimize_frequencies(to_abi(secs), lam3(L), target)
        want = F.optimize(secs, L, target)
        assert got[free] == 1.0
        for a, b in zip(got, want):
            assert math.isclose(a, b, rel_tol=1e-12, abs_tol=1e-15), (target, got, want)
        assert abft.attn_abft_unsafe_probability(to_abi(secs), lam3(L), got) <= target * (1 + 1e-9)
