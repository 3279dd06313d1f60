"""Adaptive ABFT detection frequencies (paper Sec. 4.5, Algorithm 1).

TEST INFRASTRUCTURE ONLY (see the package header).

Model. Errors of type e (INF, NaN, near-INF) strike an operation OP of
n_OP flops as a Poisson process of rate lambda_e per flop, so the chance of
k errors is P(k) = exp(-lambda n) (lambda n)^k / k!. A protection section
S = {OP_1..OP_m} survives when it sees no error (R_free) or exactly one
error (R_e(i): one error of type e in OP_i, none elsewhere), and that one
error is either handled (ABFT enabled, probability f_S) or, unhandled,
harmless: it leads to a non-trainable state with probability p_i^e (the
paper's Table 4). Two or more errors in a section count as failure. So

    FC_S(f) = R_free + sum_i sum_e R_e(i) * (f + (1 - f) * (1 - p_i^e))
    FC_att  = prod_S FC_S(f_S)

FC sits within ~1e-13 of 1 at real error rates while targets are ~1e-11
failures per execution, so everything here is computed as a failure
probability U = 1 - FC, from small terms, never as a difference of numbers
near 1:

    U_S(f) = P_S(>= 2 errors) + (1 - f) * sum_i sum_e R_e(i) p_i^e
    U_att  = 1 - prod_S (1 - U_S)

Readings (the printed formulas are inconsistent):
  * H_i^e. The text defines phi as the probability that an error leads to
    a non-trainable state and then writes H = f + (1 - f) phi for the
    probability that an error is handled or harmless; harmless is 1 - phi,
    so H = f + (1 - f)(1 - p) here.
  * FCE. FC_S is linear in f_S, so the coverage gained per unit of ABFT
    time is the constant FCE_S = (dFC_S/df_S) / T_S = sum R_e(i) p_i^e / T_S
    (the printed numerator's R_free term is not a derivative and is left
    out; its 1 - phi matches the printed H, with phi read as above).
  * Algorithm 1. Start from the coverage with every section off, then take
    the sections in descending FCE: all of T_S while the remaining deficit
    is at least FCE_S T_S, else the fraction that closes it, and nothing
    once the target is met. This is the greedy (fractional-knapsack)
    solution of the first-order expansion of FC_att; the cross terms of the
    product are O(U^2), far below the target's resolution.
  * A target that even full protection misses (U_att(1, .., 1) above it)
    checks every section always.
  * An operation missing from Table 4 (O) takes p = 1 (every unhandled
    error is taken as fatal).
"""
from __future__ import annotations

import math
from dataclasses import dataclass
from typing import Dict, List, Sequence

TYPES = ("INF", "NaN", "nINF")


@dataclass
class Op:
    name: str
    flops: float
    p: Dict[str, float]          # Table 4: P(non-trainable | one error of type e)


@dataclass
class Section:
    name: str
    ops: List[Op]
    cost: float                  # T_S: ABFT time of the section when always on


def poisson(k: int, mean: float) -> float:
    """P(k) of a Poisson law of the given mean (Sec. 4.5)."""
    return math.exp(-mean) * mean ** k / math.factorial(k)


def mean_errors(sec: Section, lam: Dict[str, float]) -> float:
    return sum(lam[e] * op.flops for op in sec.ops for e in TYPES)


def r_free(sec: Section, lam: Dict[str, float]) -> float:
    """Probability of no error in any operation of the section."""
    r = 1.0
    for op in sec.ops:
        for e in TYPES:
            r *= poisson(0, lam[e] * op.flops)
    return r


def r_single(sec: Section, lam: Dict[str, float], j: int, e: str) -> float:
    """Exactly one error, of type e, in operation j; none anywhere else."""
    op = sec.ops[j]
    r = 1.0
    for t in TYPES:
        r *= poisson(1 if t == e else 0, lam[t] * op.flops)
    rest = Section(sec.name, [o for i, o in enumerate(sec.ops) if i != j], sec.cost)
    return r * r_free(rest, lam)


def p_two_or_more(mu: float) -> float:
    """P(k >= 2) of a Poisson law of mean mu, without cancellation: the
    series exp(-mu) sum_{k>=2} mu^k / k! for small mu."""
    if mu > 0.5:
        return 1.0 - math.exp(-mu) * (1.0 + mu)
    term, acc, k = mu * mu / 2.0, 0.0, 2
    while term > 0.0 and term > acc * 1e-18:
        acc += term
        k += 1
        term *= mu / k
    return math.exp(-mu) * acc


def harmful_single(sec: Section, lam: Dict[str, float]) -> float:
    """sum_i sum_e R_e(i) p_i^e: one error, fatal unless handled."""
    return sum(r_single(sec, lam, j, e) * op.p[e] for j, op in enumerate(sec.ops) for e in TYPES)


def unsafe_section(sec: Section, lam: Dict[str, float], f: float) -> float:
    """U_S(f) = 1 - FC_S(f)."""
    return p_two_or_more(mean_errors(sec, lam)) + (1.0 - f) * harmful_single(sec, lam)


def fc_section(sec: Section, lam: Dict[str, float], f: float) -> float:
    """FC_S(f) as printed (a sum of probabilities; use unsafe_section for
    its complement near 1)."""
    fc = r_free(sec, lam)
    for j, op in enumerate(sec.ops):
        for e in TYPES:
            fc += r_single(sec, lam, j, e) * (f + (1.0 - f) * (1.0 - op.p[e]))
    return fc


def unsafe_att(secs: Sequence[Section], lam: Dict[str, float], freqs: Sequence[float]) -> float:
    """U_att = 1 - prod_S FC_S(f_S)."""
    return -math.expm1(sum(math.log1p(-unsafe_section(s, lam, f)) for s, f in zip(secs, freqs)))


def fce(sec: Section, lam: Dict[str, float]) -> float:
    """Coverage gained per unit of ABFT time spent on the section."""
    return harmful_single(sec, lam) / sec.cost if sec.cost > 0 else math.inf


def optimize(secs: Sequence[Section], lam: Dict[str, float], fail_target: float) -> List[float]:
    """Algorithm 1 (reading above), with the target given as the allowed
    failure probability per execution (1 - FC_target); returns f_S per
    section in the input order."""
    if fail_target <= unsafe_att(secs, lam, [1.0] * len(secs)):
        return [1.0] * len(secs)   # unreachable: check every section always
    deficit = unsafe_att(secs, lam, [0.0] * len(secs)) - fail_target
    f = [0.0] * len(secs)
    # a section whose check costs nothing is always checked: its whole
    # coverage gain comes first and for free
    for i, s in enumerate(secs):
        if s.cost <= 0.0:
            f[i] = 1.0
            deficit -= harmful_single(s, lam)
    paid = [i for i, s in enumerate(secs) if s.cost > 0.0]
    for i in sorted(paid, key=lambda i: -fce(secs[i], lam)):
        s = secs[i]
        if deficit <= 0.0:
            break
        gain = fce(s, lam)
        if gain * s.cost <= deficit:
            f[i] = 1.0
            deficit -= gain * s.cost
        else:
            f[i] = deficit / (gain * s.cost)
            deficit = 0.0
    return f


def schedule(freq: float, step: int) -> bool:
    """Whether a section of frequency freq is checked at a given step: on
    when floor((k+1) f) > floor(k f), which holds on a fraction f of any
    long run of steps, spread evenly."""
    return math.floor((step + 1) * freq) > math.floor(step * freq)


# ---- the paper's inputs ------------------------------------------------

# Table 4: probability of a non-trainable state after one error, per model,
# error type and injected matrix (Q, K, V, AS, CL)
TABLE4 = {
    "Bert":    {"INF": (1.000, 1.000, 1.000, 1.000, 1.000),
                "NaN": (1.000, 1.000, 1.000, 1.000, 1.000),
                "nINF": (0.459, 0.434, 0.063, 0.002, 0.006)},
    "GPT-2":   {"INF": (0.918, 0.868, 1.000, 0.569, 1.000),
                "NaN": (1.000, 1.000, 1.000, 0.547, 1.000),
                "nINF": (0.384, 0.372, 0.010, 0.005, 0.007)},
    "Neo":     {"INF": (1.000, 0.856, 1.000, 0.547, 1.000),
                "NaN": (1.000, 1.000, 1.000, 0.547, 1.000),
                "nINF": (0.103, 0.144, 0.058, 0.112, 0.096)},
    "Roberta": {"INF": (1.000, 0.999, 1.000, 1.000, 1.000),
                "NaN": (1.000, 1.000, 1.000, 1.000, 1.000),
                "nINF": (0.540, 0.499, 0.036, 0.055, 0.004)},
}
MATRICES = ("Q", "K", "V", "AS", "CL")


def table4_p(model: str, matrix: str) -> Dict[str, float]:
    if matrix not in MATRICES:
        return {e: 1.0 for e in TYPES}
    k = MATRICES.index(matrix)
    return {e: TABLE4[model][e][k] for e in TYPES}


def layer_sections(B: int, S: int, H: int, nh: int, causal: bool, model: str,
                   costs: Dict[str, float]) -> List[Section]:
    """The forward's three protection sections (Sec. 4.4) at a layer shape:
    S_AS = {X W^Q, X W^K, Q K^T}, S_CL = {X W^V, AP V}, S_O = {CL W^O};
    flops are 2 M N K per GEMM (unmasked score pairs only)."""
    T, d = B * S, H // nh
    P = S * (S + 1) // 2 if causal else S * S
    proj = 2.0 * T * H * H
    score = 2.0 * B * nh * d * P

    def op(name, n):
        return Op(name, n, table4_p(model, name))

    return [
        Section("AS", [op("Q", proj), op("K", proj), op("AS", score)], costs["AS"]),
        Section("CL", [op("V", proj), op("CL", score)], costs["CL"]),
        Section("O", [op("O", proj)], costs["O"]),
    ]
