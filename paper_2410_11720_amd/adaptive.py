"""Inputs of the adaptive detection frequencies (paper Sec. 4.5) for one
attention layer: the operations of each protection section with their
flops and vulnerabilities, in the form attn_abft_optimize_frequencies
takes. The optimiser and the per-step masks are the library's
(attn_abft_optimize_frequencies, attn_abft_sections_for_step)."""
from __future__ import annotations

# Table 4 (Sec. 3.3): probability that one error of type INF / NaN /
# near-INF in the given output leads to a non-trainable state.
VULNERABILITY = {
    "Bert":    {"Q": (1.000, 1.000, 0.459), "K": (1.000, 1.000, 0.434),
                "V": (1.000, 1.000, 0.063), "AS": (1.000, 1.000, 0.002),
                "CL": (1.000, 1.000, 0.006)},
    "GPT-2":   {"Q": (0.918, 1.000, 0.384), "K": (0.868, 1.000, 0.372),
                "V": (1.000, 1.000, 0.010), "AS": (0.569, 0.547, 0.005),
                "CL": (1.000, 1.000, 0.007)},
    "Neo":     {"Q": (1.000, 1.000, 0.103), "K": (0.856, 1.000, 0.144),
                "V": (1.000, 1.000, 0.058), "AS": (0.547, 0.547, 0.112),
                "CL": (1.000, 1.000, 0.096)},
    "Roberta": {"Q": (1.000, 1.000, 0.540), "K": (0.999, 1.000, 0.499),
                "V": (1.000, 1.000, 0.036), "AS": (1.000, 1.000, 0.055),
                "CL": (1.000, 1.000, 0.004)},
}
FATAL = (1.0, 1.0, 1.0)   # outputs the table does not cover (O, the backward)


def layer_sections(batch, seq, hidden, heads, causal, costs, model="GPT-2", backward=True):
    """[(T_S, [(flops, (p_INF, p_NaN, p_nINF)), ...]), ...] for S_AS, S_CL,
    S_O and, with backward=True, the backward as one more section.
    costs: check time of each section when run every step, same order."""
    T, d = batch * seq, hidden // heads
    P = seq * (seq + 1) // 2 if causal else seq * seq
    proj = 2.0 * T * hidden * hidden
    score = 2.0 * batch * heads * d * P
    v = VULNERABILITY[model]
    secs = [
        (costs[0], [(proj, v["Q"]), (proj, v["K"]), (score, v["AS"])]),
        (costs[1], [(proj, v["V"]), (score, v["CL"])]),
        (costs[2], [(proj, FATAL)]),
    ]
    if backward:
        fwd = 4 * proj + 2 * score
        secs.append((costs[3], [(2.0 * fwd, FATAL)]))
    return secs
