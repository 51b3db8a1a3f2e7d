"""Oracle: the paper's metrics (Sec. 5.1.3).  TEST INFRASTRUCTURE ONLY.

omega(gamma, alpha): expected number of tokens produced by one verification
of a gamma-token chain when each drafted token is accepted independently with
probability alpha (the geometric sum 1 + alpha + ... + alpha^gamma).
speedup_ratio: normal-decoding time over speculative-decoding time for N
output tokens including the prompt-processing time, with per-token target
time T_p, draft time T_q per drafted token and verification time T_v.
tau: mean tokens emitted per draft-verify cycle.
n_alpha: acceptance rate of the n-th drafted token of chain drafts (one token
per draft forward, Sec. 5.1.3): of the cycles whose first n-1 drafted tokens
were accepted, so that the n-th was judged, the fraction that accepted it.
"""


def omega(gamma, alpha):
    if alpha == 1.0:
        return float(gamma + 1)
    return (1.0 - alpha ** (gamma + 1)) / (1.0 - alpha)


def speedup_ratio(N, T_p, T_q, T_v, gamma, alpha, T_prompt):
    w = omega(gamma, alpha)
    return (N * T_p + T_prompt) / (N * (gamma * T_q + T_v) / w + T_prompt)


def tau(emitted_per_cycle):
    n = len(emitted_per_cycle)
    return sum(emitted_per_cycle) / n if n else 0.0


def n_alpha(accepted_per_cycle, gamma):
    """[n-alpha for n = 1..gamma] from the number of accepted drafted tokens
    of each chain cycle (None where no cycle reached position n)."""
    out = []
    for n in range(1, gamma + 1):
        judged = sum(1 for a in accepted_per_cycle if a >= n - 1)
        accepted = sum(1 for a in accepted_per_cycle if a >= n)
        out.append(accepted / judged if judged else None)
    return out

