"""Oracle: the paper's metrics (Sec. 5.1.3).  TEST INFRASTRUCTURE ONLY.

omega(gamma, alpha): expected number of tokens produced by one verification
of a gamma-token chain when each drafted token is accepted independently with
probability alpha (the geometric sum 1 + alpha + ... + alpha^gamma).
speedup_ratio: normal-decoding time over speculative-decoding time for N
output tokens including the prompt-processing time, with per-token target
time T_p, draft time T_q per drafted token and verification time T_v.
tau: mean tokens emitted per draft-verify cycle.
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
