"""MetaKV's per-prompt configuration choice and its success metric.

Section 2.3 describes the choice: predicted end-to-end latency and peak memory of every
candidate configuration pass a budget filter (at most L_max and M_max); uncompressed FP16 is
taken whenever it passes; otherwise only the least compressed passing setting of each method
stays, and the one left, or the one an accuracy predictor rates highest, is taken.  When nothing
passes, the configuration with the smallest relative violation
v_c = L_c / L_max + M_c / M_max is taken, the accuracy prediction breaking ties.  Readings:
"least compressed" is the lowest compression level within a method (more bits, a larger H2O
budget, a smaller RocketKV ratio); ties that remain go to the candidate listed first.

Section 3.1 defines the constrained success rate: the fraction of prompts answered correctly
with latency at most L_max and peak memory at most M_max.

TEST INFRASTRUCTURE ONLY (see the package docstring).
"""


def select(cands, l_max, m_max):
    """cands: list of dicts with method, level, latency, memory, p_correct.
    -> (index of the chosen candidate, True when no candidate met both budgets)."""
    passing = [i for i, c in enumerate(cands) if c["latency"] <= l_max and c["memory"] <= m_max]
    if not passing:
        def violation(i):
            return cands[i]["latency"] / l_max + cands[i]["memory"] / m_max
        best = 0
        for i in range(1, len(cands)):
            if violation(i) < violation(best) or (violation(i) == violation(best)
                                                 and cands[i]["p_correct"] > cands[best]["p_correct"]):
                best = i
        return best, True
    for i in passing:
        if cands[i]["method"] == "fp16":
            return i, False
    per_method = {}
    for i in passing:
        m = cands[i]["method"]
        if m not in per_method or cands[i]["level"] < cands[per_method[m]]["level"]:
            per_method[m] = i
    left = sorted(per_method.values())
    if len(left) == 1:
        return left[0], False
    best = left[0]
    for i in left[1:]:
        if cands[i]["p_correct"] > cands[best]["p_correct"]:
            best = i
    return best, False


def constrained_success_rate(correct, latency, memory, l_max, m_max):
    """Fraction of prompts i with correct[i], latency[i] <= l_max and memory[i] <= m_max."""
    n = len(correct)
    ok = sum(1 for i in range(n) if correct[i] and latency[i] <= l_max and memory[i] <= m_max)
    return ok / n
