"""Host-side planning for the interleaved A/F layer step.

Eq. 2 of the paper models the time of one layer step of the A/F pipeline
(section 4.3, "Interleaved A/F Pipeline"): with M = 1 the attention, the
hidden-state transfer and the FFN run one after the other; with M >= 2
microbatches the two stages overlap, the slower stage sets the pace and the
transfer is amortised over the microbatches:

    t_layer = t_A + t_F + t_comm              (M = 1)
    t_layer = max(t_A, t_F) + t_comm / M      (M >= 2)
"""
from __future__ import annotations


def eq2_layer_time(t_a: float, t_f: float, t_comm: float, M: int) -> float:
    if M < 1:
        raise ValueError("microbatch depth M must be >= 1")
    if M == 1:
        return t_a + t_f + t_comm
    return max(t_a, t_f) + t_comm / M


def equal_microbatches(B: int, M: int):
    """M contiguous microbatch sizes summing to B, as equal as possible."""
    if not 1 <= M <= B:
        raise ValueError("need 1 <= M <= B")
    base, rem = divmod(B, M)
    return [base + (1 if i < rem else 0) for i in range(M)]


# --------------------------------------------------------------------------
# Dynamic microbatch depth and adaptive request batching (section 4.3; the
# paper's Table 1 evaluates both): choose the number of microbatches M and
# their sizes with the lowest predicted (or measured) layer time.
# --------------------------------------------------------------------------
def candidate_splits(B: int, depths=(1, 2, 4), granularity: int = 16,
                     uneven=(0.25, 1 / 3, 2 / 3, 0.75)):
    """Contiguous microbatch splits of B: equal ones for each depth, plus
    uneven two-way splits (sizes rounded to ``granularity``)."""
    out = []
    for M in depths:
        if 1 <= M <= B:
            out.append(equal_microbatches(B, M))
    if 2 in depths:
        for f in uneven:
            n1 = int(round(B * f / granularity)) * granularity
            if 0 < n1 < B:
                out.append([n1, B - n1])
    seen, uniq = set(), []
    for s in out:
        if tuple(s) not in seen:
            seen.add(tuple(s))
            uniq.append(s)
    return uniq


def eq2_predict(sizes, t_a, t_f, t_comm: float = 0.0) -> float:
    """Eq. 2 with profiled per-stage latency curves t_a(n), t_f(n) of a
    microbatch of n requests; with M >= 2 the slower stage's total sets the pace."""
    M = len(sizes)
    if M == 1:
        return eq2_layer_time(t_a(sizes[0]), t_f(sizes[0]), t_comm, 1)
    return eq2_layer_time(sum(t_a(n) for n in sizes), sum(t_f(n) for n in sizes), t_comm, M)


def choose_split(candidates, cost):
    """The candidate with the smallest cost (ties: the earlier candidate)."""
    best, best_c = None, None
    for s in candidates:
        c = cost(s)
        if best is None or c < best_c:
            best, best_c = s, c
    return best, best_c
