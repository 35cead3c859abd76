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
