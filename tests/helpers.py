"""Test-side helpers: picking sample rows of a full-size workload (test code only)."""
import torch


def sample_rows(n_total, n, seed=0, must=()):
    g = torch.Generator().manual_seed(seed)
    picks = set(int(m) for m in must)
    perm = torch.randperm(n_total, generator=g).tolist()
    for p in perm:
        if len(picks) >= n:
            break
        picks.add(p)
    return sorted(picks)
