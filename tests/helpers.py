"""Test-side helpers: restricting a paged KV cache to a few sequences so the
oracle can evaluate sampled rows of a full-size workload on the host."""
import torch

from paper_2608_01891_amd import synth


def sub_attention(a, rows):
    """CPU AttnInputs holding only sequences ``rows`` of ``a`` (blocks re-numbered)."""
    rows = [int(r) for r in rows]
    bt = a.block_table.cpu()
    ctx = a.context_lens.cpu()
    phys, table = [], torch.full((len(rows), a.max_blocks), -1, dtype=torch.int32)
    for i, b in enumerate(rows):
        n = -(-int(ctx[b]) // a.block_size)
        ids = bt[b, :n].tolist()
        table[i, :n] = torch.arange(len(phys), len(phys) + n, dtype=torch.int32)
        phys += ids
    idx = torch.tensor(phys, dtype=torch.int64, device=a.k_cache.device)
    if len(phys) == 0:
        idx = torch.zeros(1, dtype=torch.int64, device=a.k_cache.device)
    k = a.k_cache.index_select(0, idx).cpu()
    v = a.v_cache.index_select(0, idx).cpu()
    return synth.AttnInputs(q=a.q[rows].cpu(), k_cache=k, v_cache=v, block_table=table,
                            context_lens=ctx[rows].clone(), B=len(rows), Hq=a.Hq, Hkv=a.Hkv, D=a.D,
                            block_size=a.block_size, max_blocks=a.max_blocks,
                            num_blocks=max(len(phys), 1), max_context_len=a.max_context_len)


def sample_rows(n_total, n, seed=0, must=()):
    g = torch.Generator().manual_seed(seed)
    picks = set(int(m) for m in must)
    perm = torch.randperm(n_total, generator=g).tolist()
    for p in perm:
        if len(picks) >= n:
            break
        picks.add(p)
    return sorted(picks)
