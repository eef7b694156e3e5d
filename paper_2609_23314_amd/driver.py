"""Block prompt processing and decode on top of ``vd_evict_step`` (Sec. 2.2,
Eq. block_processing): append a block of new K/V rows to every unit's cache,
then apply the eviction pass; B = T is one-shot eviction and B = 1 is
decode-time eviction.

``EvictingCache`` owns the cache tensors, the host-side token counts, the
optional running-sum state and a ``pos`` payload (the original token index of
every cached row).  Appending is a plain device copy into the tail slots; the
pass itself runs in the HIP library.
"""
from typing import Optional, Sequence

import torch

from . import vd


class EvictingCache:
    def __init__(self, num_seqs: int, num_layers: int, num_kv_heads: int, head_dim: int,
                 capacity: int, budget: Sequence[int], dtype=torch.bfloat16, device="cuda",
                 variant: str = "l2", num_q_heads: Optional[int] = None,
                 running_sum: bool = True, track_pos: bool = True):
        shape = (num_seqs, num_layers, num_kv_heads, capacity, head_dim)
        self.k = torch.zeros(shape, dtype=dtype, device=device)
        self.v = torch.zeros(shape, dtype=dtype, device=device)
        self.units = num_seqs * num_layers * num_kv_heads
        self.n = [0] * num_seqs          # cached tokens per sequence (host)
        self.seen = [0] * num_seqs       # tokens appended so far per sequence
        self.budget = [int(b) for b in budget]
        self.variant = variant
        self.num_q_heads = num_q_heads
        self.running_sum = (torch.zeros((self.units, head_dim + 1), dtype=torch.float64,
                                        device=device) if running_sum else None)
        self.pos = (torch.full((self.units, capacity), -1, dtype=torch.int32, device=device)
                    if track_pos else None)
        self.capacity = capacity

    def append(self, seq: int, k_rows: torch.Tensor, v_rows: torch.Tensor):
        """Appends [layers, kv_heads, t, head_dim] rows to sequence `seq`."""
        t = k_rows.shape[2]
        n0 = self.n[seq]
        if n0 + t > self.capacity:
            raise ValueError(f"sequence {seq}: {n0} + {t} rows exceed capacity {self.capacity}")
        self.k[seq, :, :, n0:n0 + t].copy_(k_rows)
        self.v[seq, :, :, n0:n0 + t].copy_(v_rows)
        if self.pos is not None:
            L, H = self.k.shape[1], self.k.shape[2]
            u0 = seq * L * H
            ids = torch.arange(self.seen[seq], self.seen[seq] + t, dtype=torch.int32,
                               device=self.pos.device)
            self.pos[u0:u0 + L * H, n0:n0 + t] = ids
        self.n[seq] = n0 + t
        self.seen[seq] += t

    def evict(self, scores_out=None, keep_out=None, stream=None):
        """One eviction pass over every unit; afterwards n = min(n, N)."""
        vd.vd_evict_step(self.k, self.v, self.n, self.budget, self.variant,
                         running_sum=self.running_sum, pos=self.pos, scores_out=scores_out,
                         keep_out=keep_out, num_q_heads=self.num_q_heads, stream=stream)
        self.n = [min(n, N) for n, N in zip(self.n, self.budget)]
