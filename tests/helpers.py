"""Shared test helpers: structured inputs built through the workload packer."""
from __future__ import annotations

import numpy as np
import torch

import workload
from workload import BLOCK


def bf16_round(a: np.ndarray) -> np.ndarray:
    """Round float values to the nearest bf16 (RNE) and return them as float64."""
    return torch.as_tensor(np.asarray(a, dtype=np.float32)).to(torch.bfloat16).to(torch.float64).numpy()


class Paged:
    """A batch assembled from logical per-request K/V, packed into paged caches."""

    def __init__(self, *, num_q_heads, num_kv_heads, head_dim, dtype, k_logical, v_logical,
                 q, num_drafts, window=0, seed=0, spare_blocks=3):
        self.Hq, self.Hkv, self.D = num_q_heads, num_kv_heads, head_dim
        self.dtype = dtype
        self.window = window
        tdt = workload.torch_dtype(dtype)
        x = workload.elems_per_16b(dtype)
        rng = np.random.default_rng(seed)
        self.num_drafts = np.asarray(num_drafts, dtype=np.int64)
        self.seq_lens = np.array([k.shape[0] for k in k_logical], dtype=np.int32)
        n = self.num_drafts + 1
        assert np.all(self.seq_lens >= n)
        self.q_start = np.zeros(len(k_logical) + 1, dtype=np.int32)
        self.q_start[1:] = np.cumsum(n)
        nblk = (self.seq_lens + BLOCK - 1) // BLOCK
        self.num_blocks = int(nblk.sum()) + spare_blocks
        perm = rng.permutation(self.num_blocks).astype(np.int32)
        self.block_tables = np.full((len(k_logical), max(1, int(nblk.max()))), -1, dtype=np.int32)
        off = 0
        for i in range(len(k_logical)):
            self.block_tables[i, :nblk[i]] = perm[off:off + nblk[i]]
            off += nblk[i]
        # spare blocks hold garbage that no request may read
        kc = torch.full((self.num_blocks, self.Hkv, self.D // x, BLOCK, x), 1e4, dtype=tdt)
        vc = torch.full((self.num_blocks, self.Hkv, self.D, BLOCK), -1e4, dtype=tdt)
        for i, (kl, vl) in enumerate(zip(k_logical, v_logical)):
            kl = torch.as_tensor(np.asarray(kl, dtype=np.float32)).to(tdt)
            vl = torch.as_tensor(np.asarray(vl, dtype=np.float32)).to(tdt)
            for g in range(self.Hkv):
                workload.pack_request_kv(kl[:, g, :], vl[:, g, :], self.block_tables[i], kc, vc, g)
        self.k_cache, self.v_cache = kc, vc
        self.q = torch.as_tensor(np.asarray(q, dtype=np.float32)).to(tdt)
        self.k_logical = [torch.as_tensor(np.asarray(k, dtype=np.float32)).to(tdt).to(torch.float64)
                          for k in k_logical]
        self.v_logical = [torch.as_tensor(np.asarray(v, dtype=np.float32)).to(tdt).to(torch.float64)
                          for v in v_logical]

    @property
    def total_q(self):
        return int(self.q_start[-1])

    def oracle_args(self):
        return dict(num_q_heads=self.Hq, num_kv_heads=self.Hkv, head_dim=self.D,
                    sliding_window=self.window, scale=0.0, dtype=workload.dtype_code(self.dtype),
                    q=workload.host_storage(self.q), k_cache=workload.host_storage(self.k_cache),
                    v_cache=workload.host_storage(self.v_cache), block_tables=self.block_tables,
                    seq_lens=self.seq_lens, q_start=self.q_start)


def random_paged(*, num_q_heads, num_kv_heads, head_dim, dtype, contexts, drafts, window=0,
                 seed=0, spare_blocks=3):
    rng = np.random.default_rng(1000 + seed)
    k_log, v_log = [], []
    for L, k in zip(contexts, drafts):
        S = int(L) + int(k) + 1
        k_log.append(rng.standard_normal((S, num_kv_heads, head_dim)))
        v_log.append(rng.standard_normal((S, num_kv_heads, head_dim)))
    T = int(np.sum(np.asarray(drafts) + 1))
    q = rng.standard_normal((T, num_q_heads, head_dim))
    return Paged(num_q_heads=num_q_heads, num_kv_heads=num_kv_heads, head_dim=head_dim,
                 dtype=dtype, k_logical=k_log, v_logical=v_log, q=q, num_drafts=drafts,
                 window=window, seed=seed, spare_blocks=spare_blocks)


def sdpa_reference(p: Paged, missing=None) -> np.ndarray:
    """torch scaled_dot_product_attention (float64, CPU) on the logical tensors, with
    an explicit boolean mask for the in-draft causal rule and the sliding window.
    ``missing``: optional {request: set of logical block indices} whose keys are
    left out of the mask (an unmapped block); a row left with no key is zero."""
    G = p.Hq // p.Hkv
    out = np.zeros((p.total_q, p.Hq, p.D))
    qf = p.q.to(torch.float64)
    for i in range(len(p.seq_lens)):
        q0, q1 = int(p.q_start[i]), int(p.q_start[i + 1])
        n, S = q1 - q0, int(p.seq_lens[i])
        pos = torch.arange(S - n, S)[:, None]
        t = torch.arange(S)[None, :]
        mask = t <= pos
        if p.window > 0:
            mask &= t > pos - p.window
        for b in (missing or {}).get(i, ()):
            mask &= (t // 16) != b
        qi = qf[q0:q1].permute(1, 0, 2)[None]                         # [1, Hq, n, D]
        ki = p.k_logical[i].permute(1, 0, 2).repeat_interleave(G, 0)[None]  # [1, Hq, S, D]
        vi = p.v_logical[i].permute(1, 0, 2).repeat_interleave(G, 0)[None]
        o = torch.nn.functional.scaled_dot_product_attention(qi, ki, vi, attn_mask=mask)
        o = torch.where(mask.any(dim=1)[None, None, :, None], o, torch.zeros_like(o))
        out[q0:q1] = o[0].permute(1, 0, 2).numpy()
    return out
