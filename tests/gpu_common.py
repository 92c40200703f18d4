"""Helpers for the GPU parity tests: run the HIP path and the oracle on the
same seeded inputs and compare them to the stated tolerances."""
from __future__ import annotations

import numpy as np
import torch

import oracle
import paper_2608_24004_amd as av
import workload

# Attention tolerance: per (row, head) output vector, the infinity-norm error
# relative to the infinity norm of the reference.  bf16 storage with fp32
# accumulation: 2e-2.  fp32 storage: the kernel rounds P to nothing and keeps
# fp32 throughout, so 1e-4 leaves room only for summation-order differences.
ATTN_TOL = {"bf16": 2e-2, "f32": 1e-4}
NEAR_TIE = 1e-3   # top-2 logit gap below which a row's argmax is flagged


def rel_err_rows(got: np.ndarray, ref: np.ndarray) -> np.ndarray:
    got = got.reshape(-1, got.shape[-1]).astype(np.float64)
    ref = ref.reshape(-1, ref.shape[-1])
    den = np.maximum(np.abs(ref).max(axis=1), 1e-6)
    return np.abs(got - ref).max(axis=1) / den


def assert_attention_close(got, ref, dtype: str, what: str = ""):
    err = rel_err_rows(np.asarray(got), np.asarray(ref))
    tol = ATTN_TOL[dtype]
    bad = np.nonzero(~(err <= tol))[0]
    assert bad.size == 0, "%s: %d of %d vectors above %.0e (max %.3e at %d)" % (
        what, bad.size, err.size, tol, float(np.nanmax(err)), int(bad[0]))
    return float(err.max()) if err.size else 0.0


def to_host_f64(t) -> np.ndarray:
    return t.detach().to(torch.float64).cpu().numpy()


def gpu_attention(q, kc, vc, bt, sl, qs, *, max_q_len, max_seq_len, window=0, split=0, sinks=None):
    out = av.verify_attention(q, kc, vc, bt, sl, qs, max_q_len=max_q_len, max_seq_len=max_seq_len,
                              sliding_window=window, kv_split_blocks=split, sinks=sinks)
    torch.cuda.synchronize()
    return out


def compact_for_rows(batch, layer, rows: np.ndarray):
    """Host copies holding only the KV blocks of the requests that own `rows`
    (so a sample of a very large cache can be checked on the CPU).  Returns the
    oracle keyword arguments and the rows renumbered into the compact batch."""
    reqs = np.unique(np.searchsorted(batch.q_start, rows, side="right") - 1)
    bt = batch.block_tables[reqs]
    used = np.unique(bt[bt >= 0])
    remap = np.full(batch.num_blocks, -1, dtype=np.int32)
    remap[used] = np.arange(used.size, dtype=np.int32)
    bt_c = np.where(bt >= 0, remap[np.maximum(bt, 0)], -1).astype(np.int32)
    idx = torch.as_tensor(used, dtype=torch.int64, device=layer.k_cache.device)
    kc = workload.host_storage(layer.k_cache.index_select(0, idx))
    vc = workload.host_storage(layer.v_cache.index_select(0, idx))
    n = np.diff(batch.q_start)[reqs]
    qs_c = np.zeros(reqs.size + 1, dtype=np.int32)
    qs_c[1:] = np.cumsum(n)
    old_rows = np.concatenate([np.arange(batch.q_start[r], batch.q_start[r + 1]) for r in reqs])
    qrows = torch.as_tensor(old_rows, dtype=torch.int64, device=layer.q.device)
    q_c = workload.host_storage(layer.q.index_select(0, qrows))
    new_of_old = {int(o): k for k, o in enumerate(old_rows)}
    rows_c = np.array([new_of_old[int(r)] for r in rows], dtype=np.int32)
    cfg = batch.cfg
    args = dict(num_q_heads=cfg.num_q_heads, num_kv_heads=cfg.num_kv_heads, head_dim=cfg.head_dim,
                sliding_window=layer.window, scale=0.0, dtype=workload.dtype_code(cfg.dtype),
                q=q_c, k_cache=kc, v_cache=vc, block_tables=bt_c,
                seq_lens=batch.seq_lens[reqs], q_start=qs_c,
                sinks=None if layer.sinks is None else layer.sinks.cpu().numpy())
    return args, rows_c


def sample_pairs(batch, n_pairs: int, seed: int, max_requests: int = 6):
    """(rows, heads) to check: every row of a few requests (including the ones
    with the fewest and the most drafts and the longest context), each with a
    random head, plus random extra pairs inside those requests."""
    rng = np.random.default_rng(seed)
    B, Hq = len(batch.seq_lens), batch.cfg.num_q_heads
    n = np.diff(batch.q_start)
    want = {int(np.argmin(n)), int(np.argmax(n)), int(np.argmax(batch.seq_lens))}
    others = [i for i in rng.permutation(B) if i not in want]
    reqs = sorted(list(want) + others[:max(0, max_requests - len(want))])
    rows = np.concatenate([np.arange(batch.q_start[i], batch.q_start[i + 1]) for i in reqs])
    extra = rng.choice(rows, size=n_pairs)
    rows = np.concatenate([rows, extra])
    heads = rng.integers(0, Hq, size=rows.size)
    return rows.astype(np.int32), heads.astype(np.int32)


def oracle_accept_all(logits, q_start, tokens, dtype_code):
    am, gap = oracle.argmax(workload.host_storage(logits), dtype_code)
    acc, ne, em = oracle.accept(q_start, tokens, am)
    return am, gap, acc, ne, em


def pair_schedule(batch, layer, plan):
    """(request, KV head, row group) pairs of the persistent bf16 schedule and
    whether a workgroup range boundary cuts each one (its first and last KV
    blocks belong to different workgroups), from the plan verify_attention
    reports: one launch per row class, each with the unit numbering and the
    equal-share ranges it documents over the class's requests."""
    cfg = batch.cfg
    G = cfg.num_q_heads // cfg.num_kv_heads
    n = np.diff(batch.q_start).astype(np.int64)
    S = batch.seq_lens.astype(np.int64)
    W = layer.window
    key_lo = np.maximum(0, S - n - W + 1) if W > 0 else np.zeros_like(S)
    nb = np.maximum(0, (S + 15) // 16 - key_lo // 16)
    pairs = []
    for cls in plan.get("classes", [plan]):
        rpg, rg_max, nwg = cls["rows_per_group"], cls["row_groups"], cls["workgroups"]
        lo, hi = cls.get("rows_lo", 0), cls.get("rows_hi", 2 ** 31 - 1)
        inside = (G * n >= lo) & (G * n <= hi)
        rg = np.where(inside, np.minimum(rg_max, (G * n + rpg - 1) // rpg), 0)
        units = cfg.num_kv_heads * rg * nb
        start = np.concatenate([[0], np.cumsum(units)])
        U = int(start[-1])
        N = min(nwg, max(U, 1))
        owner = lambda u: ((u + 1) * N - 1) // max(U, 1)
        for i in range(len(n)):
            for g in range(cfg.num_kv_heads):
                for r in range(int(rg[i])):
                    if nb[i] == 0:
                        continue
                    ps = int(start[i]) + (g * int(rg[i]) + r) * int(nb[i])
                    pairs.append((i, g, r, owner(ps) != owner(ps + int(nb[i]) - 1)))
    return pairs


def row_reach(plan, rows):
    """Local rows (Hq/Hkv * j + h % (Hq/Hkv)) the launch computes for a request
    with `rows` of them: its row class's row groups times rows per group."""
    if not plan["mfma"]:
        return plan["row_groups"] * plan["rows_per_item"]
    for cls in plan["classes"]:
        if cls["rows_lo"] <= rows <= cls["rows_hi"]:
            return cls["row_groups"] * cls["rows_per_group"]
    raise AssertionError("no row class holds %d rows" % rows)


def pair_vectors(batch, pair, rows_per_group):
    """(rows, heads) of the output vectors a pair computes."""
    i, g, r, _ = pair
    cfg = batch.cfg
    G = cfg.num_q_heads // cfg.num_kv_heads
    q0, q1 = int(batch.q_start[i]), int(batch.q_start[i + 1])
    local = np.arange(r * rows_per_group, min((r + 1) * rows_per_group, G * (q1 - q0)))
    return (q0 + local // G).astype(np.int32), (g * G + local % G).astype(np.int32)
