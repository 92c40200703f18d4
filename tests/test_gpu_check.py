"""verify_check_batch on the GPU: every count and the first offending request
equal a host restatement of the preconditions the header states, on the
workloads' own (valid) descriptors and on seeded corruptions of them; and the
binding's check=True refuses a bad descriptor before it launches anything."""
from __future__ import annotations

import sys

import numpy as np
import pytest
import torch

import paper_2608_24004_amd as av
import workload

pytestmark = pytest.mark.gpu
DEV = "cuda:0"
INT_MAX = 2 ** 31 - 1


def say(*a):
    print(*a, file=sys.stderr, flush=True)


def host_check(q_start, total_q, max_q_len=0, seq_lens=None, block_tables=None, num_blocks=0,
               max_seq_len=0, window=0):
    """The preconditions, request by request, as the header states them."""
    B = len(q_start) - 1
    flags = np.zeros((B, 5), dtype=bool)
    for i in range(B):
        q0, q1 = int(q_start[i]), int(q_start[i + 1])
        flags[i, 0] = (q0 < 0 or q1 < q0 or q1 > total_q or (i == 0 and q0 != 0)
                       or (i == B - 1 and q1 != total_q))
        n = max(q1 - q0, 0)
        flags[i, 1] = max_q_len > 0 and n > max_q_len
        if seq_lens is None:
            continue
        S = int(seq_lens[i])
        mb = block_tables.shape[1] if block_tables is not None else (1 << 31) // 16 - 1
        flags[i, 2] = S < n
        flags[i, 3] = S > max_seq_len or S > 16 * mb
        if block_tables is not None:
            hi = min(max(S, 0), 16 * mb)
            lo = max(0, hi - n - window + 1) if window > 0 else 0
            ids = block_tables[i, lo // 16:(hi + 15) // 16]
            flags[i, 4] = bool(np.any((ids < 0) | (ids >= num_blocks)))
    counts = dict(zip(av.CHECK_KINDS, (int(c) for c in flags.sum(axis=0))))
    bad = np.nonzero(flags.any(axis=1))[0]
    return counts, (int(bad[0]) if bad.size else -1)


def _gpu(qs, total_q, *, max_q_len=0, seq_lens=None, block_tables=None, num_blocks=0,
         max_seq_len=0, window=0):
    d = lambda a: None if a is None else torch.as_tensor(np.ascontiguousarray(a), device=DEV)
    return av.check_batch(d(qs), total_q, max_q_len=max_q_len, seq_lens=d(seq_lens),
                          block_tables=d(block_tables), num_blocks=num_blocks,
                          max_seq_len=max_seq_len, sliding_window=window)


def _both(what, qs, total_q, **kw):
    got = _gpu(qs, total_q, **kw)
    want = host_check(qs, total_q, **kw)
    assert got == want, "%s: device %s, host %s" % (what, got, want)
    return got


@pytest.mark.parametrize("name", list(workload.CONFIGS))
def test_valid_workload_descriptors_pass(name):
    cfg = workload.CONFIGS[name]
    bt = workload.make_batch(cfg, 0, DEV, with_layers=False, with_logits=False)
    T = int(bt.q_start[-1])
    for w in cfg.windows:
        counts, first = _both(name, bt.q_start, T, max_q_len=bt.max_q_len, seq_lens=bt.seq_lens,
                              block_tables=bt.block_tables, num_blocks=bt.num_blocks,
                              max_seq_len=bt.max_seq_len, window=w)
        say("check", name, "window", w, counts, first)
        assert not any(counts.values()) and first == -1
    # acceptance's view: q_start only
    assert _both(name + " q_start", bt.q_start, T) == (dict.fromkeys(av.CHECK_KINDS, 0), -1)


def _corrupt(rng, qs, sl, bt, nb):
    """One seeded corruption of a valid descriptor; returns new copies."""
    qs, sl, bt = qs.copy(), sl.copy(), bt.copy()
    B = len(sl)
    i = int(rng.integers(0, B))
    kind = int(rng.integers(0, 9))
    if kind == 0:                      # a block id past the cache, inside the read range
        nblk = (int(sl[i]) + 15) // 16
        if nblk:
            bt[i, int(rng.integers(0, nblk))] = nb + int(rng.integers(0, 3))
    elif kind == 1:                    # a negative id inside the read range
        nblk = (int(sl[i]) + 15) // 16
        if nblk:
            bt[i, nblk - 1] = -1
    elif kind == 2:                    # garbage past the read range: not an error
        nblk = (int(sl[i]) + 15) // 16
        if nblk < bt.shape[1]:
            bt[i, nblk:] = -7
    elif kind == 3:                    # S_i below n_i
        sl[i] = int(qs[i + 1] - qs[i]) - 1 - int(rng.integers(0, 2))
    elif kind == 4:                    # S_i above the host bound
        sl[i] = int(sl.max()) + 1
    elif kind == 5:                    # q_start going backwards
        if B > 1:
            j = int(rng.integers(1, B))
            qs[j] = qs[j - 1] - 1
    elif kind == 6:                    # q_start[0] != 0
        qs[0] = 1
    elif kind == 7:                    # rows past total_q
        qs[B] += 1
    else:                              # a negative q_start entry
        qs[i] = -5
    return qs, sl, bt


@pytest.mark.parametrize("name", ["qwen3_8b", "gpt_oss_20b", "dsk_distill_8b"])
def test_corrupted_descriptors_are_counted_exactly(name):
    cfg = workload.CONFIGS[name]
    bt = workload.make_batch(cfg, 1, DEV, with_layers=False, with_logits=False)
    T = int(bt.q_start[-1])
    rng = np.random.default_rng(77)
    hits = dict.fromkeys(av.CHECK_KINDS, 0)
    for trial in range(60):
        qs, sl, tb = bt.q_start, bt.seq_lens, bt.block_tables
        for _ in range(int(rng.integers(1, 4))):
            qs, sl, tb = _corrupt(rng, qs, sl, tb, bt.num_blocks)
        w = cfg.windows[trial % len(cfg.windows)]
        mq = bt.max_q_len - (trial % 3 == 0)       # sometimes a bound one too tight
        counts, first = _both("%s trial %d" % (name, trial), qs, T, max_q_len=mq, seq_lens=sl,
                              block_tables=tb, num_blocks=bt.num_blocks,
                              max_seq_len=bt.max_seq_len, window=w)
        for k, v in counts.items():
            hits[k] += v > 0
    say("check corruptions", name, "trials with each kind", hits)
    assert all(v > 0 for v in hits.values())


def test_window_limits_the_ids_checked():
    """Ids before the first row's window start are not read, so not checked;
    one inside it is."""
    qs = np.array([0, 3, 4], dtype=np.int32)
    sl = np.array([100, 40], dtype=np.int32)
    tb = np.array([[-1, -1, -1, -1, 5, 6, 7], [1, 2, 3, -1, -1, -1, -1]], dtype=np.int32)
    # request 0: rows at 97..99, window 32 -> keys from 66: blocks 4..6
    assert _both("window", qs, 4, seq_lens=sl, block_tables=tb, num_blocks=8, max_seq_len=100,
                 window=32) == (dict.fromkeys(av.CHECK_KINDS, 0), -1)
    counts, first = _both("no window", qs, 4, seq_lens=sl, block_tables=tb, num_blocks=8,
                          max_seq_len=100, window=0)
    assert counts["block_id"] == 1 and first == 0
    counts, first = _both("wider window", qs, 4, seq_lens=sl, block_tables=tb, num_blocks=8,
                          max_seq_len=100, window=40)
    assert counts["block_id"] == 1 and first == 0


def test_many_requests_grid_strided():
    """More requests than the check's grid: every one is still tested."""
    B = 9000
    rng = np.random.default_rng(3)
    n = rng.integers(1, 5, size=B)
    qs = np.concatenate([[0], np.cumsum(n)]).astype(np.int32)
    sl = (n + rng.integers(0, 40, size=B)).astype(np.int32)
    tb = np.arange(B * 3, dtype=np.int32).reshape(B, 3)
    bad = [5, 4096, 8191, 8999]
    for i in bad:
        tb[i, (int(sl[i]) - 1) // 16] = -1
    counts, first = _both("9000 requests", qs, int(qs[-1]), seq_lens=sl, block_tables=tb,
                          num_blocks=B * 3, max_seq_len=int(sl.max()))
    assert counts["block_id"] == len(bad) and first == bad[0]


def test_binding_refuses_a_bad_batch_before_launching():
    cfg = workload.CONFIGS["qwen3_8b"]
    b = workload.make_batch(cfg, 2, DEV, with_logits=False)
    layer = b.layers[0]
    T = int(b.q_start[-1])
    tb = b.block_tables.copy()
    tb[3, 0] = b.num_blocks                          # an id the kernels would skip
    t_tb = torch.as_tensor(tb, device=DEV)
    out = torch.full_like(layer.q, 7.0)
    with pytest.raises(av.BatchError) as e:
        av.verify_attention(layer.q, layer.k_cache, layer.v_cache, t_tb, b.t_seq_lens, b.t_q_start,
                            max_q_len=b.max_q_len, max_seq_len=b.max_seq_len, out=out, check=True)
    assert e.value.counts["block_id"] == 1 and e.value.first == 3
    torch.cuda.synchronize()
    assert bool((out == 7.0).all())                  # nothing was launched
    # the same call on the valid table passes the check and runs
    av.verify_attention(layer.q, layer.k_cache, layer.v_cache, b.t_block_tables, b.t_seq_lens,
                        b.t_q_start, max_q_len=b.max_q_len, max_seq_len=b.max_seq_len, out=out,
                        check=True)
    torch.cuda.synchronize()
    assert not bool((out == 7.0).any())

    # kv append: only the new tokens' blocks are checked
    k_new = torch.zeros((T, cfg.num_kv_heads, cfg.head_dim), dtype=layer.k_cache.dtype, device=DEV)
    kc0 = layer.k_cache.clone()
    tb2 = b.block_tables.copy()
    last = (int(b.seq_lens[5]) - 1) // 16
    tb2[5, last] = -1
    with pytest.raises(av.BatchError):
        av.verify_kv_append(k_new, k_new, layer.k_cache, layer.v_cache,
                            torch.as_tensor(tb2, device=DEV), b.t_seq_lens, b.t_q_start, check=True)
    torch.cuda.synchronize()
    assert torch.equal(layer.k_cache, kc0)
    tb2[5, last] = b.block_tables[5, last]
    tb2[5, 0] = -1                                   # an old block: not the append's business
    if last > 0:
        av.verify_kv_append(k_new, k_new, layer.k_cache.clone(), layer.v_cache.clone(),
                            torch.as_tensor(tb2, device=DEV), b.t_seq_lens, b.t_q_start, check=True)

    # acceptance: q_start must describe exactly total_q rows
    logits = torch.zeros((T, 1000), dtype=torch.bfloat16, device=DEV)
    qs = b.q_start.copy()
    qs[-1] -= 1
    with pytest.raises(av.BatchError) as e:
        av.verify_accept(logits, b.t_tokens, torch.as_tensor(qs, device=DEV), check=True)
    assert e.value.counts["rows"] == 1 and e.value.first == cfg.batch - 1
