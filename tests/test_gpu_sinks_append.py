"""Attention sinks and the KV append on the GPU against the oracle.

Sinks: the same batches as the attention parity tests with per-head sink
logits, both dtypes, with and without a window and across forced split
counts; sink -inf gives exactly the output without sinks, a huge sink zero.
KV append: the cache after verify_kv_append equals the oracle's bit for bit,
and verify_kv_append followed by verify_attention equals the oracle's
attention over the appended cache.
"""
from __future__ import annotations

import sys

import numpy as np
import pytest
import torch

import oracle
import paper_2608_24004_amd as av
import workload
from gpu_common import assert_attention_close, gpu_attention, to_host_f64
from helpers import random_paged

pytestmark = pytest.mark.gpu
DEV = "cuda:0"


def say(*a):
    print(*a, file=sys.stderr, flush=True)


def _dev(p):
    return dict(q=p.q.to(DEV), kc=p.k_cache.to(DEV), vc=p.v_cache.to(DEV),
                bt=torch.as_tensor(p.block_tables, device=DEV), sl=torch.as_tensor(p.seq_lens, device=DEV),
                qs=torch.as_tensor(p.q_start, device=DEV))


def _run(p, d, sinks, split=0):
    return gpu_attention(d["q"], d["kc"], d["vc"], d["bt"], d["sl"], d["qs"],
                         max_q_len=int(np.diff(p.q_start).max()), max_seq_len=int(p.seq_lens.max()),
                         window=p.window, split=split,
                         sinks=None if sinks is None else torch.as_tensor(sinks, dtype=torch.float32,
                                                                          device=DEV))


@pytest.mark.parametrize("dtype", ["bf16", "f32"])
@pytest.mark.parametrize("hq,hkv,d", [(32, 8, 128), (64, 8, 64), (8, 2, 64), (8, 1, 128)])
@pytest.mark.parametrize("window", [0, 128])
def test_sinks_match_oracle(dtype, hq, hkv, d, window):
    rng = np.random.default_rng(hq + d + window)
    say("sinks", dtype, hq, hkv, d, window)
    p = random_paged(num_q_heads=hq, num_kv_heads=hkv, head_dim=d, dtype=dtype,
                     contexts=[0, 1, 15, 300, 700, 40], drafts=[0, 4, 8, 2, 16, 32], window=window,
                     seed=int(rng.integers(1 << 20)))
    sinks = (rng.standard_normal(hq) * 2.0).astype(np.float32)
    ref = oracle.attention(sinks=sinks.astype(np.float64), **p.oracle_args())
    d_ = _dev(p)
    for split in (0, 1, 3):
        got = to_host_f64(_run(p, d_, sinks, split))
        assert_attention_close(got, ref, dtype, "sinks split=%d" % split)


def test_sink_limits_on_gpu():
    p = random_paged(num_q_heads=32, num_kv_heads=8, head_dim=128, dtype="bf16",
                     contexts=[50, 900], drafts=[8, 3], seed=12)
    d = _dev(p)
    for split in (0, 2):
        plain = _run(p, d, None, split)
        none = _run(p, d, np.full(32, -np.inf, dtype=np.float32), split)
        assert torch.equal(plain, none)
        huge = _run(p, d, np.full(32, 1e4, dtype=np.float32), split)
        assert float(huge.float().abs().max()) == 0.0


@pytest.mark.parametrize("dtype", ["bf16", "f32"])
@pytest.mark.parametrize("hq,hkv,d", [(32, 8, 128), (64, 8, 64)])
def test_kv_append_matches_oracle_and_feeds_attention(dtype, hq, hkv, d):
    rng = np.random.default_rng(hq + d)
    say("append", dtype, hq, hkv, d)
    p = random_paged(num_q_heads=hq, num_kv_heads=hkv, head_dim=d, dtype=dtype,
                     contexts=[0, 17, 250, 31], drafts=[5, 0, 32, 16], seed=3)
    T = p.total_q
    tdt = workload.torch_dtype(dtype)
    k_new = torch.randn((T, hkv, d), dtype=torch.float32).to(tdt)
    v_new = torch.randn((T, hkv, d), dtype=torch.float32).to(tdt)
    code = workload.dtype_code(dtype)
    kc_ref, vc_ref = oracle.kv_append(num_kv_heads=hkv, head_dim=d, dtype=code,
                                      k_new=workload.host_storage(k_new),
                                      v_new=workload.host_storage(v_new),
                                      block_tables=p.block_tables, seq_lens=p.seq_lens,
                                      q_start=p.q_start, k_cache=workload.host_storage(p.k_cache),
                                      v_cache=workload.host_storage(p.v_cache))
    dv = _dev(p)
    av.verify_kv_append(k_new.to(DEV), v_new.to(DEV), dv["kc"], dv["vc"], dv["bt"], dv["sl"], dv["qs"])
    torch.cuda.synchronize()
    assert np.array_equal(workload.host_storage(dv["kc"]), kc_ref)
    assert np.array_equal(workload.host_storage(dv["vc"]), vc_ref)
    # attention over the appended cache
    got = to_host_f64(_run(p, dv, None))
    args = p.oracle_args()
    args.update(k_cache=kc_ref, v_cache=vc_ref)
    ref = oracle.attention(**args)
    assert_attention_close(got, ref, dtype, "after append")


@pytest.mark.parametrize("dtype", ["bf16", "f32"])
def test_kv_append_skips_rows_without_a_slot(dtype):
    # rows whose position is negative (S < n), lies past the block table, or
    # maps to a block id outside [0, num_blocks) write nothing; every other
    # row lands in its slot, bit for bit as in the oracle
    hq, hkv, d = 16, 4, 64
    say("append skips", dtype)
    p = random_paged(num_q_heads=hq, num_kv_heads=hkv, head_dim=d, dtype=dtype,
                     contexts=[40, 100, 20, 64], drafts=[7, 3, 9, 4], seed=11)
    bt = p.block_tables.copy()
    sl = p.seq_lens.copy()
    bt[0, 2] = -1                       # positions 32..47 of request 0: no block
    bt[1, 1] = p.num_blocks + 5         # positions 16..31 of request 1: id out of range
    sl[2] = 5                           # request 2: 10 rows but only 5 keys, p < 0 for 5 rows
    sl[3] = bt.shape[1] * 16 + 3        # request 3: its last rows fall past the block table
    T = p.total_q
    tdt = workload.torch_dtype(dtype)
    g = torch.Generator().manual_seed(5)
    k_new = torch.randn((T, hkv, d), generator=g).to(tdt)
    v_new = torch.randn((T, hkv, d), generator=g).to(tdt)
    code = workload.dtype_code(dtype)
    kc_ref, vc_ref = oracle.kv_append(num_kv_heads=hkv, head_dim=d, dtype=code,
                                      k_new=workload.host_storage(k_new),
                                      v_new=workload.host_storage(v_new),
                                      block_tables=bt, seq_lens=sl, q_start=p.q_start,
                                      k_cache=workload.host_storage(p.k_cache),
                                      v_cache=workload.host_storage(p.v_cache))
    kc, vc = p.k_cache.to(DEV), p.v_cache.to(DEV)
    av.verify_kv_append(k_new.to(DEV), v_new.to(DEV), kc, vc, torch.as_tensor(bt, device=DEV),
                        torch.as_tensor(sl, device=DEV), torch.as_tensor(p.q_start, device=DEV))
    torch.cuda.synchronize()
    assert np.array_equal(workload.host_storage(kc), kc_ref)
    assert np.array_equal(workload.host_storage(vc), vc_ref)
    # something was skipped and something was written
    assert not np.array_equal(kc_ref, workload.host_storage(p.k_cache))
