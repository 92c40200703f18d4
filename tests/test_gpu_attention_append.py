"""verify_attention_append (the KV append fused into the attention launch) on
the GPU.

The new tokens' K/V are random and differ from what the cache holds at their
slots, so a kernel that read the stale cache instead of k_new / v_new, or
stored a token in the wrong slot, fails.  For every case:

* the cache after the call equals the oracle's append bit for bit;
* the output matches the oracle's attention over the appended cache (the
  attention tolerance);
* with a fixed split (kv_split_blocks > 0, so the same partition of the walk)
  and on the fp32 path, the output equals verify_kv_append followed by
  verify_attention bit for bit.
"""
from __future__ import annotations

import sys

import numpy as np
import pytest
import torch

import oracle
import paper_2608_24004_amd as av
import workload
from gpu_common import assert_attention_close, rel_err_rows, row_reach, to_host_f64
from helpers import random_paged

pytestmark = pytest.mark.gpu
DEV = "cuda:0"


def say(*a):
    print(*a, file=sys.stderr, flush=True)


def _bits(t):
    return t.reshape(-1).view(torch.uint8)


def _new_kv(T, hkv, d, dtype, seed):
    g = torch.Generator().manual_seed(seed)
    tdt = workload.torch_dtype(dtype)
    return (torch.randn((T, hkv, d), generator=g).to(tdt),
            torch.randn((T, hkv, d), generator=g).to(tdt))


def _case(p, *, bt=None, sl=None, split=0, sinks=None, what="", check_oracle=True):
    bt = p.block_tables if bt is None else bt
    sl = p.seq_lens if sl is None else sl
    code = workload.dtype_code(p.dtype)
    k_new, v_new = _new_kv(p.total_q, p.Hkv, p.D, p.dtype, seed=p.total_q + split)
    kc_ref, vc_ref = oracle.kv_append(num_kv_heads=p.Hkv, head_dim=p.D, dtype=code,
                                      k_new=workload.host_storage(k_new),
                                      v_new=workload.host_storage(v_new), block_tables=bt,
                                      seq_lens=sl, q_start=p.q_start,
                                      k_cache=workload.host_storage(p.k_cache),
                                      v_cache=workload.host_storage(p.v_cache))
    assert not np.array_equal(kc_ref, workload.host_storage(p.k_cache)), "nothing to append"
    d = lambda a: torch.as_tensor(a, device=DEV)
    t_bt, t_sl, t_qs = d(bt), d(sl), d(p.q_start)
    q = p.q.to(DEV)
    kn, vn = k_new.to(DEV), v_new.to(DEV)
    mq, ms = int(np.diff(p.q_start).max()), int(sl.max())
    sk = None if sinks is None else torch.as_tensor(sinks, device=DEV)
    kw = dict(max_q_len=mq, max_seq_len=ms, sliding_window=p.window, kv_split_blocks=split,
              sinks=sk)
    # fused
    kc, vc = p.k_cache.to(DEV), p.v_cache.to(DEV)
    out = av.verify_attention_append(q, kn, vn, kc, vc, t_bt, t_sl, t_qs, **kw)
    torch.cuda.synchronize()
    assert np.array_equal(workload.host_storage(kc), kc_ref), what + ": k cache"
    assert np.array_equal(workload.host_storage(vc), vc_ref), what + ": v cache"
    err = 0.0
    if check_oracle:
        args = p.oracle_args()
        args.update(k_cache=kc_ref, v_cache=vc_ref, block_tables=bt, seq_lens=sl, sinks=sinks)
        ref = oracle.attention(**args)
        err = assert_attention_close(to_host_f64(out), ref, p.dtype, what)
    # append, then attention
    kc2, vc2 = p.k_cache.to(DEV), p.v_cache.to(DEV)
    av.verify_kv_append(kn, vn, kc2, vc2, t_bt, t_sl, t_qs)
    out2 = av.verify_attention(q, kc2, vc2, t_bt, t_sl, t_qs, **kw)
    torch.cuda.synchronize()
    same = torch.equal(_bits(out), _bits(out2))
    if split > 0 or p.dtype == "f32":
        assert same, what + ": differs from append + attention"
    else:
        assert_attention_close(to_host_f64(out), to_host_f64(out2), p.dtype, what + " vs append + attention")
    say("  ", what, "max rel err %.2e" % err, "bitwise equal to append + attention:", same)


SHAPES = [(32, 8, 128, 0), (64, 8, 64, 128), (16, 2, 64, 5), (8, 1, 128, 0)]


@pytest.mark.parametrize("dtype", ["bf16", "f32"])
@pytest.mark.parametrize("hq,hkv,d,window", SHAPES)
def test_fused_append_matches_oracle(dtype, hq, hkv, d, window):
    say("attention append", dtype, hq, hkv, d, window)
    p = random_paged(num_q_heads=hq, num_kv_heads=hkv, head_dim=d, dtype=dtype,
                     contexts=[0, 17, 250, 31, 1000, 3], drafts=[5, 0, 32, 16, 8, 1], window=window,
                     seed=hq + d + window)
    sinks = None
    if window:
        sinks = np.random.default_rng(window).standard_normal(hq).astype(np.float32)
    for split in (0, 1, 3):
        _case(p, split=split, sinks=sinks, what="%s %s split %d" % (dtype, (hq, hkv, d, window), split))


def test_fused_append_row_classes():
    """A ragged batch in two row classes (both persistent shapes)."""
    say("attention append row classes")
    p = random_paged(num_q_heads=32, num_kv_heads=8, head_dim=128, dtype="bf16",
                     contexts=[700, 40, 1500, 3000, 9, 260, 2048, 5000],
                     drafts=[11, 12, 0, 32, 20, 3, 11, 40], seed=21)
    for split in (0, 2):
        _case(p, split=split, what="row classes split %d" % split)


def test_fused_append_scheduled_batch():
    """300 requests: the separate schedule launch runs first."""
    rng = np.random.default_rng(8)
    say("attention append 300 requests")
    p = random_paged(num_q_heads=32, num_kv_heads=8, head_dim=128, dtype="bf16",
                     contexts=list(rng.integers(0, 300, size=300)),
                     drafts=list(rng.integers(0, 9, size=300)), seed=22)
    _case(p, split=0, what="300 requests")
    _case(p, split=4, what="300 requests split 4")


@pytest.mark.parametrize("dtype", ["bf16", "f32"])
def test_fused_append_skips_rows_without_a_slot(dtype):
    """Rows with a negative position (S < n) or on a block id outside the
    cache store nothing, as in verify_kv_append, and the unmapped blocks hold
    no keys for the attention."""
    say("attention append skips", dtype)
    p = random_paged(num_q_heads=16, num_kv_heads=4, head_dim=64, dtype=dtype,
                     contexts=[40, 100, 20, 64], drafts=[7, 3, 9, 4], seed=11)
    bt = p.block_tables.copy()
    sl = p.seq_lens.copy()
    bt[0, 2] = -1                       # positions 32..47 of request 0: no block
    bt[1, 6] = p.num_blocks + 5         # request 1's new tokens: id out of range
    sl[2] = 5                           # request 2: 10 rows but 5 keys
    for split in (0, 1):
        _case(p, bt=bt, sl=sl, split=split, what="%s skips split %d" % (dtype, split))


@pytest.mark.parametrize("name", ["qwen3_8b", "dsk_distill_8b", "gpt_oss_20b"])
def test_fused_append_full_size(name):
    """Full-size workloads in the launch configuration of verify_attention:
    the cache bit for bit against verify_kv_append, the output against
    verify_kv_append + verify_attention (the fused launch may partition the
    walk differently: attention tolerance), every vector."""
    cfg = workload.CONFIGS[name]
    say("attention append full", name)
    b = workload.make_batch(cfg, 0, DEV, with_logits=False)
    T = b.total_q
    for layer in b.layers:
        k_new, v_new = (t.to(DEV) for t in _new_kv(T, cfg.num_kv_heads, cfg.head_dim, cfg.dtype, 5))
        kw = dict(max_q_len=b.max_q_len, max_seq_len=b.max_seq_len, sliding_window=layer.window,
                  sinks=layer.sinks)
        kc2, vc2 = layer.k_cache.clone(), layer.v_cache.clone()
        av.verify_kv_append(k_new, v_new, kc2, vc2, b.t_block_tables, b.t_seq_lens, b.t_q_start)
        ref = av.verify_attention(layer.q, kc2, vc2, b.t_block_tables, b.t_seq_lens, b.t_q_start, **kw)
        out = av.verify_attention_append(layer.q, k_new, v_new, layer.k_cache, layer.v_cache,
                                         b.t_block_tables, b.t_seq_lens, b.t_q_start, **kw)
        torch.cuda.synchronize()
        assert torch.equal(_bits(layer.k_cache), _bits(kc2)) and torch.equal(_bits(layer.v_cache), _bits(vc2))
        del kc2, vc2
        err = rel_err_rows(out.float().cpu().numpy(), ref.float().cpu().numpy().astype(np.float64))
        say("  window", layer.window, "max rel err vs append + attention %.2e" % err.max(),
            "bitwise", torch.equal(_bits(out), _bits(ref)))
        assert float(err.max()) <= 2e-2


@pytest.mark.parametrize("dtype", ["bf16", "f32"])
def test_fused_append_writes_every_new_token_past_max_q_len(dtype):
    """A request with more rows than max_q_len promised: the rows past the
    launch's reach are NaN, as in verify_attention, but the append still
    stores every new token (the walk covers all of the request's blocks)."""
    say("attention append past max_q_len", dtype)
    p = random_paged(num_q_heads=32, num_kv_heads=8, head_dim=128, dtype=dtype,
                     contexts=[300, 600, 50], drafts=[40, 2, 7], seed=41)
    code = workload.dtype_code(dtype)
    k_new, v_new = _new_kv(p.total_q, p.Hkv, p.D, dtype, seed=3)
    kc_ref, vc_ref = oracle.kv_append(num_kv_heads=p.Hkv, head_dim=p.D, dtype=code,
                                      k_new=workload.host_storage(k_new),
                                      v_new=workload.host_storage(v_new),
                                      block_tables=p.block_tables, seq_lens=p.seq_lens,
                                      q_start=p.q_start, k_cache=workload.host_storage(p.k_cache),
                                      v_cache=workload.host_storage(p.v_cache))
    d = lambda a: torch.as_tensor(a, device=DEV)
    q, kc, vc = p.q.to(DEV), p.k_cache.to(DEV), p.v_cache.to(DEV)
    mq = 4
    out = av.verify_attention_append(q, k_new.to(DEV), v_new.to(DEV), kc, vc, d(p.block_tables),
                                     d(p.seq_lens), d(p.q_start), max_q_len=mq,
                                     max_seq_len=int(p.seq_lens.max()))
    torch.cuda.synchronize()
    assert np.array_equal(workload.host_storage(kc), kc_ref)
    assert np.array_equal(workload.host_storage(vc), vc_ref)
    args = p.oracle_args()
    args.update(k_cache=kc_ref, v_cache=vc_ref)
    ref = oracle.attention(**args)
    got = to_host_f64(out)
    plan = av.attention_plan(q, kc, d(p.block_tables), max_q_len=mq, max_seq_len=int(p.seq_lens.max()))
    G = p.Hq // p.Hkv
    reached = np.zeros(got.shape[:2], dtype=bool)
    for i in range(len(p.seq_lens)):
        q0, q1 = int(p.q_start[i]), int(p.q_start[i + 1])
        reach = row_reach(plan, G * (q1 - q0))
        for j in range(q1 - q0):
            for h in range(p.Hq):
                reached[q0 + j, h] = j * G + h % G < reach
    assert not reached.all()
    assert np.isnan(got[~reached]).all()
    assert_attention_close(got[reached], ref[reached], dtype, "reached rows")
