"""GPU parity: the HIP path against the CPU oracle on the same seeded inputs.

Accept: argmax, accept lengths and emitted tokens bit-exact (rows whose top-2
gap is below 1e-3 are flagged; the generator's rows have a unique maximum, so
the strict comparison is made on every row and the flagged count is asserted).
Attention: per (row, head) vector within 2e-2 relative (bf16) / 1e-4 (fp32).
"""
from __future__ import annotations

import sys

import numpy as np
import pytest
import torch

import oracle
import paper_2608_24004_amd as av
import workload
from gpu_common import (NEAR_TIE, assert_attention_close, compact_for_rows, gpu_attention,
                        oracle_accept_all, pair_schedule, row_reach, to_host_f64)
from helpers import Paged, random_paged

pytestmark = pytest.mark.gpu
DEV = "cuda:0"


def say(*a):
    print(*a, file=sys.stderr, flush=True)


# --------------------------------------------------------------------------- accept


@pytest.mark.parametrize("seed", range(5))
@pytest.mark.parametrize("name", list(workload.CONFIGS))
def test_accept_full_size(name, seed):
    cfg = workload.CONFIGS[name]
    say("accept full", name, "seed", seed)
    bt = workload.make_batch(cfg, seed, DEV, with_layers=False)
    acc, ne, em, am = av.verify_accept(bt.logits, bt.t_tokens, bt.t_q_start)
    torch.cuda.synchronize()
    r_am, gap, r_acc, r_ne, r_em = oracle_accept_all(bt.logits, bt.q_start, bt.tokens,
                                                     workload.dtype_code(cfg.dtype))
    assert int((gap < NEAR_TIE).sum()) == 0
    np.testing.assert_array_equal(am.cpu().numpy(), r_am)
    np.testing.assert_array_equal(acc.cpu().numpy(), r_acc)
    np.testing.assert_array_equal(ne.cpu().numpy(), r_ne)
    np.testing.assert_array_equal(em.cpu().numpy(), r_em)


def _accept_case(rows_per_req, vocab, dtype, fill, seed):
    rng = np.random.default_rng(seed)
    n = np.asarray(rows_per_req)
    q_start = np.zeros(n.size + 1, dtype=np.int32)
    q_start[1:] = np.cumsum(n)
    T = int(q_start[-1])
    vals = fill(rng, (T, vocab)).astype(np.float32)
    logits = torch.as_tensor(vals).to(workload.torch_dtype(dtype))
    host = workload.host_storage(logits)
    am_ref, _ = oracle.argmax(host, workload.dtype_code(dtype), with_gap=False)
    # plant long accepted runs so the scan crosses 64-row chunks
    tokens = rng.integers(0, vocab, size=T).astype(np.int32)
    for i in range(n.size):
        q0 = q_start[i]
        J = int(rng.integers(0, max(1, n[i])))
        for j in range(max(0, n[i] - 1)):
            if j < J:
                tokens[q0 + j + 1] = am_ref[q0 + j]
    return logits, tokens, q_start


def _ties(rng, shape):
    return rng.integers(-3, 4, size=shape)


def _specials(rng, shape):
    x = rng.standard_normal(shape)
    T, V = shape
    for r in range(T):
        kind = r % 6
        if kind == 0:
            x[r, rng.integers(0, V, size=2)] = np.nan
        elif kind == 1:
            x[r] = -np.inf
        elif kind == 2:
            x[r] = -np.abs(x[r]) - 1
            x[r, rng.integers(0, V)] = -0.0
            x[r, rng.integers(0, V)] = 0.0
        elif kind == 3:
            x[r, rng.integers(0, V, size=3)] = np.inf
        elif kind == 4:
            x[r] = 0.0
    return x


@pytest.mark.parametrize("dtype", ["bf16", "f32"])
@pytest.mark.parametrize("vocab", [1, 7, 8, 1000, 8193, 40000, 151936])
@pytest.mark.parametrize("fill", [_ties, _specials], ids=["ties", "specials"])
def test_accept_edge_cases(dtype, vocab, fill):
    rows = [1, 3, 0, 9, 70, 1, 33, 0, 2]   # includes empty requests and > 64 rows
    if vocab >= 40000:
        rows = [1, 70, 0, 5]
    logits, tokens, q_start = _accept_case(rows, vocab, dtype, fill, seed=vocab)
    say("accept edge", dtype, vocab, fill.__name__)
    acc, ne, em, am = av.verify_accept(logits.to(DEV), torch.as_tensor(tokens, device=DEV),
                                       torch.as_tensor(q_start, device=DEV))
    torch.cuda.synchronize()
    r_am, _, r_acc, r_ne, r_em = oracle_accept_all(logits, q_start, tokens,
                                                   workload.dtype_code(dtype))
    np.testing.assert_array_equal(am.cpu().numpy(), r_am)
    np.testing.assert_array_equal(acc.cpu().numpy(), r_acc)
    np.testing.assert_array_equal(ne.cpu().numpy(), r_ne)
    np.testing.assert_array_equal(em.cpu().numpy(), r_em)


def test_accept_strided_rows():
    # logits rows with padding after the vocabulary (row stride > vocab)
    V, stride = 1000, 1024
    full = torch.randn(40, stride, device=DEV).to(torch.bfloat16)
    view = full[:, :V]
    q_start = torch.tensor([0, 9, 40], dtype=torch.int32, device=DEV)
    tokens = torch.randint(0, V, (40,), dtype=torch.int32, device=DEV)
    lib = av.library()
    import ctypes
    am = torch.empty(40, dtype=torch.int32, device=DEV)
    acc = torch.empty(2, dtype=torch.int32, device=DEV)
    ne = torch.empty(2, dtype=torch.int32, device=DEV)
    em = torch.empty(40, dtype=torch.int32, device=DEV)
    nbytes = av.accept_workspace_size(2, 40, V, av.BF16)
    ws = torch.empty(nbytes, dtype=torch.uint8, device=DEV)
    p = lambda t: ctypes.c_void_p(t.data_ptr())
    rc = lib.verify_accept(2, 40, V, stride, av.BF16, p(full), p(tokens), p(q_start), p(am), p(acc),
                           p(ne), p(em), p(ws), nbytes,
                           ctypes.c_void_p(torch.cuda.current_stream().cuda_stream))
    assert rc == 0
    torch.cuda.synchronize()
    ref, _ = oracle.argmax(workload.host_storage(view.contiguous()), av.BF16, with_gap=False)
    np.testing.assert_array_equal(am.cpu().numpy(), ref)


# --------------------------------------------------------------------------- attention


def _to_dev(p: Paged):
    return dict(q=p.q.to(DEV), kc=p.k_cache.to(DEV), vc=p.v_cache.to(DEV),
                bt=torch.as_tensor(p.block_tables, device=DEV),
                sl=torch.as_tensor(p.seq_lens, device=DEV),
                qs=torch.as_tensor(p.q_start, device=DEV))


def _check_paged(p: Paged, split=0, what=""):
    d = _to_dev(p)
    out = gpu_attention(d["q"], d["kc"], d["vc"], d["bt"], d["sl"], d["qs"],
                        max_q_len=int(np.diff(p.q_start).max()), max_seq_len=int(p.seq_lens.max()),
                        window=p.window, split=split)
    ref = oracle.attention(**p.oracle_args())
    return assert_attention_close(to_host_f64(out), ref, p.dtype, what)


SHAPES = [(8, 2, 64), (32, 8, 128), (64, 8, 64), (4, 4, 128), (8, 1, 128), (16, 2, 64)]


@pytest.mark.parametrize("dtype", ["bf16", "f32"])
@pytest.mark.parametrize("hq,hkv,d", [(8, 2, 64), (32, 8, 128)])
@pytest.mark.parametrize("split", [0, 2])
def test_attention_rows_past_max_q_len(dtype, hq, hkv, d, split):
    """max_q_len below a request's row count: the rows the launch reaches
    (computed on the host from the plan) match the oracle, the rest are NaN."""
    say("attn max_q_len too small", dtype, hq, hkv, d, split)
    p = random_paged(num_q_heads=hq, num_kv_heads=hkv, head_dim=d, dtype=dtype,
                     contexts=[40, 300, 5, 77], drafts=[8, 2, 16, 0], seed=hq + d)
    dv = _to_dev(p)
    max_q_len = 3
    out = gpu_attention(dv["q"], dv["kc"], dv["vc"], dv["bt"], dv["sl"], dv["qs"],
                        max_q_len=max_q_len, max_seq_len=int(p.seq_lens.max()), split=split)
    plan = av.attention_plan(dv["q"], dv["kc"], dv["bt"], max_q_len=max_q_len,
                             max_seq_len=int(p.seq_lens.max()), kv_split_blocks=split)
    got = to_host_f64(out)
    ref = oracle.attention(**p.oracle_args())
    G = hq // hkv
    reached = np.zeros((p.total_q, hq), dtype=bool)
    for i in range(len(p.seq_lens)):
        n_i = int(p.q_start[i + 1] - p.q_start[i])
        reach = row_reach(plan, G * n_i)
        for j in range(n_i):
            for h in range(hq):
                reached[p.q_start[i] + j, h] = j * G + h % G < reach
    assert (~reached).any() and reached.any()
    assert_attention_close(got[reached], ref[reached], dtype, "reached rows")
    assert np.isnan(got[~reached]).all()


@pytest.mark.parametrize("dtype", ["bf16", "f32"])
@pytest.mark.parametrize("hq,hkv,d", SHAPES)
@pytest.mark.parametrize("window", [0, 5, 128])
def test_attention_ragged_small(dtype, hq, hkv, d, window):
    rng = np.random.default_rng(hq * 7 + d + window)
    drafts = [0, 1, 2, 4, 8, 16, 32, 3, 0, 7]
    contexts = [0, 1, 15, 16, 31, 200, 600, 47, 333, 129]
    rng.shuffle(drafts)
    say("attn ragged", dtype, hq, hkv, d, window)
    p = random_paged(num_q_heads=hq, num_kv_heads=hkv, head_dim=d, dtype=dtype,
                     contexts=contexts, drafts=drafts, window=window, seed=int(rng.integers(1 << 30)))
    for split in (0, 1, 3):
        _check_paged(p, split=split, what="split=%d" % split)


@pytest.mark.parametrize("k", list(range(0, 33)))
def test_attention_every_draft_length(k):
    say("attn k", k)
    p = random_paged(num_q_heads=32, num_kv_heads=8, head_dim=128, dtype="bf16",
                     contexts=[5, 100, 517], drafts=[k, k, k], seed=k)
    _check_paged(p, split=4)


@pytest.mark.parametrize("hq,hkv", [(8, 2), (16, 2)])
@pytest.mark.parametrize("k", [0, 1, 3, 4, 5, 7, 8, 11, 12, 15, 16, 20, 24, 28, 31, 32])
def test_attention_every_head_dim_64_shape(hq, hkv, k):
    # head dim 64: the row count G (k + 1) walks every kernel shape of the
    # table, one to seventeen 16-row tiles
    say("attn d64 k", hq, hkv, k)
    p = random_paged(num_q_heads=hq, num_kv_heads=hkv, head_dim=64, dtype="bf16",
                     contexts=[5, 100, 517, 1100], drafts=[k, k, k, k], seed=k + hq)
    for split in (0, 4):
        _check_paged(p, split=split, what="d64 k=%d split=%d" % (k, split))


def test_attention_spiky_masks():
    # Large-norm queries and a planted key that matches them at a position just
    # after some rows: a causal or window leak changes those rows by O(1).
    rng = np.random.default_rng(9)
    Hq, Hkv, D = 8, 2, 128
    for window in (0, 24):
        ctx, k = [60, 33], [12, 20]
        k_log, v_log = [], []
        for L, kk in zip(ctx, k):
            S = L + kk + 1
            K = rng.standard_normal((S, Hkv, D)) * 0.1
            V = rng.standard_normal((S, Hkv, D))
            K[S - 3] = 3.0          # huge score for every query pointing along +1
            V[S - 3] = 50.0
            if window:
                K[S - kk - 1 - window] = 3.0   # just outside the first row's window
                V[S - kk - 1 - window] = -50.0
            k_log.append(K)
            v_log.append(V)
        T = sum(kk + 1 for kk in k)
        q = np.abs(rng.standard_normal((T, Hq, D))) * 3.0
        p = Paged(num_q_heads=Hq, num_kv_heads=Hkv, head_dim=D, dtype="bf16", k_logical=k_log,
                  v_logical=v_log, q=q, num_drafts=k, window=window, seed=3)
        for split in (0, 1, 2):
            _check_paged(p, split=split, what="spiky w=%d split=%d" % (window, split))


def test_attention_split_invariance_and_degenerate():
    # one request with no context (S = n), single keys, and requests of all sizes
    p = random_paged(num_q_heads=32, num_kv_heads=8, head_dim=128, dtype="bf16",
                     contexts=[0, 0, 1, 2000, 4000], drafts=[0, 5, 0, 9, 1], seed=77)
    for split in (0, 1, 2, 5, 16, 64, 1000):
        say("attn split", split)
        _check_paged(p, split=split, what="split=%d" % split)


@pytest.mark.parametrize("dtype", ["bf16", "f32"])
@pytest.mark.parametrize("hq,hkv,d", [(32, 8, 128), (8, 2, 64)])
def test_attention_requests_without_rows(dtype, hq, hkv, d):
    # requests with no scored row (n_i = 0, with and without cached keys)
    # between ordinary ones: they get no work and leave the others unchanged
    say("attn empty requests", dtype, hq, hkv, d)
    p = random_paged(num_q_heads=hq, num_kv_heads=hkv, head_dim=d, dtype=dtype,
                     contexts=[100, 50, 0, 700, 33, 0, 1200], drafts=[3, -1, 0, -1, 8, -1, 5],
                     seed=hq + d)
    assert (np.diff(p.q_start) == 0).sum() == 3
    for split in (0, 1, 3):
        _check_paged(p, split=split, what="empty requests split=%d" % split)


@pytest.mark.parametrize("dtype,hq,hkv,d", [("bf16", 32, 8, 128), ("bf16", 8, 2, 64), ("f32", 8, 2, 64)])
def test_attention_batches_above_the_inline_schedule(dtype, hq, hkv, d):
    # more than 256 requests: the per-request unit offsets come from the
    # separate one-workgroup schedule launch instead of each workgroup's scan
    rng = np.random.default_rng(300 + d)
    B = 300
    contexts = rng.integers(0, 200, size=B)
    drafts = rng.integers(0, 9, size=B)
    drafts[::37] = -1          # a few requests without scored rows
    say("attn 300 requests", dtype, hq, hkv, d)
    p = random_paged(num_q_heads=hq, num_kv_heads=hkv, head_dim=d, dtype=dtype,
                     contexts=contexts.tolist(), drafts=drafts.tolist(), seed=int(d))
    for split in (0, 1, 3):
        _check_paged(p, split=split, what="300 requests split=%d" % split)


@pytest.mark.parametrize("window,with_sinks", [(0, False), (40, True)])
def test_attention_batches_above_the_inline_schedule_in_row_classes(window, with_sinks):
    # more than 256 requests with draft lengths on both sides of the row-class
    # boundary: two launches, each with its own schedule launch and merge,
    # with a sliding window and sinks in one case
    rng = np.random.default_rng(301 + window)
    B = 300
    contexts = rng.integers(0, 200, size=B)
    drafts = rng.integers(0, 21, size=B)
    drafts[::37] = -1
    say("attn 300 requests, row classes", window, with_sinks)
    p = random_paged(num_q_heads=32, num_kv_heads=8, head_dim=128, dtype="bf16",
                     contexts=contexts.tolist(), drafts=drafts.tolist(), window=window, seed=7)
    sinks = (rng.standard_normal(32) * 2.0).astype(np.float32) if with_sinks else None
    d = _to_dev(p)
    max_q_len = int(np.diff(p.q_start).max())
    plan = av.attention_plan(d["q"], d["kc"], d["bt"], max_q_len=max_q_len,
                             max_seq_len=int(p.seq_lens.max()), sliding_window=window)
    assert len(plan["classes"]) == 2
    ref = oracle.attention(sinks=None if sinks is None else sinks.astype(np.float64), **p.oracle_args())
    for split in (0, 3):
        out = gpu_attention(d["q"], d["kc"], d["vc"], d["bt"], d["sl"], d["qs"], max_q_len=max_q_len,
                            max_seq_len=int(p.seq_lens.max()), window=window, split=split,
                            sinks=None if sinks is None else torch.as_tensor(sinks, device=DEV))
        assert_attention_close(to_host_f64(out), ref, "bf16", "300 requests row classes split=%d" % split)


@pytest.mark.parametrize("hq,hkv,d", [(64, 8, 64), (32, 8, 128), (16, 2, 64)])
def test_attention_long_pairs(hq, hkv, d):
    # pairs of 64 blocks and more run on the one-wavefront shapes (72 rows at
    # D 64, 36 rows at D 128); shorter pairs in the same batch, every row checked
    say("attn long pairs", hq, hkv, d)
    p = random_paged(num_q_heads=hq, num_kv_heads=hkv, head_dim=d, dtype="bf16",
                     contexts=[1500, 3100, 40, 1030, 0], drafts=[8, 8, 3, 8, 8], seed=hq + d)
    for split in (0, 1, 3, 100):
        _check_paged(p, split=split, what="long pairs split=%d" % split)


@pytest.mark.parametrize("contexts", [[1500, 3100, 40, 1030, 900, 2000, 0, 1200],
                                      [40, 300, 77, 5, 200, 130, 0, 60]])
def test_attention_row_classes(contexts):
    """A ragged batch at head dim 128 whose largest request needs the
    four-wavefront shape runs in two launches: requests with at most 48 rows
    per KV head (12 rows at Hq/Hkv = 4, the boundary itself included) on the
    three-tile shape (long contexts: one wavefront; short: two), the others on
    the four-wavefront shape; every row of both against the oracle."""
    say("attn row classes", contexts[:3])
    drafts = [11, 12, 0, 32, 20, 3, 11, 40]   # 48 | 52 | 4 | 132 | 84 | 16 | 48 | 164 rows
    p = random_paged(num_q_heads=32, num_kv_heads=8, head_dim=128, dtype="bf16",
                     contexts=contexts, drafts=drafts, seed=len(contexts) + contexts[0])
    dv = _to_dev(p)
    plan = av.attention_plan(dv["q"], dv["kc"], dv["bt"], max_q_len=int(np.diff(p.q_start).max()),
                             max_seq_len=int(p.seq_lens.max()))
    assert len(plan["classes"]) == 2 and plan["classes"][0]["rows_hi"] == 48
    for split in (0, 1, 3):
        _check_paged(p, split=split, what="row classes split=%d" % split)


@pytest.mark.parametrize("dtype", ["bf16", "f32"])
@pytest.mark.parametrize("hq,hkv,d,window", [(32, 8, 128, 0), (64, 8, 64, 128), (16, 2, 64, 20)])
def test_attention_skips_unmapped_blocks(dtype, hq, hkv, d, window):
    """Block ids outside [0, num_blocks) (negative, or past the cache) hold no
    keys: every vector against the oracle, which leaves those positions out of
    the softmax, across split settings; a request whose only block is unmapped
    gets zeros.  The drafts (up to 32) put the batch in two row classes at
    head dim 128."""
    say("attn unmapped blocks", dtype, hq, hkv, d, window)
    p = random_paged(num_q_heads=hq, num_kv_heads=hkv, head_dim=d, dtype=dtype,
                     contexts=[400, 70, 3, 900, 33], drafts=[5, 32, 4, 9, 0], window=window,
                     seed=hq + d + window)
    bt = p.block_tables.copy()
    bt[0, 3] = -1                          # request 0: a block in the middle
    bt[1, 5] = p.num_blocks + 2            # request 1: the new tokens' last block
    bt[2, 0] = -1                          # request 2: its only block
    bt[3, 0] = p.num_blocks                # request 3: the first block
    bt[3, (int(p.seq_lens[3]) - 1) // 16] = -7   # and the last
    dv = _to_dev(p)
    t_bt = torch.as_tensor(bt, device=DEV)
    args = p.oracle_args()
    args.update(block_tables=bt)
    ref = oracle.attention(**args)
    q0, q1 = p.q_start[2], p.q_start[3]
    assert np.all(ref[q0:q1] == 0.0)
    for split in (0, 1, 3):
        out = gpu_attention(dv["q"], dv["kc"], dv["vc"], t_bt, dv["sl"], dv["qs"],
                            max_q_len=int(np.diff(p.q_start).max()),
                            max_seq_len=int(p.seq_lens.max()), window=window, split=split)
        got = to_host_f64(out)
        assert_attention_close(got, ref, dtype, "unmapped split=%d" % split)
        assert np.all(got[q0:q1] == 0.0)


SEEDS = range(5)
EVERY_PAIR = ["qwen3_8b", "dsk_distill_8b", "gpt_oss_20b"]


def _attention_layers(bt):
    for layer in bt.layers:
        out = gpu_attention(layer.q, layer.k_cache, layer.v_cache, bt.t_block_tables,
                            bt.t_seq_lens, bt.t_q_start, max_q_len=bt.max_q_len,
                            max_seq_len=bt.max_seq_len, window=layer.window, sinks=layer.sinks)
        plan = av.attention_plan(layer.q, layer.k_cache, bt.t_block_tables, max_q_len=bt.max_q_len,
                                 max_seq_len=bt.max_seq_len, sliding_window=layer.window)
        yield layer, out, plan


@pytest.mark.parametrize("seed", SEEDS)
@pytest.mark.parametrize("name", EVERY_PAIR)
def test_attention_full_size_every_vector(name, seed):
    """Every (row, head) output vector of every layer at full size, in the
    launch configuration bench.py times, for five seeds; the pairs that
    workgroup range boundaries cut (merged by attn_combine_slots) are among
    them, and their count is asserted."""
    cfg = workload.CONFIGS[name]
    say("attn full every vector", name, "seed", seed)
    bt = workload.make_batch(cfg, seed, DEV, with_logits=False)
    code = workload.dtype_code(cfg.dtype)
    for layer, out, plan in _attention_layers(bt):
        got = to_host_f64(out)
        ref = oracle.attention(num_q_heads=cfg.num_q_heads, num_kv_heads=cfg.num_kv_heads,
                               head_dim=cfg.head_dim, sliding_window=layer.window, scale=0.0,
                               dtype=code, q=workload.host_storage(layer.q),
                               k_cache=workload.host_storage(layer.k_cache),
                               v_cache=workload.host_storage(layer.v_cache),
                               block_tables=bt.block_tables, seq_lens=bt.seq_lens,
                               q_start=bt.q_start,
                               sinks=None if layer.sinks is None else layer.sinks.cpu().numpy())
        err = assert_attention_close(got, ref, cfg.dtype, "%s seed %d window=%d" % (
            name, seed, layer.window))
        pairs = pair_schedule(bt, layer, plan)
        cut = sum(p[3] for p in pairs)
        say("  window", layer.window, "vectors", got.shape[0] * got.shape[1], "max rel err", err,
            "pairs", len(pairs), "cut", cut, "plan", plan)
        assert cut > 0
        del out
    torch.cuda.empty_cache()


@pytest.mark.parametrize("seed", SEEDS)
def test_attention_long_context_sampled(seed):
    """The long-context stress at full size (43 GB of KV): every (row, head)
    of sampled requests -- the fewest and most drafts, the longest context,
    and a request with a pair cut by a workgroup range boundary -- plus random
    extra vectors."""
    name = "long_context"
    cfg = workload.CONFIGS[name]
    say("attn long context", "seed", seed)
    bt = workload.make_batch(cfg, seed, DEV, with_logits=False)
    for layer, out, plan in _attention_layers(bt):
        pairs = pair_schedule(bt, layer, plan)
        cut_reqs = sorted({p[0] for p in pairs if p[3]})
        assert cut_reqs
        n = np.diff(bt.q_start)
        want = {int(np.argmin(n)), int(np.argmax(n)), int(np.argmax(bt.seq_lens)),
                cut_reqs[seed % len(cut_reqs)]}
        rng = np.random.default_rng(seed)
        others = [i for i in rng.permutation(len(n)) if i not in want]
        reqs = sorted(want | set(others[:2]))
        Hq = cfg.num_q_heads
        rows = np.concatenate([np.repeat(np.arange(bt.q_start[i], bt.q_start[i + 1]), Hq)
                               for i in reqs]).astype(np.int32)
        heads = np.concatenate([np.tile(np.arange(Hq), int(n[i])) for i in reqs]).astype(np.int32)
        extra = rng.integers(0, bt.total_q, size=64).astype(np.int32)
        xh = rng.integers(0, Hq, size=64).astype(np.int32)
        rows, heads = np.concatenate([rows, extra]), np.concatenate([heads, xh])
        got = to_host_f64(out[torch.as_tensor(rows, device=DEV, dtype=torch.int64),
                              torch.as_tensor(heads, device=DEV, dtype=torch.int64)])
        args, rows_c = compact_for_rows(bt, layer, rows)
        ref = oracle.attention(rows=rows_c, heads=heads, **args)
        err = assert_attention_close(got, ref, cfg.dtype, "%s seed %d" % (name, seed))
        say("  requests", reqs, "cut-pair requests", len(cut_reqs), "vectors", rows.size,
            "max rel err", err)
        assert torch.isfinite(out.float()).all()
        del out
    torch.cuda.empty_cache()
