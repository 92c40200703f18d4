"""GPU parity of the fused LM head + greedy acceptance (verify_lmhead_accept)
against the CPU oracle on the same seeded bf16 inputs.

The kernel sums the bf16 products in fp32, the oracle in double, so two logits
closer than fp32 rounding may compare either way.  Rows whose oracle top-2 gap
is below 1e-3 are flagged and left out of the argmax comparison; a request is
compared for acceptance when its rows 0 .. m (m = the oracle's accept length)
are unflagged.  Everything else is bit-exact: argmax, accept length, emitted
count and emitted tokens.  At full size the oracle checks sampled rows and
whole requests; a float32 torch product on the GPU checks every row.
"""
from __future__ import annotations

import sys

import numpy as np
import pytest
import torch

import oracle
import paper_2608_24004_amd as av
import workload
from gpu_common import NEAR_TIE

pytestmark = pytest.mark.gpu
DEV = "cuda:0"


def say(*a):
    print(*a, file=sys.stderr, flush=True)


def _batch(rows_per_req, vocab, seed, match=0.7):
    """q_start, designated tokens and drafts planted as them with probability `match`."""
    rng = np.random.default_rng(seed)
    n = np.asarray(rows_per_req, dtype=np.int64)
    q_start = np.zeros(n.size + 1, dtype=np.int32)
    q_start[1:] = np.cumsum(n)
    T = int(q_start[-1])
    des = rng.integers(0, vocab, size=T).astype(np.int32)
    tokens = rng.integers(0, vocab, size=T).astype(np.int32)
    for i in range(n.size):
        for j in range(int(n[i]) - 1):
            r = int(q_start[i]) + j
            if rng.random() < match:
                tokens[r + 1] = des[r]
    return q_start, des, tokens


def _run(hidden, weight, tokens, q_start):
    d = lambda a: torch.as_tensor(a, device=DEV)
    acc, ne, em, am = av.verify_lmhead_accept(hidden, weight, d(tokens), d(q_start))
    torch.cuda.synchronize()
    return am.cpu().numpy(), acc.cpu().numpy(), ne.cpu().numpy(), em.cpu().numpy()


def _check(got, ref_am, ref_gap, q_start, tokens, rows=None, what=""):
    """Compare the GPU outputs with the oracle on `rows` (all if None);
    acceptance for every request whose rows are all in `rows`."""
    am, acc, ne, em = got
    T = int(q_start[-1])
    rows = np.arange(T) if rows is None else np.asarray(rows)
    flagged = ref_gap < NEAR_TIE          # NaN gaps (NaN rows) are not flagged
    ok = ~flagged
    np.testing.assert_array_equal(am[rows][ok], ref_am[ok], err_msg=what + " argmax")
    full = np.full(T, -1, dtype=np.int64)
    full[rows] = ref_am
    fl = np.zeros(T, dtype=bool)
    fl[rows] = flagged
    have = np.zeros(T, dtype=bool)
    have[rows] = True
    checked = 0
    for i in range(q_start.size - 1):
        q0, q1 = int(q_start[i]), int(q_start[i + 1])
        if q1 == q0 or not have[q0:q1].all():
            continue
        r_acc, r_ne, r_em = oracle.accept(np.array([0, q1 - q0], dtype=np.int32), tokens[q0:q1],
                                          full[q0:q1].astype(np.int32))
        m = int(r_acc[0])
        if fl[q0:q0 + m + 1].any():
            continue
        assert acc[i] == m and ne[i] == r_ne[0], (what, i)
        np.testing.assert_array_equal(em[q0:q1], r_em, err_msg="%s request %d" % (what, i))
        checked += 1
    return int(flagged.sum()), checked


CASES = [
    # rows per request, hidden size, vocab
    ([1], 32, 1),
    ([1], 64, 3),
    ([5, 1, 3], 64, 100),
    ([9] * 4, 256, 1024),
    ([17, 0, 33, 15], 128, 5003),
    ([65], 96, 777),
    ([9] * 32, 256, 3001),               # 288 rows: one full row chunk
    ([9] * 32 + [1], 128, 3001),         # 289 rows: two chunks of 144 and 145 rows
    ([9] * 36, 256, 3001),               # 324 rows: two row chunks
    ([33] * 21, 64, 2048),               # 693 rows, 128 tiles: three chunks with 6, 5 and 5
                                         # workgroups per XCD group (a column left neutral)
    ([7] * 111, 64, 777),                # 777 rows, 49 tiles: one group of 49 workgroups, 3 chunks
    ([33] * 300, 64, 4096),              # 9900 rows: two rounds of 32 chunks
    ([9] * 20, 64, 90001),               # 180 rows, 22 tiles per workgroup: six vocabulary
                                         # tiles per wavefront (one pass, not two of five)
    ([3, 8, 1], 2880, 4099),
]


@pytest.mark.parametrize("rows,H,V", CASES)
def test_lmhead_matches_oracle(rows, H, V):
    say("lmhead", rows[:4], len(rows), H, V)
    q_start, des, tokens = _batch(rows, V, seed=H + V + len(rows))
    cfg = workload.CONFIGS["tiny"].replace(vocab=V, hidden_size=H)
    hidden, weight = workload.draw_lmhead(cfg, 7, DEV, des)
    got = _run(hidden, weight, tokens, q_start)
    ref_am, ref_gap = oracle.lmhead_argmax(workload.host_storage(hidden),
                                           workload.host_storage(weight), oracle.BF16)
    flagged, checked = _check(got, ref_am, ref_gap, q_start, tokens, what="%s/%d/%d" % (rows[:3], H, V))
    assert flagged <= max(1, int(q_start[-1]) // 50)
    assert checked >= 1 or int(q_start[-1]) == 0


def test_lmhead_ties_go_to_the_lower_index_and_nan_wins():
    H, V = 128, 700
    rng = np.random.default_rng(3)
    w = rng.standard_normal((V, H)) / np.sqrt(H)
    w[650] = w[17]                       # identical rows: identical logits on both sides
    w[300] = w[299]
    hid = np.stack([w[17] * 9.0, w[650] * 9.0, w[299] * 9.0, rng.standard_normal(H)])
    weight = torch.as_tensor(w, dtype=torch.float32).to(torch.bfloat16).to(DEV)
    hidden = torch.as_tensor(hid, dtype=torch.float32).to(torch.bfloat16).to(DEV)
    q_start = np.array([0, 2, 4], dtype=np.int32)
    tokens = np.array([5, 17, 9, 299], dtype=np.int32)
    am, acc, ne, em = _run(hidden, weight, tokens, q_start)
    assert am[:3].tolist() == [17, 17, 299]
    ref_am, _ = oracle.lmhead_argmax(workload.host_storage(hidden), workload.host_storage(weight),
                                     oracle.BF16)
    assert ref_am[:3].tolist() == [17, 17, 299]
    assert acc.tolist() == [1, 1] and em[:2].tolist() == [17, 17]
    # a NaN in a weight row makes that entry's logit NaN in every row: the
    # first NaN is every row's argmax
    w2 = w.copy()
    w2[450, 5] = np.nan
    w2[600, 0] = np.nan
    weight2 = torch.as_tensor(w2, dtype=torch.float32).to(torch.bfloat16).to(DEV)
    am2, _, _, _ = _run(hidden, weight2, tokens, q_start)
    ref2, _ = oracle.lmhead_argmax(workload.host_storage(hidden), workload.host_storage(weight2),
                                   oracle.BF16)
    assert am2.tolist() == [450] * 4 and ref2.tolist() == [450] * 4


def test_lmhead_repeated_calls_agree():
    """The same inputs give the same bits on every call (fixed summation order)."""
    q_start, des, tokens = _batch([9] * 32, 151936, seed=5)
    cfg = workload.CONFIGS["qwen3_8b"]
    hidden, weight = workload.draw_lmhead(cfg, 11, DEV, des)
    first = _run(hidden, weight, tokens, q_start)
    for _ in range(2):
        again = _run(hidden, weight, tokens, q_start)
        for a, b in zip(first, again):
            np.testing.assert_array_equal(a, b)


@pytest.mark.parametrize("name", ["qwen3_8b", "dsk_distill_8b", "gpt_oss_20b", "long_context"])
def test_lmhead_full_size(name):
    """The workload's scored rows, hidden size and vocabulary: the oracle on
    every row of the requests with the fewest and the most drafts plus random
    rows, and a float32 torch product on every row."""
    cfg = workload.CONFIGS[name]
    say("lmhead full", name)
    bt = workload.make_batch(cfg, 0, DEV, with_layers=False, with_logits=False)
    hidden, weight = workload.draw_lmhead(cfg, 0, DEV, bt.designated)
    got = _run(hidden, weight, bt.tokens, bt.q_start)
    T = bt.total_q
    rng = np.random.default_rng(1)
    n = np.diff(bt.q_start)
    reqs = {int(np.argmax(n)), int(np.argmin(n))}
    rows = np.concatenate([np.arange(bt.q_start[i], bt.q_start[i + 1]) for i in sorted(reqs)] +
                          [rng.integers(0, T, size=6)])
    rows = np.unique(rows).astype(np.int32)
    ref_am, ref_gap = oracle.lmhead_argmax(workload.host_storage(hidden), workload.host_storage(weight),
                                           oracle.BF16, rows=rows)
    flagged, checked = _check(got, ref_am, ref_gap, bt.q_start, bt.tokens, rows=rows, what=name)
    assert checked >= 1 and flagged <= 2
    # every row against a float32 product on the GPU (rows whose top-2 gap there
    # is below 1e-3 are left out)
    wf = weight.to(torch.float32)
    for r0 in range(0, T, 512):
        r1 = min(T, r0 + 512)
        lg = hidden[r0:r1].to(torch.float32) @ wf.T
        top = torch.topk(lg, 2, dim=1)
        gap = (top.values[:, 0] - top.values[:, 1]).cpu().numpy()
        ref = top.indices[:, 0].cpu().numpy()
        ok = gap >= NEAR_TIE
        np.testing.assert_array_equal(got[0][r0:r1][ok], ref[ok], err_msg="%s fp32 rows %d.." % (name, r0))
        del lg, top
    say("lmhead full %s: %d rows, %d oracle rows, %d requests checked, %d flagged" % (
        name, T, rows.size, checked, flagged))
