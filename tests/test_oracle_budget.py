"""Pins of the budget-allocation oracle (Sec. 4.2, Alg. 2) against what the
paper fixes and against an independent brute force:

* the most frequent continuation prefix, recomputed by enumerating every
  prefix of every candidate (no grouping);
* the confidence term at the properties the paper states for it: minimum
  confidence g_min with a single supporting candidate, saturation towards 1 as
  support grows, and the consensus ratio alone when g_min = 1;
* the allocation's invariants on random batches, and its degenerate cases.
"""
from __future__ import annotations

import math

import numpy as np
import pytest

import oracle


def pack(cands_per_req, max_len=None):
    """CSR layout of lists of candidate token lists."""
    rows = [c for req in cands_per_req for c in req]
    if max_len is None:
        max_len = max([len(r) for r in rows] + [1])
    start = np.cumsum([0] + [len(req) for req in cands_per_req]).astype(np.int32)
    lens = np.array([len(r) for r in rows], dtype=np.int32)
    toks = np.zeros((max(len(rows), 1), max_len), dtype=np.int32)
    for i, r in enumerate(rows):
        toks[i, :len(r)] = r
    return start, lens, toks, rows


def brute_most_frequent_prefix(cands):
    """(count, prefix) of the non-empty prefix most candidates start with;
    ties: longer, then lexicographically smaller.  (0, ()) if none."""
    best = (0, ())
    seen = set()
    for c in cands:
        for L in range(1, len(c) + 1):
            p = tuple(c[:L])
            if p in seen:
                continue
            seen.add(p)
            cnt = sum(1 for d in cands if tuple(d[:L]) == p and len(d) >= L)
            key = (cnt, L, tuple(-x for x in p))
            if key > (best[0], len(best[1]), tuple(-x for x in best[1])):
                best = (cnt, p)
    return best


def run(cands_per_req, alpha, g_min, last=None, ctx=None, max_len=None):
    start, lens, toks, rows = pack(cands_per_req, max_len)
    B = len(cands_per_req)
    last = np.arange(100, 100 + B, dtype=np.int32) if last is None else last
    return oracle.budget(start, lens, toks, last, alpha, g_min, ctx_len=ctx), rows


def test_most_frequent_prefix_matches_brute_force():
    rng = np.random.default_rng(3)
    for trial in range(300):
        B = int(rng.integers(1, 6))
        reqs = []
        for _ in range(B):
            n = int(rng.integers(0, 8))
            vocab = int(rng.integers(1, 4))   # tiny vocabularies force ties
            reqs.append([list(rng.integers(0, vocab, size=int(rng.integers(0, 7)))) for _ in range(n)])
        r, rows = run(reqs, alpha=float(rng.integers(0, 60)), g_min=float(rng.uniform(0, 1)))
        off = 0
        for i, req in enumerate(reqs):
            cnt, pref = brute_most_frequent_prefix(req)
            assert r["agree"][i] == cnt, (trial, i)
            assert r["prefix_len"][i] == len(pref), (trial, i)
            if cnt == 0:
                assert r["source"][i] == -1 and r["score"][i] == 0.0
            else:
                # the drafts come from the longest candidate starting with the
                # prefix, the lowest row among equals
                members = [off + j for j, c in enumerate(req) if tuple(c[:len(pref)]) == pref]
                longest = max(len(rows[m]) for m in members)
                assert r["source"][i] == min(m for m in members if len(rows[m]) == longest)
            off += len(req)


def test_confidence_term_properties():
    # n identical candidates: consensus ratio 1, so the score is p(n) itself
    def score_of(n, g_min):
        r, _ = run([[[7, 8, 9]] * n], alpha=10.0, g_min=g_min)
        return float(r["score"][0])

    for g_min in (0.0, 0.2, 0.5, 0.9):
        # a single supporting candidate gets exactly the minimum confidence
        assert score_of(1, g_min) == g_min
        vals = [score_of(n, g_min) for n in range(1, 41)]
        assert all(b > a for a, b in zip(vals[:20], vals[1:20]))   # more support, more confidence
        assert all(b >= a for a, b in zip(vals, vals[1:]))
        assert abs(vals[-1] - 1.0) < 1e-15          # saturation with ample support
        assert all(g_min <= v <= 1.0 for v in vals)
    # g_min = 1: no down-weighting, the score is the consensus ratio c / n
    r, _ = run([[[1, 2], [1, 3], [4], [1]], [[5], [6]]], alpha=10.0, g_min=1.0)
    assert r["score"][0] == 3 / 4 and r["score"][1] == 1 / 2


def test_worked_example_by_hand():
    """Two requests, alpha = 20 (B_t = 10 for a batch of 2), g_min = 0.5.

    Request 0: three 12-token candidates sharing only their first token:
      c = n = 3, |CT*| = 1, g0 = p(3) = 0.5 + 0.5 (1 - e^-2) = 0.93233235...
    Request 1: [3..10] and [8, 1]: two singleton groups, the longer prefix
      wins: c = 1, n = 2, |CT*| = 8, g1 = 1/2 p(2) = 1/2 (0.5 + 0.5 (1 - e^-1))
      = 0.40803013970...
    G = 1.34036249...; shares floor(10 g0 / G) = floor(6.9558) = 6 and
    floor(10 g1 / G) = floor(3.0442) = 3, so L0 = max(1, 6) = 6 and
    L1 = max(8, 3) = 8.
    """
    r0 = [[1] + list(range(2, 13)), [1] + list(range(20, 31)), [1] + list(range(40, 51))]
    r1 = [list(range(3, 11)), [8, 1]]
    r, _ = run([r0, r1], alpha=20.0, g_min=0.5, last=np.array([70, 71], np.int32),
               ctx=np.array([1000, 5], np.int32))
    assert abs(r["score"][0] - 0.9323323583816936) < 1e-15
    assert abs(r["score"][1] - 0.4080301397071394) < 1e-15
    assert r["prefix_len"].tolist() == [1, 8]
    assert r["agree"].tolist() == [3, 1]
    assert r["draft_len"].tolist() == [6, 8]
    assert r["q_start"].tolist() == [0, 7, 16]
    assert r["tokens"].tolist() == [70] + r0[0][:6] + [71] + r1[0]
    assert r["seq_lens"].tolist() == [1000 + 7, 5 + 9]


def test_allocation_invariants_random():
    rng = np.random.default_rng(11)
    for trial in range(200):
        B = int(rng.integers(1, 9))
        reqs = []
        for _ in range(B):
            n = int(rng.integers(0, 6))
            base = list(rng.integers(0, 50, size=10))
            # candidates share a random-length prefix of a common base, then diverge
            reqs.append([base[:int(rng.integers(0, 6))] + list(rng.integers(0, 50, size=int(rng.integers(0, 8))))
                         for _ in range(n)])
        alpha = float(rng.integers(0, 200))
        r, rows = run(reqs, alpha=alpha, g_min=float(rng.uniform(0, 1)),
                      ctx=rng.integers(0, 1000, size=B).astype(np.int32))
        bt = math.floor(alpha / B)
        G = float(np.sum(r["score"]))
        shares = [math.floor(bt * s / G) if G > 0 else 0 for s in r["score"]]
        assert sum(shares) <= bt
        for i in range(B):
            L, src = int(r["draft_len"][i]), int(r["source"][i])
            q0 = int(r["q_start"][i])
            assert int(r["q_start"][i + 1]) - q0 == L + 1
            assert r["tokens"][q0] == 100 + i
            if src < 0:
                assert L == 0 and r["agree"][i] == 0
                continue
            assert r["prefix_len"][i] <= L <= len(rows[src])
            assert L == min(len(rows[src]), max(int(r["prefix_len"][i]), shares[i]))
            drafts = r["tokens"][q0 + 1:q0 + 1 + L].tolist()
            assert drafts == list(rows[src][:L])
            # the agreed part of the drafts is the prefix c_i candidates share
            k = int(r["prefix_len"][i])
            agreeing = sum(1 for c in reqs[i] if len(c) >= k and list(c[:k]) == drafts[:k])
            assert agreeing == r["agree"][i]


def test_degenerate_batches():
    # no candidates anywhere: G = 0, every request verifies its last token only
    r, _ = run([[], [], []], alpha=100.0, g_min=0.3)
    assert r["draft_len"].tolist() == [0, 0, 0] and r["q_start"].tolist() == [0, 1, 2, 3]
    # empty candidates count in n but support no prefix
    r, _ = run([[[], [], [4, 5]]], alpha=100.0, g_min=1.0)
    assert r["agree"][0] == 1 and r["score"][0] == 1 / 3 and r["prefix_len"][0] == 2
    # alpha = 0: no shared budget, each request drafts its agreed prefix
    r, _ = run([[[1, 2, 3], [1, 2, 4]], [[9, 9]]], alpha=0.0, g_min=0.5)
    assert r["draft_len"].tolist() == [2, 2]
    # the budget per request shrinks with the batch: B_t = floor(alpha / bz)
    one = [[1] + list(range(100 * j, 100 * j + 30)) for j in range(1, 5)]  # agree on 1 token
    r1, _ = run([one], alpha=40.0, g_min=0.5)
    r2, _ = run([one, one], alpha=40.0, g_min=0.5)
    assert r1["draft_len"][0] == 31 and r2["draft_len"].tolist() == [10, 10]
    # empty batch
    r, _ = run([], alpha=10.0, g_min=0.5, last=np.zeros(0, np.int32))
    assert r["q_start"].tolist() == [0] and r["tokens"].size == 0


def test_rejects_bad_hyperparameters():
    with pytest.raises(ValueError):
        run([[[1]]], alpha=-1.0, g_min=0.5)
    with pytest.raises(ValueError):
        run([[[1]]], alpha=1.0, g_min=1.5)
