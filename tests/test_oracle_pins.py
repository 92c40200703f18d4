"""Pins of the CPU oracle to things other than itself (no GPU).

Attention: a library routine (torch SDPA with an explicit mask), closed forms
that expose the visible-key range, the scale, the key/value layout and the
grouped-query head map, and invariants of the definition.
Argmax: numpy.argmax (independent implementation, same tie rule) and hand cases.
Acceptance: closed-form properties and the losslessness of greedy speculative
decoding (Sec. 2.2: verification reproduces plain decoding exactly).
"""
from __future__ import annotations

import math

import numpy as np
import pytest
import torch

import oracle
import workload
from helpers import Paged, random_paged, sdpa_reference


def run_oracle(p: Paged, rows=None, heads=None):
    return oracle.attention(rows=rows, heads=heads, **p.oracle_args())


# --------------------------------------------------------------------------- attention


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
@pytest.mark.parametrize("hq,hkv,d", [(8, 2, 64), (4, 4, 16), (8, 1, 32)])
@pytest.mark.parametrize("window", [0, 5, 37])
def test_attention_matches_sdpa(dtype, hq, hkv, d, window):
    p = random_paged(num_q_heads=hq, num_kv_heads=hkv, head_dim=d, dtype=dtype,
                     contexts=[0, 3, 20, 45], drafts=[0, 4, 2, 7], window=window, seed=hq + d)
    got = run_oracle(p)
    ref = sdpa_reference(p)
    np.testing.assert_allclose(got, ref, rtol=1e-12, atol=1e-12)


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
@pytest.mark.parametrize("window", [0, 20])
def test_attention_skips_keys_on_unmapped_blocks(dtype, window):
    """A key whose block id lies outside [0, num_blocks) is no key: the oracle
    equals SDPA with those positions masked out, and a row left with no key
    (request 3's only block) is zero."""
    p = random_paged(num_q_heads=8, num_kv_heads=2, head_dim=32, dtype=dtype,
                     contexts=[40, 70, 20, 3], drafts=[5, 9, 0, 4], window=window, seed=31)
    bt = p.block_tables.copy()
    bt[0, 1] = -1                      # request 0: positions 16..31
    bt[1, 0] = p.num_blocks            # request 1: positions 0..15 (past the cache)
    bt[1, 4] = -3                      # request 1: positions 64..79 (new tokens among them)
    bt[3, 0] = -1                      # request 3: its only block
    args = p.oracle_args()
    args.update(block_tables=bt)
    got = oracle.attention(**args)
    ref = sdpa_reference(p, missing={0: {1}, 1: {0, 4}, 3: {0}})
    np.testing.assert_allclose(got, ref, rtol=1e-12, atol=1e-12)
    q0, q1 = p.q_start[3], p.q_start[4]
    assert np.all(got[q0:q1] == 0.0)
    # the unmapped keys matter: with valid ids the result differs
    assert not np.allclose(got, run_oracle(p))


def _const_keys(S, hkv, d):
    return np.ones((S, hkv, d)) * 0.25


@pytest.mark.parametrize("window", [0, 1, 7, 16, 300])
def test_equal_keys_average_exactly_the_visible_values(window):
    # Equal keys give equal weights, so each row averages V over exactly its
    # visible positions [max(0, p-W+1), p]: V_t = t makes that mean (lo+p)/2.
    ctx, drafts = [0, 5, 17, 40], [3, 0, 6, 9]
    k_log, v_log = [], []
    for L, k in zip(ctx, drafts):
        S = L + k + 1
        k_log.append(_const_keys(S, 2, 16))
        v_log.append(np.broadcast_to(np.arange(S, dtype=np.float64)[:, None, None], (S, 2, 16)).copy())
    T = sum(k + 1 for k in drafts)
    q = np.random.default_rng(0).standard_normal((T, 4, 16))
    p = Paged(num_q_heads=4, num_kv_heads=2, head_dim=16, dtype="f32", k_logical=k_log,
              v_logical=v_log, q=q, num_drafts=drafts, window=window)
    got = run_oracle(p)
    for i in range(len(ctx)):
        S, n = p.seq_lens[i], drafts[i] + 1
        for j in range(n):
            pos = S - n + j
            lo = max(0, pos - window + 1) if window > 0 else 0
            np.testing.assert_allclose(got[p.q_start[i] + j], (lo + pos) / 2.0, rtol=0, atol=1e-12)


def test_single_key_returns_its_value():
    # S = 1 (empty context, no drafts): the output is V_0 itself.
    rng = np.random.default_rng(3)
    k_log = [rng.standard_normal((1, 2, 32))]
    v_log = [rng.standard_normal((1, 2, 32))]
    q = rng.standard_normal((1, 8, 32))
    p = Paged(num_q_heads=8, num_kv_heads=2, head_dim=32, dtype="f32", k_logical=k_log,
              v_logical=v_log, q=q, num_drafts=[0])
    got = run_oracle(p)
    for h in range(8):
        np.testing.assert_array_equal(got[0, h], p.v_logical[0][0, h // 4].numpy())


def test_dominant_key_closed_form_and_scale():
    # Q = c e_3 and K_t = e_3 only at t*: score c/sqrt(D) at t*, 0 elsewhere, so
    # O = (e^{c/sqrt(D)} V_t* + sum_{t != t*} V_t) / (e^{c/sqrt(D)} + N - 1).
    D, S, tstar, c = 16, 37, 21, 6.0
    rng = np.random.default_rng(5)
    K = np.zeros((S, 1, D))
    K[tstar, 0, 3] = 1.0
    V = rng.standard_normal((S, 1, D))
    q = np.zeros((1, 1, D))
    q[0, 0, 3] = c
    p = Paged(num_q_heads=1, num_kv_heads=1, head_dim=D, dtype="f32", k_logical=[K],
              v_logical=[V], q=q, num_drafts=[0])
    got = run_oracle(p)[0, 0]
    Vr = p.v_logical[0][:, 0].numpy()
    w = math.exp(c / math.sqrt(D))
    want = (w * Vr[tstar] + Vr.sum(0) - Vr[tstar]) / (w + S - 1)
    np.testing.assert_allclose(got, want, rtol=1e-13, atol=1e-14)


def test_two_key_softmax_closed_form():
    # Two keys with dot products a and b against q: weights are the 2-way
    # softmax of (a, b)/sqrt(D); V_0 = e_0, V_1 = e_1.
    D = 64
    K = np.zeros((2, 1, D))
    K[0, 0, :2] = [1.0, 2.0]
    K[1, 0, :2] = [-3.0, 0.5]
    q = np.zeros((1, 1, D))
    q[0, 0, :2] = [2.0, -1.0]
    V = np.zeros((2, 1, D))
    V[0, 0, 0] = 1.0
    V[1, 0, 1] = 1.0
    p = Paged(num_q_heads=1, num_kv_heads=1, head_dim=D, dtype="f32", k_logical=[K],
              v_logical=[V], q=q, num_drafts=[0])
    got = run_oracle(p)[0, 0]
    a, b = (2 * 1 - 1 * 2) / 8.0, (2 * -3 - 1 * 0.5) / 8.0
    wa = 1.0 / (1.0 + math.exp(b - a))
    assert got[0] == pytest.approx(wa, abs=1e-15)
    assert got[1] == pytest.approx(1 - wa, abs=1e-15)
    assert np.all(got[2:] == 0)


def test_grouped_query_head_map():
    # KV head g carries the constant value g + 1, so q-head h must return
    # floor(h / G) + 1 (a modulo map would return h % Hkv + 1 instead).
    Hq, Hkv, D, S = 12, 3, 16, 40
    rng = np.random.default_rng(7)
    K = rng.standard_normal((S, Hkv, D))
    V = np.zeros((S, Hkv, D))
    for g in range(Hkv):
        V[:, g, :] = g + 1
    q = rng.standard_normal((3, Hq, D))
    p = Paged(num_q_heads=Hq, num_kv_heads=Hkv, head_dim=D, dtype="bf16", k_logical=[K],
              v_logical=[V], q=q, num_drafts=[2])
    got = run_oracle(p)
    for h in range(Hq):
        np.testing.assert_allclose(got[:, h, :], h // (Hq // Hkv) + 1, rtol=0, atol=1e-12)


def test_layout_each_key_dimension_is_read_from_its_slot():
    # One key carries a distinct value in every dimension; query head h is e_h
    # (Hq = D heads sharing one KV head), so head h scores that key with
    # K[t*][h]/sqrt(D) and every other key with 0.  With V_t* = 1 and V = 0
    # elsewhere the output of head h is the softmax weight of t*:
    # w / (w + S - 1), w = exp(K[t*][h]/sqrt(D)), a closed form per dimension.
    D, S, tstar = 32, 19, 17
    K = np.zeros((S, 1, D))
    K[tstar, 0, :] = (np.arange(D) - D / 2) / 4.0
    V = np.zeros((S, 1, D))
    V[tstar, 0, :] = 1.0
    q = np.zeros((1, D, D))
    for h in range(D):
        q[0, h, h] = 1.0
    for dtype in ("f32", "bf16"):
        p = Paged(num_q_heads=D, num_kv_heads=1, head_dim=D, dtype=dtype, k_logical=[K],
                  v_logical=[V], q=q, num_drafts=[0])
        got = run_oracle(p)
        for h in range(D):
            w = math.exp(K[tstar, 0, h] / math.sqrt(D))
            np.testing.assert_allclose(got[0, h], w / (w + S - 1), rtol=1e-13)


def test_block_permutation_invariance():
    a = random_paged(num_q_heads=8, num_kv_heads=2, head_dim=64, dtype="bf16",
                     contexts=[33, 70], drafts=[5, 2], seed=11)
    b = Paged(num_q_heads=8, num_kv_heads=2, head_dim=64, dtype="bf16",
              k_logical=[k.numpy() for k in a.k_logical], v_logical=[v.numpy() for v in a.v_logical],
              q=a.q.to(torch.float32).numpy(), num_drafts=[5, 2], seed=99, spare_blocks=7)
    assert not np.array_equal(a.block_tables, b.block_tables[:, :a.block_tables.shape[1]])
    np.testing.assert_array_equal(run_oracle(a), run_oracle(b))


def test_future_keys_do_not_leak():
    # Perturbing keys/values after a row's position leaves that row bit-identical.
    base = random_paged(num_q_heads=4, num_kv_heads=2, head_dim=32, dtype="f32",
                        contexts=[10], drafts=[6], seed=4)
    S = int(base.seq_lens[0])
    k2 = base.k_logical[0].numpy().copy()
    v2 = base.v_logical[0].numpy().copy()
    cut = S - 4                      # rows j with position < cut must not change
    k2[cut:] += 50.0
    v2[cut:] -= 9.0
    pert = Paged(num_q_heads=4, num_kv_heads=2, head_dim=32, dtype="f32", k_logical=[k2],
                 v_logical=[v2], q=base.q.numpy(), num_drafts=[6], seed=4)
    a, b = run_oracle(base), run_oracle(pert)
    n = 7
    for j in range(n):
        pos = S - n + j
        if pos < cut:
            np.testing.assert_array_equal(a[j], b[j])
        else:
            assert not np.array_equal(a[j], b[j])


def test_wide_window_equals_full_and_zero_drafts_is_plain_decode():
    kw = dict(num_q_heads=8, num_kv_heads=2, head_dim=64, dtype="bf16",
              contexts=[3, 50, 90], drafts=[0, 0, 3], seed=21)
    full = random_paged(window=0, **kw)
    wide = random_paged(window=10_000, **kw)
    np.testing.assert_array_equal(run_oracle(full), run_oracle(wide))
    # k = 0: one query row at the last position sees every key (plain decode):
    # SDPA with no mask at all.
    got = run_oracle(full)
    G = 4
    for i in (0, 1):
        r = int(full.q_start[i])
        qi = full.q[r].to(torch.float64)[None, :, None, :]
        ki = full.k_logical[i].permute(1, 0, 2).repeat_interleave(G, 0)[None]
        vi = full.v_logical[i].permute(1, 0, 2).repeat_interleave(G, 0)[None]
        o = torch.nn.functional.scaled_dot_product_attention(qi, ki, vi)[0, :, 0, :].numpy()
        np.testing.assert_allclose(got[r], o, rtol=1e-12, atol=1e-13)


def test_selected_pairs_match_full_run():
    p = random_paged(num_q_heads=8, num_kv_heads=2, head_dim=64, dtype="bf16",
                     contexts=[40, 9], drafts=[3, 8], seed=2)
    full = run_oracle(p)
    rows = np.array([0, 3, 5, 12, 7], dtype=np.int32)
    heads = np.array([7, 0, 3, 1, 6], dtype=np.int32)
    sel = run_oracle(p, rows=rows, heads=heads)
    np.testing.assert_array_equal(sel, full[rows, heads])


# --------------------------------------------------------------------------- argmax


def _bf16_bits(a):
    return workload.host_storage(torch.as_tensor(np.asarray(a, dtype=np.float32)).to(torch.bfloat16))


@pytest.mark.parametrize("vocab", [1, 2, 7, 64, 1000, 4099])
def test_argmax_matches_numpy_with_many_ties(vocab):
    rng = np.random.default_rng(vocab)
    vals = rng.integers(-3, 4, size=(37, vocab)).astype(np.float32)  # heavy ties
    for dtype, raw in ((oracle.F32, vals), (oracle.BF16, _bf16_bits(vals))):
        am, gap = oracle.argmax(raw, dtype)
        np.testing.assert_array_equal(am, np.argmax(vals, axis=1))
        srt = np.sort(vals, axis=1)
        want_gap = srt[:, -1] - srt[:, -2] if vocab > 1 else np.full(37, np.inf)
        np.testing.assert_array_equal(gap, want_gap)


def test_argmax_special_values():
    nan, inf = np.nan, np.inf
    rows = [
        ([-1.0, -2.0, -1.5, -0.0, -3.0, -1.0, -4.0, 0.0], 3),   # -0 == +0: lowest index
        ([-5.0, -1.0, 0.0, -2.0, -1.0, -0.0], 2),
        ([1.0, 2.0, 3.0, 0.5, nan, 9.0, 1.0, 2.0, 3.0, nan], 4),  # first NaN
        ([-inf, -inf, -inf], 0),
        ([1.0, inf, 2.0, inf], 1),
        ([-inf, -1e30, -inf], 1),
    ]
    for vals, want in rows:
        a = np.array([vals], dtype=np.float32)
        for dtype, raw in ((oracle.F32, a), (oracle.BF16, _bf16_bits(a))):
            am, _ = oracle.argmax(raw, dtype)
            assert am[0] == want, (vals, dtype)
            if not np.isnan(a).any():
                assert am[0] == np.argmax(a[0])


# --------------------------------------------------------------------------- acceptance


def _accept_case(drafts_per_req, argmax_per_req):
    q_start = np.zeros(len(drafts_per_req) + 1, dtype=np.int32)
    tokens, am = [], []
    for i, (d, a) in enumerate(zip(drafts_per_req, argmax_per_req)):
        assert len(a) == len(d) + 1
        tokens += [12345] + list(d)
        am += list(a)
        q_start[i + 1] = q_start[i] + len(d) + 1
    return q_start, np.array(tokens, np.int32), np.array(am, np.int32)


def test_accept_closed_forms():
    # k = 0: nothing proposed, the bonus token is row 0's argmax.
    # drafts equal to the argmax continuation: all accepted (m = k).
    # first divergence at draft j+1: m = j.
    reqs = [([], [77]),
            ([5, 6, 7], [5, 6, 7, 8]),
            ([5, 6, 7], [5, 9, 7, 8]),
            ([5, 6, 7], [1, 6, 7, 8]),
            ([4] * 40, [4] * 40 + [3]),
            ([4] * 40, [4] * 33 + [2] * 8)]
    q_start, tok, am = _accept_case([r[0] for r in reqs], [r[1] for r in reqs])
    acc, ne, em = oracle.accept(q_start, tok, am)
    np.testing.assert_array_equal(acc, [0, 3, 1, 0, 40, 33])
    np.testing.assert_array_equal(ne, acc + 1)
    # emitted: accepted drafts then the bonus, -1 after
    assert list(em[q_start[0]:q_start[1]]) == [77]
    assert list(em[q_start[1]:q_start[2]]) == [5, 6, 7, 8]
    assert list(em[q_start[2]:q_start[3]]) == [5, 9, -1, -1]
    assert list(em[q_start[3]:q_start[4]]) == [1, -1, -1, -1]
    assert list(em[q_start[4]:q_start[5]]) == [4] * 40 + [3]
    assert list(em[q_start[5]:q_start[6]]) == [4] * 33 + [2] + [-1] * 7
    rho = oracle.rejection_rate(acc, q_start)
    assert np.isnan(rho[0]) and rho[1] == 0 and rho[2] == pytest.approx(2 / 3) and rho[3] == 1


def test_accept_invariants_random():
    rng = np.random.default_rng(8)
    k = rng.integers(0, 20, size=300)
    q_start = np.zeros(301, np.int32)
    q_start[1:] = np.cumsum(k + 1)
    T = int(q_start[-1])
    am = rng.integers(0, 4, size=T).astype(np.int32)
    tok = rng.integers(0, 4, size=T).astype(np.int32)
    acc, ne, em = oracle.accept(q_start, tok, am)
    for i in range(300):
        q0, m = q_start[i], acc[i]
        assert 0 <= m <= k[i] and ne[i] == m + 1
        np.testing.assert_array_equal(em[q0:q0 + m], tok[q0 + 1:q0 + 1 + m])
        assert em[q0 + m] == am[q0 + m]
        if m < k[i]:
            assert am[q0 + m] != tok[q0 + m + 1]


class ToyLM:
    """Deterministic toy language model: logits are a seeded hash of the prefix."""

    def __init__(self, vocab, seed):
        self.vocab, self.seed = vocab, seed

    def logits(self, prefix):
        h = np.random.SeedSequence([self.seed] + [int(t) + 1 for t in prefix[-6:]] + [len(prefix)])
        r = np.random.default_rng(h)
        return r.integers(-4, 5, size=self.vocab).astype(np.float32)  # ties on purpose


def test_greedy_speculation_is_lossless():
    # Sec. 2.2: speculative decoding with verification reproduces exactly the
    # target's own greedy output, whatever the drafts are.
    rng = np.random.default_rng(1)
    for seed in range(6):
        lm = ToyLM(vocab=11, seed=seed)
        prompt = [3, 1, 4]
        ar = list(prompt)
        for _ in range(60):
            ar.append(int(np.argmax(lm.logits(ar))))
        seq = list(prompt)
        while len(seq) < len(ar):
            k = int(rng.integers(0, 7))
            drafts = []
            for j in range(k):
                good = len(seq) + j < len(ar) and rng.random() < 0.6
                drafts.append(ar[len(seq) + j] if good else int(rng.integers(0, 11)))
            rows = [seq + drafts[:j] for j in range(k + 1)]
            lg = np.stack([lm.logits(r) for r in rows])
            am, _ = oracle.argmax(lg, oracle.F32, with_gap=False)
            q_start = np.array([0, k + 1], np.int32)
            tokens = np.array([seq[-1]] + drafts, np.int32)
            acc, ne, em = oracle.accept(q_start, tokens, am)
            seq += list(em[:ne[0]])
        assert seq[:len(ar)] == ar
