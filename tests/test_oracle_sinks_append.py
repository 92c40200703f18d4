"""Pins of the oracle's attention sinks and KV append (no GPU).

Sinks: a softmax over the visible scores with the sink logit appended (torch
softmax and matmul, an independent implementation), the limit cases -inf (no
effect) and a huge sink (output 0), and a closed form with equal keys.
KV append: after appending the new tokens' K/V into a cache whose slots held
stale values, attention over the cache equals SDPA on the true sequences, and
exactly the new tokens' slots changed.
"""
from __future__ import annotations

import math

import numpy as np
import pytest
import torch

import oracle
import workload
from helpers import Paged, random_paged, sdpa_reference


def softmax_with_sink_reference(p: Paged, sinks) -> np.ndarray:
    """Per request and head: scores of the visible keys (torch, float64), the
    head's sink appended as one more logit, softmax, weights (without the
    sink's) times V."""
    G = p.Hq // p.Hkv
    scale = 1.0 / math.sqrt(p.D)
    out = np.zeros((p.total_q, p.Hq, p.D))
    qf = p.q.to(torch.float64)
    for i in range(len(p.seq_lens)):
        q0, q1 = int(p.q_start[i]), int(p.q_start[i + 1])
        n, S = q1 - q0, int(p.seq_lens[i])
        for j in range(n):
            pos = S - n + j
            lo = max(0, pos - p.window + 1) if p.window > 0 else 0
            for h in range(p.Hq):
                k = p.k_logical[i][lo:pos + 1, h // G, :]
                v = p.v_logical[i][lo:pos + 1, h // G, :]
                s = (k @ qf[q0 + j, h]) * scale
                logits = torch.cat([s, torch.tensor([float(sinks[h])], dtype=torch.float64)])
                w = torch.softmax(logits, dim=0)[:-1]
                out[q0 + j, h] = (w @ v).numpy()
    return out


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
@pytest.mark.parametrize("window", [0, 6])
def test_sinks_match_softmax_with_an_extra_logit(dtype, window):
    p = random_paged(num_q_heads=8, num_kv_heads=2, head_dim=32, dtype=dtype,
                     contexts=[0, 5, 30], drafts=[2, 0, 6], window=window, seed=4)
    sinks = np.random.default_rng(1).standard_normal(8) * 2.0
    got = oracle.attention(sinks=sinks, **p.oracle_args())
    ref = softmax_with_sink_reference(p, sinks)
    np.testing.assert_allclose(got, ref, rtol=1e-12, atol=1e-12)


def test_sink_limits():
    p = random_paged(num_q_heads=4, num_kv_heads=2, head_dim=16, dtype="f32",
                     contexts=[10, 40], drafts=[3, 1], seed=2)
    plain = oracle.attention(**p.oracle_args())
    none = oracle.attention(sinks=np.full(4, -np.inf), **p.oracle_args())
    assert np.array_equal(plain, none)
    huge = oracle.attention(sinks=np.full(4, 1e4), **p.oracle_args())
    assert np.abs(huge).max() < 1e-300


def test_sink_closed_form_with_equal_keys():
    # every visible key equal (k = 0.25 in every dim) and every value equal to
    # the vector v_g: O = v * m e^s / (m e^s + e^sink), m = visible keys,
    # s = q.k / sqrt(D)
    Hq, Hkv, D = 4, 2, 16
    ctx, k = [7, 20], [2, 3]
    k_log, v_log = [], []
    vvec = np.arange(Hkv * D, dtype=np.float64).reshape(Hkv, D) / 8.0   # exact in fp32
    for L, kk in zip(ctx, k):
        S = L + kk + 1
        k_log.append(np.full((S, Hkv, D), 0.25))
        v_log.append(np.broadcast_to(vvec, (S, Hkv, D)).copy())
    T = sum(kk + 1 for kk in k)
    q = np.random.default_rng(5).standard_normal((T, Hq, D))
    p = Paged(num_q_heads=Hq, num_kv_heads=Hkv, head_dim=D, dtype="f32", k_logical=k_log,
              v_logical=v_log, q=q, num_drafts=k, window=0, seed=1)
    sinks = np.array([-1.0, 0.5, 2.0, 0.0])
    got = oracle.attention(sinks=sinks, **p.oracle_args())
    qf = p.q.to(torch.float64).numpy()
    for i in range(2):
        q0, n, S = int(p.q_start[i]), k[i] + 1, ctx[i] + k[i] + 1
        for j in range(n):
            m = S - n + j + 1
            for h in range(Hq):
                s = float(qf[q0 + j, h].sum()) * 0.25 / math.sqrt(D)
                frac = m * math.exp(s) / (m * math.exp(s) + math.exp(sinks[h]))
                np.testing.assert_allclose(got[q0 + j, h], vvec[h // 2] * frac, rtol=1e-12, atol=1e-13)


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_kv_append_places_the_new_tokens(dtype):
    rng = np.random.default_rng(7)
    Hq, Hkv, D = 8, 2, 32
    p = random_paged(num_q_heads=Hq, num_kv_heads=Hkv, head_dim=D, dtype=dtype,
                     contexts=[0, 13, 40], drafts=[3, 0, 18], seed=9)
    code = workload.dtype_code(dtype)
    tdt = workload.torch_dtype(dtype)
    # the true K/V of the new tokens (the last n_i positions of each request)
    # and a cache in which those slots hold stale values
    n = np.diff(p.q_start)
    k_new = torch.cat([p.k_logical[i][-n[i]:] for i in range(3)]).to(tdt)
    v_new = torch.cat([p.v_logical[i][-n[i]:] for i in range(3)]).to(tdt)
    stale_k = [kl.clone() for kl in p.k_logical]
    stale_v = [vl.clone() for vl in p.v_logical]
    for i in range(3):
        stale_k[i][-n[i]:] = torch.as_tensor(rng.standard_normal((n[i], Hkv, D)))
        stale_v[i][-n[i]:] = torch.as_tensor(rng.standard_normal((n[i], Hkv, D)))
    stale = Paged(num_q_heads=Hq, num_kv_heads=Hkv, head_dim=D, dtype=dtype,
                  k_logical=[k.numpy() for k in stale_k], v_logical=[v.numpy() for v in stale_v],
                  q=p.q.to(torch.float64).numpy(), num_drafts=p.num_drafts, seed=9)
    assert np.array_equal(stale.block_tables, p.block_tables)
    kc, vc = oracle.kv_append(num_kv_heads=Hkv, head_dim=D, dtype=code,
                              k_new=workload.host_storage(k_new), v_new=workload.host_storage(v_new),
                              block_tables=stale.block_tables, seq_lens=stale.seq_lens,
                              q_start=stale.q_start, k_cache=workload.host_storage(stale.k_cache),
                              v_cache=workload.host_storage(stale.v_cache))
    # exactly the new tokens' slots changed ...
    before_k = workload.host_storage(stale.k_cache)
    before_v = workload.host_storage(stale.v_cache)
    changed = int((kc != before_k).sum()), int((vc != before_v).sum())
    assert changed[0] <= p.total_q * Hkv * D and changed[1] <= p.total_q * Hkv * D
    assert changed[0] > 0.9 * p.total_q * Hkv * D
    # ... and attention over the appended cache sees the true sequences
    args = stale.oracle_args()
    args.update(k_cache=kc, v_cache=vc)
    got = oracle.attention(**args)
    ref = sdpa_reference(p)
    np.testing.assert_allclose(got, ref, rtol=1e-12, atol=1e-12)
