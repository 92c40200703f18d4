"""The seeded workload generator: determinism, structure and statistics (no GPU)."""
from __future__ import annotations

import numpy as np
import pytest
import torch

import oracle
import workload


def _small(name, **kw):
    return workload.CONFIGS[name].replace(**kw)


def test_deterministic_and_seed_dependent():
    cfg = _small("qwen3_8b", batch=3, vocab=300, context=("uniform", 20, 60))
    a = workload.make_batch(cfg, 5)
    b = workload.make_batch(cfg, 5)
    c = workload.make_batch(cfg, 6)
    for x, y in ((a.layers[0].k_cache, b.layers[0].k_cache), (a.logits, b.logits)):
        assert torch.equal(x, y)
    np.testing.assert_array_equal(a.tokens, b.tokens)
    assert not torch.equal(a.layers[0].q, c.layers[0].q)


@pytest.mark.parametrize("name", list(workload.CONFIGS))
def test_structure(name):
    cfg = workload.CONFIGS[name]
    cfg = cfg.replace(batch=min(cfg.batch, 6), vocab=min(cfg.vocab, 512))
    # shrink the contexts so the CPU test stays small
    if cfg.context[0] == "uniform":
        cfg = cfg.replace(context=("uniform", 1, 300))
    elif cfg.context[0] == "lognormal":
        cfg = cfg.replace(context=("lognormal", 64, 1.0, 400))
    bt = workload.make_batch(cfg, 1)
    n = bt.num_drafts + 1
    np.testing.assert_array_equal(np.diff(bt.q_start), n)
    np.testing.assert_array_equal(bt.seq_lens, bt.context_len + n)
    used = bt.block_tables[bt.block_tables >= 0]
    assert sorted(used.tolist()) == list(range(bt.num_blocks))   # a permutation of the pool
    for i in range(cfg.batch):
        assert (bt.block_tables[i] >= 0).sum() == -(-bt.seq_lens[i] // 16)
    x = workload.elems_per_16b(cfg.dtype)
    for layer, w in zip(bt.layers, cfg.windows):
        assert layer.window == w
        assert tuple(layer.k_cache.shape) == (bt.num_blocks, cfg.num_kv_heads, cfg.head_dim // x, 16, x)
        assert tuple(layer.v_cache.shape) == (bt.num_blocks, cfg.num_kv_heads, cfg.head_dim, 16)
        assert tuple(layer.q.shape) == (bt.total_q, cfg.num_q_heads, cfg.head_dim)
    # the planted maximum is the unique row maximum (oracle argmax, zero ties)
    am, gap = oracle.argmax(workload.host_storage(bt.logits), workload.dtype_code(cfg.dtype))
    np.testing.assert_array_equal(am, bt.designated)
    assert np.all(gap > 0)


def test_logits_look_standard_normal():
    cfg = _small("qwen3_8b", batch=8, vocab=20000, context=("fixed", 16))
    bt = workload.make_batch(cfg, 3, with_layers=False)
    x = bt.logits.to(torch.float64).numpy()
    assert abs(x.mean()) < 0.01 and abs(x.std() - 1) < 0.01
    # row maxima follow the law of the maximum of V normals: mean ~ 3.8 at V = 2e4
    assert 3.4 < x.max(axis=1).mean() < 4.3


@pytest.mark.parametrize("match,k", [(("prob", 0.7), 8), (("halves", 0.8, 0.3), 9), (("prob", 0.5), 3)])
def test_mean_accept_length_matches_closed_form(match, k):
    # E[m] = sum_{j=1..k} prod_{l<=j} p_l for independent per-position matches.
    cfg = _small("qwen3_8b", batch=3000, vocab=40, context=("fixed", 1), drafts=("fixed", k),
                 match=match)
    bt = workload.make_batch(cfg, 11, with_layers=False)
    am, _ = oracle.argmax(workload.host_storage(bt.logits), oracle.BF16)
    acc, ne, em = oracle.accept(bt.q_start, bt.tokens, am)
    p = workload.match_probability(cfg, k)
    want = np.sum(np.cumprod(p))
    var_bound = np.sum(np.arange(1, k + 1) ** 2 * 1.0)  # crude bound on Var(m)
    tol = 5 * np.sqrt(min(var_bound, k * k) / cfg.batch)
    assert abs(acc.mean() - want) < tol, (acc.mean(), want, tol)


def test_divergence_recipe():
    cfg = workload.CONFIGS["tiny"].replace(batch=2000)
    bt = workload.make_batch(cfg, 2, with_layers=False)
    am, _ = oracle.argmax(workload.host_storage(bt.logits), oracle.F32)
    acc, _, _ = oracle.accept(bt.q_start, bt.tokens, am)
    # divergence point uniform on {0..k}: accept length uniform on {0..4}
    counts = np.bincount(acc, minlength=5)
    assert counts.shape[0] == 5 and np.all(np.abs(counts / 2000 - 0.2) < 0.04)
