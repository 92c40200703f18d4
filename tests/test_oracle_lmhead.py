"""Pins of the LM-head oracle (no GPU): logits <hidden[r], weight[v]> and
their argmax, checked against what fixes them independently of the oracle.

* numpy's float64 matrix product of the same exact inputs, and numpy's argmax
  (first occurrence) on it;
* a one-hot hidden state reads one column of the weight exactly;
* Cauchy-Schwarz: with +-1 weight rows (all of norm sqrt(H)), a hidden state
  equal to row d has its maximum at d;
* the tie rule (duplicated rows: the lowest index), a NaN weight row, and
  equivariance under a permutation of the vocabulary.
"""
from __future__ import annotations

import numpy as np
import pytest
import torch

import oracle
import workload


def bf16(a) -> torch.Tensor:
    return torch.as_tensor(np.asarray(a, dtype=np.float32)).to(torch.bfloat16)


def exact(t: torch.Tensor) -> np.ndarray:
    return t.to(torch.float64).numpy()


@pytest.mark.parametrize("T,H,V", [(1, 64, 1), (7, 64, 500), (12, 256, 3001), (3, 2880, 257)])
def test_matches_numpy_product(T, H, V):
    rng = np.random.default_rng(T * 1000 + H + V)
    hs = bf16(rng.standard_normal((T, H)))
    w = bf16(rng.standard_normal((V, H)) / np.sqrt(H))
    am, gap, lg = oracle.lmhead_argmax(workload.host_storage(hs), workload.host_storage(w),
                                       oracle.BF16, with_logits=True)
    ref = exact(hs) @ exact(w).T
    np.testing.assert_allclose(lg, ref, rtol=1e-12, atol=1e-12)
    np.testing.assert_array_equal(am, np.argmax(ref, axis=1))
    srt = np.sort(ref, axis=1)
    want_gap = srt[:, -1] - srt[:, -2] if V > 1 else np.full(T, np.inf)
    np.testing.assert_allclose(gap, want_gap, rtol=1e-9, atol=1e-12)


def test_selected_rows_equal_the_full_run():
    rng = np.random.default_rng(2)
    hs = bf16(rng.standard_normal((20, 128)))
    w = bf16(rng.standard_normal((900, 128)))
    full = oracle.lmhead_argmax(workload.host_storage(hs), workload.host_storage(w), oracle.BF16)
    sel = np.array([19, 0, 7, 7, 3], dtype=np.int32)
    part = oracle.lmhead_argmax(workload.host_storage(hs), workload.host_storage(w), oracle.BF16,
                                rows=sel)
    np.testing.assert_array_equal(part[0], full[0][sel])
    np.testing.assert_array_equal(part[1], full[1][sel])


def test_one_hot_hidden_reads_a_weight_column():
    rng = np.random.default_rng(3)
    H, V = 96, 700
    w = bf16(rng.standard_normal((V, H)))
    k = np.array([0, 5, 95, 40])
    hs = np.zeros((k.size, H), dtype=np.float32)
    hs[np.arange(k.size), k] = 2.0
    am, gap, lg = oracle.lmhead_argmax(workload.host_storage(bf16(hs)), workload.host_storage(w),
                                       oracle.BF16, with_logits=True)
    cols = 2.0 * exact(w)[:, k].T
    np.testing.assert_array_equal(lg, cols)
    np.testing.assert_array_equal(am, np.argmax(cols, axis=1))


def test_cauchy_schwarz_planted_rows():
    rng = np.random.default_rng(4)
    H, V, T = 256, 2000, 30
    signs = rng.choice([-1.0, 1.0], size=(V, H))
    w = bf16(signs)
    d = rng.integers(0, V, size=T)
    hs = bf16(signs[d])
    am, gap = oracle.lmhead_argmax(workload.host_storage(hs), workload.host_storage(w), oracle.BF16)
    np.testing.assert_array_equal(am, d)
    assert np.all(gap > 0)


def test_ties_nan_and_permutation():
    rng = np.random.default_rng(5)
    H, V = 64, 300
    w = rng.standard_normal((V, H))
    w[200] = w[17]                       # duplicate of a row: equal logits
    hs = np.stack([w[17], rng.standard_normal(H)])
    # the exact self-product of row 17 beats every other row for hidden = w[17]
    am, gap = oracle.lmhead_argmax(workload.host_storage(bf16(hs)), workload.host_storage(bf16(w)),
                                   oracle.BF16)
    assert am[0] == 17 and gap[0] == 0.0
    # a NaN weight entry makes that vocabulary entry's logit NaN: it wins
    wn = w.copy()
    wn[250, 3] = np.nan
    wn[260, 0] = np.nan
    am, gap = oracle.lmhead_argmax(workload.host_storage(bf16(hs)), workload.host_storage(bf16(wn)),
                                   oracle.BF16)
    assert am.tolist() == [250, 250] and np.all(np.isnan(gap))
    # permuting the vocabulary permutes the logits
    perm = rng.permutation(V)
    _, _, lg = oracle.lmhead_argmax(workload.host_storage(bf16(hs)), workload.host_storage(bf16(w)),
                                    oracle.BF16, with_logits=True)
    _, _, lgp = oracle.lmhead_argmax(workload.host_storage(bf16(hs)),
                                     workload.host_storage(bf16(w[perm])), oracle.BF16,
                                     with_logits=True)
    np.testing.assert_array_equal(lgp, lg[:, perm])


def test_rejects_bad_shapes():
    with pytest.raises(ValueError):
        oracle.lmhead_argmax(np.zeros((2, 8), np.uint16), np.zeros((5, 16), np.uint16), oracle.BF16)
