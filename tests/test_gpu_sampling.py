"""Stochastic verification on the GPU against the oracle.

verify_accept_sampled draws each row's token from softmax(logits / T) with
Gumbel-max noise that both sides compute from the same Philox4x32-10 counter
and the same fp32 steps, so the drawn tokens, the accept lengths and the
emitted tokens are compared bit for bit: at every workload's full size, on
edge-case rows (ties, NaN, +-inf, signed zeros, vocabularies that leave
ragged tails), at several temperatures, with strided rows, and across seeds
and offsets.
"""
from __future__ import annotations

import ctypes
import sys

import numpy as np
import pytest
import torch

import oracle
import paper_2608_24004_amd as av
import workload

pytestmark = pytest.mark.gpu
DEV = "cuda:0"


def say(*a):
    print(*a, file=sys.stderr, flush=True)


def _oracle_all(logits, q_start, tokens, code, T, seed, offset):
    y = oracle.sample(workload.host_storage(logits), code, T, seed=seed, offset=offset)
    acc, ne, em = oracle.accept(q_start, tokens, y)
    return y, acc, ne, em


def _check(got, want):
    for g, w, what in zip(got, want, ("sampled", "accept_len", "num_emitted", "emitted")):
        np.testing.assert_array_equal(g, w, err_msg=what)


def _gpu(logits, tokens, q_start, T, seed, offset):
    acc, ne, em, y = av.verify_accept_sampled(logits, tokens, q_start, temperature=T, seed=seed,
                                              offset=offset)
    torch.cuda.synchronize()
    return [t.cpu().numpy() for t in (y, acc, ne, em)]


def _plant(y, q_start, rng, vocab):
    """Drafts that follow the oracle's draws for a random number of leading
    positions, then one random token: long accepted runs and rejections."""
    n = np.diff(q_start)
    tokens = rng.integers(0, max(vocab, 1), size=int(q_start[-1])).astype(np.int32)
    for i in range(n.size):
        q0 = int(q_start[i])
        J = int(rng.integers(0, max(1, n[i])))
        for j in range(min(J, max(0, n[i] - 1))):
            tokens[q0 + j + 1] = y[q0 + j]
    return tokens


@pytest.mark.parametrize("name,seed", [(n, s) for n in workload.CONFIGS for s in range(5)
                                        if n != "long_context" or s < 2])
def test_sampled_full_size(name, seed):
    cfg = workload.CONFIGS[name]
    say("sampled full", name, "seed", seed)
    bt = workload.make_batch(cfg, seed, DEV, with_layers=False)
    code = workload.dtype_code(cfg.dtype)
    T, seed, offset = 0.7, 0x1234_5678_9ABC_DEF0, 11
    y_ref = oracle.sample(workload.host_storage(bt.logits), code, T, seed=seed, offset=offset)
    tokens = _plant(y_ref, bt.q_start, np.random.default_rng(1), bt.logits.shape[1])
    want = _oracle_all(bt.logits, bt.q_start, tokens, code, T, seed, offset)
    got = _gpu(bt.logits, torch.as_tensor(tokens, device=DEV), bt.t_q_start, T, seed, offset)
    _check(got, want)
    assert (want[1] > 0).mean() > 0.3      # the planted drafts are accepted


def _ties(rng, shape):
    return rng.integers(-3, 4, size=shape)


def _specials(rng, shape):
    x = rng.standard_normal(shape)
    T, V = shape
    for r in range(T):
        kind = r % 7
        if kind == 0:
            x[r, rng.integers(0, V, size=2)] = np.nan
        elif kind == 1:
            x[r] = -np.inf
        elif kind == 2:
            x[r] = -np.inf
            x[r, rng.integers(0, V, size=3)] = 0.0
        elif kind == 3:
            x[r, rng.integers(0, V, size=3)] = np.inf
        elif kind == 4:
            x[r] = 0.0
            x[r, rng.integers(0, V, size=V // 2 + 1)] = -0.0
        elif kind == 5:
            x[r] *= 40.0            # peaked rows: near-greedy at low T
    return x


@pytest.mark.parametrize("dtype", ["bf16", "f32"])
@pytest.mark.parametrize("vocab", [1, 7, 8, 1000, 8193, 151936])
@pytest.mark.parametrize("fill", [_ties, _specials], ids=["ties", "specials"])
@pytest.mark.parametrize("T", [0.05, 1.0, 3.0])
def test_sampled_edge_cases(dtype, vocab, fill, T):
    rows = [1, 3, 0, 9, 70, 1, 33, 0, 2]
    if vocab >= 100000:
        rows = [1, 70, 0, 5]
    rng = np.random.default_rng(vocab + int(T * 100))
    n = np.asarray(rows)
    q_start = np.zeros(n.size + 1, dtype=np.int32)
    q_start[1:] = np.cumsum(n)
    vals = fill(rng, (int(q_start[-1]), vocab)).astype(np.float32)
    logits = torch.as_tensor(vals).to(workload.torch_dtype(dtype))
    code = workload.dtype_code(dtype)
    seed, offset = int(rng.integers(0, 1 << 63)), int(rng.integers(0, 1 << 32))
    y_ref = oracle.sample(workload.host_storage(logits), code, T, seed=seed, offset=offset)
    tokens = _plant(y_ref, q_start, rng, vocab)
    say("sampled edge", dtype, vocab, fill.__name__, T)
    want = _oracle_all(logits, q_start, tokens, code, T, seed, offset)
    got = _gpu(logits.to(DEV), torch.as_tensor(tokens, device=DEV),
               torch.as_tensor(q_start, device=DEV), T, seed, offset)
    _check(got, want)


def test_sampled_seeds_offsets_and_extreme_temperatures():
    rng = np.random.default_rng(5)
    V, R = 5000, 96
    x = torch.as_tensor(rng.standard_normal((R, V)).astype(np.float32) * 3.0).to(torch.bfloat16)
    q_start = np.arange(0, R + 1, 8, dtype=np.int32)
    tokens = rng.integers(0, V, size=R).astype(np.int32)
    xd, td, qd = x.to(DEV), torch.as_tensor(tokens, device=DEV), torch.as_tensor(q_start, device=DEV)
    seen = []
    for T, seed, offset in ((1.0, 0, 0), (1.0, 1, 0), (1.0, 1 << 32, 0), (1.0, 0, 1),
                            (1.0, (1 << 64) - 1, (1 << 32) - 1), (1e-30, 7, 3), (1e30, 7, 3)):
        want = _oracle_all(x, q_start, tokens, av.BF16, T, seed, offset)
        got = _gpu(xd, td, qd, T, seed, offset)
        _check(got, want)
        seen.append(got[0])
    # each change of seed or offset redraws most rows
    for other in seen[1:5]:
        assert np.mean(other != seen[0]) > 0.5
    # T -> 0 is the argmax (on rows whose maximum is unique)
    am, gap = oracle.argmax(workload.host_storage(x), av.BF16)
    unique = gap > 0
    assert unique.mean() > 0.5
    np.testing.assert_array_equal(seen[5][unique], am[unique])


def test_sampled_strided_rows():
    V, stride, R = 1000, 1024, 40
    full = torch.randn(R, stride, device=DEV).to(torch.bfloat16)
    q_start = torch.tensor([0, 9, R], dtype=torch.int32, device=DEV)
    tokens = torch.randint(0, V, (R,), dtype=torch.int32, device=DEV)
    outs = [torch.empty(n, dtype=torch.int32, device=DEV) for n in (R, 2, 2, R)]
    nbytes = av.accept_workspace_size(2, R, V, av.BF16)
    ws = torch.empty(nbytes, dtype=torch.uint8, device=DEV)
    p = lambda t: ctypes.c_void_p(t.data_ptr())
    rc = av.library().verify_accept_sampled(
        2, R, V, stride, av.BF16, p(full), p(tokens), p(q_start), 0.9, 99, 5, *[p(o) for o in outs],
        p(ws), nbytes, ctypes.c_void_p(torch.cuda.current_stream().cuda_stream))
    assert rc == 0
    torch.cuda.synchronize()
    y_ref = oracle.sample(workload.host_storage(full[:, :V].contiguous()), av.BF16, 0.9, seed=99,
                          offset=5)
    np.testing.assert_array_equal(outs[0].cpu().numpy(), y_ref)
    acc, ne, em = oracle.accept(q_start.cpu().numpy(), tokens.cpu().numpy(), y_ref)
    np.testing.assert_array_equal(outs[1].cpu().numpy(), acc)
    np.testing.assert_array_equal(outs[3].cpu().numpy(), em)


def test_more_rows_than_one_launch_holds():
    # 70 000 scored rows: the per-chunk kernels run in slices of at most 65 535
    # rows (the grid's y limit); the draws depend on the absolute row index
    rng = np.random.default_rng(70000)
    n = np.full(7000, 10)
    q_start = np.zeros(n.size + 1, dtype=np.int32)
    q_start[1:] = np.cumsum(n)
    V = 24
    logits = torch.as_tensor(rng.standard_normal((int(q_start[-1]), V)).astype(np.float32)).to(
        torch.bfloat16)
    code = workload.dtype_code("bf16")
    seed, offset = 1234567, 9
    y_ref = oracle.sample(workload.host_storage(logits), code, 0.8, seed=seed, offset=offset)
    tokens = _plant(y_ref, q_start, rng, V)
    say("sampled 70000 rows")
    want = _oracle_all(logits, q_start, tokens, code, 0.8, seed, offset)
    d_logits, d_tok, d_qs = (logits.to(DEV), torch.as_tensor(tokens, device=DEV),
                             torch.as_tensor(q_start, device=DEV))
    _check(_gpu(d_logits, d_tok, d_qs, 0.8, seed, offset), want)
    acc, ne, em, am = av.verify_accept(d_logits, d_tok, d_qs)
    torch.cuda.synchronize()
    am_ref, _ = oracle.argmax(workload.host_storage(logits), code, with_gap=False)
    r_acc, r_ne, r_em = oracle.accept(q_start, tokens, am_ref)
    np.testing.assert_array_equal(am.cpu().numpy(), am_ref)
    np.testing.assert_array_equal(acc.cpu().numpy(), r_acc)
    np.testing.assert_array_equal(ne.cpu().numpy(), r_ne)
    np.testing.assert_array_equal(em.cpu().numpy(), r_em)
