"""CPU oracle for the batched speculative-verification step.

TEST INFRASTRUCTURE ONLY: the tests, the smoke check and the CPU-baseline leg of
the benchmark may use this package; the product path (the HIP library and its
Python binding) never imports it, and this package never imports the product.

The arithmetic lives in ``oracle.c`` (plain C, double precision), compiled with
gcc into ``liboracle.so``.  This module only marshals numpy arrays to it.

Functions (each restates the paper's definition; see ``oracle.c``):
  attention(...)  -- softmax attention of selected (row, head) pairs against
                     the paged KV cache (speculative verification scores all
                     k+1 positions in one target pass, Sec. 2.2).
  kv_append(...)  -- the new tokens' K/V written into their paged-cache slots.
  argmax(...)     -- lowest index of the row maximum, plus the top-2 gap.
  sample(...)     -- stochastic verification's per-row sample from softmax(x/T)
                     (Gumbel-max with Philox4x32-10 noise).
  accept(...)     -- greedy acceptance: longest matching draft prefix plus one
                     bonus token; rejection rate = rejected / proposed (Sec. 3.1).
  budget(...)     -- redundancy-aware draft budget (Sec. 4.2, Alg. 2) and the
                     verify-step descriptor built from the draft lengths.
"""
from __future__ import annotations

import ctypes
import os
import subprocess

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "oracle.c")
_LIB = os.path.join(_HERE, "liboracle.so")

F32 = 0
BF16 = 1

_lib = None


def build(force: bool = True) -> str:
    """Compile oracle.c with gcc (OpenMP) into liboracle.so; return its path."""
    if force or not os.path.exists(_LIB):
        tmp = _LIB + ".tmp%d" % os.getpid()
        subprocess.run(
            ["gcc", "-O2", "-fopenmp", "-fPIC", "-shared", "-Wall", "-o", tmp, _SRC, "-lm"],
            check=True,
        )
        os.replace(tmp, _LIB)
    return _LIB


def _load():
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(_LIB):
        build(force=True)
    lib = ctypes.CDLL(_LIB)
    i32, i64, f64, vp = ctypes.c_int32, ctypes.c_int64, ctypes.c_double, ctypes.c_void_p
    lib.oracle_kv_append.argtypes = [i32, i32, i32, i32, i32, i32, vp, vp, vp, vp, vp, vp, vp]
    lib.oracle_kv_append.restype = ctypes.c_int
    lib.oracle_attention.argtypes = [i32, i32, i32, i32, i32, i32, i32, f64, i32, vp, vp, vp, vp,
                                     vp, vp, i64, vp, vp, vp, vp]
    lib.oracle_attention.restype = ctypes.c_int
    lib.oracle_argmax.argtypes = [i64, i64, i64, i32, vp, vp, vp]
    lib.oracle_argmax.restype = ctypes.c_int
    lib.oracle_lmhead_argmax.argtypes = [i64, vp, i32, i64, i32, vp, vp, vp, vp, vp]
    lib.oracle_lmhead_argmax.restype = ctypes.c_int
    lib.oracle_accept.argtypes = [i32, vp, vp, vp, vp, vp, vp]
    lib.oracle_accept.restype = ctypes.c_int
    lib.oracle_budget.argtypes = [i32, i32, vp, vp, vp, vp, vp, f64, f64, vp, vp, vp, vp, vp, vp, vp,
                                  vp]
    lib.oracle_budget.restype = ctypes.c_int
    lib.oracle_sample.argtypes = [i64, i64, i64, i32, vp, ctypes.c_float, ctypes.c_uint64,
                                  ctypes.c_uint32, vp]
    lib.oracle_sample.restype = ctypes.c_int
    lib.oracle_philox4x32_10.argtypes = [vp, vp, vp]
    lib.oracle_philox4x32_10.restype = None
    lib.oracle_sample_log.argtypes = [i64, vp, vp]
    lib.oracle_sample_log.restype = None
    lib.oracle_gumbel_of_word.argtypes = [i64, vp, vp, vp]
    lib.oracle_gumbel_of_word.restype = None
    lib.oracle_num_threads.argtypes = []
    lib.oracle_num_threads.restype = ctypes.c_int
    _lib = lib
    return lib


def _ptr(a: np.ndarray):
    return a.ctypes.data_as(ctypes.c_void_p)


def _raw(a: np.ndarray, dtype_code: int) -> np.ndarray:
    """Element storage as expected by the C side: float32, or bf16 bits as uint16."""
    a = np.ascontiguousarray(a)
    if dtype_code == F32:
        if a.dtype != np.float32:
            raise TypeError("expected float32 storage, got %s" % a.dtype)
    else:
        if a.dtype not in (np.uint16, np.int16):
            raise TypeError("expected bf16 bit storage (uint16/int16), got %s" % a.dtype)
    return a


def num_threads() -> int:
    return int(_load().oracle_num_threads())


def attention(*, num_q_heads: int, num_kv_heads: int, head_dim: int, sliding_window: int,
              scale: float, dtype: int, q, k_cache, v_cache, block_tables, seq_lens, q_start,
              rows=None, heads=None, sinks=None) -> np.ndarray:
    """Attention output (float64) for the given (row, head) pairs.

    ``rows``/``heads`` are equal-length int arrays; both None means every pair in
    row-major order, returned with shape [T, Hq, D]; otherwise shape [P, D].
    ``sinks``: optional [Hq] sink logits (one extra softmax logit per head with
    a zero value, in the units of the scaled scores).
    """
    lib = _load()
    q = _raw(q, dtype)
    k_cache = _raw(k_cache, dtype)
    v_cache = _raw(v_cache, dtype)
    bt = np.ascontiguousarray(block_tables, dtype=np.int32)
    sl = np.ascontiguousarray(seq_lens, dtype=np.int32)
    qs = np.ascontiguousarray(q_start, dtype=np.int32)
    num_seqs = sl.shape[0]
    total_q = int(qs[-1])
    full = rows is None and heads is None
    if full:
        rr, hh = np.meshgrid(np.arange(total_q, dtype=np.int32),
                             np.arange(num_q_heads, dtype=np.int32), indexing="ij")
        rows, heads = rr.reshape(-1), hh.reshape(-1)
    rows = np.ascontiguousarray(rows, dtype=np.int32)
    heads = np.ascontiguousarray(heads, dtype=np.int32)
    out = np.zeros((rows.shape[0], head_dim), dtype=np.float64)
    sk = None if sinks is None else np.ascontiguousarray(sinks, dtype=np.float64)
    if sk is not None and sk.shape != (num_q_heads,):
        raise ValueError("sinks must have one entry per query head")
    num_blocks = k_cache.size // (num_kv_heads * head_dim * 16)
    rc = lib.oracle_attention(num_seqs, num_q_heads, num_kv_heads, head_dim, bt.shape[1],
                              num_blocks, sliding_window, float(scale), dtype, _ptr(q), _ptr(k_cache),
                              _ptr(v_cache), _ptr(bt), _ptr(sl), _ptr(qs), rows.shape[0],
                              _ptr(rows), _ptr(heads), _ptr(sk) if sk is not None else None,
                              _ptr(out))
    if rc != 0:
        raise ValueError("oracle_attention rejected its arguments")
    if full:
        return out.reshape(total_q, num_q_heads, head_dim)
    return out


def kv_append(*, num_kv_heads: int, head_dim: int, dtype: int, k_new, v_new, block_tables,
              seq_lens, q_start, k_cache, v_cache):
    """Copies of k_cache / v_cache (storage bits) with the new tokens' K/V
    written into their slots (see oracle_kv_append)."""
    lib = _load()
    kn = _raw(k_new, dtype)
    vn = _raw(v_new, dtype)
    kc = np.array(_raw(k_cache, dtype), copy=True, order="C")
    vc = np.array(_raw(v_cache, dtype), copy=True, order="C")
    bt = np.ascontiguousarray(block_tables, dtype=np.int32)
    sl = np.ascontiguousarray(seq_lens, dtype=np.int32)
    qs = np.ascontiguousarray(q_start, dtype=np.int32)
    rc = lib.oracle_kv_append(sl.shape[0], num_kv_heads, head_dim, bt.shape[1], kc.shape[0], dtype,
                              _ptr(kn), _ptr(vn), _ptr(bt), _ptr(sl), _ptr(qs), _ptr(kc), _ptr(vc))
    if rc != 0:
        raise ValueError("oracle_kv_append rejected its arguments")
    return kc, vc


def argmax(logits, dtype: int, with_gap: bool = True):
    """(argmax[int32], gap[float64] or None) for a [rows, vocab] logits array."""
    lib = _load()
    lg = _raw(logits, dtype)
    rows, vocab = lg.shape
    am = np.zeros(rows, dtype=np.int32)
    gap = np.zeros(rows, dtype=np.float64) if with_gap else None
    rc = lib.oracle_argmax(rows, vocab, vocab, dtype, _ptr(lg), _ptr(am),
                           _ptr(gap) if with_gap else None)
    if rc != 0:
        raise ValueError("oracle_argmax rejected its arguments")
    return am, gap


def lmhead_argmax(hidden_states, weight, dtype: int, rows=None, with_logits: bool = False):
    """Argmax (and gap to the runner-up) of the logits <hidden[r], weight[v]>
    for the selected rows (all if None), computed in double from the
    storage arrays hidden_states [T, H] and weight [V, H].  Returns
    (argmax, gap) or (argmax, gap, logits [n, V]) with with_logits."""
    lib = _load()
    hs = _raw(hidden_states, dtype)
    w = _raw(weight, dtype)
    T, H = hs.shape
    V, H2 = w.shape
    if H != H2:
        raise ValueError("hidden sizes differ: %d vs %d" % (H, H2))
    sel = np.arange(T, dtype=np.int32) if rows is None else np.ascontiguousarray(rows, dtype=np.int32)
    if sel.size and (sel.min() < 0 or sel.max() >= T):
        raise ValueError("selected row out of range")
    am = np.zeros(sel.size, dtype=np.int32)
    gap = np.zeros(sel.size, dtype=np.float64)
    lg = np.zeros((sel.size, V), dtype=np.float64) if with_logits else None
    rc = lib.oracle_lmhead_argmax(sel.size, _ptr(sel), H, V, dtype, _ptr(hs), _ptr(w), _ptr(am),
                                  _ptr(gap), _ptr(lg) if with_logits else None)
    if rc != 0:
        raise ValueError("oracle_lmhead_argmax rejected its arguments")
    return (am, gap, lg) if with_logits else (am, gap)


def inv_temperature(temperature: float) -> np.float32:
    """The fp32 1/T both sides multiply the logits by."""
    return np.float32(1.0 / float(temperature))


def sample(logits, dtype: int, temperature: float, seed: int, offset: int = 0) -> np.ndarray:
    """Each row's token drawn from softmax(logits / T) by the Gumbel-max rule
    (see oracle_sample): the stochastic verification's per-row sample."""
    lib = _load()
    lg = _raw(logits, dtype)
    rows, vocab = lg.shape
    out = np.zeros(rows, dtype=np.int32)
    rc = lib.oracle_sample(rows, vocab, vocab, dtype, _ptr(lg), float(inv_temperature(temperature)),
                           int(seed) & ((1 << 64) - 1), int(offset) & 0xFFFFFFFF, _ptr(out))
    if rc != 0:
        raise ValueError("oracle_sample rejected its arguments")
    return out


def philox4x32_10(ctr, key) -> np.ndarray:
    """One Philox4x32-10 block: 4 counter words, 2 key words -> 4 output words."""
    c = np.ascontiguousarray(ctr, dtype=np.uint32)
    k = np.ascontiguousarray(key, dtype=np.uint32)
    out = np.zeros(4, dtype=np.uint32)
    _load().oracle_philox4x32_10(_ptr(c), _ptr(k), _ptr(out))
    return out


def sample_log(x) -> np.ndarray:
    """The fp32 natural log the sampler's Gumbel noise uses."""
    a = np.ascontiguousarray(x, dtype=np.float32)
    out = np.zeros_like(a)
    _load().oracle_sample_log(a.size, _ptr(a), _ptr(out))
    return out


def gumbel_of_word(w):
    """(u, g): the uniform and the Gumbel noise term the sampler derives from
    raw Philox output words."""
    a = np.ascontiguousarray(w, dtype=np.uint32)
    u = np.zeros(a.shape, dtype=np.float32)
    g = np.zeros(a.shape, dtype=np.float32)
    _load().oracle_gumbel_of_word(a.size, _ptr(a), _ptr(u), _ptr(g))
    return u, g


def accept(q_start, tokens, argmax_rows):
    """(accept_len, num_emitted, emitted) for greedy acceptance."""
    lib = _load()
    qs = np.ascontiguousarray(q_start, dtype=np.int32)
    tok = np.ascontiguousarray(tokens, dtype=np.int32)
    am = np.ascontiguousarray(argmax_rows, dtype=np.int32)
    num_seqs = qs.shape[0] - 1
    acc = np.zeros(num_seqs, dtype=np.int32)
    ne = np.zeros(num_seqs, dtype=np.int32)
    em = np.zeros(tok.shape[0], dtype=np.int32)
    lib.oracle_accept(num_seqs, _ptr(qs), _ptr(tok), _ptr(am), _ptr(acc), _ptr(ne), _ptr(em))
    return acc, ne, em


def budget(cand_start, cand_len, cand_tokens, last_token, alpha: float, g_min: float,
           ctx_len=None):
    """Draft lengths of the next verify step (see oracle_budget in oracle.c).

    cand_tokens is [C, max_len]; returns a dict of numpy arrays: score,
    agree, prefix_len, source, draft_len, q_start, tokens (and seq_lens when
    ctx_len is given)."""
    lib = _load()
    cs = np.ascontiguousarray(cand_start, dtype=np.int32)
    cl = np.ascontiguousarray(cand_len, dtype=np.int32)
    ct = np.ascontiguousarray(cand_tokens, dtype=np.int32)
    if ct.ndim != 2:
        raise ValueError("cand_tokens must be [candidates, max_len]")
    lt = np.ascontiguousarray(last_token, dtype=np.int32)
    B = cs.shape[0] - 1
    max_len = ct.shape[1]
    cx = None if ctx_len is None else np.ascontiguousarray(ctx_len, dtype=np.int32)
    out = dict(score=np.zeros(B, np.float64), agree=np.zeros(B, np.int32),
               prefix_len=np.zeros(B, np.int32), source=np.zeros(B, np.int32),
               draft_len=np.zeros(B, np.int32), q_start=np.zeros(B + 1, np.int32),
               tokens=np.zeros(B * (max_len + 1), np.int32))
    if cx is not None:
        out["seq_lens"] = np.zeros(B, np.int32)
    rc = lib.oracle_budget(B, max_len, _ptr(cs), _ptr(cl), _ptr(ct), _ptr(lt),
                           _ptr(cx) if cx is not None else None, float(alpha), float(g_min),
                           _ptr(out["score"]), _ptr(out["agree"]), _ptr(out["prefix_len"]),
                           _ptr(out["source"]), _ptr(out["draft_len"]), _ptr(out["q_start"]),
                           _ptr(out["tokens"]), _ptr(out["seq_lens"]) if cx is not None else None)
    if rc != 0:
        raise ValueError("oracle_budget rejected its arguments")
    out["tokens"] = out["tokens"][: out["q_start"][-1]]
    return out


def rejection_rate(accept_len, q_start):
    """Per-request rejected / proposed drafts (NaN where no draft was proposed)."""
    k = np.diff(np.asarray(q_start)) - 1
    acc = np.asarray(accept_len)
    with np.errstate(invalid="ignore", divide="ignore"):
        return np.where(k > 0, (k - acc) / np.maximum(k, 1), np.nan)
