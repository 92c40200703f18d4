"""MI355X-native batched speculative-verification step (AgentSpec hot path).

Thin ctypes binding over the C ABI in ``include/agentspec_verify.h``: argument
marshalling only.  Every step of the verify pass runs in the HIP kernels of
``libagentspec_verify.so``; PyTorch supplies device memory and the stream.
If the library is missing, every entry point raises -- there is no fallback.

    verify_attention(...)      paged multi-query GQA attention of all scored rows
    verify_accept(...)         vocabulary argmax + greedy acceptance of the drafts
    verify_lmhead_accept(...)  the same acceptance fed by the LM head, logits
                               never stored
    verify_accept_sampled(...), verify_budget(...), verify_kv_append(...)
    verify_attention_append(...) the append and the attention in one launch
    check_batch(...)           the batch descriptor's preconditions, checked on
                               the device (the calls above take ``check=True``,
                               or every call does with AGENTSPEC_VERIFY_CHECK=1)
"""
from __future__ import annotations

import ctypes
import os
from typing import Optional

from .build import LIB_PATH

__all__ = ["verify_attention", "verify_accept", "verify_accept_noalloc", "verify_accept_sampled",
           "verify_lmhead_accept",
           "verify_budget", "verify_kv_append", "verify_attention_append",
           "attention_workspace_size", "attention_plan",
           "accept_workspace_size",
           "lmhead_accept_workspace_size", "check_batch", "BatchError", "VerifyError", "library",
           "abi_version", "F32", "BF16"]

OK, EINVAL, EUNSUPPORTED, EWORKSPACE, EHIP = 0, -1, -2, -3, -4
NOALLOC_SCRATCH_BYTES = 4 << 20  # VERIFY_NOALLOC_SCRATCH_BYTES of the C header
F32, BF16 = 0, 1
# verify_check_batch's counts, in the order of VERIFY_CHECK_ROWS .. _BLOCK_ID,
# then the first offending request (VERIFY_CHECK_FIRST)
CHECK_KINDS = ("rows", "q_len", "short_seq", "long_seq", "block_id")
CHECK_COUNTS = 6
CHECK_BY_DEFAULT = os.environ.get("AGENTSPEC_VERIFY_CHECK", "0") == "1"


class VerifyError(RuntimeError):
    def __init__(self, status: int, where: str):
        self.status = status
        super().__init__("%s: %s (status %d)" % (where, _status_string(status), status))


class BatchError(ValueError):
    """A batch descriptor that fails verify_check_batch: ``counts`` maps each
    kind in CHECK_KINDS to its number of offending requests, ``first`` is the
    lowest offending request."""

    def __init__(self, where: str, counts: dict, first: int):
        self.counts, self.first = counts, first
        bad = ", ".join("%s %d" % (k, v) for k, v in counts.items() if v)
        super().__init__("%s: bad batch descriptor (%s; first request %d)" % (where, bad, first))


class AttnParams(ctypes.Structure):
    _fields_ = [
        ("num_seqs", ctypes.c_int32),
        ("num_q_heads", ctypes.c_int32),
        ("num_kv_heads", ctypes.c_int32),
        ("head_dim", ctypes.c_int32),
        ("block_size", ctypes.c_int32),
        ("max_blocks_per_seq", ctypes.c_int32),
        ("num_blocks", ctypes.c_int32),
        ("sliding_window", ctypes.c_int32),
        ("scale", ctypes.c_float),
        ("dtype", ctypes.c_int32),
        ("kv_split_blocks", ctypes.c_int32),
    ]


_lib = None


def library(path: Optional[str] = None):
    """Load (once) and return the ctypes handle of the HIP library."""
    global _lib
    if _lib is not None and path is None:
        return _lib
    path = path or os.environ.get("AGENTSPEC_VERIFY_LIB", LIB_PATH)
    if not os.path.exists(path):
        raise RuntimeError("verify library not built: %s is missing "
                           "(run `python -m paper_2608_24004_amd.build`)" % path)
    lib = ctypes.CDLL(path)
    i32, i64, vp, sz = ctypes.c_int32, ctypes.c_int64, ctypes.c_void_p, ctypes.c_size_t
    P = ctypes.POINTER(AttnParams)
    lib.verify_attention_workspace_size.argtypes = [P, i32, i32, i32, ctypes.POINTER(sz)]
    lib.verify_attention_workspace_size.restype = ctypes.c_int
    lib.verify_attention.argtypes = [P, i32, i32, i32, vp, vp, vp, vp, vp, vp, vp, vp, vp, sz, vp]
    lib.verify_attention.restype = ctypes.c_int
    lib.verify_attention_plan.argtypes = [P, i32, i32, i32, ctypes.POINTER(i32)]
    lib.verify_attention_plan.restype = ctypes.c_int
    lib.verify_kv_append.argtypes = [P, i32, vp, vp, vp, vp, vp, vp, vp, vp]
    lib.verify_attention_append.argtypes = [P, i32, i32, i32, vp, vp, vp, vp, vp, vp, vp, vp, vp, vp,
                                            vp, sz, vp]
    lib.verify_attention_append.restype = ctypes.c_int
    lib.verify_kv_append.restype = ctypes.c_int
    lib.verify_accept_workspace_size.argtypes = [i32, i32, i64, i32, ctypes.POINTER(sz)]
    lib.verify_accept_workspace_size.restype = ctypes.c_int
    lib.verify_accept.argtypes = [i32, i32, i64, i64, i32, vp, vp, vp, vp, vp, vp, vp, vp, sz, vp]
    lib.verify_accept.restype = ctypes.c_int
    lib.verify_accept_noalloc.argtypes = [i32, i32, i64, i64, i32, vp, vp, vp, vp, vp, vp, vp, vp]
    lib.verify_accept_noalloc.restype = ctypes.c_int
    lib.verify_accept_sampled.argtypes = [i32, i32, i64, i64, i32, vp, vp, vp, ctypes.c_float,
                                          ctypes.c_uint64, ctypes.c_uint32, vp, vp, vp, vp, vp, sz, vp]
    lib.verify_accept_sampled.restype = ctypes.c_int
    f64 = ctypes.c_double
    lib.verify_lmhead_accept_workspace_size.argtypes = [i32, i32, i32, i64, i32, ctypes.POINTER(sz)]
    lib.verify_lmhead_accept_workspace_size.restype = ctypes.c_int
    lib.verify_lmhead_accept.argtypes = [i32, i32, i32, i64, i32, vp, vp, vp, vp, vp, vp, vp, vp, vp,
                                         sz, vp]
    lib.verify_lmhead_accept.restype = ctypes.c_int
    lib.verify_budget.argtypes = [i32, i32, i32, vp, vp, vp, vp, vp, f64, f64, vp, vp, vp, vp, vp, vp,
                                  vp, i64, vp, vp]
    lib.verify_budget.restype = ctypes.c_int
    lib.verify_check_batch.argtypes = [i32, i32, i32, vp, P, i32, vp, vp, vp, vp]
    lib.verify_check_batch.restype = ctypes.c_int
    lib.verify_status_string.argtypes = [ctypes.c_int]
    lib.verify_status_string.restype = ctypes.c_char_p
    lib.verify_abi_version.argtypes = []
    lib.verify_abi_version.restype = ctypes.c_int
    if path == LIB_PATH or _lib is None:
        _lib = lib
    return lib


def _status_string(status: int) -> str:
    try:
        return library().verify_status_string(status).decode()
    except Exception:
        return "status %d" % status


def abi_version() -> int:
    return int(library().verify_abi_version())


def _check(status: int, where: str):
    if status != OK:
        raise VerifyError(status, where)


def _dtype_code(t) -> int:
    import torch
    if t.dtype == torch.bfloat16:
        return BF16
    if t.dtype == torch.float32:
        return F32
    raise TypeError("unsupported storage dtype %s (bf16 or fp32)" % t.dtype)


def _dev_ptr(t, name, dtype=None):
    if t is None:
        return None
    if not t.is_cuda:
        raise ValueError("%s must be a device tensor" % name)
    if not t.is_contiguous():
        raise ValueError("%s must be contiguous" % name)
    if dtype is not None and t.dtype != dtype:
        raise TypeError("%s must be %s, got %s" % (name, dtype, t.dtype))
    return ctypes.c_void_p(t.data_ptr())


def _expect(t, name, shape=None, dtype=None, device=None):
    """Check a caller tensor before its pointer crosses the ABI.

    The kernels index device memory by the sizes passed beside the pointers,
    so a tensor smaller than those sizes would be read or written out of
    bounds, and one on another device would be read through the wrong
    address space."""
    if t is None:
        raise ValueError("%s is required" % name)
    if shape is not None and tuple(t.shape) != tuple(shape):
        raise ValueError("%s must have shape %s, got %s" % (name, tuple(shape), tuple(t.shape)))
    if dtype is not None and t.dtype != dtype:
        raise TypeError("%s must be %s, got %s" % (name, dtype, t.dtype))
    if device is not None and t.device != device:
        raise ValueError("%s is on %s, the call runs on %s" % (name, t.device, device))


def _check_attention_tensors(q, k_cache, v_cache, block_tables, seq_lens=None, q_start=None,
                             sinks=None, out=None, workspace=None):
    import torch
    if q.dim() != 3:
        raise ValueError("q must be [T, Hq, D], got %s" % (tuple(q.shape),))
    T, Hq, D = q.shape
    if k_cache.dim() != 5:
        raise ValueError("k_cache must be [num_blocks, Hkv, D/x, 16, x], got %s" % (tuple(k_cache.shape),))
    nb, hkv = k_cache.shape[0], k_cache.shape[1]
    x = 16 // q.element_size()
    dev, i32 = q.device, torch.int32
    _expect(k_cache, "k_cache", (nb, hkv, D // x, 16, x), q.dtype, dev)
    _expect(v_cache, "v_cache", (nb, hkv, D, 16), q.dtype, dev)
    if block_tables.dim() != 2:
        raise ValueError("block_tables must be [B, max_blocks], got %s" % (tuple(block_tables.shape),))
    B = block_tables.shape[0]
    _expect(block_tables, "block_tables", None, i32, dev)
    if seq_lens is not None:
        _expect(seq_lens, "seq_lens", (B,), i32, dev)
    if q_start is not None:
        _expect(q_start, "q_start", (B + 1,), i32, dev)
    if sinks is not None:
        _expect(sinks, "sinks", (Hq,), torch.float32, dev)
    if out is not None:
        _expect(out, "out", tuple(q.shape), q.dtype, dev)
    if workspace is not None:
        _expect(workspace, "workspace", None, None, dev)


def _stream_ptr(stream, device):
    import torch
    s = stream if stream is not None else torch.cuda.current_stream(device)
    return ctypes.c_void_p(s.cuda_stream)


def _attn_params(q, k_cache, block_tables, sliding_window, scale, kv_split_blocks):
    T, Hq, D = q.shape
    params = AttnParams()
    params.num_seqs = block_tables.shape[0]
    params.num_q_heads = Hq
    params.num_kv_heads = k_cache.shape[1]
    params.head_dim = D
    params.block_size = k_cache.shape[3]
    params.max_blocks_per_seq = block_tables.shape[1]
    params.num_blocks = k_cache.shape[0]
    params.sliding_window = int(sliding_window)
    params.scale = float(scale)
    params.dtype = _dtype_code(q)
    params.kv_split_blocks = int(kv_split_blocks)
    return params


def check_batch(q_start, total_q: int, *, max_q_len: int = 0, seq_lens=None, block_tables=None,
                num_blocks: int = 0, max_seq_len: int = 0, sliding_window: int = 0, stream=None):
    """The batch descriptor's preconditions, checked on the device by
    verify_check_batch.  Waits for the call's stream and returns (counts,
    first): offending requests per kind of CHECK_KINDS, and the lowest
    offending request (-1 if none).

    Only q_start (and n_i <= max_q_len when max_q_len > 0) is checked unless
    seq_lens is given; then also n_i <= S_i <= max_seq_len, and with
    block_tables and num_blocks the ids of every block the rows can read
    (keys from the first row's window start, sliding_window > 0, or 0)."""
    import torch
    i32 = torch.int32
    if q_start.dim() != 1 or q_start.shape[0] < 1:
        raise ValueError("q_start must be [B + 1], got %s" % (tuple(q_start.shape),))
    B = q_start.shape[0] - 1
    dev = q_start.device
    params = None
    if seq_lens is not None:
        _expect(seq_lens, "seq_lens", (B,), i32, dev)
        params = AttnParams(num_seqs=B, block_size=16, num_blocks=int(num_blocks),
                            sliding_window=int(sliding_window),
                            max_blocks_per_seq=(1 << 31) // 16 - 1)
        if block_tables is not None:
            if block_tables.dim() != 2 or block_tables.shape[0] != B or block_tables.shape[1] < 1:
                raise ValueError("block_tables must be [B, max_blocks], got %s"
                                 % (tuple(block_tables.shape),))
            _expect(block_tables, "block_tables", None, i32, dev)
            params.max_blocks_per_seq = block_tables.shape[1]
    elif block_tables is not None:
        raise ValueError("block_tables are checked against seq_lens, which is missing")
    counts = torch.empty(CHECK_COUNTS, dtype=i32, device=dev)
    rc = library().verify_check_batch(
        B, int(total_q), int(max_q_len), _dev_ptr(q_start, "q_start", i32),
        ctypes.byref(params) if params is not None else None, int(max_seq_len),
        _dev_ptr(seq_lens, "seq_lens", i32), _dev_ptr(block_tables, "block_tables", i32),
        _dev_ptr(counts, "counts", i32), _stream_ptr(stream, dev))
    _check(rc, "verify_check_batch")
    (stream if stream is not None else torch.cuda.current_stream(dev)).synchronize()
    c = counts.cpu().tolist()
    return dict(zip(CHECK_KINDS, c[:len(CHECK_KINDS)])), (c[-1] if c[-1] != 2 ** 31 - 1 else -1)


def _checked(check, where, **kw):
    """Raise BatchError before `where` launches anything if the descriptor
    fails verify_check_batch (with check=True, or by default when
    AGENTSPEC_VERIFY_CHECK=1)."""
    if not (CHECK_BY_DEFAULT if check is None else check):
        return
    counts, first = check_batch(**kw)
    if any(counts.values()):
        raise BatchError(where, counts, first)


def attention_workspace_size(q, k_cache, block_tables, *, max_q_len: int, max_seq_len: int,
                             sliding_window: int = 0, scale: float = 0.0,
                             kv_split_blocks: int = 0) -> int:
    params = _attn_params(q, k_cache, block_tables, sliding_window, scale, kv_split_blocks)
    n = ctypes.c_size_t(0)
    _check(library().verify_attention_workspace_size(ctypes.byref(params), q.shape[0], int(max_q_len),
                                                     int(max_seq_len), ctypes.byref(n)),
           "verify_attention_workspace_size")
    return int(n.value)


PLAN_INFO = 11  # entries of verify_attention_plan's info array


def attention_plan(q, k_cache, block_tables, *, max_q_len: int, max_seq_len: int,
                   sliding_window: int = 0, scale: float = 0.0, kv_split_blocks: int = 0) -> dict:
    """The work decomposition verify_attention would use (nothing is launched)."""
    p = _attn_params(q, k_cache, block_tables, sliding_window, scale, kv_split_blocks)
    info = (ctypes.c_int32 * PLAN_INFO)()
    _check(library().verify_attention_plan(ctypes.byref(p), int(q.shape[0]), int(max_q_len),
                                           int(max_seq_len), info), "verify_attention_plan")
    v = [int(x) for x in info]
    if not v[0]:
        return dict(zip(("mfma", "splits", "rows_per_item", "row_groups", "split_blocks"), v[:5]))
    # bf16: one persistent launch per row class (requests by Hq/Hkv * n_i)
    keys = ("workgroups", "rows_per_group", "row_groups", "units_per_workgroup")
    classes = [dict(zip(keys, v[1:5]), rows_lo=0, rows_hi=v[10])]
    if v[5] > 1:
        classes.append(dict(zip(keys, v[6:10]), rows_lo=v[10] + 1, rows_hi=2 ** 31 - 1))
    return dict(mfma=1, classes=classes, **classes[0])


def verify_attention(q, k_cache, v_cache, block_tables, seq_lens, q_start, *, max_q_len: int,
                     max_seq_len: int, sliding_window: int = 0, scale: float = 0.0,
                     kv_split_blocks: int = 0, sinks=None, out=None, workspace=None,
                     stream=None, check=None):
    """Attention of every packed query row against its request's paged KV cache.

    q [T, Hq, D]; k_cache [NB, Hkv, D/x, 16, x]; v_cache [NB, Hkv, D, 16] (bf16 or
    fp32, x = 16 bytes / element); block_tables [B, MB], seq_lens [B], q_start
    [B+1] int32 on the device.  max_q_len / max_seq_len are host upper bounds of
    n_i = q_start[i+1]-q_start[i] and S_i = seq_lens[i].  sinks: optional [Hq]
    float32 device tensor of per-head sink logits.  Returns `out`.  check:
    validate the descriptor on the device first (check_batch; raises
    BatchError, waits for the stream).
    """
    import torch
    _check_attention_tensors(q, k_cache, v_cache, block_tables, seq_lens, q_start, sinks, out,
                             workspace)
    _checked(check, "verify_attention", q_start=q_start, total_q=q.shape[0], max_q_len=max_q_len,
             seq_lens=seq_lens, block_tables=block_tables, num_blocks=k_cache.shape[0],
             max_seq_len=max_seq_len, sliding_window=sliding_window, stream=stream)
    params = _attn_params(q, k_cache, block_tables, sliding_window, scale, kv_split_blocks)
    if out is None:
        out = torch.empty_like(q)
    ws_bytes = attention_workspace_size(q, k_cache, block_tables, max_q_len=max_q_len,
                                        max_seq_len=max_seq_len, sliding_window=sliding_window,
                                        scale=scale, kv_split_blocks=kv_split_blocks)
    if workspace is None and ws_bytes > 0:
        workspace = torch.empty(ws_bytes, dtype=torch.uint8, device=q.device)
    ws_have = workspace.numel() * workspace.element_size() if workspace is not None else 0
    i32 = torch.int32
    rc = library().verify_attention(
        ctypes.byref(params), q.shape[0], int(max_q_len), int(max_seq_len),
        _dev_ptr(q, "q"), _dev_ptr(k_cache, "k_cache", q.dtype), _dev_ptr(v_cache, "v_cache", q.dtype),
        _dev_ptr(block_tables, "block_tables", i32), _dev_ptr(seq_lens, "seq_lens", i32),
        _dev_ptr(q_start, "q_start", i32), _dev_ptr(sinks, "sinks", torch.float32),
        _dev_ptr(out, "out", q.dtype), _dev_ptr(workspace, "workspace"), ws_have,
        _stream_ptr(stream, q.device))
    _check(rc, "verify_attention")
    return out


def verify_attention_append(q, k_new, v_new, k_cache, v_cache, block_tables, seq_lens, q_start, *,
                            max_q_len: int, max_seq_len: int, sliding_window: int = 0,
                            scale: float = 0.0, kv_split_blocks: int = 0, sinks=None, out=None,
                            workspace=None, stream=None, check=None):
    """verify_kv_append and verify_attention in one launch sequence: the new
    tokens' K/V (k_new, v_new [T, Hkv, D], the cache's dtype) are stored into
    k_cache / v_cache in place while the attention reads them from k_new /
    v_new.  Same arguments and result as verify_attention; returns `out`."""
    import torch
    _check_attention_tensors(q, k_cache, v_cache, block_tables, seq_lens, q_start, sinks, out,
                             workspace)
    shape = (q.shape[0], k_cache.shape[1], q.shape[2])
    _expect(k_new, "k_new", shape, q.dtype, q.device)
    _expect(v_new, "v_new", shape, q.dtype, q.device)
    _checked(check, "verify_attention_append", q_start=q_start, total_q=q.shape[0],
             max_q_len=max_q_len, seq_lens=seq_lens, block_tables=block_tables,
             num_blocks=k_cache.shape[0], max_seq_len=max_seq_len, sliding_window=sliding_window,
             stream=stream)
    params = _attn_params(q, k_cache, block_tables, sliding_window, scale, kv_split_blocks)
    if out is None:
        out = torch.empty_like(q)
    ws_bytes = attention_workspace_size(q, k_cache, block_tables, max_q_len=max_q_len,
                                        max_seq_len=max_seq_len, sliding_window=sliding_window,
                                        scale=scale, kv_split_blocks=kv_split_blocks)
    if workspace is None and ws_bytes > 0:
        workspace = torch.empty(ws_bytes, dtype=torch.uint8, device=q.device)
    ws_have = workspace.numel() * workspace.element_size() if workspace is not None else 0
    i32 = torch.int32
    rc = library().verify_attention_append(
        ctypes.byref(params), q.shape[0], int(max_q_len), int(max_seq_len), _dev_ptr(q, "q"),
        _dev_ptr(k_new, "k_new", q.dtype), _dev_ptr(v_new, "v_new", q.dtype),
        _dev_ptr(k_cache, "k_cache", q.dtype), _dev_ptr(v_cache, "v_cache", q.dtype),
        _dev_ptr(block_tables, "block_tables", i32), _dev_ptr(seq_lens, "seq_lens", i32),
        _dev_ptr(q_start, "q_start", i32), _dev_ptr(sinks, "sinks", torch.float32),
        _dev_ptr(out, "out", q.dtype), _dev_ptr(workspace, "workspace"), ws_have,
        _stream_ptr(stream, q.device))
    _check(rc, "verify_attention_append")
    return out


def accept_workspace_size(num_seqs: int, total_q: int, vocab: int, dtype_code: int) -> int:
    n = ctypes.c_size_t(0)
    _check(library().verify_accept_workspace_size(int(num_seqs), int(total_q), int(vocab),
                                                  int(dtype_code), ctypes.byref(n)),
           "verify_accept_workspace_size")
    return int(n.value)


def _accept_buffers(logits, q_start, argmax_out, accept_len, num_emitted, emitted, workspace,
                    need_workspace=True):
    import torch
    if logits.dim() != 2:
        raise ValueError("logits must be [T, V], got %s" % (tuple(logits.shape),))
    T, V = logits.shape
    if q_start.dim() != 1 or q_start.shape[0] < 1:
        raise ValueError("q_start must be [B + 1], got %s" % (tuple(q_start.shape),))
    B = q_start.shape[0] - 1
    dev = logits.device
    i32 = torch.int32
    _expect(q_start, "q_start", None, i32, dev)
    for name, t, n in (("argmax_out", argmax_out, T), ("accept_len", accept_len, B),
                       ("num_emitted", num_emitted, B), ("emitted", emitted, T)):
        if t is not None:
            _expect(t, name, (n,), i32, dev)
    if workspace is not None:
        _expect(workspace, "workspace", None, None, dev)
    code = _dtype_code(logits)
    if argmax_out is None:
        argmax_out = torch.empty(T, dtype=i32, device=dev)
    if accept_len is None:
        accept_len = torch.empty(B, dtype=i32, device=dev)
    if num_emitted is None:
        num_emitted = torch.empty(B, dtype=i32, device=dev)
    if emitted is None:
        emitted = torch.empty(T, dtype=i32, device=dev)
    ws_bytes = accept_workspace_size(B, T, V, code) if need_workspace else 0
    if workspace is None and ws_bytes > 0:
        workspace = torch.empty(ws_bytes, dtype=torch.uint8, device=dev)
    ws_have = workspace.numel() * workspace.element_size() if workspace is not None else 0
    return B, T, V, code, argmax_out, accept_len, num_emitted, emitted, workspace, ws_have


def verify_accept(logits, tokens, q_start, *, argmax_out=None, accept_len=None, num_emitted=None,
                  emitted=None, workspace=None, stream=None, check=None):
    """Vocabulary argmax of every row and greedy acceptance of the drafts.

    logits [T, V] (bf16 or fp32), tokens [T] and q_start [B+1] int32 on the
    device.  Returns (accept_len [B], num_emitted [B], emitted [T], argmax [T]).
    check: validate q_start on the device first (check_batch).
    """
    import torch
    i32 = torch.int32
    B, T, V, code, argmax_out, accept_len, num_emitted, emitted, workspace, ws_have = \
        _accept_buffers(logits, q_start, argmax_out, accept_len, num_emitted, emitted, workspace)
    _expect(tokens, "tokens", (T,), i32, logits.device)
    _checked(check, "verify_accept", q_start=q_start, total_q=T, stream=stream)
    rc = library().verify_accept(
        B, T, V, V, code, _dev_ptr(logits, "logits"), _dev_ptr(tokens, "tokens", i32),
        _dev_ptr(q_start, "q_start", i32), _dev_ptr(argmax_out, "argmax_out", i32),
        _dev_ptr(accept_len, "accept_len", i32), _dev_ptr(num_emitted, "num_emitted", i32),
        _dev_ptr(emitted, "emitted", i32), _dev_ptr(workspace, "workspace"), ws_have,
        _stream_ptr(stream, logits.device))
    _check(rc, "verify_accept")
    return accept_len, num_emitted, emitted, argmax_out


def verify_accept_noalloc(logits, tokens, q_start, *, argmax_out=None, accept_len=None,
                          num_emitted=None, emitted=None, stream=None, check=None):
    """verify_accept without a workspace: the library's per-GPU scratch array
    holds the partial maxima (for callers that cannot allocate; calls that
    overlap on one GPU race).  Outputs not passed in are allocated here, by
    torch, before the call; the C call allocates nothing.  Returns
    (accept_len [B], num_emitted [B], emitted [T], argmax [T])."""
    import torch
    i32 = torch.int32
    B, T, V, code, argmax_out, accept_len, num_emitted, emitted, _, _ = \
        _accept_buffers(logits, q_start, argmax_out, accept_len, num_emitted, emitted, None,
                        need_workspace=False)
    _expect(tokens, "tokens", (T,), i32, logits.device)
    _checked(check, "verify_accept_noalloc", q_start=q_start, total_q=T, stream=stream)
    rc = library().verify_accept_noalloc(
        B, T, V, V, code, _dev_ptr(logits, "logits"), _dev_ptr(tokens, "tokens", i32),
        _dev_ptr(q_start, "q_start", i32), _dev_ptr(argmax_out, "argmax_out", i32),
        _dev_ptr(accept_len, "accept_len", i32), _dev_ptr(num_emitted, "num_emitted", i32),
        _dev_ptr(emitted, "emitted", i32), _stream_ptr(stream, logits.device))
    _check(rc, "verify_accept_noalloc")
    return accept_len, num_emitted, emitted, argmax_out


def verify_accept_sampled(logits, tokens, q_start, *, temperature: float, seed: int, offset: int = 0,
                          sampled_out=None, accept_len=None, num_emitted=None, emitted=None,
                          workspace=None, stream=None, check=None):
    """Stochastic verification at temperature T > 0: every row draws
    y ~ softmax(logits / T) (Gumbel-max with Philox4x32-10 noise keyed by
    `seed`, counter (v / 4, row, offset, 0)) and a request accepts its drafts
    up to the first one that differs from its row's draw.

    Same layouts as verify_accept.  Returns (accept_len [B], num_emitted [B],
    emitted [T], sampled [T]).
    """
    import torch
    i32 = torch.int32
    if not 0 <= int(seed) < (1 << 64) or not 0 <= int(offset) < (1 << 32):
        raise ValueError("seed must fit 64 bits and offset 32 bits, unsigned")
    B, T, V, code, sampled_out, accept_len, num_emitted, emitted, workspace, ws_have = \
        _accept_buffers(logits, q_start, sampled_out, accept_len, num_emitted, emitted, workspace)
    _expect(tokens, "tokens", (T,), i32, logits.device)
    _checked(check, "verify_accept_sampled", q_start=q_start, total_q=T, stream=stream)
    rc = library().verify_accept_sampled(
        B, T, V, V, code, _dev_ptr(logits, "logits"), _dev_ptr(tokens, "tokens", i32),
        _dev_ptr(q_start, "q_start", i32), float(temperature), int(seed), int(offset),
        _dev_ptr(sampled_out, "sampled_out", i32), _dev_ptr(accept_len, "accept_len", i32),
        _dev_ptr(num_emitted, "num_emitted", i32), _dev_ptr(emitted, "emitted", i32),
        _dev_ptr(workspace, "workspace"), ws_have, _stream_ptr(stream, logits.device))
    _check(rc, "verify_accept_sampled")
    return accept_len, num_emitted, emitted, sampled_out


def lmhead_accept_workspace_size(num_seqs: int, total_q: int, hidden_size: int, vocab: int,
                                 dtype_code: int = BF16) -> int:
    n = ctypes.c_size_t(0)
    _check(library().verify_lmhead_accept_workspace_size(int(num_seqs), int(total_q), int(hidden_size),
                                                         int(vocab), int(dtype_code), ctypes.byref(n)),
           "verify_lmhead_accept_workspace_size")
    return int(n.value)


def verify_lmhead_accept(hidden, weight, tokens, q_start, *, argmax_out=None, accept_len=None,
                         num_emitted=None, emitted=None, workspace=None, stream=None, check=None):
    """LM head fused with greedy acceptance: logits <hidden[r], weight[v]> are
    reduced to each row's argmax inside the kernel (never stored), then the
    drafts are accepted as in verify_accept.

    hidden [T, H] and weight [V, H] bf16, tokens [T] and q_start [B+1] int32,
    all on the device.  Returns (accept_len [B], num_emitted [B], emitted [T],
    argmax [T]).
    """
    import torch
    i32 = torch.int32
    if hidden.dim() != 2 or weight.dim() != 2:
        raise ValueError("hidden must be [T, H] and weight [V, H]")
    T, H = hidden.shape
    V, H2 = weight.shape
    if H != H2:
        raise ValueError("hidden sizes differ: %d vs %d" % (H, H2))
    if q_start.dim() != 1 or q_start.shape[0] < 1:
        raise ValueError("q_start must be [B + 1], got %s" % (tuple(q_start.shape),))
    B = q_start.shape[0] - 1
    dev = hidden.device
    _expect(weight, "weight", None, hidden.dtype, dev)
    _expect(tokens, "tokens", (T,), i32, dev)
    _expect(q_start, "q_start", None, i32, dev)
    for name, t, n in (("argmax_out", argmax_out, T), ("accept_len", accept_len, B),
                       ("num_emitted", num_emitted, B), ("emitted", emitted, T)):
        if t is not None:
            _expect(t, name, (n,), i32, dev)
    if workspace is not None:
        _expect(workspace, "workspace", None, None, dev)
    _checked(check, "verify_lmhead_accept", q_start=q_start, total_q=T, stream=stream)
    code = _dtype_code(hidden)
    if argmax_out is None:
        argmax_out = torch.empty(T, dtype=i32, device=dev)
    if accept_len is None:
        accept_len = torch.empty(B, dtype=i32, device=dev)
    if num_emitted is None:
        num_emitted = torch.empty(B, dtype=i32, device=dev)
    if emitted is None:
        emitted = torch.empty(T, dtype=i32, device=dev)
    ws_bytes = lmhead_accept_workspace_size(B, T, H, V, code)
    if workspace is None and ws_bytes > 0:
        workspace = torch.empty(ws_bytes, dtype=torch.uint8, device=dev)
    ws_have = workspace.numel() * workspace.element_size() if workspace is not None else 0
    rc = library().verify_lmhead_accept(
        B, T, H, V, code, _dev_ptr(hidden, "hidden"), _dev_ptr(weight, "weight", hidden.dtype),
        _dev_ptr(tokens, "tokens", i32), _dev_ptr(q_start, "q_start", i32),
        _dev_ptr(argmax_out, "argmax_out", i32), _dev_ptr(accept_len, "accept_len", i32),
        _dev_ptr(num_emitted, "num_emitted", i32), _dev_ptr(emitted, "emitted", i32),
        _dev_ptr(workspace, "workspace"), ws_have, _stream_ptr(stream, dev))
    _check(rc, "verify_lmhead_accept")
    return accept_len, num_emitted, emitted, argmax_out


def verify_budget(cand_start, cand_len, cand_tokens, last_token, *, alpha: float, g_min: float,
                  ctx_len=None, out=None, stream=None):
    """Redundancy-aware draft lengths (Sec. 4.2, Alg. 2) and the next verify
    step's descriptor.

    cand_start [B+1], cand_len [C], cand_tokens [C, max_len], last_token [B]
    and ctx_len [B] (optional) are int32 device tensors.  Returns a dict of
    device tensors: score (float64), agree, prefix_len, source, draft_len,
    q_start, tokens (capacity B * (max_len + 1); q_start[-1] entries used) and,
    with ctx_len, seq_lens.  ``out`` may hold preallocated tensors by name.
    """
    import torch
    if cand_start.dim() != 1 or cand_start.shape[0] < 1 or cand_tokens.dim() != 2:
        raise ValueError("cand_start must be [B + 1] and cand_tokens [C, max_len]")
    B = cand_start.shape[0] - 1
    C, max_len = cand_tokens.shape
    dev = cand_start.device
    i32 = torch.int32
    _expect(cand_len, "cand_len", (C,), i32, dev)
    _expect(cand_tokens, "cand_tokens", None, i32, dev)
    _expect(last_token, "last_token", (B,), i32, dev)
    if ctx_len is not None:
        _expect(ctx_len, "ctx_len", (B,), i32, dev)
    o = dict(out or {})
    shapes = dict(score=(B, torch.float64), agree=(B, i32), prefix_len=(B, i32), source=(B, i32),
                  draft_len=(B, i32), q_start=(B + 1, i32), tokens=(B * (max_len + 1), i32))
    if ctx_len is not None:
        shapes["seq_lens"] = (B, i32)
    for k, (n, dt) in shapes.items():
        if k not in o:
            o[k] = torch.empty(max(n, 1) if k == "tokens" else n, dtype=dt, device=dev)
        elif k == "tokens":
            # the capacity is passed to the call, which checks it
            _expect(o[k], k, None, dt, dev)
            if o[k].dim() != 1:
                raise ValueError("tokens must be one-dimensional")
        else:
            _expect(o[k], k, (n,), dt, dev)
    rc = library().verify_budget(
        B, C, max_len, _dev_ptr(cand_start, "cand_start", i32), _dev_ptr(cand_len, "cand_len", i32),
        _dev_ptr(cand_tokens, "cand_tokens", i32), _dev_ptr(last_token, "last_token", i32),
        _dev_ptr(ctx_len, "ctx_len", i32), float(alpha), float(g_min),
        _dev_ptr(o["score"], "score", torch.float64), _dev_ptr(o["agree"], "agree", i32),
        _dev_ptr(o["prefix_len"], "prefix_len", i32), _dev_ptr(o["source"], "source", i32),
        _dev_ptr(o["draft_len"], "draft_len", i32), _dev_ptr(o["q_start"], "q_start", i32),
        _dev_ptr(o["tokens"], "tokens", i32), o["tokens"].numel(),
        _dev_ptr(o.get("seq_lens"), "seq_lens", i32), _stream_ptr(stream, dev))
    _check(rc, "verify_budget")
    return o


def verify_kv_append(k_new, v_new, k_cache, v_cache, block_tables, seq_lens, q_start, *,
                     stream=None, check=None):
    """Write the new tokens' K/V ([T, Hkv, D], the cache's dtype) into their
    paged-cache slots (position S_i - n_i + j for row j of request i), in place.
    check: validate the descriptor and the new tokens' block ids on the device
    first (check_batch with a one-key window: only those blocks)."""
    import torch
    if k_new.dim() != 3:
        raise ValueError("k_new must be [T, Hkv, D], got %s" % (tuple(k_new.shape),))
    _expect(v_new, "v_new", tuple(k_new.shape), k_new.dtype, k_new.device)
    if q_start.dim() != 1 or q_start.shape[0] < 1:
        raise ValueError("q_start must be [B + 1], got %s" % (tuple(q_start.shape),))
    probe = torch.empty((0, k_new.shape[1], k_new.shape[2]), dtype=k_new.dtype, device=k_new.device)
    _check_attention_tensors(probe, k_cache, v_cache, block_tables, seq_lens, q_start)
    if k_cache.shape[1] != k_new.shape[1]:
        raise ValueError("k_new has %d KV heads, the cache %d" % (k_new.shape[1], k_cache.shape[1]))
    params = _attn_params(probe, k_cache, block_tables, 0, 0.0, 0)
    i32 = torch.int32
    _checked(check, "verify_kv_append", q_start=q_start, total_q=k_new.shape[0], seq_lens=seq_lens,
             block_tables=block_tables, num_blocks=k_cache.shape[0],
             max_seq_len=16 * block_tables.shape[1], sliding_window=1, stream=stream)
    rc = library().verify_kv_append(
        ctypes.byref(params), k_new.shape[0], _dev_ptr(k_new, "k_new"),
        _dev_ptr(v_new, "v_new", k_new.dtype), _dev_ptr(block_tables, "block_tables", i32),
        _dev_ptr(seq_lens, "seq_lens", i32), _dev_ptr(q_start, "q_start", i32),
        _dev_ptr(k_cache, "k_cache", k_new.dtype), _dev_ptr(v_cache, "v_cache", k_new.dtype),
        _stream_ptr(stream, k_new.device))
    _check(rc, "verify_kv_append")
