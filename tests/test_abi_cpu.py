"""The C-ABI library on the host: it loads, exports every declared symbol, and
rejects bad arguments with the documented status before touching the GPU."""
from __future__ import annotations

import ctypes
import glob
import os
import re

import pytest
import torch

import paper_2608_24004_amd as av

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def declared_symbols():
    names = set()
    for h in glob.glob(os.path.join(ROOT, "include", "*.h")):
        src = open(h).read()
        src = re.sub(r"/\*.*?\*/", "", src, flags=re.S)
        for m in re.finditer(r"^\s*(?:const\s+)?\w+\s*\*?\s*(verify_\w+)\s*\(", src, flags=re.M):
            names.add(m.group(1))
    return names


def test_header_declares_the_entry_points():
    names = declared_symbols()
    for n in ("verify_attention", "verify_accept", "verify_accept_sampled", "verify_budget",
              "verify_kv_append", "verify_attention_workspace_size",
              "verify_accept_workspace_size", "verify_lmhead_accept", "verify_accept_noalloc",
              "verify_lmhead_accept_workspace_size", "verify_check_batch", "verify_attention_append",
              "verify_status_string",
              "verify_abi_version"):
        assert n in names


def test_library_exports_every_declared_symbol():
    lib = av.library()
    for name in declared_symbols():
        assert hasattr(lib, name), name
    assert av.abi_version() == 10800
    assert lib.verify_status_string(0) == b"ok"
    assert lib.verify_status_string(-3) == b"workspace too small"


def test_binding_constants_match_the_header():
    """The binding's copies of the header's constants and enum values."""
    src = open(os.path.join(ROOT, "include", "agentspec_verify.h")).read()
    defs = {m.group(1): m.group(2).strip() for m in re.finditer(r"#define\s+(VERIFY_\w+)\s+([^\n]+)", src)}
    assert int(defs["VERIFY_ATTN_PLAN_INFO"]) == av.PLAN_INFO
    assert int(defs["VERIFY_CHECK_COUNTS"]) == av.CHECK_COUNTS == len(av.CHECK_KINDS) + 1
    m = re.fullmatch(r"\(\s*(\d+)u?\s*<<\s*(\d+)\s*\)", defs["VERIFY_NOALLOC_SCRATCH_BYTES"])
    assert m and int(m.group(1)) << int(m.group(2)) == av.NOALLOC_SCRATCH_BYTES
    order = ["VERIFY_CHECK_ROWS", "VERIFY_CHECK_QLEN", "VERIFY_CHECK_SHORT", "VERIFY_CHECK_LONG",
             "VERIFY_CHECK_BLOCK_ID"]
    assert [int(defs[k]) for k in order] == list(range(len(av.CHECK_KINDS)))
    assert int(defs["VERIFY_CHECK_FIRST"]) == len(av.CHECK_KINDS)
    enums = dict(re.findall(r"(VERIFY_E?\w+)\s*=\s*(-?\d+)", src))
    assert (int(enums["VERIFY_OK"]), int(enums["VERIFY_EINVAL"]), int(enums["VERIFY_EUNSUPPORTED"]),
            int(enums["VERIFY_EWORKSPACE"]), int(enums["VERIFY_EHIP"])) == (
        av.OK, av.EINVAL, av.EUNSUPPORTED, av.EWORKSPACE, av.EHIP)
    assert (int(enums["VERIFY_F32"]), int(enums["VERIFY_BF16"])) == (av.F32, av.BF16)


def test_missing_library_fails_loudly(tmp_path):
    with pytest.raises(RuntimeError, match="not built"):
        av.library(str(tmp_path / "nope.so"))


def _params(**kw):
    p = av.AttnParams()
    base = dict(num_seqs=4, num_q_heads=32, num_kv_heads=8, head_dim=128, block_size=16,
                max_blocks_per_seq=64, num_blocks=1000, sliding_window=0, scale=0.0,
                dtype=av.BF16, kv_split_blocks=0)
    base.update(kw)
    for k, v in base.items():
        setattr(p, k, v)
    return p


def _ws(p, total_q=36, max_q=9, max_s=1000):
    n = ctypes.c_size_t(0)
    rc = av.library().verify_attention_workspace_size(ctypes.byref(p), total_q, max_q, max_s,
                                                      ctypes.byref(n))
    return rc, n.value


@pytest.mark.parametrize("kw,want", [
    (dict(head_dim=96), av.EUNSUPPORTED),
    (dict(block_size=32), av.EUNSUPPORTED),
    (dict(dtype=7), av.EUNSUPPORTED),
    (dict(num_q_heads=30), av.EINVAL),        # not a multiple of Hkv
    (dict(num_kv_heads=0), av.EINVAL),
    (dict(num_seqs=-1), av.EINVAL),
    (dict(sliding_window=-5), av.EINVAL),
    (dict(scale=-1.0), av.EINVAL),
    (dict(scale=float("nan")), av.EINVAL),
    (dict(kv_split_blocks=-2), av.EINVAL),
    (dict(max_blocks_per_seq=0), av.EINVAL),
])
def test_attention_argument_validation(kw, want):
    rc, _ = _ws(_params(**kw))
    assert rc == want
    # the launch entry point reports the same status (it validates first)
    rc2 = av.library().verify_attention(ctypes.byref(_params(**kw)), 36, 9, 1000, *([None] * 8),
                                        None, 0, None)
    assert rc2 == want


def test_attention_workspace_query_and_checks():
    lib = av.library()
    # fp32 (split-K VALU path): 63 blocks / 8 per split -> 8 splits of fp32
    # partial outputs and log-sum-exps; a single split needs no workspace
    rc, n = _ws(_params(dtype=av.F32, kv_split_blocks=8), total_q=36, max_q=9, max_s=1000)
    assert rc == 0 and n >= 36 * 32 * 8 * (128 + 1) * 4
    rc, n1 = _ws(_params(dtype=av.F32, kv_split_blocks=1000), total_q=36, max_q=9, max_s=1000)
    assert rc == 0 and n1 == 0
    # bf16 (persistent MFMA path): per-request unit offsets plus partial slots,
    # growing with the number of workgroups (fewer units per workgroup)
    rc, a = _ws(_params(kv_split_blocks=64), total_q=36, max_q=9, max_s=1000)
    rc2, b = _ws(_params(kv_split_blocks=8), total_q=36, max_q=9, max_s=1000)
    assert rc == 0 and rc2 == 0 and 0 < a < b
    rc, auto = _ws(_params(), total_q=36, max_q=9, max_s=1000)
    assert rc == 0 and auto > 0
    assert lib.verify_attention_workspace_size(ctypes.byref(_params()), 36, 9, 1000, None) == av.EINVAL
    assert lib.verify_attention_workspace_size(None, 36, 9, 1000, ctypes.byref(ctypes.c_size_t())) == av.EINVAL
    # too small a workspace is refused before any launch (dummy non-null pointers)
    dummy = ctypes.c_void_p(0x1000)
    for kw, need in ((dict(dtype=av.F32, kv_split_blocks=8), n), (dict(kv_split_blocks=8), b)):
        rc = lib.verify_attention(ctypes.byref(_params(**kw)), 36, 9, 1000, dummy, dummy, dummy,
                                  dummy, dummy, dummy, None, dummy, dummy, need - 1, None)
        assert rc == av.EWORKSPACE
    # null required pointers
    rc = lib.verify_attention(ctypes.byref(_params()), 36, 9, 1000, None, dummy, dummy, dummy,
                              dummy, dummy, None, dummy, dummy, auto, None)
    assert rc == av.EINVAL
    # negative host sizes
    assert _ws(_params(), total_q=-1)[0] == av.EINVAL
    assert _ws(_params(), max_s=-1)[0] == av.EINVAL
    # units beyond the 32-bit unit index are refused
    assert _ws(_params(num_seqs=65535, max_blocks_per_seq=1 << 20), max_s=1 << 24)[0] == av.EUNSUPPORTED


def test_accept_argument_validation():
    lib = av.library()
    n = ctypes.c_size_t(0)
    assert lib.verify_accept_workspace_size(4, 40, 151936, av.BF16, ctypes.byref(n)) == 0
    assert n.value >= 40 * 8
    assert lib.verify_accept_workspace_size(4, 40, 0, av.BF16, ctypes.byref(n)) == av.EINVAL
    assert lib.verify_accept_workspace_size(4, 40, 1 << 31, av.BF16, ctypes.byref(n)) == av.EINVAL
    assert lib.verify_accept_workspace_size(4, 40, 100, 5, ctypes.byref(n)) == av.EUNSUPPORTED
    assert lib.verify_accept_workspace_size(-1, 40, 100, av.F32, ctypes.byref(n)) == av.EINVAL
    dummy = ctypes.c_void_p(0x1000)
    args = [dummy] * 7
    # row stride shorter than the vocabulary
    assert lib.verify_accept(4, 40, 100, 50, av.F32, *args, dummy, 1 << 20, None) == av.EINVAL
    # missing outputs
    assert lib.verify_accept(4, 40, 100, 0, av.F32, dummy, dummy, dummy, dummy, None, dummy, dummy,
                             dummy, 1 << 20, None) == av.EINVAL
    # small workspace
    lib.verify_accept_workspace_size(4, 40, 100, av.F32, ctypes.byref(n))
    assert lib.verify_accept(4, 40, 100, 0, av.F32, *args, dummy, n.value - 1, None) == av.EWORKSPACE
    # empty batch is a no-op
    assert lib.verify_accept(0, 0, 100, 0, av.F32, *([None] * 8), 0, None) == 0


def test_accept_noalloc_limits_checked_before_any_device_call():
    """verify_accept_noalloc rejects, on the host, a call whose scratch need
    exceeds the fixed per-GPU array, and bad arguments, before touching HIP."""
    lib = av.library()
    n = ctypes.c_size_t(0)
    dummy = ctypes.c_void_p(0x1000)
    # the largest bf16 row count the scratch holds, and one beyond it
    fits, over = 0, 0
    for rows in (100_000, 300_000, 400_000, 600_000):
        assert lib.verify_accept_workspace_size(4, rows, 151936, av.BF16, ctypes.byref(n)) == 0
        if n.value <= av.NOALLOC_SCRATCH_BYTES:
            fits = rows
        elif not over:
            over = rows
    assert fits >= 300_000 and over
    assert lib.verify_accept_noalloc(4, over, 151936, 0, av.BF16, *([dummy] * 7), None) == \
        av.EWORKSPACE
    assert lib.verify_accept_noalloc(4, 40, 151936, 0, 7, *([dummy] * 7), None) == av.EUNSUPPORTED
    assert lib.verify_accept_noalloc(4, 40, 0, 0, av.BF16, *([dummy] * 7), None) == av.EINVAL
    assert lib.verify_accept_noalloc(-1, 40, 100, 0, av.F32, *([dummy] * 7), None) == av.EINVAL


def test_accept_sampled_argument_validation():
    lib = av.library()
    n = ctypes.c_size_t(0)
    lib.verify_accept_workspace_size(4, 40, 100, av.F32, ctypes.byref(n))
    d = ctypes.c_void_p(0x1000)

    def call(temperature=1.0, stride=0, dtype=av.F32, ws=n.value, accept=d, logits=d):
        return lib.verify_accept_sampled(4, 40, 100, stride, dtype, logits, d, d, temperature,
                                         (1 << 64) - 1, (1 << 32) - 1, None, accept, d, d, d, ws,
                                         None)

    for t in (0.0, -1.0, float("nan"), float("inf"), 1e-45):   # 1e-45: 1/T overflows fp32
        assert call(temperature=t) == av.EINVAL, t
    assert call(stride=50) == av.EINVAL
    assert call(accept=None) == av.EINVAL
    assert call(logits=None) == av.EINVAL
    assert call(dtype=9) == av.EUNSUPPORTED
    assert call(ws=n.value - 1) == av.EWORKSPACE
    assert lib.verify_accept_sampled(0, 0, 100, 0, av.F32, *([None] * 3), 0.7, 1, 0,
                                     *([None] * 5), 0, None) == 0
    with pytest.raises(ValueError):
        av.verify_accept_sampled(None, None, None, temperature=1.0, seed=-1)


def test_lmhead_accept_argument_validation():
    lib = av.library()
    n = ctypes.c_size_t(0)
    assert lib.verify_lmhead_accept_workspace_size(4, 40, 4096, 151936, av.BF16, ctypes.byref(n)) == 0
    assert n.value >= 40 * 8
    for args, want in (((4, 40, 4096, 151936, av.F32), av.EUNSUPPORTED),
                       ((4, 40, 4096, 151936, 7), av.EINVAL),
                       ((4, 40, 4100, 151936, av.BF16), av.EINVAL),    # hidden not a multiple of 32
                       ((4, 40, 0, 151936, av.BF16), av.EINVAL),
                       ((4, 40, 4096, 0, av.BF16), av.EINVAL),
                       ((4, 40, 4096, 1 << 31, av.BF16), av.EINVAL),
                       ((-1, 40, 4096, 100, av.BF16), av.EINVAL)):
        assert lib.verify_lmhead_accept_workspace_size(*args, ctypes.byref(n)) == want, args
    lib.verify_lmhead_accept_workspace_size(4, 40, 256, 1000, av.BF16, ctypes.byref(n))
    d = ctypes.c_void_p(0x1000)

    def call(dtype=av.BF16, hid=d, w=d, acc=d, ws=n.value, H=256):
        return lib.verify_lmhead_accept(4, 40, H, 1000, dtype, hid, w, d, d, None, acc, d, d, d, ws,
                                        None)

    assert call(dtype=av.F32) == av.EUNSUPPORTED
    assert call(hid=None) == av.EINVAL
    assert call(w=None) == av.EINVAL
    assert call(acc=None) == av.EINVAL
    assert call(hid=ctypes.c_void_p(0x1008)) == av.EINVAL   # rows are copied in 16-byte pieces
    assert call(H=250) == av.EINVAL
    assert call(ws=n.value - 1) == av.EWORKSPACE
    assert lib.verify_lmhead_accept(0, 0, 256, 1000, av.BF16, *([None] * 8), None, 0, None) == 0


def test_budget_argument_validation():
    lib = av.library()
    d = ctypes.c_void_p(0x1000)
    ok = dict(num_seqs=4, num_cands=10, max_len=8, cs=d, cl=d, ct=d, lt=d, cx=None, alpha=10.0,
              g_min=0.5, score=d, agree=d, prefix=d, source=d, dl=d, qs=d, tok=d, cap=4 * 9, sl=None)

    def call(**kw):
        a = dict(ok)
        a.update(kw)
        return lib.verify_budget(a["num_seqs"], a["num_cands"], a["max_len"], a["cs"], a["cl"], a["ct"],
                                 a["lt"], a["cx"], a["alpha"], a["g_min"], a["score"], a["agree"],
                                 a["prefix"], a["source"], a["dl"], a["qs"], a["tok"], a["cap"], a["sl"],
                                 None)

    assert call(num_seqs=-1) == av.EINVAL
    assert call(num_cands=-1) == av.EINVAL
    assert call(max_len=0) == av.EINVAL
    assert call(alpha=-1.0) == av.EINVAL
    assert call(alpha=float("nan")) == av.EINVAL
    assert call(g_min=1.5) == av.EINVAL
    assert call(g_min=-0.1) == av.EINVAL
    assert call(cap=4 * 9 - 1) == av.EINVAL           # tokens capacity below B * (max_len + 1)
    assert call(qs=None) == av.EINVAL
    assert call(source=None) == av.EINVAL
    assert call(ct=None) == av.EINVAL
    assert call(cx=d) == av.EINVAL                    # ctx_len without seq_lens
    assert call(sl=d) == av.EINVAL                    # seq_lens without ctx_len
    assert call(num_seqs=1 << 20, max_len=4096, cap=1 << 40) == av.EUNSUPPORTED


def test_attention_append_argument_validation():
    """verify_attention_append: verify_attention's checks, and the new tokens'
    arrays are required once there are rows."""
    lib = av.library()
    d = ctypes.c_void_p(0x1000)
    sz = ctypes.c_size_t(1 << 30)
    args = lambda kn, vn: (ctypes.byref(_params()), 36, 9, 1000, d, kn, vn, d, d, d, d, d, None, d, d,
                           sz, None)
    assert lib.verify_attention_append(*args(None, d)) == av.EINVAL
    assert lib.verify_attention_append(*args(d, None)) == av.EINVAL
    bad = (ctypes.byref(_params(head_dim=96)), 36, 9, 1000, d, d, d, d, d, d, d, d, None, d, d, sz, None)
    assert lib.verify_attention_append(*bad) == av.EUNSUPPORTED
    small = (ctypes.byref(_params()), 36, 9, 1000, d, d, d, d, d, d, d, d, None, d, d,
             ctypes.c_size_t(0), None)
    assert lib.verify_attention_append(*small) == av.EWORKSPACE
    # no rows: nothing to enqueue, and no q / K / V arrays needed
    none = (ctypes.byref(_params(num_seqs=0)), 0, 0, 0) + (None,) * 10 + (d, sz, None)
    assert lib.verify_attention_append(*none) == 0


def test_kv_append_argument_validation():
    lib = av.library()
    d = ctypes.c_void_p(0x1000)
    for kw, want in ((dict(head_dim=96), av.EUNSUPPORTED), (dict(num_kv_heads=0), av.EINVAL),
                     (dict(dtype=7), av.EUNSUPPORTED)):
        assert lib.verify_kv_append(ctypes.byref(_params(**kw)), 36, d, d, d, d, d, d, d, None) == want
    for i in range(7):
        ptrs = [d] * 7
        ptrs[i] = None
        assert lib.verify_kv_append(ctypes.byref(_params()), 36, *ptrs, None) == av.EINVAL
    assert lib.verify_kv_append(ctypes.byref(_params()), -1, d, d, d, d, d, d, d, None) == av.EINVAL
    # nothing to append: a no-op that needs no pointers
    assert lib.verify_kv_append(ctypes.byref(_params()), 0, *([None] * 7), None) == 0


def test_check_batch_argument_validation():
    """verify_check_batch refuses bad arguments before any device call."""
    lib = av.library()
    d = ctypes.c_void_p(0x1000)
    P = ctypes.byref
    ok = lambda **kw: _params(num_seqs=4, **kw)
    # negative sizes, no counts, no q_start
    assert lib.verify_check_batch(-1, 10, 0, d, None, 0, None, None, d, None) == av.EINVAL
    assert lib.verify_check_batch(4, -1, 0, d, None, 0, None, None, d, None) == av.EINVAL
    assert lib.verify_check_batch(4, 10, -1, d, None, 0, None, None, d, None) == av.EINVAL
    assert lib.verify_check_batch(4, 10, 0, d, None, 0, None, None, None, None) == av.EINVAL
    assert lib.verify_check_batch(4, 10, 0, None, None, 0, None, None, d, None) == av.EINVAL
    # seq_lens or block tables need the layer's shape
    assert lib.verify_check_batch(4, 10, 0, d, None, 0, d, None, d, None) == av.EINVAL
    assert lib.verify_check_batch(4, 10, 0, d, None, 0, None, d, d, None) == av.EINVAL
    # params that disagree with the call, or without seq_lens
    assert lib.verify_check_batch(4, 10, 0, d, P(_params(num_seqs=5)), 100, d, d, d, None) == av.EINVAL
    assert lib.verify_check_batch(4, 10, 0, d, P(ok(block_size=32)), 100, d, d, d, None) == av.EINVAL
    assert lib.verify_check_batch(4, 10, 0, d, P(ok(max_blocks_per_seq=0)), 100, d, d, d, None) == av.EINVAL
    assert lib.verify_check_batch(4, 10, 0, d, P(ok(sliding_window=-1)), 100, d, d, d, None) == av.EINVAL
    assert lib.verify_check_batch(4, 10, 0, d, P(ok()), -1, d, d, d, None) == av.EINVAL
    assert lib.verify_check_batch(4, 10, 0, d, P(ok()), 100, None, d, d, None) == av.EINVAL
    # the binding: block tables without seq_lens
    qs = torch.zeros(5, dtype=torch.int32)
    with pytest.raises(ValueError, match="seq_lens"):
        av.check_batch(qs, 0, block_tables=torch.zeros((4, 2), dtype=torch.int32))


def test_binding_checks_tensor_shapes_dtypes_and_devices():
    """The binding refuses tensors whose sizes disagree with what the call
    derives from the others (the kernels would index past them).  Meta
    tensors carry shapes without storage, so every check runs without a GPU;
    tensors that pass them stop at the device-memory check."""
    import torch
    m = dict(device="meta")
    bf, i32 = torch.bfloat16, torch.int32
    base = dict(q=torch.empty(36, 32, 128, dtype=bf, **m),
                k_cache=torch.empty(100, 8, 16, 16, 8, dtype=bf, **m),
                v_cache=torch.empty(100, 8, 128, 16, dtype=bf, **m),
                block_tables=torch.empty(4, 30, dtype=i32, **m),
                seq_lens=torch.empty(4, dtype=i32, **m), q_start=torch.empty(5, dtype=i32, **m))

    def attn(**kw):
        args = dict(base)
        args.update(kw)
        av.verify_attention(**args, max_q_len=9, max_seq_len=480)

    with pytest.raises(ValueError, match="q must be a device tensor"):
        attn()
    with pytest.raises(ValueError, match="v_cache must have shape"):
        attn(v_cache=torch.empty(100, 8, 128, 8, dtype=bf, **m))
    with pytest.raises(ValueError, match="k_cache must have shape"):
        attn(k_cache=torch.empty(100, 8, 8, 16, 16, dtype=bf, **m))
    with pytest.raises(ValueError, match="q_start must have shape"):
        attn(q_start=torch.empty(4, dtype=i32, **m))
    with pytest.raises(TypeError, match="seq_lens must be"):
        attn(seq_lens=torch.empty(4, dtype=torch.int64, **m))
    with pytest.raises(ValueError, match="out must have shape"):
        attn(out=torch.empty(35, 32, 128, dtype=bf, **m))
    with pytest.raises(ValueError, match="sinks must have shape"):
        attn(sinks=torch.empty(8, dtype=torch.float32, **m))
    with pytest.raises(ValueError, match="block_tables is on cpu"):
        attn(block_tables=torch.empty(4, 30, dtype=i32))

    logits = torch.empty(36, 1000, dtype=bf, **m)
    qs = torch.empty(5, dtype=i32, **m)
    with pytest.raises(ValueError, match="tokens must have shape"):
        av.verify_accept(logits, torch.empty(35, dtype=i32, **m), qs)
    with pytest.raises(ValueError, match="emitted must have shape"):
        av.verify_accept(logits, torch.empty(36, dtype=i32, **m), qs,
                         emitted=torch.empty(30, dtype=i32, **m))
    with pytest.raises(ValueError, match="accept_len must have shape"):
        av.verify_accept_sampled(logits, torch.empty(36, dtype=i32, **m), qs, temperature=0.7, seed=1,
                                 accept_len=torch.empty(5, dtype=i32, **m))
    with pytest.raises(ValueError, match="tokens must have shape"):
        av.verify_lmhead_accept(torch.empty(36, 64, dtype=bf, **m), torch.empty(1000, 64, dtype=bf, **m),
                                torch.empty(30, dtype=i32, **m), qs)
    with pytest.raises(ValueError, match="last_token must have shape"):
        av.verify_budget(torch.empty(5, dtype=i32, **m), torch.empty(9, dtype=i32, **m),
                         torch.empty(9, 16, dtype=i32, **m), torch.empty(3, dtype=i32, **m),
                         alpha=64.0, g_min=0.3)
    with pytest.raises(ValueError, match="v_new must have shape"):
        av.verify_kv_append(torch.empty(36, 8, 128, dtype=bf, **m), torch.empty(36, 8, 64, dtype=bf, **m),
                            base["k_cache"], base["v_cache"], base["block_tables"], base["seq_lens"],
                            base["q_start"])


def _plan(p, total_q, max_q, max_s):
    info = (ctypes.c_int32 * av.PLAN_INFO)()
    assert av.library().verify_attention_plan(ctypes.byref(p), total_q, max_q, max_s, info) == 0
    return [int(x) for x in info]


def test_attention_plan_row_classes():
    """The host side of the bf16 schedule (no GPU needed: without one the
    library assumes 256 compute units and two resident workgroups each)."""
    # Qwen-shaped: 36 rows per KV head, long contexts -> one launch, the
    # one-wavefront three-tile shape (48 rows per group), one row group
    q = _plan(_params(num_seqs=32, max_blocks_per_seq=1026), 288, 9, 16393)
    assert q[0] == 1 and q[5] == 1 and q[2] == 48 and q[3] == 1 and q[10] == 2 ** 31 - 1
    # ragged drafts up to 32 (132 rows): two launches, requests of up to 48
    # rows on the three-tile shape, the rest on the four-wavefront shape
    # (128 rows per group, two row groups)
    r = _plan(_params(num_seqs=32, max_blocks_per_seq=1026), 500, 33, 16393)
    assert r[5] == 2 and r[10] == 48
    assert r[2] == 48 and r[3] == 1 and r[7] == 128 and r[8] == 2
    # short contexts (fewer than 64 blocks): the first class takes the
    # two-wavefront two-tile shape instead
    s = _plan(_params(num_seqs=32, max_blocks_per_seq=64), 500, 33, 900)
    assert s[5] == 2 and s[2] == 64 and s[7] == 128
    # the long-context batch (8195 blocks at most): its classes own up to
    # 128 * 8 * 8195 and twice that many units, 4 and 8 times 4096 per
    # resident workgroup (512), so they launch 4 and 8 times as many
    lc = _plan(_params(num_seqs=128, max_blocks_per_seq=8196), 2200, 33, 131105)
    assert lc[5] == 2 and lc[1] == 4 * 512 and lc[6] == 8 * 512
    # the Qwen-shaped batch stays at the resident count
    assert q[1] == 512
    # at most 12 rows per KV head with G = 4 stays one launch; 20 rows at
    # G = 4 (five tiles) splits
    assert _plan(_params(num_seqs=8, max_blocks_per_seq=1026), 100, 12, 16393)[5] == 1
    assert _plan(_params(num_seqs=8, max_blocks_per_seq=1026), 100, 20, 16393)[5] == 2
    # head dim 64 keeps one launch at any draft length
    d64 = _plan(_params(num_seqs=8, num_q_heads=64, head_dim=64, max_blocks_per_seq=1026), 300, 33, 16393)
    assert d64[5] == 1
    # the binding reports the classes with their row bounds
    qt = torch.zeros(500, 32, 128, dtype=torch.bfloat16)
    kc = torch.zeros(40, 8, 16, 16, 8, dtype=torch.bfloat16)
    bt = torch.zeros(32, 1026, dtype=torch.int32)
    plan = av.attention_plan(qt, kc, bt, max_q_len=33, max_seq_len=16393)
    assert [c["rows_lo"] for c in plan["classes"]] == [0, 49]
    assert plan["classes"][0]["rows_hi"] == 48 and plan["rows_per_group"] == 48
