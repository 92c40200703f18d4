"""Buffer guards for every entry point of the library.

Each output and each workspace sits between two canary regions of known
bytes.  Every call runs twice on the same inputs, after its outputs and its
workspace were filled with different garbage.  Then:

* the canaries are intact: nothing is written outside the buffers passed;
* the inputs are bit-identical to what they were: only outputs are written;
* the two calls' outputs are bit-identical: every output element the
  interface defines is written, no result depends on what the workspace held
  before, and the kernels are deterministic.

The attention and acceptance cases cover both row classes, forced splits,
the separate schedule launch (300 requests), sliding windows with sinks, rows
a launch does not reach (written as NaN), the fp32 path, and bf16 and fp32
logits."""
from __future__ import annotations

import sys

import numpy as np
import pytest
import torch

import paper_2608_24004_amd as av
from helpers import random_paged

pytestmark = pytest.mark.gpu
DEV = "cuda:0"
PAD = 4096          # canary bytes before and after every guarded buffer
CANARY = 0xC3


def say(*a):
    print(*a, file=sys.stderr, flush=True)


def _bytes(t):
    return t.reshape(-1).view(torch.uint8)


class Arena:
    """Guarded device buffers: each is a view into a larger byte buffer whose
    first and last PAD bytes hold CANARY."""

    def __init__(self):
        self.bufs = []

    def take(self, name, shape, dtype):
        n = int(np.prod(shape)) * torch.empty((), dtype=dtype).element_size()
        raw = torch.full((PAD + n + PAD,), CANARY, dtype=torch.uint8, device=DEV)
        view = raw[PAD:PAD + n].view(dtype).view(shape)
        self.bufs.append((name, raw, n))
        return view

    def fill(self, byte):
        for _, raw, n in self.bufs:
            raw[PAD:PAD + n].fill_(byte)

    def check(self, what):
        torch.cuda.synchronize()
        for name, raw, n in self.bufs:
            for side, part in (("before", raw[:PAD]), ("after", raw[PAD + n:])):
                bad = int((part != CANARY).sum())
                assert bad == 0, "%s: %d canary bytes %s %s changed" % (what, bad, side, name)


def _snapshot(inputs):
    return [t.clone() for t in inputs]


def _assert_unchanged(inputs, before, what):
    for k, (t, t0) in enumerate(zip(inputs, before)):
        assert torch.equal(_bytes(t), _bytes(t0)), "%s: input %d changed" % (what, k)


def _twice(call, arena, inputs, outputs, what, fills=((0xA5, 0x5A), (0x5A, 0xFF))):
    """Run `call` twice, outputs and workspace pre-filled with different bytes
    each time; check canaries, inputs and bitwise agreement.  `outputs` maps a
    name to (tensor, number of leading elements the interface defines)."""
    before = _snapshot(inputs)
    results = []
    for out_byte, ws_byte in fills:
        arena.fill(out_byte)
        for name, raw, n in arena.bufs:
            if name == "workspace":
                raw[PAD:PAD + n].fill_(ws_byte)
        call()
        arena.check(what)
        results.append({k: _bytes(t.reshape(-1)[:m]).clone() for k, (t, m) in outputs.items()})
    _assert_unchanged(inputs, before, what)
    for k in outputs:
        assert torch.equal(results[0][k], results[1][k]), \
            "%s: output %s differs between calls (unwritten elements or workspace dependence)" % (what, k)
    say("  ", what, "ok:", ", ".join("%s %d" % (k, m) for k, (t, m) in outputs.items()))


def _attention_case(p, *, max_q_len=None, split=0, sinks=False):
    q = p.q.to(DEV)
    kc, vc = p.k_cache.to(DEV), p.v_cache.to(DEV)
    bt = torch.as_tensor(p.block_tables, device=DEV)
    sl = torch.as_tensor(p.seq_lens, device=DEV)
    qs = torch.as_tensor(p.q_start, device=DEV)
    sk = None
    if sinks:
        g = torch.Generator().manual_seed(7)
        sk = torch.randn(p.Hq, generator=g, dtype=torch.float32).to(DEV)
    mq = int(np.diff(p.q_start).max()) if max_q_len is None else max_q_len
    ms = int(p.seq_lens.max())
    arena = Arena()
    out = arena.take("out", tuple(q.shape), q.dtype)
    nbytes = av.attention_workspace_size(q, kc, bt, max_q_len=mq, max_seq_len=ms,
                                         sliding_window=p.window, kv_split_blocks=split)
    ws = arena.take("workspace", (max(nbytes, 1),), torch.uint8)
    call = lambda: av.verify_attention(q, kc, vc, bt, sl, qs, max_q_len=mq, max_seq_len=ms,
                                       sliding_window=p.window, kv_split_blocks=split, sinks=sk,
                                       out=out, workspace=ws)
    inputs = [q, kc, vc, bt, sl, qs] + ([sk] if sk is not None else [])
    plan = av.attention_plan(q, kc, bt, max_q_len=mq, max_seq_len=ms, sliding_window=p.window,
                             kv_split_blocks=split)
    return call, arena, inputs, {"out": (out, out.numel())}, plan


ATTENTION_CASES = [
    # (label, shape (Hq, Hkv, D), dtype, contexts, drafts, window, split, sinks, max_q_len)
    ("row classes", (32, 8, 128), "bf16", [700, 40, 1500, 3000, 9, 260, 2048, 5000],
     [11, 12, 0, 32, 20, 3, 11, 40], 0, 0, False, None),
    ("row classes split 3", (32, 8, 128), "bf16", [700, 40, 1500, 3000, 9, 260, 2048, 5000],
     [11, 12, 0, 32, 20, 3, 11, 40], 0, 3, False, None),
    ("window and sinks", (64, 8, 64), "bf16", [4000, 130, 17, 900], [5, 0, 16, 9], 128, 0, True, None),
    ("unreached rows", (32, 8, 128), "bf16", [300, 600, 50], [40, 2, 7], 0, 1, False, 4),
    ("fp32", (32, 8, 128), "f32", [700, 40, 1500], [11, 0, 32], 0, 2, False, None),
]


@pytest.mark.parametrize("case", ATTENTION_CASES, ids=[c[0] for c in ATTENTION_CASES])
def test_attention_guards(case):
    label, (hq, hkv, d), dtype, contexts, drafts, window, split, sinks, mq = case
    say("guards attention", label)
    p = random_paged(num_q_heads=hq, num_kv_heads=hkv, head_dim=d, dtype=dtype, contexts=contexts,
                     drafts=drafts, window=window, seed=11)
    call, arena, inputs, outputs, plan = _attention_case(p, max_q_len=mq, split=split, sinks=sinks)
    if label.startswith("row classes"):
        assert len(plan["classes"]) == 2
    _twice(call, arena, inputs, outputs, "attention " + label)
    if mq is not None:
        # the unreached rows are NaN on both calls (checked equal above); some exist
        assert bool(torch.isnan(outputs["out"][0].float()).any())


def test_attention_guards_scheduled_batch():
    """300 requests: above the inline schedule, so a separate schedule launch
    writes the unit table into the workspace first."""
    rng = np.random.default_rng(5)
    contexts = list(rng.integers(0, 400, size=300))
    drafts = list(rng.integers(0, 9, size=300))
    say("guards attention 300 requests")
    p = random_paged(num_q_heads=32, num_kv_heads=8, head_dim=128, dtype="bf16", contexts=contexts,
                     drafts=drafts, seed=12)
    call, arena, inputs, outputs, plan = _attention_case(p)
    _twice(call, arena, inputs, outputs, "attention 300 requests")


def test_kv_append_guards():
    """The caches are the outputs: both calls start from the same cache, and
    nothing outside them (or in the other inputs) changes."""
    p = random_paged(num_q_heads=32, num_kv_heads=8, head_dim=128, dtype="bf16",
                     contexts=[100, 0, 33, 700], drafts=[4, 0, 31, 9], seed=13)
    say("guards kv_append")
    g = torch.Generator().manual_seed(3)
    T = p.total_q
    k_new = torch.randn((T, p.Hkv, p.D), generator=g).to(torch.bfloat16).to(DEV)
    v_new = torch.randn((T, p.Hkv, p.D), generator=g).to(torch.bfloat16).to(DEV)
    bt = torch.as_tensor(p.block_tables, device=DEV)
    sl = torch.as_tensor(p.seq_lens, device=DEV)
    qs = torch.as_tensor(p.q_start, device=DEV)
    arena = Arena()
    kc = arena.take("k_cache", tuple(p.k_cache.shape), torch.bfloat16)
    vc = arena.take("v_cache", tuple(p.v_cache.shape), torch.bfloat16)
    kc0, vc0 = p.k_cache.to(DEV), p.v_cache.to(DEV)
    inputs = [k_new, v_new, bt, sl, qs, kc0, vc0]
    before = _snapshot(inputs)
    results = []
    for _ in range(2):
        kc.copy_(kc0)
        vc.copy_(vc0)
        av.verify_kv_append(k_new, v_new, kc, vc, bt, sl, qs)
        arena.check("kv_append")
        results.append((_bytes(kc).clone(), _bytes(vc).clone()))
    _assert_unchanged(inputs, before, "kv_append")
    assert torch.equal(results[0][0], results[1][0]) and torch.equal(results[0][1], results[1][1])
    assert not torch.equal(results[0][0], _bytes(kc0))   # the append wrote something


def _accept_inputs(T_per_req, V, dtype, seed):
    g = torch.Generator().manual_seed(seed)
    n = np.asarray(T_per_req, dtype=np.int64)
    q_start = np.zeros(n.size + 1, dtype=np.int32)
    q_start[1:] = np.cumsum(n)
    T = int(q_start[-1])
    logits = torch.randn((T, V), generator=g).to(dtype).to(DEV)
    am = logits.float().argmax(dim=1).int().cpu().numpy()
    tokens = torch.randint(0, V, (T,), generator=g, dtype=torch.int32).numpy()
    for i in range(n.size):            # accept a few drafts of each request
        for j in range(min(int(n[i]) - 1, 2 + i % 3)):
            tokens[q_start[i] + j + 1] = am[q_start[i] + j]
    return logits, torch.as_tensor(tokens, device=DEV), torch.as_tensor(q_start, device=DEV)


def _accept_outputs(arena, B, T):
    return dict(argmax=arena.take("argmax_out", (T,), torch.int32),
                accept_len=arena.take("accept_len", (B,), torch.int32),
                num_emitted=arena.take("num_emitted", (B,), torch.int32),
                emitted=arena.take("emitted", (T,), torch.int32))


@pytest.mark.parametrize("dtype", [torch.bfloat16, torch.float32], ids=["bf16", "f32"])
@pytest.mark.parametrize("mode", ["greedy", "noalloc", "sampled"])
def test_accept_guards(mode, dtype):
    rows = [1, 9, 33, 0, 5, 17, 2]
    V = 50021
    say("guards accept", mode, dtype)
    logits, tokens, qs = _accept_inputs(rows, V, dtype, seed=21)
    B, T = len(rows), int(sum(rows))
    arena = Arena()
    o = _accept_outputs(arena, B, T)
    code = av.BF16 if dtype == torch.bfloat16 else av.F32
    ws = None
    if mode != "noalloc":
        ws = arena.take("workspace", (max(av.accept_workspace_size(B, T, V, code), 1),), torch.uint8)
    kw = dict(argmax_out=o["argmax"], accept_len=o["accept_len"], num_emitted=o["num_emitted"],
              emitted=o["emitted"])
    if mode == "greedy":
        call = lambda: av.verify_accept(logits, tokens, qs, workspace=ws, **kw)
    elif mode == "noalloc":
        call = lambda: av.verify_accept_noalloc(logits, tokens, qs, **kw)
    else:
        kw["sampled_out"] = kw.pop("argmax_out")
        call = lambda: av.verify_accept_sampled(logits, tokens, qs, temperature=0.7, seed=99,
                                                offset=3, workspace=ws, **kw)
    outputs = {k: (t, t.numel()) for k, t in o.items()}
    _twice(call, arena, [logits, tokens, qs], outputs, "accept %s %s" % (mode, dtype))


def test_lmhead_guards():
    rows = [9, 1, 33, 0, 17]
    V, H = 20011, 512
    say("guards lmhead")
    g = torch.Generator().manual_seed(31)
    T, B = int(sum(rows)), len(rows)
    hidden = torch.randn((T, H), generator=g).to(torch.bfloat16).to(DEV)
    weight = (torch.randn((V, H), generator=g) * 0.05).to(torch.bfloat16).to(DEV)
    qs = torch.as_tensor(np.concatenate([[0], np.cumsum(rows)]).astype(np.int32), device=DEV)
    tokens = torch.randint(0, V, (T,), generator=g, dtype=torch.int32).to(DEV)
    arena = Arena()
    o = _accept_outputs(arena, B, T)
    ws = arena.take("workspace", (max(av.lmhead_accept_workspace_size(B, T, H, V), 1),), torch.uint8)
    call = lambda: av.verify_lmhead_accept(hidden, weight, tokens, qs, argmax_out=o["argmax"],
                                           accept_len=o["accept_len"], num_emitted=o["num_emitted"],
                                           emitted=o["emitted"], workspace=ws)
    outputs = {k: (t, t.numel()) for k, t in o.items()}
    _twice(call, arena, [hidden, weight, tokens, qs], outputs, "lmhead")


def test_budget_guards():
    rng = np.random.default_rng(41)
    B, max_len = 37, 12
    cand_per_req = rng.integers(0, 6, size=B)
    start = np.concatenate([[0], np.cumsum(cand_per_req)]).astype(np.int32)
    C = int(start[-1])
    lens = rng.integers(0, max_len + 1, size=C).astype(np.int32)
    toks = rng.integers(0, 5, size=(C, max_len)).astype(np.int32)
    last = rng.integers(0, 5, size=B).astype(np.int32)
    ctx = rng.integers(1, 5000, size=B).astype(np.int32)
    say("guards budget")
    d = lambda a: torch.as_tensor(a, device=DEV)
    inputs = [d(start), d(lens), d(toks), d(last), d(ctx)]
    arena = Arena()
    i32 = torch.int32
    out = dict(score=arena.take("score", (B,), torch.float64), agree=arena.take("agree", (B,), i32),
               prefix_len=arena.take("prefix_len", (B,), i32), source=arena.take("source", (B,), i32),
               draft_len=arena.take("draft_len", (B,), i32), q_start=arena.take("q_start", (B + 1,), i32),
               tokens=arena.take("tokens", (B * (max_len + 1),), i32),
               seq_lens=arena.take("seq_lens", (B,), i32))
    call = lambda: av.verify_budget(*inputs[:4], ctx_len=inputs[4], alpha=96.0, g_min=0.1, out=out)
    call()
    torch.cuda.synchronize()
    used = int(out["q_start"][-1])           # tokens beyond q_start[B] are not defined
    outputs = {k: (t, t.numel()) for k, t in out.items() if k != "tokens"}
    outputs["tokens"] = (out["tokens"], used)
    _twice(call, arena, inputs, outputs, "budget")


@pytest.mark.parametrize("dtype", ["bf16", "f32"])
def test_attention_append_guards(dtype):
    """The fused append: caches, output and workspace guarded; both calls
    start from the same cache, with different garbage in the output and the
    workspace, and must agree bit for bit."""
    p = random_paged(num_q_heads=32, num_kv_heads=8, head_dim=128, dtype=dtype,
                     contexts=[700, 40, 1500, 3000, 9, 260], drafts=[11, 12, 0, 32, 20, 3], seed=14)
    say("guards attention append", dtype)
    tdt = p.q.dtype
    g = torch.Generator().manual_seed(4)
    T = p.total_q
    k_new = torch.randn((T, p.Hkv, p.D), generator=g).to(tdt).to(DEV)
    v_new = torch.randn((T, p.Hkv, p.D), generator=g).to(tdt).to(DEV)
    q = p.q.to(DEV)
    bt = torch.as_tensor(p.block_tables, device=DEV)
    sl = torch.as_tensor(p.seq_lens, device=DEV)
    qs = torch.as_tensor(p.q_start, device=DEV)
    mq, ms = int(np.diff(p.q_start).max()), int(p.seq_lens.max())
    arena = Arena()
    kc = arena.take("k_cache", tuple(p.k_cache.shape), tdt)
    vc = arena.take("v_cache", tuple(p.v_cache.shape), tdt)
    out = arena.take("out", tuple(q.shape), tdt)
    nbytes = av.attention_workspace_size(q, kc, bt, max_q_len=mq, max_seq_len=ms)
    ws = arena.take("workspace", (max(nbytes, 1),), torch.uint8)
    kc0, vc0 = p.k_cache.to(DEV), p.v_cache.to(DEV)
    inputs = [q, k_new, v_new, bt, sl, qs, kc0, vc0]
    before = _snapshot(inputs)
    results = []
    for out_byte, ws_byte in ((0xA5, 0x5A), (0x5A, 0xFF)):
        arena.fill(out_byte)
        for name, raw, n in arena.bufs:
            if name == "workspace":
                raw[PAD:PAD + n].fill_(ws_byte)
        kc.copy_(kc0)
        vc.copy_(vc0)
        av.verify_attention_append(q, k_new, v_new, kc, vc, bt, sl, qs, max_q_len=mq, max_seq_len=ms,
                                   out=out, workspace=ws)
        arena.check("attention append " + dtype)
        results.append([_bytes(t).clone() for t in (kc, vc, out)])
    _assert_unchanged(inputs, before, "attention append " + dtype)
    for a_, b_ in zip(*results):
        assert torch.equal(a_, b_)
    assert not torch.equal(results[0][0], _bytes(kc0))   # the append wrote something
