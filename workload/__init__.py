"""Seeded synthetic workloads for the batched speculative-verification step.

This module only draws random inputs and lays them out in memory.  It holds
none of the verification arithmetic (no attention, no argmax, no acceptance),
so that the HIP path and the CPU oracle, which both consume its output, stay
independent of each other.

Every workload is a batch of decode requests.  Request i has a prior context of
L_i tokens and k_i >= 0 draft tokens, so the verify pass scores n_i = k_i + 1
positions and reads S_i = L_i + n_i cached keys (the caller has already
appended the K/V of the n_i new tokens).  Query rows are packed request by
request: rows q_start[i] .. q_start[i+1]-1 belong to request i.

Inputs follow the recipe of the workloads the paper measures (Sec. 5.1: agentic
code generation, deep research, SWE-Bench and GAIA traces, which are not
available here); shapes follow the models the paper serves (Qwen-3-8B,
DeepSeek-R1-Distill-Llama-8B, GPT-OSS-20B):
  * Q, K, V ~ N(0, 1), drawn in fp32 and rounded to the storage dtype; the
    GPT-OSS-shaped workload adds per-head attention sink logits ~ N(0, 1);
  * the paged KV cache holds sum_i ceil(S_i/16) physical 16-token blocks, handed
    to requests through a random permutation (fragmented placement);
  * logits ~ N(0, 1) i.i.d. per row, with the position of the row maximum drawn
    uniformly (order-statistic construction below), so the generator knows the
    row's argmax without computing one;
  * draft j+1 of a request equals the argmax of row j with the configured match
    probability, else a uniform token different from it.

Paged layouts (x = 16 bytes / element size, so 8 for bf16 and 4 for fp32):
  k_cache [num_blocks, Hkv, D/x, 16, x]   (token t, dim d of a block at [d/x, t, d%x])
  v_cache [num_blocks, Hkv, D, 16]        (token t, dim d of a block at [d, t])
"""
from __future__ import annotations

import dataclasses
import math
import zlib
from dataclasses import dataclass, field
from typing import List, Optional, Tuple

import numpy as np

BLOCK = 16


@dataclass(frozen=True)
class Config:
    name: str
    batch: int
    num_q_heads: int
    num_kv_heads: int
    head_dim: int
    dtype: str                      # "bf16" or "f32": Q/K/V/O storage and logits
    vocab: int
    context: Tuple                  # ("fixed", L) | ("uniform", lo, hi) | ("lognormal", median, sigma, cap)
    drafts: Tuple                   # ("fixed", k) | ("choice", (k, ...)) | ("uniform", lo, hi)
    match: Tuple                    # ("divergence",) | ("prob", p) | ("halves", p_first, p_second)
    windows: Tuple[int, ...] = (0,)  # one attention layer per entry; 0 = full causal
    sinks: bool = False             # per-head attention sink logits in every layer
    hidden_size: int = 4096         # model width: rows of the LM-head weight
    description: str = ""

    def replace(self, **kw) -> "Config":
        return dataclasses.replace(self, **kw)


# Workloads, smallest first.  "qwen3_8b" is the throughput workload; the others
# are parity cases.  Readings of under-specified recipe details:
#   "2k", "16k", ... are powers of two and ranges are integer-uniform inclusive;
#   the log-normal context uses sigma = 1 (natural log) and is clipped to [16, cap];
#   "first half of each draft" means draft positions j < ceil(k/2).
CONFIGS = {
    "tiny": Config(
        name="tiny", batch=4, num_q_heads=8, num_kv_heads=2, head_dim=64, dtype="f32",
        vocab=1024, context=("fixed", 256), drafts=("fixed", 4), match=("divergence",),
        hidden_size=256,
        description="single layer, fp32, drafts planted as argmax up to a random divergence point"),
    "qwen3_8b": Config(
        name="qwen3_8b", batch=32, num_q_heads=32, num_kv_heads=8, head_dim=128, dtype="bf16",
        vocab=151936, context=("uniform", 2048, 16384), drafts=("fixed", 8), match=("prob", 0.7),
        description="Qwen-3-8B-shaped verify step, one layer"),
    "dsk_distill_8b": Config(
        name="dsk_distill_8b", batch=64, num_q_heads=32, num_kv_heads=8, head_dim=128,
        dtype="bf16", vocab=128256, context=("lognormal", 8192, 1.0, 32768),
        drafts=("choice", (0, 2, 4, 8, 16)), match=("prob", 0.6),
        description="Llama-3-8B-shaped (DeepSeek-R1-Distill-Llama-8B) verify step, ragged drafts"),
    "gpt_oss_20b": Config(
        name="gpt_oss_20b", batch=64, num_q_heads=64, num_kv_heads=8, head_dim=64, dtype="bf16",
        vocab=201088, context=("uniform", 4096, 65536), drafts=("fixed", 8), match=("prob", 0.5),
        windows=(128, 0), sinks=True, hidden_size=2880,
        description="GPT-OSS-20B-shaped verify step: a 128-token sliding-window layer and a full "
                    "layer, both with per-head attention sinks"),
    "long_context": Config(
        name="long_context", batch=128, num_q_heads=32, num_kv_heads=8, head_dim=128,
        dtype="bf16", vocab=151936, context=("uniform", 32768, 131072), drafts=("uniform", 0, 32),
        match=("halves", 0.8, 0.3),
        description="long-context agent stress: Qwen-3-8B shapes, ragged drafts 0-32"),
}


@dataclass
class Layer:
    window: int
    q: object          # torch tensor [T, Hq, D]
    k_cache: object    # torch tensor [num_blocks, Hkv, D/x, 16, x]
    v_cache: object    # torch tensor [num_blocks, Hkv, D, 16]
    sinks: object = None  # torch float32 [Hq] sink logits, or None


@dataclass
class Batch:
    cfg: Config
    seed: int
    device: str
    context_len: np.ndarray       # [B] L_i
    num_drafts: np.ndarray        # [B] k_i
    seq_lens: np.ndarray          # [B] S_i = L_i + k_i + 1
    q_start: np.ndarray           # [B+1]
    block_tables: np.ndarray      # [B, max_blocks] int32, -1 padded
    num_blocks: int
    designated: np.ndarray        # [T] planted position of each logits row's maximum
    planted_match: np.ndarray     # [T] bool: draft after this row was planted equal to it
    tokens: np.ndarray            # [T] row inputs: last committed token then the drafts
    logits: object                # torch [T, V]
    layers: List[Layer] = field(default_factory=list)
    t_seq_lens: object = None     # torch int32 copies on `device`
    t_q_start: object = None
    t_block_tables: object = None
    t_tokens: object = None

    @property
    def total_q(self) -> int:
        return int(self.q_start[-1])

    @property
    def max_seq_len(self) -> int:
        return int(self.seq_lens.max()) if self.seq_lens.size else 0

    @property
    def max_q_len(self) -> int:
        return int((self.num_drafts + 1).max()) if self.num_drafts.size else 0


def torch_dtype(name: str):
    import torch
    return {"bf16": torch.bfloat16, "f32": torch.float32}[name]


def elems_per_16b(name: str) -> int:
    return {"bf16": 8, "f32": 4}[name]


def _stream_seed(seed: int, tag: str) -> int:
    """Independent 63-bit seed per (seed, tensor tag)."""
    ss = np.random.SeedSequence([seed & 0xFFFFFFFF, zlib.crc32(tag.encode())])
    return int(ss.generate_state(1, dtype=np.uint64)[0]) & ((1 << 63) - 1)


def _torch_gen(device: str, seed: int, tag: str):
    import torch
    g = torch.Generator(device=device)
    g.manual_seed(_stream_seed(seed, tag))
    return g


def draw_context(cfg: Config, rng: np.random.Generator, b: int) -> np.ndarray:
    kind = cfg.context[0]
    if kind == "fixed":
        return np.full(b, cfg.context[1], dtype=np.int64)
    if kind == "uniform":
        return rng.integers(cfg.context[1], cfg.context[2] + 1, size=b, dtype=np.int64)
    if kind == "lognormal":
        med, sigma, cap = cfg.context[1], cfg.context[2], cfg.context[3]
        x = np.exp(rng.normal(math.log(med), sigma, size=b))
        return np.clip(np.rint(x), 16, cap).astype(np.int64)
    raise ValueError(kind)


def draw_drafts(cfg: Config, rng: np.random.Generator, b: int) -> np.ndarray:
    kind = cfg.drafts[0]
    if kind == "fixed":
        return np.full(b, cfg.drafts[1], dtype=np.int64)
    if kind == "choice":
        return rng.choice(np.asarray(cfg.drafts[1], dtype=np.int64), size=b)
    if kind == "uniform":
        return rng.integers(cfg.drafts[1], cfg.drafts[2] + 1, size=b, dtype=np.int64)
    raise ValueError(kind)


def match_probability(cfg: Config, k: int) -> np.ndarray:
    """Per-draft-position probability that draft j+1 is planted equal to row j's argmax."""
    kind = cfg.match[0]
    if kind == "prob":
        return np.full(k, cfg.match[1])
    if kind == "halves":
        j = np.arange(k)
        return np.where(j < (k + 1) // 2, cfg.match[1], cfg.match[2])
    raise ValueError(kind)


def _pred_bits(x, dtype_name: str):
    """Largest value of the storage dtype strictly below x (elementwise, finite x)."""
    import torch
    if dtype_name == "bf16":
        bits = x.view(torch.int16).to(torch.int32)
        sign_mask, max_mag, it = 0x8000, 0x7FFF, torch.int16
    else:
        bits = x.view(torch.int32).to(torch.int64)
        sign_mask, max_mag, it = 0x80000000, 0x7FFFFFFF, torch.int32
    ubits = bits & ((sign_mask << 1) - 1)
    neg = (ubits & sign_mask) != 0
    mag = ubits & max_mag
    zero = mag == 0
    new = torch.where(zero, torch.full_like(ubits, sign_mask | 1),
                      torch.where(neg, ubits + 1, ubits - 1))
    # back to signed storage
    new = torch.where(new >= sign_mask, new - (sign_mask << 1), new)
    return new.to(it).view(x.dtype)


def draw_logits(cfg: Config, seed: int, device: str, rows: int, vocab: int,
                designated: np.ndarray, row_chunk: int = 256):
    """i.i.d. N(0,1) logits rows whose maximum sits at `designated[r]`.

    Order-statistic construction: the row maximum of V i.i.d. normals has CDF
    Phi(x)^V, so it is drawn as Phi^{-1}(u^{1/V}); the other V-1 entries are
    normals conditioned to lie below it (rejection: redraw any that do not).
    After rounding to the storage dtype, entries that rounded up to the maximum
    are moved one ulp below it, so the designated entry is the unique maximum.
    """
    import torch
    from scipy.special import ndtri
    dt = torch_dtype(cfg.dtype)
    rng = np.random.default_rng(_stream_seed(seed, "logits-max"))
    u = rng.random(rows)
    eps = -np.expm1(np.log(u) / vocab)          # 1 - u^{1/V}, computed without cancellation
    xmax = -ndtri(eps)                          # Phi^{-1}(1 - eps)
    out = torch.empty((rows, vocab), dtype=dt, device=device)
    g = _torch_gen(device, seed, "logits")
    xmax_t = torch.as_tensor(xmax, dtype=torch.float32, device=device)
    des_t = torch.as_tensor(designated, dtype=torch.int64, device=device)
    for r0 in range(0, rows, row_chunk):
        r1 = min(rows, r0 + row_chunk)
        x = torch.randn((r1 - r0, vocab), generator=g, device=device, dtype=torch.float32)
        lim = xmax_t[r0:r1, None]
        bad = x >= lim
        while bool(bad.any()):
            x[bad] = torch.randn(int(bad.sum()), generator=g, device=device, dtype=torch.float32)
            bad = x >= lim
        xs = x.to(dt)
        mb = xmax_t[r0:r1].to(dt)
        xs = torch.minimum(xs, _pred_bits(mb, cfg.dtype)[:, None])
        xs.scatter_(1, des_t[r0:r1, None], mb[:, None])
        out[r0:r1] = xs
    return out


def draw_lmhead(cfg: Config, seed: int, device: str, designated: np.ndarray, *,
                alpha: float = 8.0, peaked: float = 0.75, vocab: Optional[int] = None,
                hidden_size: Optional[int] = None):
    """Final hidden states and an LM-head weight (both bf16) for the fused
    LM-head path: (hidden [T, H], weight [V, H]).

    weight ~ N(0, 1/H) elementwise, so every row has norm about 1 and the
    logits <hidden, weight[v]> of an N(0, I) hidden state are about N(0, 1).
    A fraction `peaked` of the rows (chosen at random) adds alpha * weight[d]
    for the row's designated token d: its logit gains about alpha and, at
    alpha = 8, beats the maximum of 10^5 - 10^6 others in nearly every row,
    so drafts planted as d are mostly accepted, as on a confident model.  The
    other rows are flat.  No logit is computed here.
    """
    import torch
    V = cfg.vocab if vocab is None else int(vocab)
    H = cfg.hidden_size if hidden_size is None else int(hidden_size)
    T = int(designated.shape[0])
    g = _torch_gen(device, seed, "lmhead")
    w = torch.empty((V, H), dtype=torch.bfloat16, device=device)
    scale = 1.0 / math.sqrt(H)
    step = max(1, (1 << 26) // H)
    for v0 in range(0, V, step):
        v1 = min(V, v0 + step)
        w[v0:v1] = (torch.randn((v1 - v0, H), generator=g, device=device,
                                dtype=torch.float32) * scale).to(torch.bfloat16)
    hs = torch.randn((T, H), generator=g, device=device, dtype=torch.float32)
    rng = np.random.default_rng(_stream_seed(seed, "lmhead-peaked"))
    pk = rng.random(T) < peaked
    if T and pk.any():
        rows = torch.as_tensor(np.nonzero(pk)[0], dtype=torch.int64, device=device)
        des = torch.as_tensor(designated.astype(np.int64)[pk], device=device)
        hs[rows] += alpha * w[des].to(torch.float32)
    return hs.to(torch.bfloat16), w


def make_batch(cfg: Config, seed: int, device: str = "cpu", *,
               context_len: Optional[np.ndarray] = None,
               num_drafts: Optional[np.ndarray] = None,
               with_layers: bool = True, with_logits: bool = True) -> Batch:
    """Draw one verify step of workload `cfg` (deterministic in (cfg, seed, device))."""
    import torch
    rng = np.random.default_rng(_stream_seed(seed, "meta"))
    b = cfg.batch
    L = np.asarray(context_len, dtype=np.int64) if context_len is not None else draw_context(cfg, rng, b)
    k = np.asarray(num_drafts, dtype=np.int64) if num_drafts is not None else draw_drafts(cfg, rng, b)
    b = L.shape[0]
    n = k + 1
    S = L + n
    q_start = np.zeros(b + 1, dtype=np.int32)
    q_start[1:] = np.cumsum(n)
    T = int(q_start[-1])
    nblk = (S + BLOCK - 1) // BLOCK
    num_blocks = int(nblk.sum())
    perm = rng.permutation(num_blocks).astype(np.int32)
    max_blocks = int(nblk.max()) if b else 1
    bt = np.full((b, max_blocks), -1, dtype=np.int32)
    off = 0
    for i in range(b):
        bt[i, :nblk[i]] = perm[off:off + nblk[i]]
        off += nblk[i]

    V = cfg.vocab
    designated = rng.integers(0, V, size=T, dtype=np.int64)
    tokens = np.zeros(T, dtype=np.int32)
    planted = np.zeros(T, dtype=bool)
    for i in range(b):
        q0 = int(q_start[i])
        ki = int(k[i])
        tokens[q0] = rng.integers(0, V)
        if cfg.match[0] == "divergence":
            J = int(rng.integers(0, ki + 1))
            hit = np.arange(ki) < J
        else:
            hit = rng.random(ki) < match_probability(cfg, ki)
        for j in range(ki):
            row = q0 + j
            if hit[j] or V == 1:
                tokens[row + 1] = designated[row]
                planted[row] = True
            else:
                o = int(rng.integers(0, V - 1))
                tokens[row + 1] = o if o < designated[row] else o + 1

    batch = Batch(cfg=cfg, seed=seed, device=device, context_len=L, num_drafts=k,
                  seq_lens=S.astype(np.int32), q_start=q_start, block_tables=bt,
                  num_blocks=num_blocks, designated=designated.astype(np.int32),
                  planted_match=planted, tokens=tokens, logits=None)
    batch.t_seq_lens = torch.as_tensor(batch.seq_lens, device=device)
    batch.t_q_start = torch.as_tensor(q_start, device=device)
    batch.t_block_tables = torch.as_tensor(bt, device=device)
    batch.t_tokens = torch.as_tensor(tokens, device=device)
    if with_logits:
        batch.logits = draw_logits(cfg, seed, device, T, V, designated)
    if with_layers:
        dt = torch_dtype(cfg.dtype)
        D, Hq, Hkv = cfg.head_dim, cfg.num_q_heads, cfg.num_kv_heads
        x = elems_per_16b(cfg.dtype)
        for li, w in enumerate(cfg.windows):
            g = _torch_gen(device, seed, "layer%d" % li)
            q = torch.randn((T, Hq, D), generator=g, device=device, dtype=torch.float32).to(dt)
            kc = _randn_storage((num_blocks, Hkv, D // x, BLOCK, x), g, device, dt)
            vc = _randn_storage((num_blocks, Hkv, D, BLOCK), g, device, dt)
            # sink logits ~ N(0, 1), drawn after the caches so that adding them
            # leaves every other tensor of the stream unchanged
            sk = (torch.randn(Hq, generator=g, device=device, dtype=torch.float32)
                  if cfg.sinks else None)
            batch.layers.append(Layer(window=w, q=q, k_cache=kc, v_cache=vc, sinks=sk))
    return batch


def _randn_storage(shape, g, device, dt, chunk_elems: int = 1 << 28):
    """N(0,1) drawn in fp32 and rounded to `dt`, chunked to bound fp32 temporaries."""
    import torch
    out = torch.empty(shape, dtype=dt, device=device)
    flat = out.view(-1)
    for s in range(0, flat.numel(), chunk_elems):
        e = min(flat.numel(), s + chunk_elems)
        flat[s:e] = torch.randn(e - s, generator=g, device=device, dtype=torch.float32).to(dt)
    return out


def pack_request_kv(k_logical, v_logical, block_row: np.ndarray, k_cache, v_cache, kv_head: int):
    """Write one request's logical K/V ([S, D] tensors, one KV head) into the paged caches."""
    import torch
    S, D = k_logical.shape
    x = k_cache.shape[-1]
    t = torch.arange(S)
    b = torch.as_tensor(np.asarray(block_row)[(t // BLOCK).numpy()], dtype=torch.int64)
    o = t % BLOCK
    k_cache[b, kv_head, :, o, :] = k_logical.reshape(S, D // x, x).to(k_cache.dtype)
    v_cache[b, kv_head, :, o] = v_logical.to(v_cache.dtype)


def host_storage(t) -> np.ndarray:
    """numpy view of a CPU tensor's storage: float32 as float32, bf16 as uint16 bits."""
    import torch
    t = t.detach().cpu().contiguous()
    if t.dtype == torch.bfloat16:
        return t.view(torch.int16).numpy().view(np.uint16)
    if t.dtype == torch.float32:
        return t.numpy()
    raise TypeError(t.dtype)


def dtype_code(name: str) -> int:
    """Storage dtype code shared by the C ABI and the oracle: 0 = fp32, 1 = bf16."""
    return {"f32": 0, "bf16": 1}[name]


def draw_candidates(seed: int, batch: int, max_cands: int = 16, max_len: int = 32,
                    vocab: int = 151936, agree_vocab: int = 4):
    """Seeded candidate continuations for the budget allocation (Sec. 4.2), in
    the CSR layout verify_budget takes: (cand_start [B+1], cand_len [C],
    cand_tokens [C, max_len]) int32 numpy arrays.

    Request i gets U{0..max_cands} candidates.  Each candidate starts with a
    U{0..max_len/2}-token prefix of a per-request base continuation whose first
    token comes from a small set (so that candidates agree in varying numbers,
    the redundancy the method scores), then continues with uniform tokens up
    to U{0..max_len} tokens in all.
    """
    rng = np.random.default_rng([seed, 0xB0D6E7])
    starts = [0]
    rows = []
    for _ in range(batch):
        n = int(rng.integers(0, max_cands + 1))
        base = rng.integers(0, vocab, size=max_len)
        base[0] = int(rng.integers(0, agree_vocab))
        for _ in range(n):
            k = int(rng.integers(0, max_len // 2 + 1))
            total = int(rng.integers(k, max_len + 1))
            c = np.concatenate([base[:k], rng.integers(0, vocab, size=total - k)])
            if total > 0 and k == 0:
                c[0] = int(rng.integers(0, agree_vocab))
            rows.append(c)
        starts.append(len(rows))
    C = max(1, len(rows))
    lens = np.zeros(C, dtype=np.int32)
    toks = np.zeros((C, max_len), dtype=np.int32)
    for r, c in enumerate(rows):
        lens[r] = len(c)
        toks[r, :len(c)] = c
    return np.array(starts, dtype=np.int32), lens, toks
