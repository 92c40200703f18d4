"""Throughput of the batched speculative-verification step on one MI355X.

    python bench.py [--gpus 1] [--steps K] [--warmup W] [--config qwen3_8b] [--seeds 0,1,2,3,4]

One step = every attention layer of the workload (verify_attention) followed by
verify_accept (vocabulary argmax + greedy acceptance) over one batch of
synthetic inputs already resident in HBM.  Every seed draws its own batch; per
seed, W untimed steps, then K steps back to back with a HIP event between
consecutive steps.  Prints one JSON line:

  value         verified tokens/s: per seed sum_i (accept_len_i + 1) / the
                median step time, then the mean over seeds
  roofline      the attention call: algorithmic bytes per launch / mean launch
                time (K calls back to back on the launch stream between two HIP
                events, after the timed steps; mean over seeds) vs 8 TB/s HBM,
                and the same-run ceilings of a torch gather of the walk's K/V
                tiles and of a plain device copy
  cpu_baseline  the CPU oracle on a bounded sample of the first seed's step
                (first requests of the batch, all their heads and logits rows)
"""
from __future__ import annotations

import argparse
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

HBM_PEAK_GBS = 8000.0   # MI355X HBM3E datasheet peak
MFMA_BF16_PEAK_TFLOPS = 2500.0  # MI355X dense bf16 matrix peak
CALIB_BYTES = 256 << 20  # the plain elementwise kernel of --copy-calibration reads and writes this
# sources whose change invalidates a stored traffic measurement of the attention call
KERNEL_SOURCES = ("paper_2608_24004_amd/csrc/verify_attention.hip",
                  "paper_2608_24004_amd/csrc/common.h", "paper_2608_24004_amd/build.py")
# ... and a stored instruction count of the sampled acceptance kernel
ACCEPT_SOURCES = ("paper_2608_24004_amd/csrc/verify_accept.hip",
                  "paper_2608_24004_amd/csrc/common.h", "paper_2608_24004_amd/build.py")
# vector-ALU issue peak: 256 CUs x 4 SIMDs x 16 lanes x 2.4 GHz lane-instructions/s (a wave64
# instruction holds a 16-lane SIMD for 4 cycles)
VALU_PEAK_LANE_OPS = 256 * 4 * 16 * 2.4e9


def log(*a):
    print(*a, file=sys.stderr, flush=True)


def attention_bytes(bt, layer) -> float:
    """Algorithmic HBM bytes of one attention layer: the visible keys' K and V
    (union over the request's rows), Q read once, O written once, and the
    block-table entries walked."""
    import numpy as np
    cfg = bt.cfg
    e = 2 if cfg.dtype == "bf16" else 4
    n = np.diff(bt.q_start).astype(np.int64)
    S = bt.seq_lens.astype(np.int64)
    vis = S if layer.window == 0 else np.minimum(S, layer.window + n - 1)
    kv = float(vis.sum()) * 2 * cfg.num_kv_heads * cfg.head_dim * e
    qo = 2.0 * bt.total_q * cfg.num_q_heads * cfg.head_dim * e
    first = S - vis
    blocks = ((S + 15) // 16 - first // 16).sum()
    return kv + qo + 4.0 * float(blocks)


def accept_bytes(bt) -> float:
    cfg = bt.cfg
    e = 2 if cfg.dtype == "bf16" else 4
    T, B = bt.total_q, len(bt.seq_lens)
    return float(T) * cfg.vocab * e + 4.0 * (4 * T + 3 * B + 1)


def kernel_source_hash(sources=KERNEL_SOURCES) -> str:
    import hashlib
    h = hashlib.sha256()
    for f in sources:
        with open(os.path.join(ROOT, f), "rb") as fh:
            h.update(fh.read())
    return h.hexdigest()


def traffic_file(workload: str) -> str:
    return os.path.join(ROOT, "profiles", "traffic_verify_attention_%s.txt" % workload)


def stored_traffic(workload: str):
    """HBM bytes per verify_attention call from the committed counter summary,
    or None when there is none or the kernel sources changed since it was taken."""
    try:
        kv = dict(l.split(":", 1) for l in open(traffic_file(workload)) if ":" in l)
    except OSError:
        return None
    if kv.get("source_sha256", "").strip() != kernel_source_hash():
        return None
    return float(kv["traffic_bytes_per_call"])


def stored_sample_instructions(workload: str):
    """VALU instructions of one sample_chunks dispatch from the committed
    counter summary, or None when there is none or the sources changed."""
    path = os.path.join(ROOT, "profiles", "counters_verify_step_%s.md" % workload)
    try:
        kv = dict(l.split(":", 1) for l in open(path) if l.startswith(("accept_source_sha256:",
                                                                     "valu_instructions_sample_chunks:")))
    except OSError:
        return None
    if kv.get("accept_source_sha256", "").strip() != kernel_source_hash(ACCEPT_SOURCES):
        return None
    return float(kv["valu_instructions_sample_chunks"])


def summarize_pmc(fetch_csv: str, write_csv: str, workload: str) -> None:
    """Turn two rocprofv3 --pmc runs of `bench.py --copy-calibration` (FETCH_SIZE,
    then WRITE_SIZE; KiB per dispatch) into HBM bytes per verify_attention call.
    Each counter is scaled by what it reads for the calibration kernel, which
    moves CALIB_BYTES in each direction.  Prints the summary text."""
    import collections
    import csv
    import re

    # the kernels one verify_attention call launches (the append is a separate
    # call).  A call launches each of them once per row class and layer, with a
    # grid of its own, so they are told apart by template arguments and grid;
    # the fused append's kernels (a side call) are not part of it.
    call_kernels = ("attn_schedule", "attn_persist", "attn_combine_slots", "attn_valu", "attn_combine")

    def per_kernel(path, counter):
        by_dispatch = collections.defaultdict(float)
        names, grids = {}, {}
        for r in csv.DictReader(open(path)):
            if r["Counter_Name"] != counter:
                continue
            d = r["Dispatch_Id"]
            by_dispatch[d] += float(r["Counter_Value"])
            names[d] = r["Kernel_Name"]
            grids[d] = r.get("Grid_Size", "")
        groups = collections.defaultdict(list)
        calib = None
        for d in sorted(by_dispatch, key=int):
            n = names[d]
            m = re.search(r"averify::\(anonymous namespace\)::(\w+)(<[^>]*>)?", n)
            if m:
                key = m.group(1)
                if key in call_kernels:
                    key = "%s%s grid %s" % (key, (m.group(2) or "").replace(" ", ""), grids[d])
                groups[key].append(by_dispatch[d])
            elif "bitwise_not" in n:
                calib = by_dispatch[d]
        return {k: sum(v) / len(v) for k, v in groups.items()}, \
               {k: len(v) for k, v in groups.items()}, calib

    fk, fn, fcal = per_kernel(fetch_csv, "FETCH_SIZE")
    wk, wn, wcal = per_kernel(write_csv, "WRITE_SIZE")
    if not fcal or not wcal:
        raise SystemExit("no calibration dispatch (run bench.py with --copy-calibration)")
    ff = CALIB_BYTES / (fcal * 1024.0)
    wf = CALIB_BYTES / (wcal * 1024.0)
    attn = [k for k in fk if k.split("<")[0].split(" ")[0] in call_kernels and ",true>" not in k]
    total = 0.0
    lines = []
    for k in sorted(attn):
        fb = fk[k] * 1024.0 * ff
        wb = wk.get(k, 0.0) * 1024.0 * wf
        total += fb + wb
        lines.append("  %-48s dispatches %3d  FETCH %10.1f KiB  WRITE %9.1f KiB  -> %.4f GB read, "
                     "%.4f GB written" % (k, fn[k], fk[k], wk.get(k, 0.0), fb / 1e9, wb / 1e9))
    for k in sorted(set(fk) - set(attn)):
        lines.append("  %-48s dispatches %3d  FETCH %10.1f KiB  WRITE %9.1f KiB  (not this call)" % (
            k, fn[k], fk[k], wk.get(k, 0.0)))
    print("workload: %s" % workload)
    print("source_sha256: %s" % kernel_source_hash())
    print("traffic_bytes_per_call: %.0f" % total)
    print("calibration_fetch_factor: %.4f" % ff)
    print("calibration_write_factor: %.4f" % wf)
    print("calibration: bitwise_not over %d MiB int32 reads %.1f KiB, writes %.1f KiB" % (
        CALIB_BYTES >> 20, fcal, wcal))
    print("per-kernel mean per dispatch:")
    print("\n".join(lines))


def graph_time_us(fn, steps: int) -> float:
    """Mean device time of fn() (one short call): `steps` calls captured back
    to back in one HIP graph, the replay timed with events (a call shorter
    than its host-side launch would otherwise measure the launch)."""
    import torch
    torch.cuda.synchronize()
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph):
        for _ in range(steps):
            fn()
    graph.replay()
    torch.cuda.synchronize()
    stream = torch.cuda.current_stream()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record(stream)
    graph.replay()
    e1.record(stream)
    torch.cuda.synchronize()
    return e0.elapsed_time(e1) * 1e3 / steps


def kv_append_timing(av, bt, steps: int):
    """Device time of writing the step's new tokens' K/V ([T, Hkv, D] each)
    into the first layer's cache (verify_kv_append), and its bytes: the new
    K/V read once and written once; and the append fused into the attention
    launch (verify_attention_append) against the append then the attention.  The calls rotate over enough copies of
    the new K/V (more than the 256 MB Infinity Cache holds) that every call
    reads its inputs from HBM."""
    import torch
    cfg = bt.cfg
    l = bt.layers[0]
    T = bt.total_q
    g = torch.Generator(device=l.q.device)
    g.manual_seed(5)
    k_new = torch.randn((T, cfg.num_kv_heads, cfg.head_dim), generator=g, device=l.q.device).to(l.q.dtype)
    v_new = torch.randn_like(k_new)
    one = 2 * k_new.numel() * k_new.element_size()
    copies = max(2, -(-(640 << 20) // one))
    ks = [k_new.clone() for _ in range(copies)]
    vs = [v_new.clone() for _ in range(copies)]
    # the cache is modified in place: append into copies of the cache
    kc, vc = l.k_cache.clone(), l.v_cache.clone()
    it = [0]

    def fn():
        c = it[0] % copies
        it[0] += 1
        av.verify_kv_append(ks[c], vs[c], kc, vc, bt.t_block_tables, bt.t_seq_lens, bt.t_q_start)
    fn()
    us = graph_time_us(fn, max(steps, 2 * copies))
    nbytes = 2 * one

    # the append fused into the attention launch (verify_attention_append)
    # against the append followed by the attention, on the same cache copy:
    # `steps` calls of each captured in a HIP graph and replayed (device time,
    # without the host's launch cost), the two alternated over two rounds, the
    # last round reported
    kw = dict(max_q_len=bt.max_q_len, max_seq_len=bt.max_seq_len, sliding_window=l.window,
              sinks=l.sinks)
    out = torch.empty_like(l.q)
    ws = torch.empty(max(1, av.attention_workspace_size(l.q, kc, bt.t_block_tables, max_q_len=bt.max_q_len,
                                                        max_seq_len=bt.max_seq_len,
                                                        sliding_window=l.window)),
                     dtype=torch.uint8, device=l.q.device)

    def two():
        c = it[0] % copies
        it[0] += 1
        av.verify_kv_append(ks[c], vs[c], kc, vc, bt.t_block_tables, bt.t_seq_lens, bt.t_q_start)
        av.verify_attention(l.q, kc, vc, bt.t_block_tables, bt.t_seq_lens, bt.t_q_start, out=out,
                            workspace=ws, **kw)

    def fused():
        c = it[0] % copies
        it[0] += 1
        av.verify_attention_append(l.q, ks[c], vs[c], kc, vc, bt.t_block_tables, bt.t_seq_lens,
                                   bt.t_q_start, out=out, workspace=ws, **kw)

    two()
    fused()
    for _ in range(2):
        t_two, t_fused = graph_time_us(two, steps), graph_time_us(fused, steps)
    del kc, vc, ks, vs, out, ws
    return {"us": us, "bytes": nbytes, "GBps": nbytes / (us * 1e-6) / 1e9, "rows": T,
            "input_copies": copies, "append_then_attention_us": t_two,
            "fused_attention_append_us": t_fused}


def accept_timing(av, bt, steps: int, aws):
    """Device time of the acceptance calls on the step's logits: greedy
    (verify_accept) and stochastic at T = 0.7 (verify_accept_sampled), with
    the logits' bytes per microsecond each reaches.  The calls rotate over
    copies of the logits totalling more than twice the 256 MB Infinity Cache,
    so that every call streams its logits from HBM, as in the step.  The
    sampled call scores every logit with its own Gumbel noise, so it is bound
    by vector ALU work, not by HBM."""
    import torch
    T, V = bt.logits.shape
    dev = bt.logits.device
    B = len(bt.q_start) - 1
    nbytes = T * V * bt.logits.element_size()
    copies = max(2, -(-(640 << 20) // max(1, nbytes)))
    lg = [bt.logits] + [bt.logits.clone() for _ in range(copies - 1)]
    outs = [torch.empty(n, dtype=torch.int32, device=dev) for n in (B, B, T, T)]
    it = [0]

    def nxt():
        c = it[0] % copies
        it[0] += 1
        return lg[c]
    greedy = lambda: av.verify_accept(nxt(), bt.t_tokens, bt.t_q_start, accept_len=outs[0],
                                      num_emitted=outs[1], emitted=outs[2], argmax_out=outs[3],
                                      workspace=aws)
    sampled = lambda: av.verify_accept_sampled(nxt(), bt.t_tokens, bt.t_q_start, temperature=0.7,
                                               seed=1234, offset=1, accept_len=outs[0],
                                               num_emitted=outs[1], emitted=outs[2],
                                               sampled_out=outs[3], workspace=aws)
    res = {"logits_bytes": nbytes, "rows": T, "vocab": V, "logits_copies": copies}
    for name, fn in (("greedy", greedy), ("sampled_T0.7", sampled)):
        fn()
        us = graph_time_us(fn, max(steps, 2 * copies))
        res[name] = {"us": us, "GBps": nbytes / (us * 1e-6) / 1e9,
                     "logits_per_ns": T * V / (us * 1e3)}
    # the sampled call is bound by vector-ALU issue: its counted instructions
    # (64 lanes each) per second against the issue peak
    ninst = stored_sample_instructions(bt.cfg.name)
    if ninst is not None:
        sus = res["sampled_T0.7"]["us"]  # the whole call (sample_chunks + accept_scan)
        achieved = ninst * 64 / (sus * 1e-6)
        res["sampled_T0.7"]["roofline"] = {
            "bound": "alu", "achieved": achieved / 1e12, "peak": VALU_PEAK_LANE_OPS / 1e12,
            "unit": "T VALU lane-instructions/s", "frac": achieved / VALU_PEAK_LANE_OPS,
            "instructions": ninst}
    del lg
    return res


def walk_tiles(bt, layer):
    """(block, KV head) tile ids of every K/V tile one attention call walks,
    request by request, head by head, block by block (visible blocks only)."""
    import numpy as np
    cfg = bt.cfg
    Hkv = cfg.num_kv_heads
    ids = []
    n = np.diff(bt.q_start)
    for i in range(len(bt.seq_lens)):
        S = int(bt.seq_lens[i])
        lo = 0 if layer.window == 0 else max(0, S - int(n[i]) - layer.window + 1)
        blocks = bt.block_tables[i, lo // 16:(S + 15) // 16].astype(np.int64)
        blocks = blocks[blocks >= 0]
        for g in range(Hkv):
            ids.append(blocks * Hkv + g)
    return np.concatenate(ids) if ids else np.zeros(0, np.int64)


def ceilings(bt, layer, reps: int = 10):
    """Same-run bandwidth ceilings of the attention call's access pattern:
    a torch index_select gather of every K and V tile the call walks (4 KiB
    tiles at D 128 bf16, through the block table, in the walk's order), and a
    plain device-to-device copy of 2 GiB.  Both count bytes read plus bytes
    written; each is the mean over `reps` back-to-back calls."""
    import torch
    dev = layer.q.device
    tile = layer.k_cache[0, 0].numel()
    ktiles = layer.k_cache.view(-1, tile)
    vtiles = layer.v_cache.view(-1, tile)
    idx = torch.as_tensor(walk_tiles(bt, layer), device=dev)
    ko = torch.empty((idx.numel(), tile), dtype=ktiles.dtype, device=dev)
    vo = torch.empty_like(ko)

    def timed(fn):
        fn()
        torch.cuda.synchronize()
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record()
        for _ in range(reps):
            fn()
        e1.record()
        torch.cuda.synchronize()
        return e0.elapsed_time(e1) * 1e-3 / reps

    t = timed(lambda: (torch.index_select(ktiles, 0, idx, out=ko),
                       torch.index_select(vtiles, 0, idx, out=vo)))
    gbytes = 2.0 * 2 * ko.numel() * ko.element_size()
    del ko, vo
    src = torch.empty(1 << 30, dtype=torch.bfloat16, device=dev)
    src.fill_(1.0)
    dst = torch.empty_like(src)
    tc = timed(lambda: dst.copy_(src))
    cbytes = 2.0 * src.numel() * src.element_size()
    del src, dst
    return {"gather_GBps": gbytes / t / 1e9, "gather_bytes": gbytes,
            "copy_GBps": cbytes / tc / 1e9, "copy_bytes": cbytes}


def host_info():
    """CPU model and host RAM of this machine (for the CPU baseline)."""
    model, ram = None, None
    try:
        for line in open("/proc/cpuinfo"):
            if line.startswith("model name"):
                model = line.split(":", 1)[1].strip()
                break
        for line in open("/proc/meminfo"):
            if line.startswith("MemTotal:"):
                ram = round(int(line.split()[1]) * 1024 / 1e9, 1)
                break
    except OSError:
        pass
    return model, ram


def lmhead_timing(av, workload, bt, steps: int):
    """Device time of the LM head fused with greedy acceptance
    (verify_lmhead_accept) for the step's scored rows: hidden [T, H] and the
    model's LM-head weight [V, H] in bf16.  Its roofline is the larger of the
    weight stream over HBM (every weight byte is read once per call while the
    rows fit one row chunk) and the dense bf16 MFMA work 2 T H V."""
    import torch
    cfg = bt.cfg
    dev = bt.logits.device
    hidden, weight = workload.draw_lmhead(cfg, 0, str(dev), bt.designated)
    T, H = hidden.shape
    V = weight.shape[0]
    B = len(bt.q_start) - 1
    outs = [torch.empty(n, dtype=torch.int32, device=dev) for n in (B, B, T, T)]
    ws = torch.empty(max(1, av.lmhead_accept_workspace_size(B, T, H, V)), dtype=torch.uint8,
                     device=dev)
    fn = lambda: av.verify_lmhead_accept(hidden, weight, bt.t_tokens, bt.t_q_start,
                                         accept_len=outs[0], num_emitted=outs[1], emitted=outs[2],
                                         argmax_out=outs[3], workspace=ws)
    fn()
    us = graph_time_us(fn, steps)
    nbytes = float(V * H * 2 + T * H * 2)
    flops = 2.0 * T * H * V
    t_hbm, t_mfma = nbytes / (HBM_PEAK_GBS * 1e3), flops / (MFMA_BF16_PEAK_TFLOPS * 1e6)
    bound = "hbm" if t_hbm >= t_mfma else "mfma"
    res = {"us": us, "rows": T, "hidden": H, "vocab": V, "bytes": nbytes, "flops": flops,
           "GBps": nbytes / (us * 1e-6) / 1e9, "TFLOPs": flops / (us * 1e-6) / 1e12,
           "bound": bound, "roofline_us": max(t_hbm, t_mfma),
           "frac": max(t_hbm, t_mfma) / us}
    del hidden, weight, ws
    return res


def budget_timing(av, workload, *, oracle_ok: bool, batch: int, steps: int, dev: str):
    """Mean device time of one verify_budget call (Sec. 4.2, Alg. 2) on seeded
    candidate sets for the batch, and the oracle's time for the same call.  The
    call is latency-bound (one small launch), so it has no roofline."""
    import numpy as np
    import torch
    start, lens, toks = workload.draw_candidates(1, batch)
    rng = np.random.default_rng(2)
    last = rng.integers(0, 151936, size=batch).astype(np.int32)
    ctx = rng.integers(2048, 16385, size=batch).astype(np.int32)
    d = lambda a: torch.as_tensor(a, device=dev)
    args = (d(start), d(lens), d(toks), d(last))
    ctx_d = d(ctx)
    # B_t = floor(alpha / bz) is the whole batch's budget: eight drafts per
    # request on average, as in the verify workload
    alpha = 8.0 * batch * batch
    out = av.verify_budget(*args, alpha=alpha, g_min=0.3, ctx_len=ctx_d)
    us = graph_time_us(lambda: av.verify_budget(*args, alpha=alpha, g_min=0.3, ctx_len=ctx_d,
                                                out=out), steps)
    res = {"us": us, "batch": batch,
           "candidates": int(start[-1]), "max_len": int(toks.shape[1]), "alpha": alpha, "g_min": 0.3,
           "mean_draft_len": float(out["draft_len"].float().mean().item())}
    if oracle_ok:
        import oracle
        t0 = time.perf_counter()
        reps = 0
        while time.perf_counter() - t0 < 0.5:
            oracle.budget(start, lens, toks, last, alpha, 0.3, ctx_len=ctx)
            reps += 1
        res["oracle_us"] = (time.perf_counter() - t0) / reps * 1e6
    return res


def cpu_baseline(bt, budget_s: float):
    """Time the oracle (as it stands) on the same step: request by request, all
    heads, every layer, and the request's logits rows, until the whole batch is
    done or about `budget_s` seconds have passed.  If the whole batch takes less
    than that, the pass is repeated (up to 5 times) and the median pass is used.
    Reports verified tokens/s of the processed requests."""
    import numpy as np
    import oracle
    import workload
    cfg = bt.cfg
    code = workload.dtype_code(cfg.dtype)
    host = []
    for layer in bt.layers:
        host.append(dict(q=workload.host_storage(layer.q), k=workload.host_storage(layer.k_cache),
                         v=workload.host_storage(layer.v_cache), window=layer.window,
                         sinks=None if layer.sinks is None else layer.sinks.cpu().numpy()))
    logits = workload.host_storage(bt.logits)
    B = len(bt.seq_lens)
    passes = []
    spent = 0.0
    while spent < budget_s and len(passes) < 5:
        done, emitted, elapsed = 0, 0, 0.0
        while done < B and spent + elapsed < budget_s * 2:
            i = done
            q0, q1 = int(bt.q_start[i]), int(bt.q_start[i + 1])
            rows = np.repeat(np.arange(q0, q1, dtype=np.int32), cfg.num_q_heads)
            heads = np.tile(np.arange(cfg.num_q_heads, dtype=np.int32), q1 - q0)
            t0 = time.perf_counter()
            for h in host:
                oracle.attention(num_q_heads=cfg.num_q_heads, num_kv_heads=cfg.num_kv_heads,
                                 head_dim=cfg.head_dim, sliding_window=h["window"], scale=0.0,
                                 dtype=code, q=h["q"], k_cache=h["k"], v_cache=h["v"],
                                 block_tables=bt.block_tables, seq_lens=bt.seq_lens,
                                 q_start=bt.q_start, rows=rows, heads=heads, sinks=h["sinks"])
            am, _ = oracle.argmax(logits[q0:q1], code, with_gap=False)
            qs = np.array([0, q1 - q0], dtype=np.int32)
            acc, ne, _ = oracle.accept(qs, bt.tokens[q0:q1], am)
            elapsed += time.perf_counter() - t0
            emitted += int(ne[0])
            done += 1
        spent += elapsed
        passes.append((emitted / elapsed, done, elapsed))
        if done < B:
            break
    passes.sort()
    value, done, elapsed = passes[len(passes) // 2]
    model, ram = host_info()
    return dict(value=value, unit="verified tokens/s", cores=oracle.num_threads(), kind="oracle",
                cpu_model=model, host_ram_GB=ram,
                sample="%d of %d requests (all %d heads, %d layer(s), their logits rows); "
                       "median of %d pass(es), %.2f s per pass" % (
                           done, B, cfg.num_q_heads, len(bt.layers), len(passes), elapsed))


def summarize_trace(csv_path: str, layers: int) -> None:
    """Inter-kernel idle time inside the timed verify steps, from the kernel
    trace of a rocprofv3 --kernel-trace run of bench.py.  A step is a run of
    attention kernels (per layer and row class: attn_schedule for large
    batches, attn_persist, attn_combine_slots; at least two per layer) ended by
    argmax_chunks, accept_scan, issued back to back.  The most frequent such
    kernel sequence is the step (the timed steps and the warm-up steps have
    it; the attention-only calls timed after them do not)."""
    import collections
    import csv
    import re
    import statistics as st
    rows = []
    for r in csv.DictReader(open(csv_path)):
        m = re.search(r"averify::\(anonymous namespace\)::(\w+)", r["Kernel_Name"])
        name = m.group(1) if m else "other"
        rows.append((int(r["Start_Timestamp"]), int(r["End_Timestamp"]), name))
    rows.sort()
    names = [x[2] for x in rows]
    attention = {"attn_schedule", "attn_persist", "attn_combine_slots"}
    found = []
    for j in range(len(rows) - 1):
        if names[j] == "argmax_chunks" and names[j + 1] == "accept_scan":
            k = j
            while k > 0 and names[k - 1] in attention:
                k -= 1
            if j - k >= 2 * layers:
                found.append((k, j + 2))
    if not found:
        raise SystemExit("no verify step found in %s" % csv_path)
    sig = list(collections.Counter(tuple(names[a:b]) for a, b in found).most_common(1)[0][0])
    steps = [rows[a:b] for a, b in found if names[a:b] == sig]
    dur = collections.defaultdict(list)
    gaps = collections.defaultdict(list)
    spans, busy, between = [], [], []
    for k, stp in enumerate(steps):
        for j, (t0, t1, n) in enumerate(stp):
            dur["%d %s" % (j, n)].append((t1 - t0) / 1e3)
            if j:
                gaps["%s -> %s" % (stp[j - 1][2], n)].append((t0 - stp[j - 1][1]) / 1e3)
        spans.append((stp[-1][1] - stp[0][0]) / 1e3)
        busy.append(sum(t1 - t0 for t0, t1, _ in stp) / 1e3)
        if k and steps[k - 1][-1][1] <= stp[0][0] and stp[0][0] - steps[k - 1][-1][1] < 100e3:
            between.append((stp[0][0] - steps[k - 1][-1][1]) / 1e3)
    print("steps found: %d (kernel sequence %s)" % (len(steps), ", ".join(sig)))
    print("")
    print("| in-step kernel | median us |")
    print("|---|---|")
    for k in sorted(dur, key=lambda x: int(x.split()[0])):
        print("| %s | %.1f |" % (k.split(" ", 1)[1], st.median(dur[k])))
    print("")
    print("| idle gap | median us |")
    print("|---|---|")
    for k, v in gaps.items():
        print("| %s | %.2f |" % (k, st.median(v)))
    if between:
        print("| accept_scan -> next step's attn_persist | %.2f |" % st.median(between))
    print("")
    print("median step span %.1f us, of which kernels busy %.1f us, idle %.1f us" % (
        st.median(spans), st.median(busy), st.median([a - b for a, b in zip(spans, busy)])))


def summarize_counters(paths) -> None:
    """Mean per dispatch of every counter of rocprofv3 --pmc runs, per kernel of
    this library (KiB counters as read, before any calibration)."""
    import collections
    import csv
    import re
    agg = collections.defaultdict(lambda: collections.defaultdict(list))
    for p in paths:
        per = collections.defaultdict(float)
        names = {}
        for r in csv.DictReader(open(p)):
            m = re.search(r"averify::\(anonymous namespace\)::(\w+)", r["Kernel_Name"])
            if not m:
                continue
            key = (r["Dispatch_Id"], r["Counter_Name"])
            per[key] += float(r["Counter_Value"])
            names[r["Dispatch_Id"]] = m.group(1)
        for (d, c), v in per.items():
            agg[names[d]][c].append(v)
    mean = {k: {c: sum(v) / len(v) for c, v in agg[k].items()} for k in agg}
    # derived figures per dispatch: the counters sum over the chip's 8 XCDs and
    # 1024 SIMDs; SQ_WAVE_CYCLES and the SQ wait/active counters count in units
    # of 4 cycles
    need = ("GRBM_GUI_ACTIVE", "SQ_VALU_MFMA_BUSY_CYCLES", "SQ_INSTS_VALU", "SQ_WAIT_INST_ANY",
            "SQ_WAVE_CYCLES", "SQ_LDS_IDX_ACTIVE", "SQ_LDS_BANK_CONFLICT", "TA_BUSY_avr", "TCC_HIT_sum",
            "TCC_MISS_sum", "SQ_WAVES", "SQ_INSTS_SALU", "SQ_INSTS_VMEM", "SQ_INSTS_MFMA")
    print("| kernel | cycles per XCD | waves | MFMA busy | VALU busy | waiting | LDS active | "
          "LDS conflict share | TA busy | L2 hit | VALU / SALU / VMEM / MFMA instr per wave |")
    print("|---|---|---|---|---|---|---|---|---|---|---|")
    for k in sorted(mean):
        m = mean[k]
        if not all(c in m for c in need):
            continue
        cyc = m["GRBM_GUI_ACTIVE"] / 8
        waves = max(m["SQ_WAVES"], 1.0)
        print("| `%s` | %.0f | %.0f | %.2f | %.2f | %.2f | %.2f | %.2f | %.2f | %.2f | %.0f / %.0f / %.0f / %.0f |" % (
            k, cyc, m["SQ_WAVES"], m["SQ_VALU_MFMA_BUSY_CYCLES"] / 1024 / cyc,
            4 * m["SQ_INSTS_VALU"] / 1024 / cyc, m["SQ_WAIT_INST_ANY"] / max(m["SQ_WAVE_CYCLES"], 1.0),
            m["SQ_LDS_IDX_ACTIVE"] / 256 / cyc, m["SQ_LDS_BANK_CONFLICT"] / max(m["SQ_LDS_IDX_ACTIVE"], 1.0),
            m["TA_BUSY_avr"] / cyc, m["TCC_HIT_sum"] / max(m["TCC_HIT_sum"] + m["TCC_MISS_sum"], 1.0),
            m["SQ_INSTS_VALU"] / waves, m["SQ_INSTS_SALU"] / waves, m["SQ_INSTS_VMEM"] / waves,
            m["SQ_INSTS_MFMA"] / waves))
    if "sample_chunks" in mean and "SQ_INSTS_VALU" in mean["sample_chunks"]:
        print()
        print("valu_instructions_sample_chunks: %.0f" % mean["sample_chunks"]["SQ_INSTS_VALU"])
        print("accept_source_sha256: %s" % kernel_source_hash(ACCEPT_SOURCES))
    print()
    print("Raw means per dispatch:")
    print()
    print("```")
    for k in sorted(agg):
        print("%s:" % k)
        for c in sorted(agg[k]):
            v = agg[k][c]
            print("  %-28s %16.1f  (mean of %d dispatches)" % (c, sum(v) / len(v), len(v)))
    print("```")


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--config", default="qwen3_8b")
    ap.add_argument("--seeds", default="0,1,2,3,4",
                    help="comma-separated seeds; each draws its own batch (default: five)")
    ap.add_argument("--cpu-budget", type=float, default=12.0,
                    help="seconds of oracle work for the CPU baseline (0 = skip)")
    ap.add_argument("--side", action=argparse.BooleanOptionalAction, default=True,
                    help="also time the other entry points and the same-run ceilings")
    ap.add_argument("--graph", action=argparse.BooleanOptionalAction, default=False,
                    help="replay the step as one captured HIP graph instead of launching its "
                         "kernels one by one (measured slower on this step)")
    ap.add_argument("--copy-calibration", action="store_true",
                    help="after the timed steps, run one plain elementwise kernel that reads "
                         "and writes %d MiB (scale for the HBM byte counters)" % (CALIB_BYTES >> 20))
    ap.add_argument("--summarize-pmc", nargs=2, metavar=("FETCH_CSV", "WRITE_CSV"),
                    help="print the HBM traffic summary of two rocprofv3 --pmc runs and exit")
    ap.add_argument("--summarize-trace", metavar="KERNEL_TRACE_CSV",
                    help="print the in-step kernel times and idle gaps of a rocprofv3 "
                         "--kernel-trace run and exit")
    ap.add_argument("--summarize-counters", nargs="+", metavar="COUNTER_CSV",
                    help="print per-kernel means of rocprofv3 --pmc runs and exit")
    args = ap.parse_args()

    if args.summarize_pmc:
        summarize_pmc(args.summarize_pmc[0], args.summarize_pmc[1], args.config)
        return
    if args.summarize_counters:
        summarize_counters(args.summarize_counters)
        return

    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) != 1:
        print("bench.py measures one GPU: the verify step runs on a single MI355X "
              "(--gpus %d requested; the verify step here runs and is measured on one GPU)" % args.gpus,
              file=sys.stderr)
        sys.exit(2)

    import workload
    cfg = workload.CONFIGS[args.config]
    if args.summarize_trace:
        summarize_trace(args.summarize_trace, len(cfg.windows))
        return

    import statistics
    import numpy as np
    import torch
    import paper_2608_24004_amd as av

    dev = "cuda:0"
    torch.cuda.set_device(0)
    seeds = [int(x) for x in args.seeds.split(",") if x.strip()]
    lib = av.library()
    stream = torch.cuda.current_stream()
    code = workload.dtype_code(cfg.dtype)
    K = args.steps
    per_seed = []
    first = None   # the first seed's batch and buffers, kept for the side measurements
    for seed in seeds:
        log("config", cfg.name, "seed", seed)
        bt = workload.make_batch(cfg, seed, dev)
        torch.cuda.synchronize()
        outs = [torch.empty_like(l.q) for l in bt.layers]
        ws = []
        for l in bt.layers:
            nb = av.attention_workspace_size(l.q, l.k_cache, bt.t_block_tables, max_q_len=bt.max_q_len,
                                             max_seq_len=bt.max_seq_len, sliding_window=l.window)
            ws.append(torch.empty(max(nb, 1), dtype=torch.uint8, device=dev))
        T, B = bt.total_q, len(bt.seq_lens)
        acc = torch.empty(B, dtype=torch.int32, device=dev)
        ne = torch.empty(B, dtype=torch.int32, device=dev)
        em = torch.empty(T, dtype=torch.int32, device=dev)
        am = torch.empty(T, dtype=torch.int32, device=dev)
        aws = torch.empty(max(1, av.accept_workspace_size(B, T, cfg.vocab, code)), dtype=torch.uint8,
                          device=dev)

        def attention(li, bt=bt, outs=outs, ws=ws):
            l = bt.layers[li]
            av.verify_attention(l.q, l.k_cache, l.v_cache, bt.t_block_tables, bt.t_seq_lens,
                                bt.t_q_start, max_q_len=bt.max_q_len, max_seq_len=bt.max_seq_len,
                                sliding_window=l.window, sinks=l.sinks, out=outs[li], workspace=ws[li])

        def step(bt=bt, acc=acc, ne=ne, em=em, am=am, aws=aws, attention=attention):
            for li in range(len(bt.layers)):
                attention(li)
            av.verify_accept(bt.logits, bt.t_tokens, bt.t_q_start, argmax_out=am, accept_len=acc,
                             num_emitted=ne, emitted=em, workspace=aws)

        for _ in range(args.warmup):
            step()
        torch.cuda.synchronize()
        run_step = step
        if args.graph:
            # The step's launches, captured once: a serving loop replays them
            # without per-kernel launch work on the host.
            graph = torch.cuda.CUDAGraph()
            with torch.cuda.graph(graph):
                step()
            graph.replay()
            torch.cuda.synchronize()
            run_step = graph.replay

        # timed region: K whole steps back to back, one HIP event between
        # consecutive steps (no other synchronisation inside)
        evs = [torch.cuda.Event(enable_timing=True) for _ in range(K + 1)]
        torch.cuda.synchronize()
        wall0 = time.perf_counter()
        evs[0].record(stream)
        for k in range(K):
            run_step()
            evs[k + 1].record(stream)
        torch.cuda.synchronize()
        wall = time.perf_counter() - wall0
        step_ms = [evs[k].elapsed_time(evs[k + 1]) for k in range(K)]
        med_ms = statistics.median(step_ms)
        mean_ms = evs[0].elapsed_time(evs[K]) / K
        # the same K steps with events only at the two ends (what an event
        # between steps costs shows as the difference to mean_ms)
        torch.cuda.synchronize()
        evs[0].record(stream)
        for k in range(K):
            run_step()
        evs[1].record(stream)
        torch.cuda.synchronize()
        plain_ms = evs[0].elapsed_time(evs[1]) / K

        # average duration of one attention call (roofline): K calls of the
        # layer launched back to back on the launch stream, HIP events at the
        # two ends of that region, after the timed steps
        attn_ms = []
        for li in range(len(bt.layers)):
            e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            torch.cuda.synchronize()
            e0.record(stream)
            for _ in range(K):
                attention(li)
            e1.record(stream)
            torch.cuda.synchronize()
            attn_ms.append(e0.elapsed_time(e1) / K)

        emitted = int(ne.sum().item())
        proposed = int(bt.num_drafts.sum())
        accepted = int(acc.sum().item())
        abytes = [attention_bytes(bt, l) for l in bt.layers]
        dom = int(np.argmax(abytes))
        step_bytes = sum(abytes) + accept_bytes(bt)
        r = dict(seed=seed, median_ms=med_ms, mean_ms=mean_ms, plain_ms=plain_ms, min_ms=min(step_ms),
                 max_ms=max(step_ms), wall_ms=wall / K * 1e3, emitted=emitted, proposed=proposed,
                 accepted=accepted, T=T, value=emitted / (med_ms * 1e-3), attn_ms=attn_ms,
                 abytes=abytes, dom=dom, achieved=abytes[dom] / (attn_ms[dom] * 1e-3) / 1e9,
                 step_bytes=step_bytes, mean_context=float(bt.context_len.mean()))
        per_seed.append(r)
        log("seed %d: step median %.4f ms (mean %.4f, without inner events %.4f, min %.4f, max %.4f; "
            "wall %.4f); attention "
            "calls timed alone %s ms; emitted %d -> %.0f verified tok/s; attention layer %d %.3f GB "
            "-> %.0f GB/s" % (seed, med_ms, mean_ms, plain_ms, r["min_ms"], r["max_ms"], r["wall_ms"],
                              ["%.4f" % x for x in attn_ms], emitted, r["value"], dom,
                              abytes[dom] / 1e9, r["achieved"]))
        if first is None:
            first = dict(bt=bt, aws=aws, abytes=abytes, dom=dom)
        else:
            del bt, outs, ws, aws, step, attention, run_step
            torch.cuda.empty_cache()

    bt, aws, abytes, dom = first["bt"], first["aws"], first["abytes"], first["dom"]
    T, B = bt.total_q, len(bt.seq_lens)
    mean = lambda k: float(np.mean([r[k] for r in per_seed]))
    value = mean("value")
    ms_step = mean("median_ms")
    achieved = mean("achieved")
    step_frac = float(np.mean([r["step_bytes"] / r["median_ms"] / 1e6 / HBM_PEAK_GBS for r in per_seed]))
    proposed, accepted = sum(r["proposed"] for r in per_seed), sum(r["accepted"] for r in per_seed)
    log("over %d seed(s): %.0f verified tok/s (mean of per-seed medians), step %.4f ms, attention "
        "%.0f GB/s (%.3f of peak), step %.3f of peak; drafts proposed %d accepted %d" % (
            len(seeds), value, ms_step, achieved, achieved / HBM_PEAK_GBS, step_frac, proposed,
            accepted))

    if args.copy_calibration:
        x = torch.zeros(CALIB_BYTES // 4, dtype=torch.int32, device=dev)
        y = torch.empty_like(x)
        torch.cuda.synchronize()
        torch.bitwise_not(x, out=y)
        torch.cuda.synchronize()
        del x, y

    ceil = budget = append = accept_t = lmhead = None
    if args.side:
        ceil = ceilings(bt, bt.layers[dom])
        log("same-run ceilings:", ceil)
        budget = budget_timing(av, workload, oracle_ok=args.cpu_budget > 0, batch=B, steps=K, dev=dev)
        log("budget allocation (verify_budget):", budget)
        append = kv_append_timing(av, bt, K)
        log("KV append (verify_kv_append):", append)
        accept_t = accept_timing(av, bt, K, aws)
        log("acceptance calls:", accept_t)
        lmhead = lmhead_timing(av, workload, bt, K) if cfg.dtype == "bf16" else None
        log("LM head fused with acceptance (verify_lmhead_accept):", lmhead)

    traffic = stored_traffic(cfg.name)
    if traffic is not None:
        log("HBM traffic per attention call (counters, seed 0): %.4f GB vs algorithmic %.4f GB" % (
            traffic / 1e9, abytes[dom] / 1e9))

    cpu = None
    if args.cpu_budget > 0:
        log("cpu baseline (oracle) ...")
        cpu = cpu_baseline(bt, args.cpu_budget)
        log("cpu baseline", cpu)

    roof = {"bound": "hbm", "achieved": achieved, "peak": HBM_PEAK_GBS, "unit": "GB/s",
            "frac": achieved / HBM_PEAK_GBS, "traffic": traffic,
            "algorithmic_bytes": mean("abytes") if len(bt.layers) == 1 else abytes[dom],
            "kernel": "verify_attention call (attn_persist + attn_combine_slots), layer %d" % dom}
    if ceil:
        roof.update(ceiling_GBps=ceil["gather_GBps"], ceiling_frac=achieved / ceil["gather_GBps"],
                    ceiling_kind="torch index_select of the call's K/V tiles through the block "
                                 "table, bytes read + written",
                    copy_ceiling_GBps=ceil["copy_GBps"],
                    copy_ceiling_frac=achieved / ceil["copy_GBps"])
    res = {
        "metric": "verified tokens/sec per verify step (1 GPU) + achieved HBM GB/s vs peak",
        "value": value,
        "unit": "verified tokens/s",
        "n_gpus": 1,
        "steps": K,
        "warmup": args.warmup,
        "ms_per_step": ms_step,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16" if cfg.dtype == "bf16" else "f32",
        "data": "synthetic",
        "config": {"workload": cfg.name, "description": cfg.description, "batch": B,
                   "total_q": T, "mean_context": mean("mean_context"),
                   "num_q_heads": cfg.num_q_heads, "num_kv_heads": cfg.num_kv_heads,
                   "head_dim": cfg.head_dim, "vocab": cfg.vocab, "layers": len(bt.layers),
                   "seeds": seeds, "hip_graph": bool(args.graph)},
        "roofline": roof,
        "step_hbm_frac": step_frac,
        "scored_positions_per_s": float(np.mean([r["T"] / (r["median_ms"] * 1e-3) for r in per_seed])),
        "rejection_rate": 1 - accepted / max(1, proposed),
        "per_seed": [{k: r[k] for k in ("seed", "median_ms", "mean_ms", "plain_ms", "min_ms", "max_ms",
                                        "emitted",
                                        "value", "achieved")} for r in per_seed],
        "cpu_baseline": cpu,
        "budget_alloc": budget,
        "kv_append": append,
        "accept": accept_t,
        "lmhead_accept": lmhead,
    }
    print(json.dumps(res), flush=True)


if __name__ == "__main__":
    main()
