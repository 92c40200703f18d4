"""The verify step captured in a HIP graph and replayed: every replay must give
the eager call's results exactly (the kernels are deterministic), with other
eager work and synchronisations between the replays."""
from __future__ import annotations

import numpy as np
import pytest
import torch

import paper_2608_24004_amd as av
import workload
DEV = "cuda:0"


def say(*a):
    print(*a, flush=True)


pytestmark = pytest.mark.gpu


def test_graph_replays_match_eager():
    cfg = workload.CONFIGS["qwen3_8b"].replace(batch=6, context=("uniform", 100, 3000))
    bt = workload.make_batch(cfg, 5, DEV)
    layer = bt.layers[0]
    T, B = bt.total_q, len(bt.seq_lens)
    code = workload.dtype_code(cfg.dtype)
    nb = av.attention_workspace_size(layer.q, layer.k_cache, bt.t_block_tables,
                                     max_q_len=bt.max_q_len, max_seq_len=bt.max_seq_len)
    ws = torch.empty(max(nb, 1), dtype=torch.uint8, device=DEV)
    aws = torch.empty(max(1, av.accept_workspace_size(B, T, cfg.vocab, code)), dtype=torch.uint8,
                      device=DEV)

    def outputs():
        return dict(out=torch.empty_like(layer.q), am=torch.empty(T, dtype=torch.int32, device=DEV),
                    acc=torch.empty(B, dtype=torch.int32, device=DEV),
                    ne=torch.empty(B, dtype=torch.int32, device=DEV),
                    em=torch.empty(T, dtype=torch.int32, device=DEV))

    def step(o):
        av.verify_attention(layer.q, layer.k_cache, layer.v_cache, bt.t_block_tables, bt.t_seq_lens,
                            bt.t_q_start, max_q_len=bt.max_q_len, max_seq_len=bt.max_seq_len,
                            out=o["out"], workspace=ws)
        av.verify_accept(bt.logits, bt.t_tokens, bt.t_q_start, argmax_out=o["am"],
                         accept_len=o["acc"], num_emitted=o["ne"], emitted=o["em"], workspace=aws)

    ref = outputs()
    step(ref)
    torch.cuda.synchronize()
    ref = {k: v.clone() for k, v in ref.items()}

    got = outputs()
    for v in got.values():
        v.fill_(-7 if v.dtype == torch.int32 else 0)
    torch.cuda.synchronize()
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph):
        step(got)
    torch.cuda.synchronize()
    for r in range(4):
        say("graph replay", r)
        for v in got.values():  # replays must rewrite every output
            v.fill_(-7 if v.dtype == torch.int32 else 0)
        graph.replay()
        torch.cuda.synchronize()
        for k in ref:
            assert torch.equal(got[k], ref[k]), (r, k)
        # eager work between replays, on other buffers
        other = outputs()
        step(other)
        torch.cuda.synchronize()
        for k in ref:
            assert torch.equal(other[k], ref[k]), (r, k)


def test_graph_replays_of_the_fused_append_match_eager():
    """verify_attention_append captured and replayed: every replay rewrites the
    output and leaves the cache as the eager call did (appending the same
    tokens again is idempotent), with eager calls on a cache copy between
    replays."""
    cfg = workload.CONFIGS["qwen3_8b"].replace(batch=6, context=("uniform", 100, 3000))
    bt = workload.make_batch(cfg, 6, DEV, with_logits=False)
    layer = bt.layers[0]
    T = bt.total_q
    g = torch.Generator(device=DEV)
    g.manual_seed(9)
    kn = torch.randn((T, cfg.num_kv_heads, cfg.head_dim), generator=g, device=DEV).to(layer.q.dtype)
    vn = torch.randn((T, cfg.num_kv_heads, cfg.head_dim), generator=g, device=DEV).to(layer.q.dtype)
    kw = dict(max_q_len=bt.max_q_len, max_seq_len=bt.max_seq_len)
    nb = av.attention_workspace_size(layer.q, layer.k_cache, bt.t_block_tables, **kw)
    ws = torch.empty(max(nb, 1), dtype=torch.uint8, device=DEV)
    kc0, vc0 = layer.k_cache.clone(), layer.v_cache.clone()

    def call(kc, vc, out):
        av.verify_attention_append(layer.q, kn, vn, kc, vc, bt.t_block_tables, bt.t_seq_lens,
                                   bt.t_q_start, out=out, workspace=ws, **kw)

    ref_k, ref_v, ref_o = kc0.clone(), vc0.clone(), torch.empty_like(layer.q)
    call(ref_k, ref_v, ref_o)
    torch.cuda.synchronize()
    kc, vc, out = kc0.clone(), vc0.clone(), torch.zeros_like(layer.q)
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph):
        call(kc, vc, out)
    torch.cuda.synchronize()
    for r in range(4):
        say("fused append graph replay", r)
        out.zero_()
        graph.replay()
        torch.cuda.synchronize()
        assert torch.equal(out, ref_o) and torch.equal(kc, ref_k) and torch.equal(vc, ref_v), r
        ok, ov, oo = kc0.clone(), vc0.clone(), torch.empty_like(layer.q)
        call(ok, ov, oo)
        torch.cuda.synchronize()
        assert torch.equal(oo, ref_o) and torch.equal(ok, ref_k), r
