"""verify_accept_noalloc (no workspace: the library's per-GPU scratch array)
against verify_accept with a caller-owned workspace, bit for bit, on two calls
in a row -- the second smaller than the first, so that it runs over what the
first left in the scratch -- and a third call in the other storage dtype."""
from __future__ import annotations

import sys

import numpy as np
import pytest
import torch

import paper_2608_24004_amd as av
import workload

pytestmark = pytest.mark.gpu
DEV = "cuda:0"


def say(*a):
    print(*a, file=sys.stderr, flush=True)


def _case(rows_per_req, vocab, dtype, seed):
    """Seeded logits with drafts planted to agree with a random prefix of the
    rows' argmax (the argmax taken by torch on the device: it only shapes the
    drafts; both calls under test read the same logits)."""
    g = torch.Generator(device=DEV)
    g.manual_seed(seed)
    n = np.asarray(rows_per_req)
    q_start = np.zeros(n.size + 1, dtype=np.int32)
    q_start[1:] = np.cumsum(n)
    T = int(q_start[-1])
    logits = torch.randn((T, vocab), generator=g, device=DEV).to(workload.torch_dtype(dtype))
    am = logits.float().argmax(dim=1).cpu().numpy().astype(np.int32)
    rng = np.random.default_rng(seed)
    tokens = rng.integers(0, vocab, size=T).astype(np.int32)
    for i in range(n.size):
        q0, k = int(q_start[i]), int(n[i]) - 1
        keep = int(rng.integers(0, k + 1)) if k > 0 else 0
        for j in range(1, k + 1):
            tokens[q0 + j] = am[q0 + j - 1] if j <= keep else (am[q0 + j - 1] + 1) % vocab
    return (logits, torch.as_tensor(tokens, device=DEV), torch.as_tensor(q_start, device=DEV))


def _outputs(B, T):
    i32 = torch.int32
    return dict(accept_len=torch.full((B,), -7, dtype=i32, device=DEV),
                num_emitted=torch.full((B,), -7, dtype=i32, device=DEV),
                emitted=torch.full((T,), -7, dtype=i32, device=DEV),
                argmax_out=torch.full((T,), -7, dtype=i32, device=DEV))


def _check_same(logits, tokens, q_start, what):
    B, T = q_start.numel() - 1, logits.shape[0]
    ref = av.verify_accept(logits, tokens, q_start, **_outputs(B, T))
    got = av.verify_accept_noalloc(logits, tokens, q_start, **_outputs(B, T))
    torch.cuda.synchronize()
    for name, a, b in zip(("accept_len", "num_emitted", "emitted", "argmax"), got, ref):
        np.testing.assert_array_equal(a.cpu().numpy(), b.cpu().numpy(), err_msg="%s %s" % (what, name))
    say(what, "ok: rows", T, "accepted", int(ref[0].sum().item()))


def test_noalloc_matches_workspace_call_twice_then_smaller():
    # first call: the Qwen-3-8B-shaped step's acceptance (32 requests x 9 rows,
    # vocabulary 151936, bf16), the largest scratch use of the three
    say("no-alloc call 1: 32 x 9 rows, V 151936 bf16")
    _check_same(*_case([9] * 32, 151936, "bf16", 11), "call 1")
    # second call, smaller: ragged rows (one request with no row), V 5003
    say("no-alloc call 2: ragged 7 requests, V 5003 bf16")
    _check_same(*_case([1, 3, 0, 17, 2, 9, 5], 5003, "bf16", 12), "call 2")
    # third: fp32 logits, vocabulary below one chunk
    say("no-alloc call 3: 3 requests, V 300 fp32")
    _check_same(*_case([4, 1, 6], 300, "f32", 13), "call 3")


def test_noalloc_rejects_oversized_calls():
    logits = torch.zeros((1, 8), dtype=torch.bfloat16, device=DEV)
    lib = av.library()
    rc = lib.verify_accept_noalloc(1, 600_000, 151936, 0, av.BF16, logits.data_ptr(),
                                   logits.data_ptr(), logits.data_ptr(), None, logits.data_ptr(),
                                   logits.data_ptr(), logits.data_ptr(), None)
    assert rc == av.EWORKSPACE
