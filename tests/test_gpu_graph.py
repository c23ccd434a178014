"""The verify path captured in a HIP graph: every replay equals eager launches.

The bench runs the step as a graph.  The library's kernels clear their own
scratch (the acceptance ticket counters are zeroed by a kernel, split-K
partials are overwritten), so a replay must reproduce the eager result bit for
bit.  The graph is replayed several times with new inputs copied into the
captured buffers, with eager work and synchronizations in between, and each
replay is compared with an eager run on the same inputs.
"""

import numpy as np
import pytest
import torch

import workloads as wl
from tests.gpu_util import dev_bf16, dev_i32, dev_f32, need_gpu, say

pytestmark = pytest.mark.gpu


def test_graph_replays_match_eager():
    p = need_gpu()
    M, K1, N1, K2 = 80, 1024, 2 * 1536, 1536        # gate|up then down (split-K shape)
    N2 = 1024
    B, k, V, T = 8, 3, 20000, 0.7
    dev = "cuda"
    # captured (static) buffers
    x = torch.empty((M, K1), dtype=torch.bfloat16, device=dev)
    w1q = torch.empty((N1, K1), dtype=torch.uint8, device=dev)
    w1s = torch.empty((N1,), dtype=torch.float32, device=dev)
    w2q = torch.empty((N2, K2), dtype=torch.uint8, device=dev)
    w2s = torch.empty((N2,), dtype=torch.float32, device=dev)
    zt = torch.empty((B, k + 1, V), dtype=torch.bfloat16, device=dev)
    zd = torch.empty((B, k, V), dtype=torch.bfloat16, device=dev)
    xt = torch.empty((B, k), dtype=torch.int32, device=dev)
    u = torch.empty((B, k + 1), dtype=torch.float32, device=dev)
    q1 = torch.empty((M, K1), dtype=torch.uint8, device=dev)
    s1 = torch.empty((M,), dtype=torch.float32, device=dev)
    y1 = torch.empty((M, N1), dtype=torch.bfloat16, device=dev)
    q2 = torch.empty((M, K2), dtype=torch.uint8, device=dev)
    s2 = torch.empty((M,), dtype=torch.float32, device=dev)
    y2 = torch.empty((M, N2), dtype=torch.float32, device=dev)
    gws = torch.empty((max(p.gemm_workspace_bytes(M, N1, K1), p.gemm_workspace_bytes(M, N2, K2), 16),),
                      dtype=torch.uint8, device=dev)
    assert p.gemm_workspace_bytes(M, N2, K2) > 0       # the down shape splits K
    aws = torch.empty((p.accept_workspace_bytes(B, k, V),), dtype=torch.uint8, device=dev)
    out = torch.empty((B, k + 1), dtype=torch.int32, device=dev)
    num = torch.empty((B,), dtype=torch.int32, device=dev)

    def load(seed):
        x.copy_(dev_bf16(wl.linear_activations(M, K1, seed, 0.01, 20.0)))
        a, s = p.quantize(dev_bf16(wl.linear_weights(N1, K1, seed + 1, 0.02)))
        w1q.copy_(a); w1s.copy_(s)
        a, s = p.quantize(dev_bf16(wl.linear_weights(N2, K2, seed + 2, 0.02)))
        w2q.copy_(a); w2s.copy_(s)
        t_, d_ = wl.accept_logits(B, k, V, seed + 3, 0.8)
        zt.copy_(dev_bf16(t_)); zd.copy_(dev_bf16(d_))
        xt.copy_(dev_i32(wl.draft_tokens_sampled(d_, T, seed=seed + 4)))
        u.copy_(dev_f32(wl.philox_uniforms((B, k + 1), seed=seed + 5)))

    def step():
        p.quantize(x, out=q1, scales=s1)
        p.gemm(q1, s1, w1q, w1s, out=y1, workspace=gws)
        p.quantize(y1, silu_mul=True, out=q2, scales=s2)
        p.gemm(q2, s2, w2q, w2s, out_dtype=torch.float32, out=y2, workspace=gws)
        p.verify_accept(zt, zd, xt, u, T, workspace=aws, out_tokens=out, num_accepted=num)

    def snapshot():
        torch.cuda.synchronize()
        return [t.detach().clone() for t in (q1, s1, y1, q2, s2, y2, out, num)]

    load(100)
    step()                                            # warm up outside the capture
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        step()
    torch.cuda.synchronize()
    for rep, seed in enumerate((200, 300, 300, 400)):
        say(f"graph replay {rep} (inputs seed {seed})")
        load(seed)
        step()                                        # eager reference
        ref = snapshot()
        for t in (q1, s1, y1, q2, s2, y2, out, num):  # poison the outputs
            t.fill_(0) if t.dtype != torch.float32 else t.fill_(float("nan"))
        torch.cuda.synchronize()
        g.replay()
        got = snapshot()
        names = ("q1", "s1", "y1", "q2", "s2", "y2", "out", "num")
        for n, a, b in zip(names, got, ref):
            assert torch.equal(a.view(torch.uint8) if a.dtype == torch.bfloat16 else a,
                               b.view(torch.uint8) if b.dtype == torch.bfloat16 else b), (rep, n)
        # eager work between replays on the same buffers
        p.gemm(q1, s1, w1q, w1s, out=y1, workspace=gws)
        torch.cuda.synchronize()
