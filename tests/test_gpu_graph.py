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
    M, K1, N1, K2 = 80, 1024, 2 * 4096, 4096        # gate|up then down (split-K shape)
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
    gws = torch.zeros((max(p.gemm_workspace_bytes(M, N1, K1), p.gemm_workspace_bytes(M, N2, K2), 16),),
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


def test_graph_replays_of_the_lm_head_and_tree_paths():
    """The LM head with statistics followed by the acceptance from those
    statistics, and the token-tree acceptance (greedy and sampling), captured
    once and replayed with new inputs: every replay equals eager launches, and
    two eager runs agree (determinism)."""
    p = need_gpu()
    dev = "cuda"
    B, k, K, V, T = 6, 3, 512, 3000, 0.8
    M = B * (k + 1)
    N = 9
    par = torch.tensor([-1, -1, 0, 0, 1, 2, 2, 4, 5], dtype=torch.int32, device=dev).repeat(B, 1).contiguous()
    hq = torch.empty((M, K), dtype=torch.uint8, device=dev)
    hs = torch.empty((M,), dtype=torch.float32, device=dev)
    wq = torch.empty((V, K), dtype=torch.uint8, device=dev)
    wsc = torch.empty((V,), dtype=torch.float32, device=dev)
    zd = torch.empty((B, k, V), dtype=torch.bfloat16, device=dev)
    xt = torch.empty((B, k), dtype=torch.int32, device=dev)
    u = torch.empty((B, k + 1), dtype=torch.float32, device=dev)
    zt_tree = torch.empty((B, N + 1, V), dtype=torch.bfloat16, device=dev)
    x_tree = torch.empty((B, N), dtype=torch.int32, device=dev)
    u_tree = torch.empty((B, N + 1), dtype=torch.float32, device=dev)
    logits = torch.empty((M, V), dtype=torch.bfloat16, device=dev)
    stats = torch.empty((M, p.logit_stats_count(M, V, K), 2), dtype=torch.float32, device=dev)
    aws = torch.empty((p.accept_workspace_bytes(B, k, V),), dtype=torch.uint8, device=dev)
    tws = torch.empty((p.accept_tree_workspace_bytes(B, N, V),), dtype=torch.uint8, device=dev)
    outs = [torch.empty((B, k + 1), dtype=torch.int32, device=dev), torch.empty((B,), dtype=torch.int32, device=dev),
            torch.empty((B, N + 1), dtype=torch.int32, device=dev), torch.empty((B, N), dtype=torch.int32, device=dev),
            torch.empty((B,), dtype=torch.int32, device=dev), torch.empty((B, N + 1), dtype=torch.int32, device=dev),
            torch.empty((B, N), dtype=torch.int32, device=dev), torch.empty((B,), dtype=torch.int32, device=dev)]

    def load(seed):
        a, s = p.quantize(dev_bf16(wl.linear_activations(M, K, seed, 0.01, 20.0)))
        hq.copy_(a); hs.copy_(s)
        a, s = p.quantize(dev_bf16(wl.linear_weights(V, K, seed + 1, 0.1)))
        wq.copy_(a); wsc.copy_(s)
        _, d_ = wl.accept_logits(B, k, V, seed + 2, 0.8)
        zd.copy_(dev_bf16(d_))
        xt.copy_(dev_i32(wl.draft_tokens_sampled(d_, T, seed=seed + 3)))
        u.copy_(dev_f32(wl.philox_uniforms((B, k + 1), seed=seed + 4)))
        t_, dd = wl.accept_logits(B, N, V, seed + 5, 0.95)
        zt_tree.copy_(dev_bf16(t_))
        x_tree.copy_(dev_i32(wl.tree_tokens_topk(dd, par[0].cpu().numpy())))
        u_tree.copy_(dev_f32(wl.philox_uniforms((B, N + 1), seed=seed + 6)))

    def step():
        p.gemm_logit_stats(hq, hs, wq, wsc, T, out=logits, stats=stats)
        p.verify_accept(logits.view(B, k + 1, V), zd, xt, u, T, workspace=aws, out_tokens=outs[0],
                        num_accepted=outs[1], target_stats=stats)
        p.verify_accept_tree(zt_tree, par, x_tree, None, 0.0, workspace=tws, out_tokens=outs[2],
                             accepted_nodes=outs[3], num_accepted=outs[4])
        p.verify_accept_tree(zt_tree, par, x_tree, u_tree, T, workspace=tws, out_tokens=outs[5],
                             accepted_nodes=outs[6], num_accepted=outs[7])

    def snapshot():
        torch.cuda.synchronize()
        return [t.detach().clone() for t in [logits, stats] + outs]

    load(10)
    step()
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        step()
    torch.cuda.synchronize()
    for rep, seed in enumerate((20, 30, 30)):
        say(f"graph replay {rep} (inputs seed {seed})")
        load(seed)
        step()
        ref = snapshot()
        step()
        again = snapshot()
        for a, b in zip(again, ref):
            assert torch.equal(a.view(torch.uint8), b.view(torch.uint8)), rep     # deterministic
        for t in outs:
            t.fill_(-7)
        stats.fill_(float("nan"))
        torch.cuda.synchronize()
        g.replay()
        got = snapshot()
        for i, (a, b) in enumerate(zip(got, ref)):
            assert torch.equal(a.view(torch.uint8), b.view(torch.uint8)), (rep, i)


def test_graph_replays_of_kv_cache_tree_mask_and_clip_count():
    """The FP8 KV-cache write, the tree attention masks and the clip count
    (its counter cleared by a fill kernel inside the graph) replayed with new
    inputs, each replay equal to eager calls on the same inputs."""
    p = need_gpu()
    T, H, D, S = 40, 8, 128, 96
    N, B = 25, 16
    dev = "cuda"
    kx = torch.empty((T, H, D), dtype=torch.bfloat16, device=dev)
    vx = torch.empty_like(kx)
    slots = torch.empty((T,), dtype=torch.int64, device=dev)
    kc = torch.zeros((S, H, D), dtype=torch.uint8, device=dev)
    vc = torch.zeros_like(kc)
    ks = torch.zeros((S, H), dtype=torch.float32, device=dev)
    vs = torch.zeros_like(ks)
    par = torch.empty((B, N), dtype=torch.int32, device=dev)
    mask = torch.empty((B, N), dtype=torch.int64, device=dev)
    depth = torch.empty((B, N), dtype=torch.int32, device=dev)
    scale = torch.empty((1,), dtype=torch.float32, device=dev)
    cnt = torch.zeros((1,), dtype=torch.int64, device=dev)

    def load(seed):
        rng = np.random.default_rng(seed)
        kx.copy_(dev_bf16(wl.linear_activations(T, H * D, seed, 0.01, 20.0)).view(T, H, D))
        vx.copy_(dev_bf16(wl.linear_activations(T, H * D, seed + 1)).view(T, H, D))
        sl = rng.choice(S, T, replace=False).astype(np.int64)
        sl[3] = -1
        slots.copy_(torch.from_numpy(sl))
        par.copy_(dev_i32(np.array([[int(rng.integers(-1, n)) if n else -1 for n in range(N)]
                                    for _ in range(B)], np.int32)))
        scale.copy_(dev_f32([0.02 + 0.01 * (seed % 3)]))

    def run():
        kc.zero_(); vc.zero_(); ks.zero_(); vs.zero_(); cnt.zero_()
        p.kv_cache_write(kx, vx, slots, kc, vc, ks, vs)
        p.tree_attention_mask(par, mask=mask, depth=depth)
        p.clip_count(kx.view(T, H * D), scale, count=cnt)

    def snap():
        torch.cuda.synchronize()
        return [t.clone() for t in (kc, vc, ks, vs, mask, depth, cnt)]

    load(1)
    run()
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        run()
    for rep, seed in enumerate((5, 6, 6, 9)):
        say(f"graph replay {rep} (inputs seed {seed})")
        load(seed)
        run()
        ref = snap()
        load(seed)
        g.replay()
        got = snap()
        for a, b in zip(got, ref):
            assert torch.equal(a, b)
        torch.cuda.synchronize()
