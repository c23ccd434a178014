"""Every kernel run twice on the same inputs gives bit-identical results (an
LDS race or an order-dependent reduction would show here): the GEMM in every
tile configuration the planner picks (including split K and the grouped
large-M order), its statistics and SiLU epilogues, tree sampling, the FP8
KV-cache write and the clip count."""

import numpy as np
import pytest
import torch

import workloads as wl
from tests.gpu_util import dev_bf16, dev_f32, dev_i32, need_gpu, say

pytestmark = pytest.mark.gpu


def _q(p, M, K, seed):
    return p.quantize(dev_bf16(wl.linear_activations(M, K, seed, 0.01, 20.0)))


@pytest.mark.parametrize("M,N,K", [
    (8, 1024, 512), (64, 4096, 4096), (80, 6144, 1024), (80, 28672, 512),   # small M, split K, wide N
    (320, 28672, 1024), (320, 4096, 4096), (320, 6144, 1024), (320, 4096, 2048),
    (1300, 672, 256),                                                         # grouped large-M order
    (4096, 4096, 256), (2048, 7168, 512),                                     # 256x256, 256x224 in-place-refill tiles
    (300, 60096, 256),                                                        # 160x192 tiles, wide N
])
def test_gemm_twice(M, N, K):
    p = need_gpu()
    say(f"gemm twice M={M} N={N} K={K}")
    a, sa = _q(p, M, K, M + N)
    w, sw = _q(p, N, K, K + 1)
    y1 = p.gemm(a, sa, w, sw, out_dtype=torch.float32)
    y2 = p.gemm(a, sa, w, sw, out_dtype=torch.float32)
    torch.cuda.synchronize()
    assert torch.equal(y1, y2)


def test_epilogues_twice():
    p = need_gpu()
    M, V, K, I = 320, 13000, 512, 2056
    a, sa = _q(p, M, K, 5)
    w, sw = _q(p, V, K, 6)
    l1, s1 = p.gemm_logit_stats(a, sa, w, sw, 0.7)
    l2, s2 = p.gemm_logit_stats(a, sa, w, sw, 0.7)
    wg, swg = _q(p, 2 * I, K, 7)
    h1 = p.gemm_silu_mul(a, sa, wg, swg)
    h2 = p.gemm_silu_mul(a, sa, wg, swg)
    torch.cuda.synchronize()
    assert torch.equal(l1, l2) and torch.equal(s1, s2) and torch.equal(h1, h2)


def test_tree_kv_and_clip_twice():
    p = need_gpu()
    B, V = 12, 5000
    par = np.asarray(wl.TREE25, np.int32)
    N = len(par)
    zt, zd = wl.accept_logits(B, N, V, 3, 0.95, scale=2.0)
    x = dev_i32(wl.tree_tokens_topk(zd, par))
    parents = dev_i32(np.tile(par, (B, 1)))
    u = dev_f32(wl.philox_uniforms((B, N + 1), seed=4))
    dzt = dev_bf16(zt)
    r1 = p.verify_accept_tree(dzt, parents, x, u, 0.7)
    r2 = p.verify_accept_tree(dzt, parents, x, u, 0.7)
    T, H, D, S = 100, 8, 128, 256
    kx = dev_bf16(wl.linear_activations(T, H * D, 8, 0.01, 20.0)).view(T, H, D)
    slots = torch.from_numpy(np.random.default_rng(9).choice(S, T, replace=False).astype(np.int64)).cuda()
    outs = []
    for _ in range(2):
        kc = torch.zeros((S, H, D), dtype=torch.uint8, device="cuda")
        ks = torch.zeros((S, H), dtype=torch.float32, device="cuda")
        p.kv_cache_write(kx, kx, slots, kc, kc.clone(), ks, ks.clone())
        outs.append((kc, ks))
    c1 = p.clip_count(kx.view(T, H * D), dev_f32([0.01]))
    c2 = p.clip_count(kx.view(T, H * D), dev_f32([0.01]))
    torch.cuda.synchronize()
    assert all(torch.equal(a, b) for a, b in zip(r1, r2))
    assert torch.equal(outs[0][0], outs[1][0]) and torch.equal(outs[0][1], outs[1][1])
    assert torch.equal(c1, c2)
