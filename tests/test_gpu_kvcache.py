"""GPU parity of spec_fp8_kv_cache_write (the FP8 KV-cache write of the
verify step's new keys and values) against oracle/kvcache.py.

Codes and scales are bit-exact over the whole cache: the stored slots hold
the oracle's codes, and every other slot keeps its sentinel bytes (padding
slots, slots beyond the cache and untouched slots are never written).
Head sizes cover every lane-group width of the kernel (D/8 rounded up to a
power of two from 1 to 64), including groups with idle lanes."""

import numpy as np
import pytest
import torch

import workloads as wl
from oracle import kvcache as ok, quantize as oq
from tests.gpu_util import dev_bf16, dev_f32, host, need_gpu, say

pytestmark = pytest.mark.gpu

SENT_CODE = 0xAB
SENT_SCALE = -1.0


def _slots(T, num_slots, seed):
    rng = np.random.default_rng(seed)
    s = rng.choice(num_slots, T, replace=False).astype(np.int64)
    if T >= 3:
        s[1] = -1                     # padding token
        s[T - 1] = num_slots + 5      # beyond the cache: skipped
    return s


def _run(p, kb, vb, slots, H, D, num_slots, static=None):
    """Device and oracle writes from sentinel-filled caches; returns both."""
    T = kb.shape[0]
    kc = torch.full((num_slots, H, D), SENT_CODE, dtype=torch.uint8, device="cuda")
    vc = torch.full_like(kc, SENT_CODE)
    dk = dev_bf16(kb)[:, :H * D].view(T, H, D) if kb.shape[1] == H * D else None
    dv = dev_bf16(vb)[:, :H * D].view(T, H, D) if vb.shape[1] == H * D else None
    dslots = torch.from_numpy(slots).cuda()
    if static is None:
        ks = torch.full((num_slots, H), SENT_SCALE, dtype=torch.float32, device="cuda")
        vs = torch.full_like(ks, SENT_SCALE)
    else:
        ks, vs = dev_f32([static[0]]), dev_f32([static[1]])
    p.kv_cache_write(dk, dv, dslots, kc, vc, ks, vs, per_tensor=static is not None)
    rk = np.full((num_slots, H, D), SENT_CODE, np.uint8)
    rv = rk.copy()
    rks = np.full((num_slots, H), SENT_SCALE, np.float32)
    rvs = rks.copy()
    ok.kv_cache_write(kb, slots, H, D, rk, rks, None if static is None else static[0])
    ok.kv_cache_write(vb, slots, H, D, rv, rvs, None if static is None else static[1])
    return (host(kc), host(vc), host(ks), host(vs)), (rk, rv, rks, rvs)


@pytest.mark.parametrize("T,H,D,seed", [
    (5, 8, 128, 0),          # 16-lane groups, the Llama head
    (37, 4, 64, 1),          # 8-lane groups
    (13, 3, 80, 2),          # 10 of 16 lanes live
    (9, 2, 256, 3),          # 32-lane groups
    (7, 1, 512, 4),          # 64-lane groups, one head
    (11, 5, 8, 5),           # one lane per row
    (3, 2, 24, 6),           # 3 of 4 lanes live
    (1, 8, 128, 7),          # one token
])
def test_kv_cache_write_per_row_vs_oracle(T, H, D, seed):
    p = need_gpu()
    say(f"kv cache write per-row T={T} H={H} D={D}")
    kb = wl.linear_activations(T, H * D, seed, 0.02, 20.0)
    vb = wl.linear_activations(T, H * D, seed + 100)
    num_slots = 2 * T + 3
    dev, ref = _run(p, kb, vb, _slots(T, num_slots, seed), H, D, num_slots)
    for name, a, b in zip(("k codes", "v codes", "k scales", "v scales"), dev, ref):
        np.testing.assert_array_equal(a, b, err_msg=name)


@pytest.mark.parametrize("T,H,D,seed", [(5, 8, 128, 10), (13, 3, 80, 11), (7, 1, 512, 12)])
def test_kv_cache_write_static_scale_vs_oracle(T, H, D, seed):
    """Static per-tensor scales calibrated on the device (spec_fp8_quantize,
    CALIBRATE) over the first tokens; the later tokens exceed that range and
    saturate."""
    p = need_gpu()
    say(f"kv cache write static T={T} H={H} D={D}")
    kf = wl.f32_from_bf16_bits(wl.linear_activations(T, H * D, seed, 0.02, 20.0))
    kf[T // 2:] *= 3.0
    kb = wl.bf16_bits_from_f32(kf)
    vb = wl.linear_activations(T, H * D, seed + 100)
    cal = (T + 1) // 2
    scales = []
    for x in (kb, vb):
        run = torch.zeros(1, dtype=torch.float32, device="cuda")
        p.calibrate(dev_bf16(x[:cal]), run)
        s_ref = oq.calibrate_per_tensor([x[:cal]])
        assert host(run)[0] == s_ref
        scales.append(float(s_ref))
    num_slots = 2 * T + 3
    dev, ref = _run(p, kb, vb, _slots(T, num_slots, seed), H, D, num_slots, static=scales)
    for name, a, b in zip(("k codes", "v codes"), dev[:2], ref[:2]):
        np.testing.assert_array_equal(a, b, err_msg=name)


def test_kv_cache_write_full_size_from_qkv_columns():
    """The verify step's T = 320 new tokens (B = 64, k = 4) of 8 KV heads of
    128, read in place from the K and V column blocks of the QKV projection
    output [320, 6144], written into a paged cache of 16-token blocks."""
    p = need_gpu()
    c = wl.CONFIGS["KV"]
    B, T, H, D, bs = c["B"], c["T"], c["H"], c["D"], c["block_size"]
    n_new = T // B
    rng = np.random.default_rng(c["seed"])
    ctx = rng.integers(c["ctx_min"], c["ctx_max"] + 1, size=B)
    slots, num_slots = wl.paged_slot_mapping(B, n_new, ctx, bs, seed=c["seed"] + 1)
    say(f"kv cache write full size T={T} H={H} D={D} slots={num_slots}")
    q_cols = 4096
    qkv = wl.linear_activations(T, q_cols + 2 * H * D, c["seed"] + 2, c["key_outlier_frac"],
                                c["key_outlier_scale"])
    dqkv = dev_bf16(qkv)
    dk = dqkv[:, q_cols:q_cols + H * D].view(T, H, D)
    dv = dqkv[:, q_cols + H * D:].view(T, H, D)
    kc = torch.full((num_slots, H, D), SENT_CODE, dtype=torch.uint8, device="cuda")
    vc = torch.full_like(kc, SENT_CODE)
    ks = torch.full((num_slots, H), SENT_SCALE, dtype=torch.float32, device="cuda")
    vs = torch.full_like(ks, SENT_SCALE)
    dslots = torch.from_numpy(slots).cuda()
    p.kv_cache_write(dk, dv, dslots, kc, vc, ks, vs)
    torch.cuda.synchronize()
    kb = np.ascontiguousarray(qkv[:, q_cols:q_cols + H * D])
    vb = np.ascontiguousarray(qkv[:, q_cols + H * D:])
    for dev_c, dev_s, xb in ((kc, ks, kb), (vc, vs, vb)):
        rc = np.zeros((num_slots, H, D), np.uint8)
        rs = np.zeros((num_slots, H), np.float32)
        ok.kv_cache_write(xb, slots, H, D, rc, rs)
        np.testing.assert_array_equal(host(dev_c[dslots]), rc[slots])
        np.testing.assert_array_equal(host(dev_s[dslots]), rs[slots])
        mask = torch.ones(num_slots, dtype=torch.bool, device="cuda")
        mask[dslots] = False
        assert int((dev_c[mask] != SENT_CODE).sum()) == 0
        assert int((dev_s[mask] != SENT_SCALE).sum()) == 0


def test_kv_cache_write_empty_calls():
    p = need_gpu()
    H, D = 2, 16
    kc = torch.full((4, H, D), SENT_CODE, dtype=torch.uint8, device="cuda")
    vc = torch.full_like(kc, SENT_CODE)
    ks = torch.zeros((4, H), dtype=torch.float32, device="cuda")
    vs = torch.zeros_like(ks)
    empty = torch.zeros((0, H, D), dtype=torch.bfloat16, device="cuda")
    p.kv_cache_write(empty, empty, torch.zeros(0, dtype=torch.int64, device="cuda"), kc, vc, ks, vs)
    k = torch.ones((3, H, D), dtype=torch.bfloat16, device="cuda")
    p.kv_cache_write(k, k, torch.full((3,), -1, dtype=torch.int64, device="cuda"), kc, vc, ks, vs)
    assert int((kc != SENT_CODE).sum()) == 0 and int((vc != SENT_CODE).sum()) == 0
