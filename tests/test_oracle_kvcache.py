"""Pins of the oracle's FP8 KV-cache write (oracle/kvcache.py).

Against torch's own float8_e4m3fn cast (an implementation independent of the
oracle's encoder) on explicitly sliced head columns, the E4M3 error bound of
every stored row, the amax -> 448 property per head, the paged slot layout
(positions mapped through the page table by hand), and the skip rule."""

import numpy as np
import torch

import workloads as wl
from oracle import e4m3, kvcache as ok, quantize as oq


def _heads(T, H, D, seed):
    return wl.linear_activations(T, H * D, seed, outlier_frac=0.01, outlier_scale=20.0)


def test_rows_match_torch_cast_at_their_slots():
    T, H, D = 9, 4, 64
    x = _heads(T, H, D, 3)
    slots = np.array([7, 0, 12, 3, 5, 1, 9, 14, 2], np.int64)
    cache = np.full((16, H, D), 0xAB, np.uint8)
    scales = np.full((16, H), -1.0, np.float32)
    ok.kv_cache_write(x, slots, H, D, cache, scales)
    xf = oq.bf16_to_f32(x)
    for t in range(T):
        for h in range(H):
            row = xf[t, h * D:(h + 1) * D]
            s = np.float32(np.float64(np.max(np.abs(row))) / 448.0)
            assert scales[slots[t], h] == s
            inv = np.float32(1.0 / np.float64(s))
            ref = torch.clamp(torch.from_numpy(row) * torch.tensor(inv), -448.0, 448.0) \
                .to(torch.float8_e4m3fn).view(torch.uint8).numpy()
            np.testing.assert_array_equal(cache[slots[t], h], ref)
    untouched = np.setdiff1d(np.arange(16), slots)
    assert np.all(cache[untouched] == 0xAB) and np.all(scales[untouched] == -1.0)


def test_error_bound_and_amax_per_head():
    T, H, D = 20, 8, 128
    x = _heads(T, H, D, 4)
    slots = np.arange(T, dtype=np.int64)[::-1].copy()
    cache = np.zeros((T, H, D), np.uint8)
    scales = np.zeros((T, H), np.float32)
    ok.kv_cache_write(x, slots, H, D, cache, scales)
    xf = oq.bf16_to_f32(x).astype(np.float64).reshape(T, H, D)
    got = e4m3.decode(cache[slots]) * scales[slots][..., None].astype(np.float64)
    y = np.abs(xf) / scales[slots][..., None]
    normal = y >= 2.0 ** -6
    err = np.abs(got - xf)
    assert np.all(err[normal] <= 2.0 ** -4 * np.abs(xf[normal]) * (1 + 2.0 ** -20))
    sub_bound = (2.0 ** -10) * np.broadcast_to(scales[slots][..., None], xf.shape) * (1 + 2.0 ** -20)
    assert np.all(err[~normal] <= sub_bound[~normal])
    top = np.argmax(np.abs(xf), axis=2)
    codes = np.take_along_axis(cache[slots], top[..., None], axis=2)[..., 0]
    assert np.all((codes & 0x7F) == 0x7E)


def test_heads_are_independent_rows():
    """Scaling one head by 2^3 scales only that head's scale; no code changes."""
    T, H, D = 4, 3, 32
    xf = oq.bf16_to_f32(_heads(T, H, D, 5))
    x2 = xf.copy()
    x2[:, D:2 * D] *= 8.0
    slots = np.arange(T, dtype=np.int64)
    c1, s1 = ok.kv_cache_write(wl.bf16_bits_from_f32(xf), slots, H, D, np.zeros((T, H, D), np.uint8),
                               np.zeros((T, H), np.float32))
    c2, s2 = ok.kv_cache_write(wl.bf16_bits_from_f32(x2), slots, H, D, np.zeros((T, H, D), np.uint8),
                               np.zeros((T, H), np.float32))
    np.testing.assert_array_equal(c1, c2)
    np.testing.assert_array_equal(s2[:, 1], s1[:, 1] * 8)
    np.testing.assert_array_equal(s2[:, [0, 2]], s1[:, [0, 2]])


def test_static_scale_saturates_and_skips():
    T, H, D = 6, 2, 16
    xf = oq.bf16_to_f32(_heads(T, H, D, 6))
    xf[4:] *= 3.0                                          # the last tokens exceed the calibration range
    scale = np.float32(np.max(np.abs(xf[:3])) / 448.0)      # calibrated on the first half only
    slots = np.array([4, -1, 2, 99, 0, 5], np.int64)         # -1: padding; 99: beyond the cache
    cache = np.full((6, H, D), 0x55, np.uint8)
    ok.kv_cache_write(wl.bf16_bits_from_f32(xf), slots, H, D, cache, static_scale=scale)
    for t in (0, 2, 4, 5):
        inv = np.float32(1.0 / np.float64(scale))
        ref = torch.clamp(torch.from_numpy(xf[t]) * torch.tensor(inv), -448.0, 448.0) \
            .to(torch.float8_e4m3fn).view(torch.uint8).numpy().reshape(H, D)
        np.testing.assert_array_equal(cache[slots[t]], ref)
    assert np.all(cache[[1, 3]] == 0x55)
    big = np.abs(xf[4:]) > np.max(np.abs(xf[:3])) * (1 + 2.0 ** -4)
    assert big.any()
    stored = cache[[0, 5]].reshape(2, -1)                   # tokens 4 and 5 (slots 0 and 5)
    assert np.all((stored[big] & 0x7F) == 0x7E)             # beyond the range: saturated to +-448


def test_paged_slots_follow_the_page_table():
    B, n, bs = 4, 5, 16
    ctx = [0, 15, 31, 100]
    slots, num_slots = wl.paged_slot_mapping(B, n, ctx, bs, seed=1)
    assert len(set(slots.tolist())) == B * n and slots.max() < num_slots
    for b in range(B):
        s = slots[b * n:(b + 1) * n]
        pos = ctx[b] + np.arange(n)
        # consecutive positions inside one block take consecutive slots
        same = pos[1:] // bs == pos[:-1] // bs
        assert np.all(s[1:][same] == s[:-1][same] + 1)
        assert np.all(s % bs == pos % bs)
