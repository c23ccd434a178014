"""The seeded generators are deterministic and have the stated distributions."""

import numpy as np

import workloads as wl


def test_generators_are_deterministic():
    a = wl.linear_activations(8, 512, seed=0, outlier_frac=0.01, outlier_scale=20.0)
    b = wl.linear_activations(8, 512, seed=0, outlier_frac=0.01, outlier_scale=20.0)
    np.testing.assert_array_equal(a, b)
    zt1, zd1 = wl.accept_logits(2, 3, 256, seed=0, c=0.5, scale=2.0)
    zt2, zd2 = wl.accept_logits(2, 3, 256, seed=0, c=0.5, scale=2.0)
    np.testing.assert_array_equal(zt1, zt2)
    np.testing.assert_array_equal(zd1, zd2)
    np.testing.assert_array_equal(wl.philox_uniforms((2, 4), 7), wl.philox_uniforms((2, 4), 7))


def test_outlier_channels():
    x = wl.f32_from_bf16_bits(wl.linear_activations(2048, 1000, seed=3, outlier_frac=0.01,
                                                    outlier_scale=20.0))
    std = x.std(axis=0)
    big = std > 5
    assert big.sum() == 10
    assert np.allclose(std[big].mean(), 20.0, rtol=0.1)
    assert np.allclose(std[~big].mean(), 1.0, rtol=0.05)


def test_accept_logits_marginals_and_correlation():
    zt, zd = wl.accept_logits(64, 2, 4000, seed=1, c=0.8, scale=3.0)
    t = wl.f32_from_bf16_bits(zt)
    d = wl.f32_from_bf16_bits(zd)
    assert abs(t.std() - 3.0) < 0.2
    r = np.corrcoef(t[:, :2].ravel(), d.ravel())[0, 1]
    assert abs(r - 0.64) < 0.06                     # corr = c^2 (Var S = 1 on average)


def test_sampled_drafts_follow_softmax():
    V = 6
    z = np.log(np.array([0.05, 0.1, 0.15, 0.2, 0.2, 0.3], np.float32))
    zb = wl.bf16_bits_from_f32(np.tile(z, (20000, 1, 1)))
    x = wl.draft_tokens_sampled(zb, 1.0, seed=2).ravel()
    freq = np.bincount(x, minlength=V) / len(x)
    p = np.exp(wl.f32_from_bf16_bits(wl.bf16_bits_from_f32(z)).astype(np.float64))
    p /= p.sum()
    assert np.max(np.abs(freq - p)) < 0.015


def test_fp8_code_bytes_cover_every_non_nan_pattern():
    c = wl.fp8_code_bytes(600, 512, seed=9)
    assert c.dtype == np.uint8 and c.shape == (600, 512)
    vals = np.unique(c)
    assert len(vals) == 254 and 0x7F not in vals and 0xFF not in vals
    np.testing.assert_array_equal(c, wl.fp8_code_bytes(600, 512, seed=9))
    assert not np.array_equal(c, wl.fp8_code_bytes(600, 512, seed=10))


def test_uniform_scales_range_and_determinism():
    s = wl.uniform_scales(1000, seed=4)
    assert s.dtype == np.float32 and np.all(s >= 1e-3) and np.all(s < 2e-3)
    np.testing.assert_array_equal(s, wl.uniform_scales(1000, seed=4))
