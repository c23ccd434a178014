"""C5, the long-prompt prefill / calibration workload, at full size (M=4096).

The paper's own FP8 scheme is static: one per-tensor activation scale from a
min-max calibration pass (section 3.2, FP8 Post-Training Quantization; the
calibration study of section 5).  Here the two FFN GEMMs of the target model
(4096 -> 14336 and 14336 -> 4096) run on a held-out batch of 4096 heavy-tailed
Student-t(3) activation rows, once with the static scale calibrated on 32
seeded batches and once with dynamic per-token scales.  Checked against the
oracle:
  * the calibrated scale, bit-exactly (device: spec_fp8_quantize CALIBRATE);
  * the codes of sampled rows of the held-out batch, static and dynamic,
    bit-exactly;
  * sampled GEMM outputs of both schemes, to the 2e-3 tolerance and the
    device's accumulation bound.
The paper's calibration metric (clip rate of the held-out batch against the
calibrated range) and the error of each scheme against the bf16 product are
printed.
"""

import numpy as np
import pytest
import torch

import workloads as wl
from oracle import gemm as og, quantize as oq
from tests.fp8_mfma_model import error_bound
from tests.gpu_util import dev_bf16, host, need_gpu, say

pytestmark = pytest.mark.gpu

TOL = 2e-3
CAL_ROWS = 64      # 32 batches x 64 rows = 2048 calibration tokens (the paper's largest calibration length)


@pytest.mark.parametrize("name", ["up", "down"])
def test_c5_static_vs_dynamic_full_size(name):
    p = need_gpu()
    c = wl.CONFIGS["C5"]
    M = c["M"]
    K, N = (c["K1"], c["N1"]) if name == "up" else (c["K2"], c["N2"])
    seed = c["seed"] + (0 if name == "up" else 500)
    say(f"C5 {name}: M={M} K={K} N={N}, {c['n_calib']} calibration batches of {CAL_ROWS} rows")

    # static min-max calibration over the seeded batches
    batches = [wl.student_t_activations(CAL_ROWS, K, seed + 1 + i, c["df"]) for i in range(c["n_calib"])]
    running = torch.zeros(1, dtype=torch.float32, device="cuda")
    for xb in batches:
        p.calibrate(dev_bf16(xb), running)
    s_static = host(running)[0]
    s_ref = oq.calibrate_per_tensor(batches)
    assert s_static.tobytes() == np.float32(s_ref).tobytes(), (s_static, s_ref)
    lo, hi = oq.calibrate_minmax(batches)
    del batches

    # held-out batch, static and dynamic quantization
    xb = wl.student_t_activations(M, K, seed, c["df"])
    x = dev_bf16(xb)
    a_st, _ = p.quantize(x, per_tensor_scale=running)
    a_dy, sa_dy = p.quantize(x)
    wb = wl.linear_weights(N, K, seed + 99, c["w_std"])
    wt = dev_bf16(wb)
    w, sw = p.quantize(wt)
    del wt
    y_st = host(p.gemm(a_st, running, w, sw, out_dtype=torch.float32))
    y_dy = host(p.gemm(a_dy, sa_dy, w, sw, out_dtype=torch.float32))

    rng = np.random.default_rng(seed)
    rows = np.unique(np.concatenate([[0, M - 1], rng.choice(M, 6, replace=False)]))
    cols = np.unique(np.concatenate([[0, N - 1], rng.choice(N, 128, replace=False)]))
    qst_ref = oq.quantize_per_tensor(xb[rows], s_ref)
    qdy_ref, sdy_ref = oq.quantize_rows(xb[rows])
    qw_ref, sw_ref = oq.quantize_rows(wb[cols])
    np.testing.assert_array_equal(host(a_st)[rows], qst_ref)
    np.testing.assert_array_equal(host(a_dy)[rows], qdy_ref)
    np.testing.assert_array_equal(host(sa_dy)[rows], sdy_ref)
    np.testing.assert_array_equal(host(w)[cols], qw_ref)
    np.testing.assert_array_equal(host(sw)[cols], sw_ref)

    r_idx, c_idx = np.arange(len(rows)), np.arange(len(cols))
    sst = np.full(len(rows), s_ref, np.float32)
    for label, y, qa, sa in (("static", y_st, qst_ref, sst), ("dynamic", y_dy, qdy_ref, sdy_ref)):
        y_ref = og.gemm(qa, sa, qw_ref, sw_ref)
        err = og.rel_error(y[np.ix_(rows, cols)], y_ref)
        assert err <= TOL, (label, err)
        bound = error_bound(qa, sa, qw_ref, sw_ref, r_idx, c_idx)
        assert np.all(np.abs(y[np.ix_(rows, cols)] - y_ref) <= bound), label

    # the paper's calibration metric and the end-to-end error of each scheme
    clip = oq.clip_rate(xb, lo, hi)
    xf = oq.bf16_to_f32(xb[rows]).astype(np.float64)
    wf = oq.bf16_to_f32(wb[cols]).astype(np.float64)
    y_bf16 = xf @ wf.T
    e_st = og.rel_error(y_st[np.ix_(rows, cols)], y_bf16)
    e_dy = og.rel_error(y_dy[np.ix_(rows, cols)], y_bf16)
    say(f"C5 {name}: static scale {float(s_ref):.6g}, clip rate {clip:.3e}; rel error vs bf16 product: "
        f"static {e_st:.3e}, dynamic {e_dy:.3e}")
    # both schemes keep the FP8 GEMM close to the bf16 product; a held-out
    # batch of heavy-tailed activations only rarely leaves the calibrated range
    assert clip < 1e-3
    assert e_st < 0.1 and e_dy < 0.1
