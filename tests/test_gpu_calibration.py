"""GPU parity of spec_fp8_clip_count and of the static-calibration study
workflow (calibrate on L tokens, count the clipped values of a test set)
against the oracle."""

import numpy as np
import pytest
import torch

import workloads as wl
from oracle import quantize as oq
from tests.gpu_util import dev_bf16, dev_f32, host, need_gpu, say

pytestmark = pytest.mark.gpu


@pytest.mark.parametrize("rows,cols,seed", [(1, 8, 0), (37, 1000, 1), (300, 4096, 2), (5, 14336, 3)])
def test_clip_count_bit_exact(rows, cols, seed):
    p = need_gpu()
    say(f"clip count rows={rows} cols={cols}")
    xb = wl.student_t_activations(rows, cols, seed, df=3.0)
    x = dev_bf16(xb)
    amax = float(np.max(np.abs(oq.bf16_to_f32(xb))))
    for frac in (1.0, 0.5, 0.1, 0.01):
        s = np.float32(amax * frac / 448.0)
        got = int(host(p.clip_count(x, dev_f32([s])))[0])
        assert got == oq.clip_count_static(xb, s), frac
    # strided rows: a column window of a wider tensor; the counter accumulates over calls
    wide = dev_bf16(wl.student_t_activations(rows, cols + 24, seed + 7, df=3.0))
    view = wide[:, 8:8 + cols]
    s = np.float32(amax * 0.2 / 448.0)
    cnt = p.clip_count(view, dev_f32([s]))
    p.clip_count(view, dev_f32([s]), count=cnt)
    ref = oq.clip_count_static(host(view.contiguous().view(torch.int16)).view(np.uint16), s)
    assert int(host(cnt)[0]) == 2 * ref


def test_calibration_study_workflow_small():
    """Device calibration over L tokens of each synthetic set, then the clip
    count of an in-domain-like test set, equal to the oracle at every L."""
    p = need_gpu()
    c = wl.CONFIGS["CALSTUDY"]
    K, test_tokens = 512, 1024
    test = wl.student_t_activations(test_tokens, K, c["seed"] + 100, c["indomain_df"])
    dtest = dev_bf16(test)
    for L in (32, 256):
        sets = wl.calibration_sets(L, K, c["seed"], c["public_outlier_frac"], c["public_outlier_scale"],
                                   c["indomain_df"])
        for name, cal in sets.items():
            run = torch.zeros(1, dtype=torch.float32, device="cuda")
            p.calibrate(dev_bf16(cal), run)
            s_ref = oq.calibrate_per_tensor([cal])
            assert host(run)[0] == s_ref, (L, name)
            got = int(host(p.clip_count(dtest, run))[0])
            assert got == oq.clip_count_static(test, s_ref), (L, name)
            say(f"  L={L} {name}: clip rate {got / test.size:.3e}")
