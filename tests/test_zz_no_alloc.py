"""spec_verify_accept_noalloc (the acceptance on the library's fixed device
scratch, for callers that cannot allocate) against spec_verify_accept (the
caller's workspace): the same kernels on the same inputs, so the results
must be identical bit for bit.  Two calls in a row on the shared scratch,
the second on a smaller problem, for greedy and speculative sampling with
and without draft logits."""

import numpy as np
import pytest
import torch

import workloads as wl
from tests.gpu_util import dev_bf16, dev_f32, dev_i32, host, need_gpu, say

pytestmark = pytest.mark.gpu


def _case(B, k, V, seed, T, with_draft):
    zt, zd = wl.accept_logits(B, k, V, seed, 0.99, scale=3.0)
    x = wl.draft_tokens_sampled(zd, T if T > 0 else 0.7, seed=seed + 1)
    u = wl.philox_uniforms((B, k + 1), seed=seed + 2)
    return (dev_bf16(zt), dev_bf16(zd) if with_draft else None, dev_i32(x),
            dev_f32(u) if T > 0 else None)


@pytest.mark.parametrize("T,with_draft", [(0.7, True), (0.7, False), (0.0, False)])
def test_noalloc_equals_workspace_entry_point(T, with_draft):
    p = need_gpu()
    for (B, k, V, seed) in [(64, 4, 128256, 7), (5, 2, 20000, 3)]:      # the second call is smaller
        say(f"noalloc T={T} draft_logits={with_draft} B={B} k={k} V={V}")
        zt, zd, x, u = _case(B, k, V, seed, T, with_draft)
        out_n = torch.full((B, k + 1), -7, dtype=torch.int32, device="cuda")
        num_n = torch.full((B,), -7, dtype=torch.int32, device="cuda")
        p.verify_accept_noalloc(zt, zd, x, u, T, out_n, num_n)
        out_w, num_w = p.verify_accept(zt, zd, x, u, T)
        np.testing.assert_array_equal(host(out_n), host(out_w))
        np.testing.assert_array_equal(host(num_n), host(num_w))
        assert np.all(host(num_n) >= 0)


def test_noalloc_refuses_calls_beyond_the_scratch():
    p = need_gpu()
    from paper_2606_18502_amd import _lib
    B, k, V = 64, 4, 1 << 22
    assert p.accept_workspace_bytes(B, k, V) > _lib.ACCEPT_SCRATCH_BYTES
    zt = torch.zeros((B, k + 1, V), dtype=torch.bfloat16, device="cuda")
    x = torch.zeros((B, k), dtype=torch.int32, device="cuda")
    out = torch.empty((B, k + 1), dtype=torch.int32, device="cuda")
    num = torch.empty((B,), dtype=torch.int32, device="cuda")
    with pytest.raises(_lib.SpecError) as e:
        p.verify_accept_noalloc(zt, None, x, None, 0.0, out, num)
    assert e.value.status == 9
