"""The C-ABI library loads, exports every symbol include/spec_fp8.h declares,
and rejects every invalid argument on the host before any HIP call (these
calls never reach a kernel, so they run without a GPU)."""

import ctypes
import os
import re

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "spec_fp8.h")

OK, NULL, SHAPE, UNSUP, ENUM, ALIGN, WS, HIP, VALUE, SCRATCH = range(10)
A16 = 0x10000            # fake, 16-byte aligned device address: never dereferenced here
A1 = 0x10001             # misaligned


@pytest.fixture(scope="module")
def lib():
    import paper_2606_18502_amd as p
    san = os.environ.get("SPECFP8_ABI_LIB")
    if san:            # the host-only build under sanitizers (tests/test_host_sanitizers.py)
        from paper_2606_18502_amd import _lib
        return _lib.declare(ctypes.CDLL(san))
    if not os.path.exists(p.LIB_PATH):
        from paper_2606_18502_amd import build
        build.build()
    return p.load_library()


def _declared():
    text = open(HEADER).read()
    return sorted(set(re.findall(r"\b(spec_[a-z0-9_]+)\s*\(", text)))


def test_exports_every_declared_symbol(lib):
    names = _declared()
    assert len(names) >= 9
    for n in names:
        assert hasattr(lib, n), n
    from paper_2606_18502_amd import _lib
    assert set(_lib.EXPORTS) == set(names)


def test_version_and_status_strings(lib):
    assert lib.spec_version() == 510
    for s in range(10):
        assert lib.spec_status_string(s)
    assert lib.spec_status_string(9) != b"unknown status"
    assert lib.spec_status_string(99) == b"unknown status"
    assert lib.spec_last_hip_error() == 0


def q(lib, x=A16, rows=4, cols=64, ld_x=64, kind=0, mode=0, scales=A16, qp=A16, ld_q=64):
    return lib.spec_fp8_quantize(x, rows, cols, ld_x, kind, mode, scales, qp, ld_q, None)


def test_quantize_validation(lib):
    assert q(lib, kind=2) == ENUM
    assert q(lib, mode=5) == ENUM
    assert q(lib, rows=-1) == SHAPE
    assert q(lib, cols=0) == SHAPE
    assert q(lib, ld_x=32) == SHAPE
    assert q(lib, kind=1, ld_x=64) == SHAPE            # SiLU input needs 2*cols
    assert q(lib, ld_q=32) == SHAPE
    assert q(lib, cols=60, ld_x=64, ld_q=64) == UNSUP  # cols % 8
    assert q(lib, x=None) == NULL
    assert q(lib, scales=None) == NULL
    assert q(lib, qp=None) == NULL
    assert q(lib, x=A1) == ALIGN
    assert q(lib, ld_x=68) == ALIGN
    assert q(lib, scales=A16 + 2) == ALIGN
    assert q(lib, rows=0, x=None, scales=None, qp=None) == OK   # empty: no-op
    # static calibration writes no codes: q and ld_q are not checked
    assert q(lib, mode=3) == ENUM
    assert q(lib, mode=2, rows=0, qp=None, ld_q=0) == OK
    assert q(lib, mode=2, x=None, qp=None, ld_q=0) == NULL
    assert q(lib, mode=2, scales=None, qp=None, ld_q=0) == NULL
    assert q(lib, mode=2, x=A1, qp=None, ld_q=0) == ALIGN
    assert q(lib, mode=2, ld_x=32, qp=None, ld_q=0) == SHAPE


def kv(lib, k=A16, ld_k=1024, v=A16, ld_v=1024, slots=A16, T=4, H=8, D=128, num_slots=64, mode=0,
       ks=A16, vs=A16, kc=A16, vc=A16):
    return lib.spec_fp8_kv_cache_write(k, ld_k, v, ld_v, slots, T, H, D, num_slots, mode, ks, vs, kc, vc, None)


def test_kv_cache_write_validation(lib):
    assert kv(lib, mode=2) == ENUM                    # calibration is spec_fp8_quantize's
    assert kv(lib, mode=7) == ENUM
    assert kv(lib, T=-1) == SHAPE
    assert kv(lib, H=0) == SHAPE
    assert kv(lib, D=0) == SHAPE
    assert kv(lib, num_slots=-1) == SHAPE
    assert kv(lib, ld_k=1016) == SHAPE                # ld < H*D
    assert kv(lib, ld_v=8) == SHAPE
    assert kv(lib, D=100, ld_k=800, ld_v=800) == UNSUP  # D % 8
    assert kv(lib, D=520, ld_k=4160, ld_v=4160) == UNSUP  # D > 512
    assert kv(lib, H=(1 << 31), D=8, ld_k=1 << 34, ld_v=1 << 34) == UNSUP
    assert kv(lib, num_slots=(1 << 62)) == UNSUP      # cache bytes beyond int64
    assert kv(lib, k=None) == NULL
    assert kv(lib, v=None) == NULL
    assert kv(lib, slots=None) == NULL
    assert kv(lib, ks=None) == NULL
    assert kv(lib, vs=None) == NULL
    assert kv(lib, kc=None) == NULL
    assert kv(lib, vc=None) == NULL
    assert kv(lib, k=A1) == ALIGN
    assert kv(lib, v=A16 + 8) == ALIGN
    assert kv(lib, ld_k=1028) == ALIGN
    assert kv(lib, kc=A16 + 8) == ALIGN
    assert kv(lib, slots=A16 + 4) == ALIGN
    assert kv(lib, ks=A16 + 2) == ALIGN
    assert kv(lib, T=0, k=None, v=None, slots=None, ks=None, vs=None, kc=None, vc=None) == OK  # no-op
    assert kv(lib, num_slots=0) == OK                 # every token skipped: nothing enqueued


def test_tree_mask_validation(lib):
    f = lib.spec_tree_attention_mask
    assert f(A16, -1, 5, A16, A16, None) == SHAPE
    assert f(A16, 4, 0, A16, A16, None) == SHAPE
    assert f(A16, 4, 65, A16, A16, None) == UNSUP
    assert f(A16, 1 << 40, 5, A16, A16, None) == UNSUP
    assert f(None, 4, 5, A16, A16, None) == NULL
    assert f(A16, 4, 5, None, A16, None) == NULL
    assert f(A16, 4, 5, A16, None, None) == NULL
    assert f(A16 + 2, 4, 5, A16, A16, None) == ALIGN
    assert f(A16, 4, 5, A16 + 4, A16, None) == ALIGN
    assert f(A16, 4, 5, A16, A16 + 2, None) == ALIGN
    assert f(None, 0, 5, None, None, None) == OK


def test_clip_count_validation(lib):
    f = lib.spec_fp8_clip_count
    assert f(A16, -1, 64, 64, A16, A16, None) == SHAPE
    assert f(A16, 4, 0, 64, A16, A16, None) == SHAPE
    assert f(A16, 4, 64, 32, A16, A16, None) == SHAPE
    assert f(A16, 4, 60, 64, A16, A16, None) == UNSUP
    assert f(None, 4, 64, 64, A16, A16, None) == NULL
    assert f(A16, 4, 64, 64, None, A16, None) == NULL
    assert f(A16, 4, 64, 64, A16, None, None) == NULL
    assert f(A1, 4, 64, 64, A16, A16, None) == ALIGN
    assert f(A16, 4, 64, 68, A16, A16, None) == ALIGN
    assert f(A16, 4, 64, 64, A16 + 2, A16, None) == ALIGN
    assert f(A16, 4, 64, 64, A16, A16 + 4, None) == ALIGN
    assert f(None, 0, 64, 64, None, None, None) == OK


def test_silu_mul_validation(lib):
    f = lib.spec_silu_mul_bf16
    assert f(A16, 4, 64, 64, A16, 64, None) == SHAPE          # ld_x < 2*cols
    assert f(A16, 4, 60, 120, A16, 64, None) == UNSUP
    assert f(None, 4, 64, 128, A16, 64, None) == NULL
    assert f(A1, 4, 64, 128, A16, 64, None) == ALIGN
    assert f(None, 0, 64, 128, None, 64, None) == OK


def g(lib, a=A16, lda=512, sa=A16, am=0, w=A16, ldw=512, sw=A16, wm=0, M=8, N=1024, K=512,
      y=A16, ldy=1024, od=0, ws=None, wsb=0):
    return lib.spec_fp8_gemm(a, lda, sa, am, w, ldw, sw, wm, M, N, K, y, ldy, od, ws, wsb, None)


def test_gemm_validation(lib):
    assert g(lib, am=3) == ENUM
    assert g(lib, am=2) == ENUM        # calibration is a quantize mode only
    assert g(lib, wm=2) == ENUM
    assert g(lib, wm=-1) == ENUM
    assert g(lib, od=7) == ENUM
    assert g(lib, M=-1) == SHAPE
    assert g(lib, N=0) == SHAPE
    assert g(lib, K=0) == SHAPE
    assert g(lib, lda=256) == SHAPE
    assert g(lib, ldy=512) == SHAPE
    assert g(lib, K=500, lda=512, ldw=512) == UNSUP
    assert g(lib, a=None) == NULL
    assert g(lib, sw=None) == NULL
    assert g(lib, y=None) == NULL
    assert g(lib, a=A1) == ALIGN
    assert g(lib, lda=520) == ALIGN
    assert g(lib, ldy=1028) == ALIGN
    assert g(lib, M=0, a=None, sa=None, w=None, sw=None, y=None) == OK
    # a shape that splits K needs a workspace
    need = lib.spec_fp8_gemm_workspace_bytes(320, 1024, 4096)
    assert need > 0
    assert g(lib, M=320, N=1024, K=4096, lda=4096, ldw=4096, ldy=1024) == WS
    assert g(lib, M=320, N=1024, K=4096, lda=4096, ldw=4096, ldy=1024, ws=A16, wsb=need - 1) == WS
    assert g(lib, M=320, N=1024, K=4096, lda=4096, ldw=4096, ldy=1024, ws=A1, wsb=need) == ALIGN
    assert lib.spec_fp8_gemm_workspace_bytes(8, 1024, 100) == 0
    # more output tiles than an int grid holds
    big = (1 << 31) - 1
    assert g(lib, M=big, N=big, K=128, lda=128, ldw=128, ldy=big + 1) == UNSUP


def acc(lib, zt=A16, zd=A16, x=A16, u=A16, B=2, k=3, V=256, T=0.7, out=A16, num=A16, ws=A16, wsb=1 << 20):
    return lib.spec_verify_accept(zt, zd, x, u, B, k, V, ctypes.c_float(T), out, num, ws, wsb, None)


def test_accept_validation(lib):
    assert acc(lib, T=float("nan")) == VALUE
    assert acc(lib, T=-0.5) == VALUE
    assert acc(lib, T=float("inf")) == VALUE
    assert acc(lib, k=0) == SHAPE
    assert acc(lib, B=-1) == SHAPE
    assert acc(lib, V=0) == SHAPE
    assert acc(lib, k=17) == UNSUP
    assert acc(lib, V=1 << 31) == UNSUP
    assert acc(lib, V=(1 << 22) + 8) == UNSUP
    assert acc(lib, V=1 << 22, ws=None) == WS        # the largest V passes the shape checks
    assert acc(lib, B=20000, k=4) == UNSUP
    assert acc(lib, zt=None) == NULL
    assert acc(lib, x=None) == NULL
    assert acc(lib, u=None) == NULL                 # T > 0 needs uniforms
    assert acc(lib, zt=A1) == ALIGN
    assert acc(lib, num=A16 + 2) == ALIGN
    need = lib.spec_verify_accept_workspace_bytes(2, 3, 256)
    assert need > 0
    assert acc(lib, ws=None) == WS
    assert acc(lib, wsb=need - 1) == WS
    assert acc(lib, ws=A16 + 8, wsb=need) == ALIGN
    assert acc(lib, B=0, zt=None, zd=None, x=None, u=None, out=None, num=None, ws=None, wsb=0) == OK


def accn(lib, zt=A16, zd=A16, x=A16, u=A16, B=2, k=3, V=256, T=0.7, out=A16, num=A16):
    return lib.spec_verify_accept_noalloc(zt, zd, x, u, B, k, V, ctypes.c_float(T), out, num, None)


def test_accept_noalloc_validation(lib):
    # the argument checks of spec_verify_accept, before any HIP call
    assert accn(lib, T=float("nan")) == VALUE
    assert accn(lib, k=0) == SHAPE
    assert accn(lib, k=17) == UNSUP
    assert accn(lib, zt=None) == NULL
    assert accn(lib, u=None) == NULL
    assert accn(lib, zt=A1) == ALIGN
    assert accn(lib, B=0, zt=None, zd=None, x=None, u=None, out=None, num=None) == OK
    # then the fixed scratch's size: the C4 workload fits, a call needing more is refused
    from paper_2606_18502_amd import _lib
    limit = _lib.ACCEPT_SCRATCH_BYTES
    assert lib.spec_verify_accept_workspace_bytes(64, 4, 128256) <= limit
    assert lib.spec_verify_accept_workspace_bytes(64, 4, 1 << 22) > limit
    assert accn(lib, B=64, k=4, V=1 << 22) == SCRATCH
    assert accn(lib, B=64, k=4, V=1 << 22, T=0.0, u=None) == SCRATCH


def test_workspace_sizes_grow_with_problem(lib):
    assert lib.spec_verify_accept_workspace_bytes(64, 4, 128256) > lib.spec_verify_accept_workspace_bytes(2, 3, 256)
    assert lib.spec_verify_accept_workspace_bytes(0, 3, 256) == 0
    assert lib.spec_fp8_gemm_workspace_bytes(4096, 14336, 4096) == 0     # enough tiles: no split


def ls(lib, a=A16, lda=512, sa=A16, am=0, w=A16, ldw=512, sw=A16, wm=0, M=8, V=1024, K=512, T=0.7,
       y=A16, ldy=1024, st=A16, ldst=None):
    if ldst is None:
        ldst = lib.spec_logit_stats_count(M, V, K)
    return lib.spec_fp8_gemm_logit_stats(a, lda, sa, am, w, ldw, sw, wm, M, V, K, ctypes.c_float(T), y, ldy, st,
                                         ldst, None)


def test_logit_stats_gemm_validation(lib):
    G = lib.spec_logit_stats_count(8, 1024, 512)
    assert G >= 1
    assert lib.spec_logit_stats_count(320, 128256, 4096) >= 128256 // 224      # one group per wave column
    assert lib.spec_logit_stats_count(8, 1024, 100) == 0                         # K % 128
    assert lib.spec_logit_stats_count(0, 1024, 512) == 0
    # the GEMM operand checks come first and are those of spec_fp8_gemm
    assert ls(lib, am=2) == ENUM
    assert ls(lib, K=500, lda=512, ldw=512) == UNSUP
    assert ls(lib, ldy=512) == SHAPE
    assert ls(lib, a=None) == NULL
    assert ls(lib, ldy=1028) == ALIGN
    # then the statistics' own
    assert ls(lib, T=float("nan")) == VALUE
    assert ls(lib, T=-1.0) == VALUE
    assert ls(lib, ldst=G - 1) == SHAPE
    assert ls(lib, st=None) == NULL
    assert ls(lib, st=A16 + 4) == ALIGN
    assert ls(lib, M=0, a=None, sa=None, w=None, sw=None, y=None, st=None, ldst=G) == OK
    # the LM head's 160 x 384 tile addresses a tile's operand rows with 32-bit
    # offsets: 159 lda + 128 and 383 ldw + 128 must not exceed 2^32
    lm = dict(M=320, V=128256, K=4096, ldy=128256)
    assert ls(lib, lda=1 << 25, ldw=4096, **lm) == UNSUP
    assert ls(lib, lda=4096, ldw=1 << 24, **lm) == UNSUP


def accs(lib, zt=A16, ts=A16, n=4, ldn=4, zd=A16, x=A16, u=A16, B=2, k=3, V=256, T=0.7, out=A16, num=A16, ws=A16,
         wsb=1 << 20):
    return lib.spec_verify_accept_stats(zt, ts, n, ldn, zd, x, u, B, k, V, ctypes.c_float(T), out, num, ws, wsb, None)


def test_accept_stats_validation(lib):
    # the checks of spec_verify_accept come first
    assert accs(lib, T=-0.5) == VALUE
    assert accs(lib, k=0) == SHAPE
    assert accs(lib, zt=None) == NULL
    # then the target statistics
    assert accs(lib, n=0) == SHAPE
    assert accs(lib, n=5, ldn=4) == SHAPE
    assert accs(lib, n=1 << 31, ldn=1 << 31) == UNSUP
    assert accs(lib, ts=None) == NULL
    assert accs(lib, ts=A16 + 4) == ALIGN
    assert accs(lib, ws=None) == WS
    assert accs(lib, B=0, zt=None, ts=None, zd=None, x=None, u=None, out=None, num=None, ws=None, wsb=0) == OK
    assert accs(lib, T=0.0, u=None, zd=None, ws=None) == WS             # greedy: no uniforms, no draft logits


def tr(lib, zt=A16, par=A16, tok=A16, u=A16, B=2, N=5, V=256, T=0.7, out=A16, nodes=A16, num=A16, ws=A16,
       wsb=1 << 20):
    return lib.spec_verify_accept_tree(zt, par, tok, u, B, N, V, ctypes.c_float(T), out, nodes, num, ws, wsb, None)


def test_accept_tree_validation(lib):
    assert tr(lib, T=float("nan")) == VALUE
    assert tr(lib, T=-1.0) == VALUE
    assert tr(lib, N=0) == SHAPE
    assert tr(lib, B=-1) == SHAPE
    assert tr(lib, V=0) == SHAPE
    assert tr(lib, N=65) == UNSUP
    assert tr(lib, V=(1 << 22) + 8) == UNSUP
    assert tr(lib, B=70000) == UNSUP
    assert tr(lib, B=65535, N=64, V=1 << 22) == UNSUP      # more than 2^31 streaming items
    assert tr(lib, B=1000, N=64, V=1 << 22, ws=None) == WS   # within the item limit
    assert tr(lib, par=None) == NULL
    assert tr(lib, tok=None) == NULL
    assert tr(lib, nodes=None) == NULL
    assert tr(lib, u=None) == NULL                  # T > 0 needs uniforms
    assert tr(lib, T=0.0, u=None, ws=None) == WS     # greedy needs none
    assert tr(lib, zt=A1) == ALIGN
    assert tr(lib, par=A16 + 2) == ALIGN
    need = lib.spec_verify_accept_tree_workspace_bytes(2, 5, 256)
    assert need > 0
    assert tr(lib, wsb=need - 1) == WS
    assert tr(lib, ws=A16 + 8, wsb=need) == ALIGN
    assert tr(lib, B=0, zt=None, par=None, tok=None, u=None, out=None, nodes=None, num=None, ws=None, wsb=0) == OK


def gs(lib, a=A16, lda=512, sa=A16, am=0, w=A16, ldw=512, sw=A16, wm=0, M=8, I=512, K=512, h=A16, ldh=512):
    return lib.spec_fp8_gemm_silu_mul(a, lda, sa, am, w, ldw, sw, wm, M, I, K, h, ldh, None)


def test_gemm_silu_mul_validation(lib):
    assert gs(lib, I=0) == SHAPE
    assert gs(lib, I=36, ldh=40) == UNSUP           # I % 8
    assert gs(lib, ldh=256) == SHAPE                # ldh < I
    assert gs(lib, am=2) == ENUM
    assert gs(lib, K=500) == UNSUP
    assert gs(lib, a=None) == NULL
    assert gs(lib, h=None) == NULL
    assert gs(lib, h=A1) == ALIGN
    assert gs(lib, ldh=516) == ALIGN
    assert gs(lib, M=0, a=None, sa=None, w=None, sw=None, h=None) == OK
