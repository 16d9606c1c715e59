"""Host-side checks of the C ABI (no GPU): the library loads, exports every
symbol the header declares, and rejects bad arguments before touching HIP."""
import ctypes
import os
import re
from fractions import Fraction

import numpy as np
import pytest

import oracle
from paper_2512_02901_amd import binding

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "fairy2i.h")

# A non-null dummy device address: every call below fails validation before
# the pointer could be used.
P = ctypes.c_void_p(0x1000)


@pytest.fixture(scope="module")
def lib():
    return binding.load()


def declared_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(fairy2i_[a-z0-9_]+)\s*\(", text)))


def test_every_declared_symbol_is_exported(lib):
    names = declared_functions()
    assert len(names) >= 9
    for n in names:
        assert hasattr(lib, n), n
    assert set(names) == set(binding._SIGNATURES), "binding and header disagree"


def test_status_strings(lib):
    for s in range(8):
        assert lib.fairy2i_status_string(s)
    assert lib.fairy2i_status_string(99) == b"unknown status"
    assert lib.fairy2i_abi_version() == 5


def test_to_widely_linear_validation(lib):
    f = lib.fairy2i_to_widely_linear
    assert f(None, 4, 4, P, P, None) == binding.ERR_NULL
    assert f(P, 4, 4, None, P, None) == binding.ERR_NULL
    assert f(P, 3, 4, P, P, None) == binding.ERR_SHAPE
    assert f(P, 4, 5, P, P, None) == binding.ERR_SHAPE
    assert f(P, 0, 4, P, P, None) == binding.ERR_SHAPE
    assert f(P, -2, 4, P, P, None) == binding.ERR_SHAPE


def test_quantize_validation(lib):
    f = lib.fairy2i_quantize
    wsb = lib.fairy2i_quantize_workspace_bytes(8, 8, 2)
    assert wsb > 0
    assert f(None, 8, 8, 2, P, P, P, wsb, None) == binding.ERR_NULL
    assert f(P, 8, 6, 2, P, P, P, wsb, None) == binding.ERR_SHAPE   # K % 4
    assert f(P, 0, 8, 2, P, P, P, wsb, None) == binding.ERR_SHAPE
    assert f(P, 1 << 20, 1 << 12, 2, P, P, P, 1 << 30, None) == binding.ERR_SHAPE  # N*K > 2^31
    assert f(P, 8, 8, 0, P, P, P, wsb, None) == binding.ERR_STAGES
    assert f(P, 8, 8, 5, P, P, P, wsb, None) == binding.ERR_STAGES
    assert f(P, 8, 8, 2, P, P, None, wsb, None) == binding.ERR_WORKSPACE
    assert f(P, 8, 8, 2, P, P, P, wsb - 1, None) == binding.ERR_WORKSPACE


def test_act_quant_validation(lib):
    f = lib.fairy2i_quantize_act_int8
    assert f(None, 0, 1, 8, P, P, None) == binding.ERR_NULL
    assert f(P, 0, 0, 8, P, P, None) == binding.ERR_SHAPE
    assert f(P, 2, 1, 8, P, P, None) == binding.ERR_DTYPE
    assert f(P, 7, 1, 8, P, P, None) == binding.ERR_DTYPE


def test_wl_matmul_validation(lib):
    f = lib.fairy2i_wl_matmul
    ok = dict(cu=P, su=P, cw=P, sw=P, T=2, N=8, K=16, x=P, xs=None, dt=binding.ACT_F32, B=1, y=P)

    def call(**kw):
        a = dict(ok, **kw)
        return f(a["cu"], a["su"], a["cw"], a["sw"], a["T"], a["N"], a["K"], a["x"], a["xs"],
                 a["dt"], a["B"], a["y"], None, 0, None)
    assert call(cu=None) == binding.ERR_NULL
    assert call(sw=None) == binding.ERR_NULL
    assert call(y=None) == binding.ERR_NULL
    assert call(K=18) == binding.ERR_SHAPE
    assert call(N=0) == binding.ERR_SHAPE
    assert call(B=0) == binding.ERR_SHAPE
    assert call(T=0) == binding.ERR_STAGES
    assert call(T=5) == binding.ERR_STAGES
    assert call(dt=3) == binding.ERR_DTYPE
    assert call(B=17) == binding.ERR_UNSUPPORTED                     # float needs decode batch
    assert call(B=17, dt=binding.ACT_BF16) == binding.ERR_UNSUPPORTED
    assert call(xs=P) == binding.ERR_UNSUPPORTED                     # x_scale with float acts
    assert call(dt=binding.ACT_I8) == binding.ERR_NULL               # int8 needs x_scale
    assert lib.fairy2i_wl_matmul_workspace_bytes(8, 16, 2, 1, 0) == 0


def test_int8_accumulators_validation(lib):
    f = lib.fairy2i_wl_int8_accumulators
    assert f(None, P, 2, 8, 16, P, 1, P, None, 0, None) == binding.ERR_NULL
    assert f(P, P, 2, 8, 16, P, 1, None, None, 0, None) == binding.ERR_NULL
    assert f(P, P, 2, 8, 14, P, 1, P, None, 0, None) == binding.ERR_SHAPE
    assert f(P, P, 9, 8, 16, P, 1, P, None, 0, None) == binding.ERR_STAGES


def _host_mean(lib, v):
    v = np.ascontiguousarray(v, dtype=np.float64)
    out = ctypes.c_float(-1.0)
    st = lib.fairy2i_host_exact_mean_f32(v.ctypes.data_as(ctypes.c_void_p), v.size, ctypes.byref(out))
    assert st == binding.OK
    return np.float32(out.value)


def test_scale_rounding_matches_oracle_exact_rationals(lib):
    """The library's exact-mean rounding (the code its GPU finalize kernel
    runs, here on the host) against the oracle's rational arithmetic."""
    rng = np.random.default_rng(0)
    cases = [
        np.abs(rng.standard_normal(1000)) * 0.02,
        np.abs(rng.standard_normal(7)) * np.exp2(rng.integers(-140, 120, 7)),
        np.array([5e-324] * 3),
        np.array([1e-310, 3e-320, 7e-315]),
        np.array([1.0, 1.0 + 2.0 ** -24]),                  # exact tie -> even
        np.array([1.0 + 2.0 ** -23, 1.0 + 2.0 ** -22]),
        np.array([3.0e38, 3.4e38]),                          # near float32 max
        np.array([1e39, 1e39]),                              # overflow -> inf
        np.array([1.0e-45, 2.0e-45, 0.0]),                   # float32 subnormal result
        np.array([2.0 ** -150, 2.0 ** -150]),                # rounds to 0 (tie, even)
        np.array([2.0 ** -150 * 1.5]),                       # rounds up to the smallest subnormal
        np.abs(rng.standard_normal(5000)) * np.exp2(rng.integers(-1000, 1000, 5000)),
    ]
    for v in cases:
        got = _host_mean(lib, v)
        want = oracle.round_to_f32(oracle.exact_sum(np.abs(v)) / v.size)
        assert (np.isinf(got) and np.isinf(want)) or got == want, (v[:4], got, want)
    assert _host_mean(lib, np.zeros(0)) == 0


def test_scale_rounding_random_ties(lib):
    """Many means that land exactly on float32 rounding ties."""
    rng = np.random.default_rng(1)
    for _ in range(200):
        base = np.float32(rng.uniform(0.001, 0.1))
        ulp = float(np.nextafter(base, np.float32(1)) - base)
        n = int(rng.integers(1, 40))
        target = Fraction(float(base)) + Fraction(ulp) / 2   # exact midpoint
        vals = np.full(n, float(target), dtype=np.float64)
        assert Fraction(float(vals[0])) == target
        got = _host_mean(lib, vals)
        assert got == oracle.round_to_f32(target)


def _layer(**kw):
    d = dict(codes_U=0x1000, scales_U=0x1000, codes_W=0x1000, scales_W=0x1000, x=0x1000, x_scale=None,
             y=0x1000, N=64, K=128, layout=binding.LAYOUT_D3, group_size=0)
    d.update(kw)
    return binding.WlLayer(d["codes_U"], d["scales_U"], d["codes_W"], d["scales_W"], d["x"], d["x_scale"],
                           d["y"], d["N"], d["K"], d["layout"], d["group_size"])


def test_group_build_validation(lib):
    """fairy2i_wl_group_build_table checks every layer on the host."""
    def build(layers, T=2, dt=binding.ACT_BF16, B=1, ws=P, wsb=1 << 30, tb=None):
        arr = (binding.WlLayer * max(1, len(layers)))(*layers)
        n = len(layers)
        tbytes = lib.fairy2i_wl_group_table_bytes(max(n, 1)) if tb is None else tb
        buf = (ctypes.c_uint8 * max(1, tbytes))()
        return lib.fairy2i_wl_group_build_table(ctypes.byref(arr), n, T, dt, B, ws, wsb, ctypes.byref(buf), tbytes)
    good = [_layer(), _layer(N=200, K=1088)]
    assert build(good) == binding.OK
    assert lib.fairy2i_wl_group_workspace_bytes(ctypes.byref((binding.WlLayer * 2)(*good)), 2, 2, 1, 1) > 0
    assert build([]) == binding.ERR_SHAPE
    assert build(good, T=5) == binding.ERR_STAGES
    assert build(good, dt=7) == binding.ERR_DTYPE
    assert build(good, dt=binding.ACT_F32) == binding.ERR_UNSUPPORTED     # float32 not on the matrix cores
    assert build([_layer(K=100)]) == binding.ERR_UNSUPPORTED               # K % 64
    assert build(good, B=17) == binding.ERR_UNSUPPORTED
    assert build([_layer(codes_W=None)]) == binding.ERR_NULL
    assert build([_layer(x_scale=0x1000)]) == binding.ERR_UNSUPPORTED      # x_scale with bf16
    assert build([_layer()], dt=binding.ACT_I8) == binding.ERR_NULL        # int8 needs x_scale
    assert build(good, ws=None) == binding.ERR_WORKSPACE
    assert build(good, wsb=16) == binding.ERR_WORKSPACE
    assert build(good, tb=8) == binding.ERR_WORKSPACE
    assert build([_layer(layout=binding.LAYOUT_TILED), _layer(N=200, K=1088)]) == binding.OK
    fp4 = binding.LAYOUT_TILED_FP4
    assert build([_layer(layout=fp4), _layer(layout=fp4, N=200, K=1088)]) == binding.OK
    assert build([_layer(layout=fp4)], B=2) == binding.OK
    assert build([_layer(layout=fp4)], B=4) == binding.OK                   # one one-band tile
    assert build([_layer(layout=fp4)], B=8) == binding.OK                   # 5..8 tokens: two one-band tiles
    assert build([_layer(layout=fp4)], B=16) == binding.OK                  # 9..16 tokens: four (T <= 2)
    assert build([_layer(layout=fp4)], B=9, T=3) == binding.ERR_UNSUPPORTED
    assert build([_layer(layout=fp4)], B=17) == binding.ERR_UNSUPPORTED
    assert build([_layer(layout=fp4)], B=4, T=4) == binding.OK
    assert build([_layer(layout=fp4)], B=5, T=4) == binding.ERR_UNSUPPORTED  # two tiles need T <= 3
    assert build([_layer(layout=fp4)], B=2, T=4) == binding.OK
    assert build([_layer(layout=fp4, x_scale=0x1000)], dt=binding.ACT_I8) == binding.ERR_UNSUPPORTED
    assert build([_layer(layout=fp4), _layer()]) == binding.ERR_UNSUPPORTED  # fp4 for every layer or none
    assert build([_layer(), _layer(layout=fp4)]) == binding.ERR_UNSUPPORTED
    assert build([_layer(layout=3)]) == binding.ERR_UNSUPPORTED
    assert build([_layer(group_size=1)]) == binding.ERR_UNSUPPORTED       # not whole 256-code steps
    assert build([_layer(group_size=256)]) == binding.ERR_UNSUPPORTED     # per-group scales need fp4 codes
    assert build([_layer(group_size=-256)]) == binding.ERR_UNSUPPORTED


def test_repack_validation_and_size(lib):
    b = lib.fairy2i_repack_tiled_bytes
    assert b(16, 256, 1) == 1024
    assert b(17, 256, 2) == 2 * 2 * 1024             # 2 row blocks
    assert b(2048, 5504, 2) == 2 * 128 * 22 * 1024   # K = 5504: 21.5 steps -> 22
    assert b(0, 256, 1) == 0 and b(16, 6, 1) == 0 and b(16, 256, 5) == 0
    f = lib.fairy2i_repack_tiled
    assert f(None, 16, 256, 1, P, 1024, None) == binding.ERR_NULL
    assert f(P, 16, 256, 1, None, 1024, None) == binding.ERR_NULL
    assert f(P, 16, 258, 1, P, 1 << 20, None) == binding.ERR_SHAPE
    assert f(P, 0, 256, 1, P, 1 << 20, None) == binding.ERR_SHAPE
    assert f(P, 16, 256, 0, P, 1 << 20, None) == binding.ERR_STAGES
    assert f(P, 16, 256, 1, P, 1023, None) == binding.ERR_WORKSPACE
    f4 = lib.fairy2i_repack_tiled_fp4
    assert f4(None, 16, 256, 1, P, 1024, None) == binding.ERR_NULL
    assert f4(P, 16, 256, 1, None, 1024, None) == binding.ERR_NULL
    assert f4(P, 16, 258, 1, P, 1 << 20, None) == binding.ERR_SHAPE
    assert f4(P, 16, 256, 5, P, 1 << 20, None) == binding.ERR_STAGES
    assert f4(P, 16, 256, 1, P, 1023, None) == binding.ERR_WORKSPACE


def test_group_call_validation(lib):
    buf = (ctypes.c_uint8 * 256)()
    assert lib.fairy2i_wl_matmul_group(None, P, None) == binding.ERR_NULL
    assert lib.fairy2i_wl_matmul_group(ctypes.byref(buf), P, None) == binding.ERR_UNSUPPORTED  # not a table
    ev = (ctypes.c_void_p * 4)(0x1000, 0x1000, None, 0x1000)
    assert lib.fairy2i_wl_matmul_group_timed(ctypes.byref(buf), P, None, ev) == binding.ERR_NULL
    assert lib.fairy2i_wl_matmul_group_timed(ctypes.byref(buf), P, None, None) == binding.ERR_NULL


def test_cgemm_validation(lib):
    """Both complex GEMM entry points reject bad operands, sizes and
    workspaces before any GPU work; the planar workspace covers the three
    bf16 planes of each operand (K padded to 64), the three float32 products
    and the library's 32 MiB."""
    op = binding.CgemmOperand
    M, N, K = 70, 90, 100

    def ops(a=None, b=None):
        A = (op * 2)(op(P, K, binding.ACT_F32, 0, 0, 0), op(P, K, binding.ACT_F32, 0, 0, 0))
        B = (op * 2)(op(P, K, binding.ACT_BF16, 0, 1, 0), op(P, K, binding.ACT_BF16, 0, 1, 0))
        if a is not None:
            A[0] = a
        if b is not None:
            B[0] = b
        return A, B

    Ks = (ctypes.c_int64 * 2)(K, 36)
    for planar in (False, True):
        def call(A, B, nseg=1, m=M, n=N, C=P, ldc=N, acc=0, ws=P, wsb=1 << 40):
            if planar:
                return lib.fairy2i_cgemm_gauss_planar(ctypes.byref(A), ctypes.byref(B), ctypes.byref(Ks), nseg, m, n,
                                                      C, ldc, acc, ws, wsb, None)
            return lib.fairy2i_cgemm_gauss(ctypes.byref(A), ctypes.byref(B), ctypes.byref(Ks), nseg, m, n, C, ldc,
                                           acc, None)
        assert call(*ops(), C=None) == binding.ERR_NULL
        assert call(*ops(a=op(None, K, binding.ACT_F32, 0, 0, 0))) == binding.ERR_NULL
        assert call(*ops(), nseg=0) == binding.ERR_SHAPE
        assert call(*ops(), nseg=3) == binding.ERR_SHAPE
        assert call(*ops(), m=0) == binding.ERR_SHAPE
        assert call(*ops(), ldc=N - 1) == binding.ERR_SHAPE
        assert call(*ops(), acc=2) == binding.ERR_SHAPE
        assert call(*ops(a=op(P, K - 1, binding.ACT_F32, 0, 0, 0))) == binding.ERR_SHAPE    # ld < K
        assert call(*ops(a=op(P, M - 1, binding.ACT_F32, 1, 0, 0))) == binding.ERR_SHAPE    # ld < rows
        assert call(*ops(b=op(P, K, 7, 0, 0, 0))) == binding.ERR_SHAPE                      # dtype
        assert call(*ops(b=op(P, K, binding.ACT_F32, 0, 2, 0))) == binding.ERR_SHAPE        # conj flag
        assert call(*ops(b=op(P, K, binding.ACT_F32, 0, 0, 1))) == binding.ERR_SHAPE        # reserved
        if planar:
            assert call(*ops(), ws=None) == binding.ERR_WORKSPACE
            need = lib.fairy2i_cgemm_gauss_planar_workspace_bytes(ctypes.byref(Ks), 1, M, N)
            assert call(*ops(), wsb=need - 1) == binding.ERR_WORKSPACE
    wsb = lib.fairy2i_cgemm_gauss_planar_workspace_bytes
    a256 = lambda b: (b + 255) // 256 * 256
    Kp = 192   # 100 + 36 padded to 64
    assert wsb(ctypes.byref(Ks), 2, M, N) == (a256(3 * M * Kp * 2) + a256(3 * N * Kp * 2) + a256(3 * M * N * 4)
                                              + (32 << 20))
    assert wsb(ctypes.byref(Ks), 0, M, N) == 0
    assert wsb(ctypes.byref(Ks), 1, 0, N) == 0
    assert wsb(ctypes.byref((ctypes.c_int64 * 2)(0, 5)), 1, M, N) == 0


def test_probe_mfma_validation(lib):
    """The matrix-core rate probe rejects bad arguments before any launch and
    names the operations of a launch only when it launches."""
    ops = ctypes.c_double(-1.0)
    probe = lib.fairy2i_probe_mfma
    assert probe(binding.PROBE_MFMA_I8, 4, 8, None, ctypes.byref(ops), None) == binding.ERR_NULL
    assert probe(binding.PROBE_MFMA_I8, 4, 8, P, None, None) == binding.ERR_NULL
    assert probe(7, 4, 8, P, ctypes.byref(ops), None) == binding.ERR_UNSUPPORTED
    assert probe(binding.PROBE_MFMA_F8F4, 0, 8, P, ctypes.byref(ops), None) == binding.ERR_SHAPE
    assert probe(binding.PROBE_MFMA_F8F4, 4, 0, P, ctypes.byref(ops), None) == binding.ERR_SHAPE
    assert probe(binding.PROBE_MFMA_I8, (1 << 20) + 1, 8, P, ctypes.byref(ops), None) == binding.ERR_SHAPE
    assert ops.value == -1.0


def test_real_form_validation(lib):
    """The real-form entries reject bad arguments before any launch."""
    assert lib.fairy2i_wl_realify(None, P, binding.ACT_F32, 4, 4, P, None) == binding.ERR_NULL
    assert lib.fairy2i_wl_realify(P, P, binding.ACT_I8, 4, 4, P, None) == binding.ERR_DTYPE
    assert lib.fairy2i_wl_realify(P, P, binding.ACT_F32, 0, 4, P, None) == binding.ERR_SHAPE
    assert lib.fairy2i_wl_realify(P, P, binding.ACT_BF16, 1 << 16, 1 << 15, P, None) == binding.ERR_SHAPE
    assert lib.fairy2i_wl_unrealify_grad(P, 4, 4, None, P, None) == binding.ERR_NULL
    assert lib.fairy2i_wl_unrealify_grad(P, 4, -1, P, P, None) == binding.ERR_SHAPE
    assert lib.fairy2i_f32_to_bf16(P, 0, P, None) == binding.ERR_SHAPE
    assert lib.fairy2i_f32_to_bf16(None, 8, P, None) == binding.ERR_NULL
    wsb = lib.fairy2i_gemm_bf16_workspace_bytes()
    assert wsb >= 1 << 20

    def g(A=P, lda=64, ta=0, B=P, ldb=32, tb=0, M=16, N=32, K=64, C=P, ldc=32, ws=P, n=None):
        return lib.fairy2i_gemm_bf16(A, lda, ta, B, ldb, tb, M, N, K, C, ldc, ws, wsb if n is None else n, None)
    assert g(C=None) == binding.ERR_NULL
    assert g(ta=2) == binding.ERR_SHAPE
    assert g(M=0) == binding.ERR_SHAPE
    assert g(lda=63) == binding.ERR_SHAPE            # op(A) = A: lda >= K
    assert g(ta=1, lda=15) == binding.ERR_SHAPE      # A stored K x M: lda >= M
    assert g(ldb=31) == binding.ERR_SHAPE            # op(B) = B: ldb >= N
    assert g(tb=1, ldb=63) == binding.ERR_SHAPE      # B stored N x K: ldb >= K
    assert g(ldc=31) == binding.ERR_SHAPE
    assert g(n=wsb - 1) == binding.ERR_WORKSPACE
    assert g(ws=None) == binding.ERR_WORKSPACE
    tune = lib.fairy2i_gemm_bf16_tune
    assert tune(P, 64, 0, P, 32, 0, 16, 32, 64, None, 32, P, wsb, None, None) == binding.ERR_NULL
    assert tune(P, 63, 0, P, 32, 0, 16, 32, 64, P, 32, P, wsb, None, None) == binding.ERR_SHAPE
    assert tune(P, 64, 0, P, 32, 0, 16, 32, 64, P, 32, P, wsb - 1, None, None) == binding.ERR_WORKSPACE


def test_realify_codes_validation(lib):
    rc = lib.fairy2i_wl_realify_codes
    assert rc(None, P, P, P, 2, 4, 8, P, None) == binding.ERR_NULL
    assert rc(P, P, P, P, 0, 4, 8, P, None) == binding.ERR_STAGES
    assert rc(P, P, P, P, 5, 4, 8, P, None) == binding.ERR_STAGES
    assert rc(P, P, P, P, 2, 4, 6, P, None) == binding.ERR_SHAPE        # K % 4
    assert rc(P, P, P, P, 2, 0, 8, P, None) == binding.ERR_SHAPE
    assert rc(P, P, P, P, 2, 4, 8, ctypes.c_void_p(0x1008), None) == binding.ERR_SHAPE   # R not 16-byte aligned
