"""The CPU table-lookup kernel (Sec. 3.4, lookup tables for CPU inference)
against the oracle.  Host code only: these tests run without a GPU.

Bar: the int32 axis sums are exact, so they must equal the oracle's
integer products (``int8_accumulators``) bit for bit; y is the oracle's
combine of those sums (``combine_accumulators``, float64) rounded once to
complex64, and within 1e-6 of the full-precision product
``wl_matmul_int8``."""
import numpy as np
import pytest

from oracle import fairy2i as O

f2 = pytest.importorskip("paper_2512_02901_amd")


@pytest.fixture(scope="module")
def lib():
    from paper_2512_02901_amd import binding
    try:
        return binding.load()
    except (RuntimeError, OSError) as e:  # not built in this checkout
        pytest.skip(str(e))


def _case(rng, T, N, K, B, q=None):
    codes_U = rng.integers(0, 4, (T, N, K))
    codes_W = rng.integers(0, 4, (T, N, K))
    su = (rng.random((T, 2)) + 0.01).astype(np.float32)
    sw = (rng.random((T, 2)) + 0.01).astype(np.float32)
    if q is None:
        q = rng.integers(-127, 128, (B, K, 2)).astype(np.int8)
    f = (rng.random(B) + 0.01).astype(np.float32)
    return codes_U, su, codes_W, sw, q, f


def _check(codes_U, su, codes_W, sw, q, f, threads=0):
    cu, cw = O.pack(codes_U), O.pack(codes_W)
    y, acc = f2.cpu_lut_wl_matmul(cu, su, cw, sw, q, f, want_acc=True, threads=threads)
    P = O.int8_accumulators(codes_U, codes_W, q)
    np.testing.assert_array_equal(acc, P)
    y_comb = O.combine_accumulators(P, su, sw, f)
    np.testing.assert_array_equal(y, y_comb.astype(np.complex64))
    y_ref = O.wl_matmul_int8(codes_U, su, codes_W, sw, q, f)
    err = np.linalg.norm(y - y_ref) / max(np.linalg.norm(y_ref), 1e-30)
    assert err <= 1e-6, err
    return y, acc


# shapes span one group (K = 4), row chunks with a ragged tail (N % 32),
# table windows and int16 flush blocks with ragged tails (K / 4 % 32), every
# T and odd / even / maximal B
@pytest.mark.parametrize("T,N,K,B", [
    (1, 1, 4, 1), (1, 5, 12, 1), (2, 37, 260, 1), (2, 64, 2048, 2), (3, 33, 516, 3),
    (4, 17, 1024, 16), (2, 100, 5504, 5), (2, 65, 4100, 1), (3, 31, 132, 7), (1, 96, 8192, 1),
])
def test_lut_matches_oracle(lib, T, N, K, B):
    rng = np.random.default_rng(1000 * T + N + K + B)
    _check(*_case(rng, T, N, K, B))


def test_lut_extreme_activations(lib):
    """Every code equal and every activation at the int8 extremes: the
    largest sums a table entry (4 * 128) and a flush block can hold."""
    T, N, K, B = 2, 8, 5504, 2
    rng = np.random.default_rng(7)
    for code in range(4):
        codes = np.full((T, N, K), code)
        for val in (-128, 127):
            q = np.full((B, K, 2), val, dtype=np.int8)
            q[1, :, 1] = -128 if val == 127 else 127
            _, su, _, sw, _, f = _case(rng, T, N, K, B, q=q)
            _check(codes, su, codes, sw, q, f)


def test_lut_zero_tokens(lib):
    rng = np.random.default_rng(8)
    codes_U, su, codes_W, sw, _, f = _case(rng, 2, 40, 256, 3)
    q = np.zeros((3, 256, 2), dtype=np.int8)
    y, acc = _check(codes_U, su, codes_W, sw, q, f)
    assert not np.any(acc) and not np.any(y)


def test_lut_thread_count_does_not_change_results(lib):
    rng = np.random.default_rng(9)
    codes_U, su, codes_W, sw, q, f = _case(rng, 2, 300, 1028, 4)
    cu, cw = O.pack(codes_U), O.pack(codes_W)
    outs = [f2.cpu_lut_wl_matmul(cu, su, cw, sw, q, f, want_acc=True, threads=n) for n in (1, 3, 0, 2)]
    for y, acc in outs[1:]:
        np.testing.assert_array_equal(y, outs[0][0])
        np.testing.assert_array_equal(acc, outs[0][1])


def test_lut_quantised_llama_layer(lib):
    """A quantised LLaMA-shaped layer (Student-t weights with outlier
    columns, the oracle's quantiser) at the q-projection width, with the
    int8 token of an N(0,1) bf16-like activation."""
    import synth
    rng = np.random.default_rng(11)
    A = synth.llama_weight(512, 4096, (11,))
    U, W = O.to_widely_linear(A)
    T = 2
    codes_U, su = O.quantize(U.astype(np.complex128), T)
    codes_W, sw = O.quantize(W.astype(np.complex128), T)
    x = rng.standard_normal((1, 2048)) + 1j * rng.standard_normal((1, 2048))
    q, f = O.quantize_act_int8(x)
    _check(codes_U, su, codes_W, sw, q, f)


@pytest.mark.slow
def test_lut_full_q_shape(lib):
    """The full q-projection layer (complex 2048 x 2048, T = 2, B = 1)."""
    rng = np.random.default_rng(12)
    _check(*_case(rng, 2, 2048, 2048, 1))


def test_lut_workspace_reuse_and_errors(lib):
    rng = np.random.default_rng(13)
    codes_U, su, codes_W, sw, q, f = _case(rng, 2, 16, 64, 1)
    cu, cw = O.pack(codes_U), O.pack(codes_W)
    ws = np.empty(f2.cpu_lut_workspace_bytes(2, 64, 1), dtype=np.uint8)
    y1, _ = f2.cpu_lut_wl_matmul(cu, su, cw, sw, q, f, workspace=ws)
    y2, _ = f2.cpu_lut_wl_matmul(cu, su, cw, sw, q, f, workspace=ws)
    np.testing.assert_array_equal(y1, y2)
    assert f2.cpu_lut_workspace_bytes(2, 66, 1) == 0          # K % 4 != 0
    assert f2.cpu_lut_workspace_bytes(5, 64, 1) == 0          # T > 4
    assert f2.cpu_lut_workspace_bytes(2, 64, 17) == 0         # B > 16
    assert f2.cpu_lut_workspace_bytes(2, 64, 16) > f2.cpu_lut_workspace_bytes(2, 64, 1)


def test_lut_abi_validation(lib):
    import ctypes
    from paper_2512_02901_amd import binding
    b = np.zeros(64, dtype=np.uint8)
    p = b.ctypes.data_as(ctypes.c_void_p)
    need = lib.fairy2i_cpu_lut_workspace_bytes(1, 16, 1, 1)
    ws = np.zeros(need, dtype=np.uint8)
    w = ws.ctypes.data_as(ctypes.c_void_p)
    call = lib.fairy2i_cpu_lut_wl_matmul
    # no output at all
    assert call(p, p, p, p, 1, 4, 16, p, p, 1, None, None, w, need, 1) == binding.ERR_NULL
    # y without scales
    assert call(p, None, p, p, 1, 4, 16, p, p, 1, p, None, w, need, 1) == binding.ERR_NULL
    assert call(p, p, p, p, 0, 4, 16, p, p, 1, p, None, w, need, 1) == binding.ERR_STAGES
    assert call(p, p, p, p, 1, 4, 18, p, p, 1, p, None, w, need, 1) == binding.ERR_SHAPE
    assert call(p, p, p, p, 1, 0, 16, p, p, 1, p, None, w, need, 1) == binding.ERR_SHAPE
    assert call(p, p, p, p, 1, 4, 16, p, p, 17, p, None, w, need, 1) == binding.ERR_SHAPE
    assert call(p, p, p, p, 1, 4, 16, p, p, 1, p, None, w, need - 1, 1) == binding.ERR_WORKSPACE
