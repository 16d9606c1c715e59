"""GPU parity of the QAT kernels against the CPU oracle (oracle/qat.py).

Bars:
* fake-quant forward: codes and scales bit-exact (the quantiser); W^ equal
  to the oracle's float64 sum rounded once (float32 output bit-exact, bf16
  output bit-exact against a single rounding of the float64 value);
* straight-through backward: relative L2 <= 1e-6 (the GPU keeps the running
  gradient in float32 between stages);
* Gauss GEMM (the single kernel and the planar path through the vendor
  library, which round the operands alike): exact for small-integer operands (every product and sum is an
  integer below 2^24, so any wrong index, sign or lane shows); otherwise,
  element by element, within the bound of its roundings: the operands and
  the two sums Ar + Ai, Br + Bi rounded to bf16 (2^-9 each) and float32
  accumulation, |dC| <= 2^-7 sum_k (|Ar||Br| + |Ai||Bi| + |Ar + Ai||Br + Bi|)
  (a factor 2 over the first-order bound), which holds at any size.
"""
import numpy as np
import pytest

import oracle
from oracle import qat as oq

pytestmark = pytest.mark.gpu


def dev(a, gpu):
    import torch
    return torch.from_numpy(np.ascontiguousarray(a)).to(gpu)


def host(t):
    return t.detach().cpu().numpy()


def rel_l2(got, want):
    got = np.asarray(got, dtype=np.complex128)
    want = np.asarray(want, dtype=np.complex128)
    den = np.linalg.norm(want)
    return np.linalg.norm(got - want) / (den if den > 0 else 1.0)


def bf16_once(v):
    """float64 -> bf16 bits, nearest with ties to even, one rounding
    (normal range)."""
    v = np.asarray(v, dtype=np.float64)
    u = v.view(np.uint64)
    a = u & np.uint64(0x7FFFFFFFFFFFFFFF)
    r = (a + np.uint64((1 << 44) - 1) + ((a >> np.uint64(45)) & np.uint64(1))) >> np.uint64(45)
    b = r - np.uint64((1023 - 127) << 7)
    out = np.where(a == 0, np.uint64(0), b) | ((u >> np.uint64(48)) & np.uint64(0x8000))
    return out.astype(np.uint16)


def bf16_bits_to_f64(bits):
    return (np.asarray(bits, dtype=np.uint32) << 16).view(np.float32).astype(np.float64)


def cplx(rng, *shape):
    return rng.standard_normal(shape) + 1j * rng.standard_normal(shape)


def to_bf16_pairs(z, gpu):
    """complex -> bf16 pairs [.., 2] on the device (round to nearest even)."""
    import torch
    z = np.asarray(z, dtype=np.complex128)
    bits = np.stack([bf16_once(z.real), bf16_once(z.imag)], axis=-1)
    return dev(bits.view(np.int16), gpu).view(torch.bfloat16)


def bf16_value(z):
    z = np.asarray(z, dtype=np.complex128)
    return bf16_bits_to_f64(bf16_once(z.real)) + 1j * bf16_bits_to_f64(bf16_once(z.imag))


# ------------------------------------------------------------ fake quant ---

@pytest.mark.parametrize("N,K,T", [(64, 256, 1), (33, 100, 2), (128, 1024, 3), (17, 64, 4)])
def test_fake_quant_matches_oracle(gpu, N, K, T):
    import torch
    import paper_2512_02901_amd as f2
    import synth
    A = synth.llama_weight(2 * N, 2 * K, (N, K, T, 1))
    U, _ = oracle.to_widely_linear(A)
    w_hat, codes, scales = oq.fake_quant(U, T)
    g32, c32, s32 = f2.qat_fake_quant(dev(U, gpu), T, out_dtype=f2.ACT_F32)
    np.testing.assert_array_equal(host(c32), oracle.pack(codes))
    np.testing.assert_array_equal(host(s32), scales)
    np.testing.assert_array_equal(host(g32), w_hat.astype(np.complex64))
    g16, _, _ = f2.qat_fake_quant(dev(U, gpu), T, out_dtype=f2.ACT_BF16)
    got = host(g16.view(torch.int16)).view(np.uint16)
    np.testing.assert_array_equal(got[..., 0], bf16_once(w_hat.real))
    np.testing.assert_array_equal(got[..., 1], bf16_once(w_hat.imag))


# --------------------------------------------------------- STE backward ---

@pytest.mark.parametrize("N,K,T", [(64, 256, 1), (33, 100, 2), (256, 2048, 2), (40, 512, 3), (9, 36, 4)])
def test_ste_backward_matches_oracle(gpu, N, K, T):
    import paper_2512_02901_amd as f2
    import synth
    rng = np.random.default_rng(N + K + T)
    A = synth.llama_weight(2 * N, 2 * K, (N, K, T, 2))
    U, _ = oracle.to_widely_linear(A)
    _, codes, scales = oq.fake_quant(U, T)
    G = cplx(rng, N, K).astype(np.complex64)
    want = oq.ste_backward(codes, scales, G.astype(np.complex128))
    _, c, s = f2.qat_fake_quant(dev(U, gpu), T, out_dtype=f2.ACT_F32)
    got = f2.qat_ste_backward(c, s, dev(G, gpu))
    assert rel_l2(host(got), want) <= 1e-6
    # repeat: bitwise equal (fixed-order reductions)
    np.testing.assert_array_equal(host(f2.qat_ste_backward(c, s, dev(G, gpu))), host(got))
    # g_hat 8 bytes off 16-byte alignment: the one-value-at-a-time loads, same sums in the same order
    import torch
    buf = torch.empty(N * K + 1, dtype=torch.complex64, device=gpu)
    buf[1:] = dev(G, gpu).reshape(-1)
    g_off = buf[1:].view(N, K)
    assert g_off.data_ptr() % 16 == 8
    np.testing.assert_array_equal(host(f2.qat_ste_backward(c, s, g_off)), host(got))


# ------------------------------------------------------------- Gauss GEMM ---

def gemm_bound(A, B):
    """Per-element bound of the bf16 + float32 roundings for C = A B^T
    (A [M, K], B [N, K], the values the kernel rounds)."""
    ar, ai, br, bi = np.abs(A.real), np.abs(A.imag), np.abs(B.real), np.abs(B.imag)
    asum, bsum = np.abs(A.real + A.imag), np.abs(B.real + B.imag)
    t = ar @ br.T + ai @ bi.T
    return 2.0 ** -7 * t, 2.0 ** -7 * (t + asum @ bsum.T)


def operand(z, dtype, trans, gpu):
    """z is the logical [rows, K] operand; stored as [K, rows] when trans."""
    import torch
    import paper_2512_02901_amd as f2
    st = z.T if trans else z
    if dtype == f2.ACT_F32:
        return dev(st.astype(np.complex64), gpu)
    return to_bf16_pairs(st, gpu)


def logical(z, dtype, conj):
    """The operand's values as the kernel reads them (before its own rounding)."""
    import paper_2512_02901_amd as f2
    v = z.astype(np.complex64).astype(np.complex128) if dtype == f2.ACT_F32 else bf16_value(z)
    return np.conj(v) if conj else v


@pytest.mark.parametrize("M,N,K", [(64, 64, 32), (100, 37, 70), (5, 130, 257), (256, 192, 1024)])
@pytest.mark.parametrize("layout", [(0, 0), (1, 0), (0, 1), (1, 1)])
@pytest.mark.parametrize("planar", [False, True])
def test_gauss_gemm_integers_exact(gpu, M, N, K, layout, planar):
    """Small integers: every bf16 value, product and sum is exact, so the
    kernel must reproduce the complex product bit for bit."""
    import paper_2512_02901_amd as f2
    rng = np.random.default_rng(M * 7 + N + K + 10 * layout[0] + layout[1])
    A = rng.integers(-8, 9, (M, K)) + 1j * rng.integers(-8, 9, (M, K))
    B = rng.integers(-8, 9, (N, K)) + 1j * rng.integers(-8, 9, (N, K))
    for dt in (f2.ACT_BF16, f2.ACT_F32):
        for conj in ((0, 0), (1, 0), (0, 1)):
            C = f2.cgemm_gauss([(operand(A, dt, layout[0], gpu), layout[0], conj[0],
                                 operand(B, dt, layout[1], gpu), layout[1], conj[1], K)], M, N, planar=planar)
            want = (np.conj(A) if conj[0] else A) @ (np.conj(B) if conj[1] else B).T
            np.testing.assert_array_equal(host(C), want.astype(np.complex64))


@pytest.mark.parametrize("M,N,K", [(64, 64, 64), (200, 130, 300), (512, 256, 2048)])
@pytest.mark.parametrize("planar", [False, True])
def test_gauss_gemm_within_rounding_bound(gpu, M, N, K, planar):
    import paper_2512_02901_amd as f2
    rng = np.random.default_rng(M + N + K)
    A, B = cplx(rng, M, K), cplx(rng, N, K)
    for dt in (f2.ACT_BF16, f2.ACT_F32):
        for lay in ((0, 0), (1, 1)):
            C = host(f2.cgemm_gauss([(operand(A, dt, lay[0], gpu), lay[0], 1, operand(B, dt, lay[1], gpu), lay[1], 0,
                                      K)], M, N, planar=planar))
            a, b = logical(A, dt, 1), logical(B, dt, 0)
            want = a @ b.T
            br, bi = gemm_bound(a, b)
            assert np.all(np.abs(C.real - want.real) <= br)
            assert np.all(np.abs(C.imag - want.imag) <= bi)
            assert rel_l2(C, want) <= 1e-2


@pytest.mark.parametrize("planar", [False, True])
def test_gauss_gemm_two_segments_and_accumulate(gpu, planar):
    import paper_2512_02901_amd as f2
    rng = np.random.default_rng(3)
    M, N, K0, K1 = 70, 90, 100, 36
    A0, B0, A1, B1 = cplx(rng, M, K0), cplx(rng, N, K0), cplx(rng, M, K1), cplx(rng, N, K1)
    C0 = rng.standard_normal((M, N)) + 1j * rng.standard_normal((M, N))
    out = dev(C0.astype(np.complex64), gpu)
    f2.cgemm_gauss([(operand(A0, f2.ACT_BF16, 0, gpu), 0, 0, operand(B0, f2.ACT_BF16, 0, gpu), 0, 0, K0),
                    (operand(A1, f2.ACT_BF16, 1, gpu), 1, 1, operand(B1, f2.ACT_F32, 0, gpu), 0, 1, K1)],
                   M, N, out=out, accumulate=True, planar=planar)
    a0, b0 = logical(A0, f2.ACT_BF16, 0), logical(B0, f2.ACT_BF16, 0)
    a1, b1 = logical(A1, f2.ACT_BF16, 1), logical(B1, f2.ACT_F32, 1)
    want = C0.astype(np.complex64).astype(np.complex128) + a0 @ b0.T + a1 @ b1.T
    r0, i0 = gemm_bound(a0, b0)
    r1, i1 = gemm_bound(a1, b1)
    got = host(out)
    assert np.all(np.abs(got.real - want.real) <= r0 + r1 + 1e-6)
    assert np.all(np.abs(got.imag - want.imag) <= i0 + i1 + 1e-6)


@pytest.mark.parametrize("planar", [False, True])
def test_qat_layer_step_matches_oracle(gpu, planar):
    """One training step of a widely-linear layer on the GPU: fake-quant
    forward of both masters, Y = X U^T + conj(X) W^T, then from G_Y the
    input gradient and the two weight gradients (one Gauss GEMM each) and
    the straight-through gradients of the masters; against the oracle on
    the same inputs."""
    import torch
    import paper_2512_02901_amd as f2
    import synth
    rng = np.random.default_rng(11)
    Bt, N, K, T = 96, 128, 256, 2
    A = synth.llama_weight(2 * N, 2 * K, (Bt, N, K))
    U, W = oracle.to_widely_linear(A)
    X = cplx(rng, Bt, K)
    GY = cplx(rng, Bt, N)
    dU, dW = dev(U, gpu), dev(W, gpu)
    Uh, cu, su = f2.qat_fake_quant(dU, T)
    Wh, cw, sw = f2.qat_fake_quant(dW, T)
    Xb = to_bf16_pairs(X, gpu)
    GYb = to_bf16_pairs(GY, gpu)
    Y = f2.cgemm_gauss([(Xb, 0, 0, Uh, 0, 0, K), (Xb, 0, 1, Wh, 0, 0, K)], Bt, N, planar=planar)
    GX = f2.cgemm_gauss([(GYb, 0, 0, Uh, 1, 1, N), (GYb, 0, 1, Wh, 1, 0, N)], Bt, K, planar=planar)
    GUW = [f2.cgemm_gauss([(GYb, 1, 0, Xb, 1, c, Bt)], N, K, planar=planar) for c in (1, 0)]
    gU = f2.qat_ste_backward(cu, su, GUW[0])
    gW = f2.qat_ste_backward(cw, sw, GUW[1])
    torch.cuda.synchronize()
    # oracle on the values the kernels read: bf16 W^, X, G_Y
    Uh_o, codes_u, sc_u = oq.fake_quant(U, T)
    Wh_o, codes_w, sc_w = oq.fake_quant(W, T)
    Uq, Wq, Xq, GYq = bf16_value(Uh_o), bf16_value(Wh_o), bf16_value(X), bf16_value(GY)
    Y_o = oq.layer_forward(Uq, Wq, Xq)
    GX_o, GU_o, GW_o = oq.layer_backward(Uq, Wq, Xq, GYq)
    for got, want in ((Y, Y_o), (GX, GX_o), (GUW[0], GU_o), (GUW[1], GW_o)):
        assert rel_l2(host(got), want) <= 1e-2
    # the straight-through step on the GPU's own weight gradients
    gU_o = oq.ste_backward(codes_u, sc_u, host(GUW[0]).astype(np.complex128))
    gW_o = oq.ste_backward(codes_w, sc_w, host(GUW[1]).astype(np.complex128))
    assert rel_l2(host(gU), gU_o) <= 1e-6
    assert rel_l2(host(gW), gW_o) <= 1e-6
