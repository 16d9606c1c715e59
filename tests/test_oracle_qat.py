"""Pins of the QAT oracle (oracle/qat.py) to facts outside it.

* The straight-through backward equals torch autograd (CPU, float64) on the
  forward graph written with the usual straight-through construction
  b = r + (b_hard - r).detach() and the scales as masked means of |Re r|,
  |Im r| -- a different route (automatic differentiation of the forward)
  to the same gradient as the oracle's hand-written reverse recursion.
* Gauss's product equals the plain complex product, and its three real
  products are the ones remark (iii) names.
* The layer gradients equal torch autograd of the real form [Re y; Im y] =
  R [Re x; Im x] (Eq. R-sum), and of the complex form, for a real loss."""
import numpy as np
import pytest

from oracle import fairy2i as O
from oracle import qat as Q

torch = pytest.importorskip("torch")


def _cplx(rng, *shape):
    return rng.standard_normal(shape) + 1j * rng.standard_normal(shape)


def _torch_fake_quant(Mr, Mi, T, codes):
    """The STE forward graph in torch: per stage, hard codes from the oracle
    (the projection is piecewise constant), b = r + (b_hard - r).detach(),
    scales as masked means with the masks fixed."""
    Rr, Ri = Mr, Mi
    hat_r = torch.zeros_like(Mr)
    hat_i = torch.zeros_like(Mi)
    for t in range(T):
        b_re, b_im = O.code_planes(codes[t])
        b_re = torch.from_numpy(b_re)
        b_im = torch.from_numpy(b_im)
        m_re, m_im = b_re != 0, b_im != 0
        s_re = (Rr.abs() * m_re).sum() / max(int(m_re.sum()), 1) if m_re.any() else Rr.sum() * 0
        s_im = (Ri.abs() * m_im).sum() / max(int(m_im.sum()), 1) if m_im.any() else Ri.sum() * 0
        br = Rr + (b_re - Rr).detach()
        bi = Ri + (b_im - Ri).detach()
        qr, qi = s_re * br, s_im * bi
        hat_r = hat_r + qr
        hat_i = hat_i + qi
        Rr, Ri = Rr - qr, Ri - qi
    return hat_r, hat_i


@pytest.mark.parametrize("N,K,T", [(3, 8, 1), (4, 12, 2), (5, 16, 3), (2, 20, 4)])
def test_ste_backward_matches_autograd(N, K, T):
    rng = np.random.default_rng(N * 100 + K + T)
    M = _cplx(rng, N, K).astype(np.complex64)
    W_hat, codes, scales = Q.fake_quant(M, T)
    G = _cplx(rng, N, K)
    got = Q.ste_backward(codes, scales, G)
    Mr = torch.tensor(M.real.astype(np.float64), requires_grad=True)
    Mi = torch.tensor(M.imag.astype(np.float64), requires_grad=True)
    hr, hi = _torch_fake_quant(Mr, Mi, T, codes)
    # the forward values agree with the oracle's (scales in float64 here)
    np.testing.assert_allclose(hr.detach().numpy() + 1j * hi.detach().numpy(), W_hat, rtol=1e-6, atol=1e-7)
    loss = (hr * torch.from_numpy(G.real)).sum() + (hi * torch.from_numpy(G.imag)).sum()
    loss.backward()
    want = Mr.grad.numpy() + 1j * Mi.grad.numpy()
    # the oracle uses the stored float32 scales, autograd the float64 means
    np.testing.assert_allclose(got, want, rtol=1e-6, atol=1e-6)


def test_ste_backward_t1_closed_form():
    """T = 1: g = (s_re Re G + b_re <Re G, b_re>/n_re) + i (...)."""
    rng = np.random.default_rng(5)
    M = _cplx(rng, 6, 10).astype(np.complex64)
    _, codes, scales = Q.fake_quant(M, 1)
    G = _cplx(rng, 6, 10)
    b_re, b_im = O.code_planes(codes[0])
    want_r = scales[0, 0] * G.real + b_re * (G.real * b_re).sum() / np.count_nonzero(b_re)
    want_i = scales[0, 1] * G.imag + b_im * (G.imag * b_im).sum() / np.count_nonzero(b_im)
    np.testing.assert_allclose(Q.ste_backward(codes, scales, G), want_r + 1j * want_i, rtol=1e-12)


def test_gauss_is_the_complex_product():
    rng = np.random.default_rng(6)
    A, B = _cplx(rng, 7, 9), _cplx(rng, 9, 5)
    np.testing.assert_allclose(Q.gauss_matmul(A, B), A @ B, rtol=1e-12, atol=1e-12)
    # scalar case of remark (iii)
    a, b, c, d = 1.5, -2.0, 0.25, 3.0
    z = Q.gauss_matmul(np.array([[a + 1j * b]]), np.array([[c + 1j * d]]))[0, 0]
    assert z == (a + 1j * b) * (c + 1j * d)


def test_layer_gradients_match_autograd_of_the_real_form():
    rng = np.random.default_rng(7)
    Bt, N, K = 3, 4, 5
    U, W, X, GY = _cplx(rng, N, K), _cplx(rng, N, K), _cplx(rng, Bt, K), _cplx(rng, Bt, N)
    Y = Q.layer_forward(U, W, X)
    R = O.realify_lin(U) + O.realify_conj(W)
    Xt = np.concatenate([X.real, X.imag], axis=1)
    np.testing.assert_allclose(np.concatenate([Y.real, Y.imag], axis=1), Xt @ R.T, rtol=1e-12, atol=1e-12)
    tU_r = torch.tensor(U.real, requires_grad=True)
    tU_i = torch.tensor(U.imag, requires_grad=True)
    tW_r = torch.tensor(W.real, requires_grad=True)
    tW_i = torch.tensor(W.imag, requires_grad=True)
    tX_r = torch.tensor(X.real, requires_grad=True)
    tX_i = torch.tensor(X.imag, requires_grad=True)
    # the real form, built from the blocks of Eq. (realify-ops)
    top = torch.cat([tU_r + tW_r, tW_i - tU_i], dim=1)
    bot = torch.cat([tU_i + tW_i, tU_r - tW_r], dim=1)
    Rt = torch.cat([top, bot], dim=0)
    Yt = torch.cat([tX_r, tX_i], dim=1) @ Rt.T
    loss = (Yt * torch.from_numpy(np.concatenate([GY.real, GY.imag], axis=1))).sum()
    loss.backward()
    G_X, G_U, G_W = Q.layer_backward(U, W, X, GY)
    np.testing.assert_allclose(G_X, tX_r.grad.numpy() + 1j * tX_i.grad.numpy(), rtol=1e-12, atol=1e-12)
    np.testing.assert_allclose(G_U, tU_r.grad.numpy() + 1j * tU_i.grad.numpy(), rtol=1e-12, atol=1e-12)
    np.testing.assert_allclose(G_W, tW_r.grad.numpy() + 1j * tW_i.grad.numpy(), rtol=1e-12, atol=1e-12)
