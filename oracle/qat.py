"""CPU oracle of the quantisation-aware-training pieces of one widely-linear
layer (TEST INFRASTRUCTURE ONLY: imported by tests/, never by the product
path).

What it follows (arXiv 2512.02901):
  * Sec. 3.2, QAT paragraph, and Sec. 3.3 (the QAT remarks after the
    formal definition): full-precision masters; the forward pass uses the
    dequantised sum of the T-stage recursion; the backward pass is a
    straight-through estimator for the projection b(.); the scales are
    recomputed every step and differentiated through their dependence on
    the residuals;
  * Sec. 3.2, remark (iii): Gauss's three-multiplication complex product,
    Re = ac - bd, Im = (a + b)(c + d) - ac - bd;
  * the layer y = U x + W conj(x) (Sec. 3.1) with its gradients.

Readings (the paper does not fix these):
  * the straight-through estimator takes b(.) as the identity map of the
    complex entry (its real 2x2 Jacobian is I at every entry, whatever the
    entry's code); the paper's "small neighbourhood" is given no radius, so
    no clipping is applied;
  * s_re = mean |Re r| over the entries coded +-1 is differentiated with
    the set held fixed: d s_re / d Re r_j = b_re_j / n_re for those entries
    (b_re_j, the sign the projection chose, is the derivative of |Re r_j|;
    at Re r_j = 0 the projection gives +1 and so does this rule), likewise
    s_im; an empty axis group has scale 0 and contributes nothing;
  * gradients of a real loss with respect to a complex array are written
    g = dL/dRe + i dL/dIm.
"""
from __future__ import annotations

import numpy as np

from .fairy2i import code_planes, dequantize, quantize


def fake_quant(M: np.ndarray, T: int):
    """Forward of the fake quantiser: (W^ = sum_t s_t b_t (complex128),
    codes [T, N, K], scales [T, 2]) with the quantiser of Sec. 3.3."""
    codes, scales = quantize(M, T)
    return dequantize(codes, scales), codes, scales


def ste_backward(codes: np.ndarray, scales: np.ndarray, g_hat: np.ndarray) -> np.ndarray:
    """Gradient with respect to the master from g_hat = dL/dW^ (complex,
    [N, K]), through the recursion W^ = sum_t Q_t, Q_t = q_t(R_t),
    R_{t+1} = R_t - Q_t, R_0 = master.  Per stage, with the straight-through
    b and the scales' dependence on R_t:
        dL/dRe R_t += s_re Re G_Q + b_re (sum_j Re G_Q_j b_re_j) / n_re
        dL/dIm R_t += s_im Im G_Q + b_im (sum_j Im G_Q_j b_im_j) / n_im
    where G_Q = dL/dQ_t = g_hat - dL/dR_{t+1} (Q_t enters W^ directly and
    R_{t+1} with a minus sign).  Stages in reverse order; complex128."""
    T = codes.shape[0]
    g_hat = np.asarray(g_hat, dtype=np.complex128)
    H = np.zeros_like(g_hat)            # dL/dR_{t+1}, zero for R_T
    for t in reversed(range(T)):
        b_re, b_im = code_planes(codes[t])
        s_re, s_im = float(scales[t, 0]), float(scales[t, 1])
        GQ = g_hat - H
        n_re = int(np.count_nonzero(b_re))
        n_im = int(np.count_nonzero(b_im))
        d_re = np.sum(GQ.real * b_re) / n_re if n_re else 0.0
        d_im = np.sum(GQ.imag * b_im) / n_im if n_im else 0.0
        H = H + (s_re * GQ.real + b_re * d_re) + 1j * (s_im * GQ.imag + b_im * d_im)
    return H


def gauss_matmul(A: np.ndarray, B: np.ndarray) -> np.ndarray:
    """Remark (iii): C = A B for complex A [M, K], B [K, N] with three real
    products: P1 = Ar Br, P2 = Ai Bi, P3 = (Ar + Ai)(Br + Bi);
    C = (P1 - P2) + i (P3 - P1 - P2).  float64, no rounding of the sums."""
    A = np.asarray(A, dtype=np.complex128)
    B = np.asarray(B, dtype=np.complex128)
    P1 = A.real @ B.real
    P2 = A.imag @ B.imag
    P3 = (A.real + A.imag) @ (B.real + B.imag)
    return (P1 - P2) + 1j * (P3 - P1 - P2)


def layer_forward(U_hat, W_hat, X):
    """Y = X U^T + conj(X) W^T for tokens X [B, K] (y = U x + W conj(x) per
    token)."""
    X = np.asarray(X, dtype=np.complex128)
    return X @ np.asarray(U_hat).T + np.conj(X) @ np.asarray(W_hat).T


def layer_backward(U_hat, W_hat, X, G_Y):
    """Gradients of a real loss through Y = X U^T + conj(X) W^T, from
    G_Y = dL/dY:  G_X = G_Y conj(U) + conj(G_Y) W,  G_U = G_Y^T conj(X),
    G_W = G_Y^T X."""
    X = np.asarray(X, dtype=np.complex128)
    G_Y = np.asarray(G_Y, dtype=np.complex128)
    U_hat = np.asarray(U_hat, dtype=np.complex128)
    W_hat = np.asarray(W_hat, dtype=np.complex128)
    G_X = G_Y @ np.conj(U_hat) + np.conj(G_Y) @ W_hat
    G_U = G_Y.T @ np.conj(X)
    G_W = G_Y.T @ X
    return G_X, G_U, G_W
