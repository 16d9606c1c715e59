"""CPU oracle of the Fairy2i widely-linear quantised layer (arXiv 2512.02901).

TEST INFRASTRUCTURE ONLY.  This module is imported by ``tests/``, by
``__graft_entry__.smoke()`` and by the ``cpu_baseline`` leg of ``bench.py``.
The product path (the HIP library and its Python binding) never imports,
links or calls anything here, and nothing here imports the product path.

It is written to be read against the paper: plain NumPy in float64 (or exact
integer / rational arithmetic where a result has to be exact), no blocking,
no fusion, no reordering.  Every function names the passage it follows.

Notation (paper Sec. 3.1, with N = complex output dim, K = complex input dim):
  real layer      A in R^{2N x 2K}  (the paper's R), row = output, col = input
  complex pair    U, W in C^{N x K},  y = U x + W conj(x)
  codes           k in {0,1,2,3} stands for the codeword i^k
                  (0 -> +1, 1 -> +i, 2 -> -1, 3 -> -i)
  stages          t = 0 .. T-1 of recursive residual quantisation (Sec. 3.3)

Readings taken where the paper does not fix a detail (each one is a choice
of this implementation, listed with its reason in the design notes):
  * real/imag pairing is the stacked-halves split of Sec. 3.1
    (x~ = [Re x; Im x]), so R11 = A[:N,:K] etc.;
  * U, W are stored as complex64, i.e. the exact values of Eq. (UW-from-R)
    rounded once to float32;
  * projection ties follow the floor formula of Eq. (ifairy-proj)
    (each tie goes counter-clockwise), and w = 0 maps to +1;
  * an axis scale is the exact mean of its group rounded once to float32,
    0 when the group is empty; the residual subtracts that stored value;
  * int8 activations use a per-token absmax over the 2K real components,
    symmetric range [-127, 127], computed in float32.
"""
from __future__ import annotations

from fractions import Fraction

import numpy as np

# ---------------------------------------------------------------------------
# Sec. 3.1 -- widely-linear form of a real layer
# ---------------------------------------------------------------------------


def _split_blocks(A: np.ndarray):
    """The four N x K blocks R11, R12, R21, R22 of A (Sec. 3.1, block
    partition), promoted to float64."""
    A = np.asarray(A)
    rows, cols = A.shape
    assert rows % 2 == 0 and cols % 2 == 0, "real dims must be even (pad, Sec. 3.1 remarks)"
    N, K = rows // 2, cols // 2
    R = A.astype(np.float64)
    return R[:N, :K], R[:N, K:], R[N:, :K], R[N:, K:]


def to_widely_linear_f64(A: np.ndarray):
    """Eq. (UW-from-R): Re U = (R11+R22)/2, Im U = (R21-R12)/2,
    Re W = (R11-R22)/2, Im W = (R12+R21)/2.  complex128 result.

    For float32 input every sum here is exact in float64 (or, when the two
    exponents are more than 29 apart, off by less than the float32 grain),
    and halving is exact."""
    R11, R12, R21, R22 = _split_blocks(A)
    U = 0.5 * (R11 + R22) + 1j * (0.5 * (R21 - R12))
    W = 0.5 * (R11 - R22) + 1j * (0.5 * (R12 + R21))
    return U, W


def to_widely_linear(A: np.ndarray):
    """Eq. (UW-from-R) stored as complex64 (the precision the library emits):
    each component is the exact value rounded once to float32."""
    U, W = to_widely_linear_f64(A)
    return U.astype(np.complex64), W.astype(np.complex64)


def realify_lin(U: np.ndarray) -> np.ndarray:
    """Eq. (realify-ops): R_lin(U) = [[Re U, -Im U], [Im U, Re U]]."""
    U = np.asarray(U, dtype=np.complex128)
    return np.block([[U.real, -U.imag], [U.imag, U.real]])


def realify_conj(W: np.ndarray) -> np.ndarray:
    """Eq. (realify-ops): R_conj(W) = [[Re W, Im W], [Im W, -Re W]]."""
    W = np.asarray(W, dtype=np.complex128)
    return np.block([[W.real, W.imag], [W.imag, -W.real]])


def stack_real(x: np.ndarray) -> np.ndarray:
    """x~ = [Re x; Im x] (Sec. 3.1) for the last axis of x."""
    x = np.asarray(x, dtype=np.complex128)
    return np.concatenate([x.real, x.imag], axis=-1)


# ---------------------------------------------------------------------------
# Sec. 3.2 -- PhaseQuant projection, axis scales, dequantisation
# ---------------------------------------------------------------------------

CODEWORDS = np.array([1.0 + 0j, 1j, -1.0 + 0j, -1j], dtype=np.complex128)  # i^k


def project(w: np.ndarray) -> np.ndarray:
    """Eq. (ifairy-proj): code k of the codeword nearest to w by angle.

    Uses the paper's equivalent floor form k = floor(2 Arg(w)/pi + 1/2) taken
    modulo 4, with Arg in (-pi, pi], evaluated by exact comparisons of
    a = Re w and b = Im w instead of atan2:
        k = 1  iff  b > 0  and  -b <  a <= b     (Arg in [pi/4, 3pi/4))
        k = 2  iff  a < 0  and   a <  b <= -a    (Arg in [3pi/4, pi] or (-pi, -3pi/4))
        k = 3  iff  b < 0  and   b <= a <  -b    (Arg in [-3pi/4, -pi/4))
        k = 0  otherwise                          (Arg in [-pi/4, pi/4), and w = 0)
    """
    w = np.asarray(w, dtype=np.complex128)
    a, b = w.real, w.imag
    k = np.zeros(w.shape, dtype=np.uint8)
    k[(b > 0) & (-b < a) & (a <= b)] = 1
    k[(a < 0) & (a < b) & (b <= -a)] = 2
    k[(b < 0) & (b <= a) & (a < -b)] = 3
    return k


def exact_sum(values: np.ndarray) -> Fraction:
    """Exact rational sum of finite float64 values.

    Each value is m * 2**e with an integer m of at most 53 bits (np.frexp);
    the integers are summed per exponent with Python's unbounded ints."""
    v = np.asarray(values, dtype=np.float64).ravel()
    if v.size == 0:
        return Fraction(0)
    assert np.all(np.isfinite(v))
    m, e = np.frexp(v)
    mant = np.ldexp(m, 53).astype(np.int64)          # exact integers
    ex = e.astype(np.int64) - 53
    emin = int(ex.min())
    total = 0
    for x in np.unique(ex):
        total += sum(mant[ex == x].tolist()) << int(x - emin)
    return Fraction(total) * (Fraction(2) ** emin)


def round_to_f32(q: Fraction) -> np.float32:
    """Round an exact rational to the nearest float32, ties to even.

    Takes float32(float64(q)) and then checks it and its two float32
    neighbours against q exactly, so the double rounding through float64
    cannot leak in."""
    approx = np.float32(float(q))
    if not np.isfinite(approx):
        return approx
    cands = [np.nextafter(approx, np.float32(-np.inf)), approx,
             np.nextafter(approx, np.float32(np.inf))]
    best = None
    for c in cands:
        if not np.isfinite(c):
            continue
        d = abs(Fraction(float(c)) - q)
        if best is None or d < best[0] or (
                d == best[0] and (int(np.float32(c).view(np.uint32)) & 1) == 0):
            best = (d, np.float32(c))
    return best[1]


def axis_scales(r: np.ndarray, k: np.ndarray):
    """Eq. (ifairy-scale), per tensor (Sec. 3.2 footnote):
        s_re = mean of |Re r| over entries coded +-1   (k even),
        s_im = mean of |Im r| over entries coded +-i   (k odd).
    Each mean is exact and then rounded once to float32; an empty group
    gives 0.  Returns (s_re, s_im) as np.float32."""
    r = np.asarray(r, dtype=np.complex128)
    even = (k % 2) == 0
    odd = ~even
    out = []
    for vals in (np.abs(r.real[even]), np.abs(r.imag[odd])):
        n = vals.size
        out.append(np.float32(0.0) if n == 0 else round_to_f32(exact_sum(vals) / n))
    return out[0], out[1]


def code_planes(k: np.ndarray):
    """b = i^k = b_re + i b_im with b_re, b_im in {-1, 0, +1} (Sec. 3.2)."""
    b = CODEWORDS[np.asarray(k, dtype=np.int64)]
    return b.real, b.imag


def dequantize_stage(k: np.ndarray, s_re, s_im) -> np.ndarray:
    """Eq. (ifairy-dequant): w^ = s_re b_re + i s_im b_im (complex128)."""
    b_re, b_im = code_planes(k)
    return float(s_re) * b_re + 1j * (float(s_im) * b_im)


# ---------------------------------------------------------------------------
# Sec. 3.3 -- recursive residual quantisation
# ---------------------------------------------------------------------------


def quantize(M: np.ndarray, T: int):
    """Recursive residual quantisation of one complex matrix (Sec. 3.3,
    formal definition): R(0) = M; for t < T: codes(t) = project(R(t)),
    (s_re, s_im)(t) = axis_scales(R(t), codes(t)),
    R(t+1) = R(t) - (s_re b_re + i s_im b_im).

    M is taken at its stored complex64 values; the residual is kept in
    float64 and subtracts the stored float32 scales.
    Returns codes uint8 [T, N, K] and scales float32 [T, 2] = (s_re, s_im)."""
    R = np.asarray(M).astype(np.complex64).astype(np.complex128)
    N, K = R.shape
    codes = np.zeros((T, N, K), dtype=np.uint8)
    scales = np.zeros((T, 2), dtype=np.float32)
    for t in range(T):
        k = project(R)
        s_re, s_im = axis_scales(R, k)
        codes[t] = k
        scales[t] = (s_re, s_im)
        b_re, b_im = code_planes(k)
        R = (R.real - np.float64(s_re) * b_re) + 1j * (R.imag - np.float64(s_im) * b_im)
    return codes, scales


def quantize_with_residuals(M: np.ndarray, T: int):
    """As ``quantize`` but also returns the residuals R(0..T) (for pins)."""
    R = np.asarray(M).astype(np.complex64).astype(np.complex128)
    res = [R]
    codes, scales = quantize(M, T)
    for t in range(T):
        b_re, b_im = code_planes(codes[t])
        R = (R.real - np.float64(scales[t, 0]) * b_re) + 1j * (R.imag - np.float64(scales[t, 1]) * b_im)
        res.append(R)
    return codes, scales, res


def dequantize(codes: np.ndarray, scales: np.ndarray) -> np.ndarray:
    """Eq. (res-sum): the deployed matrix sum_t W^(t), complex128."""
    T = codes.shape[0]
    out = np.zeros(codes.shape[1:], dtype=np.complex128)
    for t in range(T):
        out += dequantize_stage(codes[t], scales[t, 0], scales[t, 1])
    return out


# ---------------------------------------------------------------------------
# Sec. 3.4 -- storage: 2-bit codes
# ---------------------------------------------------------------------------


def pack(codes: np.ndarray) -> np.ndarray:
    """Pack codes [T, N, K] into bytes [T, N, K/4]: code (t, i, j) sits in
    byte j // 4 of row i at bits 2*(j % 4) .. 2*(j % 4)+1 (2 bits per complex
    weight, Sec. 3.4 storage paragraph)."""
    codes = np.asarray(codes, dtype=np.uint8)
    T, N, K = codes.shape
    assert K % 4 == 0
    out = np.zeros((T, N, K // 4), dtype=np.uint8)
    for j in range(4):
        out |= (codes[:, :, j::4] & 3) << (2 * j)
    return out


def unpack(packed: np.ndarray, K: int) -> np.ndarray:
    """Inverse of ``pack``."""
    packed = np.asarray(packed, dtype=np.uint8)
    T, N, KB = packed.shape
    assert KB * 4 == K
    codes = np.zeros((T, N, K), dtype=np.uint8)
    for j in range(4):
        codes[:, :, j::4] = (packed >> (2 * j)) & 3
    return codes


# ---------------------------------------------------------------------------
# Widely-linear product with the quantised pair (Eq. widely-linear with the
# deployed sum of Eq. res-sum; Algorithm 1 computes the same product)
# ---------------------------------------------------------------------------


def wl_matmul(codes_U, scales_U, codes_W, scales_W, x: np.ndarray) -> np.ndarray:
    """y = U^ x + W^ conj(x) for every token (row) of x [B, K], where
    U^ = sum_t (s_re b_re + i s_im b_im) over U's stages and W^ likewise.
    complex128 [B, N]."""
    U = dequantize(codes_U, scales_U)
    W = dequantize(codes_W, scales_W)
    x = np.asarray(x, dtype=np.complex128)
    return x @ U.T + np.conj(x) @ W.T


def dense_real_matrix(codes_U, scales_U, codes_W, scales_W) -> np.ndarray:
    """Eq. (R-sum) for the quantised pair: R^ = R_lin(U^) + R_conj(W^)."""
    return realify_lin(dequantize(codes_U, scales_U)) + realify_conj(dequantize(codes_W, scales_W))


# ---------------------------------------------------------------------------
# INT8 activations (named in the CPU look-up-table paragraph of Sec. 3.4;
# the quantiser itself is this implementation's reading)
# ---------------------------------------------------------------------------


def quantize_act_int8(x: np.ndarray):
    """Per-token symmetric absmax quantisation, in float32:
        g   = max over the 2K real components |x|
        inv = float32(127 / g)
        q   = clamp(round_half_even(float32(x * inv)), -127, 127)
        f   = float32(g / 127)          (dequantisation factor)
    g = 0 gives q = 0 and f = 0.  x is complex [B, K] with float32 parts.
    Returns q int8 [B, K, 2] (interleaved re, im) and f float32 [B]."""
    x = np.asarray(x)
    B, K = x.shape
    comps = np.stack([x.real.astype(np.float32), x.imag.astype(np.float32)], axis=-1)  # [B,K,2]
    q = np.zeros((B, K, 2), dtype=np.int8)
    f = np.zeros(B, dtype=np.float32)
    for b in range(B):
        g = np.float32(np.max(np.abs(comps[b])))
        if g == 0:
            continue
        inv = np.float32(np.float32(127.0) / g)
        v = (comps[b] * inv).astype(np.float32)
        q[b] = np.clip(np.rint(v), -127, 127).astype(np.int8)
        f[b] = np.float32(g / np.float32(127.0))
    return q, f


def int8_as_complex(q: np.ndarray) -> np.ndarray:
    q = np.asarray(q, dtype=np.int64)
    return q[..., 0].astype(np.float64) + 1j * q[..., 1].astype(np.float64)


def int8_accumulators(codes_U, codes_W, q: np.ndarray) -> np.ndarray:
    """Exact integer products of each ternary code plane with the int8
    activations: P[M, t, p, b, i, c] = sum_j B^{M,t}_p[i, j] * q[b, j, c]
    with M in (U, W), p in (re-axis plane b_re, im-axis plane b_im) and
    c in (re, im) component of q.  int64 [2, T, 2, B, N, 2]."""
    q = np.asarray(q, dtype=np.int64)
    B, K, _ = q.shape
    T, N, _ = codes_U.shape
    P = np.zeros((2, T, 2, B, N, 2), dtype=np.int64)
    for m, codes in enumerate((codes_U, codes_W)):
        for t in range(T):
            b_re, b_im = code_planes(codes[t])
            for p, plane in enumerate((b_re, b_im)):
                pl = plane.astype(np.int64)
                for c in range(2):
                    P[m, t, p, :, :, c] = q[:, :, c] @ pl.T
    return P


def combine_accumulators(P: np.ndarray, scales_U, scales_W, f) -> np.ndarray:
    """y from the integer products: expands (s_re b_re + i s_im b_im)(q_re +- i q_im)
    for U (with q) and W (with conj q), sums the stages and multiplies by the
    token's dequantisation factor.  float64 complex [B, N]."""
    T = P.shape[1]
    y = np.zeros(P.shape[3:5], dtype=np.complex128)
    for t in range(T):
        su_re, su_im = float(scales_U[t, 0]), float(scales_U[t, 1])
        sw_re, sw_im = float(scales_W[t, 0]), float(scales_W[t, 1])
        Ur, Ui = P[0, t, 0].astype(np.float64), P[0, t, 1].astype(np.float64)
        Wr, Wi = P[1, t, 0].astype(np.float64), P[1, t, 1].astype(np.float64)
        re = (su_re * Ur[..., 0] - su_im * Ui[..., 1]) + (sw_re * Wr[..., 0] + sw_im * Wi[..., 1])
        im = (su_re * Ur[..., 1] + su_im * Ui[..., 0]) + (-sw_re * Wr[..., 1] + sw_im * Wi[..., 0])
        y += re + 1j * im
    return y * np.asarray(f, dtype=np.float64)[:, None]


def wl_matmul_int8(codes_U, scales_U, codes_W, scales_W, q, f) -> np.ndarray:
    """y = f_b (U^ q_b + W^ conj(q_b)) with q_b the int8 token as a complex
    vector: the same product as ``wl_matmul`` on dequantised activations."""
    y = wl_matmul(codes_U, scales_U, codes_W, scales_W, int8_as_complex(q))
    return y * np.asarray(f, dtype=np.float64)[:, None]
