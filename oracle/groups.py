"""CPU oracle of the quantiser and product with per-group axis scales
(TEST INFRASTRUCTURE ONLY: imported by tests/, never by the product path).

The paper uses one pair of axis scales per tensor (Sec. 3.2, the footnote
to Eq. ifairy-scale) and names per-group scale sharing as the alternative
(Sec. 1 and the footnote).  The reading taken here: a group is G consecutive
input columns of one output row, j in [g G, min((g + 1) G, K)), so a row of K
columns has ceil(K / G) groups and the last one may be shorter.  Every group
gets its own pair (s_re, s_im) of Eq. (ifairy-scale), computed over the
group's entries only, at every stage of the recursion of Sec. 3.3; the
projection of Eq. (ifairy-proj) is per entry and does not change.  The
dequantised entry (Eq. ifairy-dequant) uses the scales of its own group.

Scales are float32 [T, N, ceil(K / G), 2] = (s_re, s_im) per stage, row and
group; each is the exact group mean rounded once to float32, 0 for an empty
axis group, and the residual subtracts the stored value (the same readings
as the per-tensor quantiser).
"""
from __future__ import annotations

import numpy as np

from .fairy2i import axis_scales, code_planes, project


def n_groups(K: int, G: int) -> int:
    return -(-K // G)


def group_bounds(K: int, G: int):
    """[(start, stop)] of the column groups of a row."""
    return [(g * G, min(K, (g + 1) * G)) for g in range(n_groups(K, G))]


def quantize_grouped(M: np.ndarray, T: int, G: int):
    """Sec. 3.3 recursion with per-group scales: R(0) = M (complex64 values);
    for t < T: codes(t) = project(R(t)); for each row i and group g the
    scales of Eq. (ifairy-scale) over that group's entries; then
    R(t+1) = R(t) - (s_re[i, g(j)] b_re + i s_im[i, g(j)] b_im).
    Returns codes uint8 [T, N, K] and scales float32 [T, N, ngroups, 2]."""
    R = np.asarray(M).astype(np.complex64).astype(np.complex128)
    N, K = R.shape
    bounds = group_bounds(K, G)
    codes = np.zeros((T, N, K), dtype=np.uint8)
    scales = np.zeros((T, N, len(bounds), 2), dtype=np.float32)
    for t in range(T):
        k = project(R)
        codes[t] = k
        s_re = np.zeros((N, K))
        s_im = np.zeros((N, K))
        for i in range(N):
            for g, (a, b) in enumerate(bounds):
                sr, si = axis_scales(R[i, a:b], k[i, a:b])
                scales[t, i, g] = (sr, si)
                s_re[i, a:b] = np.float64(sr)
                s_im[i, a:b] = np.float64(si)
        b_re, b_im = code_planes(k)
        R = (R.real - s_re * b_re) + 1j * (R.imag - s_im * b_im)
    return codes, scales


def dequantize_grouped(codes: np.ndarray, scales: np.ndarray, G: int) -> np.ndarray:
    """Eq. (res-sum) with per-group scales: sum_t (s_re b_re + i s_im b_im),
    each entry scaled by its row's and group's pair.  complex128 [N, K]."""
    T, N, K = codes.shape
    out = np.zeros((N, K), dtype=np.complex128)
    for t in range(T):
        b_re, b_im = code_planes(codes[t])
        for g, (a, b) in enumerate(group_bounds(K, G)):
            sr = scales[t, :, g, 0].astype(np.float64)[:, None]
            si = scales[t, :, g, 1].astype(np.float64)[:, None]
            out[:, a:b] += sr * b_re[:, a:b] + 1j * (si * b_im[:, a:b])
    return out


def wl_matmul_grouped(codes_U, scales_U, codes_W, scales_W, x: np.ndarray, G: int) -> np.ndarray:
    """y = U^ x + W^ conj(x) with the per-group dequantised pair, for every
    token (row) of x [B, K].  complex128 [B, N]."""
    U = dequantize_grouped(codes_U, scales_U, G)
    W = dequantize_grouped(codes_W, scales_W, G)
    x = np.asarray(x, dtype=np.complex128)
    return x @ U.T + np.conj(x) @ W.T
