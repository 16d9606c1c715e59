"""CPU oracle of one widely-linear decoder block for one decode token
(TEST INFRASTRUCTURE ONLY: imported by tests/, __graft_entry__.smoke() and
bench.py's cpu_baseline leg; the product path never imports it).

What it follows (arXiv 2512.02901):
  * Sec. 1: every linear layer of a LLaMA-style block (q, k, v, o, gate, up,
    down) becomes a widely-linear layer y = U x + W conj(x);
  * Sec. 3.1, self-attention paragraph, Eq. (hermitian-score): scores are
    S = Re(q^H k) / sqrt(d_k), equal to the real dot product of the stacked
    parts; softmax and value aggregation act on the real and imaginary parts
    separately; the output projection is widely-linear too.
The non-linear parts are those of the LLaMA block the paper converts
(RMSNorm, rotary position embedding, SwiGLU), written on the complex
representation: a complex vector x of length n stands for the real vector
[Re x ; Im x] of length 2n (Sec. 3.1 pairing), and every element-wise real
operation acts on Re and Im parts alike.

Readings (the paper leaves these open):
  * head pairing: complex entry c = h dc + j of a q, k, v or attention output
    (head h, j < dc = dh / 2) holds real dims h dh + j (Re) and
    h dh + dc + j (Im) of head h, i.e. each head's two halves.  Then the
    Hermitian score of a head equals that head's real score, and the rotary
    embedding that rotates dim j with dim j + dh/2 (the half-split rotary
    form) is the complex rotation c -> c e^{i pos theta_j};
  * rotary frequencies theta_j = base^(-2 j / dh), base 10000, dh = real
    head dim; the score scale is 1 / sqrt(dh);
  * RMSNorm over the 2n real components: x / sqrt(mean(x^2) + eps) * gamma,
    gamma given in stacked order [gamma_re ; gamma_im];
  * SwiGLU: silu(Re g) Re u + i silu(Im g) Im u;
  * the inputs of the quantised layers (the normed vectors, the attention
    output and the SwiGLU output) are rounded to bf16, as the decode kernels
    take bf16 activations; everything else is float64.

``block_decode`` is the widely-linear form the GPU path computes;
``block_decode_real`` is the textbook real LLaMA block on the dequantised real
matrices (Eq. R-sum) with the stacked vectors, used only to pin the former.
"""
from __future__ import annotations

import numpy as np

from .fairy2i import dense_real_matrix, wl_matmul

PROJ = ("q", "k", "v", "o", "gate", "up", "down")


def bf16_round(v: np.ndarray) -> np.ndarray:
    """Round values to bf16 (nearest, ties to even) the way a float32
    producer does: first to float32, then to bf16."""
    v32 = np.asarray(v, dtype=np.float64).astype(np.float32)
    u = v32.view(np.uint32).astype(np.uint64)
    r = ((u + 0x7FFF + ((u >> 16) & 1)) >> 16) << 16
    return r.astype(np.uint32).view(np.float32).astype(np.float64)


def bf16_round_complex(x: np.ndarray) -> np.ndarray:
    x = np.asarray(x, dtype=np.complex128)
    return bf16_round(x.real) + 1j * bf16_round(x.imag)


def rms_norm(x: np.ndarray, gamma: np.ndarray, eps: float) -> np.ndarray:
    """RMSNorm of complex x [B, n] over its 2n real components; gamma [2n] in
    stacked order."""
    x = np.asarray(x, dtype=np.complex128)
    n = x.shape[-1]
    g = np.asarray(gamma, dtype=np.float64)
    ms = (np.sum(x.real ** 2, axis=-1) + np.sum(x.imag ** 2, axis=-1)) / (2 * n)
    r = 1.0 / np.sqrt(ms + eps)
    return (x.real * r[:, None]) * g[:n] + 1j * ((x.imag * r[:, None]) * g[n:])


def rope_angles(pos: int, dh: int, base: float = 10000.0) -> np.ndarray:
    """pos * theta_j for j < dh / 2, theta_j = base^(-2 j / dh)."""
    j = np.arange(dh // 2, dtype=np.float64)
    return pos * base ** (-2.0 * j / dh)


def rope(xh: np.ndarray, pos: int, dh: int, base: float = 10000.0) -> np.ndarray:
    """Rotary embedding of complex per-head vectors xh [..., H, dh/2] at
    position pos: entry j times e^{i pos theta_j}."""
    a = rope_angles(pos, dh, base)
    return np.asarray(xh, dtype=np.complex128) * (np.cos(a) + 1j * np.sin(a))


def hermitian_attention(q: np.ndarray, k_cache: np.ndarray, v_cache: np.ndarray, n_ctx: int,
                        dh: int) -> np.ndarray:
    """Eq. (hermitian-score) for one query per head: q [H, dc];
    k_cache, v_cache [H, S, dc] with positions 0 .. n_ctx - 1 valid.
    s_n = Re(q^H k_n) / sqrt(dh); p = softmax(s); o = sum_n p_n v_n (the real
    weights act on Re v and Im v alike).  Returns o [H, dc]."""
    q = np.asarray(q, dtype=np.complex128)
    K = np.asarray(k_cache[:, :n_ctx], dtype=np.complex128)
    V = np.asarray(v_cache[:, :n_ctx], dtype=np.complex128)
    s = np.einsum("hj,hnj->hn", np.conj(q), K).real / np.sqrt(dh)
    s = s - s.max(axis=1, keepdims=True)
    p = np.exp(s)
    p = p / p.sum(axis=1, keepdims=True)
    return np.einsum("hn,hnj->hj", p, V.real) + 1j * np.einsum("hn,hnj->hj", p, V.imag)


def silu(v: np.ndarray) -> np.ndarray:
    return v / (1.0 + np.exp(-v))


def block_decode(x, layers, norm_attn, norm_mlp, k_cache, v_cache, pos: int, n_heads: int,
                 eps: float = 1e-5, base: float = 10000.0, act_round: bool = True):
    """One decode token through the widely-linear block.

    x: complex [1, n] (residual stream, n = complex model width);
    layers: {name: (codes_U, scales_U, codes_W, scales_W)} for PROJ, codes
    unpacked [T, N, K]; norm_attn, norm_mlp: float [2n] (stacked order);
    k_cache, v_cache: complex [H, S, dc] holding positions 0 .. pos - 1.
    Writes the token's rotated key and its value at position pos of copies of
    the caches and returns (out [1, n], k_cache', v_cache', trace) where
    trace holds the intermediate vectors.  act_round=False skips the bf16
    rounding of the layer inputs (used by the real-form pin)."""
    x = np.asarray(x, dtype=np.complex128)
    rnd = bf16_round_complex if act_round else (lambda a: np.asarray(a, dtype=np.complex128))
    n = x.shape[-1]
    H = n_heads
    dc = n // H
    dh = 2 * dc

    def wl(name, a):
        cu, su, cw, sw = layers[name]
        return wl_matmul(cu, su, cw, sw, a)

    z = rnd(rms_norm(x, norm_attn, eps))
    q = rope(wl("q", z).reshape(H, dc), pos, dh, base)
    k = rope(wl("k", z).reshape(H, dc), pos, dh, base)
    v = wl("v", z).reshape(H, dc)
    kc = np.array(k_cache, dtype=np.complex128, copy=True)
    vc = np.array(v_cache, dtype=np.complex128, copy=True)
    kc[:, pos] = k
    vc[:, pos] = v
    o = rnd(hermitian_attention(q, kc, vc, pos + 1, dh).reshape(1, n))
    h1 = x + wl("o", o)
    z2 = rnd(rms_norm(h1, norm_mlp, eps))
    g = wl("gate", z2)
    u = wl("up", z2)
    act = rnd(silu(g.real) * u.real + 1j * (silu(g.imag) * u.imag))
    out = h1 + wl("down", act)
    trace = {"z": z, "q": q, "k": k, "v": v, "o": o, "h1": h1, "z2": z2, "g": g, "u": u, "act": act}
    return out, kc, vc, trace


# ---------------------------------------------------------------------------
# The same block as a real LLaMA block (pin only)
# ---------------------------------------------------------------------------


def head_pairing(n_complex: int, n_heads: int) -> np.ndarray:
    """perm [2n]: stacked component s of a per-head-paired complex vector is
    real head-major dim perm[s] (Re of entry h dc + j -> h dh + j, Im ->
    h dh + dc + j)."""
    dc = n_complex // n_heads
    dh = 2 * dc
    perm = np.zeros(2 * n_complex, dtype=np.int64)
    for h in range(n_heads):
        for j in range(dc):
            perm[h * dc + j] = h * dh + j
            perm[n_complex + h * dc + j] = h * dh + dc + j
    return perm


def rope_real_half_split(r: np.ndarray, pos: int, dh: int, base: float = 10000.0) -> np.ndarray:
    """Rotary embedding of real head vectors r [..., dh] rotating dim j with
    dim j + dh/2 by pos theta_j (x cos + rotate_half(x) sin, rotate_half(x) =
    [-x2, x1])."""
    a = rope_angles(pos, dh, base)
    c = np.concatenate([np.cos(a), np.cos(a)])
    s = np.concatenate([np.sin(a), np.sin(a)])
    x1, x2 = r[..., : dh // 2], r[..., dh // 2:]
    return r * c + np.concatenate([-x2, x1], axis=-1) * s


def block_decode_real(x, layers, norm_attn, norm_mlp, k_cache_real, v_cache_real, pos: int,
                      n_heads: int, eps: float = 1e-5, base: float = 10000.0, act_round: bool = True):
    """The real block on stacked vectors: x [1, n] complex is taken as
    x~ = [Re x; Im x]; each projection is the dequantised real matrix
    R^ = R_lin(U^) + R_conj(W^) (Eq. R-sum), whose q/k/v output rows and o
    input columns are read in head-major real order through head_pairing;
    real RMSNorm, real rotary embedding, softmax(q.k / sqrt(dh)) v per head,
    real SwiGLU.  Caches are real head-major [H, S, dh].  Returns (out x~ [1,
    2n], k_cache', v_cache')."""
    x = np.asarray(x, dtype=np.complex128)
    n = x.shape[-1]
    H = n_heads
    dh = 2 * n // H
    perm = head_pairing(n, H)
    inv = np.argsort(perm)

    def R(name):
        cu, su, cw, sw = layers[name]
        return dense_real_matrix(cu, su, cw, sw)

    def stack(v):
        return np.concatenate([v.real, v.imag], axis=-1)

    def bf16(v):
        return bf16_round(v) if act_round else v

    xt = stack(x)
    ms = np.mean(xt ** 2, axis=-1, keepdims=True)
    zt = bf16(xt / np.sqrt(ms + eps) * norm_attn)
    # stacked outputs -> head-major real order
    qh = (zt @ R("q").T)[:, inv].reshape(H, dh)
    kh = (zt @ R("k").T)[:, inv].reshape(H, dh)
    vh = (zt @ R("v").T)[:, inv].reshape(H, dh)
    qh = rope_real_half_split(qh, pos, dh, base)
    kh = rope_real_half_split(kh, pos, dh, base)
    kc = np.array(k_cache_real, dtype=np.float64, copy=True)
    vc = np.array(v_cache_real, dtype=np.float64, copy=True)
    kc[:, pos] = kh
    vc[:, pos] = vh
    s = np.einsum("hd,hnd->hn", qh, kc[:, :pos + 1]) / np.sqrt(dh)
    p = np.exp(s - s.max(axis=1, keepdims=True))
    p = p / p.sum(axis=1, keepdims=True)
    oh = np.einsum("hn,hnd->hd", p, vc[:, :pos + 1]).reshape(1, 2 * n)
    ot = bf16(oh[:, perm])                      # head-major -> stacked input of o
    h1 = xt + ot @ R("o").T
    ms2 = np.mean(h1 ** 2, axis=-1, keepdims=True)
    z2 = bf16(h1 / np.sqrt(ms2 + eps) * norm_mlp)
    g = z2 @ R("gate").T
    u = z2 @ R("up").T
    act = bf16(silu(g) * u)
    out = h1 + act @ R("down").T
    return out, kc, vc
