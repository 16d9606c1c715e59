"""Pins of the decoder-block oracle (oracle/block.py) against what the paper
and textbook formulas fix, on the CPU:
  * the widely-linear block equals the real LLaMA block (pre-norm, rotary
    embedding rotating dim j with j + dh/2, softmax(q.k / sqrt(dh)) v per head,
    SwiGLU) applied to the stacked vectors with the dequantised real matrices
    of Eq. (R-sum): Sec. 3.1's claim that Re(q^H k) equals the real score;
  * the complex rotary embedding equals the real half-split rotation;
  * attention special cases: one position gives o = v; equal keys give the
    mean of the values; a dominant key gives its value;
  * RMSNorm: unit gamma gives mean square 1 / (1 + eps / ms).
"""
import numpy as np
import pytest

import oracle
from oracle import block as ob
import synth


def _layers(n, f, T, key):
    shapes = {"q": (n, n), "k": (n, n), "v": (n, n), "o": (n, n), "gate": (f, n), "up": (f, n), "down": (n, f)}
    out = {}
    for i, name in enumerate(ob.PROJ):
        N, K = shapes[name]
        A = synth.llama_weight(2 * N, 2 * K, (key, i))
        U, W = oracle.to_widely_linear(A)
        cu, su = oracle.quantize(U, T)
        cw, sw = oracle.quantize(W, T)
        out[name] = (cu, su, cw, sw)
    return out


def _caches(H, S, dc, pos, key):
    rng = np.random.default_rng(key)
    kr = np.zeros((H, S, 2 * dc))
    vr = np.zeros((H, S, 2 * dc))
    kr[:, :pos] = rng.standard_normal((H, pos, 2 * dc))
    vr[:, :pos] = rng.standard_normal((H, pos, 2 * dc))
    # per-head pairing: entry j = dim j + i dim j + dc
    kc = kr[..., :dc] + 1j * kr[..., dc:]
    vc = vr[..., :dc] + 1j * vr[..., dc:]
    return kr, vr, kc, vc


@pytest.mark.parametrize("act_round", [False, True])
def test_block_equals_real_llama_block(act_round):
    n, f, H, T, S, pos = 128, 344, 4, 2, 16, 9
    dc = n // H
    layers = _layers(n, f, T, 70)
    rng = np.random.default_rng(71)
    x = (rng.standard_normal((1, n)) + 1j * rng.standard_normal((1, n))) * 2.0
    na = 1.0 + 0.1 * rng.standard_normal(2 * n)
    nm = 1.0 + 0.1 * rng.standard_normal(2 * n)
    kr, vr, kc, vc = _caches(H, S, dc, pos, 72)
    out, kc2, vc2, _ = ob.block_decode(x, layers, na, nm, kc, vc, pos, H, act_round=act_round)
    outr, kr2, vr2 = ob.block_decode_real(x, layers, na, nm, kr, vr, pos, H, act_round=act_round)
    got = np.concatenate([out.real, out.imag], axis=-1)
    err = np.abs(got - outr).max() / np.abs(outr).max()
    # bf16 rounding of a value computed two ways can land on either side of a tie
    assert err <= (1e-12 if not act_round else 1e-5), err
    np.testing.assert_allclose(kc2[..., :].real, kr2[..., :dc], rtol=0, atol=1e-10)
    np.testing.assert_allclose(kc2.imag, kr2[..., dc:], rtol=0, atol=1e-10)
    np.testing.assert_allclose(vc2.real, vr2[..., :dc], rtol=0, atol=1e-10)


def test_rope_complex_equals_half_split_rotation():
    rng = np.random.default_rng(73)
    H, dh = 3, 128
    r = rng.standard_normal((H, dh))
    c = r[:, :dh // 2] + 1j * r[:, dh // 2:]
    for pos in (0, 1, 7, 4095):
        rc = ob.rope(c, pos, dh)
        rr = ob.rope_real_half_split(r, pos, dh)
        np.testing.assert_allclose(rc.real, rr[:, :dh // 2], rtol=0, atol=1e-12)
        np.testing.assert_allclose(rc.imag, rr[:, dh // 2:], rtol=0, atol=1e-12)
    # position 0 is the identity; the rotation keeps every entry's magnitude
    np.testing.assert_array_equal(ob.rope(c, 0, dh), c)
    np.testing.assert_allclose(np.abs(ob.rope(c, 123, dh)), np.abs(c), rtol=1e-14)


def test_hermitian_score_equals_stacked_dot_product():
    rng = np.random.default_rng(74)
    q = rng.standard_normal(64) + 1j * rng.standard_normal(64)
    k = rng.standard_normal(64) + 1j * rng.standard_normal(64)
    assert abs(np.real(np.vdot(q, k)) - (q.real @ k.real + q.imag @ k.imag)) < 1e-12


def test_attention_special_cases():
    rng = np.random.default_rng(75)
    H, S, dc, dh = 2, 8, 16, 32
    q = rng.standard_normal((H, dc)) + 1j * rng.standard_normal((H, dc))
    K = rng.standard_normal((H, S, dc)) + 1j * rng.standard_normal((H, S, dc))
    V = rng.standard_normal((H, S, dc)) + 1j * rng.standard_normal((H, S, dc))
    np.testing.assert_allclose(ob.hermitian_attention(q, K, V, 1, dh), V[:, 0], rtol=1e-15)
    Ke = np.repeat(K[:, :1], S, axis=1)
    np.testing.assert_allclose(ob.hermitian_attention(q, Ke, V, 5, dh), V[:, :5].mean(axis=1), rtol=1e-13)
    Kd = np.zeros_like(K)
    Kd[:, 3] = q * 1e3       # score of position 3 is |q|^2 1e3 / sqrt(dh): the softmax picks it
    np.testing.assert_allclose(ob.hermitian_attention(q, Kd, V, 6, dh), V[:, 3], rtol=1e-12)


def test_rms_norm_unit_gamma():
    rng = np.random.default_rng(76)
    x = rng.standard_normal((3, 50)) + 1j * rng.standard_normal((3, 50))
    eps = 1e-5
    y = ob.rms_norm(x, np.ones(100), eps)
    ms = (np.abs(x) ** 2).sum(axis=1) / 100
    np.testing.assert_allclose((np.abs(y) ** 2).sum(axis=1) / 100, ms / (ms + eps), rtol=1e-13)
