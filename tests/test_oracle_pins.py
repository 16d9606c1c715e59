"""Pins of the CPU oracle against what the paper and mathematics fix.

None of these re-types an oracle formula: each checks the oracle against a
different characterisation (hand-worked values, brute force, closed-form
identities, exact rational arithmetic, or an independent textbook route).
"""
import json
import math
import os
from fractions import Fraction

import numpy as np
import pytest

import oracle
import synth

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def _golden(name):
    with open(os.path.join(GOLDEN, name)) as f:
        return json.load(f)


def _rand_complex(rng, shape, scale=1.0):
    return ((rng.standard_normal(shape) + 1j * rng.standard_normal(shape)) * scale)


# ---------------------------------------------------------------- Sec. 3.1 ---

def test_widely_linear_hand_example():
    g = _golden("widely_linear_2x2.json")
    U, W = oracle.to_widely_linear(np.array(g["A"], dtype=np.float32))
    assert U.shape == (1, 1) and W.shape == (1, 1)
    assert (U[0, 0].real, U[0, 0].imag) == tuple(g["U"])
    assert (W[0, 0].real, W[0, 0].imag) == tuple(g["W"])


@pytest.mark.parametrize("shape", [(2, 2), (8, 6), (256, 256), (64, 200)])
def test_exact_equivalence_theorem(shape):
    """Theorem (exact equivalence): [Re y; Im y] = A x~ <=> y = U x + W conj(x),
    checked to float64 rounding for random A and x."""
    rng = np.random.default_rng(sum(shape))
    A = rng.standard_normal(shape).astype(np.float32)
    N, K = shape[0] // 2, shape[1] // 2
    U, W = oracle.to_widely_linear_f64(A)
    x = _rand_complex(rng, (5, K))
    y = x @ U.T + np.conj(x) @ W.T
    y_real = oracle.stack_real(x) @ A.astype(np.float64).T
    err = np.abs(oracle.stack_real(y) - y_real).max()
    assert err <= 1e-13 * max(1.0, np.abs(y_real).max())


def test_round_trip_R_sum_is_exact():
    """Eq. (R-sum): A = R_lin(U) + R_conj(W), bit for bit."""
    rng = np.random.default_rng(7)
    A = rng.standard_normal((64, 96)).astype(np.float32)
    U, W = oracle.to_widely_linear_f64(A)
    R = oracle.realify_lin(U) + oracle.realify_conj(W)
    np.testing.assert_array_equal(R, A.astype(np.float64))


def test_realify_ops_act_as_complex_maps():
    """Eq. (realify-eval): R_lin(U) x~ stacks U x, R_conj(W) x~ stacks W conj(x)."""
    rng = np.random.default_rng(3)
    U = _rand_complex(rng, (5, 7))
    W = _rand_complex(rng, (5, 7))
    x = _rand_complex(rng, (7,))
    np.testing.assert_allclose(oracle.realify_lin(U) @ oracle.stack_real(x), oracle.stack_real(U @ x), rtol=1e-13, atol=1e-13)
    np.testing.assert_allclose(oracle.realify_conj(W) @ oracle.stack_real(x), oracle.stack_real(W @ np.conj(x)), rtol=1e-13, atol=1e-13)


def test_uniqueness_special_cases():
    """Uniqueness: a complex-linear A gives W = 0 exactly, a conjugate-linear A
    gives U = 0 exactly, and each recovers its generator."""
    rng = np.random.default_rng(11)
    U0 = _rand_complex(rng, (6, 10)).astype(np.complex64)
    W0 = _rand_complex(rng, (6, 10)).astype(np.complex64)
    U, W = oracle.to_widely_linear(oracle.realify_lin(U0).astype(np.float32))
    np.testing.assert_array_equal(U, U0)
    assert not np.any(W)
    U, W = oracle.to_widely_linear(oracle.realify_conj(W0).astype(np.float32))
    np.testing.assert_array_equal(W, W0)
    assert not np.any(U)


def test_complex64_storage_is_single_rounding():
    """U, W are the exact block averages rounded once to float32; checked with
    exact rationals, including operands whose exponents are far apart."""
    rng = np.random.default_rng(5)
    A = rng.standard_normal((8, 8)).astype(np.float32)
    A[0, 0], A[4, 4] = np.float32(3.0e38), np.float32(1.0e-38)      # R11, R22 far apart
    A[1, 5], A[5, 1] = np.float32(1.1754944e-38), np.float32(-7.0)  # R12, R21
    A[2, 2], A[6, 6] = np.float32(1.5e-45), np.float32(1.5e-45)     # subnormals
    U, W = oracle.to_widely_linear(A)
    N = K = 4
    F = [[Fraction(float(v)) for v in row] for row in A]
    for i in range(N):
        for j in range(K):
            r11, r12, r21, r22 = F[i][j], F[i][j + K], F[i + N][j], F[i + N][j + K]
            assert U[i, j].real == oracle.round_to_f32((r11 + r22) / 2)
            assert U[i, j].imag == oracle.round_to_f32((r21 - r12) / 2)
            assert W[i, j].real == oracle.round_to_f32((r11 - r22) / 2)
            assert W[i, j].imag == oracle.round_to_f32((r12 + r21) / 2)


# ---------------------------------------------------------------- Sec. 3.2 ---

def test_projection_matches_brute_force_argmax():
    """Eq. (ifairy-proj) argmax form: the codeword s maximising Re(w conj(s)),
    found by trying all four, on random points (ties have probability 0)."""
    rng = np.random.default_rng(0)
    w = _rand_complex(rng, (100000,)) * np.exp(rng.uniform(-3, 3, 100000))
    scores = np.stack([(w * np.conj(s)).real for s in oracle.CODEWORDS])  # [4, n]
    np.testing.assert_array_equal(oracle.project(w), np.argmax(scores, axis=0))


def test_projection_matches_floor_formula():
    """Eq. (ifairy-proj) floor form with theta = atan2 (off the tie lines)."""
    rng = np.random.default_rng(1)
    w = _rand_complex(rng, (100000,))
    theta = np.arctan2(w.imag, w.real)
    k = np.floor(2 * theta / np.pi + 0.5).astype(np.int64) % 4
    np.testing.assert_array_equal(oracle.project(w), k)


def test_projection_nearest_codeword_distance():
    """Nearest codeword in the complex plane = nearest by angle (|s| = 1)."""
    rng = np.random.default_rng(2)
    w = _rand_complex(rng, (20000,))
    d = np.stack([np.abs(w - s) for s in oracle.CODEWORDS])
    np.testing.assert_array_equal(oracle.project(w), np.argmin(d, axis=0))


def test_projection_ties_and_zeros():
    g = _golden("projection_ties.json")
    for c in g["cases"]:
        re, im = float(c["re"]), float(c["im"])
        w = np.array([complex(re, im)])
        w.real[0], w.imag[0] = re, im  # keep signed zeros
        assert oracle.project(w)[0] == c["code"], c


def test_projection_figure2():
    g = _golden("fig2_projection.json")
    for c in g["cases"]:
        w = c["magnitude"] * np.exp(1j * np.deg2rad(c["angle_deg"]))
        assert oracle.project(np.array([w]))[0] == c["code"]


def test_scales_are_least_squares_optimal_and_correctly_rounded():
    """Given the codes, s_re (s_im) minimises sum |w - s b(w)|^2 over the +-1
    (+-i) group; the stored float32 is the float32 with the smallest exact
    objective, i.e. no float32 neighbour does better."""
    rng = np.random.default_rng(4)
    r = _rand_complex(rng, (40, 33), 0.03)
    k = oracle.project(r)
    s_re, s_im = oracle.axis_scales(r, k)
    b = oracle.CODEWORDS[k]
    for s, grp in ((s_re, (k % 2) == 0), (s_im, (k % 2) == 1)):
        ws, bs = r[grp], b[grp]

        def obj(sv):
            sv = Fraction(float(sv))
            tot = Fraction(0)
            for wv, bv in zip(ws, bs):
                dr = Fraction(float(wv.real)) - sv * Fraction(int(bv.real))
                di = Fraction(float(wv.imag)) - sv * Fraction(int(bv.imag))
                tot += dr * dr + di * di
            return tot
        o = obj(s)
        assert o <= obj(np.nextafter(s, np.float32(0)))
        assert o <= obj(np.nextafter(s, np.float32(1)))


def test_scale_of_empty_group_is_zero():
    r = np.array([[1.0 + 0.1j, -2.0 + 0.5j, 0.3 - 0.1j, 0.0]])
    k = oracle.project(r)
    assert np.all(k % 2 == 0)
    s_re, s_im = oracle.axis_scales(r, k)
    assert s_im == 0 and s_re > 0


def test_exact_sum_against_fractions():
    rng = np.random.default_rng(9)
    v = np.abs(rng.standard_normal(500)) * np.exp2(rng.integers(-60, 60, 500))
    v[:5] = [5e-324, 0.0, 1e300, 2.2250738585072014e-308, 1e-310]
    assert oracle.exact_sum(v) == sum(Fraction(float(t)) for t in v)


def test_round_to_f32_ties_and_neighbours():
    one = Fraction(1)
    ulp = Fraction(1, 2 ** 23)
    assert oracle.round_to_f32(one + ulp / 2) == np.float32(1.0)            # tie -> even
    assert oracle.round_to_f32(one + 3 * ulp / 2) == np.float32(1.0) + np.float32(2.0 ** -22)  # tie -> even (up)
    assert oracle.round_to_f32(one + ulp / 2 + Fraction(1, 2 ** 80)) == np.nextafter(np.float32(1), np.float32(2))
    # a value where rounding through float64 first would give the wrong float32
    q = Fraction(1) + ulp / 2 + Fraction(1, 2 ** 60)   # float64(q) = 1 + ulp/2 exactly -> tie -> 1.0
    assert float(q) == 1 + 2.0 ** -24
    assert oracle.round_to_f32(q) == np.nextafter(np.float32(1), np.float32(2))


# ---------------------------------------------------------------- Sec. 3.3 ---

def test_residual_energy_identity_and_monotone():
    """||R(t+1)||^2 = ||R(t)||^2 - sum_even(2 s_re |Re r| - s_re^2)
    - sum_odd(2 s_im |Im r| - s_im^2), exactly (rationals); hence non-increasing."""
    rng = np.random.default_rng(6)
    M = _rand_complex(rng, (12, 16), 0.02).astype(np.complex64)
    codes, scales, res = oracle.quantize_with_residuals(M, 4)

    def fr(v):
        return Fraction(float(v))
    for t in range(4):
        R, Rn = res[t], res[t + 1]
        k = codes[t]
        s_re, s_im = fr(scales[t, 0]), fr(scales[t, 1])
        e0 = sum(fr(v.real) ** 2 + fr(v.imag) ** 2 for v in R.ravel())
        # the residual is carried in float64, so compare with the float64 residual's
        # exact energy: the identity holds for the exact update, and the float64
        # update is exact here (operands within 29 binary orders of each other)
        e1 = sum(fr(v.real) ** 2 + fr(v.imag) ** 2 for v in Rn.ravel())
        dec = Fraction(0)
        for v, kk in zip(R.ravel(), k.ravel()):
            if kk % 2 == 0:
                dec += 2 * s_re * abs(fr(v.real)) - s_re * s_re
            else:
                dec += 2 * s_im * abs(fr(v.imag)) - s_im * s_im
        assert e1 == e0 - dec
        assert e1 <= e0


def test_residual_norm_nonincreasing_over_stages_full_distribution():
    A = synth.llama_weight(128, 256, (99, 0, 0))
    U, W = oracle.to_widely_linear(A)
    for M in (U, W):
        _, _, res = oracle.quantize_with_residuals(M, 4)
        norms = [np.linalg.norm(R) for R in res]
        assert all(norms[t + 1] <= norms[t] for t in range(4))
        assert norms[2] < 0.75 * norms[0]


def test_codebook_matrix_recovered_exactly():
    """M = c * i^k: stage 0 returns the codes and s_re = s_im = c; the stage-1
    residual is 0, so every stage-1 code is +1 (code 0) with zero scales."""
    rng = np.random.default_rng(8)
    k = rng.integers(0, 4, (9, 12)).astype(np.uint8)
    c = np.float32(0.0371)
    M = (np.float64(c) * oracle.CODEWORDS[k]).astype(np.complex64)
    codes, scales = oracle.quantize(M, 2)
    np.testing.assert_array_equal(codes[0], k)
    assert scales[0, 0] == c and scales[0, 1] == c
    assert not np.any(codes[1]) and not np.any(scales[1])
    np.testing.assert_array_equal(oracle.dequantize(codes, scales), M.astype(np.complex128))


def test_T1_single_stage_error_and_phasequant():
    """T = 1 is plain PhaseQuant: every dequantised weight lies on its codeword's
    axis with the group's scale, and its direction is the projected one."""
    rng = np.random.default_rng(10)
    M = _rand_complex(rng, (20, 24), 0.05).astype(np.complex64)
    codes, scales = oracle.quantize(M, 1)
    D = oracle.dequantize(codes, scales)
    np.testing.assert_array_equal(oracle.project(D), codes[0])
    on_re = (codes[0] % 2) == 0
    assert np.all(np.abs(D.real[on_re]) == np.float64(scales[0, 0]))
    assert np.all(D.imag[on_re] == 0)
    assert np.all(np.abs(D.imag[~on_re]) == np.float64(scales[0, 1]))


# ---------------------------------------------------------------- Sec. 3.4 ---

def test_packing_golden_and_round_trip():
    g = _golden("packing.json")
    codes = np.array(g["rows"], dtype=np.uint8)[None]
    np.testing.assert_array_equal(oracle.pack(codes)[0], np.array(g["bytes"], dtype=np.uint8))
    rng = np.random.default_rng(12)
    c = rng.integers(0, 4, (3, 7, 32)).astype(np.uint8)
    p = oracle.pack(c)
    assert p.nbytes == 3 * 7 * 32 // 4          # T bits per real parameter per matrix half
    np.testing.assert_array_equal(oracle.unpack(p, 32), c)


def test_storage_is_T_bits_per_real_parameter():
    A = synth.llama_weight(64, 128, (98, 0, 0))
    U, W = oracle.to_widely_linear(A)
    for T in (1, 2, 3):
        nbytes = oracle.pack(oracle.quantize(U, T)[0]).nbytes + oracle.pack(oracle.quantize(W, T)[0]).nbytes
        assert nbytes * 8 == T * A.size


def test_code_multiplication_is_swap_and_negate():
    """Algorithm 1's multiplication-free rule: x1 keeps (a, b), xi gives (-b, a),
    x-1 gives (-a, -b), x-i gives (b, -a); applied to x and to conj(x)."""
    rule = {0: lambda a, b: (a, b), 1: lambda a, b: (-b, a),
            2: lambda a, b: (-a, -b), 3: lambda a, b: (b, -a)}
    rng = np.random.default_rng(13)
    for z in _rand_complex(rng, (50,)):
        for k in range(4):
            for v in (z, np.conj(z)):
                re, im = rule[k](v.real, v.imag)
                p = oracle.CODEWORDS[k] * v
                assert (re, im) == (p.real, p.imag)


def _quantized_pair(shape, T, seed):
    A = synth.llama_weight(shape[0], shape[1], (97, seed, 0))
    U, W = oracle.to_widely_linear(A)
    cu, su = oracle.quantize(U, T)
    cw, sw = oracle.quantize(W, T)
    return A, U, W, cu, su, cw, sw


@pytest.mark.parametrize("T", [1, 2, 3])
def test_codes_path_equals_dense_real_path(T):
    """y from the codes equals the real matrix-vector product R^ x~ with
    R^ = sum_t R_lin(U^(t)) + R_conj(W^(t)) (Eq. realify-ops, R-sum)."""
    A, U, W, cu, su, cw, sw = _quantized_pair((96, 160), T, T)
    rng = np.random.default_rng(T)
    x = _rand_complex(rng, (3, 80))
    y = oracle.wl_matmul(cu, su, cw, sw, x)
    Rq = oracle.dense_real_matrix(cu, su, cw, sw)
    np.testing.assert_allclose(oracle.stack_real(y), oracle.stack_real(x) @ Rq.T, rtol=1e-12, atol=1e-12)


def test_quantisation_error_bound():
    """||A x~ - R^ x~|| <= (||R_U(T)||_F + ||R_W(T)||_F) ||x|| (the residuals
    are exactly what the deployed sum misses)."""
    A = synth.llama_weight(128, 128, (96, 0, 0))
    U, W = oracle.to_widely_linear(A)
    rng = np.random.default_rng(14)
    x = _rand_complex(rng, (64,))
    for T in (1, 2, 3):
        cu, su, ru = oracle.quantize_with_residuals(U, T)
        cw, sw, rw = oracle.quantize_with_residuals(W, T)
        y = oracle.wl_matmul(cu, su, cw, sw, x[None])[0]
        y_true = oracle.stack_real(x) @ A.astype(np.float64).T
        err = np.linalg.norm(oracle.stack_real(y) - y_true)
        bound = (np.linalg.norm(ru[-1]) + np.linalg.norm(rw[-1])) * np.linalg.norm(x)
        assert err <= bound * (1 + 1e-6) + 1e-5 * np.linalg.norm(y_true)


def test_int8_accumulators_brute_force():
    """Integer products by explicit loops over the unpacked codes."""
    rng = np.random.default_rng(15)
    T, N, K, B = 2, 3, 8, 2
    cu = rng.integers(0, 4, (T, N, K)).astype(np.uint8)
    cw = rng.integers(0, 4, (T, N, K)).astype(np.uint8)
    q = rng.integers(-127, 128, (B, K, 2)).astype(np.int8)
    P = oracle.int8_accumulators(cu, cw, q)
    plane_val = {0: (1, 0), 1: (0, 1), 2: (-1, 0), 3: (0, -1)}
    for m, codes in enumerate((cu, cw)):
        for t in range(T):
            for p in range(2):
                for b in range(B):
                    for i in range(N):
                        for c in range(2):
                            s = 0
                            for j in range(K):
                                s += plane_val[int(codes[t, i, j])][p] * int(q[b, j, c])
                            assert P[m, t, p, b, i, c] == s


def test_accumulator_epilogue_equals_complex_product():
    """Combining the integer products with the axis scales gives the same y
    as the complex product on the dequantised matrices."""
    A, U, W, cu, su, cw, sw = _quantized_pair((64, 96), 2, 5)
    x = synth.activations(4, 48, (95, 0))
    q, f = oracle.quantize_act_int8(x)
    P = oracle.int8_accumulators(cu, cw, q)
    y1 = oracle.combine_accumulators(P, su, sw, f)
    y2 = oracle.wl_matmul_int8(cu, su, cw, sw, q, f)
    np.testing.assert_allclose(y1, y2, rtol=1e-12, atol=1e-12)
    assert np.abs(P).max() <= 127 * 48


def test_activation_quantizer_properties():
    x = synth.activations(6, 100, (94, 0))
    x[3] = 0
    q, f = oracle.quantize_act_int8(x)
    assert q.dtype == np.int8 and f.dtype == np.float32
    for b in range(6):
        comps = np.stack([x[b].real, x[b].imag], -1).astype(np.float64)
        if b == 3:
            assert not np.any(q[b]) and f[b] == 0
            continue
        g = np.abs(comps).max()
        assert np.abs(q[b]).max() == 127
        assert np.all(np.sign(q[b]) == np.sign(np.where(np.abs(comps) * 127 / g >= 0.5, comps, 0)))
        # reconstruction error at most half a step (+ float32 slack)
        assert np.abs(q[b] * (g / 127) - comps).max() <= (g / 127) * (0.5 + 1e-5)
        assert abs(float(f[b]) - g / 127) <= 1e-7 * g


def test_act_quant_ties_to_even():
    """Reading S10, worked by hand: a token whose largest magnitude is 127
    has inv = 127/127 = 1 exactly, so every x * inv is x itself and the
    half-integers are exact ties; round-half-to-even gives 2.5 -> 2,
    3.5 -> 4, -2.5 -> -2, 0.5 -> 0, -0.5 -> 0, 1.5 -> 2, 126.5 -> 126
    (round-half-away would give 3, 4, -3, 1, -1, 2, 127)."""
    re = np.array([127.0, 2.5, 3.5, -2.5, 0.5, -0.5, 1.5, 126.5], np.float32)
    x = (re + 0j).astype(np.complex64).reshape(1, -1)
    q, f = oracle.quantize_act_int8(x)
    assert q[0, :, 0].tolist() == [127, 2, 4, -2, 0, 0, 2, 126]
    assert not np.any(q[0, :, 1])
    assert f[0] == np.float32(1.0)


def test_act_quant_product_rounded_to_float32():
    """Reading S10, worked by hand: gamma = 2.614424 (float32 0x402752B9)
    gives inv = fl32(127 / gamma) = 48.576664 (0x42424E81).  For
    x = 1.6983464 (0x3FD9636A) the exact product inv * x is 82.5000012..., and
    its float32 rounding is 82.5 (float32 spacing there is 2^-17), an exact
    tie that rounds to the even 82.  Rounding the exact product instead would
    give 83, and so would the other order of operations,
    fl32(fl32(x / gamma) * 127) = 82.50001."""
    g = np.uint32(0x402752B9).view(np.float32)
    xv = np.uint32(0x3FD9636A).view(np.float32)
    inv = np.float32(np.float32(127.0) / g)
    assert inv.view(np.uint32) == 0x42424E81
    assert Fraction(float(inv)) * Fraction(float(xv)) - Fraction(165, 2) < Fraction(1, 2 ** 19)
    x = np.array([[complex(g, 0.0), complex(xv, 0.0)]], np.complex64)
    q, f = oracle.quantize_act_int8(x)
    assert q[0, 0, 0] == 127 and q[0, 1, 0] == 82


def test_residual_subtracts_stored_float32_scale():
    """Reading S5, worked by hand: one row (1, 1, 1, (1 + 2^-23) + i 7 2^-26).
    Stage 0 codes every entry +1 (real axis); the exact mean of |Re| is
    1 + 2^-25, whose float32 rounding is 1 (half an ulp of 1 is 2^-24), so
    s_re = 1 and s_im = 0 (empty group).  The last entry's stage-1 residual is
    then 2^-23 + i 7 2^-26 with |Re| > |Im|: code 0 (+1).  Subtracting the
    exact mean instead would leave 3 2^-25 + i 7 2^-26 with |Im| > |Re|:
    code 1 (+i).  Stage 1's scales: s_re = mean(0, 0, 0, 2^-23) = 2^-25."""
    M = np.array([[1.0, 1.0, 1.0, complex(1.0 + 2.0 ** -23, 7 * 2.0 ** -26)]], np.complex64)
    assert M[0, 3].real == np.float32(1.0 + 2.0 ** -23) and M[0, 3].imag == np.float32(7 * 2.0 ** -26)
    codes, scales = oracle.quantize(M, 2)
    assert codes[0].tolist() == [[0, 0, 0, 0]]
    assert scales[0].tolist() == [1.0, 0.0]
    assert codes[1].tolist() == [[0, 0, 0, 0]]
    assert scales[1].tolist() == [2.0 ** -25, 0.0]


def test_small_layer_end_to_end_error():
    """The 256x256 case end to end: with T = 2 the codes path stays close to
    the real layer it approximates (sanity on the whole chain)."""
    A, x = synth.small_layer()
    U, W = oracle.to_widely_linear(A)
    cu, su = oracle.quantize(U, 2)
    cw, sw = oracle.quantize(W, 2)
    y = oracle.wl_matmul(cu, su, cw, sw, x)
    y_true = oracle.stack_real(x) @ A.astype(np.float64).T
    rel = np.linalg.norm(oracle.stack_real(y) - y_true) / np.linalg.norm(y_true)
    rel1 = np.linalg.norm(oracle.stack_real(oracle.wl_matmul(cu[:1], su[:1], cw[:1], sw[:1], x)) - y_true) / np.linalg.norm(y_true)
    assert rel < rel1 < 1.0


def test_oracle_imports_nothing_from_the_product():
    src_dir = os.path.join(os.path.dirname(os.path.dirname(__file__)), "oracle")
    for fn in os.listdir(src_dir):
        if fn.endswith(".py"):
            text = open(os.path.join(src_dir, fn)).read()
            assert "paper_2512_02901_amd" not in text and "torch" not in text, fn
