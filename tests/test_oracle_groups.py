"""Pins of the per-group oracle (oracle/groups.py) to facts outside it.

Each group's recursion involves only that group's entries, so the grouped
quantiser must equal the per-tensor quantiser (itself pinned in
test_oracle_pins.py) run on every one-row column block; the grouped product
must equal the sum of per-tensor products over those blocks; stage-1 group
scales are least-squares optimal per group, so they can only lower the
error of the per-tensor scales; a single group per row of a one-row matrix
is the per-tensor quantiser itself."""
import numpy as np
import pytest

from oracle import fairy2i as O
from oracle import groups as Gq


def _matrix(rng, N, K, heavy=False):
    if heavy:
        re = rng.standard_t(4, (N, K)) * 0.02
        im = rng.standard_t(4, (N, K)) * 0.02
        re[:, rng.choice(K, max(1, K // 50), replace=False)] *= 10
    else:
        re, im = rng.standard_normal((N, K)), rng.standard_normal((N, K))
    return (re + 1j * im).astype(np.complex64)


@pytest.mark.parametrize("N,K,G,T", [(3, 32, 8, 1), (4, 44, 16, 2), (2, 40, 12, 3), (5, 64, 64, 2),
                                     (3, 36, 100, 2), (2, 1024, 256, 2), (1, 20, 4, 4)])
def test_groups_are_independent_per_tensor_problems(N, K, G, T):
    rng = np.random.default_rng(N * 1000 + K + G + T)
    M = _matrix(rng, N, K, heavy=(K >= 64))
    codes, scales = Gq.quantize_grouped(M, T, G)
    assert scales.shape == (T, N, Gq.n_groups(K, G), 2)
    for i in range(N):
        for g, (a, b) in enumerate(Gq.group_bounds(K, G)):
            c1, s1 = O.quantize(M[i:i + 1, a:b], T)
            np.testing.assert_array_equal(codes[:, i, a:b], c1[:, 0])
            np.testing.assert_array_equal(scales[:, i, g], s1)


def test_group_bounds_cover_the_row():
    for K, G in [(40, 12), (36, 100), (5504, 256), (2048, 256), (8, 8)]:
        b = Gq.group_bounds(K, G)
        assert b[0][0] == 0 and b[-1][1] == K
        assert all(b[i][1] == b[i + 1][0] for i in range(len(b) - 1))
        assert all(0 < hi - lo <= G for lo, hi in b)
        assert len(b) == -(-K // G)


def test_one_group_one_row_is_per_tensor():
    rng = np.random.default_rng(3)
    M = _matrix(rng, 1, 48)
    for G in (48, 64, 1000):
        codes, scales = Gq.quantize_grouped(M, 3, G)
        c1, s1 = O.quantize(M, 3)
        np.testing.assert_array_equal(codes, c1)
        np.testing.assert_array_equal(scales[:, 0, 0], s1)


def test_stage1_group_scales_never_raise_the_error():
    """At T = 1 the codes do not depend on the scales; each group's pair is
    the least-squares optimum for its entries (Eq. ifairy-scale), so the
    grouped error is at most the per-tensor error."""
    rng = np.random.default_rng(4)
    for G in (8, 32, 100):
        M = _matrix(rng, 6, 200, heavy=True)
        cg, sg = Gq.quantize_grouped(M, 1, G)
        ct, st = O.quantize(M, 1)
        np.testing.assert_array_equal(cg, ct)
        Mg = M.astype(np.complex128)
        eg = np.linalg.norm(Mg - Gq.dequantize_grouped(cg, sg, G))
        et = np.linalg.norm(Mg - O.dequantize(ct, st))
        assert eg <= et * (1 + 1e-12)


def test_grouped_product_is_the_sum_of_block_products():
    rng = np.random.default_rng(5)
    N, K, G, T, B = 4, 40, 12, 2, 3
    MU, MW = _matrix(rng, N, K), _matrix(rng, N, K)
    cu, su = Gq.quantize_grouped(MU, T, G)
    cw, sw = Gq.quantize_grouped(MW, T, G)
    x = rng.standard_normal((B, K)) + 1j * rng.standard_normal((B, K))
    y = Gq.wl_matmul_grouped(cu, su, cw, sw, x, G)
    ref = np.zeros((B, N), dtype=np.complex128)
    for i in range(N):
        for g, (a, b) in enumerate(Gq.group_bounds(K, G)):
            ref[:, i:i + 1] += O.wl_matmul(cu[:, i:i + 1, a:b], su[:, i, g], cw[:, i:i + 1, a:b], sw[:, i, g],
                                           x[:, a:b])
    np.testing.assert_allclose(y, ref, rtol=1e-13, atol=1e-13)


def test_broadcast_per_tensor_scales_reproduce_the_per_tensor_product():
    rng = np.random.default_rng(6)
    N, K, G, T = 5, 64, 16, 2
    cu, su = O.quantize(_matrix(rng, N, K), T)
    cw, sw = O.quantize(_matrix(rng, N, K), T)
    ng = Gq.n_groups(K, G)
    bu = np.broadcast_to(su[:, None, None, :], (T, N, ng, 2)).copy()
    bw = np.broadcast_to(sw[:, None, None, :], (T, N, ng, 2)).copy()
    x = rng.standard_normal((2, K)) + 1j * rng.standard_normal((2, K))
    np.testing.assert_allclose(Gq.wl_matmul_grouped(cu, bu, cw, bw, x, G), O.wl_matmul(cu, su, cw, sw, x),
                               rtol=1e-13, atol=1e-13)
