"""GPU parity: the HIP path (through the C ABI) against the CPU oracle on the
same seeded inputs.

Bars: packed codes, scales, int8 activations and integer accumulators
bit-exact; y within relative L2 1e-5 for float32 and int8 activations and
1e-3 for bf16 activations (the oracle consumes the same bf16-rounded values).
"""
import numpy as np
import pytest

import oracle
import synth

pytestmark = pytest.mark.gpu

TOL_F32 = 1e-5
TOL_BF16 = 1e-3


def rel_l2(got, want):
    got = np.asarray(got, dtype=np.complex128)
    want = np.asarray(want, dtype=np.complex128)
    den = np.linalg.norm(want)
    return np.linalg.norm(got - want) / (den if den > 0 else 1.0)


def dev(a, gpu):
    import torch
    return torch.from_numpy(np.ascontiguousarray(a)).to(gpu)


def host(t):
    return t.detach().cpu().numpy()


def oracle_layer(A, T):
    U, W = oracle.to_widely_linear(A)
    cu, su = oracle.quantize(U, T)
    cw, sw = oracle.quantize(W, T)
    return U, W, cu, su, cw, sw


def upload_layer(cu, su, cw, sw, gpu):
    return (dev(oracle.pack(cu), gpu), dev(su, gpu), dev(oracle.pack(cw), gpu), dev(sw, gpu))


def bf16_dev(x, gpu):
    """complex64 [B, K] with bf16-exact parts -> bf16 [B, K, 2] device tensor."""
    import torch
    bits = np.stack([synth.bf16_bits(x.real.astype(np.float32)),
                     synth.bf16_bits(x.imag.astype(np.float32))], axis=-1)
    return dev(bits.view(np.int16), gpu).view(torch.bfloat16)


# ------------------------------------------------------------- to_wl ---

@pytest.mark.parametrize("shape", [(256, 256), (2, 2), (6, 10), (130, 68), (4096, 4096)])
def test_to_widely_linear_bit_exact(gpu, shape):
    import paper_2512_02901_amd as f2
    if shape == (256, 256):
        A = synth.small_layer()[0]
    else:
        A = synth.llama_weight(shape[0], shape[1], (1, *shape))
    U, W = f2.to_widely_linear(dev(A, gpu))
    Uo, Wo = oracle.to_widely_linear(A)
    np.testing.assert_array_equal(host(U), Uo)
    np.testing.assert_array_equal(host(W), Wo)


def test_to_widely_linear_extremes(gpu):
    import paper_2512_02901_amd as f2
    A = np.zeros((8, 8), np.float32)
    A[0, 0], A[4, 4] = 3.0e38, 1.0e-38
    A[1, 5], A[5, 1] = 1.1754944e-38, -7.0
    A[2, 2], A[6, 6] = 1.5e-45, 1.5e-45
    A[3, 7], A[7, 3] = -3.4e38, -3.4e38
    U, W = f2.to_widely_linear(dev(A, gpu))
    Uo, Wo = oracle.to_widely_linear(A)
    np.testing.assert_array_equal(host(U).view(np.uint32), Uo.view(np.uint32))
    np.testing.assert_array_equal(host(W).view(np.uint32), Wo.view(np.uint32))


# ---------------------------------------------------------- quantize ---

def _check_quantize(M, T, gpu):
    import paper_2512_02901_amd as f2
    codes, scales = f2.quantize(dev(M, gpu), T)
    co, so = oracle.quantize(M, T)
    np.testing.assert_array_equal(host(scales).view(np.uint32), so.view(np.uint32))
    np.testing.assert_array_equal(host(codes), oracle.pack(co))


@pytest.mark.parametrize("T", [1, 2, 3, 4])
def test_quantize_small_layer(gpu, T):
    A = synth.small_layer()[0]
    U, W = oracle.to_widely_linear(A)
    _check_quantize(U, T, gpu)
    _check_quantize(W, T, gpu)


@pytest.mark.parametrize("shape", [(1, 4), (3, 20), (37, 100), (64, 1028)])
def test_quantize_ragged(gpu, shape):
    rng = np.random.default_rng(shape[1])
    M = ((rng.standard_normal(shape) + 1j * rng.standard_normal(shape)) * 0.03).astype(np.complex64)
    _check_quantize(M, 3, gpu)


def test_quantize_degenerate(gpu):
    # all zeros: every code +1, all scales 0
    _check_quantize(np.zeros((8, 16), np.complex64), 2, gpu)
    # codebook-valued: exact at stage 0, zero residual after
    rng = np.random.default_rng(3)
    k = rng.integers(0, 4, (16, 32))
    M = (np.float64(np.float32(0.0371)) * oracle.CODEWORDS[k]).astype(np.complex64)
    _check_quantize(M, 3, gpu)
    # exact ties on the diagonals and signed zeros
    vals = np.array([1 + 1j, -1 + 1j, -1 - 1j, 1 - 1j, 0, complex(-0.0, 0.0), complex(0.0, -0.0),
                     -1, 1j, -1j, 2 + 2j, -3 + 3j], dtype=np.complex64)
    M = np.resize(vals, (6, 16)).astype(np.complex64)
    M[1].real = -0.0
    _check_quantize(M, 4, gpu)
    # one group empty at stage 0 (all on the real axis)
    M = (np.resize(np.array([1.0, -2.0, 0.5, -0.25]), (4, 8)) + 0.01j).astype(np.complex64)
    _check_quantize(M, 2, gpu)


def test_quantize_llama_q_shape(gpu):
    """4096x4096 real layer -> 2048x2048 U and W, T = 2 (full size)."""
    import paper_2512_02901_amd as f2
    A = synth.llama_weight(4096, 4096, synth.layer_key(2, 0, "q"))
    U, W = f2.to_widely_linear(dev(A, gpu))
    Uo, Wo = oracle.to_widely_linear(A)
    for Md, Mo in ((U, Uo), (W, Wo)):
        codes, scales = f2.quantize(Md, 2)
        co, so = oracle.quantize(Mo, 2)
        np.testing.assert_array_equal(host(scales).view(np.uint32), so.view(np.uint32))
        np.testing.assert_array_equal(host(codes), oracle.pack(co))


# ----------------------------------------------------- act quant ---

def test_act_quant_bit_exact(gpu):
    import paper_2512_02901_amd as f2
    x = synth.activations(9, 300, (4, 0))
    x[4] = 0
    x[6, 17] = complex(-50.0, 0)     # outlier sets the scale
    q, xs = f2.quantize_act_int8(dev(x, gpu))
    qo, fo = oracle.quantize_act_int8(x)
    np.testing.assert_array_equal(host(q), qo)
    np.testing.assert_array_equal(host(xs).view(np.uint32), fo.view(np.uint32))
    xb = synth.bf16_round_complex(x)
    q, xs = f2.quantize_act_int8(bf16_dev(xb, gpu))
    qo, fo = oracle.quantize_act_int8(xb)
    np.testing.assert_array_equal(host(q), qo)
    np.testing.assert_array_equal(host(xs).view(np.uint32), fo.view(np.uint32))


# -------------------------------------------------------- products ---

def test_small_layer_f32(gpu):
    """256x256 real layer, T = 2, one float32 token: the whole chain on GPU."""
    import paper_2512_02901_amd as f2
    A, x = synth.small_layer()
    U, W = f2.to_widely_linear(dev(A, gpu))
    cu, su = f2.quantize(U, 2)
    cw, sw = f2.quantize(W, 2)
    y = f2.wl_matmul(cu, su, cw, sw, dev(x, gpu))
    _, _, cuo, suo, cwo, swo = oracle_layer(A, 2)
    yo = oracle.wl_matmul(cuo, suo, cwo, swo, x)
    assert rel_l2(host(y), yo) <= TOL_F32


@pytest.mark.parametrize("T", [1, 2, 3, 4])
@pytest.mark.parametrize("B", [1, 3, 16])
@pytest.mark.parametrize("NK", [(128, 128), (100, 20), (70, 1100)])
def test_decode_float_paths(gpu, T, B, NK):
    import paper_2512_02901_amd as f2
    N, K = NK
    A = synth.llama_weight(2 * N, 2 * K, (5, N, K))
    _, _, cu, su, cw, sw = oracle_layer(A, T)
    d = upload_layer(cu, su, cw, sw, gpu)
    x = synth.activations(B, K, (6, B, K))
    y = f2.wl_matmul(*d, dev(x, gpu))
    assert rel_l2(host(y), oracle.wl_matmul(cu, su, cw, sw, x)) <= TOL_F32
    xb = synth.bf16_round_complex(x)
    y = f2.wl_matmul(*d, bf16_dev(xb, gpu))
    err = rel_l2(host(y), oracle.wl_matmul(cu, su, cw, sw, xb))
    assert err <= TOL_BF16
    assert err <= TOL_F32   # fp32 accumulation of exact bf16 values: far inside the bar


@pytest.mark.parametrize("T", [1, 2, 3, 4])
@pytest.mark.parametrize("B", [1, 5, 16, 17, 64, 100, 130])
@pytest.mark.parametrize("NK", [(128, 128), (48, 68), (96, 1040), (100, 192), (37, 1088)])
def test_int8_paths_bit_exact(gpu, T, B, NK):
    """Decode (B <= 16) and prefill (B > 16) int8 products: accumulators
    bit-exact, y within 1e-5."""
    import paper_2512_02901_amd as f2
    N, K = NK
    A = synth.llama_weight(2 * N, 2 * K, (7, N, K))
    _, _, cu, su, cw, sw = oracle_layer(A, T)
    d = upload_layer(cu, su, cw, sw, gpu)
    x = synth.activations(B, K, (8, B, K))
    qo, fo = oracle.quantize_act_int8(x)
    q, xs = dev(qo, gpu), dev(fo, gpu)
    acc = f2.int8_accumulators(d[0], d[2], q)
    np.testing.assert_array_equal(host(acc), oracle.int8_accumulators(cu, cw, qo))
    y = f2.wl_matmul(*d, q, xs)
    assert rel_l2(host(y), oracle.wl_matmul_int8(cu, su, cw, sw, qo, fo)) <= TOL_F32


def test_zero_activations_and_zero_scales(gpu):
    import paper_2512_02901_amd as f2
    A = synth.llama_weight(64, 64, (9, 0, 0))
    _, _, cu, su, cw, sw = oracle_layer(A, 2)
    d = upload_layer(cu, su, cw, sw, gpu)
    x = np.zeros((3, 32), np.complex64)
    y = f2.wl_matmul(*d, dev(x, gpu))
    assert not np.any(host(y))
    q, xs = f2.quantize_act_int8(dev(x, gpu))
    assert not np.any(host(q)) and not np.any(host(xs))
    y = f2.wl_matmul(*d, q, xs)
    assert not np.any(host(y))
    y = f2.wl_matmul(d[0], dev(np.zeros((2, 2), np.float32), gpu), d[2],
                     dev(np.zeros((2, 2), np.float32), gpu), dev(synth.activations(2, 32, (9, 1)), gpu))
    assert not np.any(host(y))


def test_deterministic(gpu):
    import paper_2512_02901_amd as f2
    A = synth.llama_weight(512, 1024, (10, 0, 0))
    _, _, cu, su, cw, sw = oracle_layer(A, 2)
    d = upload_layer(cu, su, cw, sw, gpu)
    xb = synth.bf16_round_complex(synth.activations(4, 512, (10, 1)))
    y1 = host(f2.wl_matmul(*d, bf16_dev(xb, gpu)))
    y2 = host(f2.wl_matmul(*d, bf16_dev(xb, gpu)))
    np.testing.assert_array_equal(y1.view(np.uint32), y2.view(np.uint32))


# ------------------------------------------------- full LLaMA shapes ---

@pytest.mark.parametrize("proj", ["q", "gate", "down"])
def test_decode_llama_shapes_bf16(gpu, proj):
    """Full-size LLaMA-2-7B projections, T = 2, bf16 decode at B = 1, 4, 16."""
    import paper_2512_02901_amd as f2
    rows, cols = synth.LLAMA2_7B_PROJ[proj]
    A = synth.llama_weight(rows, cols, synth.layer_key(3, 0, proj))
    U, W = f2.to_widely_linear(dev(A, gpu))
    cu, su = f2.quantize(U, 2)
    cw, sw = f2.quantize(W, 2)
    # the oracle's reference is built from the oracle's own codes
    _, _, cuo, suo, cwo, swo = oracle_layer(A, 2)
    np.testing.assert_array_equal(host(cu), oracle.pack(cuo))
    np.testing.assert_array_equal(host(cw), oracle.pack(cwo))
    Uo = oracle.dequantize(cuo, suo)
    Wo = oracle.dequantize(cwo, swo)
    for B in (1, 4, 16):
        xb = synth.bf16_round_complex(synth.activations(B, cols // 2, (3, B, cols)))
        y = host(f2.wl_matmul(cu, su, cw, sw, bf16_dev(xb, gpu)))
        xo = xb.astype(np.complex128)
        yo = xo @ Uo.T + np.conj(xo) @ Wo.T
        assert rel_l2(y, yo) <= TOL_BF16


def test_prefill_llama_q_shape_sampled(gpu):
    """2048 tokens x the 4096x4096 projection (complex 2048x2048), T = 2,
    int8: accumulators bit-exact and y within 1e-5 on 24 sampled tokens."""
    import paper_2512_02901_amd as f2
    A = synth.llama_weight(4096, 4096, synth.layer_key(4, 0, "q"))
    _, _, cu, su, cw, sw = oracle_layer(A, 2)
    d = upload_layer(cu, su, cw, sw, gpu)
    x = synth.activations(2048, 2048, (4, 1))
    q, xs = f2.quantize_act_int8(dev(x, gpu))
    qo, fo = oracle.quantize_act_int8(x)
    np.testing.assert_array_equal(host(q), qo)
    y = host(f2.wl_matmul(*d, q, xs))
    acc = host(f2.int8_accumulators(d[0], d[2], q))
    rng = np.random.default_rng(0)
    toks = np.sort(rng.choice(2048, 24, replace=False))
    toks[0], toks[-1] = 0, 2047
    np.testing.assert_array_equal(acc[:, :, :, toks], oracle.int8_accumulators(cu, cw, qo[toks]))
    assert rel_l2(y[toks], oracle.wl_matmul_int8(cu, su, cw, sw, qo[toks], fo[toks])) <= TOL_F32


# ------------------------------------- decode on the int8 matrix cores ---

@pytest.mark.parametrize("T", [1, 2, 3, 4])
@pytest.mark.parametrize("B", [1, 2, 3, 8, 9, 16])
@pytest.mark.parametrize("NK", [(64, 64), (100, 320), (48, 1088)])
def test_mfma_decode_bf16_and_int8(gpu, T, B, NK):
    """K % 64 == 0 routes bf16 and int8 decode to the matrix cores: ragged
    row blocks (N % 16), K not a multiple of 256 or 512, several tiles."""
    import paper_2512_02901_amd as f2
    N, K = NK
    A = synth.llama_weight(2 * N, 2 * K, (11, N, K))
    _, _, cu, su, cw, sw = oracle_layer(A, T)
    d = upload_layer(cu, su, cw, sw, gpu)
    x = synth.activations(B, K, (12, B, K))
    xb = synth.bf16_round_complex(x)
    y = host(f2.wl_matmul(*d, bf16_dev(xb, gpu)))
    assert rel_l2(y, oracle.wl_matmul(cu, su, cw, sw, xb)) <= TOL_F32
    qo, fo = oracle.quantize_act_int8(x)
    q, xs = dev(qo, gpu), dev(fo, gpu)
    np.testing.assert_array_equal(host(f2.int8_accumulators(d[0], d[2], q)),
                                  oracle.int8_accumulators(cu, cw, qo))
    y = host(f2.wl_matmul(*d, q, xs))
    assert rel_l2(y, oracle.wl_matmul_int8(cu, su, cw, sw, qo, fo)) <= TOL_F32


@pytest.mark.parametrize("B", [1, 3, 9])
def test_mfma_decode_misaligned_activations(gpu, B):
    """Activations whose address is not 16-byte aligned take the element-wise
    load path of the operand preparation; results are bitwise those of an
    aligned copy."""
    import torch
    import paper_2512_02901_amd as f2
    N, K = 48, 320
    A = synth.llama_weight(2 * N, 2 * K, (14, N, K))
    _, _, cu, su, cw, sw = oracle_layer(A, 2)
    d = upload_layer(cu, su, cw, sw, gpu)
    x = synth.activations(B, K, (15, B, K))
    xb = synth.bf16_round_complex(x)
    qo, fo = oracle.quantize_act_int8(x)
    for xa, xs, want in ((bf16_dev(xb, gpu), None, oracle.wl_matmul(cu, su, cw, sw, xb)),
                         (dev(qo, gpu), dev(fo, gpu), oracle.wl_matmul_int8(cu, su, cw, sw, qo, fo))):
        buf = torch.zeros(xa.numel() + 8, dtype=xa.dtype, device=xa.device)
        xm = buf[1:1 + xa.numel()].view(xa.shape)
        xm.copy_(xa)
        assert xm.data_ptr() % 16 != 0
        y0 = host(f2.wl_matmul(*d, xa, xs))
        y1 = host(f2.wl_matmul(*d, xm, xs))
        np.testing.assert_array_equal(y1, y0)
        assert rel_l2(y1, want) <= TOL_F32


def test_prefill_misaligned_activations(gpu):
    """int8 activations at an address that is not 16-byte aligned take the
    element-wise path of the prefill operand preparation: bitwise the same."""
    import torch
    import paper_2512_02901_amd as f2
    N, K, B = 40, 192, 37
    A = synth.llama_weight(2 * N, 2 * K, (18, N, K))
    _, _, cu, su, cw, sw = oracle_layer(A, 2)
    d = upload_layer(cu, su, cw, sw, gpu)
    qo, fo = oracle.quantize_act_int8(synth.activations(B, K, (19, B, K)))
    q, xs = dev(qo, gpu), dev(fo, gpu)
    buf = torch.zeros(q.numel() + 16, dtype=torch.int8, device=gpu)
    qm = buf[5:5 + q.numel()].view(q.shape)
    qm.copy_(q)
    y0 = host(f2.wl_matmul(*d, q, xs))
    np.testing.assert_array_equal(host(f2.wl_matmul(*d, qm, xs)), y0)
    np.testing.assert_array_equal(host(f2.int8_accumulators(d[0], d[2], qm)), oracle.int8_accumulators(cu, cw, qo))
    assert rel_l2(y0, oracle.wl_matmul_int8(cu, su, cw, sw, qo, fo)) <= TOL_F32


def test_mfma_decode_bf16_wide_dynamic_range(gpu):
    """A token whose values span 2^-40 .. 2^3: values more than 2^14 below the
    token's largest magnitude are rounded to its 2^-E grid; the error stays
    far inside the bf16 bar."""
    import paper_2512_02901_amd as f2
    N, K = 32, 256
    A = synth.llama_weight(2 * N, 2 * K, (13, 0, 0))
    _, _, cu, su, cw, sw = oracle_layer(A, 2)
    d = upload_layer(cu, su, cw, sw, gpu)
    rng = np.random.default_rng(13)
    mag = np.exp2(rng.uniform(-40, 3, (1, K))) * np.sign(rng.standard_normal((1, K)))
    x = synth.bf16_round_complex((mag + 1j * mag[:, ::-1]).astype(np.complex64))
    y = host(f2.wl_matmul(*d, bf16_dev(x, gpu)))
    assert rel_l2(y, oracle.wl_matmul(cu, su, cw, sw, x)) <= 1e-5


def test_group_matches_single_layer_calls(gpu):
    """One grouped call over layers of different shapes matches the per-layer
    calls (up to split-K rounding) and the oracle; repeated calls are
    bitwise identical."""
    import torch
    import paper_2512_02901_amd as f2
    shapes = [(128, 256), (200, 64), (48, 1088), (64, 2048)]
    for B, mk in ((1, "bf16"), (4, "bf16"), (11, "i8")):
        layers, refs = [], []
        for i, (N, K) in enumerate(shapes):
            A = synth.llama_weight(2 * N, 2 * K, (14, i, N))
            _, _, cu, su, cw, sw = oracle_layer(A, 2)
            d = upload_layer(cu, su, cw, sw, gpu)
            x = synth.activations(B, K, (15, i, B))
            if mk == "bf16":
                xv = synth.bf16_round_complex(x)
                xd, xs = bf16_dev(xv, gpu), None
                yo = oracle.wl_matmul(cu, su, cw, sw, xv)
            else:
                qo, fo = oracle.quantize_act_int8(x)
                xd, xs = dev(qo, gpu), dev(fo, gpu)
                yo = oracle.wl_matmul_int8(cu, su, cw, sw, qo, fo)
            y = torch.empty((B, N), dtype=torch.complex64, device=gpu)
            layers.append((*d, xd, xs, y))
            refs.append((host(f2.wl_matmul(*d, xd, xs)), yo))
        grp = f2.WlGroup(layers, T=2, B=B)
        grp.run()
        first = [host(l[6]).copy() for l in layers]
        grp.run()   # second call reuses workspace and table: bitwise identical
        for (cu, su, cw, sw, xd, xs, y), (ys, yo), y1 in zip(layers, refs, first):
            np.testing.assert_array_equal(host(y).view(np.uint32), y1.view(np.uint32))
            assert rel_l2(host(y), ys) <= 1e-6     # same products, K possibly sliced differently
            assert rel_l2(host(y), yo) <= TOL_F32


# ------------------------------------------------------ tiled layout ---

def tile_reference(packed, N, K):
    """The tiled decode layout of D3 bytes [T, N, K/4], written out with
    numpy: tile (row block, 256-code step, stage) of 1024 bytes holds, at
    byte 16 (16 g + r) + e, D3 byte 64 s + 16 g + e of row 16 rb + r."""
    T = packed.shape[0]
    nrb, nk4, rowbytes = -(-N // 16), -(-K // 256), K // 4
    pad = np.zeros((T, nrb * 16, nk4 * 64), np.uint8)
    pad[:, :N, :rowbytes] = packed
    a = pad.reshape(T, nrb, 16, nk4, 4, 16)            # t, rb, r, s, g, e
    return np.ascontiguousarray(a.transpose(1, 3, 0, 4, 2, 5)).reshape(-1)


@pytest.mark.parametrize("NKT", [(16, 256, 1), (100, 320, 2), (48, 1088, 3), (37, 100, 2), (5, 4, 4),
                                 (2048, 5504, 2)])
def test_repack_tiled_bit_exact(gpu, NKT):
    """fairy2i_repack_tiled is a byte permutation of D3 with zero padding:
    ragged row blocks, K not a multiple of 256 or of 64 (byte path), and an
    unaligned source."""
    import torch
    import paper_2512_02901_amd as f2
    N, K, T = NKT
    rng = np.random.default_rng(N * 7 + K)
    packed = rng.integers(0, 256, (T, N, K // 4), dtype=np.uint8)
    want = tile_reference(packed, N, K)
    got = host(f2.repack_tiled(dev(packed, gpu)))
    assert got.shape == want.shape == (f2.repack_tiled_bytes(N, K, T),)
    np.testing.assert_array_equal(got, want)
    buf = torch.zeros(packed.size + 16, dtype=torch.uint8, device=gpu)
    src = buf[3:3 + packed.size].view(packed.shape)
    src.copy_(dev(packed, gpu))
    np.testing.assert_array_equal(host(f2.repack_tiled(src)), want)


def test_group_tiled_matches_d3(gpu):
    """A grouped call over tiled copies of the codes gives bitwise the same y
    as over the D3 codes (same kernels and K slicing, other addresses), for
    the streaming (one activation tile) and the register (several tiles)
    product kernels; both match the oracle."""
    import torch
    import paper_2512_02901_amd as f2
    shapes = [(128, 256), (200, 64), (48, 1088), (64, 2048), (37, 5504)]
    for T in (1, 2, 3):
        qlayers = []
        for i, (N, K) in enumerate(shapes):
            _, _, cu, su, cw, sw = oracle_layer(synth.llama_weight(2 * N, 2 * K, (16, i, N)), T)
            d = upload_layer(cu, su, cw, sw, gpu)
            qlayers.append((cu, su, cw, sw, d, (f2.repack_tiled(d[0]), d[1], f2.repack_tiled(d[2]), d[3])))
        for B, mk in ((1, "bf16"), (2, "bf16"), (3, "bf16"), (16, "bf16"), (1, "i8"), (8, "i8"), (9, "i8")):
            d3, tl, refs = [], [], []
            for i, ((N, K), (cu, su, cw, sw, d, dt)) in enumerate(zip(shapes, qlayers)):
                x = synth.activations(B, K, (17, i, B))
                if mk == "bf16":
                    xv = synth.bf16_round_complex(x)
                    xd, xs = bf16_dev(xv, gpu), None
                    yo = oracle.wl_matmul(cu, su, cw, sw, xv)
                else:
                    qo, fo = oracle.quantize_act_int8(x)
                    xd, xs = dev(qo, gpu), dev(fo, gpu)
                    yo = oracle.wl_matmul_int8(cu, su, cw, sw, qo, fo)
                y0 = torch.empty((B, N), dtype=torch.complex64, device=gpu)
                y1 = torch.empty((B, N), dtype=torch.complex64, device=gpu)
                d3.append((*d, xd, xs, y0))
                tl.append((*dt, xd, xs, y1))
                refs.append(yo)
            f2.WlGroup(d3, T=T, B=B).run()
            f2.WlGroup(tl, T=T, B=B, tiled=True).run()
            for a, b, yo in zip(d3, tl, refs):
                np.testing.assert_array_equal(host(b[6]).view(np.uint32), host(a[6]).view(np.uint32))
                assert rel_l2(host(b[6]), yo) <= TOL_F32
