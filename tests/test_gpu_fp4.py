"""GPU parity of the fp4 decode path (codes in the fp4 tiled layout, bf16
activations on the fp8 x fp4 matrix cores) against the CPU oracle.

Bars: the repacked bytes bit-exact against the layout's definition written
out with numpy; y against the oracle within relative L2 TOL_FP4.  The path
scales each token by a power of two so that its largest magnitude m lies in
[2^7, 2^8), splits the scaled values into two magnitude bands (>= 1, and < 1
taken times 2^8) and writes each as an e4m3 digit pair (hi, lo) with
u = hi + 2^-5 lo.  Every value down to 2^-22 m is held exactly.  The matrix
cores multiply the digits exactly and add a group's products with a narrow
adder (bits more than about 2^13 below the group's largest product are
dropped); the bands keep every hi-digit group inside that window, so y
matches the oracle to float32 rounding for any token: measured about 1e-7
for N(0,1) tokens, tokens spread over 2^14 and tokens with 3000-sigma
channels.  TOL_FP4 = 1e-6 leaves a factor 10; the bar for bf16 activations is
1e-3.
"""
import numpy as np
import pytest

import oracle
import synth

pytestmark = pytest.mark.gpu

TOL_FP4 = 1e-6
# Five or more tokens per call (three or more at T = 4): one band of (hi, lo)
# digits per value, four columns per token.  Every bf16 value is still held
# exactly, but the matrix
# core's narrow adder may drop the low bits of a small product that shares
# an MFMA group with one near the token's largest magnitude (at most about
# 2^-13 of that product).  Measured about 4e-6 for N(0,1) tokens and up to
# 1.5e-4 with a 300-sigma channel; TOL_ONE_BAND keeps a factor 2 to the 1e-3
# bar for bf16 activations, TOL_ONE_BAND_TYPICAL applies to N(0,1) tokens.
TOL_ONE_BAND = 5e-4
TOL_ONE_BAND_TYPICAL = 2e-5


def two_bands(B, T):
    """The library's choice: two bands (exact) for up to 2 tokens, and up to
    4 tokens when T <= 3."""
    return B <= 2 or (B <= 4 and T <= 3)


def tol_for(B, typical=False, T=2):
    if two_bands(B, T):
        return TOL_FP4
    return TOL_ONE_BAND_TYPICAL if typical else TOL_ONE_BAND


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


def bf16_dev(x, gpu):
    import torch
    bits = np.stack([synth.bf16_bits(x.real.astype(np.float32)),
                     synth.bf16_bits(x.imag.astype(np.float32))], axis=-1)
    return dev(bits.view(np.int16), gpu).view(torch.bfloat16)


def quantized_layer(N, K, T, key):
    A = synth.llama_weight(2 * N, 2 * K, key)
    U, W = oracle.to_widely_linear(A)
    cu, su = oracle.quantize(U, T)
    cw, sw = oracle.quantize(W, T)
    return cu, su, cw, sw


def fp4_reference(packed, N, K):
    """The fp4 tiled layout of D3 bytes [T, N, K/4], written out from its
    definition: lane (g, r) of tile (rb, s, t) holds codes
    256 s + 128 kb + 32 g + n of row 16 rb + r; n = 16 h + 8 a + m goes to
    word 2 kb + h, nibble m, bits (q, p) at (3, 1) for a = 0, (2, 0) for a = 1."""
    T = packed.shape[0]
    nrb, nk4 = -(-N // 16), -(-K // 256)
    codes = np.zeros((T, nrb * 16, nk4 * 256), np.uint32)
    unpacked = (packed[..., None] >> (2 * np.arange(4, dtype=np.uint8))) & 3   # [T, N, K/4, 4]
    codes[:, :N, :K] = unpacked.reshape(T, N, K)
    p, q = codes & 1, codes >> 1
    out = np.zeros((nrb, nk4, T, 4, 16, 4), np.uint32)          # rb, s, t, g, r, word
    for kb in range(2):
        for n in range(32):
            h, a, m = n // 16, (n // 8) % 2, n % 8
            k = np.arange(nk4)[:, None] * 256 + 128 * kb + 32 * np.arange(4)[None, :] + n   # [s, g]
            pk = p[:, :, k]          # [T, rows, s, g]
            qk = q[:, :, k]
            nib = (qk << 3) | (pk << 1) if a == 0 else (qk << 2) | pk
            nib = nib.reshape(T, nrb, 16, nk4, 4).transpose(1, 3, 0, 4, 2)   # rb, s, t, g, r
            out[..., 2 * kb + h] |= nib << (4 * m)
    return out.astype("<u4").view(np.uint8).reshape(-1)


@pytest.mark.parametrize("NKT", [(16, 256, 1), (100, 320, 2), (48, 1088, 3), (37, 100, 2), (5, 4, 4),
                                 (2048, 5504, 2)])
def test_repack_tiled_fp4_bit_exact(gpu, NKT):
    """fairy2i_repack_tiled_fp4 against the layout's definition: ragged row
    blocks, K not a multiple of 256 or of 32, an unaligned source."""
    import torch
    import paper_2512_02901_amd as f2
    N, K, T = NKT
    rng = np.random.default_rng(N * 11 + K)
    packed = rng.integers(0, 256, (T, N, K // 4), dtype=np.uint8)
    want = fp4_reference(packed, N, K)
    got = host(f2.repack_tiled_fp4(dev(packed, gpu)))
    assert got.shape == want.shape == (f2.repack_tiled_bytes(N, K, T),)
    np.testing.assert_array_equal(got, want)
    buf = torch.zeros(packed.size + 16, dtype=torch.uint8, device=gpu)
    src = buf[3:3 + packed.size].view(packed.shape)
    src.copy_(dev(packed, gpu))
    np.testing.assert_array_equal(host(f2.repack_tiled_fp4(src)), want)


SHAPES = [(128, 256), (200, 64), (48, 1088), (64, 2048), (37, 5504), (1, 64)]


def run_fp4_group(layers, T, B, gpu, x_of):
    """layers: [(N, K, cu, su, cw, sw)]; x_of(i, N, K) -> bf16-exact complex
    activations [B, K].  Returns (y list, oracle list, group)."""
    import torch
    import paper_2512_02901_amd as f2
    args, refs = [], []
    for i, (N, K, cu, su, cw, sw) in enumerate(layers):
        x = x_of(i, N, K)
        d_cu, d_cw = dev(oracle.pack(cu), gpu), dev(oracle.pack(cw), gpu)
        y = torch.empty((B, N), dtype=torch.complex64, device=gpu)
        args.append((f2.repack_tiled_fp4(d_cu), dev(su, gpu), f2.repack_tiled_fp4(d_cw), dev(sw, gpu),
                     bf16_dev(x, gpu), None, y))
        refs.append(oracle.wl_matmul(cu, su, cw, sw, x))
    grp = f2.WlGroup(args, T=T, B=B, layout=f2.LAYOUT_TILED_FP4)
    grp.run()
    return [a[6] for a in args], refs, grp


@pytest.mark.parametrize("T", [1, 2, 3, 4])
def test_group_fp4_matches_oracle(gpu, T):
    """One grouped fp4 call over layers of several shapes (ragged row blocks,
    K with a partial 256-code step, one row), 1 to 16 tokens (two-band tiles
    of 1 or 2 tokens up to 4 tokens at T <= 3, else one-band tiles of 4),
    against the oracle; a repeated
    call is bitwise identical."""
    layers = [(N, K, *quantized_layer(N, K, T, (40, i, N))) for i, (N, K) in enumerate(SHAPES)]
    Bs = {1: (1, 2, 3, 4, 5, 8, 9, 16), 2: (1, 2, 3, 4, 5, 7, 8, 12, 16), 3: (1, 2, 3, 4, 5, 8), 4: (1, 2, 3, 4)}[T]
    for B in Bs:   # B > 4: two tiles (T <= 3); B > 8: four tiles (T <= 2)
        ys, refs, grp = run_fp4_group(layers, T, B, gpu,
                                      lambda i, N, K: synth.bf16_round_complex(synth.activations(B, K, (41, i, B))))
        first = [host(y).copy() for y in ys]
        errs = [rel_l2(host(y), yo) for y, yo in zip(ys, refs)]
        print(f"T={T} B={B} rel-L2 per layer:", " ".join(f"{e:.2e}" for e in errs))
        assert max(errs) <= tol_for(B, typical=True, T=T)
        grp.run()
        for y, y1 in zip(ys, first):
            np.testing.assert_array_equal(host(y).view(np.uint32), y1.view(np.uint32))


def representable_tokens(B, K, key):
    """bf16 tokens whose values all lie within a factor 2^14 of the token's
    largest magnitude (magnitudes in [1, 2^14), random signs): every value is
    represented exactly by its two e4m3 digits."""
    rng = np.random.default_rng(key)
    mag = np.exp2(rng.uniform(0.0, 14.0, (B, K, 2)))
    v = mag * np.where(rng.random((B, K, 2)) < 0.5, -1.0, 1.0)
    return synth.bf16_round_complex((v[..., 0] + 1j * v[..., 1]).astype(np.complex64))


def test_group_fp4_exact_for_representable_tokens(gpu):
    """Tokens spanning 2^14, every value held exactly by its digits: y
    matches the oracle and the int8 tiled path (exact integer products of the
    same values on the int8 matrix cores) to float32 rounding."""
    import torch
    import paper_2512_02901_amd as f2
    T = 2
    layers = [(N, K, *quantized_layer(N, K, T, (42, i, N))) for i, (N, K) in enumerate(SHAPES)]
    for B in (1, 2):
        xs = {}

        def x_of(i, N, K):
            xs[i] = representable_tokens(B, K, 43 * 100 + 10 * i + B)
            return xs[i]
        ys, refs, _ = run_fp4_group(layers, T, B, gpu, x_of)
        errs = [rel_l2(host(y), yo) for y, yo in zip(ys, refs)]
        print(f"B={B} rel-L2 per layer:", " ".join(f"{e:.2e}" for e in errs))
        tol = TOL_FP4
        assert max(errs) <= tol
        # the same products through the int8 matrix cores (tiled layout)
        args = []
        for i, (N, K, cu, su, cw, sw) in enumerate(layers):
            y = torch.empty((B, N), dtype=torch.complex64, device=gpu)
            args.append((f2.repack_tiled(dev(oracle.pack(cu), gpu)), dev(su, gpu),
                         f2.repack_tiled(dev(oracle.pack(cw), gpu)), dev(sw, gpu), bf16_dev(xs[i], gpu), None, y))
        f2.WlGroup(args, T=T, B=B, tiled=True).run()
        for y, a in zip(ys, args):
            assert rel_l2(host(y), host(a[6])) <= tol


@pytest.mark.parametrize("T", [2, 3])
def test_group_fp4_outlier_channels(gpu, T):
    """Tokens of N(0,1) values with one complex channel multiplied by 30, 300
    or 3000 (the crest factors of LLaMA-style activation outliers), at
    K = 2048 and K = 5504, 1 to 16 tokens per call: with two bands (1 to 4
    tokens) every value keeps its own 8 significant bits and y matches to
    float32 rounding; with one band (5 or more tokens) y stays inside the
    bf16 bar with a factor 2 to spare."""
    shapes = [(64, 2048), (48, 5504)]
    layers = [(N, K, *quantized_layer(N, K, T, (49, i, N))) for i, (N, K) in enumerate(shapes)]
    for mult in (30.0, 300.0, 3000.0):
        for B in ((1, 2, 3, 4, 6, 8, 16) if T <= 2 else (1, 2, 3, 4, 6, 8)):
            def x_of(i, N, K):
                x = synth.activations(B, K, (50, i, B, int(mult)))
                rng = np.random.default_rng((51, i, B, int(mult)))
                for b in range(B):
                    x[b, rng.integers(K)] *= np.float32(mult)
                return synth.bf16_round_complex(x)
            ys, refs, _ = run_fp4_group(layers, T, B, gpu, x_of)
            errs = [rel_l2(host(y), yo) for y, yo in zip(ys, refs)]
            print(f"T={T} x{mult:g} B={B} rel-L2:", " ".join(f"{e:.2e}" for e in errs))
            assert max(errs) <= tol_for(B, T=T)


def test_group_fp4_edge_tokens(gpu):
    """A zero token gives y = 0 (and does not disturb its neighbour); a token
    spanning 2^-40 .. 2^3 (its values below 2^-22 m rounded) and a single huge
    or tiny token (scaled without overflow) match to float32 rounding."""
    T = 2
    N, K = 48, 1088
    layer = [(N, K, *quantized_layer(N, K, T, (44, 0, N)))]
    rng = np.random.default_rng(45)
    mag = np.exp2(rng.uniform(-40, 3, (1, K))) * np.sign(rng.standard_normal((1, K)))
    wide = synth.bf16_round_complex((mag + 1j * mag[:, ::-1]).astype(np.complex64))
    normal = synth.bf16_round_complex(synth.activations(1, K, (46,)))
    cases = {
        "zero+normal": np.concatenate([np.zeros((1, K), np.complex64), normal]),
        "wide": wide,
        "huge": synth.bf16_round_complex((normal * np.float32(2.0 ** 100)).astype(np.complex64)),
        "tiny": synth.bf16_round_complex((normal * np.float32(2.0 ** -100)).astype(np.complex64)),
    }
    cases["zero+normal x3"] = np.concatenate([cases["zero+normal"], normal])  # two two-band tiles
    for name, x in cases.items():
        B = x.shape[0]
        ys, refs, _ = run_fp4_group(layer, T, B, gpu, lambda i, N_, K_: x)
        y, yo = host(ys[0]), refs[0]
        err = rel_l2(y, yo)
        print(f"{name}: rel-L2 {err:.2e}")
        assert np.all(np.isfinite(y.view(np.float32)))
        if name.startswith("zero+normal"):
            assert np.all(y[0] == 0)
            assert rel_l2(y[1], yo[1]) <= tol_for(B, typical=True)
        else:
            assert err <= TOL_FP4


def test_group_many_one_step_layers(gpu):
    """Many consecutive one-step work items (K = 64 layers): at T = 1 the load
    side of the streaming kernels runs three items ahead of the output side,
    the deepest their item queue gets.  Both the fp4 and the int8 streaming
    kernel against the oracle, and a repeated call bitwise identical."""
    import torch
    import paper_2512_02901_amd as f2
    T, B = 1, 1
    shapes = [(16 * (1 + i % 3), 64) for i in range(48)] + [(37, 320), (5, 64)]
    layers = [(N, K, *quantized_layer(N, K, T, (47, i, N))) for i, (N, K) in enumerate(shapes)]
    xs = [synth.bf16_round_complex(synth.activations(B, K, (48, i))) for i, (N, K) in enumerate(shapes)]
    ys, refs, grp = run_fp4_group(layers, T, B, gpu, lambda i, N, K: xs[i])
    first = [host(y).copy() for y in ys]
    for y, yo in zip(ys, refs):
        assert rel_l2(host(y), yo) <= TOL_FP4
    grp.run()
    for y, y1 in zip(ys, first):
        np.testing.assert_array_equal(host(y).view(np.uint32), y1.view(np.uint32))
    args = []
    for i, (N, K, cu, su, cw, sw) in enumerate(layers):
        y = torch.empty((B, N), dtype=torch.complex64, device=gpu)
        args.append((f2.repack_tiled(dev(oracle.pack(cu), gpu)), dev(su, gpu),
                     f2.repack_tiled(dev(oracle.pack(cw), gpu)), dev(sw, gpu), bf16_dev(xs[i], gpu), None, y))
    f2.WlGroup(args, T=T, B=B, tiled=True).run()
    for a, yo in zip(args, refs):
        assert rel_l2(host(a[6]), yo) <= 1e-5


def test_coop_kernel_full_k_group(gpu):
    """A group large enough for full-K work items (70 LLaMA-2-7B-shaped
    layers, 13,280 row blocks) with 1 to 16 tokens: the block-cooperative
    kernel (four waves on consecutive row blocks of one layer sharing one
    activation ring; the last groups claimed at run time) against the oracle
    on sampled layers, and a repeated call bitwise identical (which blocks
    take the claimed groups changes from call to call)."""
    import torch
    import paper_2512_02901_amd as f2
    T = 2
    shapes = []
    for layer in range(10):
        for p in synth.PROJ_ORDER:
            rows, cols = synth.LLAMA2_7B_PROJ[p]
            shapes.append((rows // 2, cols // 2))
    assert sum((N + 15) // 16 for N, _ in shapes) >= 12288
    mats = []
    for i, (N, K) in enumerate(shapes):
        A = synth.torch_llama_weight(2 * N, 2 * K, 8000 + i, gpu)
        U, W = f2.to_widely_linear(A)
        cu, su = f2.quantize(U, T)
        cw, sw = f2.quantize(W, T)
        mats.append((N, K, cu, su, cw, sw, f2.repack_tiled_fp4(cu), f2.repack_tiled_fp4(cw)))
        del A, U, W
    # the table lists the 22-step down projections first; the last 35 % of the
    # group steps (2048-wide layers of the last projections) are claimed at
    # run time, so the sample covers both parts
    check = [0, 4, 6, 60, 64, 66, 68, 69]
    for B in (1, 2, 3, 4, 5, 8, 16):
        rng = np.random.default_rng(B)
        args, xs = [], []
        for (N, K, cu, su, cw, sw, cu4, cw4) in mats:
            x = synth.bf16_round_complex((rng.standard_normal((B, K)) + 1j * rng.standard_normal((B, K)))
                                         .astype(np.complex64))
            y = torch.empty((B, N), dtype=torch.complex64, device=gpu)
            args.append((cu4, su, cw4, sw, bf16_dev(x, gpu), None, y))
            xs.append(x)
        grp = f2.WlGroup(args, T=T, B=B, layout=f2.LAYOUT_TILED_FP4)
        grp.run()
        torch.cuda.synchronize()
        first = [host(a[6]).copy() for a in args]
        errs = []
        for i in check:
            N, K, cu, su, cw, sw, _, _ = mats[i]
            want = oracle.wl_matmul(oracle.unpack(host(cu), K), host(su), oracle.unpack(host(cw), K), host(sw), xs[i])
            errs.append(rel_l2(first[i], want))
        print(f"B={B} coop rel-L2:", " ".join(f"{e:.2e}" for e in errs))
        assert max(errs) <= tol_for(B, typical=True)
        grp.run()
        torch.cuda.synchronize()
        for a, y1 in zip(args, first):
            np.testing.assert_array_equal(host(a[6]).view(np.uint32), y1.view(np.uint32))
        del grp, args
