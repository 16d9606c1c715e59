"""GPU parity of one widely-linear decoder block for one decode token
(fairy2i_block_decode: RMSNorm, grouped fp4 projections, rotary embedding,
Hermitian-score attention over the caches, SwiGLU, residuals) against the
block oracle (oracle/block.py, pinned to the real LLaMA block on the CPU).

Both sides round the inputs of the quantised layers to bf16 at the same four
points.  The GPU computes the values it rounds in float32, the oracle in
float64, so a value within float32 error of a bf16 tie can round either way,
and one such flip perturbs the next stage, which then flips more (at the
LLaMA shape the end-to-end difference reaches about 1e-3).  The parity check
is therefore stage by stage: each stage of the oracle takes the GPU's own
input to that stage (read back with fairy2i_block_intermediates), float
outputs must match within TOL_STAGE, and a bf16 output may differ from the
oracle's rounding only by one step at a near-tie (the oracle's unrounded
value within TOL_TIE times the stage's RMS of the midpoint).  The end-to-end difference is
printed and held to a loose sanity bound.
"""
import numpy as np
import pytest

import oracle
from oracle import block as ob
import synth

pytestmark = pytest.mark.gpu

TOL_STAGE = 1e-6   # float32 stages against float64
TOL_TIE = 1e-5     # how close to a bf16 midpoint a differently rounded value must be
TOL_END = 1e-2     # end-to-end sanity (see the module docstring)


def rel_l2(got, want):
    got = np.asarray(got, dtype=np.complex128)
    want = np.asarray(want, dtype=np.complex128)
    den = np.linalg.norm(want)
    return np.linalg.norm(got - want) / (den if den > 0 else 1.0)


def host(t):
    return t.detach().cpu().numpy()


def dev(a, gpu):
    import torch
    return torch.from_numpy(np.ascontiguousarray(a)).to(gpu)


def shapes(n, f):
    return {"q": (n, n), "k": (n, n), "v": (n, n), "o": (n, n), "gate": (f, n), "up": (f, n), "down": (n, f)}


def cpu_layers(n, f, T, key):
    out = {}
    for i, (name, (N, K)) in enumerate(shapes(n, f).items()):
        A = synth.llama_weight(2 * N, 2 * K, (key, i))
        U, W = oracle.to_widely_linear(A)
        out[name] = (*oracle.quantize(U, T), *oracle.quantize(W, T))
    return {k: (v[0], v[1], v[2], v[3]) for k, v in out.items()}


def gpu_block(layers_cpu, n, f, H, T, max_ctx, gpu, norm_a, norm_m):
    import paper_2512_02901_amd as f2
    dl = {}
    for name, (cu, su, cw, sw) in layers_cpu.items():
        dl[name] = (f2.repack_tiled_fp4(dev(oracle.pack(cu), gpu)), dev(su, gpu),
                    f2.repack_tiled_fp4(dev(oracle.pack(cw), gpu)), dev(sw, gpu))
    return f2.WlBlock(dl, dev(norm_a.astype(np.float32), gpu), dev(norm_m.astype(np.float32), gpu),
                      n=n, n_ff=f, n_heads=H, T=T, max_ctx=max_ctx)


def make_inputs(n, H, max_ctx, pos, key):
    rng = np.random.default_rng(key)
    dc = n // H
    x = (rng.standard_normal((1, n)) + 1j * rng.standard_normal((1, n))).astype(np.complex64)
    norm_a = (1.0 + 0.1 * rng.standard_normal(2 * n)).astype(np.float32)
    norm_m = (1.0 + 0.1 * rng.standard_normal(2 * n)).astype(np.float32)
    kc = np.zeros((H, max_ctx, dc), np.complex64)
    vc = np.zeros((H, max_ctx, dc), np.complex64)
    kc[:, :pos] = (rng.standard_normal((H, pos, dc)) + 1j * rng.standard_normal((H, pos, dc))) * 2
    vc[:, :pos] = rng.standard_normal((H, pos, dc)) + 1j * rng.standard_normal((H, pos, dc))
    return x, norm_a, norm_m, kc, vc


def bf16_check(got, want, what):
    """got: complex bf16 values from the GPU; want: the oracle's unrounded
    values.  Every component equals the oracle's rounding, except one bf16
    step away at a near-tie.  Returns the number of such flips."""
    g = np.concatenate([got.real.ravel(), got.imag.ravel()])
    w = np.concatenate([np.asarray(want).real.ravel(), np.asarray(want).imag.ravel()])
    r = ob.bf16_round(w)
    diff = g != r
    if np.any(diff):
        # float32 error is bounded relative to the stage's magnitude (an
        # element near zero can be a cancelling sum), so the tie distance is too
        scale = np.sqrt(np.mean(w ** 2))
        mid = 0.5 * (g[diff] + r[diff])
        near = np.abs(w[diff] - mid) <= TOL_TIE * scale
        ulp = np.abs(g[diff] - r[diff]) <= np.abs(r[diff]) * 2.0 ** -7
        bad = ~(near & ulp)
        assert not np.any(bad), f"{what}: {int(bad.sum())} components off the oracle's bf16 rounding"
    return int(diff.sum())


def as_complex(t):
    """bf16 [len, 2] or complex64 tensor -> complex128 numpy."""
    import torch
    if t.dtype == torch.bfloat16:
        v = t.float().cpu().numpy().astype(np.float64)
        return v[:, 0] + 1j * v[:, 1]
    return t.cpu().numpy().astype(np.complex128)


def check_stages(blk, layers, x, na, nm, kc_before, kc_after, vc_after, pos, H, y):
    """Every stage of the block against the oracle fed the GPU's input to
    that stage; returns the flips per bf16 point."""
    im = {k: as_complex(v) for k, v in blk.intermediates().items()}
    n = x.shape[-1]
    dc = n // H

    def wl(name, a):
        cu, su, cw, sw = layers[name]
        return oracle.wl_matmul(cu, su, cw, sw, a.reshape(1, -1)).ravel()

    flips = {}
    flips["z"] = bf16_check(im["z"], ob.rms_norm(x, na, 1e-5).ravel(), "z")
    assert rel_l2(im["k"], wl("k", im["z"])) <= TOL_STAGE
    assert rel_l2(im["v"], wl("v", im["z"])) <= TOL_STAGE
    assert rel_l2(im["q_rot"], ob.rope(wl("q", im["z"]).reshape(H, dc), pos, 2 * dc).ravel()) <= TOL_STAGE
    assert rel_l2(kc_after[:, pos], ob.rope(im["k"].reshape(H, dc), pos, 2 * dc)) <= TOL_STAGE
    np.testing.assert_array_equal(vc_after[:, pos], im["v"].reshape(H, dc).astype(np.complex64))
    np.testing.assert_array_equal(kc_after[:, :pos], kc_before[:, :pos])
    o_want = ob.hermitian_attention(im["q_rot"].reshape(H, dc), kc_after, vc_after, pos + 1, 2 * dc)
    flips["o"] = bf16_check(im["o"], o_want.ravel(), "o")
    assert rel_l2(im["a"], wl("o", im["o"])) <= TOL_STAGE
    assert rel_l2(im["h1"], x.ravel() + im["a"]) <= TOL_STAGE
    flips["z2"] = bf16_check(im["z2"], ob.rms_norm(im["h1"].reshape(1, -1), nm, 1e-5).ravel(), "z2")
    assert rel_l2(im["g"], wl("gate", im["z2"])) <= TOL_STAGE
    assert rel_l2(im["u"], wl("up", im["z2"])) <= TOL_STAGE
    act = ob.silu(im["g"].real) * im["u"].real + 1j * (ob.silu(im["g"].imag) * im["u"].imag)
    flips["act"] = bf16_check(im["act"], act, "act")
    assert rel_l2(im["d"], wl("down", im["act"])) <= TOL_STAGE
    assert rel_l2(y.ravel(), im["h1"] + im["d"]) <= TOL_STAGE
    return flips


@pytest.mark.parametrize("pos", [0, 63, 64, 130])
def test_block_small(gpu, pos):
    """n = 256 complex (512 real), 4 heads of 128 real dims, FFN 704 complex,
    T = 2; caches of 200 positions holding `pos` earlier tokens (one, several
    and ragged 64-position attention slices)."""
    n, f, H, T, max_ctx = 256, 704, 4, 2, 200
    layers = cpu_layers(n, f, T, 80)
    x, na, nm, kc, vc = make_inputs(n, H, max_ctx, pos, 81 + pos)
    blk = gpu_block(layers, n, f, H, T, max_ctx, gpu, na, nm)
    dk, dv = dev(kc, gpu), dev(vc, gpu)
    y = host(blk.decode(dev(x, gpu), dk, dv, pos))
    flips = check_stages(blk, layers, x, na, nm, kc, host(dk), host(dv), pos, H, y)
    yo, _, _, _ = ob.block_decode(x, layers, na, nm, kc, vc, pos, H)
    err = rel_l2(y, yo)
    print(f"pos {pos}: end-to-end rel-L2 {err:.2e}, bf16 flips {flips}")
    assert err <= TOL_END
    # a repeated call gives the same bits
    y2 = host(blk.decode(dev(x, gpu), dev(kc, gpu), dev(vc, gpu), pos))
    np.testing.assert_array_equal(y.view(np.uint32), y2.view(np.uint32))


def test_block_token_sequence(gpu):
    """Five tokens decoded one after another from empty caches, each output
    fed back as the next input (the caches grow by one position per call),
    every stage of every call checked."""
    n, f, H, T, max_ctx = 128, 320, 2, 2, 16
    layers = cpu_layers(n, f, T, 82)
    x, na, nm, kc, vc = make_inputs(n, H, max_ctx, 0, 83)
    blk = gpu_block(layers, n, f, H, T, max_ctx, gpu, na, nm)
    dk, dv = dev(kc, gpu), dev(vc, gpu)
    xg = dev(x, gpu)
    for pos in range(5):
        kb = host(dk)
        yg = blk.decode(xg, dk, dv, pos)
        flips = check_stages(blk, layers, host(xg), na, nm, kb, host(dk), host(dv), pos, H, host(yg))
        print(f"token {pos}: bf16 flips {flips}")
        xg = yg.clone()


def test_block_llama_shape(gpu):
    """LLaMA-2-7B block shape: n = 2048 complex (4096 real), 32 heads of 128
    real dims, FFN 5504 complex, T = 2, quantised on the GPU; 1500 cached
    positions of a 2048-position cache."""
    import torch
    import paper_2512_02901_amd as f2
    n, f, H, T, max_ctx, pos = 2048, 5504, 32, 2, 2048, 1500
    dl, cl = {}, {}
    for i, (name, (N, K)) in enumerate(shapes(n, f).items()):
        A = synth.torch_llama_weight(2 * N, 2 * K, 8400 + i, gpu)
        U, W = f2.to_widely_linear(A)
        cu, su = f2.quantize(U, T)
        cw, sw = f2.quantize(W, T)
        dl[name] = (f2.repack_tiled_fp4(cu), su, f2.repack_tiled_fp4(cw), sw)
        cl[name] = (oracle.unpack(host(cu), K), host(su), oracle.unpack(host(cw), K), host(sw))
        del A, U, W
    x, na, nm, kc, vc = make_inputs(n, H, max_ctx, pos, 85)
    blk = f2.WlBlock(dl, dev(na, gpu), dev(nm, gpu), n=n, n_ff=f, n_heads=H, T=T, max_ctx=max_ctx)
    dk, dv = dev(kc, gpu), dev(vc, gpu)
    y = host(blk.decode(dev(x, gpu), dk, dv, pos))
    torch.cuda.synchronize()
    flips = check_stages(blk, cl, x, na, nm, kc, host(dk), host(dv), pos, H, y)
    yo, _, _, _ = ob.block_decode(x, cl, na, nm, kc, vc, pos, H)
    err = rel_l2(y, yo)
    print(f"LLaMA block: end-to-end rel-L2 {err:.2e}, bf16 flips {flips}")
    assert err <= TOL_END


def test_block_general_path_wide_heads(gpu):
    """The unfused path: an FFN of 8256 complex entries, past the fused
    path's 8192 (separate norm, preparation, reduction and SwiGLU kernels),
    with 2 heads of 256 real dims (the attention kernel's wide variant),
    quantised on the GPU; 70 cached positions."""
    import torch
    import paper_2512_02901_amd as f2
    n, f, H, T, max_ctx, pos = 256, 8256, 2, 2, 80, 70
    dl, cl = {}, {}
    for i, (name, (N, K)) in enumerate(shapes(n, f).items()):
        A = synth.torch_llama_weight(2 * N, 2 * K, 8500 + i, gpu)
        U, W = f2.to_widely_linear(A)
        cu, su = f2.quantize(U, T)
        cw, sw = f2.quantize(W, T)
        dl[name] = (f2.repack_tiled_fp4(cu), su, f2.repack_tiled_fp4(cw), sw)
        cl[name] = (oracle.unpack(host(cu), K), host(su), oracle.unpack(host(cw), K), host(sw))
        del A, U, W
    x, na, nm, kc, vc = make_inputs(n, H, max_ctx, pos, 86)
    blk = f2.WlBlock(dl, dev(na, gpu), dev(nm, gpu), n=n, n_ff=f, n_heads=H, T=T, max_ctx=max_ctx)
    dk, dv = dev(kc, gpu), dev(vc, gpu)
    y = host(blk.decode(dev(x, gpu), dk, dv, pos))
    torch.cuda.synchronize()
    flips = check_stages(blk, cl, x, na, nm, kc, host(dk), host(dv), pos, H, y)
    yo, _, _, _ = ob.block_decode(x, cl, na, nm, kc, vc, pos, H)
    err = rel_l2(y, yo)
    print(f"general path: end-to-end rel-L2 {err:.2e}, bf16 flips {flips}")
    assert err <= TOL_END
    y2 = host(blk.decode(dev(x, gpu), dev(kc, gpu), dev(vc, gpu), pos))
    np.testing.assert_array_equal(y.view(np.uint32), y2.view(np.uint32))
