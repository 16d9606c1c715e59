"""fairy2i_wl_matmul_noalloc (the library's own device array as workspace,
nothing allocated) against fairy2i_wl_matmul with a caller workspace: the
same kernels, so y is compared bit for bit.  Each case runs two calls in a
row, the second with a smaller input, so the second call finds the first
call's contents in the shared array."""
import numpy as np
import pytest

import oracle
import synth

pytestmark = pytest.mark.gpu


def host(t):
    return t.detach().cpu().numpy()


def dev(a, gpu):
    import torch
    return torch.from_numpy(np.ascontiguousarray(a)).to(gpu)


def layer(N, K, T, key, gpu):
    A = synth.llama_weight(2 * N, 2 * K, key)
    U, W = oracle.to_widely_linear(A)
    cu, su = oracle.quantize(U, T)
    cw, sw = oracle.quantize(W, T)
    return (dev(oracle.pack(cu), gpu), dev(su, gpu), dev(oracle.pack(cw), gpu), dev(sw, gpu)), (cu, su, cw, sw)


def bf16_dev(x, gpu):
    import torch
    bits = np.stack([synth.bf16_bits(x.real.astype(np.float32)),
                     synth.bf16_bits(x.imag.astype(np.float32))], axis=-1)
    return dev(bits.view(np.int16), gpu).view(torch.bfloat16)


def same_bits(a, b):
    np.testing.assert_array_equal(host(a).view(np.uint32), host(b).view(np.uint32))


@pytest.mark.parametrize("kind", ["bf16_decode", "int8_prefill", "int8_decode", "f32_decode"])
def test_noalloc_matches_wl_matmul(gpu, kind):
    import torch
    import paper_2512_02901_amd as f2
    T = 2
    # (N, K, B): a larger call, then a smaller one on the same array
    shapes = {"bf16_decode": [(2048, 5504, 4), (100, 320, 1)],
              "int8_prefill": [(512, 2048, 600), (48, 1088, 40)],
              "int8_decode": [(1024, 2048, 16), (37, 256, 3)],
              "f32_decode": [(300, 640, 2), (16, 64, 1)]}[kind]
    for i, (N, K, B) in enumerate(shapes):
        d, ref = layer(N, K, T, (61, i, N, K), gpu)
        x = synth.activations(B, K, (62, i, B))
        if kind == "bf16_decode":
            args = (bf16_dev(synth.bf16_round_complex(x), gpu), None)
        elif kind == "f32_decode":
            args = (dev(x, gpu), None)
        else:
            args = f2.quantize_act_int8(dev(x, gpu))
        y_ref = f2.wl_matmul(*d, *args)
        y = torch.full((B, N), float("nan"), dtype=torch.complex64, device=gpu)
        f2.wl_matmul_noalloc(*d, *args, out=y)
        torch.cuda.synchronize()
        same_bits(y, y_ref)
        if i == 0:
            assert f2.wl_matmul_workspace_bytes(N, K, T, B, f2.binding._act_dtype(args[0])) > 0 or kind == "f32_decode"


def test_noalloc_rejects_oversized_workspace(gpu):
    """A call that would need more than the fixed array is refused on the
    host (nothing launched): 4096 int8 tokens at K = 5504."""
    import torch
    import paper_2512_02901_amd as f2
    N, K, B, T = 64, 5504, 4096, 2
    assert f2.wl_matmul_workspace_bytes(N, K, T, B, f2.ACT_I8) > f2.binding.NOALLOC_SCRATCH_BYTES
    codes = torch.zeros((T, N, K // 4), dtype=torch.uint8, device=gpu)
    scales = torch.zeros((T, 2), dtype=torch.float32, device=gpu)
    q = torch.zeros((B, K, 2), dtype=torch.int8, device=gpu)
    xs = torch.zeros((B,), dtype=torch.float32, device=gpu)
    with pytest.raises(f2.Fairy2iError) as e:
        f2.wl_matmul_noalloc(codes, scales, codes, scales, q, xs)
    assert e.value.status == f2.binding.ERR_WORKSPACE
