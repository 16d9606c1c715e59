"""Thin ctypes binding of libfairy2i.so (declared in include/fairy2i.h).

Argument marshalling only: torch tensors supply device pointers and the
current HIP stream; every step of the computation runs in the library's
kernels.  There is no fallback: if the library is missing, ``load()`` raises.
"""
from __future__ import annotations

import ctypes
import os

import numpy as np

_LIB_PATH = os.path.join(os.path.dirname(os.path.abspath(__file__)), "libfairy2i.so")
_lib = None

OK, ERR_NULL, ERR_SHAPE, ERR_STAGES, ERR_DTYPE, ERR_UNSUPPORTED, ERR_WORKSPACE, ERR_HIP = range(8)
ACT_F32, ACT_BF16, ACT_I8 = 0, 1, 2
LAYOUT_D3, LAYOUT_TILED, LAYOUT_TILED_FP4 = 0, 1, 2
MAX_STAGES = 4
MAX_DECODE_BATCH = 16

_c_i32, _c_i64, _c_size, _c_p = ctypes.c_int32, ctypes.c_int64, ctypes.c_size_t, ctypes.c_void_p

_SIGNATURES = {
    "fairy2i_status_string": (ctypes.c_char_p, [_c_i32]),
    "fairy2i_abi_version": (_c_i32, []),
    "fairy2i_to_widely_linear": (_c_i32, [_c_p, _c_i64, _c_i64, _c_p, _c_p, _c_p]),
    "fairy2i_quantize_workspace_bytes": (_c_size, [_c_i64, _c_i64, _c_i32]),
    "fairy2i_quantize": (_c_i32, [_c_p, _c_i64, _c_i64, _c_i32, _c_p, _c_p, _c_p, _c_size, _c_p]),
    "fairy2i_quantize_grouped": (_c_i32, [_c_p, _c_i64, _c_i64, _c_i32, _c_i64, _c_p, _c_p, _c_p]),
    "fairy2i_repack_tiled_bytes": (_c_size, [_c_i64, _c_i64, _c_i32]),
    "fairy2i_repack_tiled": (_c_i32, [_c_p, _c_i64, _c_i64, _c_i32, _c_p, _c_size, _c_p]),
    "fairy2i_repack_tiled_fp4": (_c_i32, [_c_p, _c_i64, _c_i64, _c_i32, _c_p, _c_size, _c_p]),
    "fairy2i_quantize_act_int8": (_c_i32, [_c_p, _c_i32, _c_i64, _c_i64, _c_p, _c_p, _c_p]),
    "fairy2i_wl_matmul_workspace_bytes": (_c_size, [_c_i64, _c_i64, _c_i32, _c_i64, _c_i32]),
    "fairy2i_wl_matmul": (_c_i32, [_c_p, _c_p, _c_p, _c_p, _c_i32, _c_i64, _c_i64, _c_p, _c_p,
                                   _c_i32, _c_i64, _c_p, _c_p, _c_size, _c_p]),
    "fairy2i_wl_matmul_noalloc": (_c_i32, [_c_p, _c_p, _c_p, _c_p, _c_i32, _c_i64, _c_i64, _c_p, _c_p,
                                           _c_i32, _c_i64, _c_p, _c_p]),
    "fairy2i_wl_int8_accumulators": (_c_i32, [_c_p, _c_p, _c_i32, _c_i64, _c_i64, _c_p, _c_i64,
                                              _c_p, _c_p, _c_size, _c_p]),
    "fairy2i_host_exact_mean_f32": (_c_i32, [_c_p, _c_i64, _c_p]),
    "fairy2i_wl_group_workspace_bytes": (_c_size, [_c_p, _c_i32, _c_i32, _c_i32, _c_i64]),
    "fairy2i_wl_group_table_bytes": (_c_size, [_c_i32]),
    "fairy2i_wl_group_build_table": (_c_i32, [_c_p, _c_i32, _c_i32, _c_i32, _c_i64, _c_p, _c_size,
                                              _c_p, _c_size]),
    "fairy2i_wl_matmul_group": (_c_i32, [_c_p, _c_p, _c_p]),
    "fairy2i_wl_matmul_group_timed": (_c_i32, [_c_p, _c_p, _c_p, _c_p]),
    "fairy2i_block_workspace_bytes": (_c_size, [_c_p]),
    "fairy2i_block_plan_bytes": (_c_size, [_c_p]),
    "fairy2i_block_build_plan": (_c_i32, [_c_p, _c_p, _c_size, _c_p, _c_size]),
    "fairy2i_block_decode": (_c_i32, [_c_p, _c_p, _c_p, _c_p, _c_p, _c_i64, _c_p, _c_p]),
    "fairy2i_block_intermediates": (_c_i32, [_c_p, _c_p]),
    "fairy2i_qat_fake_quant": (_c_i32, [_c_p, _c_i64, _c_i64, _c_i32, _c_p, _c_p, _c_p, _c_i32, _c_p, _c_size,
                                        _c_p]),
    "fairy2i_qat_ste_workspace_bytes": (_c_size, [_c_i64, _c_i64]),
    "fairy2i_qat_ste_backward": (_c_i32, [_c_p, _c_p, _c_i32, _c_i64, _c_i64, _c_p, _c_p, _c_p, _c_size, _c_p]),
    "fairy2i_cgemm_gauss": (_c_i32, [_c_p, _c_p, _c_p, _c_i32, _c_i64, _c_i64, _c_p, _c_i64, _c_i32, _c_p]),
    "fairy2i_cgemm_gauss_planar_workspace_bytes": (_c_size, [_c_p, _c_i32, _c_i64, _c_i64]),
    "fairy2i_cgemm_gauss_planar": (_c_i32, [_c_p, _c_p, _c_p, _c_i32, _c_i64, _c_i64, _c_p, _c_i64, _c_i32, _c_p,
                                            _c_size, _c_p]),
    "fairy2i_probe_mfma": (_c_i32, [_c_i32, _c_i32, _c_i32, _c_p, _c_p, _c_p]),
    "fairy2i_wl_realify": (_c_i32, [_c_p, _c_p, _c_i32, _c_i64, _c_i64, _c_p, _c_p]),
    "fairy2i_wl_realify_codes": (_c_i32, [_c_p, _c_p, _c_p, _c_p, _c_i32, _c_i64, _c_i64, _c_p, _c_p]),
    "fairy2i_wl_unrealify_grad": (_c_i32, [_c_p, _c_i64, _c_i64, _c_p, _c_p, _c_p]),
    "fairy2i_f32_to_bf16": (_c_i32, [_c_p, _c_i64, _c_p, _c_p]),
    "fairy2i_gemm_bf16_workspace_bytes": (_c_size, []),
    "fairy2i_gemm_bf16_tune": (_c_i32, [_c_p, _c_i64, _c_i32, _c_p, _c_i64, _c_i32, _c_i64, _c_i64, _c_i64, _c_p,
                                        _c_i64, _c_p, _c_size, _c_p, _c_p]),
    "fairy2i_gemm_bf16": (_c_i32, [_c_p, _c_i64, _c_i32, _c_p, _c_i64, _c_i32, _c_i64, _c_i64, _c_i64, _c_p, _c_i64,
                                   _c_p, _c_size, _c_p]),
    "fairy2i_cpu_lut_workspace_bytes": (_c_size, [_c_i32, _c_i64, _c_i64, _c_i32]),
    "fairy2i_cpu_lut_wl_matmul": (_c_i32, [_c_p, _c_p, _c_p, _c_p, _c_i32, _c_i64, _c_i64, _c_p, _c_p, _c_i64,
                                           _c_p, _c_p, _c_p, _c_size, _c_i32]),
}


class WlLayer(ctypes.Structure):
    """fairy2i_wl_layer of include/fairy2i.h."""
    _fields_ = [("codes_U", _c_p), ("scales_U", _c_p), ("codes_W", _c_p), ("scales_W", _c_p),
                ("x", _c_p), ("x_scale", _c_p), ("y", _c_p), ("N", _c_i64), ("K", _c_i64),
                ("layout", _c_i32), ("group_size", _c_i32)]


class CgemmOperand(ctypes.Structure):
    """fairy2i_cgemm_operand of include/fairy2i.h."""
    _fields_ = [("data", _c_p), ("ld", _c_i64), ("dtype", _c_i32), ("trans", _c_i32), ("conj", _c_i32),
                ("reserved", _c_i32)]


class BlockDesc(ctypes.Structure):
    """fairy2i_block_desc of include/fairy2i.h."""
    _fields_ = [("n", _c_i64), ("n_ff", _c_i64), ("n_heads", _c_i32), ("T", _c_i32), ("max_ctx", _c_i64),
                ("eps", ctypes.c_float), ("reserved", _c_i32), ("rope_base", ctypes.c_double),
                ("codes_U", _c_p * 7), ("scales_U", _c_p * 7), ("codes_W", _c_p * 7), ("scales_W", _c_p * 7),
                ("norm_attn", _c_p), ("norm_mlp", _c_p)]


class Fairy2iError(RuntimeError):
    def __init__(self, status: int, where: str):
        self.status = status
        msg = _lib.fairy2i_status_string(status).decode() if _lib is not None else str(status)
        super().__init__(f"{where}: status {status} ({msg})")


def lib_path() -> str:
    return _LIB_PATH


def load():
    """Load libfairy2i.so (once).  Raises if it has not been built."""
    global _lib
    if _lib is None:
        if not os.path.exists(_LIB_PATH):
            raise RuntimeError(f"{_LIB_PATH} is missing: build it with "
                               "`python -m paper_2512_02901_amd.build`")
        lib = ctypes.CDLL(_LIB_PATH)
        for name, (res, args) in _SIGNATURES.items():
            fn = getattr(lib, name)
            fn.restype = res
            fn.argtypes = args
        _lib = lib
    return _lib


def _check(status: int, where: str):
    if status != OK:
        raise Fairy2iError(status, where)


# --------------------------------------------------------------- helpers ---

def _torch():
    import torch
    return torch


def _stream_ptr(tensor) -> int:
    torch = _torch()
    return torch.cuda.current_stream(tensor.device).cuda_stream


def _ptr(t):
    return None if t is None else ctypes.c_void_p(t.data_ptr())


def _require(t, dtype, name, device=None):
    torch = _torch()
    if not isinstance(t, torch.Tensor):
        raise TypeError(f"{name} must be a torch.Tensor")
    if not t.is_cuda:
        raise ValueError(f"{name} must be a device tensor")
    if dtype is not None and t.dtype != dtype:
        raise TypeError(f"{name} must be {dtype}, got {t.dtype}")
    if not t.is_contiguous():
        raise ValueError(f"{name} must be contiguous")
    if device is not None and t.device != device:
        raise ValueError(f"{name} is on {t.device}, expected {device}")


# ------------------------------------------------------------------ API ---

def wl_realify(U, W, out=None):
    """U, W: [N, K] complex64 or bf16 [N, K, 2] device tensors -> R: bf16
    [2N, 2K], the layer's real map with (re, im) rows and columns
    interleaved (fairy2i_wl_realify; out: such a tensor to write)."""
    torch = _torch()
    lib = load()
    if U.dtype == torch.complex64:
        dt = ACT_F32
        N, K = U.shape
    else:
        dt = ACT_BF16
        N, K = U.shape[0], U.shape[1]
    for t, n in ((U, "U"), (W, "W")):
        _require(t, U.dtype, n, U.device)
        if t.shape != U.shape or (dt == ACT_BF16 and (t.dim() != 3 or t.shape[2] != 2 or t.dtype != torch.bfloat16)):
            raise ValueError(f"{n} must be [N, K] complex64 or [N, K, 2] bf16")
    R = torch.empty((2 * N, 2 * K), dtype=torch.bfloat16, device=U.device) if out is None else out
    _require(R, torch.bfloat16, "out", U.device)
    if tuple(R.shape) != (2 * N, 2 * K):
        raise ValueError("out must be [2N, 2K]")
    _check(lib.fairy2i_wl_realify(_ptr(U), _ptr(W), dt, N, K, _ptr(R), _stream_ptr(U)), "fairy2i_wl_realify")
    return R


def wl_realify_codes(codes_U, scales_U, codes_W, scales_W, out=None):
    """The layer's real map R (bf16 [2N, 2K]) straight from the quantised
    pair: canonical codes uint8 [T, N, K/4] and scales float32 [T, 2] of U
    and of W (fairy2i_wl_realify_codes)."""
    torch = _torch()
    lib = load()
    _require(codes_U, torch.uint8, "codes_U")
    T, N, K4 = codes_U.shape
    d = codes_U.device
    _require(codes_W, torch.uint8, "codes_W", d)
    for t, n in ((scales_U, "scales_U"), (scales_W, "scales_W")):
        _require(t, torch.float32, n, d)
        if tuple(t.shape) != (T, 2):
            raise ValueError(f"{n} must be [T, 2]")
    if tuple(codes_W.shape) != (T, N, K4):
        raise ValueError("codes_W must match codes_U")
    K = 4 * K4
    R = torch.empty((2 * N, 2 * K), dtype=torch.bfloat16, device=d) if out is None else out
    _require(R, torch.bfloat16, "out", d)
    if tuple(R.shape) != (2 * N, 2 * K):
        raise ValueError("out must be [2N, 2K]")
    _check(lib.fairy2i_wl_realify_codes(_ptr(codes_U), _ptr(scales_U), _ptr(codes_W), _ptr(scales_W), T, N, K,
                                        _ptr(R), _stream_ptr(codes_U)), "fairy2i_wl_realify_codes")
    return R


def wl_unrealify_grad(G_R, N, K, out=None):
    """G_R: float32 [2N, 2K] -> (G_U, G_W) complex64 [N, K] (out: a pair
    of such tensors to write)."""
    torch = _torch()
    lib = load()
    _require(G_R, torch.float32, "G_R")
    if tuple(G_R.shape) != (2 * N, 2 * K):
        raise ValueError("G_R must be [2N, 2K]")
    if out is None:
        G_U = torch.empty((N, K), dtype=torch.complex64, device=G_R.device)
        G_W = torch.empty_like(G_U)
    else:
        G_U, G_W = out
        for t, n in ((G_U, "G_U"), (G_W, "G_W")):
            _require(t, torch.complex64, n, G_R.device)
            if tuple(t.shape) != (N, K):
                raise ValueError(f"{n} must be [N, K]")
    _check(lib.fairy2i_wl_unrealify_grad(_ptr(G_R), N, K, _ptr(G_U), _ptr(G_W), _stream_ptr(G_R)),
           "fairy2i_wl_unrealify_grad")
    return G_U, G_W


def f32_to_bf16(x, out=None):
    """float32 (or complex64, as its float pairs) device tensor -> bf16 of
    the same number of values, nearest even; complex input gives [..., 2]."""
    torch = _torch()
    lib = load()
    _require(x, None, "x")
    xf = torch.view_as_real(x) if x.dtype == torch.complex64 else x
    if xf.dtype != torch.float32:
        raise TypeError("x must be float32 or complex64")
    if out is None:
        out = torch.empty(xf.shape, dtype=torch.bfloat16, device=x.device)
    _require(out, torch.bfloat16, "out", x.device)
    if out.numel() != xf.numel():
        raise ValueError("out must hold as many values as x")
    _check(lib.fairy2i_f32_to_bf16(ctypes.c_void_p(xf.data_ptr()), xf.numel(), _ptr(out), _stream_ptr(x)),
           "fairy2i_f32_to_bf16")
    return out


def gemm_bf16(A, B, transA=False, transB=False, out=None, workspace=None, tune=False):
    """C (float32 M x N) = op(A) op(B) for bf16 row-major 2-D device tensors
    (fairy2i_gemm_bf16); op(X) is X or X^T.  tune=True first times the
    library's candidate algorithms for this problem (fairy2i_gemm_bf16_tune,
    which synchronises) and keeps the fastest."""
    torch = _torch()
    lib = load()
    _require(A, torch.bfloat16, "A")
    _require(B, torch.bfloat16, "B", A.device)
    if A.dim() != 2 or B.dim() != 2:
        raise ValueError("A and B must be 2-D")
    M, K = (A.shape[1], A.shape[0]) if transA else (A.shape[0], A.shape[1])
    Kb, N = (B.shape[1], B.shape[0]) if transB else (B.shape[0], B.shape[1])
    if Kb != K:
        raise ValueError("inner dimensions differ")
    if out is None:
        out = torch.empty((M, N), dtype=torch.float32, device=A.device)
    _require(out, torch.float32, "out", A.device)
    if tuple(out.shape) != (M, N):
        raise ValueError("out must be M x N")
    ws, wsb = _workspace(lib.fairy2i_gemm_bf16_workspace_bytes(), workspace, A.device)
    if tune:
        _check(lib.fairy2i_gemm_bf16_tune(_ptr(A), A.shape[1], int(transA), _ptr(B), B.shape[1], int(transB), M, N,
                                          K, _ptr(out), N, _ptr(ws), wsb, None, _stream_ptr(A)),
               "fairy2i_gemm_bf16_tune")
    _check(lib.fairy2i_gemm_bf16(_ptr(A), A.shape[1], int(transA), _ptr(B), B.shape[1], int(transB), M, N, K,
                                 _ptr(out), N, _ptr(ws), wsb, _stream_ptr(A)), "fairy2i_gemm_bf16")
    return out


PROBE_MFMA_I8 = 0    # v_mfma_i32_16x16x64_i8 (the prefill GEMM's instruction)
PROBE_MFMA_F8F4 = 1  # v_mfma_scale_f32_16x16x128_f8f6f4, e4m3 x e2m1 (the decode product's)
PROBE_MFMA_I8_32X32 = 2  # v_mfma_i32_32x32x32_i8


def probe_mfma(kind: int, blocks: int, iters: int, sink) -> float:
    """Launch the matrix-core rate probe on the current stream of sink's
    device (sink: int32 device tensor of at least blocks * 256 words);
    returns the operations of the launch, for the caller to time."""
    torch = _torch()
    lib = load()
    _require(sink, torch.int32, "sink")
    if sink.numel() < blocks * 256:
        raise ValueError("sink needs blocks * 256 words")
    ops = ctypes.c_double()
    _check(lib.fairy2i_probe_mfma(kind, blocks, iters, _ptr(sink), ctypes.byref(ops), _stream_ptr(sink)),
           "fairy2i_probe_mfma")
    return ops.value


def to_widely_linear(A):
    """A: float32 [2N, 2K] device tensor -> (U, W) complex64 [N, K]."""
    torch = _torch()
    lib = load()
    _require(A, torch.float32, "A")
    rows, cols = A.shape
    U = torch.empty((rows // 2, cols // 2), dtype=torch.complex64, device=A.device)
    W = torch.empty_like(U)
    _check(lib.fairy2i_to_widely_linear(_ptr(A), rows, cols, _ptr(U), _ptr(W), _stream_ptr(A)),
           "fairy2i_to_widely_linear")
    return U, W


def quantize(M, T: int):
    """M: complex64 [N, K] -> (codes uint8 [T, N, K/4], scales float32 [T, 2])."""
    torch = _torch()
    lib = load()
    _require(M, torch.complex64, "M")
    N, K = M.shape
    codes = torch.empty((T, N, K // 4), dtype=torch.uint8, device=M.device)
    scales = torch.empty((T, 2), dtype=torch.float32, device=M.device)
    wsb = lib.fairy2i_quantize_workspace_bytes(N, K, T)
    ws = torch.empty(max(int(wsb), 1), dtype=torch.uint8, device=M.device)
    _check(lib.fairy2i_quantize(_ptr(M), N, K, T, _ptr(codes), _ptr(scales), _ptr(ws), wsb,
                                _stream_ptr(M)), "fairy2i_quantize")
    return codes, scales


def quantize_grouped(M, T: int, G: int):
    """M: complex64 [N, K] -> (codes uint8 [T, N, K/4], scales float32
    [T, N, ceil(K/G), 2]): one pair of axis scales per group of G input
    columns of a row."""
    torch = _torch()
    lib = load()
    _require(M, torch.complex64, "M")
    N, K = M.shape
    ng = -(-K // G) if G > 0 else 0
    codes = torch.empty((T, N, K // 4), dtype=torch.uint8, device=M.device)
    scales = torch.empty((T, N, max(ng, 1), 2), dtype=torch.float32, device=M.device)
    _check(lib.fairy2i_quantize_grouped(_ptr(M), N, K, T, G, _ptr(codes), _ptr(scales), _stream_ptr(M)),
           "fairy2i_quantize_grouped")
    return codes, scales


def _act_dtype(x):
    torch = _torch()
    if x.dtype == torch.complex64:
        return ACT_F32
    if x.dtype == torch.bfloat16:
        return ACT_BF16
    if x.dtype == torch.int8:
        return ACT_I8
    raise TypeError(f"unsupported activation dtype {x.dtype}")


def _act_shape(x):
    """(B, K) of an activation tensor: complex64 [B, K] or bf16/int8 [B, K, 2]."""
    if x.dim() == 2:
        return x.shape[0], x.shape[1]
    if x.dim() == 3 and x.shape[2] == 2:
        return x.shape[0], x.shape[1]
    raise ValueError("activations must be complex64 [B, K] or bf16/int8 [B, K, 2]")


def quantize_act_int8(x):
    """x: complex64 [B, K] or bf16 [B, K, 2] -> (q int8 [B, K, 2], x_scale float32 [B])."""
    torch = _torch()
    lib = load()
    _require(x, None, "x")
    dt = _act_dtype(x)
    B, K = _act_shape(x)
    q = torch.empty((B, K, 2), dtype=torch.int8, device=x.device)
    xs = torch.empty((B,), dtype=torch.float32, device=x.device)
    _check(lib.fairy2i_quantize_act_int8(_ptr(x), dt, B, K, _ptr(q), _ptr(xs), _stream_ptr(x)),
           "fairy2i_quantize_act_int8")
    return q, xs


def wl_matmul_workspace_bytes(N, K, T, B, dtype) -> int:
    return int(load().fairy2i_wl_matmul_workspace_bytes(N, K, T, B, dtype))


def wl_matmul(codes_U, scales_U, codes_W, scales_W, x, x_scale=None, out=None, workspace=None):
    """y = sum_t U^(t) x + W^(t) conj(x) for each token; complex64 [B, N]."""
    torch = _torch()
    lib = load()
    for t, n in ((codes_U, "codes_U"), (codes_W, "codes_W")):
        _require(t, torch.uint8, n)
    for t, n in ((scales_U, "scales_U"), (scales_W, "scales_W")):
        _require(t, torch.float32, n)
    _require(x, None, "x")
    T, N, KB = codes_U.shape
    if codes_W.shape != codes_U.shape or scales_U.shape != (T, 2) or scales_W.shape != (T, 2):
        raise ValueError("codes/scales shapes disagree")
    dt = _act_dtype(x)
    B, K = _act_shape(x)
    if K != 4 * KB:
        raise ValueError(f"activations have K={K}, codes have K={4 * KB}")
    dev_ = x.device
    for t, n in ((codes_U, "codes_U"), (codes_W, "codes_W"), (scales_U, "scales_U"), (scales_W, "scales_W")):
        _require(t, None, n, dev_)
    if x_scale is not None:
        _require(x_scale, torch.float32, "x_scale", dev_)
        if tuple(x_scale.shape) != (B,):
            raise ValueError(f"x_scale must have shape ({B},), got {tuple(x_scale.shape)}")
    if out is None:
        out = torch.empty((B, N), dtype=torch.complex64, device=dev_)
    else:
        _require(out, torch.complex64, "out", dev_)
        if tuple(out.shape) != (B, N):
            raise ValueError(f"out must have shape ({B}, {N}), got {tuple(out.shape)}")
    workspace, wsb = _workspace(lib.fairy2i_wl_matmul_workspace_bytes(N, K, T, B, dt), workspace, dev_)
    _check(lib.fairy2i_wl_matmul(_ptr(codes_U), _ptr(scales_U), _ptr(codes_W), _ptr(scales_W), T, N, K,
                                 _ptr(x), _ptr(x_scale), dt, B, _ptr(out), _ptr(workspace), wsb,
                                 _stream_ptr(x)), "fairy2i_wl_matmul")
    return out


NOALLOC_SCRATCH_BYTES = 32 << 20


def wl_matmul_noalloc(codes_U, scales_U, codes_W, scales_W, x, x_scale=None, out=None):
    """wl_matmul without a workspace: the library's fixed device array
    (NOALLOC_SCRATCH_BYTES per GPU) serves as one; allocates nothing when
    ``out`` is given.  Calls that overlap on one GPU race."""
    torch = _torch()
    lib = load()
    for t, n in ((codes_U, "codes_U"), (codes_W, "codes_W")):
        _require(t, torch.uint8, n, x.device)
    for t, n in ((scales_U, "scales_U"), (scales_W, "scales_W")):
        _require(t, torch.float32, n, x.device)
    _require(x, None, "x")
    T, N, KB = codes_U.shape
    if codes_W.shape != codes_U.shape or scales_U.shape != (T, 2) or scales_W.shape != (T, 2):
        raise ValueError("codes/scales shapes disagree")
    dt = _act_dtype(x)
    B, K = _act_shape(x)
    if K != 4 * KB:
        raise ValueError(f"activations have K={K}, codes have K={4 * KB}")
    if x_scale is not None:
        _require(x_scale, torch.float32, "x_scale", x.device)
        if tuple(x_scale.shape) != (B,):
            raise ValueError(f"x_scale must have shape ({B},), got {tuple(x_scale.shape)}")
    if out is None:
        out = torch.empty((B, N), dtype=torch.complex64, device=x.device)
    else:
        _require(out, torch.complex64, "out", x.device)
        if tuple(out.shape) != (B, N):
            raise ValueError(f"out must have shape ({B}, {N}), got {tuple(out.shape)}")
    _check(lib.fairy2i_wl_matmul_noalloc(_ptr(codes_U), _ptr(scales_U), _ptr(codes_W), _ptr(scales_W), T, N, K,
                                         _ptr(x), _ptr(x_scale), dt, B, _ptr(out), _stream_ptr(x)),
           "fairy2i_wl_matmul_noalloc")
    return out


def _workspace(need, workspace, device):
    """(workspace tensor or None, its size in bytes): a fresh uint8 device
    buffer of `need` bytes when none is given, else the caller's, checked."""
    torch = _torch()
    need = int(need)
    if workspace is None:
        if need == 0:
            return None, 0
        workspace = torch.empty(need, dtype=torch.uint8, device=device)
    _require(workspace, torch.uint8, "workspace", device)
    return workspace, workspace.numel()


def repack_tiled_bytes(N, K, T) -> int:
    return int(load().fairy2i_repack_tiled_bytes(N, K, T))


def _repack(fn, codes, out):
    torch = _torch()
    lib = load()
    _require(codes, torch.uint8, "codes")
    T, N, KB = codes.shape
    nb = repack_tiled_bytes(N, 4 * KB, T)
    if out is None:
        out = torch.empty(nb, dtype=torch.uint8, device=codes.device)
    else:
        _require(out, torch.uint8, "out")
    _check(getattr(lib, fn)(_ptr(codes), N, 4 * KB, T, _ptr(out), out.numel(), _stream_ptr(codes)), fn)
    return out


def repack_tiled(codes, out=None):
    """D3 codes [T, N, K/4] -> the tiled decode layout (1-D uint8 tensor of
    fairy2i_repack_tiled_bytes bytes)."""
    return _repack("fairy2i_repack_tiled", codes, out)


def repack_tiled_fp4(codes, out=None):
    """D3 codes [T, N, K/4] -> the fp4 tiled decode layout (1-D uint8 tensor
    of fairy2i_repack_tiled_bytes bytes)."""
    return _repack("fairy2i_repack_tiled_fp4", codes, out)


def int8_accumulators(codes_U, codes_W, q, workspace=None):
    """Exact int32 products acc[M][t][p][b][i][c] behind the int8 path."""
    torch = _torch()
    lib = load()
    _require(codes_U, torch.uint8, "codes_U")
    _require(codes_W, torch.uint8, "codes_W")
    _require(q, torch.int8, "q")
    T, N, KB = codes_U.shape
    B, K = _act_shape(q)
    if K != 4 * KB:
        raise ValueError("K mismatch")
    _require(codes_W, None, "codes_W", q.device)
    _require(codes_U, None, "codes_U", q.device)
    if codes_W.shape != codes_U.shape:
        raise ValueError("codes_U and codes_W shapes disagree")
    acc = torch.empty((2, T, 2, B, N, 2), dtype=torch.int32, device=q.device)
    workspace, wsb = _workspace(lib.fairy2i_wl_matmul_workspace_bytes(N, K, T, B, ACT_I8), workspace, q.device)
    _check(lib.fairy2i_wl_int8_accumulators(_ptr(codes_U), _ptr(codes_W), T, N, K, _ptr(q), B,
                                            _ptr(acc), _ptr(workspace), wsb, _stream_ptr(q)),
           "fairy2i_wl_int8_accumulators")
    return acc


def host_exact_mean_f32(values) -> np.float32:
    """Host-side self-check of the scale rounding (no GPU involved)."""
    lib = load()
    v = np.ascontiguousarray(values, dtype=np.float64)
    out = ctypes.c_float(0.0)
    _check(lib.fairy2i_host_exact_mean_f32(v.ctypes.data_as(ctypes.c_void_p), v.size,
                                           ctypes.byref(out)), "fairy2i_host_exact_mean_f32")
    return np.float32(out.value)


def qat_fake_quant(M, T: int, out_dtype: int = ACT_BF16):
    """Fake-quant forward of a complex64 master [N, K]: (W^, codes, scales);
    W^ is bf16 pairs [N, K, 2] (ACT_BF16) or complex64 [N, K] (ACT_F32)."""
    torch = _torch()
    lib = load()
    _require(M, torch.complex64, "M")
    N, K = M.shape
    codes = torch.empty((T, N, K // 4), dtype=torch.uint8, device=M.device)
    scales = torch.empty((T, 2), dtype=torch.float32, device=M.device)
    if out_dtype == ACT_BF16:
        w_hat = torch.empty((N, K, 2), dtype=torch.bfloat16, device=M.device)
    else:
        w_hat = torch.empty((N, K), dtype=torch.complex64, device=M.device)
    wsb = lib.fairy2i_quantize_workspace_bytes(N, K, T)
    ws = torch.empty(max(int(wsb), 1), dtype=torch.uint8, device=M.device)
    _check(lib.fairy2i_qat_fake_quant(_ptr(M), N, K, T, _ptr(codes), _ptr(scales), _ptr(w_hat), out_dtype, _ptr(ws),
                                      wsb, _stream_ptr(M)), "fairy2i_qat_fake_quant")
    return w_hat, codes, scales


def qat_ste_backward(codes, scales, g_hat):
    """dL/dM from dL/dW^ (complex64 [N, K]) through the fake quantiser."""
    torch = _torch()
    lib = load()
    _require(g_hat, torch.complex64, "g_hat")
    N, K = g_hat.shape
    T = codes.shape[0]
    _require(codes, torch.uint8, "codes", g_hat.device)
    _require(scales, torch.float32, "scales", g_hat.device)
    if tuple(codes.shape) != (T, N, K // 4) or tuple(scales.shape) != (T, 2):
        raise ValueError("codes [T, N, K/4] and scales [T, 2] must match g_hat")
    out = torch.empty_like(g_hat)
    wsb = lib.fairy2i_qat_ste_workspace_bytes(N, K)
    ws = torch.empty(max(int(wsb), 1), dtype=torch.uint8, device=g_hat.device)
    _check(lib.fairy2i_qat_ste_backward(_ptr(codes), _ptr(scales), T, N, K, _ptr(g_hat), _ptr(out), _ptr(ws), wsb,
                                        _stream_ptr(g_hat)), "fairy2i_qat_ste_backward")
    return out


def _cgemm_operand(t, trans, conj, rows, K, name):
    """A complex operand tensor: complex64 [a, b] or bf16 pairs [a, b, 2],
    contiguous; [rows, K] when trans == 0, [K, rows] when trans == 1."""
    torch = _torch()
    _require(t, None, name)
    if t.dtype == torch.complex64 and t.dim() == 2:
        dt = ACT_F32
    elif t.dtype == torch.bfloat16 and t.dim() == 3 and t.shape[2] == 2:
        dt = ACT_BF16
    else:
        raise TypeError(f"{name} must be complex64 [a, b] or bf16 [a, b, 2]")
    want = (K, rows) if trans else (rows, K)
    if tuple(t.shape[:2]) != want:
        raise ValueError(f"{name} has shape {tuple(t.shape[:2])}, expected {want}")
    return CgemmOperand(t.data_ptr(), t.shape[1], dt, int(trans), int(conj), 0)


def cgemm_gauss_planar_workspace_bytes(Ks, M: int, N: int) -> int:
    k = (ctypes.c_int64 * 2)(*(list(Ks) + [0] * (2 - len(Ks))))
    return int(load().fairy2i_cgemm_gauss_planar_workspace_bytes(ctypes.byref(k), len(Ks), M, N))


def cgemm_gauss(segments, M: int, N: int, out=None, accumulate: bool = False, planar: bool = False,
                workspace=None):
    """C [M, N] complex64 (+)= sum over segments of op(A) op(B)^T with
    Gauss's three real products.  segments: up to two tuples
    (A, a_trans, a_conj, B, b_trans, b_conj, K); see _cgemm_operand.
    planar: bf16 planes and one batched library GEMM
    (fairy2i_cgemm_gauss_planar, with a uint8 device workspace of
    cgemm_gauss_planar_workspace_bytes, allocated here when not given);
    else the single-kernel fairy2i_cgemm_gauss."""
    torch = _torch()
    lib = load()
    if not 1 <= len(segments) <= 2:
        raise ValueError("one or two segments")
    dev = segments[0][0].device
    A = (CgemmOperand * 2)()
    Bo = (CgemmOperand * 2)()
    Ks = (ctypes.c_int64 * 2)()
    for i, (a, at, ac, b, bt, bc, K) in enumerate(segments):
        A[i] = _cgemm_operand(a, at, ac, M, K, f"segments[{i}].A")
        Bo[i] = _cgemm_operand(b, bt, bc, N, K, f"segments[{i}].B")
        Ks[i] = K
    if out is None:
        out = torch.zeros((M, N), dtype=torch.complex64, device=dev) if accumulate else \
            torch.empty((M, N), dtype=torch.complex64, device=dev)
    _require(out, torch.complex64, "out", dev)
    if tuple(out.shape) != (M, N):
        raise ValueError(f"out must have shape ({M}, {N})")
    if not planar:
        _check(lib.fairy2i_cgemm_gauss(ctypes.byref(A), ctypes.byref(Bo), ctypes.byref(Ks), len(segments), M, N,
                                       _ptr(out), N, int(accumulate), _stream_ptr(out)), "fairy2i_cgemm_gauss")
        return out
    need = int(lib.fairy2i_cgemm_gauss_planar_workspace_bytes(ctypes.byref(Ks), len(segments), M, N))
    if workspace is None:
        workspace = torch.empty(max(need, 1), dtype=torch.uint8, device=dev)
    _require(workspace, torch.uint8, "workspace", dev)
    _check(lib.fairy2i_cgemm_gauss_planar(ctypes.byref(A), ctypes.byref(Bo), ctypes.byref(Ks), len(segments), M, N,
                                          _ptr(out), N, int(accumulate), _ptr(workspace),
                                          workspace.numel(), _stream_ptr(out)), "fairy2i_cgemm_gauss_planar")
    return out


def _host(a, dtype, name, shape=None):
    """A C-contiguous numpy view of a host array or CPU tensor, checked."""
    if hasattr(a, "is_cuda"):
        if a.is_cuda:
            raise ValueError(f"{name} must be host memory")
        a = a.numpy()
    if not isinstance(a, np.ndarray) or a.dtype != dtype or not a.flags.c_contiguous:
        raise TypeError(f"{name} must be a C-contiguous {np.dtype(dtype).name} array")
    if shape is not None and a.shape != tuple(shape):
        raise ValueError(f"{name} has shape {a.shape}, expected {tuple(shape)}")
    return a


def _hp(a):
    return None if a is None else a.ctypes.data_as(ctypes.c_void_p)


def cpu_lut_workspace_bytes(T: int, K: int, B: int, threads: int = 0) -> int:
    return int(load().fairy2i_cpu_lut_workspace_bytes(T, K, B, threads))


def cpu_lut_wl_matmul(codes_U, scales_U, codes_W, scales_W, q, x_scale, want_y=True, want_acc=False,
                      threads: int = 0, workspace=None):
    """The CPU table-lookup product (host arrays only): codes uint8 [T, N,
    K/4], scales float32 [T, 2], q int8 [B, K, 2], x_scale float32 [B].
    Returns (y complex64 [B, N] or None, acc int32 [2, T, 2, B, N, 2] or
    None).  ``workspace``: optional uint8 host array to reuse across calls."""
    lib = load()
    codes_U = _host(codes_U, np.uint8, "codes_U")
    if codes_U.ndim != 3:
        raise ValueError("codes_U must be [T, N, K/4]")
    T, N, K4 = codes_U.shape
    K = 4 * K4
    codes_W = _host(codes_W, np.uint8, "codes_W", (T, N, K4))
    q = _host(q, np.int8, "q")
    if q.ndim != 3 or q.shape[1:] != (K, 2):
        raise ValueError(f"q must be [B, {K}, 2], got {q.shape}")
    B = q.shape[0]
    su = sw = xs = None
    y = acc = None
    if want_y:
        su = _host(scales_U, np.float32, "scales_U", (T, 2))
        sw = _host(scales_W, np.float32, "scales_W", (T, 2))
        xs = _host(x_scale, np.float32, "x_scale", (B,))
        y = np.empty((B, N), dtype=np.complex64)
    if want_acc:
        acc = np.empty((2, T, 2, B, N, 2), dtype=np.int32)
    need = cpu_lut_workspace_bytes(T, K, B, threads)
    if need == 0:
        raise ValueError(f"unsupported shape T={T} K={K} B={B}")
    if workspace is None or workspace.nbytes < need:
        workspace = np.empty(need, dtype=np.uint8)
    _host(workspace, np.uint8, "workspace")
    _check(lib.fairy2i_cpu_lut_wl_matmul(_hp(codes_U), _hp(su), _hp(codes_W), _hp(sw), T, N, K, _hp(q), _hp(xs), B,
                                         _hp(y), _hp(acc), _hp(workspace), workspace.nbytes, threads),
           "fairy2i_cpu_lut_wl_matmul")
    return y, acc


class WlGroup:
    """A table of independent layers decoded by one fairy2i_wl_matmul_group
    call.  ``layers`` is a list of (codes_U, scales_U, codes_W, scales_W, x,
    x_scale, y) device tensors (x_scale None for bf16); the object keeps them,
    the workspace and both copies of the table alive.  ``layout``: LAYOUT_D3
    (codes [T, N, K/4]), LAYOUT_TILED or LAYOUT_TILED_FP4 (repacked copies,
    a 1-D uint8 tensor per matrix; N is then taken from y); ``tiled=True``
    is LAYOUT_TILED.  ``group_size`` G > 0: every layer has per-group scales
    [T, N, ceil(K/G), 2] (fairy2i_quantize_grouped; LAYOUT_TILED_FP4 only)."""

    def __init__(self, layers, T: int, B: int, tiled: bool = False, layout=None, group_size: int = 0):
        if layout is None:
            layout = LAYOUT_TILED if tiled else LAYOUT_D3
        tiled = layout != LAYOUT_D3
        torch = _torch()
        lib = load()
        if not layers:
            raise ValueError("empty group")
        dt = _act_dtype(layers[0][4])
        dev = layers[0][4].device
        self._keep = [t for layer in layers for t in layer if t is not None]
        arr = (WlLayer * len(layers))()
        for i, (cu, su, cw, sw, x, xs, y) in enumerate(layers):
            _require(x, None, f"layers[{i}].x", dev)
            Bx, K = _act_shape(x)
            if Bx != B or _act_dtype(x) != dt:
                raise ValueError("all layers of a group share B and the activation dtype")
            for t, n in ((cu, "codes_U"), (cw, "codes_W")):
                _require(t, torch.uint8, f"layers[{i}].{n}", dev)
            _require(y, torch.complex64, f"layers[{i}].y", dev)
            if y.dim() != 2 or y.shape[0] != B:
                raise ValueError(f"layers[{i}].y must have shape ({B}, N)")
            N = y.shape[1]
            sshape = (T, 2) if group_size == 0 else (T, N, -(-K // group_size) if group_size > 0 else 0, 2)
            for t, n in ((su, "scales_U"), (sw, "scales_W")):
                _require(t, torch.float32, f"layers[{i}].{n}", dev)
                if tuple(t.shape) != sshape:
                    raise ValueError(f"layers[{i}].{n} must have shape {sshape}")
            if xs is not None:
                _require(xs, torch.float32, f"layers[{i}].x_scale", dev)
                if tuple(xs.shape) != (B,):
                    raise ValueError(f"layers[{i}].x_scale must have shape ({B},)")
            if tiled:
                need = repack_tiled_bytes(N, K, T)
                if cu.numel() < need or cw.numel() < need:
                    raise ValueError("tiled codes smaller than fairy2i_repack_tiled_bytes")
            elif tuple(cu.shape) != (T, N, K // 4) or tuple(cw.shape) != (T, N, K // 4):
                raise ValueError(f"layers[{i}] codes must have shape ({T}, {N}, {K // 4})")
            arr[i] = WlLayer(cu.data_ptr(), su.data_ptr(), cw.data_ptr(), sw.data_ptr(), x.data_ptr(),
                             None if xs is None else xs.data_ptr(), y.data_ptr(), N, K,
                             layout, group_size)
        self.n = len(layers)
        wsb = int(lib.fairy2i_wl_group_workspace_bytes(ctypes.byref(arr), self.n, T, dt, B))
        self.workspace = torch.empty(max(wsb, 1), dtype=torch.uint8, device=dev)
        tb = int(lib.fairy2i_wl_group_table_bytes(self.n))
        self._table = (ctypes.c_uint8 * tb)()
        _check(lib.fairy2i_wl_group_build_table(ctypes.byref(arr), self.n, T, dt, B,
                                                _ptr(self.workspace), wsb, ctypes.byref(self._table), tb),
               "fairy2i_wl_group_build_table")
        host = torch.frombuffer(bytearray(bytes(self._table)), dtype=torch.uint8)
        self.table_device = host.to(dev)
        torch.cuda.synchronize(dev)
        self._layers = arr

    def run(self, events=None):
        """One grouped call.  ``events``: optional 4 torch.cuda.Event already
        recorded once (so they exist); the library re-records them around its
        three kernels on the current stream."""
        lib = load()
        stream = _stream_ptr(self.table_device)
        if events is None:
            _check(lib.fairy2i_wl_matmul_group(ctypes.byref(self._table), _ptr(self.table_device), stream),
                   "fairy2i_wl_matmul_group")
            return
        handles = (_c_p * 4)(*[e.cuda_event for e in events])
        _check(lib.fairy2i_wl_matmul_group_timed(ctypes.byref(self._table), _ptr(self.table_device), stream,
                                                 handles), "fairy2i_wl_matmul_group_timed")


BLOCK_PROJ = ("q", "k", "v", "o", "gate", "up", "down")


class WlBlock:
    """One widely-linear decoder block for one decode token
    (fairy2i_block_decode).  ``layers``: {name: (codes_U, scales_U, codes_W,
    scales_W)} for q, k, v, o, gate, up, down, codes in the fp4 tiled layout
    (repack_tiled_fp4); ``norm_attn``, ``norm_mlp``: float32 [2n] device
    tensors.  Keeps the weights, the workspace and both plan copies alive."""

    def __init__(self, layers, norm_attn, norm_mlp, n, n_ff, n_heads, T, max_ctx, eps=1e-5, rope_base=10000.0):
        torch = _torch()
        lib = load()
        dev = norm_attn.device
        d = BlockDesc()
        d.n, d.n_ff, d.n_heads, d.T, d.max_ctx = n, n_ff, n_heads, T, max_ctx
        d.eps, d.reserved, d.rope_base = eps, 0, rope_base
        self._keep = []
        for i, name in enumerate(BLOCK_PROJ):
            cu, su, cw, sw = layers[name]
            for t, nm, dt in ((cu, "codes_U", torch.uint8), (cw, "codes_W", torch.uint8),
                              (su, "scales_U", torch.float32), (sw, "scales_W", torch.float32)):
                _require(t, dt, f"{name}.{nm}", dev)
            N = n_ff if name in ("gate", "up") else n
            K = n_ff if name == "down" else n
            need = repack_tiled_bytes(N, K, T)
            if cu.numel() < need or cw.numel() < need or tuple(su.shape) != (T, 2) or tuple(sw.shape) != (T, 2):
                raise ValueError(f"{name}: codes or scales do not match a {N}x{K} layer with T={T}")
            d.codes_U[i], d.scales_U[i] = cu.data_ptr(), su.data_ptr()
            d.codes_W[i], d.scales_W[i] = cw.data_ptr(), sw.data_ptr()
            self._keep += [cu, su, cw, sw]
        for t, nm in ((norm_attn, "norm_attn"), (norm_mlp, "norm_mlp")):
            _require(t, torch.float32, nm, dev)
            if t.numel() != 2 * n:
                raise ValueError(f"{nm} must hold 2n = {2 * n} gains")
        d.norm_attn, d.norm_mlp = norm_attn.data_ptr(), norm_mlp.data_ptr()
        self._keep += [norm_attn, norm_mlp]
        self.n, self.n_ff, self.n_heads, self.max_ctx = n, n_ff, n_heads, max_ctx
        self._desc = d
        wsb = int(lib.fairy2i_block_workspace_bytes(ctypes.byref(d)))
        pb = int(lib.fairy2i_block_plan_bytes(ctypes.byref(d)))
        if wsb == 0 or pb == 0:
            raise Fairy2iError(ERR_SHAPE, "fairy2i_block_workspace_bytes")
        self.workspace = torch.empty(wsb, dtype=torch.uint8, device=dev)
        self._plan = (ctypes.c_uint8 * pb)()
        _check(lib.fairy2i_block_build_plan(ctypes.byref(d), _ptr(self.workspace), wsb, ctypes.byref(self._plan), pb),
               "fairy2i_block_build_plan")
        self.plan_device = torch.frombuffer(bytearray(bytes(self._plan)), dtype=torch.uint8).to(dev)
        torch.cuda.synchronize(dev)

    BLOCK_INTERMEDIATES = (("z", "bf16", "n"), ("q_rot", "c64", "n"), ("v", "c64", "n"), ("o", "bf16", "n"),
                           ("a", "c64", "n"), ("h1", "c64", "n"), ("z2", "bf16", "n"), ("g", "c64", "f"),
                           ("u", "c64", "f"), ("act", "bf16", "f"), ("d", "c64", "n"), ("k", "c64", "n"))

    def intermediates(self):
        """Views of the workspace buffers that the last decode left
        (fairy2i_block_intermediates): {name: tensor}, complex64 [len] or
        bf16 [len, 2]."""
        torch = _torch()
        lib = load()
        ptrs = (_c_p * 12)()
        _check(lib.fairy2i_block_intermediates(ctypes.byref(self._plan), ptrs), "fairy2i_block_intermediates")
        base = self.workspace.data_ptr()
        out = {}
        for (name, kind, ln), p in zip(self.BLOCK_INTERMEDIATES, ptrs):
            count = self.n if ln == "n" else self.n_ff
            off = int(p) - base
            if kind == "c64":
                out[name] = self.workspace[off:off + 8 * count].view(torch.complex64)
            else:
                out[name] = self.workspace[off:off + 4 * count].view(torch.bfloat16).view(count, 2)
        return out

    def decode(self, x, k_cache, v_cache, pos, out=None):
        """x: complex64 [1, n]; caches complex64 [n_heads, max_ctx, n / n_heads];
        returns out complex64 [1, n]."""
        torch = _torch()
        lib = load()
        dev = self.plan_device.device
        dc = self.n // self.n_heads
        _require(x, torch.complex64, "x", dev)
        if x.numel() != self.n:
            raise ValueError(f"x must hold {self.n} complex entries")
        for t, nm in ((k_cache, "k_cache"), (v_cache, "v_cache")):
            _require(t, torch.complex64, nm, dev)
            if tuple(t.shape) != (self.n_heads, self.max_ctx, dc):
                raise ValueError(f"{nm} must have shape ({self.n_heads}, {self.max_ctx}, {dc})")
        if out is None:
            out = torch.empty((1, self.n), dtype=torch.complex64, device=dev)
        else:
            _require(out, torch.complex64, "out", dev)
            if out.numel() != self.n:
                raise ValueError(f"out must hold {self.n} complex entries")
        _check(lib.fairy2i_block_decode(ctypes.byref(self._plan), _ptr(self.plan_device), _ptr(x), _ptr(k_cache),
                                        _ptr(v_cache), int(pos), _ptr(out), _stream_ptr(x)), "fairy2i_block_decode")
        return out
