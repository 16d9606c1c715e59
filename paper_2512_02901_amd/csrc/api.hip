// C-ABI entry points: argument checks on the host, then launches on the
// caller's stream.  Nothing here allocates, frees or synchronises.
#include <stddef.h>

#include <algorithm>
#include <mutex>
#include <vector>

#include "common.h"
#include "decode.h"
#include "superacc.h"

using namespace fairy2i;

namespace {

inline hipStream_t as_stream(void* s) { return static_cast<hipStream_t>(s); }

inline fairy2i_status hip_status(hipError_t e) { return e == hipSuccess ? FAIRY2I_OK : FAIRY2I_ERR_HIP; }

fairy2i_status check_wl_common(const uint8_t* cu, const uint8_t* cw, int32_t T, int64_t N, int64_t K,
                               const void* x, int64_t B, const void* out) {
  if (!cu || !cw || !x || !out) return FAIRY2I_ERR_NULL;
  if (N <= 0 || K <= 0 || B <= 0 || (K % 4) != 0) return FAIRY2I_ERR_SHAPE;
  // int32 accumulators: |sum| <= 127 K must stay below 2^31; grid limits.
  if (K > ((int64_t)1 << 24) || N > ((int64_t)1 << 31) - 64 || B > ((int64_t)1 << 31) - 64)
    return FAIRY2I_ERR_SHAPE;
  if (T < 1 || T > FAIRY2I_MAX_STAGES) return FAIRY2I_ERR_STAGES;
  return FAIRY2I_OK;
}

// Decode on the int8 matrix cores: bf16 / int8 activations, K % 64 == 0.
bool use_mfma_decode(int32_t dtype, int64_t N, int64_t K, int64_t B) {
  return (dtype == FAIRY2I_ACT_BF16 || dtype == FAIRY2I_ACT_I8) && (K % 64) == 0 &&
         B <= FAIRY2I_MAX_DECODE_BATCH && N <= ((int64_t)1 << 26) &&
         N * K / 4 < ((int64_t)1 << 31);  // 32-bit buffer ranges per code plane
}

int dec_mode(int32_t dtype) { return dtype == FAIRY2I_ACT_BF16 ? kModeBf16 : kModeI8; }

DecLayer dec_layer(const uint8_t* cu, const float* su, const uint8_t* cw, const float* sw, int64_t N,
                   int64_t K, const void* x, const float* xs, float* y) {
  DecLayer l{};
  l.codes[0] = cu;
  l.codes[1] = cw;
  l.scales[0] = su;
  l.scales[1] = sw;
  l.x = x;
  l.x_scale_in = xs;
  l.y = reinterpret_cast<float2*>(y);
  l.N = (int32_t)N;
  l.K = (int32_t)K;
  return l;
}

// Workspace of a one-layer decode call (the same for the y and the
// accumulator-export variants: the larger of the two layouts).
size_t single_decode_bytes(int64_t N, int64_t K, int32_t T, int64_t B, int32_t dtype) {
  size_t best = 0;
  for (int ex = 0; ex < 2; ++ex) {
    DecLayer l{};
    l.N = (int32_t)N;
    l.K = (int32_t)K;
    const size_t b = dec_layer_setup(l, dec_header(T, dec_mode(dtype), B, ex != 0), true, nullptr);
    if (b > best) best = b;
  }
  return best;
}

fairy2i_status run_single_decode(DecLayer l, int32_t T, int32_t dtype, int64_t B, void* ws,
                                 size_t ws_bytes, int32_t* acc, hipStream_t stream) {
  DecHeader h = dec_header(T, dec_mode(dtype), B, acc != nullptr);
  const size_t need = dec_layer_setup(l, h, true, nullptr);
  if (!ws || ws_bytes < need) return FAIRY2I_ERR_WORKSPACE;
  dec_layer_setup(l, h, true, static_cast<char*>(ws));
  l.acc = acc;
  l.item0 = 0;
  l.step0 = 0;
  h.n_layers = 1;
  h.total_items = (int64_t)l.nrb * l.nkc;
  h.total_steps = (int64_t)l.nrb * l.nk4;
  h.max_nk4 = l.nk4;
  const int64_t acc_elems = acc ? (int64_t)2 * T * 2 * B * l.N * 2 : 0;
  return hip_status(launch_decode(h, l, nullptr, l.nkc > 1, B * (int64_t)l.N, acc != nullptr, acc_elems,
                                  acc, stream));
}


// ------------------------------------------------ allocation-free call ---
// fairy2i_wl_matmul_noalloc runs fairy2i_wl_matmul with this array as its
// workspace.  Every GPU the library runs on holds its own copy until the
// process ends.  In host code `scratch` names a host-side stand-in, not the
// device memory: the device address of the current device's copy is taken
// once per device with hipGetSymbolAddress and only that address is used.
constexpr size_t kNoAllocScratchBytes = FAIRY2I_NOALLOC_SCRATCH_BYTES;
static __device__ __align__(256) unsigned char scratch[kNoAllocScratchBytes];

constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
void* g_scratch_dev[kMaxDevices] = {};  // device address of `scratch` per device, once looked up

// Device address of the current device's scratch array (looked up on the
// first call for that device).
fairy2i_status current_scratch(void** out) {
  int dev = -1;
  if (hipGetDevice(&dev) != hipSuccess) return FAIRY2I_ERR_HIP;
  if (dev < 0 || dev >= kMaxDevices) return FAIRY2I_ERR_UNSUPPORTED;
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  if (!g_scratch_dev[dev]) {
    void* p = nullptr;
    if (hipGetSymbolAddress(&p, HIP_SYMBOL(scratch)) != hipSuccess || !p) return FAIRY2I_ERR_HIP;
    g_scratch_dev[dev] = p;
  }
  *out = g_scratch_dev[dev];
  return FAIRY2I_OK;
}

}  // namespace

extern "C" {

const char* fairy2i_status_string(fairy2i_status s) {
  switch (s) {
    case FAIRY2I_OK: return "ok";
    case FAIRY2I_ERR_NULL: return "null pointer argument";
    case FAIRY2I_ERR_SHAPE: return "dimension out of range";
    case FAIRY2I_ERR_STAGES: return "number of stages T out of range";
    case FAIRY2I_ERR_DTYPE: return "unknown activation dtype";
    case FAIRY2I_ERR_UNSUPPORTED: return "unsupported argument combination";
    case FAIRY2I_ERR_WORKSPACE: return "workspace missing or too small";
    case FAIRY2I_ERR_HIP: return "HIP runtime error";
    default: return "unknown status";
  }
}

int32_t fairy2i_abi_version(void) { return 5; }

fairy2i_status fairy2i_to_widely_linear(const float* A, int64_t rows, int64_t cols, float* U,
                                        float* W, void* stream) {
  if (!A || !U || !W) return FAIRY2I_ERR_NULL;
  if (rows <= 0 || cols <= 0 || (rows % 2) != 0 || (cols % 2) != 0) return FAIRY2I_ERR_SHAPE;
  return hip_status(launch_to_widely_linear(A, rows / 2, cols / 2, reinterpret_cast<float2*>(U),
                                            reinterpret_cast<float2*>(W), as_stream(stream)));
}

size_t fairy2i_quantize_workspace_bytes(int64_t N, int64_t K, int32_t T) {
  (void)T;
  if (N <= 0 || K <= 0) return 0;
  return quantize_workspace_bytes(N, K);
}

fairy2i_status fairy2i_quantize(const float* M, int64_t N, int64_t K, int32_t T, uint8_t* codes,
                                float* scales, void* workspace, size_t workspace_bytes, void* stream) {
  if (!M || !codes || !scales) return FAIRY2I_ERR_NULL;
  if (N <= 0 || K <= 0 || (K % 4) != 0 || N > FAIRY2I_MAX_QUANTIZE_ENTRIES / K)
    return FAIRY2I_ERR_SHAPE;
  if (T < 1 || T > FAIRY2I_MAX_STAGES) return FAIRY2I_ERR_STAGES;
  if (!workspace || workspace_bytes < quantize_workspace_bytes(N, K)) return FAIRY2I_ERR_WORKSPACE;
  return hip_status(launch_quantize(reinterpret_cast<const float2*>(M), N, K, T, codes, scales,
                                    workspace, as_stream(stream)));
}

fairy2i_status fairy2i_quantize_grouped(const float* M, int64_t N, int64_t K, int32_t T, int64_t G,
                                        uint8_t* codes, float* scales, void* stream) {
  if (!M || !codes || !scales) return FAIRY2I_ERR_NULL;
  if (N <= 0 || K <= 0 || (K % 4) != 0 || N > FAIRY2I_MAX_QUANTIZE_ENTRIES / K || G < 4 || (G % 4) != 0)
    return FAIRY2I_ERR_SHAPE;
  if (T < 1 || T > FAIRY2I_MAX_STAGES) return FAIRY2I_ERR_STAGES;
  return hip_status(launch_quantize_grouped(reinterpret_cast<const float2*>(M), N, K, T, G < K ? G : K, codes,
                                            scales, as_stream(stream)));
}

static bool repack_shape_ok(int64_t N, int64_t K) {
  return N >= 1 && K >= 4 && (K % 4) == 0 && N <= FAIRY2I_MAX_QUANTIZE_ENTRIES / K;
}

size_t fairy2i_repack_tiled_bytes(int64_t N, int64_t K, int32_t T) {
  if (!repack_shape_ok(N, K) || T < 1 || T > FAIRY2I_MAX_STAGES) return 0;
  return repack_tiled_bytes(N, K, T);
}

fairy2i_status fairy2i_repack_tiled(const uint8_t* codes, int64_t N, int64_t K, int32_t T, uint8_t* tiled,
                                    size_t tiled_bytes, void* stream) {
  if (!codes || !tiled) return FAIRY2I_ERR_NULL;
  if (!repack_shape_ok(N, K)) return FAIRY2I_ERR_SHAPE;
  if (T < 1 || T > FAIRY2I_MAX_STAGES) return FAIRY2I_ERR_STAGES;
  if (tiled_bytes < repack_tiled_bytes(N, K, T)) return FAIRY2I_ERR_WORKSPACE;
  return hip_status(launch_repack_tiled(codes, N, K, T, tiled, as_stream(stream)));
}

fairy2i_status fairy2i_repack_tiled_fp4(const uint8_t* codes, int64_t N, int64_t K, int32_t T, uint8_t* out,
                                        size_t out_bytes, void* stream) {
  if (!codes || !out) return FAIRY2I_ERR_NULL;
  if (!repack_shape_ok(N, K)) return FAIRY2I_ERR_SHAPE;
  if (T < 1 || T > FAIRY2I_MAX_STAGES) return FAIRY2I_ERR_STAGES;
  if (out_bytes < repack_tiled_bytes(N, K, T)) return FAIRY2I_ERR_WORKSPACE;
  return hip_status(launch_repack_fp4(codes, N, K, T, out, as_stream(stream)));
}

fairy2i_status fairy2i_quantize_act_int8(const void* x, int32_t dtype, int64_t B, int64_t K,
                                         int8_t* q, float* x_scale, void* stream) {
  if (!x || !q || !x_scale) return FAIRY2I_ERR_NULL;
  if (B <= 0 || K <= 0 || B > ((int64_t)1 << 31) - 1) return FAIRY2I_ERR_SHAPE;
  if (dtype != FAIRY2I_ACT_F32 && dtype != FAIRY2I_ACT_BF16) return FAIRY2I_ERR_DTYPE;
  return hip_status(launch_quantize_act_int8(x, dtype, B, K, q, x_scale, as_stream(stream)));
}

size_t fairy2i_wl_matmul_workspace_bytes(int64_t N, int64_t K, int32_t T, int64_t B, int32_t dtype) {
  if (N <= 0 || K <= 0 || B <= 0 || T < 1 || T > FAIRY2I_MAX_STAGES) return 0;
  if (use_mfma_decode(dtype, N, K, B)) return single_decode_bytes(N, K, T, B, dtype);
  if (dtype == FAIRY2I_ACT_I8 && B > FAIRY2I_MAX_DECODE_BATCH) return gemm_workspace_bytes(N, K, B);
  return 0;
}

fairy2i_status fairy2i_wl_matmul(const uint8_t* codes_U, const float* scales_U,
                                 const uint8_t* codes_W, const float* scales_W, int32_t T,
                                 int64_t N, int64_t K, const void* x, const float* x_scale,
                                 int32_t dtype, int64_t B, float* y, void* workspace,
                                 size_t workspace_bytes, void* stream) {
  fairy2i_status st = check_wl_common(codes_U, codes_W, T, N, K, x, B, y);
  if (st != FAIRY2I_OK) return st;
  if (!scales_U || !scales_W) return FAIRY2I_ERR_NULL;
  if (dtype != FAIRY2I_ACT_F32 && dtype != FAIRY2I_ACT_BF16 && dtype != FAIRY2I_ACT_I8)
    return FAIRY2I_ERR_DTYPE;
  if (dtype == FAIRY2I_ACT_I8 && !x_scale) return FAIRY2I_ERR_NULL;
  if (dtype != FAIRY2I_ACT_I8 && x_scale) return FAIRY2I_ERR_UNSUPPORTED;
  if (dtype != FAIRY2I_ACT_I8 && B > FAIRY2I_MAX_DECODE_BATCH) return FAIRY2I_ERR_UNSUPPORTED;
  if (workspace_bytes < fairy2i_wl_matmul_workspace_bytes(N, K, T, B, dtype) ||
      (fairy2i_wl_matmul_workspace_bytes(N, K, T, B, dtype) > 0 && !workspace))
    return FAIRY2I_ERR_WORKSPACE;
  if (use_mfma_decode(dtype, N, K, B))
    return run_single_decode(dec_layer(codes_U, scales_U, codes_W, scales_W, N, K, x, x_scale, y), T,
                             dtype, B, workspace, workspace_bytes, nullptr, as_stream(stream));
  WlArgs a{};
  a.codes[0] = codes_U;
  a.codes[1] = codes_W;
  a.scales[0] = scales_U;
  a.scales[1] = scales_W;
  a.T = T;
  a.N = N;
  a.K = K;
  a.B = B;
  a.x = x;
  a.x_scale = x_scale;
  a.dtype = dtype;
  a.y = reinterpret_cast<float2*>(y);
  a.acc = nullptr;
  const hipError_t e = (B <= FAIRY2I_MAX_DECODE_BATCH) ? launch_gemv(a, as_stream(stream))
                                                       : launch_gemm_i8(a, workspace, as_stream(stream));
  return hip_status(e);
}

fairy2i_status fairy2i_wl_matmul_noalloc(const uint8_t* codes_U, const float* scales_U,
                                         const uint8_t* codes_W, const float* scales_W, int32_t T,
                                         int64_t N, int64_t K, const void* x, const float* x_scale,
                                         int32_t dtype, int64_t B, float* y, void* stream) {
  // argument errors first, exactly as fairy2i_wl_matmul reports them
  fairy2i_status st = check_wl_common(codes_U, codes_W, T, N, K, x, B, y);
  if (st != FAIRY2I_OK) return st;
  if (!scales_U || !scales_W) return FAIRY2I_ERR_NULL;
  if (dtype != FAIRY2I_ACT_F32 && dtype != FAIRY2I_ACT_BF16 && dtype != FAIRY2I_ACT_I8)
    return FAIRY2I_ERR_DTYPE;
  const size_t need = fairy2i_wl_matmul_workspace_bytes(N, K, T, B, dtype);
  if (need > kNoAllocScratchBytes) return FAIRY2I_ERR_WORKSPACE;
  void* ws = nullptr;
  if (need > 0 && (st = current_scratch(&ws)) != FAIRY2I_OK) return st;
  return fairy2i_wl_matmul(codes_U, scales_U, codes_W, scales_W, T, N, K, x, x_scale, dtype, B, y, ws,
                           need > 0 ? kNoAllocScratchBytes : 0, stream);
}

fairy2i_status fairy2i_wl_int8_accumulators(const uint8_t* codes_U, const uint8_t* codes_W, int32_t T,
                                            int64_t N, int64_t K, const int8_t* q, int64_t B,
                                            int32_t* acc, void* workspace, size_t workspace_bytes,
                                            void* stream) {
  fairy2i_status st = check_wl_common(codes_U, codes_W, T, N, K, q, B, acc);
  if (st != FAIRY2I_OK) return st;
  if (workspace_bytes < fairy2i_wl_matmul_workspace_bytes(N, K, T, B, FAIRY2I_ACT_I8) ||
      (fairy2i_wl_matmul_workspace_bytes(N, K, T, B, FAIRY2I_ACT_I8) > 0 && !workspace))
    return FAIRY2I_ERR_WORKSPACE;
  if (use_mfma_decode(FAIRY2I_ACT_I8, N, K, B))
    return run_single_decode(dec_layer(codes_U, nullptr, codes_W, nullptr, N, K, q, nullptr, nullptr), T,
                             FAIRY2I_ACT_I8, B, workspace, workspace_bytes, acc, as_stream(stream));
  WlArgs a{};
  a.codes[0] = codes_U;
  a.codes[1] = codes_W;
  a.T = T;
  a.N = N;
  a.K = K;
  a.B = B;
  a.x = q;
  a.dtype = FAIRY2I_ACT_I8;
  a.acc = acc;
  const hipError_t e = (B <= FAIRY2I_MAX_DECODE_BATCH) ? launch_gemv(a, as_stream(stream))
                                                       : launch_gemm_i8(a, workspace, as_stream(stream));
  return hip_status(e);
}


size_t fairy2i_wl_group_table_bytes(int32_t n_layers) {
  if (n_layers < 1) return 0;
  return sizeof(GroupTableHeader) + (size_t)n_layers * sizeof(DecLayer);
}

static fairy2i_status check_group(const fairy2i_wl_layer* layers, int32_t n_layers, int32_t T,
                                  int32_t dtype, int64_t B) {
  if (!layers) return FAIRY2I_ERR_NULL;
  if (n_layers < 1) return FAIRY2I_ERR_SHAPE;
  if (T < 1 || T > FAIRY2I_MAX_STAGES) return FAIRY2I_ERR_STAGES;
  if (dtype != FAIRY2I_ACT_F32 && dtype != FAIRY2I_ACT_BF16 && dtype != FAIRY2I_ACT_I8)
    return FAIRY2I_ERR_DTYPE;
  if (B <= 0) return FAIRY2I_ERR_SHAPE;
  for (int32_t i = 0; i < n_layers; ++i) {
    const fairy2i_wl_layer& L = layers[i];
    fairy2i_status st = check_wl_common(L.codes_U, L.codes_W, T, L.N, L.K, L.x, B, L.y);
    if (st != FAIRY2I_OK) return st;
    if (!L.scales_U || !L.scales_W) return FAIRY2I_ERR_NULL;
    if (dtype == FAIRY2I_ACT_I8 && !L.x_scale) return FAIRY2I_ERR_NULL;
    if (dtype != FAIRY2I_ACT_I8 && L.x_scale) return FAIRY2I_ERR_UNSUPPORTED;
    if (!use_mfma_decode(dtype, L.N, L.K, B) || L.N > ((int64_t)1 << 30) || L.K > ((int64_t)1 << 24))
      return FAIRY2I_ERR_UNSUPPORTED;
    // per-group scales: fp4 path, every layer or none, groups of whole 256-code steps
    if (L.group_size < 0 || L.group_size % 256 != 0) return FAIRY2I_ERR_UNSUPPORTED;
    if ((L.group_size != 0) != (layers[0].group_size != 0)) return FAIRY2I_ERR_UNSUPPORTED;
    if (L.group_size != 0 && L.layout != FAIRY2I_LAYOUT_TILED_FP4) return FAIRY2I_ERR_UNSUPPORTED;
    // the kernel addresses a scale array with 32-bit offsets
    if (L.group_size != 0 && (int64_t)T * L.N * ((L.K + L.group_size - 1) / L.group_size) * 8 >= ((int64_t)1 << 31))
      return FAIRY2I_ERR_UNSUPPORTED;
    if (L.layout != FAIRY2I_LAYOUT_D3 && L.layout != FAIRY2I_LAYOUT_TILED && L.layout != FAIRY2I_LAYOUT_TILED_FP4)
      return FAIRY2I_ERR_UNSUPPORTED;
    // the decode kernels address a matrix with 32-bit offsets
    if (L.layout != FAIRY2I_LAYOUT_D3 && repack_tiled_bytes(L.N, L.K, T) >= ((size_t)1 << 31))
      return FAIRY2I_ERR_UNSUPPORTED;
    // fp4 tiled codes: every layer, bf16 activations, one or two activation tiles of 2 tokens
    if ((L.layout == FAIRY2I_LAYOUT_TILED_FP4) != (layers[0].layout == FAIRY2I_LAYOUT_TILED_FP4))
      return FAIRY2I_ERR_UNSUPPORTED;
    if (L.layout == FAIRY2I_LAYOUT_TILED_FP4 &&
        (dtype != FAIRY2I_ACT_BF16 || B > 16 || (B > 8 && T > 2) || (B > 4 && T > 3)))
      return FAIRY2I_ERR_UNSUPPORTED;
  }
  return FAIRY2I_OK;
}

// Decode mode of a checked group.
static int group_mode(const fairy2i_wl_layer* layers, int32_t dtype) {
  return layers[0].layout == FAIRY2I_LAYOUT_TILED_FP4 ? kModeBf16F4 : dec_mode(dtype);
}

// Steps per K slice for a checked group: kSliceFullK (every layer of at most
// kMaxFullKSteps steps as one work item per row block) on the fp4 path when
// the group has enough row blocks to keep every wave busy without K slices;
// otherwise 8, halved while the group has fewer than kMinGroupItems items.
static int group_slice(const fairy2i_wl_layer* layers, int32_t n_layers, const DecHeader& h) {
  int64_t rbs = 0;
  for (int32_t i = 0; i < n_layers; ++i) rbs += (layers[i].N + 15) / 16;
  if (h.mode == kModeBf16F4 && rbs >= kFullKMinItems) return kSliceFullK;
  int slice = 8;
  while (slice > 1) {
    int64_t items = 0;
    for (int32_t i = 0; i < n_layers; ++i) {
      const int64_t nk4 = (layers[i].K + 255) / 256;
      items += (layers[i].N + 15) / 16 * ((nk4 + slice - 1) / slice);
    }
    if (items >= kMinGroupItems) break;
    slice /= 2;
  }
  return slice;
}

size_t fairy2i_wl_group_workspace_bytes(const fairy2i_wl_layer* layers, int32_t n_layers, int32_t T,
                                        int32_t dtype, int64_t B) {
  if (check_group(layers, n_layers, T, dtype, B) != FAIRY2I_OK) return 0;
  const DecHeader h = dec_header(T, group_mode(layers, dtype), B, false);
  const int slice = group_slice(layers, n_layers, h);
  size_t total = kGroupCallBytes;
  for (int32_t i = 0; i < n_layers; ++i) {
    DecLayer l{};
    l.N = (int32_t)layers[i].N;
    l.K = (int32_t)layers[i].K;
    total += dec_layer_setup(l, h, false, nullptr, slice);
  }
  return total;
}

fairy2i_status fairy2i_wl_group_build_table(const fairy2i_wl_layer* layers, int32_t n_layers, int32_t T,
                                            int32_t dtype, int64_t B, void* workspace,
                                            size_t workspace_bytes, void* table, size_t table_bytes) {
  fairy2i_status st = check_group(layers, n_layers, T, dtype, B);
  if (st != FAIRY2I_OK) return st;
  if (!table) return FAIRY2I_ERR_NULL;
  if (table_bytes < fairy2i_wl_group_table_bytes(n_layers)) return FAIRY2I_ERR_WORKSPACE;
  const size_t need = fairy2i_wl_group_workspace_bytes(layers, n_layers, T, dtype, B);
  if (!workspace || workspace_bytes < need) return FAIRY2I_ERR_WORKSPACE;
  auto* hdr = static_cast<GroupTableHeader*>(table);
  auto* tab = reinterpret_cast<DecLayer*>(hdr + 1);
  DecHeader h = dec_header(T, group_mode(layers, dtype), B, false);
  const int slice = group_slice(layers, n_layers, h);
  char* ws = static_cast<char*>(workspace);
  h.coop_ctr = reinterpret_cast<uint32_t*>(ws);
  ws += kGroupCallBytes;
  // descriptors in table order; on the fp4 path the table lists the layers by
  // decreasing work-item length (stable), so that the blocks of the product
  // kernel claim their long items first and end on short ones
  std::vector<DecLayer> ls((size_t)n_layers);
  for (int32_t i = 0; i < n_layers; ++i) {
    const fairy2i_wl_layer& L = layers[i];
    DecLayer& l = ls[(size_t)i];
    l = dec_layer(L.codes_U, L.scales_U, L.codes_W, L.scales_W, L.N, L.K, L.x, L.x_scale, L.y);
    l.tiled = L.layout != FAIRY2I_LAYOUT_D3 ? 1 : 0;
    l.gsteps = L.group_size / 256;
    ws += dec_layer_setup(l, h, false, ws, slice);
    l.acc = nullptr;
  }
  if (h.mode == kModeBf16F4)
    std::stable_sort(ls.begin(), ls.end(), [](const DecLayer& a, const DecLayer& b) { return a.kc4 > b.kc4; });
  int64_t items = 0, steps = 0, sitems = 0, ssteps = 0;
  int32_t min_nk4 = INT32_MAX;
  int any_split = 0;
  int64_t max_BN = 0;
  for (int32_t i = 0; i < n_layers; ++i) {
    DecLayer l = ls[(size_t)i];
    l.item0 = items;
    l.step0 = steps;
    l.sitem0 = sitems;
    l.sstep0 = ssteps;
    items += (int64_t)l.nrb * l.nkc;
    steps += (int64_t)l.nrb * l.nk4;
    const int rbg = coop_row_blocks(h.ntile);
    const int64_t groups = ((int64_t)l.nrb + rbg - 1) / rbg;
    sitems += groups;
    ssteps += groups * l.nk4;
    if (l.nk4 < min_nk4) min_nk4 = l.nk4;
    if (l.nk4 > h.max_nk4) h.max_nk4 = l.nk4;
    if (l.nkc > 1) any_split = 1;
    if (B * (int64_t)l.N > max_BN) max_BN = B * (int64_t)l.N;
    tab[i] = l;
  }
  // the decode kernels index a call's work items with 32-bit offsets
  if (items >= ((int64_t)1 << 31)) return FAIRY2I_ERR_UNSUPPORTED;
  *hdr = GroupTableHeader{};
  hdr->magic = kGroupMagic;
  hdr->abi = (uint32_t)fairy2i_abi_version();
  h.n_layers = n_layers;
  h.total_items = items;
  h.total_steps = steps;
  h.total_ssteps = ssteps;
  h.grouped = layers[0].group_size != 0 ? 1 : 0;
  h.coop = (h.mode == kModeBf16F4 && slice == kSliceFullK && !any_split) ? 1 : 0;
  h.coop_rb = coop_row_blocks(h.ntile);
  // Run-time claims need every group to last more steps than the kernel's
  // ring holds (a claim is answered kCoopSlots steps after it is made); the
  // claimed region starts at the first group at or after the static
  // fraction of the group steps (the table is sorted by decreasing length,
  // so it holds the shortest groups).
  h.coop_groups = sitems;
  h.coop_dyn0 = sitems;
  h.coop_dyn_steps = ssteps;
  if (h.coop && min_nk4 > kCoopSlots) {
    const int64_t target = (int64_t)(kCoopStaticFrac * (double)ssteps);
    const int rbg = h.coop_rb;
    for (int32_t i = 0; i < n_layers; ++i) {
      const DecLayer& l = tab[i];
      const int64_t groups = ((int64_t)l.nrb + rbg - 1) / rbg;
      if (l.sstep0 + groups * l.nk4 <= target) continue;
      const int64_t g = l.sstep0 >= target ? 0 : (target - l.sstep0 + l.nk4 - 1) / l.nk4;
      h.coop_dyn0 = l.sitem0 + g;
      h.coop_dyn_steps = l.sstep0 + g * l.nk4;
      break;
    }
  }
  hdr->h = h;
  hdr->any_split = any_split;
  hdr->max_BN = max_BN;
  return FAIRY2I_OK;
}

static fairy2i_status run_group(const void* table, const void* table_device, void* stream,
                                void* const* events) {
  if (!table || !table_device) return FAIRY2I_ERR_NULL;
  const auto* hdr = static_cast<const GroupTableHeader*>(table);
  if (hdr->magic != kGroupMagic || hdr->abi != (uint32_t)fairy2i_abi_version())
    return FAIRY2I_ERR_UNSUPPORTED;
  const auto* tab_dev = reinterpret_cast<const DecLayer*>(static_cast<const char*>(table_device) +
                                                          sizeof(GroupTableHeader));
  DecLayer none{};
  return hip_status(launch_decode(hdr->h, none, tab_dev, hdr->any_split, hdr->max_BN, false, 0, nullptr,
                                  as_stream(stream), reinterpret_cast<hipEvent_t const*>(events)));
}

fairy2i_status fairy2i_wl_matmul_group(const void* table, const void* table_device, void* stream) {
  return run_group(table, table_device, stream, nullptr);
}

fairy2i_status fairy2i_wl_matmul_group_timed(const void* table, const void* table_device, void* stream,
                                             void* const* events) {
  if (!events || !events[0] || !events[1] || !events[2] || !events[3]) return FAIRY2I_ERR_NULL;
  return run_group(table, table_device, stream, events);
}

fairy2i_status fairy2i_host_exact_mean_f32(const double* values, int64_t n_values, float* out) {
  if (!out || (n_values > 0 && !values)) return FAIRY2I_ERR_NULL;
  if (n_values < 0 || n_values > FAIRY2I_MAX_QUANTIZE_ENTRIES) return FAIRY2I_ERR_SHAPE;
  if (n_values == 0) {
    *out = 0.0f;
    return FAIRY2I_OK;
  }
  std::vector<uint64_t> limbs(SA_LIMBS, 0);
  for (int64_t i = 0; i < n_values; ++i) {
    double v = values[i] < 0 ? -values[i] : values[i];
    if (v == 0.0) continue;
    int limb;
    uint32_t lo, mid, hi;
    sa_split(v, &limb, &lo, &mid, &hi);
    limbs[limb] += lo;
    limbs[limb + 1] += mid;
    limbs[limb + 2] += hi;
  }
  *out = sa_mean_to_f32(limbs.data(), (uint64_t)n_values);
  return FAIRY2I_OK;
}

}  // extern "C"
