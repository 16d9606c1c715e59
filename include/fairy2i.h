/*
 * fairy2i.h -- C ABI of the MI355X (gfx950) library for the Fairy2i
 * quantised widely-linear layer (arXiv 2512.02901).
 *
 * The layer: a real linear map y~ = A x~ with A in R^{2N x 2K} (Sec. 3.1,
 * real-layer equation) is rewritten exactly as y = U x + W conj(x) with
 * U, W in C^{N x K} (Sec. 3.1, Eq. UW-from-R and the exact-equivalence
 * theorem).  U and W are quantised independently (Sec. 3.3, last paragraph)
 * by T stages of recursive residual PhaseQuant (Sec. 3.2 Eq. ifairy-proj,
 * ifairy-scale, ifairy-dequant; Sec. 3.3 formal definition) to 2-bit codes
 * over {+1, +i, -1, -i} with one (s_re, s_im) pair per matrix and stage.
 * Inference computes y = sum_t (U^(t) x + W^(t) conj(x)) from the codes
 * without multiplying by weights (Sec. 3.4, Algorithm 1, extended here with
 * the W conj(x) term and a batch of tokens).
 *
 * Conventions shared by every call
 * --------------------------------
 *  - N is the complex output dimension, K the complex input dimension; the
 *    real layer is 2N x 2K.  Real vectors pair as stacked halves:
 *    x~ = [Re x ; Im x] (Sec. 3.1).
 *  - Every pointer argument is DEVICE memory, owned and allocated by the
 *    caller; the library never keeps a pointer after the call returns and
 *    never allocates, frees or synchronises.
 *  - `stream` is a borrowed hipStream_t (NULL = the default stream); all
 *    work is enqueued on it and the call returns without waiting.
 *  - Argument checks run on the host before anything is enqueued; a failed
 *    check returns its status and enqueues nothing.  A HIP launch error
 *    returns FAIRY2I_ERR_HIP.  No exception or abort crosses the ABI.
 *  - Complex arrays are interleaved (re, im) float pairs, row-major
 *    (the memory of torch.complex64).
 *  - Codes: code k in {0,1,2,3} stands for the codeword i^k
 *    (0 -> +1, 1 -> +i, 2 -> -1, 3 -> -i).  Packed layout per matrix:
 *    uint8 codes[T][N][K/4]; code (t, i, j) is in byte (i*K + j)/4 at bits
 *    2*(j%4) and 2*(j%4)+1.  T*N*K/4 bytes per matrix, i.e. T bits per real
 *    parameter for the pair (Sec. 3.4, storage paragraph).
 *  - Scales: float32 scales[T][2] = (s_re, s_im) per matrix.
 *  - Calls are stateless and may be issued from several host threads.
 */
#ifndef FAIRY2I_H
#define FAIRY2I_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef int32_t fairy2i_status;

enum {
  FAIRY2I_OK = 0,
  FAIRY2I_ERR_NULL = 1,        /* a required pointer is NULL               */
  FAIRY2I_ERR_SHAPE = 2,       /* a dimension is out of range              */
  FAIRY2I_ERR_STAGES = 3,      /* T outside [1, FAIRY2I_MAX_STAGES]        */
  FAIRY2I_ERR_DTYPE = 4,       /* unknown activation dtype                 */
  FAIRY2I_ERR_UNSUPPORTED = 5, /* valid but not implemented combination    */
  FAIRY2I_ERR_WORKSPACE = 6,   /* workspace missing or too small           */
  FAIRY2I_ERR_HIP = 7          /* a HIP runtime call or launch failed      */
};

/* Activation element types for fairy2i_wl_matmul / fairy2i_quantize_act_int8. */
enum {
  FAIRY2I_ACT_F32 = 0,  /* float32 pairs (re, im): B*K*2 floats            */
  FAIRY2I_ACT_BF16 = 1, /* bf16 pairs (re, im): B*K*2 uint16 bf16 patterns  */
  FAIRY2I_ACT_I8 = 2    /* int8 pairs (re, im): B*K*2 int8, plus a float32
                           dequantisation factor per token                  */
};

/* Device layouts of packed codes.  D3 is the canonical one (what
 * fairy2i_quantize writes and every call accepts); TILED and TILED_FP4 are
 * the decode layouts written by fairy2i_repack_tiled and
 * fairy2i_repack_tiled_fp4, accepted by the grouped decode. */
enum {
  FAIRY2I_LAYOUT_D3 = 0,
  FAIRY2I_LAYOUT_TILED = 1,
  FAIRY2I_LAYOUT_TILED_FP4 = 2
};

#define FAIRY2I_MAX_STAGES 4
/* Largest token count served by the decode kernels for float activations;
 * larger batches need int8 activations (the prefill GEMM). */
#define FAIRY2I_MAX_DECODE_BATCH 16
/* Largest N*K (complex entries per matrix) the quantiser accepts. */
#define FAIRY2I_MAX_QUANTIZE_ENTRIES ((int64_t)1 << 31)

/* Human-readable name of a status code (static storage, never NULL). */
const char* fairy2i_status_string(fairy2i_status status);

/* Version of this ABI (incremented on any incompatible change). */
int32_t fairy2i_abi_version(void);

/*
 * Real layer -> widely-linear pair.  Sec. 3.1, Eq. (UW-from-R):
 *   R11 = A[:N,:K], R12 = A[:N,K:], R21 = A[N:,:K], R22 = A[N:,K:],
 *   Re U = (R11+R22)/2, Im U = (R21-R12)/2, Re W = (R11-R22)/2, Im W = (R12+R21)/2.
 * A: float32 [rows][cols] row-major, rows = 2N (outputs), cols = 2K (inputs).
 * U, W: complex64 [N][K] outputs; each component is the exact value rounded
 * once to float32.  rows and cols must be even and > 0 (the paper pads an odd
 * dimension with a zero channel: Sec. 3.1 remarks; the caller does that).
 * Errors: NULL pointer -> FAIRY2I_ERR_NULL; odd or non-positive dims ->
 * FAIRY2I_ERR_SHAPE.
 */
fairy2i_status fairy2i_to_widely_linear(const float* A, int64_t rows, int64_t cols,
                                        float* U, float* W, void* stream);

/* Bytes of device workspace fairy2i_quantize needs for an N x K matrix. */
size_t fairy2i_quantize_workspace_bytes(int64_t N, int64_t K, int32_t T);

/*
 * Recursive residual PhaseQuant of ONE complex matrix (call it once for U and
 * once for W).  Sec. 3.3 formal definition, with Sec. 3.2:
 *   R(0) = M;  for t < T:
 *     k(t)  = code of the nearest codeword by angle (Eq. ifairy-proj; ties
 *             take the floor form's counter-clockwise codeword, 0 -> +1),
 *     s_re  = mean |Re r| over entries coded +-1, s_im = mean |Im r| over
 *             entries coded +-i (Eq. ifairy-scale, per tensor); each mean is
 *             computed exactly and rounded once to float32; 0 if empty,
 *     R(t+1) = R(t) - (s_re b_re + i s_im b_im) with the stored float32
 *             scales, carried in float64.
 * M: complex64 [N][K] input.  codes: uint8 [T][N][K/4] output (packed
 * layout above).  scales: float32 [T][2] output.  workspace: device buffer
 * of at least fairy2i_quantize_workspace_bytes(N, K, T) bytes, contents
 * ignored on entry.  Results are bitwise deterministic.
 * Errors: FAIRY2I_ERR_NULL; FAIRY2I_ERR_SHAPE if N, K <= 0, K % 4 != 0 or
 * N*K > FAIRY2I_MAX_QUANTIZE_ENTRIES; FAIRY2I_ERR_STAGES; FAIRY2I_ERR_WORKSPACE.
 */
fairy2i_status fairy2i_quantize(const float* M, int64_t N, int64_t K, int32_t T,
                                uint8_t* codes, float* scales,
                                void* workspace, size_t workspace_bytes, void* stream);

/*
 * fairy2i_quantize with per-group axis scales (Sec. 1 and the footnote to
 * Eq. ifairy-scale name per-group scale sharing; the paper itself uses one
 * pair per tensor).  A group is G consecutive input columns of one output
 * row, j in [g G, min((g+1) G, K)), so a row has ngroups = ceil(K / G)
 * groups and the last may be shorter.  Each stage projects every entry as
 * above; each group gets its own (s_re, s_im), the exact mean over the
 * group's entries rounded once to float32 (0 for an empty axis group); the
 * residual subtracts the stored scales of the entry's own group.
 * M: complex64 [N][K].  codes: uint8 [T][N][K/4] output (packed layout
 * above).  scales: float32 [T][N][ngroups][2] output.  No workspace.
 * Results are bitwise deterministic.
 * Errors: FAIRY2I_ERR_NULL; FAIRY2I_ERR_SHAPE if N, K <= 0, K % 4 != 0,
 * N*K > FAIRY2I_MAX_QUANTIZE_ENTRIES, G < 4 or G % 4 != 0;
 * FAIRY2I_ERR_STAGES.
 */
fairy2i_status fairy2i_quantize_grouped(const float* M, int64_t N, int64_t K, int32_t T, int64_t G,
                                        uint8_t* codes, float* scales, void* stream);

/*
 * Per-token int8 activations (the paper names INT8 activations for its
 * look-up-table inference paragraph in Sec. 3.4 without defining the
 * quantiser; this is the library's definition).  For token b, in float32:
 *   g = max over the 2K real components |x|,  inv = 127 / g (IEEE division),
 *   q = clamp(rint(x * inv), -127, 127)  (round half to even),
 *   x_scale[b] = g / 127;  g = 0 gives q = 0 and x_scale = 0.
 * x: B*K*2 values of `dtype` (FAIRY2I_ACT_F32 or FAIRY2I_ACT_BF16),
 * interleaved (re, im).  q: int8 [B][K][2] output.  x_scale: float32 [B].
 * Errors: FAIRY2I_ERR_NULL; FAIRY2I_ERR_SHAPE if B or K <= 0;
 * FAIRY2I_ERR_DTYPE for any other dtype.
 */
fairy2i_status fairy2i_quantize_act_int8(const void* x, int32_t dtype, int64_t B, int64_t K,
                                         int8_t* q, float* x_scale, void* stream);

/* Bytes of device workspace fairy2i_wl_matmul needs (0 if none). */
size_t fairy2i_wl_matmul_workspace_bytes(int64_t N, int64_t K, int32_t T, int64_t B,
                                         int32_t dtype);

/*
 * Quantised widely-linear product for a batch of B tokens (Sec. 3.4,
 * Algorithm 1, read with the dequantisation of Eq. ifairy-dequant and the
 * deployed sum of Eq. res-sum, and with the W conj(x) term of
 * Eq. widely-linear):
 *   y[b] = sum_t ( U^(t) x_b + W^(t) conj(x_b) ),
 *   U^(t) = s^U_re(t) B_re(t) + i s^U_im(t) B_im(t)   (W^(t) likewise).
 * codes_U, codes_W: uint8 [T][N][K/4]; scales_U, scales_W: float32 [T][2].
 * x: B*K*2 activations of `dtype`, interleaved (re, im).  For
 * FAIRY2I_ACT_I8, x_scale is float32 [B] (dequantisation factor per token,
 * as produced by fairy2i_quantize_act_int8) and y[b] is multiplied by it;
 * for the float dtypes x_scale must be NULL.
 * y: complex64 [B][N] output.
 * Accumulation is exact integer arithmetic on the matrix cores, or float32
 * in the vector kernel, always in a fixed order: results are bitwise
 * reproducible run to run.
 * B <= FAIRY2I_MAX_DECODE_BATCH runs the decode kernels: bf16 and int8
 * activations with K % 64 == 0 go to the int8 matrix cores (bf16 tokens as
 * a 23-bit block fixed point, exact for every value within 2^14 of the
 * token's largest magnitude, smaller values rounded to that grid), other
 * cases to a float32 / int32 vector kernel.  Larger B needs FAIRY2I_ACT_I8
 * and runs the int8-MFMA prefill GEMM: with K % 64 == 0 (and sizes within
 * 32-bit offsets) a workspace holds the activations in the matrix-core
 * operand layout and the GEMM streams operands through LDS; otherwise a
 * direct kernel runs without workspace.
 * workspace: at least fairy2i_wl_matmul_workspace_bytes(...) bytes of
 * device memory (may be NULL when that is 0), contents ignored on entry.
 * Errors: FAIRY2I_ERR_NULL; FAIRY2I_ERR_SHAPE if N, K, B <= 0 or K % 4;
 * FAIRY2I_ERR_STAGES; FAIRY2I_ERR_DTYPE; FAIRY2I_ERR_UNSUPPORTED for
 * B > FAIRY2I_MAX_DECODE_BATCH with float activations, or a non-NULL
 * x_scale with float activations; FAIRY2I_ERR_WORKSPACE.
 */
fairy2i_status fairy2i_wl_matmul(const uint8_t* codes_U, const float* scales_U,
                                 const uint8_t* codes_W, const float* scales_W,
                                 int32_t T, int64_t N, int64_t K,
                                 const void* x, const float* x_scale, int32_t dtype, int64_t B,
                                 float* y, void* workspace, size_t workspace_bytes,
                                 void* stream);

/*
 * fairy2i_wl_matmul for callers that cannot allocate device memory (code
 * under HIP graph capture, serving loops, harnesses that forbid hipMalloc):
 * the same arguments without the workspace, which is taken from a device
 * array of FAIRY2I_NOALLOC_SCRATCH_BYTES that the library holds on every GPU
 * it runs on until the process ends (the array of the current device is used;
 * `stream` must belong to that device).  Nothing is allocated or freed.
 * Results are bitwise those of fairy2i_wl_matmul.  All calls on one GPU share
 * that GPU's array: calls that overlap on one GPU (other streams, other host
 * threads) race and must be serialised by the caller.  The workspace's
 * contents are never read before being written, so no clearing is needed.
 * Errors: as fairy2i_wl_matmul; FAIRY2I_ERR_WORKSPACE when the call would
 * need more than FAIRY2I_NOALLOC_SCRATCH_BYTES of workspace
 * (fairy2i_wl_matmul_workspace_bytes; for example more than about 2900
 * int8 tokens at K = 5504); FAIRY2I_ERR_HIP if the array's address cannot be
 * obtained.
 */
#define FAIRY2I_NOALLOC_SCRATCH_BYTES ((size_t)32 << 20)
fairy2i_status fairy2i_wl_matmul_noalloc(const uint8_t* codes_U, const float* scales_U,
                                         const uint8_t* codes_W, const float* scales_W,
                                         int32_t T, int64_t N, int64_t K,
                                         const void* x, const float* x_scale, int32_t dtype, int64_t B,
                                         float* y, void* stream);

/*
 * The exact integer products behind the int8 path of fairy2i_wl_matmul,
 * exported so they can be compared bit for bit:
 *   acc[M][t][p][b][i][c] = sum_j B^{M,t}_p[i][j] * q[b][j][c]
 * with M in {0 = U, 1 = W}, p in {0 = b_re plane, 1 = b_im plane} (entries in
 * {-1, 0, +1}, the 2x2 real blocks of Eq. realify-ops split by axis) and
 * c in {0 = re, 1 = im}.  acc: int32 [2][T][2][B][N][2] output.
 * It runs the same kernels as fairy2i_wl_matmul with FAIRY2I_ACT_I8 and the
 * same B (decode for B <= FAIRY2I_MAX_DECODE_BATCH, prefill above), with the
 * epilogue replaced by a store of the accumulators.
 * Errors: as fairy2i_wl_matmul.
 */
fairy2i_status fairy2i_wl_int8_accumulators(const uint8_t* codes_U, const uint8_t* codes_W,
                                            int32_t T, int64_t N, int64_t K,
                                            const int8_t* q, int64_t B, int32_t* acc,
                                            void* workspace, size_t workspace_bytes,
                                            void* stream);

/*
 * One layer of a grouped decode call (fairy2i_wl_matmul_group): the same
 * arguments fairy2i_wl_matmul takes for one layer.  All pointers are device
 * memory; x is B*K*2 activations of the group's dtype, x_scale is float32 [B]
 * for FAIRY2I_ACT_I8 and NULL otherwise, y is complex64 [B][N].
 */
typedef struct fairy2i_wl_layer {
  const uint8_t* codes_U;
  const float* scales_U;
  const uint8_t* codes_W;
  const float* scales_W;
  const void* x;
  const float* x_scale;
  float* y;
  int64_t N;
  int64_t K;
  int32_t layout;    /* FAIRY2I_LAYOUT_D3, _TILED or _TILED_FP4, for both
                        codes_U and codes_W (same T as the call)           */
  int32_t group_size; /* 0: scales_U, scales_W are float32 [T][2] (one pair
                        per stage).  G > 0: per-group scales as written by
                        fairy2i_quantize_grouped, float32
                        [T][N][ceil(K / G)][2]; G a multiple of 256 and
                        layout FAIRY2I_LAYOUT_TILED_FP4 (see below)          */
} fairy2i_wl_layer;

/*
 * Grouped decode: the product of fairy2i_wl_matmul for many independent
 * layers (for example every projection of a decoder stack, each with its own
 * input) in a fixed number of kernel launches, so the weight stream of all
 * layers runs back to back instead of paying a launch per layer.
 * Restrictions: dtype FAIRY2I_ACT_BF16 or FAIRY2I_ACT_I8, 1 <= B <= 16,
 * every K a multiple of 64.  Each layer's codes are in the
 * layout its `layout` field names (same layout for U and W).  With
 * FAIRY2I_LAYOUT_TILED_FP4 every layer of the group must use it, with dtype
 * FAIRY2I_ACT_BF16 and B <= 16 (B <= 8 for T = 3, B <= 4 for T = 4); the
 * product then runs on the
 * fp8 x fp4 matrix cores.  Each token is scaled by a power of two 2^S so that
 * its largest magnitude m lies in [2^7, 2^8).  For B <= 4 (B <= 2 when T = 4)
 * a scaled value v is split by magnitude into two bands (|v| >= 1, and |v| < 1 taken times 2^8),
 * and each band value u is written as two e4m3 digits, hi = e4m3(u) and
 * lo = e4m3((u - hi) * 2^5) (round to nearest even), u = hi + 2^-5 lo.  Every
 * value down to 2^-22 m is represented exactly, smaller ones to within
 * 2^-30 m.  The digit products are exact and are summed in float32 on the
 * matrix cores; y matches the exact product of the bf16 inputs to float32
 * rounding (relative L2 about 1e-7, also for tokens with 3000-sigma
 * channels).  For 5 <= B <= 16 (3 <= B <= 4 when T = 4) each value gets one
 * (hi, lo) pair (four tokens per 16-column tile): still exact per value, but
 * the matrix core's narrow adder may drop the low bits of a small product
 * next to one near m in the same group of products, at most about 2^-13 of
 * the larger; relative L2 about 3e-6 for N(0,1) tokens and up to 1.8e-4
 * with a 3000-sigma channel, inside the 1e-3 bar for bf16 activations.
 * Per-group scales (group_size G > 0) are supported on this fp4 path only,
 * for every layer of the group or for none (G may differ between layers).
 * The products of each 256-code step then start from zero and are folded,
 * in float32, into sums scaled by the step's group scales (Eq. ifairy-dequant
 * per group); the scale arrays are read alongside the codes (8 bytes per
 * row, group, stage and matrix).
 *
 * Use: size the workspace with fairy2i_wl_group_workspace_bytes and the
 * table with fairy2i_wl_group_table_bytes; fairy2i_wl_group_build_table
 * (host only, enqueues nothing) checks every layer and writes the table into
 * HOST memory `table`; copy those bytes unchanged to device memory; then each
 * fairy2i_wl_matmul_group(table, table_device, stream) computes every layer's
 * y.  The workspace and both table copies must stay alive and unchanged while
 * calls that use them run; calls sharing a workspace must not overlap.
 * Results equal fairy2i_wl_matmul on each layer up to the float32 rounding
 * of the split-K sums (a one-layer call may cut K into more slices to fill
 * the GPU); repeated calls are bitwise identical.
 * Errors: as fairy2i_wl_matmul, checked per layer by the build call;
 * FAIRY2I_ERR_UNSUPPORTED for the restrictions above; FAIRY2I_ERR_SHAPE if
 * n_layers < 1; fairy2i_wl_matmul_group returns FAIRY2I_ERR_NULL for a NULL
 * table and FAIRY2I_ERR_UNSUPPORTED for bytes that are not a built table.
 */
/*
 * Tiled decode layout of one matrix's packed codes (the code values and
 * their packing into bytes are those of D3; only the byte order changes).
 * Codes are cut into tiles of 16 rows x 256 codes (1024 bytes per stage);
 * tile (row block rb, 256-code step s, stage t) is stored at byte offset
 *     ((rb * ceil(K/256) + s) * T + t) * 1024
 * and byte 16 * (16 g + r) + e of the tile is D3 byte 64 s + 16 g + e of
 * row 16 rb + r of stage t (g < 4, r < 16, e < 16); bytes past row N - 1 or
 * past the row's K/4 bytes are 0.  A 256-code step of one row block is then
 * one contiguous 1024-byte run per stage, which is what one wave of the
 * decode product loads at once.
 * fairy2i_repack_tiled_bytes: bytes of the tiled copy, T * ceil(N/16) *
 * ceil(K/256) * 1024 (0 for invalid sizes).
 * fairy2i_repack_tiled: codes (D3, T*N*K/4 bytes) -> tiled (device memory,
 * tiled_bytes >= fairy2i_repack_tiled_bytes); enqueued on `stream`.
 * Errors: FAIRY2I_ERR_NULL; FAIRY2I_ERR_SHAPE for N < 1, K < 4, K % 4 != 0;
 * FAIRY2I_ERR_STAGES; FAIRY2I_ERR_WORKSPACE if tiled_bytes is too small;
 * FAIRY2I_ERR_HIP.
 */
size_t fairy2i_repack_tiled_bytes(int64_t N, int64_t K, int32_t T);
fairy2i_status fairy2i_repack_tiled(const uint8_t* codes, int64_t N, int64_t K, int32_t T,
                                    uint8_t* tiled, size_t tiled_bytes, void* stream);

/*
 * Fp4 tiled decode layout of one matrix's packed codes (Sec. 3.4 codes
 * i^k; same tiles and size as the tiled layout, fairy2i_repack_tiled_bytes).
 * Lane (g, r) (g < 4, r < 16) owns bytes 16 * (16 g + r) .. + 15 of tile
 * (rb, s, t), read as four little-endian 32-bit words; it holds codes
 * 256 s + 128 kb + 32 g + n (kb < 2, n < 32) of row 16 rb + r of stage t.
 * Writing n = 16 h + 8 a + m (h, a < 2, m < 8), code n is in word 2 kb + h,
 * nibble m (bits 4m .. 4m+3), with its bits p = k & 1 and q = k >> 1 at
 * nibble bits (1, 3) for a = 0 and (0, 2) for a = 1.  Codes past row N - 1 or
 * past K are 0.  A nibble masked to bits (3, 1), or to bit 3 with bit 1 set,
 * is then an e2m1 value of (1 - 2q) p or 1 - 2q, which the decode product
 * feeds to v_mfma_f32_16x16x128_f8f6f4 with five ALU instructions per
 * 16 codes.
 * fairy2i_repack_tiled_fp4: codes (D3, T*N*K/4 bytes) -> out (device memory,
 * out_bytes >= fairy2i_repack_tiled_bytes(N, K, T)); enqueued on `stream`.
 * Errors: as fairy2i_repack_tiled.
 */
fairy2i_status fairy2i_repack_tiled_fp4(const uint8_t* codes, int64_t N, int64_t K, int32_t T,
                                        uint8_t* out, size_t out_bytes, void* stream);

size_t fairy2i_wl_group_workspace_bytes(const fairy2i_wl_layer* layers, int32_t n_layers,
                                        int32_t T, int32_t dtype, int64_t B);
size_t fairy2i_wl_group_table_bytes(int32_t n_layers);
fairy2i_status fairy2i_wl_group_build_table(const fairy2i_wl_layer* layers, int32_t n_layers,
                                            int32_t T, int32_t dtype, int64_t B,
                                            void* workspace, size_t workspace_bytes,
                                            void* table, size_t table_bytes);
fairy2i_status fairy2i_wl_matmul_group(const void* table, const void* table_device, void* stream);

/*
 * fairy2i_wl_matmul_group with timing marks: records events[0] before the
 * first launch, events[1] after the activation-operand kernel, events[2]
 * after the product kernel and events[3] after the split-K reduction (each
 * on `stream`, with hipEventRecord), so a caller can time each kernel of the
 * call.  events: 4 hipEvent_t created by the caller.
 * Errors: as fairy2i_wl_matmul_group; FAIRY2I_ERR_NULL for NULL events.
 */
fairy2i_status fairy2i_wl_matmul_group_timed(const void* table, const void* table_device,
                                             void* stream, void* const* events);

/*
 * One widely-linear decoder block for one decode token (Sec. 1: every linear
 * layer of the LLaMA-style block converted; Sec. 3.1, self-attention
 * paragraph, Eq. hermitian-score).  With x the complex residual stream
 * (n entries standing for the 2n real components [Re x ; Im x]):
 *   z   = bf16(RMSNorm(x; norm_attn))            over the 2n real components
 *   q, k, v = the q, k, v widely-linear layers of z (grouped fp4 decode)
 *   q, k turned by the rotary embedding: entry j of a head times
 *        e^{i pos theta_j}, theta_j = rope_base^(-2 j / dh)
 *   k, v stored at position pos of the caches
 *   per head: s_m = Re(q^H k_m) / sqrt(dh) for m = 0 .. pos, p = softmax(s),
 *        o = sum_m p_m v_m;  o rounded to bf16
 *   h1  = x + o-layer(o)
 *   z2  = bf16(RMSNorm(h1; norm_mlp)); g, u = gate/up layers of z2
 *   act = bf16(silu(Re g) Re u + i silu(Im g) Im u)
 *   out = h1 + down-layer(act)
 * A head owns dc = n / n_heads consecutive complex entries; entry j holds the
 * head's real dims j and j + dc (dh = 2 dc), which makes the Hermitian score
 * the head's real dot-product score and the rotary embedding the half-split
 * rotation of those dims.  Caches: complex64 [n_heads][max_ctx][dc] each,
 * positions 0 .. pos - 1 filled by earlier calls.  All pointers are device
 * memory except where noted.  Reductions run in a fixed order: results are
 * bitwise reproducible.
 *
 * Use: fill fairy2i_block_desc (codes in the fp4 tiled layout of
 * fairy2i_repack_tiled_fp4, B = 1); size the workspace with
 * fairy2i_block_workspace_bytes and the plan with fairy2i_block_plan_bytes;
 * fairy2i_block_build_plan (host only, enqueues nothing) writes the plan into
 * HOST memory; copy those bytes unchanged to device memory; then each
 * fairy2i_block_decode(plan, plan_device, x, k_cache, v_cache, pos, out,
 * stream) runs the block for one token.  The workspace, the weights and both
 * plan copies must stay alive and unchanged while calls that use them run;
 * calls sharing a workspace must not overlap.
 * Errors: FAIRY2I_ERR_NULL; FAIRY2I_ERR_SHAPE for sizes that are not
 * positive, n % n_heads != 0, dc odd or above 256, n or n_ff not a multiple
 * of 64, T out of range, max_ctx above 262144, or pos outside [0, max_ctx);
 * FAIRY2I_ERR_WORKSPACE;
 * FAIRY2I_ERR_UNSUPPORTED for a plan not built by this library version;
 * FAIRY2I_ERR_HIP.
 */
typedef struct fairy2i_block_desc {
  int64_t n;          /* complex width of the residual stream (2n real)        */
  int64_t n_ff;       /* complex width of the gate/up outputs and down input   */
  int32_t n_heads;    /* attention heads                                       */
  int32_t T;          /* stages of every projection                            */
  int64_t max_ctx;    /* positions each cache holds                            */
  float eps;          /* RMSNorm epsilon                                       */
  int32_t reserved;   /* 0                                                     */
  double rope_base;   /* rotary base                                           */
  /* per projection, in the order q, k, v, o, gate, up, down: fp4 tiled codes
     and float32 [T][2] scales of U and W */
  const uint8_t* codes_U[7];
  const float* scales_U[7];
  const uint8_t* codes_W[7];
  const float* scales_W[7];
  const float* norm_attn;  /* float32 [2n]: gains of Re parts, then of Im parts */
  const float* norm_mlp;   /* float32 [2n] */
} fairy2i_block_desc;

size_t fairy2i_block_workspace_bytes(const fairy2i_block_desc* desc);
size_t fairy2i_block_plan_bytes(const fairy2i_block_desc* desc);
fairy2i_status fairy2i_block_build_plan(const fairy2i_block_desc* desc, void* workspace, size_t workspace_bytes,
                                        void* plan, size_t plan_bytes);
fairy2i_status fairy2i_block_decode(const void* plan, const void* plan_device, const float* x /* [n] complex64 */,
                                    float* k_cache, float* v_cache, int64_t pos, float* out /* [n] complex64 */,
                                    void* stream);
/*
 * Test export: the device addresses of the block's intermediate vectors in
 * its workspace, as the last fairy2i_block_decode on that workspace left
 * them: ptrs[0..11] = z (bf16 pairs [n]), q after the rotary embedding
 * (complex64 [n]), v (complex64 [n]), o (bf16 pairs [n]), o-layer output a,
 * h1, z2 (bf16 pairs [n]), g, u (complex64 [n_ff]), act (bf16 pairs [n_ff]),
 * down-layer output d (complex64 [n]), k before the rotary embedding
 * (complex64 [n]).  Host-only; enqueues nothing.
 * Errors: FAIRY2I_ERR_NULL; FAIRY2I_ERR_UNSUPPORTED for a foreign plan.
 */
fairy2i_status fairy2i_block_intermediates(const void* plan, void** ptrs);

/*
 * Host-side self-check of the exact-mean rounding used by fairy2i_quantize
 * for the axis scales: *out = float32 nearest (ties to even) to
 * (sum of |values[i]|) / n_values, with the sum taken exactly; 0 when
 * n_values == 0.  values is HOST memory (n_values finite doubles).  Runs on
 * the CPU with the same code the GPU uses; enqueues nothing.
 * Errors: FAIRY2I_ERR_NULL; FAIRY2I_ERR_SHAPE if n_values < 0 or
 * n_values > FAIRY2I_MAX_QUANTIZE_ENTRIES.
 */
fairy2i_status fairy2i_host_exact_mean_f32(const double* values, int64_t n_values, float* out);

/*
 * Quantisation-aware training of one widely-linear layer (Sec. 3.2, QAT
 * paragraph and remark (iii); Sec. 3.3, the QAT remarks after the formal
 * definition): full-precision masters, a fake-quantised forward pass, a
 * straight-through backward pass, and complex GEMMs with Gauss's three real
 * products.
 *
 * fairy2i_qat_fake_quant: the quantiser of fairy2i_quantize (same codes,
 * scales, workspace and errors) followed by the dequantised sum
 * W^ = sum_t (s_re b_re + i s_im b_im) of every entry (Eq. res-sum), summed
 * in double and rounded once to out_dtype: FAIRY2I_ACT_F32 (complex64
 * [N][K]) or FAIRY2I_ACT_BF16 (bf16 pairs [N][K][2]).  The codes and scales
 * are what fairy2i_qat_ste_backward takes.
 * Errors: as fairy2i_quantize; FAIRY2I_ERR_DTYPE for another out_dtype.
 */
fairy2i_status fairy2i_qat_fake_quant(const float* M, int64_t N, int64_t K, int32_t T, uint8_t* codes,
                                      float* scales, void* w_hat, int32_t out_dtype, void* workspace,
                                      size_t workspace_bytes, void* stream);

/*
 * Straight-through backward of the fake quantiser: from g_hat = dL/dW^
 * (complex64 [N][K], g = dL/dRe + i dL/dIm) to g_master = dL/dM (complex64
 * [N][K] output), through W^ = sum_t Q_t, Q_t = s_t b(R_t), R_{t+1} = R_t -
 * Q_t, R_0 = M, taking b(.) as the identity map of the complex entry (no
 * clipping radius) and each scale as the masked mean of Eq. (ifairy-scale)
 * with its mask fixed (d s_re / d Re r_j = b_re_j / n_re on the entries
 * coded +-1, likewise s_im).  Stage t, in reverse order, with H = dL/dR_{t+1}
 * (0 for t = T-1) and G_Q = g_hat - H:
 *   H += (s_re Re G_Q + b_re d_re) + i (s_im Im G_Q + b_im d_im),
 *   d_re = sum_j Re(G_Q_j) b_re_j / n_re,  d_im likewise (0 when empty).
 * The sums are taken in double in a fixed order (bitwise reproducible); H is
 * kept in g_master as complex64.  codes, scales: as written by
 * fairy2i_qat_fake_quant.  workspace: fairy2i_qat_ste_workspace_bytes(N, K).
 * Errors: FAIRY2I_ERR_NULL; FAIRY2I_ERR_SHAPE (as fairy2i_quantize);
 * FAIRY2I_ERR_STAGES; FAIRY2I_ERR_WORKSPACE.
 */
size_t fairy2i_qat_ste_workspace_bytes(int64_t N, int64_t K);
fairy2i_status fairy2i_qat_ste_backward(const uint8_t* codes, const float* scales, int32_t T, int64_t N, int64_t K,
                                        const float* g_hat, float* g_master, void* workspace,
                                        size_t workspace_bytes, void* stream);

/*
 * One operand of fairy2i_cgemm_gauss: `rows` x K complex values (rows = M
 * for A, N for B), either with K contiguous (trans = 0: element (r, k) at
 * index r * ld + k, ld >= K) or with the rows contiguous (trans = 1: element
 * (r, k) at index k * ld + r, ld >= rows).  dtype FAIRY2I_ACT_F32 (complex64
 * values) or FAIRY2I_ACT_BF16 (bf16 pairs); conj = 1 takes the conjugate.
 */
typedef struct fairy2i_cgemm_operand {
  const void* data;
  int64_t ld;
  int32_t dtype;
  int32_t trans;
  int32_t conj;
  int32_t reserved; /* 0 */
} fairy2i_cgemm_operand;

/*
 * Complex GEMM with Gauss's three real products (Sec. 3.2, remark (iii)):
 *   C[m][n] (+)= sum over segments s < nseg, k < K[s] of A[s](m, k) B[s](n, k)
 * with each complex product formed as P1 = Ar Br, P2 = Ai Bi,
 * P3 = (Ar + Ai)(Br + Bi), C = (P1 - P2) + i (P3 - P1 - P2): three real
 * products instead of four.  The operands are rounded to bf16 (the sums
 * Ar + Ai and Br + Bi formed in float32 from the inputs and rounded once)
 * and multiplied on the bf16 matrix cores with float32 accumulation.  Two
 * segments cover the widely-linear layer in one call: Y = X U^T + conj(X)
 * W^T (forward), G_X = G_Y conj(U) + conj(G_Y) W and [G_U | G_W] =
 * G_Y^T [conj(X) | X] (backward).  C: complex64 [M][ldc]; accumulate = 1
 * adds to C.  Error: the real part as exact as float32 accumulation of the
 * bf16 operands; the imaginary part carries the bf16 rounding of the two
 * sums, at most about 2^-8 sum_k |Ar + Ai| |Br + Bi| per element.
 * Errors: FAIRY2I_ERR_NULL; FAIRY2I_ERR_SHAPE for nseg outside [1, 2],
 * M, N, K[s] <= 0, ldc < N, an ld below its minimum, or a bad dtype / trans
 * / conj / reserved field; FAIRY2I_ERR_UNSUPPORTED for M above 4,194,240
 * (65,535 tiles of 64 rows) or N above 2^31.
 */
fairy2i_status fairy2i_cgemm_gauss(const fairy2i_cgemm_operand* A, const fairy2i_cgemm_operand* B, const int64_t* K,
                                   int32_t nseg, int64_t M, int64_t N, float* C, int64_t ldc, int32_t accumulate,
                                   void* stream);

/*
 * The same product as fairy2i_cgemm_gauss (Sec. 3.2, remark (iii)), with
 * the three real products run as plain GEMMs: a kernel writes each operand
 * as three bf16 planes (Re, Im, Re + Im, rounded exactly as in
 * fairy2i_cgemm_gauss, K padded to a multiple of 64 with zeros), one batched
 * bf16 GEMM of the vendor library (hipBLASLt, float32 accumulation) forms
 * P1, P2, P3, and a kernel writes C (+)= (P1 - P2) + i (P3 - P1 - P2).  The
 * result differs from fairy2i_cgemm_gauss only in the order of the float32
 * accumulation.  Arguments as fairy2i_cgemm_gauss, plus workspace: device
 * memory of at least fairy2i_cgemm_gauss_planar_workspace_bytes(K, nseg,
 * M, N) bytes, 256-byte aligned (the planes, the three float32 products and
 * the library's own 32 MiB), caller-owned; its contents are scratch.
 * fairy2i_cgemm_gauss_planar_workspace_bytes returns 0 for invalid sizes.
 * The first call on a device creates the library's handle there, and the
 * first call of a shape asks the library for its algorithm (kept for later
 * calls of that shape); neither is allowed under stream capture.
 * Errors: as fairy2i_cgemm_gauss; FAIRY2I_ERR_WORKSPACE for a missing or
 * short workspace; FAIRY2I_ERR_UNSUPPORTED for M or N above 4,194,240 or no
 * library algorithm for the shape; FAIRY2I_ERR_HIP for a library error.
 */
size_t fairy2i_cgemm_gauss_planar_workspace_bytes(const int64_t* K, int32_t nseg, int64_t M, int64_t N);
fairy2i_status fairy2i_cgemm_gauss_planar(const fairy2i_cgemm_operand* A, const fairy2i_cgemm_operand* B,
                                          const int64_t* K, int32_t nseg, int64_t M, int64_t N, float* C,
                                          int64_t ldc, int32_t accumulate, void* workspace, size_t workspace_bytes,
                                          void* stream);

/*
 * Real form of the layer's training products (Sec. 3.1, Eq. UW-from-R read
 * backwards, with Eq. realify-ops).  y = U x + W conj(x) is the real map of
 * (Re, Im) pairs whose 2 x 2 block for output n and input k is
 *   [ Re U + Re W   Im W - Im U ]
 *   [ Im U + Im W   Re U - Re W ]
 * fairy2i_wl_realify writes it as R: bf16 [2N][2K] row-major, entry
 * (2n + a, 2k + b) = block (a, b) of (n, k), each the exact sum or
 * difference of the two inputs rounded once (nearest even).  U, W: [N][K]
 * complex, float32 pairs (dtype FAIRY2I_ACT_F32) or bf16 pairs
 * (FAIRY2I_ACT_BF16), device memory.  With tokens stored as (re, im) pairs,
 * a [M][K] complex matrix is a real M x 2K matrix in place, and the three
 * products of a training step are plain real GEMMs (fairy2i_gemm_bf16):
 *   Y   [M][N] complex = X R^T     (forward; X bf16 pairs)
 *   G_X [M][K] complex = G_Y R     (G_Y rounded to bf16 pairs first)
 *   G_R [2N][2K] float = G_Y^T X
 * and fairy2i_wl_unrealify_grad reads G_U = G_Y^T conj(X) and
 * G_W = G_Y^T X (complex64 [N][K], device) off G_R's blocks:
 *   Re G_U = G_R[2n][2k] + G_R[2n+1][2k+1], Im G_U = G_R[2n+1][2k] - G_R[2n][2k+1],
 *   Re G_W = G_R[2n][2k] - G_R[2n+1][2k+1], Im G_W = G_R[2n][2k+1] + G_R[2n+1][2k].
 * These are the products fairy2i_cgemm_gauss computes with Gauss's three
 * real products per complex product; the real form needs four real products'
 * work for both segments instead of six, and no operand planes.
 * fairy2i_wl_realify_codes writes the same R straight from the quantised
 * pair (canonical packed codes uint8 [T][N][K/4] and scales float32 [T][2]
 * of U and of W, as fairy2i_quantize writes them; K % 4 == 0, R 16-byte
 * aligned): each entry of U^ and W^ is Eq. (res-sum) summed over the stages
 * in increasing order in double, each block entry formed from those and
 * rounded once to bf16 (no float32 U^, W^ in between, so a training step
 * that needs W^ only for its products can skip writing and reading it).
 * fairy2i_f32_to_bf16: out[i] = in[i] rounded to bf16 (nearest even),
 * n values, device memory.
 * Errors: FAIRY2I_ERR_NULL; FAIRY2I_ERR_DTYPE; FAIRY2I_ERR_STAGES;
 * FAIRY2I_ERR_SHAPE for non-positive sizes or N K > 2^30 (realify,
 * realify_codes, unrealify), K % 4 != 0 or a misaligned R (realify_codes),
 * n <= 0 (f32_to_bf16); FAIRY2I_ERR_HIP if a launch fails.
 */
fairy2i_status fairy2i_wl_realify(const void* U, const void* W, int32_t dtype, int64_t N, int64_t K, void* R,
                                  void* stream);
fairy2i_status fairy2i_wl_realify_codes(const uint8_t* codes_U, const float* scales_U, const uint8_t* codes_W,
                                        const float* scales_W, int32_t T, int64_t N, int64_t K, void* R,
                                        void* stream);
fairy2i_status fairy2i_wl_unrealify_grad(const float* G_R, int64_t N, int64_t K, float* G_U, float* G_W,
                                         void* stream);
fairy2i_status fairy2i_f32_to_bf16(const float* in, int64_t n, void* out, void* stream);

/*
 * Plain real GEMM on the matrix cores, for the real form above (the
 * vendor library, hipBLASLt, bf16 operands, float32 accumulation and
 * output): C = op(A) op(B), every matrix row-major in device memory:
 * op(A) is M x K, A itself (transA = 0, lda >= K) or the transpose of a
 * stored K x M matrix (transA = 1, lda >= M); op(B) is K x N, B itself
 * (transB = 0, ldb >= N) or the transpose of a stored N x K matrix
 * (transB = 1, ldb >= K); C: float32 M x N, ldc >= N, overwritten.
 * workspace: device buffer of at least fairy2i_gemm_bf16_workspace_bytes()
 * bytes for the library.  The library's first heuristic choice per problem
 * shape is kept for the process, unless fairy2i_gemm_bf16_tune chose one.
 * Errors: FAIRY2I_ERR_NULL; FAIRY2I_ERR_SHAPE (sizes, transposition flags,
 * leading dimensions); FAIRY2I_ERR_WORKSPACE; FAIRY2I_ERR_UNSUPPORTED if the
 * library offers no algorithm; FAIRY2I_ERR_HIP.
 */
size_t fairy2i_gemm_bf16_workspace_bytes(void);
/*
 * Tuning for fairy2i_gemm_bf16 (same arguments, C overwritten): times up to
 * 16 of the library's candidate algorithms for the problem on `stream`
 * (each run 2 + 5 times) and keeps the fastest for later calls of the same
 * problem in this process; *best_us (host, may be NULL) receives its time
 * per call.  This call SYNCHRONISES the stream (outside any graph capture);
 * without it a problem gets the library's first heuristic choice.
 * Errors: as fairy2i_gemm_bf16.
 */
fairy2i_status fairy2i_gemm_bf16_tune(const void* A, int64_t lda, int32_t transA, const void* B, int64_t ldb,
                                      int32_t transB, int64_t M, int64_t N, int64_t K, float* C, int64_t ldc,
                                      void* workspace, size_t workspace_bytes, float* best_us, void* stream);
fairy2i_status fairy2i_gemm_bf16(const void* A, int64_t lda, int32_t transA, const void* B, int64_t ldb,
                                 int32_t transB, int64_t M, int64_t N, int64_t K, float* C, int64_t ldc,
                                 void* workspace, size_t workspace_bytes, void* stream);

/*
 * CPU table-lookup product for int8 activations (Sec. 3.4, the paragraph on
 * lookup tables for CPU inference): every four consecutive codes of a row
 * (one byte of the canonical packed layout) index a 256-entry table of their
 * partial sums with the token's int8 activations, built once per token and
 * column group, so the row loop is table fetches and integer adds.  Host
 * code; every pointer is HOST memory and nothing runs on the GPU.
 *
 *   codes_U, codes_W: canonical packed codes, uint8 [T][N][K/4] each;
 *   scales_U, scales_W: float32 [T][2] (s_re, s_im); q: int8 [B][K][2]
 *   (re, im) as written by fairy2i_quantize_act_int8; x_scale: float32 [B]
 *   per-token dequantisation factors; y: complex64 [B][N] output, or NULL;
 *   acc: int32 [2][T][2][B][N][2] output (the layout of
 *   fairy2i_wl_int8_accumulators), or NULL.  At least one of y and acc.
 *   y is Eq. (ifairy-dequant) applied to the exact integer sums in double,
 *   stages in increasing order, U with q and W with conj(q), times x_scale,
 *   rounded once to float32.
 *   workspace: host scratch of at least fairy2i_cpu_lut_workspace_bytes(T,
 *   K, B, n_threads) bytes (the table plus per-thread accumulators), 16-byte
 *   aligned; n_threads <= 0 uses every CPU in the calling thread's affinity
 *   mask (at most 256).
 * The threads are a persistent pool owned by the library; concurrent calls
 * are serialised.
 * Errors: FAIRY2I_ERR_NULL; FAIRY2I_ERR_STAGES; FAIRY2I_ERR_SHAPE if N, K <=
 * 0, K % 4 != 0 or B outside [1, FAIRY2I_MAX_DECODE_BATCH];
 * FAIRY2I_ERR_WORKSPACE if the workspace is too small.
 */
size_t fairy2i_cpu_lut_workspace_bytes(int32_t T, int64_t K, int64_t B, int32_t n_threads);
fairy2i_status fairy2i_cpu_lut_wl_matmul(const uint8_t* codes_U, const float* scales_U,
                                         const uint8_t* codes_W, const float* scales_W,
                                         int32_t T, int64_t N, int64_t K,
                                         const int8_t* q, const float* x_scale, int64_t B,
                                         float* y, int32_t* acc,
                                         void* workspace, size_t workspace_bytes, int32_t n_threads);

/*
 * Matrix-core rate probe, for the roofline figures (not part of the method):
 * the sustained rate of the prefill GEMM's instruction (kind
 * FAIRY2I_PROBE_MFMA_I8: v_mfma_i32_16x16x64_i8, 32768 operations), of the
 * decode product's (FAIRY2I_PROBE_MFMA_F8F4: v_mfma_scale_f32_16x16x128_f8f6f4
 * with e4m3 x e2m1 operands, 65536 operations) or of the larger int8 shape
 * (FAIRY2I_PROBE_MFMA_I8_32X32: v_mfma_i32_32x32x32_i8, 65536 operations) on
 * this GPU at the clock it holds under that load.  Launches `blocks` blocks
 * of 256 threads on `stream`; every wave issues `iters` x 8 independent
 * MFMAs (x 4 for the 32 x 32 shape) with no memory traffic and writes one
 * int32 of their sums to sink[block * 256 + thread]
 * (device memory, blocks * 256 words, contents meaningless).  *ops (host)
 * receives the operations one launch performs; the caller times the launch.
 * Errors: FAIRY2I_ERR_NULL; FAIRY2I_ERR_UNSUPPORTED for another kind;
 * FAIRY2I_ERR_SHAPE unless 1 <= blocks <= 2^20 and 1 <= iters <= 2^24;
 * FAIRY2I_ERR_HIP if the launch fails.
 */
#define FAIRY2I_PROBE_MFMA_I8 0
#define FAIRY2I_PROBE_MFMA_F8F4 1
#define FAIRY2I_PROBE_MFMA_I8_32X32 2
fairy2i_status fairy2i_probe_mfma(int32_t kind, int32_t blocks, int32_t iters, int32_t* sink, double* ops,
                                  void* stream);

#ifdef __cplusplus
}
#endif

#endif /* FAIRY2I_H */
