// Decode (1..16 token) product on the int8 matrix cores: internal layer
// descriptors shared by the C-ABI layer and decode.hip.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace fairy2i {

constexpr int kModeBf16 = 0;  // bf16 activations as 3 base-256 digits of a 23-bit fixed point
constexpr int kModeI8 = 1;    // int8 activations with a per-token factor
constexpr int kModeBf16F4 = 2;  // bf16 activations as e4m3 digit pairs in two magnitude bands,
                                // codes in the fp4 tiled layout (fp8 x fp4 matrix cores)

constexpr int kCoopSlots = 4;     // steps in the cooperative kernel's ring
// Cooperative fp4 kernel geometry by its activation tiles per call (NT = 1,
// 2 or 4; three tiles run as four): waves per block (four for one or two
// tiles, three or two blocks per CU, whose barriers are independent; eight
// for four tiles, one block per CU, so that more row blocks share each
// step's activation operand), waves per row block (with four tiles two: one
// for the U planes, one for the W planes) and row blocks per group.
constexpr int coop_nt(int ntile) { return ntile >= 3 ? 4 : ntile; }
constexpr int coop_waves(int nt) { return nt >= 4 ? 8 : 4; }
constexpr int coop_plane_split(int nt) { return nt >= 4 ? 2 : 1; }
constexpr int coop_row_blocks(int ntile) { return coop_waves(coop_nt(ntile)) / coop_plane_split(coop_nt(ntile)); }
constexpr int kKernelReg = 0;     // codes staged in registers; any batch, accumulator export
constexpr int kKernelStream = 1;  // codes streamed through an LDS ring; one activation tile
constexpr int kRegKc4 = 2;        // 256-code steps per work item of the register kernel

// One layer of a decode call.  Workspace pointers (xf, xs, part) are carved
// out of the caller's workspace by the host code.
struct DecLayer {
  const uint8_t* codes[2];   // U, W: [T][N][K/4]
  const float* scales[2];    // U, W: [T][2]
  const void* x;             // [B][K][2] bf16 or int8
  const float* x_scale_in;   // int8: [B] dequantisation factors
  float2* y;                 // [B][N]
  int32_t* acc;              // accumulator export [2][T][2][B][N][2], else null
  int8_t* xf;                // activation operand [ntile][nk4][4][4][nc][16]
  float* xs;                 // per-token output factor [B]
  float2* part;              // split-K partials [nkc][B][N] (nkc > 1)
  int32_t N, K;
  int32_t nrb, nk4, nkc, kc4;  // 16-row blocks, 256-code steps, K slices, steps per slice
  int32_t tiled;             // codes in a tiled layout (tiled or fp4 tiled; else D3)
  int32_t gsteps;            // per-group scales: 256-code steps per group (scales [T][N][groups][2]);
                             // 0: one pair per stage (scales [T][2])
  int64_t item0;             // index of this layer's first work item
  int64_t step0;             // 256-code steps of all work items before item0
  int64_t sitem0;            // block-cooperative kernel: first group of coop_row_blocks row blocks
  int64_t sstep0;            //   and the group steps (groups x nk4) of all layers before this one
};

struct DecHeader {
  int32_t n_layers, T, mode, B;
  int32_t ntile;   // 16-column activation tiles
  int32_t nc;      // stored columns per tile (the first tile's valid columns)
  int32_t kernel;  // kKernelReg or kKernelStream
  int32_t grouped;  // every layer has per-group scales (fp4 path only)
  int32_t bands;    // fp4 path: activation digit bands per token (2: 8 columns, 1: 4 columns)
  int32_t max_nk4;  // the most 256-code steps of a layer of the call
  int64_t total_items;
  int64_t total_steps;  // 256-code steps of all work items
  int64_t total_ssteps; // block-cooperative kernel: steps of all row-block groups
  int32_t coop;         // every layer is one full-K item per row block: the cooperative kernel may run
  int32_t coop_rb;      // row blocks per group of the cooperative kernel
  // Cooperative kernel: groups [0, coop_dyn0) (coop_dyn_steps group steps) are
  // split over the blocks in equal shares of steps; the rest are claimed one
  // at a time at run time from *coop_ctr (zeroed by the activation
  // preparation of the same call).  coop_dyn0 == coop_groups: no claims.
  uint32_t* coop_ctr;
  int64_t coop_groups;
  int64_t coop_dyn0;
  int64_t coop_dyn_steps;
};

// Bytes at the start of a group call's workspace that hold the cooperative
// kernel's claim counter.
constexpr size_t kGroupCallBytes = 256;
// Fraction of a cooperative call's group steps split statically (the rest is
// claimed at run time, where the shortest groups sit).
constexpr double kCoopStaticFrac = 0.65;

// Group table of fairy2i_wl_group_build_table: this header followed by the
// layer descriptors (the device copy is read by the kernels at the same
// offsets).
constexpr uint32_t kGroupMagic = 0xFA112101u;
struct GroupTableHeader {
  uint32_t magic, abi;
  DecHeader h;
  int32_t any_split, pad0_;
  int64_t max_BN;
};
static_assert(sizeof(GroupTableHeader) % 16 == 0, "table header alignment");

int dec_f4_bands(int T, int64_t B);
int dec_ntile(int mode, int64_t B, int T);
int dec_ncols(int mode, int64_t B);
// Tiles of 16 activation columns processed per pass of the register kernel.
int dec_tiles_per_group(int T, int ntile);

// Header fields that do not depend on the layers (n_layers, total_items = 0).
DecHeader dec_header(int T, int mode, int64_t B, bool export_acc);

// Fill the geometry fields of `l` (N, K set) for header h and return its
// workspace bytes; with `ws` non-null also carve xf, xs, part out of it.
// `single`: a one-layer call (slices chosen to give the GPU enough items).
// `slice`: steps per K slice chosen for a whole group: 0 for the default
// (8), kSliceFullK for a group with enough row blocks that a layer of at most
// kMaxFullKSteps steps is not split along K (no partials, no reduction).
constexpr int kSliceFullK = -1;
constexpr int kMaxFullKSteps = 32;
constexpr int64_t kFullKMinItems = 12288;
constexpr int64_t kMinGroupItems = 2048;  // a small group gets shorter slices until it has this many items
size_t dec_layer_setup(DecLayer& l, const DecHeader& h, bool single, char* ws, int slice = 0);

// The fp8 x fp4 path (decode_f4.hip): activation operand and product
// launches of a kModeBf16F4 call (errors are left for hipGetLastError).
void launch_f4_prep(const DecHeader& h, const DecLayer& inl, const DecLayer* tab, hipStream_t s);
void launch_f4_product(const DecHeader& h, const DecLayer& inl, const DecLayer* tab, hipStream_t s);

hipError_t launch_decode(const DecHeader& h, const DecLayer& inl, const DecLayer* tab,
                         int any_split, int64_t max_BN, bool export_acc, int64_t acc_elems,
                         int32_t* acc, hipStream_t s, hipEvent_t const* events = nullptr);

}  // namespace fairy2i
