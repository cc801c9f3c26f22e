// Internal declarations shared by the gfx950 kernels and the C ABI layer.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace saf3r {

constexpr int kHeadDim = 64;
constexpr int kBlock = 64;
constexpr int kMaxHeads = 256;
constexpr int kMaxBlocks = 16384;  // select keeps one score row per query block in LDS

enum Pattern : int32_t {
  kDense = 0,
  kFrameLocal = 1,
  kTopK = 2,
  kAnchor = 3,
  kStride = 4,
  kGlobalProbe = 5,
  kCosineTopK = 6
};

constexpr int kMaxCosineDim = 4096;   // feature width accepted by the cosine selection
constexpr int kMaxCosinePerFrame = 64;  // key blocks kept per frame by a cosine head
constexpr int kNmseParts = 128;         // NMSE partial sums per head (workspace pairs)
// Device array of saf3r_nmse_noalloc's partial sums: every head count the
// library accepts (one float64 pair per part).
constexpr int64_t kNmseScratchBytes = (int64_t)kMaxHeads * kNmseParts * 16;

// ---------------------------------------------------------------- launches

struct PoolArgs {
  int64_t n;            // tokens per head
  int32_t nb;           // blocks per head
  int32_t n_heads;      // heads to pool (the Top-K heads)
  int16_t head[kMaxHeads];
};

struct TopKArgs {
  int64_t n;
  int32_t nb;
  int32_t cap;
  int32_t rows_per_group;  // query blocks scored together by one workgroup
  int32_t n_heads;
  int16_t head[kMaxHeads];
  int32_t topk[kMaxHeads];
};

struct StaticArgs {
  int64_t n;
  int32_t nb;
  int32_t cap;
  int32_t tokens_per_frame;
  int32_t n_heads;
  int16_t head[kMaxHeads];
  int8_t pattern[kMaxHeads];
  int32_t param[kMaxHeads];  // ANCHOR: anchor frame; STRIDE: key stride
};

// Paper-literal query probe: one probe per head over all N queries.
struct GlobalArgs {
  int64_t n;
  int32_t nb;
  int32_t cap;
  int32_t n_heads;
  int16_t head[kMaxHeads];
  int32_t topk[kMaxHeads];
};

// Key-range split of long lists: on a layer of at least kSplitMinExtent key
// blocks, a list head whose list can hold kSplitMinBlocks or more key blocks
// runs as kSplitChunks work items per query block, item c walking the list
// entries in key blocks [c nb / C, (c + 1) nb / C). The waves that run together on an XCD then
// read K and V from one key range instead of the head's whole extent. Each
// item writes its unnormalised output and softmax statistics to a workspace
// and a merge launch combines the chunks in a fixed order.
constexpr int kSplitMinBlocks = 384;
constexpr int kSplitMinExtent = 4096;
constexpr int kSplitChunks = 4;
// Load balance: a list or dense head whose items walk at least
// kBalanceMinBlocks (bf16) or kBalanceMinBlocksF32 key blocks is also split
// when one item is longer than twice the layer's work spread over the chip's
// wave slots (256 CUs x 4 SIMDs x 2 waves), i.e. when its rows, not the total
// work, would set the launch's length. An fp32 tile costs about eight times
// a bf16 one (fp32 matrix cores, one wave per SIMD), so shorter fp32 rows
// are worth splitting.
constexpr int kBalanceMinBlocks = 32;
constexpr int kBalanceMinBlocksF32 = 8;
constexpr int64_t kWaveSlots = 2048;
constexpr int64_t kSplitItemBytes = (int64_t)kBlock * kHeadDim * 4 + (int64_t)kBlock * 2 * 4;

struct AttnArgs {
  int64_t n;
  int32_t nb;
  int32_t cap;
  int32_t heads;          // heads in this launch (entries of order[])
  int32_t slab;           // query blocks of one head handled by one XCD: ceil(nb / 8)
  int32_t mode;           // 0: lists or dense per head; 1: every head dense; 2: STRIDE heads
  int32_t splits;         // key ranges of a split head (kSplitChunks)
  float scale_log2;       // log2(e) / sqrt(64)
  float* part_o;          // split items' O^T accumulators, 64 x 64 fp32 each
  float* part_ml;         // split items' (running max, row sum) per query
  int16_t order[kMaxHeads];        // heads of this launch, longest work item first
  int16_t split_pos[kMaxHeads];    // by order position: index among split heads, or -1
  int32_t unit_start[kMaxHeads + 1];  // by order position: first work unit (slab units)
  int8_t dense[kMaxHeads];    // by head index: 1 = iterate all key blocks
  int32_t stride[kMaxHeads];  // by head index: key stride of a STRIDE head
};

// The merge of split heads: one wave per (split head, query block).
struct MergeArgs {
  int64_t n;
  int32_t nb;
  int32_t splits;
  int32_t n_split;
  int32_t dtype;  // of the output rows: 1 bf16, 0 fp32
  int16_t head[kMaxHeads];  // by split index: head
};

// Block-wise DINO Top-K on caller-supplied per-token features.
struct CosineArgs {
  int64_t n;
  int32_t nb;
  int32_t cap;
  int32_t dim;  // feature width
  int32_t tokens_per_frame;
  int32_t n_groups;                     // cosine heads grouped by per-frame count
  int32_t group_k[kMaxHeads];           // key blocks kept per frame by group g
  int16_t group_start[kMaxHeads + 1];   // group g: head[group_start[g] .. group_start[g + 1])
  int16_t head[kMaxHeads];
};

// List check of the listed heads: one wave per (head, query block).
struct ValidateArgs {
  int32_t nb;
  int32_t cap;
  int32_t n_heads;
  int16_t head[kMaxHeads];
  int32_t expect[kMaxHeads];  // by slot: the exact count a row must hold, or -1 (any)
};

hipError_t launch_pool(int dtype, const void* q, const void* k, double* qp, double* kp,
                       const PoolArgs& a, hipStream_t s);
hipError_t launch_select_topk(const double* qp, const double* kpT, int32_t* idx, int32_t* cnt,
                              double* scores, const TopKArgs& a, size_t lds_bytes, hipStream_t s);
hipError_t launch_select_static(int32_t* idx, int32_t* cnt, const StaticArgs& a, hipStream_t s);
// The list check on `s`, then its result copied to the host and the stream
// waited for: out[0] = rows that fail, out[1] = the lowest failing row
// (h * nb + i). `result` is the caller's 8-byte device workspace.
hipError_t run_validate_index(const int32_t* idx, const int32_t* cnt, int32_t* result,
                              const ValidateArgs& a, int32_t out[2], hipStream_t s);
hipError_t launch_select_global(const double* qp, const double* kpT, int32_t* idx, int32_t* cnt,
                                double* scores, const GlobalArgs& a, hipStream_t s);
hipError_t launch_cosine(int dtype, const void* f, double* fb, double* sim, int32_t* idx,
                         int32_t* cnt, const CosineArgs& a, hipStream_t s);
hipError_t launch_nmse(int dtype, const void* ref, const void* test, void* workspace, double* out,
                       int heads, int64_t n, hipStream_t s);
// Device address of the current device's NMSE scratch array (resolved on the
// first call on that device).
hipError_t nmse_scratch(void** ptr);
hipError_t launch_attention(int dtype, const void* q, const void* k, const void* v,
                            const int32_t* idx, const int32_t* cnt, void* out, float* lse,
                            const AttnArgs& a, hipStream_t s);
hipError_t launch_attention_merge(const float* part_o, const float* part_ml, void* out,
                                  float* lse, const MergeArgs& a, hipStream_t s);

// Top-K selection sizes, shared by the kernels and the host layer. Key
// slots per lane for a row of nb blocks: ceil(nb / 64) rounded up to a
// multiple of 4; a row occupies 64 * row_chunk(nb) words (LDS or workspace).
__host__ __device__ constexpr int row_chunk(int nb) { return ((nb + 63) / 64 + 3) & ~3; }
// LDS entries after the last row, so that every lane may read its C slots
// rounded up to a multiple of 8 unconditionally.
constexpr int kRowPad = 128;
// Bytes of LDS the single-launch Top-K selection needs for `rows` query blocks.
inline size_t topk_lds_bytes(int rows, int nb) {
  return ((size_t)rows * 64 * row_chunk(nb) + kRowPad) * sizeof(uint32_t);
}
// Threads per workgroup of the single-launch Top-K selection for `rows` query blocks.
inline int topk_threads(int rows) { return rows >= 16 ? 512 : 256; }
// Workspace path of the Top-K selection: bytes of one query block's key row.
inline size_t topk_ws_row_bytes(int nb) { return (size_t)64 * row_chunk(nb) * sizeof(uint32_t); }
// The workspace path's two launches (scores into `keys`, then one wave per row).
hipError_t launch_select_topk_ws(const double* qp, const double* kpT, uint32_t* keys, int32_t* idx,
                                 int32_t* cnt, double* scores, const TopKArgs& a, hipStream_t s);

}  // namespace saf3r
