// Block-sparse attention over the kept key blocks (Sec. 4.1: the Top-K and
// static kernels compute only the scores between the queries and the
// selected keys, and the softmax is renormalised over that set), with the
// dense ("Full") case as the same loop over every key block.
//
// One wave owns one (head, 64-query block) and walks its kept-block list in
// half tiles of 32 keys with an online softmax:
//   S^T = K Q^T      (keys x queries) on MFMA, so a lane owns one query
//                    column and the row sum stays inside the lane pair
//                    (lane, lane ^ 32);
//   O^T += V^T P^T   (head dim x queries) on MFMA, P^T taken straight from
//                    the S^T accumulators, V^T read from LDS with the gfx950
//                    transposing LDS read so V is never transposed in memory.
// The half-tile steps are software-pipelined: step t issues S^T of half t+1
// and the P V product of half t-1 on the matrix cores while the VALU runs
// the softmax of half t, and the scheduler is told to interleave the two
// streams. Q sits in registers for the whole loop; K and V half tiles are
// staged in LDS by the direct buffer-to-LDS load two steps ahead. Every
// global access of Q, K, V and O is a buffer instruction whose range-checked
// offsets (vector and immediate, never the unchecked scalar offset) are
// bounded by the head's extent, so a partial last block reads zeros and a
// corrupt index list cannot touch memory outside the head.
//
// Launch order: workgroup b runs on XCD b % 8; each XCD takes a contiguous
// slab of query blocks of every head (neighbouring query blocks share kept
// key blocks, which then hit in that XCD's L2), longest work items first.
//
// Long lists can run split into key ranges: a work item is then (head, key
// range c of splits, query block) and walks only its list's entries inside
// range c (a dense head's item walks every block of the range), ranges in
// order within a head, so the waves that run together on an XCD read K and V
// from one range rather than the head's whole extent, and no item of a small
// layer is much longer than the others.
// Such an item stores its unnormalised O^T and (running max, row sum) per
// query in a workspace; attn_merge_kernel combines the ranges of each query
// block in range order.
//
// A launch in which every head is dense runs attn_bf16_dense_kernel: four
// waves take four neighbouring query blocks of one head, and since all four
// walk every key block in order, each K and V half tile is staged in LDS
// once for the four (one barrier per half-tile step).
#include <type_traits>

#include "saf3r_internal.h"

namespace saf3r {
namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x4 __attribute__((ext_vector_type(4)));
typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
typedef float f32x2 __attribute__((ext_vector_type(2)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef int i32x4 __attribute__((ext_vector_type(4)));
typedef int i32x2 __attribute__((ext_vector_type(2)));
typedef __attribute__((address_space(3))) bf16x4 lds_bf16x4;

constexpr uint32_t kRsrcWord3 = 0x00020000u;  // gfx9 buffer descriptor: 32-bit raw data
constexpr int kFStride = 65;                   // fp32 per LDS row (fp32 path)
constexpr float kNegInf = -__builtin_inff();
constexpr float kLn2 = 0.6931471805599453f;

__device__ inline __amdgpu_buffer_rsrc_t make_rsrc(const void* base, uint32_t bytes) {
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(base), (short)0, (int)bytes,
                                           (int)kRsrcWord3);
}

__device__ inline bf16x8 load_b128(__amdgpu_buffer_rsrc_t r, uint32_t byte_off) {
  return __builtin_bit_cast(bf16x8, __builtin_amdgcn_raw_buffer_load_b128(r, (int)byte_off, 0, 0));
}

__device__ inline float fast_exp2(float x) { return __builtin_amdgcn_exp2f(x); }

struct Work {
  int h, i;
  int chunk;  // key range of a split head's item, or -1
  int item;   // split item index (partials), or -1
  bool valid;
};

// Work unit u = b / 8 of order position hh covers unit_start[hh] <= u <
// unit_start[hh + 1]: slab units per key range, key ranges in order, so the
// items that run together on an XCD share one key range of one head.
__device__ inline Work work_item(const AttnArgs& a) {
  const int xcd = blockIdx.x & 7;
  const int u = blockIdx.x >> 3;
  Work w;
  w.valid = u < a.unit_start[a.heads];
  if (!w.valid) return w;
  int lo = 0, hi = a.heads;  // the last order position with unit_start <= u
  while (hi - lo > 1) {
    const int mid = (lo + hi) >> 1;
    if (a.unit_start[mid] <= u) lo = mid;
    else hi = mid;
  }
  const int r = u - a.unit_start[lo];
  const int chunk = r / a.slab;
  const int i = xcd * a.slab + (r - chunk * a.slab);
  w.valid = i < a.nb;
  w.h = a.order[lo];
  w.i = i;
  const int sp = a.split_pos[lo];
  w.chunk = sp >= 0 ? chunk : -1;
  w.item = sp >= 0 ? (sp * a.splits + chunk) * a.nb + i : -1;
  return w;
}

// A split item's share of its row: key blocks [c nb / splits, (c + 1) nb /
// splits) of range c. A dense head's item walks every block of the range
// (from dense_lo); a list head's item keeps its list's entries inside the
// range: in an ascending list, the entries after those below jlo and before
// the first at or above jhi (any other list still yields a sub-range of the
// row, read within it).
__device__ inline void split_range(const Work& w, const AttnArgs& a, bool dense,
                                   const int32_t*& list, int& count, int& dense_lo, int lane) {
  const int nb = a.nb;
  const int jlo = (int)(((int64_t)w.chunk * nb) / a.splits);
  const int jhi = (int)(((int64_t)(w.chunk + 1) * nb) / a.splits);
  if (dense) {
    dense_lo = jlo;
    count = jhi - jlo;
    return;
  }
  int below_lo = 0, below_hi = 0;
  for (int base = 0; base < count; base += 64) {
    const int p = base + lane;
    const int j = p < count ? list[p] : 0x7fffffff;
    below_lo += __popcll(__ballot(j < jlo));
    below_hi += __popcll(__ballot(j < jhi));
  }
  list += below_lo;
  count = max(below_hi - below_lo, 0);
}

typedef float f32x4_t __attribute__((ext_vector_type(4)));
typedef float f32x2_t __attribute__((ext_vector_type(2)));

// A split item's result: its O^T accumulators as they stand, relative to its
// own running max (register-major: 16 stores of 64 lanes x 16 B), and the
// (running max, row sum) of each query. An empty range writes only the
// statistics (-inf, 0), and the merge never reads its accumulators.
template <typename Acc>
__device__ inline void store_partials(const Acc (&o)[2][2], const float (&m)[2], const float (&lt)[2],
                                      const AttnArgs& a, int64_t item, bool empty, int lane) {
  const int l32 = lane & 31;
  if (!empty) {
    float* const po = a.part_o + item * (kBlock * kHeadDim);
#pragma unroll
    for (int c = 0; c < 2; ++c)
#pragma unroll
      for (int tq = 0; tq < 2; ++tq)
#pragma unroll
        for (int g = 0; g < 4; ++g)
          *(f32x4_t*)(po + (((c * 2 + tq) * 4 + g) * 64 + lane) * 4) =
              f32x4_t{o[c][tq][4 * g], o[c][tq][4 * g + 1], o[c][tq][4 * g + 2], o[c][tq][4 * g + 3]};
  }
  if ((lane >> 5) == 0) {
#pragma unroll
    for (int tq = 0; tq < 2; ++tq)
      *(f32x2_t*)(a.part_ml + (item * kBlock + 32 * tq + l32) * 2) =
          empty ? f32x2_t{-__builtin_inff(), 0.f} : f32x2_t{m[tq], lt[tq]};
  }
}

// fp32 output of one query block from the O^T accumulators (register e of
// tile [c][tq] of lane (l32, hf) is head dim 32c + 8(e/4) + 4hf + e%4 of
// query 32tq + l32), scaled by inv; lse_row, if not null, is the head's LSE
// row (natural log).
template <typename Acc>
__device__ inline void write_out_tile_f32(const Acc (&o)[2][2], const float (&inv)[2],
                                          const float (&lse_val)[2], __amdgpu_buffer_rsrc_t ro,
                                          float* lse_row, int i, int64_t n, int lane) {
  const int l32 = lane & 31;
  const int hf = lane >> 5;
#pragma unroll
  for (int tq = 0; tq < 2; ++tq) {
    const int query = i * kBlock + 32 * tq + l32;
#pragma unroll
    for (int c = 0; c < 2; ++c)
#pragma unroll
      for (int g = 0; g < 4; ++g) {
        f32x4_t ov;
#pragma unroll
        for (int r = 0; r < 4; ++r) ov[r] = o[c][tq][4 * g + r] * inv[tq];
        __builtin_amdgcn_raw_buffer_store_b128(__builtin_bit_cast(i32x4, ov), ro,
                                               (query * kHeadDim + 32 * c + 8 * g + 4 * hf) * 4, 0, 0);
      }
    if (lse_row && hf == 0 && query < n) lse_row[query] = lse_val[tq];
  }
}

// ------------------------------------------------------------------ bf16

typedef __attribute__((address_space(3))) void lds_void;
typedef __attribute__((address_space(3))) char lds_char;
typedef __attribute__((address_space(3))) const bf16x8 lds_bf16x8;

// LDS tiles: rows of 128 B; 16-byte chunk c of row r is stored at slot
// c ^ f(r), f(r) = (bit2(r), bit1(r), bit0(r) ^ bit1(r) ^ bit3(r)). With it
// the MFMA operand reads (16 rows at one chunk) and the transposing reads
// (4 rows x 2 chunks per 16 lanes, 4 x 4 per 32) touch every bank once,
// whether the LDS serves 128 or 256 bytes per clock.
__device__ inline int swz_f(int r) {
  return ((r >> 2) & 1) | (r & 2) | (((r ^ (r >> 1) ^ (r >> 3)) & 1) << 2);
}
__device__ inline int swz(int r, int c) { return r * 128 + ((c ^ swz_f(r)) << 4); }

// Direct buffer-to-LDS loads of 8-row groups: instruction n fills LDS bytes
// [1024n, 1024n + 1024), lane l its 16 bytes at 16l, i.e. row 8n + l/8,
// slot l%8, which must hold chunk (l%8) ^ f(8n + l/8) = (l%8) ^ f(l/8) ^ (4
// if n is odd). The lane's byte offset inside its 8-row group depends only
// on the parity of n; the group offset 1024n is the instruction's immediate
// offset, which the hardware adds to both the memory and the LDS address.
struct DmaLaneOffsets {
  int even, odd;
};
__device__ inline DmaLaneOffsets dma_lane_offset(int lane) {
  const int r = lane >> 3;
  const int c = (lane & 7) ^ swz_f(r);
  return {(r * kHeadDim + c * 8) * 2, (r * kHeadDim + (c ^ 4) * 8) * 2};
}
// max / sum of a value over the lane pair (l, l ^ 32) that shares a query
__device__ inline float pair_max(float x) {
  const auto s = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  return fmaxf(__uint_as_float(s[0]), __uint_as_float(s[1]));
}
__device__ inline float pair_sum(float x) {
  const auto s = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  return __uint_as_float(s[0]) + __uint_as_float(s[1]);
}

constexpr bf16x2 kOnes = {(__bf16)1.0f, (__bf16)1.0f};

// Waits expressed as s_waitcnt immediates (gfx9 encoding: vmcnt in bits 3:0
// and 15:14, expcnt 6:4, lgkmcnt 11:8).
constexpr int kWaitVm8 = 0x0F78;   // vmcnt(8)
constexpr int kWaitVm0 = 0x0F70;   // vmcnt(0)
constexpr int kWaitLgkm0 = 0xC07F; // lgkmcnt(0)

// One 32-row half tile (rows 64j + 32h .. of the head) into an LDS half
// buffer with the direct buffer-to-LDS load: four 1 KB instructions. The
// tile's offset goes into the base and extent of a descriptor built for this
// tile in scalar registers, and the scalar offset operand stays 0: the
// hardware range-checks the vector and immediate offsets against the extent
// but not the scalar offset. So rows past the head's last token (a partial
// last block) read zeros, and a block index outside [0, nb) reads a tile of
// zeros instead of memory outside the head.
// head_bytes - t, or 0 when t is at or past the end, on the scalar unit: as
// plain C the compiler lowers this saturating subtract of two scalars to a
// copy, a clamped vector subtract and a readfirstlane, three VALU
// instructions per tile load in the loop. The borrow of s_sub_u32 sets SCC.
__device__ inline uint32_t rem_bytes(uint32_t head_bytes, uint32_t t) {
  uint32_t r;
  asm("s_sub_u32 %0, %1, %2\n\ts_cselect_b32 %0, 0, %0" : "=&s"(r) : "s"(head_bytes), "s"(t) : "scc");
  return r;
}

__device__ inline void dma_half(const uint16_t* head, uint32_t head_bytes, int nb, int j, int h,
                                lds_char* buf, DmaLaneOffsets off) {
  const uint32_t t = __builtin_amdgcn_readfirstlane(
      (uint32_t)j < (uint32_t)nb ? ((uint32_t)j * kBlock + 32u * h) * (kHeadDim * 2) : head_bytes);
  const uint32_t rem = rem_bytes(head_bytes, t);
  const __amdgpu_buffer_rsrc_t r = make_rsrc(reinterpret_cast<const char*>(head) + t, rem);
  __builtin_amdgcn_raw_ptr_buffer_load_lds(r, (lds_void*)buf, 16, off.even, 0, 0, 0);
  __builtin_amdgcn_raw_ptr_buffer_load_lds(r, (lds_void*)buf, 16, off.odd, 0, 1024, 0);
  __builtin_amdgcn_raw_ptr_buffer_load_lds(r, (lds_void*)buf, 16, off.even, 0, 2048, 0);
  __builtin_amdgcn_raw_ptr_buffer_load_lds(r, (lds_void*)buf, 16, off.odd, 0, 3072, 0);
}

// Key sets a launch walks: per-head lists or all blocks (kLists), every block
// of every head (kAllDense), or the keys 0, s, 2s, ... of STRIDE heads taken
// 64 at a time as virtual blocks (kStrided).
enum AttnMode { kLists = 0, kAllDense = 1, kStrided = 2 };

// One 32-row half of virtual key block j of a STRIDE head: key rows
// (64j + 32h + r) * stride, r < 32, into an LDS half buffer (same slot layout
// as dma_half). Rows at or past token n load as zeros (offset past the
// buffer's extent).
__device__ inline void dma_half_strided(__amdgpu_buffer_rsrc_t r, int j, int h, lds_char* buf,
                                        int lane, int64_t stride, int64_t n, uint32_t head_bytes) {
  const int rr = lane >> 3;
  const int c = (lane & 7) ^ swz_f(rr);
#pragma unroll
  for (int g = 0; g < 4; ++g) {
    const int64_t row = ((int64_t)j * kBlock + 32 * h + 8 * g + rr) * stride;
    const uint32_t off = row < n ? (uint32_t)(row * kHeadDim * 2) + (uint32_t)(((g & 1) ? (c ^ 4) : c) * 16)
                                 : head_bytes;
    __builtin_amdgcn_raw_ptr_buffer_load_lds(r, (lds_void*)(buf + 1024 * g), 16, (int)off, 0, 0, 0);
  }
}

// Output of one query block from the O^T accumulators (register e of tile
// [c][tq] of lane (l32, hf) holds head dim 32c + 8(e/4) + 4hf + e%4 of query
// 32tq + l32): scaled by inv, rounded to bf16 into two idle LDS half buffers
// (query rows 0..31 in b0, 32..63 in b1, same swizzle as the K tiles), then
// stored as full 128-byte rows, eight 1 KB stores. lse_row, if not null, is
// the head's LSE row; lse_val is in natural log.
__device__ inline void write_out_tile(const f32x16 (&o)[2][2], const float (&inv)[2],
                                      const float (&lse_val)[2], lds_char* b0, lds_char* b1,
                                      __amdgpu_buffer_rsrc_t ro, float* lse_row, int i, int64_t n,
                                      int lane) {
  const int l32 = lane & 31;
  const int hf = lane >> 5;
#pragma unroll
  for (int tq = 0; tq < 2; ++tq) {
    const int query = i * kBlock + 32 * tq + l32;
    lds_char* const ob = tq ? b1 : b0;
#pragma unroll
    for (int c = 0; c < 2; ++c)
#pragma unroll
      for (int g = 0; g < 4; ++g) {
        bf16x4 ov;
#pragma unroll
        for (int r = 0; r < 4; ++r) ov[r] = (__bf16)(o[c][tq][4 * g + r] * inv[tq]);
        *(lds_bf16x4*)(ob + swz(l32, 4 * c + g) + 8 * hf) = ov;
      }
    if (lse_row && hf == 0 && query < n) lse_row[query] = lse_val[tq];
  }
#pragma unroll
  for (int nn = 0; nn < 8; ++nn) {
    const int row = 8 * nn + (lane >> 3);
    const int chunk = lane & 7;
    lds_char* const ob = row >= 32 ? b1 : b0;
    const bf16x8 val = *(lds_bf16x8*)(ob + swz(row & 31, chunk));
    __builtin_amdgcn_raw_buffer_store_b128(__builtin_bit_cast(i32x4, val), ro,
                                           (int)(((i * kBlock + row) * kHeadDim + 8 * chunk) * 2), 0, 0);
  }
}

// Per-wave state and building blocks of the bf16 walk over one 64-query
// block: Q^T in registers, the O^T accumulators, the running max and row-sum
// share of each query half, and the lane's LDS operand offsets.
template <bool kPin>
struct Bf16Walk {
  bf16x8 qB[2][4];  // Q^T as the B operand: qB[tq][s] = Q[64i + 32tq + l32][16s + 8hf + (0..7)]
  f32x16 o[2][2];   // O^T tiles [head-dim half c][query half tq]
  float nm[2];      // minus the running max of the log2-scaled scores (the fma's addend)
  float l[2];       // this lane's share of the running row sum
  float sc;
  int l32, hf;
  int tr_row, tr_col;  // transposing-read position of this lane in a 4-row x 16-column group
  // Lane parts of the LDS operand addresses: the K read of chunk pair st (row
  // l32), and the transposing V reads of column half c, rows +0 / +8 of a
  // 16-row group (the 16-row group's 2 KB is an immediate offset). With kPin
  // an empty asm redefines a part at each use, so the buffer's base also
  // goes into the immediate offset instead of one hoisted address register
  // per (buffer, part): eight registers in all for a ring of eight buffers.
  // With two buffers per tensor the hoisted addresses measured faster.
  int kpart[4];
  int vpart[2][2];

  __device__ __forceinline__ void init(__amdgpu_buffer_rsrc_t rq, int i, int lane, float scale) {
    l32 = lane & 31;
    hf = lane >> 5;
    sc = scale;
#pragma unroll
    for (int tq = 0; tq < 2; ++tq)
#pragma unroll
      for (int s = 0; s < 4; ++s)
        qB[tq][s] = load_b128(
            rq, (uint32_t)(((i * kBlock + 32 * tq + l32) * kHeadDim + 16 * s + 8 * hf) * 2));
#pragma unroll
    for (int c = 0; c < 2; ++c)
#pragma unroll
      for (int tq = 0; tq < 2; ++tq)
#pragma unroll
        for (int e = 0; e < 16; ++e) o[c][tq][e] = 0.f;
    nm[0] = nm[1] = -kNegInf;
    l[0] = l[1] = 0.f;
    tr_row = 4 * hf + ((lane & 15) >> 2);
    tr_col = 16 * ((lane >> 4) & 1) + 4 * (lane & 3);
#pragma unroll
    for (int st = 0; st < 4; ++st) kpart[st] = swz(l32, 2 * st + hf);
#pragma unroll
    for (int c = 0; c < 2; ++c)
#pragma unroll
      for (int r8 = 0; r8 < 2; ++r8)
        vpart[c][r8] = swz(tr_row + 8 * r8, (32 * c + tr_col) >> 3) + (tr_col & 7) * 2;
  }

  // S^T of a key half (32 keys x 64 queries) from an LDS K half buffer
  __device__ __forceinline__ void read_k(lds_char* kb, bf16x8 (&kA)[4]) {
#pragma unroll
    for (int st = 0; st < 4; ++st) {
      if constexpr (kPin) asm volatile("" : "+v"(kpart[st]));
      kA[st] = *(lds_bf16x8*)(kb + kpart[st]);
    }
  }
  __device__ __forceinline__ void read_v(lds_char* vb, bf16x8 (&vA)[2][2]) {
    if constexpr (kPin) {
#pragma unroll
      for (int c = 0; c < 2; ++c)
#pragma unroll
        for (int r8 = 0; r8 < 2; ++r8) asm volatile("" : "+v"(vpart[c][r8]));
    }
#pragma unroll
    for (int u = 0; u < 2; ++u)
#pragma unroll
      for (int c = 0; c < 2; ++c) {
        const bf16x4 lo = __builtin_amdgcn_ds_read_tr16_b64_v4bf16((lds_bf16x4*)(vb + 2048 * u + vpart[c][0]));
        const bf16x4 hi = __builtin_amdgcn_ds_read_tr16_b64_v4bf16((lds_bf16x4*)(vb + 2048 * u + vpart[c][1]));
        vA[u][c] = bf16x8{lo[0], lo[1], lo[2], lo[3], hi[0], hi[1], hi[2], hi[3]};
      }
  }
  __device__ __forceinline__ void mfma_s(const bf16x8 (&kA)[4], f32x16 (&s)[2]) {
    f32x16 acc0 = {}, acc1 = {};
#pragma unroll
    for (int st = 0; st < 4; ++st) {
      acc0 = __builtin_amdgcn_mfma_f32_32x32x16_bf16(kA[st], qB[0][st], acc0, 0, 0, 0);
      acc1 = __builtin_amdgcn_mfma_f32_32x32x16_bf16(kA[st], qB[1][st], acc1, 0, 0, 0);
    }
    s[0] = acc0;
    s[1] = acc1;
  }
  __device__ __forceinline__ void mfma_pv(const bf16x8 (&vA)[2][2], const bf16x8 (&p)[2][2]) {
#pragma unroll
    for (int u = 0; u < 2; ++u)
#pragma unroll
      for (int c = 0; c < 2; ++c)
#pragma unroll
        for (int tq = 0; tq < 2; ++tq)
          o[c][tq] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(vA[u][c], p[u][tq], o[c][tq], 0, 0, 0);
  }
  // Online-softmax step over one key half. P = exp2(s*sc - m) is taken with
  // the running max as it stands and rounded to bf16; the row sum adds the
  // rounded values (one bf16 dot with (1, 1) per pair), so the normaliser
  // matches the weights the P V product uses. Only when some lane's share of
  // the row sum leaves [0, 2^12] (a new larger max, or the first half where
  // the max is still -inf and the sum is inf or NaN) is the half's max taken:
  // the running max moves to it, O and l are rescaled (after the P V of the
  // previous half, which is already issued) and P is recomputed. Keys at or
  // past `valid` (a partial last block) get P = 0.
  __device__ __forceinline__ void probs(const f32x16 (&s)[2], bf16x8 (&p)[2][2], float (&rs)[2]) {
#pragma unroll
    for (int tq = 0; tq < 2; ++tq) {
      const float nmcur = nm[tq];
      float r = 0.f;
#pragma unroll
      for (int u = 0; u < 2; ++u) {
        bf16x2 pr[4];
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          const f32x2 pf = {fast_exp2(fmaf(s[tq][8 * u + 2 * e], sc, nmcur)),
                            fast_exp2(fmaf(s[tq][8 * u + 2 * e + 1], sc, nmcur))};
          pr[e] = __builtin_convertvector(pf, bf16x2);
          r = __builtin_amdgcn_fdot2_f32_bf16(pr[e], kOnes, r, false);
        }
        p[u][tq] = bf16x8{pr[0][0], pr[0][1], pr[1][0], pr[1][1],
                          pr[2][0], pr[2][1], pr[3][0], pr[3][1]};
      }
      rs[tq] = r;
    }
  }
  __device__ __forceinline__ void mask_keys(f32x16 (&s)[2], int valid) {
    if (valid < 32) {
#pragma unroll
      for (int e = 0; e < 16; ++e) {
        const int key = 8 * (e >> 2) + 4 * hf + (e & 3);
        if (key >= valid) {
          s[0][e] = kNegInf;
          s[1][e] = kNegInf;
        }
      }
    }
  }
  __device__ __forceinline__ void fixup(f32x16 (&s)[2], bf16x8 (&p)[2][2], float (&rs)[2]) {
    // 0x45800000 is 2^12; inf and NaN compare above it as unsigned bits
    if (__ballot(__float_as_uint(rs[0]) > 0x45800000u || __float_as_uint(rs[1]) > 0x45800000u)) {
#pragma unroll
      for (int tq = 0; tq < 2; ++tq) {
        float mx = fmaxf(fmaxf(s[tq][0], s[tq][1]), s[tq][2]);
#pragma unroll
        for (int e = 3; e < 15; e += 2) mx = fmaxf(fmaxf(mx, s[tq][e]), s[tq][e + 1]);
        mx = fmaxf(mx, s[tq][15]);
        // -max(x, m) = min(-x, -m) and (-m) - (-m') = m' - m, exactly
        const float nmnew = fminf(-(pair_max(mx) * sc), nm[tq]);
        const float alpha = fast_exp2(nmnew - nm[tq]);
        nm[tq] = nmnew;
        l[tq] *= alpha;
#pragma unroll
        for (int c = 0; c < 2; ++c) o[c][tq] *= alpha;
      }
      probs(s, p, rs);
    }
    l[0] += rs[0];
    l[1] += rs[1];
  }

  // One half-tile step t: Sᵀ of half t+1 (from kb, if kNext) and O += Vᵀ Pᵀ
  // of half t-1 (from vb) on the matrix cores while the VALU runs the softmax
  // of half t (s_cur, keys past `valid` masked); then s_cur and p_prev move
  // on by one half. Both are issued in one scheduling region: the 12 LDS
  // operand reads first (mask 0x100), ten softmax VALU ops (0x002) while they
  // land, then each of the 16 MFMAs (0x008) followed by four VALU ops, so the
  // matrix cores and the VALU work on independent data side by side.
  template <bool kNext>
  __device__ __forceinline__ void step(lds_char* kb, lds_char* vb, int valid, f32x16 (&s_cur)[2],
                       bf16x8 (&p_prev)[2][2]) {
    bf16x8 kA[4];
    bf16x8 vA[2][2];
    if constexpr (kNext) read_k(kb, kA);
    read_v(vb, vA);
    f32x16 s_next[2];
    if constexpr (kNext) mfma_s(kA, s_next);
    mfma_pv(vA, p_prev);
    bf16x8 p_new[2][2];
    mask_keys(s_cur, valid);
    float rs[2];
    probs(s_cur, p_new, rs);
    __builtin_amdgcn_sched_group_barrier(0x100, 12, 0);
    __builtin_amdgcn_sched_group_barrier(0x002, 10, 0);
#pragma unroll
    for (int g = 0; g < 16; ++g) {
      __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
      __builtin_amdgcn_sched_group_barrier(0x002, 4, 0);
    }
    fixup(s_cur, p_new, rs);
#pragma unroll
    for (int u = 0; u < 2; ++u)
#pragma unroll
      for (int tq = 0; tq < 2; ++tq) p_prev[u][tq] = p_new[u][tq];
    if constexpr (kNext) {
      s_cur[0] = s_next[0];
      s_cur[1] = s_next[1];
    }
  }
  // The last step: no half t+1; O += Vᵀ Pᵀ of half t-1, the softmax of half
  // t, then the P V of half t itself.
  __device__ __forceinline__ void last_step(lds_char* vb_prev, lds_char* vb_cur, int valid, f32x16 (&s_cur)[2],
                            const bf16x8 (&p_prev)[2][2]) {
    bf16x8 vA[2][2];
    read_v(vb_prev, vA);
    mfma_pv(vA, p_prev);
    bf16x8 p_new[2][2];
    mask_keys(s_cur, valid);
    float rs[2];
    probs(s_cur, p_new, rs);
    fixup(s_cur, p_new, rs);
    read_v(vb_cur, vA);
    mfma_pv(vA, p_new);
  }
  __device__ __forceinline__ void running_max(float (&m)[2]) const {
    m[0] = -nm[0];
    m[1] = -nm[1];
  }
  // the row sums of the two query halves (the lane pair's shares added)
  __device__ __forceinline__ void row_sums(float (&lt)[2]) const {
    lt[0] = pair_sum(l[0]);
    lt[1] = pair_sum(l[1]);
  }
};

template <int kMode>
__global__ __launch_bounds__(64) __attribute__((amdgpu_waves_per_eu(2, 2))) void attn_bf16_kernel(const uint16_t* __restrict__ q,
                                                      const uint16_t* __restrict__ k,
                                                      const uint16_t* __restrict__ v,
                                                      const int32_t* __restrict__ idx,
                                                      const int32_t* __restrict__ cnt,
                                                      uint16_t* __restrict__ out,
                                                      float* __restrict__ lse, AttnArgs a) {
  // Four LDS half tiles of 32 rows: K half 0 / 1 and V half 0 / 1 of the
  // tiles in flight. Separate objects, so the compiler sees which DMA writes
  // can alias which reads.
  __shared__ __attribute__((aligned(1024))) char k0_buf[32 * 128];
  __shared__ __attribute__((aligned(1024))) char k1_buf[32 * 128];
  __shared__ __attribute__((aligned(1024))) char v0_buf[32 * 128];
  __shared__ __attribute__((aligned(1024))) char v1_buf[32 * 128];
  lds_char* const kbuf0 = (lds_char*)k0_buf;
  lds_char* const kbuf1 = (lds_char*)k1_buf;
  lds_char* const vbuf0 = (lds_char*)v0_buf;
  lds_char* const vbuf1 = (lds_char*)v1_buf;

  const Work w = work_item(a);
  if (!w.valid) return;
  const int lane = threadIdx.x;
  const int l32 = lane & 31;
  const int hf = lane >> 5;
  const int nb = a.nb;
  const bool dense = kMode != kLists || a.dense[w.h] != 0;
  const int32_t* list = idx + ((int64_t)w.h * nb + w.i) * a.cap;
  // STRIDE heads: nkeys sampled keys in count virtual blocks of 64
  const int64_t stride = kMode == kStrided ? a.stride[w.h] : 1;
  const int64_t nkeys = kMode == kStrided ? (a.n + stride - 1) / stride : a.n;
  int count = kMode == kStrided ? (int)((nkeys + kBlock - 1) / kBlock) : nb;
  if (!dense) count = min(max(cnt[(int64_t)w.h * nb + w.i], 0), a.cap);
  int dense_lo = 0;  // first key block of a dense head's item
  if constexpr (kMode == kLists) {
    if (w.chunk >= 0) split_range(w, a, dense, list, count, dense_lo, lane);
  }

  const int64_t head_off = (int64_t)w.h * a.n * kHeadDim;
  const uint32_t head_bytes = (uint32_t)(a.n * kHeadDim * 2);
  const __amdgpu_buffer_rsrc_t rk = make_rsrc(k + head_off, head_bytes);
  const __amdgpu_buffer_rsrc_t rv = make_rsrc(v + head_off, head_bytes);
  const __amdgpu_buffer_rsrc_t ro = make_rsrc(out + head_off, head_bytes);
  const uint16_t* const kh = k + head_off;
  const uint16_t* const vh = v + head_off;
  auto load_half = [&](bool is_v, int j, int h, lds_char* buf, DmaLaneOffsets off) {
    if constexpr (kMode == kStrided)
      dma_half_strided(is_v ? rv : rk, j, h, buf, threadIdx.x, stride, a.n, head_bytes);
    else
      dma_half(is_v ? vh : kh, head_bytes, nb, j, h, buf, off);
  };

  Bf16Walk<false> wk;
  wk.init(make_rsrc(q + head_off, head_bytes), w.i, lane, a.scale_log2);

  const DmaLaneOffsets dma_off = dma_lane_offset(lane);
  // tile of list position it, clamped to the last kept tile: loads past the
  // end of the list refetch that tile into a buffer no later step reads
  auto tile_at = [&](int it) -> int {
    const int c = min(it, count - 1);
    return dense ? dense_lo + c : list[c];
  };

  if (count <= 0) {  // an empty list: no keys, zero output, LSE -inf
    if constexpr (kMode == kLists) {
      if (w.chunk >= 0) {  // an empty key range: statistics only, the merge skips it
        float m[2];
        wk.running_max(m);
        store_partials(wk.o, m, wk.l, a, w.item, true, lane);
        return;
      }
    }
#pragma unroll
    for (int tq = 0; tq < 2; ++tq) {
      const int query = w.i * kBlock + 32 * tq + l32;
#pragma unroll
      for (int c = 0; c < 2; ++c)
#pragma unroll
        for (int g = 0; g < 4; ++g)
          __builtin_amdgcn_raw_buffer_store_b64(i32x2{0, 0}, ro,
              (int)((query * kHeadDim + 32 * c + 8 * g + 4 * hf) * 2), 0, 0);
      if (lse && hf == 0 && query < a.n) lse[(int64_t)w.h * a.n + query] = kNegInf;
    }
    return;
  }

  // the last (virtual) key block may hold fewer than 64 keys
  const int last_block = kMode == kStrided ? count - 1 : nb - 1;
  const bool tail = (nkeys % kBlock) != 0;
  const int valid_last = (int)(nkeys - (int64_t)last_block * kBlock);

  // ---- pipeline
  // Half-tile steps t = 2j + h (tile j of the list, key half h). Step t
  // reads K half t+1 and V half t-1, then refills the buffers it read: K
  // half t+3 (same parity as t+1) and V half t+1 (parity of t-1). Every step
  // issues eight DMA loads, so at the start of a step the loads of the step
  // before last, which it reads, are done after vmcnt(8).
  f32x16 s_cur[2];
  bf16x8 p_prev[2][2];
#pragma unroll
  for (int u = 0; u < 2; ++u)
#pragma unroll
    for (int tq = 0; tq < 2; ++tq) p_prev[u][tq] = bf16x8{};  // P of half -1: nothing

  int j0 = tile_at(0), j1 = tile_at(1), j2 = tile_at(2);
  {
    // prologue: S^T of half 0, then the loads steps -2 and -1 would issue
    load_half(false, j0, 0, kbuf0, dma_off);
    __builtin_amdgcn_s_waitcnt(kWaitVm0);
    bf16x8 kA[4];
    wk.read_k(kbuf0, kA);
    wk.mfma_s(kA, s_cur);
    __builtin_amdgcn_s_waitcnt(kWaitLgkm0);
    load_half(false, j0, 1, kbuf1, dma_off);   // K half 1 (tile 0)
    load_half(true, j0, 1, vbuf1, dma_off);   // V of half -1: any tile (its P is 0)
    load_half(false, j1, 0, kbuf0, dma_off);   // K half 2 (tile 1)
    load_half(true, j0, 0, vbuf0, dma_off);   // V half 0 (tile 0)
  }

  // kNext: there is a half t+1; kMask: half t may be the partial last block
  auto step = [&](auto h_c, auto next_c, auto mask_c, int jcur, int jkn, int jvn) {
    constexpr int h = decltype(h_c)::value;
    constexpr bool kNext = decltype(next_c)::value;
    constexpr bool kMask = decltype(mask_c)::value;
    lds_char* const kb = h == 0 ? kbuf1 : kbuf0;  // K half t+1
    lds_char* const vb = h == 0 ? vbuf1 : vbuf0;  // V half t-1
    __builtin_amdgcn_s_waitcnt(kWaitVm8);
    int valid = 32;
    if constexpr (kMask) {
      if (tail && jcur == last_block) valid = valid_last - 32 * h;
    }
    wk.template step<kNext>(kb, vb, valid, s_cur, p_prev);
    // refill the two buffers this step read
    __builtin_amdgcn_s_waitcnt(kWaitLgkm0);
    if constexpr (kNext) {
      load_half(false, jkn, h ^ 1, kb, dma_off);
      load_half(true, jvn, h ^ 1, vb, dma_off);
    }
  };

  using F = std::false_type;
  using T = std::true_type;
  using H0 = std::integral_constant<int, 0>;
  using H1 = std::integral_constant<int, 1>;
  for (int it = 0; it + 1 < count; ++it) {
    // tiles it (j0), it+1 (j1), it+2 (j2)
    const int j3 = tile_at(it + 3);
    step(H0{}, T{}, F{}, j0, j1, j0);  // half 2it:   loads K(it+1,1), V(it,1)
    step(H1{}, T{}, F{}, j0, j2, j1);  // half 2it+1: loads K(it+2,0), V(it+1,0)
    j0 = j1;
    j1 = j2;
    j2 = j3;
  }
  // last tile: its halves may hold the partial last block
  step(H0{}, T{}, T{}, j0, j1, j0);
  __builtin_amdgcn_s_waitcnt(kWaitVm0);
  wk.last_step(vbuf0, vbuf1, tail && j0 == last_block ? valid_last - 32 : 32, s_cur, p_prev);

  float lt[2], m[2];
  wk.row_sums(lt);
  wk.running_max(m);
  if constexpr (kMode == kLists) {
    if (w.chunk >= 0) {  // a split item: the merge combines the ranges
      store_partials(wk.o, m, lt, a, w.item, false, lane);
      return;
    }
  }
  const float inv[2] = {1.0f / lt[0], 1.0f / lt[1]};
  const float lse_val[2] = {(m[0] + __log2f(lt[0])) * kLn2, (m[1] + __log2f(lt[1])) * kLn2};
  write_out_tile(wk.o, inv, lse_val, kbuf0, kbuf1, ro, lse ? lse + (int64_t)w.h * a.n : nullptr, w.i,
                 a.n, lane);
}

// ---- every head dense: kDenseWaves waves per workgroup sharing the K / V tiles
//
// A workgroup takes kDenseWaves neighbouring query blocks of one head, and
// since every one of them walks every key block in order, each K and V half
// tile is staged in LDS once for all of them. Wave w owns query block
// kDenseWaves * group + w; a block past the head's last one runs the last
// block again and stores nothing, so every wave meets every barrier. The K and
// V half tiles go into a ring of four LDS buffers per tensor (K half x in
// kring[x % 4], V half x in vring[x % 4]). Step t reads K half t+1 and V half
// t-1; right after the step's barrier the waves refill the buffers step t-1
// read (K half t+4, V half t+2), each wave issuing its share of the eight 1 KB
// DMA instructions, three steps before those buffers are read. Before the
// barrier each wave waits for its own loads of three steps back, so after it
// every wave's loads for the step have landed, and every wave has finished
// the reads of step t-1.
constexpr int kDenseWaves = 4;

// Group g (rows 8g .. 8g+7) of the 32-row half h of block j into buf: one 1 KB
// DMA instruction. The descriptor starts at the group and extends over what
// is left of the head, so rows past the head, and any j outside [0, nb),
// read zeros.
__device__ inline void dma_group(const uint16_t* head, uint32_t head_bytes, int nb, int j, int h,
                                 int g, lds_char* buf, int lane_off) {
  const uint32_t t = __builtin_amdgcn_readfirstlane(
      (uint32_t)j < (uint32_t)nb ? ((uint32_t)j * kBlock + 32u * h + 8u * g) * (kHeadDim * 2)
                                 : head_bytes);
  const uint32_t rem = rem_bytes(head_bytes, t);
  const __amdgpu_buffer_rsrc_t r = make_rsrc(reinterpret_cast<const char*>(head) + t, rem);
  __builtin_amdgcn_raw_ptr_buffer_load_lds(r, (lds_void*)(buf + 1024 * g), 16, lane_off, 0, 0, 0);
}

__global__ __launch_bounds__(64 * kDenseWaves) __attribute__((amdgpu_waves_per_eu(2, 2))) void attn_bf16_dense_kernel(
    const uint16_t* __restrict__ q, const uint16_t* __restrict__ k, const uint16_t* __restrict__ v,
    uint16_t* __restrict__ out, float* __restrict__ lse, AttnArgs a) {
  __shared__ __attribute__((aligned(1024))) char kr0[32 * 128];
  __shared__ __attribute__((aligned(1024))) char kr1[32 * 128];
  __shared__ __attribute__((aligned(1024))) char kr2[32 * 128];
  __shared__ __attribute__((aligned(1024))) char kr3[32 * 128];
  __shared__ __attribute__((aligned(1024))) char vr0[32 * 128];
  __shared__ __attribute__((aligned(1024))) char vr1[32 * 128];
  __shared__ __attribute__((aligned(1024))) char vr2[32 * 128];
  __shared__ __attribute__((aligned(1024))) char vr3[32 * 128];
  lds_char* const kring[4] = {(lds_char*)kr0, (lds_char*)kr1, (lds_char*)kr2, (lds_char*)kr3};
  lds_char* const vring[4] = {(lds_char*)vr0, (lds_char*)vr1, (lds_char*)vr2, (lds_char*)vr3};
  constexpr int kW = kDenseWaves;

  // workgroup b runs on XCD b % 8; each XCD takes a contiguous run of the
  // (head, group) units, so the workgroups it runs at once walk one head
  const int nb = a.nb;
  const int groups = (nb + kW - 1) / kW;
  const int total = a.heads * groups;
  const int per_xcd = (total + 7) / 8;
  const int unit = (blockIdx.x & 7) * per_xcd + (blockIdx.x >> 3);
  if (unit >= total) return;  // the whole workgroup
  const int hpos = unit / groups;
  const int hidx = a.order[hpos];
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int lane = threadIdx.x & 63;
  const int l32 = lane & 31;
  const int hf = lane >> 5;
  const int i_own = (unit - hpos * groups) * kW + wave;
  const bool valid_block = i_own < nb;

  const int64_t head_off = (int64_t)hidx * a.n * kHeadDim;
  const uint32_t head_bytes = (uint32_t)(a.n * kHeadDim * 2);
  const uint16_t* const kh = k + head_off;
  const uint16_t* const vh = v + head_off;

  Bf16Walk<true> wk;
  wk.init(make_rsrc(q + head_off, head_bytes), valid_block ? i_own : nb - 1, lane, a.scale_log2);

  // this wave's share of a step's eight DMA instructions n = wave, wave + kW,
  // ... (n < 4: K group n, else V group n - 4); its group is wave % 4 either way
  const DmaLaneOffsets dma_off = dma_lane_offset(lane);
  const int dma_g = wave & 3;
  const int dma_lane = (dma_g & 1) ? dma_off.odd : dma_off.even;
  auto issue = [&](int jk, int hk, lds_char* kb, int jv, int hv, lds_char* vb) {
#pragma unroll
    for (int n0 = 0; n0 < 8; n0 += kW) {
      if (n0 + wave < 4) dma_group(kh, head_bytes, nb, jk, hk, dma_g, kb, dma_lane);
      else dma_group(vh, head_bytes, nb, jv, hv, dma_g, vb, dma_lane);
    }
  };
  // this wave's loads up to `pending` instructions back have landed and its
  // LDS reads are done; then the workgroup meets (the asm's memory clobber
  // keeps LDS accesses on their side of the barrier)
  auto sync = [&](auto pending_c) {
    constexpr int pending = decltype(pending_c)::value;
    __builtin_amdgcn_s_waitcnt((0x0F70 | pending) & kWaitLgkm0);
    asm volatile("s_barrier" ::: "memory");
  };
  constexpr int kPending = 2 * (8 / kW);  // two steps of this wave's loads

  const bool tail = (a.n % kBlock) != 0;
  const int valid_last = (int)(a.n - (int64_t)(nb - 1) * kBlock);

  f32x16 s_cur[2];
  bf16x8 p_prev[2][2];
#pragma unroll
  for (int u = 0; u < 2; ++u)
#pragma unroll
    for (int tq = 0; tq < 2; ++tq) p_prev[u][tq] = bf16x8{};  // P of half -1: nothing

  // prologue: K halves 0-3 into kring[0..3]; V half -1 (any data, its P is 0:
  // V half 1) into vring[3], V halves 0 and 1 into vring[0] and vring[1]
  issue(0, 0, kring[0], 0, 1, vring[3]);
  issue(0, 1, kring[1], 0, 0, vring[0]);
  issue(1, 0, kring[2], 0, 1, vring[1]);
  issue(1, 1, kring[3], 0, 1, vring[1]);
  sync(std::integral_constant<int, 0>{});
  {
    bf16x8 kA[4];
    wk.read_k(kring[0], kA);
    wk.mfma_s(kA, s_cur);
  }

  // step t = 2j + h with P = t % 4 (the ring slots are then fixed)
  auto step = [&](auto p_c, auto mask_c, int j) {
    constexpr int P = decltype(p_c)::value;
    constexpr int h = P & 1;
    constexpr bool kMask = decltype(mask_c)::value;
    sync(std::integral_constant<int, kPending>{});
    // refill what step t-1 read: K half t+4 (block j+2, half h), V half t+2 (block j+1, half h)
    issue(j + 2, h, kring[P], j + 1, h, vring[(P + 2) & 3]);
    const int valid = kMask && tail ? valid_last - 32 * h : 32;
    wk.template step<true>(kring[(P + 1) & 3], vring[(P + 3) & 3], valid, s_cur, p_prev);
  };
  // the last step t = 2nb - 1, P = t % 4
  auto last = [&](auto p_c) {
    constexpr int P = decltype(p_c)::value;
    sync(std::integral_constant<int, 0>{});
    wk.last_step(vring[(P + 3) & 3], vring[P], tail ? valid_last - 32 : 32, s_cur, p_prev);
  };

  using F = std::false_type;
  using T = std::true_type;
  using P0 = std::integral_constant<int, 0>;
  using P1 = std::integral_constant<int, 1>;
  using P2 = std::integral_constant<int, 2>;
  using P3 = std::integral_constant<int, 3>;
  int it = 0;  // tiles it and it + 1 per iteration, it even
  for (; it + 2 < nb; it += 2) {
    step(P0{}, F{}, it);
    step(P1{}, F{}, it);
    step(P2{}, F{}, it + 1);
    step(P3{}, F{}, it + 1);
  }
  if (nb - it == 2) {
    step(P0{}, F{}, it);
    step(P1{}, F{}, it);
    step(P2{}, T{}, it + 1);
    last(P3{});
  } else {
    step(P0{}, T{}, it);
    last(P1{});
  }

  if (!valid_block) return;
  float lt[2];
  wk.row_sums(lt);
  const __amdgpu_buffer_rsrc_t ro = make_rsrc(out + head_off, head_bytes);
  float* const lse_row = lse ? lse + (int64_t)hidx * a.n : nullptr;
  // straight from the registers: 8-byte stores, once per walk of nb blocks
#pragma unroll
  for (int tq = 0; tq < 2; ++tq) {
    const int query = i_own * kBlock + 32 * tq + l32;
    const float inv = 1.0f / lt[tq];
#pragma unroll
    for (int c = 0; c < 2; ++c)
#pragma unroll
      for (int g = 0; g < 4; ++g) {
        bf16x4 ov;
#pragma unroll
        for (int r = 0; r < 4; ++r) ov[r] = (__bf16)(wk.o[c][tq][4 * g + r] * inv);
        __builtin_amdgcn_raw_buffer_store_b64(__builtin_bit_cast(i32x2, ov), ro,
                                              (int)((query * kHeadDim + 32 * c + 8 * g + 4 * hf) * 2), 0, 0);
      }
    if (lse_row && hf == 0 && query < a.n) lse_row[query] = (__log2f(lt[tq]) - wk.nm[tq]) * kLn2;
  }
}

// Combines the key ranges of split heads: per query, M = max of the ranges'
// running maxima, weights 2^(m_c - M), O = sum_c w_c O_c / sum_c w_c l_c, in
// range order; rows written in the layer's dtype. One wave per (split head,
// query block).
template <bool kBf16>
__global__ __launch_bounds__(64) void attn_merge_kernel(const float* __restrict__ part_o,
                                                       const float* __restrict__ part_ml,
                                                       void* __restrict__ out,
                                                       float* __restrict__ lse, MergeArgs a) {
  __shared__ __attribute__((aligned(1024))) char b0[32 * 128];
  __shared__ __attribute__((aligned(1024))) char b1[32 * 128];
  const int sp = blockIdx.x / a.nb;
  const int i = blockIdx.x - sp * a.nb;
  if (sp >= a.n_split) return;
  const int h = a.head[sp];
  const int lane = threadIdx.x;
  const int l32 = lane & 31;
  auto ml_at = [&](int c, int tq) -> f32x2 {
    const int64_t item = (int64_t)(sp * a.splits + c) * a.nb + i;
    return *(const f32x2*)(part_ml + (item * kBlock + 32 * tq + l32) * 2);
  };
  float mx[2] = {kNegInf, kNegInf};
  for (int c = 0; c < a.splits; ++c)
#pragma unroll
    for (int tq = 0; tq < 2; ++tq) mx[tq] = fmaxf(mx[tq], ml_at(c, tq)[0]);
  float lt[2] = {0.f, 0.f};
  f32x16 o[2][2];
#pragma unroll
  for (int c = 0; c < 2; ++c)
#pragma unroll
    for (int tq = 0; tq < 2; ++tq)
#pragma unroll
      for (int e = 0; e < 16; ++e) o[c][tq][e] = 0.f;
  for (int c = 0; c < a.splits; ++c) {
    float wgt[2];
#pragma unroll
    for (int tq = 0; tq < 2; ++tq) {
      const f32x2 ml = ml_at(c, tq);
      wgt[tq] = ml[0] == kNegInf ? 0.f : fast_exp2(ml[0] - mx[tq]);
      lt[tq] = fmaf(wgt[tq], ml[1], lt[tq]);
    }
    // an empty range (every query's max is -inf) wrote no accumulators
    if (!__ballot(wgt[0] != 0.f || wgt[1] != 0.f)) continue;
    const float* const po = part_o + ((int64_t)(sp * a.splits + c) * a.nb + i) * (kBlock * kHeadDim);
#pragma unroll
    for (int c2 = 0; c2 < 2; ++c2)
#pragma unroll
      for (int tq = 0; tq < 2; ++tq)
#pragma unroll
        for (int g = 0; g < 4; ++g) {
          const f32x4 val = *(const f32x4*)(po + (((c2 * 2 + tq) * 4 + g) * 64 + lane) * 4);
#pragma unroll
          for (int r = 0; r < 4; ++r) o[c2][tq][4 * g + r] = fmaf(wgt[tq], val[r], o[c2][tq][4 * g + r]);
        }
  }
  float inv[2], lse_val[2];
#pragma unroll
  for (int tq = 0; tq < 2; ++tq) {
    inv[tq] = lt[tq] > 0.f ? 1.0f / lt[tq] : 0.f;
    lse_val[tq] = lt[tq] > 0.f ? (mx[tq] + __log2f(lt[tq])) * kLn2 : kNegInf;
  }
  const int64_t head_off = (int64_t)h * a.n * kHeadDim;
  float* const lse_row = lse ? lse + (int64_t)h * a.n : nullptr;
  if constexpr (kBf16) {
    const __amdgpu_buffer_rsrc_t ro =
        make_rsrc(static_cast<uint16_t*>(out) + head_off, (uint32_t)(a.n * kHeadDim * 2));
    write_out_tile(o, inv, lse_val, (lds_char*)b0, (lds_char*)b1, ro, lse_row, i, a.n, lane);
  } else {
    const __amdgpu_buffer_rsrc_t ro =
        make_rsrc(static_cast<float*>(out) + head_off, (uint32_t)(a.n * kHeadDim * 4));
    write_out_tile_f32(o, inv, lse_val, ro, lse_row, i, a.n, lane);
  }
}

// ------------------------------------------------------------------ fp32

// Same structure with v_mfma_f32_32x32x2_f32 and fp32 softmax operands; K and
// V tiles both go through LDS (one wave, no barrier).
template <int kMode>
__global__ __launch_bounds__(64) void attn_f32_kernel(const float* __restrict__ q,
                                                     const float* __restrict__ k,
                                                     const float* __restrict__ v,
                                                     const int32_t* __restrict__ idx,
                                                     const int32_t* __restrict__ cnt,
                                                     float* __restrict__ out,
                                                     float* __restrict__ lse, AttnArgs a) {
  __shared__ float ks[kBlock * kFStride];
  __shared__ float vsf[kBlock * kFStride];

  const Work w = work_item(a);
  if (!w.valid) return;
  const int lane = threadIdx.x;
  const int l32 = lane & 31;
  const int hf = lane >> 5;
  const int nb = a.nb;
  const bool dense = kMode != kLists || a.dense[w.h] != 0;
  const int32_t* list = idx + ((int64_t)w.h * nb + w.i) * a.cap;
  const int64_t stride = kMode == kStrided ? a.stride[w.h] : 1;
  const int64_t nkeys = kMode == kStrided ? (a.n + stride - 1) / stride : a.n;
  int count = kMode == kStrided ? (int)((nkeys + kBlock - 1) / kBlock) : nb;
  if (!dense) count = min(max(cnt[(int64_t)w.h * nb + w.i], 0), a.cap);
  int dense_lo = 0;  // first key block of a dense head's item
  if constexpr (kMode == kLists) {
    if (w.chunk >= 0) split_range(w, a, dense, list, count, dense_lo, lane);
  }
  const int last_block = kMode == kStrided ? count - 1 : nb - 1;

  const int64_t head_off = (int64_t)w.h * a.n * kHeadDim;
  const uint32_t head_bytes = (uint32_t)(a.n * kHeadDim * 4);
  const __amdgpu_buffer_rsrc_t rq = make_rsrc(q + head_off, head_bytes);
  const __amdgpu_buffer_rsrc_t rk = make_rsrc(k + head_off, head_bytes);
  const __amdgpu_buffer_rsrc_t rv = make_rsrc(v + head_off, head_bytes);
  const __amdgpu_buffer_rsrc_t ro = make_rsrc(out + head_off, head_bytes);

  // Q^T B operand: qB[tq][s] = Q[64i + 32tq + l32][2s + hf]
  float qB[2][32];
#pragma unroll
  for (int tq = 0; tq < 2; ++tq)
#pragma unroll
    for (int s4 = 0; s4 < 8; ++s4) {
      // dims 8*s4 .. 8*s4+7 of this query: the lane half picks odd or even
      const int row = w.i * kBlock + 32 * tq + l32;
      const f32x4 x0 = __builtin_bit_cast(
          f32x4, __builtin_amdgcn_raw_buffer_load_b128(rq, (row * kHeadDim + 8 * s4) * 4, 0, 0));
      const f32x4 x1 = __builtin_bit_cast(
          f32x4, __builtin_amdgcn_raw_buffer_load_b128(rq, (row * kHeadDim + 8 * s4 + 4) * 4, 0, 0));
      qB[tq][4 * s4 + 0] = hf ? x0[1] : x0[0];
      qB[tq][4 * s4 + 1] = hf ? x0[3] : x0[2];
      qB[tq][4 * s4 + 2] = hf ? x1[1] : x1[0];
      qB[tq][4 * s4 + 3] = hf ? x1[3] : x1[2];
    }

  f32x16 o[2][2];
#pragma unroll
  for (int c = 0; c < 2; ++c)
#pragma unroll
    for (int tq = 0; tq < 2; ++tq)
#pragma unroll
      for (int e = 0; e < 16; ++e) o[c][tq][e] = 0.f;
  float m[2] = {kNegInf, kNegInf};
  float l[2] = {0.f, 0.f};
  const bool tail = (nkeys % kBlock) != 0;
  const float sc = a.scale_log2;

  for (int it = 0; it < count; ++it) {
    const int j = dense ? dense_lo + it : list[it];
    // stage K and V tiles: rows 4n + lane/16, float4 chunk lane%16 (a STRIDE
    // head's row r of virtual block j is token (64j + r) * stride; tokens at
    // or past n read as zeros through an offset past the buffer's extent)
#pragma unroll
    for (int n4 = 0; n4 < 16; ++n4) {
      const int row = 4 * n4 + (lane >> 4);
      const int64_t tok = ((int64_t)j * kBlock + row) * stride;
      const int off = kMode == kStrided && tok >= a.n
                          ? (int)head_bytes
                          : (int)((tok * kHeadDim + (lane & 15) * 4) * 4);
      const f32x4 kx = __builtin_bit_cast(f32x4, __builtin_amdgcn_raw_buffer_load_b128(rk, off, 0, 0));
      const f32x4 vx = __builtin_bit_cast(f32x4, __builtin_amdgcn_raw_buffer_load_b128(rv, off, 0, 0));
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        ks[row * kFStride + (lane & 15) * 4 + e] = kx[e];
        vsf[row * kFStride + (lane & 15) * 4 + e] = vx[e];
      }
    }

    f32x16 s[2][2];
#pragma unroll
    for (int tk = 0; tk < 2; ++tk)
#pragma unroll
      for (int tq = 0; tq < 2; ++tq) {
        f32x16 acc = {};
#pragma unroll
        for (int st = 0; st < 32; ++st)
          acc = __builtin_amdgcn_mfma_f32_32x32x2f32(ks[(32 * tk + l32) * kFStride + 2 * st + hf],
                                                     qB[tq][st], acc, 0, 0, 0);
        s[tk][tq] = acc;
      }

    if (tail && j == last_block) {
      const int valid_keys = (int)(nkeys - (int64_t)j * kBlock);
#pragma unroll
      for (int tk = 0; tk < 2; ++tk)
#pragma unroll
        for (int e = 0; e < 16; ++e) {
          const int key = 32 * tk + 8 * (e >> 2) + 4 * hf + (e & 3);
          if (key >= valid_keys) {
            s[tk][0][e] = kNegInf;
            s[tk][1][e] = kNegInf;
          }
        }
    }

#pragma unroll
    for (int tq = 0; tq < 2; ++tq) {
      float mx = s[0][tq][0];
#pragma unroll
      for (int e = 1; e < 16; ++e) mx = fmaxf(mx, s[0][tq][e]);
#pragma unroll
      for (int e = 0; e < 16; ++e) mx = fmaxf(mx, s[1][tq][e]);
      mx = fmaxf(mx, __shfl_xor(mx, 32));
      const float mnew = fmaxf(m[tq], mx * sc);
      const float alpha = exp2f(m[tq] - mnew);
      m[tq] = mnew;
      float rs = 0.f;
#pragma unroll
      for (int tk = 0; tk < 2; ++tk)
#pragma unroll
        for (int e = 0; e < 16; ++e) {
          const float p = exp2f(fmaf(s[tk][tq][e], sc, -mnew));
          s[tk][tq][e] = p;
          rs += p;
        }
      l[tq] = fmaf(l[tq], alpha, rs);
#pragma unroll
      for (int c = 0; c < 2; ++c) o[c][tq] *= alpha;
    }

    // O^T[c][tq] += V^T P^T; k-step (tk, g, r) pairs key 32tk+8g+r (lane half
    // 0) with key 32tk+8g+4+r (lane half 1), i.e. S^T register 4g+r.
#pragma unroll
    for (int c = 0; c < 2; ++c)
#pragma unroll
      for (int tk = 0; tk < 2; ++tk)
#pragma unroll
        for (int e = 0; e < 16; ++e) {
          const int key = 32 * tk + 8 * (e >> 2) + 4 * hf + (e & 3);
          const float va = vsf[key * kFStride + 32 * c + l32];
#pragma unroll
          for (int tq = 0; tq < 2; ++tq)
            o[c][tq] = __builtin_amdgcn_mfma_f32_32x32x2f32(va, s[tk][tq][e], o[c][tq], 0, 0, 0);
        }
  }

  float lt[2];
#pragma unroll
  for (int tq = 0; tq < 2; ++tq) lt[tq] = l[tq] + __shfl_xor(l[tq], 32);
  if constexpr (kMode == kLists) {
    if (w.chunk >= 0) {  // a split item: the merge combines the ranges
      store_partials(o, m, lt, a, w.item, count <= 0, lane);
      return;
    }
  }
  // an empty list (no keys) gives a zero output and LSE -inf
  float inv[2], lse_val[2];
#pragma unroll
  for (int tq = 0; tq < 2; ++tq) {
    inv[tq] = lt[tq] > 0.f ? 1.0f / lt[tq] : 0.f;
    lse_val[tq] = lt[tq] > 0.f ? (m[tq] + log2f(lt[tq])) * kLn2 : kNegInf;
  }
  write_out_tile_f32(o, inv, lse_val, ro, lse ? lse + (int64_t)w.h * a.n : nullptr, w.i, a.n, lane);
}

}  // namespace

hipError_t launch_attention(int dtype, const void* q, const void* k, const void* v,
                            const int32_t* idx, const int32_t* cnt, void* out, float* lse,
                            const AttnArgs& a, hipStream_t s) {
  const int64_t groups = 8LL * a.unit_start[a.heads];
  if (groups == 0) return hipSuccess;
  const dim3 grid((unsigned)groups);
  if (dtype == 1) {
    if (a.mode == kAllDense) {
      const int64_t units = (int64_t)a.heads * ((a.nb + kDenseWaves - 1) / kDenseWaves);
      hipLaunchKernelGGL(attn_bf16_dense_kernel, dim3((unsigned)(8 * ((units + 7) / 8))),
                         dim3(64 * kDenseWaves), 0, s, static_cast<const uint16_t*>(q),
                         static_cast<const uint16_t*>(k), static_cast<const uint16_t*>(v),
                         static_cast<uint16_t*>(out), lse, a);
      return hipGetLastError();
    }
    auto kern = a.mode == kStrided ? attn_bf16_kernel<kStrided> : attn_bf16_kernel<kLists>;
    hipLaunchKernelGGL(kern, grid, dim3(64), 0, s, static_cast<const uint16_t*>(q),
                       static_cast<const uint16_t*>(k), static_cast<const uint16_t*>(v), idx, cnt,
                       static_cast<uint16_t*>(out), lse, a);
  } else {
    auto kern = a.mode == kStrided ? attn_f32_kernel<kStrided> : attn_f32_kernel<kLists>;
    hipLaunchKernelGGL(kern, grid, dim3(64), 0, s, static_cast<const float*>(q),
                       static_cast<const float*>(k), static_cast<const float*>(v), idx, cnt,
                       static_cast<float*>(out), lse, a);
  }
  return hipGetLastError();
}

hipError_t launch_attention_merge(const float* part_o, const float* part_ml, void* out,
                                  float* lse, const MergeArgs& a, hipStream_t s) {
  const int64_t groups = (int64_t)a.n_split * a.nb;
  if (groups == 0) return hipSuccess;
  if (a.dtype == 1)
    hipLaunchKernelGGL(attn_merge_kernel<true>, dim3((unsigned)groups), dim3(64), 0, s, part_o,
                       part_ml, out, lse, a);
  else
    hipLaunchKernelGGL(attn_merge_kernel<false>, dim3((unsigned)groups), dim3(64), 0, s, part_o,
                       part_ml, out, lse, a);
  return hipGetLastError();
}

}  // namespace saf3r
