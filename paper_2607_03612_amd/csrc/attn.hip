// Block-sparse attention over the kept key blocks (Sec. 4.1: the Top-K and
// static kernels compute only the scores between the queries and the
// selected keys, and the softmax is renormalised over that set), with the
// dense ("Full") case as the same loop over every key block.
//
// One wave owns one (head, 64-query block) and walks its kept-block list with
// an online softmax:
//   S^T = K Q^T      (keys x queries) on MFMA, so a lane owns one query
//                    column and the row max / row sum stay inside the lane
//                    pair (lane, lane ^ 32);
//   O^T += V^T P^T   (head dim x queries) on MFMA, P^T taken straight from
//                    the S^T accumulators, V^T read from LDS with the gfx950
//                    transposing LDS read so V is never transposed in memory.
// Q sits in registers for the whole loop, K tiles are loaded straight into
// the MFMA operand layout (prefetched one tile ahead), V goes through a
// per-wave LDS tile. All global accesses use buffer instructions bounded by
// the head's extent, so a partial last block reads zeros and a corrupt index
// list cannot touch memory outside the head.
//
// Launch order: workgroup b runs on XCD b % 8; each XCD takes a contiguous
// slab of query blocks of every head (neighbouring query blocks share kept
// key blocks, which then hit in that XCD's L2), heads in decreasing cost.
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
  bool valid;
};

__device__ inline Work work_item(const AttnArgs& a) {
  const int xcd = blockIdx.x & 7;
  const int u = blockIdx.x >> 3;
  const int hh = u / a.slab;
  const int i = xcd * a.slab + (u - hh * a.slab);
  Work w;
  w.valid = hh < a.heads && i < a.nb;
  w.h = w.valid ? a.order[hh] : 0;
  w.i = i;
  return w;
}

// ------------------------------------------------------------------ bf16

typedef __attribute__((address_space(3))) void lds_void;
typedef __attribute__((address_space(3))) char lds_char;
typedef __attribute__((address_space(3))) const bf16x8 lds_bf16x8;

// LDS tiles: 64 rows x 128 B; 16-byte chunk c of row r is stored at slot
// c ^ f(r), f(r) = (bit2(r), bit1(r), bit0(r) ^ bit1(r) ^ bit3(r)). With it
// the MFMA operand reads (16 rows at one chunk) and the transposing reads
// (4 rows x 2 chunks per 16 lanes, 4 x 4 per 32) touch every bank once,
// whether the LDS serves 128 or 256 bytes per clock.
__device__ inline int swz_f(int r) {
  return ((r >> 2) & 1) | (r & 2) | (((r ^ (r >> 1) ^ (r >> 3)) & 1) << 2);
}
__device__ inline int swz(int r, int c) { return r * 128 + ((c ^ swz_f(r)) << 4); }

// One 64x64 bf16 tile (rows 64j.. of the head) into LDS with the direct
// buffer-to-LDS load: instruction n fills LDS bytes [1024n, 1024n + 1024),
// lane l its 16 bytes at 16l, i.e. row 8n + l/8, slot l%8, which must hold
// chunk (l%8) ^ f(8n + l/8) = (l%8) ^ f(l/8) ^ (4 if n is odd). Rows past
// the head read as zeros. The lane's byte offset inside its 8-row group
// depends only on the parity of n; the tile and group offsets are
// wave-uniform and go in the scalar offset.
struct DmaLaneOffsets {
  int even, odd;
};
__device__ inline DmaLaneOffsets dma_lane_offset(int lane) {
  const int r = lane >> 3;
  const int c = (lane & 7) ^ swz_f(r);
  return {(r * kHeadDim + c * 8) * 2, (r * kHeadDim + (c ^ 4) * 8) * 2};
}
__device__ inline void dma_tile(__amdgpu_buffer_rsrc_t r, int j, lds_char* tile,
                                DmaLaneOffsets off) {
  const int base = __builtin_amdgcn_readfirstlane(j * kBlock * kHeadDim * 2);  // j is wave-uniform
#pragma unroll
  for (int n = 0; n < 8; ++n)
    __builtin_amdgcn_raw_ptr_buffer_load_lds(r, (lds_void*)(tile + 1024 * n), 16,
                                             (n & 1) ? off.odd : off.even,
                                             base + n * 8 * kHeadDim * 2, 0, 0);
}

// Waits on the direct-to-LDS loads. Vector memory loads complete in issue
// order, and each tile is eight loads, so "all but the last eight" means "all
// but the tile issued last".
__device__ inline void wait_all_but_last_tile() { asm volatile("s_waitcnt vmcnt(8)" ::: "memory"); }
__device__ inline void wait_all_loads() { asm volatile("s_waitcnt vmcnt(0)" ::: "memory"); }
__device__ inline void wait_lds() { asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory"); }
__device__ inline void compiler_fence() { asm volatile("" ::: "memory"); }

// max / sum of a value over the lane pair (l, l ^ 32) that shares a query
__device__ inline float pair_max(float x) {
  const auto s = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  return fmaxf(__uint_as_float(s[0]), __uint_as_float(s[1]));
}
__device__ inline float pair_sum(float x) {
  const auto s = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  return __uint_as_float(s[0]) + __uint_as_float(s[1]);
}

// The running max is only raised when a tile's max exceeds it by more than
// this (log2 units): P stays <= 2^8 and O is rescaled rarely.
constexpr float kRescaleSlack = 8.0f;
constexpr bf16x2 kOnes = {(__bf16)1.0f, (__bf16)1.0f};

template <bool kAllDense>
__global__ __launch_bounds__(64) __attribute__((amdgpu_waves_per_eu(2, 2))) void attn_bf16_kernel(const uint16_t* __restrict__ q,
                                                      const uint16_t* __restrict__ k,
                                                      const uint16_t* __restrict__ v,
                                                      const int32_t* __restrict__ idx,
                                                      const int32_t* __restrict__ cnt,
                                                      uint16_t* __restrict__ out,
                                                      float* __restrict__ lse, AttnArgs a) {
  // LDS pointers stay in address space 3 (no generic-pointer casts). K and V
  // are separate objects, so the compiler can see that refilling one tile
  // does not alias reads of the other.
  __shared__ __attribute__((aligned(1024))) char k_tile[64 * 128];
  __shared__ __attribute__((aligned(1024))) char v_tile[64 * 128];
  lds_char* const ks = (lds_char*)k_tile;
  lds_char* const vs = (lds_char*)v_tile;

  const Work w = work_item(a);
  if (!w.valid) return;
  const int lane = threadIdx.x;
  const int l32 = lane & 31;
  const int hf = lane >> 5;
  const int nb = a.nb;
  const bool dense = kAllDense || a.dense[w.h] != 0;
  const int32_t* list = idx + ((int64_t)w.h * nb + w.i) * a.cap;
  int count = nb;
  if (!dense) count = min(max(cnt[(int64_t)w.h * nb + w.i], 0), a.cap);

  const int64_t head_off = (int64_t)w.h * a.n * kHeadDim;
  const uint32_t head_bytes = (uint32_t)(a.n * kHeadDim * 2);
  const __amdgpu_buffer_rsrc_t rq = make_rsrc(q + head_off, head_bytes);
  const __amdgpu_buffer_rsrc_t rk = make_rsrc(k + head_off, head_bytes);
  const __amdgpu_buffer_rsrc_t rv = make_rsrc(v + head_off, head_bytes);
  const __amdgpu_buffer_rsrc_t ro = make_rsrc(out + head_off, head_bytes);

  // Q^T as the B operand: qB[tq][s] = Q[64i + 32tq + l32][16s + 8hf + (0..7)]
  bf16x8 qB[2][4];
#pragma unroll
  for (int tq = 0; tq < 2; ++tq)
#pragma unroll
    for (int s = 0; s < 4; ++s)
      qB[tq][s] = load_b128(
          rq, (uint32_t)(((w.i * kBlock + 32 * tq + l32) * kHeadDim + 16 * s + 8 * hf) * 2));

  // load order from here on: K tile, V tile, next K tile, next V tile, ...
  compiler_fence();
  const DmaLaneOffsets dma_off = dma_lane_offset(lane);
  int j = count > 0 ? (dense ? 0 : list[0]) : 0;
  dma_tile(rk, j, ks, dma_off);
  dma_tile(rv, j, vs, dma_off);

  f32x16 o[2][2];  // O^T tiles [head-dim half c][query half tq]
#pragma unroll
  for (int c = 0; c < 2; ++c)
#pragma unroll
    for (int tq = 0; tq < 2; ++tq)
#pragma unroll
      for (int e = 0; e < 16; ++e) o[c][tq][e] = 0.f;
  float m[2] = {kNegInf, kNegInf};  // running max of the log2-scaled scores
  float l[2] = {0.f, 0.f};          // this lane's share of the running row sum

  const bool tail = (a.n % kBlock) != 0;
  const float sc = a.scale_log2;
  // transposing-read position of this lane inside a 4-row x 16-column group
  const int tr_row = 4 * hf + ((lane & 15) >> 2);
  const int tr_col = 16 * ((lane >> 4) & 1) + 4 * (lane & 3);

  // One step of the online softmax over kept tile `it`. Only the last step
  // can meet the partial last key block (lists are ascending), so only the
  // peeled last step carries the key mask.
  auto step = [&](int it, auto last) {
    constexpr bool kLast = decltype(last)::value;
    const int jcur = j;
    constexpr bool more = !kLast;
    if constexpr (more) j = dense ? it + 1 : list[it + 1];
    wait_all_but_last_tile();  // the K tile of jcur is in LDS (its V tile may be in flight)

    // S^T[tk][tq] = K Q^T (keys 32tk.., queries 32tq..); K rows as A operand
    f32x16 s[2][2];
#pragma unroll
    for (int tk = 0; tk < 2; ++tk) {
      bf16x8 kA[4];
#pragma unroll
      for (int st = 0; st < 4; ++st)
        kA[st] = *(lds_bf16x8*)(ks + swz(32 * tk + l32, 2 * st + hf));
#pragma unroll
      for (int tq = 0; tq < 2; ++tq) {
        f32x16 acc = {};
#pragma unroll
        for (int st = 0; st < 4; ++st)
          acc = __builtin_amdgcn_mfma_f32_32x32x16_bf16(kA[st], qB[tq][st], acc, 0, 0, 0);
        s[tk][tq] = acc;
      }
    }
    // the K operands are in registers: refill the K tile for the next step
    if constexpr (more) {
      wait_lds();
      dma_tile(rk, j, ks, dma_off);
    }

    if constexpr (kLast) {
      if (tail && jcur == nb - 1) {
        const int valid_keys = (int)(a.n - (int64_t)jcur * kBlock);
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
    }

    // online softmax per query column (lanes l and l ^ 32 share it). P is
    // rounded to bf16 here, and the row sum adds the rounded values (one
    // bf16 dot with (1, 1) per pair), so the normaliser matches the weights
    // the P V product actually uses.
    bf16x8 pB[2][2][2];  // [tk][u][tq]: keys 32tk + 16u.. as the B operand
#pragma unroll
    for (int tq = 0; tq < 2; ++tq) {
      float mx = fmaxf(fmaxf(s[0][tq][0], s[0][tq][1]), s[0][tq][2]);
#pragma unroll
      for (int e = 3; e < 15; e += 2) mx = fmaxf(fmaxf(mx, s[0][tq][e]), s[0][tq][e + 1]);
      mx = fmaxf(fmaxf(mx, s[0][tq][15]), s[1][tq][0]);
#pragma unroll
      for (int e = 1; e < 15; e += 2) mx = fmaxf(fmaxf(mx, s[1][tq][e]), s[1][tq][e + 1]);
      mx = fmaxf(mx, s[1][tq][15]);
      const float tile_max = pair_max(mx) * sc;
      const float mnew = tile_max > m[tq] + kRescaleSlack ? tile_max : m[tq];
      if (__ballot(mnew != m[tq])) {  // wave-uniform: rescale only when some max moved
        const float alpha = fast_exp2(m[tq] - mnew);
        m[tq] = mnew;
        l[tq] *= alpha;
#pragma unroll
        for (int c = 0; c < 2; ++c) o[c][tq] *= alpha;
      }
      const float mcur = m[tq];
      float rs = 0.f;
#pragma unroll
      for (int tk = 0; tk < 2; ++tk)
#pragma unroll
        for (int u = 0; u < 2; ++u) {
          bf16x2 pr[4];
#pragma unroll
          for (int e = 0; e < 4; ++e) {
            const f32x2 pf = {fast_exp2(fmaf(s[tk][tq][8 * u + 2 * e], sc, -mcur)),
                              fast_exp2(fmaf(s[tk][tq][8 * u + 2 * e + 1], sc, -mcur))};
            pr[e] = __builtin_convertvector(pf, bf16x2);
            rs = __builtin_amdgcn_fdot2_f32_bf16(pr[e], kOnes, rs, false);
          }
          pB[tk][u][tq] = bf16x8{pr[0][0], pr[0][1], pr[1][0], pr[1][1],
                                 pr[2][0], pr[2][1], pr[3][0], pr[3][1]};
        }
      l[tq] += rs;
    }

    // the V tile of jcur is in LDS (the next K tile, if any, may be in flight)
    if constexpr (more) wait_all_but_last_tile(); else wait_all_loads();

    // O^T[c][tq] += V^T[c][keys] P^T[keys][tq]
#pragma unroll
    for (int tk = 0; tk < 2; ++tk)
#pragma unroll
      for (int u = 0; u < 2; ++u) {
        const int krow = 32 * tk + 16 * u + tr_row;
#pragma unroll
        for (int c = 0; c < 2; ++c) {
          const int col = 32 * c + tr_col;
          const bf16x4 lo = __builtin_amdgcn_ds_read_tr16_b64_v4bf16(
              (lds_bf16x4*)(vs + swz(krow, col >> 3) + (col & 7) * 2));
          const bf16x4 hi = __builtin_amdgcn_ds_read_tr16_b64_v4bf16(
              (lds_bf16x4*)(vs + swz(krow + 8, col >> 3) + (col & 7) * 2));
          const bf16x8 vA = {lo[0], lo[1], lo[2], lo[3], hi[0], hi[1], hi[2], hi[3]};
#pragma unroll
          for (int tq = 0; tq < 2; ++tq)
            o[c][tq] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(vA, pB[tk][u][tq], o[c][tq], 0, 0, 0);
        }
      }
    // the V operands are consumed: refill the V tile for the next step
    if constexpr (more) {
      wait_lds();
      dma_tile(rv, j, vs, dma_off);
    }
  };
  for (int it = 0; it + 1 < count; ++it) step(it, std::false_type{});
  if (count > 0) step(count - 1, std::true_type{});

  // epilogue: normalise, round to bf16, store; log-sum-exp in natural log
#pragma unroll
  for (int tq = 0; tq < 2; ++tq) {
    const float lt = pair_sum(l[tq]);
    const float inv = 1.0f / lt;
    const int query = w.i * kBlock + 32 * tq + l32;
#pragma unroll
    for (int c = 0; c < 2; ++c)
#pragma unroll
      for (int g = 0; g < 4; ++g) {
        bf16x4 ov;
#pragma unroll
        for (int r = 0; r < 4; ++r) ov[r] = (__bf16)(o[c][tq][4 * g + r] * inv);
        __builtin_amdgcn_raw_buffer_store_b64(
            __builtin_bit_cast(i32x2, ov), ro,
            (int)((query * kHeadDim + 32 * c + 8 * g + 4 * hf) * 2), 0, 0);
      }
    if (lse && hf == 0 && query < a.n)
      lse[(int64_t)w.h * a.n + query] = (m[tq] + __log2f(lt)) * kLn2;
  }
}

// ------------------------------------------------------------------ fp32

// Same structure with v_mfma_f32_32x32x2_f32 and fp32 softmax operands; K and
// V tiles both go through LDS (one wave, no barrier).
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
  const bool dense = a.dense[w.h] != 0;
  const int32_t* list = idx + ((int64_t)w.h * nb + w.i) * a.cap;
  int count = nb;
  if (!dense) count = min(max(cnt[(int64_t)w.h * nb + w.i], 0), a.cap);

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
  const bool tail = (a.n % kBlock) != 0;
  const float sc = a.scale_log2;

  for (int it = 0; it < count; ++it) {
    const int j = dense ? it : list[it];
    // stage K and V tiles: rows 4n + lane/16, float4 chunk lane%16
#pragma unroll
    for (int n4 = 0; n4 < 16; ++n4) {
      const int row = 4 * n4 + (lane >> 4);
      const int off = ((j * kBlock + row) * kHeadDim + (lane & 15) * 4) * 4;
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

    if (tail && j == nb - 1) {
      const int valid_keys = (int)(a.n - (int64_t)j * kBlock);
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

#pragma unroll
  for (int tq = 0; tq < 2; ++tq) {
    const float lt = l[tq] + __shfl_xor(l[tq], 32);
    const float inv = 1.0f / lt;
    const int query = w.i * kBlock + 32 * tq + l32;
#pragma unroll
    for (int c = 0; c < 2; ++c)
#pragma unroll
      for (int g = 0; g < 4; ++g) {
        f32x4 ov;
#pragma unroll
        for (int r = 0; r < 4; ++r) ov[r] = o[c][tq][4 * g + r] * inv;
        __builtin_amdgcn_raw_buffer_store_b128(__builtin_bit_cast(i32x4, ov), ro,
                                               (query * kHeadDim + 32 * c + 8 * g + 4 * hf) * 4, 0, 0);
      }
    if (lse && hf == 0 && query < a.n)
      lse[(int64_t)w.h * a.n + query] = (m[tq] + log2f(lt)) * kLn2;
  }
}

}  // namespace

hipError_t launch_attention(int dtype, const void* q, const void* k, const void* v,
                            const int32_t* idx, const int32_t* cnt, void* out, float* lse,
                            const AttnArgs& a, hipStream_t s) {
  const int64_t groups = 8LL * a.heads * a.slab;
  if (groups == 0) return hipSuccess;
  bool all_dense = true;
  for (int h = 0; h < a.heads; ++h) all_dense = all_dense && a.dense[h];
  if (dtype == 1) {
    auto kern = all_dense ? attn_bf16_kernel<true> : attn_bf16_kernel<false>;
    hipLaunchKernelGGL(kern, dim3((unsigned)groups), dim3(64), 0, s,
                       static_cast<const uint16_t*>(q), static_cast<const uint16_t*>(k),
                       static_cast<const uint16_t*>(v), idx, cnt, static_cast<uint16_t*>(out),
                       lse, a);
  } else {
    hipLaunchKernelGGL(attn_f32_kernel, dim3((unsigned)groups), dim3(64), 0, s,
                       static_cast<const float*>(q), static_cast<const float*>(k),
                       static_cast<const float*>(v), idx, cnt, static_cast<float*>(out), lse, a);
  }
  return hipGetLastError();
}

}  // namespace saf3r
