// DINO Top-K kernel, block-wise form (Sec. 4.1 and Sec. 4.3): per query block,
// the key blocks of every frame whose features are most similar to its own.
//
// The features are the caller's per-token vectors (the paper uses the last
// DINO block's patch features). Every token's feature is scaled to unit
// length and averaged over its block; the dot product of two block means is
// then the mean cosine similarity over the tile of token pairs, the same
// linearity argument as the query probe. All of it runs in float64:
//   1. cosine_pool_kernel: one workgroup per block writes the block's mean
//      unit feature, dimension-major [D][nb];
//   2. cosine_sim_mfma_kernel: the block similarity matrix [nb][nb], the
//      product of that matrix with itself on the fp64 matrix cores (upper
//      tiles only, mirrored);
//   3. cosine_topk_kernel: one wave per (per-frame count k, query block), one
//      lane per frame (a key block counts under the frame of its first
//      token): k scans find the frame's k-th best (similarity desc, index
//      asc) pair; the frame's kept blocks go out ascending at an offset from
//      a prefix sum over the frames, into every head that keeps k per frame.
// The lists depend on the features only, so they are computed once per
// sequence and reused by every layer.
#include <algorithm>

#include "saf3r_internal.h"

namespace saf3r {
namespace {

constexpr int kPoolThreads = 256;

template <typename T>
__device__ inline double feat_at(const T* f, int64_t i);
template <>
__device__ inline double feat_at<uint16_t>(const uint16_t* f, int64_t i) {
  return (double)__uint_as_float((uint32_t)f[i] << 16);
}
template <>
__device__ inline double feat_at<float>(const float* f, int64_t i) {
  return (double)f[i];
}

// Mean unit feature of block b: fb[d][b] = (1/n_b) sum_t f[t][d] / |f[t]|.
// kVec: rows are whole 16-byte vectors (feat_dim * element size a multiple
// of 16, 16-byte aligned base), read 16 bytes per lane; otherwise one element
// per lane.
template <typename T, bool kVec>
__global__ __launch_bounds__(kPoolThreads) void cosine_pool_kernel(const T* __restrict__ f,
                                                                  double* __restrict__ fb,
                                                                  CosineArgs a) {
  constexpr int kPer = 16 / (int)sizeof(T);  // elements per 16-byte vector
  __shared__ double inv_norm[kBlock];
  const int b = blockIdx.x;
  const int t = threadIdx.x, lane = t & 63, wave = t >> 6;
  const int64_t row0 = (int64_t)b * kBlock;
  const int rows = (int)min<int64_t>(kBlock, a.n - row0);
  const int vecs = a.dim / kPer;  // 16-byte vectors per row (kVec)
  // 1/|f_t| for the block's tokens: one wave per token
  for (int r = wave; r < rows; r += kPoolThreads / 64) {
    double ss = 0.0;
    if constexpr (kVec) {
      const uint4* row = reinterpret_cast<const uint4*>(f + (row0 + r) * a.dim);
      for (int c = lane; c < vecs; c += 64) {
        const uint4 u = row[c];
        const T* e = reinterpret_cast<const T*>(&u);
#pragma unroll
        for (int q = 0; q < kPer; ++q) {
          const double x = feat_at(e, q);
          ss = fma(x, x, ss);
        }
      }
    } else {
      for (int d = lane; d < a.dim; d += 64) {
        const double x = feat_at(f, (row0 + r) * a.dim + d);
        ss = fma(x, x, ss);
      }
    }
#pragma unroll
    for (int m = 32; m >= 1; m >>= 1) ss += __shfl_xor(ss, m);
    if (lane == 0) inv_norm[r] = 1.0 / sqrt(ss);
  }
  __syncthreads();
  if constexpr (kVec) {
    // thread t: dimensions [kPer c, kPer c + kPer) for c = t, t + 256, ...
    for (int c = t; c < vecs; c += kPoolThreads) {
      double acc[kPer];
#pragma unroll
      for (int q = 0; q < kPer; ++q) acc[q] = 0.0;
      const uint4* col = reinterpret_cast<const uint4*>(f + row0 * a.dim) + c;
      for (int r = 0; r < rows; ++r) {
        const uint4 u = col[(int64_t)r * vecs];
        const T* e = reinterpret_cast<const T*>(&u);
#pragma unroll
        for (int q = 0; q < kPer; ++q) acc[q] = fma(feat_at(e, q), inv_norm[r], acc[q]);
      }
#pragma unroll
      for (int q = 0; q < kPer; ++q) fb[(int64_t)(kPer * c + q) * a.nb + b] = acc[q] / (double)rows;
    }
  } else {
    for (int d = t; d < a.dim; d += kPoolThreads) {
      double acc = 0.0;
      for (int r = 0; r < rows; ++r) acc = fma(feat_at(f, (row0 + r) * a.dim + d), inv_norm[r], acc);
      fb[(int64_t)d * a.nb + b] = acc / (double)rows;
    }
  }
}

typedef double f64x4 __attribute__((ext_vector_type(4)));

// sim[i][j] = sum_d fb[d][i] fb[d][j] on the fp64 matrix cores: a 64x64
// tile per workgroup, a 32x32 quarter per wave as 2x2 tiles of
// v_mfma_f64_16x16x4f64 (A: 16 row blocks x 4 dimensions, one double per
// lane; B: 4 dimensions x 16 column blocks; both read 16 consecutive blocks
// of one dimension, 128 B). The matrix is symmetric: only tiles on or above
// the diagonal are computed, and an off-diagonal tile is also stored
// transposed.
__global__ __launch_bounds__(256) void cosine_sim_mfma_kernel(const double* __restrict__ fb,
                                                             double* __restrict__ sim,
                                                             CosineArgs a) {
  const int tiles = (a.nb + 63) / 64;
  const int ti = blockIdx.x / tiles, tj = blockIdx.x - (blockIdx.x / tiles) * tiles;
  if (ti > tj) return;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int r0 = ti * 64 + 32 * (wave >> 1), c0 = tj * 64 + 32 * (wave & 1);
  const int nb = a.nb;
  const int sub = lane >> 4;  // dimension within a group of 4
  auto operand = [&](int d0, int blk) -> double {
    const int d = d0 + sub;
    return d < a.dim && blk < nb ? fb[(int64_t)d * nb + blk] : 0.0;
  };
  f64x4 acc[2][2];
#pragma unroll
  for (int x = 0; x < 2; ++x)
#pragma unroll
    for (int y = 0; y < 2; ++y) acc[x][y] = f64x4{0.0, 0.0, 0.0, 0.0};
  // 16 dimensions per step (four MFMA groups), the next 16 loading meanwhile
  constexpr int kSteps = 4;
  double an[kSteps][2], bn[kSteps][2];
  auto load_step = [&](int d0, double (&ax)[kSteps][2], double (&bx)[kSteps][2]) {
#pragma unroll
    for (int u = 0; u < kSteps; ++u)
#pragma unroll
      for (int x = 0; x < 2; ++x) {
        ax[u][x] = operand(d0 + 4 * u, r0 + 16 * x + (lane & 15));
        bx[u][x] = operand(d0 + 4 * u, c0 + 16 * x + (lane & 15));
      }
  };
  load_step(0, an, bn);
  for (int d0 = 0; d0 < a.dim; d0 += 4 * kSteps) {
    double ac[kSteps][2], bc[kSteps][2];
#pragma unroll
    for (int u = 0; u < kSteps; ++u)
#pragma unroll
      for (int x = 0; x < 2; ++x) {
        ac[u][x] = an[u][x];
        bc[u][x] = bn[u][x];
      }
    load_step(d0 + 4 * kSteps, an, bn);
#pragma unroll
    for (int u = 0; u < kSteps; ++u) {
      acc[0][0] = __builtin_amdgcn_mfma_f64_16x16x4f64(ac[u][0], bc[u][0], acc[0][0], 0, 0, 0);
      acc[0][1] = __builtin_amdgcn_mfma_f64_16x16x4f64(ac[u][0], bc[u][1], acc[0][1], 0, 0, 0);
      acc[1][0] = __builtin_amdgcn_mfma_f64_16x16x4f64(ac[u][1], bc[u][0], acc[1][0], 0, 0, 0);
      acc[1][1] = __builtin_amdgcn_mfma_f64_16x16x4f64(ac[u][1], bc[u][1], acc[1][1], 0, 0, 0);
    }
  }
  // element e of a lane: row (lane / 16) + 4e, column lane % 16 of the tile
#pragma unroll
  for (int x = 0; x < 2; ++x)
#pragma unroll
    for (int y = 0; y < 2; ++y)
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        const int i = r0 + 16 * x + sub + 4 * e;
        const int j = c0 + 16 * y + (lane & 15);
        if (i < nb && j < nb) {
          sim[(int64_t)i * nb + j] = acc[x][y][e];
          if (ti != tj) sim[(int64_t)j * nb + i] = acc[x][y][e];
        }
      }
}

// (value, index) order of the selection: higher value first, then lower index
__device__ inline bool ranks_before(double v, int j, double w, int k) {
  return v > w || (v == w && j < k);
}

// Inclusive prefix sum over the 64 lanes.
__device__ inline int lane_scan_incl(int v) {
#pragma unroll
  for (int d = 1; d < 64; d <<= 1) {
    const int o = __shfl_up(v, d);
    if ((threadIdx.x & 63) >= d) v += o;
  }
  return v;
}

// One wave per (group of cosine heads with one per-frame count k, query
// block). Lane f handles frame f (64 frames per pass): k scans of the frame's
// blocks find its k-th best (similarity desc, index asc) pair, a prefix sum
// of the per-frame kept counts gives the frame's offset in the row, and the
// lane writes the frame's kept blocks there in ascending order, into the row
// of every head of the group.
// kLds: the wave first copies its similarity row into its own LDS row
// (coalesced), and the lanes' frame scans read LDS instead of scattered
// global words (rows up to kTopkLdsRow doubles). The row's list is built in
// the wave's LDS list (cap entries) and then copied, coalesced, into the row
// of every head of the group.
constexpr int kTopkLdsRow = 8192;

// list entries kept in LDS: a row keeps at most nb blocks
__host__ __device__ inline int topk_list_len(const CosineArgs& a) { return a.cap < a.nb ? a.cap : a.nb; }

template <bool kLds>
__global__ __launch_bounds__(256) void cosine_topk_kernel(const double* __restrict__ sim,
                                                         int32_t* __restrict__ idx,
                                                         int32_t* __restrict__ cnt,
                                                         CosineArgs a) {
  extern __shared__ double srow[];  // [waves][nb] doubles when kLds, then [waves][cap] ints
  const int lane = threadIdx.x & 63;
  const int wl = threadIdx.x >> 6;
  const int wpg = blockDim.x >> 6;
  const int64_t wave = (int64_t)blockIdx.x * wpg + wl;
  if (wave >= (int64_t)a.n_groups * a.nb) return;  // whole waves; no barrier below
  const int g = (int)(wave / a.nb);
  const int i = (int)(wave - (int64_t)g * a.nb);
  const int k = a.group_k[g];
  const int q0 = a.group_start[g], q1 = a.group_start[g + 1];
  const double* grow = sim + (int64_t)i * a.nb;
  double* lrow = srow + (int64_t)wl * a.nb;
  const int list_len = topk_list_len(a);
  int* llist = reinterpret_cast<int*>(srow + (kLds ? (int64_t)wpg * a.nb : 0)) + (int64_t)wl * list_len;
  if constexpr (kLds) {
    for (int j = lane; j < a.nb; j += 64) lrow[j] = grow[j];
    asm volatile("" ::: "memory");  // a wave's LDS accesses run in order
  }
  const double* row = kLds ? lrow : grow;
  const int64_t T = a.tokens_per_frame;
  const int frames = (int)((a.n + T - 1) / T);
  int base = 0;
  for (int f0 = 0; f0 < frames; f0 += 64) {
    // key blocks whose first token lies in frame f
    const int f = f0 + lane;
    int j_lo = 0, j_hi = 0;
    if (f < frames) {
      j_lo = (int)(((int64_t)f * T + kBlock - 1) / kBlock);
      j_hi = (int)min<int64_t>(((int64_t)(f + 1) * T + kBlock - 1) / kBlock, a.nb);
    }
    const int kk = min(k, max(j_hi - j_lo, 0));
    // the kk-th pair: each scan takes the best pair ranked after the last
    double tv = __builtin_inf();
    int tj = -1;
    for (int p = 0; p < kk; ++p) {
      double bv = -__builtin_inf();
      int bj = a.nb;
      for (int j = j_lo; j < j_hi; ++j) {
        const double v = row[j];
        if (ranks_before(tv, tj, v, j) && ranks_before(v, j, bv, bj)) {
          bv = v;
          bj = j;
        }
      }
      tv = bv;
      tj = bj;
    }
    // kept: every pair ranked at or before (tv, tj)
    int kept = 0;
    if (kk > 0)
      for (int j = j_lo; j < j_hi; ++j) kept += ranks_before(tv, tj, row[j], j) ? 0 : 1;
    const int incl = lane_scan_incl(kept);
    int pos = base + incl - kept;
    if (kept > 0) {
      for (int j = j_lo; j < j_hi; ++j) {
        if (ranks_before(tv, tj, row[j], j)) continue;
        if (pos < list_len) llist[pos] = j;
        ++pos;
      }
    }
    base += __shfl(incl, 63);
  }
  asm volatile("" ::: "memory");  // the list's LDS writes, then the wave's reads
  for (int q = q0; q < q1; ++q) {
    const int h = a.head[q];
    int32_t* dst = idx + ((int64_t)h * a.nb + i) * a.cap;
    for (int p = lane; p < a.cap; p += 64) dst[p] = p < base ? llist[p] : -1;
    if (lane == 0) cnt[(int64_t)h * a.nb + i] = base;
  }
}

}  // namespace

hipError_t launch_cosine(int dtype, const void* f, double* fb, double* sim, int32_t* idx,
                         int32_t* cnt, const CosineArgs& a, hipStream_t s) {
  if (a.n_groups == 0) return hipSuccess;
  const int esz = dtype == 1 ? 2 : 4;
  const bool vec = ((int64_t)a.dim * esz) % 16 == 0 && (reinterpret_cast<uintptr_t>(f) & 15) == 0;
  const dim3 grid((unsigned)a.nb), block(kPoolThreads);
  if (dtype == 1) {
    const uint16_t* fp = static_cast<const uint16_t*>(f);
    if (vec)
      hipLaunchKernelGGL((cosine_pool_kernel<uint16_t, true>), grid, block, 0, s, fp, fb, a);
    else
      hipLaunchKernelGGL((cosine_pool_kernel<uint16_t, false>), grid, block, 0, s, fp, fb, a);
  } else {
    const float* fp = static_cast<const float*>(f);
    if (vec)
      hipLaunchKernelGGL((cosine_pool_kernel<float, true>), grid, block, 0, s, fp, fb, a);
    else
      hipLaunchKernelGGL((cosine_pool_kernel<float, false>), grid, block, 0, s, fp, fb, a);
  }
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  const int tiles = (a.nb + 63) / 64;
  hipLaunchKernelGGL(cosine_sim_mfma_kernel, dim3((unsigned)(tiles * tiles)), dim3(256), 0, s, fb, sim, a);
  e = hipGetLastError();
  if (e != hipSuccess) return e;
  const int64_t waves = (int64_t)a.n_groups * a.nb;
  // per wave: the similarity row (kLds) and the list; waves per workgroup
  // such that a workgroup takes at most 96 KB of LDS, at most four
  const bool lds_row = a.nb <= kTopkLdsRow;
  const size_t wave_bytes = (lds_row ? (size_t)a.nb * sizeof(double) : 0) +
                            (size_t)topk_list_len(a) * sizeof(int);
  const int wpg = (int)std::max<size_t>(1, std::min<size_t>(4, (96 * 1024) / wave_bytes));
  const size_t lds = (size_t)wpg * wave_bytes;
  const dim3 tgrid((unsigned)((waves + wpg - 1) / wpg)), tblock(64 * wpg);
  auto go = [&](auto kern) -> hipError_t {
    hipError_t e2 = hipFuncSetAttribute(reinterpret_cast<const void*>(kern),
                                        hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
    if (e2 != hipSuccess) return e2;
    hipLaunchKernelGGL(kern, tgrid, tblock, lds, s, sim, idx, cnt, a);
    return hipGetLastError();
  };
  return lds_row ? go(cosine_topk_kernel<true>) : go(cosine_topk_kernel<false>);
}

}  // namespace saf3r
