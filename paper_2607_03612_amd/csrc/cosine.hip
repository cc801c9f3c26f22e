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
//   2. cosine_sim_kernel: the block similarity matrix [nb][nb] as a 64x64
//      register-tiled product of that matrix with itself;
//   3. cosine_topk_kernel: one wave per (head, query block); for every frame
//      (a key block counts under the frame of its first token) it finds the
//      k-th best (similarity desc, index asc) pair by k passes of a wave-wide
//      argmax and writes the frame's kept blocks ascending.
// The lists depend on the features only, so they are computed once per
// sequence and reused by every layer.
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
template <typename T>
__global__ __launch_bounds__(kPoolThreads) void cosine_pool_kernel(const T* __restrict__ f,
                                                                  double* __restrict__ fb,
                                                                  CosineArgs a) {
  __shared__ double inv_norm[kBlock];
  __shared__ double part[kPoolThreads / 64];
  const int b = blockIdx.x;
  const int t = threadIdx.x, lane = t & 63, wave = t >> 6;
  const int64_t row0 = (int64_t)b * kBlock;
  const int rows = (int)min<int64_t>(kBlock, a.n - row0);
  // 1/|f_t| for the block's tokens: one wave per token
  for (int r = wave; r < rows; r += kPoolThreads / 64) {
    double ss = 0.0;
    for (int d = lane; d < a.dim; d += 64) {
      const double x = feat_at(f, (row0 + r) * a.dim + d);
      ss = fma(x, x, ss);
    }
#pragma unroll
    for (int m = 32; m >= 1; m >>= 1) ss += __shfl_xor(ss, m);
    if (lane == 0) inv_norm[r] = 1.0 / sqrt(ss);
  }
  __syncthreads();
  for (int d = t; d < a.dim; d += kPoolThreads) {
    double acc = 0.0;
    for (int r = 0; r < rows; ++r) acc = fma(feat_at(f, (row0 + r) * a.dim + d), inv_norm[r], acc);
    fb[(int64_t)d * a.nb + b] = acc / (double)rows;
  }
  (void)part;
}

// sim[i][j] = sum_d fb[d][i] fb[d][j]: 64x64 tiles, 16x16 threads of 4x4.
__global__ __launch_bounds__(256) void cosine_sim_kernel(const double* __restrict__ fb,
                                                        double* __restrict__ sim, CosineArgs a) {
  __shared__ double as[16][64];
  __shared__ double bs[16][64];
  const int tiles = (a.nb + 63) / 64;
  const int ti = blockIdx.x / tiles, tj = blockIdx.x - (blockIdx.x / tiles) * tiles;
  const int i0 = ti * 64, j0 = tj * 64;
  const int tx = threadIdx.x & 15, ty = threadIdx.x >> 4;
  double acc[4][4];
#pragma unroll
  for (int x = 0; x < 4; ++x)
#pragma unroll
    for (int y = 0; y < 4; ++y) acc[x][y] = 0.0;
  for (int d0 = 0; d0 < a.dim; d0 += 16) {
    // stage 16 dimensions of the 64 rows and 64 columns
    for (int e = threadIdx.x; e < 16 * 64; e += 256) {
      const int dd = e >> 6, c = e & 63;
      const int d = d0 + dd;
      as[dd][c] = d < a.dim && i0 + c < a.nb ? fb[(int64_t)d * a.nb + i0 + c] : 0.0;
      bs[dd][c] = d < a.dim && j0 + c < a.nb ? fb[(int64_t)d * a.nb + j0 + c] : 0.0;
    }
    __syncthreads();
#pragma unroll
    for (int dd = 0; dd < 16; ++dd) {
      double av[4], bv[4];
#pragma unroll
      for (int x = 0; x < 4; ++x) av[x] = as[dd][4 * ty + x];
#pragma unroll
      for (int y = 0; y < 4; ++y) bv[y] = bs[dd][4 * tx + y];
#pragma unroll
      for (int x = 0; x < 4; ++x)
#pragma unroll
        for (int y = 0; y < 4; ++y) acc[x][y] = fma(av[x], bv[y], acc[x][y]);
    }
    __syncthreads();
  }
#pragma unroll
  for (int x = 0; x < 4; ++x) {
    const int i = i0 + 4 * ty + x;
    if (i >= a.nb) continue;
#pragma unroll
    for (int y = 0; y < 4; ++y) {
      const int j = j0 + 4 * tx + y;
      if (j < a.nb) sim[(int64_t)i * a.nb + j] = acc[x][y];
    }
  }
}

// (value, index) order of the selection: higher value first, then lower index
__device__ inline bool ranks_before(double v, int j, double w, int k) {
  return v > w || (v == w && j < k);
}

// One wave per (cosine head, query block): per-frame Top-K, ascending output.
__global__ __launch_bounds__(256) void cosine_topk_kernel(const double* __restrict__ sim,
                                                         int32_t* __restrict__ idx,
                                                         int32_t* __restrict__ cnt,
                                                         CosineArgs a) {
  const int lane = threadIdx.x & 63;
  const int64_t wave = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6);
  if (wave >= (int64_t)a.n_heads * a.nb) return;
  const int slot = (int)(wave / a.nb);
  const int i = (int)(wave - (int64_t)slot * a.nb);
  const int h = a.head[slot];
  const int k = a.topk[slot];
  const double* row = sim + (int64_t)i * a.nb;
  int32_t* dst = idx + ((int64_t)h * a.nb + i) * a.cap;
  const int64_t T = a.tokens_per_frame;
  const int frames = (int)((a.n + T - 1) / T);
  int pos = 0;
  for (int f = 0; f < frames; ++f) {
    // key blocks whose first token lies in frame f
    const int j_lo = (int)(((int64_t)f * T + kBlock - 1) / kBlock);
    const int j_hi = (int)min<int64_t>(((int64_t)(f + 1) * T + kBlock - 1) / kBlock, a.nb);
    const int size = j_hi - j_lo;
    if (size <= 0) continue;
    const int kk = min(k, size);
    // k-th pair in (value desc, index asc) order: kk passes of a wave argmax
    // over the pairs ranked after the previous pass's pair
    double tv = __builtin_inf();
    int tj = -1;
    for (int p = 0; p < kk; ++p) {
      double bv = -__builtin_inf();
      int bj = a.nb;
      for (int j = j_lo + lane; j < j_hi; j += 64) {
        const double v = row[j];
        if (ranks_before(tv, tj, v, j) && ranks_before(v, j, bv, bj)) {
          bv = v;
          bj = j;
        }
      }
#pragma unroll
      for (int m = 32; m >= 1; m >>= 1) {
        const double ov = __shfl_xor(bv, m);
        const int oj = __shfl_xor(bj, m);
        if (ranks_before(ov, oj, bv, bj)) {
          bv = ov;
          bj = oj;
        }
      }
      tv = bv;
      tj = bj;
    }
    // the frame's kept blocks: every pair ranked at or before (tv, tj)
    for (int j0 = j_lo; j0 < j_hi; j0 += 64) {
      const int j = j0 + lane;
      const bool keep = j < j_hi && !ranks_before(tv, tj, row[j < j_hi ? j : j_lo], j);
      const uint64_t m = __ballot(keep);
      const int at = pos + __popcll(m & ((1ull << lane) - 1));
      if (keep && at < a.cap) dst[at] = j;
      pos += __popcll(m);
    }
  }
  for (int p = pos + lane; p < a.cap; p += 64) dst[p] = -1;
  if (lane == 0) cnt[(int64_t)h * a.nb + i] = pos;
}

}  // namespace

hipError_t launch_cosine(int dtype, const void* f, double* fb, double* sim, int32_t* idx,
                         int32_t* cnt, const CosineArgs& a, hipStream_t s) {
  if (a.n_heads == 0) return hipSuccess;
  if (dtype == 1)
    hipLaunchKernelGGL(cosine_pool_kernel<uint16_t>, dim3((unsigned)a.nb), dim3(kPoolThreads), 0, s,
                       static_cast<const uint16_t*>(f), fb, a);
  else
    hipLaunchKernelGGL(cosine_pool_kernel<float>, dim3((unsigned)a.nb), dim3(kPoolThreads), 0, s,
                       static_cast<const float*>(f), fb, a);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  const int tiles = (a.nb + 63) / 64;
  hipLaunchKernelGGL(cosine_sim_kernel, dim3((unsigned)(tiles * tiles)), dim3(256), 0, s, fb, sim, a);
  e = hipGetLastError();
  if (e != hipSuccess) return e;
  const int64_t waves = (int64_t)a.n_heads * a.nb;
  hipLaunchKernelGGL(cosine_topk_kernel, dim3((unsigned)((waves + 3) / 4)), dim3(256), 0, s, sim,
                     idx, cnt, a);
  return hipGetLastError();
}

}  // namespace saf3r
