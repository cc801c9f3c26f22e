// Block pooling for the query-probe estimate (Sec. 4.3): the probe of a set
// of queries is their mean; SAF3R's online stage pools every 64-token block of
// Q and K of each Top-K head.
//
// HBM-bound: each 64x64 tile is read once with 16-byte coalesced nontemporal
// loads (one wave per tile, eight rows of 128 B per load instruction) and summed in
// float64, which is exact for bf16 inputs (8-bit significands summed in a
// 53-bit significand), then divided by the block's own token count. Pooled Q
// is written [H][nb][64]; pooled K dimension-major [H][64][nb], the layout
// the scoring reads coalesce on.
#include "saf3r_internal.h"

namespace saf3r {
namespace {

constexpr int kWavesPerGroup = 4;

typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));

__device__ inline float bf16_lo(uint32_t w) { return __uint_as_float(w << 16); }
__device__ inline float bf16_hi(uint32_t w) { return __uint_as_float(w & 0xffff0000u); }

// One wave pools one 64-token block of one head of Q or K.
__global__ __launch_bounds__(256) void pool_bf16_kernel(const uint16_t* __restrict__ q,
                                                        const uint16_t* __restrict__ k,
                                                        double* __restrict__ qp,
                                                        double* __restrict__ kp, PoolArgs a) {
  const int lane = threadIdx.x & 63;
  const int64_t wave = (int64_t)blockIdx.x * kWavesPerGroup + (threadIdx.x >> 6);
  const int64_t per_tensor = (int64_t)a.n_heads * a.nb;
  if (wave >= 2 * per_tensor) return;
  const int tensor = wave >= per_tensor ? 1 : 0;
  const int64_t w = wave - tensor * per_tensor;
  const int slot = (int)(w / a.nb);
  const int b = (int)(w - (int64_t)slot * a.nb);
  const int h = a.head[slot];
  const int64_t row0 = (int64_t)b * kBlock;
  const int rows = (int)min<int64_t>(kBlock, a.n - row0);

  const uint16_t* src = (tensor ? k : q) + ((int64_t)h * a.n + row0) * kHeadDim;
  const int r = lane >> 3;  // row within each group of 8 rows
  const int c = lane & 7;   // 16-byte chunk = 8 columns

  // rows past a partial last block load a clamped valid row (so all eight
  // loads issue back to back) and are zeroed afterwards; the loads are
  // nontemporal (each tile is read once here), which keeps them from
  // displacing other lines and makes the stream faster from a cold cache
  u32x4 v[8];
#pragma unroll
  for (int it = 0; it < 8; ++it) {
    const int row = r + 8 * it;
    v[it] = __builtin_nontemporal_load(
        reinterpret_cast<const u32x4*>(src + min(row, rows - 1) * kHeadDim + c * 8));
  }
#pragma unroll
  for (int it = 0; it < 8; ++it)
    if (r + 8 * it >= rows) v[it] = u32x4{0u, 0u, 0u, 0u};
  double acc[8];
#pragma unroll
  for (int e = 0; e < 8; ++e) acc[e] = 0.0;
#pragma unroll
  for (int it = 0; it < 8; ++it) {
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      acc[2 * e] += (double)bf16_lo(v[it][e]);
      acc[2 * e + 1] += (double)bf16_hi(v[it][e]);
    }
  }
  // lanes c, c+8, ..., c+56 hold partial sums of the same 8 columns
#pragma unroll
  for (int m = 8; m < 64; m <<= 1) {
#pragma unroll
    for (int e = 0; e < 8; ++e) acc[e] += __shfl_xor(acc[e], m);
  }
  if (r == 0) {
    const double nrows = (double)rows;
    if (tensor == 0) {
      double* dst = qp + ((int64_t)h * a.nb + b) * kHeadDim + c * 8;
#pragma unroll
      for (int e = 0; e < 8; e += 2) {
        double2 o;
        o.x = acc[e] / nrows;
        o.y = acc[e + 1] / nrows;
        *reinterpret_cast<double2*>(dst + e) = o;
      }
    } else {  // dimension-major [H][64][nb]
      double* dst = kp + ((int64_t)h * kHeadDim + c * 8) * a.nb + b;
#pragma unroll
      for (int e = 0; e < 8; ++e) dst[(int64_t)e * a.nb] = acc[e] / nrows;
    }
  }
}

__global__ __launch_bounds__(256) void pool_f32_kernel(const float* __restrict__ q,
                                                       const float* __restrict__ k,
                                                       double* __restrict__ qp,
                                                       double* __restrict__ kp, PoolArgs a) {
  const int lane = threadIdx.x & 63;
  const int64_t wave = (int64_t)blockIdx.x * kWavesPerGroup + (threadIdx.x >> 6);
  const int64_t per_tensor = (int64_t)a.n_heads * a.nb;
  if (wave >= 2 * per_tensor) return;
  const int tensor = wave >= per_tensor ? 1 : 0;
  const int64_t w = wave - tensor * per_tensor;
  const int slot = (int)(w / a.nb);
  const int b = (int)(w - (int64_t)slot * a.nb);
  const int h = a.head[slot];
  const int64_t row0 = (int64_t)b * kBlock;
  const int rows = (int)min<int64_t>(kBlock, a.n - row0);

  const float* src = (tensor ? k : q) + ((int64_t)h * a.n + row0) * kHeadDim;
  const int r = lane >> 4;  // row within each group of 4 rows
  const int c = lane & 15;  // 16-byte chunk = 4 columns

  double acc[4] = {0.0, 0.0, 0.0, 0.0};
#pragma unroll
  for (int it = 0; it < 16; ++it) {
    const int row = r + 4 * it;
    float4 x = *reinterpret_cast<const float4*>(src + min(row, rows - 1) * kHeadDim + c * 4);
    if (row >= rows) x = make_float4(0.f, 0.f, 0.f, 0.f);
    acc[0] += (double)x.x;
    acc[1] += (double)x.y;
    acc[2] += (double)x.z;
    acc[3] += (double)x.w;
  }
#pragma unroll
  for (int m = 16; m < 64; m <<= 1) {
#pragma unroll
    for (int e = 0; e < 4; ++e) acc[e] += __shfl_xor(acc[e], m);
  }
  if (r == 0) {
    const double nrows = (double)rows;
    if (tensor == 0) {
      double* dst = qp + ((int64_t)h * a.nb + b) * kHeadDim + c * 4;
      double2 o0, o1;
      o0.x = acc[0] / nrows;
      o0.y = acc[1] / nrows;
      o1.x = acc[2] / nrows;
      o1.y = acc[3] / nrows;
      *reinterpret_cast<double2*>(dst) = o0;
      *reinterpret_cast<double2*>(dst + 2) = o1;
    } else {  // dimension-major [H][64][nb]
      double* dst = kp + ((int64_t)h * kHeadDim + c * 4) * a.nb + b;
#pragma unroll
      for (int e = 0; e < 4; ++e) dst[(int64_t)e * a.nb] = acc[e] / nrows;
    }
  }
}

}  // namespace

hipError_t launch_pool(int dtype, const void* q, const void* k, double* qp, double* kp,
                       const PoolArgs& a, hipStream_t s) {
  const int64_t waves = 2 * (int64_t)a.n_heads * a.nb;
  if (waves == 0) return hipSuccess;
  const dim3 grid((unsigned)((waves + kWavesPerGroup - 1) / kWavesPerGroup));
  if (dtype == 1) {
    hipLaunchKernelGGL(pool_bf16_kernel, grid, dim3(256), 0, s, static_cast<const uint16_t*>(q),
                       static_cast<const uint16_t*>(k), qp, kp, a);
  } else {
    hipLaunchKernelGGL(pool_f32_kernel, grid, dim3(256), 0, s, static_cast<const float*>(q),
                       static_cast<const float*>(k), qp, kp, a);
  }
  return hipGetLastError();
}

}  // namespace saf3r
