// Approximation cost of a sparse configuration (Sec. 4.2, Eq. 1): per head,
//   E = ||O_full - O_sparse||^2 / ||O_full||^2
// summed in float64 over the head's N x 64 outputs. One workgroup per head
// (a fixed reduction order, so the result is deterministic); 16-byte loads.
#include "saf3r_internal.h"

namespace saf3r {
namespace {

constexpr int kNmseThreads = 1024;

__device__ inline void add_pairs(uint32_t a, uint32_t b, double& num, double& den) {
  const double a0 = (double)__uint_as_float(a << 16), a1 = (double)__uint_as_float(a & 0xffff0000u);
  const double b0 = (double)__uint_as_float(b << 16), b1 = (double)__uint_as_float(b & 0xffff0000u);
  num = fma(a0 - b0, a0 - b0, num);
  num = fma(a1 - b1, a1 - b1, num);
  den = fma(a0, a0, den);
  den = fma(a1, a1, den);
}

template <bool kBf16>
__global__ __launch_bounds__(kNmseThreads) void nmse_kernel(const uint4* __restrict__ ref,
                                                           const uint4* __restrict__ test,
                                                           double* __restrict__ out,
                                                           int64_t vec_per_head) {
  __shared__ double part[2][kNmseThreads / 64];
  const int h = blockIdx.x;
  const uint4* r = ref + (int64_t)h * vec_per_head;
  const uint4* t = test + (int64_t)h * vec_per_head;
  double num = 0.0, den = 0.0;
  for (int64_t e = threadIdx.x; e < vec_per_head; e += kNmseThreads) {
    const uint4 a = r[e], b = t[e];
    if constexpr (kBf16) {
      add_pairs(a.x, b.x, num, den);
      add_pairs(a.y, b.y, num, den);
      add_pairs(a.z, b.z, num, den);
      add_pairs(a.w, b.w, num, den);
    } else {
      const uint32_t av[4] = {a.x, a.y, a.z, a.w}, bv[4] = {b.x, b.y, b.z, b.w};
#pragma unroll
      for (int c = 0; c < 4; ++c) {
        const double x = (double)__uint_as_float(av[c]), y = (double)__uint_as_float(bv[c]);
        num = fma(x - y, x - y, num);
        den = fma(x, x, den);
      }
    }
  }
#pragma unroll
  for (int m = 32; m >= 1; m >>= 1) {
    num += __shfl_xor(num, m);
    den += __shfl_xor(den, m);
  }
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  if (lane == 0) {
    part[0][wave] = num;
    part[1][wave] = den;
  }
  __syncthreads();
  if (threadIdx.x == 0) {
    double sn = 0.0, sd = 0.0;
    for (int w = 0; w < kNmseThreads / 64; ++w) {
      sn += part[0][w];
      sd += part[1][w];
    }
    out[h] = sn / sd;
  }
}

}  // namespace

hipError_t launch_nmse(int dtype, const void* ref, const void* test, double* out, int heads,
                       int64_t n, hipStream_t s) {
  const int64_t esz = dtype == 1 ? 2 : 4;
  const int64_t vec = n * kHeadDim * esz / 16;  // N x 64 elements per head, 16-byte vectors
  if (dtype == 1)
    hipLaunchKernelGGL(nmse_kernel<true>, dim3((unsigned)heads), dim3(kNmseThreads), 0, s,
                       static_cast<const uint4*>(ref), static_cast<const uint4*>(test), out, vec);
  else
    hipLaunchKernelGGL(nmse_kernel<false>, dim3((unsigned)heads), dim3(kNmseThreads), 0, s,
                       static_cast<const uint4*>(ref), static_cast<const uint4*>(test), out, vec);
  return hipGetLastError();
}

}  // namespace saf3r
