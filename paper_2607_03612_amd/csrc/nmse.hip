// Approximation cost of a sparse configuration (Sec. 4.2, Eq. 1): per head,
//   E = ||O_full - O_sparse||^2 / ||O_full||^2
// summed in float64 over the head's N x 64 outputs.
//
// Two launches with a fixed reduction order (the result is deterministic):
//   1. kNmseParts workgroups per head each sum one contiguous slice of the
//      head's outputs (16-byte loads, four in flight per thread) and write
//      their (numerator, denominator) pair to the workspace;
//   2. one wave per head adds its kNmseParts pairs and divides.
#include <atomic>

#include "saf3r_internal.h"

namespace saf3r {

// Partial sums of saf3r_nmse_noalloc: the (numerator, denominator) pairs of
// up to kMaxHeads heads, kNmseScratchBytes (512 KB), which each GPU the
// library runs on holds until the process ends. Host code never passes this
// name to a kernel (on the host it is a stand-in, not a device address): the
// array's device address comes from hipGetSymbolAddress, once per device.
static __device__ __align__(256) double2 scratch[kMaxHeads * kNmseParts];
static_assert(sizeof(scratch) == kNmseScratchBytes, "scratch size");

namespace {

constexpr int kNmseThreads = 256;
constexpr int kNmseUnroll = 4;

__device__ inline void add_pairs(uint32_t a, uint32_t b, double& num, double& den) {
  const double a0 = (double)__uint_as_float(a << 16), a1 = (double)__uint_as_float(a & 0xffff0000u);
  const double b0 = (double)__uint_as_float(b << 16), b1 = (double)__uint_as_float(b & 0xffff0000u);
  num = fma(a0 - b0, a0 - b0, num);
  num = fma(a1 - b1, a1 - b1, num);
  den = fma(a0, a0, den);
  den = fma(a1, a1, den);
}

template <bool kBf16>
__device__ inline void add_vec(const uint4& a, const uint4& b, double& num, double& den) {
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

// Workgroup (h, p): 16-byte vectors [p * chunk, min((p + 1) * chunk, vec)) of head h.
template <bool kBf16>
__global__ __launch_bounds__(kNmseThreads) void nmse_part_kernel(const uint4* __restrict__ ref,
                                                                const uint4* __restrict__ test,
                                                                double2* __restrict__ part,
                                                                int64_t vec_per_head,
                                                                int64_t chunk) {
  __shared__ double red[2][kNmseThreads / 64];
  const int h = blockIdx.x / kNmseParts;
  const int p = blockIdx.x - h * kNmseParts;
  const int64_t lo = (int64_t)p * chunk;
  const int64_t hi = min(lo + chunk, vec_per_head);
  const uint4* r = ref + (int64_t)h * vec_per_head;
  const uint4* t = test + (int64_t)h * vec_per_head;
  double num = 0.0, den = 0.0;
  int64_t e = lo + threadIdx.x;
  for (; e + (kNmseUnroll - 1) * kNmseThreads < hi; e += kNmseUnroll * kNmseThreads) {
    uint4 a[kNmseUnroll], b[kNmseUnroll];
#pragma unroll
    for (int u = 0; u < kNmseUnroll; ++u) {
      a[u] = r[e + u * kNmseThreads];
      b[u] = t[e + u * kNmseThreads];
    }
#pragma unroll
    for (int u = 0; u < kNmseUnroll; ++u) add_vec<kBf16>(a[u], b[u], num, den);
  }
  for (; e < hi; e += kNmseThreads) add_vec<kBf16>(r[e], t[e], num, den);
#pragma unroll
  for (int m = 32; m >= 1; m >>= 1) {
    num += __shfl_xor(num, m);
    den += __shfl_xor(den, m);
  }
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  if (lane == 0) {
    red[0][wave] = num;
    red[1][wave] = den;
  }
  __syncthreads();
  if (threadIdx.x == 0) {
    double sn = 0.0, sd = 0.0;
#pragma unroll
    for (int w = 0; w < kNmseThreads / 64; ++w) {
      sn += red[0][w];
      sd += red[1][w];
    }
    part[blockIdx.x] = double2{sn, sd};
  }
}

// One wave per head: lane l adds parts l, l + 64, ...; then a butterfly.
__global__ __launch_bounds__(64) void nmse_final_kernel(const double2* __restrict__ part,
                                                        double* __restrict__ out) {
  const int h = blockIdx.x;
  double num = 0.0, den = 0.0;
  for (int p = threadIdx.x; p < kNmseParts; p += 64) {
    const double2 v = part[(int64_t)h * kNmseParts + p];
    num += v.x;
    den += v.y;
  }
#pragma unroll
  for (int m = 32; m >= 1; m >>= 1) {
    num += __shfl_xor(num, m);
    den += __shfl_xor(den, m);
  }
  if (threadIdx.x == 0) out[h] = num / den;
}

}  // namespace

hipError_t nmse_scratch(void** ptr) {
  // one resolved address per device, kept for the life of the process
  constexpr int kMaxDevices = 64;
  static std::atomic<void*> resolved[kMaxDevices];
  int dev = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return e;
  if (dev < 0 || dev >= kMaxDevices) return hipErrorInvalidDevice;
  void* p = resolved[dev].load(std::memory_order_acquire);
  if (p == nullptr) {
    e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess) return e;
    if (p == nullptr) return hipErrorInvalidSymbol;
    resolved[dev].store(p, std::memory_order_release);
  }
  *ptr = p;
  return hipSuccess;
}

hipError_t launch_nmse(int dtype, const void* ref, const void* test, void* workspace, double* out,
                       int heads, int64_t n, hipStream_t s) {
  const int64_t esz = dtype == 1 ? 2 : 4;
  const int64_t vec = n * kHeadDim * esz / 16;  // N x 64 elements per head, 16-byte vectors
  const int64_t chunk = (vec + kNmseParts - 1) / kNmseParts;
  double2* part = static_cast<double2*>(workspace);
  const dim3 grid((unsigned)(heads * kNmseParts));
  if (dtype == 1)
    hipLaunchKernelGGL(nmse_part_kernel<true>, grid, dim3(kNmseThreads), 0, s,
                       static_cast<const uint4*>(ref), static_cast<const uint4*>(test), part, vec,
                       chunk);
  else
    hipLaunchKernelGGL(nmse_part_kernel<false>, grid, dim3(kNmseThreads), 0, s,
                       static_cast<const uint4*>(ref), static_cast<const uint4*>(test), part, vec,
                       chunk);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(nmse_final_kernel, dim3((unsigned)heads), dim3(64), 0, s, part, out);
  return hipGetLastError();
}

}  // namespace saf3r
