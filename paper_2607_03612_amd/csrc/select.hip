// Kept-key-block selection per query block (Sec. 4.1 static and
// query-probe Top-K kernels, block scores from Sec. 4.3).
//
// Top-K heads: a workgroup scores R query blocks of one head against every
// key block in float64 (s = qbar . kbar / 8, the exact tile mean of the
// pre-softmax scores), keeps the R score rows in LDS as order-preserving
// 64-bit keys, then one wave per row finds the k-th largest key by bisection
// over the key range with wave-wide counts and compacts the kept indices in
// ascending order with ballots. Ties at the threshold go to the lower block
// index, so the result is unique and matches a stable sort by (score desc,
// index asc).
//
// Frame-local heads: the kept blocks of query block i are the contiguous
// range of key blocks whose tokens overlap the frames touched by block i.
#include "saf3r_internal.h"

namespace saf3r {
namespace {

constexpr int kThreads = 256;
constexpr int kWaves = kThreads / 64;

__device__ inline uint64_t order_key(double s) {
  s += 0.0;  // -0 -> +0 so that equal scores give equal keys
  const uint64_t b = (uint64_t)__double_as_longlong(s);
  return (b >> 63) ? ~b : (b | 0x8000000000000000ull);
}

__device__ inline int wave_sum(int v) {
#pragma unroll
  for (int m = 1; m < 64; m <<= 1) v += __shfl_xor(v, m);
  return v;
}
__device__ inline uint64_t wave_min(uint64_t v) {
#pragma unroll
  for (int m = 1; m < 64; m <<= 1) {
    const uint64_t o = __shfl_xor(v, m);
    v = o < v ? o : v;
  }
  return v;
}
__device__ inline uint64_t wave_max(uint64_t v) {
#pragma unroll
  for (int m = 1; m < 64; m <<= 1) {
    const uint64_t o = __shfl_xor(v, m);
    v = o > v ? o : v;
  }
  return v;
}

// Number of keys >= t in one LDS row, summed over the wave.
__device__ inline int count_ge(const uint64_t* row, int nb, uint64_t t, int lane) {
  int c = 0;
  for (int j = lane; j < nb; j += 64) c += row[j] >= t ? 1 : 0;
  return wave_sum(c);
}

template <int R>
__global__ __launch_bounds__(kThreads) void select_topk_kernel(const double* __restrict__ qp,
                                                              const double* __restrict__ kp,
                                                              int32_t* __restrict__ idx,
                                                              int32_t* __restrict__ cnt,
                                                              double* __restrict__ scores,
                                                              TopKArgs a) {
  extern __shared__ __attribute__((aligned(16))) double lds[];
  const int nb = a.nb;
  const int groups = (nb + R - 1) / R;
  const int slot = blockIdx.x / groups;
  const int i0 = (blockIdx.x - slot * groups) * R;
  const int rows = min(R, nb - i0);
  const int h = a.head[slot];
  const int k = a.topk[slot];

  double* qs = lds;                                       // [R][64]
  uint64_t* keys = reinterpret_cast<uint64_t*>(lds + R * kHeadDim);  // [R][nb]

  const double* qsrc = qp + ((int64_t)h * nb + i0) * kHeadDim;
  for (int t = threadIdx.x; t < R * kHeadDim; t += kThreads)
    qs[t] = t < rows * kHeadDim ? qsrc[t] : 0.0;
  __syncthreads();

  // ---- scores: one key block per thread, R query blocks at once
  const double* khead = kp + (int64_t)h * nb * kHeadDim;
  for (int j = threadIdx.x; j < nb; j += kThreads) {
    double acc[R];
#pragma unroll
    for (int r = 0; r < R; ++r) acc[r] = 0.0;
    const double2* krow = reinterpret_cast<const double2*>(khead + (int64_t)j * kHeadDim);
#pragma unroll 4
    for (int d2 = 0; d2 < kHeadDim / 2; ++d2) {
      const double2 kv = krow[d2];
#pragma unroll
      for (int r = 0; r < R; ++r) {
        acc[r] = fma(qs[r * kHeadDim + 2 * d2], kv.x, acc[r]);
        acc[r] = fma(qs[r * kHeadDim + 2 * d2 + 1], kv.y, acc[r]);
      }
    }
#pragma unroll
    for (int r = 0; r < R; ++r) {
      if (r < rows) {
        const double s = acc[r] * 0.125;  // 1/sqrt(64), exact
        keys[r * nb + j] = order_key(s);
        if (scores) scores[((int64_t)h * nb + i0 + r) * nb + j] = s;
      }
    }
  }
  __syncthreads();

  // ---- selection: one wave per query block
  const int lane = threadIdx.x & 63;
  const uint64_t lanemask_lt = (1ull << lane) - 1ull;
  for (int r = threadIdx.x >> 6; r < rows; r += kWaves) {
    const uint64_t* row = keys + r * nb;
    int32_t* dst = idx + ((int64_t)h * nb + i0 + r) * a.cap;

    // Threshold t and the number of keys equal to t to take (lowest j first).
    uint64_t t = 0;
    int take_equal = 0;
    if (k >= nb) {
      t = 0;  // every key is > 0 after order_key
    } else {
      uint64_t lo = ~0ull, hi = 0;
      for (int j = lane; j < nb; j += 64) {
        const uint64_t x = row[j];
        lo = x < lo ? x : lo;
        hi = x > hi ? x : hi;
      }
      lo = wave_min(lo);
      hi = wave_max(hi) + 1;  // count(>= lo) = nb >= k, count(>= hi) = 0 < k
      int c_hi = 0;
      bool exact = false;
      while (hi - lo > 1) {
        const uint64_t mid = lo + (hi - lo) / 2;
        const int c = count_ge(row, nb, mid, lane);
        if (c == k) {  // {key >= mid} is exactly the top k
          t = mid - 1;
          exact = true;
          break;
        }
        if (c > k) {
          lo = mid;
        } else {
          hi = mid;
          c_hi = c;
        }
      }
      if (!exact) {
        t = lo;  // the k-th largest key; c_hi keys are strictly larger
        take_equal = k - c_hi;
      }
    }

    int out_base = 0, eq_base = 0;
    for (int j0 = 0; j0 < nb; j0 += 64) {
      const int j = j0 + lane;
      const bool valid = j < nb;
      const uint64_t x = valid ? row[j] : 0ull;
      const bool is_eq = valid && x == t;
      const uint64_t b_eq = __ballot(is_eq);
      const int eq_before = eq_base + __popcll(b_eq & lanemask_lt);
      const bool sel = valid && (x > t || (is_eq && eq_before < take_equal));
      const uint64_t b_sel = __ballot(sel);
      const int pos = out_base + __popcll(b_sel & lanemask_lt);
      if (sel && pos < a.cap) dst[pos] = j;
      out_base += __popcll(b_sel);
      eq_base += __popcll(b_eq);
    }
    for (int p = out_base + lane; p < a.cap; p += 64) dst[p] = -1;
    if (lane == 0) cnt[(int64_t)h * nb + i0 + r] = out_base;
  }
}

// One wave per (head, query block) of the non-Top-K heads.
__global__ __launch_bounds__(kThreads) void select_static_kernel(int32_t* __restrict__ idx,
                                                                int32_t* __restrict__ cnt,
                                                                StaticArgs a) {
  const int lane = threadIdx.x & 63;
  const int64_t wave = (int64_t)blockIdx.x * kWaves + (threadIdx.x >> 6);
  if (wave >= (int64_t)a.n_heads * a.nb) return;
  const int slot = (int)(wave / a.nb);
  const int i = (int)(wave - (int64_t)slot * a.nb);
  const int h = a.head[slot];
  const int64_t row = (int64_t)h * a.nb + i;
  if (a.pattern[slot] == kDense) {
    if (lane == 0) cnt[row] = a.nb;
    return;
  }
  const int64_t T = a.tokens_per_frame;
  const int64_t first = (int64_t)i * kBlock;
  const int64_t last = min(first + kBlock, a.n) - 1;
  const int64_t tok_lo = (first / T) * T;
  const int64_t tok_hi = min((last / T + 1) * T, a.n) - 1;
  const int j_lo = (int)(tok_lo / kBlock);
  const int len = (int)(tok_hi / kBlock) - j_lo + 1;
  int32_t* dst = idx + row * a.cap;
  for (int p = lane; p < a.cap; p += 64) dst[p] = p < len ? j_lo + p : -1;
  if (lane == 0) cnt[row] = len;
}

template <int R>
hipError_t launch_topk_r(const double* qp, const double* kp, int32_t* idx, int32_t* cnt,
                         double* scores, const TopKArgs& a, size_t lds, hipStream_t s) {
  auto kern = select_topk_kernel<R>;
  hipError_t e = hipFuncSetAttribute(reinterpret_cast<const void*>(kern),
                                     hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
  if (e != hipSuccess) return e;
  const int groups = (a.nb + R - 1) / R;
  hipLaunchKernelGGL(kern, dim3((unsigned)(groups * a.n_heads)), dim3(kThreads), lds, s, qp, kp,
                     idx, cnt, scores, a);
  return hipGetLastError();
}

}  // namespace

size_t topk_lds_bytes(int rows, int nb) {
  return (size_t)rows * (kHeadDim + nb) * sizeof(double);
}

hipError_t launch_select_topk(const double* qp, const double* kp, int32_t* idx, int32_t* cnt,
                              double* scores, const TopKArgs& a, size_t lds, hipStream_t s) {
  if (a.n_heads == 0) return hipSuccess;
  switch (a.rows_per_group) {
    case 8: return launch_topk_r<8>(qp, kp, idx, cnt, scores, a, lds, s);
    case 4: return launch_topk_r<4>(qp, kp, idx, cnt, scores, a, lds, s);
    case 2: return launch_topk_r<2>(qp, kp, idx, cnt, scores, a, lds, s);
    case 1: return launch_topk_r<1>(qp, kp, idx, cnt, scores, a, lds, s);
    default: return hipErrorInvalidValue;
  }
}

hipError_t launch_select_static(int32_t* idx, int32_t* cnt, const StaticArgs& a, hipStream_t s) {
  const int64_t waves = (int64_t)a.n_heads * a.nb;
  if (waves == 0) return hipSuccess;
  hipLaunchKernelGGL(select_static_kernel, dim3((unsigned)((waves + kWaves - 1) / kWaves)),
                     dim3(kThreads), 0, s, idx, cnt, a);
  return hipGetLastError();
}

}  // namespace saf3r
