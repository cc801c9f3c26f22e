// Kept-key-block selection per query block (Sec. 4.1 static and
// query-probe Top-K kernels, block scores from Sec. 4.3).
//
// Top-K heads. A workgroup scores R <= 16 query blocks of one head against
// every key block in float64 (s = qbar . kbar / 8, the exact tile mean of the
// pre-softmax scores) on the fp64 matrix cores: 16x16 score tiles from
// v_mfma_f64_16x16x4f64 with the pooled queries held in registers as the A
// operand and the dimension-major pooled keys as coalesced B columns. Scores
// become order-preserving 64-bit keys; LDS keeps only their high 32 bits.
// One wave per query block then:
//   1. loads its row of high keys into registers and finds, by bisection
//      with wave-wide counts, the k-th largest high key T;
//   2. if more keys share T than are still needed, recomputes the score
//      tiles of that bucket with the same instruction sequence (so the fp64
//      values are bit-identical) and bisects their low 32 bits the same way
//      (the low halves overwrite the bucket's LDS slots; a per-lane bitmask
//      remembers the bucket, whose high half is T);
//   3. compacts the kept indices in ascending order with ballots; keys equal
//      in all 64 bits go to the lower block index.
// The result equals a stable sort by (score desc, index asc), first k.
//
// Frame-local heads: the kept blocks of query block i are the contiguous
// range of key blocks whose tokens overlap the frames touched by block i.
#include "saf3r_internal.h"

namespace saf3r {
namespace {

constexpr int kStaticThreads = 256;

__device__ inline uint64_t order_key(double s) {
  s += 0.0;  // -0 -> +0 so that equal scores give equal keys
  const uint64_t b = (uint64_t)__double_as_longlong(s);
  return (b >> 63) ? ~b : (b | 0x8000000000000000ull);
}

__device__ inline uint32_t wave_min_u32(uint32_t v) {
#pragma unroll
  for (int m = 1; m < 64; m <<= 1) v = min(v, (uint32_t)__shfl_xor((int)v, m));
  return v;
}
__device__ inline uint32_t wave_max_u32(uint32_t v) {
#pragma unroll
  for (int m = 1; m < 64; m <<= 1) v = max(v, (uint32_t)__shfl_xor((int)v, m));
  return v;
}

typedef double f64x4 __attribute__((ext_vector_type(4)));

// A operand of the score tiles: pooled query rows i0 + lane%16, dimensions
// 4s + lane/16 for s = 0..15 (rows past the head's blocks are zero).
struct QOperand {
  double a[16];
};

__device__ inline QOperand load_q_operand(const double* qp_head, int i0, int nb, int lane) {
  QOperand q;
  const int row = i0 + (lane & 15);
#pragma unroll
  for (int s = 0; s < 16; ++s)
    q.a[s] = row < nb ? qp_head[(int64_t)row * kHeadDim + 4 * s + (lane >> 4)] : 0.0;
  return q;
}

// 16x16 tile of raw scores (before the 1/8): element e of a lane is row
// i0 + lane/16 + 4e (the fp64 MFMA output order), key block 16c + lane%16. Always this instruction sequence, so a tile is
// bit-identical whenever it is recomputed.
// Columns past the last key block read a clamped (valid) address and are
// never stored, so every load is unconditional.
struct KColumn {
  double b[16];
};
__device__ inline KColumn load_k_column(const double* kT, int nb, int c, int lane) {
  const int j = min(16 * c + (lane & 15), nb - 1);
  const double* col = kT + (int64_t)(lane >> 4) * nb + j;
  KColumn k;
#pragma unroll
  for (int s = 0; s < 16; ++s) k.b[s] = col[(int64_t)(4 * s) * nb];
  return k;
}
// 16x16 tile of raw scores (before the 1/8): element e of a lane is row
// i0 + lane/16 + 4e (the fp64 MFMA output order), key block 16c + lane%16.
// Two accumulation chains (even and odd dimension groups) summed at the end;
// always this instruction sequence, so a recomputed tile is bit-identical.
__device__ inline f64x4 score_tile(const QOperand& q, const KColumn& k) {
  f64x4 a0 = {0.0, 0.0, 0.0, 0.0}, a1 = {0.0, 0.0, 0.0, 0.0};
#pragma unroll
  for (int s = 0; s < 16; s += 2) {
    a0 = __builtin_amdgcn_mfma_f64_16x16x4f64(q.a[s], k.b[s], a0, 0, 0, 0);
    a1 = __builtin_amdgcn_mfma_f64_16x16x4f64(q.a[s + 1], k.b[s + 1], a1, 0, 0, 0);
  }
  return a0 + a1;
}

// Row of high keys of one query block, j = 64e + lane: in registers for the
// bisection counts when it has at most MAXK chunks of 64 (MAXK > 0), else
// counted straight from LDS. Slots past the last block hold 0, below every
// valid key.
template <int MAXK>
struct RowKeys {
  uint32_t r[MAXK > 0 ? MAXK : 1];
  const uint32_t* lds;
  int chunks, lane;

  __device__ inline void init(const uint32_t* row, int nb, int lane_) {
    lds = row;
    lane = lane_;
    chunks = (nb + 63) / 64;
    if constexpr (MAXK > 0) {
#pragma unroll
      for (int e = 0; e < MAXK; ++e) {
        const int j = 64 * e + lane;
        r[e] = j < nb ? row[j] : 0u;
      }
    }
  }
  // f(e, key) for every chunk e < chunks, from the registers (unrolled) or
  // from LDS
  template <typename F>
  __device__ inline void each(F&& f, int nb) const {
    if constexpr (MAXK > 0) {
#pragma unroll
      for (int e = 0; e < MAXK; ++e)
        if (e < chunks) f(e, r[e]);
    } else {
      for (int e = 0; e < chunks; ++e) {
        const int j = 64 * e + lane;
        f(e, j < nb ? lds[j] : 0u);
      }
    }
  }
  // number of keys >= t (t >= 1), wave-wide: one compare per chunk into a
  // lane mask, popcounts summed on the scalar unit
  __device__ inline int count_ge(uint32_t t, int nb) const {
    int c = 0;
    if constexpr (MAXK > 0) {
#pragma unroll
      for (int e = 0; e < MAXK; ++e) c += __popcll(__ballot(r[e] >= t));
    } else {
      for (int e = 0; e < chunks; ++e) {
        const int j = 64 * e + lane;
        c += __popcll(__ballot(j < nb && lds[j] >= t));
      }
    }
    return c;
  }
};

// k-th largest of the wave's 32-bit values (only lanes/elements passing
// `valid` count). Returns T and sets *gt = number of values > T, or returns
// with *exact set when {values >= T} has exactly k members.
template <typename CountGe>
__device__ inline uint32_t kth_largest(uint32_t lo, uint32_t hi_incl, int k, CountGe count_ge,
                                       int* gt, bool* exact) {
  uint64_t lo64 = lo, hi64 = (uint64_t)hi_incl + 1;  // count(>= lo) >= k, count(>= hi) < k
  int c_hi = 0;
  *exact = false;
  while (hi64 - lo64 > 1) {
    const uint64_t mid = lo64 + (hi64 - lo64) / 2;
    const int c = count_ge((uint32_t)mid);
    if (c == k) {
      *exact = true;
      *gt = c;
      return (uint32_t)mid;
    }
    if (c > k) {
      lo64 = mid;
    } else {
      hi64 = mid;
      c_hi = c;
    }
  }
  *gt = c_hi;
  return (uint32_t)lo64;
}

template <int R, int THREADS, int MAXK>
__global__ __launch_bounds__(THREADS) void select_topk_kernel(const double* __restrict__ qp,
                                                             const double* __restrict__ kpT,
                                                             int32_t* __restrict__ idx,
                                                             int32_t* __restrict__ cnt,
                                                             double* __restrict__ scores,
                                                             TopKArgs a) {
  extern __shared__ __attribute__((aligned(16))) double lds[];
  constexpr int kWaves = THREADS / 64;
  const int nb = a.nb;
  const int groups = (nb + R - 1) / R;
  const int slot = blockIdx.x / groups;
  const int i0 = (blockIdx.x - slot * groups) * R;
  const int rows = min(R, nb - i0);
  const int h = a.head[slot];
  const int k = a.topk[slot];

  uint32_t* keys = reinterpret_cast<uint32_t*>(lds);  // [R][nb] high halves

  // ---- scores: 16x16 fp64 MFMA tiles, one chunk of 16 key blocks per step
  const int lane = threadIdx.x & 63;
  const int wave = threadIdx.x >> 6;
  const double* kT = kpT + (int64_t)h * kHeadDim * nb;
  const double* qp_head = qp + (int64_t)h * nb * kHeadDim;
  const int chunks16 = (nb + 15) / 16;
  {
    const QOperand qa = load_q_operand(qp_head, i0, nb, lane);
    KColumn next = load_k_column(kT, nb, min(wave, chunks16 - 1), lane);
    for (int c = wave; c < chunks16; c += kWaves) {
      const KColumn cur = next;
      next = load_k_column(kT, nb, min(c + kWaves, chunks16 - 1), lane);  // prefetch
      const f64x4 t = score_tile(qa, cur);
      const int j = 16 * c + (lane & 15);
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        const int r = (lane >> 4) + 4 * e;
        if (r < rows && j < nb) {
          const double s = t[e] * 0.125;  // 1/sqrt(64), exact
          keys[r * nb + j] = (uint32_t)(order_key(s) >> 32);
          if (scores) scores[((int64_t)h * nb + i0 + r) * nb + j] = s;
        }
      }
    }
  }
  __syncthreads();

  // ---- selection: one wave per query block
  const uint64_t lanemask_lt = (1ull << lane) - 1ull;
  constexpr int kMaskWords = MAXK > 0 ? 1 : 4;  // chunks <= 48, or <= 256 (nb <= 16384)
  for (int r = wave; r < rows; r += kWaves) {
    uint32_t* lrow = keys + r * nb;
    int32_t* dst = idx + ((int64_t)h * nb + i0 + r) * a.cap;
    RowKeys<MAXK> row;
    row.init(lrow, nb, lane);
    const int chunks = row.chunks;

    // stage 1: T = k-th largest high key. Kept: hi > T, plus `need` of the
    // hi == T bucket (all of it, or the best by stage 2)
    uint32_t T = 1;
    bool take_ge = true;  // exact split: keep every hi >= T
    int need = 0;
    bool stage2 = false;
    uint32_t T2 = 0;
    int need2 = 0;
    uint64_t memb[kMaskWords];  // bit e of word e/64: slot (e, lane) is in the bucket
#pragma unroll
    for (int w = 0; w < kMaskWords; ++w) memb[w] = 0;
    if (k < nb) {
      uint32_t mn = 0xffffffffu, mx = 0u;
      row.each([&](int, uint32_t x) {
        if (x != 0u) {  // 0 marks a slot past the last block
          mn = min(mn, x);
          mx = max(mx, x);
        }
      }, nb);
      mn = wave_min_u32(mn);
      mx = wave_max_u32(mx);
      int gt;
      bool exact;
      T = kth_largest(mn, mx, k, [&](uint32_t t) { return row.count_ge(t, nb); }, &gt, &exact);
      if (!exact) {
        take_ge = false;
        need = k - gt;
        int bucket = 0;
        row.each([&](int e, uint32_t x) {
          const bool m = x == T;
          if (m) memb[e >> 6] |= 1ull << (e & 63);
          bucket += __popcll(__ballot(m));
        }, nb);
        if (bucket > need) {
          // stage 2: exact low halves of the bucket members from their
          // recomputed score tiles, written over the members' LDS slots
          stage2 = true;
          const QOperand qa = load_q_operand(qp_head, i0, nb, lane);
          uint32_t lmn = 0xffffffffu, lmx = 0u;
          for (int e = 0; e < chunks; ++e) {
            uint64_t members = __ballot((memb[e >> 6] >> (e & 63)) & 1);
            while (members) {
              const int b = __ffsll((unsigned long long)members) - 1;
              members &= members - 1;
              const int j = 64 * e + b;
              const f64x4 t = score_tile(qa, load_k_column(kT, nb, j >> 4, lane));
              const double v = __shfl(t[r >> 2], (j & 15) + 16 * (r & 3));
              const uint32_t lo = (uint32_t)order_key(v * 0.125);
              if (lane == 0) lrow[j] = lo;
              lmn = min(lmn, lo);
              lmx = max(lmx, lo);
            }
          }
          auto count_lo = [&](uint32_t t) {
            int c = 0;
            for (int e = 0; e < chunks; ++e) {
              const bool m = (memb[e >> 6] >> (e & 63)) & 1;
              c += __popcll(__ballot(m && lrow[64 * e + lane] >= t));
            }
            return c;
          };
          int gt2;
          bool exact2;
          T2 = kth_largest(lmn, lmx, need, count_lo, &gt2, &exact2);
          need2 = exact2 ? 0 : need - gt2;
          if (exact2) T2 = T2 - 1;  // members with lo > T2 are exactly the ones needed
        }
      }
    }

    int out_base = 0, eq_base = 0;
    const int take = stage2 ? need2 : need;
    // slots past the last block hold key 0 < T and are never selected
    row.each([&](int e, uint32_t key_hi) {
      const int j = 64 * e + lane;
      const bool member = (memb[e >> 6] >> (e & 63)) & 1;
      const uint32_t x = member ? T : key_hi;
      bool sel, is_eq;
      if (take_ge) {
        sel = x >= T;
        is_eq = false;
      } else if (!stage2) {
        is_eq = member;
        sel = x > T;
      } else {
        const uint32_t lo = member ? lrow[j] : 0u;
        is_eq = member && lo == T2;
        sel = x > T || (member && lo > T2);
      }
      const uint64_t b_eq = __ballot(is_eq);
      const int eq_before = eq_base + __popcll(b_eq & lanemask_lt);
      sel = sel || (is_eq && eq_before < take);
      const uint64_t b_sel = __ballot(sel);
      const int pos = out_base + __popcll(b_sel & lanemask_lt);
      if (sel && pos < a.cap) dst[pos] = j;
      out_base += __popcll(b_sel);
      eq_base += __popcll(b_eq);
    }, nb);
    for (int p = out_base + lane; p < a.cap; p += 64) dst[p] = -1;
    if (lane == 0) cnt[(int64_t)h * nb + i0 + r] = out_base;
  }
}

// One wave per (head, query block) of the non-Top-K heads.
__global__ __launch_bounds__(kStaticThreads) void select_static_kernel(int32_t* __restrict__ idx,
                                                                      int32_t* __restrict__ cnt,
                                                                      StaticArgs a) {
  constexpr int kWaves = kStaticThreads / 64;
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

template <int R, int THREADS, int MAXK>
hipError_t launch_topk(const double* qp, const double* kpT, int32_t* idx, int32_t* cnt,
                       double* scores, const TopKArgs& a, size_t lds, hipStream_t s) {
  auto kern = select_topk_kernel<R, THREADS, MAXK>;
  hipError_t e = hipFuncSetAttribute(reinterpret_cast<const void*>(kern),
                                     hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
  if (e != hipSuccess) return e;
  const int groups = (a.nb + R - 1) / R;
  hipLaunchKernelGGL(kern, dim3((unsigned)(groups * a.n_heads)), dim3(THREADS), lds, s, qp, kpT,
                     idx, cnt, scores, a);
  return hipGetLastError();
}

template <int R, int THREADS>
hipError_t launch_topk_rows(const double* qp, const double* kpT, int32_t* idx, int32_t* cnt,
                            double* scores, const TopKArgs& a, size_t lds, hipStream_t s) {
  const int chunks = (a.nb + 63) / 64;
  if (chunks <= 4) return launch_topk<R, THREADS, 4>(qp, kpT, idx, cnt, scores, a, lds, s);
  if (chunks <= 16) return launch_topk<R, THREADS, 16>(qp, kpT, idx, cnt, scores, a, lds, s);
  if (chunks <= 48) return launch_topk<R, THREADS, 48>(qp, kpT, idx, cnt, scores, a, lds, s);
  return launch_topk<R, THREADS, 0>(qp, kpT, idx, cnt, scores, a, lds, s);
}

}  // namespace

size_t topk_lds_bytes(int rows, int nb) { return (size_t)rows * nb * sizeof(uint32_t); }

int topk_threads(int rows) { return rows >= 16 ? 512 : 256; }

hipError_t launch_select_topk(const double* qp, const double* kpT, int32_t* idx, int32_t* cnt,
                              double* scores, const TopKArgs& a, size_t lds, hipStream_t s) {
  if (a.n_heads == 0) return hipSuccess;
  switch (a.rows_per_group) {
    case 16: return launch_topk_rows<16, 512>(qp, kpT, idx, cnt, scores, a, lds, s);
    case 8: return launch_topk_rows<8, 256>(qp, kpT, idx, cnt, scores, a, lds, s);
    case 4: return launch_topk_rows<4, 256>(qp, kpT, idx, cnt, scores, a, lds, s);
    case 2: return launch_topk_rows<2, 256>(qp, kpT, idx, cnt, scores, a, lds, s);
    case 1: return launch_topk_rows<1, 256>(qp, kpT, idx, cnt, scores, a, lds, s);
    default: return hipErrorInvalidValue;
  }
}

hipError_t launch_select_static(int32_t* idx, int32_t* cnt, const StaticArgs& a, hipStream_t s) {
  const int64_t waves = (int64_t)a.n_heads * a.nb;
  if (waves == 0) return hipSuccess;
  constexpr int kWaves = kStaticThreads / 64;
  hipLaunchKernelGGL(select_static_kernel, dim3((unsigned)((waves + kWaves - 1) / kWaves)),
                     dim3(kStaticThreads), 0, s, idx, cnt, a);
  return hipGetLastError();
}

}  // namespace saf3r
