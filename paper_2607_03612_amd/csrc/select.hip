// Kept-key-block selection per query block (Sec. 4.1 static and
// query-probe Top-K kernels, block scores from Sec. 4.3).
//
// Top-K heads. A workgroup scores R <= 16 query blocks of one head against
// every key block in float64 (s = qbar . kbar / 8, the exact tile mean of the
// pre-softmax scores) on the fp64 matrix cores: 16x16 score tiles from
// v_mfma_f64_16x16x4f64 with the pooled queries held in registers as the A
// operand and the dimension-major pooled keys as coalesced B columns. Scores
// become order-preserving 64-bit keys; LDS keeps only their high 32 bits.
// One wave per query block then, with its row of high keys in registers (lane
// l holds blocks [l*C, l*C + C), C = ceil(nb / 64) rounded up to a multiple
// of 4, read as 16-byte LDS words):
//   1. brackets the k-th largest high key between two pivots read off a
//      stratified sample (one key per lane), checks the bracket with one
//      counting pass and, once it holds at most 512 keys, packs those into
//      LDS; bisection over the packed keys with wave-wide counts (per-lane
//      VALU counts summed by a DPP scan) then finds the k-th largest high
//      key T, or stops early at a threshold kept by exactly k keys;
//   2. if more keys share T than are still needed, recomputes the score
//      tiles of that bucket with the same instruction sequence (so the fp64
//      values are bit-identical) and bisects their low 32 bits the same way
//      (the low halves overwrite the bucket's LDS slots; a per-lane bitmask
//      remembers the bucket, whose high half is T);
//   3. writes the kept indices in ascending order: a wave prefix sum of the
//      per-lane kept counts gives each lane its output offset; keys equal in
//      all 64 bits go to the lower block index.
// The result equals a stable sort by (score desc, index asc), first k.
//
// Frame-local heads: the kept blocks of query block i are the contiguous
// range of key blocks whose tokens overlap the frames touched by block i.
// Anchor heads: the contiguous range of key blocks of the anchor frame.
//
// Global-probe heads (the query probe of Sec. 4.3 as stated: one probe, the
// mean of all N queries, per head): one workgroup per head forms the probe
// from the pooled queries (sum of n_b * qbar_b over the blocks, over N),
// scores every key block in float64, finds the k-th largest order key exactly
// by an 8-bit-digit radix select over the 64-bit keys, writes the kept
// blocks ascending (keys equal to the k-th go to the lowest indices), and a
// second launch copies that list to every query block.
#include <algorithm>

#include "saf3r_internal.h"

namespace saf3r {
namespace {

constexpr int kStaticThreads = 256;

__device__ inline uint64_t order_key(double s) {
  s += 0.0;  // -0 -> +0 so that equal scores give equal keys
  const uint64_t b = (uint64_t)__double_as_longlong(s);
  return (b >> 63) ? ~b : (b | 0x8000000000000000ull);
}

// Lanes of one wave exchange values through LDS. The hardware runs a wave's
// LDS instructions in order; this keeps the compiler from moving an LDS access
// across the hand-over (it only sees each lane's own accesses).
__device__ inline void wave_lds_handover() { asm volatile("" ::: "memory"); }

// Inclusive prefix sum over the 64 lanes: shifts within rows of 16 lanes,
// then the broadcasts of lane 15 into rows 1 and 3 and of lane 31 into rows 2
// and 3 (DPP row_shr, row_bcast:15, row_bcast:31).
__device__ inline uint32_t wave_scan_incl(uint32_t v) {
  v += (uint32_t)__builtin_amdgcn_update_dpp(0, (int)v, 0x111, 0xf, 0xf, true);
  v += (uint32_t)__builtin_amdgcn_update_dpp(0, (int)v, 0x112, 0xf, 0xf, true);
  v += (uint32_t)__builtin_amdgcn_update_dpp(0, (int)v, 0x114, 0xf, 0xf, true);
  v += (uint32_t)__builtin_amdgcn_update_dpp(0, (int)v, 0x118, 0xf, 0xf, true);
  v += (uint32_t)__builtin_amdgcn_update_dpp(0, (int)v, 0x142, 0xa, 0xf, false);
  v += (uint32_t)__builtin_amdgcn_update_dpp(0, (int)v, 0x143, 0xc, 0xf, false);
  return v;
}
__device__ inline uint32_t wave_total(uint32_t v) {
  return (uint32_t)__builtin_amdgcn_readlane((int)wave_scan_incl(v), 63);
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

// Row of high keys of one query block; lane l owns blocks l*C + e, e < C,
// with C = ceil(nb / 64) rounded up to a multiple of 4 so that a lane's
// chunk is whole 16-byte LDS words. Held in registers when C <= MAXK
// (MAXK > 0), else read from LDS on every pass. Slots past the last block
// hold 0, below every valid key.
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));


template <int MAXK>
struct RowKeys {
  uint32_t r[MAXK > 0 ? MAXK : 1];
  const uint32_t* lds;
  int C, base, nb;

  __device__ inline void init(const uint32_t* row, int nb_, int lane) {
    lds = row;
    nb = nb_;
    C = row_chunk(nb);
    base = lane * C;
    if constexpr (MAXK > 0) {
      static_assert(MAXK % 4 == 0, "slots are read four at a time");
#pragma unroll
      for (int e = 0; e < MAXK; ++e) r[e] = 0u;
      // the lane's chunk as 16-byte LDS reads (rows are 64*C words long)
      const u32x4* src = reinterpret_cast<const u32x4*>(row + base);
#pragma unroll
      for (int q = 0; q < MAXK / 4; ++q) {
        if (4 * q < C) {
          const u32x4 x = src[q];
#pragma unroll
          for (int t = 0; t < 4; ++t) r[4 * q + t] = base + 4 * q + t < nb ? x[t] : 0u;
        }
      }
    }
  }
  // g(e) for every slot e < C, in groups of 8 behind one uniform branch
  template <typename G>
  __device__ inline void each_slot(G&& g) const {
#pragma unroll
    for (int e0 = 0; e0 < MAXK; e0 += 8) {
      if (e0 < C) {
#pragma unroll
        for (int e = e0; e < e0 + 8 && e < MAXK; ++e) g(e);
      }
    }
  }
  // f(e, key) for every slot (padding slots included, with key 0)
  template <typename F>
  __device__ inline void each(F&& f) const {
    if constexpr (MAXK > 0) {
      each_slot([&](int e) { f(e, r[e]); });
    } else {
      for (int e = 0; e < C; ++e) {
        const int j = base + e;
        f(e, j < nb ? lds[j] : 0u);
      }
    }
  }
  // this lane's keys >= t (t >= 1)
  __device__ inline uint32_t lane_count_ge(uint32_t t) const {
    uint32_t c = 0;
    each([&](int, uint32_t x) { c += x >= t ? 1u : 0u; });
    return c;
  }
};

// k-th largest of the wave's 32-bit values by bisection over [lo, hi_incl]
// (count_ge(lo) >= k). Returns T and sets *gt = number of values > T, or
// returns with *exact set when {values >= T} has exactly k members.
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


// Candidates packed per wave once the bracket holds at most this many keys
// (8 per lane), and the pivots' distance from the target sample rank.
constexpr int kPackedKeys = 512;
constexpr int kPivotSlack = 4;

// The kept blocks of one query block (row r of the 16-row group at i0) from
// its high keys in `row`. `lrow` is LDS scratch of 64 * row_chunk(nb)
// words, free to overwrite (the keys are in registers, or for MAXK = 0 are
// the row itself, whose bucket slots stage 2 overwrites with low halves).
// Writes the ascending list to dst[0, cap) (padded with -1) and the count to
// *cnt_row.
template <int MAXK>
__device__ inline void select_row(RowKeys<MAXK>& row, uint32_t* lrow, int32_t* dst,
                                  int32_t* cnt_row, const double* qp_head, const double* kT,
                                  int i0, int r, int k, int nb, int cap, int lane) {
  constexpr int kMaskWords = MAXK > 0 ? (MAXK + 63) / 64 : 4;  // C <= MAXK, or <= 256 (nb <= 16384)
  const int C = row.C;

  // Kept: hi > T, plus `need` of the hi == T bucket (the best by stage 2),
  // or every hi >= T when a threshold splits off exactly k keys.
  uint32_t T = 1;
  bool take_ge = true;
  int need = 0;
  uint32_t T2 = 0;
  int need2 = 0;
  uint64_t memb[kMaskWords];  // bit e of word e/64: slot e of this lane is in the bucket
#pragma unroll
  for (int w = 0; w < kMaskWords; ++w) memb[w] = 0;
  if (k < nb) {
    // bracket: count(>= lo) > k > count(>= hi); thresholds are 33-bit so
    // that hi = 2^32 (counted by nobody) fits
    uint64_t lo = 1, hi = 1ull << 32;
    int c_lo = nb, c_hi = 0;
    bool exact = false;
    if constexpr (MAXK > 8) {
      if (C >= 8) {
        // pivots from the sample of keys l*C (made distinct by the lane
        // in the low 6 bits): ranks about kPivotSlack samples on either
        // side of the expected rank k*64/nb of the k-th key
        const uint32_t xs = (row.r[0] & 0xffffffc0u) | (uint32_t)lane;
        wave_lds_handover();
        lrow[lane] = xs;  // the row is in registers; its LDS is scratch now
        wave_lds_handover();
        int g = 0;
#pragma unroll
        for (int s2 = 0; s2 < 64; ++s2) g += lrow[s2] > xs ? 1 : 0;
        const int64_t k64 = (int64_t)k * 64;
        const int rank_hi = k64 >= (int64_t)kPivotSlack * nb
                                ? (int)((k64 - (int64_t)kPivotSlack * nb) / nb) : -1;
        const int rank_lo = (int)((k64 + (int64_t)kPivotSlack * nb + nb - 1) / nb);
        uint64_t p_lo = 1, p_hi = 1ull << 32;
        if (rank_hi >= 0)
          p_hi = (uint64_t)(uint32_t)__builtin_amdgcn_readlane(
                     (int)xs, __builtin_ctzll(__ballot(g == rank_hi))) + 1;
        if (rank_lo <= 63)
          p_lo = max((uint32_t)__builtin_amdgcn_readlane(
                         (int)xs, __builtin_ctzll(__ballot(g == rank_lo))) & 0xffffffc0u, 1u);
        // one pass counts both pivots (count(>= p_lo) in the low half)
        const bool hi_inf = p_hi >> 32;
        const uint32_t t_lo = (uint32_t)p_lo, t_hi = (uint32_t)p_hi;
        uint32_t pc = 0;
        row.each([&](int, uint32_t x) {
          pc += (x >= t_lo ? 1u : 0u) + (!hi_inf && x >= t_hi ? 0x10000u : 0u);
        });
        const uint32_t tot = wave_total(pc);
        const int cl = (int)(tot & 0xffffu), ch = (int)(tot >> 16);
        if (cl == k) {
          exact = true;
          T = t_lo;
        } else if (!hi_inf && ch == k) {
          exact = true;
          T = t_hi;
        } else {
          if (ch > k) {
            lo = p_hi;
            c_lo = ch;
          } else if (cl > k) {
            lo = p_lo;
            c_lo = cl;
          }
          if (cl < k) {
            hi = p_lo;
            c_hi = cl;
          } else if (ch < k) {
            hi = p_hi;
            c_hi = ch;
          }
        }
      }
    }
    bool packed = false;
    int c_above = 0;  // keys at or above the packed bracket's top
    uint32_t pk[kPackedKeys / 64];
#pragma unroll
    for (int q = 0; q < kPackedKeys / 64; ++q) pk[q] = 0u;
    while (!exact && hi - lo > 1) {
      if constexpr (MAXK > 8) {
        // pack the bracket's keys into LDS slots [0, c_lo - c_hi); keys
        // outside it go to a per-lane dummy slot at the row's end
        if (!packed && C >= 10 && c_lo - c_hi <= kPackedKeys) {
          const uint32_t lo32 = (uint32_t)lo, span = (uint32_t)(hi - lo - 1);
          uint32_t n = 0;
          row.each([&](int, uint32_t x) { n += x - lo32 <= span ? 1u : 0u; });
          uint32_t pos = wave_scan_incl(n) - n;
          const uint32_t dummy = (uint32_t)(nb - 64 + lane);
          wave_lds_handover();
          row.each([&](int, uint32_t x) {
            const bool in = x - lo32 <= span;
            lrow[in ? pos : dummy] = x;
            pos += in ? 1u : 0u;
          });
          wave_lds_handover();
          const int ncand = c_lo - c_hi;
#pragma unroll
          for (int q = 0; q < kPackedKeys / 64; ++q)
            pk[q] = 64 * q + lane < ncand ? lrow[64 * q + lane] : 0u;
          c_above = c_hi;
          packed = true;
        }
      }
      const uint64_t mid = lo + (hi - lo) / 2;
      const uint32_t t = (uint32_t)mid;
      int c;
      if (packed) {
        uint32_t n = 0;
#pragma unroll
        for (int q = 0; q < kPackedKeys / 64; ++q) n += pk[q] >= t ? 1u : 0u;
        c = c_above + (int)wave_total(n);
      } else {
        c = (int)wave_total(row.lane_count_ge(t));
      }
      if (c == k) {
        exact = true;
        T = t;
      } else if (c > k) {
        lo = mid;
        c_lo = c;
      } else {
        hi = mid;
        c_hi = c;
      }
    }
    if (!exact) {
      // hi == lo + 1: the bucket of high key T holds c_lo - c_hi > need
      // keys. Stage 2: exact low halves of its members from their
      // recomputed score tiles, written over the members' LDS slots.
      take_ge = false;
      T = (uint32_t)lo;
      need = k - c_hi;
      row.each([&](int e, uint32_t x) {
        if (x == T) memb[e >> 6] |= 1ull << (e & 63);
      });
      const QOperand qa = load_q_operand(qp_head, i0, nb, lane);
      uint32_t lmn = 0xffffffffu, lmx = 0u;
      wave_lds_handover();
      for (int e = 0; e < C; ++e) {
        uint64_t members = __ballot((memb[e >> 6] >> (e & 63)) & 1);
        while (members) {
          const int b = __ffsll((unsigned long long)members) - 1;
          members &= members - 1;
          const int j = b * C + e;
          const f64x4 t = score_tile(qa, load_k_column(kT, nb, j >> 4, lane));
          const double v = __shfl(t[r >> 2], (j & 15) + 16 * (r & 3));
          const uint32_t lo_key = (uint32_t)order_key(v * 0.125);
          if (lane == 0) lrow[j] = lo_key;
          lmn = min(lmn, lo_key);
          lmx = max(lmx, lo_key);
        }
      }
      wave_lds_handover();
      auto count_lo = [&](uint32_t t) {
        uint32_t c = 0;
        for (int e = 0; e < C; ++e) {
          if ((memb[e >> 6] >> (e & 63)) & 1) c += lrow[min(row.base + e, nb - 1)] >= t ? 1u : 0u;
        }
        return (int)wave_total(c);
      };
      int gt2;
      bool exact2;
      T2 = kth_largest(lmn, lmx, need, count_lo, &gt2, &exact2);
      need2 = exact2 ? 0 : need - gt2;
      if (exact2) T2 = T2 - 1;  // members with lo > T2 are exactly the ones needed
    }
  }

  // ascending output
  if (MAXK > 0 && take_ge && k + 64 <= nb) {
    // every key >= T, k of them: each lane writes its kept indices to LDS
    // slots [0, k) from its prefix-sum offset (others to a dummy slot among
    // the row's last 64), then the list goes out coalesced
    const uint32_t n = row.lane_count_ge(T);
    uint32_t pos = wave_scan_incl(n) - n;
    const uint32_t dummy = (uint32_t)(nb - 64 + lane);
    wave_lds_handover();
    row.each([&](int e, uint32_t x) {
      const bool kept = x >= T;
      lrow[kept ? pos : dummy] = (uint32_t)(row.base + e);
      pos += kept ? 1u : 0u;
    });
    wave_lds_handover();
    for (int p = lane; p < cap; p += 64) dst[p] = p < k ? (int32_t)lrow[p] : -1;
    if (lane == 0) *cnt_row = k;
    return;
  }
  // general case: per-lane counts of keys kept outright (low half) and
  // of tie-set keys (high half), prefix-summed over the wave
  auto classify = [&](int e, uint32_t key_hi, bool* strict, bool* is_eq) {
    const bool member = (memb[e >> 6] >> (e & 63)) & 1;
    if (take_ge) {
      *strict = key_hi >= T;
      *is_eq = false;
    } else {
      const uint32_t lo_key = member ? lrow[min(row.base + e, nb - 1)] : 0u;
      *strict = (!member && key_hi > T) || (member && lo_key > T2);
      *is_eq = member && lo_key == T2;
    }
  };
  uint32_t packed_counts = 0;
  row.each([&](int e, uint32_t key_hi) {
    bool strict, is_eq;
    classify(e, key_hi, &strict, &is_eq);
    packed_counts += (strict ? 1u : 0u) + (is_eq ? 0x10000u : 0u);
  });
  const uint32_t incl = wave_scan_incl(packed_counts);
  const uint32_t excl = incl - packed_counts;
  const uint32_t total = (uint32_t)__builtin_amdgcn_readlane((int)incl, 63);
  const int take = take_ge ? 0 : need2;
  int eq_before = (int)(excl >> 16);
  int pos = (int)(excl & 0xffffu) + min(eq_before, take);
  const int out_total = (int)(total & 0xffffu) + min((int)(total >> 16), take);
  row.each([&](int e, uint32_t key_hi) {
    bool strict, is_eq;
    classify(e, key_hi, &strict, &is_eq);
    const bool sel = strict || (is_eq && eq_before < take);
    if (sel && pos < cap) dst[pos] = row.base + e;
    pos += sel ? 1 : 0;
    eq_before += is_eq ? 1 : 0;
  });
  for (int p = out_total + lane; p < cap; p += 64) dst[p] = -1;
  if (lane == 0) *cnt_row = out_total;
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

  uint32_t* keys = reinterpret_cast<uint32_t*>(lds);  // [R][ld] high halves
  const int ld = 64 * row_chunk(nb);

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
          keys[r * ld + j] = (uint32_t)(order_key(s) >> 32);
          if (scores) scores[((int64_t)h * nb + i0 + r) * nb + j] = s;
        }
      }
    }
  }
  __syncthreads();

  // ---- selection: one wave per query block
  for (int r = wave; r < rows; r += kWaves) {
    uint32_t* lrow = keys + r * ld;
    RowKeys<MAXK> row;
    row.init(lrow, nb, lane);
    select_row<MAXK>(row, lrow, idx + ((int64_t)h * nb + i0 + r) * a.cap,
                     cnt + (int64_t)h * nb + i0 + r, qp_head, kT, i0, r, k, nb, a.cap, lane);
  }
}

// Top-K heads with a workspace: the same scores and the same selection in two
// launches, so that neither phase leaves the other's units idle on a CU.
//   1. topk_score_kernel: eight waves score 16 query blocks of one head
//      (the tiles of select_topk_kernel) and store the high keys as rows of
//      64 * row_chunk(nb) words in the workspace;
//   2. topk_rows_kernel: one wave per query block loads its row of keys
//      (into registers, or into its own LDS row when C > MAXK) and runs
//      select_row; with little LDS per wave, many rows are in flight per CU.
constexpr int kScoreWaves = 8;

__global__ __launch_bounds__(kScoreWaves * 64) void topk_score_kernel(
    const double* __restrict__ qp, const double* __restrict__ kpT, uint32_t* __restrict__ keys,
    double* __restrict__ scores, TopKArgs a) {
  const int nb = a.nb;
  const int groups = (nb + 15) / 16;
  const int slot = blockIdx.x / groups;
  const int i0 = (blockIdx.x - slot * groups) * 16;
  const int rows = min(16, nb - i0);
  const int h = a.head[slot];
  const int lane = threadIdx.x & 63;
  const int wave = threadIdx.x >> 6;
  const int64_t ld = 64 * row_chunk(nb);
  const double* kT = kpT + (int64_t)h * kHeadDim * nb;
  const double* qp_head = qp + (int64_t)h * nb * kHeadDim;
  uint32_t* ws = keys + ((int64_t)slot * nb + i0) * ld;
  const int chunks16 = (nb + 15) / 16;
  const QOperand qa = load_q_operand(qp_head, i0, nb, lane);
  KColumn next = load_k_column(kT, nb, min(wave, chunks16 - 1), lane);
  for (int c = wave; c < chunks16; c += kScoreWaves) {
    const KColumn cur = next;
    next = load_k_column(kT, nb, min(c + kScoreWaves, chunks16 - 1), lane);  // prefetch
    const f64x4 t = score_tile(qa, cur);
    const int j = 16 * c + (lane & 15);
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      const int r = (lane >> 4) + 4 * e;
      if (r < rows && j < nb) {
        const double s = t[e] * 0.125;  // 1/sqrt(64), exact
        ws[r * ld + j] = (uint32_t)(order_key(s) >> 32);
        if (scores) scores[((int64_t)h * nb + i0 + r) * nb + j] = s;
      }
    }
  }
}

template <int MAXK>
__global__ __launch_bounds__(256) void topk_rows_kernel(const double* __restrict__ qp,
                                                       const double* __restrict__ kpT,
                                                       const uint32_t* __restrict__ keys,
                                                       int32_t* __restrict__ idx,
                                                       int32_t* __restrict__ cnt, TopKArgs a) {
  extern __shared__ __attribute__((aligned(16))) uint32_t srow[];  // [waves][ld]
  const int nb = a.nb;
  const int lane = threadIdx.x & 63;
  const int wl = threadIdx.x >> 6;
  const int64_t w = (int64_t)blockIdx.x * (blockDim.x >> 6) + wl;
  if (w >= (int64_t)a.n_heads * nb) return;  // whole waves; no barrier below
  const int slot = (int)(w / nb);
  const int i = (int)(w - (int64_t)slot * nb);
  const int h = a.head[slot];
  const int64_t ld = 64 * row_chunk(nb);
  uint32_t* lrow = srow + wl * ld;
  const uint32_t* grow = keys + ((int64_t)slot * nb + i) * ld;
  RowKeys<MAXK> row;
  if constexpr (MAXK > 0) {
    row.init(grow, nb, lane);
  } else {
    for (int64_t q = lane; q < ld / 4; q += 64)
      reinterpret_cast<u32x4*>(lrow)[q] = reinterpret_cast<const u32x4*>(grow)[q];
    wave_lds_handover();
    row.init(lrow, nb, lane);
  }
  select_row<MAXK>(row, lrow, idx + ((int64_t)h * nb + i) * a.cap, cnt + (int64_t)h * nb + i,
                   qp + (int64_t)h * nb * kHeadDim, kpT + (int64_t)h * kHeadDim * nb, i & ~15,
                   i & 15, a.topk[slot], nb, a.cap, lane);
}

// One wave per (head, query block) of the static-pattern heads (DENSE,
// FRAME_LOCAL, ANCHOR, STRIDE).
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
  const int pattern = a.pattern[slot];
  if (pattern == kDense) {
    if (lane == 0) cnt[row] = a.nb;
    return;
  }
  if (pattern == kStride) {  // token-level sampling: count of 64-key groups, no list
    const int64_t keys = (a.n + a.param[slot] - 1) / a.param[slot];
    if (lane == 0) cnt[row] = (int)((keys + kBlock - 1) / kBlock);
    return;
  }
  const int64_t T = a.tokens_per_frame;
  int64_t tok_lo, tok_hi;  // token range whose blocks are kept
  if (pattern == kAnchor) {
    tok_lo = (int64_t)a.param[slot] * T;
    tok_hi = min(tok_lo + T, a.n) - 1;
  } else {  // frame-local: the frames touched by block i
    const int64_t first = (int64_t)i * kBlock;
    const int64_t last = min(first + kBlock, a.n) - 1;
    tok_lo = (first / T) * T;
    tok_hi = min((last / T + 1) * T, a.n) - 1;
  }
  const int j_lo = (int)(tok_lo / kBlock);
  const int len = (int)(tok_hi / kBlock) - j_lo + 1;
  int32_t* dst = idx + row * a.cap;
  for (int p = lane; p < a.cap; p += 64) dst[p] = p < len ? j_lo + p : -1;
  if (lane == 0) cnt[row] = len;
}

// The list check: result[0] counts failing rows, result[1] keeps the lowest
// one (INT32_MAX while none fails).
__global__ __launch_bounds__(64) void validate_init_kernel(int32_t* __restrict__ result) {
  if (threadIdx.x == 0) {
    result[0] = 0;
    result[1] = 0x7fffffff;
  }
}

// One wave per (listed head, query block): the row's count lies in [0, cap]
// (and equals the class's exact count where it has one), its first count
// entries rise strictly inside [0, nb), and the rest of the row is -1. The
// wave reads only its own row, whatever the row holds.
__global__ __launch_bounds__(256) void validate_index_kernel(const int32_t* __restrict__ idx,
                                                             const int32_t* __restrict__ cnt,
                                                             int32_t* __restrict__ result,
                                                             ValidateArgs a) {
  const int lane = threadIdx.x & 63;
  const int64_t wave = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6);
  if (wave >= (int64_t)a.n_heads * a.nb) return;
  const int slot = (int)(wave / a.nb);
  const int i = (int)(wave - (int64_t)slot * a.nb);
  const int64_t row = (int64_t)a.head[slot] * a.nb + i;
  const int c = cnt[row];
  bool bad = c < 0 || c > a.cap || (a.expect[slot] >= 0 && c != a.expect[slot]);
  if (!bad) {  // c is the same in every lane
    const int32_t* list = idx + row * a.cap;
    for (int p = lane; p < a.cap; p += 64) {
      const int v = list[p];
      if (p < c) bad = bad || v < 0 || v >= a.nb || (p > 0 && list[p - 1] >= v);
      else bad = bad || v != -1;
    }
  }
  if (__ballot(bad) != 0 && lane == 0) {
    atomicAdd(&result[0], 1);
    atomicMin(&result[1], (int32_t)row);
  }
}

constexpr int kGlobalThreads = 1024;
constexpr int kGlobalWaves = kGlobalThreads / 64;

// One workgroup per global-probe head; writes row 0 of the head's lists.
__global__ __launch_bounds__(kGlobalThreads) void select_global_kernel(const double* __restrict__ qp,
                                                                      const double* __restrict__ kpT,
                                                                      int32_t* __restrict__ idx,
                                                                      int32_t* __restrict__ cnt,
                                                                      double* __restrict__ scores,
                                                                      GlobalArgs a) {
  extern __shared__ __attribute__((aligned(16))) uint64_t skeys[];  // [nb] order keys
  __shared__ double part[kGlobalWaves][kHeadDim];
  __shared__ double qbar[kHeadDim];
  __shared__ uint32_t hist[256];
  __shared__ uint32_t wave_tot[kGlobalWaves][2];
  __shared__ int sel_digit, sel_above;
  const int t = threadIdx.x, lane = t & 63, wave = t >> 6;
  const int h = a.head[blockIdx.x];
  const int k = a.topk[blockIdx.x];
  const int nb = a.nb;
  const double* qh = qp + (int64_t)h * nb * kHeadDim;
  const double* kT = kpT + (int64_t)h * kHeadDim * nb;

  // probe: mean of all queries = sum over blocks of (block size) * block mean,
  // over N. Wave w sums blocks w, w + 16, ... in two interleaved chains; the
  // partial sums are added in a fixed order.
  double acc0 = 0.0, acc1 = 0.0;
  int b = wave;
  for (; b + 7 * kGlobalWaves < nb; b += 8 * kGlobalWaves) {
    double x[8];  // eight loads in flight, then the two chains
#pragma unroll
    for (int u = 0; u < 8; ++u) x[u] = qh[(int64_t)(b + u * kGlobalWaves) * kHeadDim + lane];
#pragma unroll
    for (int u = 0; u < 8; u += 2) {
      acc0 = fma((double)kBlock, x[u], acc0);
      const int b1 = b + (u + 1) * kGlobalWaves;
      const double n1 = b1 == nb - 1 ? (double)(a.n - (int64_t)(nb - 1) * kBlock) : (double)kBlock;
      acc1 = fma(n1, x[u + 1], acc1);
    }
  }
  for (; b < nb; b += kGlobalWaves) {
    const double n0 = b == nb - 1 ? (double)(a.n - (int64_t)(nb - 1) * kBlock) : (double)kBlock;
    acc0 = fma(n0, qh[(int64_t)b * kHeadDim + lane], acc0);
  }
  part[wave][lane] = acc0 + acc1;
  __syncthreads();
  if (t < kHeadDim) {
    double sum = 0.0;
#pragma unroll
    for (int w = 0; w < kGlobalWaves; ++w) sum += part[w][t];
    qbar[t] = sum / (double)a.n;
  }
  __syncthreads();

  // scores of every key block, in float64 (four interleaved chains over the
  // dimensions, added in a fixed order), kept as order keys
  for (int j = t; j < nb; j += kGlobalThreads) {
    double s4[4] = {0.0, 0.0, 0.0, 0.0};
#pragma unroll
    for (int d = 0; d < kHeadDim; ++d) s4[d & 3] = fma(qbar[d], kT[(int64_t)d * nb + j], s4[d & 3]);
    const double sj = ((s4[0] + s4[1]) + (s4[2] + s4[3])) * 0.125;  // 1/sqrt(64), exact
    skeys[j] = order_key(sj);
    if (scores) scores[(int64_t)h * nb * nb + j] = sj;
  }
  __syncthreads();

  // k-th largest key, one 8-bit digit at a time from the top
  uint64_t prefix = 0, mask = 0;
  int remaining = k;
  for (int shift = 56; shift >= 0; shift -= 8) {
    if (t < 256) hist[t] = 0;
    __syncthreads();
    for (int j = t; j < nb; j += kGlobalThreads) {
      const uint64_t key = skeys[j];
      if ((key & mask) == prefix) atomicAdd(&hist[(key >> shift) & 255], 1u);
    }
    __syncthreads();
    // digit of the k-th key: the first d, from 255 down, at which the count
    // of keys with digit >= d reaches `remaining` (a scan over the bins in
    // descending order by the first four waves; digit 0 if none does)
    if (t < 256) {
      const uint32_t hv = hist[255 - t];
      const uint32_t incl = wave_scan_incl(hv);
      if (lane == 63) wave_tot[wave][0] = incl;
    }
    __syncthreads();
    if (t < 256) {
      const uint32_t hv = hist[255 - t];
      uint32_t incl = wave_scan_incl(hv);
      for (int w = 0; w < wave; ++w) incl += wave_tot[w][0];
      const bool reach = (int)incl >= remaining;
      const uint32_t prev = incl - hv;
      // the first lane (lowest t) that reaches; t = 255 (digit 0) always takes
      // the rest
      const bool first = (reach && (int)prev < remaining) || (t == 255 && (int)prev < remaining && !reach);
      if (first) {
        sel_digit = 255 - t;
        sel_above = (int)prev;
      }
    }
    __syncthreads();
    prefix |= (uint64_t)sel_digit << shift;
    mask |= 0xffull << shift;
    remaining -= sel_above;
    __syncthreads();
  }
  // prefix is the k-th largest key; keep keys above it and the `remaining`
  // lowest-index keys equal to it, in ascending block order
  int32_t* dst = idx + (int64_t)h * nb * a.cap;
  int out_pos = 0, eq_seen = 0;
  for (int j0 = 0; j0 < nb; j0 += kGlobalThreads) {
    const int j = j0 + t;
    const uint64_t key = j < nb ? skeys[j] : 0ull;
    const bool gt = j < nb && key > prefix;
    const bool eq = j < nb && key == prefix;
    const uint64_t below = (1ull << lane) - 1;
    const uint64_t eq_mask = __ballot(eq);
    if (lane == 0) wave_tot[wave][0] = (uint32_t)__popcll(eq_mask);
    __syncthreads();
    int eq_before = eq_seen + __popcll(eq_mask & below);
    for (int w = 0; w < wave; ++w) eq_before += (int)wave_tot[w][0];
    const bool kept = gt || (eq && eq_before < remaining);
    const uint64_t kept_mask = __ballot(kept);
    if (lane == 0) wave_tot[wave][1] = (uint32_t)__popcll(kept_mask);
    __syncthreads();
    int pos = out_pos + __popcll(kept_mask & below);
    for (int w = 0; w < wave; ++w) pos += (int)wave_tot[w][1];
    if (kept && pos < a.cap) dst[pos] = j;
    int eq_chunk = 0, kept_chunk = 0;
#pragma unroll
    for (int w = 0; w < kGlobalWaves; ++w) {
      eq_chunk += (int)wave_tot[w][0];
      kept_chunk += (int)wave_tot[w][1];
    }
    eq_seen += eq_chunk;
    out_pos += kept_chunk;
    __syncthreads();
  }
  for (int p = out_pos + t; p < a.cap; p += kGlobalThreads) dst[p] = -1;
  if (t == 0) cnt[(int64_t)h * nb] = out_pos;
}

// Copies row 0 of every global-probe head to its other query blocks: one
// wave per (head, row >= 1).
__global__ __launch_bounds__(256) void select_global_broadcast_kernel(int32_t* __restrict__ idx,
                                                                    int32_t* __restrict__ cnt,
                                                                    GlobalArgs a) {
  const int lane = threadIdx.x & 63;
  const int64_t wave = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6);
  const int64_t rows = (int64_t)a.n_heads * (a.nb - 1);
  if (wave >= rows) return;
  const int slot = (int)(wave / (a.nb - 1));
  const int i = 1 + (int)(wave - (int64_t)slot * (a.nb - 1));
  const int h = a.head[slot];
  const int32_t* src = idx + (int64_t)h * a.nb * a.cap;
  int32_t* dst = idx + ((int64_t)h * a.nb + i) * a.cap;
  for (int p = lane; p < a.cap; p += 64) dst[p] = src[p];
  if (lane == 0) cnt[(int64_t)h * a.nb + i] = cnt[(int64_t)h * a.nb];
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
  const int chunks = row_chunk(a.nb);
  if (chunks <= 4) return launch_topk<R, THREADS, 4>(qp, kpT, idx, cnt, scores, a, lds, s);
  if (chunks <= 16) return launch_topk<R, THREADS, 16>(qp, kpT, idx, cnt, scores, a, lds, s);
  if (chunks <= 48) return launch_topk<R, THREADS, 48>(qp, kpT, idx, cnt, scores, a, lds, s);
  return launch_topk<R, THREADS, 0>(qp, kpT, idx, cnt, scores, a, lds, s);
}

}  // namespace


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


hipError_t launch_select_topk_ws(const double* qp, const double* kpT, uint32_t* keys, int32_t* idx,
                                 int32_t* cnt, double* scores, const TopKArgs& a, hipStream_t s) {
  if (a.n_heads == 0) return hipSuccess;
  const int groups = (a.nb + 15) / 16;
  hipLaunchKernelGGL(topk_score_kernel, dim3((unsigned)(groups * a.n_heads)),
                     dim3(kScoreWaves * 64), 0, s, qp, kpT, keys, scores, a);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  // waves per workgroup: as many rows as fit in 64 KB of LDS, at most four
  const size_t row_bytes = topk_ws_row_bytes(a.nb);
  const int wpg = (int)std::max<size_t>(1, std::min<size_t>(4, (64 * 1024) / row_bytes));
  const size_t lds = (size_t)wpg * row_bytes;
  const int64_t waves = (int64_t)a.n_heads * a.nb;
  const dim3 grid((unsigned)((waves + wpg - 1) / wpg)), block(64 * wpg);
  auto go = [&](auto kern) -> hipError_t {
    hipError_t e2 = hipFuncSetAttribute(reinterpret_cast<const void*>(kern),
                                        hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
    if (e2 != hipSuccess) return e2;
    hipLaunchKernelGGL(kern, grid, block, lds, s, qp, kpT, keys, idx, cnt, a);
    return hipGetLastError();
  };
  const int chunks = row_chunk(a.nb);
  if (chunks <= 4) return go(topk_rows_kernel<4>);
  if (chunks <= 16) return go(topk_rows_kernel<16>);
  if (chunks <= 48) return go(topk_rows_kernel<48>);
  if (chunks <= 72) return go(topk_rows_kernel<72>);
  return go(topk_rows_kernel<0>);
}

hipError_t launch_select_global(const double* qp, const double* kpT, int32_t* idx, int32_t* cnt,
                                double* scores, const GlobalArgs& a, hipStream_t s) {
  if (a.n_heads == 0) return hipSuccess;
  const size_t lds = (size_t)a.nb * sizeof(uint64_t);
  hipError_t e = hipFuncSetAttribute(reinterpret_cast<const void*>(select_global_kernel),
                                     hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(select_global_kernel, dim3((unsigned)a.n_heads), dim3(kGlobalThreads), lds, s,
                     qp, kpT, idx, cnt, scores, a);
  e = hipGetLastError();
  if (e != hipSuccess || a.nb == 1) return e;
  const int64_t waves = (int64_t)a.n_heads * (a.nb - 1);
  hipLaunchKernelGGL(select_global_broadcast_kernel, dim3((unsigned)((waves + 3) / 4)), dim3(256),
                     0, s, idx, cnt, a);
  return hipGetLastError();
}

hipError_t run_validate_index(const int32_t* idx, const int32_t* cnt, int32_t* result,
                              const ValidateArgs& a, int32_t out[2], hipStream_t s) {
  hipLaunchKernelGGL(validate_init_kernel, dim3(1), dim3(64), 0, s, result);
  const int64_t waves = (int64_t)a.n_heads * a.nb;
  if (waves > 0)
    hipLaunchKernelGGL(validate_index_kernel, dim3((unsigned)((waves + 3) / 4)), dim3(256), 0, s,
                       idx, cnt, result, a);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  e = hipMemcpyAsync(out, result, 2 * sizeof(int32_t), hipMemcpyDeviceToHost, s);
  if (e != hipSuccess) return e;
  return hipStreamSynchronize(s);
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
