// Launch stand-ins for the host-layer sanitizer build: the C ABI layer
// (csrc/api.cpp) compiled by g++ with AddressSanitizer and
// UndefinedBehaviorSanitizer and linked against these functions instead of
// the HIP kernels, so every validation, sizing and launch-ordering path of
// the ABI runs on the CPU. Each stand-in checks the arguments the host layer
// built for its kernel (counts inside their arrays, heads in range and
// distinct, ordered prefix sums, workspace offsets inside the workspace the
// caller declared) and returns hipErrorInvalidValue when one is off, which
// the ABI reports as SAF3R_ERR_HIP. Nothing here touches a GPU.
#include <stdint.h>

#include <vector>

#include "../../paper_2607_03612_amd/csrc/saf3r_internal.h"

namespace saf3r {
namespace {

bool heads_ok(const int16_t* head, int n, int limit) {
  if (n < 0 || n > kMaxHeads) return false;
  std::vector<char> seen(kMaxHeads, 0);
  for (int i = 0; i < n; ++i) {
    if (head[i] < 0 || head[i] >= limit || seen[head[i]]) return false;
    seen[head[i]] = 1;
  }
  return true;
}

bool blocks_ok(int64_t n, int nb) { return n >= 1 && nb == (int)((n + kBlock - 1) / kBlock); }

hipError_t launch_status(bool ok) { return ok ? hipSuccess : hipErrorInvalidValue; }

}  // namespace

hipError_t launch_pool(int dtype, const void* q, const void* k, double* qp, double* kp,
                       const PoolArgs& a, hipStream_t) {
  return launch_status((dtype == 0 || dtype == 1) && q && k && qp && kp && blocks_ok(a.n, a.nb) &&
                 heads_ok(a.head, a.n_heads, kMaxHeads));
}

hipError_t launch_select_topk(const double* qp, const double* kpT, int32_t* idx, int32_t* cnt,
                              double*, const TopKArgs& a, size_t lds_bytes, hipStream_t) {
  bool ok = qp && kpT && idx && cnt && blocks_ok(a.n, a.nb) && heads_ok(a.head, a.n_heads, kMaxHeads);
  ok = ok && (a.rows_per_group == 1 || a.rows_per_group == 2 || a.rows_per_group == 4 ||
              a.rows_per_group == 8 || a.rows_per_group == 16);
  ok = ok && lds_bytes == topk_lds_bytes(a.rows_per_group, a.nb) && lds_bytes <= 160 * 1024;
  for (int i = 0; ok && i < a.n_heads; ++i) ok = a.topk[i] >= 1 && a.topk[i] <= a.nb && a.topk[i] <= a.cap;
  return launch_status(ok);
}

hipError_t launch_select_topk_ws(const double* qp, const double* kpT, uint32_t* keys, int32_t* idx,
                                 int32_t* cnt, double*, const TopKArgs& a, hipStream_t) {
  bool ok = qp && kpT && keys && idx && cnt && blocks_ok(a.n, a.nb) &&
            heads_ok(a.head, a.n_heads, kMaxHeads) && a.n_heads >= 1;
  for (int i = 0; ok && i < a.n_heads; ++i) ok = a.topk[i] >= 1 && a.topk[i] <= a.nb && a.topk[i] <= a.cap;
  return launch_status(ok);
}

hipError_t launch_select_static(int32_t* idx, int32_t* cnt, const StaticArgs& a, hipStream_t) {
  bool ok = idx && cnt && blocks_ok(a.n, a.nb) && heads_ok(a.head, a.n_heads, kMaxHeads) &&
            a.tokens_per_frame >= 1;
  for (int i = 0; ok && i < a.n_heads; ++i)
    ok = a.pattern[i] == kDense || a.pattern[i] == kFrameLocal || a.pattern[i] == kAnchor ||
         a.pattern[i] == kStride;
  return launch_status(ok);
}

hipError_t launch_select_global(const double* qp, const double* kpT, int32_t* idx, int32_t* cnt,
                                double*, const GlobalArgs& a, hipStream_t) {
  bool ok = qp && kpT && idx && cnt && blocks_ok(a.n, a.nb) && heads_ok(a.head, a.n_heads, kMaxHeads);
  for (int i = 0; ok && i < a.n_heads; ++i) ok = a.topk[i] >= 1 && a.topk[i] <= a.nb && a.topk[i] <= a.cap;
  return launch_status(ok);
}

hipError_t launch_cosine(int dtype, const void* f, double* fb, double* sim, int32_t* idx,
                         int32_t* cnt, const CosineArgs& a, hipStream_t) {
  bool ok = (dtype == 0 || dtype == 1) && f && fb && idx && cnt && blocks_ok(a.n, a.nb) &&
            a.dim >= 1 && a.dim <= kMaxCosineDim && sim == fb + (int64_t)a.dim * a.nb &&
            a.n_groups >= 0 && a.n_groups <= kMaxHeads && a.group_start[0] == 0;
  for (int g = 0; ok && g < a.n_groups; ++g)
    ok = a.group_start[g + 1] > a.group_start[g] && a.group_k[g] >= 1 &&
         a.group_k[g] <= kMaxCosinePerFrame && (g == 0 || a.group_k[g] > a.group_k[g - 1]);
  ok = ok && heads_ok(a.head, a.group_start[a.n_groups], kMaxHeads);
  return launch_status(ok);
}

hipError_t launch_nmse(int dtype, const void* ref, const void* test, void* workspace, double* out,
                       int heads, int64_t n, hipStream_t) {
  return launch_status((dtype == 0 || dtype == 1) && ref && test && workspace && out && heads >= 1 &&
                 heads <= kMaxHeads && n >= 1);
}

hipError_t nmse_scratch(void** ptr) {
  static double2 fake[kMaxHeads * kNmseParts];  // host stand-in, never written
  *ptr = fake;
  return hipSuccess;
}

hipError_t launch_attention(int dtype, const void* q, const void* k, const void* v,
                            const int32_t*, const int32_t*, void* out, float*, const AttnArgs& a,
                            hipStream_t) {
  bool ok = (dtype == 0 || dtype == 1) && q && k && v && out && blocks_ok(a.n, a.nb) &&
            a.slab == (a.nb + 7) / 8 && a.splits == kSplitChunks && a.mode >= 0 && a.mode <= 2 &&
            heads_ok(a.order, a.heads, kMaxHeads) && a.unit_start[0] == 0;
  int n_split = 0;
  for (int i = 0; ok && i < a.heads; ++i) {
    const bool split = a.split_pos[i] >= 0;
    ok = a.unit_start[i + 1] == a.unit_start[i] + a.slab * (split ? a.splits : 1) &&
         a.split_pos[i] >= -1 && a.split_pos[i] < kMaxHeads && (!split || a.part_o);
    if (split) {
      ok = ok && a.split_pos[i] == n_split && a.mode == 0;
      ++n_split;
    }
    if (a.mode == 2) ok = ok && a.stride[a.order[i]] >= 1 && a.stride[a.order[i]] <= a.n;
  }
  // the partials of split items start after the O accumulators
  if (ok && n_split > 0)
    ok = a.part_ml == a.part_o + (int64_t)n_split * a.splits * a.nb * kBlock * kHeadDim;
  return launch_status(ok);
}

// the check's result as the device would report it for lists that pass
hipError_t run_validate_index(const int32_t* idx, const int32_t* cnt, int32_t* result,
                              const ValidateArgs& a, int32_t out[2], hipStream_t) {
  bool ok = idx && cnt && result && out && a.nb >= 1 && a.nb <= kMaxBlocks && a.cap >= 1 &&
            a.n_heads >= 1 && heads_ok(a.head, a.n_heads, kMaxHeads);
  for (int i = 0; ok && i < a.n_heads; ++i) ok = a.expect[i] == -1 || (a.expect[i] >= 1 && a.expect[i] <= a.nb);
  out[0] = 0;
  out[1] = 0x7fffffff;
  return launch_status(ok);
}

hipError_t launch_attention_merge(const float* part_o, const float* part_ml, void* out, float*,
                                  const MergeArgs& a, hipStream_t) {
  return launch_status(part_o && part_ml && out && blocks_ok(a.n, a.nb) && a.splits == kSplitChunks &&
                 (a.dtype == 0 || a.dtype == 1) &&
                 heads_ok(a.head, a.n_split, kMaxHeads) && a.n_split >= 1 &&
                 part_ml == part_o + (int64_t)a.n_split * a.splits * a.nb * kBlock * kHeadDim);
}

}  // namespace saf3r
