// C ABI of the SAF3R hot path: host-side validation, launch geometry and
// work ordering. Every check runs before any launch, so a call that returns
// an error has enqueued nothing.
#include <math.h>
#include <stdint.h>

#include <algorithm>
#include <numeric>
#include <vector>

#include "../../include/saf3r.h"
#include "saf3r_internal.h"

namespace {

using saf3r::kMaxBlocks;
using saf3r::kMaxHeads;

constexpr int64_t kMaxTokens = (int64_t)kMaxBlocks * saf3r::kBlock;  // 1,048,576

// Problem sizes after validation.
struct Shape {
  int heads;
  int64_t n;
  int nb;
  int frames;
  int tokens_per_frame;
  int dtype;
};

saf3r_status check_problem(const saf3r_problem* p, Shape* out) {
  if (!p) return SAF3R_ERR_INVALID_ARGUMENT;
  if (p->heads <= 0 || p->frames <= 0 || p->tokens_per_frame <= 0) return SAF3R_ERR_INVALID_ARGUMENT;
  if (p->dtype != SAF3R_F32 && p->dtype != SAF3R_BF16) return SAF3R_ERR_INVALID_ARGUMENT;
  if (p->head_dim != saf3r::kHeadDim || p->block != saf3r::kBlock) return SAF3R_ERR_UNSUPPORTED;
  if (p->heads > kMaxHeads) return SAF3R_ERR_UNSUPPORTED;
  const int64_t n = (int64_t)p->frames * p->tokens_per_frame;
  if (n > kMaxTokens) return SAF3R_ERR_UNSUPPORTED;
  out->heads = p->heads;
  out->n = n;
  out->nb = (int)((n + saf3r::kBlock - 1) / saf3r::kBlock);
  out->frames = p->frames;
  out->tokens_per_frame = p->tokens_per_frame;
  out->dtype = p->dtype;
  return SAF3R_OK;
}

saf3r_status check_table(const Shape& s, const saf3r_head_cfg* t) {
  if (!t) return SAF3R_ERR_INVALID_ARGUMENT;
  for (int h = 0; h < s.heads; ++h) {
    const int32_t p = t[h].param;
    switch (t[h].pattern) {
      case SAF3R_DENSE:
      case SAF3R_FRAME_LOCAL:
      case SAF3R_SKIP:
        break;
      case SAF3R_TOPK:
      case SAF3R_GLOBAL_PROBE:
        if (p < 1 || p > s.nb) return SAF3R_ERR_BAD_TABLE;
        break;
      case SAF3R_ANCHOR:
        if (p < 0 || p >= s.frames) return SAF3R_ERR_BAD_TABLE;
        break;
      case SAF3R_STRIDE:
        if (p < 1 || (int64_t)p > s.n) return SAF3R_ERR_BAD_TABLE;
        break;
      case SAF3R_COSINE_TOPK:
        if (p < 1 || p > saf3r::kMaxCosinePerFrame) return SAF3R_ERR_BAD_TABLE;
        break;
      default:
        return SAF3R_ERR_BAD_TABLE;
    }
  }
  return SAF3R_OK;
}

// Kept blocks of query block i of a frame-local head: the key blocks whose
// tokens overlap the frames touched by block i (a contiguous range).
int frame_local_len(const Shape& s, int i) {
  const int64_t T = s.tokens_per_frame;
  const int64_t first = (int64_t)i * saf3r::kBlock;
  const int64_t last = std::min<int64_t>(first + saf3r::kBlock, s.n) - 1;
  const int64_t tok_lo = (first / T) * T;
  const int64_t tok_hi = std::min<int64_t>((last / T + 1) * T, s.n) - 1;
  return (int)(tok_hi / saf3r::kBlock - tok_lo / saf3r::kBlock + 1);
}

int max_frame_local_len(const Shape& s) {
  int best = 0;
  for (int i = 0; i < s.nb; ++i) best = std::max(best, frame_local_len(s, i));
  return best;
}

// Kept blocks of an ANCHOR head: the key blocks holding a token of frame a.
int anchor_len(const Shape& s, int a) {
  const int64_t lo = (int64_t)a * s.tokens_per_frame;
  const int64_t hi = std::min<int64_t>(lo + s.tokens_per_frame, s.n) - 1;
  return (int)(hi / saf3r::kBlock - lo / saf3r::kBlock + 1);
}

// Kept blocks of a COSINE_TOPK head keeping k per frame (a key block counts
// under the frame of its first token): sum over frames of min(k, blocks).
int cosine_len(const Shape& s, int k) {
  const int64_t T = s.tokens_per_frame;
  int total = 0;
  for (int64_t f = 0; f * T < s.n; ++f) {
    const int64_t lo = (f * T + saf3r::kBlock - 1) / saf3r::kBlock;
    const int64_t hi = std::min<int64_t>(((f + 1) * T + saf3r::kBlock - 1) / saf3r::kBlock, s.nb);
    if (hi > lo) total += (int)std::min<int64_t>(k, hi - lo);
  }
  return total;
}

int capacity(const Shape& s, const saf3r_head_cfg* t) {
  int cap = 1;
  bool any_fl = false;
  for (int h = 0; h < s.heads; ++h) {
    const int p = t[h].pattern;
    if (p == SAF3R_TOPK || p == SAF3R_GLOBAL_PROBE) cap = std::max(cap, t[h].param);
    if (p == SAF3R_ANCHOR) cap = std::max(cap, anchor_len(s, t[h].param));
    if (p == SAF3R_COSINE_TOPK) cap = std::max(cap, cosine_len(s, t[h].param));
    if (p == SAF3R_FRAME_LOCAL) any_fl = true;
  }
  if (any_fl) cap = std::max(cap, max_frame_local_len(s));
  return cap;
}

bool pooled_class(int pattern) { return pattern == SAF3R_TOPK || pattern == SAF3R_GLOBAL_PROBE; }

// True when p is null or a multiple of `bytes`: the kernels read and write
// Q/K/V/O, the pooled arrays, the NMSE inputs and the workspaces with
// 16-byte vector accesses, the other arrays element by element.
bool aligned(const void* p, uintptr_t bytes) { return reinterpret_cast<uintptr_t>(p) % bytes == 0; }

saf3r_status hip_status(hipError_t e) { return e == hipSuccess ? SAF3R_OK : SAF3R_ERR_HIP; }

}  // namespace

extern "C" {

int32_t saf3r_num_blocks(const saf3r_problem* problem) {
  Shape s;
  const saf3r_status st = check_problem(problem, &s);
  return st == SAF3R_OK ? s.nb : (int32_t)st;
}

int32_t saf3r_index_capacity(const saf3r_problem* problem, const saf3r_head_cfg* table) {
  Shape s;
  saf3r_status st = check_problem(problem, &s);
  if (st != SAF3R_OK) return st;
  st = check_table(s, table);
  if (st != SAF3R_OK) return st;
  return capacity(s, table);
}

saf3r_status saf3r_estimate_blocks(const saf3r_problem* problem, const saf3r_head_cfg* table,
                                   const void* q, const void* k, double* q_pooled,
                                   double* k_pooled, void* stream) {
  Shape s;
  saf3r_status st = check_problem(problem, &s);
  if (st != SAF3R_OK) return st;
  st = check_table(s, table);
  if (st != SAF3R_OK) return st;
  if (!q || !k || !q_pooled || !k_pooled) return SAF3R_ERR_INVALID_ARGUMENT;
  if (!aligned(q, 16) || !aligned(k, 16) || !aligned(q_pooled, 16) || !aligned(k_pooled, 8))
    return SAF3R_ERR_INVALID_ARGUMENT;
  saf3r::PoolArgs a{};
  a.n = s.n;
  a.nb = s.nb;
  for (int h = 0; h < s.heads; ++h)
    if (pooled_class(table[h].pattern)) a.head[a.n_heads++] = (int16_t)h;
  return hip_status(saf3r::launch_pool(s.dtype, q, k, q_pooled, k_pooled, a,
                                       static_cast<hipStream_t>(stream)));
}

int64_t saf3r_select_workspace_bytes(const saf3r_problem* problem, const saf3r_head_cfg* table) {
  Shape s;
  saf3r_status st = check_problem(problem, &s);
  if (st != SAF3R_OK) return st;
  st = check_table(s, table);
  if (st != SAF3R_OK) return st;
  int64_t topk_heads = 0;
  for (int h = 0; h < s.heads; ++h) topk_heads += table[h].pattern == SAF3R_TOPK ? 1 : 0;
  return topk_heads * s.nb * (int64_t)saf3r::topk_ws_row_bytes(s.nb);
}

saf3r_status saf3r_select_blocks(const saf3r_problem* problem, const saf3r_head_cfg* table,
                                 const double* q_pooled, const double* k_pooled,
                                 int32_t* block_idx, int32_t* block_cnt, int32_t cap,
                                 double* scores_or_null, void* workspace_or_null,
                                 int64_t workspace_bytes, void* stream) {
  Shape s;
  saf3r_status st = check_problem(problem, &s);
  if (st != SAF3R_OK) return st;
  st = check_table(s, table);
  if (st != SAF3R_OK) return st;
  if (!q_pooled || !k_pooled || !block_idx || !block_cnt) return SAF3R_ERR_INVALID_ARGUMENT;
  if (!aligned(q_pooled, 8) || !aligned(k_pooled, 8) || !aligned(block_idx, 4) ||
      !aligned(block_cnt, 4) || !aligned(scores_or_null, 8) || !aligned(workspace_or_null, 16))
    return SAF3R_ERR_INVALID_ARGUMENT;
  if (cap < capacity(s, table)) return SAF3R_ERR_CAPACITY;

  saf3r::TopKArgs ta{};
  ta.n = s.n;
  ta.nb = s.nb;
  ta.cap = cap;
  saf3r::StaticArgs sa{};
  sa.n = s.n;
  sa.nb = s.nb;
  sa.cap = cap;
  sa.tokens_per_frame = s.tokens_per_frame;
  saf3r::GlobalArgs ga{};
  ga.n = s.n;
  ga.nb = s.nb;
  ga.cap = cap;
  for (int h = 0; h < s.heads; ++h) {
    if (table[h].pattern == SAF3R_TOPK) {
      ta.head[ta.n_heads] = (int16_t)h;
      ta.topk[ta.n_heads++] = table[h].param;
    } else if (table[h].pattern == SAF3R_GLOBAL_PROBE) {
      ga.head[ga.n_heads] = (int16_t)h;
      ga.topk[ga.n_heads++] = table[h].param;
    } else if (table[h].pattern == SAF3R_COSINE_TOPK || table[h].pattern == SAF3R_SKIP) {
      // cosine lists come from saf3r_cosine_select; skipped heads stay as they are
    } else {
      sa.head[sa.n_heads] = (int16_t)h;
      sa.pattern[sa.n_heads] = (int8_t)table[h].pattern;
      sa.param[sa.n_heads++] = table[h].param;
    }
  }
  // Without a workspace: query blocks scored per workgroup, the most (up to
  // 16) whose score rows fit in LDS; each key-block read is then shared by
  // that many rows. With one: as many Top-K heads per pair of launches as
  // the workspace holds.
  constexpr size_t kLdsBudget = 150 * 1024;
  int rows = 16;
  while (rows > 1 && saf3r::topk_lds_bytes(rows, s.nb) > kLdsBudget) rows /= 2;
  ta.rows_per_group = rows;
  const size_t lds = saf3r::topk_lds_bytes(rows, s.nb);
  const int64_t head_bytes = (int64_t)s.nb * (int64_t)saf3r::topk_ws_row_bytes(s.nb);
  int batch = ta.n_heads;
  if (workspace_or_null) {
    if (workspace_bytes < 0) return SAF3R_ERR_INVALID_ARGUMENT;
    if (ta.n_heads > 0 && workspace_bytes < head_bytes) return SAF3R_ERR_CAPACITY;
    if (ta.n_heads > 0) batch = (int)std::min<int64_t>(ta.n_heads, workspace_bytes / head_bytes);
  } else if (lds > kLdsBudget) {
    return SAF3R_ERR_UNSUPPORTED;
  }

  hipStream_t hs = static_cast<hipStream_t>(stream);
  hipError_t e = saf3r::launch_select_static(block_idx, block_cnt, sa, hs);
  if (e != hipSuccess) return SAF3R_ERR_HIP;
  e = saf3r::launch_select_global(q_pooled, k_pooled, block_idx, block_cnt, scores_or_null, ga, hs);
  if (e != hipSuccess) return SAF3R_ERR_HIP;
  if (!workspace_or_null)
    return hip_status(saf3r::launch_select_topk(q_pooled, k_pooled, block_idx, block_cnt,
                                                scores_or_null, ta, lds, hs));
  for (int b0 = 0; b0 < ta.n_heads; b0 += batch) {
    saf3r::TopKArgs tb = ta;
    tb.n_heads = std::min(batch, ta.n_heads - b0);
    for (int q = 0; q < tb.n_heads; ++q) {
      tb.head[q] = ta.head[b0 + q];
      tb.topk[q] = ta.topk[b0 + q];
    }
    e = saf3r::launch_select_topk_ws(q_pooled, k_pooled, static_cast<uint32_t*>(workspace_or_null),
                                     block_idx, block_cnt, scores_or_null, tb, hs);
    if (e != hipSuccess) return SAF3R_ERR_HIP;
  }
  return SAF3R_OK;
}

// Key blocks one query block of head h walks (its work if not split).
static int attention_cost(const Shape& s, const saf3r_head_cfg* table, int h, int fl_len) {
  const int p = table[h].pattern;
  switch (p) {
    case SAF3R_DENSE: return s.nb;
    case SAF3R_FRAME_LOCAL: return fl_len;
    case SAF3R_ANCHOR: return anchor_len(s, table[h].param);
    case SAF3R_COSINE_TOPK: return cosine_len(s, table[h].param);
    case SAF3R_STRIDE:
      return (int)((((s.n + table[h].param - 1) / table[h].param) + saf3r::kBlock - 1) /
                   saf3r::kBlock);
    default: return table[h].param;  // TOPK, GLOBAL_PROBE
  }
}

static bool listed_class(int p) {
  return p == SAF3R_FRAME_LOCAL || p == SAF3R_TOPK || p == SAF3R_ANCHOR ||
         p == SAF3R_GLOBAL_PROBE || p == SAF3R_COSINE_TOPK;
}

// Key blocks walked by all query blocks of the list and dense heads (the
// work of the launch that may split).
static int64_t listed_work(const Shape& s, const saf3r_head_cfg* table, int fl_len) {
  int64_t total = 0;
  for (int h = 0; h < s.heads; ++h) {
    const int p = table[h].pattern;
    if (p == SAF3R_DENSE || listed_class(p)) total += (int64_t)s.nb * attention_cost(s, table, h, fl_len);
  }
  return total;
}

// A list or dense head runs split into key ranges: (bf16, locality) on a
// layer of at least kSplitMinExtent key blocks when its list can reach
// kSplitMinBlocks key blocks; (load balance, both dtypes) when its items walk
// at least kBalanceMinBlocks (bf16) or kBalanceMinBlocksF32 (fp32) blocks,
// more than twice the layer's work per wave slot.
static bool attention_split(const Shape& s, const saf3r_head_cfg* table, int h, int cost,
                            int64_t work) {
  const int p = table[h].pattern;
  if (!(listed_class(p) || p == SAF3R_DENSE)) return false;
  const bool bf16 = s.dtype == SAF3R_BF16;
  if (bf16 && listed_class(p) && s.nb >= saf3r::kSplitMinExtent && cost >= saf3r::kSplitMinBlocks)
    return true;
  const int min_blocks = bf16 ? saf3r::kBalanceMinBlocks : saf3r::kBalanceMinBlocksF32;
  return cost >= min_blocks && (int64_t)cost * saf3r::kWaveSlots > 2 * work;
}

int64_t saf3r_attention_workspace_bytes(const saf3r_problem* problem, const saf3r_head_cfg* table) {
  Shape s;
  saf3r_status st = check_problem(problem, &s);
  if (st != SAF3R_OK) return st;
  st = check_table(s, table);
  if (st != SAF3R_OK) return st;
  const int fl_len = max_frame_local_len(s);
  const int64_t work = listed_work(s, table, fl_len);
  int64_t n_split = 0;
  for (int h = 0; h < s.heads; ++h)
    n_split += attention_split(s, table, h, attention_cost(s, table, h, fl_len), work) ? 1 : 0;
  return n_split * saf3r::kSplitChunks * s.nb * saf3r::kSplitItemBytes;
}

saf3r_status saf3r_sparse_attention(const saf3r_problem* problem, const saf3r_head_cfg* table,
                                    const void* q, const void* k, const void* v,
                                    const int32_t* block_idx, const int32_t* block_cnt,
                                    int32_t cap, void* out, float* lse_or_null,
                                    void* workspace_or_null, int64_t workspace_bytes,
                                    void* stream) {
  Shape s;
  saf3r_status st = check_problem(problem, &s);
  if (st != SAF3R_OK) return st;
  st = check_table(s, table);
  if (st != SAF3R_OK) return st;
  if (!q || !k || !v || !out) return SAF3R_ERR_INVALID_ARGUMENT;
  if (!aligned(q, 16) || !aligned(k, 16) || !aligned(v, 16) || !aligned(out, 16) ||
      !aligned(block_idx, 4) || !aligned(block_cnt, 4) || !aligned(lse_or_null, 4))
    return SAF3R_ERR_INVALID_ARGUMENT;
  bool needs_lists = false;
  for (int h = 0; h < s.heads; ++h) {
    const int p = table[h].pattern;
    needs_lists = needs_lists || (p != SAF3R_DENSE && p != SAF3R_STRIDE && p != SAF3R_SKIP);
  }
  if (needs_lists) {
    if (!block_idx || !block_cnt) return SAF3R_ERR_INVALID_ARGUMENT;
    if (cap < capacity(s, table)) return SAF3R_ERR_CAPACITY;
  }
  const int64_t split_bytes = saf3r_attention_workspace_bytes(problem, table);
  if (split_bytes < 0) return (saf3r_status)split_bytes;
  const bool split = workspace_or_null != nullptr && split_bytes > 0;
  if (workspace_or_null) {
    if (workspace_bytes < 0 || !aligned(workspace_or_null, 16)) return SAF3R_ERR_INVALID_ARGUMENT;
    if (workspace_bytes < split_bytes) return SAF3R_ERR_CAPACITY;
  }

  // Up to three launches: heads with block lists or dense (one kernel, work
  // items in decreasing length so the longest start first; split heads as
  // kSplitChunks items per query block), the merge of split heads, then
  // STRIDE heads (token-sampled keys).
  saf3r::AttnArgs a{};
  a.n = s.n;
  a.nb = s.nb;
  a.cap = cap;
  a.slab = (s.nb + 7) / 8;
  a.splits = saf3r::kSplitChunks;
  a.scale_log2 = (float)(1.4426950408889634 / sqrt((double)saf3r::kHeadDim));
  saf3r::AttnArgs sa = a;
  std::vector<int> item_cost(s.heads, 0);
  std::vector<char> is_split(s.heads, 0);
  const int fl_len = max_frame_local_len(s);
  const int64_t work = listed_work(s, table, fl_len);
  std::vector<int> listed, strided;
  bool all_dense = true;
  for (int h = 0; h < s.heads; ++h) {
    const int p = table[h].pattern;
    if (p == SAF3R_SKIP) continue;
    a.dense[h] = p == SAF3R_DENSE ? 1 : 0;
    sa.stride[h] = p == SAF3R_STRIDE ? table[h].param : 1;
    const int cost = attention_cost(s, table, h, fl_len);
    is_split[h] = split && attention_split(s, table, h, cost, work) ? 1 : 0;
    item_cost[h] = is_split[h] ? (cost + saf3r::kSplitChunks - 1) / saf3r::kSplitChunks : cost;
    if (p == SAF3R_STRIDE) {
      strided.push_back(h);
    } else {
      listed.push_back(h);
      all_dense = all_dense && p == SAF3R_DENSE;
    }
  }
  auto by_cost = [&](int x, int y) { return item_cost[x] > item_cost[y]; };
  std::stable_sort(listed.begin(), listed.end(), by_cost);
  std::stable_sort(strided.begin(), strided.end(), by_cost);
  saf3r::MergeArgs ma{};
  ma.n = s.n;
  ma.nb = s.nb;
  ma.splits = saf3r::kSplitChunks;
  ma.dtype = s.dtype;
  a.heads = (int)listed.size();
  bool any_split = false;
  for (int h : listed) any_split = any_split || is_split[h];
  a.mode = all_dense && !any_split ? 1 : 0;  // split items run in the list mode
  a.unit_start[0] = 0;
  for (size_t i = 0; i < listed.size(); ++i) {
    const int h = listed[i];
    a.order[i] = (int16_t)h;
    a.split_pos[i] = is_split[h] ? (int16_t)ma.n_split : (int16_t)-1;
    if (is_split[h]) ma.head[ma.n_split++] = (int16_t)h;
    a.unit_start[i + 1] = a.unit_start[i] + a.slab * (is_split[h] ? saf3r::kSplitChunks : 1);
  }
  const int64_t part_o_bytes =
      (int64_t)ma.n_split * saf3r::kSplitChunks * s.nb * saf3r::kBlock * saf3r::kHeadDim * 4;
  a.part_o = split ? static_cast<float*>(workspace_or_null) : nullptr;
  a.part_ml = split ? reinterpret_cast<float*>(static_cast<char*>(workspace_or_null) + part_o_bytes)
                    : nullptr;
  sa.heads = (int)strided.size();
  sa.mode = 2;
  sa.unit_start[0] = 0;
  for (size_t i = 0; i < strided.size(); ++i) {
    sa.order[i] = (int16_t)strided[i];
    sa.split_pos[i] = -1;
    sa.unit_start[i + 1] = sa.unit_start[i] + sa.slab;
  }

  hipStream_t hs = static_cast<hipStream_t>(stream);
  hipError_t e = saf3r::launch_attention(s.dtype, q, k, v, block_idx, block_cnt, out, lse_or_null,
                                         a, hs);
  if (e != hipSuccess) return SAF3R_ERR_HIP;
  if (ma.n_split > 0) {
    e = saf3r::launch_attention_merge(a.part_o, a.part_ml, out, lse_or_null, ma, hs);
    if (e != hipSuccess) return SAF3R_ERR_HIP;
  }
  return hip_status(saf3r::launch_attention(s.dtype, q, k, v, block_idx, block_cnt, out,
                                            lse_or_null, sa, hs));
}

saf3r_status saf3r_validate_index(const saf3r_problem* problem, const saf3r_head_cfg* table,
                                  const int32_t* block_idx, const int32_t* block_cnt, int32_t cap,
                                  int32_t* workspace, int32_t* first_bad_or_null, void* stream) {
  Shape s;
  saf3r_status st = check_problem(problem, &s);
  if (st != SAF3R_OK) return st;
  st = check_table(s, table);
  if (st != SAF3R_OK) return st;
  if (!block_idx || !block_cnt || !workspace || cap < 1) return SAF3R_ERR_INVALID_ARGUMENT;
  if (!aligned(block_idx, 4) || !aligned(block_cnt, 4) || !aligned(workspace, 4))
    return SAF3R_ERR_INVALID_ARGUMENT;
  saf3r::ValidateArgs a{};
  a.nb = s.nb;
  a.cap = cap;
  for (int h = 0; h < s.heads; ++h) {
    const int p = table[h].pattern;
    if (!listed_class(p)) continue;  // DENSE, STRIDE and SKIP heads have no list
    a.head[a.n_heads] = (int16_t)h;
    a.expect[a.n_heads] = p == SAF3R_TOPK || p == SAF3R_GLOBAL_PROBE ? table[h].param : -1;
    ++a.n_heads;
  }
  if (a.n_heads == 0) return SAF3R_OK;
  int32_t result[2] = {0, 0};
  if (saf3r::run_validate_index(block_idx, block_cnt, workspace, a, result,
                                static_cast<hipStream_t>(stream)) != hipSuccess)
    return SAF3R_ERR_HIP;
  if (result[0] == 0) return SAF3R_OK;
  if (first_bad_or_null) *first_bad_or_null = result[1];
  return SAF3R_ERR_CORRUPT_INDEX;
}

int64_t saf3r_cosine_workspace_bytes(const saf3r_problem* problem, int32_t feat_dim) {
  Shape s;
  const saf3r_status st = check_problem(problem, &s);
  if (st != SAF3R_OK) return st;
  if (feat_dim < 1 || feat_dim > saf3r::kMaxCosineDim) return SAF3R_ERR_INVALID_ARGUMENT;
  return ((int64_t)feat_dim * s.nb + (int64_t)s.nb * s.nb) * (int64_t)sizeof(double);
}

saf3r_status saf3r_cosine_select(const saf3r_problem* problem, const saf3r_head_cfg* table,
                                 const void* features, int32_t feat_dim, void* workspace,
                                 int64_t workspace_bytes, int32_t* block_idx, int32_t* block_cnt,
                                 int32_t cap, void* stream) {
  Shape s;
  saf3r_status st = check_problem(problem, &s);
  if (st != SAF3R_OK) return st;
  st = check_table(s, table);
  if (st != SAF3R_OK) return st;
  if (!features || !workspace || !block_idx || !block_cnt) return SAF3R_ERR_INVALID_ARGUMENT;
  if (feat_dim < 1 || feat_dim > saf3r::kMaxCosineDim) return SAF3R_ERR_INVALID_ARGUMENT;
  if (!aligned(features, s.dtype == SAF3R_BF16 ? 2 : 4) || !aligned(workspace, 8) ||
      !aligned(block_idx, 4) || !aligned(block_cnt, 4))
    return SAF3R_ERR_INVALID_ARGUMENT;
  const int64_t need = saf3r_cosine_workspace_bytes(problem, feat_dim);
  if (workspace_bytes < need) return SAF3R_ERR_CAPACITY;
  if (cap < capacity(s, table)) return SAF3R_ERR_CAPACITY;
  saf3r::CosineArgs a{};
  a.n = s.n;
  a.nb = s.nb;
  a.cap = cap;
  a.dim = feat_dim;
  a.tokens_per_frame = s.tokens_per_frame;
  // the lists depend on the features and the per-frame count only: heads
  // with equal counts form one group, whose lists are found once
  std::vector<int> cos;
  for (int h = 0; h < s.heads; ++h)
    if (table[h].pattern == SAF3R_COSINE_TOPK) cos.push_back(h);
  std::stable_sort(cos.begin(), cos.end(),
                   [&](int x, int y) { return table[x].param < table[y].param; });
  for (size_t q = 0; q < cos.size(); ++q) {
    a.head[q] = (int16_t)cos[q];
    if (q == 0 || table[cos[q]].param != table[cos[q - 1]].param) {
      a.group_start[a.n_groups] = (int16_t)q;
      a.group_k[a.n_groups++] = table[cos[q]].param;
    }
  }
  a.group_start[a.n_groups] = (int16_t)cos.size();
  double* fb = static_cast<double*>(workspace);
  double* sim = fb + (int64_t)feat_dim * s.nb;
  return hip_status(saf3r::launch_cosine(s.dtype, features, fb, sim, block_idx, block_cnt, a,
                                         static_cast<hipStream_t>(stream)));
}

int64_t saf3r_nmse_workspace_bytes(const saf3r_problem* problem) {
  Shape s;
  const saf3r_status st = check_problem(problem, &s);
  if (st != SAF3R_OK) return st;
  return (int64_t)s.heads * saf3r::kNmseParts * 2 * (int64_t)sizeof(double);
}

saf3r_status saf3r_nmse(const saf3r_problem* problem, const void* o_full, const void* o_sparse,
                        void* workspace, int64_t workspace_bytes, double* nmse_out,
                        void* stream) {
  Shape s;
  const saf3r_status st = check_problem(problem, &s);
  if (st != SAF3R_OK) return st;
  if (!o_full || !o_sparse || !workspace || !nmse_out) return SAF3R_ERR_INVALID_ARGUMENT;
  if (!aligned(o_full, 16) || !aligned(o_sparse, 16) || !aligned(workspace, 16) ||
      !aligned(nmse_out, 8))
    return SAF3R_ERR_INVALID_ARGUMENT;
  if (workspace_bytes < saf3r_nmse_workspace_bytes(problem)) return SAF3R_ERR_CAPACITY;
  return hip_status(saf3r::launch_nmse(s.dtype, o_full, o_sparse, workspace, nmse_out, s.heads,
                                       s.n, static_cast<hipStream_t>(stream)));
}

saf3r_status saf3r_nmse_noalloc(const saf3r_problem* problem, const void* o_full,
                                const void* o_sparse, double* nmse_out, void* stream) {
  Shape s;
  const saf3r_status st = check_problem(problem, &s);
  if (st != SAF3R_OK) return st;
  if (!o_full || !o_sparse || !nmse_out) return SAF3R_ERR_INVALID_ARGUMENT;
  if (!aligned(o_full, 16) || !aligned(o_sparse, 16) || !aligned(nmse_out, 8))
    return SAF3R_ERR_INVALID_ARGUMENT;
  if (saf3r_nmse_workspace_bytes(problem) > saf3r::kNmseScratchBytes) return SAF3R_ERR_CAPACITY;
  void* scratch = nullptr;
  if (saf3r::nmse_scratch(&scratch) != hipSuccess) return SAF3R_ERR_HIP;
  return hip_status(saf3r::launch_nmse(s.dtype, o_full, o_sparse, scratch, nmse_out, s.heads, s.n,
                                       static_cast<hipStream_t>(stream)));
}

const char* saf3r_status_string(int32_t status) {
  switch (status) {
    case SAF3R_OK: return "ok";
    case SAF3R_ERR_INVALID_ARGUMENT: return "invalid argument (null or misaligned pointer, size or dtype)";
    case SAF3R_ERR_UNSUPPORTED: return "unsupported (head_dim/block must be 64; size limits)";
    case SAF3R_ERR_CAPACITY: return "index capacity or workspace smaller than required";
    case SAF3R_ERR_HIP: return "HIP runtime error on launch";
    case SAF3R_ERR_BAD_TABLE: return "bad pattern table (class or class parameter)";
    case SAF3R_ERR_CORRUPT_INDEX: return "corrupt kept-block list (count, order, range or padding)";
    default: return "unknown status";
  }
}

}  // extern "C"
