// Internal interface between the C-ABI host layer (host_api.cpp) and the kernel
// translation units.  Everything here is validated by the host layer first.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace sparstar {

constexpr int kMaxKeep = 8;
constexpr int kMaxHeads = 256;

// Forced key blocks as disjoint, ascending block-index ranges [begin, end).
struct KeepBlocks {
  int n;
  int begin[kMaxKeep];
  int end[kMaxKeep];
};

// Per-head top-k budgets (Eq. 5), evaluated on the host.
struct HeadBudgets {
  int k[kMaxHeads];
};

// Pooled blocks are stored split for the fp16 matrix cores: row i of qbar (and
// of kbar) is 2^e_i (hi_i + lo_i) with hi_i = fp16(2^-e_i qbar_i), lo_i =
// fp16(2^-e_i qbar_i - hi_i) and e_i chosen so that the row's largest
// magnitude scales into [2^13, 2^14): hi + lo carries 22 significant bits.
// Layout per row: D fp16 hi values, then D fp16 lo values; e_i in its own
// int32 array.
struct PoolArgs {
  const uint16_t* q;  // [BH, Lq, D] bf16
  const uint16_t* k;  // [BH, Lk, D] bf16
  uint16_t* q_bar;    // [BH, n_q, 2 D] fp16 (hi, lo)
  uint16_t* k_bar;    // [BH, n_k, 2 D] fp16 (hi, lo)
  int32_t* q_exp;     // [BH, n_q]
  int32_t* k_exp;     // [BH, n_k]
  int64_t lq, lk;
  int bh, n_q, n_k;
  KeepBlocks keep;    // key blocks that are never pooled or scored
};

struct ScoreArgs {
  const uint16_t* q_bar;  // [BH, n_q, 2 D] fp16 (hi, lo)
  const uint16_t* k_bar;  // [BH, n_k, 2 D] fp16 (hi, lo)
  const int32_t* q_exp;   // [BH, n_q]
  const int32_t* k_exp;   // [BH, n_k]
  float* s;               // [BH, n_q, s_stride]
  int bh, n_q, n_k;
  int s_stride;           // floats per row of S (>= n_k)
  float tau;           // D^-1/2
  KeepBlocks keep;
};

struct SelectArgs {
  const float* s;          // [BH, n_q, s_stride]
  int32_t* kv_num_blocks;  // [BH, n_q]
  int32_t* kv_indices;     // [BH, n_q, stride]
  int64_t rows;            // BH * n_q
  int n_q, n_k, heads, stride;
  int n_sel;               // selectable key blocks per row (Eq. 4)
  int s_stride;            // floats per row of S (>= n_k)
  KeepBlocks keep;
  HeadBudgets budget;
};

// Scores and selection in one kernel (S kept in LDS): kFusedRows query blocks
// of one head per work-group, one wave per row for the selection.  Rows of up
// to kFusedMaxBlocks key blocks (16 rows x 2304 x 4 B = 144 KB of LDS).
constexpr int kFusedRows = 16;
constexpr int kFusedMaxBlocks = 2304;

struct ScoreSelectArgs {
  const uint16_t* q_bar;   // [BH, n_q, 2 D] fp16 (hi, lo)
  const uint16_t* k_bar;   // [BH, n_k, 2 D] fp16 (hi, lo)
  const int32_t* q_exp;    // [BH, n_q]
  const int32_t* k_exp;    // [BH, n_k]
  int32_t* kv_num_blocks;  // [BH, n_q]
  int32_t* kv_indices;     // [BH, n_q, stride]
  int bh, n_q, n_k, heads, stride, d;
  int n_sel;               // selectable key blocks per row (Eq. 4)
  float tau;               // D^-1/2
  KeepBlocks keep;
  HeadBudgets budget;
};

struct AttnArgs {
  const uint16_t* q;  // [BH, Lq, D]
  const uint16_t* k;  // [BH, Lk, D]
  const uint16_t* v;  // [BH, Lk, D]
  uint16_t* o;        // [BH, Lq, D]
  float* lse;         // [BH, Lq] or null
  const int32_t* kv_num_blocks;  // [BH, n_q] (sparse only)
  const int32_t* kv_indices;     // [BH, n_q, stride] (sparse only)
  int64_t lq, lk;
  int bh, n_q, n_k, stride;
  float scale_log2;   // softmax scale * log2(e)
  // Key-range split: with part_o set, work item (bh, query block, r) covers key
  // blocks [r n_k / n_splits, (r + 1) n_k / n_splits) and writes a partial
  // result that a merge kernel combines; otherwise one pass writes O and lse.
  uint16_t* part_o;   // [BH * n_q, n_splits, BLK, D] fp16: the range's unnormalised P V times 2^-e per row
  float* part_meta;   // [BH * n_q, n_splits, BLK, 4]: running max (log2 units), row sum of the bf16 P,
                      // row sum of the fp32 p, e (the row's power-of-two scale, as a float)
  int n_splits;       // key ranges per query block: 8 or kSplits
};

// Key ranges per query block: each XCD takes n_splits / 8 of them (x, x + 8, ...)
// one after the other, so that its 4 MB L2 holds about one range of a head's
// K/V at a time.  kSplits
// is the most (and the workspace is sized for it); short lists take 8 ranges,
// where the per-range fixed cost (list scan, Q load, epilogue, partial result
// and its merge) outweighs the L2 locality of the narrower ranges.
constexpr int kSplits = 16;
// Lists that can hold fewer keys than this (kv_stride x block size) take 8 ranges.
constexpr int64_t kFewRangesBelowKeys = 24576;

// Bytes of the fp16 partial-O region of the split workspace (256-byte aligned;
// the per-row records follow it).
inline size_t attn_partial_o_bytes(int64_t rows, int d) { return (size_t(rows * d) * 2 + 255) & ~size_t(255); }

// Bytes of attention workspace for the key-range split (0 when it is not used).
size_t attn_workspace_bytes(int64_t bh, int64_t n_q, int64_t n_k, int d, int block);

// Token-wise top-n mass (the upper bound of the retained-mass analysis) for a
// few sampled query rows per head.
constexpr int kTopkMaxRows = 16;

struct TopkArgs {
  const uint16_t* q;        // [BH, Lq, D] bf16
  const uint16_t* k;        // [BH, Lk, D] bf16
  const int32_t* n_tokens;  // [BH, n_rows]
  const float* lse_all;     // [BH, Lq] dense log-sum-exp
  float* scores;            // [BH, n_rows, Lk] fp32 logits (workspace)
  float* mass;              // [BH, n_rows]
  int64_t lq, lk;
  int64_t bh;
  int n_rows;
  int64_t rows[kTopkMaxRows];  // sampled query positions, shared by every head
  float scale;
};

hipError_t launch_pool(const PoolArgs& a, int d, int block, hipStream_t stream);
hipError_t launch_score(const ScoreArgs& a, int d, hipStream_t stream);
hipError_t launch_select(const SelectArgs& a, hipStream_t stream);
hipError_t launch_score_select(const ScoreSelectArgs& a, hipStream_t stream);
hipError_t launch_attn(const AttnArgs& a, int d, int block, bool dense, hipStream_t stream);
hipError_t launch_retained_mass(const float* lse_sel, const float* lse_all, int64_t n, float* mass,
                                hipStream_t stream);
hipError_t launch_topk_mass(const TopkArgs& a, int d, hipStream_t stream);

}  // namespace sparstar
