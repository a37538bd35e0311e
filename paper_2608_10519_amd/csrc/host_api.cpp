// C ABI of libsparstar: host-side validation, the keep-set and budget logic of
// Eq. (3)-(5), workspace layout, and kernel launches.  Every argument check runs
// before the first HIP call, so invalid calls return an error without touching
// the device.
#include <math.h>
#include <stdarg.h>
#include <stdio.h>

#include <algorithm>
#include <string>
#include <vector>

#include "../../include/sparstar.h"
#include "host_internal.h"
#include "launch.h"

namespace {

thread_local std::string g_error;

int fail(int code, const char* fmt, ...) {
  char buf[512];
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(buf, sizeof buf, fmt, ap);
  va_end(ap);
  g_error = buf;
  return code;
}

int ok() {
  g_error.clear();
  return SPARSTAR_OK;
}

int64_t ceil_div(int64_t a, int64_t b) { return (a + b - 1) / b; }
size_t align256(size_t x) { return (x + 255) & ~size_t(255); }
bool aligned16(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }

// Shared size checks.  Limits keep every derived index inside int32 where the
// kernels use int (block indices, list positions) and inside int64 elsewhere.
int check_sizes(int B, int H, int64_t Lq, int64_t Lk, int D, int block_size) {
  if (B < 1 || H < 1) return fail(SPARSTAR_ERR_INVALID_ARG, "B and H must be >= 1 (got B=%d, H=%d)", B, H);
  if (Lq < 0) return fail(SPARSTAR_ERR_INVALID_ARG, "Lq must be >= 0 (got %lld)", (long long)Lq);
  if (Lk < 1) return fail(SPARSTAR_ERR_INVALID_ARG, "Lk must be >= 1 (got %lld)", (long long)Lk);
  if (D != 64 && D != 128) return fail(SPARSTAR_ERR_UNSUPPORTED, "head dim %d not supported (64 or 128)", D);
  if (block_size != 64 && block_size != 128)
    return fail(SPARSTAR_ERR_UNSUPPORTED, "block size %d not supported (64 or 128)", block_size);
  if (Lq > (int64_t(1) << 30) || Lk > (int64_t(1) << 30))
    return fail(SPARSTAR_ERR_INVALID_ARG, "sequence length above 2^30");
  const int64_t bh = int64_t(B) * H;
  const int64_t nq = ceil_div(Lq, block_size), nk = ceil_div(Lk, block_size);
  if (bh * std::max(Lq, Lk) * D > (int64_t(1) << 46)) return fail(SPARSTAR_ERR_INVALID_ARG, "tensor too large");
  if (bh * (nq + nk) >= (int64_t(1) << 31) || bh * nq * nk >= (int64_t(1) << 40))
    return fail(SPARSTAR_ERR_INVALID_ARG, "too many blocks");
  return SPARSTAR_OK;
}

// Eq. (5), with the reading that a product within 1e-9 * max(1, n_sel) of an
// integer counts as that integer.
int budget_k(double rho, int64_t n_sel) {
  const double p = rho * double(n_sel);
  const double r = nearbyint(p);
  const double c = fabs(p - r) <= 1e-9 * double(std::max<int64_t>(1, n_sel)) ? r : ceil(p);
  const int64_t k = std::min<int64_t>(n_sel, std::max<int64_t>(1, int64_t(c)));
  return int(k);
}

}  // namespace


// Keep set (Eq. 3), selectable count (Eq. 4) and per-head budgets (Eq. 5).
struct Plan {
  sparstar::KeepBlocks keep;
  sparstar::HeadBudgets budgets;
  int64_t n_keep_blocks, n_sel;
  int max_k;
};

static int plan_selection(int H, int64_t Lk, int block_size, const double* budget, int n_budget,
                          const sparstar_range* keep, int n_keep, Plan& plan) {
  using namespace sparstar;
  if (H < 1 || H > SPARSTAR_MAX_HEADS) return fail(SPARSTAR_ERR_UNSUPPORTED, "H must be in [1, %d] (got %d)",
                                                   SPARSTAR_MAX_HEADS, H);
  if (!budget) return fail(SPARSTAR_ERR_INVALID_ARG, "budget must be non-null");
  if (n_budget != 1 && n_budget != H)
    return fail(SPARSTAR_ERR_INVALID_ARG, "n_budget must be 1 or H (got %d, H=%d)", n_budget, H);
  for (int i = 0; i < n_budget; ++i)
    if (!(budget[i] >= 0.0 && budget[i] <= 1.0))
      return fail(SPARSTAR_ERR_INVALID_ARG, "budget[%d] = %g is outside [0, 1]", i, budget[i]);
  if (n_keep < 0 || n_keep > SPARSTAR_MAX_KEEP_RANGES)
    return fail(SPARSTAR_ERR_INVALID_ARG, "n_keep must be in [0, %d] (got %d)", SPARSTAR_MAX_KEEP_RANGES, n_keep);
  if (n_keep > 0 && !keep) return fail(SPARSTAR_ERR_INVALID_ARG, "keep is null with n_keep = %d", n_keep);
  for (int i = 0; i < n_keep; ++i)
    if (keep[i].begin < 0 || keep[i].begin > keep[i].end || keep[i].end > Lk)
      return fail(SPARSTAR_ERR_INVALID_ARG, "keep[%d] = [%lld, %lld) is not inside [0, Lk=%lld]", i,
                  (long long)keep[i].begin, (long long)keep[i].end, (long long)Lk);
  const int64_t nk = ceil_div(Lk, block_size);
  // Block j meets [begin, end) iff floor(begin/b) <= j < ceil(end/b).
  std::vector<char> is_keep(size_t(nk), 0);
  for (int i = 0; i < n_keep; ++i) {
    if (keep[i].begin == keep[i].end) continue;
    const int64_t j0 = keep[i].begin / block_size, j1 = ceil_div(keep[i].end, block_size);
    for (int64_t j = j0; j < j1; ++j) is_keep[size_t(j)] = 1;
  }
  plan.keep = KeepBlocks{};
  plan.n_keep_blocks = 0;
  for (int64_t j = 0; j < nk;) {
    if (!is_keep[size_t(j)]) { ++j; continue; }
    int64_t e = j;
    while (e < nk && is_keep[size_t(e)]) ++e;
    // merged intervals never outnumber the (<= kMaxKeep) input ranges
    plan.keep.begin[plan.keep.n] = int(j);
    plan.keep.end[plan.keep.n] = int(e);
    ++plan.keep.n;
    plan.n_keep_blocks += e - j;
    j = e;
  }
  plan.n_sel = nk - plan.n_keep_blocks;
  plan.budgets = HeadBudgets{};
  plan.max_k = 0;
  for (int h = 0; h < H; ++h) {
    plan.budgets.k[h] = budget_k(budget[n_budget == 1 ? 0 : h], plan.n_sel);
    plan.max_k = std::max(plan.max_k, plan.budgets.k[h]);
  }
  return SPARSTAR_OK;
}

extern "C" int64_t sparstar_kv_stride(int H, int64_t Lk, int block_size, const double* budget, int n_budget,
                                      const sparstar_range* keep, int n_keep) {
  if (Lk < 1 || Lk > (int64_t(1) << 30)) return fail(SPARSTAR_ERR_INVALID_ARG, "Lk must be in [1, 2^30]");
  if (block_size != 64 && block_size != 128)
    return fail(SPARSTAR_ERR_UNSUPPORTED, "block size %d not supported (64 or 128)", block_size);
  Plan plan;
  if (int rc = plan_selection(H, Lk, block_size, budget, n_budget, keep, n_keep, plan)) return rc;
  ok();
  return plan.n_keep_blocks + plan.max_k;
}

extern "C" int sparstar_clip_keep_ranges(int clip, sparstar_range text, sparstar_range ref, sparstar_range* out,
                                         int cap) {
  if (clip < 1) return fail(SPARSTAR_ERR_INVALID_ARG, "clip index starts at 1 (got %d)", clip);
  if (text.begin < 0 || text.begin > text.end || ref.begin < 0 || ref.begin > ref.end)
    return fail(SPARSTAR_ERR_INVALID_ARG, "ranges need 0 <= begin <= end");
  const int n = clip == 1 ? 2 : 1;  // Eq. 3: text and reference for clip 1, text only after
  if (!out || cap < n) return fail(SPARSTAR_ERR_INVALID_ARG, "out needs room for %d ranges", n);
  out[0] = text;
  if (n == 2) out[1] = ref;
  ok();
  return n;
}

extern "C" int sparstar_scale_densities(const int64_t* scale_lq, int n_scales, const double* finest_rho, int n_finest,
                                        double* rho_out) {
  if (n_scales < 0 || n_finest < 0 || n_finest > n_scales)
    return fail(SPARSTAR_ERR_INVALID_ARG, "need 0 <= n_finest <= n_scales (got %d, %d)", n_finest, n_scales);
  if (n_scales > 0 && (!scale_lq || !rho_out)) return fail(SPARSTAR_ERR_INVALID_ARG, "null scale arrays");
  if (n_finest > 0 && !finest_rho) return fail(SPARSTAR_ERR_INVALID_ARG, "null densities");
  // lookup table query length -> density, from the finest scales
  std::vector<std::pair<int64_t, double>> table;
  for (int i = 0; i < n_finest; ++i) {
    const double rho = finest_rho[i];
    if (!(rho >= 0.0 && rho <= 1.0)) return fail(SPARSTAR_ERR_INVALID_ARG, "density %g outside [0, 1]", rho);
    const int64_t lq = scale_lq[n_scales - n_finest + i];
    bool found = false;
    for (const auto& e : table)
      if (e.first == lq) {
        if (e.second != rho)
          return fail(SPARSTAR_ERR_INVALID_ARG, "scales of %lld tokens given densities %g and %g", (long long)lq,
                      e.second, rho);
        found = true;
      }
    if (!found) table.push_back({lq, rho});
  }
  for (int s = 0; s < n_scales; ++s) {
    rho_out[s] = -1.0;
    for (const auto& e : table)
      if (e.first == scale_lq[s]) rho_out[s] = e.second;
  }
  return ok();
}

extern "C" const char* sparstar_last_error(void) { return g_error.c_str(); }

// Selector workspace: the pooled blocks split into fp16 hi and lo parts (4 D
// bytes per block), their power-of-two scales, then S with its rows padded to
// whole 128-byte lines (an S passed in by the caller keeps rows of n_k).
struct WsLayout {
  size_t q_bar, k_bar, q_exp, k_exp, s, total;
};

static int64_t s_row_stride(int64_t nk) { return (nk + 31) / 32 * 32; }

static WsLayout ws_layout(int B, int H, int64_t Lq, int64_t Lk, int D, int block_size) {
  const int64_t bh = int64_t(B) * H;
  const int64_t nq = ceil_div(Lq, block_size), nk = ceil_div(Lk, block_size);
  WsLayout w;
  w.q_bar = 0;
  w.k_bar = align256(size_t(bh * nq * D) * 4);
  w.q_exp = w.k_bar + align256(size_t(bh * nk * D) * 4);
  w.k_exp = w.q_exp + align256(size_t(bh * nq) * sizeof(int32_t));
  w.s = w.k_exp + align256(size_t(bh * nk) * sizeof(int32_t));
  w.total = w.s + align256(size_t(bh * nq * s_row_stride(nk)) * sizeof(float));
  return w;
}

extern "C" size_t sparstar_score_workspace_bytes(int B, int H, int64_t Lq, int64_t Lk, int D, int block_size) {
  if (check_sizes(B, H, Lq, Lk, D, block_size) != SPARSTAR_OK) return 0;
  return ws_layout(B, H, Lq, Lk, D, block_size).total;
}

// s_outside: S may live in the caller's `scores` output instead of the
// workspace, which then only needs the pooled blocks.  validate_only: check
// every argument (the workspace by its size only) and launch nothing.
static int score_common(const void* q, const void* k, int B, int H, int64_t Lq, int64_t Lk, int D, int block_size,
                        const double* budget, int n_budget, const sparstar_range* keep, int n_keep,
                        int32_t* kv_num_blocks, int32_t* kv_indices, int kv_stride, float* scores, void* workspace,
                        size_t workspace_bytes, void* stream, bool fused, bool s_outside = false,
                        bool validate_only = false) {
  using namespace sparstar;
  if (int rc = check_sizes(B, H, Lq, Lk, D, block_size)) return rc;
  // With Lq == 0 there is nothing to read or write on the query side.
  if (!k || (Lq > 0 && !q)) return fail(SPARSTAR_ERR_INVALID_ARG, "q and k must be non-null");
  if (!aligned16(q) || !aligned16(k)) return fail(SPARSTAR_ERR_INVALID_ARG, "q and k must be 16-byte aligned");
  if (Lq > 0 && (!kv_num_blocks || !kv_indices))
    return fail(SPARSTAR_ERR_INVALID_ARG, "kv_num_blocks and kv_indices must be non-null");
  Plan plan;
  if (int rc = plan_selection(H, Lk, block_size, budget, n_budget, keep, n_keep, plan)) return rc;
  const int64_t nq = ceil_div(Lq, block_size), nk = ceil_div(Lk, block_size);
  const KeepBlocks& kb = plan.keep;
  const HeadBudgets& hb = plan.budgets;
  const int64_t n_keep_blocks = plan.n_keep_blocks, n_sel = plan.n_sel;
  const int max_k = plan.max_k;
  if (int64_t(kv_stride) < n_keep_blocks + max_k || kv_stride < 1)
    return fail(SPARSTAR_ERR_INVALID_ARG, "kv_stride %d < |J_keep| + max k = %lld", kv_stride,
                (long long)(n_keep_blocks + max_k));
  const WsLayout wl = ws_layout(B, H, Lq, Lk, D, block_size);
  const size_t need = (s_outside && scores) ? wl.s : wl.total;
  if (!validate_only) {
    if (!workspace) return fail(SPARSTAR_ERR_WORKSPACE, "workspace is null");
    if ((reinterpret_cast<uintptr_t>(workspace) & 255u) != 0)
      return fail(SPARSTAR_ERR_WORKSPACE, "workspace must be 256-byte aligned");
  }
  if (workspace_bytes < need)
    return fail(SPARSTAR_ERR_WORKSPACE, "workspace of %zu bytes < %zu required", workspace_bytes, need);
  if (scores && (reinterpret_cast<uintptr_t>(scores) & 3u) != 0)
    return fail(SPARSTAR_ERR_INVALID_ARG, "scores must be 4-byte aligned");
  if (fused && nk > kFusedMaxBlocks)
    return fail(SPARSTAR_ERR_UNSUPPORTED, "fused scores and selection take at most %d key blocks (got %lld)",
                kFusedMaxBlocks, (long long)nk);
  if (nq == 0 || validate_only) return ok();

  const int bh = B * H;
  char* ws = static_cast<char*>(workspace);
  uint16_t* q_bar = reinterpret_cast<uint16_t*>(ws + wl.q_bar);
  uint16_t* k_bar = reinterpret_cast<uint16_t*>(ws + wl.k_bar);
  int32_t* q_exp = reinterpret_cast<int32_t*>(ws + wl.q_exp);
  int32_t* k_exp = reinterpret_cast<int32_t*>(ws + wl.k_exp);
  float* s = scores ? scores : reinterpret_cast<float*>(ws + wl.s);
  const int s_stride = int(scores ? nk : s_row_stride(nk));
  hipStream_t st = static_cast<hipStream_t>(stream);

  PoolArgs pa{static_cast<const uint16_t*>(q), static_cast<const uint16_t*>(k), q_bar, k_bar, q_exp, k_exp, Lq, Lk,
              bh, int(nq), int(nk), kb};
  hipError_t e = launch_pool(pa, D, block_size, st);
  if (e != hipSuccess) return fail(SPARSTAR_ERR_HIP, "pool launch: %s", hipGetErrorString(e));
  const float tau = float(1.0 / sqrt(double(D)));
  if (fused) {
    // scores and selection in one kernel, S kept in LDS
    ScoreSelectArgs fa{q_bar, k_bar, q_exp, k_exp, kv_num_blocks, kv_indices, bh, int(nq), int(nk), H, kv_stride, D,
                       int(n_sel), tau, kb, hb};
    e = launch_score_select(fa, st);
    if (e != hipSuccess) return fail(SPARSTAR_ERR_HIP, "score/select launch: %s", hipGetErrorString(e));
    return ok();
  }
  if (n_sel > 0) {
    ScoreArgs sa{q_bar, k_bar, q_exp, k_exp, s, bh, int(nq), int(nk), s_stride, tau, kb};
    e = launch_score(sa, D, st);
    if (e != hipSuccess) return fail(SPARSTAR_ERR_HIP, "score launch: %s", hipGetErrorString(e));
  }
  SelectArgs sel{s, kv_num_blocks, kv_indices, int64_t(bh) * nq, int(nq), int(nk), H, kv_stride, int(n_sel),
                 s_stride, kb, hb};
  e = launch_select(sel, st);
  if (e != hipSuccess) return fail(SPARSTAR_ERR_HIP, "select launch: %s", hipGetErrorString(e));
  return ok();
}

extern "C" int sparstar_score_blocks(const void* q, const void* k, int B, int H, int64_t Lq, int64_t Lk, int D,
                                     int block_size, const double* budget, int n_budget, const sparstar_range* keep,
                                     int n_keep, int32_t* kv_num_blocks, int32_t* kv_indices, int kv_stride,
                                     float* scores, void* workspace, size_t workspace_bytes, void* stream) {
  return score_common(q, k, B, H, Lq, Lk, D, block_size, budget, n_budget, keep, n_keep, kv_num_blocks, kv_indices,
                      kv_stride, scores, workspace, workspace_bytes, stream, false);
}

namespace sparstar {

int score_blocks_internal(const void* q, const void* k, int B, int H, int64_t Lq, int64_t Lk, int D, int block_size,
                          const double* budget, int n_budget, const sparstar_range* keep, int n_keep,
                          int32_t* kv_num_blocks, int32_t* kv_indices, int kv_stride, float* scores, void* workspace,
                          size_t workspace_bytes, void* stream, bool validate_only) {
  return score_common(q, k, B, H, Lq, Lk, D, block_size, budget, n_budget, keep, n_keep, kv_num_blocks, kv_indices,
                      kv_stride, scores, workspace, workspace_bytes, stream, false, true, validate_only);
}

int report_error(int code, const char* msg) { return fail(code, "%s", msg); }

size_t score_pooled_bytes(int B, int H, int64_t Lq, int64_t Lk, int D, int block_size) {
  if (check_sizes(B, H, Lq, Lk, D, block_size) != SPARSTAR_OK) return 0;
  return ws_layout(B, H, Lq, Lk, D, block_size).s;
}

}  // namespace sparstar

extern "C" int sparstar_score_blocks_fused(const void* q, const void* k, int B, int H, int64_t Lq, int64_t Lk, int D,
                                           int block_size, const double* budget, int n_budget,
                                           const sparstar_range* keep, int n_keep, int32_t* kv_num_blocks,
                                           int32_t* kv_indices, int kv_stride, void* workspace,
                                           size_t workspace_bytes, void* stream) {
  return score_common(q, k, B, H, Lq, Lk, D, block_size, budget, n_budget, keep, n_keep, kv_num_blocks, kv_indices,
                      kv_stride, nullptr, workspace, workspace_bytes, stream, true);
}

size_t sparstar::attn_workspace_bytes(int64_t bh, int64_t n_q, int64_t n_k, int d, int block) {
  if (n_k < kSplits) return 0;  // fewer key blocks than ranges: single pass
  const int64_t rows = bh * n_q * kSplits * block;
  return attn_partial_o_bytes(rows, d) + size_t(rows) * 4 * sizeof(float);
}

extern "C" size_t sparstar_attn_workspace_bytes(int B, int H, int64_t Lq, int64_t Lk, int D, int block_size) {
  if (check_sizes(B, H, Lq, Lk, D, block_size) != SPARSTAR_OK) return 0;
  return sparstar::attn_workspace_bytes(int64_t(B) * H, ceil_div(Lq, block_size), ceil_div(Lk, block_size), D,
                                        block_size);
}

static int attn_common(const void* q, const void* k, const void* v, int B, int H, int64_t Lq, int64_t Lk, int D,
                       int block_size, const int32_t* kv_num_blocks, const int32_t* kv_indices, int kv_stride,
                       float softmax_scale, void* o, float* lse, void* workspace, size_t workspace_bytes,
                       void* stream, bool dense) {
  using namespace sparstar;
  if (int rc = check_sizes(B, H, Lq, Lk, D, block_size)) return rc;
  if (!k || !v || (Lq > 0 && (!q || !o))) return fail(SPARSTAR_ERR_INVALID_ARG, "q, k, v and o must be non-null");
  if (!aligned16(q) || !aligned16(k) || !aligned16(v) || !aligned16(o))
    return fail(SPARSTAR_ERR_INVALID_ARG, "q, k, v and o must be 16-byte aligned");
  if (lse && (reinterpret_cast<uintptr_t>(lse) & 3u) != 0)
    return fail(SPARSTAR_ERR_INVALID_ARG, "lse must be 4-byte aligned");
  if (!dense && Lq > 0) {
    if (!kv_num_blocks || !kv_indices)
      return fail(SPARSTAR_ERR_INVALID_ARG, "kv_num_blocks and kv_indices must be non-null");
    if (kv_stride < 1) return fail(SPARSTAR_ERR_INVALID_ARG, "kv_stride must be >= 1 (got %d)", kv_stride);
  }
  if (!(softmax_scale == softmax_scale) || isinf(softmax_scale))
    return fail(SPARSTAR_ERR_INVALID_ARG, "softmax_scale must be finite");
  const int64_t nq = ceil_div(Lq, block_size), nk = ceil_div(Lk, block_size);
  const size_t need = attn_workspace_bytes(int64_t(B) * H, nq, nk, D, block_size);
  const bool split = workspace != nullptr && need > 0;
  if (split) {
    if ((reinterpret_cast<uintptr_t>(workspace) & 255u) != 0)
      return fail(SPARSTAR_ERR_WORKSPACE, "workspace must be 256-byte aligned");
    if (workspace_bytes < need)
      return fail(SPARSTAR_ERR_WORKSPACE, "workspace of %zu bytes < %zu required", workspace_bytes, need);
  }
  if (nq == 0) return ok();
  const double sc = softmax_scale > 0.f ? double(softmax_scale) : 1.0 / sqrt(double(D));
  AttnArgs a{};
  a.q = static_cast<const uint16_t*>(q);
  a.k = static_cast<const uint16_t*>(k);
  a.v = static_cast<const uint16_t*>(v);
  a.o = static_cast<uint16_t*>(o);
  a.lse = lse;
  a.kv_num_blocks = kv_num_blocks;
  a.kv_indices = kv_indices;
  a.lq = Lq;
  a.lk = Lk;
  a.bh = B * H;
  a.n_q = int(nq);
  a.n_k = int(nk);
  a.stride = dense ? 0 : kv_stride;
  a.scale_log2 = float(sc * 1.4426950408889634074);
  if (split) {
    const int64_t rows = int64_t(B) * H * nq * kSplits * block_size;
    char* ws = static_cast<char*>(workspace);
    a.part_o = reinterpret_cast<uint16_t*>(ws);
    a.part_meta = reinterpret_cast<float*>(ws + attn_partial_o_bytes(rows, D));
    // The dense call lists every key block, so it takes the rule of a full list.
    const int64_t list_keys = (dense ? nk : int64_t(kv_stride)) * block_size;
    a.n_splits = list_keys < kFewRangesBelowKeys ? 8 : kSplits;
  }
  hipError_t e = launch_attn(a, D, block_size, dense, static_cast<hipStream_t>(stream));
  if (e != hipSuccess) return fail(SPARSTAR_ERR_HIP, "attention launch: %s", hipGetErrorString(e));
  return ok();
}

extern "C" int sparstar_sparse_attn_fwd(const void* q, const void* k, const void* v, int B, int H, int64_t Lq,
                                        int64_t Lk, int D, int block_size, const int32_t* kv_num_blocks,
                                        const int32_t* kv_indices, int kv_stride, float softmax_scale, void* o,
                                        float* lse, void* workspace, size_t workspace_bytes, void* stream) {
  return attn_common(q, k, v, B, H, Lq, Lk, D, block_size, kv_num_blocks, kv_indices, kv_stride, softmax_scale, o,
                     lse, workspace, workspace_bytes, stream, false);
}

extern "C" int sparstar_dense_attn_fwd(const void* q, const void* k, const void* v, int B, int H, int64_t Lq,
                                       int64_t Lk, int D, int block_size, float softmax_scale, void* o, float* lse,
                                       void* workspace, size_t workspace_bytes, void* stream) {
  return attn_common(q, k, v, B, H, Lq, Lk, D, block_size, nullptr, nullptr, 0, softmax_scale, o, lse, workspace,
                     workspace_bytes, stream, true);
}

extern "C" int sparstar_retained_mass(const float* lse_sel, const float* lse_all, int64_t n, float* mass,
                                      void* stream) {
  if (n < 0) return fail(SPARSTAR_ERR_INVALID_ARG, "n must be >= 0 (got %lld)", (long long)n);
  if (n > 0 && (!lse_sel || !lse_all || !mass))
    return fail(SPARSTAR_ERR_INVALID_ARG, "lse_sel, lse_all and mass must be non-null");
  const uintptr_t mis = reinterpret_cast<uintptr_t>(lse_sel) | reinterpret_cast<uintptr_t>(lse_all) |
                        reinterpret_cast<uintptr_t>(mass);
  if (mis & 3u) return fail(SPARSTAR_ERR_INVALID_ARG, "lse_sel, lse_all and mass must be 4-byte aligned");
  hipError_t e = sparstar::launch_retained_mass(lse_sel, lse_all, n, mass, static_cast<hipStream_t>(stream));
  if (e != hipSuccess) return fail(SPARSTAR_ERR_HIP, "retained-mass launch: %s", hipGetErrorString(e));
  return ok();
}

static_assert(sparstar::kTopkMaxRows == SPARSTAR_MAX_MASS_ROWS, "sampled-row limit");
static_assert(sparstar::kFusedMaxBlocks == SPARSTAR_FUSED_MAX_BLOCKS, "fused row limit");

static int check_topk_sizes(int B, int H, int64_t Lk, int n_rows) {
  if (B < 1 || H < 1 || int64_t(B) * H > 65535)
    return fail(SPARSTAR_ERR_INVALID_ARG, "need B, H >= 1 and B * H <= 65535 (got B=%d, H=%d)", B, H);
  if (Lk < 1 || Lk > (int64_t(1) << 30)) return fail(SPARSTAR_ERR_INVALID_ARG, "Lk must be in [1, 2^30]");
  if (n_rows < 1 || n_rows > SPARSTAR_MAX_MASS_ROWS)
    return fail(SPARSTAR_ERR_INVALID_ARG, "n_rows must be in [1, %d] (got %d)", SPARSTAR_MAX_MASS_ROWS, n_rows);
  if (int64_t(B) * H * n_rows * Lk > (int64_t(1) << 40)) return fail(SPARSTAR_ERR_INVALID_ARG, "too many logits");
  return SPARSTAR_OK;
}

extern "C" size_t sparstar_token_topk_workspace_bytes(int B, int H, int64_t Lk, int n_rows) {
  if (check_topk_sizes(B, H, Lk, n_rows) != SPARSTAR_OK) return 0;
  return size_t(int64_t(B) * H * n_rows * Lk) * sizeof(float);
}

extern "C" int sparstar_token_topk_mass(const void* q, const void* k, int B, int H, int64_t Lq, int64_t Lk, int D,
                                        const int64_t* rows, int n_rows, const int32_t* n_tokens,
                                        const float* lse_all, float softmax_scale, float* mass, void* workspace,
                                        size_t workspace_bytes, void* stream) {
  using namespace sparstar;
  if (int rc = check_topk_sizes(B, H, Lk, n_rows)) return rc;
  if (Lq < 1 || Lq > (int64_t(1) << 30)) return fail(SPARSTAR_ERR_INVALID_ARG, "Lq must be in [1, 2^30]");
  if (D != 64 && D != 128) return fail(SPARSTAR_ERR_UNSUPPORTED, "head dim %d not supported (64 or 128)", D);
  if (int64_t(B) * H * std::max(Lq, Lk) * D > (int64_t(1) << 46))
    return fail(SPARSTAR_ERR_INVALID_ARG, "tensor too large");
  if (!q || !k || !rows || !n_tokens || !lse_all || !mass)
    return fail(SPARSTAR_ERR_INVALID_ARG, "q, k, rows, n_tokens, lse_all and mass must be non-null");
  if (!aligned16(q) || !aligned16(k)) return fail(SPARSTAR_ERR_INVALID_ARG, "q and k must be 16-byte aligned");
  const uintptr_t mis = reinterpret_cast<uintptr_t>(n_tokens) | reinterpret_cast<uintptr_t>(lse_all) |
                        reinterpret_cast<uintptr_t>(mass);
  if (mis & 3u) return fail(SPARSTAR_ERR_INVALID_ARG, "n_tokens, lse_all and mass must be 4-byte aligned");
  for (int r = 0; r < n_rows; ++r)
    if (rows[r] < 0 || rows[r] >= Lq)
      return fail(SPARSTAR_ERR_INVALID_ARG, "rows[%d] = %lld is outside [0, Lq=%lld)", r, (long long)rows[r],
                  (long long)Lq);
  if (!(softmax_scale == softmax_scale) || isinf(softmax_scale))
    return fail(SPARSTAR_ERR_INVALID_ARG, "softmax_scale must be finite");
  const size_t need = sparstar_token_topk_workspace_bytes(B, H, Lk, n_rows);
  if (!workspace) return fail(SPARSTAR_ERR_WORKSPACE, "workspace is null");
  if (reinterpret_cast<uintptr_t>(workspace) & 3u)
    return fail(SPARSTAR_ERR_WORKSPACE, "workspace must be 4-byte aligned");
  if (workspace_bytes < need)
    return fail(SPARSTAR_ERR_WORKSPACE, "workspace of %zu bytes < %zu required", workspace_bytes, need);
  TopkArgs a{};
  a.q = static_cast<const uint16_t*>(q);
  a.k = static_cast<const uint16_t*>(k);
  a.n_tokens = n_tokens;
  a.lse_all = lse_all;
  a.scores = static_cast<float*>(workspace);
  a.mass = mass;
  a.lq = Lq;
  a.lk = Lk;
  a.bh = int64_t(B) * H;
  a.n_rows = n_rows;
  for (int r = 0; r < n_rows; ++r) a.rows[r] = rows[r];
  a.scale = float(softmax_scale > 0.f ? double(softmax_scale) : 1.0 / sqrt(double(D)));
  hipError_t e = launch_topk_mass(a, D, static_cast<hipStream_t>(stream));
  if (e != hipSuccess) return fail(SPARSTAR_ERR_HIP, "token top-n mass launch: %s", hipGetErrorString(e));
  return ok();
}
