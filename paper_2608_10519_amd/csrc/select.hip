// Retained support A_i = J_keep  U  TopKIdx_{j in J_sel}(S_ij, k_h)  (Eq. 6),
// written as the forward-only block mask of Section 5.3: kv_num_blocks and the
// ascending kv_indices row.
//
// One wavefront per score row.  The k-th largest selectable score is found
// exactly by a 4-pass radix select (8 bits per pass) on order-preserving 32-bit
// keys, with the digit histogram in LDS.  Equal scores are broken toward the
// lower block index.  A final pass walks the row in ascending block order and
// compacts {forced} U {selected} with wave ballots, so the list comes out
// sorted without a sort.
#include "device_common.h"

namespace sparstar {

constexpr int kSelWaves = 4;

// fp32 -> unsigned key with the same order (-0 is folded onto +0).
__device__ __forceinline__ uint32_t order_key(float f) {
  uint32_t u = __float_as_uint(f == 0.f ? 0.f : f);
  return (u & 0x80000000u) ? ~u : (u | 0x80000000u);
}

__device__ __forceinline__ int lanes_below(uint64_t mask) {
  return __builtin_amdgcn_mbcnt_hi((uint32_t)(mask >> 32), __builtin_amdgcn_mbcnt_lo((uint32_t)mask, 0u));
}

__global__ __launch_bounds__(64 * kSelWaves) void select_kernel(SelectArgs a) {
  __shared__ uint32_t hist[kSelWaves][256];
  const int wave = threadIdx.x / 64, lane = threadIdx.x % 64;
  const int64_t row = (int64_t)blockIdx.x * kSelWaves + wave;
  const bool live = row < a.rows;  // every wave runs the same loop trip counts
  const int64_t r = live ? row : 0;
  const int h = (int)((r / a.n_q) % a.heads);
  const int kk = a.budget.k[h];
  const float* s = a.s + r * a.n_k;
  const int chunks = (a.n_k + 63) / 64;

  uint32_t prefix = 0, mask = 0;
  uint32_t rem = (uint32_t)kk;
  for (int shift = 24; shift >= 0; shift -= 8) {
#pragma unroll
    for (int e = 0; e < 4; ++e) hist[wave][lane * 4 + e] = 0;
    __syncthreads();
    for (int c = 0; c < chunks; ++c) {
      const int j = c * 64 + lane;
      if (j < a.n_k && !keep_block(a.keep, j)) {
        const uint32_t key = order_key(s[j]);
        if ((key & mask) == prefix) atomicAdd(&hist[wave][(key >> shift) & 255u], 1u);
      }
    }
    __syncthreads();
    // The digit d of the rem-th largest key: count(bins > d) < rem <= count(bins >= d).
    uint32_t cnt[4], own = 0;
#pragma unroll
    for (int e = 0; e < 4; ++e) { cnt[e] = hist[wave][lane * 4 + e]; own += cnt[e]; }
    uint32_t suffix = own;  // sum over lanes >= lane
#pragma unroll
    for (int off = 1; off < 64; off <<= 1) {
      const uint32_t o = __shfl_down(suffix, off, 64);
      if (lane + off < 64) suffix += o;
    }
    uint32_t above = suffix - own;  // keys in bins above this lane's four
    int found = -1;
    uint32_t new_rem = 0;
#pragma unroll
    for (int e = 3; e >= 0; --e) {
      if (found < 0 && rem > 0 && above < rem && above + cnt[e] >= rem) {
        found = lane * 4 + e;
        new_rem = rem - above;
      }
      above += cnt[e];
    }
    const uint64_t who = __ballot(found >= 0);
    if (who != 0) {
      const int src = __builtin_ctzll(who);
      const int digit = __shfl(found, src, 64);
      rem = (uint32_t)__shfl((int)new_rem, src, 64);
      prefix |= (uint32_t)digit << shift;
      mask |= 255u << shift;
    }
    __syncthreads();
  }
  // kk == 0 (no selectable block): select nothing.
  const uint32_t thr = kk > 0 ? prefix : 0xffffffffu;
  const uint32_t take_ties = kk > 0 ? rem : 0u;

  if (!live) return;
  int32_t* out = a.kv_indices + r * a.stride;
  int pos = 0;
  uint32_t ties = 0;
  for (int c = 0; c < chunks; ++c) {
    const int j = c * 64 + lane;
    const bool valid = j < a.n_k;
    const bool forced = valid && keep_block(a.keep, j);
    const bool cand = valid && !forced;
    const uint32_t key = cand ? order_key(s[j]) : 0u;
    const bool tie = cand && key == thr;
    const uint64_t tie_mask = __ballot(tie);
    const uint32_t tie_rank = ties + (uint32_t)lanes_below(tie_mask);
    const bool take = forced || (cand && (key > thr || (tie && tie_rank < take_ties)));
    const uint64_t take_mask = __ballot(take);
    if (take) out[pos + lanes_below(take_mask)] = j;
    pos += __popcll(take_mask);
    ties += (uint32_t)__popcll(tie_mask);
  }
  if (lane == 0) a.kv_num_blocks[r] = pos;
}

// Rows of up to kSelCachedMaxBlocks blocks: each wave reads its row once,
// keeps the order keys in LDS (forced blocks as 0, corrected for in the
// counts) and walks it four keys per lane per LDS read in all five passes.
constexpr int kSelCachedMaxBlocks = 3584;  // 4 waves x 3584 x 4 B = 56 KB (+ 4 KB of histograms)

// sum of v over the lanes below this one, for 0 <= v <= 7
__device__ __forceinline__ uint32_t lanes_below_sum(uint32_t v) {
  uint32_t r = 0;
#pragma unroll
  for (int b = 0; b < 3; ++b) r += (uint32_t)lanes_below(__ballot((v >> b) & 1u)) << b;
  return r;
}

__global__ __launch_bounds__(64 * kSelWaves) void select_cached_kernel(SelectArgs a) {
  __shared__ uint32_t hist[kSelWaves][256];
  extern __shared__ uint4 row_keys[];  // [kSelWaves][quads] order keys, 4 per entry
  const int wave = threadIdx.x / 64, lane = threadIdx.x % 64;
  const int64_t row = (int64_t)blockIdx.x * kSelWaves + wave;
  const bool live = row < a.rows;  // every wave runs the same loop trip counts
  const int64_t r = live ? row : 0;
  const int h = (int)((r / a.n_q) % a.heads);
  const int kk = a.budget.k[h];
  const float* s = a.s + r * a.n_k;
  const int quads = (a.n_k + 3) / 4;
  const int rounds = (quads + 63) / 64;  // 256 keys per round
  uint4* const keys = row_keys + (size_t)wave * quads;

  // fill: key of block j at keys[j / 4].(j % 4); forced and padding blocks 0
  uint32_t n_forced = 0;
  for (int q = lane; q < quads; q += 64) {
    uint32_t k4[4];
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      const int j = 4 * q + e;
      const bool forced = j < a.n_k && keep_block(a.keep, j);
      k4[e] = (j < a.n_k && !forced) ? order_key(s[j]) : 0u;
      n_forced += forced;
    }
    keys[q] = make_uint4(k4[0], k4[1], k4[2], k4[3]);
  }
  n_forced = (uint32_t)__reduce_add_sync(~0ull, n_forced);

  uint32_t prefix = 0, mask = 0;
  uint32_t rem = (uint32_t)kk;
  for (int shift = 24; shift >= 0; shift -= 8) {
#pragma unroll
    for (int e = 0; e < 4; ++e) hist[wave][lane * 4 + e] = 0;
    __syncthreads();
    for (int c = 0; c < rounds; ++c) {
      const int q = c * 64 + lane;
      if (q < quads) {
        const uint4 v = keys[q];
        const uint32_t k4[4] = {v.x, v.y, v.z, v.w};
#pragma unroll
        for (int e = 0; e < 4; ++e)
          if ((k4[e] & mask) == prefix) atomicAdd(&hist[wave][(k4[e] >> shift) & 255u], 1u);
      }
    }
    __syncthreads();
    // forced blocks and the padding past n_k were counted as key 0
    if (lane == 0 && prefix == 0) hist[wave][0] -= n_forced + (uint32_t)(4 * quads - a.n_k);
    __syncthreads();
    // The digit d of the rem-th largest key: count(bins > d) < rem <= count(bins >= d).
    uint32_t cnt[4], own = 0;
#pragma unroll
    for (int e = 0; e < 4; ++e) { cnt[e] = hist[wave][lane * 4 + e]; own += cnt[e]; }
    uint32_t suffix = own;  // sum over lanes >= lane
#pragma unroll
    for (int off = 1; off < 64; off <<= 1) {
      const uint32_t o = __shfl_down(suffix, off, 64);
      if (lane + off < 64) suffix += o;
    }
    uint32_t above = suffix - own;  // keys in bins above this lane's four
    int found = -1;
    uint32_t new_rem = 0;
#pragma unroll
    for (int e = 3; e >= 0; --e) {
      if (found < 0 && rem > 0 && above < rem && above + cnt[e] >= rem) {
        found = lane * 4 + e;
        new_rem = rem - above;
      }
      above += cnt[e];
    }
    const uint64_t who = __ballot(found >= 0);
    if (who != 0) {
      const int src = __builtin_ctzll(who);
      const int digit = __shfl(found, src, 64);
      rem = (uint32_t)__shfl((int)new_rem, src, 64);
      prefix |= (uint32_t)digit << shift;
      mask |= 255u << shift;
    }
    __syncthreads();
  }
  // kk == 0 (no selectable block): select nothing.
  const uint32_t thr = kk > 0 ? prefix : 0xffffffffu;
  const uint32_t take_ties = kk > 0 ? rem : 0u;

  if (!live) return;
  // compaction in ascending block order: lane L holds blocks 4 (64 c + L) + e,
  // so a block's rank is (lanes below) + (earlier e of the same lane)
  int32_t* out = a.kv_indices + r * a.stride;
  int pos = 0;
  uint32_t ties = 0;
  for (int c = 0; c < rounds; ++c) {
    const int q = c * 64 + lane;
    const uint4 v = q < quads ? keys[q] : make_uint4(0, 0, 0, 0);
    const uint32_t k4[4] = {v.x, v.y, v.z, v.w};
    bool forced[4], cand[4], tie[4];
    uint32_t n_tie = 0;
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      const int j = 4 * q + e;
      const bool valid = j < a.n_k;
      forced[e] = valid && keep_block(a.keep, j);
      cand[e] = valid && !forced[e];
      tie[e] = cand[e] && k4[e] == thr;
      n_tie += tie[e];
    }
    uint32_t tie_rank = ties + lanes_below_sum(n_tie);
    bool take[4];
    uint32_t n_take = 0;
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      take[e] = forced[e] || (cand[e] && (k4[e] > thr || (tie[e] && tie_rank < take_ties)));
      tie_rank += tie[e];
      n_take += take[e];
    }
    uint32_t at = (uint32_t)pos + lanes_below_sum(n_take);
#pragma unroll
    for (int e = 0; e < 4; ++e)
      if (take[e]) out[at++] = 4 * q + e;
    pos += (int)__reduce_add_sync(~0ull, n_take);
    ties += (uint32_t)__reduce_add_sync(~0ull, n_tie);
  }
  if (lane == 0) a.kv_num_blocks[r] = pos;
}

hipError_t launch_select(const SelectArgs& a, hipStream_t stream) {
  const int64_t grid = (a.rows + kSelWaves - 1) / kSelWaves;
  if (grid == 0) return hipSuccess;
  if (a.n_k <= kSelCachedMaxBlocks)
    select_cached_kernel<<<grid, 64 * kSelWaves, (size_t)kSelWaves * ((a.n_k + 3) / 4) * sizeof(uint4), stream>>>(a);
  else
    select_kernel<<<grid, 64 * kSelWaves, 0, stream>>>(a);
  return hipGetLastError();
}

}  // namespace sparstar
