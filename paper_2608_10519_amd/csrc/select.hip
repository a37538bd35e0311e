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

hipError_t launch_select(const SelectArgs& a, hipStream_t stream) {
  const int64_t grid = (a.rows + kSelWaves - 1) / kSelWaves;
  if (grid == 0) return hipSuccess;
  select_kernel<<<grid, 64 * kSelWaves, 0, stream>>>(a);
  return hipGetLastError();
}

}  // namespace sparstar
