// Retained support A_i = J_keep  U  TopKIdx_{j in J_sel}(S_ij, k_h)  (Eq. 6),
// written as the forward-only block mask of Section 5.3: kv_num_blocks and the
// ascending kv_indices row.
//
// One wavefront per score row, on order-preserving 32-bit keys of the fp32
// scores.  Equal scores are broken toward the lower block index.  A final pass
// walks the row in ascending block order and compacts {forced} U {selected}
// with wave ballots, so the list comes out sorted without a sort.
//
// Rows of up to kSelRegMaxBlocks blocks keep their keys in registers (key c of
// lane L is block 64 c + L) and find the k-th largest key bit by bit from the
// top: a candidate threshold t is kept when at least k keys are >= t, counted
// with one compare and one ballot popcount per 64 keys, with no atomics.  The
// search stops early once exactly k keys are >= t.  Longer rows stream from
// memory through a 4-pass radix select (8 bits per pass) with the digit
// histogram in LDS.
#include "device_common.h"

namespace sparstar {

constexpr int kSelWaves = 4;
constexpr int kSelRegMaxBlocks = 3584;  // 56 keys per lane

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

// Forced blocks and blocks past n_k hold key 0, below every real key (the
// smallest order key of a non-NaN float is 0x007fffff), so they never count.
//
// Selection of one row whose keys sit in registers: key[c] of lane L is the key
// of block 64 c + L.  Every lane of the wave calls it.
template <int C>
__device__ __forceinline__ void select_row_regs(const uint32_t (&key)[C], int n_k, int kk, const KeepBlocks& keep,
                                                int lane, int32_t* out, int32_t* num_out) {
  // thr, take_ties: take every candidate with key > thr and the first
  // take_ties candidates (in block order) with key == thr
  uint32_t thr = 0xffffffffu, take_ties = 0;  // kk == 0: nothing selectable
  if (kk > 0) {
    uint32_t t = 0;
    bool exact = false;
    for (int b = 31; b >= 0; --b) {
      const uint32_t tt = t | (1u << b);
      int n = 0;
#pragma unroll
      for (int c = 0; c < C; ++c) n += __builtin_popcountll(__ballot(key[c] >= tt));
      if (n >= kk) {
        t = tt;
        if (n == kk) {
          exact = true;
          break;
        }
      }
    }
    // t >= 1 here: the kk <= n_sel real keys are all >= 1
    if (exact) {
      thr = t - 1;  // the keys >= t are exactly the kk largest
    } else {
      // t is the kk-th largest key; the keys above it are all taken
      int n_gt = 0;
      if (t != 0xffffffffu) {
#pragma unroll
        for (int c = 0; c < C; ++c) n_gt += __builtin_popcountll(__ballot(key[c] > t));
      }
      thr = t;
      take_ties = (uint32_t)(kk - n_gt);
    }
  }
  int pos = 0;
  uint32_t ties = 0;
#pragma unroll
  for (int c = 0; c < C; ++c) {
    if (64 * c >= n_k) break;
    const int j = 64 * c + lane;
    const bool valid = j < n_k;
    const bool forced = valid && keep_block(keep, j);
    const bool cand = valid && !forced;
    const bool tie = cand && key[c] == thr;
    const uint64_t tie_mask = __ballot(tie);
    const uint32_t tie_rank = ties + (uint32_t)lanes_below(tie_mask);
    const bool take = forced || (cand && (key[c] > thr || (tie && tie_rank < take_ties)));
    const uint64_t take_mask = __ballot(take);
    if (take) out[pos + lanes_below(take_mask)] = j;
    pos += __popcll(take_mask);
    ties += (uint32_t)__popcll(tie_mask);
  }
  if (lane == 0) *num_out = pos;
}

// Rows of up to 64 C blocks: one wave per row reads its row of S straight
// into registers (coalesced, 256 bytes per load).
template <int C>
__global__ __launch_bounds__(64 * kSelWaves) void select_reg_kernel(SelectArgs a) {
  const int wave = threadIdx.x / 64, lane = threadIdx.x % 64;
  const int64_t row = (int64_t)blockIdx.x * kSelWaves + wave;
  if (row >= a.rows) return;  // wave-uniform; no barrier below
  const int h = (int)((row / a.n_q) % a.heads);
  const float* s = a.s + row * a.n_k;
  // all loads first (in bounds, independent), then the keys
  float sv[C];
#pragma unroll
  for (int c = 0; c < C; ++c) {
    const int j = 64 * c + lane;
    sv[c] = s[j < a.n_k ? j : a.n_k - 1];
  }
  uint32_t key[C];
#pragma unroll
  for (int c = 0; c < C; ++c) {
    const int j = 64 * c + lane;
    key[c] = (j < a.n_k && !keep_block(a.keep, j)) ? order_key(sv[c]) : 0u;
  }
  select_row_regs<C>(key, a.n_k, a.budget.k[h], a.keep, lane, a.kv_indices + row * a.stride,
                     a.kv_num_blocks + row);
}

// ---------------------------------------------------------------------------
// Fused scores and selection: S_ij = tau qbar_i . kbar_j (Eq. 2) for the
// kFusedRows query blocks of one head goes into LDS as order keys, and each
// wave then selects one row from there (Eq. 6), so S never leaves the CU.
//
// Scores on v_mfma_f32_16x16x32_f16 over the split pooled rows (hi.hi + hi.lo
// + lo.hi, fp32 accumulation, as the separate score kernel): per 16-key tile,
// A = kbar (16 keys x 32 d), B = qbar^T (32 d x 16 query blocks), C = S^T
// (16 keys x 16 query blocks).  Lane l (g = l / 16) supplies the 8 fp16 values
// d = 32 s + 8 g + i of key (A) or query block (B) l % 16, and receives
// C[4 g + r][l % 16], r = 0..3: four consecutive keys of one row, stored as one
// 16-byte LDS write.  The 16-key tiles go round-robin over the waves.
// Work-groups are numbered so that each XCD runs consecutive groups of query
// blocks (one head's kbar at a time in its L2).
// ---------------------------------------------------------------------------
template <int D, int C>
__global__ __launch_bounds__(64 * kFusedRows) void score_select_kernel(ScoreSelectArgs a) {
  extern __shared__ uint32_t fused_keys[];  // [kFusedRows][row_len] order keys
  const int wave = threadIdx.x / 64, lane = threadIdx.x % 64;
  const int groups = (a.n_q + kFusedRows - 1) / kFusedRows;
  const int64_t wl = xcd_linear(blockIdx.x, (int64_t)gridDim.x);
  const int64_t bh = wl / groups;
  const int i0 = (int)(wl % groups) * kFusedRows;
  const int row_len = (a.n_k + 15) / 16 * 16;  // whole 16-key tiles

  constexpr int KS = D / 32;  // k-steps
  const int n16 = lane % 16, g = lane / 16;
  // B operand: qbar of query block i0 + n16 (hi and lo), zeros past n_q
  const int qi = i0 + n16;
  const bool q_ok = qi < a.n_q;
  const uint16_t* qrow = a.q_bar + (bh * a.n_q + (q_ok ? qi : 0)) * (2 * D);
  // element-wise (a select of whole uint4 values goes through scratch memory)
  auto keep_if = [](bool ok, uint4 v) {
    return make_uint4(ok ? v.x : 0u, ok ? v.y : 0u, ok ? v.z : 0u, ok ? v.w : 0u);
  };
  uint4 qh[KS], ql[KS];
#pragma unroll
  for (int s = 0; s < KS; ++s) {
    const uint4 vh = *reinterpret_cast<const uint4*>(qrow + 32 * s + 8 * g);
    const uint4 vl = *reinterpret_cast<const uint4*>(qrow + D + 32 * s + 8 * g);
    qh[s] = keep_if(q_ok, vh);
    ql[s] = keep_if(q_ok, vl);
  }
  const int eq = q_ok ? a.q_exp[bh * a.n_q + qi] : 0;

  const uint16_t* kb = a.k_bar + bh * (int64_t)a.n_k * (2 * D);
  const int32_t* kexp = a.k_exp + bh * (int64_t)a.n_k;
  const int tiles = row_len / 16;
  // kbar rows of tile kt (zeros past n_k); the next tile's loads are issued
  // before the current tile's MFMAs
  auto load_k = [&](int kt, uint4 (&kh)[KS], uint4 (&kl)[KS]) {
    const int kj = kt * 16 + n16;
    const bool ok = kt < tiles && kj < a.n_k;
    const uint16_t* krow = kb + (int64_t)(ok ? kj : 0) * (2 * D);
#pragma unroll
    for (int s = 0; s < KS; ++s) {
      const uint4 vh = *reinterpret_cast<const uint4*>(krow + 32 * s + 8 * g);
      const uint4 vl = *reinterpret_cast<const uint4*>(krow + D + 32 * s + 8 * g);
      kh[s] = keep_if(ok, vh);
      kl[s] = keep_if(ok, vl);
    }
  };
  uint4 nh[KS], nl[KS];
  load_k(wave, nh, nl);
  for (int kt = wave; kt < tiles; kt += kFusedRows) {
    uint4 kh[KS], kl[KS];
#pragma unroll
    for (int s = 0; s < KS; ++s) {
      kh[s] = nh[s];
      kl[s] = nl[s];
    }
    load_k(kt + kFusedRows, nh, nl);
    f32x4 acc = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int s = 0; s < KS; ++s) {
      const f16x8 ah = __builtin_bit_cast(f16x8, kh[s]), al = __builtin_bit_cast(f16x8, kl[s]);
      const f16x8 bh_ = __builtin_bit_cast(f16x8, qh[s]), bl = __builtin_bit_cast(f16x8, ql[s]);
      acc = __builtin_amdgcn_mfma_f32_16x16x32_f16(ah, bh_, acc, 0, 0, 0);
      acc = __builtin_amdgcn_mfma_f32_16x16x32_f16(ah, bl, acc, 0, 0, 0);
      acc = __builtin_amdgcn_mfma_f32_16x16x32_f16(al, bh_, acc, 0, 0, 0);
    }
    // keys 16 kt + 4 g + r of row n16; forced blocks and blocks past n_k get key 0
    uint32_t k4[4];
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      const int j = 16 * kt + 4 * g + r;
      const bool live = j < a.n_k && !keep_block(a.keep, j);
      k4[r] = live ? order_key(a.tau * __builtin_amdgcn_ldexpf(acc[r], eq + kexp[live ? j : 0])) : 0u;
    }
    *reinterpret_cast<uint4*>(fused_keys + (size_t)n16 * row_len + 16 * kt + 4 * g) =
        make_uint4(k4[0], k4[1], k4[2], k4[3]);
  }
  __syncthreads();

  const int i = i0 + wave;
  if (i >= a.n_q) return;  // wave-uniform; no barrier below
  const uint32_t* rk = fused_keys + (size_t)wave * row_len;
  uint32_t key[C];
#pragma unroll
  for (int c = 0; c < C; ++c) {
    const int j = 64 * c + lane;
    const uint32_t v = rk[j < row_len ? j : row_len - 1];  // in bounds, independent reads
    key[c] = j < a.n_k ? v : 0u;
  }
  const int64_t r = bh * a.n_q + i;
  select_row_regs<C>(key, a.n_k, a.budget.k[(int)(bh % a.heads)], a.keep, lane, a.kv_indices + r * a.stride,
                     a.kv_num_blocks + r);
}

size_t score_select_lds_bytes(int n_k) { return (size_t)kFusedRows * ((n_k + 15) / 16 * 16) * sizeof(uint32_t); }

template <int D>
static hipError_t launch_fused_d(const ScoreSelectArgs& a, int64_t grid, hipStream_t stream) {
  const size_t lds = score_select_lds_bytes(a.n_k);
  if (a.n_k <= 512) score_select_kernel<D, 8><<<grid, 64 * kFusedRows, lds, stream>>>(a);
  else if (a.n_k <= 1024) score_select_kernel<D, 16><<<grid, 64 * kFusedRows, lds, stream>>>(a);
  else if (a.n_k <= 1536) score_select_kernel<D, 24><<<grid, 64 * kFusedRows, lds, stream>>>(a);
  else score_select_kernel<D, 36><<<grid, 64 * kFusedRows, lds, stream>>>(a);
  return hipGetLastError();
}

hipError_t launch_score_select(const ScoreSelectArgs& a, hipStream_t stream) {
  static_assert(kFusedMaxBlocks <= 64 * 36, "fused rows fit the largest register count");
  static_assert((size_t)kFusedRows * kFusedMaxBlocks * 4 <= 160 * 1024, "fused rows fit in LDS");
  const int64_t grid = (int64_t)a.bh * ((a.n_q + kFusedRows - 1) / kFusedRows);
  if (grid == 0) return hipSuccess;
  if (a.n_k > kFusedMaxBlocks) return hipErrorInvalidValue;
  if (a.d == 128) return launch_fused_d<128>(a, grid, stream);
  if (a.d == 64) return launch_fused_d<64>(a, grid, stream);
  return hipErrorInvalidValue;
}

hipError_t launch_select(const SelectArgs& a, hipStream_t stream) {
  const int64_t grid = (a.rows + kSelWaves - 1) / kSelWaves;
  if (grid == 0) return hipSuccess;
  if (a.n_k <= 512) select_reg_kernel<8><<<grid, 64 * kSelWaves, 0, stream>>>(a);
  else if (a.n_k <= 1024) select_reg_kernel<16><<<grid, 64 * kSelWaves, 0, stream>>>(a);
  else if (a.n_k <= 1536) select_reg_kernel<24><<<grid, 64 * kSelWaves, 0, stream>>>(a);
  else if (a.n_k <= 2304) select_reg_kernel<36><<<grid, 64 * kSelWaves, 0, stream>>>(a);
  else if (a.n_k <= kSelRegMaxBlocks) select_reg_kernel<kSelRegMaxBlocks / 64><<<grid, 64 * kSelWaves, 0, stream>>>(a);
  else select_kernel<<<grid, 64 * kSelWaves, 0, stream>>>(a);
  return hipGetLastError();
}

}  // namespace sparstar
