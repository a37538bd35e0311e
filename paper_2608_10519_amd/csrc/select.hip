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

// The same key from the float's bits.
__device__ __forceinline__ uint32_t order_key_bits(uint32_t u) {
  u = u == 0x80000000u ? 0u : u;
  return u ^ ((uint32_t)((int32_t)u >> 31) | 0x80000000u);
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
  const float* s = a.s + r * a.s_stride;
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
// The keys of a row sit in registers: key[c] of lane L is the key of block
// 64 c + L.  Every helper below is called by every lane of the wave.

// Number of keys >= x (wave-uniform).
template <int C>
__device__ __forceinline__ int count_ge(const uint32_t (&key)[C], uint32_t x) {
  int n = 0;
#pragma unroll
  for (int c = 0; c < C; ++c) n += __builtin_popcountll(__ballot(key[c] >= x));
  return n;
}

// Top-down bit search: from t (bits above b0 already fixed, count_ge(t) >= kk),
// the largest t with count_ge(t) >= kk, decided one bit at a time.  It stops
// early when some t has exactly kk keys >= t, and then sets `exact`.
template <int C>
__device__ __forceinline__ uint32_t bit_search(const uint32_t (&key)[C], int kk, uint32_t t, int b0, bool& exact) {
  exact = false;
  for (int b = b0; b >= 0; --b) {
    const uint32_t tt = t | (1u << b);
    const int n = count_ge<C>(key, tt);
    if (n >= kk) {
      t = tt;
      if (n == kk) {
        exact = true;
        break;
      }
    }
  }
  return t;
}

// The selection rule of a row: take every candidate key > thr and the first
// take_ties candidates (in block order) whose key equals thr.
struct SelRule {
  uint32_t thr, take_ties;
};

// The rule for the kk largest keys (1 <= kk <= number of real keys) by a bit
// search over the whole row.
template <int C>
__device__ __forceinline__ SelRule rule_full(const uint32_t (&key)[C], int kk) {
  bool exact;
  const uint32_t t = bit_search<C>(key, kk, 0u, 31, exact);
  if (exact) return {t - 1, 0u};  // the keys >= t are exactly the kk largest
  // t is the kk-th largest key (>= 1); the keys above it are all taken
  const int n_gt = t != 0xffffffffu ? count_ge<C>(key, t + 1) : 0;
  return {t, (uint32_t)(kk - n_gt)};
}

// Candidate keys per lane for the bracketed search (1024 per row).
constexpr int kSelCand = 16;

template <int M>
__device__ __forceinline__ SelRule rule_from_candidates(const uint32_t* buf, int m, int lane, int kk, int g_hi,
                                                        uint32_t t_lo, uint32_t upper) {
  uint32_t cand[M];
#pragma unroll
  for (int i = 0; i < M; ++i) cand[i] = 64 * i + lane < m ? buf[64 * i + lane] : 0u;
  // the kc-th largest candidate is the kk-th largest key
  const int kc = kk - g_hi;
  const uint32_t diff = t_lo ^ upper;  // the range shares the bits above b0
  const int b0 = diff == 0 ? -1 : 31 - __builtin_clz(diff);
  const uint32_t t0 = b0 == 31 ? 0u : (b0 < 0 ? t_lo : (t_lo & ~((2u << b0) - 1u)));
  bool exact;
  uint32_t t = bit_search<M>(cand, kc, t0, b0, exact);
  if (exact) {
    // exactly kc candidates are >= t; below t_lo that also counts keys outside
    // the range, so the rule starts at t_lo at the lowest
    t = t < t_lo ? t_lo : t;
    return {t - 1, 0u};
  }
  const int n_gt = g_hi + (t != 0xffffffffu ? count_ge<M>(cand, t + 1) : 0);
  return {t, (uint32_t)(kk - n_gt)};
}

// The 128 sampled keys in descending order across the wave: element
// e = 64 j + lane is s[j] of lane `lane`.  A bitonic network: at distance d the
// partner of e is e ^ d, the lane's other register for d = 64 and lane ^ d
// otherwise; e keeps the larger key when its block of k elements runs
// descending ((e & k) == 0) and e is the lower index of the pair.
__device__ __forceinline__ void sort_samples_desc(uint32_t (&s)[2], int lane) {
#pragma unroll
  for (int k = 2; k <= 128; k <<= 1) {
#pragma unroll
    for (int d = k >> 1; d >= 1; d >>= 1) {
      if (d == 64) {  // only at k = 128, where every pair runs descending
        const uint32_t hi = s[0] > s[1] ? s[0] : s[1], lo = s[0] > s[1] ? s[1] : s[0];
        s[0] = hi;
        s[1] = lo;
      } else {
#pragma unroll
        for (int j = 0; j < 2; ++j) {
          const int e = 64 * j + lane;
          const uint32_t pv = (uint32_t)__shfl_xor((int)s[j], d, 64);
          const bool keep_max = ((e & k) == 0) == ((e & d) == 0);
          const uint32_t mx = s[j] > pv ? s[j] : pv, mn = s[j] > pv ? pv : s[j];
          s[j] = keep_max ? mx : mn;
        }
      }
    }
  }
}

// The rule for the kk largest keys, bracketed from a sample first.  samp[] holds
// the keys of 128 evenly spaced blocks of the row (samp[0] of lane L: sample L,
// samp[1]: sample 64 + L; 0 for forced ones).  The sampled keys of the ranks
// around the expected rank of the kk-th key (a margin of about 2.2 standard
// deviations of the binomial count), read off the sorted sample, give
// thresholds t_lo <= t_hi; two counts over the row
// check that the kk-th key lies in [t_lo, t_hi), and the keys there (a few
// hundred) are compacted through the wave's LDS buffer `buf` (64 kSelCand
// words) and searched alone.  When the bracket misses or holds too many keys,
// the whole row is searched.
template <int C>
__device__ __forceinline__ SelRule rule_sampled(const uint32_t (&key)[C], int kk, int n_sel, const uint32_t (&samp)[2],
                                                uint32_t* buf, int lane) {
  const int s_real = count_ge<2>(samp, 1u);
  if (s_real >= 16 && n_sel > 0 && kk < n_sel) {
    const float p = (float)kk / (float)n_sel;
    const float mid = p * (float)s_real;  // expected number of sampled keys >= the kk-th key
    const int margin = (int)(2.2f * sqrtf((float)s_real * p * (1.f - p))) + 2;
    const int r1 = (int)mid - margin, r2 = (int)mid + 1 + margin;
    const bool has_hi = r1 >= 1;
    // the r-th largest sampled key (1 <= r <= 128, wave-uniform)
    uint32_t ss[2] = {samp[0], samp[1]};
    sort_samples_desc(ss, lane);
    auto kth = [&](int r) -> uint32_t {
      const int e = __builtin_amdgcn_readfirstlane(r - 1);
      return e < 64 ? (uint32_t)__builtin_amdgcn_readlane((int)ss[0], e)
                    : (uint32_t)__builtin_amdgcn_readlane((int)ss[1], e - 64);
    };
    const uint32_t t_hi = has_hi ? kth(r1) : 0u;
    const uint32_t t_lo = r2 <= s_real ? kth(r2) : 1u;
    const int g_hi = has_hi ? count_ge<C>(key, t_hi) : 0;  // keys above the range
    const int g_lo = count_ge<C>(key, t_lo);
    const int m = g_lo - g_hi;                             // keys in [t_lo, t_hi)
    if (g_hi < kk && kk <= g_lo && m <= 64 * kSelCand) {
      int base = 0;
#pragma unroll
      for (int c = 0; c < C; ++c) {
        const bool in = key[c] >= t_lo && (!has_hi || key[c] < t_hi);
        const uint64_t mask = __ballot(in);
        if (in) buf[base + lanes_below(mask)] = key[c];
        base += __popcll(mask);
      }
      const uint32_t upper = has_hi ? t_hi - 1 : 0xffffffffu;
      if (m <= 64 * 4) return rule_from_candidates<4>(buf, m, lane, kk, g_hi, t_lo, upper);
      if (m <= 64 * 8) return rule_from_candidates<8>(buf, m, lane, kk, g_hi, t_lo, upper);
      return rule_from_candidates<kSelCand>(buf, m, lane, kk, g_hi, t_lo, upper);
    }
  }
  return rule_full<C>(key, kk);
}

// Writes the row's list: the forced blocks and the selected ones, ascending.
// A block is forced when it lies below n_k and holds key 0 (real keys are
// >= 0x007fffff).  Without ties to break (take_ties == 0, the usual case) a
// block is taken when forced or above thr.
template <int C>
__device__ __forceinline__ void emit_row(const uint32_t (&key)[C], int n_k, SelRule rule, int lane, int32_t* out,
                                         int32_t* num_out) {
  int pos = 0;
  if (rule.take_ties == 0) {
#pragma unroll
    for (int c = 0; c < C; ++c) {
      if (64 * c >= n_k) break;
      const bool valid = 64 * c + 64 <= n_k || 64 * c + lane < n_k;
      const bool take = key[c] > rule.thr || (key[c] == 0u && valid);
      const uint64_t take_mask = __ballot(take);
      if (take) out[pos + lanes_below(take_mask)] = 64 * c + lane;
      pos += __popcll(take_mask);
    }
  } else {
    uint32_t ties = 0;
#pragma unroll
    for (int c = 0; c < C; ++c) {
      if (64 * c >= n_k) break;
      const bool valid = 64 * c + 64 <= n_k || 64 * c + lane < n_k;
      const bool tie = key[c] == rule.thr;  // thr >= 1: never a forced block
      const uint64_t tie_mask = __ballot(tie);
      const uint32_t tie_rank = ties + (uint32_t)lanes_below(tie_mask);
      const bool take = key[c] > rule.thr || (tie && tie_rank < rule.take_ties) || (key[c] == 0u && valid);
      const uint64_t take_mask = __ballot(take);
      if (take) out[pos + lanes_below(take_mask)] = 64 * c + lane;
      pos += __popcll(take_mask);
      ties += (uint32_t)__popcll(tie_mask);
    }
  }
  if (lane == 0) *num_out = pos;
}

// Bit c of lane L: whether block 64 c + L (c < 64) is forced.
__device__ __forceinline__ uint64_t forced_mask(const KeepBlocks& kb, int lane) {
  auto below = [](int x) -> uint64_t {  // bits [0, x)
    return x <= 0 ? 0ull : (x >= 64 ? ~0ull : (1ull << x) - 1ull);
  };
  uint64_t m = 0;
#pragma unroll
  for (int t = 0; t < kMaxKeep; ++t) {
    if (t >= kb.n) break;  // uniform: a kernel argument
    // the chunks c with begin <= 64 c + lane < end
    const int c_lo = kb.begin[t] <= lane ? 0 : (kb.begin[t] - lane + 63) / 64;
    const int c_hi = kb.end[t] <= lane ? 0 : (kb.end[t] - lane + 63) / 64;
    m |= below(c_hi) & ~below(c_lo);
  }
  return m;
}

// Sample i (0..127) of a row of n_k blocks: the middle block of the i-th of 128
// equal segments.
__device__ __forceinline__ int sample_block(int i, int n_k) { return (int)(((2 * (int64_t)i + 1) * n_k) / 256); }

// Rows of up to 64 C blocks: one wave per row reads its row of S straight
// into registers (coalesced, 256 bytes per load) through one buffer
// descriptor, so that loads past n_k need no clamp (they read 0).
template <int C>
__global__ __launch_bounds__(64 * kSelWaves) void select_reg_kernel(SelectArgs a) {
  __shared__ uint32_t cbuf[kSelWaves][64 * kSelCand];
  // the wave index as a scalar, so that the row's descriptor is one too
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x / 64), lane = threadIdx.x % 64;
  const int64_t row = (int64_t)blockIdx.x * kSelWaves + wave;
  if (row >= a.rows) return;  // wave-uniform; no barrier below
  const int h = (int)((row / a.n_q) % a.heads);
  const __amdgpu_buffer_rsrc_t rs =
      __builtin_amdgcn_make_buffer_rsrc(const_cast<float*>(a.s + row * a.s_stride), (short)0, a.n_k * 4, 0x00020000);
  // all loads first (independent), then the keys in place; S is read once
  // (cache policy 2: non-temporal)
  uint32_t key[C];
#pragma unroll
  for (int c = 0; c < C; ++c) key[c] = __builtin_amdgcn_raw_buffer_load_b32(rs, (64 * c + lane) * 4, 0, 2);
  const int b0 = sample_block(lane, a.n_k), b1 = sample_block(64 + lane, a.n_k);
  const uint32_t sp0 = __builtin_amdgcn_raw_buffer_load_b32(rs, b0 * 4, 0, 0);
  const uint32_t sp1 = __builtin_amdgcn_raw_buffer_load_b32(rs, b1 * 4, 0, 0);
  const uint64_t fm = forced_mask(a.keep, lane);
#pragma unroll
  for (int c = 0; c < C; ++c) {
    const bool real = (64 * c + 64 <= a.n_k || 64 * c + lane < a.n_k) && !((fm >> c) & 1ull);
    key[c] = real ? order_key_bits(key[c]) : 0u;
  }
  const uint32_t samp[2] = {keep_block(a.keep, b0) ? 0u : order_key_bits(sp0),
                            keep_block(a.keep, b1) ? 0u : order_key_bits(sp1)};
  const int kk = a.budget.k[h];
  // kk == 0: nothing selectable
  const SelRule rule = kk > 0 ? rule_sampled<C>(key, kk, a.n_sel, samp, cbuf[wave], lane) : SelRule{0xffffffffu, 0u};
  emit_row<C>(key, a.n_k, rule, lane, a.kv_indices + row * a.stride, a.kv_num_blocks + row);
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
  uint32_t* rk = fused_keys + (size_t)wave * row_len;
  uint32_t key[C];
#pragma unroll
  for (int c = 0; c < C; ++c) {
    const int j = 64 * c + lane;
    const uint32_t v = rk[j < row_len ? j : row_len - 1];  // in bounds, independent reads
    key[c] = j < a.n_k ? v : 0u;
  }
  const uint32_t samp[2] = {rk[sample_block(lane, a.n_k)], rk[sample_block(64 + lane, a.n_k)]};
  const int64_t r = bh * a.n_q + i;
  const int kk = a.budget.k[(int)(bh % a.heads)];
  // the row's own LDS keys are in registers now: their space holds the
  // bracketed candidates (at most min(n_k, 64 kSelCand) of them)
  const SelRule rule = kk > 0 ? rule_sampled<C>(key, kk, a.n_sel, samp, rk, lane) : SelRule{0xffffffffu, 0u};
  emit_row<C>(key, a.n_k, rule, lane, a.kv_indices + r * a.stride, a.kv_num_blocks + r);
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
