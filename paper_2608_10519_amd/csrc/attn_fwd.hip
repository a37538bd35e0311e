// Block-sparse attention forward (Eq. 7, Section 5.3) and its dense variant.
//
// One work-group per (batch*head, query block of BLK rows); BLK/32 wavefronts,
// each owning 32 query rows.  The work-group walks the ascending key-block list
// of its query block; per key block:
//   1. the K tile (BLK x D) is staged row-major in LDS and the V tile
//      transposed (D x BLK), from registers prefetched during the previous
//      tile's math;
//   2. S^T = K Q^T on v_mfma_f32_32x32x16_bf16 (fp32 accumulate).  Computing
//      the transpose leaves each lane holding 16 keys of ONE query column, which
//      is exactly the B-operand layout P^T needs below, so the softmax state
//      (running max m and sum l) is lane-local;
//   3. online softmax in the log2 domain; P is rounded to bf16 once.  Two row
//      sums are kept: over the rounded values (normalises O, so the weights
//      applied to V sum to one and V == 1 gives O == 1 exactly) and over the
//      fp32 values (for the log-sum-exp);
//   4. O^T += V^T P^T on the same MFMA (O^T accumulators keep a lane's query
//      column together, so the rescale by exp2(m_old - m_new) is lane-local).
// The epilogue writes O = O^T / l in bf16 and lse = ln2 * (m + log2 l_fp32).
//
// MFMA layouts used (v_mfma_f32_32x32x16_bf16, lane l, h = l / 32):
//   A[m][k]: m = l % 32, k = 8h + i (i = 0..7 of the lane's bf16x8)
//   B[k][n]: n = l % 32, k = 8h + i
//   C[m][n]: n = l % 32, m = 8 (a / 4) + 4h + (a % 4) for accumulator a = 0..15
// The contraction only needs A and B to agree on k, so keys may be permuted
// consistently: the P^T operand reuses the S^T C layout directly and the V^T
// operand reads the same key permutation from LDS.
#include "device_common.h"

namespace sparstar {

template <int D, int BLK>
struct AttnCfg {
  static constexpr int NW = BLK / 32;         // wavefronts (32 query rows each)
  static constexpr int NT = NW * 64;          // threads
  static constexpr int KLD = D + 8;           // K tile row pitch (bf16), padded
  static constexpr int VLD = BLK + 8;         // V^T tile row pitch (bf16), padded
  static constexpr int KCH = BLK * D / 8 / NT;          // 16-byte K chunks per thread
  static constexpr int VGR = (BLK / 4) * (D / 8) / NT;  // 4-key x 8-d V groups per thread
  static constexpr int KT = BLK / 32;         // 32-key sub-tiles per key block
  static constexpr int DS = D / 16;           // MFMA k-steps over D
  static constexpr int DT = D / 32;           // 32-row d tiles of O^T
  static_assert(KCH * NT * 8 == BLK * D, "K tile split");
  static_assert(VGR * NT * 32 == BLK * D, "V tile split");
};

template <int D, int BLK, bool DENSE>
__global__ __launch_bounds__(BLK * 2) void attn_fwd_kernel(AttnArgs a) {
  using C = AttnCfg<D, BLK>;
  __shared__ __attribute__((aligned(16))) uint16_t ks[BLK * C::KLD];
  __shared__ __attribute__((aligned(16))) uint16_t vt[D * C::VLD];

  const int64_t nwork = (int64_t)a.bh * a.n_q;
  const int64_t work = xcd_linear(blockIdx.x, nwork);
  const int64_t bh = work / a.n_q;
  const int qb = (int)(work % a.n_q);

  const int tid = threadIdx.x, wave = tid / 64, lane = tid % 64;
  const int l32 = lane % 32, hh = lane / 32;

  const uint16_t* kbase = a.k + bh * a.lk * D;
  const uint16_t* vbase = a.v + bh * a.lk * D;

  // ---- list of key blocks
  int nblk;
  const int32_t* list = nullptr;
  if constexpr (DENSE) {
    nblk = a.n_k;
  } else {
    const int64_t r = bh * a.n_q + qb;
    nblk = a.kv_num_blocks[r];
    nblk = nblk < 0 ? 0 : (nblk > a.stride ? a.stride : nblk);
    list = a.kv_indices + r * a.stride;
  }
  auto block_at = [&](int it) -> int {
    if constexpr (DENSE) return it;
    int j = __builtin_amdgcn_readfirstlane(list[it]);
    return (j >= 0 && j < a.n_k) ? j : -1;
  };

  // ---- Q fragment (B operand of S^T = K Q^T): Q[q][16 s + 8 hh .. +7]
  const int64_t q_row = (int64_t)qb * BLK + wave * 32 + l32;
  const bool q_ok = q_row < a.lq;
  const uint16_t* qp = a.q + (bh * a.lq + (q_row < a.lq ? q_row : 0)) * D;
  bf16x8 qf[C::DS];
#pragma unroll
  for (int s = 0; s < C::DS; ++s) {
    uint4 u = q_ok ? *reinterpret_cast<const uint4*>(qp + 16 * s + 8 * hh) : make_uint4(0, 0, 0, 0);
    qf[s] = __builtin_bit_cast(bf16x8, u);
  }

  f32x16 acc_o[C::DT];
#pragma unroll
  for (int t = 0; t < C::DT; ++t)
#pragma unroll
    for (int e = 0; e < 16; ++e) acc_o[t][e] = 0.f;
  float m_run = -INFINITY, l_run = 0.f, le_run = 0.f;

  // ---- global -> register prefetch of one key block
  uint4 kreg[C::KCH];
  uint4 vreg[C::VGR][4];
  auto load_tile = [&](int blk) {
    const int64_t key0 = (int64_t)blk * BLK;
#pragma unroll
    for (int r = 0; r < C::KCH; ++r) {
      const int c = tid + C::NT * r;
      const int row = c / (D / 8), col = c % (D / 8);
      const int64_t key = key0 + row;
      kreg[r] = key < a.lk ? *reinterpret_cast<const uint4*>(kbase + key * D + col * 8) : make_uint4(0, 0, 0, 0);
    }
#pragma unroll
    for (int r = 0; r < C::VGR; ++r) {
      const int g = tid + C::NT * r;
      const int dg = g % (D / 8), kg = g / (D / 8);
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        const int64_t key = key0 + 4 * kg + e;
        vreg[r][e] = key < a.lk ? *reinterpret_cast<const uint4*>(vbase + key * D + dg * 8) : make_uint4(0, 0, 0, 0);
      }
    }
  };
  auto store_tile = [&]() {
#pragma unroll
    for (int r = 0; r < C::KCH; ++r) {
      const int c = tid + C::NT * r;
      const int row = c / (D / 8), col = c % (D / 8);
      *reinterpret_cast<uint4*>(&ks[row * C::KLD + col * 8]) = kreg[r];
    }
#pragma unroll
    for (int r = 0; r < C::VGR; ++r) {
      const int g = tid + C::NT * r;
      const int dg = g % (D / 8), kg = g / (D / 8);
      const uint32_t w0[4] = {vreg[r][0].x, vreg[r][0].y, vreg[r][0].z, vreg[r][0].w};
      const uint32_t w1[4] = {vreg[r][1].x, vreg[r][1].y, vreg[r][1].z, vreg[r][1].w};
      const uint32_t w2[4] = {vreg[r][2].x, vreg[r][2].y, vreg[r][2].z, vreg[r][2].w};
      const uint32_t w3[4] = {vreg[r][3].x, vreg[r][3].y, vreg[r][3].z, vreg[r][3].w};
#pragma unroll
      for (int p = 0; p < 4; ++p) {
        // d = 8 dg + 2p (low halves) and 8 dg + 2p + 1 (high halves); keys 4 kg .. 4 kg + 3
        uint2 lo, hi;
        lo.x = (w0[p] & 0xffffu) | (w1[p] << 16);
        lo.y = (w2[p] & 0xffffu) | (w3[p] << 16);
        hi.x = (w0[p] >> 16) | (w1[p] & 0xffff0000u);
        hi.y = (w2[p] >> 16) | (w3[p] & 0xffff0000u);
        *reinterpret_cast<uint2*>(&vt[(8 * dg + 2 * p) * C::VLD + 4 * kg]) = lo;
        *reinterpret_cast<uint2*>(&vt[(8 * dg + 2 * p + 1) * C::VLD + 4 * kg]) = hi;
      }
    }
  };

  // find the first valid block
  int it = 0;
  int cur = -1;
  while (it < nblk && (cur = block_at(it)) < 0) ++it;
  if (cur >= 0) load_tile(cur);

  const float sl2 = a.scale_log2;
  while (cur >= 0) {
    // next valid block
    int it_next = it + 1, nxt = -1;
    while (it_next < nblk && (nxt = block_at(it_next)) < 0) ++it_next;

    __syncthreads();  // previous tile fully consumed
    store_tile();
    __syncthreads();
    if (nxt >= 0) load_tile(nxt);

    // ---- S^T = K Q^T
    f32x16 acc_s[C::KT];
#pragma unroll
    for (int kt = 0; kt < C::KT; ++kt) {
#pragma unroll
      for (int e = 0; e < 16; ++e) acc_s[kt][e] = 0.f;
#pragma unroll
      for (int s = 0; s < C::DS; ++s) {
        const uint4 u = *reinterpret_cast<const uint4*>(&ks[(kt * 32 + l32) * C::KLD + 16 * s + 8 * hh]);
        acc_s[kt] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(__builtin_bit_cast(bf16x8, u), qf[s], acc_s[kt], 0, 0, 0);
      }
    }

    // ---- online softmax (log2 domain); keys >= Lk masked
    const int64_t key0 = (int64_t)cur * BLK;
    const bool partial = key0 + BLK > a.lk;
    float mx = -INFINITY;
#pragma unroll
    for (int kt = 0; kt < C::KT; ++kt)
#pragma unroll
      for (int e = 0; e < 16; ++e) {
        float z = acc_s[kt][e] * sl2;
        if (partial) {
          const int key = kt * 32 + 8 * (e / 4) + 4 * hh + (e % 4);
          if (key0 + key >= a.lk) z = -INFINITY;
        }
        acc_s[kt][e] = z;
        mx = fmaxf(mx, z);
      }
    mx = fmaxf(mx, __shfl_xor(mx, 32, 64));
    const float m_new = fmaxf(m_run, mx);
    const float m_use = m_new == -INFINITY ? 0.f : m_new;
    const float alpha = exp2f(m_run - m_use);

    float ls = 0.f, le = 0.f;
    uint32_t pk[C::KT][8];  // bf16 pairs of P^T, per 32-key sub-tile
#pragma unroll
    for (int kt = 0; kt < C::KT; ++kt)
#pragma unroll
      for (int e = 0; e < 16; e += 2) {
        const float p0 = exp2f(acc_s[kt][e] - m_use), p1 = exp2f(acc_s[kt][e + 1] - m_use);
        const uint32_t w = pack_bf16(p0, p1);
        pk[kt][e / 2] = w;
        ls += bf16_lo(w) + bf16_hi(w);
        le += p0 + p1;
      }
    ls += __shfl_xor(ls, 32, 64);
    le += __shfl_xor(le, 32, 64);
    l_run = l_run * alpha + ls;
    le_run = le_run * alpha + le;
    m_run = m_new;
#pragma unroll
    for (int t = 0; t < C::DT; ++t)
#pragma unroll
      for (int e = 0; e < 16; ++e) acc_o[t][e] *= alpha;

    // ---- O^T += V^T P^T over 16-key k-steps
#pragma unroll
    for (int kt = 0; kt < C::KT; ++kt)
#pragma unroll
      for (int half = 0; half < 2; ++half) {
        // accumulators a = 8 half + i of sub-tile kt hold keys
        //   32 kt + 16 half + 4 hh + i       (i = 0..3)
        //   32 kt + 16 half + 8 + 4 hh + i-4 (i = 4..7)
        uint4 pu;
        pu.x = pk[kt][4 * half + 0];
        pu.y = pk[kt][4 * half + 1];
        pu.z = pk[kt][4 * half + 2];
        pu.w = pk[kt][4 * half + 3];
        const bf16x8 pb = __builtin_bit_cast(bf16x8, pu);
        const int kcol = 32 * kt + 16 * half + 4 * hh;
#pragma unroll
        for (int t = 0; t < C::DT; ++t) {
          const uint16_t* vr = &vt[(32 * t + l32) * C::VLD + kcol];
          const uint2 v0 = *reinterpret_cast<const uint2*>(vr);
          const uint2 v1 = *reinterpret_cast<const uint2*>(vr + 8);
          const uint4 vu = make_uint4(v0.x, v0.y, v1.x, v1.y);
          acc_o[t] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(__builtin_bit_cast(bf16x8, vu), pb, acc_o[t], 0, 0, 0);
        }
      }

    it = it_next;
    cur = nxt;
  }

  // ---- epilogue
  if (q_ok) {
    const float inv = l_run > 0.f ? 1.f / l_run : 0.f;
    uint16_t* op = a.o + (bh * a.lq + q_row) * D;
#pragma unroll
    for (int t = 0; t < C::DT; ++t)
#pragma unroll
      for (int g = 0; g < 4; ++g) {
        const int d = 32 * t + 8 * g + 4 * hh;
        uint2 w;
        w.x = pack_bf16(acc_o[t][4 * g + 0] * inv, acc_o[t][4 * g + 1] * inv);
        w.y = pack_bf16(acc_o[t][4 * g + 2] * inv, acc_o[t][4 * g + 3] * inv);
        *reinterpret_cast<uint2*>(op + d) = w;
      }
    if (a.lse != nullptr && hh == 0)
      a.lse[bh * a.lq + q_row] = le_run > 0.f ? (m_run + log2f(le_run)) * 0.69314718055994530942f : -INFINITY;
  }
}

template <int D, int BLK>
static hipError_t launch_cfg(const AttnArgs& a, bool dense, hipStream_t stream) {
  const int64_t grid = (int64_t)a.bh * a.n_q;
  if (grid == 0) return hipSuccess;
  if (dense) attn_fwd_kernel<D, BLK, true><<<grid, AttnCfg<D, BLK>::NT, 0, stream>>>(a);
  else attn_fwd_kernel<D, BLK, false><<<grid, AttnCfg<D, BLK>::NT, 0, stream>>>(a);
  return hipGetLastError();
}

hipError_t launch_attn(const AttnArgs& a, int d, int block, bool dense, hipStream_t stream) {
  if (d == 128 && block == 64) return launch_cfg<128, 64>(a, dense, stream);
  if (d == 128 && block == 128) return launch_cfg<128, 128>(a, dense, stream);
  if (d == 64 && block == 64) return launch_cfg<64, 64>(a, dense, stream);
  if (d == 64 && block == 128) return launch_cfg<64, 128>(a, dense, stream);
  return hipErrorInvalidValue;
}

}  // namespace sparstar
