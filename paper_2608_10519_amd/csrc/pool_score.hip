// Block pooling (Section 5.1) and aggregated query-key block scores (Eq. 2).
//
// pool:  qbar_i = b^-1 sum_r q~_{i,r}, kbar_j likewise; the final partial block
//        is zero-padded and still divided by the nominal b.  One work-group per
//        block streams its b x D bf16 tile once with 16-byte loads (HBM-bound;
//        algorithmic bytes = 2*D per token read + 4*D + 4 per block written).
//        The mean is written split for the fp16 matrix cores (launch.h):
//        2^e (hi + lo) with e the row's power-of-two scale.
// score: S_ij = tau * qbar_i . kbar_j for selectable j, on fp16 MFMA with
//        fp32 accumulation as hi.hi + hi.lo + lo.hi: the dropped lo.lo term
//        and the split leave a relative error near 2^-21 of sum |q k|, the
//        level of an fp32 dot product; forced key blocks are neither pooled
//        nor scored (Section 5.2), their S columns are left untouched.
#include "device_common.h"

namespace sparstar {

// ---------------------------------------------------------------------------
// pool: grid = BH*n_q + BH*n_k work-groups (query blocks first), 256 threads.
// Thread t owns the 16-byte column chunk (t % CH) of rows g, g + RG, ... with
// g = t / CH, CH = D/8 chunks per row and RG = 256/CH row groups.
// ---------------------------------------------------------------------------
template <int D, int BLK>
__global__ __launch_bounds__(256) void pool_kernel(PoolArgs a) {
  constexpr int CH = D / 8;
  constexpr int RG = 256 / CH;
  constexpr int RPT = BLK / RG;
  __shared__ float red[RG][D + 1];
  __shared__ float wmax[4];

  const int64_t wg = blockIdx.x;
  const int64_t nqb = (int64_t)a.bh * a.n_q;
  const bool is_q = wg < nqb;
  const int64_t w = is_q ? wg : wg - nqb;
  const int nb = is_q ? a.n_q : a.n_k;
  const int64_t bh = w / nb;
  const int blk = (int)(w % nb);
  if (!is_q && keep_block(a.keep, blk)) return;  // uniform over the work-group

  const int64_t len = is_q ? a.lq : a.lk;
  const uint16_t* src = (is_q ? a.q : a.k) + (bh * len + (int64_t)blk * BLK) * D;
  const int t = threadIdx.x, c = t % CH, g = t / CH;
  const int64_t rows_left = len - (int64_t)blk * BLK;

  // all loads in flight at once (rows past the end re-read the last row, then
  // count as zeros); Q and K are read once here, so the loads are non-temporal
  // and do not displace what the caches hold
  typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));
  uint4 v[RPT];
#pragma unroll
  for (int r = 0; r < RPT; ++r) {
    const int row = g + r * RG;
    const int64_t rr = row < rows_left ? row : rows_left - 1;
    const u32x4 t4 = __builtin_nontemporal_load(reinterpret_cast<const u32x4*>(src + rr * D + c * 8));
    v[r] = make_uint4(t4[0], t4[1], t4[2], t4[3]);
  }
#pragma unroll
  for (int r = 0; r < RPT; ++r)
    if (g + r * RG >= rows_left) v[r] = make_uint4(0, 0, 0, 0);
  float acc[8];
#pragma unroll
  for (int e = 0; e < 8; ++e) acc[e] = 0.f;
#pragma unroll
  for (int r = 0; r < RPT; ++r) {
    const uint32_t w4[4] = {v[r].x, v[r].y, v[r].z, v[r].w};
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      acc[2 * e] += bf16_lo(w4[e]);
      acc[2 * e + 1] += bf16_hi(w4[e]);
    }
  }
#pragma unroll
  for (int e = 0; e < 8; ++e) red[g][c * 8 + e] = acc[e];
  __syncthreads();
  float x = 0.f;  // element t of the block mean
  if (t < D) {
    float s = 0.f;
#pragma unroll
    for (int r = 0; r < RG; ++r) s += red[r][t];
    x = s * (1.0f / BLK);
  }
  // the row's largest magnitude (a wave maximum, then over the four waves)
  // fixes its scale 2^e: |x| 2^-e < 2^14, inside fp16's range
  float m = fabsf(x);
#pragma unroll
  for (int off = 32; off > 0; off >>= 1) m = fmaxf(m, __shfl_xor(m, off, 64));
  if (t % 64 == 0) wmax[t / 64] = m;
  __syncthreads();
  m = fmaxf(fmaxf(wmax[0], wmax[1]), fmaxf(wmax[2], wmax[3]));
  const int ex = (m > 0.f && m <= 3.402823466e38f) ? __builtin_amdgcn_frexp_expf(m) - 14 : 0;
  const int64_t row = bh * nb + blk;
  if (t < D) {
    const float xs = __builtin_amdgcn_ldexpf(x, -ex);
    const _Float16 hi = (_Float16)xs;
    const _Float16 lo = (_Float16)(xs - (float)hi);  // the difference is exact in fp32
    uint16_t* dst = (is_q ? a.q_bar : a.k_bar) + row * (2 * D);
    dst[t] = __builtin_bit_cast(uint16_t, hi);
    dst[D + t] = __builtin_bit_cast(uint16_t, lo);
  }
  if (t == 0) (is_q ? a.q_exp : a.k_exp)[row] = ex;
}

// ---------------------------------------------------------------------------
// score: one work-group per (bh, 64 query blocks, 64 key blocks) tile of S,
// four waves, each a 32 x 32 sub-tile on v_mfma_f32_32x32x16_f16.  Every
// thread issues all of its global loads (its row's 16-byte pieces of the hi and
// lo parts, for all of D) at once, so a work-group waits for memory once; D
// then goes through LDS in chunks of SKC columns, each LDS row holding the
// chunk's hi then lo values of one pooled row, padded to 144 bytes: 16
// consecutive rows read at one 16-byte offset then fall on 16 disjoint groups
// of four banks.
//
// MFMA operands (lane l, h = l / 32): A[m][k] = qbar[m = l % 32][d],
// B[k][n] = kbar[n = l % 32][d], k = 8 h + i over the lane's 8 fp16 values at
// d = 16 s + 8 h + i of k-step s.  C[m][n] sits at accumulator a with
// n = l % 32, m = 8 (a / 4) + 4 h + (a % 4).
// ---------------------------------------------------------------------------
constexpr int ST = 64;   // tile edge (query blocks and key blocks)
constexpr int SKC = 32;  // D chunk

template <int D>
__global__ __launch_bounds__(256) void score_kernel(ScoreArgs a) {
  constexpr int RB = 144;  // padded LDS row (bytes): SKC hi + SKC lo fp16
  __shared__ __attribute__((aligned(16))) unsigned char qs[ST * RB];
  __shared__ __attribute__((aligned(16))) unsigned char ks[ST * RB];
  __shared__ int qe[ST], ke[ST];
  const int tiles_i = (a.n_q + ST - 1) / ST;
  const int tiles_j = (a.n_k + ST - 1) / ST;
  // consecutive tiles (one head's, key tiles fastest) on the same XCD, whose
  // L2 then holds that head's pooled blocks
  int64_t wg = xcd_linear(blockIdx.x, (int64_t)gridDim.x);
  const int tj = (int)(wg % tiles_j);
  wg /= tiles_j;
  const int ti = (int)(wg % tiles_i);
  const int64_t bh = wg / tiles_i;
  const int i0 = ti * ST, j0 = tj * ST;

  const int t = threadIdx.x;
  const int wave = t / 64, lane = t % 64, l32 = lane % 32, h = lane / 32;
  const int wq = wave / 2, wk = wave % 2;  // the wave's 32 x 32 sub-tile
  // loader: thread t stages row lr, 16-byte piece lc of the chunk's hi and lo
  // parts.  Rows past the end re-read a valid row and are zeroed when staged.
  const int lr = t / 4, lc = t % 4;
  const bool q_ok = i0 + lr < a.n_q, k_ok = j0 + lr < a.n_k;
  const uint16_t* const qrow = a.q_bar + (bh * a.n_q + (q_ok ? i0 + lr : 0)) * (2 * D) + 8 * lc;
  const uint16_t* const krow = a.k_bar + (bh * a.n_k + (k_ok ? j0 + lr : 0)) * (2 * D) + 8 * lc;
  auto ld = [](const uint16_t* p) { return *reinterpret_cast<const uint4*>(p); };
  // element-wise (a select of whole uint4 values goes through scratch memory)
  auto keep_if = [](bool ok, uint4 v) {
    return make_uint4(ok ? v.x : 0u, ok ? v.y : 0u, ok ? v.z : 0u, ok ? v.w : 0u);
  };
  constexpr int NC = D / SKC;
  uint4 qh[NC], ql[NC], kh[NC], kl[NC];
#pragma unroll
  for (int c = 0; c < NC; ++c) {
    qh[c] = ld(qrow + c * SKC);
    ql[c] = ld(qrow + D + c * SKC);
    kh[c] = ld(krow + c * SKC);
    kl[c] = ld(krow + D + c * SKC);
  }
  if (t < ST) qe[t] = i0 + t < a.n_q ? a.q_exp[bh * a.n_q + i0 + t] : 0;
  else if (t < 2 * ST) ke[t - ST] = j0 + t - ST < a.n_k ? a.k_exp[bh * a.n_k + j0 + t - ST] : 0;

  f32x16 acc;
#pragma unroll
  for (int e = 0; e < 16; ++e) acc[e] = 0.f;
#pragma unroll
  for (int c = 0; c < NC; ++c) {
    if (c > 0) __syncthreads();  // the previous chunk's reads are done
    *reinterpret_cast<uint4*>(qs + lr * RB + 16 * lc) = keep_if(q_ok, qh[c]);
    *reinterpret_cast<uint4*>(qs + lr * RB + 64 + 16 * lc) = keep_if(q_ok, ql[c]);
    *reinterpret_cast<uint4*>(ks + lr * RB + 16 * lc) = keep_if(k_ok, kh[c]);
    *reinterpret_cast<uint4*>(ks + lr * RB + 64 + 16 * lc) = keep_if(k_ok, kl[c]);
    __syncthreads();
    const unsigned char* qa = qs + (wq * 32 + l32) * RB + 16 * h;
    const unsigned char* kc = ks + (wk * 32 + l32) * RB + 16 * h;
#pragma unroll
    for (int s = 0; s < SKC / 16; ++s) {
      const f16x8 ah = *reinterpret_cast<const f16x8*>(qa + 32 * s);
      const f16x8 al = *reinterpret_cast<const f16x8*>(qa + 64 + 32 * s);
      const f16x8 bh_ = *reinterpret_cast<const f16x8*>(kc + 32 * s);
      const f16x8 bl = *reinterpret_cast<const f16x8*>(kc + 64 + 32 * s);
      acc = __builtin_amdgcn_mfma_f32_32x32x16_f16(ah, bh_, acc, 0, 0, 0);
      acc = __builtin_amdgcn_mfma_f32_32x32x16_f16(ah, bl, acc, 0, 0, 0);
      acc = __builtin_amdgcn_mfma_f32_32x32x16_f16(al, bh_, acc, 0, 0, 0);
    }
  }

  const int j = j0 + wk * 32 + l32;
  if (j >= a.n_k || keep_block(a.keep, j)) return;  // no barrier below
  const int ej = ke[wk * 32 + l32];
  float* scol = a.s + bh * (int64_t)a.n_q * a.s_stride + j;
#pragma unroll
  for (int e = 0; e < 16; ++e) {
    const int r = wq * 32 + 8 * (e / 4) + 4 * h + (e % 4);
    const int i = i0 + r;
    if (i < a.n_q) scol[(int64_t)i * a.s_stride] = a.tau * __builtin_amdgcn_ldexpf(acc[e], qe[r] + ej);
  }
}

hipError_t launch_pool(const PoolArgs& a, int d, int block, hipStream_t stream) {
  const int64_t grid = (int64_t)a.bh * (a.n_q + a.n_k);
  if (grid == 0) return hipSuccess;
  if (d == 128 && block == 64) pool_kernel<128, 64><<<grid, 256, 0, stream>>>(a);
  else if (d == 128 && block == 128) pool_kernel<128, 128><<<grid, 256, 0, stream>>>(a);
  else if (d == 64 && block == 64) pool_kernel<64, 64><<<grid, 256, 0, stream>>>(a);
  else if (d == 64 && block == 128) pool_kernel<64, 128><<<grid, 256, 0, stream>>>(a);
  else return hipErrorInvalidValue;
  return hipGetLastError();
}

hipError_t launch_score(const ScoreArgs& a, int d, hipStream_t stream) {
  const int64_t grid = (int64_t)a.bh * ((a.n_q + ST - 1) / ST) * ((a.n_k + ST - 1) / ST);
  if (grid == 0) return hipSuccess;
  if (d == 128) score_kernel<128><<<grid, 256, 0, stream>>>(a);
  else if (d == 64) score_kernel<64><<<grid, 256, 0, stream>>>(a);
  else return hipErrorInvalidValue;
  return hipGetLastError();
}

}  // namespace sparstar
