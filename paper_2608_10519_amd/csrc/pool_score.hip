// Block pooling (Section 5.1) and aggregated query-key block scores (Eq. 2).
//
// pool:  qbar_i = b^-1 sum_r q~_{i,r}, kbar_j likewise; the final partial block
//        is zero-padded and still divided by the nominal b.  One work-group per
//        block streams its b x D bf16 tile once with 16-byte loads (HBM-bound;
//        algorithmic bytes = 2*D per token read + 4*D per block written).
// score: S_ij = tau * qbar_i . kbar_j in fp32 (MFMA) for selectable j; forced key
//        blocks are neither pooled nor scored (Section 5.2), their S columns are
//        left untouched.
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

  // all loads in flight at once (rows past the end re-read the last row, then count as zeros)
  uint4 v[RPT];
#pragma unroll
  for (int r = 0; r < RPT; ++r) {
    const int row = g + r * RG;
    const int64_t rr = row < rows_left ? row : rows_left - 1;
    v[r] = *reinterpret_cast<const uint4*>(src + rr * D + c * 8);
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
  if (t < D) {
    float s = 0.f;
#pragma unroll
    for (int r = 0; r < RG; ++r) s += red[r][t];
    float* dst = (is_q ? a.q_bar : a.k_bar) + (bh * nb + blk) * D;
    dst[t] = s * (1.0f / BLK);
  }
}

// ---------------------------------------------------------------------------
// score: one work-group per (bh, 64 query blocks, 64 key blocks) tile of S,
// four waves, each a 32 x 32 sub-tile on v_mfma_f32_32x32x2_f32 (fp32
// products, fp32 accumulation).  D is streamed through LDS in chunks of SKC
// columns (coalesced 16-byte loads), which keeps a work-group at 18 KB of LDS
// so that many share a CU; rows are padded by 4 floats, which makes the
// per-lane row reads below free of bank conflicts.
//
// MFMA operands (lane l, h = l / 32): A[m][k] = qbar[m = l % 32][d],
// B[k][n] = kbar[n = l % 32][d] with k = h; within a chunk MFMA s reads
// d = (SKC/2) h + s, so each lane walks its own half-row with 16-byte reads.
// C[m][n] sits at accumulator a with n = l % 32, m = 8 (a / 4) + 4 h + (a % 4).
// ---------------------------------------------------------------------------
constexpr int ST = 64;   // tile edge (query blocks and key blocks)
constexpr int SKC = 32;  // D chunk

template <int D>
__global__ __launch_bounds__(256) void score_kernel(ScoreArgs a) {
  constexpr int RS = SKC + 4;  // padded LDS row (floats)
  __shared__ __attribute__((aligned(16))) float qs[ST * RS];
  __shared__ __attribute__((aligned(16))) float ks[ST * RS];
  const int tiles_i = (a.n_q + ST - 1) / ST;
  const int tiles_j = (a.n_k + ST - 1) / ST;
  int64_t wg = blockIdx.x;
  const int tj = (int)(wg % tiles_j);
  wg /= tiles_j;
  const int ti = (int)(wg % tiles_i);
  const int64_t bh = wg / tiles_i;
  const int i0 = ti * ST, j0 = tj * ST;

  const float* qb = a.q_bar + bh * (int64_t)a.n_q * D;
  const float* kb = a.k_bar + bh * (int64_t)a.n_k * D;
  const int t = threadIdx.x;
  const int wave = t / 64, lane = t % 64, l32 = lane % 32, h = lane / 32;
  const int wq = wave / 2, wk = wave % 2;  // the wave's 32 x 32 sub-tile
  // loader: 64 rows x SKC floats = 512 float4 per tile; thread t loads rows lr and lr + 32.
  // Rows past the end re-read a valid row and are zeroed when staged; the
  // next chunk's loads are in flight while the current chunk is multiplied.
  const int lr = t / 8, lc = (t % 8) * 4;
  const bool q0_ok = i0 + lr < a.n_q, q1_ok = i0 + lr + 32 < a.n_q;
  const bool k0_ok = j0 + lr < a.n_k, k1_ok = j0 + lr + 32 < a.n_k;
  const float* const qr0 = qb + (int64_t)(q0_ok ? i0 + lr : 0) * D + lc;
  const float* const qr1 = qb + (int64_t)(q1_ok ? i0 + lr + 32 : 0) * D + lc;
  const float* const kr0 = kb + (int64_t)(k0_ok ? j0 + lr : 0) * D + lc;
  const float* const kr1 = kb + (int64_t)(k1_ok ? j0 + lr + 32 : 0) * D + lc;
  float4 q0 = *reinterpret_cast<const float4*>(qr0), q1 = *reinterpret_cast<const float4*>(qr1);
  float4 k0 = *reinterpret_cast<const float4*>(kr0), k1 = *reinterpret_cast<const float4*>(kr1);
  // element-wise (a select of whole float4 values goes through scratch memory)
  auto keep_if = [](bool ok, float4 v) {
    return make_float4(ok ? v.x : 0.f, ok ? v.y : 0.f, ok ? v.z : 0.f, ok ? v.w : 0.f);
  };

  f32x16 acc;
#pragma unroll
  for (int e = 0; e < 16; ++e) acc[e] = 0.f;
#pragma unroll
  for (int d0 = 0; d0 < D; d0 += SKC) {
    if (d0 > 0) __syncthreads();  // the previous chunk's reads are done
    *reinterpret_cast<float4*>(qs + lr * RS + lc) = keep_if(q0_ok, q0);
    *reinterpret_cast<float4*>(qs + (lr + 32) * RS + lc) = keep_if(q1_ok, q1);
    *reinterpret_cast<float4*>(ks + lr * RS + lc) = keep_if(k0_ok, k0);
    *reinterpret_cast<float4*>(ks + (lr + 32) * RS + lc) = keep_if(k1_ok, k1);
    __syncthreads();
    if (d0 + SKC < D) {
      q0 = *reinterpret_cast<const float4*>(qr0 + d0 + SKC);
      q1 = *reinterpret_cast<const float4*>(qr1 + d0 + SKC);
      k0 = *reinterpret_cast<const float4*>(kr0 + d0 + SKC);
      k1 = *reinterpret_cast<const float4*>(kr1 + d0 + SKC);
    }
    const float* qa = qs + (wq * 32 + l32) * RS + (SKC / 2) * h;
    const float* kc = ks + (wk * 32 + l32) * RS + (SKC / 2) * h;
#pragma unroll
    for (int i = 0; i < SKC / 8; ++i) {
      const float4 x = *reinterpret_cast<const float4*>(qa + 4 * i);
      const float4 y = *reinterpret_cast<const float4*>(kc + 4 * i);
      acc = __builtin_amdgcn_mfma_f32_32x32x2f32(x.x, y.x, acc, 0, 0, 0);
      acc = __builtin_amdgcn_mfma_f32_32x32x2f32(x.y, y.y, acc, 0, 0, 0);
      acc = __builtin_amdgcn_mfma_f32_32x32x2f32(x.z, y.z, acc, 0, 0, 0);
      acc = __builtin_amdgcn_mfma_f32_32x32x2f32(x.w, y.w, acc, 0, 0, 0);
    }
  }

  const int j = j0 + wk * 32 + l32;
  if (j >= a.n_k || keep_block(a.keep, j)) return;  // no barrier below
  float* scol = a.s + bh * (int64_t)a.n_q * a.n_k + j;
#pragma unroll
  for (int e = 0; e < 16; ++e) {
    const int i = i0 + wq * 32 + 8 * (e / 4) + 4 * h + (e % 4);
    if (i < a.n_q) scol[(int64_t)i * a.n_k] = a.tau * acc[e];
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
