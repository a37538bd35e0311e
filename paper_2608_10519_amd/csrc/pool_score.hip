// Block pooling (Section 5.1) and aggregated query-key block scores (Eq. 2).
//
// pool:  qbar_i = b^-1 sum_r q~_{i,r}, kbar_j likewise; the final partial block
//        is zero-padded and still divided by the nominal b.  One work-group per
//        block streams its b x D bf16 tile once with 16-byte loads (HBM-bound;
//        algorithmic bytes = 2*D per token read + 4*D per block written).
// score: S_ij = tau * qbar_i . kbar_j in fp32 FMA for selectable j; forced key
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

  uint4 v[RPT];
#pragma unroll
  for (int r = 0; r < RPT; ++r) {
    const int row = g + r * RG;
    v[r] = row < rows_left ? *reinterpret_cast<const uint4*>(src + (int64_t)row * D + c * 8)
                           : make_uint4(0, 0, 0, 0);
  }
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
// score: one work-group per (bh, 64 query blocks, 64 key blocks) tile,
// 256 threads, each a 4x4 sub-tile; D streamed through LDS in chunks of 32.
// ---------------------------------------------------------------------------
constexpr int ST = 64;   // tile edge (query blocks and key blocks)
constexpr int SKC = 32;  // D chunk

template <int D>
__global__ __launch_bounds__(256) void score_kernel(ScoreArgs a) {
  __shared__ float qs[SKC][ST + 4];
  __shared__ float ks[SKC][ST + 4];
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
  const int t = threadIdx.x, tx = t % 16, ty = t / 16;

  float acc[4][4];
#pragma unroll
  for (int r = 0; r < 4; ++r)
#pragma unroll
    for (int c = 0; c < 4; ++c) acc[r][c] = 0.f;

  // loader: 64 rows x 32 floats = 512 float4; thread t loads rows lr and lr + 32
  const int lr = t / 8, lc = (t % 8) * 4;
  for (int d0 = 0; d0 < D; d0 += SKC) {
#pragma unroll
    for (int h = 0; h < 2; ++h) {
      const int row = lr + 32 * h;
      float4 qv = make_float4(0.f, 0.f, 0.f, 0.f), kv = qv;
      if (i0 + row < a.n_q) qv = *reinterpret_cast<const float4*>(qb + (int64_t)(i0 + row) * D + d0 + lc);
      if (j0 + row < a.n_k) kv = *reinterpret_cast<const float4*>(kb + (int64_t)(j0 + row) * D + d0 + lc);
      qs[lc + 0][row] = qv.x; qs[lc + 1][row] = qv.y; qs[lc + 2][row] = qv.z; qs[lc + 3][row] = qv.w;
      ks[lc + 0][row] = kv.x; ks[lc + 1][row] = kv.y; ks[lc + 2][row] = kv.z; ks[lc + 3][row] = kv.w;
    }
    __syncthreads();
#pragma unroll 8
    for (int d = 0; d < SKC; ++d) {
      const float4 qv = *reinterpret_cast<const float4*>(&qs[d][ty * 4]);
      const float4 kv = *reinterpret_cast<const float4*>(&ks[d][tx * 4]);
      const float qa[4] = {qv.x, qv.y, qv.z, qv.w};
      const float ka[4] = {kv.x, kv.y, kv.z, kv.w};
#pragma unroll
      for (int r = 0; r < 4; ++r)
#pragma unroll
        for (int c = 0; c < 4; ++c) acc[r][c] = fmaf(qa[r], ka[c], acc[r][c]);
    }
    __syncthreads();
  }

  float* srow = a.s + bh * (int64_t)a.n_q * a.n_k;
#pragma unroll
  for (int c = 0; c < 4; ++c) {
    const int j = j0 + tx * 4 + c;
    if (j >= a.n_k || keep_block(a.keep, j)) continue;
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      const int i = i0 + ty * 4 + r;
      if (i < a.n_q) srow[(int64_t)i * a.n_k + j] = a.tau * acc[r][c];
    }
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
