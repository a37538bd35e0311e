// Retained attention mass (Section 4, Analysis): the share of each query's
// dense softmax mass that a block selection keeps, and the token-wise upper
// bound -- the largest share any equally many single keys can hold.
//
//   mass_kernel          mass_t = exp(lse_sel_t - lse_all_t), elementwise.
//   topk_scores_kernel   logits s_t,u = scale * q_t . k_u in fp32 for a few
//                        sampled query rows of a head against every key: one
//                        work-group per (head, 1024-key chunk), the sampled
//                        rows held in LDS as fp32, K streamed once.
//   topk_mass_kernel     per (head, sampled row): the n-th largest logit by a
//                        4-pass 8-bit radix select on order-preserving keys,
//                        then sum over the top n of exp(s - lse_all).
#include "device_common.h"

namespace sparstar {

__global__ __launch_bounds__(256) void mass_kernel(const float* lse_sel, const float* lse_all, int64_t n,
                                                   float* mass) {
  for (int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x; i < n; i += (int64_t)gridDim.x * 256) {
    const float a = lse_sel[i];
    mass[i] = a == -INFINITY ? 0.f : expf(a - lse_all[i]);
  }
}

template <int D>
__global__ __launch_bounds__(256) void topk_scores_kernel(TopkArgs a) {
  constexpr int CHUNK = 1024;  // keys per work-group
  __shared__ float qs[kTopkMaxRows * D];
  const int64_t bh = blockIdx.y;
  const int64_t key0 = (int64_t)blockIdx.x * CHUNK;
  const int tid = threadIdx.x;
  for (int i = tid; i < a.n_rows * D; i += 256) {
    const int r = i / D, d = i % D;
    const uint16_t bits = a.q[(bh * a.lq + a.rows[r]) * D + d];
    qs[i] = __uint_as_float((uint32_t)bits << 16);
  }
  __syncthreads();
  for (int m = 0; m < CHUNK / 256; ++m) {
    const int64_t u = key0 + m * 256 + tid;
    if (u >= a.lk) break;
    float kf[D];
    const uint4* kp = reinterpret_cast<const uint4*>(a.k + (bh * a.lk + u) * D);
#pragma unroll
    for (int c = 0; c < D / 8; ++c) {
      const uint4 w = kp[c];
      kf[8 * c + 0] = bf16_lo(w.x);
      kf[8 * c + 1] = bf16_hi(w.x);
      kf[8 * c + 2] = bf16_lo(w.y);
      kf[8 * c + 3] = bf16_hi(w.y);
      kf[8 * c + 4] = bf16_lo(w.z);
      kf[8 * c + 5] = bf16_hi(w.z);
      kf[8 * c + 6] = bf16_lo(w.w);
      kf[8 * c + 7] = bf16_hi(w.w);
    }
    for (int r = 0; r < a.n_rows; ++r) {
      float acc = 0.f;
#pragma unroll
      for (int d = 0; d < D; ++d) acc = fmaf(qs[r * D + d], kf[d], acc);
      a.scores[(bh * a.n_rows + r) * a.lk + u] = acc * a.scale;
    }
  }
}

// fp32 -> uint32 with the same order (-0 folded onto +0)
__device__ __forceinline__ uint32_t order_key(float x) {
  uint32_t u = __float_as_uint(x == 0.f ? 0.f : x);
  return (u & 0x80000000u) ? ~u : (u | 0x80000000u);
}

__global__ __launch_bounds__(256) void topk_mass_kernel(TopkArgs a) {
  __shared__ uint32_t hist[256];
  __shared__ uint32_t sel[2];  // chosen digit, count of keys above it
  __shared__ float part[256];
  const int64_t row = blockIdx.x;  // bh * n_rows + r
  const int64_t bh = row / a.n_rows;
  const int r = (int)(row % a.n_rows);
  const int tid = threadIdx.x;
  const float* s = a.scores + row * a.lk;
  int64_t want = a.n_tokens[row];
  want = want < 0 ? 0 : (want > a.lk ? a.lk : want);
  const float lse = a.lse_all[bh * a.lq + a.rows[r]];
  if (want == 0) {
    if (tid == 0) a.mass[row] = 0.f;
    return;
  }
  // radix select of the want-th largest key, most significant digit first
  uint32_t prefix = 0, pmask = 0;
  uint32_t above = 0;  // keys known to be larger than the selected prefix
  for (int shift = 24; shift >= 0; shift -= 8) {
    hist[tid] = 0;
    __syncthreads();
    for (int64_t u = tid; u < a.lk; u += 256) {
      const uint32_t key = order_key(s[u]);
      if ((key & pmask) == prefix) atomicAdd(&hist[(key >> shift) & 255u], 1u);
    }
    __syncthreads();
    if (tid == 0) {
      uint32_t acc = above;
      int dgt = 255;
      for (; dgt > 0; --dgt) {
        if (acc + hist[dgt] >= (uint32_t)want) break;
        acc += hist[dgt];
      }
      sel[0] = (uint32_t)dgt;
      sel[1] = acc;
    }
    __syncthreads();
    prefix |= sel[0] << shift;
    pmask |= 255u << shift;
    above = sel[1];
    __syncthreads();
  }
  // prefix is the want-th largest key; `above` keys are strictly larger
  float sum = 0.f;
  for (int64_t u = tid; u < a.lk; u += 256) {
    const float x = s[u];
    if (order_key(x) > prefix) sum += expf(x - lse);
  }
  part[tid] = sum;
  __syncthreads();
  for (int w = 128; w > 0; w >>= 1) {
    if (tid < w) part[tid] += part[tid + w];
    __syncthreads();
  }
  if (tid == 0) {
    // the ties at the threshold fill the remaining places
    const uint32_t k = prefix;
    const uint32_t u = (k & 0x80000000u) ? (k & 0x7fffffffu) : ~k;
    const float t = __uint_as_float(u);
    a.mass[row] = part[0] + (float)(want - (int64_t)above) * expf(t - lse);
  }
}

hipError_t launch_retained_mass(const float* lse_sel, const float* lse_all, int64_t n, float* mass,
                                hipStream_t stream) {
  if (n == 0) return hipSuccess;
  int64_t blocks = (n + 255) / 256;
  if (blocks > 65536) blocks = 65536;
  mass_kernel<<<blocks, 256, 0, stream>>>(lse_sel, lse_all, n, mass);
  return hipGetLastError();
}

hipError_t launch_topk_mass(const TopkArgs& a, int d, hipStream_t stream) {
  if (a.bh == 0 || a.n_rows == 0) return hipSuccess;
  const dim3 grid((unsigned)((a.lk + 1023) / 1024), (unsigned)a.bh);
  if (d == 128) topk_scores_kernel<128><<<grid, 256, 0, stream>>>(a);
  else if (d == 64) topk_scores_kernel<64><<<grid, 256, 0, stream>>>(a);
  else return hipErrorInvalidValue;
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  topk_mass_kernel<<<(unsigned)(a.bh * a.n_rows), 256, 0, stream>>>(a);
  return hipGetLastError();
}

}  // namespace sparstar
