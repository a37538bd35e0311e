// Block-sparse attention forward (Eq. 7, Section 5.3) and its dense variant.
//
// Work decomposition.  One work-group per (batch*head, query block of BLK
// rows), launched head-major so that all eight XCDs work on the same head at a
// time and that head's K/V (74 MB at the 720p shape) stays resident in the
// 256 MB last-level cache.  The work-group has 2 * BLK/32 wavefronts: wave w
// owns the 32-row query slice (w % (BLK/32)) and the key half (w / (BLK/32)) of
// every key block, so each wave touches only half of each K and V tile and two
// waves per SIMD stay resident (<= 256 VGPRs each).
//
// Per key block of the query block's ascending list:
//   * K and V tiles (BLK x D each) are copied row-major into LDS with coalesced
//     16-byte loads and stores (row pitches padded so that the operand reads
//     below are bank-conflict-free).  LDS is double-buffered: the tile of step
//     t+1 is written while step t computes (one barrier per step) and the global
//     loads of step t+2 are in flight during the whole step;
//   * S^T = K Q^T on v_mfma_f32_32x32x16_bf16 (fp32 accumulate).  The
//     transpose leaves each lane holding 16 keys of ONE query column -- exactly
//     the B-operand layout P^T needs -- so the softmax state is lane-local up to
//     one cross-half (lane l <-> l+32) max per step (v_permlane32_swap);
//   * online softmax in the log2 domain: the scale is folded into one FMA, the
//     exponential is the bare v_exp_f32, and O is rescaled lazily, only when a
//     query's running maximum grows by more than 2^8 (P then stays <= 256,
//     harmless in fp32 and bf16), which skips nearly all rescales;
//   * O^T += V^T P^T on the same MFMA (P rounded to bf16 once).  The V^T
//     operand comes straight from the row-major V tile through the LDS
//     transpose read ds_read_b64_tr_b16 (in each 16-lane group, source lane s
//     points at V[r0 + s/4][4 (c0 + s%4)], and lane j receives
//     V[r0 .. r0+3][4 c0 + j]: 4 keys of one d column).
// The two key halves of a query slice each hold a partial (m, l, O); they are
// merged once through LDS at the end.  O = O^T / l in bf16, lse = ln2*(m + log2 l).
//
// MFMA layouts (v_mfma_f32_32x32x16_bf16, lane l, h = l / 32):
//   A[m][k]: m = l % 32, k = 8h + i (i = 0..7 of the lane's bf16x8)
//   B[k][n]: n = l % 32, k = 8h + i
//   C[m][n]: n = l % 32, m = 8 (a / 4) + 4h + (a % 4), accumulator a = 0..15
// A and B only need to agree on k, so keys may be permuted consistently: the
// P^T operand reuses the S^T C layout directly, and the V^T operand reads the
// same key permutation.
#include <type_traits>

#include "device_common.h"

namespace sparstar {

typedef short s16x4 __attribute__((ext_vector_type(4)));
typedef short s16x8 __attribute__((ext_vector_type(8)));
typedef float f32x2 __attribute__((ext_vector_type(2)));
typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
typedef _Float16 f16x4 __attribute__((ext_vector_type(4)));
typedef _Float16 f16x8 __attribute__((ext_vector_type(8)));

template <int D, int BLK>
struct AttnCfg {
  static constexpr int NQS = BLK / 32;        // 32-row query slices
  static constexpr int NW = 2 * NQS;          // waves: (query slice, key half)
  static constexpr int NT = 64 * NW;          // threads
  static constexpr int KH = BLK / 2;          // keys per key half
  static constexpr int KT = KH / 32;          // 32-key sub-tiles per wave and step
  static constexpr int DS = D / 16;           // MFMA k-steps over D
  static constexpr int DT = D / 32;           // 32-row d tiles of O^T
  static constexpr int KLD = D + 8;           // K row pitch (bf16): consecutive rows 4 banks apart
  static constexpr int VLD = D + 32;          // V row pitch (bf16): consecutive rows 16 banks apart, so the
                                              // two 16-lane groups of a transpose read fill disjoint banks
  static constexpr int K_ELEMS = BLK * KLD;
  static constexpr int V_ELEMS = BLK * VLD;
  static constexpr int STAGE = K_ELEMS + V_ELEMS;
  static constexpr int CPR = D / 8;                 // 16-byte chunks per row
  static constexpr int CH = BLK * CPR / NT;         // chunks per thread, for each of K and V
  static constexpr int ROWS_PER_PASS = NT / CPR;    // rows covered by one chunk pass
  static_assert(CH * NT == BLK * CPR, "tile split");
};

__device__ __forceinline__ float half_swap_max(float x) {
  const auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  return fmaxf(__uint_as_float(r[0]), __uint_as_float(r[1]));
}

__device__ __forceinline__ float half_swap_sum(float x) {
  const auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  return __uint_as_float(r[0]) + __uint_as_float(r[1]);
}

__device__ __forceinline__ uint32_t pack2_bf16(float lo, float hi) {
  return __builtin_bit_cast(uint32_t, __builtin_convertvector((f32x2){lo, hi}, bf16x2));
}

__device__ __forceinline__ s16x4 lds_read_tr(const uint16_t* p) {
  return __builtin_amdgcn_ds_read_tr16_b64_v4i16(
      (__attribute__((address_space(3))) s16x4*)(const_cast<uint16_t*>(p)));
}

__device__ __forceinline__ __amdgpu_buffer_rsrc_t make_rsrc(const void* base, uint32_t bytes) {
  // raw (stride 0) buffer; reads past `bytes` return zeros
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(base), (short)0, (int)bytes, 0x00020000);
}

__device__ __forceinline__ uint4 buf_load16(__amdgpu_buffer_rsrc_t r, uint32_t voff, uint32_t soff) {
  return __builtin_bit_cast(uint4, __builtin_amdgcn_raw_buffer_load_b128(r, voff, soff, 0));
}

template <int D, int BLK, bool DENSE, bool SPLIT>
__global__ __launch_bounds__(BLK * 4) __attribute__((amdgpu_waves_per_eu(2, 2)))
void attn_fwd_kernel(AttnArgs a) {
  using C = AttnCfg<D, BLK>;
  // K double buffer, then V double buffer.  Step t reads K of tile t+1 (for the
  // scores one step ahead) and V of tile t, while K of t+2 and V of t+1 are
  // written into the other halves.
  __shared__ __attribute__((aligned(16))) uint16_t smem[2 * C::K_ELEMS + 2 * C::V_ELEMS];
  __shared__ int list_pos[2];

  // Work item.  Work-groups are dispatched round-robin over the eight XCDs, so
  // with the key-range split the work-group id decodes as
  //   id = ((bh * S + s) * n_q + qb) * 8 + x,  range r = 8 s + x,  S = kSplits / 8:
  // XCD x runs range x of every query block of head bh, then range 8 + x, ...,
  // and its L2 holds one range of the head's K/V at a time.
  int split = 0;
  int64_t work = blockIdx.x;
  if constexpr (SPLIT) {
    constexpr int S = kSplits / 8;
    const int64_t x = blockIdx.x % 8, rest = blockIdx.x / 8;
    const int64_t qbi = rest % a.n_q, rest2 = rest / a.n_q;
    split = (int)((rest2 % S) * 8 + x);
    work = (rest2 / S) * a.n_q + qbi;
  }
  const int64_t bh = work / a.n_q;
  const int qb = (int)(work % a.n_q);
  const int blk_lo = SPLIT ? (int)((int64_t)split * a.n_k / kSplits) : 0;
  const int blk_hi = SPLIT ? (int)((int64_t)(split + 1) * a.n_k / kSplits) : a.n_k;

  const int tid = threadIdx.x, wave = tid / 64, lane = tid % 64;
  const int l32 = lane % 32, hh = lane / 32;
  const int qs = wave % C::NQS;   // query slice
  const int kh = wave / C::NQS;   // key half

  // ---- list positions [pos_lo, pos_hi) that may hold blocks of [blk_lo, blk_hi)
  int pos_lo, pos_hi;
  const int32_t* list = nullptr;
  if constexpr (DENSE) {
    pos_lo = blk_lo;
    pos_hi = blk_hi;
  } else {
    const int64_t r = bh * a.n_q + qb;
    int nblk = a.kv_num_blocks[r];
    nblk = nblk < 0 ? 0 : (nblk > a.stride ? a.stride : nblk);
    list = a.kv_indices + r * a.stride;
    if constexpr (SPLIT) {
      // an ascending list: the range starts after the entries < blk_lo and ends
      // after the entries < blk_hi
      if (tid < 2) list_pos[tid] = 0;
      __syncthreads();
      int c_lo = 0, c_hi = 0;
      for (int i = tid; i < nblk; i += C::NT) {
        const int j = list[i];
        c_lo += j < blk_lo;
        c_hi += j < blk_hi;
      }
#pragma unroll
      for (int off = 32; off > 0; off >>= 1) {
        c_lo += __shfl_xor(c_lo, off, 64);
        c_hi += __shfl_xor(c_hi, off, 64);
      }
      if (lane == 0) {
        atomicAdd(&list_pos[0], c_lo);
        atomicAdd(&list_pos[1], c_hi);
      }
      __syncthreads();
      pos_lo = list_pos[0];
      pos_hi = list_pos[1];
    } else {
      pos_lo = 0;
      pos_hi = nblk;
    }
  }

  // ---- block cursor: the next list entry is prefetched one call ahead with a
  // vector-memory load, so its latency hides behind a whole step
  int cur_pos = pos_lo;
  // (the range check covers the vector offset, so the position goes there:
  // reading one past the end returns 0 instead of touching memory)
  const __amdgpu_buffer_rsrc_t list_rs = make_rsrc(list, DENSE ? 0u : (uint32_t)pos_hi * 4u);
  uint32_t pf = 0;
  if constexpr (!DENSE) pf = __builtin_amdgcn_raw_buffer_load_b32(list_rs, (uint32_t)cur_pos * 4u, 0u, 0);
  // next block of [blk_lo, blk_hi) in list order, or -1
  auto fetch_next = [&]() -> int {
    if constexpr (DENSE) {
      return cur_pos < pos_hi ? cur_pos++ : -1;
    } else {
      while (cur_pos < pos_hi) {
        const int j = __builtin_amdgcn_readfirstlane((int)pf);
        ++cur_pos;
        pf = __builtin_amdgcn_raw_buffer_load_b32(list_rs, (uint32_t)cur_pos * 4u, 0u, 0);
        if (j >= blk_lo && j < blk_hi) return j;
      }
      return -1;
    }
  };

  // ---- Q fragment (B operand of S^T = K Q^T): Q[q][16 s + 8 hh .. +7]
  const int64_t q_row = (int64_t)qb * BLK + qs * 32 + l32;
  const bool q_ok = q_row < a.lq;
  const uint16_t* qp = a.q + (bh * a.lq + (q_ok ? q_row : 0)) * D;
  bf16x8 qf[C::DS];
#pragma unroll
  for (int s = 0; s < C::DS; ++s) {
    const uint4 u = q_ok ? *reinterpret_cast<const uint4*>(qp + 16 * s + 8 * hh) : make_uint4(0, 0, 0, 0);
    qf[s] = __builtin_bit_cast(bf16x8, u);
  }

  f32x16 acc_o[C::DT];
#pragma unroll
  for (int t = 0; t < C::DT; ++t)
#pragma unroll
    for (int e = 0; e < 16; ++e) acc_o[t][e] = 0.f;
  float m_run = -INFINITY;  // running max (log2 domain), shared by both lane halves
  float l_run = 0.f;        // this lane's partial row sum of the bf16 P it applied

  // ---- tile copy through buffer loads: thread tid moves chunk
  // (row0 + p * ROWS_PER_PASS, col8) of a tile.  Each tile gets its own
  // descriptor (base at the tile, records = bytes left in the head), so rows
  // past Lk read as zeros; the per-lane offsets stay in the range-checked
  // vector offset.
  const int row0 = tid / C::CPR, col8 = (tid % C::CPR) * 8;
  const uint16_t* const kbase = a.k + bh * a.lk * D;
  const uint16_t* const vbase = a.v + bh * a.lk * D;
  constexpr uint32_t TILE_BYTES = BLK * D * 2;
  uint32_t voff[C::CH];
#pragma unroll
  for (int p = 0; p < C::CH; ++p) voff[p] = (uint32_t)((row0 + p * C::ROWS_PER_PASS) * D + col8) * 2u;
  const uint32_t last_bytes = (uint32_t)(a.lk - (int64_t)(a.n_k - 1) * BLK) * (D * 2);
  auto tile_bytes = [&](int blk) -> uint32_t { return blk == a.n_k - 1 ? last_bytes : TILE_BYTES; };
  uint4 kreg[C::CH], vreg[C::CH];
  auto load_k = [&](int blk) {
    const __amdgpu_buffer_rsrc_t rs = make_rsrc(kbase + (int64_t)blk * BLK * D, tile_bytes(blk));
#pragma unroll
    for (int p = 0; p < C::CH; ++p) kreg[p] = buf_load16(rs, voff[p], 0u);
  };
  auto load_v = [&](int blk) {
    const __amdgpu_buffer_rsrc_t rs = make_rsrc(vbase + (int64_t)blk * BLK * D, tile_bytes(blk));
#pragma unroll
    for (int p = 0; p < C::CH; ++p) vreg[p] = buf_load16(rs, voff[p], 0u);
  };
  uint16_t* const kst = smem + row0 * C::KLD + col8;
  uint16_t* const vst = smem + 2 * C::K_ELEMS + row0 * C::VLD + col8;
  auto store_k = [&](int buf) {
#pragma unroll
    for (int p = 0; p < C::CH; ++p)
      *reinterpret_cast<uint4*>(kst + buf * C::K_ELEMS + p * C::ROWS_PER_PASS * C::KLD) = kreg[p];
  };
  auto store_v = [&](int buf) {
#pragma unroll
    for (int p = 0; p < C::CH; ++p)
      *reinterpret_cast<uint4*>(vst + buf * C::V_ELEMS + p * C::ROWS_PER_PASS * C::VLD) = vreg[p];
  };

  // per-lane LDS read bases (buffer 0)
  const uint16_t* const k_rd = smem + (kh * C::KH + l32) * C::KLD + 8 * hh;
  const int grp = lane >> 4, sl = lane & 15;
  const uint16_t* const v_rd =
      smem + 2 * C::K_ELEMS + (kh * C::KH + 4 * hh + (sl >> 2)) * C::VLD + 16 * (grp & 1) + 4 * (sl & 3);

  // ---- S^T = K Q^T for this wave's keys of the K tile in buffer kb
  auto scores = [&](int kb, f32x16* acc) {
    const uint16_t* ks = k_rd + kb * C::K_ELEMS;
#pragma unroll
    for (int kt = 0; kt < C::KT; ++kt) {
#pragma unroll
      for (int e = 0; e < 16; ++e) acc[kt][e] = 0.f;
#pragma unroll
      for (int s = 0; s < C::DS; ++s) {
        const uint4 u = *reinterpret_cast<const uint4*>(ks + kt * 32 * C::KLD + 16 * s);
        acc[kt] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(__builtin_bit_cast(bf16x8, u), qf[s], acc[kt], 0, 0, 0);
      }
    }
  };

  const float sl2 = a.scale_log2;
  const bf16x2 ones = {(__bf16)1.0f, (__bf16)1.0f};

  // keys >= Lk of a partial last block get -inf scores
  auto mask_tail = [&](f32x16* acc, int blk) {
    const int64_t key0 = (int64_t)blk * BLK;
    if (key0 + BLK > a.lk) {
#pragma unroll
      for (int kt = 0; kt < C::KT; ++kt)
#pragma unroll
        for (int e = 0; e < 16; ++e) {
          const int key = kh * C::KH + kt * 32 + 8 * (e / 4) + 4 * hh + (e % 4);
          if (key0 + key >= a.lk) acc[kt][e] = -INFINITY;
        }
    }
  };
  // running max for a new score tile, with lazy rescaling: O and l are only
  // rescaled when a query's maximum grows by more than 2^8
  auto update_max = [&](const f32x16* acc) {
    float mx = -INFINITY;
#pragma unroll
    for (int kt = 0; kt < C::KT; ++kt)
#pragma unroll
      for (int e = 0; e < 16; ++e) mx = fmaxf(mx, acc[kt][e]);
    mx = half_swap_max(mx) * sl2;  // the tile's max logit (log2 domain) for the lane's query
    if (__any(mx > m_run + 8.0f)) {
      const float m_new = fmaxf(m_run, mx);
      const float alpha = m_run == -INFINITY ? 0.f : __builtin_amdgcn_exp2f(m_run - m_new);
      l_run *= alpha;
#pragma unroll
      for (int t = 0; t < C::DT; ++t)
#pragma unroll
        for (int e = 0; e < 16; ++e) acc_o[t][e] *= alpha;
      m_run = m_new;
    }
  };

  // ---- prologue: K of tiles 0 and 1 and V of tile 0 staged, K of tile 2 and
  // V of tile 1 in flight, S of tile 0 computed and its max applied
  int b0 = fetch_next();
  int b1 = fetch_next();
  int b2 = fetch_next();
  f32x16 acc_s[C::KT];
  if (b0 >= 0) {
    load_k(b0);
    load_v(b0);
    store_k(0);
    store_v(0);
  }
  if (b1 >= 0) {
    load_k(b1);
    store_k(1);
    load_v(b1);
  }
  if (b2 >= 0) load_k(b2);
  __syncthreads();
  if (b0 >= 0) {
    scores(0, acc_s);
    mask_tail(acc_s, b0);
    update_max(acc_s);
  }
  __syncthreads();  // K buffer 0 is rewritten in the first step

  // One step: P and O += P V of tile t (block b0) while the scores of tile t+1
  // (block b1) run on the matrix cores.  The compute block has no branch, and
  // sched_group_barrier interleaves each score MFMA with the exponentials of
  // the current tile and each P V MFMA with a row-sum update, so the VALU work
  // hides under the matrix-core work of the same wave.
  auto step = [&](auto parity) {
    constexpr int P = decltype(parity)::value;
    f32x16 acc_n[C::KT];
    const float neg_m = m_run == -INFINITY ? 0.f : -m_run;

    // K of tile t+1 (buffer 1-P; stale but harmless when there is no such tile)
    uint4 kf[C::KT][C::DS];
    const uint16_t* ks = k_rd + (1 - P) * C::K_ELEMS;
#pragma unroll
    for (int kt = 0; kt < C::KT; ++kt)
#pragma unroll
      for (int s = 0; s < C::DS; ++s) kf[kt][s] = *reinterpret_cast<const uint4*>(ks + kt * 32 * C::KLD + 16 * s);

    uint32_t pk[C::KT][8];  // bf16 pairs of P^T, per 32-key sub-tile
#pragma unroll
    for (int kt = 0; kt < C::KT; ++kt) {
#pragma unroll
      for (int e = 0; e < 16; ++e) acc_n[kt][e] = 0.f;
#pragma unroll
      for (int s = 0; s < C::DS; ++s)
        acc_n[kt] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(__builtin_bit_cast(bf16x8, kf[kt][s]), qf[s], acc_n[kt],
                                                            0, 0, 0);
#pragma unroll
      for (int e = 0; e < 16; e += 2) {
        const float p0 = __builtin_amdgcn_exp2f(fmaf(acc_s[kt][e], sl2, neg_m));
        const float p1 = __builtin_amdgcn_exp2f(fmaf(acc_s[kt][e + 1], sl2, neg_m));
        pk[kt][e / 2] = __builtin_bit_cast(uint32_t, __builtin_convertvector((f32x2){p0, p1}, bf16x2));
      }
    }

    // O^T += V^T P^T over 16-key k-steps (V tile of block b0 in buffer P)
    const uint16_t* vs = v_rd + P * C::V_ELEMS;
#pragma unroll
    for (int kt = 0; kt < C::KT; ++kt)
#pragma unroll
      for (int half = 0; half < 2; ++half) {
        // accumulators a = 8 half + i of sub-tile kt hold keys
        //   base + 4 hh + i (i = 0..3) and base + 8 + 4 hh + (i - 4) (i = 4..7),
        // base = kh * KH + 32 kt + 16 half; the two transpose reads fetch the
        // same keys of V for d = 32 t + l % 32.
        uint4 pu;
        pu.x = pk[kt][4 * half + 0];
        pu.y = pk[kt][4 * half + 1];
        pu.z = pk[kt][4 * half + 2];
        pu.w = pk[kt][4 * half + 3];
        const bf16x8 pb = __builtin_bit_cast(bf16x8, pu);
#pragma unroll
        for (int t = 0; t < C::DT; ++t) {
          const uint16_t* vr = vs + (32 * kt + 16 * half) * C::VLD + 32 * t;
          const s16x4 v0 = lds_read_tr(vr);
          const s16x4 v1 = lds_read_tr(vr + 8 * C::VLD);
          const s16x8 vv = __builtin_shufflevector(v0, v1, 0, 1, 2, 3, 4, 5, 6, 7);
          acc_o[t] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(__builtin_bit_cast(bf16x8, vv), pb, acc_o[t], 0, 0, 0);
        }
#pragma unroll
        for (int i = 0; i < 4; ++i)
          l_run = __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(bf16x2, pk[kt][4 * half + i]), ones, l_run,
                                                  false);
      }
    if constexpr (C::KT == 1 && C::DS == 8 && C::DT == 4) {
      // K reads first; then 8 x (score MFMA + 5 VALU of the exponentials + 2 V
      // transpose reads, so the V operands land while the exponentials run);
      // then 8 x (P V MFMA + 1 row-sum VALU)
      __builtin_amdgcn_sched_group_barrier(0x100, 8, 0);
#pragma unroll
      for (int i = 0; i < 8; ++i) {
        __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
        __builtin_amdgcn_sched_group_barrier(0x002, 5, 0);
        __builtin_amdgcn_sched_group_barrier(0x100, 2, 0);
      }
#pragma unroll
      for (int i = 0; i < 8; ++i) {
        __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
        __builtin_amdgcn_sched_group_barrier(0x002, 1, 0);
      }
    }

    // scores of tile t+1: tail mask and running max (rescales O if needed)
    if (b1 >= 0) {
      mask_tail(acc_n, b1);
      update_max(acc_n);
    }

    // stage K of t+2 and V of t+1, start the loads of K of t+3 and V of t+2
    if (b2 >= 0) store_k(P);
    if (b1 >= 0) store_v(1 - P);
    const int b3 = fetch_next();
    if (b3 >= 0) load_k(b3);
    if (b2 >= 0) load_v(b2);
    __syncthreads();
#pragma unroll
    for (int kt = 0; kt < C::KT; ++kt) acc_s[kt] = acc_n[kt];
    b0 = b1;
    b1 = b2;
    b2 = b3;
  };

  while (b0 >= 0) {
    step(std::integral_constant<int, 0>{});
    if (b0 < 0) break;
    step(std::integral_constant<int, 1>{});
  }

  // ---- merge the two key halves of each query slice, then write O and lse
  l_run = half_swap_sum(l_run);  // both lane halves now hold the slice's partial sum
  float* mrg = reinterpret_cast<float*>(smem);  // [NQS][2 + 16 DT][64] floats; tile buffers are free now
  constexpr int MR = 2 + 16 * C::DT;
  static_assert(C::NQS * MR * 64 * 4 <= (2 * C::K_ELEMS + 2 * C::V_ELEMS) * 2, "merge buffer fits in LDS");
  float* my = mrg + qs * MR * 64;
  if (kh == 1) {
    my[0 * 64 + lane] = m_run;
    my[1 * 64 + lane] = l_run;
#pragma unroll
    for (int t = 0; t < C::DT; ++t)
#pragma unroll
      for (int e = 0; e < 16; ++e) my[(2 + 16 * t + e) * 64 + lane] = acc_o[t][e];
  }
  __syncthreads();
  if (kh == 0) {
    const float m1 = my[0 * 64 + lane], l1 = my[1 * 64 + lane];
    const float mm = fmaxf(m_run, m1);
    const float a0 = m_run == -INFINITY ? 0.f : exp2f(m_run - mm);
    const float a1 = m1 == -INFINITY ? 0.f : exp2f(m1 - mm);
    const float l = l_run * a0 + l1 * a1;
    const float inv = l > 0.f ? 1.f / l : 0.f;
    if (SPLIT && q_ok) {
      const int64_t prow = (work * kSplits + split) * BLK + qs * 32 + l32;
      _Float16* po = reinterpret_cast<_Float16*>(a.part_o) + prow * D;
#pragma unroll
      for (int t = 0; t < C::DT; ++t)
#pragma unroll
        for (int g = 0; g < 4; ++g) {
          const int d = 32 * t + 8 * g + 4 * hh;
          f16x4 w;
#pragma unroll
          for (int e = 0; e < 4; ++e)
            w[e] = (_Float16)((acc_o[t][4 * g + e] * a0 + my[(2 + 16 * t + 4 * g + e) * 64 + lane] * a1) * inv);
          *reinterpret_cast<f16x4*>(po + d) = w;
        }
      if (hh == 0) {
        a.part_ml[2 * prow] = mm;
        a.part_ml[2 * prow + 1] = l;
      }
    }
    if (!SPLIT && q_ok) {
      uint16_t* op = a.o + (bh * a.lq + q_row) * D;
#pragma unroll
      for (int t = 0; t < C::DT; ++t)
#pragma unroll
        for (int g = 0; g < 4; ++g) {
          const int d = 32 * t + 8 * g + 4 * hh;
          float o[4];
#pragma unroll
          for (int e = 0; e < 4; ++e)
            o[e] = (acc_o[t][4 * g + e] * a0 + my[(2 + 16 * t + 4 * g + e) * 64 + lane] * a1) * inv;
          uint2 w;
          w.x = pack2_bf16(o[0], o[1]);
          w.y = pack2_bf16(o[2], o[3]);
          *reinterpret_cast<uint2*>(op + d) = w;
        }
      if (a.lse != nullptr && hh == 0)
        a.lse[bh * a.lq + q_row] = l > 0.f ? (mm + log2f(l)) * 0.69314718055994530942f : -INFINITY;
    }
  }
}

// Combines the kSplits partial results of one query block:
//   O = sum_r w_r O_r / sum_r w_r,  w_r = l_r 2^(m_r - M),  M = max_r m_r,
//   lse = ln2 (M + log2 sum_r w_r).
// Ranges with no visible key (l_r = 0) have weight 0 and their O_r is not read.
template <int D, int BLK>
__global__ __launch_bounds__(256) void attn_merge_kernel(AttnArgs a) {
  __shared__ float wts[kSplits][BLK];
  const int64_t work = blockIdx.x;
  const int64_t bh = work / a.n_q;
  const int qb = (int)(work % a.n_q);
  const int tid = threadIdx.x;
  const int64_t rows = a.lq - (int64_t)qb * BLK;
  for (int row = tid; row < BLK; row += 256) {
    float m[kSplits], l[kSplits], mm = -INFINITY;
#pragma unroll
    for (int r = 0; r < kSplits; ++r) {
      const int64_t prow = (work * kSplits + r) * BLK + row;
      m[r] = a.part_ml[2 * prow];
      l[r] = a.part_ml[2 * prow + 1];
      if (l[r] > 0.f) mm = fmaxf(mm, m[r]);
    }
    float tot = 0.f;
#pragma unroll
    for (int r = 0; r < kSplits; ++r) {
      const float w = l[r] > 0.f ? l[r] * exp2f(m[r] - mm) : 0.f;
      wts[r][row] = w;
      tot += w;
    }
    const float inv = tot > 0.f ? 1.f / tot : 0.f;
#pragma unroll
    for (int r = 0; r < kSplits; ++r) wts[r][row] *= inv;
    if (row < rows && a.lse != nullptr)
      a.lse[bh * a.lq + (int64_t)qb * BLK + row] = tot > 0.f ? (mm + log2f(tot)) * 0.69314718055994530942f : -INFINITY;
  }
  __syncthreads();
  constexpr int CPR = D / 8;
  for (int c = tid; c < BLK * CPR; c += 256) {
    const int row = c / CPR, d0 = (c % CPR) * 8;
    if (row >= rows) continue;
    float acc[8] = {0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int r = 0; r < kSplits; ++r) {
      const float w = wts[r][row];
      if (w == 0.f) continue;
      const int64_t prow = (work * kSplits + r) * BLK + row;
      const f16x8 v = *reinterpret_cast<const f16x8*>(reinterpret_cast<const _Float16*>(a.part_o) + prow * D + d0);
#pragma unroll
      for (int e = 0; e < 8; ++e) acc[e] = fmaf(w, (float)v[e], acc[e]);
    }
    uint4 o;
    o.x = pack2_bf16(acc[0], acc[1]);
    o.y = pack2_bf16(acc[2], acc[3]);
    o.z = pack2_bf16(acc[4], acc[5]);
    o.w = pack2_bf16(acc[6], acc[7]);
    *reinterpret_cast<uint4*>(a.o + (bh * a.lq + (int64_t)qb * BLK + row) * D + d0) = o;
  }
}

template <int D, int BLK>
static hipError_t launch_cfg(const AttnArgs& a, bool dense, hipStream_t stream) {
  const int64_t items = (int64_t)a.bh * a.n_q;
  if (items == 0) return hipSuccess;
  constexpr int NT = AttnCfg<D, BLK>::NT;
  if (a.part_o != nullptr) {
    if (dense) attn_fwd_kernel<D, BLK, true, true><<<items * kSplits, NT, 0, stream>>>(a);
    else attn_fwd_kernel<D, BLK, false, true><<<items * kSplits, NT, 0, stream>>>(a);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    attn_merge_kernel<D, BLK><<<items, 256, 0, stream>>>(a);
  } else {
    if (dense) attn_fwd_kernel<D, BLK, true, false><<<items, NT, 0, stream>>>(a);
    else attn_fwd_kernel<D, BLK, false, false><<<items, NT, 0, stream>>>(a);
  }
  return hipGetLastError();
}

size_t attn_workspace_bytes(int64_t bh, int64_t n_q, int64_t n_k, int d, int block) {
  if (n_k < kSplits) return 0;  // fewer key blocks than ranges: single pass
  const int64_t rows = bh * n_q * kSplits * block;
  const size_t o_bytes = (size_t(rows * d) * 2 + 255) & ~size_t(255);
  return o_bytes + size_t(rows) * 2 * sizeof(float);
}

hipError_t launch_attn(const AttnArgs& a, int d, int block, bool dense, hipStream_t stream) {
  if (d == 128 && block == 64) return launch_cfg<128, 64>(a, dense, stream);
  if (d == 128 && block == 128) return launch_cfg<128, 128>(a, dense, stream);
  if (d == 64 && block == 64) return launch_cfg<64, 64>(a, dense, stream);
  if (d == 64 && block == 128) return launch_cfg<64, 128>(a, dense, stream);
  return hipErrorInvalidValue;
}

}  // namespace sparstar
