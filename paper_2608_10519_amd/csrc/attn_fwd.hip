// Block-sparse attention forward (Eq. 7, Section 5.3) and its dense variant.
//
// Work decomposition.  One work-group per (batch*head, query block of BLK
// rows, key range), launched so that the eight XCDs stream disjoint key ranges
// of the same head (see the work-item decode below).  The work-group has one
// wavefront per 32-row query slice (two for 64-row blocks, four for 128-row
// blocks), and every wave takes the whole of each key tile, so no key is ever
// split between waves.  Keys come in tiles of KB = BLK / 2 (32 keys for 64-row
// blocks, 64 for 128-row blocks; a key block is two tiles), which sizes the LDS
// ring at 40 KB (80 KB) per work-group at D = 128: four (two) work-groups per
// CU, two waves per SIMD, each under 256 VGPRs.
//
// Per tile of the query block's ascending key-block list:
//   * K and V tiles (KB x D) go from global memory straight into LDS
//     (buffer_load ... lds, 1 KB per wave instruction, coalesced), with no
//     VGPR staging.  LDS holds a ring of three K tiles and two V tiles; each
//     step has two barrier phases (scores, then P V), and each phase's barrier
//     frees the slot the next loads go into;
//   * S^T = K Q^T on v_mfma_f32_32x32x16_bf16 (fp32 accumulate).  The
//     transpose leaves each lane holding 16 keys of ONE query column -- exactly
//     the B-operand layout P^T needs -- so the softmax state is lane-local up to
//     one cross-half (lane l <-> l+32) max per step (v_permlane32_swap);
//   * online softmax in the log2 domain: the scale is folded into one FMA, the
//     exponential is the bare v_exp_f32, and the running maximum is not taken
//     per tile: P is formed against the current one, and only when some lane's
//     sum of a sub-tile's P exceeds 2^8 (so that some p might) is the tile's
//     max taken, O and the sums rescaled by a power of two, and P formed
//     again -- nearly never after the first tiles;
//   * O^T += V^T P^T on the same MFMA (P rounded to bf16 once).  The V^T
//     operand comes straight from the row-major V tile through the LDS
//     transpose read ds_read_b64_tr_b16 (in each 16-lane group, source lane s
//     points at V[r0 + s/4][4 (c0 + s%4)], and lane j receives
//     V[r0 .. r0+3][4 c0 + j]: 4 keys of one d column).
// O = O^T / l in bf16 with l the row sum of the bf16-rounded P, and
// lse = ln2*(m + log2 le) with le the row sum of the unrounded fp32 p.
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

template <int D, int BLK>
struct AttnCfg {
  static constexpr int KB = BLK / 2;          // keys per K/V tile
  static constexpr int SUB = BLK / KB;        // tiles per key block (list entry)
  static constexpr int NQS = BLK / 32;        // 32-row query slices
  static constexpr int NW = NQS;              // waves: one per query slice
  static constexpr int NT = 64 * NW;          // threads
  static constexpr int KT = KB / 32;          // 32-key sub-tiles per step
  static constexpr int DS = D / 16;           // MFMA k-steps over D
  static constexpr int DT = D / 32;           // 32-row d tiles of O^T
  static constexpr int RB = D * 2;            // bytes per K/V row
  static constexpr int CPR = D / 8;           // 16-byte chunks per row
  static constexpr int RPB = 256 / RB;        // rows per 256 bytes (one pass over the 64 LDS banks)
  static constexpr int TILE = KB * D;         // elements per K or V tile
  static constexpr int TILE_BYTES = TILE * 2;
  static constexpr int RPD = 1024 / RB;       // rows per direct-to-LDS wave load (64 lanes x 16 B)
  static constexpr int DPW = TILE_BYTES / 1024 / NW;  // direct loads per wave and tile
  static_assert(DPW * NW * 1024 == TILE_BYTES, "tile split over the waves");
  static_assert(KT * 32 == KB, "32-key sub-tiles");
  static_assert(SUB * KB == BLK, "whole tiles per key block");
};

// LDS tiles are stored unpadded (a direct-to-LDS load writes 1 KB contiguous
// per wave), with the 16-byte chunks of each row XOR-permuted so that both
// operand reads are free of bank conflicts:
//   K (ds_read_b128, 16 lanes per pass: 16 consecutive rows, one chunk):
//     physical chunk = c ^ (r / RPB mod CPR)
//   V (ds_read_b64_tr_b16, 32 lanes per pass: 4 consecutive rows x 4 chunks):
//     physical chunk = c ^ ((r / RPB mod 4) * 4 mod CPR)
template <int D, int BLK>
__device__ __forceinline__ int k_swz(int r) {
  using C = AttnCfg<D, BLK>;
  return (r / C::RPB) % C::CPR;
}
template <int D, int BLK>
__device__ __forceinline__ int v_swz(int r) {
  using C = AttnCfg<D, BLK>;
  return (((r / C::RPB) & 3) << 2) & (C::CPR - 1);
}

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

// Buffer descriptor as four dwords (raw buffer, stride 0, `bytes` records):
// the form the inline-asm direct-to-LDS load takes.
typedef int i32x4 __attribute__((ext_vector_type(4)));
__device__ __forceinline__ i32x4 raw_rsrc(const void* base, uint32_t bytes) {
  const uint64_t p = reinterpret_cast<uint64_t>(base);
  i32x4 r;
  r[0] = __builtin_amdgcn_readfirstlane((int)(uint32_t)p);
  r[1] = __builtin_amdgcn_readfirstlane((int)((uint32_t)(p >> 32) & 0xffffu));
  r[2] = __builtin_amdgcn_readfirstlane((int)bytes);
  r[3] = 0x00020000;
  return r;
}

__device__ __forceinline__ uint32_t lds_addr(const void* p) {
  return (uint32_t)reinterpret_cast<uintptr_t>((const __attribute__((address_space(3))) void*)p);
}

// Direct-to-LDS loads: lane l of a wave-wide load copies 16 bytes from
// buffer offset voff (+ the instruction offset) to LDS byte m0 (+ the same
// instruction offset) + 16 l.  Written as inline assembly so that the compiler
// does not order every later LDS read behind them; each caller waits for these
// loads explicitly (vmcnt) before a barrier makes the tile visible.
//
// A wave's share of one tile: N wave-wide loads after a single M0 write.  The
// instruction offset moves the LDS destination and the memory address alike,
// so load i goes to LDS m0 + 1024 i + 16 l and reads voff[i] + 1024 i (the
// callers pass voff[i] already reduced by 1024 i).
template <int N>
__device__ __forceinline__ void dma_tile(uint32_t m0, const uint32_t* voff, i32x4 rsrc) {
  static_assert(N == 1 || N == 2 || N == 4, "loads per wave and tile");
  if constexpr (N == 1) {
    asm volatile(
        "s_mov_b32 m0, %0\n\t"
        "s_nop 0\n\t"
        "buffer_load_dwordx4 %1, %2, 0 offen lds"
        :
        : "s"(m0), "v"(voff[0]), "s"(rsrc)
        : "memory", "m0");
  } else if constexpr (N == 2) {
    asm volatile(
        "s_mov_b32 m0, %0\n\t"
        "s_nop 0\n\t"
        "buffer_load_dwordx4 %1, %3, 0 offen lds\n\t"
        "buffer_load_dwordx4 %2, %3, 0 offen offset:1024 lds"
        :
        : "s"(m0), "v"(voff[0]), "v"(voff[1]), "s"(rsrc)
        : "memory", "m0");
  } else {
    asm volatile(
        "s_mov_b32 m0, %0\n\t"
        "s_nop 0\n\t"
        "buffer_load_dwordx4 %1, %5, 0 offen lds\n\t"
        "buffer_load_dwordx4 %2, %5, 0 offen offset:1024 lds\n\t"
        "buffer_load_dwordx4 %3, %5, 0 offen offset:2048 lds\n\t"
        "buffer_load_dwordx4 %4, %5, 0 offen offset:3072 lds"
        :
        : "s"(m0), "v"(voff[0]), "v"(voff[1]), "v"(voff[2]), "v"(voff[3]), "s"(rsrc)
        : "memory", "m0");
  }
}

// s_waitcnt with only the vector-memory counter constrained (<= n outstanding)
template <int N>
__device__ __forceinline__ void wait_vmcnt() {
  static_assert(N >= 0 && N < 64, "vmcnt range");
  __builtin_amdgcn_s_waitcnt((N & 15) | ((N >> 4) << 14) | (7 << 4) | (15 << 8));
}

template <int D, int BLK, bool DENSE, bool SPLIT>
__global__ __launch_bounds__(BLK * 2) __attribute__((amdgpu_waves_per_eu(2, 2)))
void attn_fwd_kernel(AttnArgs a) {
  using C = AttnCfg<D, BLK>;
  // Ring of three K tiles and two V tiles.  Step t reads K of tile t+1 (the
  // scores one step ahead) and V of tile t; at its start it issues the
  // direct-to-LDS loads of V of tile t+1 and K of tile t+3 into the slots that
  // the previous step released.  K(j) lives in slot j mod 3, V(j) in j mod 2.
  __shared__ __attribute__((aligned(1024))) uint16_t ks0[C::TILE], ks1[C::TILE], ks2[C::TILE];
  __shared__ __attribute__((aligned(1024))) uint16_t vs0[C::TILE], vs1[C::TILE];

  // Work item.  Work-groups are dispatched round-robin over the eight XCDs, so
  // with the key-range split the work-group id decodes as
  //   id = ((bh * S + s) * n_q + qb) * 8 + x,  range r = 8 s + x,  S = n_splits / 8:
  // XCD x runs range x of every query block of head bh, then range 8 + x, ...,
  // and its L2 holds one range of the head's K/V at a time.
  int split = 0;
  int64_t work = blockIdx.x;
  if constexpr (SPLIT) {
    const int S = a.n_splits / 8;
    const int64_t x = blockIdx.x % 8, rest = blockIdx.x / 8;
    const int64_t qbi = rest % a.n_q, rest2 = rest / a.n_q;
    split = (int)((rest2 % S) * 8 + x);
    work = (rest2 / S) * a.n_q + qbi;
  }
  const int64_t bh = work / a.n_q;
  const int qb = (int)(work % a.n_q);
  const int blk_lo = SPLIT ? (int)((int64_t)split * a.n_k / a.n_splits) : 0;
  const int blk_hi = SPLIT ? (int)((int64_t)(split + 1) * a.n_k / a.n_splits) : a.n_k;

  const int tid = threadIdx.x, lane = tid % 64;
  const int wave = __builtin_amdgcn_readfirstlane(tid / 64);
  const int l32 = lane % 32, hh = lane / 32;
  const int qs = wave;  // query slice

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

  // ---- the list positions [pos_lo, pos_lo + cnt) that hold the blocks of
  // [blk_lo, blk_hi): an ascending list has them after the entries < blk_lo and
  // before the entries >= blk_hi (every wave counts them itself)
  int pos_lo, cnt;
  const int32_t* list = nullptr;
  if constexpr (DENSE) {
    pos_lo = blk_lo;
    cnt = blk_hi - blk_lo;
  } else {
    const int64_t r = bh * a.n_q + qb;
    int nblk = a.kv_num_blocks[r];
    nblk = nblk < 0 ? 0 : (nblk > a.stride ? a.stride : nblk);
    list = a.kv_indices + r * a.stride;
    // 64 x U entries per pass, all loads independent (one memory latency per
    // pass); the counts come from ballots, so they are wave-uniform at once
    constexpr int U = 12;
    int c_lo = 0, c_hi = 0;
    // (the first pass does not wait for the count: it reads up to the stride)
    for (int base = 0; base == 0 || base < nblk; base += 64 * U) {
      int v[U];
#pragma unroll
      for (int u = 0; u < U; ++u) {
        const int i = base + 64 * u + lane;
        v[u] = i < a.stride ? list[i] : 0x7fffffff;
      }
#pragma unroll
      for (int u = 0; u < U; ++u) {
        const bool in = base + 64 * u + lane < nblk;
        c_lo += __builtin_popcountll(__builtin_amdgcn_ballot_w64(in && v[u] < blk_lo));
        c_hi += __builtin_popcountll(__builtin_amdgcn_ballot_w64(in && v[u] < blk_hi));
      }
    }
    pos_lo = __builtin_amdgcn_readfirstlane(c_lo);
    cnt = __builtin_amdgcn_readfirstlane(c_hi) - pos_lo;
  }

  // ---- the key tiles of the item.  Tile j (KB keys) is tile j % SUB of the key
  // block at list position pos_lo + j / SUB.  The entries are held 64 at a time
  // in a VGPR (lane i: entry lbase + i) and picked out with v_readlane, so the
  // loop issues no memory load of its own except one batch load per 64
  // entries.  j >= cnt * SUB, and an entry outside [blk_lo, blk_hi) -- only
  // possible in a list that is not ascending --, give -1: a tile that is
  // loaded as zeros and fully masked.
  int lreg = -1, lbase = 0;
  auto load_batch = [&](int base) {
    lbase = base;
    if constexpr (!DENSE) {
      lreg = base + lane < cnt ? list[pos_lo + base + lane] : -1;
      // consume the load here, so that its wait stays on this rare path and is
      // not merged into the common path of the loop
      asm volatile("; list batch %0" ::"v"(lreg));
    }
  };
  const int ntiles = cnt * C::SUB;
  auto fetch = [&](int j) -> int {
    if (j >= ntiles) return -1;
    const int e = j / C::SUB, sub = j % C::SUB;
    if constexpr (DENSE) {
      int kt = (blk_lo + e) * C::SUB + sub;
      // At 128-row blocks the tile index is hidden from the compiler, which
      // would otherwise precompute the addresses of all six unrolled steps and
      // spill registers to scratch.
      if constexpr (BLK == 128) asm volatile("" : "+s"(kt));
      return kt;
    } else {
      if (e >= lbase + 64) load_batch(lbase + 64);
      const int b = __builtin_amdgcn_readlane(lreg, e - lbase);
      return (b >= blk_lo && b < blk_hi) ? b * C::SUB + sub : -1;
    }
  };

  f32x16 acc_o[C::DT];
#pragma unroll
  for (int t = 0; t < C::DT; ++t)
#pragma unroll
    for (int e = 0; e < 16; ++e) acc_o[t][e] = 0.f;
  float m_run = -INFINITY;  // running max (log2 domain), shared by both lane halves
  // Two row sums per lane (each over the lane's half of the keys):
  //   l_run:  of the bf16-rounded P that multiplies V, so that O = (P V) / l_run
  //           is an exact convex combination of the rounded weights (V = 1 gives
  //           O = 1 exactly);
  //   le_run: of the unrounded fp32 p, for the log-sum-exp.
  float l_run = 0.f;
  float le_run = 0.f;

  // ---- direct-to-LDS tile loads: load i of wave w fills LDS bytes
  // [(DPW w + i) KB, +1 KB); lane l writes 16 bytes at +16 l, i.e. physical
  // chunk l % CPR of row RPD (DPW w + i) + l / CPR, and so reads the logical
  // chunk that the XOR permutation puts there.  Each tile gets its own
  // descriptor (records = bytes of the tile that exist), so rows past Lk and
  // the tiles past the end of the list arrive as zeros.  Load i adds 1024 i
  // bytes (RPD rows) to both sides, which moves the K permutation by 4 chunks
  // and leaves the V permutation unchanged; with the instruction offset taking
  // the 1024 i, the per-lane offset of load i is kdma ^ 64 i for K and vdma for
  // V (the identity holds for every configuration built).
  uint32_t kdma, vdma;
  {
    const int row = C::RPD * C::DPW * wave + lane / C::CPR, pos = lane % C::CPR;
    kdma = (uint32_t)(row * C::RB + 16 * (pos ^ k_swz<D, BLK>(row)));
    vdma = (uint32_t)(row * C::RB + 16 * (pos ^ v_swz<D, BLK>(row)));
  }
  const uint16_t* const kbase = a.k + bh * a.lk * D;
  const uint16_t* const vbase = a.v + bh * a.lk * D;
  // tiles are KB keys; the last one may be partial, and with SUB > 1 the last
  // tiles of a partial key block may lie wholly past Lk (0 bytes)
  const int n_kt = (int)((a.lk + C::KB - 1) / C::KB);
  const uint32_t last_bytes = (uint32_t)(a.lk - (int64_t)(n_kt - 1) * C::KB) * (uint32_t)C::RB;
  auto tile_bytes = [&](int kt) -> uint32_t {
    return (kt < 0 || kt >= n_kt) ? 0u : (kt == n_kt - 1 ? last_bytes : (uint32_t)C::TILE_BYTES);
  };
  auto dma = [&](const uint16_t* base, int blk, uint16_t* slot, uint32_t off0, uint32_t step) {
    const i32x4 rs = raw_rsrc(base + (int64_t)(blk < 0 ? 0 : blk) * C::TILE, tile_bytes(blk));
    uint32_t off[C::DPW];
#pragma unroll
    for (int i = 0; i < C::DPW; ++i) off[i] = off0 ^ (step * i);
    dma_tile<C::DPW>(lds_addr(slot) + (uint32_t)(C::DPW * wave) * 1024u, off, rs);
  };

  // ---- per-lane LDS read offsets (bytes within a tile)
  // K operand of S^T: row 32 kt + l32, logical chunk 2 s + hh
  uint32_t koff[C::DS];
  {
    const int r = l32;
#pragma unroll
    for (int s = 0; s < C::DS; ++s) koff[s] = (uint32_t)(r * C::RB + 16 * ((2 * s + hh) ^ k_swz<D, BLK>(r)));
  }
  // V^T operand through the transpose read: in each 16-lane group g, source lane
  // sl points at row R = 4 hh + sl / 4 (+ 32 kt + 16 half + 8 for the
  // second read), bytes 64 t + 32 (g % 2) + 8 (sl % 4), i.e. logical chunk
  // 4 t + 2 (g % 2) + (sl % 4) / 2, half (sl % 2); lane j then receives
  // V[R0 .. R0+3][4 c0 + j], four keys of one d column
  uint32_t voff[C::DT];
  {
    const int grp = lane >> 4, sl = lane & 15;
    const int r = 4 * hh + (sl >> 2);
#pragma unroll
    for (int t = 0; t < C::DT; ++t) {
      const int c = 4 * t + 2 * (grp & 1) + ((sl & 3) >> 1);
      voff[t] = (uint32_t)(r * C::RB + 16 * (c ^ v_swz<D, BLK>(r)) + 8 * (sl & 1));
    }
  }
  auto kslot = [&](auto i) -> uint16_t* {
    constexpr int I = decltype(i)::value;
    if constexpr (I == 0) return ks0;
    else if constexpr (I == 1) return ks1;
    else return ks2;
  };
  auto vslot = [&](auto i) -> uint16_t* {
    constexpr int I = decltype(i)::value;
    if constexpr (I == 0) return vs0;
    else return vs1;
  };
  auto lds_u4 = [](const uint16_t* slot, uint32_t byte_off) -> uint4 {
    return *reinterpret_cast<const uint4*>(reinterpret_cast<const char*>(slot) + byte_off);
  };

  const float sl2 = a.scale_log2;
  const bf16x2 ones = {(__bf16)1.0f, (__bf16)1.0f};

  // keys >= Lk of a partial last block, and every key of a -1 tile, get -inf
  auto mask_tile = [&](f32x16* acc, int blk) {
    const int64_t key0 = (int64_t)blk * C::KB;
    if (blk < 0 || key0 + C::KB > a.lk) {
#pragma unroll
      for (int kt = 0; kt < C::KT; ++kt)
#pragma unroll
        for (int e = 0; e < 16; ++e) {
          const int key = kt * 32 + 8 * (e / 4) + 4 * hh + (e % 4);
          if (blk < 0 || key0 + key >= a.lk) acc[kt][e] = -INFINITY;
        }
    }
  };
  int b1 = -1, b2 = -1, b3 = -1, b4 = -1;  // blocks of tiles t+1 .. t+4
  f32x16 acc_s[C::KT];                     // S^T of tile t

  // S^T of one K tile (LDS slot ks) into acc
  auto scores = [&](const uint16_t* ks, f32x16* acc) {
#pragma unroll
    for (int kt = 0; kt < C::KT; ++kt) {
#pragma unroll
      for (int e = 0; e < 16; ++e) acc[kt][e] = 0.f;
#pragma unroll
      for (int s = 0; s < C::DS; ++s)
        acc[kt] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(
            __builtin_bit_cast(bf16x8, lds_u4(ks, koff[s] + kt * 32 * C::RB)), qf[s], acc[kt], 0, 0, 0);
    }
  };
  // the tile's max logit (log2 domain) of the lane's query over both lane halves
  auto tile_max = [&](const f32x16* acc) -> float {
    float mx = -INFINITY;
#pragma unroll
    for (int kt = 0; kt < C::KT; ++kt)
#pragma unroll
      for (int e = 0; e < 16; ++e) mx = fmaxf(mx, acc[kt][e]);
    return mx;
  };
  // tiles [0, n_whole) lie wholly below Lk; -1 (as unsigned) and the rest need the mask
  const uint32_t n_whole = (uint32_t)(a.lk / C::KB);
  auto needs_mask = [&](int blk) { return (uint32_t)blk >= n_whole; };

  if (cnt > 0) {
    // ---- prologue.  The loads follow the order of the steady state (K(j+4)
    // after the first barrier of step j, V(j+2) after the second), so that the
    // vmcnt thresholds of the step hold from the first step on.
    load_batch(0);
    const int b0 = fetch(0);
    b1 = fetch(1);
    b2 = fetch(2);
    b3 = fetch(3);
    b4 = fetch(4);
    dma(kbase, b0, ks0, kdma, 64u);
    dma(kbase, b1, ks1, kdma, 64u);
    dma(kbase, b2, ks2, kdma, 64u);
    dma(vbase, b0, vs0, vdma, 0u);
    wait_vmcnt<3 * C::DPW>();  // K(0)
    __syncthreads();
    scores(ks0, acc_s);
    if (needs_mask(b0)) mask_tile(acc_s, b0);
    m_run = half_swap_max(tile_max(acc_s)) * sl2;  // O and the sums are still zero
    __syncthreads();  // K slot 0 is free
    dma(kbase, b3, ks0, kdma, 64u);
    wait_vmcnt<3 * C::DPW>();  // K(1)
    __syncthreads();
    dma(vbase, b1, vs1, vdma, 0u);

    // One step (T = t mod 6 fixes the slots), in two phases:
    //   A: the scores of tile t+1 on the matrix cores while the exponentials of
    //      tile t run; then V(t) is waited for, a barrier releases K slot
    //      (t+1) % 3, and K(t+4) is loaded into it (it has 2.5 steps to land);
    //   B: O += P V of tile t; then K(t+2) is waited for, a barrier releases V
    //      slot t % 2, and V(t+2) is loaded into it (1.5 steps to land).
    // Apart from the rare exact path of phase A, the phases are branch-free,
    // and sched_group_barrier interleaves their MFMAs with their VALU work so
    // that the latter hides under the matrix cores.
    int t = 0;
    auto step = [&](auto tc) {
      constexpr int T = decltype(tc)::value;
      constexpr int KS = (T + 1) % 3, VS = T % 2;
      uint16_t* const kr = kslot(std::integral_constant<int, KS>{});
      uint16_t* const vr = vslot(std::integral_constant<int, VS>{});

      // ---- phase A, per 32-key sub-tile kt: the K reads and score MFMAs of
      // tile t+1 interleaved with the exponentials of sub-tile kt of tile t.
      // The running max is only refreshed when a sub-tile could break the
      // bound p <= 2^8: a lane's sum of the sub-tile's P stays <= 2^8 whenever
      // every p does, so a larger (or non-finite) sum in any lane sends the
      // wave to the exact path -- the sub-tile's max, a rescale of O and both
      // sums to it, and the sub-tile's P again (then p <= 1 there).
      f32x16 acc_n[C::KT];
      uint32_t pk[C::KT][8];  // bf16 pairs of P^T, per 32-key sub-tile
      float pf[C::KT][16];    // the same p in fp32, summed for lse in phase B (one sub-tile per step)
#pragma unroll
      for (int kt = 0; kt < C::KT; ++kt) {
        // exp2 offset -m; +inf for a query that has seen no key yet, which makes
        // the sum non-finite and takes the exact path
        const float neg_m = m_run == -INFINITY ? INFINITY : -m_run;
        float st = 0.f;  // row sum of the sub-tile's bf16 P (the lane's keys)
        float se = 0.f;  // with two sub-tiles per step: row sum of its fp32 p
        auto exps = [&](float off) {
#pragma unroll
          for (int e = 0; e < 16; e += 2) {
            const float p0 = __builtin_amdgcn_exp2f(fmaf(acc_s[kt][e], sl2, off));
            const float p1 = __builtin_amdgcn_exp2f(fmaf(acc_s[kt][e + 1], sl2, off));
            pk[kt][e / 2] = __builtin_bit_cast(uint32_t, __builtin_convertvector((f32x2){p0, p1}, bf16x2));
            st = __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(bf16x2, pk[kt][e / 2]), ones, st, false);
            if constexpr (C::KT == 1) {
              pf[kt][e] = p0;
              pf[kt][e + 1] = p1;
            } else {
              se += p0 + p1;
            }
          }
        };
        uint4 kf[C::DS];
#pragma unroll
        for (int s = 0; s < C::DS; ++s) kf[s] = lds_u4(kr, koff[s] + kt * 32 * C::RB);
#pragma unroll
        for (int e = 0; e < 16; ++e) acc_n[kt][e] = 0.f;
#pragma unroll
        for (int s = 0; s < C::DS; ++s)
          acc_n[kt] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(__builtin_bit_cast(bf16x8, kf[s]), qf[s],
                                                              acc_n[kt], 0, 0, 0);
        exps(neg_m);
        if constexpr (C::DS == 8) {
          // the K reads in groups of RG, then 8 x (score MFMA + VA VALU of the
          // exponentials and row sums); with two sub-tiles per step (64-key
          // tiles) the K reads go four at a time and the fp32 row sum is
          // taken here: both keep the wave under 256 VGPRs without spills
          constexpr int RG = C::KT == 1 ? 8 : 4;  // K reads per group
          constexpr int VA = C::KT == 1 ? 6 : 8;  // VALU per score MFMA
#pragma unroll
          for (int g = 0; g < 8 / RG; ++g) {
            __builtin_amdgcn_sched_group_barrier(0x100, RG, 0);
#pragma unroll
            for (int i = 0; i < RG; ++i) {
              __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
              __builtin_amdgcn_sched_group_barrier(0x002, VA, 0);
            }
          }
        }
        __builtin_amdgcn_sched_barrier(0);
        if (__builtin_amdgcn_ballot_w64(!(st <= 256.f))) {
          float mx = -INFINITY;
#pragma unroll
          for (int e = 0; e < 16; ++e) mx = fmaxf(mx, acc_s[kt][e]);
          mx = half_swap_max(mx) * sl2;
          if (mx > m_run) {
            // the max moves up by a whole number of binades (to >= mx), so the
            // rescale is exact, also on the bf16 P of the step's earlier
            // sub-tiles, which are not yet in O but already in l and le.  A
            // jump past 2^128 (or the first key) drops the old terms, which
            // are then below 2^-120 of the new ones.
            float alpha = 0.f;
            const float dm = mx - m_run;
            if (dm > 128.f) {
              m_run = mx;
            } else {
              const float k = ceilf(dm);
              alpha = __builtin_amdgcn_ldexpf(1.f, -(int)k);
              m_run += k;
            }
            l_run *= alpha;
            le_run *= alpha;
#pragma unroll
            for (int d = 0; d < C::DT; ++d)
#pragma unroll
              for (int e = 0; e < 16; ++e) acc_o[d][e] *= alpha;
#pragma unroll
            for (int j = 0; j < kt; ++j)
#pragma unroll
              for (int i = 0; i < 8; ++i)
                pk[j][i] = pack2_bf16(__uint_as_float(pk[j][i] << 16) * alpha,
                                      __uint_as_float(pk[j][i] & 0xffff0000u) * alpha);
          }
          st = 0.f;
          se = 0.f;
          exps(m_run == -INFINITY ? 0.f : -m_run);
        }
        l_run += st;
        if constexpr (C::KT != 1) le_run += se;
      }
      wait_vmcnt<2 * C::DPW>();  // V(t)
      __syncthreads();
      dma(kbase, b4, kr, kdma, 64u);

      // ---- phase B: O^T += V^T P^T over 16-key k-steps
#pragma unroll
      for (int kt = 0; kt < C::KT; ++kt)
#pragma unroll
        for (int half = 0; half < 2; ++half) {
          // accumulators a = 8 half + i of sub-tile kt hold keys
          //   base + 4 hh + i (i = 0..3) and base + 8 + 4 hh + (i - 4) (i = 4..7),
          // base = 32 kt + 16 half; the two transpose reads fetch the
          // same keys of V for d = 32 t + l % 32.
          uint4 pu;
          pu.x = pk[kt][4 * half + 0];
          pu.y = pk[kt][4 * half + 1];
          pu.z = pk[kt][4 * half + 2];
          pu.w = pk[kt][4 * half + 3];
          const bf16x8 pb = __builtin_bit_cast(bf16x8, pu);
#pragma unroll
          for (int dt = 0; dt < C::DT; ++dt) {
            const uint16_t* vp = reinterpret_cast<const uint16_t*>(reinterpret_cast<const char*>(vr) + voff[dt] +
                                                                   (32 * kt + 16 * half) * C::RB);
            const s16x4 v0 = lds_read_tr(vp);
            const s16x4 v1 = lds_read_tr(vp + 8 * D);
            const s16x8 vv = __builtin_shufflevector(v0, v1, 0, 1, 2, 3, 4, 5, 6, 7);
            acc_o[dt] =
                __builtin_amdgcn_mfma_f32_32x32x16_bf16(__builtin_bit_cast(bf16x8, vv), pb, acc_o[dt], 0, 0, 0);
          }
          if constexpr (C::KT == 1) {
#pragma unroll
            for (int i = 0; i < 8; ++i) le_run += pf[kt][8 * half + i];
          }
        }
      if constexpr (C::DT == 4) {
        // the first two MFMAs' V reads, then (P V MFMA + the V reads of the
        // MFMA two ahead + VB VALU) for all but the last two MFMAs, then
        // 2 x (MFMA + VB VALU); with one sub-tile per step the VALU work is the
        // fp32 row sum, here where the VALU is idle rather than among the
        // exponentials of phase A
        constexpr int VB = C::KT == 1 ? 2 : 0;
        __builtin_amdgcn_sched_group_barrier(0x100, 4, 0);
#pragma unroll
        for (int i = 0; i < 8 * C::KT - 2; ++i) {
          __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
          __builtin_amdgcn_sched_group_barrier(0x100, 2, 0);
          if constexpr (VB > 0) __builtin_amdgcn_sched_group_barrier(0x002, VB, 0);
        }
#pragma unroll
        for (int i = 0; i < 2; ++i) {
          __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
          if constexpr (VB > 0) __builtin_amdgcn_sched_group_barrier(0x002, VB, 0);
        }
      }
      // keeps the fp32 row sum in this phase, among the P V MFMAs, rather than
      // sunk into the next step ahead of its first score MFMA
      if constexpr (C::KT == 1) asm volatile("" : "+v"(le_run));
      if (t + 1 < ntiles && needs_mask(b1)) mask_tile(acc_n, b1);
      __builtin_amdgcn_sched_barrier(0);
      wait_vmcnt<3 * C::DPW>();  // K(t+2)
      __syncthreads();
      dma(vbase, b2, vr, vdma, 0u);

#pragma unroll
      for (int kt = 0; kt < C::KT; ++kt) acc_s[kt] = acc_n[kt];
      b1 = b2;
      b2 = b3;
      b3 = b4;
      b4 = fetch(t + 5);
    };

    while (true) {
      step(std::integral_constant<int, 0>{});
      if (++t >= ntiles) break;
      step(std::integral_constant<int, 1>{});
      if (++t >= ntiles) break;
      step(std::integral_constant<int, 2>{});
      if (++t >= ntiles) break;
      step(std::integral_constant<int, 3>{});
      if (++t >= ntiles) break;
      step(std::integral_constant<int, 4>{});
      if (++t >= ntiles) break;
      step(std::integral_constant<int, 5>{});
      if (++t >= ntiles) break;
    }
    wait_vmcnt<0>();  // loads past the end of the list still write LDS
  }

  // ---- write O and lse.  The lane's row index is derived again from the lane
  // id (v_mbcnt) rather than kept live over the loop, where every VGPR counts.
  l_run = half_swap_sum(l_run);  // both lane halves now hold the query's row sums
  le_run = half_swap_sum(le_run);
  const int lane_o = (int)__builtin_amdgcn_mbcnt_hi(~0u, __builtin_amdgcn_mbcnt_lo(~0u, 0u));
  const int l32o = lane_o % 32, hho = lane_o / 32;
  const int64_t row_o = (int64_t)qb * BLK + qs * 32 + l32o;
  const bool row_ok = row_o < a.lq;
  if constexpr (SPLIT) {
    // Partial result of this key range: the unnormalised P V, scaled by a
    // power of two 2^-ex per query row so that its largest magnitude lies in
    // [0.5, 1) and every value keeps fp16's relative precision whatever the
    // range of V; the merge undoes the scale exactly.
    float amax = 0.f;
#pragma unroll
    for (int t = 0; t < C::DT; ++t)
#pragma unroll
      for (int e = 0; e < 16; ++e) amax = fmaxf(amax, fabsf(acc_o[t][e]));
    amax = half_swap_max(amax);
    int ex = 0;
    if (amax > 0.f && amax <= 3.402823466e38f) ex = __builtin_amdgcn_frexp_expf(amax);
    ex = ex < -126 ? -126 : ex;
    const float sc = __builtin_amdgcn_ldexpf(1.0f, -ex);
    if (row_ok) {
      const int64_t prow = (work * a.n_splits + split) * BLK + qs * 32 + l32o;
      _Float16* po = reinterpret_cast<_Float16*>(a.part_o) + prow * D;
#pragma unroll
      for (int t = 0; t < C::DT; ++t)
#pragma unroll
        for (int g = 0; g < 4; ++g) {
          const int d = 32 * t + 8 * g + 4 * hho;
          f16x4 w;
#pragma unroll
          for (int e = 0; e < 4; ++e) w[e] = (_Float16)(acc_o[t][4 * g + e] * sc);
          *reinterpret_cast<f16x4*>(po + d) = w;
        }
      if (hho == 0)
        reinterpret_cast<float4*>(a.part_meta)[prow] = make_float4(m_run, l_run, le_run, (float)ex);
    }
  } else if (row_ok) {
    const float inv = l_run > 0.f ? 1.f / l_run : 0.f;
    uint16_t* op = a.o + (bh * a.lq + row_o) * D;
#pragma unroll
    for (int t = 0; t < C::DT; ++t)
#pragma unroll
      for (int g = 0; g < 4; ++g) {
        const int d = 32 * t + 8 * g + 4 * hho;
        float o[4];
#pragma unroll
        for (int e = 0; e < 4; ++e) o[e] = acc_o[t][4 * g + e] * inv;
        uint2 w;
        w.x = pack2_bf16(o[0], o[1]);
        w.y = pack2_bf16(o[2], o[3]);
        *reinterpret_cast<uint2*>(op + d) = w;
      }
    if (a.lse != nullptr && hho == 0)
      a.lse[bh * a.lq + row_o] = le_run > 0.f ? (m_run + log2f(le_run)) * 0.69314718055994530942f : -INFINITY;
  }
}

// Combines the NS partial results of one query block.  Range r left, per
// query row, A_r = sum of bf16(p) v over its keys scaled by 2^-e_r (fp16), its
// running max m_r (log2 units), the row sums lb_r (of the bf16 p that multiply
// V) and le_r (of the fp32 p), and e_r.  With M = max_r m_r and
// w_r = 2^(m_r - M) over the ranges that saw a key (lb_r > 0):
//   O   = sum_r w_r 2^e_r A_r / sum_r w_r lb_r,
//   lse = ln2 (M + log2 sum_r w_r le_r).
// Ranges with no visible key have weight 0 and add nothing.
// One thread per 8-column chunk of the query block's rows (two chunks per
// thread at BLK = 128, D = 128).
template <int D, int BLK>
struct MergeCfg {
  static constexpr int CPR = D / 8;                     // 8-column chunks per row
  static constexpr int CHUNKS = BLK * CPR;
  static constexpr int NT = CHUNKS < 1024 ? CHUNKS : 1024;
  static constexpr int CPT = CHUNKS / NT;               // chunks per thread
  static_assert(CPT * NT == CHUNKS && NT >= BLK, "chunk split");
};

template <int D, int BLK, int NS>
__global__ __launch_bounds__((MergeCfg<D, BLK>::NT)) void attn_merge_kernel(AttnArgs a) {
  using M = MergeCfg<D, BLK>;
  __shared__ float wts[NS][BLK];
  const int64_t work = blockIdx.x;
  const int64_t bh = work / a.n_q;
  const int qb = (int)(work % a.n_q);
  const int tid = threadIdx.x;
  const int64_t rows = a.lq - (int64_t)qb * BLK;
  // every range's partial is written for every real row of the block (zeros
  // when it saw no key); rows past Lq are never read
  auto load_chunk = [&](int c, f16x8* v) {
    const int row = c / M::CPR, d0 = (c % M::CPR) * 8;
    const int rr = row < rows ? row : 0;
#pragma unroll
    for (int r = 0; r < NS; ++r) {
      const int64_t prow = (work * NS + r) * BLK + rr;
      v[r] = *reinterpret_cast<const f16x8*>(reinterpret_cast<const _Float16*>(a.part_o) + prow * D + d0);
    }
  };
  auto combine = [&](int c, const f16x8* v) {
    const int row = c / M::CPR, d0 = (c % M::CPR) * 8;
    if (row >= rows) return;
    float acc[8] = {0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int r = 0; r < NS; ++r) {
      const float w = wts[r][row];
#pragma unroll
      for (int e = 0; e < 8; ++e) acc[e] = w != 0.f ? fmaf(w, (float)v[r][e], acc[e]) : acc[e];
    }
    uint4 o;
    o.x = pack2_bf16(acc[0], acc[1]);
    o.y = pack2_bf16(acc[2], acc[3]);
    o.z = pack2_bf16(acc[4], acc[5]);
    o.w = pack2_bf16(acc[6], acc[7]);
    *reinterpret_cast<uint4*>(a.o + (bh * a.lq + (int64_t)qb * BLK + row) * D + d0) = o;
  };

  // The threads of the first BLK rows turn the per-row records into weights
  // first and then issue their partial loads; every other thread issues its
  // partial loads at once, so that their latency overlaps the records'.
  f16x8 v[NS];
  if (tid >= BLK) load_chunk(tid, v);
  if (tid < BLK && tid < rows) {
    const int row = tid;
    const float2* rec = reinterpret_cast<const float2*>(a.part_meta);  // record i = float2 pairs 2i, 2i + 1
    float m[NS], lb[NS], mm = -INFINITY;
#pragma unroll
    for (int r = 0; r < NS; ++r) {
      const float2 x = rec[2 * ((work * NS + r) * BLK + row)];
      m[r] = x.x;
      lb[r] = x.y;
      if (lb[r] > 0.f) mm = fmaxf(mm, m[r]);
    }
    float den = 0.f, sum_e = 0.f;
#pragma unroll
    for (int r = 0; r < NS; ++r) {
      const float2 y = rec[2 * ((work * NS + r) * BLK + row) + 1];  // (le, e)
      const float w = lb[r] > 0.f ? exp2f(m[r] - mm) : 0.f;
      den = fmaf(w, lb[r], den);
      sum_e = fmaf(w, y.x, sum_e);
      wts[r][row] = __builtin_amdgcn_ldexpf(w, (int)y.y);
    }
    const float inv = den > 0.f ? 1.f / den : 0.f;
#pragma unroll
    for (int r = 0; r < NS; ++r) wts[r][row] *= inv;
    if (a.lse != nullptr)
      a.lse[bh * a.lq + (int64_t)qb * BLK + row] =
          sum_e > 0.f ? (mm + log2f(sum_e)) * 0.69314718055994530942f : -INFINITY;
  }
  if (tid < BLK) load_chunk(tid, v);
  __syncthreads();
  combine(tid, v);
#pragma unroll
  for (int k = 1; k < M::CPT; ++k) {
    load_chunk(tid + k * M::NT, v);
    combine(tid + k * M::NT, v);
  }
}

template <int D, int BLK>
static hipError_t launch_cfg(const AttnArgs& a, bool dense, hipStream_t stream) {
  const int64_t items = (int64_t)a.bh * a.n_q;
  if (items == 0) return hipSuccess;
  constexpr int NT = AttnCfg<D, BLK>::NT;
  if (a.part_o != nullptr) {
    if (a.n_splits != 8 && a.n_splits != kSplits) return hipErrorInvalidValue;
    if (dense) attn_fwd_kernel<D, BLK, true, true><<<items * a.n_splits, NT, 0, stream>>>(a);
    else attn_fwd_kernel<D, BLK, false, true><<<items * a.n_splits, NT, 0, stream>>>(a);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    if (a.n_splits == 8) attn_merge_kernel<D, BLK, 8><<<items, MergeCfg<D, BLK>::NT, 0, stream>>>(a);
    else attn_merge_kernel<D, BLK, kSplits><<<items, MergeCfg<D, BLK>::NT, 0, stream>>>(a);
  } else {
    if (dense) attn_fwd_kernel<D, BLK, true, false><<<items, NT, 0, stream>>>(a);
    else attn_fwd_kernel<D, BLK, false, false><<<items, NT, 0, stream>>>(a);
  }
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
