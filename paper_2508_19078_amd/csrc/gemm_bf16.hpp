// bf16 grouped-GEMM core for gfx950: 8-wave blocks with a three-stage
// direct-to-LDS pipeline.
//
// A block of 512 threads (8 waves, two per SIMD) computes an RA x RB output
// tile, RA, RB in {128, 256}, of C = sum_k A(r, k) B(n, k); each wave owns a
// 64 x 64 sub-tile as 2 x 2 v_mfma_f32_32x32x16_bf16 tiles (the bf16 shape that
// reaches the chip's MFMA peak), operands swapped so that a lane holds groups of
// four consecutive output columns.
//
// * Tiles go straight from global memory to LDS (global_load_lds_dwordx4: each
//   lane moves 16 bytes to LDS base + 16 * lane), three 64-deep K slabs in the
//   ring: two are in flight while the third is multiplied.  Per-lane addresses
//   are resolved once per tile; a slab only adds a uniform stride.
// * K-contiguous tiles are stored [row][64 k] (128-byte rows) with the 16-byte
//   chunk index XOR-swizzled by (row >> 1) & 7: the fragment reads of 16
//   consecutive rows hit 16 distinct 4-bank groups.
// * MN-contiguous tiles (weights in the NN products, both operands of the
//   weight-gradient products) are stored k-major, [64 k][R rows], with the chunk
//   index XOR-swizzled by (k & 3) << 2, and read with ds_read_b64_tr_b16, which
//   hands each lane four k-consecutive elements of one row; two such reads form
//   a fragment, so nothing is transposed on the way in.
// * An operand may interleave two matrices in 32-row blocks (gate and up
//   weights; the two dSwiGLU gradients), so that the pairs the epilogue needs sit
//   in one lane.
// * Rows past the operand's extent read a clamped (valid) address and only feed
//   outputs that are never stored; k past K is zeroed in the A fragments of the
//   last slab, so the clamped B data meets zeros.
#pragma once

#include "gemm.hpp"

namespace fm {

constexpr int B16_BK = 64;                      // k per slab
constexpr int B16_NS = 3;                       // LDS stages
constexpr int B16_THREADS = 512;                // 8 waves

#define FM_LDS __attribute__((address_space(3)))
typedef short i16x4_t __attribute__((ext_vector_type(4)));
typedef float f32x16_t __attribute__((ext_vector_type(16)));

// s_waitcnt with only vmcnt limited (expcnt / lgkmcnt left at their maxima).
template <int N> __device__ __forceinline__ void wait_vmcnt() {
  static_assert(N >= 0 && N < 64, "vmcnt range");
  __builtin_amdgcn_s_waitcnt((N & 15) | ((N >> 4) << 14) | (7 << 4) | (15 << 8));
}

// Workgroup barrier without the memory fences of __syncthreads: the fences
// would wait for every outstanding load, including the slabs still in flight.
// LDS reads of the previous slab have completed (their MFMAs consumed them) and
// this slab's DMA completion is waited for explicitly before the barrier.
__device__ __forceinline__ void barrier_lds() { asm volatile("s_barrier" ::: "memory"); }

__device__ __forceinline__ void dma16(const void* g, FM_LDS void* l) {
  __builtin_amdgcn_global_load_lds((const FM_GLOBAL void*)g, l, 16, 0, 0);
}

// Wave index as a uniform (scalar) value.
__device__ __forceinline__ int wave_id() { return __builtin_amdgcn_readfirstlane(threadIdx.x >> 6); }

__device__ __forceinline__ int swz_kc(int row) { return (row >> 1) & 7; }
// A transposed read of one 16-lane group touches 4 k-rows and 2 adjacent
// chunks; the two groups served together (rows +16) touch the next 2 chunks.
// Moving k & 3 into bits 2-3 of the chunk position spreads the 4 x 4 chunk
// reads of the pair over 16 positions (all 64 banks).
__device__ __forceinline__ int swz_mn(int k) { return (k & 3) << 2; }

// One operand of the bf16 core: logical [R rows][K].  Element (r, k) lives at
// p[r * ld + k] (K-contiguous) or p[k * ld + r] (MN-contiguous), relative to
// the tile origin.  With p2 set, the logical rows alternate in blocks of 32
// between p (even blocks) and p2 (odd blocks): logical row r is physical row
// 32 (r / 64) + r % 32 of matrix (r / 32) % 2.  rows = physical rows valid from
// the origin (per matrix).
struct B16Src {
  const bf16* p;
  const bf16* p2;
  int ld;
  int rows;
  int K;
};

__device__ __forceinline__ const bf16* b16_row(const B16Src& s, int r, int& pr) {
  if (s.p2) {
    pr = 32 * (r >> 6) + (r & 31);
    return (r >> 5) & 1 ? s.p2 : s.p;
  }
  pr = r;
  return s.p;
}

// Direct-to-LDS loading of one R-row operand: the tile is R/8 blocks of 1 KB,
// NI = R/64 of them per wave and slab.
template <bool KC, int R> struct B16Dma {
  static constexpr int NI = R / 64;
  const char* ptr[NI];
  size_t step;

  __device__ __forceinline__ void init(const B16Src& s) {
    const int lane = lane_id(), wave = wave_id();
#pragma unroll
    for (int u = 0; u < NI; ++u) {
      const int ins = wave * NI + u;
      if (KC) {
        const int r = ins * 8 + (lane >> 3);            // 8 rows of 128 bytes
        const int c = (lane & 7) ^ swz_kc(r);           // chunk this lane fetches
        int pr;
        const bf16* base = b16_row(s, r, pr);
        ptr[u] = (const char*)(base + (size_t)min(pr, s.rows - 1) * s.ld + 8 * c);
      } else {
        constexpr int CPR = R / 8;                       // 16-byte chunks per k-row
        const int kr = ins * (64 / CPR) + lane / CPR;
        const int c = (lane % CPR) ^ swz_mn(kr);
        int pr;
        const bf16* base = b16_row(s, 8 * c, pr);
        ptr[u] = (const char*)(base + (size_t)kr * s.ld + min(pr, s.rows - 8));
      }
    }
    step = KC ? (size_t)B16_BK * 2 : (size_t)B16_BK * s.ld * 2;
  }

  __device__ __forceinline__ void issue_full(int slab, FM_LDS char* tile) const {
    const int wave = wave_id();
    const size_t adv = step * (size_t)slab;
#pragma unroll
    for (int u = 0; u < NI; ++u) dma16(ptr[u] + adv, tile + (wave * NI + u) * 1024);
  }

  __device__ __forceinline__ void issue_tail(const B16Src& s, int k0, FM_LDS char* tile) const {
    const int lane = lane_id(), wave = wave_id();
#pragma unroll
    for (int u = 0; u < NI; ++u) {
      const int ins = wave * NI + u;
      if (KC) {
        const int r = ins * 8 + (lane >> 3);
        const int c = (lane & 7) ^ swz_kc(r);
        int pr;
        const bf16* base = b16_row(s, r, pr);
        dma16(base + (size_t)min(pr, s.rows - 1) * s.ld + min(k0 + 8 * c, s.K - 8), tile + ins * 1024);
      } else {
        constexpr int CPR = R / 8;
        const int kr = ins * (64 / CPR) + lane / CPR;
        const int c = (lane % CPR) ^ swz_mn(kr);
        int pr;
        const bf16* base = b16_row(s, 8 * c, pr);
        dma16(base + (size_t)min(k0 + kr, s.K - 1) * s.ld + min(pr, s.rows - 8), tile + ins * 1024);
      }
    }
  }
};

// MFMA fragments of a wave's 64 rows (two 32-row blocks) of an R-row tile: a
// fragment is 32 rows x 16 k, 8 k per lane: lane l holds row r0 + l % 32 and
// k 16 ks + 8 (l / 32) + 0..7 of the slab.  Offsets are per lane, computed once.
template <bool KC, int R> struct B16Frag {
  uint32_t off[2][KC ? 4 : 1];   // [i][ks] for K-contiguous, [i] for MN-contiguous

  __device__ __forceinline__ void init(int w) {
    const int lane = lane_id();
#pragma unroll
    for (int i = 0; i < 2; ++i) {
      const int r0 = w * 64 + i * 32;
      if (KC) {
        const int r = r0 + (lane & 31);
#pragma unroll
        for (int ks = 0; ks < 4; ++ks) {
          const int c = ks * 2 + (lane >> 5);
          off[i][ks] = (uint32_t)(r * 128 + ((c ^ swz_kc(r)) << 4));
        }
      } else {
        // ds_read_b64_tr_b16: in each 16-lane group, output lane i element j
        // comes from the address of lane 4j + i/4, offset i % 4.  Group g covers
        // rows r0 + 16 (g & 1) + [0, 16) and k 8 (g >> 1) + [0, 8) of the k-step;
        // lane L of the group points at (k = kbase + L/4, row = rbase + 4 (L % 4)).
        // The swizzle depends only on k & 3, which the k-step (16 ks) and the
        // half (4 h) leave unchanged: those enter as constant offsets.
        const int g = lane >> 4, L = lane & 15;
        const int n = r0 + 16 * (g & 1) + 4 * (L & 3);
        const int k = 8 * (g >> 1) + (L >> 2);
        off[i][0] = (uint32_t)(k * (R * 2) + (((n >> 3) ^ swz_mn(k)) << 4) + ((n >> 2) & 1) * 8);
      }
    }
  }

  __device__ __forceinline__ bf16x8_t read(const FM_LDS char* tile, int i, int ks) const {
    if (KC) {
      return __builtin_bit_cast(bf16x8_t, *(const FM_LDS u32x4_t*)(tile + off[i][ks]));
    } else {
      const FM_LDS char* p = tile + off[i][0] + ks * 16 * (R * 2);
      const i16x4_t v0 = __builtin_amdgcn_ds_read_tr16_b64_v4i16((FM_LDS i16x4_t*)p);
      const i16x4_t v1 = __builtin_amdgcn_ds_read_tr16_b64_v4i16((FM_LDS i16x4_t*)(p + 4 * (R * 2)));
      const u32x2_t w0 = __builtin_bit_cast(u32x2_t, v0), w1 = __builtin_bit_cast(u32x2_t, v1);
      return __builtin_bit_cast(bf16x8_t, u32x4_t{w0[0], w0[1], w1[0], w1[1]});
    }
  }
};

// Zeroes the k >= K elements of an A fragment (k-step ks of the slab at k0).
__device__ __forceinline__ bf16x8_t b16_mask_k(bf16x8_t f, int k0, int ks, int K) {
  const int kf = k0 + ks * 16 + 8 * (lane_id() >> 5);
  if (kf + 8 <= K) return f;
  u32x4_t w = __builtin_bit_cast(u32x4_t, f);
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const uint32_t lo = (kf + 2 * i < K) ? 0x0000FFFFu : 0u;
    const uint32_t hi = (kf + 2 * i + 1 < K) ? 0xFFFF0000u : 0u;
    w[i] &= (lo | hi);
  }
  return __builtin_bit_cast(bf16x8_t, w);
}

// Accumulator of a wave's 64 x 64 sub-tile: 2 x 2 MFMA tiles of 32 x 32.
// Register r of tile (i, j) holds sub-tile row i*32 + lane % 32 and column
// j*32 + 8 (r / 4) + 4 (lane / 32) + r % 4.
struct B16Acc {
  f32x16_t v[2][2];
  __device__ __forceinline__ void zero() {
#pragma unroll
    for (int i = 0; i < 2; ++i)
#pragma unroll
      for (int j = 0; j < 2; ++j)
#pragma unroll
        for (int r = 0; r < 16; ++r) v[i][j][r] = 0.f;
  }
  // quad g = (i, j, q): i = g >> 3, j = (g >> 2) & 1, register group q = g & 3
  __device__ __forceinline__ f32x4_t quad(int g) const {
    const f32x16_t& t = v[g >> 3][(g >> 2) & 1];
    const int q = g & 3;
    return f32x4_t{t[4 * q], t[4 * q + 1], t[4 * q + 2], t[4 * q + 3]};
  }
};

// Block-tile coordinates of quad g: the row, and the first of 4 columns.
template <int RA> __device__ __forceinline__ AccCoord b16_quad_coord(int g) {
  const int lane = lane_id(), wave = wave_id();
  const int wm = wave % (RA / 64), wn = wave / (RA / 64);
  const int i = g >> 3, j = (g >> 2) & 1, q = g & 3;
  return AccCoord{wm * 64 + i * 32 + (lane & 31), wn * 64 + j * 32 + 8 * q + 4 * (lane >> 5)};
}

template <bool AKC, bool BKC, int RA, int RB, bool TAIL>
__device__ __forceinline__ void b16_mma_slab(const FM_LDS char* buf, const B16Frag<AKC, RA>& fa_off,
                                             const B16Frag<BKC, RB>& fb_off, B16Acc& acc, int k0, int K) {
#pragma unroll
  for (int ks = 0; ks < 4; ++ks) {
    bf16x8_t fa[2], fb[2];
#pragma unroll
    for (int i = 0; i < 2; ++i) {
      fa[i] = fa_off.read(buf, i, ks);
      if (TAIL) fa[i] = b16_mask_k(fa[i], k0, ks, K);
    }
#pragma unroll
    for (int j = 0; j < 2; ++j) fb[j] = fb_off.read(buf + RA * 128, j, ks);
#pragma unroll
    for (int i = 0; i < 2; ++i)
#pragma unroll
      for (int j = 0; j < 2; ++j)
        acc.v[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(fb[j], fa[i], acc.v[i][j], 0, 0, 0);
  }
}

// LDS bytes of the bf16 core for an RA x RB tile.
template <int RA, int RB> struct B16Lds {
  static constexpr int value = B16_NS * (RA + RB) * 128;
};

// k loop over [0, K), accumulating into acc.  Ends with a barrier so the LDS
// can be reused by a following call.
template <bool AKC, bool BKC, int RA, int RB>
__device__ __forceinline__ void b16_gemm(const B16Src& A, const B16Src& B, int K, FM_LDS char* lds,
                                         B16Acc& acc) {
  static_assert((RA / 64) * (RB / 64) == 8, "8 waves of 64 x 64");
  constexpr int STAGE = (RA + RB) * 128;
  constexpr int PER_STAGE = RA / 64 + RB / 64;   // DMA instructions per wave and stage
  const int nk = (K + B16_BK - 1) / B16_BK;
  if (nk <= 0) return;
  const int nfull = K / B16_BK;                  // slabs with no k past K
  const int wave = wave_id();
  B16Frag<AKC, RA> fa;
  B16Frag<BKC, RB> fb;
  fa.init(wave % (RA / 64));
  fb.init(wave / (RA / 64));
  B16Dma<AKC, RA> da;
  B16Dma<BKC, RB> db;
  da.init(A);
  db.init(B);
  auto issue = [&](int s) {
    FM_LDS char* buf = lds + (s % B16_NS) * STAGE;
    if (s < nfull) {
      da.issue_full(s, buf);
      db.issue_full(s, buf + RA * 128);
    } else {
      da.issue_tail(A, s * B16_BK, buf);
      db.issue_tail(B, s * B16_BK, buf + RA * 128);
    }
  };
  // Slab kt is ready once at most one later slab is still in flight; the
  // barrier also tells every wave that slab kt-1's buffer is free again.
  auto ready = [&](int kt) {
    if (kt + 1 < nk) wait_vmcnt<PER_STAGE>();
    else wait_vmcnt<0>();
    barrier_lds();
    if (kt + 2 < nk) issue(kt + 2);
  };
  issue(0);
  if (nk > 1) issue(1);
  int kt = 0;
  for (; kt < nfull; ++kt) {
    ready(kt);
    b16_mma_slab<AKC, BKC, RA, RB, false>(lds + (kt % B16_NS) * STAGE, fa, fb, acc, kt * B16_BK, K);
  }
  if (kt < nk) {   // the partial last slab
    ready(kt);
    b16_mma_slab<AKC, BKC, RA, RB, true>(lds + (kt % B16_NS) * STAGE, fa, fb, acc, kt * B16_BK, K);
  }
  barrier_lds();
}

}  // namespace fm
