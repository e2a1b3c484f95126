// bf16 main loop of the grouped-GEMM core for gfx950: a three-stage
// direct-to-LDS pipeline.
//
// Same block shape as gemm.hpp (256 threads, 2 x 2 waves of 64 x 64, 128 x 128
// output tile), with v_mfma_f32_32x32x16_bf16 (the bf16 shape that reaches the
// chip's MFMA peak; 16x16x32 issues measurably slower), operands swapped so each
// lane owns groups of four consecutive output columns, and a K slab of 64:
//
// * Global tiles go straight to LDS with global_load_lds_dwordx4 (each lane
//   moves 16 bytes to LDS base + 16 * lane), three slabs deep: two slabs are in
//   flight while the third is multiplied, with no staging registers.
// * K-contiguous tiles are stored [row][64 k] (128-byte rows) with the 16-byte
//   chunk index XOR-swizzled by (row >> 1) & 7, so the 16-byte fragment reads of
//   16 consecutive rows hit 16 distinct 4-bank groups.
// * MN-contiguous tiles (weights in the NN products, both operands of the
//   weight-gradient products) are stored k-major, [64 k][128 rows] (256-byte
//   rows), with the chunk index XOR-swizzled by (k & 3) << 2, and read with
//   ds_read_b64_tr_b16, which hands each lane four k-consecutive elements of
//   one row: two such reads form an MFMA fragment, so no transposing writes.
// * Rows and columns past the operand's extent read a clamped (valid) address
//   and only feed outputs that are never stored; k past K is zeroed in the A
//   fragments of the last slab, so the clamped B data meets zeros.
#pragma once

#include "gemm.hpp"

namespace fm {

constexpr int B16_BK = 64;                      // k per slab
constexpr int B16_NS = 3;                       // LDS stages
constexpr int B16_TILE = 128 * B16_BK * 2;      // bytes of one operand tile (16 KB)

#define FM_LDS __attribute__((address_space(3)))
typedef short i16x4_t __attribute__((ext_vector_type(4)));

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

// swizzles (16-byte chunk positions)
__device__ __forceinline__ int swz_kc(int row) { return (row >> 1) & 7; }
// MN-contiguous tiles: a transposed read of one 16-lane group touches 4 k-rows
// and 2 adjacent chunks; the two groups served together (rows +16) touch the
// next 2 chunks.  Moving k & 3 into bits 2-3 of the chunk position spreads the
// 4 x 4 chunk reads of the pair over all 16 positions (all 64 banks).
__device__ __forceinline__ int swz_mn(int k) { return (k & 3) << 2; }

// Wave index as a uniform (scalar) value.
__device__ __forceinline__ int wave_id() { return __builtin_amdgcn_readfirstlane(threadIdx.x >> 6); }

// Direct-to-LDS loading of one operand: this wave moves 4 of the tile's 16
// 1 KB blocks per slab.  init() resolves the per-lane global addresses of the
// first slab once per tile (rows past the operand clamped); a full slab then
// only adds a uniform stride.  The last, partial slab clamps k as well.
template <bool KC> struct DmaOp {
  const char* ptr[4];
  size_t step;     // bytes per slab

  __device__ __forceinline__ void init(const Opnd<bf16>& op) {
    const int lane = lane_id(), wave = wave_id();
#pragma unroll
    for (int u = 0; u < 4; ++u) {
      const int ins = wave * 4 + u;
      if (KC) {
        const int r = ins * 8 + (lane >> 3);          // 8 rows of 128 bytes
        const int c = (lane & 7) ^ swz_kc(r);         // chunk this lane fetches
        ptr[u] = (const char*)(op.p + (size_t)min(r, op.rows - 1) * op.ld + 8 * c);
      } else {
        const int kr = ins * 4 + (lane >> 4);         // 4 k-rows of 256 bytes
        const int c = (lane & 15) ^ swz_mn(kr);
        ptr[u] = (const char*)(op.p + (size_t)kr * op.ld + min(8 * c, op.rows - 8));
      }
    }
    step = KC ? (size_t)B16_BK * 2 : (size_t)B16_BK * op.ld * 2;
  }

  __device__ __forceinline__ void issue_full(int s, FM_LDS char* tile) const {
    const int wave = wave_id();
    const size_t adv = step * (size_t)s;
#pragma unroll
    for (int u = 0; u < 4; ++u) dma16(ptr[u] + adv, tile + (wave * 4 + u) * 1024);
  }

  __device__ __forceinline__ void issue_tail(const Opnd<bf16>& op, int k0, FM_LDS char* tile) const {
    const int lane = lane_id(), wave = wave_id();
#pragma unroll
    for (int u = 0; u < 4; ++u) {
      const int ins = wave * 4 + u;
      if (KC) {
        const int r = ins * 8 + (lane >> 3);
        const int c = (lane & 7) ^ swz_kc(r);
        dma16(op.p + (size_t)min(r, op.rows - 1) * op.ld + min(k0 + 8 * c, op.K - 8), tile + ins * 1024);
      } else {
        const int kr = ins * 4 + (lane >> 4);
        const int c = (lane & 15) ^ swz_mn(kr);
        dma16(op.p + (size_t)min(k0 + kr, op.K - 1) * op.ld + min(8 * c, op.rows - 8), tile + ins * 1024);
      }
    }
  }
};

typedef float f32x16_t __attribute__((ext_vector_type(16)));

// 64 x 64 wave tile as 2 x 2 MFMA tiles of 32 x 32 (16 accumulators per lane).
// Register r of tile (i, j) holds row i*32 + (lane & 31) and column
// j*32 + 8*(r/4) + 4*(lane/32) + r%4 of the wave tile.
template <int NA, int NB> struct Acc<bf16, NA, NB> {
  f32x16_t v[NA * NB][2][2];
  __device__ __forceinline__ void zero() {
#pragma unroll
    for (int x = 0; x < NA * NB; ++x)
#pragma unroll
      for (int i = 0; i < 2; ++i)
#pragma unroll
        for (int j = 0; j < 2; ++j)
#pragma unroll
          for (int r = 0; r < 16; ++r) v[x][i][j][r] = 0.f;
  }
  __device__ __forceinline__ f32x4_t quad(int x, int g) const {
    const f32x16_t& t = v[x][g >> 3][(g >> 2) & 1];
    const int q = g & 3;
    return f32x4_t{t[4 * q], t[4 * q + 1], t[4 * q + 2], t[4 * q + 3]};
  }
};
// quad g = (i, j, q): i = g >> 3, j = (g >> 2) & 1, register group q = g & 3
template <> __device__ __forceinline__ AccCoord quad_coord<bf16>(int g) {
  const int lane = lane_id(), wave = threadIdx.x >> 6;
  const int i = g >> 3, j = (g >> 2) & 1, q = g & 3;
  return AccCoord{(wave & 1) * 64 + i * 32 + (lane & 31), (wave >> 1) * 64 + j * 32 + 8 * q + 4 * (lane >> 5)};
}

// One MFMA fragment is 32 rows x 16 k, 8 k per lane: lane l holds row
// r0 + l%32 and k 16 ks + 8 (l/32) + 0..7 of the slab.  FragOff holds the
// per-lane byte offsets inside a tile for the wave's two 32-row blocks
// (r0 = 64 w + 32 i), computed once per kernel.
template <bool KC> struct FragOff {
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
        // The swizzle of k depends only on k & 3, which the k-step (16 ks) and
        // the half (4 h) leave unchanged: those enter as constant offsets.
        const int g = lane >> 4, L = lane & 15;
        const int n = r0 + 16 * (g & 1) + 4 * (L & 3);
        const int k = 8 * (g >> 1) + (L >> 2);
        off[i][0] = (uint32_t)(k * 256 + (((n >> 3) ^ swz_mn(k)) << 4) + ((n >> 2) & 1) * 8);
      }
    }
  }

  __device__ __forceinline__ bf16x8_t read(const FM_LDS char* tile, int i, int ks) const {
    if (KC) {
      return __builtin_bit_cast(bf16x8_t, *(const FM_LDS u32x4_t*)(tile + off[i][ks]));
    } else {
      const FM_LDS char* p = tile + off[i][0] + ks * 16 * 256;
      const i16x4_t v0 = __builtin_amdgcn_ds_read_tr16_b64_v4i16((FM_LDS i16x4_t*)p);
      const i16x4_t v1 = __builtin_amdgcn_ds_read_tr16_b64_v4i16((FM_LDS i16x4_t*)(p + 4 * 256));
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

template <bool AKC, bool BKC, int NA, int NB, bool TAIL>
__device__ __forceinline__ void b16_mma_slab(const FM_LDS char* buf, const FragOff<AKC>& fo_a,
                                             const FragOff<BKC>& fo_b, Acc<bf16, NA, NB>& acc, int k0,
                                             int K) {
#pragma unroll
  for (int ks = 0; ks < 4; ++ks) {
    bf16x8_t fa[NA][2], fb[NB][2];
#pragma unroll
    for (int a = 0; a < NA; ++a)
#pragma unroll
      for (int i = 0; i < 2; ++i) {
        fa[a][i] = fo_a.read(buf + a * B16_TILE, i, ks);
        if (TAIL) fa[a][i] = b16_mask_k(fa[a][i], k0, ks, K);
      }
#pragma unroll
    for (int b = 0; b < NB; ++b)
#pragma unroll
      for (int j = 0; j < 2; ++j) fb[b][j] = fo_b.read(buf + (NA + b) * B16_TILE, j, ks);
#pragma unroll
    for (int a = 0; a < NA; ++a)
#pragma unroll
      for (int b = 0; b < NB; ++b)
#pragma unroll
        for (int i = 0; i < 2; ++i)
#pragma unroll
          for (int j = 0; j < 2; ++j)
            acc.v[a * NB + b][i][j] =
                __builtin_amdgcn_mfma_f32_32x32x16_bf16(fb[b][j], fa[a][i], acc.v[a * NB + b][i][j], 0, 0, 0);
  }
}

// LDS bytes needed by the bf16 main loop for NA + NB operands.
template <int NA, int NB> struct B16Lds {
  static constexpr int bytes = B16_NS * (NA + NB) * B16_TILE;
};

// k loop over [0, K).  `lds` holds B16_NS stages of (NA + NB) tiles.  Ends with
// a barrier so the LDS can be reused.
template <bool AKC, bool BKC, int NA, int NB>
__device__ __forceinline__ void gemm_mainloop_b16(const Opnd<bf16> (&A)[NA], const Opnd<bf16> (&B)[NB],
                                                  int K, FM_LDS char* lds, Acc<bf16, NA, NB>& acc) {
  constexpr int STAGE = (NA + NB) * B16_TILE;
  constexpr int PER_STAGE = 4 * (NA + NB);      // DMA instructions per wave and stage
  const int nk = (K + B16_BK - 1) / B16_BK;
  if (nk <= 0) return;
  const int nfull = K / B16_BK;                 // slabs with no k past K
  const int wave = wave_id();
  FragOff<AKC> fo_a;
  FragOff<BKC> fo_b;
  fo_a.init(wave & 1);
  fo_b.init(wave >> 1);
  DmaOp<AKC> da[NA];
  DmaOp<BKC> db[NB];
#pragma unroll
  for (int a = 0; a < NA; ++a) da[a].init(A[a]);
#pragma unroll
  for (int b = 0; b < NB; ++b) db[b].init(B[b]);
  auto issue = [&](int s) {
    FM_LDS char* buf = lds + (s % B16_NS) * STAGE;
    if (s < nfull) {
#pragma unroll
      for (int a = 0; a < NA; ++a) da[a].issue_full(s, buf + a * B16_TILE);
#pragma unroll
      for (int b = 0; b < NB; ++b) db[b].issue_full(s, buf + (NA + b) * B16_TILE);
    } else {
#pragma unroll
      for (int a = 0; a < NA; ++a) da[a].issue_tail(A[a], s * B16_BK, buf + a * B16_TILE);
#pragma unroll
      for (int b = 0; b < NB; ++b) db[b].issue_tail(B[b], s * B16_BK, buf + (NA + b) * B16_TILE);
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
    b16_mma_slab<AKC, BKC, NA, NB, false>(lds + (kt % B16_NS) * STAGE, fo_a, fo_b, acc, kt * B16_BK, K);
  }
  if (kt < nk) {   // the partial last slab
    ready(kt);
    b16_mma_slab<AKC, BKC, NA, NB, true>(lds + (kt % B16_NS) * STAGE, fo_a, fo_b, acc, kt * B16_BK, K);
  }
  barrier_lds();
}

// Dispatch: the bf16 pipeline above, or the register-staged core of gemm.hpp.
template <typename T, int NA, int NB> struct LdsBytes {
  static constexpr int value = 2 * (NA + NB) * GemmCfg<T>::TILE * (int)sizeof(T);
};
template <int NA, int NB> struct LdsBytes<bf16, NA, NB> {
  static constexpr int value = B16_NS * (NA + NB) * B16_TILE;
};

template <typename T, bool AKC, bool BKC, int NA, int NB>
__device__ __forceinline__ void run_gemm(const Opnd<T> (&A)[NA], const Opnd<T> (&B)[NB], int K, char* lds,
                                         Acc<T, NA, NB>& acc) {
  if constexpr (sizeof(T) == 2)
    gemm_mainloop_b16<AKC, BKC, NA, NB>(A, B, K, (FM_LDS char*)lds, acc);
  else
    gemm_mainloop<T, AKC, BKC, NA, NB>(A, B, K, (T*)lds, acc);
}

}  // namespace fm
