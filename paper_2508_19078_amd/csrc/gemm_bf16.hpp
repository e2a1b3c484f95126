// bf16 main loop of the grouped-GEMM core for gfx950: a three-stage
// direct-to-LDS pipeline.
//
// Same block shape and accumulator layout as gemm.hpp (256 threads, 2 x 2
// waves, 128 x 128 output tile, operands swapped in the MFMA so each lane owns
// four consecutive output columns), with a K slab of 64:
//
// * Global tiles go straight to LDS with global_load_lds_dwordx4 (each lane
//   moves 16 bytes to LDS base + 16 * lane), three slabs deep: two slabs are in
//   flight while the third is multiplied, with no staging registers.
// * K-contiguous tiles are stored [row][64 k] (128-byte rows) with the 16-byte
//   chunk index XOR-swizzled by (row >> 1) & 7, so the 16-byte fragment reads of
//   16 consecutive rows hit 16 distinct 4-bank groups.
// * MN-contiguous tiles (weights in the NN products, both operands of the
//   weight-gradient products) are stored k-major, [64 k][128 rows] (256-byte
//   rows), with the chunk index XOR-swizzled by a function of k, and read with
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
__device__ __forceinline__ int swz_mn(int k) { return ((k & 3) << 1) | (((k >> 3) & 1) << 3); }

// Issues this wave's share (4 x 1 KB) of one operand tile for the slab at k0.
template <bool KC>
__device__ __forceinline__ void b16_issue_tile(const Opnd<bf16>& op, int k0, FM_LDS char* tile) {
  const int lane = lane_id(), wave = threadIdx.x >> 6;
#pragma unroll
  for (int u = 0; u < 4; ++u) {
    const int ins = wave * 4 + u;               // 1 KB block of the tile
    FM_LDS char* dst = tile + ins * 1024;
    if (KC) {
      const int r = ins * 8 + (lane >> 3);      // 8 rows of 128 bytes
      const int c = (lane & 7) ^ swz_kc(r);     // global chunk this lane fetches
      const int rr = min(r, op.rows - 1);
      const int col = min(k0 + 8 * c, op.K - 8);
      dma16(op.p + (size_t)rr * op.ld + col, dst);
    } else {
      const int kr = ins * 4 + (lane >> 4);     // 4 k-rows of 256 bytes
      const int c = (lane & 15) ^ swz_mn(kr);
      const int kk = min(k0 + kr, op.K - 1);
      const int rc = min(8 * c, op.rows - 8);
      dma16(op.p + (size_t)kk * op.ld + rc, dst);
    }
  }
}

// One MFMA fragment (16 rows x 8 k) of rows [r0, r0+16) at k-step ks (0/1).
template <bool KC>
__device__ __forceinline__ bf16x8_t b16_frag(const FM_LDS char* tile, int r0, int ks) {
  const int lane = lane_id(), r16 = lane & 15, q4 = lane >> 4;
  if (KC) {
    const int r = r0 + r16;
    const int c = ks * 4 + q4;
    const FM_LDS char* p = tile + r * 128 + ((c ^ swz_kc(r)) << 4);
    return __builtin_bit_cast(bf16x8_t, *(const FM_LDS u32x4_t*)p);
  } else {
    // ds_read_b64_tr_b16: in each 16-lane group, output lane i element j comes
    // from the address of lane 4j + i/4, offset i % 4.  Lane L therefore points
    // at (k = kbase + L/4, row = r0 + 4 (L % 4)).
    const int L = r16;
    const int n = r0 + 4 * (L & 3);
    const int half = (n >> 2) & 1;
    const int chunk = n >> 3;
    u32x4_t out;
#pragma unroll
    for (int h = 0; h < 2; ++h) {
      const int k = ks * 32 + 8 * q4 + 4 * h + (L >> 2);
      const FM_LDS char* p = tile + k * 256 + ((chunk ^ swz_mn(k)) << 4) + half * 8;
      const i16x4_t v = __builtin_amdgcn_ds_read_tr16_b64_v4i16((FM_LDS i16x4_t*)p);
      const u32x2_t w = __builtin_bit_cast(u32x2_t, v);
      out[2 * h] = w[0];
      out[2 * h + 1] = w[1];
    }
    return __builtin_bit_cast(bf16x8_t, out);
  }
}

// Zeroes the k >= K elements of an A fragment (k-step ks of the slab at k0).
__device__ __forceinline__ bf16x8_t b16_mask_k(bf16x8_t f, int k0, int ks, int K) {
  const int kf = k0 + ks * 32 + 8 * (lane_id() >> 4);
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

template <bool AKC, bool BKC, int NA, int NB>
__device__ __forceinline__ void b16_mma_slab(const FM_LDS char* buf, Acc<bf16, NA, NB>& acc, int k0,
                                             int K, bool tail) {
  const int wave = threadIdx.x >> 6;
  const int wm = wave & 1, wn = wave >> 1;
#pragma unroll
  for (int ks = 0; ks < 2; ++ks) {
    bf16x8_t fa[NA][4], fb[NB][4];
#pragma unroll
    for (int a = 0; a < NA; ++a)
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        fa[a][i] = b16_frag<AKC>(buf + a * B16_TILE, wm * 64 + i * 16, ks);
        if (tail) fa[a][i] = b16_mask_k(fa[a][i], k0, ks, K);
      }
#pragma unroll
    for (int b = 0; b < NB; ++b)
#pragma unroll
      for (int j = 0; j < 4; ++j) fb[b][j] = b16_frag<BKC>(buf + (NA + b) * B16_TILE, wn * 64 + j * 16, ks);
#pragma unroll
    for (int a = 0; a < NA; ++a)
#pragma unroll
      for (int b = 0; b < NB; ++b)
#pragma unroll
        for (int i = 0; i < 4; ++i)
#pragma unroll
          for (int j = 0; j < 4; ++j)
            acc.v[a * NB + b][i][j] =
                __builtin_amdgcn_mfma_f32_16x16x32_bf16(fb[b][j], fa[a][i], acc.v[a * NB + b][i][j], 0, 0, 0);
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
  auto issue = [&](int s) {
    FM_LDS char* buf = lds + (s % B16_NS) * STAGE;
#pragma unroll
    for (int a = 0; a < NA; ++a) b16_issue_tile<AKC>(A[a], s * B16_BK, buf + a * B16_TILE);
#pragma unroll
    for (int b = 0; b < NB; ++b) b16_issue_tile<BKC>(B[b], s * B16_BK, buf + (NA + b) * B16_TILE);
  };
  issue(0);
  if (nk > 1) issue(1);
  for (int kt = 0; kt < nk; ++kt) {
    if (kt + 1 < nk) wait_vmcnt<PER_STAGE>();
    else wait_vmcnt<0>();
    barrier_lds();
    if (kt + 2 < nk) issue(kt + 2);
    const int k0 = kt * B16_BK;
    b16_mma_slab<AKC, BKC, NA, NB>(lds + (kt % B16_NS) * STAGE, acc, k0, K, k0 + B16_BK > K);
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
