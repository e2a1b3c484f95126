// bf16 grouped-GEMM core for gfx950: persistent blocks of 4 or 8 waves, a
// multi-stage direct-to-LDS ring and register double-buffered MFMA fragments.
//
// A block of WM x WN waves computes an RA x RB output tile of
// C = sum_k A(r, k) B(n, k).  The waves form a WM x WN grid; each owns
// a TM x TN sub-tile as MI x NJ v_mfma_f32_32x32x16_bf16 tiles (the bf16 shape
// that reaches the chip's MFMA peak), operands swapped so that a lane holds
// groups of four consecutive output columns.
//
// * Tiles go straight from global memory to LDS (global_load_lds_dwordx4: each
//   lane moves 16 bytes to LDS base + 16 * lane), 64-k slabs in two rings: NSA
//   slabs of A, NSB = NSA - 1 of B.
//   Per-lane offsets are resolved once per tile; a slab only advances uniform
//   bases held in scalar registers.
// * Every DMA instruction fetches 64 bytes from each of 16 rows, and the next
//   instruction of the same wave fetches the other 64 bytes of the same 128-byte
//   lines.  Inside this kernel the pairing measured faster than instructions
//   that fetch whole lines; a standalone DMA loop moves the same bytes per clock
//   from L2 with either pattern (94-116 bytes per clock per CU).
// * Two products summed into one accumulator can run as one K loop (KJ): the
//   DMA of A and B adds a fixed jump to the second matrix pair from slab kj / 64
//   on (dX = dA_g W_gate + dA_u W_up: one prologue and one drain per tile).
// * K-contiguous slabs are stored as two halves [R rows][32 k] (64-byte rows),
//   the 16-byte chunk index XOR-swizzled by (row >> 2) & 3 so that the fragment
//   reads of 16 consecutive rows hit 16 distinct 4-bank groups.
// * MN-contiguous slabs (weights in the NN products, both operands of the
//   weight-gradient products) are stored as R/32 column blocks [64 k][32 rows]
//   and read with ds_read_b64_tr_b16, which hands each lane four k-consecutive
//   elements of one row; two such reads form a fragment, so nothing is
//   transposed on the way in.  A 32-lane read touches four 64-byte k-rows, 32
//   bytes of each, which already covers the 64 banks once.
// * Fragments are read one 16-k step ahead of the MFMAs that use them, into a
//   second register set.  In the steady state the two waves of each SIMD take
//   turns: one issues a k-step's MFMAs while the other reads its next
//   fragments and issues refills, a block barrier between turns (see b16_gemm).
// * An operand may interleave two matrices in 32-row blocks (gate and up
//   weights; the two dSwiGLU gradients), so that the pairs the epilogue needs sit
//   in one lane.  A DMA instruction always stays inside one 32-row block.
// * With BE = 1 the B operand is int8 (the quantised forward's weight codes,
//   K-contiguous): 64-byte slab rows, one DMA instruction per 16 rows, and each
//   lane widens its 8 codes to bf16 (exactly) as it reads the fragment.
// * Rows past the operand's extent read a clamped (valid) address and only feed
//   outputs that are never stored; k past K is zeroed in the A fragments of the
//   last slab, so the clamped B data meets zeros.
#pragma once

#include <type_traits>

#include "gemm.hpp"

namespace fm {

#define FM_LDS __attribute__((address_space(3)))
typedef short i16x4_t __attribute__((ext_vector_type(4)));
typedef float f32x16_t __attribute__((ext_vector_type(16)));

// Tile configuration: RA x RB block tile, WM x WN waves, BK k per slab,
// separate LDS rings of NSA slabs for A and NSB slabs for B (NSA = NSB + 1: the
// A operand, the one that streams, gets one more slab of latency tolerance).
// BE = bytes per B element: 2 (bf16) or 1 (int8 codes, K-contiguous only,
// widened exactly to bf16 as fragments are read).
template <int RA_, int RB_, int WM_, int WN_, int BK_, int NSA_, int NSB_, int BE_ = 2> struct B16Cfg {
  static constexpr int RA = RA_, RB = RB_, WM = WM_, WN = WN_, BK = BK_, NSA = NSA_, NSB = NSB_, BE = BE_;
  static constexpr int NW = WM * WN, THREADS = 64 * NW;
  static constexpr int TM = RA / WM, TN = RB / WN;    // wave sub-tile
  static constexpr int MI = TM / 32, NJ = TN / 32;    // MFMA tiles per wave
  static constexpr int KS = BK / 16;                  // MFMA k-steps per slab
  static constexpr int A_BYTES = RA * BK * 2, B_BYTES = RB * BK * BE;
  static constexpr int B_BASE = NSA * A_BYTES;        // B ring follows the A ring
  static constexpr int LDS = NSA * A_BYTES + NSB * B_BYTES;
  static constexpr int A_INS = RA * BK * 2 / 1024 / NW;   // DMA instructions per wave and slab
  static constexpr int B_INS = RB * BK * BE / 1024 / NW;
  static_assert(BE == 1 || BE == 2, "bf16 or int8 B");
  static_assert((NW == 4 || NW == 8) && TM % 32 == 0 && TN % 32 == 0, "4 or 8 waves of 32-multiples");
  static_assert(BK == 64, "slab depth: two 32-k halves per slab");
  static_assert(A_INS >= 1 && B_INS >= 1 && KS % 2 == 0, "whole DMA instructions per wave");
  static_assert(NSB >= 2 && NSA == NSB + 1 && LDS <= 160 * 1024, "LDS rings");
};

// s_waitcnt with only vmcnt limited (expcnt / lgkmcnt left at their maxima).
template <int N> __device__ __forceinline__ void wait_vmcnt() {
  static_assert(N >= 0 && N < 64, "vmcnt range");
  __builtin_amdgcn_s_waitcnt((N & 15) | ((N >> 4) << 14) | (7 << 4) | (15 << 8));
}
// s_waitcnt lgkmcnt(0) (vmcnt / expcnt left at their maxima).
__device__ __forceinline__ void wait_lgkm0() { __builtin_amdgcn_s_waitcnt(15 | (3 << 14) | (7 << 4)); }

// Workgroup barrier without the memory fences of __syncthreads: the fences
// would wait for every outstanding load, including the slabs still in flight.
// Each wave waits for its own DMA and LDS reads explicitly before it.
__device__ __forceinline__ void barrier_lds() { asm volatile("s_barrier" ::: "memory"); }

// One global_load_lds_dwordx4: 16 bytes per lane from g to LDS l + 16 * lane
// (l uniform, through M0).  Written as inline assembly so that the compiler's
// wait-count bookkeeping does not see it: it would count the LDS write as an
// out-of-order LDS event and then wait for every pending LDS read before each
// MFMA.  The DMA's own completion is waited for explicitly (vmcnt, then a
// barrier) before its data is read.  M0 is restored; s_nop covers the wait
// state required between writing M0 and an LDS DMA.
__device__ __forceinline__ void dma16(const void* g, FM_LDS void* l) {
  uint32_t saved;
  asm volatile(
      "s_mov_b32 %0, m0\n\t"
      "s_mov_b32 m0, %2\n\t"
      "s_nop 0\n\t"
      "global_load_lds_dwordx4 %1, off\n\t"
      "s_mov_b32 m0, %0"
      : "=&s"(saved)
      : "v"(g), "s"((uint32_t)(uintptr_t)l)
      : "memory");
}

// Keeps the instruction scheduler from moving anything across this point, so
// that fragment reads stay ahead of the MFMAs they overlap.
__device__ __forceinline__ void sched_fence() { __builtin_amdgcn_sched_barrier(0); }

// A wave-uniform pointer held in scalar registers (the compiler cannot always
// prove that a pointer read from memory is uniform).
__device__ __forceinline__ const void* uniform_ptr(const void* p) {
  const uint64_t v = (uint64_t)(uintptr_t)p;
  const uint32_t lo = __builtin_amdgcn_readfirstlane((uint32_t)v);
  const uint32_t hi = __builtin_amdgcn_readfirstlane((uint32_t)(v >> 32));
  return (const void*)(uintptr_t)(((uint64_t)hi << 32) | lo);
}

// The same with a uniform 64-bit base and a 32-bit per-lane byte offset.
__device__ __forceinline__ void dma16s(const void* base, uint32_t off, FM_LDS void* l) {
  base = uniform_ptr(base);
  uint32_t saved;
  asm volatile(
      "s_mov_b32 %0, m0\n\t"
      "s_mov_b32 m0, %3\n\t"
      "s_nop 0\n\t"
      "global_load_lds_dwordx4 %1, %2\n\t"
      "s_mov_b32 m0, %0"
      : "=&s"(saved)
      : "v"(off), "s"(base), "s"((uint32_t)(uintptr_t)l)
      : "memory");
}

// Lane index computed where it is used: volatile, so it cannot be hoisted.
__device__ __forceinline__ int lane_id_here() {
  int l;
  asm volatile("v_mbcnt_lo_u32_b32 %0, -1, 0\n\tv_mbcnt_hi_u32_b32 %0, -1, %0" : "=v"(l));
  return l;
}

// Wave index as a uniform (scalar) value.
__device__ __forceinline__ int wave_id() { return __builtin_amdgcn_readfirstlane(threadIdx.x >> 6); }

// Chunk swizzle of a K-contiguous half-slab row (4 chunks of 16 bytes): 16
// consecutive rows at one logical chunk land on 16 distinct 4-bank groups.
__device__ __forceinline__ int swz_kc(int row) { return (row >> 2) & 3; }

// One operand of the bf16 core: logical [R rows][K].  Element (r, k) lives at
// p[r * ld + k] (K-contiguous) or p[k * ld + r] (MN-contiguous), relative to
// the tile origin.  With p2 set, the logical rows alternate in blocks of 32
// between p (even blocks) and p2 (odd blocks): logical row r is physical row
// 32 (r / 64) + r % 32 of matrix (r / 32) % 2.  rows = physical rows valid from
// the origin (per matrix).  With pk set (a product run with KJ), k >= kj reads
// the matrix at pk (same layout and ld) at k - kj: two products summed into one
// accumulator as a single K loop; kj is a whole number of slabs.
struct B16Src {
  const bf16* p;
  const bf16* p2;
  int ld;
  int rows;
  int K;
  const bf16* pk;
  int kj;
};

__device__ __forceinline__ const bf16* b16_row(const B16Src& s, int r, int& pr) {
  if (s.p2) {
    pr = 32 * (r >> 6) + (r & 31);
    return (r >> 5) & 1 ? s.p2 : s.p;
  }
  pr = r;
  return s.p;
}

// Direct-to-LDS loading of one R-row operand: a slab is R * 128 bytes, R / 8
// instructions of 1 KB, NI = R / 64 per wave.  Instruction `ins` moves:
//   KC: rows 16 (ins / 2) + [0, 16), k-half ins % 2 (32 k), to half
//       ins % 2 at row 16 (ins / 2);
//   MN: k-rows 16 (ins / CB) + [0, 16) of a column block (32 rows), to that
//       block's k-rows; CB = R / 32 column blocks.
// Consecutive instructions of a wave cover the two 64-byte halves of the same
// 16 lines.  Each takes a uniform 64-bit base plus a 32-bit per-lane offset.
template <bool KC, int R, int NI, bool INTER, bool KJ = false> struct B16Dma {
  static constexpr int CB = R / 32;
  static_assert(!(KJ && INTER), "one second matrix");
  const char* base[NI];      // uniform
  uint32_t off[NI];          // per lane
  size_t step;
  size_t jump;               // KJ: added to the address of slabs nj and later
  int nj;

  // Column block of an MN instruction.  With two interleaved matrices the
  // blocks of one matrix alternate, so consecutive instructions take blocks
  // c and c + 2 (the two halves of the same lines): 0, 2, 1, 3, 4, 6, 5, 7, ...
  __device__ __forceinline__ static int cblk(int ins) {
    const int c = ins % CB;
    return INTER ? (c & ~3) | ((c & 1) << 1) | ((c >> 1) & 1) : c;
  }
  // The 32-row block an instruction reads (uniform), and its matrix.
  __device__ __forceinline__ static int block_of(int ins) { return KC ? (ins >> 1) >> 1 : cblk(ins); }
  __device__ __forceinline__ static const bf16* matrix(const B16Src& s, int ins) {
    return (INTER && (block_of(ins) & 1)) ? s.p2 : s.p;
  }
  // Physical row (within its matrix) of logical row r.
  __device__ __forceinline__ static int phys_row(int r) { return INTER ? 32 * (r >> 6) + (r & 31) : r; }

  // Lane's source in slab 0: KC (row, k), MN (k-row, first row).
  __device__ __forceinline__ static void chunk(int ins, int lane, int& a, int& b) {
    if (KC) {
      a = 16 * (ins >> 1) + (lane >> 2);
      b = 32 * (ins & 1) + 8 * ((lane & 3) ^ swz_kc(a));
    } else {
      a = 16 * (ins / CB) + (lane >> 2);
      b = 32 * cblk(ins) + 8 * (lane & 3);
    }
  }
  __device__ __forceinline__ static uint32_t lane_off(const B16Src& s, int ins, int lane, int k0) {
    int a, b;
    chunk(ins, lane, a, b);
    if (KC) {
      // K - 8 >= k0: both are multiples of 8 and the slab starts below K
      return (uint32_t)(((size_t)min(phys_row(a), s.rows - 1) * s.ld + min(b, s.K - 8 - k0)) * 2);
    }
    return (uint32_t)(((size_t)min(a, s.K - 1 - k0) * s.ld + min(phys_row(b), s.rows - 8)) * 2);
  }

  __device__ __forceinline__ void init(const B16Src& s) {
    const int lane = lane_id(), wave = wave_id();
#pragma unroll
    for (int u = 0; u < NI; ++u) {
      const int ins = wave * NI + u;
      base[u] = (const char*)matrix(s, ins);
      off[u] = lane_off(s, ins, lane, 0);
    }
    step = KC ? (size_t)64 * 2 : (size_t)64 * s.ld * 2;
    if (KJ) {
      nj = s.kj / 64;
      jump = (size_t)((uintptr_t)s.pk - (uintptr_t)s.p) - step * (size_t)nj;
    }
  }

  __device__ __forceinline__ static int lds_block(int ins) {
    return KC ? (ins & 1) * (R / 16) + (ins >> 1) : cblk(ins) * 4 + ins / CB;
  }

  __device__ __forceinline__ void issue_full(int slab, FM_LDS char* tile) const { issue_part<0, NI>(slab, tile); }
  // Instructions [U0, U1) of a whole slab (a slab's issue can be spread out).
  template <int U0, int U1>
  __device__ __forceinline__ void issue_part(int slab, FM_LDS char* tile) const {
    const int wave = wave_id();
    const size_t adv = step * (size_t)slab + (KJ && slab >= nj ? jump : 0);
#pragma unroll
    for (int u = U0; u < U1; ++u) dma16s(base[u] + adv, off[u], tile + lds_block(wave * NI + u) * 1024);
  }

  // A slab that reaches past K: k is clamped to the last valid element.  The
  // lane index is re-read here (opaque to the optimiser), so that these address
  // computations are not hoisted and kept live through the main loop.
  __device__ __forceinline__ void issue_tail(const B16Src& s, int k0, FM_LDS char* tile) const {
    const int lane = lane_id_here(), wave = wave_id();
#pragma unroll
    for (int u = 0; u < NI; ++u) {
      const int ins = wave * NI + u;
      const bool second = KJ && k0 >= s.kj;
      const bf16* m = second ? s.pk : matrix(s, ins);
      const int km = second ? k0 - s.kj : k0;
      const char* bt = (const char*)(KC ? m + km : m + (size_t)km * s.ld);
      dma16s(bt, lane_off(s, ins, lane, k0), tile + lds_block(ins) * 1024);
    }
  }
};

// MFMA fragments of a wave's NB 32-row blocks of an R-row tile: a fragment is
// 32 rows x 16 k, 8 k per lane: lane l holds row r0 + l % 32 and k
// 16 ks + 8 (l / 32) + 0..7 of the slab.  Offsets are per lane, computed once:
// for K-contiguous slabs k-step ks lies in half ks / 2 and flips bit 5 of the
// offset (the chunk index is 2 (ks % 2) + l / 32 and the swizzle XORs it); for
// MN-contiguous slabs it adds 16 k-rows.
template <bool KC, int R, int NB> struct B16Frag {
  uint32_t off[NB];

  __device__ __forceinline__ void init(int row0) {
    const int lane = lane_id();
#pragma unroll
    for (int i = 0; i < NB; ++i) {
      const int r0 = row0 + i * 32;
      if (KC) {
        const int r = r0 + (lane & 31);
        off[i] = (uint32_t)(r * 64 + (((lane >> 5) ^ swz_kc(r)) << 4));
      } else {
        // ds_read_b64_tr_b16: in each 16-lane group, output lane i element j
        // comes from the address of lane 4j + i/4, offset i % 4.  Group g covers
        // rows r0 + 16 (g & 1) + [0, 16) and k 8 (g >> 1) + [0, 8) of the k-step;
        // lane L of the group points at (k = kbase + L/4, row = rbase + 4 (L % 4)).
        const int g = lane >> 4, L = lane & 15;
        const int n = r0 + 16 * (g & 1) + 4 * (L & 3);
        const int k = 8 * (g >> 1) + (L >> 2);
        off[i] = (uint32_t)((n >> 5) * (64 * 64) + k * 64 + (n & 31) * 2);
      }
    }
  }

  __device__ __forceinline__ bf16x8_t read(const FM_LDS char* tile, int i, int ks) const {
    if (KC) {
      const FM_LDS char* p = tile + (ks >> 1) * (R * 64) + (off[i] ^ (uint32_t)((ks & 1) << 5));
      return __builtin_bit_cast(bf16x8_t, *(const FM_LDS u32x4_t*)p);
    } else {
      const FM_LDS char* p = tile + off[i] + ks * 16 * 64;
      const i16x4_t v0 = __builtin_amdgcn_ds_read_tr16_b64_v4i16((FM_LDS i16x4_t*)p);
      const i16x4_t v1 = __builtin_amdgcn_ds_read_tr16_b64_v4i16((FM_LDS i16x4_t*)(p + 4 * 64));
      const u32x2_t w0 = __builtin_bit_cast(u32x2_t, v0), w1 = __builtin_bit_cast(u32x2_t, v1);
      return __builtin_bit_cast(bf16x8_t, u32x4_t{w0[0], w0[1], w1[0], w1[1]});
    }
  }
};

// int8 K-contiguous operand (the weights of the quantised forward), logical
// [R rows][K] bytes with the same row / interleave conventions as B16Src (ld
// and K in bytes; the pointers are byte pointers).  A slab is R rows x 64 k =
// 64 bytes per row, stored [R][64 B] with the 16-byte chunk index XOR-swizzled
// by (row >> 2) & 3; instruction ins moves rows 16 ins + [0, 16), 64 bytes of
// each (half of a 128-byte line: the other half belongs to the next slab).
template <int R, int NI, bool INTER> struct I8Dma {
  const char* base[NI];      // uniform
  uint32_t off[NI];          // per lane
  size_t step;

  __device__ __forceinline__ static const char* matrix(const B16Src& s, int ins) {
    return (const char*)((INTER && ((ins >> 1) & 1)) ? s.p2 : s.p);   // 32-row block ins / 2
  }
  __device__ __forceinline__ static int phys_row(int r) { return INTER ? 32 * (r >> 6) + (r & 31) : r; }
  __device__ __forceinline__ static uint32_t lane_off(const B16Src& s, int ins, int lane, int k0) {
    const int a = 16 * ins + (lane >> 2);
    const int b = 16 * ((lane & 3) ^ swz_kc(a));
    // K - 16 >= k0: K is a multiple of 16 and the slab starts below K
    return (uint32_t)((size_t)min(phys_row(a), s.rows - 1) * s.ld + min(b, s.K - 16 - k0));
  }
  __device__ __forceinline__ void init(const B16Src& s) {
    const int lane = lane_id(), wave = wave_id();
#pragma unroll
    for (int u = 0; u < NI; ++u) {
      const int ins = wave * NI + u;
      base[u] = matrix(s, ins);
      off[u] = lane_off(s, ins, lane, 0);
    }
    step = 64;
  }
  __device__ __forceinline__ void issue_full(int slab, FM_LDS char* tile) const { issue_part<0, NI>(slab, tile); }
  template <int U0, int U1>
  __device__ __forceinline__ void issue_part(int slab, FM_LDS char* tile) const {
    const int wave = wave_id();
    const size_t adv = step * (size_t)slab;
#pragma unroll
    for (int u = U0; u < U1; ++u) dma16s(base[u] + adv, off[u], tile + (wave * NI + u) * 1024);
  }
  __device__ __forceinline__ void issue_tail(const B16Src& s, int k0, FM_LDS char* tile) const {
    const int lane = lane_id_here(), wave = wave_id();
#pragma unroll
    for (int u = 0; u < NI; ++u) {
      const int ins = wave * NI + u;
      dma16s(matrix(s, ins) + k0, lane_off(s, ins, lane, k0), tile + ins * 1024);
    }
  }
};

// Eight int8 codes -> eight bf16 (exact: |q| <= 128 has at most 8 significant bits).
__device__ __forceinline__ bf16x8_t widen_i8x8(u32x2_t raw) {
  u32x4_t v;
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const uint32_t x = raw[i >> 1];
    const int sh = (i & 1) * 16;
    const float lo = (float)(int8_t)((x >> sh) & 0xFF);
    const float hi = (float)(int8_t)((x >> (sh + 8)) & 0xFF);
    v[i] = (__float_as_uint(lo) >> 16) | (__float_as_uint(hi) & 0xFFFF0000u);
  }
  return __builtin_bit_cast(bf16x8_t, v);
}

// Fragments of an int8 slab: lane l holds row r0 + l % 32 and k 16 ks +
// 8 (l / 32) + 0..7, i.e. 8 bytes of chunk ks (swizzled), widened to bf16.
// Sixteen consecutive rows read 16 distinct 2-bank groups.
template <int R, int NB> struct I8Frag {
  uint32_t off[NB];
  __device__ __forceinline__ void init(int row0) {
    const int lane = lane_id();
#pragma unroll
    for (int i = 0; i < NB; ++i) {
      const int r = row0 + i * 32 + (lane & 31);
      off[i] = (uint32_t)(r * 64 + (swz_kc(r) << 4) + 8 * (lane >> 5));
    }
  }
  __device__ __forceinline__ bf16x8_t read(const FM_LDS char* tile, int i, int ks) const {
    return widen_i8x8(*(const FM_LDS u32x2_t*)(tile + (off[i] ^ (uint32_t)(ks << 4))));
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

// Accumulator of a wave's sub-tile: MI x NJ MFMA tiles of 32 x 32.  Register
// r of tile (i, j) holds sub-tile row i*32 + lane % 32 and column
// j*32 + 8 (r / 4) + 4 (lane / 32) + r % 4.
template <int MI, int NJ> struct B16Acc {
  f32x16_t v[MI][NJ];
  __device__ __forceinline__ void zero() {
#pragma unroll
    for (int i = 0; i < MI; ++i)
#pragma unroll
      for (int j = 0; j < NJ; ++j)
#pragma unroll
        for (int r = 0; r < 16; ++r) v[i][j][r] = 0.f;
  }
  // registers 4q .. 4q+3 of tile (i, j)
  __device__ __forceinline__ f32x4_t quad(int i, int j, int q) const {
    const f32x16_t& t = v[i][j];
    return f32x4_t{t[4 * q], t[4 * q + 1], t[4 * q + 2], t[4 * q + 3]};
  }
};

// Block-tile coordinates of quad (i, j, q): the row, and the first of 4 columns.
template <class C> __device__ __forceinline__ AccCoord b16_coord(int i, int j, int q) {
  const int lane = lane_id(), wave = wave_id();
  const int wm = wave % C::WM, wn = wave / C::WM;
  return AccCoord{wm * C::TM + i * 32 + (lane & 31), wn * C::TN + j * 32 + 8 * q + 4 * (lane >> 5)};
}

// Output staging.  Stores straight from the accumulator layout write 8 bytes
// per lane scattered over 32 rows; instead a tile is put into LDS (row-major,
// the 16-byte chunk index XOR-swizzled by the row) and copied out with every
// lane storing 16 consecutive bytes and each row written whole.  T is the
// element type of the output (bf16 or float), COLS the tile width.
template <typename T, int COLS> struct Stage {
  static constexpr int EPC = 16 / sizeof(T);         // elements per 16-byte chunk
  static constexpr int CPR = COLS / EPC;             // chunks per row
  static constexpr int ROW_BYTES = COLS * (int)sizeof(T);
  static_assert(CPR == 16 || CPR == 32 || CPR == 64, "chunks per row");

  // LDS byte offset of the 4 values at (row, col), col a multiple of 4.
  static __device__ __forceinline__ uint32_t at(int row, int col) {
    const int c = col / EPC;
    return (uint32_t)(row * ROW_BYTES + ((c ^ (row & (CPR - 1))) << 4) + (col % EPC) * (int)sizeof(T));
  }
  static __device__ __forceinline__ void put4(FM_LDS char* lds, int row, int col, f32x4_t v) {
    FM_LDS char* p = lds + at(row, col);
    if (sizeof(T) == 2) {
      *(FM_LDS u32x2_t*)p = u32x2_t{pk_bf16(v[0], v[1]), pk_bf16(v[2], v[3])};
    } else {
      *(FM_LDS f32x4_t*)p = v;
    }
  }
  // Copies rows [0, ROWS) of the staged tile out with NT threads: row r goes to
  // row_ptr(r) (nullptr: not stored), columns below cols_valid (a multiple of
  // EPC); with accumulate (float only) the values are added to what the output
  // holds.
  template <int ROWS, int NT, class RowPtr>
  static __device__ __forceinline__ void copy_rows(const FM_LDS char* lds, RowPtr row_ptr, int cols_valid,
                                                   bool accumulate = false) {
    constexpr int TOTAL = ROWS * CPR;
    // thread index re-read here (opaque): per-lane addresses stay out of the
    // registers of a surrounding tile loop
    const int tid = wave_id() * 64 + lane_id_here();
#pragma unroll 4
    for (int idx = tid; idx < TOTAL; idx += NT) {
      const int row = idx / CPR, c = idx % CPR;
      u32x4_t v = *(const FM_LDS u32x4_t*)(lds + row * ROW_BYTES + ((c ^ (row & (CPR - 1))) << 4));
      T* out = row_ptr(row);
      if (out != nullptr && c * EPC < cols_valid) {
        T* dst = out + c * EPC;
        if (sizeof(T) == 4 && accumulate) {
          const f32x4_t o = *(const FM_GLOBAL f32x4_t*)dst;
          v = __builtin_bit_cast(u32x4_t, __builtin_bit_cast(f32x4_t, v) + o);
        }
        st16(dst, v);
      }
    }
  }
  // Rows [0, ROWS) to out[row * ld + col] for row < rows_valid.
  template <int ROWS, int NT>
  static __device__ __forceinline__ void copy_out(const FM_LDS char* lds, T* out, size_t ld, int rows_valid,
                                                  int cols_valid) {
    copy_rows<ROWS, NT>(lds, [=](int row) { return row < rows_valid ? out + (size_t)row * ld : (T*)nullptr; },
                    cols_valid);
  }
};

// Barrier that also makes this wave's LDS writes visible to the block.
__device__ __forceinline__ void barrier_lds_writes() {
  wait_lgkm0();
  barrier_lds();
}

// k loop over [0, K), accumulating into acc.  Ends with a barrier so the LDS
// can be reused by a following call.
//
// DMA order.  At the barrier that ends slab kt the block issues B(kt + NSB),
// then A(kt + NSA) (when they exist).  Slab kt + 1 is then complete once every
// DMA instruction issued before A(kt + NSA - 1) has landed: the waits count the
// A instructions issued after B(kt + 1) (s_waitcnt vmcnt is in issue order).
//
// Steady state (slab kt, while both refills are whole slabs): the two waves of
// each SIMD take turns on its matrix pipe.  Group P (waves 0 .. NW/2-1) and
// group Q (the others, one per SIMD) run the same straight-line loop one
// block barrier apart: Q passes one extra barrier before the loop, P one after
// it.  The loop alternates an MFMA burst (the 16 products of two k-steps) with
// the next two k-steps' fragment reads plus the refills, a barrier after each
// (four per slab), so while P multiplies Q reads and the other way round, and
// neither wave runs a slab's last k-steps alone.  (Left to the hardware, the
// first wave of a SIMD took the pipe for whole bursts and finished its k-steps
// about 800 clocks per slab before the second, which then could not keep the
// pipe busy by itself.)  Each wave's reads, MFMAs and refills keep their order
// (accumulation order and vmcnt counting as before).  The slab's buffers are
// released by the barrier after P's last burst, which is the barrier after Q's
// last reads: both of those phases end with the wave's reads of the slab and
// its DMA of the next slab complete.  The last slabs (and the partial one)
// drain through a general version of the step with every wave in step.
// The DMA side of one product: slab issue into the two rings.
template <class C, bool AKC, bool BKC, bool AI, bool BI, bool KJ = false> struct B16Pipe {
  static constexpr int BK = C::BK, NSA = C::NSA, NSB = C::NSB;
  static_assert(C::BE == 2 || BKC, "int8 B is K-contiguous");
  static_assert(C::BE == 2 || !KJ, "bf16 operands only");
  using DmaB = std::conditional_t<C::BE == 1, I8Dma<C::RB, C::B_INS, BI>, B16Dma<BKC, C::RB, C::B_INS, BI, KJ>>;
  B16Dma<AKC, C::RA, C::A_INS, AI, KJ> da;
  DmaB db;
  const B16Src& A;
  const B16Src& B;
  FM_LDS char* lds;
  int nk, nfull;

  __device__ __forceinline__ B16Pipe(const B16Src& A_, const B16Src& B_, int K, FM_LDS char* lds_)
      : A(A_), B(B_), lds(lds_) {
    nk = (K + BK - 1) / BK;
    nfull = K / BK;
    if (nk > 0) {
      da.init(A);
      db.init(B);
    }
  }
  __device__ __forceinline__ FM_LDS char* abuf(int s) const { return lds + (s % NSA) * C::A_BYTES; }
  __device__ __forceinline__ FM_LDS char* bbuf(int s) const { return lds + C::B_BASE + (s % NSB) * C::B_BYTES; }
  __device__ __forceinline__ void issue_a(int s) const {
    if (s < nfull) da.issue_full(s, abuf(s));
    else da.issue_tail(A, s * BK, abuf(s));
  }
  __device__ __forceinline__ void issue_b(int s) const {
    if (s < nfull) db.issue_full(s, bbuf(s));
    else db.issue_tail(B, s * BK, bbuf(s));
  }
  // B(0) A(0) B(1) A(1) ... B(NSB-1) A(NSB-1) A(NSA-1), as far as there are slabs.
  __device__ __forceinline__ void prologue() const {
#pragma nounroll
    for (int s = 0; s < NSA && s < nk; ++s) {
      if (s < NSB) issue_b(s);
      issue_a(s);
    }
  }
};

// Issues the prologue of a product ahead of its b16_gemm call (which then takes
// EXTRA >= 0): a persistent kernel starts the next tile's first slabs before the
// previous tile's epilogue stores, so those stores drain while the slabs land.
// The LDS rings must be free (no reads or DMA of the previous tile pending).
template <class C, bool AKC, bool BKC, bool AI = false, bool BI = false>
__device__ __forceinline__ void b16_prologue(const B16Src& A, const B16Src& B, int K, FM_LDS char* lds) {
  const B16Pipe<C, AKC, BKC, AI, BI> pp(A, B, K, lds);
  pp.prologue();
}

// EXTRA < 0: the product issues its own prologue.  EXTRA >= 0: b16_prologue
// issued it already (same A, B, K); with extra_issued the wave has issued at
// least EXTRA more vector-memory instructions since, which may stay in flight
// at the first wait.  KJ: A and B switch to their second matrices (pk) at k = kj.
template <class C, bool AKC, bool BKC, bool AI = false, bool BI = false, int EXTRA = -1, bool KJ = false>
__device__ __forceinline__ void b16_gemm(const B16Src& A, const B16Src& B, int K, FM_LDS char* lds,
                                         B16Acc<C::MI, C::NJ>& acc, bool extra_issued = true) {
  constexpr int BK = C::BK, NSA = C::NSA, NSB = C::NSB, KS = C::KS, MI = C::MI, NJ = C::NJ;
  constexpr int PA = C::A_INS, PB = C::B_INS;   // DMA instructions per wave and slab
  constexpr int XW = EXTRA < 0 ? 0 : EXTRA;
  static_assert((NSB - 1) * (PA + PB) + PA + XW < 64, "vmcnt range");
  const B16Pipe<C, AKC, BKC, AI, BI, KJ> pp(A, B, K, lds);
  const int nk = pp.nk;
  if (nk <= 0) return;
  const int nfull = pp.nfull;
  const int wave = wave_id();
  B16Frag<AKC, C::RA, MI> fa;
  std::conditional_t<C::BE == 1, I8Frag<C::RB, NJ>, B16Frag<BKC, C::RB, NJ>> fb;
  fa.init((wave % C::WM) * C::TM);
  fb.init((wave / C::WM) * C::TN);
  const auto& da = pp.da;
  const auto& db = pp.db;

  auto abuf = [&](int s) { return pp.abuf(s); };
  auto bbuf = [&](int s) { return pp.bbuf(s); };
  auto issue_a = [&](int s) { pp.issue_a(s); };
  auto issue_b = [&](int s) { pp.issue_b(s); };
  bf16x8_t xa[2][MI], xb[2][NJ];
  auto read = [&](int set, int s, int ks) {
    const FM_LDS char* ab = abuf(s);
    const FM_LDS char* bb = bbuf(s);
#pragma unroll
    for (int i = 0; i < MI; ++i) xa[set][i] = fa.read(ab, i, ks);
#pragma unroll
    for (int j = 0; j < NJ; ++j) xb[set][j] = fb.read(bb, j, ks);
  };
  // MFMAs of register set `set` for A tiles [i0, i1).
  auto mma = [&](int set, int i0, int i1, bool tail, int k0, int ks) {
#pragma unroll
    for (int i = i0; i < i1; ++i) {
      const bf16x8_t a = tail ? b16_mask_k(xa[set][i], k0, ks, K) : xa[set][i];
#pragma unroll
      for (int j = 0; j < NJ; ++j)
        acc.v[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(xb[set][j], a, acc.v[i][j], 0, 0, 0);
    }
  };
  constexpr int LAST = (KS - 1) & 1;           // register set of the last k-step

  if (EXTRA < 0) pp.prologue();
  // slab 0 is complete once everything issued after A(0) is at most in flight
  if (XW > 0 && extra_issued) {
    if (nk >= NSA) wait_vmcnt<(NSB - 1) * (PA + PB) + PA + XW>();
    else if (nk >= NSB) wait_vmcnt<(NSB - 1) * (PA + PB) + XW>();   // A(NSA - 1) does not exist
    else wait_vmcnt<XW>();
  } else {
    if (nk >= NSA) wait_vmcnt<(NSB - 1) * (PA + PB) + PA>();
    else if (nk >= NSB) wait_vmcnt<(NSB - 1) * (PA + PB)>();
    else wait_vmcnt<0>();
  }
  wait_lgkm0();   // no scalar loads pending: LDS-read waits in the loop can count
  barrier_lds();
  read(0, 0, 0);

  int kt = 0;
  const int nsteady = nfull - NSA;             // refills A(kt + NSA), B(kt + NSB) whole
  // Per slab each wave issues A(kt + 2) with its reads of k-steps 2 and 3, and
  // B(kt + 2) right after the slab barrier that frees B's buffer, so that the
  // slab-end wait (at most A(kt + 2) in flight) finds B(kt + 1) issued a whole
  // read phase and burst earlier.
  static_assert(KS == 4, "two k-steps per burst");
  const bool P = wave < C::NW / 2;
  auto bar = [&]() { sched_fence(); barrier_lds(); sched_fence(); };
  if (nsteady > 0) read(1, 0, 1);              // the first burst multiplies k-steps 0 and 1
  if (nsteady > 0 && !P) bar();
  for (; kt < nsteady; ++kt) {
    // 1: k-steps 0 and 1
    mma(0, 0, MI, false, 0, 0);
    mma(1, 0, MI, false, 0, 0);
    bar();
    // 2: read k-steps 2 and 3; A(kt + 2); this slab's reads and the next slab's DMA done
    read(0, kt, 2);
    read(1, kt, 3);
    if (kt > 0) da.issue_full(kt + NSA - 1, abuf(kt + NSA - 1));
    sched_fence();
    wait_lgkm0();
    wait_vmcnt<PA>();                          // A(kt + NSA - 1) may still be in flight
    bar();                                     // Q: the slab barrier
    // 3: k-steps 2 and 3
    mma(0, 0, MI, false, 0, 0);
    mma(1, 0, MI, false, 0, 0);
    sched_fence();
    wait_lgkm0();
    wait_vmcnt<PA>();
    bar();                                     // P: the slab barrier
    // 4: B(kt + 2) into this slab's B buffer; the next slab's k-steps 0 and 1
    db.issue_full(kt + NSB, bbuf(kt + NSB));
    read(0, kt + 1, 0);
    read(1, kt + 1, 1);
    bar();
  }
  if (nsteady > 0 && P) bar();
  // Refills still owed by the last steady slab.
  if (kt > 0 && kt == nsteady) da.issue_full(kt + NSA - 1, abuf(kt + NSA - 1));
  // Drain: the slabs whose refills pass the end, and the partial slab.
  for (; kt < nk; ++kt) {
    const bool tail = kt >= nfull;
#pragma unroll
    for (int ks = 0; ks + 1 < KS; ++ks) {
      read((ks & 1) ^ 1, kt, ks + 1);
      mma(ks & 1, 0, MI, tail, kt * BK, ks);
    }
    if (kt + 1 < nk) {
      wait_lgkm0();
      // A(kt + NSA - 1), issued right after B(kt + 1), may stay in flight
      if (kt + NSA - 1 < nk) wait_vmcnt<PA>();
      else wait_vmcnt<0>();
      barrier_lds();
      if (kt + NSB < nk) issue_b(kt + NSB);
      if (kt + NSA < nk) issue_a(kt + NSA);
      read(LAST ^ 1, kt + 1, 0);
    }
    mma(LAST, 0, MI, tail, kt * BK, KS - 1);
  }
  barrier_lds();
}

}  // namespace fm
