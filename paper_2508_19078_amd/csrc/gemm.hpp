// Block-level MFMA GEMM core for the grouped expert FFN (gfx950, wave64).
//
// A block of 256 threads (4 waves, 2 x 2) computes a BM x BN = 128 x 128 tile
// of C = sum_k A(m, k) B(n, k) for NA A-operands and NB B-operands at once
// (NA * NB accumulators: the gate and up projections share their A tile, the
// two weight gradients dW_gate / dW_up share their B tile).  Each operand is
// either K-contiguous (element (r, k) at p[r * ld + k]) or MN-contiguous
// (element (r, k) at p[k * ld + r]); both are staged through LDS as [r][k]
// rows, so every MFMA fragment is one 16-byte LDS read.  MN-contiguous tiles
// are transposed on the way in: a thread loads two k-rows of 16 bytes and
// writes (k, k+1) pairs.  Global tiles are double-buffered through registers:
// the next k-slab is in flight while the current one is multiplied.
//
// MFMA: v_mfma_f32_16x16x32_bf16 (bf16) or 4 x v_mfma_f32_16x16x4_f32 (fp32),
// with the operands swapped (B first) so that each lane's four accumulator
// values are four consecutive output columns of one row: stores are 8 or 16
// bytes wide.  Out-of-range rows, columns and k are loaded as zeros.
#pragma once

#include "common.hpp"

namespace fm {

constexpr int G_BM = 128, G_BN = 128, G_THREADS = 256;

template <typename T> struct GemmCfg {
  static constexpr int V = 16 / sizeof(T);   // elements per 16 bytes
  static constexpr int BK = 4 * V;           // k per slab: one MFMA k-step
  static constexpr int LDSS = BK + V;        // LDS row stride (elements), 16-byte pad
  static constexpr int TILE = 128 * LDSS;    // elements of one staged operand tile
};

template <typename T> struct Opnd {
  const T* p;   // tile origin (r = 0, k = 0)
  int ld;       // row stride (K-contiguous) or k stride (MN-contiguous), elements
  int rows;     // valid r extent from the origin (<= 0: none)
  int K;        // valid k extent
};

template <typename T> struct frag_of;
template <> struct frag_of<bf16> { typedef bf16x8_t type; };
template <> struct frag_of<float> { typedef f32x4_t type; };

__device__ __forceinline__ f32x4_t mfma_step(bf16x8_t b, bf16x8_t a, f32x4_t c) {
  return __builtin_amdgcn_mfma_f32_16x16x32_bf16(b, a, c, 0, 0, 0);
}
__device__ __forceinline__ f32x4_t mfma_step(f32x4_t b, f32x4_t a, f32x4_t c) {
#pragma unroll
  for (int i = 0; i < 4; ++i) c = __builtin_amdgcn_mfma_f32_16x16x4f32(b[i], a[i], c, 0, 0, 0);
  return c;
}

// Global -> registers -> LDS staging of one 128 x BK operand tile.
template <typename T, bool KC> struct Stager {
  typedef GemmCfg<T> C;
  static constexpr int V = C::V, BK = C::BK;
  static constexpr int NCH = 128 * BK / V / G_THREADS;   // 16-byte loads per thread (2)
  u32x4_t reg[NCH];

  __device__ __forceinline__ void load(const Opnd<T>& op, int k0) {
    const int tid = threadIdx.x;
    if (KC) {
#pragma unroll
      for (int u = 0; u < NCH; ++u) {
        const int c = tid + G_THREADS * u;
        const int r = c / (BK / V), kc = (c % (BK / V)) * V;
        const bool ok = r < op.rows && k0 + kc < op.K;
        reg[u] = ok ? ld16(op.p + (size_t)r * op.ld + k0 + kc) : u32x4_t{0, 0, 0, 0};
      }
    } else {
#pragma unroll
      for (int u = 0; u < NCH / 2; ++u) {
        const int c = tid + G_THREADS * u;
        const int rc = (c % (128 / V)) * V, kp = 2 * (c / (128 / V));
        const bool rok = rc < op.rows;
        const int ka = k0 + kp, kb = k0 + kp + 1;
        reg[2 * u] = (rok && ka < op.K) ? ld16(op.p + (size_t)ka * op.ld + rc) : u32x4_t{0, 0, 0, 0};
        reg[2 * u + 1] = (rok && kb < op.K) ? ld16(op.p + (size_t)kb * op.ld + rc) : u32x4_t{0, 0, 0, 0};
      }
    }
  }

  __device__ __forceinline__ void store(T* lds) const {
    const int tid = threadIdx.x;
    if (KC) {
#pragma unroll
      for (int u = 0; u < NCH; ++u) {
        const int c = tid + G_THREADS * u;
        const int r = c / (BK / V), kc = (c % (BK / V)) * V;
        *reinterpret_cast<u32x4_t*>(lds + r * C::LDSS + kc) = reg[u];   // LDS
      }
    } else {
#pragma unroll
      for (int u = 0; u < NCH / 2; ++u) {
        const int c = tid + G_THREADS * u;
        const int rc = (c % (128 / V)) * V, kp = 2 * (c / (128 / V));
        const u32x4_t a = reg[2 * u], b = reg[2 * u + 1];
        if (sizeof(T) == 2) {
#pragma unroll
          for (int i = 0; i < V; ++i) {
            const uint32_t lo = (a[i / 2] >> (16 * (i & 1))) & 0xFFFFu;
            const uint32_t hi = (b[i / 2] >> (16 * (i & 1))) & 0xFFFFu;
            *reinterpret_cast<uint32_t*>(lds + (rc + i) * C::LDSS + kp) = lo | (hi << 16);
          }
        } else {
#pragma unroll
          for (int i = 0; i < V; ++i)
            *reinterpret_cast<uint2*>(lds + (rc + i) * C::LDSS + kp) = make_uint2(a[i], b[i]);
        }
      }
    }
  }
};

// acc[a * NB + b][i][j]: wave sub-tile (i, j) of operand pair (a, b), 16 x 16
// MFMA tiles (the fp32 core).  The bf16 core specialises this with 32 x 32 tiles.
template <typename T, int NA, int NB> struct Acc {
  f32x4_t v[NA * NB][4][4];
  __device__ __forceinline__ void zero() {
#pragma unroll
    for (int x = 0; x < NA * NB; ++x)
#pragma unroll
      for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int j = 0; j < 4; ++j) v[x][i][j] = f32x4_t{0, 0, 0, 0};
  }
  __device__ __forceinline__ f32x4_t quad(int x, int g) const { return v[x][g >> 2][g & 3]; }
};

// Multiplies the staged slab in `lds` (operand tiles A0..A{NA-1}, B0..B{NB-1}).
template <typename T, int NA, int NB>
__device__ __forceinline__ void mma_slab(const T* lds, Acc<T, NA, NB>& acc) {
  typedef GemmCfg<T> C;
  typedef typename frag_of<T>::type frag;
  const int lane = lane_id(), wave = threadIdx.x >> 6;
  const int wm = wave & 1, wn = wave >> 1;
  const int r16 = lane & 15, q4 = lane >> 4;
  frag fa[NA][4], fb[NB][4];
#pragma unroll
  for (int a = 0; a < NA; ++a)
#pragma unroll
    for (int i = 0; i < 4; ++i)
      fa[a][i] = *reinterpret_cast<const frag*>(lds + a * C::TILE +
                                                (wm * 64 + i * 16 + r16) * C::LDSS + q4 * C::V);
#pragma unroll
  for (int b = 0; b < NB; ++b)
#pragma unroll
    for (int j = 0; j < 4; ++j)
      fb[b][j] = *reinterpret_cast<const frag*>(lds + (NA + b) * C::TILE +
                                                (wn * 64 + j * 16 + r16) * C::LDSS + q4 * C::V);
#pragma unroll
  for (int a = 0; a < NA; ++a)
#pragma unroll
    for (int b = 0; b < NB; ++b)
#pragma unroll
      for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int j = 0; j < 4; ++j)
          acc.v[a * NB + b][i][j] = mfma_step(fb[b][j], fa[a][i], acc.v[a * NB + b][i][j]);
}

// Runs the k loop over [0, K) for the given operands, accumulating into acc.
// `lds` holds 2 buffers of (NA + NB) tiles.  Ends with a barrier so the LDS can
// be reused by a following call.
template <typename T, bool AKC, bool BKC, int NA, int NB>
__device__ __forceinline__ void gemm_mainloop(const Opnd<T> (&A)[NA], const Opnd<T> (&B)[NB], int K,
                                              T* lds, Acc<T, NA, NB>& acc) {
  typedef GemmCfg<T> C;
  constexpr int BUF = (NA + NB) * C::TILE;
  const int nk = (K + C::BK - 1) / C::BK;
  if (nk <= 0) return;
  Stager<T, AKC> sa[NA];
  Stager<T, BKC> sb[NB];
#pragma unroll
  for (int a = 0; a < NA; ++a) sa[a].load(A[a], 0);
#pragma unroll
  for (int b = 0; b < NB; ++b) sb[b].load(B[b], 0);
#pragma unroll
  for (int a = 0; a < NA; ++a) sa[a].store(lds + a * C::TILE);
#pragma unroll
  for (int b = 0; b < NB; ++b) sb[b].store(lds + (NA + b) * C::TILE);
  __syncthreads();
  for (int kt = 0; kt < nk; ++kt) {
    const int cur = kt & 1;
    const bool more = kt + 1 < nk;
    if (more) {
#pragma unroll
      for (int a = 0; a < NA; ++a) sa[a].load(A[a], (kt + 1) * C::BK);
#pragma unroll
      for (int b = 0; b < NB; ++b) sb[b].load(B[b], (kt + 1) * C::BK);
    }
    mma_slab<T, NA, NB>(lds + cur * BUF, acc);
    if (more) {
#pragma unroll
      for (int a = 0; a < NA; ++a) sa[a].store(lds + (cur ^ 1) * BUF + a * C::TILE);
#pragma unroll
      for (int b = 0; b < NB; ++b) sb[b].store(lds + (cur ^ 1) * BUF + (NA + b) * C::TILE);
    }
    __syncthreads();
  }
}

// Epilogues walk an accumulator as 16 "quads": four consecutive output columns
// of one row.  quad_coord<T>(g) gives the row and first column of quad g within
// the 128 x 128 block tile; acc.quad(x, g) the four values of operand pair x.
struct AccCoord;
template <typename T> __device__ __forceinline__ AccCoord quad_coord(int g);

// Output coordinates of accumulator element r of wave sub-tile (i, j):
// row = wm*64 + i*16 + (lane & 15), columns col4 .. col4+3 with
// col4 = wn*64 + j*16 + 4*(lane >> 4).
struct AccCoord {
  int row, col4;
};
__device__ __forceinline__ AccCoord acc_coord(int i, int j) {
  const int lane = lane_id(), wave = threadIdx.x >> 6;
  return AccCoord{(wave & 1) * 64 + i * 16 + (lane & 15), (wave >> 1) * 64 + j * 16 + 4 * (lane >> 4)};
}
template <> __device__ __forceinline__ AccCoord quad_coord<float>(int g) { return acc_coord(g >> 2, g & 3); }

// 4 consecutive values <-> global memory of T.
__device__ __forceinline__ void store4(bf16* p, f32x4_t v) {
  u32x2_t o;
  o[0] = pk_bf16(v[0], v[1]);
  o[1] = pk_bf16(v[2], v[3]);
  *(FM_GLOBAL u32x2_t*)(p) = o;
}
__device__ __forceinline__ void store4(float* p, f32x4_t v) { *(FM_GLOBAL f32x4_t*)(p) = v; }
__device__ __forceinline__ f32x4_t load4(const bf16* p) {
  const u32x2_t w = *(const FM_GLOBAL u32x2_t*)(p);
  return f32x4_t{__uint_as_float(w[0] << 16), __uint_as_float(w[0] & 0xFFFF0000u),
                 __uint_as_float(w[1] << 16), __uint_as_float(w[1] & 0xFFFF0000u)};
}
__device__ __forceinline__ f32x4_t load4(const float* p) { return *(const FM_GLOBAL f32x4_t*)(p); }

}  // namespace fm
