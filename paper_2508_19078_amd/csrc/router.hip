// Router (softmax top-k gate), int8 router quantiser and the activation
// histogram of the int8 profiling router.
//
// One kernel family serves both the full-precision router and the int8
// profiling router: a block accumulates the logits of a tile of tokens against
// every expert on MFMA.  For bf16 activations with at most 64 experts and d a
// multiple of 256 the operands stream through an LDS ring: k_route_p keeps one
// persistent block per compute unit walking 32-token tiles (64-token tiles once
// every compute unit gets one) and issues the next tile's first slabs before
// the current tile's selection; k_route_lds, one 32-token tile per block, is
// kept for the int8 histogram at smaller T, where it measured faster.
// Otherwise (fp32, wider routers) the waves split the hidden dimension into
// 16-byte-per-lane register chunks (k_route).  The waves' partial sums are
// added in a fixed order, so the logits do not depend on scheduling.  Then 16
// lanes per token select the top k by (logit desc, index asc) with branch-free
// 64-bit key reductions, and either write idx/gate or add the selection to an
// LDS histogram that is flushed to the global counts with one integer atomic
// per expert and block.
#include "common.hpp"
#include "gemm_bf16.hpp"

namespace fm {
namespace {

constexpr int RT_TOK = 32;      // tokens per block
constexpr int RT_GROUPS = 4;    // partial sums reduced in RT_GROUPS fixed-order groups
// Waves per block (splitting d) and chunks in flight per wave, by the number
// of 16-expert column tiles: as many loads in flight per CU as the
// accumulators leave registers for (about 200 KB for up to 64 experts).
template <int NE> struct RtShape {
  static constexpr int WAVES = NE <= 4 ? 16 : NE <= 8 ? 8 : 4;
  static constexpr int P = NE <= 2 ? 4 : NE <= 8 ? 2 : 1;
};

template <int N> struct fragv;
template <> struct fragv<8> { typedef bf16x8_t type; };   // 8 bf16 per lane
template <> struct fragv<4> { typedef f32x4_t type; };    // 4 fp32 per lane

// A-operand fragment of X: 16 bytes of one row.
__device__ __forceinline__ bf16x8_t load_x_frag(const bf16* p, bool ok) {
  u32x4_t v = ok ? ld16(p) : u32x4_t{0, 0, 0, 0};
  return __builtin_bit_cast(bf16x8_t, v);
}
__device__ __forceinline__ f32x4_t load_x_frag(const float* p, bool ok) {
  u32x4_t v = ok ? ld16(p) : u32x4_t{0, 0, 0, 0};
  return __builtin_bit_cast(f32x4_t, v);
}

// B-operand fragment of the router weight, same element count as X's.
__device__ __forceinline__ bf16x8_t load_w_frag(const bf16* p, bool ok, bf16x8_t) {
  return load_x_frag(p, ok);
}
__device__ __forceinline__ f32x4_t load_w_frag(const float* p, bool ok, f32x4_t) {
  return load_x_frag(p, ok);
}
// int8 codes widened exactly to bf16 (|q| <= 127 has at most 7 significant bits).
__device__ __forceinline__ bf16x8_t load_w_frag(const int8_t* p, bool ok, bf16x8_t) {
  u32x2_t raw = ok ? *(const FM_GLOBAL u32x2_t*)(p) : u32x2_t{0, 0};
  u32x4_t v;
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    uint32_t w = i < 2 ? raw[0] : raw[1];
    int sh = (i & 1) * 16;
    float lo = (float)(int8_t)((w >> sh) & 0xFF);
    float hi = (float)(int8_t)((w >> (sh + 8)) & 0xFF);
    v[i] = (__float_as_uint(lo) >> 16) | (__float_as_uint(hi) & 0xFFFF0000u);
  }
  return __builtin_bit_cast(bf16x8_t, v);
}
__device__ __forceinline__ f32x4_t load_w_frag(const int8_t* p, bool ok, f32x4_t) {
  uint32_t raw = ok ? *(const FM_GLOBAL uint32_t*)(p) : 0u;
  f32x4_t v;
#pragma unroll
  for (int i = 0; i < 4; ++i) v[i] = (float)(int8_t)((raw >> (8 * i)) & 0xFF);
  return v;
}

// Order-preserving map of a finite fp32 (with -0.0 folded into +0.0 by the
// caller) to uint32, and its inverse.
__device__ __forceinline__ uint32_t ordered_key(float v) {
  const uint32_t u = __float_as_uint(v);
  return (u & 0x80000000u) ? ~u : (u | 0x80000000u);
}
__device__ __forceinline__ float key_value(uint32_t k) {
  return __uint_as_float((k & 0x80000000u) ? (k & 0x7FFFFFFFu) : ~k);
}
// Rotation of a value within each row of 16 lanes (DPP row_ror).
template <int N> __device__ __forceinline__ uint32_t row_ror_u(uint32_t x) {
  return (uint32_t)__builtin_amdgcn_update_dpp(0, (int)x, 0x120 + N, 0xF, 0xF, false);
}
template <int N> __device__ __forceinline__ float row_ror(float x) {
  return __uint_as_float(row_ror_u<N>(__float_as_uint(x)));
}
// (hi, lo) <- max((hi, lo), rotated (hi, lo)) as a 64-bit key.
template <int N> __device__ __forceinline__ void key_max_row(uint32_t& hi, uint32_t& lo) {
  const uint32_t h2 = row_ror_u<N>(hi), l2 = row_ror_u<N>(lo);
  const bool tk = h2 > hi || (h2 == hi && l2 > lo);
  hi = tk ? h2 : hi;
  lo = tk ? l2 : lo;
}

// acc (16x16 tile) += A(16 x kc) * B(kc x 16)
__device__ __forceinline__ f32x4_t mma(bf16x8_t a, bf16x8_t b, f32x4_t c) {
  return __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, b, c, 0, 0, 0);
}
__device__ __forceinline__ f32x4_t mma(f32x4_t a, f32x4_t b, f32x4_t c) {
#pragma unroll
  for (int i = 0; i < 4; ++i) c = __builtin_amdgcn_mfma_f32_16x16x4f32(a[i], b[i], c, 0, 0, 0);
  return c;
}

// Top-k selection and outputs for the block's RT_TOK tokens starting at t0,
// WAVES waves.  The logit of (token tl, expert e) is the sum, in order, of
// NPART partials part[p * PSTRIDE + tl * EP + e], times scale[e] and plus
// bias[e] when those are given (LDS arrays); with logits != nullptr (MODE 0)
// the logits are also written out.
//
// 16 lanes per token: lane gl of the group holds experts gl, gl+16, ...  Keys
// order (value desc, index asc): the high word maps the fp32 value
// monotonically to uint32 (-0.0 == +0.0), the low word is 0xFFFF - expert.
// Each of the k selection rounds takes the group maximum with four DPP row
// rotations; the owner lane then drops it.  A group handles TPL tokens at once
// (independent chains for the scheduler to interleave).
// TT tokens (RT_TOK by default).  With FLUSH the LDS histogram is added to the
// global counts at the end (MODE != 0); a persistent kernel passes false and
// flushes once after its last tile.
template <int NE, int KMAX, int MODE, int WAVES, int NPART, int TT = RT_TOK, bool FLUSH = true>
__device__ __forceinline__ void route_select(const float* part, int PSTRIDE, int EP, const float* scale,
                                             const float* bias, int t0, int T, int E, int k,
                                             int32_t* __restrict__ idx, float* __restrict__ gate,
                                             float* __restrict__ logits, int32_t* __restrict__ counts,
                                             int* hist) {
  constexpr int RT_TOK = TT;
  constexpr int TPL = (RT_TOK + WAVES * 4 - 1) / (WAVES * 4);
  const int lane = lane_id();
  const int wave = threadIdx.x >> 6;
  const int grp = lane >> 4, gl = lane & 15;
  uint32_t khi[TPL][NE], klo[TPL][NE];
  int tl[TPL];
#pragma unroll
  for (int u = 0; u < TPL; ++u) {
    tl[u] = u * WAVES * 4 + wave * 4 + grp;
    const bool on = tl[u] < RT_TOK;
    const int tc = on ? tl[u] : 0;
#pragma unroll
    for (int i = 0; i < NE; ++i) {
      const int e = gl + 16 * i;
      float v = 0.f;
      if (e < E) {
        v = part[tc * EP + e];
#pragma unroll
        for (int p = 1; p < NPART; ++p) v += part[p * PSTRIDE + tc * EP + e];
        if (scale) v *= scale[e];
        if (bias) v += bias[e];
        if (MODE == 0 && logits && on && t0 + tc < T) logits[(size_t)(t0 + tc) * E + e] = v;
      }
      v += 0.0f;
      khi[u][i] = (on && e < E) ? ordered_key(v) : 0u;
      klo[u][i] = (on && e < E) ? 0xFFFFu - (uint32_t)e : 0u;
    }
  }
  float myv[TPL], v0[TPL];
  int mye[TPL];
#pragma unroll
  for (int u = 0; u < TPL; ++u) {
    myv[u] = 0.f;
    v0[u] = 0.f;
    mye[u] = 0;
  }
#pragma unroll
  for (int j = 0; j < KMAX; ++j) {
    if (j < k) {
#pragma unroll
      for (int u = 0; u < TPL; ++u) {
        uint32_t bh = khi[u][0], bl = klo[u][0];
#pragma unroll
        for (int i = 1; i < NE; ++i) {
          const bool tk = khi[u][i] > bh || (khi[u][i] == bh && klo[u][i] > bl);
          bh = tk ? khi[u][i] : bh;
          bl = tk ? klo[u][i] : bl;
        }
        key_max_row<8>(bh, bl);
        key_max_row<4>(bh, bl);
        key_max_row<2>(bh, bl);
        key_max_row<1>(bh, bl);
        const int e = 0xFFFF - (int)bl;
        const float v = key_value(bh);
        if (j == 0) v0[u] = v;
        if (gl == j) {
          myv[u] = v;
          mye[u] = e;
        }
#pragma unroll
        for (int i = 0; i < NE; ++i)
          if (gl + 16 * i == e) {
            khi[u][i] = 0u;
            klo[u][i] = 0u;
          }
      }
    }
  }
#pragma unroll
  for (int u = 0; u < TPL; ++u) {
    const int t = t0 + tl[u];
    const bool mine = gl < k && tl[u] < RT_TOK && t < T;
    if (MODE != 1) {                 // idx and the softmax gate over the k selected
      float g = gl < k ? expf(myv[u] - v0[u]) : 0.f;
      float sum = g;
      sum += row_ror<8>(sum);
      sum += row_ror<4>(sum);
      sum += row_ror<2>(sum);
      sum += row_ror<1>(sum);
      if (mine) {
        idx[(size_t)t * k + gl] = mye[u];
        gate[(size_t)t * k + gl] = g / sum;
      }
    }
    if (MODE != 0 && mine) {         // histogram (+ idx alone in MODE 1)
      atomicAdd(&hist[mye[u]], 1);
      if (MODE == 1 && idx) idx[(size_t)t * k + gl] = mye[u];
    }
  }
  if (MODE != 0 && FLUSH) {
    __syncthreads();
    for (int e = threadIdx.x; e < E; e += blockDim.x)
      if (hist[e]) atomicAdd(&counts[e], hist[e]);
  }
}

// Selection in small lane groups, for the logits of TT tokens in LDS (the sum,
// in order, of NPART partials stage[p * PSTRIDE + token * EP + expert], times
// scale and plus bias as in route_select).  LPT = 2, 4 or 8 lanes per token;
// lane q of a group holds experts [q NQ, (q+1) NQ) as 64-bit keys (ordered
// fp32 value, 0xFFFF - expert; -0.0 == +0.0), so that a selection round is a
// local maximum over the lane's NQ keys (a tree of independent compares) and
// log2(LPT) lane exchanges (DPP quad permutations, then a swizzle across
// quads), and the k rounds of a token run in one lane group with no loop over
// tokens (16 lanes per token and one token after another left each round a
// chain of dependent row rotations that one wave per SIMD could not hide).
// Rank j of a token lands in lane j % LPT of its group.  The selected experts
// and their order are those of route_select; the softmax denominator adds
// each lane's ranks in order, then the group's lanes by the same exchanges
// (so a gate may differ from route_select's in its last bit).
template <int CTRL> __device__ __forceinline__ uint64_t quad_perm64(uint64_t x) {
  const uint32_t lo = (uint32_t)__builtin_amdgcn_update_dpp(0, (int)(uint32_t)x, CTRL, 0xF, 0xF, false);
  const uint32_t hi = (uint32_t)__builtin_amdgcn_update_dpp(0, (int)(uint32_t)(x >> 32), CTRL, 0xF, 0xF, false);
  return ((uint64_t)hi << 32) | lo;
}
template <int CTRL> __device__ __forceinline__ float quad_perm_f(float x) {
  return __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(x), CTRL, 0xF, 0xF, false));
}
constexpr int QP_SWAP1 = 0xB1;   // quad_perm [1, 0, 3, 2]
constexpr int QP_SWAP2 = 0x4E;   // quad_perm [2, 3, 0, 1]

template <int LPT> __device__ __forceinline__ uint64_t group_max64(uint64_t b) {
  uint64_t o = quad_perm64<QP_SWAP1>(b);
  b = o > b ? o : b;
  if (LPT == 2) return b;
  o = quad_perm64<QP_SWAP2>(b);
  b = o > b ? o : b;
  if (LPT == 8) {
    const uint32_t lo = (uint32_t)__shfl_xor((int)(uint32_t)b, 4);
    const uint32_t hi = (uint32_t)__shfl_xor((int)(uint32_t)(b >> 32), 4);
    o = ((uint64_t)hi << 32) | lo;
    b = o > b ? o : b;
  }
  return b;
}
template <int LPT> __device__ __forceinline__ float group_sum(float x) {
  x += quad_perm_f<QP_SWAP1>(x);
  if (LPT == 2) return x;
  x += quad_perm_f<QP_SWAP2>(x);
  if (LPT == 8) x += __shfl_xor(x, 4);
  return x;
}

template <int LPT, int NQ, int KMAX, int MODE, int WAVES, int TT, int NPART = 1>
__device__ __forceinline__ void route_select_q(const float* stage, int PSTRIDE, int EP, const float* scale,
                                               const float* bias,
                                               int t0, int T, int E, int k, int32_t* __restrict__ idx,
                                               float* __restrict__ gate, float* __restrict__ logits,
                                               int* hist) {
  static_assert(LPT == 2 || LPT == 4 || LPT == 8, "2, 4 or 8 lanes per token");
  constexpr int GPW = 64 / LPT;                                 // lane groups per wave
  constexpr int TPL = (TT + WAVES * GPW - 1) / (WAVES * GPW);   // tokens per lane group
  constexpr int RPL = (KMAX + LPT - 1) / LPT;                   // ranks held per lane
  const int lane = lane_id(), wave = threadIdx.x >> 6;
  const int grp = lane / LPT, q = lane % LPT;
#pragma unroll
  for (int u = 0; u < TPL; ++u) {
    const int tl = u * WAVES * GPW + wave * GPW + grp;
    const bool on = tl < TT;
    const int tc = on ? tl : 0;
    uint64_t key[NQ];
#pragma unroll
    for (int i = 0; i < NQ; ++i) {
      const int e = q * NQ + i;
      float v = 0.f;
      if (e < E) {
        v = stage[tc * EP + e];
#pragma unroll
        for (int p = 1; p < NPART; ++p) v += stage[p * PSTRIDE + tc * EP + e];
        if (scale) v *= scale[e];
        if (bias) v += bias[e];
        if (MODE == 0 && logits && on && t0 + tc < T) logits[(size_t)(t0 + tc) * E + e] = v;
      }
      v += 0.0f;
      key[i] = (on && e < E) ? (((uint64_t)ordered_key(v) << 32) | (uint64_t)(0xFFFFu - (uint32_t)e)) : 0ull;
    }
    float rv[RPL], v0 = 0.f;
    int re[RPL];
#pragma unroll
    for (int r = 0; r < RPL; ++r) {
      rv[r] = 0.f;
      re[r] = 0;
    }
#pragma unroll
    for (int j = 0; j < KMAX; ++j) {
      if (j < k) {
        uint64_t m[NQ];
#pragma unroll
        for (int i = 0; i < NQ; ++i) m[i] = key[i];
#pragma unroll
        for (int w = NQ / 2; w > 0; w >>= 1)
#pragma unroll
          for (int i = 0; i < w; ++i) m[i] = m[i + w] > m[i] ? m[i + w] : m[i];
        const uint64_t b = group_max64<LPT>(m[0]);
        const int e = 0xFFFF - (int)(uint32_t)(b & 0xFFFFu);
        const float v = key_value((uint32_t)(b >> 32));
        if (j == 0) v0 = v;
        if (q == j % LPT) {
          rv[j / LPT] = v;
          re[j / LPT] = e;
        }
#pragma unroll
        for (int i = 0; i < NQ; ++i)
          if (q * NQ + i == e) key[i] = 0ull;
      }
    }
    const int t = t0 + tl;
    if (MODE != 1) {                 // idx and the softmax gate over the k selected
      float g[RPL], sum = 0.f;
#pragma unroll
      for (int r = 0; r < RPL; ++r) {
        g[r] = LPT * r + q < k ? expf(rv[r] - v0) : 0.f;
        sum += g[r];
      }
      sum = group_sum<LPT>(sum);
#pragma unroll
      for (int r = 0; r < RPL; ++r) {
        const int j = LPT * r + q;
        if (j < k && on && t < T) {
          idx[(size_t)t * k + j] = re[r];
          gate[(size_t)t * k + j] = g[r] / sum;
        }
      }
    }
    if (MODE != 0) {                 // histogram (+ idx alone in MODE 1)
#pragma unroll
      for (int r = 0; r < RPL; ++r) {
        const int j = LPT * r + q;
        if (j < k && on && t < T) {
          atomicAdd(&hist[re[r]], 1);
          if (MODE == 1 && idx) idx[(size_t)t * k + j] = re[r];
        }
      }
    }
  }
}

// MODE 0: write idx/gate (+logits).  MODE 1: histogram (+idx).  MODE 2:
// histogram, idx and gate.
template <typename TX, typename TW, int NE, int KMAX, int MODE>
__global__ __launch_bounds__(RtShape<NE>::WAVES * 64) void k_route(
    const TX* __restrict__ X, const TW* __restrict__ W, const float* __restrict__ wscale,
    const float* __restrict__ bias, int T, int d, int E, int k,
    int32_t* __restrict__ idx, float* __restrict__ gate, float* __restrict__ logits,
    int32_t* __restrict__ counts) {
  constexpr int V = 16 / sizeof(TX);           // elements per lane per chunk
  constexpr int KC = 4 * V;                    // hidden columns per chunk
  constexpr int EP = NE * 16 + 1;              // padded LDS row
  constexpr int RT_WAVES = RtShape<NE>::WAVES;
  typedef typename fragv<V>::type frag_t;
  __shared__ float red[RT_GROUPS][RT_TOK * EP];
  __shared__ int hist[NE * 16];

  const int lane = lane_id();
  const int wave = threadIdx.x >> 6;
  const int t0 = blockIdx.x * RT_TOK;
  const int r16 = lane & 15, q4 = lane >> 4;

  if (MODE != 0)
    for (int e = threadIdx.x; e < NE * 16; e += blockDim.x) hist[e] = 0;

  f32x4_t acc[2][NE];
#pragma unroll
  for (int r = 0; r < 2; ++r)
#pragma unroll
    for (int j = 0; j < NE; ++j) acc[r][j] = f32x4_t{0, 0, 0, 0};

  const int nchunks = d / KC;
  const int tail = d - nchunks * KC;           // multiple of 8 (d % 8 == 0)
  // Rows past T and experts past E read a clamped (valid) row: their logits
  // are never used, so the main loop needs no predicated loads.
  const TX* xrow[2];
#pragma unroll
  for (int r = 0; r < 2; ++r) xrow[r] = X + (size_t)min(t0 + r * 16 + r16, T - 1) * d;
  const TW* wrow[NE];
#pragma unroll
  for (int j = 0; j < NE; ++j) wrow[j] = W + (size_t)min(j * 16 + r16, E - 1) * d;

  // Chunks go in pairs: chunks 2u and 2u + 1 are the two 64-byte halves of
  // the same 128-byte lines of every row, and their loads are issued back to
  // back (the CU moves about twice the bytes per clock from L2 that way).
  // This wave's pairs are wave, wave + RT_WAVES, ...; PU of them in flight.
  constexpr int PU = RtShape<NE>::P > 1 ? RtShape<NE>::P / 2 : 1;
  const int npairs = nchunks / 2;
  const int nw = npairs > wave ? (npairs - wave + RT_WAVES - 1) / RT_WAVES : 0;
  frag_t ra[PU][2][2], rb[PU][2][NE];
  auto issue = [&](int u, int i) {
    const int pi = min(i, nw - 1);
    const int col = (wave + RT_WAVES * pi) * 2 * KC + q4 * V;
#pragma unroll
    for (int r = 0; r < 2; ++r) {
      ra[u][0][r] = load_x_frag(xrow[r] + col, true);
      ra[u][1][r] = load_x_frag(xrow[r] + col + KC, true);
    }
#pragma unroll
    for (int j = 0; j < NE; ++j) {
      rb[u][0][j] = load_w_frag(wrow[j] + col, true, frag_t{});
      rb[u][1][j] = load_w_frag(wrow[j] + col + KC, true, frag_t{});
    }
  };
  if (nw > 0) {
#pragma unroll
    for (int u = 0; u < PU; ++u) issue(u, u);
    for (int i0 = 0; i0 < nw; i0 += PU) {
#pragma unroll
      for (int u = 0; u < PU; ++u) {
        if (i0 + u < nw) {
#pragma unroll
          for (int h = 0; h < 2; ++h)
#pragma unroll
            for (int r = 0; r < 2; ++r)
#pragma unroll
              for (int j = 0; j < NE; ++j) acc[r][j] = mma(ra[u][h][r], rb[u][h][j], acc[r][j]);
        }
        issue(u, i0 + u + PU);
      }
    }
  }
  // An odd last whole chunk and the zero-filled partial chunk, if any, go to
  // the wave next in the round-robin.
  if (wave == npairs % RT_WAVES) {
    for (int c = 2 * npairs; c < nchunks + (tail > 0); ++c) {
      const int col = c * KC + q4 * V;
      const bool cok = col < d;
      frag_t a[2], b[NE];
#pragma unroll
      for (int r = 0; r < 2; ++r) a[r] = load_x_frag(xrow[r] + col, cok);
#pragma unroll
      for (int j = 0; j < NE; ++j) b[j] = load_w_frag(wrow[j] + col, cok, frag_t{});
#pragma unroll
      for (int r = 0; r < 2; ++r)
#pragma unroll
        for (int j = 0; j < NE; ++j) acc[r][j] = mma(a[r], b[j], acc[r][j]);
    }
  }

  // Fixed-order reduction of the partial sums: group g adds waves
  // g, g + 4, g + 8, g + 12 in that order, then g0 + g1 + g2 + g3.
  constexpr int PER_GROUP = RT_WAVES / RT_GROUPS;
  const int grp_id = wave % RT_GROUPS;
  for (int step = 0; step < PER_GROUP; ++step) {
    if (wave / RT_GROUPS == step) {
#pragma unroll
      for (int r = 0; r < 2; ++r)
#pragma unroll
        for (int j = 0; j < NE; ++j)
#pragma unroll
          for (int i = 0; i < 4; ++i) {
            // MFMA output: row (token) 4*q4 + i, column (expert) r16
            float* p = &red[grp_id][(r * 16 + 4 * q4 + i) * EP + j * 16 + r16];
            *p = (step == 0) ? acc[r][j][i] : *p + acc[r][j][i];
          }
    }
    __syncthreads();
  }

  // finalise logits: sum of the groups, scale (int8 router) and bias
  for (int i = threadIdx.x; i < RT_TOK * E; i += blockDim.x) {
    int tl = i / E, e = i - tl * E;
    float v = red[0][tl * EP + e];
#pragma unroll
    for (int g = 1; g < RT_GROUPS; ++g) v += red[g][tl * EP + e];
    if (wscale) v *= wscale[e];
    if (bias) v += bias[e];
    red[0][tl * EP + e] = v;
    if (MODE == 0 && logits && t0 + tl < T) logits[(size_t)(t0 + tl) * E + e] = v;
  }
  __syncthreads();

  route_select<NE, KMAX, MODE, RT_WAVES, 1>(red[0], 0, EP, nullptr, nullptr, t0, T, E, k, idx, gate, nullptr,
                                           counts, hist);
}

// The same router for bf16 activations with E <= 64 and d a multiple of 256,
// with its operands staged through LDS: every block needs all of W for its 32
// tokens, which makes the per-CU load path (not HBM) the limit of the
// register-fed kernel above.  Slabs of 256 columns of the block's 32 X rows
// and of W's rows move global -> LDS with global_load_lds_dwordx4, each
// instruction 64 bytes of 16 rows and the same wave's next one the other
// halves of those lines (the pairing that doubles the CU's L2 -> LDS rate),
// chunk index XOR-swizzled by (row >> 2) & 3; a ring of three slabs, two in
// flight.  Wave w multiplies columns [64 w, 64 w + 64) of each slab with
// v_mfma_f32_32x32x16_bf16 (int8 W widened exactly to bf16 on the way in);
// the four partial sums are added in wave order.
template <typename TW> struct RtLds;
template <> struct RtLds<bf16> {
  static constexpr int WB = 512;                     // bytes of a W row per slab
  static __device__ __forceinline__ bf16x8_t frag(const FM_LDS char* blk, int rr, int w, int cc) {
    // line w, chunk cc of the row
    const int h = cc >> 2, q = cc & 3;
    return *(const FM_LDS bf16x8_t*)(blk + ((w * 2 + h) * 1024) + rr * 64 + ((q ^ ((rr >> 2) & 3)) << 4));
  }
};
template <> struct RtLds<int8_t> {
  static constexpr int WB = 256;
  static __device__ __forceinline__ bf16x8_t frag(const FM_LDS char* blk, int rr, int w, int cc) {
    // columns 64 w + 8 cc .. +8 are bytes 64 w + 8 cc of the 256-byte row:
    // line w / 2, half w % 2, 16-byte chunk cc / 2, 8 bytes at (cc % 2) * 8
    const int q = cc >> 1;
    const u32x2_t raw = *(const FM_LDS u32x2_t*)(blk + (((w >> 1) * 2 + (w & 1)) * 1024) + rr * 64 +
                                                 ((q ^ ((rr >> 2) & 3)) << 4) + (cc & 1) * 8);
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
};

constexpr int RL_COLS = 256, RL_XB = 512, RL_NS = 3;

template <typename TW, int NB, int KMAX, int MODE>
__global__ __launch_bounds__(256) void k_route_lds(const bf16* __restrict__ X, const TW* __restrict__ W,
                                                   const float* __restrict__ wscale, const float* __restrict__ bias,
                                                   int T, int d, int E, int k, int32_t* __restrict__ idx,
                                                   float* __restrict__ gate, float* __restrict__ logits,
                                                   int32_t* __restrict__ counts) {
  constexpr int WB = RtLds<TW>::WB;
  constexpr int WLINES = WB / 128;                   // 128-byte lines of a W row per slab
  constexpr int XBYTES = RT_TOK * RL_XB;             // 16 KB
  constexpr int SLAB = XBYTES + NB * 32 * WB;
  constexpr int NIX = 2 * 4 * 2;                     // X: 2 row groups x 4 lines x 2 halves
  constexpr int NIW = 2 * NB * WLINES * 2;           // W: 2 NB row groups x lines x 2 halves
  constexpr int INS = (NIX + NIW) / 4;               // DMA instructions per wave and slab
  static_assert((NIX + NIW) % 4 == 0, "whole instructions per wave");
  constexpr int EP = NB * 32 + 1;
  static_assert(RL_NS * SLAB <= 160 * 1024 && 4 * RT_TOK * EP * 4 <= RL_NS * SLAB, "LDS");
  __shared__ __align__(1024) char lds_raw[RL_NS * SLAB];
  __shared__ int hist[NB * 32];
  __shared__ float s_scale[NB * 32], s_bias[NB * 32];
  FM_LDS char* lds = (FM_LDS char*)lds_raw;
  const int lane = lane_id_here(), wave = wave_id();
  const int t0 = blockIdx.x * RT_TOK;
  if (MODE != 0)
    for (int e = threadIdx.x; e < NB * 32; e += blockDim.x) hist[e] = 0;
  // the epilogue's per-expert scale and bias, fetched while the slabs stream
  if (threadIdx.x < E) {
    s_scale[threadIdx.x] = wscale ? wscale[threadIdx.x] : 1.f;
    s_bias[threadIdx.x] = bias ? bias[threadIdx.x] : 0.f;
  }

  // DMA plan: instruction u = wave * INS + q; X instructions first.
  const char* gp[INS];
  uint32_t dst[INS];
#pragma unroll
  for (int q = 0; q < INS; ++q) {
    const int u = wave * INS + q;
    const int rr = lane >> 2;
    if (u < NIX) {
      const int g = u >> 3, m = (u >> 1) & 3, h = u & 1;
      const int row = min(t0 + g * 16 + rr, T - 1);
      gp[q] = (const char*)(X + (size_t)row * d) + m * 128 + h * 64 + (((lane & 3) ^ ((rr >> 2) & 3)) << 4);
      dst[q] = (uint32_t)(((g * 4 + m) * 2 + h) * 1024);
    } else {
      const int v = u - NIX, g = v / (WLINES * 2), m = (v >> 1) % WLINES, h = v & 1;
      const int row = min(g * 16 + rr, E - 1);
      gp[q] = (const char*)(W + (size_t)row * d) + m * 128 + h * 64 + (((lane & 3) ^ ((rr >> 2) & 3)) << 4);
      dst[q] = (uint32_t)(XBYTES + ((g * WLINES + m) * 2 + h) * 1024);
    }
  }
  const int nslab = d / RL_COLS;
  // Blocks start at different slabs (their rank within the XCD), so that the
  // CUs sharing an L2 do not all ask for the same lines of W at once.
  const int s_off = (int)(blockIdx.x >> 3) % nslab;
  auto issue = [&](int s) {
    FM_LDS char* slab = lds + (s % RL_NS) * SLAB;
    int sg = s + s_off;
    sg -= sg >= nslab ? nslab : 0;
#pragma unroll
    for (int q = 0; q < INS; ++q) {
      const bool isx = wave * INS + q < NIX;
      dma16(gp[q] + (size_t)sg * (isx ? RL_XB : WB), slab + dst[q]);
    }
  };
  f32x16_t acc[NB];
#pragma unroll
  for (int b = 0; b < NB; ++b)
#pragma unroll
    for (int r = 0; r < 16; ++r) acc[b][r] = 0.f;

  const int pre = min(RL_NS - 1, nslab);
  for (int s = 0; s < pre; ++s) issue(s);
  const int i = lane & 31, hf = lane >> 5;
  for (int s = 0; s < nslab; ++s) {
    if (s + 1 < nslab) wait_vmcnt<INS>();
    else wait_vmcnt<0>();
    barrier_lds();
    if (s + RL_NS - 1 < nslab) issue(s + RL_NS - 1);
    const FM_LDS char* slab = lds + (s % RL_NS) * SLAB;
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const int cc = 2 * j + hf;
      // X row i: group i >> 4, row i & 15 of that group's blocks
      const bf16x8_t xa = RtLds<bf16>::frag(slab + (i >> 4) * 8 * 1024, i & 15, wave, cc);
#pragma unroll
      for (int b = 0; b < NB; ++b) {
        const int R = 32 * b + i;
        const bf16x8_t wb = RtLds<TW>::frag(slab + XBYTES + (R >> 4) * WLINES * 2 * 1024, R & 15, wave, cc);
        acc[b] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(xa, wb, acc[b], 0, 0, 0);
      }
    }
  }
  __syncthreads();

  // partial sums of the four waves, added in wave order; then scale and bias.
  // Register r of lane L holds token 8 (r / 4) + 4 (L / 32) + r % 4, expert 32 b + L % 32.
  float* red = (float*)lds_raw;                      // [wave][token][EP]
  {
    const int L = lane_id();
#pragma unroll
    for (int b = 0; b < NB; ++b)
#pragma unroll
      for (int r = 0; r < 16; ++r)
        red[(wave * RT_TOK + 8 * (r >> 2) + 4 * (L >> 5) + (r & 3)) * EP + 32 * b + (L & 31)] = acc[b][r];
  }
  __syncthreads();
  // 8 lanes per token: the block's 256 lanes hold its 32 tokens
  route_select_q<8, NB * 32 / 8, KMAX, MODE, 4, RT_TOK, 4>(red, RT_TOK * EP, EP, wscale ? s_scale : nullptr,
                                                           bias ? s_bias : nullptr, t0, T, E, k, idx, gate, logits,
                                                           hist);
  if (MODE != 0) {
    __syncthreads();
    for (int e = threadIdx.x; e < E; e += blockDim.x)
      if (hist[e]) atomicAdd(&counts[e], hist[e]);
  }
}

// Persistent router for bf16 activations, E <= 64 and d a multiple of the slab
// width (256 columns for 32-token tiles, 128 for 64-token tiles).
// A block owns tiles of TT tokens (32, or 64 once every compute unit gets a
// whole 64-token tile) and walks tiles blockIdx.x, blockIdx.x + gridDim.x, ...
// Slabs of the tile's X rows and of the router's rows (padded to
// NEG * 32, rows past E clamped) stream global -> LDS through a ring of NS slabs
// with paired-half DMA (each instruction 64 bytes of 16 rows, the same wave's
// next one the other halves of those lines; 16-byte chunks XOR-swizzled by
// (row >> 2) & 3).  The four waves split the work as expert groups of 32 x
// NKS parts of each slab's eight 16-column k-steps; each wave keeps a 32 x 32
// accumulator per 32 tokens of the tile (v_mfma_f32_32x32x16_bf16), so every
// router fragment is read, and int8 codes widened exactly to bf16, by one wave
// only; the NKS partial sums meet in LDS in a fixed order.  With 64-token tiles each router row read from L2 serves twice
// the tokens.  Once a tile's last slab is read, the next tile's first NS - 1
// slabs are issued, and the selection of the finished tile (a separate LDS
// region) overlaps their latency.  The LDS histogram of MODE 1 and 2 is
// flushed to `counts` once, after the block's last tile.
template <typename TW> struct RpW;
template <> struct RpW<bf16> {
  static __device__ __forceinline__ bf16x8_t frag(const FM_LDS char* grp, int rr, int ks, int hf) {
    // columns 16 ks + 8 hf .. + 8 (bytes 32 ks + 16 hf of the 256-byte slab row)
    const int m = ks >> 2, h = (ks >> 1) & 1, q = ((ks & 1) << 1) | hf;
    return *(const FM_LDS bf16x8_t*)(grp + (m * 2 + h) * 1024 + rr * 64 + ((q ^ ((rr >> 2) & 3)) << 4));
  }
};
template <> struct RpW<int8_t> {
  static __device__ __forceinline__ bf16x8_t frag(const FM_LDS char* grp, int rr, int ks, int hf) {
    // codes 16 ks + 8 hf .. + 8: bytes 16 ks + 8 hf of the slab row (line ks / 8)
    const int m = ks >> 3, h = (ks >> 2) & 1, q = ks & 3;
    const u32x2_t raw =
        *(const FM_LDS u32x2_t*)(grp + (m * 2 + h) * 1024 + rr * 64 + ((q ^ ((rr >> 2) & 3)) << 4) + hf * 8);
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
};

// Slabs of COLS hidden columns: 256 for 32-token tiles (half the slab steps),
// 128 for 64- and 128-token tiles (measured faster than 256 with int8 codes,
// and a 256-column bf16 slab would leave room for two in the ring).  The selection's
// staging area lives in ring slot NS - 1, which is free while the next tile's
// first NS - 1 slabs land.
template <typename TW, int TT, int NEG> struct RpCfg {
  static constexpr int COLS = TT == 32 ? 256 : 128;
  static constexpr int NTG = TT / 32;                          // token groups (accumulators per wave)
  static constexpr int NKS = 4 / NEG;                          // parts of a slab's k-steps
  static constexpr int KSTEPS = COLS / 16;                     // 16-column MFMA k-steps per slab
  static constexpr int KSP = KSTEPS / NKS;                     // k-steps per part
  static constexpr int XROW = COLS * 2;                        // bytes of an X row per slab
  static constexpr int WB = COLS * (int)sizeof(TW);            // bytes of a router row per slab
  static constexpr int XLINES = XROW / 128, WLINES = WB / 128; // 128-byte lines per slab row
  static constexpr int XBYTES = TT * XROW;
  static constexpr int SLAB = XBYTES + NEG * 32 * WB;
  static constexpr int NIX = (TT / 16) * XLINES * 2;           // X: row groups x lines x halves
  static constexpr int NIW = NEG * 2 * WLINES * 2;             // W: row groups x lines x halves
  static constexpr int INS = (NIX + NIW) / 4;                  // DMA instructions per wave and slab
  static constexpr int EP = NEG * 32 + 1;                      // padded logit row
  static constexpr int STAGE = TT * EP * 4;
  static constexpr int NS0 = (159 * 1024) / SLAB;
  static constexpr int NS = NS0 > 6 ? 6 : NS0;                 // ring depth
  static_assert(NEG * NKS == 4 && (NIX + NIW) % 4 == 0 && NS >= 3, "router tile");
  static_assert(STAGE <= SLAB && NS * SLAB + 3 * NEG * 32 * 4 <= 160 * 1024, "LDS");
  static_assert((NS - 2) * INS < 64, "vmcnt range");
};

template <int N> __device__ __forceinline__ void wait_vm_upto(int n) {
  // s_waitcnt vmcnt(n * N) for a small runtime n (0..5)
  switch (n) {
    case 0: wait_vmcnt<0>(); break;
    case 1: wait_vmcnt<N>(); break;
    case 2: wait_vmcnt<2 * N>(); break;
    case 3: wait_vmcnt<3 * N>(); break;
    case 4: wait_vmcnt<4 * N>(); break;
    default: wait_vmcnt<5 * N>(); break;
  }
}

template <typename TW, int TT, int NEG, int KMAX, int MODE>
__global__ __launch_bounds__(256) void k_route_p(const bf16* __restrict__ X, const TW* __restrict__ W,
                                                 const float* __restrict__ wscale, const float* __restrict__ bias,
                                                 int T, int d, int E, int k, int32_t* __restrict__ idx,
                                                 float* __restrict__ gate, float* __restrict__ logits,
                                                 int32_t* __restrict__ counts) {
  using C = RpCfg<TW, TT, NEG>;
  constexpr int NS = C::NS, INS = C::INS, EP = C::EP;
  __shared__ __align__(1024) char lds_raw[NS * C::SLAB];
  float* const stage = (float*)(lds_raw + (NS - 1) * C::SLAB);   // ring slot NS - 1
  __shared__ int hist[NEG * 32];
  __shared__ float s_scale[NEG * 32], s_bias[NEG * 32];
  FM_LDS char* ring = (FM_LDS char*)lds_raw;
  const int lane = lane_id_here(), wave = wave_id();
  const int ntiles = (T + TT - 1) / TT;
  if (MODE != 0)
    for (int e = threadIdx.x; e < NEG * 32; e += blockDim.x) hist[e] = 0;
  if (threadIdx.x < E) {
    s_scale[threadIdx.x] = wscale ? wscale[threadIdx.x] : 1.f;
    s_bias[threadIdx.x] = bias ? bias[threadIdx.x] : 0.f;
  }
  // This wave's DMA instructions: u = wave * INS + q, X ones first.  Per lane:
  // the row within the 16-row group and the swizzled 16-byte chunk.
  const int rr = lane >> 2;
  const uint32_t cb = (uint32_t)(((lane & 3) ^ ((rr >> 2) & 3)) << 4);
  const char* gp[INS];
  uint32_t dst[INS];
  bool isx[INS];
  const int nslab = d / C::COLS;
  auto plan = [&](int t0) {
#pragma unroll
    for (int q = 0; q < INS; ++q) {
      const int u = wave * INS + q;
      isx[q] = u < C::NIX;
      if (u < C::NIX) {
        const int h = u & 1, m = (u >> 1) % C::XLINES, g = (u >> 1) / C::XLINES;
        const int row = min(t0 + g * 16 + rr, T - 1);
        gp[q] = (const char*)(X + (size_t)row * d) + m * 128 + h * 64 + cb;
        dst[q] = (uint32_t)(((g * C::XLINES + m) * 2 + h) * 1024);
      } else {
        const int v = u - C::NIX, h = v & 1, m = (v >> 1) % C::WLINES, g = (v >> 1) / C::WLINES;
        const int row = min(g * 16 + rr, E - 1);
        gp[q] = (const char*)(W + (size_t)row * d) + m * 128 + h * 64 + cb;
        dst[q] = (uint32_t)(C::XBYTES + ((g * C::WLINES + m) * 2 + h) * 1024);
      }
    }
  };
  // Blocks of one XCD start at different slabs (their rank within the XCD), so
  // that the CUs sharing an L2 do not all ask for the same router lines at once.
  const int s_off = (int)(blockIdx.x >> 3) % nslab;
  auto issue = [&](int s) {
    FM_LDS char* slab = ring + (s % NS) * C::SLAB;
    int sg = s + s_off;
    sg -= sg >= nslab ? nslab : 0;
#pragma unroll
    for (int q = 0; q < INS; ++q) dma16(gp[q] + (size_t)sg * (isx[q] ? C::XROW : C::WB), slab + dst[q]);
  };
  // this wave's share: an expert group and a part of every slab's k-steps, for
  // all TT tokens (NTG accumulators), so that every router fragment is read,
  // and for int8 widened, by one wave only
  const int eg = wave % NEG, kp = wave / NEG;
  const int i = lane & 31, hf = lane >> 5;
  const int wr = eg * 32 + i;

  int tile = blockIdx.x;
  if (tile < ntiles) {
    plan(tile * TT);
    for (int s = 0; s < NS - 1 && s < nslab; ++s) issue(s);
  }
  bool first = true;
  while (tile < ntiles) {
    const int t0 = tile * TT;
    // two independent accumulator chains per wave (token groups, or even and
    // odd k-steps of a single token group), so consecutive MFMAs do not wait on
    // each other's results
    constexpr int NCH = C::NTG == 1 ? 2 : 1;
    f32x16_t acc[C::NTG][NCH];
#pragma unroll
    for (int g = 0; g < C::NTG; ++g)
#pragma unroll
      for (int c = 0; c < NCH; ++c)
#pragma unroll
        for (int r = 0; r < 16; ++r) acc[g][c][r] = 0.f;
    for (int s = 0; s < nslab; ++s) {
      // slabs issued after s and possibly still in flight: min(NS - 2, nslab - 1 - s);
      // the first slab of a later tile also waits for the epilogue's stores
      const int after = min(NS - 2, nslab - 1 - s);
      if (s == 0 && !first) wait_vmcnt<0>();
      else wait_vm_upto<INS>(after);
      barrier_lds();
      const FM_LDS char* slab = ring + (s % NS) * C::SLAB;
      const FM_LDS char* wg = slab + C::XBYTES + (wr >> 4) * C::WLINES * 2 * 1024;
      // all of this part's fragments are requested at once, then the refill is
      // issued while they land, then the MFMAs run (they retire while the wave
      // waits for the next slab)
      bf16x8_t xa[C::KSP][C::NTG], wb[C::KSP];
#pragma unroll
      for (int j = 0; j < C::KSP; ++j) {
        const int ks = kp * C::KSP + j;
        wb[j] = RpW<TW>::frag(wg, wr & 15, ks, hf);
#pragma unroll
        for (int g = 0; g < C::NTG; ++g) {
          const int xr = g * 32 + i;
          xa[j][g] = RpW<bf16>::frag(slab + (xr >> 4) * C::XLINES * 2 * 1024, xr & 15, ks, hf);
        }
      }
      sched_fence();
      if (s + NS - 1 < nslab) issue(s + NS - 1);
      sched_fence();
#pragma unroll
      for (int j = 0; j < C::KSP; ++j)
#pragma unroll
        for (int g = 0; g < C::NTG; ++g)
          acc[g][j % NCH] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(xa[j][g], wb[j], acc[g][j % NCH], 0, 0, 0);
    }
    if (NCH == 2)
#pragma unroll
      for (int g = 0; g < C::NTG; ++g) acc[g][0] += acc[g][NCH - 1];
    first = false;
    // every wave is done with the ring: start the next tile's first slabs
    barrier_lds();
    const int next = tile + gridDim.x;
    if (next < ntiles) {
      plan(next * TT);
      for (int s = 0; s < NS - 1 && s < nslab; ++s) issue(s);
    }
    // the parts' partial sums meet in the stage, the last part first and part 0
    // last (a fixed order): register r of lane L is token 32 g + 8 (r / 4) +
    // 4 (L / 32) + r % 4, expert 32 eg + L % 32
    for (int p = C::NKS - 1; p >= 0; --p) {
      if (kp == p) {
#pragma unroll
        for (int g = 0; g < C::NTG; ++g)
#pragma unroll
          for (int r = 0; r < 16; ++r) {
            float* q = &stage[(g * 32 + 8 * (r >> 2) + 4 * hf + (r & 3)) * EP + eg * 32 + i];
            *q = (p == C::NKS - 1) ? acc[g][0][r] : *q + acc[g][0][r];
          }
      }
      __syncthreads();
    }
    // lanes per token: every lane of the block has a token (TT = 32: 8, 64: 4, 128: 2)
    constexpr int LPT = 256 / TT;
    route_select_q<LPT, NEG * 32 / LPT, KMAX, MODE, 4, TT>(stage, 0, EP, wscale ? s_scale : nullptr,
                                                           bias ? s_bias : nullptr, t0, T, E, k, idx, gate,
                                                           logits, hist);
    __syncthreads();   // the stage is free again
    tile = next;
  }
  if (MODE != 0) {
    __syncthreads();
    for (int e = threadIdx.x; e < E; e += blockDim.x)
      if (hist[e]) atomicAdd(&counts[e], hist[e]);
  }
}

// Per-row symmetric int8 quantiser: one wave per row, 16-byte loads.
template <typename T>
__global__ __launch_bounds__(256) void k_quantize(const T* __restrict__ W, int E, int d,
                                                  int8_t* __restrict__ q, float* __restrict__ s) {
  constexpr int V = 16 / sizeof(T);   // elements per 16-byte chunk (d % 8 == 0)
  const int row = blockIdx.x * 4 + (threadIdx.x >> 6);
  const int lane = lane_id();
  if (row >= E) return;
  const T* w = W + (size_t)row * d;
  float m = 0.f;
  for (int c = lane * V; c < d; c += 64 * V) {
    float f[V];
    unpack16(ld16(w + c), f, (T*)nullptr);
#pragma unroll
    for (int i = 0; i < V; ++i) m = fmaxf(m, fabsf(f[i]));
  }
#pragma unroll
  for (int off = 32; off > 0; off >>= 1) m = fmaxf(m, __shfl_xor(m, off));
  const float sc = m / 127.0f;
  if (lane == 0) s[row] = sc;
  for (int c = lane * V; c < d; c += 64 * V) {
    float f[V];
    unpack16(ld16(w + c), f, (T*)nullptr);
    uint32_t packed[V / 4];
#pragma unroll
    for (int i = 0; i < V; ++i) {
      int v = 0;
      if (sc > 0.f) {
        const float r = rintf(f[i] / sc);
        v = (int)fminf(fmaxf(r, -127.f), 127.f);
      }
      if (i % 4 == 0) packed[i / 4] = 0;
      packed[i / 4] |= ((uint32_t)v & 0xFFu) << (8 * (i % 4));
    }
    if (V == 8) *(FM_GLOBAL u32x2_t*)(q + (size_t)row * d + c) = u32x2_t{packed[0], packed[V / 4 - 1]};
    else *(FM_GLOBAL uint32_t*)(q + (size_t)row * d + c) = packed[0];
  }
}

int route_cu_count() {
  int dev = 0, n = 0;
  if (hipGetDevice(&dev) != hipSuccess ||
      hipDeviceGetAttribute(&n, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess || n <= 0)
    n = 256;
  return n;
}

template <typename TX, typename TW, int MODE>
int launch_route(const TX* X, const TW* W, const float* ws, const float* bias, int T, int d,
                 int E, int k, int32_t* idx, float* gate, float* logits, int32_t* counts,
                 hipStream_t st) {
  dim3 grid(cdiv(T, RT_TOK));
  if constexpr (std::is_same<TX, bf16>::value) {
    const int ncu = route_cu_count();
    const bool wide = T >= 64 * ncu;
    const bool wider = T >= 128 * ncu;
    // the int8 profiling router keeps the 32-token kernel below when tiles are
    // 32 tokens (measured faster there: 19.2 against 21.7 us at T = 8192, d = 2048)
    if (E <= 64 && d % (wide ? 128 : 256) == 0 && (MODE == 0 || wide)) {
      // 128-token tiles once every compute unit gets one (the router is read
      // once per CU), else 64-token ones, else 32; one block per CU
      const int tiles = wider ? cdiv(T, 128) : wide ? cdiv(T, 64) : cdiv(T, 32);
      const dim3 pg(tiles < ncu ? tiles : ncu);
#define FM_RP(TT, NEG, KM)                                                                                \
  hipLaunchKernelGGL((k_route_p<TW, TT, NEG, KM, MODE>), pg, dim3(256), 0, st, X, W, ws, bias, T, d, E, k, \
                     idx, gate, logits, counts)
#define FM_RP_K(TT, NEG)             \
  if (k <= 2) FM_RP(TT, NEG, 2);      \
  else if (k <= 4) FM_RP(TT, NEG, 4); \
  else if (k <= 8) FM_RP(TT, NEG, 8); \
  else FM_RP(TT, NEG, 16);
      if (wider) {
        if (E <= 32) { FM_RP_K(128, 1) } else { FM_RP_K(128, 2) }
      } else if (wide) {
        if (E <= 32) { FM_RP_K(64, 1) } else { FM_RP_K(64, 2) }
      } else {
        if (E <= 32) { FM_RP_K(32, 1) } else { FM_RP_K(32, 2) }
      }
#undef FM_RP_K
#undef FM_RP
      return check_launch(MODE == 0 ? "moe_route_topk" : MODE == 1 ? "moe_profile_hist" : "moe_profile_route");
    }
    if (E <= 64 && d % RL_COLS == 0) {
#define FM_RL(NB, KM)                                                                          \
  hipLaunchKernelGGL((k_route_lds<TW, NB, KM, MODE>), grid, dim3(256), 0, st, X, W, ws, bias, T, d, E, k, \
                     idx, gate, logits, counts)
#define FM_RL_K(NB)              \
  if (k <= 2) FM_RL(NB, 2);      \
  else if (k <= 4) FM_RL(NB, 4); \
  else if (k <= 8) FM_RL(NB, 8); \
  else FM_RL(NB, 16);
      if (E <= 32) { FM_RL_K(1) }
      else { FM_RL_K(2) }
#undef FM_RL_K
#undef FM_RL
      return check_launch(MODE == 0 ? "moe_route_topk" : MODE == 1 ? "moe_profile_hist" : "moe_profile_route");
    }
  }
  const int ne = cdiv(E, 16);
#define FM_RT(NE, KM)                                                                          \
  hipLaunchKernelGGL((k_route<TX, TW, NE, KM, MODE>), grid, dim3(RtShape<NE>::WAVES * 64), 0, st, X, W, \
                     ws, bias, T, d, E, k, idx, gate, logits, counts)
#define FM_RT_K(NE)              \
  if (k <= 2) FM_RT(NE, 2);      \
  else if (k <= 4) FM_RT(NE, 4); \
  else if (k <= 8) FM_RT(NE, 8); \
  else FM_RT(NE, 16);
  if (ne <= 1) { FM_RT_K(1) }
  else if (ne <= 2) { FM_RT_K(2) }
  else if (ne <= 4) { FM_RT_K(4) }
  else if (ne <= 8) { FM_RT_K(8) }
  else { FM_RT_K(16) }
#undef FM_RT_K
#undef FM_RT
  return check_launch(MODE == 0 ? "moe_route_topk" : MODE == 1 ? "moe_profile_hist" : "moe_profile_route");
}

// Router backward with the top-k selection held fixed: for the k selected
// experts dlogit_j = g_j (dg_j - sum_i g_i dg_i) (the softmax Jacobian-vector
// product), and dX[t] = (accumulate ? dX[t] : 0) + sum_j dlogit_j Wr[idx_j].
// One wave per token; the k router rows of a 16-byte column chunk are loaded
// together (Wr stays in L2); fp32 sums in j order, one rounding to T.  (Staging
// the router in LDS per 32-token block cuts the L2 reads threefold but left one
// block of four waves per CU waiting on a serial chain of chunks: measured
// slower.)
template <typename T, int KMAX>
__global__ __launch_bounds__(256) void k_route_bwd(const float* __restrict__ gate, const int32_t* __restrict__ idx,
                                                   const float* __restrict__ dgate, const T* __restrict__ Wr, int Tn,
                                                   int d, int E, int k, int accumulate, T* __restrict__ dX) {
  constexpr int V = 16 / sizeof(T);
  const int t = blockIdx.x * 4 + (threadIdx.x >> 6);
  if (t >= Tn) return;
  float g[KMAX], dl[KMAX];
  const T* wrow[KMAX];
  float inner = 0.f;
#pragma unroll
  for (int j = 0; j < KMAX; ++j) {
    const bool on = j < k;
    g[j] = on ? gate[(size_t)t * k + j] : 0.f;
    dl[j] = on ? dgate[(size_t)t * k + j] : 0.f;
    // an expert index outside [0, E) (a caller error) is clamped, not followed
    wrow[j] = on ? Wr + (size_t)min(max(idx[(size_t)t * k + j], 0), E - 1) * d : nullptr;
    inner = fmaf(g[j], dl[j], inner);
  }
#pragma unroll
  for (int j = 0; j < KMAX; ++j) dl[j] = g[j] * (dl[j] - inner);
  // The row in groups of G 16-byte chunks per lane: the group's dX chunks (from
  // HBM) are all requested first, and the router rows of chunk u + 1 (from L2)
  // before chunk u is summed, so a wave waits for one HBM round trip per group
  // instead of one per chunk.
  constexpr int G = 4;
  const int lane = lane_id();
  T* xrow = dX + (size_t)t * d;
  for (int c0 = lane * V; c0 < d; c0 += G * 64 * V) {
    u32x4_t xr[G];
    if (accumulate) {
#pragma unroll
      for (int u = 0; u < G; ++u)
        if (c0 + u * 64 * V < d) xr[u] = ld16(xrow + c0 + u * 64 * V);
    }
    u32x4_t raw[2][KMAX];
#pragma unroll
    for (int j = 0; j < KMAX; ++j)
      if (wrow[j]) raw[0][j] = ld16(wrow[j] + c0);
#pragma unroll
    for (int u = 0; u < G; ++u) {
      const int c = c0 + u * 64 * V;
      if (c >= d) break;
      if (u + 1 < G && c + 64 * V < d) {
#pragma unroll
        for (int j = 0; j < KMAX; ++j)
          if (wrow[j]) raw[(u + 1) & 1][j] = ld16(wrow[j] + c + 64 * V);
      }
      float acc[V];
      if (accumulate) {
        unpack16(xr[u], acc, (T*)nullptr);
      } else {
#pragma unroll
        for (int i = 0; i < V; ++i) acc[i] = 0.f;
      }
#pragma unroll
      for (int j = 0; j < KMAX; ++j) {
        if (!wrow[j]) continue;
        float w[V];
        unpack16(raw[u & 1][j], w, (T*)nullptr);
#pragma unroll
        for (int i = 0; i < V; ++i) acc[i] = fmaf(dl[j], w[i], acc[i]);
      }
      st16(xrow + c, pack16(acc, (T*)nullptr));
    }
  }
}

template <typename T>
void launch_route_bwd(const float* gate, const int32_t* idx, const float* dgate, const T* Wr, int Tn, int d, int E,
                      int k, int accumulate, T* dX, hipStream_t st) {
  const dim3 grid(cdiv(Tn, 4)), block(256);
#define FM_RB(KM) \
  hipLaunchKernelGGL((k_route_bwd<T, KM>), grid, block, 0, st, gate, idx, dgate, Wr, Tn, d, E, k, accumulate, dX)
  if (k <= 2) FM_RB(2);
  else if (k <= 4) FM_RB(4);
  else if (k <= 8) FM_RB(8);
  else FM_RB(16);
#undef FM_RB
}

int check_route_shape(int T, int d, int E, int k) {
  if (T < 0 || d <= 0 || E <= 0 || k <= 0) return fail(MOE_ERR_ARG, "T=%d d=%d E=%d k=%d", T, d, E, k);
  if (E > 256) return fail(MOE_ERR_UNSUPPORTED, "E=%d > 256", E);
  if (k > 16 || k > E) return fail(MOE_ERR_UNSUPPORTED, "k=%d must be <= min(E, 16)", k);
  if (d % 8) return fail(MOE_ERR_UNSUPPORTED, "d=%d not a multiple of 8", d);
  return MOE_OK;
}

}  // namespace
}  // namespace fm

using namespace fm;

extern "C" int moe_route_topk(const void* X, const void* Wr, int dtype, const float* bias,
                              int T, int d, int E, int k, int32_t* idx, float* gate,
                              float* logits, void* stream) {
  clear_error();
  FM_TRY(check_route_shape(T, d, E, k));
  FM_TRY(need_dtype_float(dtype, "dtype"));
  if (T == 0) return MOE_OK;
  FM_TRY(need(X, "X")); FM_TRY(need(Wr, "Wr")); FM_TRY(need(idx, "idx")); FM_TRY(need(gate, "gate"));
  FM_TRY(need_aligned(X, "X")); FM_TRY(need_aligned(Wr, "Wr")); FM_TRY(need_aligned(bias, "bias"));
  FM_TRY(need_aligned(idx, "idx")); FM_TRY(need_aligned(gate, "gate")); FM_TRY(need_aligned(logits, "logits"));
  hipStream_t st = as_stream(stream);
  if (dtype == MOE_BF16)
    return launch_route<bf16, bf16, 0>((const bf16*)X, (const bf16*)Wr, nullptr, bias, T, d, E, k,
                                       idx, gate, logits, nullptr, st);
  return launch_route<float, float, 0>((const float*)X, (const float*)Wr, nullptr, bias, T, d, E, k,
                                       idx, gate, logits, nullptr, st);
}

extern "C" int moe_quantize_int8(const void* W, int dtype, int E, int d, int8_t* Wq, float* scale,
                                 void* stream) {
  clear_error();
  if (E <= 0 || d <= 0) return fail(MOE_ERR_ARG, "E=%d d=%d", E, d);
  if (d % 8) return fail(MOE_ERR_UNSUPPORTED, "d=%d not a multiple of 8", d);
  FM_TRY(need_dtype_float(dtype, "dtype"));
  FM_TRY(need(W, "W")); FM_TRY(need(Wq, "Wq")); FM_TRY(need(scale, "scale"));
  FM_TRY(need_aligned(W, "W")); FM_TRY(need_aligned(Wq, "Wq")); FM_TRY(need_aligned(scale, "scale"));
  hipStream_t st = as_stream(stream);
  dim3 grid(cdiv(E, 4)), block(256);
  if (dtype == MOE_BF16)
    hipLaunchKernelGGL(k_quantize<bf16>, grid, block, 0, st, (const bf16*)W, E, d, Wq, scale);
  else
    hipLaunchKernelGGL(k_quantize<float>, grid, block, 0, st, (const float*)W, E, d, Wq, scale);
  return check_launch("moe_quantize_int8");
}

extern "C" int moe_profile_hist(const void* X, int x_dtype, const int8_t* Wq, const float* scale,
                                const float* bias, int T, int d, int E, int k, int32_t* counts,
                                int32_t* idx, void* stream) {
  clear_error();
  FM_TRY(check_route_shape(T, d, E, k));
  FM_TRY(need_dtype_float(x_dtype, "x_dtype"));
  if (T == 0) return MOE_OK;
  FM_TRY(need(X, "X")); FM_TRY(need(Wq, "Wq")); FM_TRY(need(scale, "scale")); FM_TRY(need(counts, "counts"));
  FM_TRY(need_aligned(X, "X")); FM_TRY(need_aligned(Wq, "Wq")); FM_TRY(need_aligned(scale, "scale"));
  FM_TRY(need_aligned(bias, "bias")); FM_TRY(need_aligned(counts, "counts")); FM_TRY(need_aligned(idx, "idx"));
  hipStream_t st = as_stream(stream);
  if (x_dtype == MOE_BF16)
    return launch_route<bf16, int8_t, 1>((const bf16*)X, Wq, scale, bias, T, d, E, k, idx, nullptr,
                                         nullptr, counts, st);
  return launch_route<float, int8_t, 1>((const float*)X, Wq, scale, bias, T, d, E, k, idx, nullptr,
                                        nullptr, counts, st);
}

extern "C" int moe_profile_route(const void* X, int x_dtype, const int8_t* Wq, const float* scale,
                                 const float* bias, int T, int d, int E, int k, int32_t* counts,
                                 int32_t* idx, float* gate, void* stream) {
  clear_error();
  FM_TRY(check_route_shape(T, d, E, k));
  FM_TRY(need_dtype_float(x_dtype, "x_dtype"));
  if (T == 0) return MOE_OK;
  FM_TRY(need(X, "X")); FM_TRY(need(Wq, "Wq")); FM_TRY(need(scale, "scale")); FM_TRY(need(counts, "counts"));
  FM_TRY(need(idx, "idx")); FM_TRY(need(gate, "gate"));
  FM_TRY(need_aligned(X, "X")); FM_TRY(need_aligned(Wq, "Wq")); FM_TRY(need_aligned(scale, "scale"));
  FM_TRY(need_aligned(bias, "bias")); FM_TRY(need_aligned(counts, "counts")); FM_TRY(need_aligned(idx, "idx"));
  FM_TRY(need_aligned(gate, "gate"));
  hipStream_t st = as_stream(stream);
  if (x_dtype == MOE_BF16)
    return launch_route<bf16, int8_t, 2>((const bf16*)X, Wq, scale, bias, T, d, E, k, idx, gate, nullptr,
                                         counts, st);
  return launch_route<float, int8_t, 2>((const float*)X, Wq, scale, bias, T, d, E, k, idx, gate, nullptr,
                                        counts, st);
}

extern "C" int moe_route_bwd(const float* gate, const int32_t* idx, const float* dgate, const void* Wr, int dtype,
                             int T, int d, int E, int k, void* dX, int accumulate, void* stream) {
  clear_error();
  FM_TRY(check_route_shape(T, d, E, k));
  FM_TRY(need_dtype_float(dtype, "dtype"));
  if (T == 0) return MOE_OK;
  FM_TRY(need(gate, "gate")); FM_TRY(need(idx, "idx")); FM_TRY(need(dgate, "dgate"));
  FM_TRY(need(Wr, "Wr")); FM_TRY(need(dX, "dX"));
  FM_TRY(need_aligned(gate, "gate")); FM_TRY(need_aligned(idx, "idx")); FM_TRY(need_aligned(dgate, "dgate"));
  FM_TRY(need_aligned(Wr, "Wr")); FM_TRY(need_aligned(dX, "dX"));
  hipStream_t st = as_stream(stream);
  if (dtype == MOE_BF16)
    launch_route_bwd<bf16>(gate, idx, dgate, (const bf16*)Wr, T, d, E, k, accumulate != 0, (bf16*)dX, st);
  else
    launch_route_bwd<float>(gate, idx, dgate, (const float*)Wr, T, d, E, k, accumulate != 0, (float*)dX, st);
  return check_launch("moe_route_bwd");
}
