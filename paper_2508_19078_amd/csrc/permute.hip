// Gate re-routing and token permutation into per-slot buckets, the combine,
// and their backward passes.
//
// Permute runs in two launches (three when slots x count blocks exceed 16384),
// all deterministic:
//   count          a block of 256 tokens counts its rows per slot (LDS integer
//                  atomics)
//   [scan]         for large tables, one block turns the per-block counts into
//                  global row positions: a wave scan per slot over the blocks,
//                  then an exclusive scan over the slots (the bucket offsets)
//   place+scatter  a block of 16 or 32 tokens ranks its rows within each slot in
//                  token order, writes the maps and copies X[t] to every row t
//                  opens (16-byte accesses, the row loads issued first); for
//                  small tables it sums the count table itself
// Combine and the two backward gathers run one wave per token.
#include <stdlib.h>

#include <mutex>
#include <vector>

#include "common.hpp"
#include "debug.hpp"

namespace fm {
namespace {

constexpr int PM_TOK = 256;   // tokens (threads) per block of count/place
constexpr int PM_SMAX = 512;  // slots count and place support
constexpr int PM_FUSE = 16384;  // place sums the count table itself up to this many entries
constexpr int PS_THREADS = 512;  // place + scatter: 8 waves of 16 or 32 tokens per block

template <int KMAX>
struct TokenSlots {
  int s[KMAX];        // slot of choice j
  bool first[KMAX];   // choice j opens its row (first choice of this slot)
  int owner[KMAX];    // j' of the choice that opened the row of choice j
};

template <int KMAX>
__device__ __forceinline__ void token_slots(const int32_t* __restrict__ idx,
                                            const int32_t* __restrict__ emap, int t, int k,
                                            TokenSlots<KMAX>& ts) {
#pragma unroll
  for (int j = 0; j < KMAX; ++j) {
    ts.s[j] = -1;
    ts.first[j] = false;
    ts.owner[j] = j;
    if (j < k) {
      int e = idx[(size_t)t * k + j];
      ts.s[j] = emap ? emap[e] : e;
    }
  }
#pragma unroll
  for (int j = 0; j < KMAX; ++j) {
    bool f = j < k;
#pragma unroll
    for (int i = 0; i < KMAX; ++i)
      if (i < j && f && ts.s[i] == ts.s[j]) {
        f = false;
        ts.owner[j] = ts.owner[i];
      }
    ts.first[j] = f;
  }
}

template <int KMAX>
__global__ __launch_bounds__(PM_TOK) void k_perm_count(const int32_t* __restrict__ idx,
                                                    const int32_t* __restrict__ emap, int T, int k,
                                                    int S, int32_t* __restrict__ bc, int nblk) {
  __shared__ int cnt[PM_SMAX];
  for (int s = threadIdx.x; s < S; s += blockDim.x) cnt[s] = 0;
  __syncthreads();
  const int t = blockIdx.x * PM_TOK + threadIdx.x;
  if (t < T) {
    TokenSlots<KMAX> ts;
    token_slots<KMAX>(idx, emap, t, k, ts);
#pragma unroll
    for (int j = 0; j < KMAX; ++j)
      if (ts.first[j]) atomicAdd(&cnt[ts.s[j]], 1);
  }
  __syncthreads();
  // slot-major layout: bc[s * nblk + block]
  for (int s = threadIdx.x; s < S; s += blockDim.x) bc[(size_t)s * nblk + blockIdx.x] = cnt[s];
}

// One block of 1024 threads.
__global__ __launch_bounds__(1024) void k_perm_scan(int32_t* __restrict__ bc, int nblk, int S,
                                                    int32_t* __restrict__ offsets) {
  __shared__ int tot[513];
  const int lane = lane_id(), wave = threadIdx.x >> 6, nw = blockDim.x >> 6;
  for (int s = wave; s < S; s += nw) {
    int carry = 0;
    for (int b0 = 0; b0 < nblk; b0 += 64) {
      const int b = b0 + lane;
      const int v = b < nblk ? bc[(size_t)s * nblk + b] : 0;
      int x = v;
#pragma unroll
      for (int off = 1; off < 64; off <<= 1) {
        int y = __shfl_up(x, off);
        if (lane >= off) x += y;
      }
      if (b < nblk) bc[(size_t)s * nblk + b] = carry + x - v;
      carry += __shfl(x, 63);
    }
    if (lane == 0) tot[s] = carry;
  }
  __syncthreads();
  if (threadIdx.x == 0) {
    int run = 0;
    for (int s = 0; s < S; ++s) {
      int v = tot[s];
      tot[s] = run;
      offsets[s] = run;
      run += v;
    }
    offsets[S] = run;
  }
  __syncthreads();
  for (size_t i = threadIdx.x; i < (size_t)S * nblk; i += blockDim.x) bc[i] += tot[i / nblk];
}

// Places the rows of PS_TOK (16 or 32) tokens and copies them: block = 8 waves,
// wave w owns tokens t0 + w * PS_TOK / 8 onwards.  (16-token blocks when
// 32-token ones would leave compute units idle.)
//   1. every wave starts loading the first 4 KB of its four rows (they do not
//      depend on the maps), while the first 256 threads take the slots of the
//      count block's tokens up to the end of this block;
//   2. the rows the count block's earlier tokens open are counted per slot (LDS
//      integer atomics); this block's own tokens OR their bit into one 64-bit
//      mask per slot, so a row's rank among them is a popcount (order-free);
//      with SCAN the block also folds the count table into the slot totals and
//      the rows of the count blocks before its own (and block 0 writes the
//      bucket offsets), otherwise bc already holds those positions;
//   3. the maps are written and each row is stored at every position its token
//      opens.
// s + the squares of the 16 bytes' elements (bf16, or fp32 when f32), in order.
__device__ __forceinline__ float sq_acc(const u32x4_t& v, bool f32, float s) {
  if (f32) {
    float f[4];
    unpack16(v, f, (float*)nullptr);
#pragma unroll
    for (int i = 0; i < 4; ++i) s = fmaf(f[i], f[i], s);
  } else {
    float f[8];
    unpack16(v, f, (bf16*)nullptr);
#pragma unroll
    for (int i = 0; i < 8; ++i) s = fmaf(f[i], f[i], s);
  }
  return s;
}

template <int KMAX, bool SCAN, int PS_TOK>
__global__ __launch_bounds__(PS_THREADS) void k_place_scatter(
    const int32_t* __restrict__ idx, const float* __restrict__ gate, const int32_t* __restrict__ emap,
    int T, int k, int S, const int32_t* __restrict__ bc, int nblk, int32_t* __restrict__ offsets,
    int32_t* __restrict__ perm_token, float* __restrict__ perm_gate, int32_t* __restrict__ inv,
    const char* __restrict__ X, int row_bytes, char* __restrict__ Xp, bool xf32, float* __restrict__ x_sq) {
  constexpr int NTW = PS_TOK / (PS_THREADS / 64);   // tokens per wave
  constexpr int U = 4;                              // 16-byte chunks per lane and row per pass
  __shared__ unsigned long long msk[PM_SMAX];       // this block's tokens, one bit each, per slot
  __shared__ int pre[PM_SMAX];                      // rows of the count block's earlier tokens
  __shared__ int base[PM_SMAX];                     // this block's first row in each slot
  __shared__ int tot[SCAN ? PM_SMAX : 1];           // rows of each slot over all tokens
  __shared__ int posl[PS_TOK][KMAX];                // row of each choice that opens one, else -1
  const int tid = threadIdx.x, lane = lane_id(), wave = tid >> 6;
  const int t0 = blockIdx.x * PS_TOK;
  const int grp = t0 / PM_TOK;
  // 1. first pass of this wave's rows
  u32x4_t v[NTW][U];
#pragma unroll
  for (int x = 0; x < NTW; ++x) {
    const int t = t0 + wave * NTW + x;
    const char* src = X + (size_t)t * row_bytes;
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const int c = (lane + 64 * u) * 16;
      if (t < T && c < row_bytes) v[x][u] = ld16(src + c);
    }
  }
  const int tg = grp * PM_TOK + tid;
  const bool mine = tid < PM_TOK && tg >= t0 && tg < t0 + PS_TOK && tg < T;
  const bool earlier = tid < PM_TOK && tg < t0;
  TokenSlots<KMAX> ts;
  if (mine || earlier) {
    token_slots<KMAX>(idx, emap, tg, k, ts);
  } else {
#pragma unroll
    for (int j = 0; j < KMAX; ++j) { ts.s[j] = -1; ts.first[j] = false; ts.owner[j] = j; }
  }
  float g[KMAX];
#pragma unroll
  for (int j = 0; j < KMAX; ++j) g[j] = (mine && j < k) ? gate[(size_t)tg * k + j] : 0.f;
  const int n = SCAN ? S * nblk : 0;
  int cv[4];
#pragma unroll
  for (int u = 0; u < 4; ++u) {
    const int i = u * PS_THREADS + tid;
    cv[u] = i < n ? bc[i] : 0;
  }
  for (int s = tid; s < S; s += PS_THREADS) {
    msk[s] = 0ull;
    pre[s] = 0;
    if (SCAN) tot[s] = 0;
    base[s] = SCAN ? 0 : bc[(size_t)s * nblk + grp];
  }
  __syncthreads();
  // 2. counts and masks
  const int me = tg - t0;
#pragma unroll
  for (int j = 0; j < KMAX; ++j) {
    if (!ts.first[j]) continue;
    if (earlier) atomicAdd(&pre[ts.s[j]], 1);
    else atomicOr(&msk[ts.s[j]], 1ull << me);
  }
  for (int i0 = 0; i0 < n; i0 += 4 * PS_THREADS) {
    if (i0 > 0) {
#pragma unroll
      for (int u = 0; u < 4; ++u) {
        const int i = i0 + u * PS_THREADS + tid;
        cv[u] = i < n ? bc[i] : 0;
      }
    }
#pragma unroll
    for (int u = 0; u < 4; ++u) {
      const int i = i0 + u * PS_THREADS + tid;
      if (i < n && cv[u]) {
        const int s = i / nblk;
        atomicAdd(&tot[s], cv[u]);
        if (i - s * nblk < grp) atomicAdd(&base[s], cv[u]);
      }
    }
  }
  __syncthreads();
  if (SCAN) {
    if (wave == 0) {
      // exclusive scan of the slot totals: lane l takes a run of consecutive slots
      const int per = (S + 63) / 64, s0 = min(S, lane * per), s1 = min(S, s0 + per);
      int loc = 0;
      for (int s = s0; s < s1; ++s) loc += tot[s];
      int inc = loc;
#pragma unroll
      for (int off = 1; off < 64; off <<= 1) {
        const int y = __shfl_up(inc, off);
        if (lane >= off) inc += y;
      }
      int run = inc - loc;
      for (int s = s0; s < s1; ++s) {
        base[s] += run + pre[s];
        if (blockIdx.x == 0) offsets[s] = run;
        run += tot[s];
      }
      if (blockIdx.x == 0 && lane == 63) offsets[S] = inc;
    }
  } else {
    for (int s = tid; s < S; s += PS_THREADS) base[s] += pre[s];
  }
  __syncthreads();
  // 3. maps, then rows
  if (mine) {
    const unsigned long long lt = (1ull << me) - 1ull;
    int pos[KMAX];
#pragma unroll
    for (int j = 0; j < KMAX; ++j) {
      pos[j] = 0;
      if (ts.first[j]) pos[j] = base[ts.s[j]] + __popcll(msk[ts.s[j]] & lt);
    }
#pragma unroll
    for (int j = 0; j < KMAX; ++j) {
      if (!ts.first[j]) continue;
      float sum = 0.f;                 // gates of every choice folded into this row, j order
#pragma unroll
      for (int i = 0; i < KMAX; ++i)
        if (i < k && ts.s[i] == ts.s[j]) sum += g[i];
      perm_token[pos[j]] = tg;
      perm_gate[pos[j]] = sum;
    }
#pragma unroll
    for (int j = 0; j < KMAX; ++j) {
      posl[me][j] = ts.first[j] ? pos[j] : -1;
      if (j >= k) continue;
      int p = 0;
#pragma unroll
      for (int i = 0; i < KMAX; ++i)
        if (i == ts.owner[j]) p = pos[i];
      inv[(size_t)tg * k + j] = ts.first[j] ? p : -2 - p;
    }
  }
  __syncthreads();
#pragma unroll
  for (int x = 0; x < NTW; ++x) {
    const int tl = wave * NTW + x, t = t0 + tl;
    if (t >= T) break;
    float ss = 0.f;                  // ||X[t]||^2: the lane's chunks in order, then the wave
    for (int j = 0; j < k; ++j) {
      const int p = posl[tl][j];
      if (p < 0) continue;
      char* dst = Xp + (size_t)p * row_bytes;
#pragma unroll
      for (int u = 0; u < U; ++u) {
        const int c = (lane + 64 * u) * 16;
        if (c < row_bytes) st16(dst + c, v[x][u]);
      }
    }
    if (x_sq) {
#pragma unroll
      for (int u = 0; u < U; ++u)
        if ((lane + 64 * u) * 16 < row_bytes) ss = sq_acc(v[x][u], xf32, ss);
    }
    // rows longer than one pass
    const char* src = X + (size_t)t * row_bytes;
    for (int c0 = 64 * U * 16; c0 < row_bytes; c0 += 64 * U * 16) {
      u32x4_t w[U];
#pragma unroll
      for (int u = 0; u < U; ++u) {
        const int c = c0 + (lane + 64 * u) * 16;
        if (c < row_bytes) w[u] = ld16(src + c);
      }
      for (int j = 0; j < k; ++j) {
        const int p = posl[tl][j];
        if (p < 0) continue;
        char* dst = Xp + (size_t)p * row_bytes;
#pragma unroll
        for (int u = 0; u < U; ++u) {
          const int c = c0 + (lane + 64 * u) * 16;
          if (c < row_bytes) st16(dst + c, w[u]);
        }
      }
      if (x_sq) {
#pragma unroll
        for (int u = 0; u < U; ++u)
          if (c0 + (lane + 64 * u) * 16 < row_bytes) ss = sq_acc(w[u], xf32, ss);
      }
    }
    if (x_sq) {
#pragma unroll
      for (int off = 32; off > 0; off >>= 1) ss += __shfl_xor(ss, off);
      if (lane == 0) x_sq[t] = ss;
    }
  }
}

__global__ void k_zero_i32(int32_t* p, int n) {
  const int i = blockIdx.x * blockDim.x + threadIdx.x;
  if (i < n) p[i] = 0;
}

// Decodes inv: row of choice (t, j), folded or not.
__device__ __forceinline__ int row_of(int v) { return v >= 0 ? v : -2 - v; }

// Gathers and sums up to KMAX + S_sh rows into one token's row, U 16-byte
// chunks per lane at a time with every load of the step issued before the
// arithmetic: out[c] = sum_j w_j src[p_j][c] + sum of the shared rows.  The
// first SHMAX shared rows are loaded with the routed ones; further shared rows
// (a layer with more than SHMAX shared experts) are added one at a time.
template <typename T, int KMAX, bool WEIGHTED>
__device__ __forceinline__ void gather_sum_row(const T* __restrict__ src, const int (&p)[KMAX],
                                               const float (&g)[KMAX], size_t R, int Tn, int t, int d,
                                               int S_sh, T* __restrict__ out) {
  constexpr int V = 16 / sizeof(T), U = 2, SHMAX = 2, NS = KMAX + SHMAX;
  const T* rows[NS];
  float w[NS];
#pragma unroll
  for (int j = 0; j < KMAX; ++j) {
    rows[j] = p[j] >= 0 ? src + (size_t)p[j] * d : nullptr;
    w[j] = g[j];
  }
#pragma unroll
  for (int s = 0; s < SHMAX; ++s) {
    rows[KMAX + s] = s < S_sh ? src + (R + (size_t)s * Tn + t) * d : nullptr;
    w[KMAX + s] = 1.f;
  }
  for (int c0 = lane_id() * V; c0 < d; c0 += U * 64 * V) {
    u32x4_t raw[U][NS];
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const int c = c0 + u * 64 * V;
#pragma unroll
      for (int j = 0; j < NS; ++j)
        if (rows[j] && c < d) raw[u][j] = ld16(rows[j] + c);
    }
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const int c = c0 + u * 64 * V;
      if (c >= d) continue;
      float acc[V];
#pragma unroll
      for (int i = 0; i < V; ++i) acc[i] = 0.f;
#pragma unroll
      for (int j = 0; j < NS; ++j) {
        if (!rows[j]) continue;
        float f[V];
        unpack16(raw[u][j], f, (T*)nullptr);
#pragma unroll
        for (int i = 0; i < V; ++i) acc[i] = (WEIGHTED && j < KMAX) ? fmaf(w[j], f[i], acc[i]) : acc[i] + f[i];
      }
      for (int sh = SHMAX; sh < S_sh; ++sh) {
        float f[V];
        unpack16(ld16(src + (R + (size_t)sh * Tn + t) * d + c), f, (T*)nullptr);
#pragma unroll
        for (int i = 0; i < V; ++i) acc[i] += f[i];
      }
      st16(out + (size_t)t * d + c, pack16(acc, (T*)nullptr));
    }
  }
}

// Y[t] = sum_{first choices} perm_gate[p] O[p] + sum_shared O[shared row].
template <typename T, int KMAX>
__global__ __launch_bounds__(256) void k_combine(const T* __restrict__ O, const int32_t* __restrict__ inv,
                                                 const float* __restrict__ pg, int Tn, int k, int d,
                                                 int S_sh, T* __restrict__ Y) {
  const int t = blockIdx.x * 4 + (threadIdx.x >> 6);
  if (t >= Tn) return;
  int p[KMAX];
  float g[KMAX];
#pragma unroll
  for (int j = 0; j < KMAX; ++j) {
    p[j] = j < k ? inv[(size_t)t * k + j] : -1;
    g[j] = p[j] >= 0 ? pg[p[j]] : 0.f;
  }
  gather_sum_row<T, KMAX, true>(O, p, g, (size_t)Tn * k, Tn, t, d, S_sh, Y);
}

// dO[p] = perm_gate[p] dY[t]; shared rows get dY[t]; dgate[t,j] = <dY[t], O[row]>.
// A lane loads CB_PF chunks of dY[t] before it stores any of them, so a wave
// waits for one load latency per CB_PF chunks (one for a whole 2048-wide bf16
// row) instead of one per chunk.
constexpr int CB_PF = 4;

template <typename T, int KMAX>
__global__ __launch_bounds__(256) void k_combine_bwd(const T* __restrict__ dY, const T* __restrict__ O,
                                                     const int32_t* __restrict__ inv,
                                                     const float* __restrict__ pg, int Tn, int k,
                                                     int d, int S_sh, T* __restrict__ dO,
                                                     float* __restrict__ dgate, float* __restrict__ dy_sq) {
  constexpr int V = 16 / sizeof(T);
  const int t = blockIdx.x * 4 + (threadIdx.x >> 6);
  if (t >= Tn) return;
  const size_t R = (size_t)Tn * k;
  int p[KMAX];
  float g[KMAX], dot[KMAX];
#pragma unroll
  for (int j = 0; j < KMAX; ++j) {
    p[j] = j < k ? inv[(size_t)t * k + j] : -1;
    g[j] = p[j] >= 0 ? pg[p[j]] : 0.f;
    dot[j] = 0.f;
  }
  float ss = 0.f;                    // ||dY[t]||^2: the lane's chunks in order, then the wave
  for (int c0 = lane_id() * V; c0 < d; c0 += CB_PF * 64 * V) {
    u32x4_t rawp[CB_PF];
#pragma unroll
    for (int u = 0; u < CB_PF; ++u)
      if (c0 + u * 64 * V < d) rawp[u] = ld16(dY + (size_t)t * d + c0 + u * 64 * V);
#pragma unroll
    for (int u = 0; u < CB_PF; ++u) {
      const int c = c0 + u * 64 * V;
      if (c >= d) break;
      const u32x4_t raw = rawp[u];
      float f[V];
      unpack16(raw, f, (T*)nullptr);
      if (dy_sq) {
#pragma unroll
        for (int i = 0; i < V; ++i) ss = fmaf(f[i], f[i], ss);
      }
#pragma unroll
      for (int j = 0; j < KMAX; ++j) {
        if (j >= k) continue;
        if (p[j] >= 0) {
          float o[V];
#pragma unroll
          for (int i = 0; i < V; ++i) o[i] = g[j] * f[i];
          st16(dO + (size_t)p[j] * d + c, pack16(o, (T*)nullptr));
        }
        if (dgate) {
          float o[V];
          unpack16(ld16(O + (size_t)row_of(p[j]) * d + c), o, (T*)nullptr);
#pragma unroll
          for (int i = 0; i < V; ++i) dot[j] = fmaf(f[i], o[i], dot[j]);
        }
      }
      for (int sh = 0; sh < S_sh; ++sh) st16(dO + (R + (size_t)sh * Tn + t) * d + c, raw);
    }
  }
  if (dgate) {
#pragma unroll
    for (int j = 0; j < KMAX; ++j) {
      if (j >= k) continue;
      float v = dot[j];
#pragma unroll
      for (int off = 32; off > 0; off >>= 1) v += __shfl_xor(v, off);
      if (lane_id() == 0) dgate[(size_t)t * k + j] = v;
    }
  }
  if (dy_sq) {
#pragma unroll
    for (int off = 32; off > 0; off >>= 1) ss += __shfl_xor(ss, off);
    if (lane_id() == 0) dy_sq[t] = ss;
  }
}

// dX[t] = sum_{first choices} dX_perm[p] + sum_shared dX_perm[shared row].
template <typename T, int KMAX>
__global__ __launch_bounds__(256) void k_permute_bwd(const T* __restrict__ dXp,
                                                     const int32_t* __restrict__ inv, int Tn, int k,
                                                     int d, int S_sh, T* __restrict__ dX) {
  const int t = blockIdx.x * 4 + (threadIdx.x >> 6);
  if (t >= Tn) return;
  int p[KMAX];
  float g[KMAX];
#pragma unroll
  for (int j = 0; j < KMAX; ++j) {
    p[j] = j < k ? inv[(size_t)t * k + j] : -1;
    g[j] = 1.f;
  }
  gather_sum_row<T, KMAX, false>(dXp, p, g, (size_t)Tn * k, Tn, t, d, S_sh, dX);
}

int check_layer(const moe_layer* L) {
  if (!L) return fail(MOE_ERR_ARG, "layer must not be NULL");
  if (L->d <= 0 || L->I <= 0) return fail(MOE_ERR_ARG, "layer d=%d I=%d", L->d, L->I);
  if (L->d % 8 || L->I % 8) return fail(MOE_ERR_UNSUPPORTED, "layer d=%d I=%d must be multiples of 8", L->d, L->I);
  if (L->S_routed < 0 || L->S_shared < 0 || L->S_routed + L->S_shared < 1 || L->S_routed > 512 ||
      L->S_shared > 512)
    return fail(MOE_ERR_ARG, "layer S_routed=%d S_shared=%d", L->S_routed, L->S_shared);
  return need_dtype_float(L->dtype, "layer dtype");
}

int check_tk(int T, int k) {
  if (T < 0 || k <= 0) return fail(MOE_ERR_ARG, "T=%d k=%d", T, k);
  if (k > 16) return fail(MOE_ERR_UNSUPPORTED, "k=%d > 16", k);
  return MOE_OK;
}

#define FM_KSWITCH(k, MACRO)       \
  if ((k) <= 2) { MACRO(2); }      \
  else if ((k) <= 4) { MACRO(4); } \
  else if ((k) <= 8) { MACRO(8); } \
  else { MACRO(16); }
// The combine holds a register set per possible choice (KMAX + 2 rows of two
// chunks); an instance for k <= 6 keeps k = 6 layers at 114 instead of 137
// VGPRs (measured 65 -> 63 us cold at T = 8192, d = 2048).
#define FM_KSWITCH_COMBINE(k, MACRO) \
  if ((k) <= 2) { MACRO(2); }        \
  else if ((k) <= 4) { MACRO(4); }   \
  else if ((k) <= 6) { MACRO(6); }   \
  else if ((k) <= 8) { MACRO(8); }   \
  else { MACRO(16); }

// Compute units of the current device (256 on MI355X when the query fails).
int cu_count() {
  int dev = 0, n = 0;
  if (hipGetDevice(&dev) != hipSuccess ||
      hipDeviceGetAttribute(&n, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess || n <= 0)
    n = 256;
  return n;
}

}  // namespace
}  // namespace fm

using namespace fm;

extern "C" int moe_validate_routing(const int32_t* idx, const int32_t* expert_map, int T, int E, int k,
                                    int S_routed) {
  clear_error();
  if (T < 0 || k <= 0 || E <= 0 || S_routed <= 0) return fail(MOE_ERR_ARG, "T=%d k=%d E=%d S_routed=%d", T, k, E,
                                                               S_routed);
  if (T > 0 && !idx) return fail(MOE_ERR_ARG, "idx must not be NULL");
  if (expert_map) {
    for (int e = 0; e < E; ++e)
      if (expert_map[e] < 0 || expert_map[e] >= S_routed)
        return fail(MOE_ERR_ARG, "expert_map[%d]=%d outside [0, %d)", e, expert_map[e], S_routed);
  } else if (S_routed < E) {
    return fail(MOE_ERR_ARG, "identity map needs S_routed >= E");
  }
  for (long i = 0; i < (long)T * k; ++i)
    if (idx[i] < 0 || idx[i] >= E)
      return fail(MOE_ERR_ARG, "idx[%ld][%ld]=%d outside [0, %d)", i / k, i % k, idx[i], E);
  return MOE_OK;
}

namespace fm {
namespace {
// FLUXMOE_DEBUG_CHECKS set (and not "0"): moe_permute copies idx and
// expert_map to the host, waits for the stream, and range-checks them before
// launching anything.  Slow; for debugging callers.
int debug_check_routing(const int32_t* idx, const int32_t* expert_map, int T, int E, int k, int S_routed,
                        hipStream_t st) {
  std::vector<int32_t> hi((size_t)T * k), hm(expert_map ? E : 0);
  if (T > 0 && hipMemcpyAsync(hi.data(), idx, hi.size() * sizeof(int32_t), hipMemcpyDeviceToHost, st) != hipSuccess)
    return fail(MOE_ERR_HIP, "debug check: copy of idx failed");
  if (expert_map &&
      hipMemcpyAsync(hm.data(), expert_map, hm.size() * sizeof(int32_t), hipMemcpyDeviceToHost, st) != hipSuccess)
    return fail(MOE_ERR_HIP, "debug check: copy of expert_map failed");
  if (hipStreamSynchronize(st) != hipSuccess) return fail(MOE_ERR_HIP, "debug check: stream synchronisation failed");
  return moe_validate_routing(hi.data(), expert_map ? hm.data() : nullptr, T, E, k, S_routed);
}
}  // namespace
}  // namespace fm

extern "C" size_t moe_permute_workspace_size(int T, int k, int S_routed) {
  (void)k;
  if (T <= 0 || S_routed <= 0) return 256;
  const size_t nblk = (size_t)cdiv(T, PM_TOK);
  return ((nblk * S_routed * sizeof(int32_t) + 255) / 256) * 256;
}

namespace fm {
namespace {

// Validation of moe_permute's arguments other than the workspace.
int permute_check(const void* X, int dtype, const int32_t* idx, const float* gate, const int32_t* expert_map,
                  int T, int d, int E, int k, int S_routed, const int32_t* offsets, const int32_t* perm_token,
                  const float* perm_gate, const int32_t* inv, const void* X_perm) {
  FM_TRY(check_tk(T, k));
  if (d <= 0 || E <= 0 || S_routed <= 0) return fail(MOE_ERR_ARG, "d=%d E=%d S_routed=%d", d, E, S_routed);
  if (E > 256 || k > E) return fail(MOE_ERR_UNSUPPORTED, "E=%d k=%d", E, k);
  if (S_routed > 512) return fail(MOE_ERR_UNSUPPORTED, "S_routed=%d > 512", S_routed);
  if (!expert_map && S_routed < E) return fail(MOE_ERR_ARG, "identity map needs S_routed >= E");
  if (d % 8) return fail(MOE_ERR_UNSUPPORTED, "d=%d not a multiple of 8", d);
  FM_TRY(need_dtype_float(dtype, "dtype"));
  FM_TRY(need(offsets, "offsets"));
  if (T > 0) {
    FM_TRY(need(X, "X")); FM_TRY(need(idx, "idx")); FM_TRY(need(gate, "gate"));
    FM_TRY(need(perm_token, "perm_token")); FM_TRY(need(perm_gate, "perm_gate"));
    FM_TRY(need(inv, "inv")); FM_TRY(need(X_perm, "X_perm"));
  }
  FM_TRY(need_aligned(X, "X")); FM_TRY(need_aligned(X_perm, "X_perm"));
  FM_TRY(need_aligned(offsets, "offsets"));
  return MOE_OK;
}

// The launches of a validated permute; bc = the count table (workspace).
int permute_launch(const void* X, int dtype, const int32_t* idx, const float* gate, const int32_t* expert_map,
                   int T, int d, int E, int k, int S_routed, int32_t* offsets, int32_t* perm_token,
                   float* perm_gate, int32_t* inv, void* X_perm, float* x_sq, int32_t* bc, hipStream_t st,
                   const char* what, bool allow_debug) {
  if (T == 0) {
    hipLaunchKernelGGL(k_zero_i32, dim3(cdiv(S_routed + 1, 256)), dim3(256), 0, st, offsets,
                       S_routed + 1);
    return check_launch(what);
  }
  if (allow_debug && debug_checks()) FM_TRY(debug_check_routing(idx, expert_map, T, E, k, S_routed, st));
  const int nblk = cdiv(T, PM_TOK);
#define FM_PC(KM) \
  hipLaunchKernelGGL(k_perm_count<KM>, dim3(nblk), dim3(PM_TOK), 0, st, idx, expert_map, T, k, S_routed, bc, \
                     nblk)
  FM_KSWITCH(k, FM_PC)
#undef FM_PC
  const bool fuse = (long long)nblk * S_routed <= PM_FUSE;
  if (!fuse) hipLaunchKernelGGL(k_perm_scan, dim3(1), dim3(1024), 0, st, bc, nblk, S_routed, offsets);
  const int row_bytes = d * esize(dtype);
  // 32-token blocks once they fill every compute unit, else 16-token ones
  const bool wide = cdiv(T, 32) >= cu_count();
#define FM_PS(KM, SC, TOK)                                                                                  \
  hipLaunchKernelGGL((k_place_scatter<KM, SC, TOK>), dim3(cdiv(T, TOK)), dim3(PS_THREADS), 0, st, idx, gate, \
                     expert_map, T, k, S_routed, bc, nblk, offsets, perm_token, perm_gate, inv,             \
                     (const char*)X, row_bytes, (char*)X_perm, dtype == MOE_F32, x_sq)
#define FM_PP(KM)                       \
  if (fuse && wide) FM_PS(KM, true, 32);  \
  else if (fuse) FM_PS(KM, true, 16);     \
  else if (wide) FM_PS(KM, false, 32);    \
  else FM_PS(KM, false, 16)
  FM_KSWITCH(k, FM_PP)
#undef FM_PP
#undef FM_PS
  return check_launch(what);
}

}  // namespace
}  // namespace fm

extern "C" int moe_permute(const void* X, int dtype, const int32_t* idx, const float* gate,
                           const int32_t* expert_map, int T, int d, int E, int k, int S_routed,
                           int32_t* offsets, int32_t* perm_token, float* perm_gate, int32_t* inv,
                           void* X_perm, void* ws, size_t ws_bytes, float* x_sq, void* stream) {
  clear_error();
  FM_TRY(permute_check(X, dtype, idx, gate, expert_map, T, d, E, k, S_routed, offsets, perm_token, perm_gate, inv,
                       X_perm));
  if (T > 0) FM_TRY(need(ws, "ws"));
  FM_TRY(need_aligned(ws, "ws"));
  if (ws_bytes < moe_permute_workspace_size(T, k, S_routed))
    return fail(MOE_ERR_WORKSPACE, "workspace %zu < %zu bytes", ws_bytes,
                moe_permute_workspace_size(T, k, S_routed));
  FM_TRY(need_aligned(x_sq, "x_sq"));
  return permute_launch(X, dtype, idx, gate, expert_map, T, d, E, k, S_routed, offsets, perm_token, perm_gate, inv,
                        X_perm, x_sq, (int32_t*)ws, as_stream(stream), "moe_permute", true);
}

// ------------------------------------------------- no-allocation variant ----
//
// moe_permute_noalloc keeps its count table in a file-scope device array
// instead of a caller workspace.  In host code `scratch` names a host-side
// stand-in, not device memory: its device address is looked up per device
// (hipGetSymbolAddress, on the first call on that device) and only that
// address is handed to kernels.  Every call on a device shares the array, so
// calls that overlap on one device race; each call overwrites every entry of
// the table it reads (the count kernel stores all of them), so nothing has to
// be cleared between calls.  The debug range check of moe_permute (a host copy
// and a stream synchronisation) is not run here.
namespace fm {
namespace {
constexpr size_t PERM_SCRATCH_BYTES = size_t(1) << 20;   // count tables of up to 262144 entries
}  // namespace
}  // namespace fm

static __device__ __align__(256) char scratch[fm::PERM_SCRATCH_BYTES];

namespace fm {
namespace {
constexpr int MAX_DEVICES = 64;
std::mutex g_scratch_mu;
void* g_scratch_dev[MAX_DEVICES] = {};

// Device address of `scratch` on the current device.
int scratch_address(void** out) {
  int dev = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return fail(MOE_ERR_HIP, "moe_permute_noalloc: hipGetDevice: %s", hipGetErrorString(e));
  if (dev < 0 || dev >= MAX_DEVICES) return fail(MOE_ERR_UNSUPPORTED, "moe_permute_noalloc: device %d", dev);
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  if (!g_scratch_dev[dev]) {
    void* p = nullptr;
    e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess || !p)
      return fail(MOE_ERR_HIP, "moe_permute_noalloc: hipGetSymbolAddress(scratch): %s", hipGetErrorString(e));
    g_scratch_dev[dev] = p;
  }
  *out = g_scratch_dev[dev];
  return MOE_OK;
}
}  // namespace
}  // namespace fm

extern "C" size_t moe_permute_noalloc_max_bytes(void) { return PERM_SCRATCH_BYTES; }

extern "C" int moe_permute_noalloc(const void* X, int dtype, const int32_t* idx, const float* gate,
                                   const int32_t* expert_map, int T, int d, int E, int k, int S_routed,
                                   int32_t* offsets, int32_t* perm_token, float* perm_gate, int32_t* inv,
                                   void* X_perm, float* x_sq, void* stream) {
  clear_error();
  FM_TRY(permute_check(X, dtype, idx, gate, expert_map, T, d, E, k, S_routed, offsets, perm_token, perm_gate, inv,
                       X_perm));
  const size_t need = moe_permute_workspace_size(T, k, S_routed);
  if (need > PERM_SCRATCH_BYTES)
    return fail(MOE_ERR_UNSUPPORTED,
                "moe_permute_noalloc: T=%d tokens over S_routed=%d slots need a %zu-byte count table, above its "
                "%zu-byte scratch; use moe_permute with a workspace",
                T, S_routed, need, PERM_SCRATCH_BYTES);
  FM_TRY(need_aligned(x_sq, "x_sq"));
  void* p = nullptr;
  FM_TRY(scratch_address(&p));
  return permute_launch(X, dtype, idx, gate, expert_map, T, d, E, k, S_routed, offsets, perm_token, perm_gate, inv,
                        X_perm, x_sq, (int32_t*)p, as_stream(stream), "moe_permute_noalloc", false);
}

extern "C" int moe_unpermute(const moe_layer* L, const void* O, const int32_t* inv,
                             const float* perm_gate, int T, int k, void* Y, void* stream) {
  clear_error();
  FM_TRY(check_layer(L));
  FM_TRY(check_tk(T, k));
  if (T == 0) return MOE_OK;
  FM_TRY(need(O, "O")); FM_TRY(need(inv, "inv")); FM_TRY(need(perm_gate, "perm_gate")); FM_TRY(need(Y, "Y"));
  FM_TRY(need_aligned(O, "O")); FM_TRY(need_aligned(Y, "Y"));
  hipStream_t st = as_stream(stream);
  if (debug_checks()) FM_TRY(debug_check_inv(inv, T, k, st));
  dim3 grid(cdiv(T, 4)), block(256);
#define FM_CB(KM)                                                                                 \
  if (L->dtype == MOE_BF16)                                                                       \
    hipLaunchKernelGGL((k_combine<bf16, KM>), grid, block, 0, st, (const bf16*)O, inv, perm_gate, \
                       T, k, L->d, L->S_shared, (bf16*)Y);                                        \
  else                                                                                            \
    hipLaunchKernelGGL((k_combine<float, KM>), grid, block, 0, st, (const float*)O, inv,          \
                       perm_gate, T, k, L->d, L->S_shared, (float*)Y);
  FM_KSWITCH_COMBINE(k, FM_CB)
#undef FM_CB
  return check_launch("moe_unpermute");
}

extern "C" int moe_unpermute_bwd(const moe_layer* L, const void* dY, const void* O,
                                 const int32_t* inv, const int32_t* offsets, const float* perm_gate,
                                 int T, int k, void* dO, float* dgate, float* dy_sq, void* stream) {
  clear_error();
  FM_TRY(check_layer(L));
  FM_TRY(check_tk(T, k));
  if (T == 0) return MOE_OK;
  FM_TRY(need(dY, "dY")); FM_TRY(need(inv, "inv")); FM_TRY(need(perm_gate, "perm_gate"));
  FM_TRY(need(dO, "dO"));
  if (dgate) FM_TRY(need(O, "O"));
  (void)offsets;  // rows are addressed through inv; every routed row has one owner token
  FM_TRY(need_aligned(dY, "dY")); FM_TRY(need_aligned(O, "O")); FM_TRY(need_aligned(dO, "dO"));
  FM_TRY(need_aligned(dy_sq, "dy_sq"));
  hipStream_t st = as_stream(stream);
  if (debug_checks()) {
    FM_TRY(debug_check_inv(inv, T, k, st));
    if (offsets && L->S_routed > 0) FM_TRY(debug_check_offsets(offsets, L->S_routed, T, k, st));
  }
  dim3 grid(cdiv(T, 4)), block(256);
#define FM_CBB(KM)                                                                                  \
  if (L->dtype == MOE_BF16)                                                                         \
    hipLaunchKernelGGL((k_combine_bwd<bf16, KM>), grid, block, 0, st, (const bf16*)dY,              \
                       (const bf16*)O, inv, perm_gate, T, k, L->d, L->S_shared, (bf16*)dO, dgate, dy_sq); \
  else                                                                                              \
    hipLaunchKernelGGL((k_combine_bwd<float, KM>), grid, block, 0, st, (const float*)dY,            \
                       (const float*)O, inv, perm_gate, T, k, L->d, L->S_shared, (float*)dO,       \
                       dgate, dy_sq);
  FM_KSWITCH(k, FM_CBB)
#undef FM_CBB
  return check_launch("moe_unpermute_bwd");
}

extern "C" int moe_permute_bwd(const moe_layer* L, const void* dX_perm, const int32_t* inv, int T,
                               int k, void* dX, void* stream) {
  clear_error();
  FM_TRY(check_layer(L));
  FM_TRY(check_tk(T, k));
  if (T == 0) return MOE_OK;
  FM_TRY(need(dX_perm, "dX_perm")); FM_TRY(need(inv, "inv")); FM_TRY(need(dX, "dX"));
  FM_TRY(need_aligned(dX_perm, "dX_perm")); FM_TRY(need_aligned(dX, "dX"));
  hipStream_t st = as_stream(stream);
  if (debug_checks()) FM_TRY(debug_check_inv(inv, T, k, st));
  dim3 grid(cdiv(T, 4)), block(256);
#define FM_PB(KM)                                                                                  \
  if (L->dtype == MOE_BF16)                                                                        \
    hipLaunchKernelGGL((k_permute_bwd<bf16, KM>), grid, block, 0, st, (const bf16*)dX_perm, inv,  \
                       T, k, L->d, L->S_shared, (bf16*)dX);                                        \
  else                                                                                             \
    hipLaunchKernelGGL((k_permute_bwd<float, KM>), grid, block, 0, st, (const float*)dX_perm, inv, \
                       T, k, L->d, L->S_shared, (float*)dX);
  FM_KSWITCH(k, FM_PB)
#undef FM_PB
  return check_launch("moe_permute_bwd");
}
