// Router (softmax top-k gate), int8 router quantiser and the activation
// histogram of the int8 profiling router.
//
// One kernel serves both the full-precision router and the int8 profiling
// router: a block owns 32 tokens, its four waves split the hidden dimension
// into interleaved 16-byte-per-lane chunks and accumulate the token x expert
// logits on MFMA (16x16x32 bf16, or 16x16x4 fp32 for fp32 inputs).  The four
// partial sums are added in a fixed order in LDS, so the logits do not depend
// on scheduling.  Then one lane per token selects the top k by
// (logit desc, index asc) with an unrolled insertion list, and either writes
// idx/gate or adds the selection to an LDS histogram that is flushed to the
// global counts with one integer atomic per expert and block.
#include "common.hpp"

namespace fm {
namespace {

constexpr int RT_TOK = 32;      // tokens per block
constexpr int RT_WAVES = 4;     // waves per block, splitting d

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
  uint2 raw = ok ? *reinterpret_cast<const uint2*>(p) : make_uint2(0, 0);
  u32x4_t v;
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    uint32_t w = i < 2 ? raw.x : raw.y;
    int sh = (i & 1) * 16;
    float lo = (float)(int8_t)((w >> sh) & 0xFF);
    float hi = (float)(int8_t)((w >> (sh + 8)) & 0xFF);
    v[i] = (__float_as_uint(lo) >> 16) | (__float_as_uint(hi) & 0xFFFF0000u);
  }
  return __builtin_bit_cast(bf16x8_t, v);
}
__device__ __forceinline__ f32x4_t load_w_frag(const int8_t* p, bool ok, f32x4_t) {
  uint32_t raw = ok ? *reinterpret_cast<const uint32_t*>(p) : 0u;
  f32x4_t v;
#pragma unroll
  for (int i = 0; i < 4; ++i) v[i] = (float)(int8_t)((raw >> (8 * i)) & 0xFF);
  return v;
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

// MODE 0: write idx/gate (+logits).  MODE 1: histogram (+idx).
template <typename TX, typename TW, int NE, int KMAX, int MODE>
__global__ __launch_bounds__(256) void k_route(
    const TX* __restrict__ X, const TW* __restrict__ W, const float* __restrict__ wscale,
    const float* __restrict__ bias, int T, int d, int E, int k,
    int32_t* __restrict__ idx, float* __restrict__ gate, float* __restrict__ logits,
    int32_t* __restrict__ counts) {
  constexpr int V = 16 / sizeof(TX);           // elements per lane per chunk
  constexpr int KC = 4 * V;                    // hidden columns per chunk
  constexpr int EP = NE * 16 + 1;              // padded LDS row
  typedef typename fragv<V>::type frag_t;
  __shared__ float red[RT_TOK * EP];
  __shared__ int hist[NE * 16];

  const int lane = lane_id();
  const int wave = threadIdx.x >> 6;
  const int t0 = blockIdx.x * RT_TOK;
  const int r16 = lane & 15, q4 = lane >> 4;

  if (MODE == 1)
    for (int e = threadIdx.x; e < NE * 16; e += blockDim.x) hist[e] = 0;

  f32x4_t acc[2][NE];
#pragma unroll
  for (int r = 0; r < 2; ++r)
#pragma unroll
    for (int j = 0; j < NE; ++j) acc[r][j] = f32x4_t{0, 0, 0, 0};

  const int nchunks = d / KC;
  const int tail = d - nchunks * KC;           // multiple of 8 (d % 8 == 0)
  const TX* xrow[2];
  bool xok[2];
#pragma unroll
  for (int r = 0; r < 2; ++r) {
    int t = t0 + r * 16 + r16;
    xok[r] = t < T;
    xrow[r] = X + (size_t)(xok[r] ? t : 0) * d;
  }
  const TW* wrow[NE];
  bool wok[NE];
#pragma unroll
  for (int j = 0; j < NE; ++j) {
    int e = j * 16 + r16;
    wok[j] = e < E;
    wrow[j] = W + (size_t)(wok[j] ? e : 0) * d;
  }

  auto chunk = [&](int c0, bool full) {
    int col = c0 + q4 * V;
    bool cok = full || col < d;
    frag_t a[2], b[NE];
#pragma unroll
    for (int r = 0; r < 2; ++r) a[r] = load_x_frag(xrow[r] + col, xok[r] && cok);
#pragma unroll
    for (int j = 0; j < NE; ++j) b[j] = load_w_frag(wrow[j] + col, wok[j] && cok, frag_t{});
#pragma unroll
    for (int r = 0; r < 2; ++r)
#pragma unroll
      for (int j = 0; j < NE; ++j) acc[r][j] = mma(a[r], b[j], acc[r][j]);
  };

  int c = wave;
  for (; c + 3 * RT_WAVES < nchunks; c += 4 * RT_WAVES) {
    chunk(c * KC, true);
    chunk((c + RT_WAVES) * KC, true);
    chunk((c + 2 * RT_WAVES) * KC, true);
    chunk((c + 3 * RT_WAVES) * KC, true);
  }
  for (; c < nchunks; c += RT_WAVES) chunk(c * KC, true);
  if (tail > 0 && wave == nchunks % RT_WAVES) chunk(nchunks * KC, false);

  // fixed-order reduction of the four partial sums: ((p0 + p1) + p2) + p3
  for (int w = 0; w < RT_WAVES; ++w) {
    if (wave == w) {
#pragma unroll
      for (int r = 0; r < 2; ++r)
#pragma unroll
        for (int j = 0; j < NE; ++j)
#pragma unroll
          for (int i = 0; i < 4; ++i) {
            // MFMA output: row (token) 4*q4 + i, column (expert) r16
            float* p = &red[(r * 16 + 4 * q4 + i) * EP + j * 16 + r16];
            *p = (w == 0) ? acc[r][j][i] : *p + acc[r][j][i];
          }
    }
    __syncthreads();
  }

  // finalise logits: scale (int8 router) and bias
  for (int i = threadIdx.x; i < RT_TOK * E; i += blockDim.x) {
    int tl = i / E, e = i - tl * E;
    float v = red[tl * EP + e];
    if (wscale) v *= wscale[e];
    if (bias) v += bias[e];
    red[tl * EP + e] = v;
    if (MODE == 0 && logits && t0 + tl < T) logits[(size_t)(t0 + tl) * E + e] = v;
  }
  __syncthreads();

  // one lane per token: top-k by (value desc, index asc)
  const int tl = wave * 8 + (lane & 7);
  if (lane < 8 && t0 + tl < T) {
    float bv[KMAX];
    int bi[KMAX];
#pragma unroll
    for (int j = 0; j < KMAX; ++j) { bv[j] = -INFINITY; bi[j] = 0x7FFFFFFF; }
    const float* row = &red[tl * EP];
    for (int e = 0; e < E; ++e) {
      float v = row[e] + 0.0f;                  // -0.0 -> +0.0
      int ie = e;
#pragma unroll
      for (int j = 0; j < KMAX; ++j) {
        if (j < k && ranks_before(v, ie, bv[j], bi[j])) {
          float tv = bv[j]; int ti = bi[j];
          bv[j] = v; bi[j] = ie;
          v = tv; ie = ti;
        }
      }
    }
    const size_t t = (size_t)(t0 + tl);
    if (MODE == 0) {
      float s = 0.f, g[KMAX];
#pragma unroll
      for (int j = 0; j < KMAX; ++j) {
        g[j] = (j < k) ? expf(bv[j] - bv[0]) : 0.f;
        s += g[j];
      }
      float inv = 1.0f / s;
#pragma unroll
      for (int j = 0; j < KMAX; ++j)
        if (j < k) {
          idx[t * k + j] = bi[j];
          gate[t * k + j] = g[j] * inv;
        }
    } else {
#pragma unroll
      for (int j = 0; j < KMAX; ++j)
        if (j < k) {
          atomicAdd(&hist[bi[j]], 1);
          if (idx) idx[t * k + j] = bi[j];
        }
    }
  }
  if (MODE == 1) {
    __syncthreads();
    for (int e = threadIdx.x; e < E; e += blockDim.x)
      if (hist[e]) atomicAdd(&counts[e], hist[e]);
  }
}

// Per-row symmetric int8 quantiser: one wave per row.
template <typename T>
__global__ __launch_bounds__(256) void k_quantize(const T* __restrict__ W, int E, int d,
                                                  int8_t* __restrict__ q, float* __restrict__ s) {
  const int row = blockIdx.x * 4 + (threadIdx.x >> 6);
  const int lane = lane_id();
  if (row >= E) return;
  const T* w = W + (size_t)row * d;
  float m = 0.f;
  for (int i = lane; i < d; i += 64) m = fmaxf(m, fabsf(to_float(w[i])));
#pragma unroll
  for (int off = 32; off > 0; off >>= 1) m = fmaxf(m, __shfl_xor(m, off));
  const float sc = m / 127.0f;
  if (lane == 0) s[row] = sc;
  for (int i = lane; i < d; i += 64) {
    int v = 0;
    if (sc > 0.f) {
      float r = rintf(to_float(w[i]) / sc);
      v = (int)fminf(fmaxf(r, -127.f), 127.f);
    }
    q[(size_t)row * d + i] = (int8_t)v;
  }
}

template <typename TX, typename TW, int MODE>
int launch_route(const TX* X, const TW* W, const float* ws, const float* bias, int T, int d,
                 int E, int k, int32_t* idx, float* gate, float* logits, int32_t* counts,
                 hipStream_t st) {
  dim3 grid(cdiv(T, RT_TOK)), block(256);
  const int ne = cdiv(E, 16);
#define FM_RT(NE, KM)                                                                  \
  hipLaunchKernelGGL((k_route<TX, TW, NE, KM, MODE>), grid, block, 0, st, X, W, ws, bias, \
                     T, d, E, k, idx, gate, logits, counts)
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
  return check_launch(MODE == 0 ? "moe_route_topk" : "moe_profile_hist");
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
  FM_TRY(need(X, "X")); FM_TRY(need(Wr, "Wr")); FM_TRY(need(idx, "idx")); FM_TRY(need(gate, "gate"));
  FM_TRY(need_aligned(X, "X")); FM_TRY(need_aligned(Wr, "Wr")); FM_TRY(need_aligned(bias, "bias"));
  FM_TRY(need_aligned(idx, "idx")); FM_TRY(need_aligned(gate, "gate")); FM_TRY(need_aligned(logits, "logits"));
  if (T == 0) return MOE_OK;
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
  FM_TRY(need(X, "X")); FM_TRY(need(Wq, "Wq")); FM_TRY(need(scale, "scale")); FM_TRY(need(counts, "counts"));
  FM_TRY(need_aligned(X, "X")); FM_TRY(need_aligned(Wq, "Wq")); FM_TRY(need_aligned(scale, "scale"));
  FM_TRY(need_aligned(bias, "bias")); FM_TRY(need_aligned(counts, "counts")); FM_TRY(need_aligned(idx, "idx"));
  if (T == 0) return MOE_OK;
  hipStream_t st = as_stream(stream);
  if (x_dtype == MOE_BF16)
    return launch_route<bf16, int8_t, 1>((const bf16*)X, Wq, scale, bias, T, d, E, k, idx, nullptr,
                                         nullptr, counts, st);
  return launch_route<float, int8_t, 1>((const float*)X, Wq, scale, bias, T, d, E, k, idx, nullptr,
                                        nullptr, counts, st);
}
