// Pieces of the quantised profiling pass over a stack of MoE layers
// (Section 4.1): expert matrices dequantised from their int8 rows, the
// residual stream that couples consecutive layers, and the RMS normalisation
// of the stream in front of each layer.  The int8 routing with the
// histogram, the permutation, the grouped SwiGLU forward and the combine are
// the layer's own entry points.
#include "common.hpp"

namespace fm {
namespace {

// out[r, c] = q[r, c] * scale[r], rounded once to TO; 8 codes per thread.
template <typename TO>
__global__ __launch_bounds__(256) void k_dequant_rows(const int8_t* __restrict__ q, const float* __restrict__ scale,
                                                      long rows, int cols, TO* __restrict__ out) {
  const long n8 = rows * (long)(cols / 8);
  for (long i = (long)blockIdx.x * blockDim.x + threadIdx.x; i < n8; i += (long)gridDim.x * blockDim.x) {
    const long r = i / (cols / 8);
    const long off = i * 8;
    const u32x2_t raw = *(const FM_GLOBAL u32x2_t*)(q + off);
    const float s = scale[r];
    float f[8];
#pragma unroll
    for (int j = 0; j < 8; ++j) f[j] = (float)(int8_t)((raw[j >> 2] >> (8 * (j & 3))) & 0xFF) * s;
    if constexpr (sizeof(TO) == 2) {
      st16(out + off, pack16(f, (bf16*)nullptr));
    } else {
      st16(out + off, pack16(f, (float*)nullptr));
      st16(out + off + 4, pack16(f + 4, (float*)nullptr));
    }
  }
}

// out = X + Y in fp32, one rounding to T; 16 bytes per thread and step.
template <typename T>
__global__ __launch_bounds__(256) void k_residual_add(const T* __restrict__ X, const T* __restrict__ Y, long n,
                                                      T* __restrict__ out) {
  constexpr int V = 16 / sizeof(T);
  for (long i = ((long)blockIdx.x * blockDim.x + threadIdx.x) * V; i < n; i += (long)gridDim.x * blockDim.x * V) {
    float a[V], b[V];
    unpack16(ld16(X + i), a, (T*)nullptr);
    unpack16(ld16(Y + i), b, (T*)nullptr);
#pragma unroll
    for (int j = 0; j < V; ++j) a[j] += b[j];
    st16(out + i, pack16(a, (T*)nullptr));
  }
}

// S = X (+ Y), rounded once to T (stored when out_sum is given), and
// out_norm = S / sqrt(mean(S^2) + eps) computed from the rounded S in fp32, one
// rounding.  One wave per row, four rows per block.  The lanes' sums of squares
// run over their chunks in order and are then added by a fixed butterfly, so a
// row's scale does not depend on scheduling.  The first RN_CACHE chunks of a
// lane stay in registers between the two passes; later ones (rows longer than
// RN_CACHE * 64 * 16 bytes) are read back from out_sum (the thread's own
// stores) or recomputed from X and Y.
constexpr int RN_CACHE = 16;

template <typename T>
__global__ __launch_bounds__(256) void k_rms_norm(const T* X, const T* Y, int Tn, int d, float eps, T* out_sum,
                                                  T* __restrict__ out_norm) {
  constexpr int V = 16 / sizeof(T);
  const int row = blockIdx.x * 4 + (threadIdx.x >> 6);
  if (row >= Tn) return;
  const int lane = lane_id();
  const size_t base = (size_t)row * d;
  auto sum_chunk = [&](int c) {
    float a[V];
    unpack16(ld16(X + base + c), a, (T*)nullptr);
    if (Y) {
      float b[V];
      unpack16(ld16(Y + base + c), b, (T*)nullptr);
#pragma unroll
      for (int i = 0; i < V; ++i) a[i] += b[i];
    }
    return pack16(a, (T*)nullptr);
  };
  float ss = 0.f;
  auto square = [&](const u32x4_t& sv) {
    float r[V];
    unpack16(sv, r, (T*)nullptr);
#pragma unroll
    for (int i = 0; i < V; ++i) ss = fmaf(r[i], r[i], ss);
  };
  u32x4_t cache[RN_CACHE];
#pragma unroll
  for (int i = 0; i < RN_CACHE; ++i) {
    const int c = (i * 64 + lane) * V;
    if (c < d) {
      cache[i] = sum_chunk(c);
      if (out_sum) st16(out_sum + base + c, cache[i]);
      square(cache[i]);
    }
  }
  for (int c = (RN_CACHE * 64 + lane) * V; c < d; c += 64 * V) {
    const u32x4_t sv = sum_chunk(c);
    if (out_sum) st16(out_sum + base + c, sv);
    square(sv);
  }
#pragma unroll
  for (int off = 32; off > 0; off >>= 1) ss += __shfl_xor(ss, off);
  const float ms = ss / (float)d + eps;
  const float inv = ms > 0.f ? 1.0f / sqrtf(ms) : 0.f;   // a zero row stays zero
  auto put = [&](int c, const u32x4_t& sv) {
    float r[V];
    unpack16(sv, r, (T*)nullptr);
#pragma unroll
    for (int i = 0; i < V; ++i) r[i] *= inv;
    st16(out_norm + base + c, pack16(r, (T*)nullptr));
  };
#pragma unroll
  for (int i = 0; i < RN_CACHE; ++i) {
    const int c = (i * 64 + lane) * V;
    if (c < d) put(c, cache[i]);
  }
  for (int c = (RN_CACHE * 64 + lane) * V; c < d; c += 64 * V)
    put(c, out_sum ? ld16(out_sum + base + c) : sum_chunk(c));
}

int grid_for(long work, int per_block) {
  const long b = (work + per_block - 1) / per_block;
  return (int)(b < 65536 ? (b > 0 ? b : 1) : 65536);
}

}  // namespace
}  // namespace fm

using namespace fm;

extern "C" int moe_dequant_int8(const int8_t* q, const float* scale, long rows, int cols, int out_dtype,
                                void* out, void* stream) {
  clear_error();
  FM_TRY(need_dtype_float(out_dtype, "out_dtype"));
  if (rows < 0 || cols <= 0) return fail(MOE_ERR_ARG, "rows=%ld cols=%d", rows, cols);
  if (cols % 8) return fail(MOE_ERR_UNSUPPORTED, "cols=%d not a multiple of 8", cols);
  if (rows == 0) return MOE_OK;
  FM_TRY(need(q, "q")); FM_TRY(need(scale, "scale")); FM_TRY(need(out, "out"));
  FM_TRY(need_aligned(q, "q")); FM_TRY(need_aligned(scale, "scale")); FM_TRY(need_aligned(out, "out"));
  const long work = rows * (long)(cols / 8);
  const int grid = grid_for(work, 256);
  if (out_dtype == MOE_BF16)
    hipLaunchKernelGGL(k_dequant_rows<bf16>, dim3(grid), dim3(256), 0, as_stream(stream), q, scale, rows, cols,
                       (bf16*)out);
  else
    hipLaunchKernelGGL(k_dequant_rows<float>, dim3(grid), dim3(256), 0, as_stream(stream), q, scale, rows, cols,
                       (float*)out);
  return check_launch("moe_dequant_int8");
}

extern "C" int moe_residual_add(const void* X, const void* Y, int T, int d, int dtype, void* out, void* stream) {
  clear_error();
  FM_TRY(need_dtype_float(dtype, "dtype"));
  if (T < 0 || d <= 0) return fail(MOE_ERR_ARG, "T=%d d=%d", T, d);
  if (d % 8) return fail(MOE_ERR_UNSUPPORTED, "d=%d not a multiple of 8", d);
  if (T == 0) return MOE_OK;
  FM_TRY(need(X, "X")); FM_TRY(need(Y, "Y")); FM_TRY(need(out, "out"));
  FM_TRY(need_aligned(X, "X")); FM_TRY(need_aligned(Y, "Y")); FM_TRY(need_aligned(out, "out"));
  const long n = (long)T * d;
  const int V = dtype == MOE_BF16 ? 8 : 4;
  const int grid = grid_for(n / V, 256);
  if (dtype == MOE_BF16)
    hipLaunchKernelGGL(k_residual_add<bf16>, dim3(grid), dim3(256), 0, as_stream(stream), (const bf16*)X,
                       (const bf16*)Y, n, (bf16*)out);
  else
    hipLaunchKernelGGL(k_residual_add<float>, dim3(grid), dim3(256), 0, as_stream(stream), (const float*)X,
                       (const float*)Y, n, (float*)out);
  return check_launch("moe_residual_add");
}

extern "C" int moe_rms_norm(const void* X, const void* Y, int T, int d, int dtype, float eps, void* out_sum,
                            void* out_norm, void* stream) {
  clear_error();
  FM_TRY(need_dtype_float(dtype, "dtype"));
  if (T < 0 || d <= 0) return fail(MOE_ERR_ARG, "T=%d d=%d", T, d);
  if (d % 8) return fail(MOE_ERR_UNSUPPORTED, "d=%d not a multiple of 8", d);
  if (!(eps >= 0.f && eps < 1e30f)) return fail(MOE_ERR_ARG, "eps=%g must be finite and >= 0", (double)eps);
  if (T == 0) return MOE_OK;
  FM_TRY(need(X, "X")); FM_TRY(need(out_norm, "out_norm"));
  if (out_norm == X || (Y && out_norm == Y) || (out_sum && out_norm == out_sum))
    return fail(MOE_ERR_ARG, "out_norm must not alias X, Y or out_sum");
  FM_TRY(need_aligned(X, "X")); FM_TRY(need_aligned(Y, "Y")); FM_TRY(need_aligned(out_sum, "out_sum"));
  FM_TRY(need_aligned(out_norm, "out_norm"));
  const dim3 grid(cdiv(T, 4)), block(256);
  if (dtype == MOE_BF16)
    hipLaunchKernelGGL(k_rms_norm<bf16>, grid, block, 0, as_stream(stream), (const bf16*)X, (const bf16*)Y, T, d,
                       eps, (bf16*)out_sum, (bf16*)out_norm);
  else
    hipLaunchKernelGGL(k_rms_norm<float>, grid, block, 0, as_stream(stream), (const float*)X, (const float*)Y, T,
                       d, eps, (float*)out_sum, (float*)out_norm);
  return check_launch("moe_rms_norm");
}
