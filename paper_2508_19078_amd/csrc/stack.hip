// Pieces of the quantised profiling pass over a stack of MoE layers
// (Section 4.1): expert matrices dequantised from their int8 rows, and the
// residual stream that couples consecutive layers.  The int8 routing with the
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
