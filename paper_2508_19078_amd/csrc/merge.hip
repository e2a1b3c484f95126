// Expert merging: the frequency merge plan, the per-slot weight tables of a
// merged layer, and the importance-weighted merge of Eq. 2 (Section 5.3).
#include "common.hpp"

namespace fm {
namespace {

// One block (E <= 256 threads, one per expert).  The rank of expert e under
// (count desc, index asc) is the number of experts that rank before it.
__global__ __launch_bounds__(256) void k_merge_plan(
    const int32_t* __restrict__ counts, int E, int n_merge, int group, float total,
    int expert_base, int grp_base, int member_base, int32_t* __restrict__ expert_map,
    int32_t* __restrict__ slot_src, int32_t* __restrict__ grp_ptr,
    int32_t* __restrict__ grp_member, float* __restrict__ alpha) {
  __shared__ int c[256];
  const int e = threadIdx.x;
  if (e < E) c[e] = counts[e];
  __syncthreads();
  const int K = E - n_merge, G = n_merge / group;
  if (e < E) {
    const int ce = c[e];
    int r = 0;
    for (int o = 0; o < E; ++o) r += (c[o] > ce) || (c[o] == ce && o < e);
    int slot;
    if (r < K) {
      slot = r;
      slot_src[r] = e;
    } else {
      const int a = E - 1 - r;          // 0 = least activated
      slot = K + a / group;
      grp_member[member_base + a] = expert_base + e;
    }
    expert_map[e] = slot;
    alpha[expert_base + e] = (float)ce / total;
  }
  for (int g = threadIdx.x; g <= G; g += blockDim.x) {
    grp_ptr[grp_base + g] = member_base + g * group;
    if (g < G) slot_src[K + g] = E + g;
  }
}

__global__ void k_frequency(const int32_t* __restrict__ counts, int E, float total,
                            float* __restrict__ freq) {
  const int e = blockIdx.x * blockDim.x + threadIdx.x;
  if (e < E) freq[e] = (float)counts[e] / total;
}

__global__ void k_slot_pointers(const int32_t* __restrict__ slot_src, int S, int E,
                                size_t mat_bytes, const char* og, const char* ou,
                                const char* od, const char* mg, const char* mu, const char* md,
                                const void** wg, const void** wu, const void** wd) {
  const int s = blockIdx.x * blockDim.x + threadIdx.x;
  if (s >= S) return;
  const int src = slot_src[s];
  if (src < E) {
    wg[s] = og + (size_t)src * mat_bytes;
    wu[s] = ou + (size_t)src * mat_bytes;
    wd[s] = od + (size_t)src * mat_bytes;
  } else {
    wg[s] = mg + (size_t)(src - E) * mat_bytes;
    wu[s] = mu + (size_t)(src - E) * mat_bytes;
    wd[s] = md + (size_t)(src - E) * mat_bytes;
  }
}

constexpr int MG_UNROLL = 2;     // 16-byte chunks per thread and iteration

// grid.y = 3*G (group, matrix); grid.x strides over the matrix in 16-byte chunks.
// The group's members, pointers and coefficients are block-uniform loads.
template <typename TI, typename TO>
__global__ __launch_bounds__(256) void k_merge(const void* const* __restrict__ w_src,
                                               const int32_t* __restrict__ grp_ptr,
                                               const int32_t* __restrict__ grp_member,
                                               const float* __restrict__ alpha,
                                               void* const* __restrict__ w_dst, size_t n_elem) {
  constexpr int VI = 16 / sizeof(TI);          // input elements per 16 bytes
  const int g = blockIdx.y / 3, mat = blockIdx.y - 3 * (blockIdx.y / 3);
  const int m0 = grp_ptr[g], nm = grp_ptr[g + 1] - m0;
  float tot = 0.f;
  for (int i = 0; i < nm; ++i) tot += alpha[grp_member[m0 + i]];
  char* dst = (char*)w_dst[3 * g + mat];
  const size_t nchunk = n_elem / VI;
  const size_t stride = (size_t)gridDim.x * blockDim.x * MG_UNROLL;
  for (size_t c0 = (size_t)blockIdx.x * blockDim.x * MG_UNROLL + threadIdx.x; c0 < nchunk;
       c0 += stride) {
    float acc[MG_UNROLL][VI];
#pragma unroll
    for (int u = 0; u < MG_UNROLL; ++u)
#pragma unroll
      for (int i = 0; i < VI; ++i) acc[u][i] = 0.f;
    for (int m = 0; m < nm; ++m) {
      const int e = grp_member[m0 + m];
      const float cm = tot > 0.f ? alpha[e] / tot : 1.0f / (float)nm;
      const char* src = (const char*)w_src[3 * e + mat];
      u32x4_t v[MG_UNROLL];
#pragma unroll
      for (int u = 0; u < MG_UNROLL; ++u) {
        const size_t c = c0 + (size_t)u * blockDim.x;
        v[u] = c < nchunk ? ld16(src + c * 16) : u32x4_t{0, 0, 0, 0};
      }
#pragma unroll
      for (int u = 0; u < MG_UNROLL; ++u) {
        float f[VI];
        unpack16(v[u], f, (TI*)nullptr);
#pragma unroll
        for (int i = 0; i < VI; ++i) acc[u][i] = fmaf(cm, f[i], acc[u][i]);
      }
    }
#pragma unroll
    for (int u = 0; u < MG_UNROLL; ++u) {
      const size_t c = c0 + (size_t)u * blockDim.x;
      if (c >= nchunk) continue;
      if (sizeof(TO) == sizeof(TI)) {
        st16(dst + c * 16, pack16(acc[u], (TO*)nullptr));
      } else if (sizeof(TO) == 4) {   // bf16 in, fp32 out: 8 floats = 32 bytes
        st16(dst + c * 32, pack16(acc[u], (float*)nullptr));
        st16(dst + c * 32 + 16, pack16(acc[u] + 4, (float*)nullptr));
      } else {                        // fp32 in, bf16 out: 4 values = 8 bytes
        uint2 o;
        o.x = pk_bf16(acc[u][0], acc[u][1]);
        o.y = pk_bf16(acc[u][2], acc[u][3]);
        *reinterpret_cast<uint2*>(dst + c * 8) = o;
      }
    }
  }
}

}  // namespace
}  // namespace fm

using namespace fm;

extern "C" int moe_merge_plan(const int32_t* counts, int E, int n_merge, int group,
                              float total_tokens, int expert_base, int grp_base, int member_base,
                              int32_t* expert_map, int32_t* slot_src, int32_t* grp_ptr,
                              int32_t* grp_member, float* alpha, void* stream) {
  clear_error();
  if (E <= 0 || E > 256) return fail(MOE_ERR_UNSUPPORTED, "E=%d outside [1, 256]", E);
  if (group <= 0 || n_merge < 0 || n_merge > E || n_merge % group)
    return fail(MOE_ERR_ARG, "n_merge=%d group=%d (E=%d)", n_merge, group, E);
  if (!(total_tokens > 0.f)) return fail(MOE_ERR_ARG, "total_tokens must be > 0");
  if (expert_base < 0 || grp_base < 0 || member_base < 0) return fail(MOE_ERR_ARG, "negative base");
  FM_TRY(need(counts, "counts")); FM_TRY(need(expert_map, "expert_map"));
  FM_TRY(need(slot_src, "slot_src")); FM_TRY(need(grp_ptr, "grp_ptr"));
  FM_TRY(need(alpha, "alpha"));
  if (n_merge > 0) FM_TRY(need(grp_member, "grp_member"));
  hipLaunchKernelGGL(k_merge_plan, dim3(1), dim3(256), 0, as_stream(stream), counts, E, n_merge,
                     group, total_tokens, expert_base, grp_base, member_base, expert_map, slot_src,
                     grp_ptr, grp_member, alpha);
  return check_launch("moe_merge_plan");
}

extern "C" int moe_activation_frequency(const int32_t* counts, int E, float total_tokens, float* freq,
                                        void* stream) {
  clear_error();
  if (E <= 0) return fail(MOE_ERR_ARG, "E=%d", E);
  if (!(total_tokens > 0.f)) return fail(MOE_ERR_ARG, "total_tokens must be > 0");
  FM_TRY(need(counts, "counts")); FM_TRY(need(freq, "freq"));
  hipLaunchKernelGGL(k_frequency, dim3(cdiv(E, 256)), dim3(256), 0, as_stream(stream), counts, E,
                     total_tokens, freq);
  return check_launch("moe_activation_frequency");
}

extern "C" int moe_slot_pointers(const int32_t* slot_src, int S, int E, int d, int I, int dtype,
                                 const void* og, const void* ou, const void* od, const void* mg,
                                 const void* mu, const void* md, const void** wg, const void** wu,
                                 const void** wd, void* stream) {
  clear_error();
  if (S <= 0 || S > 512 || E <= 0 || d <= 0 || I <= 0)
    return fail(MOE_ERR_ARG, "S=%d E=%d d=%d I=%d", S, E, d, I);
  FM_TRY(need_dtype_float(dtype, "dtype"));
  FM_TRY(need(slot_src, "slot_src")); FM_TRY(need(og, "orig_gate")); FM_TRY(need(ou, "orig_up"));
  FM_TRY(need(od, "orig_down")); FM_TRY(need(wg, "w_gate")); FM_TRY(need(wu, "w_up"));
  FM_TRY(need(wd, "w_down"));
  const size_t mat_bytes = (size_t)d * I * esize(dtype);
  hipLaunchKernelGGL(k_slot_pointers, dim3(cdiv(S, 256)), dim3(256), 0, as_stream(stream),
                     slot_src, S, E, mat_bytes, (const char*)og, (const char*)ou, (const char*)od,
                     (const char*)mg, (const char*)mu, (const char*)md, wg, wu, wd);
  return check_launch("moe_slot_pointers");
}

extern "C" int moe_merge_experts(const void* const* w_src, int dtype, int d, int I, int G,
                                 const int32_t* grp_ptr, const int32_t* grp_member,
                                 const float* alpha, void* const* w_dst, int out_dtype,
                                 void* stream) {
  clear_error();
  if (d <= 0 || I <= 0 || G < 0) return fail(MOE_ERR_ARG, "d=%d I=%d G=%d", d, I, G);
  if (d % 8 || I % 8) return fail(MOE_ERR_UNSUPPORTED, "d=%d and I=%d must be multiples of 8", d, I);
  if (G > 65535 / 3) return fail(MOE_ERR_UNSUPPORTED, "G=%d too many groups", G);
  FM_TRY(need_dtype_float(dtype, "dtype"));
  FM_TRY(need_dtype_float(out_dtype, "out_dtype"));
  if (G == 0) return MOE_OK;
  FM_TRY(need(w_src, "w_src")); FM_TRY(need(grp_ptr, "grp_ptr")); FM_TRY(need(grp_member, "grp_member"));
  FM_TRY(need(alpha, "alpha")); FM_TRY(need(w_dst, "w_dst"));
  const size_t n_elem = (size_t)d * I;
  const int vi = 16 / esize(dtype);
  const size_t nchunk = n_elem / vi;
  int bx = cdiv((long)nchunk, 256L * MG_UNROLL);
  if (bx > 1024) bx = 1024;
  dim3 grid(bx, 3 * G), block(256);
  hipStream_t st = as_stream(stream);
#define FM_MG(TI, TO) \
  hipLaunchKernelGGL((k_merge<TI, TO>), grid, block, 0, st, w_src, grp_ptr, grp_member, alpha, w_dst, n_elem)
  if (dtype == MOE_BF16 && out_dtype == MOE_BF16) FM_MG(bf16, bf16);
  else if (dtype == MOE_BF16) FM_MG(bf16, float);
  else if (out_dtype == MOE_F32) FM_MG(float, float);
  else FM_MG(float, bf16);
#undef FM_MG
  return check_launch("moe_merge_experts");
}
