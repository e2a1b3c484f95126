// Grouped SwiGLU expert FFN, forward and backward, over the slots of a layer.
//
// Rows of slot s live in the per-row buffers at the slot's row range (routed:
// [offsets[s], offsets[s+1]) read from device memory; shared expert i:
// [T*k + i*T, T*k + (i+1)*T)).  A one-block kernel turns the offsets into a
// list of (slot, first row) M-tiles of 128 rows; the GEMM grids are sized by
// the host-side upper bound of that list and surplus blocks exit at once, so
// the host never waits for the bucket sizes.
//
// forward   gate_up : [A_g | A_u] = X_s [W_gate | W_up]^T, epilogue H = silu(A_g) A_u
//           down    : O = H W_down^T
// backward  dh      : dH = dO W_down, epilogue dA_g, dA_u (dSwiGLU)
//           dx      : dX_s = dA_g W_gate + dA_u W_up            (K = 2I in two passes)
//           dw_gu   : dW_gate = dA_g^T X_s, dW_up = dA_u^T X_s  (tuning slots)
//           dw_d    : dW_down = dO^T H                          (tuning slots)
#include "gemm_bf16.hpp"

namespace fm {
namespace {

struct SlotRows {
  int s;        // slot
  int m0;       // first row of this tile within the slot
  int nrows;    // rows of the slot
  long orow0;   // first row of the slot in the per-row buffers
  long xrow0;   // first row of the slot's input in X_perm (routed) or X (shared)
  bool shared;
};

__device__ __forceinline__ SlotRows slot_rows(int s, int m0, const int32_t* offsets, int S_r, int Tn,
                                              int k) {
  SlotRows r;
  r.s = s;
  r.m0 = m0;
  if (s < S_r) {
    const int b = offsets[s];
    r.nrows = offsets[s + 1] - b;
    r.orow0 = b;
    r.xrow0 = b;
    r.shared = false;
  } else {
    r.nrows = Tn;
    r.orow0 = (long)Tn * k + (long)(s - S_r) * Tn;
    r.xrow0 = 0;
    r.shared = true;
  }
  return r;
}

// tiles[0].x = number of tiles; tiles[1 + i] = (slot, first row).
__global__ __launch_bounds__(1024) void k_build_tiles(const int32_t* __restrict__ offsets, int S_r,
                                                      int S_sh, int Tn, int bm, int2* __restrict__ tiles) {
  __shared__ int base[1025];
  const int S = S_r + S_sh;
  const int s = threadIdx.x;
  int n = 0;
  if (s < S) n = s < S_r ? offsets[s + 1] - offsets[s] : Tn;
  const int nt = (n + bm - 1) / bm;
  base[s + 1] = nt;
  if (s == 0) base[0] = 0;
  __syncthreads();
  if (threadIdx.x == 0)
    for (int i = 1; i <= (int)blockDim.x; ++i) base[i] += base[i - 1];
  __syncthreads();
  if (s < S)
    for (int t = 0; t < nt; ++t) tiles[1 + base[s] + t] = make_int2(s, t * bm);
  if (threadIdx.x == 0) tiles[0] = make_int2(base[blockDim.x], 0);
}

template <typename T> struct LayerPtrs {
  const T* const* wg;
  const T* const* wu;
  const T* const* wd;
  float* const* dwg;
  float* const* dwu;
  float* const* dwd;
};

template <typename T> LayerPtrs<T> layer_ptrs(const moe_layer* L) {
  return LayerPtrs<T>{(const T* const*)L->w_gate, (const T* const*)L->w_up, (const T* const*)L->w_down,
                      L->dw_gate, L->dw_up, L->dw_down};
}

__device__ __forceinline__ float sigm(float z) { return 1.0f / (1.0f + expf(-z)); }

// ------------------------------------------------------------- forward ----

template <typename T>
__global__ __launch_bounds__(G_THREADS) void k_gate_up(LayerPtrs<T> W, const T* __restrict__ X,
                                                       const T* __restrict__ Xp,
                                                       const int32_t* __restrict__ offsets,
                                                       const int2* __restrict__ tiles, int S_r, int Tn,
                                                       int k, int d, int I, T* __restrict__ Ag,
                                                       T* __restrict__ Au, T* __restrict__ H) {
  __shared__ __align__(16) char lds[LdsBytes<T, 1, 2>::value];
  if ((int)blockIdx.y >= tiles[0].x) return;
  const int2 tl = tiles[1 + blockIdx.y];
  const SlotRows sr = slot_rows(tl.x, tl.y, offsets, S_r, Tn, k);
  const int n0 = blockIdx.x * G_BN;
  const T* xs = (sr.shared ? X : Xp) + (size_t)(sr.xrow0 + sr.m0) * d;
  Opnd<T> A[1] = {{xs, d, sr.nrows - sr.m0, d}};
  Opnd<T> B[2] = {{W.wg[sr.s] + (size_t)n0 * d, d, I - n0, d}, {W.wu[sr.s] + (size_t)n0 * d, d, I - n0, d}};
  Acc<T, 1, 2> acc;
  acc.zero();
  run_gemm<T, true, true, 1, 2>(A, B, d, lds, acc);
  const size_t ob = (size_t)(sr.orow0 + sr.m0);
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const AccCoord c = acc_coord(i, j);
      const int n = n0 + c.col4;
      if (c.row >= sr.nrows - sr.m0 || n >= I) continue;
      const f32x4_t g = acc.v[0][i][j], u = acc.v[1][i][j];
      f32x4_t h;
#pragma unroll
      for (int r = 0; r < 4; ++r) h[r] = g[r] * sigm(g[r]) * u[r];
      const size_t o = (ob + c.row) * I + n;
      store4(Ag + o, g);
      store4(Au + o, u);
      store4(H + o, h);
    }
}

template <typename T>
__global__ __launch_bounds__(G_THREADS) void k_down(LayerPtrs<T> W, const T* __restrict__ H,
                                                    const int32_t* __restrict__ offsets,
                                                    const int2* __restrict__ tiles, int S_r, int Tn,
                                                    int k, int d, int I, T* __restrict__ O) {
  __shared__ __align__(16) char lds[LdsBytes<T, 1, 1>::value];
  if ((int)blockIdx.y >= tiles[0].x) return;
  const int2 tl = tiles[1 + blockIdx.y];
  const SlotRows sr = slot_rows(tl.x, tl.y, offsets, S_r, Tn, k);
  const int n0 = blockIdx.x * G_BN;
  const size_t ob = (size_t)(sr.orow0 + sr.m0);
  Opnd<T> A[1] = {{H + ob * I, I, sr.nrows - sr.m0, I}};
  Opnd<T> B[1] = {{W.wd[sr.s] + (size_t)n0 * I, I, d - n0, I}};
  Acc<T, 1, 1> acc;
  acc.zero();
  run_gemm<T, true, true, 1, 1>(A, B, I, lds, acc);
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const AccCoord c = acc_coord(i, j);
      const int n = n0 + c.col4;
      if (c.row >= sr.nrows - sr.m0 || n >= d) continue;
      store4(O + (ob + c.row) * d + n, acc.v[0][i][j]);
    }
}

// ------------------------------------------------------------ backward ----

template <typename T>
__global__ __launch_bounds__(G_THREADS) void k_dh(LayerPtrs<T> W, const T* __restrict__ dO,
                                                  const T* __restrict__ Ag, const T* __restrict__ Au,
                                                  const int32_t* __restrict__ offsets,
                                                  const int2* __restrict__ tiles, int S_r, int Tn, int k,
                                                  int d, int I, T* __restrict__ dAg, T* __restrict__ dAu) {
  __shared__ __align__(16) char lds[LdsBytes<T, 1, 1>::value];
  if ((int)blockIdx.y >= tiles[0].x) return;
  const int2 tl = tiles[1 + blockIdx.y];
  const SlotRows sr = slot_rows(tl.x, tl.y, offsets, S_r, Tn, k);
  const int n0 = blockIdx.x * G_BN;
  const size_t ob = (size_t)(sr.orow0 + sr.m0);
  // B(n = intermediate index, k = hidden index) = W_down[k][n]: MN-contiguous
  Opnd<T> A[1] = {{dO + ob * d, d, sr.nrows - sr.m0, d}};
  Opnd<T> B[1] = {{W.wd[sr.s] + n0, I, I - n0, d}};
  Acc<T, 1, 1> acc;
  acc.zero();
  run_gemm<T, true, false, 1, 1>(A, B, d, lds, acc);
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const AccCoord c = acc_coord(i, j);
      const int n = n0 + c.col4;
      if (c.row >= sr.nrows - sr.m0 || n >= I) continue;
      const size_t o = (ob + c.row) * I + n;
      const f32x4_t dh = acc.v[0][i][j], g = load4(Ag + o), u = load4(Au + o);
      f32x4_t dg, du;
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const float s = sigm(g[r]);
        du[r] = dh[r] * g[r] * s;
        dg[r] = dh[r] * u[r] * s * (1.0f + g[r] * (1.0f - s));
      }
      store4(dAg + o, dg);
      store4(dAu + o, du);
    }
}

template <typename T>
__global__ __launch_bounds__(G_THREADS) void k_dx(LayerPtrs<T> W, const T* __restrict__ dAg,
                                                  const T* __restrict__ dAu,
                                                  const int32_t* __restrict__ offsets,
                                                  const int2* __restrict__ tiles, int S_r, int Tn, int k,
                                                  int d, int I, T* __restrict__ dXp) {
  __shared__ __align__(16) char lds[LdsBytes<T, 1, 1>::value];
  if ((int)blockIdx.y >= tiles[0].x) return;
  const int2 tl = tiles[1 + blockIdx.y];
  const SlotRows sr = slot_rows(tl.x, tl.y, offsets, S_r, Tn, k);
  const int n0 = blockIdx.x * G_BN;
  const size_t ob = (size_t)(sr.orow0 + sr.m0);
  Acc<T, 1, 1> acc;
  acc.zero();
  {  // B(n = hidden index, k = intermediate index) = W_gate[k][n]
    Opnd<T> A[1] = {{dAg + ob * I, I, sr.nrows - sr.m0, I}};
    Opnd<T> B[1] = {{W.wg[sr.s] + n0, d, d - n0, I}};
    run_gemm<T, true, false, 1, 1>(A, B, I, lds, acc);
  }
  {
    Opnd<T> A[1] = {{dAu + ob * I, I, sr.nrows - sr.m0, I}};
    Opnd<T> B[1] = {{W.wu[sr.s] + n0, d, d - n0, I}};
    run_gemm<T, true, false, 1, 1>(A, B, I, lds, acc);
  }
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const AccCoord c = acc_coord(i, j);
      const int n = n0 + c.col4;
      if (c.row >= sr.nrows - sr.m0 || n >= d) continue;
      store4(dXp + (ob + c.row) * d + n, acc.v[0][i][j]);
    }
}

__device__ __forceinline__ void store_dw(float* p, f32x4_t v, bool accumulate) {
  if (accumulate) v = v + load4(p);
  store4(p, v);
}

// grid (d / 128 column tiles, I / 128 row tiles, slots)
template <typename T>
__global__ __launch_bounds__(G_THREADS) void k_dw_gu(LayerPtrs<T> W, const T* __restrict__ X,
                                                     const T* __restrict__ Xp, const T* __restrict__ dAg,
                                                     const T* __restrict__ dAu,
                                                     const int32_t* __restrict__ offsets, int S_r, int Tn,
                                                     int k, int d, int I, int accumulate) {
  __shared__ __align__(16) char lds[LdsBytes<T, 2, 1>::value];
  const int s = blockIdx.z;
  float* dwg = W.dwg[s];
  float* dwu = W.dwu[s];
  if (!dwg || !dwu) return;
  const SlotRows sr = slot_rows(s, 0, offsets, S_r, Tn, k);
  const int n0 = blockIdx.x * G_BN, m0 = blockIdx.y * G_BM;
  // A(m = intermediate index, k = row) = dA[row][m];  B(n = hidden index, k = row) = X_s[row][n]
  Opnd<T> A[2] = {{dAg + (size_t)sr.orow0 * I + m0, I, I - m0, sr.nrows},
                  {dAu + (size_t)sr.orow0 * I + m0, I, I - m0, sr.nrows}};
  Opnd<T> B[1] = {{(sr.shared ? X : Xp) + (size_t)sr.xrow0 * d + n0, d, d - n0, sr.nrows}};
  Acc<T, 2, 1> acc;
  acc.zero();
  run_gemm<T, false, false, 2, 1>(A, B, sr.nrows, lds, acc);
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const AccCoord c = acc_coord(i, j);
      const int m = m0 + c.row, n = n0 + c.col4;
      if (m >= I || n >= d) continue;
      store_dw(dwg + (size_t)m * d + n, acc.v[0][i][j], accumulate);
      store_dw(dwu + (size_t)m * d + n, acc.v[1][i][j], accumulate);
    }
}

// grid (I / 128 column tiles, d / 128 row tiles, slots)
template <typename T>
__global__ __launch_bounds__(G_THREADS) void k_dw_d(LayerPtrs<T> W, const T* __restrict__ dO,
                                                    const T* __restrict__ H,
                                                    const int32_t* __restrict__ offsets, int S_r, int Tn,
                                                    int k, int d, int I, int accumulate) {
  __shared__ __align__(16) char lds[LdsBytes<T, 1, 1>::value];
  const int s = blockIdx.z;
  float* dwd = W.dwd[s];
  if (!dwd) return;
  const SlotRows sr = slot_rows(s, 0, offsets, S_r, Tn, k);
  const int n0 = blockIdx.x * G_BN, m0 = blockIdx.y * G_BM;
  // A(m = hidden index, k = row) = dO[row][m];  B(n = intermediate index, k = row) = H[row][n]
  Opnd<T> A[1] = {{dO + (size_t)sr.orow0 * d + m0, d, d - m0, sr.nrows}};
  Opnd<T> B[1] = {{H + (size_t)sr.orow0 * I + n0, I, I - n0, sr.nrows}};
  Acc<T, 1, 1> acc;
  acc.zero();
  run_gemm<T, false, false, 1, 1>(A, B, sr.nrows, lds, acc);
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const AccCoord c = acc_coord(i, j);
      const int m = m0 + c.row, n = n0 + c.col4;
      if (m >= d || n >= I) continue;
      store_dw(dwd + (size_t)m * I + n, acc.v[0][i][j], accumulate);
    }
}

// ------------------------------------------------------------------ host ----

int check_layer_ffn(const moe_layer* L) {
  if (!L) return fail(MOE_ERR_ARG, "layer must not be NULL");
  if (L->d <= 0 || L->I <= 0) return fail(MOE_ERR_ARG, "layer d=%d I=%d", L->d, L->I);
  if (L->d % 8 || L->I % 8)
    return fail(MOE_ERR_UNSUPPORTED, "layer d=%d I=%d must be multiples of 8", L->d, L->I);
  if (L->S_routed < 0 || L->S_shared < 0 || L->S_routed + L->S_shared < 1 || L->S_routed > 512 ||
      L->S_shared > 512)
    return fail(MOE_ERR_ARG, "layer S_routed=%d S_shared=%d", L->S_routed, L->S_shared);
  FM_TRY(need_dtype_float(L->dtype, "layer dtype"));
  FM_TRY(need(L->w_gate, "layer w_gate")); FM_TRY(need(L->w_up, "layer w_up"));
  FM_TRY(need(L->w_down, "layer w_down"));
  return MOE_OK;
}

size_t max_tiles(const moe_layer* L, int T, int k) {
  return (size_t)cdiv((long)T * k, G_BM) + L->S_routed + (size_t)L->S_shared * cdiv(T, G_BM);
}

size_t align256(size_t b) { return (b + 255) / 256 * 256; }

size_t tiles_bytes(const moe_layer* L, int T, int k) { return align256((max_tiles(L, T, k) + 1) * sizeof(int2)); }

size_t rows_total(const moe_layer* L, int T, int k) { return (size_t)T * (k + L->S_shared); }

}  // namespace
}  // namespace fm

using namespace fm;

extern "C" size_t moe_grouped_swiglu_fwd_workspace_size(const moe_layer* L, int T, int k) {
  if (!L || T < 0 || k <= 0) return 0;
  return tiles_bytes(L, T, k);
}

extern "C" size_t moe_grouped_swiglu_bwd_workspace_size(const moe_layer* L, int T, int k) {
  if (!L || T < 0 || k <= 0) return 0;
  const size_t act = align256(rows_total(L, T, k) * L->I * esize(L->dtype));
  return tiles_bytes(L, T, k) + 2 * act;
}

extern "C" int moe_grouped_swiglu_fwd(const moe_layer* L, const void* X, const void* X_perm,
                                      const int32_t* offsets, int T, int k, void* A_g, void* A_u,
                                      void* H, void* O, void* ws, size_t ws_bytes, void* stream) {
  clear_error();
  FM_TRY(check_layer_ffn(L));
  if (T < 0 || k <= 0 || k > 16) return fail(MOE_ERR_ARG, "T=%d k=%d", T, k);
  if (T == 0) return MOE_OK;
  FM_TRY(need(X, "X")); FM_TRY(need(offsets, "offsets")); FM_TRY(need(A_g, "A_g"));
  FM_TRY(need(A_u, "A_u")); FM_TRY(need(H, "H")); FM_TRY(need(O, "O")); FM_TRY(need(ws, "ws"));
  if (L->S_routed > 0) FM_TRY(need(X_perm, "X_perm"));
  FM_TRY(need_aligned(X, "X")); FM_TRY(need_aligned(X_perm, "X_perm")); FM_TRY(need_aligned(A_g, "A_g"));
  FM_TRY(need_aligned(A_u, "A_u")); FM_TRY(need_aligned(H, "H")); FM_TRY(need_aligned(O, "O"));
  FM_TRY(need_aligned(ws, "ws"));
  if (ws_bytes < moe_grouped_swiglu_fwd_workspace_size(L, T, k))
    return fail(MOE_ERR_WORKSPACE, "workspace %zu < %zu bytes", ws_bytes,
                moe_grouped_swiglu_fwd_workspace_size(L, T, k));
  const size_t mt = max_tiles(L, T, k);
  if (mt > 65535) return fail(MOE_ERR_UNSUPPORTED, "too many row tiles (%zu)", mt);
  hipStream_t st = as_stream(stream);
  int2* tiles = (int2*)ws;
  hipLaunchKernelGGL(k_build_tiles, dim3(1), dim3(1024), 0, st, offsets, L->S_routed, L->S_shared, T,
                     G_BM, tiles);
  const int d = L->d, I = L->I;
#define FM_FWD(TT)                                                                                   \
  hipLaunchKernelGGL(k_gate_up<TT>, dim3(cdiv(I, G_BN), mt), dim3(G_THREADS), 0, st,               \
                     layer_ptrs<TT>(L), (const TT*)X, (const TT*)X_perm, offsets, tiles, L->S_routed, \
                     T, k, d, I, (TT*)A_g, (TT*)A_u, (TT*)H);                                       \
  hipLaunchKernelGGL(k_down<TT>, dim3(cdiv(d, G_BN), mt), dim3(G_THREADS), 0, st, layer_ptrs<TT>(L), \
                     (const TT*)H, offsets, tiles, L->S_routed, T, k, d, I, (TT*)O);
  if (L->dtype == MOE_BF16) { FM_FWD(bf16) } else { FM_FWD(float) }
#undef FM_FWD
  return check_launch("moe_grouped_swiglu_fwd");
}

extern "C" int moe_grouped_swiglu_bwd(const moe_layer* L, const void* X, const void* X_perm,
                                      const int32_t* offsets, int T, int k, const void* A_g,
                                      const void* A_u, const void* H, const void* dO, void* dX_perm,
                                      int accumulate_dw, void* ws, size_t ws_bytes, void* stream) {
  clear_error();
  FM_TRY(check_layer_ffn(L));
  if (T < 0 || k <= 0 || k > 16) return fail(MOE_ERR_ARG, "T=%d k=%d", T, k);
  FM_TRY(need(L->dw_gate, "layer dw_gate")); FM_TRY(need(L->dw_up, "layer dw_up"));
  FM_TRY(need(L->dw_down, "layer dw_down"));
  if (T == 0 && accumulate_dw) return MOE_OK;
  FM_TRY(need(X, "X")); FM_TRY(need(offsets, "offsets")); FM_TRY(need(A_g, "A_g"));
  FM_TRY(need(A_u, "A_u")); FM_TRY(need(H, "H")); FM_TRY(need(dO, "dO"));
  FM_TRY(need(dX_perm, "dX_perm")); FM_TRY(need(ws, "ws"));
  if (L->S_routed > 0) FM_TRY(need(X_perm, "X_perm"));
  FM_TRY(need_aligned(X, "X")); FM_TRY(need_aligned(X_perm, "X_perm")); FM_TRY(need_aligned(A_g, "A_g"));
  FM_TRY(need_aligned(A_u, "A_u")); FM_TRY(need_aligned(H, "H")); FM_TRY(need_aligned(dO, "dO"));
  FM_TRY(need_aligned(dX_perm, "dX_perm")); FM_TRY(need_aligned(ws, "ws"));
  if (ws_bytes < moe_grouped_swiglu_bwd_workspace_size(L, T, k))
    return fail(MOE_ERR_WORKSPACE, "workspace %zu < %zu bytes", ws_bytes,
                moe_grouped_swiglu_bwd_workspace_size(L, T, k));
  const size_t mt = max_tiles(L, T, k);
  if (mt > 65535) return fail(MOE_ERR_UNSUPPORTED, "too many row tiles (%zu)", mt);
  hipStream_t st = as_stream(stream);
  int2* tiles = (int2*)ws;
  const size_t act = align256(rows_total(L, T, k) * L->I * esize(L->dtype));
  char* dAg = (char*)ws + tiles_bytes(L, T, k);
  char* dAu = dAg + act;
  const int d = L->d, I = L->I, S = L->S_routed + L->S_shared;
  hipLaunchKernelGGL(k_build_tiles, dim3(1), dim3(1024), 0, st, offsets, L->S_routed, L->S_shared, T,
                     G_BM, tiles);
#define FM_BWD(TT)                                                                                   \
  if (T > 0) {                                                                                       \
    hipLaunchKernelGGL(k_dh<TT>, dim3(cdiv(I, G_BN), mt), dim3(G_THREADS), 0, st, layer_ptrs<TT>(L), \
                       (const TT*)dO, (const TT*)A_g, (const TT*)A_u, offsets, tiles, L->S_routed, T, \
                       k, d, I, (TT*)dAg, (TT*)dAu);                                                \
    hipLaunchKernelGGL(k_dx<TT>, dim3(cdiv(d, G_BN), mt), dim3(G_THREADS), 0, st, layer_ptrs<TT>(L), \
                       (const TT*)dAg, (const TT*)dAu, offsets, tiles, L->S_routed, T, k, d, I,     \
                       (TT*)dX_perm);                                                               \
  }                                                                                                  \
  hipLaunchKernelGGL(k_dw_gu<TT>, dim3(cdiv(d, G_BN), cdiv(I, G_BM), S), dim3(G_THREADS), 0, st,    \
                     layer_ptrs<TT>(L), (const TT*)X, (const TT*)X_perm, (const TT*)dAg,            \
                     (const TT*)dAu, offsets, L->S_routed, T, k, d, I, accumulate_dw);               \
  hipLaunchKernelGGL(k_dw_d<TT>, dim3(cdiv(I, G_BN), cdiv(d, G_BM), S), dim3(G_THREADS), 0, st,     \
                     layer_ptrs<TT>(L), (const TT*)dO, (const TT*)H, offsets, L->S_routed, T, k, d, \
                     I, accumulate_dw);
  if (L->dtype == MOE_BF16) { FM_BWD(bf16) } else { FM_BWD(float) }
#undef FM_BWD
  return check_launch("moe_grouped_swiglu_bwd");
}
