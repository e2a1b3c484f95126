// Grouped SwiGLU expert FFN, forward and backward, over the slots of a layer.
//
// Rows of slot s live in the per-row buffers at the slot's row range (routed:
// [offsets[s], offsets[s+1]) read from device memory; shared expert i:
// [T*k + i*T, T*k + (i+1)*T)).  The host never learns the bucket sizes.
//
// forward   gate_up : [A_g | A_u] = X_s [W_gate | W_up]^T, epilogue H = silu(A_g) A_u
//           down    : O = H W_down^T
// backward  dh      : dH = dO W_down, epilogue dA_g, dA_u (dSwiGLU)
//           dx      : dX_s = dA_g W_gate + dA_u W_up            (K = 2I in two passes)
//           dw_gu   : dW_gate = dA_g^T X_s, dW_up = dA_u^T X_s  (tuning slots)
//           dw_d    : dW_down = dO^T H                          (tuning slots)
//
// Scheduling.  A one-block kernel turns the offsets into a schedule: prefix
// sums of each slot's row tiles and, for the weight gradients, of each
// tuning slot's work (its K slabs), and an order of the tuning slots by
// decreasing rows.  The GEMM kernels are persistent, one block per compute
// unit.  Blocks are dispatched to the 8 XCDs round-robin, so block b runs on
// XCD b % 8.  Row-tile products: each XCD walks its own contiguous range of the
// tile space, ordered slot-major, then in bands of row tiles (see band_order);
// concurrent blocks of an XCD thus share a band of one slot's activations and a
// few weight column tiles, which stay in that XCD's L2.  Weight-gradient
// products (whose tiles differ in cost by up to two orders of magnitude): the
// tiles of the tuning slots, largest slot first, are dealt to the XCDs
// round-robin (every XCD gets an eighth of every slot), and the blocks of an XCD
// draw its tiles from a counter, so that blocks that drew cheap tiles take more
// (see DwQueue).
#include "debug.hpp"
#include "gemm_bf16.hpp"

namespace fm {
namespace {

constexpr int N_XCD = 8;

struct SlotRows {
  int nrows;    // rows of the slot
  long orow0;   // first row of the slot in the per-row buffers
  long xrow0;   // first row of the slot's input in X_perm (routed) or X (shared)
  bool shared;
};

__device__ __forceinline__ SlotRows slot_rows(int s, const int32_t* offsets, int S_r, int Tn, int k) {
  SlotRows r;
  if (s < S_r) {
    const int b = ld_scalar(offsets + s);
    r.nrows = ld_scalar(offsets + s + 1) - b;
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

// Schedule in the workspace: mbase[0..S] (prefix of row tiles per slot),
// wbase[0..S] (prefix of weight-gradient work per slot, 64-bit), dorder[0..S]
// (the tuning slots by decreasing rows, ties by index; dorder[S] = their
// number), the tile counters of the weight-gradient kernels (DW_QUEUES
// queues of N_XCD counters, 128 bytes apart), zeroed by k_build_sched, and a
// store sink: the weight-gradient epilogues send the stores of lanes outside
// the output there, so that every wave issues the same number of stores.
constexpr int DW_QSTRIDE = 32;    // ints between two counters
constexpr int DW_QUEUES = 2;      // dW_gate/up, dW_down
constexpr int DW_QINTS = DW_QUEUES * N_XCD * DW_QSTRIDE;
constexpr int DW_SINK = 4096;      // 16-byte slots of the store sink
struct Sched {
  int32_t* mbase;
  long long* wbase;
  int32_t* dorder;
  int32_t* queues;
  float* sink;
};
inline size_t round256(size_t b) { return (b + 255) / 256 * 256; }
inline size_t sched_bytes(int S) {
  return 2 * round256(sizeof(int32_t) * (S + 1)) + round256(sizeof(long long) * (S + 1)) +
         round256(sizeof(int32_t) * DW_QINTS) + 16 * DW_SINK;
}
inline Sched sched_at(void* ws, int S) {
  Sched s;
  char* p = (char*)ws;
  s.mbase = (int32_t*)p;
  p += round256(sizeof(int32_t) * (S + 1));
  s.wbase = (long long*)p;
  p += round256(sizeof(long long) * (S + 1));
  s.dorder = (int32_t*)p;
  p += round256(sizeof(int32_t) * (S + 1));
  s.queues = (int32_t*)p;
  p += round256(sizeof(int32_t) * DW_QINTS);
  s.sink = (float*)p;
  return s;
}

// One block of 1024 threads (S <= 1024).  The weight-gradient work of a tile
// of a tuning slot is its number of 64-row K slabs + 1 (so an empty tuning slot
// still gets its zeros written); frozen slots have none.
constexpr int DW_SLAB = 64;
__global__ __launch_bounds__(1024) void k_build_sched(const int32_t* __restrict__ offsets, int S_r, int S_sh,
                                                      int Tn, int tile_rows, float* const* __restrict__ dw_tab,
                                                      int32_t* __restrict__ mbase, long long* __restrict__ wbase,
                                                      int32_t* __restrict__ dorder, int32_t* __restrict__ queues) {
  __shared__ int sm[1024];
  __shared__ long long sw[1024];
  __shared__ int skey[1024];
  const int S = S_r + S_sh, s = threadIdx.x;
  for (int i = s; i < DW_QINTS; i += 1024) queues[i] = 0;
  int n = 0;
  if (s < S) n = s < S_r ? offsets[s + 1] - offsets[s] : Tn;
  const bool tune = s < S && dw_tab && dw_tab[s];
  long long w = 0;
  if (tune) w = (n + DW_SLAB - 1) / DW_SLAB + 1;
  sm[s] = (n + tile_rows - 1) / tile_rows;
  sw[s] = w;
  skey[s] = tune ? n : -1;
  // tuning slots by decreasing rows (ties: lower index first)
  const int ntune = __syncthreads_count(tune);
  if (tune) {
    int rank = 0;
    for (int u = 0; u < S; ++u) rank += (skey[u] > n) || (skey[u] == n && u < s);
    dorder[rank] = s;
  }
  if (s == 0) dorder[S] = ntune;
  __syncthreads();
  for (int off = 1; off < 1024; off <<= 1) {   // inclusive Hillis-Steele scans
    const int a = s >= off ? sm[s - off] : 0;
    const long long b = s >= off ? sw[s - off] : 0;
    __syncthreads();
    sm[s] += a;
    sw[s] += b;
    __syncthreads();
  }
  if (s <= S) {
    mbase[s] = s == 0 ? 0 : sm[s - 1];
    wbase[s] = s == 0 ? 0 : sw[s - 1];
  }
}

// Largest s in [0, S) with base[s] <= v (base nondecreasing, base[0] = 0).
template <typename B>
__device__ __forceinline__ int find_slot(const B* base, int S, long long v) {
  int lo = 0, hi = S - 1;
  while (lo < hi) {
    const int mid = (lo + hi + 1) >> 1;
    if ((long long)ld_scalar(base + mid) <= v) lo = mid;
    else hi = mid - 1;
  }
  return lo;
}

struct Tile {
  int s, n, m;   // slot, output column tile, output row tile
};

// Order of the (row tile, column tile) pairs of one slot: bands of GM row
// tiles; inside a band column tiles advance slowest and row tiles fastest.  The
// blocks of an XCD working on one band share its GM activation tiles and a few
// weight tiles, a working set that fits the XCD's L2.
__device__ __forceinline__ void band_order(int loc, int mt, int NT, int GM, int& m, int& n) {
  const int band = loc / (GM * NT);
  const int h = min(GM, mt - band * GM);
  const int rem = loc - band * GM * NT;
  n = rem / h;
  m = band * GM + rem % h;
}

constexpr int GM_ROWS = 8;   // band height of the row-tile GEMMs
constexpr int GM_DW = 4;     // band height of the weight-gradient GEMMs

// Row-tile GEMMs: tile t of [0, M_total * NT), slot-major.
__device__ __forceinline__ Tile row_tile(const int32_t* mbase, int S, int NT, long long t) {
  Tile r;
  r.s = find_slot(mbase, S, t / NT);
  const int mb = ld_scalar(mbase + r.s);
  const int mt = ld_scalar(mbase + r.s + 1) - mb;
  band_order((int)(t - (long long)mb * NT), mt, NT, GM_ROWS, r.m, r.n);
  return r;
}

// Weight-gradient tile t: tps = MT * NT tiles per slot, bands of gm row tiles.
__device__ __forceinline__ Tile dw_tile(long long t, int tps, int MT, int gm = GM_DW) {
  Tile r;
  r.s = (int)(t / tps);
  band_order((int)(t - (long long)r.s * tps), MT, tps / MT, gm, r.m, r.n);
  return r;
}

// First weight-gradient tile whose cumulative work reaches `target`; wbase
// holds the per-tile work prefix over slots, tps tiles per slot.
__device__ __forceinline__ long long tile_at_work(const long long* wbase, int S, int tps, long long target) {
  if (target >= wbase[S] * tps) return (long long)S * tps;
  const int s = find_slot(wbase, S, target / tps);
  const long long per = wbase[s + 1] - wbase[s];
  if (per == 0) return (long long)(s + 1) * tps;
  long long i = (target - wbase[s] * tps + per - 1) / per;
  if (i > tps) i = tps;
  return (long long)s * tps + i;
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
// Logistic function with the hardware exp2 and reciprocal (about 1 ulp each),
// for epilogues whose results are rounded to bf16.
__device__ __forceinline__ float sigm_fast(float z) {
  return __builtin_amdgcn_rcpf(1.0f + __builtin_amdgcn_exp2f(-1.4426950408889634f * z));
}

struct RowArgs {
  const int32_t* offsets;
  const int32_t* mbase;
  int S_r, S, Tn, k, d, I;
  int ldA;   // row stride (elements) of the backward's dA_g, dA_u in the workspace
};

struct DwArgs {
  const int32_t* offsets;
  const long long* wbase;
  const int32_t* dorder;
  int32_t* queue;   // this kernel's N_XCD counters
  float* sink;      // DW_SINK 16-byte slots
  int S_r, S, Tn, k, d, I, accumulate;
  int ldA;          // row stride (elements) of dA_g, dA_u
};

// The range of the tile space handled by this block's XCD, and the block's
// first tile and stride inside it.
// Rows of slot s from row m0 on (a row tile with at most half a tile's rows
// left runs as a half-height tile).
__device__ __forceinline__ int rows_left(const RowArgs& ra, int s, int m0) {
  return slot_rows(s, ra.offsets, ra.S_r, ra.Tn, ra.k).nrows - m0;
}

struct TileRange {
  long long lo, hi;
  int first, step;
};
__device__ __forceinline__ TileRange row_range(const RowArgs& ra, int NT) {
  const long long total = (long long)ld_scalar(ra.mbase + ra.S) * NT;
  const int x = blockIdx.x % N_XCD;
  return TileRange{total * x / N_XCD, total * (x + 1) / N_XCD, (int)(blockIdx.x / N_XCD),
                   (int)(gridDim.x / N_XCD)};
}
__device__ __forceinline__ TileRange dw_range(const DwArgs& da, int tps) {
  const long long w = da.wbase[da.S] * tps;
  const int x = blockIdx.x % N_XCD;
  return TileRange{tile_at_work(da.wbase, da.S, tps, w * x / N_XCD),
                   tile_at_work(da.wbase, da.S, tps, w * (x + 1) / N_XCD), (int)(blockIdx.x / N_XCD),
                   (int)(gridDim.x / N_XCD)};
}

// Dynamic tile queue of the weight-gradient kernels.  XCD x owns tiles x,
// x + 8, x + 16, ... of the tuning slots' tile space (slots in dorder, largest
// first; tps tiles per slot), i.e. an eighth of every slot, so that the XCDs
// get equal work and equal shares of the costly tiles.  Its blocks take them in
// order, one atomic per tile, drawn by thread 0 a tile ahead; the draw reaches
// the other waves through LDS word 0, which is free between tiles.
struct DwQueue {
  int32_t* ctr;
  long long total;   // tiles of the tuning slots
  int x;

  __device__ __forceinline__ DwQueue(const DwArgs& da, int tps) {
    x = blockIdx.x % N_XCD;
    ctr = da.queue + x * DW_QSTRIDE;
    total = (long long)ld_scalar(da.dorder + da.S) * tps;
  }
  // Thread 0 only.  The zero offset is opaque to the compiler, so the atomic
  // stays a plain one: on a provably uniform address it would be rewritten into
  // a wave-aggregated form that waits for its result (and so for every load and
  // store of the wave still in flight) right where it is issued.
  __device__ __forceinline__ int draw() const {
    int z;
    asm volatile("v_mov_b32 %0, 0" : "=v"(z));
    return atomicAdd(ctr + z, 1);
  }
  __device__ __forceinline__ long long tile(int j) const { return (long long)j * N_XCD + x; }
  // Hands thread 0's draw to every thread (LDS word 0 must be free; the caller
  // keeps it until every wave has read it).
  __device__ __forceinline__ static int share(FM_LDS char* lds, int j) {
    if (threadIdx.x == 0) {
      wait_vmcnt<0>();
      *(FM_LDS int*)lds = j;
    }
    barrier_lds_writes();
    return *(const FM_LDS int*)lds;
  }
};

// ------------------------------------------- fp32 kernels (16x16 core) ----

template <typename T>
__global__ __launch_bounds__(G_THREADS) void kf_gate_up(LayerPtrs<T> W, const T* __restrict__ X,
                                                       const T* __restrict__ Xp, RowArgs ra,
                                                       T* __restrict__ Ag, T* __restrict__ Au,
                                                       T* __restrict__ H) {
  __shared__ __align__(16) char lds[2 * (1 + 2) * GemmCfg<T>::TILE * (int)sizeof(T)];
  const int d = ra.d, I = ra.I, NT = (I + G_BN - 1) / G_BN;
  const TileRange tr = row_range(ra, NT);
  for (long long t = tr.lo + tr.first; t < tr.hi; t += tr.step) {
    const Tile rt = row_tile(ra.mbase, ra.S, NT, t);
    const SlotRows sr = slot_rows(rt.s, ra.offsets, ra.S_r, ra.Tn, ra.k);
    const int m0 = rt.m * G_BM, n0 = rt.n * G_BN;
    const T* xs = (sr.shared ? X : Xp) + (size_t)(sr.xrow0 + m0) * d;
    Opnd<T> A[1] = {{xs, d, sr.nrows - m0, d}};
    Opnd<T> B[2] = {{ld_scalar(W.wg + rt.s) + (size_t)n0 * d, d, I - n0, d}, {ld_scalar(W.wu + rt.s) + (size_t)n0 * d, d, I - n0, d}};
    Acc<T, 1, 2> acc;
    acc.zero();
    gemm_mainloop<T, true, true, 1, 2>(A, B, d, (T*)lds, acc);
    const size_t ob = (size_t)(sr.orow0 + m0);
#pragma unroll
    for (int q = 0; q < 16; ++q) {
      const AccCoord c = quad_coord<T>(q);
      const int n = n0 + c.col4;
      if (c.row >= sr.nrows - m0 || n >= I) continue;
      const f32x4_t ag = acc.quad(0, q), u = acc.quad(1, q);
      f32x4_t h;
#pragma unroll
      for (int r = 0; r < 4; ++r) h[r] = ag[r] * sigm(ag[r]) * u[r];
      const size_t o = (ob + c.row) * I + n;
      store4(Ag + o, ag);
      store4(Au + o, u);
      store4(H + o, h);
    }
  }
}

template <typename T>
__global__ __launch_bounds__(G_THREADS) void kf_down(LayerPtrs<T> W, const T* __restrict__ H, RowArgs ra,
                                                    T* __restrict__ O) {
  __shared__ __align__(16) char lds[2 * (1 + 1) * GemmCfg<T>::TILE * (int)sizeof(T)];
  const int d = ra.d, I = ra.I, NT = (d + G_BN - 1) / G_BN;
  const TileRange tr = row_range(ra, NT);
  for (long long t = tr.lo + tr.first; t < tr.hi; t += tr.step) {
    const Tile rt = row_tile(ra.mbase, ra.S, NT, t);
    const SlotRows sr = slot_rows(rt.s, ra.offsets, ra.S_r, ra.Tn, ra.k);
    const int m0 = rt.m * G_BM, n0 = rt.n * G_BN;
    const size_t ob = (size_t)(sr.orow0 + m0);
    Opnd<T> A[1] = {{H + ob * I, I, sr.nrows - m0, I}};
    Opnd<T> B[1] = {{ld_scalar(W.wd + rt.s) + (size_t)n0 * I, I, d - n0, I}};
    Acc<T, 1, 1> acc;
    acc.zero();
    gemm_mainloop<T, true, true, 1, 1>(A, B, I, (T*)lds, acc);
#pragma unroll
    for (int q = 0; q < 16; ++q) {
      const AccCoord c = quad_coord<T>(q);
      const int n = n0 + c.col4;
      if (c.row >= sr.nrows - m0 || n >= d) continue;
      store4(O + (ob + c.row) * d + n, acc.quad(0, q));
    }
  }
}

// ------------------------------------------------------------ backward ----

// Also leaves per-row partial sums of dA_g^2 + dA_u^2 and h^2 (h = silu(a_g) a_u)
// for the expert utility: per column tile, one pair per wave column (two),
// at norms[row * 2 NT + 2 tile + wave column].
template <typename T>
__global__ __launch_bounds__(G_THREADS) void kf_dh(LayerPtrs<T> W, const T* __restrict__ dO,
                                                  const T* __restrict__ Ag, const T* __restrict__ Au,
                                                  RowArgs ra, T* __restrict__ dAg, T* __restrict__ dAu,
                                                  float2* __restrict__ norms) {
  __shared__ __align__(16) char lds[2 * (1 + 1) * GemmCfg<T>::TILE * (int)sizeof(T)];
  const int d = ra.d, I = ra.I, NT = (I + G_BN - 1) / G_BN;
  const TileRange tr = row_range(ra, NT);
  for (long long t = tr.lo + tr.first; t < tr.hi; t += tr.step) {
    const Tile rt = row_tile(ra.mbase, ra.S, NT, t);
    const SlotRows sr = slot_rows(rt.s, ra.offsets, ra.S_r, ra.Tn, ra.k);
    const int m0 = rt.m * G_BM, n0 = rt.n * G_BN;
    const size_t ob = (size_t)(sr.orow0 + m0);
    // B(n = intermediate index, k = hidden index) = W_down[k][n]: MN-contiguous
    Opnd<T> A[1] = {{dO + ob * d, d, sr.nrows - m0, d}};
    Opnd<T> B[1] = {{ld_scalar(W.wd + rt.s) + n0, I, I - n0, d}};
    Acc<T, 1, 1> acc;
    acc.zero();
    gemm_mainloop<T, true, false, 1, 1>(A, B, d, (T*)lds, acc);
    float sa[4] = {0.f, 0.f, 0.f, 0.f}, sh[4] = {0.f, 0.f, 0.f, 0.f};   // per row block i of the wave
#pragma unroll
    for (int q = 0; q < 16; ++q) {
      const AccCoord c = quad_coord<T>(q);
      const int n = n0 + c.col4;
      if (c.row >= sr.nrows - m0 || n >= I) continue;
      const size_t o = (ob + c.row) * I + n;
      const f32x4_t dh = acc.quad(0, q), ag = load4(Ag + o), u = load4(Au + o);
      f32x4_t dg, du;
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const float s = sigm(ag[r]);
        du[r] = dh[r] * ag[r] * s;
        dg[r] = dh[r] * u[r] * s * (1.0f + ag[r] * (1.0f - s));
        const float h = ag[r] * s * u[r];
        sa[q >> 2] = fmaf(dg[r], dg[r], fmaf(du[r], du[r], sa[q >> 2]));
        sh[q >> 2] = fmaf(h, h, sh[q >> 2]);
      }
      store4(dAg + o, dg);
      store4(dAu + o, du);
    }
    // quad (i, j) of lane L covers row 64 wm + 16 i + L % 16: add over the
    // four lanes L / 16 of that row, then one pair per row and wave column
    const int lane = lane_id(), wave = threadIdx.x >> 6;
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      float a = sa[i], h = sh[i];
      a += __shfl_xor(a, 16);
      h += __shfl_xor(h, 16);
      a += __shfl_xor(a, 32);
      h += __shfl_xor(h, 32);
      const int row = (wave & 1) * 64 + i * 16 + (lane & 15);
      if (lane < 16 && row < sr.nrows - m0)
        norms[(ob + row) * (2 * NT) + 2 * rt.n + (wave >> 1)] = make_float2(a, h);
    }
  }
}

template <typename T>
__global__ __launch_bounds__(G_THREADS) void kf_dx(LayerPtrs<T> W, const T* __restrict__ dAg,
                                                  const T* __restrict__ dAu, RowArgs ra,
                                                  T* __restrict__ dXp) {
  __shared__ __align__(16) char lds[2 * (1 + 1) * GemmCfg<T>::TILE * (int)sizeof(T)];
  const int d = ra.d, I = ra.I, NT = (d + G_BN - 1) / G_BN;
  const TileRange tr = row_range(ra, NT);
  for (long long t = tr.lo + tr.first; t < tr.hi; t += tr.step) {
    const Tile rt = row_tile(ra.mbase, ra.S, NT, t);
    const SlotRows sr = slot_rows(rt.s, ra.offsets, ra.S_r, ra.Tn, ra.k);
    const int m0 = rt.m * G_BM, n0 = rt.n * G_BN;
    const size_t ob = (size_t)(sr.orow0 + m0);
    Acc<T, 1, 1> acc;
    acc.zero();
    {  // B(n = hidden index, k = intermediate index) = W_gate[k][n]
      Opnd<T> A[1] = {{dAg + ob * I, I, sr.nrows - m0, I}};
      Opnd<T> B[1] = {{ld_scalar(W.wg + rt.s) + n0, d, d - n0, I}};
      gemm_mainloop<T, true, false, 1, 1>(A, B, I, (T*)lds, acc);
    }
    {
      Opnd<T> A[1] = {{dAu + ob * I, I, sr.nrows - m0, I}};
      Opnd<T> B[1] = {{ld_scalar(W.wu + rt.s) + n0, d, d - n0, I}};
      gemm_mainloop<T, true, false, 1, 1>(A, B, I, (T*)lds, acc);
    }
#pragma unroll
    for (int q = 0; q < 16; ++q) {
      const AccCoord c = quad_coord<T>(q);
      const int n = n0 + c.col4;
      if (c.row >= sr.nrows - m0 || n >= d) continue;
      store4(dXp + (ob + c.row) * d + n, acc.quad(0, q));
    }
  }
}

__device__ __forceinline__ void store_dw(float* p, f32x4_t v, bool accumulate) {
  if (accumulate) v = v + load4(p);
  store4(p, v);
}

// dW_gate = dA_g^T X_s, dW_up = dA_u^T X_s: rows over I, columns over d.
template <typename T>
__global__ __launch_bounds__(G_THREADS) void kf_dw_gu(LayerPtrs<T> W, const T* __restrict__ X,
                                                     const T* __restrict__ Xp, const T* __restrict__ dAg,
                                                     const T* __restrict__ dAu, DwArgs da) {
  __shared__ __align__(16) char lds[2 * (2 + 1) * GemmCfg<T>::TILE * (int)sizeof(T)];
  const int d = da.d, I = da.I;
  const int MT = (I + G_BM - 1) / G_BM, NT = (d + G_BN - 1) / G_BN;
  const TileRange tr = dw_range(da, MT * NT);
  for (long long t = tr.lo + tr.first; t < tr.hi; t += tr.step) {
    const Tile rt = dw_tile(t, MT * NT, MT);
    float* dwg = ld_scalar(W.dwg + rt.s);
    float* dwu = ld_scalar(W.dwu + rt.s);
    if (dwg && dwu) {
      const SlotRows sr = slot_rows(rt.s, da.offsets, da.S_r, da.Tn, da.k);
      const int m0 = rt.m * G_BM, n0 = rt.n * G_BN;
      // A(m = intermediate index, k = row) = dA[row][m];  B(n = hidden index, k = row) = X_s[row][n]
      Opnd<T> A[2] = {{dAg + (size_t)sr.orow0 * I + m0, I, I - m0, sr.nrows},
                      {dAu + (size_t)sr.orow0 * I + m0, I, I - m0, sr.nrows}};
      Opnd<T> B[1] = {{(sr.shared ? X : Xp) + (size_t)sr.xrow0 * d + n0, d, d - n0, sr.nrows}};
      Acc<T, 2, 1> acc;
      acc.zero();
      gemm_mainloop<T, false, false, 2, 1>(A, B, sr.nrows, (T*)lds, acc);
#pragma unroll
      for (int q = 0; q < 16; ++q) {
        const AccCoord c = quad_coord<T>(q);
        const int m = m0 + c.row, n = n0 + c.col4;
        if (m >= I || n >= d) continue;
        store_dw(dwg + (size_t)m * d + n, acc.quad(0, q), da.accumulate);
        store_dw(dwu + (size_t)m * d + n, acc.quad(1, q), da.accumulate);
      }
    }
  }
}

// dW_down = dO^T H: rows over d, columns over I.
template <typename T>
__global__ __launch_bounds__(G_THREADS) void kf_dw_d(LayerPtrs<T> W, const T* __restrict__ dO,
                                                    const T* __restrict__ H, DwArgs da) {
  __shared__ __align__(16) char lds[2 * (1 + 1) * GemmCfg<T>::TILE * (int)sizeof(T)];
  const int d = da.d, I = da.I;
  const int MT = (d + G_BM - 1) / G_BM, NT = (I + G_BN - 1) / G_BN;
  const TileRange tr = dw_range(da, MT * NT);
  for (long long t = tr.lo + tr.first; t < tr.hi; t += tr.step) {
    const Tile rt = dw_tile(t, MT * NT, MT);
    float* dwd = ld_scalar(W.dwd + rt.s);
    if (dwd) {
      const SlotRows sr = slot_rows(rt.s, da.offsets, da.S_r, da.Tn, da.k);
      const int m0 = rt.m * G_BM, n0 = rt.n * G_BN;
      // A(m = hidden index, k = row) = dO[row][m];  B(n = intermediate index, k = row) = H[row][n]
      Opnd<T> A[1] = {{dO + (size_t)sr.orow0 * d + m0, d, d - m0, sr.nrows}};
      Opnd<T> B[1] = {{H + (size_t)sr.orow0 * I + n0, I, I - n0, sr.nrows}};
      Acc<T, 1, 1> acc;
      acc.zero();
      gemm_mainloop<T, false, false, 1, 1>(A, B, sr.nrows, (T*)lds, acc);
#pragma unroll
      for (int q = 0; q < 16; ++q) {
        const AccCoord c = quad_coord<T>(q);
        const int m = m0 + c.row, n = n0 + c.col4;
        if (m >= d || n >= I) continue;
        store_dw(dwd + (size_t)m * I + n, acc.quad(0, q), da.accumulate);
      }
    }
  }
}

// ------------------------------------------ bf16 kernels (8-wave core) ----

typedef const bf16* cbp;

// Block tile of every bf16 product: 256 x 256, waves 2 x 4 (128 x 64 each, two
// per SIMD), 64-deep slabs, three of A and two of B in LDS (160 KB).  (One wave
// per SIMD with 128 x 128 each reads a third less LDS but measured slower: a
// lone wave cannot hide its own LDS-read and DMA-issue stalls.)
using CB = B16Cfg<256, 256, 2, 4, 64, 3, 2>;
constexpr int B16_ROWS = CB::RA;   // rows per row tile of the bf16 kernels
// Pieces of a full tile for the last round of a row-tile product: a row half
// (128 x 256) and a quarter (128 x 128), same waves and slab depth.
using CBH = B16Cfg<128, 256, 2, 4, 64, 3, 2>;
using CBQ = B16Cfg<128, 128, 2, 4, 64, 3, 2>;
// A narrow tile for a last column tile over I with at most 128 columns left
// (I = 1408: 1280..1407) in dH and dW_down: its slabs move 3/4 of a full
// tile's bytes for half the flops, where a full tile would multiply a half
// that is never written back.
using CBN = B16Cfg<256, 128, 2, 4, 64, 3, 2>;

// The XCD's share of a row-tile product (row_range) goes in rounds of one full
// tile per block.  When the last round would leave at least half of the XCD's
// blocks idle, its tiles are cut into `parts` pieces (2: row halves; 4: row and
// column halves, where the product allows them), one piece per block, so that
// the round takes about a piece's time (a slab of a piece moves 3/4 or 1/2 of a
// full tile's bytes).  cut = the first tile of that round, or tr.hi.
struct LastRound {
  long long cut;
  int parts;
};
__device__ __forceinline__ LastRound last_round(const TileRange& tr, bool quarters) {
  const long long rem = (tr.hi - tr.lo) % tr.step;
  LastRound lr{tr.hi, 0};
  if (rem > 0 && rem * 2 <= tr.step) {
    lr.cut = tr.hi - rem;
    lr.parts = quarters && rem * 4 <= tr.step ? 4 : 2;
  }
  return lr;
}

// Physical index of logical row / column c of an operand that interleaves two
// matrices in 32-blocks (the matrix is (c >> 5) & 1).
__device__ __forceinline__ int deinter(int c) { return 32 * (c >> 6) + (c & 31); }

// Writes a whole RA x RB accumulator tile (bf16) through LDS: out points at
// the tile origin, rows x cols of it are valid.
template <class C>
__device__ __forceinline__ void b16_store_staged(const B16Acc<C::MI, C::NJ>& acc, FM_LDS char* lds, bf16* out,
                                                 size_t ld, int rows, int cols) {
  using S = Stage<bf16, C::RB>;
#pragma unroll
  for (int i = 0; i < C::MI; ++i)
#pragma unroll
    for (int j = 0; j < C::NJ; ++j)
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        const AccCoord c = b16_coord<C>(i, j, q);
        S::put4(lds, c.row, c.col4, acc.quad(i, j, q));
      }
  barrier_lds_writes();
  S::template copy_out<C::RA, C::THREADS>(lds, out, ld, rows, cols);
  barrier_lds();
}

// x moved between lanes by a DPP control within each 16-lane row.
template <int CTRL> __device__ __forceinline__ float dpp_f(float x) {
  return __builtin_bit_cast(float, __builtin_amdgcn_update_dpp(0, __builtin_bit_cast(int, x), CTRL, 0xf, 0xf, false));
}

// Sum of x over aligned groups of N = 16 or 32 lanes, in every lane of the
// group: quad permutes (lane ^ 1, lane ^ 2), the half-row mirror (quad pairs)
// and the row mirror (half-row pairs) inside each row of 16, then one exchange
// across the two rows for N = 32.  Each step adds a lane's value to a partner
// holding a sum over the other, equally sized part, so every lane of the group
// ends with the same bits.
template <int N> __device__ __forceinline__ float row_lanes_sum(float x) {
  static_assert(N == 16 || N == 32, "one or two DPP rows");
  x += dpp_f<0xB1>(x);    // quad_perm [1, 0, 3, 2]
  x += dpp_f<0x4E>(x);    // quad_perm [2, 3, 0, 1]
  x += dpp_f<0x141>(x);   // row_half_mirror
  x += dpp_f<0x140>(x);   // row_mirror
  if (N == 32) x += __shfl_xor(x, 16);
  return x;
}

// SwiGLU backward of a dH tile with s = logistic(a_g): dA_u = dH a_g s,
// dA_g = dH u s (1 + a_g (1 - s)).  dH is staged through LDS rounded to bf16
// (the precision a bf16 product would hand to the elementwise step), the
// whole tile at once; every lane then takes 8-column chunks of a row (16-byte
// loads of A_g, A_u and stores of dA_g, dA_u; a wave covers whole rows).  The
// chunks go in groups of G per lane; the loads of the first group are issued
// before the tile is staged, so their latency overlaps the LDS writes.
// Pointers are at the tile origin; rows x cols are valid; A_g, A_u rows are
// ld apart, dA_g, dA_u rows ldo apart.
//
// The same pass leaves, per row of the tile, the sums over its columns of
// dA_g^2 + dA_u^2 and of h^2 with h = silu(a_g) a_u recomputed from the stored
// A_g, A_u (the factors of the expert utility, Eq. 3): the 32 lanes that share
// a row add their values by a fixed butterfly and one of them stores the pair
// at norms[row * P] (P partials per row, this column tile's slot).
template <class C>
__device__ __forceinline__ void b16_dswiglu_staged(const B16Acc<C::MI, C::NJ>& acc, FM_LDS char* lds,
                                                   const bf16* Ag, const bf16* Au, bf16* dAg, bf16* dAu,
                                                   size_t ld, size_t ldo, int rows, int cols, float2* norms,
                                                   int P) {
  using S = Stage<bf16, C::RB>;
  constexpr int CH = C::RB / 8;                     // 8-column chunks per row
  constexpr int PER = C::RA * CH / C::THREADS;      // chunks per lane
  constexpr int G = PER < 8 ? PER : 8;              // chunks in flight per lane
  static_assert(PER % G == 0 && PER * C::THREADS == C::RA * CH && C::RA * C::RB * 2 <= C::LDS &&
                    (CH == 32 || CH == 16),
                "whole chunks per lane, a row per half or quarter wave");
  // thread index re-read here (opaque), so that the per-chunk addresses are
  // not hoisted out of the tile loop and kept live through the main loop
  const int tid = wave_id() * 64 + lane_id_here();
  u32x4_t ga[G], ua[G];
  auto load = [&](int g) {
#pragma unroll
    for (int u = 0; u < G; ++u) {
      const int idx = tid + (g * G + u) * C::THREADS, r = idx / CH, c = (idx % CH) * 8;
      if (r < rows && c < cols) {
        ga[u] = ld16(Ag + (size_t)r * ld + c);
        ua[u] = ld16(Au + (size_t)r * ld + c);
      }
    }
  };
  load(0);
#pragma unroll
  for (int i = 0; i < C::MI; ++i)
#pragma unroll
    for (int j = 0; j < C::NJ; ++j)
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        const AccCoord c = b16_coord<C>(i, j, q);
        S::put4(lds, c.row, c.col4, acc.quad(i, j, q));
      }
  barrier_lds_writes();
#pragma unroll
  for (int g = 0; g < PER / G; ++g) {
    if (g > 0) load(g);
#pragma unroll
    for (int u = 0; u < G; ++u) {
      const int idx = tid + (g * G + u) * C::THREADS, r = idx / CH, c = (idx % CH) * 8;
      float sa = 0.f, sh = 0.f;
      if (r < rows && c < cols) {
        float dh[8], a[8], up[8], dg[8], du[8];
        const u32x4_t hv = *(const FM_LDS u32x4_t*)(lds + S::at(r, c));
        unpack16(hv, dh, (bf16*)nullptr);
        unpack16(ga[u], a, (bf16*)nullptr);
        unpack16(ua[u], up, (bf16*)nullptr);
#pragma unroll
        for (int e = 0; e < 8; ++e) {
          const float sg = sigm_fast(a[e]);
          const float silu = a[e] * sg;
          du[e] = dh[e] * silu;
          dg[e] = dh[e] * up[e] * sg * (1.0f + a[e] * (1.0f - sg));
          const float h = silu * up[e];
          sa = fmaf(dg[e], dg[e], fmaf(du[e], du[e], sa));
          sh = fmaf(h, h, sh);
        }
        st16(dAg + (size_t)r * ldo + c, pack16(dg, (bf16*)nullptr));
        st16(dAu + (size_t)r * ldo + c, pack16(du, (bf16*)nullptr));
      }
      // the CH lanes of this row (half or a quarter of the wave); a 128-column
      // tile gives the same sums as a 256-column tile whose other half is zero
      sa = row_lanes_sum<CH>(sa);
      sh = row_lanes_sum<CH>(sh);
      if ((tid & (CH - 1)) == 0 && r < rows) norms[(size_t)r * P] = make_float2(sa, sh);
    }
  }
  barrier_lds();
}

// [A_g | A_u] = X_s [W_gate | W_up]^T, H = silu(A_g) A_u (from A_g, A_u as
// stored in bf16, the values the backward reads).  The B tile
// interleaves 32-row blocks of W_gate and W_up (RB / 2 intermediate columns per
// tile): tile j = 2jj of a wave holds gate and j = 2jj + 1 up of the same
// columns.  One tile of shape C at rows m0 of slot s, intermediate columns n0.
template <class C>
__device__ __forceinline__ void gate_up_tile(const LayerPtrs<bf16>& W, cbp X, cbp Xp, const RowArgs& ra,
                                             FM_LDS char* lds, int s, int m0, int n0, bf16* Ag, bf16* Au,
                                             bf16* H) {
  const int d = ra.d, I = ra.I;
  const SlotRows sr = slot_rows(s, ra.offsets, ra.S_r, ra.Tn, ra.k);
  const int rows = sr.nrows - m0, cols = I - n0;
  if (rows <= 0 || cols <= 0) return;
  const B16Src A{(sr.shared ? X : Xp) + (size_t)(sr.xrow0 + m0) * d, nullptr, d, rows, d};
  const B16Src B{ld_scalar(W.wg + s) + (size_t)n0 * d, ld_scalar(W.wu + s) + (size_t)n0 * d, d, cols, d};
  B16Acc<C::MI, C::NJ> acc;
  acc.zero();
  b16_gemm<C, true, true, false, true>(A, B, d, lds, acc);
  // A_g and A_u staged side by side, then H in the first half.
  using SG = Stage<bf16, C::RB / 2>;
  FM_LDS char* sg = lds;
  FM_LDS char* su = sg + C::RA * (C::RB / 2) * 2;
  const size_t ob = (size_t)(sr.orow0 + m0);
#pragma unroll
  for (int i = 0; i < C::MI; ++i)
#pragma unroll
    for (int jj = 0; jj < C::NJ / 2; ++jj)
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        const AccCoord c = b16_coord<C>(i, 2 * jj, q);
        SG::put4(sg, c.row, deinter(c.col4), acc.quad(i, 2 * jj, q));
        SG::put4(su, c.row, deinter(c.col4), acc.quad(i, 2 * jj + 1, q));
      }
  barrier_lds_writes();
  // Each lane takes 8-column chunks of A_g and A_u, stores them, and forms H
  // from the same bf16 values (the ones the backward reads).
  constexpr int TOTAL = C::RA * SG::CPR;
  const int tid = wave_id() * 64 + lane_id_here();
#pragma unroll 4
  for (int idx = tid; idx < TOTAL; idx += C::THREADS) {
    const int row = idx / SG::CPR, c = idx % SG::CPR;
    const uint32_t off = row * SG::ROW_BYTES + ((c ^ (row & (SG::CPR - 1))) << 4);
    const u32x4_t g = *(const FM_LDS u32x4_t*)(sg + off);
    const u32x4_t u = *(const FM_LDS u32x4_t*)(su + off);
    if (row < rows && c * SG::EPC < cols) {
      const size_t o = (ob + row) * I + n0 + c * SG::EPC;
      st16(Ag + o, g);
      st16(Au + o, u);
      float a[8], v[8], h[8];
      unpack16(g, a, (bf16*)nullptr);
      unpack16(u, v, (bf16*)nullptr);
#pragma unroll
      for (int e = 0; e < 8; ++e) h[e] = a[e] * sigm_fast(a[e]) * v[e];
      st16(H + o, pack16(h, (bf16*)nullptr));
    }
  }
  barrier_lds();
}

__global__ __launch_bounds__(CB::THREADS) void kb_gate_up(LayerPtrs<bf16> W, cbp X, cbp Xp, RowArgs ra,
                                                          bf16* Ag, bf16* Au, bf16* H) {
  __shared__ __align__(16) char lds[CB::LDS];
  FM_LDS char* const l = (FM_LDS char*)lds;
  const int NT = (ra.I + CB::RB / 2 - 1) / (CB::RB / 2);
  const TileRange tr = row_range(ra, NT);
  const LastRound lr = last_round(tr, false);
  for (long long t = tr.lo + tr.first; t < lr.cut; t += tr.step) {
    const Tile rt = row_tile(ra.mbase, ra.S, NT, t);
    if (rows_left(ra, rt.s, rt.m * CB::RA) <= CBH::RA)
      gate_up_tile<CBH>(W, X, Xp, ra, l, rt.s, rt.m * CB::RA, rt.n * (CB::RB / 2), Ag, Au, H);
    else
      gate_up_tile<CB>(W, X, Xp, ra, l, rt.s, rt.m * CB::RA, rt.n * (CB::RB / 2), Ag, Au, H);
  }
  if (lr.parts && tr.first < (tr.hi - lr.cut) * 2) {   // a row half of the last round
    const Tile rt = row_tile(ra.mbase, ra.S, NT, lr.cut + tr.first / 2);
    gate_up_tile<CBH>(W, X, Xp, ra, l, rt.s, rt.m * CB::RA + (tr.first % 2) * CBH::RA, rt.n * (CB::RB / 2), Ag,
                      Au, H);
  }
}

// ------------------------------ quantised forward (int8 weights, bf16 X) ----

struct Q8Ptrs {
  const int8_t* const* qg;
  const int8_t* const* qu;
  const int8_t* const* qd;
  const float* const* sg;
  const float* const* su;
  const float* const* sd;
};

// The bf16 tile shape with int8 B slabs (16 KB instead of 32 KB each).
using CQ = B16Cfg<256, 256, 2, 4, 64, 3, 2, 1>;

// Four consecutive row scales from col (clamped so that the four stay inside
// the row count n, n >= 4; columns past n are never stored).
__device__ __forceinline__ f32x4_t scale4(const float* s, int col, int n) {
  const int c = min(col, n - 4);
  return f32x4_t{s[c], s[c + 1], s[c + 2], s[c + 3]};
}

// H = silu(s_g (X_s Q_g^T)) (s_u (X_s Q_u^T)) with int8 Q_g, Q_u interleaved
// in 32-row blocks as in kb_gate_up; the row scales of the weights scale the
// output columns.  Only H is written (no backward follows this forward).
// One such tile of shape C at rows m0 of slot s, intermediate columns n0.
template <class C>
__device__ __forceinline__ void q8_gate_up_tile(const Q8Ptrs& W, cbp X, cbp Xp, const RowArgs& ra, FM_LDS char* lds,
                                                int s, int m0, int n0, bf16* H) {
  const int d = ra.d, I = ra.I;
  const SlotRows sr = slot_rows(s, ra.offsets, ra.S_r, ra.Tn, ra.k);
  const int rows = sr.nrows - m0, cols = I - n0;
  if (rows <= 0 || cols <= 0) return;
  const B16Src A{(sr.shared ? X : Xp) + (size_t)(sr.xrow0 + m0) * d, nullptr, d, rows, d};
  // byte pointers in the B16Src fields: ld and K count bytes
  const B16Src B{(cbp)(ld_scalar(W.qg + s) + (size_t)n0 * d), (cbp)(ld_scalar(W.qu + s) + (size_t)n0 * d), d, cols,
                 d};
  B16Acc<C::MI, C::NJ> acc;
  acc.zero();
  b16_gemm<C, true, true, false, true>(A, B, d, lds, acc);
  const float* sgp = ld_scalar(W.sg + s) + n0;
  const float* sup = ld_scalar(W.su + s) + n0;
  using SG = Stage<bf16, C::RB / 2>;
  const size_t ob = (size_t)(sr.orow0 + m0);
#pragma unroll
  for (int jj = 0; jj < C::NJ / 2; ++jj)
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      const int col = deinter(b16_coord<C>(0, 2 * jj, q).col4);
      const f32x4_t cg = scale4(sgp, col, cols), cu = scale4(sup, col, cols);
#pragma unroll
      for (int i = 0; i < C::MI; ++i) {
        const AccCoord c = b16_coord<C>(i, 2 * jj, q);
        const f32x4_t ag = acc.quad(i, 2 * jj, q), u = acc.quad(i, 2 * jj + 1, q);
        f32x4_t h;
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          const float a = ag[r] * cg[r];
          h[r] = a * sigm_fast(a) * (u[r] * cu[r]);
        }
        SG::put4(lds, c.row, col, h);
      }
    }
  barrier_lds_writes();
  SG::template copy_out<C::RA, C::THREADS>(lds, H + ob * I + n0, I, rows, cols);
  barrier_lds();
}

// A 128-row int8 tile (same waves and slab depth): the last row tile of a slot
// with at most 128 rows left, and the row halves of a last round.
using CQH = B16Cfg<128, 256, 2, 4, 64, 3, 2, 1>;

// The int8 gate-up product: rounds of whole tiles per XCD as in kb_gate_up, a
// tile with at most 128 rows left taken as a 128-row tile.
__global__ __launch_bounds__(CQ::THREADS) void kq_gate_up(Q8Ptrs W, cbp X, cbp Xp, RowArgs ra, bf16* H) {
  __shared__ __align__(16) char lds[CQ::LDS];
  FM_LDS char* const l = (FM_LDS char*)lds;
  const int NT = (ra.I + CQ::RB / 2 - 1) / (CQ::RB / 2);
  const TileRange tr = row_range(ra, NT);
  const LastRound lr = last_round(tr, false);
  for (long long t = tr.lo + tr.first; t < lr.cut; t += tr.step) {
    const Tile rt = row_tile(ra.mbase, ra.S, NT, t);
    const int m0 = rt.m * CQ::RA, n0 = rt.n * (CQ::RB / 2);
    if (rows_left(ra, rt.s, m0) <= CQH::RA) q8_gate_up_tile<CQH>(W, X, Xp, ra, l, rt.s, m0, n0, H);
    else q8_gate_up_tile<CQ>(W, X, Xp, ra, l, rt.s, m0, n0, H);
  }
  if (lr.parts && tr.first < (tr.hi - lr.cut) * 2) {   // a row half of the last round
    const Tile rt = row_tile(ra.mbase, ra.S, NT, lr.cut + tr.first / 2);
    q8_gate_up_tile<CQH>(W, X, Xp, ra, l, rt.s, rt.m * CQ::RA + (tr.first % 2) * CQH::RA, rt.n * (CQ::RB / 2), H);
  }
}

// One int8-weight down tile of shape C: O = s_d (H Q_d^T).
template <class C>
__device__ __forceinline__ void q8_down_tile(const Q8Ptrs& W, cbp H, const RowArgs& ra, FM_LDS char* lds, int s,
                                             int m0, int n0, bf16* O) {
  const int d = ra.d, I = ra.I;
  const SlotRows sr = slot_rows(s, ra.offsets, ra.S_r, ra.Tn, ra.k);
  const int rows = sr.nrows - m0, cols = d - n0;
  if (rows <= 0 || cols <= 0) return;
  const size_t ob = (size_t)(sr.orow0 + m0);
  const B16Src A{H + ob * I, nullptr, I, rows, I};
  const B16Src B{(cbp)(ld_scalar(W.qd + s) + (size_t)n0 * I), nullptr, I, cols, I};
  B16Acc<C::MI, C::NJ> acc;
  acc.zero();
  b16_gemm<C, true, true>(A, B, I, lds, acc);
  const float* sdp = ld_scalar(W.sd + s) + n0;
#pragma unroll
  for (int j = 0; j < C::NJ; ++j)
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      const f32x4_t c4 = scale4(sdp, b16_coord<C>(0, j, q).col4, cols);
#pragma unroll
      for (int i = 0; i < C::MI; ++i)
#pragma unroll
        for (int r = 0; r < 4; ++r) acc.v[i][j][4 * q + r] *= c4[r];
    }
  b16_store_staged<C>(acc, lds, O + ob * d + n0, d, rows, cols);
}

// O = s_d (H Q_d^T) with int8 Q_d; tiles as in kq_gate_up.
__global__ __launch_bounds__(CQ::THREADS) void kq_down(Q8Ptrs W, cbp H, RowArgs ra, bf16* O) {
  __shared__ __align__(16) char lds[CQ::LDS];
  FM_LDS char* const l = (FM_LDS char*)lds;
  const int NT = (ra.d + CQ::RB - 1) / CQ::RB;
  const TileRange tr = row_range(ra, NT);
  const LastRound lr = last_round(tr, false);
  for (long long t = tr.lo + tr.first; t < lr.cut; t += tr.step) {
    const Tile rt = row_tile(ra.mbase, ra.S, NT, t);
    const int m0 = rt.m * CQ::RA, n0 = rt.n * CQ::RB;
    if (rows_left(ra, rt.s, m0) <= CQH::RA) q8_down_tile<CQH>(W, H, ra, l, rt.s, m0, n0, O);
    else q8_down_tile<CQ>(W, H, ra, l, rt.s, m0, n0, O);
  }
  if (lr.parts && tr.first < (tr.hi - lr.cut) * 2) {   // a row half of the last round
    const Tile rt = row_tile(ra.mbase, ra.S, NT, lr.cut + tr.first / 2);
    q8_down_tile<CQH>(W, H, ra, l, rt.s, rt.m * CQ::RA + (tr.first % 2) * CQH::RA, rt.n * CQ::RB, O);
  }
}

// O = H W_down^T, one tile of shape C at rows m0 of slot s, columns n0.
template <class C>
__device__ __forceinline__ void down_tile(const LayerPtrs<bf16>& W, cbp H, const RowArgs& ra, FM_LDS char* lds,
                                          int s, int m0, int n0, bf16* O) {
  const int d = ra.d, I = ra.I;
  const SlotRows sr = slot_rows(s, ra.offsets, ra.S_r, ra.Tn, ra.k);
  const int rows = sr.nrows - m0, cols = d - n0;
  if (rows <= 0 || cols <= 0) return;
  const size_t ob = (size_t)(sr.orow0 + m0);
  const B16Src A{H + ob * I, nullptr, I, rows, I};
  const B16Src B{ld_scalar(W.wd + s) + (size_t)n0 * I, nullptr, I, cols, I};
  B16Acc<C::MI, C::NJ> acc;
  acc.zero();
  b16_gemm<C, true, true>(A, B, I, lds, acc);
  b16_store_staged<C>(acc, lds, O + ob * d + n0, d, rows, cols);
}

__global__ __launch_bounds__(CB::THREADS) void kb_down(LayerPtrs<bf16> W, cbp H, RowArgs ra, bf16* O) {
  __shared__ __align__(16) char lds[CB::LDS];
  FM_LDS char* const l = (FM_LDS char*)lds;
  const int NT = (ra.d + CB::RB - 1) / CB::RB;
  const TileRange tr = row_range(ra, NT);
  const LastRound lr = last_round(tr, true);
  for (long long t = tr.lo + tr.first; t < lr.cut; t += tr.step) {
    const Tile rt = row_tile(ra.mbase, ra.S, NT, t);
    if (rows_left(ra, rt.s, rt.m * CB::RA) <= CBH::RA)
      down_tile<CBH>(W, H, ra, l, rt.s, rt.m * CB::RA, rt.n * CB::RB, O);
    else
      down_tile<CB>(W, H, ra, l, rt.s, rt.m * CB::RA, rt.n * CB::RB, O);
  }
  if (lr.parts && tr.first < (tr.hi - lr.cut) * lr.parts) {   // a piece of the last round
    const Tile rt = row_tile(ra.mbase, ra.S, NT, lr.cut + tr.first / lr.parts);
    const int p = tr.first % lr.parts;
    if (lr.parts == 4)
      down_tile<CBQ>(W, H, ra, l, rt.s, rt.m * CB::RA + (p >> 1) * CBQ::RA, rt.n * CB::RB + (p & 1) * CBQ::RB, O);
    else
      down_tile<CBH>(W, H, ra, l, rt.s, rt.m * CB::RA + p * CBH::RA, rt.n * CB::RB, O);
  }
}

// dH = dO W_down (B = W_down read k-major), epilogue dA_g, dA_u; one tile of
// shape C at rows m0 of slot s, column tile n (of 256 columns; C::RB = 128 for
// a last column tile with at most 128 columns left).
template <class C>
__device__ __forceinline__ void dh_tile(const LayerPtrs<bf16>& W, cbp dO, cbp Ag, cbp Au, const RowArgs& ra,
                                        FM_LDS char* lds, int s, int m0, int n, int NT, bf16* dAg, bf16* dAu,
                                        float2* norms) {
  static_assert(C::RB == CB::RB || C::RB == CBN::RB, "whole or narrow column tiles");
  const int d = ra.d, I = ra.I, n0 = n * CB::RB;
  const SlotRows sr = slot_rows(s, ra.offsets, ra.S_r, ra.Tn, ra.k);
  const int rows = sr.nrows - m0;
  if (rows <= 0) return;
  const size_t ob = (size_t)(sr.orow0 + m0);
  // B(n = intermediate index, k = hidden index) = W_down[k][n]
  const B16Src A{dO + ob * d, nullptr, d, rows, d};
  const B16Src B{ld_scalar(W.wd + s) + n0, nullptr, I, I - n0, d};
  B16Acc<C::MI, C::NJ> acc;
  acc.zero();
  b16_gemm<C, true, false>(A, B, d, lds, acc);
  b16_dswiglu_staged<C>(acc, lds, Ag + ob * I + n0, Au + ob * I + n0, dAg + ob * ra.ldA + n0,
                        dAu + ob * ra.ldA + n0, I, ra.ldA, rows, I - n0, norms + ob * NT + n, NT);
}

__global__ __launch_bounds__(CB::THREADS) void kb_dh(LayerPtrs<bf16> W, cbp dO, cbp Ag, cbp Au, RowArgs ra,
                                                     bf16* dAg, bf16* dAu, float2* norms) {
  __shared__ __align__(16) char lds[CB::LDS];
  FM_LDS char* const l = (FM_LDS char*)lds;
  const int NT = (ra.I + CB::RB - 1) / CB::RB;
  const TileRange tr = row_range(ra, NT);
  const LastRound lr = last_round(tr, false);
  for (long long t = tr.lo + tr.first; t < lr.cut; t += tr.step) {
    const Tile rt = row_tile(ra.mbase, ra.S, NT, t);
    if (ra.I - rt.n * CB::RB <= CBN::RB)
      dh_tile<CBN>(W, dO, Ag, Au, ra, l, rt.s, rt.m * CB::RA, rt.n, NT, dAg, dAu, norms);
    else if (rows_left(ra, rt.s, rt.m * CB::RA) <= CBH::RA)
      dh_tile<CBH>(W, dO, Ag, Au, ra, l, rt.s, rt.m * CB::RA, rt.n, NT, dAg, dAu, norms);
    else
      dh_tile<CB>(W, dO, Ag, Au, ra, l, rt.s, rt.m * CB::RA, rt.n, NT, dAg, dAu, norms);
  }
  if (lr.parts && tr.first < (tr.hi - lr.cut) * 2) {   // a row half of the last round
    const Tile rt = row_tile(ra.mbase, ra.S, NT, lr.cut + tr.first / 2);
    dh_tile<CBH>(W, dO, Ag, Au, ra, l, rt.s, rt.m * CB::RA + (tr.first % 2) * CBH::RA, rt.n, NT, dAg, dAu,
                 norms);
  }
}

// dX_s = dA_g W_gate + dA_u W_up (B read k-major), one tile of shape C at rows
// m0 of slot s, columns n0.  With I a whole number of slabs the two products
// run as one K loop of 2I (one prologue and one drain per tile); otherwise as
// two K passes.  Either way k runs over dA_g W_gate first: the same sums.
template <class C>
__device__ __forceinline__ void dx_tile(const LayerPtrs<bf16>& W, cbp dAg, cbp dAu, const RowArgs& ra,
                                        FM_LDS char* lds, int s, int m0, int n0, bf16* dXp) {
  const int d = ra.d, I = ra.I;
  const SlotRows sr = slot_rows(s, ra.offsets, ra.S_r, ra.Tn, ra.k);
  const int rows = sr.nrows - m0, cols = d - n0;
  if (rows <= 0 || cols <= 0) return;
  const size_t ob = (size_t)(sr.orow0 + m0);
  B16Acc<C::MI, C::NJ> acc;
  acc.zero();
  // B(n = hidden index, k = intermediate index) = W_gate[k][n], then W_up
  cbp wg = ld_scalar(W.wg + s) + n0, wu = ld_scalar(W.wu + s) + n0;
  if (I % C::BK == 0) {
    b16_gemm<C, true, false, false, false, -1, true>(
        B16Src{dAg + ob * ra.ldA, nullptr, ra.ldA, rows, 2 * I, dAu + ob * ra.ldA, I},
        B16Src{wg, nullptr, d, cols, 2 * I, wu, I}, 2 * I, lds, acc);
  } else {
    b16_gemm<C, true, false>(B16Src{dAg + ob * ra.ldA, nullptr, ra.ldA, rows, I},
                             B16Src{wg, nullptr, d, cols, I}, I, lds, acc);
    b16_gemm<C, true, false>(B16Src{dAu + ob * ra.ldA, nullptr, ra.ldA, rows, I},
                             B16Src{wu, nullptr, d, cols, I}, I, lds, acc);
  }
  b16_store_staged<C>(acc, lds, dXp + ob * d + n0, d, rows, cols);
}

__global__ __launch_bounds__(CB::THREADS) void kb_dx(LayerPtrs<bf16> W, cbp dAg, cbp dAu, RowArgs ra,
                                                     bf16* dXp) {
  __shared__ __align__(16) char lds[CB::LDS];
  FM_LDS char* const l = (FM_LDS char*)lds;
  const int NT = (ra.d + CB::RB - 1) / CB::RB;
  const TileRange tr = row_range(ra, NT);
  const LastRound lr = last_round(tr, true);
  for (long long t = tr.lo + tr.first; t < lr.cut; t += tr.step) {
    const Tile rt = row_tile(ra.mbase, ra.S, NT, t);
    if (rows_left(ra, rt.s, rt.m * CB::RA) <= CBH::RA)
      dx_tile<CBH>(W, dAg, dAu, ra, l, rt.s, rt.m * CB::RA, rt.n * CB::RB, dXp);
    else
      dx_tile<CB>(W, dAg, dAu, ra, l, rt.s, rt.m * CB::RA, rt.n * CB::RB, dXp);
  }
  if (lr.parts && tr.first < (tr.hi - lr.cut) * lr.parts) {   // a piece of the last round
    const Tile rt = row_tile(ra.mbase, ra.S, NT, lr.cut + tr.first / lr.parts);
    const int p = tr.first % lr.parts;
    if (lr.parts == 4)
      dx_tile<CBQ>(W, dAg, dAu, ra, l, rt.s, rt.m * CB::RA + (p >> 1) * CBQ::RA, rt.n * CB::RB + (p & 1) * CBQ::RB,
                   dXp);
    else
      dx_tile<CBH>(W, dAg, dAu, ra, l, rt.s, rt.m * CB::RA + p * CBH::RA, rt.n * CB::RB, dXp);
  }
}

// Weight-gradient tiles of one kernel run as a pipeline: the next tile's first
// slabs are issued (b16_prologue) before the current tile's epilogue stores,
// so the stores drain while those slabs land.  Every wave issues exactly
// MI x NJ x 4 stores per tile (lanes outside the output write to the sink),
// which the next product's first wait may leave in flight; with accumulate
// each store is preceded by a load and the wait counts none of them.
template <bool ACCUM> struct DwEpi {
  static constexpr int STORES = CB::MI * CB::NJ * 4;
  static constexpr int EXTRA = ACCUM ? 0 : STORES;
};

__device__ __forceinline__ float* dw_sink(const DwArgs& da) {
  return da.sink + (size_t)((blockIdx.x * CB::THREADS + threadIdx.x) & (DW_SINK - 1)) * 4;
}

// dW_gate = dA_g^T X_s and dW_up = dA_u^T X_s in one product: the A tile
// interleaves 32-column blocks of dA_g and dA_u (128 intermediate rows of both
// per 256-row tile), B = X_s; both read k-major.
struct DwGuTile {
  float* dwg;
  float* dwu;
  int m0, n0, K;
  bool run;
  B16Src A, B;
  __device__ __forceinline__ void init(const LayerPtrs<bf16>& W, cbp X, cbp Xp, cbp dAg, cbp dAu, const DwArgs& da,
                                      long long t, int MT, int NT) {
    Tile rt = dw_tile(t, MT * NT, MT);
    rt.s = ld_scalar(da.dorder + rt.s);
    dwg = ld_scalar(W.dwg + rt.s);
    dwu = ld_scalar(W.dwu + rt.s);
    run = dwg && dwu;
    const SlotRows sr = slot_rows(rt.s, da.offsets, da.S_r, da.Tn, da.k);
    const int d = da.d, I = da.I;
    m0 = rt.m * (CB::RA / 2);
    n0 = rt.n * CB::RB;
    K = sr.nrows;
    A = B16Src{dAg + (size_t)sr.orow0 * da.ldA + m0, dAu + (size_t)sr.orow0 * da.ldA + m0, da.ldA, I - m0,
               sr.nrows};
    B = B16Src{(sr.shared ? X : Xp) + (size_t)sr.xrow0 * d + n0, nullptr, d, d - n0, sr.nrows};
  }
};

template <bool ACCUM>
__global__ __launch_bounds__(CB::THREADS) void kb_dw_gu(LayerPtrs<bf16> W, cbp X, cbp Xp, cbp dAg, cbp dAu,
                                                        DwArgs da) {
  __shared__ __align__(16) char lds[CB::LDS];
  FM_LDS char* const l = (FM_LDS char*)lds;
  const int d = da.d, I = da.I;
  const int MT = (I + CB::RA / 2 - 1) / (CB::RA / 2), NT = (d + CB::RB - 1) / CB::RB;
  const DwQueue qu(da, MT * NT);
  float* const sink = dw_sink(da);
  int j = DwQueue::share(l, threadIdx.x == 0 ? qu.draw() : 0);
  barrier_lds();
  long long t = qu.tile(j);
  if (t < qu.total) {
    DwGuTile o;
    o.init(W, X, Xp, dAg, dAu, da, t, MT, NT);
    if (o.run) b16_prologue<CB, false, false, true, false>(o.A, o.B, o.K, l);
  }
  bool stored = false;   // the previous tile's stores may be in flight
  while (t < qu.total) {
#pragma clang diagnostic push
#pragma clang diagnostic ignored "-Wsometimes-uninitialized"
    int next;   // meaningful in thread 0 only (no default: it would cost a wait on the atomic)
    if (threadIdx.x == 0) next = qu.draw();
#pragma clang diagnostic pop
    DwGuTile o;   // tile tables are read through the scalar cache
    o.init(W, X, Xp, dAg, dAu, da, t, MT, NT);
    B16Acc<CB::MI, CB::NJ> acc;
    if (o.run) {
      acc.zero();
      b16_gemm<CB, false, false, true, false, DwEpi<ACCUM>::EXTRA>(o.A, o.B, o.K, l, acc, stored);
    }
    j = DwQueue::share(l, next);
    barrier_lds();   // every wave has read the draw before the next tile's DMA
    t = qu.tile(j);
    if (t < qu.total) {
      DwGuTile on;
      on.init(W, X, Xp, dAg, dAu, da, t, MT, NT);
      if (on.run) b16_prologue<CB, false, false, true, false>(on.A, on.B, on.K, l);
    }
    stored = o.run;
    if (o.run) {
#pragma unroll
      for (int i = 0; i < CB::MI; ++i)
#pragma unroll
        for (int jj = 0; jj < CB::NJ; ++jj)
#pragma unroll
          for (int q = 0; q < 4; ++q) {
            const AccCoord c = b16_coord<CB>(i, jj, q);
            const int m = o.m0 + deinter(c.row), n = o.n0 + c.col4;
            float* dst = (m < I && n < d) ? (((c.row >> 5) & 1) ? o.dwu : o.dwg) + (size_t)m * d + n : sink;
            store_dw(dst, acc.quad(i, jj, q), ACCUM);
          }
    }
  }
}

// dW_down = dO^T H (both read k-major).  Rows over d, columns over I; a last
// column tile with at most 128 columns left runs as a 256 x 128 tile (CBN).
// Band height of the dW_down tile order: the XCDs are dealt tiles t = 8 j + x,
// so with 8 row tiles per band (d = 2048: the whole slot) the last column's 8
// tiles of a band land on 8 different XCDs, one narrow tile each.
constexpr int GM_DWD = 8;

struct DwDTile {
  float* dwd;
  int m0, n0, K;
  bool run, narrow;
  B16Src A, B;
  __device__ __forceinline__ void init(const LayerPtrs<bf16>& W, cbp dO, cbp H, const DwArgs& da, long long t, int MT,
                                      int NT) {
    Tile rt = dw_tile(t, MT * NT, MT, GM_DWD);
    rt.s = ld_scalar(da.dorder + rt.s);
    dwd = ld_scalar(W.dwd + rt.s);
    run = dwd != nullptr;
    const SlotRows sr = slot_rows(rt.s, da.offsets, da.S_r, da.Tn, da.k);
    const int d = da.d, I = da.I;
    m0 = rt.m * CB::RA;
    n0 = rt.n * CB::RB;
    narrow = I - n0 <= CBN::RB;
    K = sr.nrows;
    A = B16Src{dO + (size_t)sr.orow0 * d + m0, nullptr, d, d - m0, sr.nrows};
    B = B16Src{H + (size_t)sr.orow0 * I + n0, nullptr, I, I - n0, sr.nrows};
  }
  __device__ __forceinline__ void prologue(FM_LDS char* l) const {
    if (!run) return;
    if (narrow) b16_prologue<CBN, false, false>(A, B, K, l);
    else b16_prologue<CB, false, false>(A, B, K, l);
  }
};

// One dW_down tile of shape C: the product (its prologue was issued with the
// same shape), the hand-over of the next draw, the next tile's prologue, then
// this tile's stores.  Every wave issues exactly DwEpi's store count (a 256 x 128
// tile has half as many outputs; its other stores go to the sink), the number
// the next product's first wait lets stay in flight.
template <class C, bool ACCUM>
__device__ __forceinline__ long long dwd_step(const LayerPtrs<bf16>& W, cbp dO, cbp H, const DwArgs& da,
                                              const DwQueue& qu, FM_LDS char* l, const DwDTile& o, int next,
                                              bool stored, int MT, int NT, float* sink) {
  static_assert(C::MI * C::NJ * 4 <= DwEpi<ACCUM>::STORES || ACCUM, "store count");
  const int d = da.d, I = da.I;
  B16Acc<C::MI, C::NJ> acc;
  if (o.run) {
    acc.zero();
    b16_gemm<C, false, false, false, false, DwEpi<ACCUM>::EXTRA>(o.A, o.B, o.K, l, acc, stored);
  }
  const int j = DwQueue::share(l, next);
  barrier_lds();
  const long long t = qu.tile(j);
  if (t < qu.total) {
    DwDTile on;
    on.init(W, dO, H, da, t, MT, NT);
    on.prologue(l);
  }
  if (o.run) {
#pragma unroll
    for (int i = 0; i < C::MI; ++i)
#pragma unroll
      for (int jj = 0; jj < C::NJ; ++jj)
#pragma unroll
        for (int q = 0; q < 4; ++q) {
          const AccCoord c = b16_coord<C>(i, jj, q);
          const int m = o.m0 + c.row, n = o.n0 + c.col4;
          float* dst = (m < d && n < I) ? o.dwd + (size_t)m * I + n : sink;
          store_dw(dst, acc.quad(i, jj, q), ACCUM);
        }
    if (!ACCUM) {   // volatile: stores to one address must not be merged away
      const f32x4_t z = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int u = C::MI * C::NJ * 4; u < DwEpi<ACCUM>::STORES; ++u) *(volatile FM_GLOBAL f32x4_t*)sink = z;
    }
  }
  return t;
}

template <bool ACCUM>
__global__ __launch_bounds__(CB::THREADS) void kb_dw_d(LayerPtrs<bf16> W, cbp dO, cbp H, DwArgs da) {
  __shared__ __align__(16) char lds[CB::LDS];
  FM_LDS char* const l = (FM_LDS char*)lds;
  const int d = da.d, I = da.I;
  const int MT = (d + CB::RA - 1) / CB::RA, NT = (I + CB::RB - 1) / CB::RB;
  const DwQueue qu(da, MT * NT);
  float* const sink = dw_sink(da);
  int j = DwQueue::share(l, threadIdx.x == 0 ? qu.draw() : 0);
  barrier_lds();
  long long t = qu.tile(j);
  if (t < qu.total) {
    DwDTile o;
    o.init(W, dO, H, da, t, MT, NT);
    o.prologue(l);
  }
  bool stored = false;
  while (t < qu.total) {
#pragma clang diagnostic push
#pragma clang diagnostic ignored "-Wsometimes-uninitialized"
    int next;   // meaningful in thread 0 only (no default: it would cost a wait on the atomic)
    if (threadIdx.x == 0) next = qu.draw();
#pragma clang diagnostic pop
    DwDTile o;
    o.init(W, dO, H, da, t, MT, NT);
    const long long tn = o.narrow ? dwd_step<CBN, ACCUM>(W, dO, H, da, qu, l, o, next, stored, MT, NT, sink)
                                  : dwd_step<CB, ACCUM>(W, dO, H, da, qu, l, o, next, stored, MT, NT, sink);
    stored = o.run;
    t = tn;
  }
}

// ----------------------------------------- expert utility (Eq. 3) ----
//
// u_s = |D_s| sqrt(mean over the slot's rows of ||g_r||^2), where the weight
// gradient of one row is three rank-one outer products, so
//   ||g_r||^2 = ||dO_r||^2 ||h_r||^2 + (||dA_g,r||^2 + ||dA_u,r||^2) ||x_r||^2.
// A slot's rows are its tokens after folding (a token whose choices share the
// slot is one row with the summed gate), so |D_s| is the slot's row count.
// The backward's dH epilogue leaves per row the partial sums of dA_g^2 + dA_u^2
// and h^2 over its column tiles; a row's x is its token's input and its dO the
// token's output gradient times the row's gate, so the rest needs only the
// tokens' ||x_t||^2 and ||dY_t||^2, which the permutation and the combine
// backward write as they read X and dY.

constexpr int UT_THREADS = 256;    // threads of the per-row pass: one row each
constexpr int UT_PB = 4;           // norm partials of a row loaded together
constexpr int US_THREADS = 1024;   // threads of the per-slot pass: one block per slot
constexpr int US_BATCH = 8;        // row values per thread loaded together

// Per-row pass over the whole row space (routed rows [0, T*k), of which the
// first offsets[S_r] are used, then T rows per shared expert): a thread forms
// its row's ||g_r||^2 in fp64 from the row's token norms, its gate and its P
// partials (in order) and stores it at vrow[row].  The token of a routed row
// is read before it is known whether the row is used (the row count is read in
// parallel); an unused row's token is clamped into [0, T) so that its norm
// loads stay in bounds, and its value is not stored.  With no routed slot the
// routed rows are skipped (the maps may then be NULL).
__global__ __launch_bounds__(UT_THREADS) void k_utility_rows(RowArgs ra, const int32_t* __restrict__ perm_token,
                                                             const float* __restrict__ perm_gate,
                                                             const float* __restrict__ x_sq,
                                                             const float* __restrict__ dy_sq,
                                                             const float2* __restrict__ norms, int P,
                                                             double* __restrict__ vrow) {
  const long R = (long)ra.Tn * ra.k;
  const long r = (long)blockIdx.x * UT_THREADS + threadIdx.x;
  if (r >= R + (long)ra.Tn * (ra.S - ra.S_r)) return;
  const bool routed = r < R;
  if (routed && ra.S_r == 0) return;   // no routed slot: the maps may be NULL
  const int used = ra.S_r > 0 ? ld_scalar(ra.offsets + ra.S_r) : 0;
  int tok;
  float g = 1.f;
  if (routed) {
    tok = min(max(perm_token[r], 0), ra.Tn - 1);
    g = perm_gate[r];
  } else {
    tok = (int)((r - R) % ra.Tn);
  }
  float sa = 0.f, sh = 0.f;
  for (int p0 = 0; p0 < P; p0 += UT_PB) {
    float2 q[UT_PB];
#pragma unroll
    for (int c = 0; c < UT_PB; ++c) q[c] = norms[r * P + min(p0 + c, P - 1)];
#pragma unroll
    for (int c = 0; c < UT_PB; ++c)
      if (p0 + c < P) {
        sa += q[c].x;
        sh += q[c].y;
      }
  }
  const float xx = x_sq[tok], yy = dy_sq[tok];
  if (!routed || r < used) vrow[r] = (double)g * g * yy * sh + (double)sa * xx;
}

// Per-slot pass, one block per slot: a thread adds the row values i, i + 1024,
// ... of the slot (US_BATCH loads in flight, added in row order); the block
// adds its threads by a fixed butterfly per wave, then the waves in order.
__global__ __launch_bounds__(US_THREADS) void k_utility_slots(RowArgs ra, const double* __restrict__ vrow,
                                                              float* __restrict__ u) {
  __shared__ double wsum[US_THREADS / 64];
  const int s = blockIdx.x, i = threadIdx.x;
  const SlotRows sr = slot_rows(s, ra.offsets, ra.S_r, ra.Tn, ra.k);
  const double* v = vrow + sr.orow0;
  double sum = 0.0;
  for (int r0 = 0; r0 < sr.nrows; r0 += US_BATCH * US_THREADS) {
    double x[US_BATCH];
#pragma unroll
    for (int e = 0; e < US_BATCH; ++e) {
      const int r = r0 + e * US_THREADS + i;
      x[e] = r < sr.nrows ? v[r] : 0.0;
    }
#pragma unroll
    for (int e = 0; e < US_BATCH; ++e)
      if (r0 + e * US_THREADS + i < sr.nrows) sum += x[e];
  }
  // the butterfly leaves the same sum in every lane (each step adds two equal
  // partial sums, in one order or the other)
#pragma unroll
  for (int off = 32; off > 0; off >>= 1) sum += __shfl_xor(sum, off);
  if ((i & 63) == 0) wsum[i >> 6] = sum;
  __syncthreads();
  if (i == 0) {
    double t = 0.0;
#pragma unroll
    for (int w = 0; w < US_THREADS / 64; ++w) t += wsum[w];
    u[s] = sr.nrows > 0 ? (float)sqrt((double)sr.nrows * t) : 0.f;
  }
}

__global__ void k_zero_f32(float* p, int n) {
  const int i = blockIdx.x * blockDim.x + threadIdx.x;
  if (i < n) p[i] = 0.f;
}

// ------------------------------------------------------------------ host ----

int check_layer_ffn(const moe_layer* L) {
  if (!L) return fail(MOE_ERR_ARG, "layer must not be NULL");
  if (L->d <= 0 || L->I <= 0) return fail(MOE_ERR_ARG, "layer d=%d I=%d", L->d, L->I);
  if (L->d % 8 || L->I % 8)
    return fail(MOE_ERR_UNSUPPORTED, "layer d=%d I=%d must be multiples of 8", L->d, L->I);
  if (L->S_routed < 0 || L->S_shared < 0 || L->S_routed + L->S_shared < 1 || L->S_routed > 512 ||
      L->S_shared > 511)
    return fail(MOE_ERR_ARG, "layer S_routed=%d S_shared=%d", L->S_routed, L->S_shared);
  FM_TRY(need_dtype_float(L->dtype, "layer dtype"));
  FM_TRY(need(L->w_gate, "layer w_gate")); FM_TRY(need(L->w_up, "layer w_up"));
  FM_TRY(need(L->w_down, "layer w_down"));
  return MOE_OK;
}


size_t rows_total(const moe_layer* L, int T, int k) { return (size_t)T * (k + L->S_shared); }
int n_slots(const moe_layer* L) { return L->S_routed + L->S_shared; }

// Persistent grid: one block per compute unit, a multiple of the XCD count.
int persistent_blocks() {
  int dev = 0, n = 0;
  if (hipGetDevice(&dev) != hipSuccess ||
      hipDeviceGetAttribute(&n, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess || n <= 0)
    n = 256;
  n = (n / N_XCD) * N_XCD;
  return n < N_XCD ? N_XCD : n;
}

}  // namespace
}  // namespace fm

using namespace fm;

extern "C" size_t moe_grouped_swiglu_fwd_workspace_size(const moe_layer* L, int T, int k) {
  if (!L || T < 0 || k <= 0) return 0;
  return sched_bytes(n_slots(L));
}

// Rows per row tile of the backward (bf16 or fp32 core).
static int bwd_tile_rows(const moe_layer* L) { return L->dtype == MOE_BF16 ? B16_ROWS : G_BM; }
// Partials of the utility's row norms per row: one per dH column tile (bf16),
// two per column tile (fp32, one per wave column).
static int norm_parts(const moe_layer* L) {
  return L->dtype == MOE_BF16 ? (L->I + CB::RB - 1) / CB::RB : 2 * ((L->I + G_BN - 1) / G_BN);
}

// Backward workspace: schedule | dA_g | dA_u | per-row norm partials (float2) |
// the utility's per-row values (double).
struct BwdWs {
  char* dAg;
  char* dAu;
  float2* norms;
  double* vrow;
};
// Row stride of dA_g and dA_u in the backward's workspace.  bf16 rows are
// padded to whole 128-byte lines (a row of I = 688 would otherwise start inside
// a line three times in four, and every 128-byte slab row of the products that
// read dA would span two lines); the padding columns are never written or read.
static int act_ld(const moe_layer* L) { return L->dtype == MOE_BF16 ? (L->I + 63) / 64 * 64 : L->I; }
static size_t bwd_act_bytes(const moe_layer* L, int T, int k) {
  return round256(rows_total(L, T, k) * act_ld(L) * esize(L->dtype));
}
static BwdWs bwd_ws_at(void* ws, const moe_layer* L, int T, int k) {
  BwdWs w;
  const size_t act = bwd_act_bytes(L, T, k);
  char* p = (char*)ws + sched_bytes(n_slots(L));
  w.dAg = p;
  w.dAu = p + act;
  p += 2 * act;
  w.norms = (float2*)p;
  p += round256(sizeof(float2) * rows_total(L, T, k) * norm_parts(L));
  w.vrow = (double*)p;
  return w;
}

extern "C" size_t moe_grouped_swiglu_bwd_workspace_size(const moe_layer* L, int T, int k) {
  if (!L || T < 0 || k <= 0) return 0;
  return sched_bytes(n_slots(L)) + 2 * bwd_act_bytes(L, T, k) +
         round256(sizeof(float2) * rows_total(L, T, k) * norm_parts(L)) +
         round256(sizeof(double) * rows_total(L, T, k));
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
  hipStream_t st = as_stream(stream);
  if (debug_checks() && L->S_routed > 0) FM_TRY(debug_check_offsets(offsets, L->S_routed, T, k, st));
  const int S = n_slots(L);
  const Sched sc = sched_at(ws, S);
  const int tile_rows = bwd_tile_rows(L);
  hipLaunchKernelGGL(k_build_sched, dim3(1), dim3(1024), 0, st, offsets, L->S_routed, L->S_shared, T, tile_rows,
                     (float* const*)nullptr, sc.mbase, sc.wbase, sc.dorder, sc.queues);
  const RowArgs ra{offsets, sc.mbase, L->S_routed, S, T, k, L->d, L->I, L->I};
  const dim3 grid(persistent_blocks()), block(G_THREADS);
#define FM_FWD(TT)                                                                                      \
  hipLaunchKernelGGL(kf_gate_up<TT>, grid, block, 0, st, layer_ptrs<TT>(L), (const TT*)X, (const TT*)X_perm, \
                     ra, (TT*)A_g, (TT*)A_u, (TT*)H);                                                   \
  hipLaunchKernelGGL(kf_down<TT>, grid, block, 0, st, layer_ptrs<TT>(L), (const TT*)H, ra, (TT*)O);
  if (L->dtype == MOE_BF16) {
    const dim3 b8(CB::THREADS);
    hipLaunchKernelGGL(kb_gate_up, grid, b8, 0, st, layer_ptrs<bf16>(L), (cbp)X, (cbp)X_perm, ra, (bf16*)A_g,
                       (bf16*)A_u, (bf16*)H);
    hipLaunchKernelGGL(kb_down, grid, b8, 0, st, layer_ptrs<bf16>(L), (cbp)H, ra, (bf16*)O);
  } else {
    FM_FWD(float)
  }
#undef FM_FWD
  return check_launch("moe_grouped_swiglu_fwd");
}

extern "C" size_t moe_grouped_swiglu_fwd_q8_workspace_size(const moe_layer_q8* L, int T, int k) {
  if (!L || T < 0 || k <= 0) return 0;
  return sched_bytes(L->S_routed + L->S_shared);
}

extern "C" int moe_grouped_swiglu_fwd_q8(const moe_layer_q8* L, const void* X, const void* X_perm,
                                         const int32_t* offsets, int T, int k, void* H, void* O, void* ws,
                                         size_t ws_bytes, void* stream) {
  clear_error();
  if (!L) return fail(MOE_ERR_ARG, "layer must not be NULL");
  if (L->d <= 0 || L->I <= 0) return fail(MOE_ERR_ARG, "layer d=%d I=%d", L->d, L->I);
  if (L->d % 16 || L->I % 16)
    return fail(MOE_ERR_UNSUPPORTED, "int8 layer d=%d I=%d must be multiples of 16", L->d, L->I);
  if (L->S_routed < 0 || L->S_shared < 0 || L->S_routed + L->S_shared < 1 || L->S_routed > 512 ||
      L->S_shared > 511)
    return fail(MOE_ERR_ARG, "layer S_routed=%d S_shared=%d", L->S_routed, L->S_shared);
  FM_TRY(need(L->q_gate, "layer q_gate")); FM_TRY(need(L->q_up, "layer q_up"));
  FM_TRY(need(L->q_down, "layer q_down")); FM_TRY(need(L->s_gate, "layer s_gate"));
  FM_TRY(need(L->s_up, "layer s_up")); FM_TRY(need(L->s_down, "layer s_down"));
  if (T < 0 || k <= 0 || k > 16) return fail(MOE_ERR_ARG, "T=%d k=%d", T, k);
  if (T == 0) return MOE_OK;
  FM_TRY(need(X, "X")); FM_TRY(need(offsets, "offsets")); FM_TRY(need(H, "H")); FM_TRY(need(O, "O"));
  FM_TRY(need(ws, "ws"));
  if (L->S_routed > 0) FM_TRY(need(X_perm, "X_perm"));
  FM_TRY(need_aligned(X, "X")); FM_TRY(need_aligned(X_perm, "X_perm")); FM_TRY(need_aligned(H, "H"));
  FM_TRY(need_aligned(O, "O")); FM_TRY(need_aligned(ws, "ws"));
  if (ws_bytes < moe_grouped_swiglu_fwd_q8_workspace_size(L, T, k))
    return fail(MOE_ERR_WORKSPACE, "workspace %zu < %zu bytes", ws_bytes,
                moe_grouped_swiglu_fwd_q8_workspace_size(L, T, k));
  hipStream_t st = as_stream(stream);
  if (debug_checks() && L->S_routed > 0) FM_TRY(debug_check_offsets(offsets, L->S_routed, T, k, st));
  const int S = L->S_routed + L->S_shared;
  const Sched sc = sched_at(ws, S);
  hipLaunchKernelGGL(k_build_sched, dim3(1), dim3(1024), 0, st, offsets, L->S_routed, L->S_shared, T, CQ::RA,
                     (float* const*)nullptr, sc.mbase, sc.wbase, sc.dorder, sc.queues);
  const RowArgs ra{offsets, sc.mbase, L->S_routed, S, T, k, L->d, L->I, L->I};
  const Q8Ptrs W{L->q_gate, L->q_up, L->q_down, L->s_gate, L->s_up, L->s_down};
  const dim3 grid(persistent_blocks()), block(CQ::THREADS);
  hipLaunchKernelGGL(kq_gate_up, grid, block, 0, st, W, (cbp)X, (cbp)X_perm, ra, (bf16*)H);
  hipLaunchKernelGGL(kq_down, grid, block, 0, st, W, (cbp)H, ra, (bf16*)O);
  return check_launch("moe_grouped_swiglu_fwd_q8");
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
  // With no tokens only the zeroing of the weight gradients runs: it reads the
  // offsets and the schedule workspace, no per-token buffer (those may be NULL).
  FM_TRY(need(offsets, "offsets")); FM_TRY(need(ws, "ws"));
  if (T > 0) {
    FM_TRY(need(X, "X")); FM_TRY(need(A_g, "A_g")); FM_TRY(need(A_u, "A_u")); FM_TRY(need(H, "H"));
    FM_TRY(need(dO, "dO")); FM_TRY(need(dX_perm, "dX_perm"));
    if (L->S_routed > 0) FM_TRY(need(X_perm, "X_perm"));
  }
  FM_TRY(need_aligned(X, "X")); FM_TRY(need_aligned(X_perm, "X_perm")); FM_TRY(need_aligned(A_g, "A_g"));
  FM_TRY(need_aligned(A_u, "A_u")); FM_TRY(need_aligned(H, "H")); FM_TRY(need_aligned(dO, "dO"));
  FM_TRY(need_aligned(dX_perm, "dX_perm")); FM_TRY(need_aligned(ws, "ws"));
  if (ws_bytes < moe_grouped_swiglu_bwd_workspace_size(L, T, k))
    return fail(MOE_ERR_WORKSPACE, "workspace %zu < %zu bytes", ws_bytes,
                moe_grouped_swiglu_bwd_workspace_size(L, T, k));
  hipStream_t st = as_stream(stream);
  if (debug_checks() && T > 0 && L->S_routed > 0) FM_TRY(debug_check_offsets(offsets, L->S_routed, T, k, st));
  const int S = n_slots(L);
  const Sched sc = sched_at(ws, S);
  const BwdWs bw = bwd_ws_at(ws, L, T, k);
  char* dAg = bw.dAg;
  char* dAu = bw.dAu;
  const int d = L->d, I = L->I;
  const int tile_rows = bwd_tile_rows(L);
  hipLaunchKernelGGL(k_build_sched, dim3(1), dim3(1024), 0, st, offsets, L->S_routed, L->S_shared, T, tile_rows,
                     L->dw_gate, sc.mbase, sc.wbase, sc.dorder, sc.queues);
  const int ldA = act_ld(L);
  const RowArgs ra{offsets, sc.mbase, L->S_routed, S, T, k, d, I, ldA};
  const DwArgs da{offsets, sc.wbase, sc.dorder, sc.queues, sc.sink, L->S_routed, S, T, k, d, I, accumulate_dw,
                  ldA};
  DwArgs da_d = da;
  da_d.queue = sc.queues + N_XCD * DW_QSTRIDE;
  const dim3 grid(persistent_blocks()), block(G_THREADS);
#define FM_BWD(TT)                                                                                        \
  if (T > 0) {                                                                                            \
    hipLaunchKernelGGL(kf_dh<TT>, grid, block, 0, st, layer_ptrs<TT>(L), (const TT*)dO, (const TT*)A_g,   \
                       (const TT*)A_u, ra, (TT*)dAg, (TT*)dAu, bw.norms);                                \
    hipLaunchKernelGGL(kf_dx<TT>, grid, block, 0, st, layer_ptrs<TT>(L), (const TT*)dAg, (const TT*)dAu, \
                       ra, (TT*)dX_perm);                                                                \
  }                                                                                                       \
  hipLaunchKernelGGL(kf_dw_gu<TT>, grid, block, 0, st, layer_ptrs<TT>(L), (const TT*)X, (const TT*)X_perm, \
                     (const TT*)dAg, (const TT*)dAu, da);                                                \
  hipLaunchKernelGGL(kf_dw_d<TT>, grid, block, 0, st, layer_ptrs<TT>(L), (const TT*)dO, (const TT*)H, da);
  if (L->dtype == MOE_BF16) {
    // dX goes last (both weight gradients first): the permutation backward
    // that follows reads dX_perm while it is still in the memory-side cache
    // (measured 79 -> 62 us for it at T = 8192, d = 2048, k = 6 + 2 shared,
    // with the 1.45 GB of fp32 weight gradients written before dX instead of
    // between dX and that read).
    const dim3 b8(CB::THREADS);
    if (T > 0)
      hipLaunchKernelGGL(kb_dh, grid, b8, 0, st, layer_ptrs<bf16>(L), (cbp)dO, (cbp)A_g, (cbp)A_u, ra,
                         (bf16*)dAg, (bf16*)dAu, bw.norms);
    if (accumulate_dw) {
      hipLaunchKernelGGL(kb_dw_d<true>, grid, b8, 0, st, layer_ptrs<bf16>(L), (cbp)dO, (cbp)H, da_d);
      hipLaunchKernelGGL(kb_dw_gu<true>, grid, b8, 0, st, layer_ptrs<bf16>(L), (cbp)X, (cbp)X_perm, (cbp)dAg,
                         (cbp)dAu, da);
    } else {
      hipLaunchKernelGGL(kb_dw_d<false>, grid, b8, 0, st, layer_ptrs<bf16>(L), (cbp)dO, (cbp)H, da_d);
      hipLaunchKernelGGL(kb_dw_gu<false>, grid, b8, 0, st, layer_ptrs<bf16>(L), (cbp)X, (cbp)X_perm, (cbp)dAg,
                         (cbp)dAu, da);
    }
    if (T > 0)
      hipLaunchKernelGGL(kb_dx, grid, b8, 0, st, layer_ptrs<bf16>(L), (cbp)dAg, (cbp)dAu, ra, (bf16*)dX_perm);
  } else {
    FM_BWD(float)
  }
#undef FM_BWD
  return check_launch("moe_grouped_swiglu_bwd");
}

extern "C" int moe_expert_utility(const moe_layer* L, const float* x_sq, const float* dy_sq,
                                  const int32_t* perm_token, const float* perm_gate, const int32_t* offsets, int T,
                                  int k, void* ws, size_t ws_bytes, float* utility, void* stream) {
  clear_error();
  FM_TRY(check_layer_ffn(L));
  if (T < 0 || k <= 0 || k > 16) return fail(MOE_ERR_ARG, "T=%d k=%d", T, k);
  FM_TRY(need(utility, "utility")); FM_TRY(need_aligned(utility, "utility"));
  const int S = n_slots(L);
  hipStream_t st = as_stream(stream);
  if (T == 0) {
    hipLaunchKernelGGL(k_zero_f32, dim3(cdiv(S, 256)), dim3(256), 0, st, utility, S);
    return check_launch("moe_expert_utility");
  }
  FM_TRY(need(x_sq, "x_sq")); FM_TRY(need(dy_sq, "dy_sq")); FM_TRY(need(offsets, "offsets"));
  FM_TRY(need(ws, "ws"));
  if (L->S_routed > 0) {
    FM_TRY(need(perm_token, "perm_token")); FM_TRY(need(perm_gate, "perm_gate"));
  }
  FM_TRY(need_aligned(x_sq, "x_sq")); FM_TRY(need_aligned(dy_sq, "dy_sq")); FM_TRY(need_aligned(ws, "ws"));
  if (ws_bytes < moe_grouped_swiglu_bwd_workspace_size(L, T, k))
    return fail(MOE_ERR_WORKSPACE, "workspace %zu < %zu bytes", ws_bytes,
                moe_grouped_swiglu_bwd_workspace_size(L, T, k));
  if (debug_checks() && L->S_routed > 0) {
    FM_TRY(debug_check_offsets(offsets, L->S_routed, T, k, st));
    int rows = 0;
    FM_TRY(debug_rows(offsets, L->S_routed, st, &rows));
    FM_TRY(debug_check_tokens(perm_token, rows, T, st));
  }
  // the per-row partials the backward left in the workspace; the row values
  // go to the space after them
  const BwdWs bw = bwd_ws_at(ws, L, T, k);
  const RowArgs ra{offsets, nullptr, L->S_routed, S, T, k, L->d, L->I, act_ld(L)};
  hipLaunchKernelGGL(k_utility_rows, dim3((unsigned)cdiv((long long)rows_total(L, T, k), UT_THREADS)),
                     dim3(UT_THREADS), 0, st, ra, perm_token, perm_gate, x_sq, dy_sq, (const float2*)bw.norms,
                     norm_parts(L), bw.vrow);
  hipLaunchKernelGGL(k_utility_slots, dim3((unsigned)S), dim3(US_THREADS), 0, st, ra, (const double*)bw.vrow,
                     utility);
  return check_launch("moe_expert_utility");
}
