// Layer-aware merging of the non-tuning experts (Section 5): the merging
// budget of each layer (Section 5.1, Eq. 1) and the similarity clustering that
// decides which experts share a group (Section 5.2): PCA features of the
// experts' parameters, then K-Means with cosine distance over every layer in
// one launch.
//
// PCA of n experts with D = 3 I d parameters each goes through the n x n Gram
// matrix of the parameter vectors (the scores are U sqrt(lambda) from the
// eigen-decomposition of the centred Gram matrix), so the only pass over the
// weights is the Gram product: an HBM-bound MFMA contraction over D, split
// into chunks of 32768 parameters, one block per (chunk, layer).  The
// per-layer eigen-decomposition (parallel cyclic Jacobi in fp64) and K-Means
// run in one block per layer; a centroid only ever meets experts of its own
// layer, which is the paper's masking of cross-layer distances.
#include "common.hpp"
#include "gemm_bf16.hpp"

namespace fm {
namespace {

constexpr int CL_NMAX = 64;        // experts per layer
constexpr int CL_RMAX = 32;        // feature dimension
constexpr int GR_ROWB = 512;       // bytes of one expert's parameters per slab
constexpr int GR_LDS = 144 * 1024; // LDS of the slab ring
constexpr long GR_KC = 32768;      // parameters per chunk
constexpr int CL_MAXL = 1024;      // layers of one budget call
constexpr int JAC_SWEEPS = 40;
constexpr int CL_TH = 1024;       // threads of the per-layer PCA / K-Means block
constexpr int CL_W = CL_TH / 64;

// ------------------------------------------------------------ Eq. 1 ------

__device__ __forceinline__ double wave_sum(double v) {
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) v += __shfl_xor(v, o);
  return v;
}
__device__ __forceinline__ int wave_sum(int v) {
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) v += __shfl_xor(v, o);
  return v;
}

// Wave-wide (value desc, index asc) maximum.
__device__ __forceinline__ void wave_argmax(double& v, int& idx) {
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) {
    const double ov = __shfl_xor(v, o);
    const int oi = __shfl_xor(idx, o);
    if (ov > v || (ov == v && oi < idx)) {
      v = ov;
      idx = oi;
    }
  }
}

// One block.  Wave w takes layers w, w + 4, ...: mean and variance of the
// frequencies by wave reductions.  Wave 0 then sums the weights and settles the
// integer budgets with wave-wide arg-max steps over the layers (lane i holds
// layers i, i + 64, ...).
__global__ __launch_bounds__(256) void k_merge_budget(const int32_t* __restrict__ counts,
                                                      const uint8_t* __restrict__ tuning, int L,
                                                      int E, double total, int B_non, double eps,
                                                      int32_t* __restrict__ budget) {
  __shared__ double sh[CL_MAXL];
  __shared__ int sB[CL_MAXL], sn[CL_MAXL];
  const int lane = lane_id(), wave = threadIdx.x >> 6;
  for (int l = wave; l < L; l += 4) {
    const int32_t* c = counts + (size_t)l * E;
    double s = 0.0;
    int n = 0;
    for (int e = lane; e < E; e += 64) {
      s += (double)c[e] / total;
      n += tuning[(size_t)l * E + e] == 0;
    }
    const double mean = wave_sum(s) / E;
    double v = 0.0;
    for (int e = lane; e < E; e += 64) {
      const double dl = (double)c[e] / total - mean;
      v += dl * dl;
    }
    v = wave_sum(v);
    n = wave_sum(n);
    if (lane == 0) {
      sh[l] = (double)(L - l) / fmax(v / E, eps);   // the paper's (L - l + 1) with l counted from 1
      sn[l] = n;
    }
  }
  __syncthreads();
  if (wave != 0) return;
  double part = 0.0;
  for (int l = lane; l < L; l += 64) part += sh[l];
  const double sum = wave_sum(part);
  long tot = 0;
  for (int l = lane; l < L; l += 64) {
    const double share = (double)B_non * sh[l] / sum;
    sh[l] = share;
    sB[l] = (int)fmin(fmax(floor(share), (double)min(1, sn[l])), (double)sn[l]);
    tot += sB[l];
  }
  for (int o = 32; o >= 1; o >>= 1) tot += __shfl_xor(tot, o);
  // Bulk of a shortfall.  Slot j of layer l beyond B_l has the value
  // share_l - (B_l + j); the settlement below takes slots in decreasing value,
  // so every slot whose value exceeds a threshold tau with at most `need` such
  // slots is taken for sure.  A bisection finds such a tau close to the
  // shortfall; the few slots left go through the settlement steps.
  if (tot < B_non) {
    const long need = (long)B_non - tot;
    auto above = [&](double tau, int l) -> int {      // #{j < room : share - (B + j) > tau}
      const int room = sn[l] - sB[l];
      if (room <= 0) return 0;
      const double x = sh[l] - sB[l] - tau;
      int j = x <= 0.0 ? 0 : (x >= room ? room : (int)ceil(x));
      while (j > 0 && !(sh[l] - (double)(sB[l] + j - 1) > tau)) --j;
      while (j < room && sh[l] - (double)(sB[l] + j) > tau) ++j;
      return j;
    };
    auto count = [&](double tau) {
      long c = 0;
      for (int l = lane; l < L; l += 64) c += above(tau, l);
      for (int o = 32; o >= 1; o >>= 1) c += __shfl_xor(c, o);
      return c;
    };
    double hi = -INFINITY, lo = INFINITY;            // the largest and smallest slot values
    for (int l = lane; l < L; l += 64)
      if (sB[l] < sn[l]) {
        hi = fmax(hi, sh[l] - sB[l]);
        lo = fmin(lo, sh[l] - (double)(sn[l] - 1));
      }
    for (int o = 32; o >= 1; o >>= 1) {
      hi = fmax(hi, __shfl_xor(hi, o));
      lo = fmin(lo, __shfl_xor(lo, o));
    }
    if (hi > -INFINITY) {
      lo -= 1.0;                                      // every slot lies above lo
      if (count(lo) <= need) {
        hi = lo;
      } else {
        for (int it = 0; it < 200; ++it) {           // count(hi) <= need < count(lo)
          const double mid = 0.5 * (lo + hi);
          if (!(mid > lo && mid < hi)) break;
          if (count(mid) <= need) hi = mid;
          else lo = mid;
        }
      }
      long got = 0;
      for (int l = lane; l < L; l += 64) {
        const int g = above(hi, l);
        sB[l] += g;
        got += g;
      }
      for (int o = 32; o >= 1; o >>= 1) got += __shfl_xor(got, o);
      tot += got;
    }
  }
  // The slots go one at a time to the layer with the largest share - B_l
  // that has room (ties: lower layer).  A layer that wins keeps winning until
  // its share - (B_l + j) falls below the best other layer's, so each step
  // hands it that whole run at once (the same result, in at most a few steps
  // per layer).
  while (tot < B_non) {
    double bv = -INFINITY, cv = -INFINITY;
    int bl = 1 << 30, cl = 1 << 30;
    for (int l = lane; l < L; l += 64)
      if (sB[l] < sn[l] && sh[l] - sB[l] > bv) {
        bv = sh[l] - sB[l];
        bl = l;
      }
    wave_argmax(bv, bl);
    if (bl >= L) break;
    for (int l = lane; l < L; l += 64)
      if (l != bl && sB[l] < sn[l] && sh[l] - sB[l] > cv) {
        cv = sh[l] - sB[l];
        cl = l;
      }
    wave_argmax(cv, cl);
    const int b0 = sB[bl];
    const long lim = min((long)(sn[bl] - b0), (long)B_non - tot);
    auto wins = [&](long j) {
      const double dj = sh[bl] - (double)(b0 + j);
      return dj > cv || (dj == cv && bl < cl);
    };
    long j = 0;                      // wins(0) holds; find the last winning j
    if (cl >= L) {
      j = lim - 1;
    } else {
      j = (long)fmax(0.0, fmin((double)(lim - 1), floor(bv - cv)));
      while (j + 1 < lim && wins(j + 1)) ++j;
      while (j > 0 && !wins(j)) --j;
    }
    if (lane == 0) sB[bl] = b0 + (int)(j + 1);
    tot += j + 1;
  }
  // Bulk of an excess, the same way: the j-th slot taken back from layer l has
  // the key share_l - (B_l - j), keys are taken in increasing order, and every
  // key below a threshold with at most `need` such keys goes for sure.
  if (tot > B_non) {
    const long need = tot - (long)B_non;
    auto below = [&](double tau, int l) -> int {      // #{j < cap : share - (B - j) < tau}
      const int cap = sB[l] - min(1, sn[l]);
      if (cap <= 0) return 0;
      const double x = tau - (sh[l] - sB[l]);
      int j = x <= 0.0 ? 0 : (x >= cap ? cap : (int)ceil(x));
      while (j > 0 && !(sh[l] - (double)(sB[l] - (j - 1)) < tau)) --j;
      while (j < cap && sh[l] - (double)(sB[l] - j) < tau) ++j;
      return j;
    };
    auto count = [&](double tau) {
      long c = 0;
      for (int l = lane; l < L; l += 64) c += below(tau, l);
      for (int o = 32; o >= 1; o >>= 1) c += __shfl_xor(c, o);
      return c;
    };
    double lo = INFINITY, hi = -INFINITY;            // the smallest and largest keys
    for (int l = lane; l < L; l += 64)
      if (sB[l] > min(1, sn[l])) {
        lo = fmin(lo, sh[l] - sB[l]);
        hi = fmax(hi, sh[l] - (double)(min(1, sn[l]) + 1));
      }
    for (int o = 32; o >= 1; o >>= 1) {
      hi = fmax(hi, __shfl_xor(hi, o));
      lo = fmin(lo, __shfl_xor(lo, o));
    }
    if (lo < INFINITY) {
      hi += 1.0;                                      // every key lies below hi
      if (count(hi) <= need) {
        lo = hi;
      } else {
        for (int it = 0; it < 200; ++it) {           // count(lo) <= need < count(hi)
          const double mid = 0.5 * (lo + hi);
          if (!(mid > lo && mid < hi)) break;
          if (count(mid) <= need) lo = mid;
          else hi = mid;
        }
      }
      long got = 0;
      for (int l = lane; l < L; l += 64) {
        const int g = below(lo, l);
        sB[l] -= g;
        got += g;
      }
      for (int o = 32; o >= 1; o >>= 1) got += __shfl_xor(got, o);
      tot -= got;
    }
  }
  // Over the total: slots are taken back one at a time from the layer with
  // the smallest share - B_l above its floor (ties: higher layer), in runs
  // the same way.  Values are negated so that the arg-max picks them.
  while (tot > B_non) {
    double bv = -INFINITY, cv = -INFINITY;
    int bl = 1 << 30, cl = 1 << 30;
    for (int l = lane; l < L; l += 64)
      if (sB[l] > min(1, sn[l]) && -(sh[l] - sB[l]) >= bv) {
        bv = -(sh[l] - sB[l]);
        bl = -l;
      }
    wave_argmax(bv, bl);
    if (bl > 0) break;
    const int lb = -bl;
    for (int l = lane; l < L; l += 64)
      if (l != lb && sB[l] > min(1, sn[l]) && -(sh[l] - sB[l]) >= cv) {
        cv = -(sh[l] - sB[l]);
        cl = -l;
      }
    wave_argmax(cv, cl);
    const int b0 = sB[lb];
    const long lim = min((long)(b0 - min(1, sn[lb])), tot - (long)B_non);
    auto wins = [&](long j) {
      const double nj = -(sh[lb] - (double)(b0 - j));
      return nj > cv || (nj == cv && bl < cl);
    };
    long j = 0;
    if (cl > 0) {
      j = lim - 1;
    } else {
      j = (long)fmax(0.0, fmin((double)(lim - 1), floor(bv - cv)));
      while (j + 1 < lim && wins(j + 1)) ++j;
      while (j > 0 && !wins(j)) --j;
    }
    if (lane == 0) sB[lb] = b0 - (int)(j + 1);
    tot -= j + 1;
  }
  for (int l = lane; l < L; l += 64) budget[l] = sB[l];
}

// -------------------------------------------------------- Gram product ----

// Wave 0 lists the layer's non-tuning experts in index order (E <= 64).
__device__ __forceinline__ int list_members(const uint8_t* tuning, int l, int E, int* mem) {
  __shared__ int s_n;
  if (threadIdx.x < 64) {
    const int e = threadIdx.x;
    const bool non = e < E && tuning[(size_t)l * E + e] == 0;
    const uint64_t m = __ballot(non);
    if (non) mem[__popcll(m & ((1ull << e) - 1ull))] = e;
    if (e == 0) s_n = __popcll(m);
  }
  __syncthreads();
  return s_n;
}

struct GramArgs {
  const void* const* w_src;   // [3 * L * E]: (gate, up, down) of expert (l, e)
  const uint8_t* tuning;      // [L * E]
  float* part;                // [L][nchunk][NT][32][32]
  long P;                     // parameters per matrix, I * d
  int E, cpm;                 // experts per layer, chunks per matrix
};

// Slab layout in LDS: [row group g (16 rows)][128-byte line m][64-byte half h]
// blocks of [16 rows][4 chunks of 16 bytes], one DMA instruction each, the
// chunk index XOR-swizzled by (row >> 2) & 3.  Wave w reads line w of every
// row (its four 16-parameter k-steps), so the waves split each slab's k range.
template <typename T> struct GramFrag;
template <> struct GramFrag<bf16> {
  typedef bf16x8_t frag;
  static __device__ __forceinline__ frag load(const FM_LDS char* p) { return *(const FM_LDS bf16x8_t*)p; }
  static __device__ __forceinline__ frag zero() { return frag{}; }
  static __device__ __forceinline__ f32x16_t mma(const frag& a, const frag& b, const f32x16_t& c) {
    return __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, c, 0, 0, 0);
  }
};
template <> struct GramFrag<float> {
  typedef f32x4_t frag;
  static __device__ __forceinline__ frag load(const FM_LDS char* p) { return *(const FM_LDS f32x4_t*)p; }
  static __device__ __forceinline__ frag zero() { return frag{0.f, 0.f, 0.f, 0.f}; }
  static __device__ __forceinline__ f32x16_t mma(const frag& a, const frag& b, f32x16_t c) {
#pragma unroll
    for (int e = 0; e < 4; ++e) c = __builtin_amdgcn_mfma_f32_32x32x2f32(a[e], b[e], c, 0, 0, 0);
    return c;
  }
};

// Waits for this wave's DMA of the slab being consumed, leaving the `ahead`
// later slabs' INS instructions each in flight (A = the most there can be).
template <int INS, int A> __device__ __forceinline__ void gram_wait(int ahead) {
  if constexpr (A == 0) {
    wait_vmcnt<0>();
  } else {
    if (ahead >= A) wait_vmcnt<A * INS>();
    else gram_wait<INS, A - 1>(ahead);
  }
}

// The slab ring of NG row groups: as many slabs as fit in GR_LDS (at most 16),
// so that fewer rows mean more slabs in flight.
template <int NG> struct GramRing {
  static constexpr int SLAB = NG * 16 * GR_ROWB;
  static constexpr int NS = GR_LDS / SLAB < 16 ? GR_LDS / SLAB : 16;
  static_assert(NS >= 3, "ring depth");
};

// NG groups of 16 rows hold the n experts (rows past n repeat row n - 1).
template <typename T, int NB, int NG>
__device__ __forceinline__ void gram_chunk(const GramArgs& a, const int* mem, int n, int l, int mat,
                                           long k0, long klen, FM_LDS char* lds, f32x16_t* acc) {
  constexpr int SLAB = GramRing<NG>::SLAB, NS = GramRing<NG>::NS;
  constexpr int EPS = GR_ROWB / (int)sizeof(T);       // parameters per row and slab
  constexpr int EPC = 16 / (int)sizeof(T);            // parameters per 16-byte chunk
  constexpr int INS = 2 * NG;                         // DMA instructions per wave and slab
  constexpr int NT = NB * (NB + 1) / 2;
  static_assert(NG >= 1 && NG <= 2 * NB, "row groups");
  typedef GramFrag<T> F;
  const int lane = lane_id_here(), wave = wave_id();
  const int nslab = (int)((klen + EPS - 1) / EPS);
  const int tail_chunks = (int)((klen - (long)(nslab - 1) * EPS) / EPC);

  // DMA plan: instruction u = wave * INS + q moves line m, half h of group g.
  const char* gp[INS];
  int cix[INS];
  uint32_t dst[INS];
#pragma unroll
  for (int q = 0; q < INS; ++q) {
    const int u = wave * INS + q, g = u >> 3, m = (u >> 1) & 3, h = u & 1;
    const int rr = lane >> 2, row = g * 16 + rr;
    const int chunk = m * 8 + h * 4 + ((lane & 3) ^ ((rr >> 2) & 3));
    const int e = mem[min(row, n - 1)];
    const char* base = (const char*)a.w_src[3 * ((size_t)l * a.E + e) + mat];
    gp[q] = base + (k0 * (long)sizeof(T)) + chunk * 16;
    cix[q] = chunk;
    dst[q] = (uint32_t)(((g * 4 + m) * 2 + h) * 1024);
  }
  auto issue = [&](int s) {
    FM_LDS char* slab = lds + (s % NS) * SLAB;
    const bool last = s == nslab - 1;
#pragma unroll
    for (int q = 0; q < INS; ++q) {
      const char* src = gp[q] + (long)s * GR_ROWB;
      if (last && cix[q] >= tail_chunks) src -= cix[q] * 16;   // any valid address: masked below
      dma16(src, slab + dst[q]);
    }
  };

  const int pre = min(NS - 1, nslab);
  for (int s = 0; s < pre; ++s) issue(s);

  // fragment addresses: lane (i, hf) reads row 32 b + i, k-steps j = 0..3 of line `wave`
  const int i = lane & 31, hf = lane >> 5;
  for (int s = 0; s < nslab; ++s) {
    gram_wait<INS, NS - 2>(min(NS - 2, nslab - 1 - s));
    barrier_lds();
    if (s + NS - 1 < nslab) issue(s + NS - 1);
    const FM_LDS char* slab = lds + (s % NS) * SLAB;
    const bool last = s == nslab - 1;
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const int cc = 2 * j + hf, h = cc >> 2, q = cc & 3;
      typename F::frag fr[NB];
#pragma unroll
      for (int b = 0; b < NB; ++b) {
        // rows past the NG loaded groups feed only outputs that are not used:
        // they read the last group
        const int R = 32 * b + i, g = min(R >> 4, NG - 1), rr = R & 15;
        fr[b] = F::load(slab + ((g * 4 + wave) * 2 + h) * 1024 + rr * 64 + ((q ^ ((rr >> 2) & 3)) << 4));
      }
      if (last && wave * 8 + cc >= tail_chunks) {
#pragma unroll
        for (int b = 0; b < NB; ++b) fr[b] = F::zero();
      }
      int t = 0;
#pragma unroll
      for (int b1 = 0; b1 < NB; ++b1)
#pragma unroll
        for (int b2 = b1; b2 < NB; ++b2) acc[t] = F::mma(fr[b1], fr[b2], acc[t]), ++t;
    }
  }
  (void)NT;
}

// Partial Gram matrix of one chunk of one matrix (gate, up or down) of the
// layer's non-tuning experts: tiles (b1 <= b2) of 32 x 32, the four waves'
// k-subranges summed in wave order.  Register r of a tile's lane L holds
// G[32 b1 + 8 (r / 4) + 4 (L / 32) + r % 4][32 b2 + L % 32].
template <typename T, int NB>
__global__ __launch_bounds__(256) void k_gram(GramArgs a) {
  constexpr int NT = NB * (NB + 1) / 2;
  __shared__ __align__(1024) char lds_raw[GR_LDS];
  __shared__ int mem[CL_NMAX];
  FM_LDS char* lds = (FM_LDS char*)lds_raw;
  const int l = blockIdx.y, c = blockIdx.x, nchunk = gridDim.x;
  const int n = list_members(a.tuning, l, a.E, mem);
  const int mat = c / a.cpm;
  const long k0 = (long)(c % a.cpm) * GR_KC;
  const long klen = a.P - k0 < GR_KC ? a.P - k0 : GR_KC;

  f32x16_t acc[NT];
#pragma unroll
  for (int t = 0; t < NT; ++t)
#pragma unroll
    for (int r = 0; r < 16; ++r) acc[t][r] = 0.f;
  const int ng = (n + 15) >> 4;
  if (ng == 1) gram_chunk<T, NB, 1>(a, mem, n, l, mat, k0, klen, lds, acc);
  else if (ng == 2) gram_chunk<T, NB, 2>(a, mem, n, l, mat, k0, klen, lds, acc);
  if constexpr (NB == 2) {
    if (ng == 3) gram_chunk<T, NB, 3>(a, mem, n, l, mat, k0, klen, lds, acc);
    else if (ng == 4) gram_chunk<T, NB, 4>(a, mem, n, l, mat, k0, klen, lds, acc);
  }
  __syncthreads();

  // sum the four waves' accumulators in wave order
  float* red = (float*)lds_raw;                        // [wave][t][r][lane]
  const int lane = lane_id(), wave = wave_id();
#pragma unroll
  for (int t = 0; t < NT; ++t)
#pragma unroll
    for (int r = 0; r < 16; ++r) red[((wave * NT + t) * 16 + r) * 64 + lane] = acc[t][r];
  __syncthreads();
  float* out = a.part + ((size_t)l * nchunk + c) * NT * 1024;
  for (int x = threadIdx.x; x < NT * 1024; x += blockDim.x) {
    const int t = x >> 10, r = (x >> 6) & 15, L = x & 63;
    float s = 0.f;
#pragma unroll
    for (int w = 0; w < 4; ++w) s += red[((w * NT + t) * 16 + r) * 64 + L];
    const int p = 8 * (r >> 2) + 4 * (L >> 5) + (r & 3), q = L & 31;
    out[t * 1024 + p * 32 + q] = s;
  }
}

// G[l][t][p][q] = sum over chunks (in chunk order, fp64) of the partials.
__global__ __launch_bounds__(256) void k_gram_sum(const float* __restrict__ part, int nchunk, int NT,
                                                  double* __restrict__ G) {
  const int l = blockIdx.y, x = blockIdx.x * blockDim.x + threadIdx.x;
  if (x >= NT * 1024) return;
  const float* p = part + (size_t)l * nchunk * NT * 1024 + x;
  const size_t st = (size_t)NT * 1024;
  double s = 0.0;
  int c = 0;
  for (; c + 16 <= nchunk; c += 16) {      // loads batched, sums kept in chunk order
    float v[16];
#pragma unroll
    for (int u = 0; u < 16; ++u) v[u] = p[(size_t)(c + u) * st];
#pragma unroll
    for (int u = 0; u < 16; ++u) s += (double)v[u];
  }
  for (; c < nchunk; ++c) s += (double)p[(size_t)c * st];
  G[(size_t)l * NT * 1024 + x] = s;
}

// ------------------------------------------- PCA and K-Means per layer ----

constexpr int LDA = CL_NMAX + 1;
constexpr int LDZ = CL_RMAX + 1;

struct ClusterLds {
  double A[CL_NMAX * LDA];      // centred Gram matrix, rotated to diagonal
  double V[CL_NMAX * LDA];      // eigenvectors (columns)
  double Z[CL_NMAX * LDZ];      // unit features
  double C[CL_NMAX * LDZ];      // centroids
  double rc[CL_NMAX / 2], rs[CL_NMAX / 2];
  int rp[CL_NMAX / 2], rq[CL_NMAX / 2];
  uint16_t tri[CL_NMAX / 2 * (CL_NMAX / 2 + 1) / 2];   // pair blocks k1 <= k2
  uint16_t pairs[(CL_NMAX - 1) * (CL_NMAX / 2)];        // round-robin (p << 8 | q) per round
  double rho[CL_NMAX], nrm2[CL_NMAX], mind[CL_NMAX], cn[CL_NMAX];
  double red[2][CL_TH];
  double bsim[CL_W][CL_NMAX];
  int bj[CL_W][CL_NMAX];
  int mem[CL_NMAX], comp[CL_RMAX], lab[CL_NMAX], chosen[CL_NMAX];
  int flag;
};

// 1 / sqrt(x) for x > 0: the hardware estimate refined by two Newton steps.
__device__ __forceinline__ double rsqrt_f64(double x) {
  double y = __builtin_amdgcn_rsq(x);
  const double hx = 0.5 * x;
  y = y * (1.5 - hx * y * y);
  y = y * (1.5 - hx * y * y);
  return y;
}

// Round-robin pairing of m indices (m even): m / 2 disjoint pairs per round,
// every pair once over m - 1 rounds.
__device__ __forceinline__ void rr_pair(int round, int k, int m, int& p, int& q) {
  int x, y;
  if (k == 0) {
    x = m - 1;
    y = round;
  } else {
    x = (round + k) % (m - 1);
    y = (round - k + (m - 1)) % (m - 1);
  }
  p = min(x, y);
  q = max(x, y);
}

struct ClusterArgs {
  const double* G;            // [L][NT][32][32]
  const uint8_t* tuning;
  const int32_t* budget;
  int32_t* labels;            // [L * E]
  float* features;            // [L * E * r] or nullptr
  int32_t* iters;             // [L] or nullptr
  int E, NB, r, max_iter;
};

__global__ __launch_bounds__(CL_TH) void k_cluster(ClusterArgs a) {
  __shared__ ClusterLds S;
  const int l = blockIdx.x, tid = threadIdx.x, lane = lane_id(), wave = wave_id();
  const int E = a.E, r = a.r;
  const int n = list_members(a.tuning, l, E, S.mem);
  const int NT = a.NB * (a.NB + 1) / 2;

  // outputs of tuning experts
  for (int e = tid; e < E; e += blockDim.x) {
    if (a.tuning[(size_t)l * E + e] != 0) {
      a.labels[(size_t)l * E + e] = -1;
      if (a.features)
        for (int j = 0; j < r; ++j) a.features[((size_t)l * E + e) * r + j] = 0.f;
    }
  }
  if (n == 0) {
    if (a.iters && tid == 0) a.iters[l] = 0;
    return;
  }
  const int B = min(max(a.budget[l], 1), n);
  const int m = n + (n & 1);

  // 1. Gram matrix (symmetrised), centred on the experts' mean.
  const double* G = a.G + (size_t)l * NT * 1024;
  auto g_at = [&](int i, int j) {
    const int b1 = i >> 5, b2 = j >> 5;
    const int t = b1 * a.NB - b1 * (b1 - 1) / 2 + (b2 - b1);
    return G[t * 1024 + (i & 31) * 32 + (j & 31)];
  };
  for (int x = tid; x < m * m; x += blockDim.x) {
    const int i = x / m, j = x % m;
    double v = 0.0;
    if (i < n && j < n) {
      if ((i >> 5) < (j >> 5)) v = g_at(i, j);
      else if ((i >> 5) > (j >> 5)) v = g_at(j, i);
      else v = 0.5 * (g_at(i, j) + g_at(j, i));
    }
    S.A[i * LDA + j] = v;
    S.V[i * LDA + j] = i == j ? 1.0 : 0.0;
  }
  __syncthreads();
  if (tid < n) {
    double s = 0.0;
#pragma unroll 8
    for (int j = 0; j < n; ++j) s += S.A[tid * LDA + j];
    S.rho[tid] = s / n;
  }
  __syncthreads();
  {
    double mu = 0.0;
    for (int i = 0; i < n; ++i) mu += S.rho[i];
    mu /= n;
    for (int x = tid; x < n * n; x += blockDim.x) {
      const int i = x / n, j = x % n;
      S.A[i * LDA + j] = S.A[i * LDA + j] - S.rho[i] - S.rho[j] + mu;
    }
  }
  __syncthreads();

  // 2. Eigen-decomposition: parallel cyclic Jacobi, A <- J^T A J, V <- V J.
  // J rotates the m / 2 disjoint pairs of a round at once, so every 2 x 2
  // block (pair k1 rows, pair k2 columns) of A and every (row, pair) of V is
  // updated from its own old values: one update phase per round.
  const int h = m / 2, ntri = h * (h + 1) / 2;
  if (tid == 0) {
    int x = 0;
    for (int k1 = 0; k1 < h; ++k1)
      for (int k2 = k1; k2 < h; ++k2) S.tri[x++] = (uint16_t)(k1 << 8 | k2);
  }
  for (int x = tid; x < (m - 1) * h; x += blockDim.x) {
    int p, q;
    rr_pair(x / h, x % h, m, p, q);
    S.pairs[x] = (uint16_t)(p << 8 | q);
  }
  __syncthreads();
  for (int sweep = 0; sweep < JAC_SWEEPS; ++sweep) {
    double off = 0.0, tot = 0.0;
    for (int x = tid; x < CL_NMAX * CL_NMAX; x += blockDim.x) {
      const int i = x >> 6, j = x & 63;
      if (i < m && j < m) {
        const double v = S.A[i * LDA + j] * S.A[i * LDA + j];
        tot += v;
        if (i != j) off += v;
      }
    }
    S.red[0][tid] = off;
    S.red[1][tid] = tot;
    __syncthreads();
    for (int hh = CL_TH / 2; hh > 0; hh >>= 1) {
      if (tid < hh) {
        S.red[0][tid] += S.red[0][tid + hh];
        S.red[1][tid] += S.red[1][tid + hh];
      }
      __syncthreads();
    }
    const bool done = S.red[0][0] <= 1e-18 * S.red[1][0];
    __syncthreads();
    if (done) break;
    for (int round = 0; round < m - 1; ++round) {
      if (tid < h) {
        const int pq = S.pairs[round * h + tid], p = pq >> 8, q = pq & 255;
        const double apq = S.A[p * LDA + q];
        double c = 1.0, s = 0.0;
        if (apq != 0.0) {
          // tan of the angle t = sgn(tau) / (|tau| + sqrt(1 + tau^2)), tau =
          // dd / e2, written without divisions: with hyp = sqrt(dd^2 + e2^2)
          // and w = |dd| + hyp, c = w / sqrt(2 hyp w), s = sgn(tau) |e2| / sqrt(2 hyp w).
          double dd = S.A[q * LDA + q] - S.A[p * LDA + p], e2 = 2.0 * apq;
          const double sg = (dd == 0.0 || (dd > 0.0) == (e2 > 0.0)) ? 1.0 : -1.0;
          const double mx = fmax(fabs(dd), fabs(e2));
          if (mx > 1e100 || mx < 1e-100) {   // c and s depend on the ratio only
            dd /= mx;
            e2 /= mx;
          }
          const double hyp = sqrt(dd * dd + e2 * e2);
          const double w = fabs(dd) + hyp;
          const double r = rsqrt_f64(2.0 * hyp * w);
          c = w * r;
          s = sg * fabs(e2) * r;
        }
        S.rc[tid] = c;
        S.rs[tid] = s;
        S.rp[tid] = p;
        S.rq[tid] = q;
      }
      __syncthreads();
      // A is symmetric: blocks k1 <= k2 are computed and stored with their
      // mirror.  Every item's loads are issued before any store, so that the
      // stores (which may alias in the compiler's view) do not serialise them.
      constexpr int NTRI = (CL_NMAX / 2 * (CL_NMAX / 2 + 1) / 2 + CL_TH - 1) / CL_TH;
      {
        double va[NTRI][4];
        int ip[NTRI][4];
        double rot[NTRI][4];
#pragma unroll
        for (int u = 0; u < NTRI; ++u) {
          const int x = min(tid + CL_TH * u, ntri - 1);
          const int k1 = S.tri[x] >> 8, k2 = S.tri[x] & 255;
          ip[u][0] = S.rp[k1]; ip[u][1] = S.rq[k1]; ip[u][2] = S.rp[k2]; ip[u][3] = S.rq[k2];
          rot[u][0] = S.rc[k1]; rot[u][1] = S.rs[k1]; rot[u][2] = S.rc[k2]; rot[u][3] = S.rs[k2];
          va[u][0] = S.A[ip[u][0] * LDA + ip[u][2]];
          va[u][1] = S.A[ip[u][0] * LDA + ip[u][3]];
          va[u][2] = S.A[ip[u][1] * LDA + ip[u][2]];
          va[u][3] = S.A[ip[u][1] * LDA + ip[u][3]];
        }
        // V: thread owns pair k = tid % 32 and rows tid / 32 + (CL_TH / 32) j
        const int k = tid & 31;
        const bool kv = k < h;
        const int kk = kv ? k : 0;
        const int vp_ = S.rp[kk], vq_ = S.rq[kk];
        const double vc = S.rc[kk], vs = S.rs[kk];
        constexpr int VR = (CL_NMAX + CL_TH / 32 - 1) / (CL_TH / 32);
        double vv[VR][2];
#pragma unroll
        for (int j = 0; j < VR; ++j) {
          const int i = min((tid >> 5) + (CL_TH / 32) * j, m - 1);
          vv[j][0] = S.V[i * LDA + vp_];
          vv[j][1] = S.V[i * LDA + vq_];
        }
#pragma unroll
        for (int u = 0; u < NTRI; ++u) {
          if (tid + CL_TH * u < ntri) {
            const double c1 = rot[u][0], s1 = rot[u][1], c2 = rot[u][2], s2 = rot[u][3];
            const double a = va[u][0], b = va[u][1], c = va[u][2], d = va[u][3];
            const double ra = c1 * a - s1 * c, rb = c1 * b - s1 * d;     // rows (pair k1)
            const double rc = s1 * a + c1 * c, rd = s1 * b + c1 * d;
            const double na = c2 * ra - s2 * rb, nb = s2 * ra + c2 * rb;  // columns (pair k2)
            const double nc = c2 * rc - s2 * rd, nd = s2 * rc + c2 * rd;
            const int p1 = ip[u][0], q1 = ip[u][1], p2 = ip[u][2], q2 = ip[u][3];
            S.A[p1 * LDA + p2] = na;
            S.A[p1 * LDA + q2] = nb;
            S.A[q1 * LDA + p2] = nc;
            S.A[q1 * LDA + q2] = nd;
            if (p1 != p2) {
              S.A[p2 * LDA + p1] = na;
              S.A[q2 * LDA + p1] = nb;
              S.A[p2 * LDA + q1] = nc;
              S.A[q2 * LDA + q1] = nd;
            }
          }
        }
        if (kv) {
#pragma unroll
          for (int j = 0; j < VR; ++j) {
            const int i = (tid >> 5) + (CL_TH / 32) * j;
            if (i < m) {
              S.V[i * LDA + vp_] = vc * vv[j][0] - vs * vv[j][1];
              S.V[i * LDA + vq_] = vs * vv[j][0] + vc * vv[j][1];
            }
          }
        }
      }
      __syncthreads();
    }
  }

  // 3. Features: scores on the r leading components (eigenvalue desc, ties
  // lower index), then scaled to unit length.
  if (tid < r) S.comp[tid] = -1;
  __syncthreads();
  if (tid < n) {
    const double li = S.A[tid * LDA + tid];
    int rank = 0;
#pragma unroll 8
    for (int q = 0; q < n; ++q) {
      const double lq = S.A[q * LDA + q];
      rank += (lq > li) || (lq == li && q < tid);
    }
    if (rank < r) S.comp[rank] = tid;
  }
  __syncthreads();
  for (int x = tid; x < n * r; x += blockDim.x) {
    const int e = x / r, j = x % r, p = S.comp[j];
    S.Z[e * LDZ + j] = p < 0 ? 0.0 : sqrt(fmax(S.A[p * LDA + p], 0.0)) * S.V[e * LDA + p];
  }
  __syncthreads();
  if (tid < n) {
    double s = 0.0;
#pragma unroll 8
    for (int j = 0; j < r; ++j) s += S.Z[tid * LDZ + j] * S.Z[tid * LDZ + j];
    S.nrm2[tid] = s;
  }
  __syncthreads();
  for (int x = tid; x < n * r; x += blockDim.x) {
    const int e = x / r, j = x % r;
    const double nr = sqrt(S.nrm2[e]);
    S.Z[e * LDZ + j] = nr > 0.0 ? S.Z[e * LDZ + j] / nr : 0.0;
  }
  __syncthreads();
  if (a.features)
    for (int x = tid; x < n * r; x += blockDim.x) {
      const int i = x / r, j = x % r;
      a.features[((size_t)l * E + S.mem[i]) * r + j] = (float)S.Z[i * LDZ + j];
    }

  // 4. Seeds: farthest-first traversal under 1 - cos, from the largest score.
  if (wave == 0) {
    const int e = lane;
    double v = e < n ? S.nrm2[e] : -1.0;
    int idx = e < n ? e : 1 << 30;
    wave_argmax(v, idx);
    int seed = idx;
    bool mine_chosen = e == seed;
    auto dist = [&](int s) {
      double d = 0.0;
#pragma unroll 8
      for (int j = 0; j < r; ++j) d += S.Z[e * LDZ + j] * S.Z[s * LDZ + j];
      return 1.0 - d;
    };
    double md = e < n ? dist(seed) : 0.0;
    if (e < r) S.C[0 * LDZ + e] = S.Z[seed * LDZ + e];
    for (int c = 1; c < B; ++c) {
      double cv = (e < n && !mine_chosen) ? md : -1.0;
      int ci = (e < n && !mine_chosen) ? e : 1 << 30;
      wave_argmax(cv, ci);
      seed = ci;
      mine_chosen = mine_chosen || e == seed;
      if (e < n) md = fmin(md, dist(seed));
      if (e < r) S.C[c * LDZ + e] = S.Z[seed * LDZ + e];
    }
  }
  __syncthreads();
  if (tid < B) {
    double s = 0.0;
#pragma unroll 8
    for (int j = 0; j < r; ++j) s += S.C[tid * LDZ + j] * S.C[tid * LDZ + j];
    S.cn[tid] = sqrt(s);
  }
  if (tid < n) S.lab[tid] = -1;
  __syncthreads();

  // 5. Lloyd passes: thread (e, w) scans centroids w, w + CL_W, ...
  int pass = 0;
  for (;;) {
    ++pass;
    {
      const int e = tid & 63, w = tid >> 6;
      double bs = -INFINITY;
      int bj = 1 << 30;
      if (e < n)
        for (int c = w; c < B; c += CL_W) {
          double d = 0.0;
#pragma unroll 8
          for (int j = 0; j < r; ++j) d += S.Z[e * LDZ + j] * S.C[c * LDZ + j];
          const double sim = S.cn[c] > 0.0 ? d / S.cn[c] : 0.0;
          if (sim > bs) {        // c increases: ties keep the lower centroid
            bs = sim;
            bj = c;
          }
        }
      S.bsim[w][e] = bs;
      S.bj[w][e] = bj;
    }
    if (tid == 0) S.flag = 0;
    __syncthreads();
    if (tid < n) {
      double bs = S.bsim[0][tid];
      int bj = S.bj[0][tid];
      for (int w = 1; w < CL_W; ++w) {
        const double v = S.bsim[w][tid];
        const int j = S.bj[w][tid];
        if (v > bs || (v == bs && j < bj)) {
          bs = v;
          bj = j;
        }
      }
      if (S.lab[tid] != bj) S.flag = 1;
      S.lab[tid] = bj;
    }
    __syncthreads();
    const bool changed = S.flag != 0;
    if ((pass > 1 && !changed) || pass >= a.max_iter) break;
    for (int x = tid; x < B * r; x += blockDim.x) {
      const int c = x / r, j = x % r;
      double s = 0.0;
      int cnt = 0;
#pragma unroll 8
      for (int e = 0; e < n; ++e)
        if (S.lab[e] == c) {
          s += S.Z[e * LDZ + j];
          ++cnt;
        }
      if (cnt) S.C[c * LDZ + j] = s / cnt;
    }
    __syncthreads();
    if (tid < B) {
      double s = 0.0;
#pragma unroll 8
      for (int j = 0; j < r; ++j) s += S.C[tid * LDZ + j] * S.C[tid * LDZ + j];
      S.cn[tid] = sqrt(s);
    }
    __syncthreads();
  }
  if (tid < n) a.labels[(size_t)l * E + S.mem[tid]] = S.lab[tid];
  if (a.iters && tid == 0) a.iters[l] = pass;
}

size_t round256(size_t x) { return (x + 255) & ~(size_t)255; }

struct ClusterSizes {
  int NB, NT, cpm, nchunk;
  size_t g_bytes, part_bytes;
};

ClusterSizes cluster_sizes(int L, int E, int d, int I) {
  ClusterSizes z;
  z.NB = E <= 32 ? 1 : 2;
  z.NT = z.NB * (z.NB + 1) / 2;
  const long P = (long)I * d;
  z.cpm = (int)((P + GR_KC - 1) / GR_KC);
  z.nchunk = 3 * z.cpm;
  z.g_bytes = round256((size_t)L * z.NT * 1024 * sizeof(double));
  z.part_bytes = round256((size_t)L * z.nchunk * z.NT * 1024 * sizeof(float));
  return z;
}

}  // namespace
}  // namespace fm

using namespace fm;

extern "C" int moe_merge_budget(const int32_t* counts, const uint8_t* tuning, int L, int E,
                                float total_tokens, int B_non, double eps, int32_t* budget,
                                void* stream) {
  clear_error();
  FM_TRY(need(counts, "counts"));
  FM_TRY(need(tuning, "tuning"));
  FM_TRY(need(budget, "budget"));
  if (L < 1 || L > CL_MAXL) return fail(MOE_ERR_UNSUPPORTED, "L=%d: 1..%d layers", L, CL_MAXL);
  if (E < 1) return fail(MOE_ERR_ARG, "E=%d", E);
  if (!(total_tokens > 0.f)) return fail(MOE_ERR_ARG, "total_tokens must be positive");
  if (B_non < 0) return fail(MOE_ERR_ARG, "B_non=%d", B_non);
  if (!(eps > 0.0)) return fail(MOE_ERR_ARG, "eps must be positive");
  hipLaunchKernelGGL(k_merge_budget, dim3(1), dim3(256), 0, as_stream(stream), counts, tuning, L, E,
                     (double)total_tokens, B_non, eps, budget);
  return check_launch("moe_merge_budget");
}

extern "C" size_t moe_cluster_workspace_size(int L, int E, int d, int I) {
  if (L < 1 || E < 1 || E > CL_NMAX || d < 1 || I < 1) return 0;
  const ClusterSizes z = cluster_sizes(L, E, d, I);
  return z.g_bytes + z.part_bytes;
}

extern "C" int moe_cluster_experts(const void* const* w_src, int dtype, int L, int E, int d, int I,
                                   const uint8_t* tuning, const int32_t* budget, int r,
                                   int max_iter, void* ws, size_t ws_bytes, int32_t* labels,
                                   float* features, int32_t* iters, void* stream) {
  clear_error();
  FM_TRY(need(w_src, "w_src"));
  FM_TRY(need(tuning, "tuning"));
  FM_TRY(need(budget, "budget"));
  FM_TRY(need(labels, "labels"));
  FM_TRY(need_dtype_float(dtype, "dtype"));
  if (!ws) return fail(MOE_ERR_WORKSPACE, "workspace is NULL");
  FM_TRY(need_aligned(ws, "ws"));
  if (L < 1 || L > 65535) return fail(MOE_ERR_UNSUPPORTED, "L=%d: 1..65535 layers", L);
  if (E < 1 || E > CL_NMAX) return fail(MOE_ERR_UNSUPPORTED, "E=%d: at most %d experts per layer", E, CL_NMAX);
  if (d < 1 || I < 1) return fail(MOE_ERR_ARG, "d=%d I=%d", d, I);
  if (((size_t)I * d * esize(dtype)) % 16 != 0)
    return fail(MOE_ERR_UNSUPPORTED, "I*d*element size must be a multiple of 16 bytes");
  if (r < 1 || r > CL_RMAX) return fail(MOE_ERR_UNSUPPORTED, "r=%d: 1..%d components", r, CL_RMAX);
  if (max_iter < 1) return fail(MOE_ERR_ARG, "max_iter=%d", max_iter);
  const ClusterSizes z = cluster_sizes(L, E, d, I);
  if (ws_bytes < z.g_bytes + z.part_bytes)
    return fail(MOE_ERR_WORKSPACE, "workspace of %zu bytes < %zu", ws_bytes, z.g_bytes + z.part_bytes);
  hipStream_t st = as_stream(stream);
  double* G = (double*)ws;
  float* part = (float*)((char*)ws + z.g_bytes);
  GramArgs ga{w_src, tuning, part, (long)I * d, E, z.cpm};
  const dim3 grid(z.nchunk, L);
  if (dtype == MOE_BF16) {
    if (z.NB == 1) hipLaunchKernelGGL((k_gram<bf16, 1>), grid, dim3(256), 0, st, ga);
    else hipLaunchKernelGGL((k_gram<bf16, 2>), grid, dim3(256), 0, st, ga);
  } else {
    if (z.NB == 1) hipLaunchKernelGGL((k_gram<float, 1>), grid, dim3(256), 0, st, ga);
    else hipLaunchKernelGGL((k_gram<float, 2>), grid, dim3(256), 0, st, ga);
  }
  FM_TRY(check_launch("moe_cluster_experts (Gram)"));
  hipLaunchKernelGGL(k_gram_sum, dim3(cdiv(z.NT * 1024, 256), L), dim3(256), 0, st, part, z.nchunk,
                     z.NT, G);
  FM_TRY(check_launch("moe_cluster_experts (Gram sum)"));
  ClusterArgs ca{G, tuning, budget, labels, features, iters, E, z.NB, r, max_iter};
  hipLaunchKernelGGL(k_cluster, dim3(L), dim3(CL_TH), 0, st, ca);
  return check_launch("moe_cluster_experts (PCA, K-Means)");
}
