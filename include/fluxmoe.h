/*
 * fluxmoe.h - C ABI of the MoE-layer hot path of Flux (federated fine-tuning of
 * sparsely activated LLMs), hand-written HIP for MI355X (gfx950).
 *
 * The layer each participant runs during local fine-tuning:
 *   route (softmax top-k gate)  ->  re-route to slots and permute into per-slot
 *   buckets  ->  grouped SwiGLU expert FFN  ->  gate-weighted combine,
 * and its backward; plus the two once-per-round steps that build the layer:
 *   int8 profiling histogram (activation frequencies)  ->  expert merging.
 *
 * Conventions shared by every entry point
 * ---------------------------------------
 * Memory.   Every tensor argument is caller-owned DEVICE memory, dense and
 *           row-major, unless the comment says "host".  Tensor pointers must be
 *           16-byte aligned (MOE_ERR_ALIGN otherwise).  The library allocates
 *           nothing: calls that need scratch take (ws, ws_bytes), sized by the
 *           matching *_workspace_size() function; too small -> MOE_ERR_WORKSPACE.
 * Streams.  `stream` is a hipStream_t passed as void* (NULL = default stream).
 *           Every call only enqueues work on it and returns; nothing
 *           synchronises the host.  The library keeps no state between calls.
 * Dtypes.   MOE_F32 or MOE_BF16 for activations and weights (one dtype per
 *           call), MOE_I8 for quantised codes.  Index arrays are int32,
 *           gates and scales fp32.  bf16 math accumulates in fp32.
 * Limits.   1 <= k <= min(E, 16), 1 <= E <= 256, d % 8 == 0, I % 8 == 0,
 *           T >= 0, routed slots <= 512, shared <= 511.  T == 0 enqueues nothing and
 *           per-token buffers may then be NULL (moe_permute still zeroes the
 *           offsets; moe_grouped_swiglu_bwd still writes zero weight
 *           gradients unless accumulating).  Anything else:
 *           MOE_ERR_UNSUPPORTED or MOE_ERR_ARG.
 * Errors.   Every function returns MOE_OK or an error code.  Arguments are
 *           validated on the host before any HIP call, so an invalid call
 *           enqueues nothing.  moe_last_error() gives a message for the last
 *           failure on the calling thread.  No C++ exception crosses the ABI.
 * Outputs.  Fully overwritten, except `counts` of moe_profile_hist and
 *           moe_profile_route (adds) and
 *           the weight gradients of moe_grouped_swiglu_bwd when accumulate_dw.
 */
#ifndef FLUXMOE_H
#define FLUXMOE_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

enum {
  MOE_OK = 0,
  MOE_ERR_ARG = 1,          /* null required pointer, negative or inconsistent size */
  MOE_ERR_UNSUPPORTED = 2,  /* outside the limits above, or an unsupported dtype */
  MOE_ERR_ALIGN = 3,        /* tensor pointer not 16-byte aligned */
  MOE_ERR_WORKSPACE = 4,    /* workspace missing or too small */
  MOE_ERR_HIP = 5           /* a HIP launch failed (message has the HIP error) */
};

enum { MOE_F32 = 0, MOE_BF16 = 1, MOE_I8 = 2 };

/* Message of the last failed call on this thread ("" if none). */
const char* moe_last_error(void);
/* ABI revision of this header. */
int moe_abi_version(void);
#define FLUXMOE_ABI_VERSION 3

/* ---------------------------------------------------------------- routing --
 * moe_route_topk: the gating network of an MoE layer (Section 2.1, "MoE":
 * tokens pass through a gating network that assigns them to experts).  The
 * paper gives no formula; this is the softmax gate with top-k:
 *   logit[t,e] = sum_i X[t,i] * Wr[e,i] + bias[e]      (fp32 accumulation)
 *   idx[t,:]   = the k experts of largest logit, in rank order; equal logits
 *                rank the lower expert index first (-0.0 equals +0.0)
 *   gate[t,j]  = exp(logit[t,idx[t,j]]) / sum_j' exp(logit[t,idx[t,j']])
 *                (= softmax over all E renormalised over the selected k)
 * X [T,d], Wr [E,d] in `dtype`; bias [E] fp32 or NULL; idx [T,k] int32;
 * gate [T,k] fp32; logits [T,E] fp32 or NULL (written when given).
 */
int moe_route_topk(const void* X, const void* Wr, int dtype, const float* bias,
                   int T, int d, int E, int k,
                   int32_t* idx, float* gate, float* logits, void* stream);

/* moe_route_bwd: the router's backward pass with the top-k selection held
 * fixed (the selection is piecewise constant in the logits; the gate of a
 * token is the softmax of its selected logits, as in moe_route_topk).  From
 * the gradient dgate of the gates (moe_unpermute_bwd's dgate):
 *   dlogit[t,j] = gate[t,j] * (dgate[t,j] - sum_i gate[t,i] * dgate[t,i])
 *   dX[t,:]     = (accumulate ? dX[t,:] : 0) + sum_j dlogit[t,j] * Wr[idx[t,j],:]
 * (fp32 sums, one rounding to `dtype`).  With accumulate = 1 this adds the
 * router's share to the expert path's dX of the same tokens.  No gradient of
 * Wr or bias is formed: the router is frozen in expert-only tuning (Section 3).
 * gate, dgate [T,k] fp32; idx [T,k] int32 as written by moe_route_topk
 * (entries outside [0, E) are clamped); Wr [E,d] and dX [T,d] in `dtype`.
 * Limits as for moe_route_topk.
 */
int moe_route_bwd(const float* gate, const int32_t* idx, const float* dgate, const void* Wr, int dtype,
                  int T, int d, int E, int k, void* dX, int accumulate, void* stream);

/* ------------------------------------------------- quantisation profiling --
 * moe_quantize_int8: the low-bit profiling copy of a weight matrix
 * (Section 4.1, quantisation-based local profiling), one symmetric scale per
 * row: scale[e] = max_i |W[e,i]| / 127 (fp32 division);
 * Wq[e,i] = clamp(round_half_even(W[e,i] / scale[e]), -127, 127) with the
 * quotient in fp32; a zero row gets scale 0 and codes 0.
 * W [E,d] in `dtype`; Wq [E,d] int8; scale [E] fp32.  Here E is any row
 * count >= 1 (not limited to 256).
 */
int moe_quantize_int8(const void* W, int dtype, int E, int d,
                      int8_t* Wq, float* scale, void* stream);

/* moe_profile_hist: expert activation histogram of the int8 profiling router
 * (Section 4.1; the activation frequency of Section 2.2, Observation 2, is
 * counts[e] / tokens).
 *   logit~[t,e] = scale[e] * sum_i X[t,i] * Wq[e,i] + bias[e]
 *   top-k of logit~ with the rule of moe_route_topk, then
 *   counts[e] += #{t : e in top-k(t)}          (ADDS to counts; int32)
 * X [T,d] in x_dtype (MOE_F32 / MOE_BF16); Wq [E,d] int8; scale [E] fp32;
 * bias [E] fp32 or NULL; counts [E] int32; idx [T,k] int32 or NULL.
 * Integer atomics only: the result does not depend on scheduling.
 */
int moe_profile_hist(const void* X, int x_dtype, const int8_t* Wq,
                     const float* scale, const float* bias,
                     int T, int d, int E, int k,
                     int32_t* counts, int32_t* idx, void* stream);

/* moe_profile_route: the int8 profiling router of moe_profile_hist that also
 * hands its routing to the profiling forward (Section 4.1: the low-bit copy
 * of the model is run, not only its routers): counts[e] += the histogram as
 * in moe_profile_hist, and idx [T,k] int32 (rank order) and gate [T,k] fp32
 * (softmax over the k selected int8 logits~, as moe_route_topk does over its
 * logits) are written.  idx and gate are required.
 */
int moe_profile_route(const void* X, int x_dtype, const int8_t* Wq,
                      const float* scale, const float* bias,
                      int T, int d, int E, int k,
                      int32_t* counts, int32_t* idx, float* gate, void* stream);

/* moe_dequant_int8: the matrices the profiling forward runs on (Section 4.1):
 *   out[r, c] = q[r, c] * scale[r]   (fp32 product, one rounding to out_dtype)
 * q [rows, cols] int8 (e.g. every expert's W_gate rows stacked: rows = E*I),
 * scale [rows] fp32 from moe_quantize_int8, out [rows, cols] in out_dtype
 * (MOE_BF16 or MOE_F32).  cols % 8 == 0.
 */
int moe_dequant_int8(const int8_t* q, const float* scale, long rows, int cols,
                     int out_dtype, void* out, void* stream);

/* moe_residual_add: out = X + Y elementwise (fp32 add, one rounding), the
 * residual stream that carries one layer's output into the next layer of the
 * profiling stack.  X, Y, out [T,d] in dtype; out may alias X.  d % 8 == 0.
 */
int moe_residual_add(const void* X, const void* Y, int T, int d, int dtype,
                     void* out, void* stream);

/* moe_rms_norm: the input of a layer of the profiling stack (Section 4.1 runs
 * the low-bit copy of the paper's models, pre-norm transformers whose MoE
 * layers read the RMS-normalised residual stream), optionally fused with the
 * residual add that produces that stream:
 *   S        = X + Y (fp32 add, one rounding to dtype), or S = X when Y is NULL
 *   out_sum  = S                                   (when out_sum != NULL)
 *   out_norm = S / sqrt(mean_i S[t,i]^2 + eps)     (per row, from the rounded S,
 *              fp32, one rounding; unit gain; a zero row stays zero)
 * X, Y, out_sum, out_norm [T,d] in dtype.  out_sum may alias X or Y; out_norm
 * aliases none of them (MOE_ERR_ARG).  eps finite and >= 0; d % 8 == 0.
 */
int moe_rms_norm(const void* X, const void* Y, int T, int d, int dtype, float eps,
                 void* out_sum, void* out_norm, void* stream);

/* ---------------------------------------------------------------- merging --
 * moe_merge_plan: which experts of one layer are merged, from its histogram
 * (Sections 5.1-5.2 decide how many and which experts share a group; this
 * entry point implements the frequency rule: the least-activated experts are
 * merged).  Experts are ranked by (counts desc, index asc).  The last n_merge
 * are merged: walked from the least activated upwards they are cut into
 * consecutive groups of `group`.  Kept experts take routed slots 0..K-1 in
 * rank order (K = E - n_merge), group g takes slot K + g.
 * Outputs (device, int32 unless noted):
 *   expert_map[E]        original expert -> routed slot (gate re-routing, Sec. 7)
 *   slot_src[K + G]      kept slot j -> its expert; group slot K+g -> E + g
 *   grp_ptr[grp_base .. grp_base+G]   CSR row pointers of the groups, values
 *                        offset by member_base (entries of the whole CSR
 *                        outside this range are not touched)
 *   grp_member[member_base .. member_base+n_merge)  expert_base + expert id
 *   alpha[expert_base .. expert_base+E) (fp32) = counts[e] / total_tokens,
 *                        the activation frequency f_e
 * Several layers write disjoint ranges of one CSR so that one
 * moe_merge_experts call merges them all.  n_merge % group == 0, group >= 1.
 */
int moe_merge_plan(const int32_t* counts, int E, int n_merge, int group,
                   float total_tokens, int expert_base, int grp_base, int member_base,
                   int32_t* expert_map, int32_t* slot_src, int32_t* grp_ptr,
                   int32_t* grp_member, float* alpha, void* stream);

/* moe_activation_frequency: freq[e] = counts[e] / total_tokens, the activation
 * frequency of Section 2.2 (Observation 2).  counts [E] int32, freq [E] fp32.
 */
int moe_activation_frequency(const int32_t* counts, int E, float total_tokens, float* freq,
                             void* stream);

/* moe_merge_experts: importance-weighted merging of grouped experts
 * (Section 5.3, Eq. 2):  W_g = sum_{e in g} (alpha_e / sum_{e' in g} alpha_e') W_e
 * for each of the expert's three matrices; a group whose alphas sum to 0 takes
 * the plain mean.  fp32 accumulation, one rounding on store.
 *   w_src: device array of 3*E_total device pointers, (gate, up, down) of
 *          expert e at [3e, 3e+1, 3e+2]; gate/up are [I,d], down is [d,I].
 *   grp_ptr[G+1], grp_member[grp_ptr[G]]: CSR of expert ids (into w_src/alpha).
 *   alpha[E_total] fp32 (the paper's f_e * a_e; any non-negative weights).
 *   w_dst: device array of 3*G device pointers, outputs in out_dtype.
 * Groups may span layers: this is the single launch that merges every layer.
 */
int moe_merge_experts(const void* const* w_src, int dtype, int d, int I, int G,
                      const int32_t* grp_ptr, const int32_t* grp_member,
                      const float* alpha, void* const* w_dst, int out_dtype,
                      void* stream);

/* moe_slot_pointers: per-slot weight pointer tables of a layer after merging.
 * Slot s < S reads from orig_*[slot_src[s]] when slot_src[s] < E and from
 * merged_*[slot_src[s] - E] otherwise (stacked [E or G][rows][cols] tensors).
 * Writes w_gate[s], w_up[s], w_down[s] (device arrays of device pointers) for
 * s in [0, S); the caller appends shared experts after them.
 */
int moe_slot_pointers(const int32_t* slot_src, int S, int E, int d, int I, int dtype,
                      const void* orig_gate, const void* orig_up, const void* orig_down,
                      const void* merged_gate, const void* merged_up,
                      const void* merged_down,
                      const void** w_gate, const void** w_up, const void** w_down,
                      void* stream);

/* ------------------------------------------------- layer-aware merging ----
 * moe_merge_budget: how many groups each layer's non-tuning experts are
 * merged into (Section 5.1, Eq. 1).  For layer l = 0..L-1 (the paper's l + 1):
 *   f_e = counts[l, e] / total_tokens,  v_l = max(population variance of f
 *   over the layer's E experts, eps),   b_l = (L - l) / v_l,
 *   share_l = B_non * b_l / sum_k b_k   (fp64; sum in layer order).
 * budget_l = floor(share_l) clamped to [min(1, n_l), n_l], n_l the layer's
 * non-tuning experts; then, while the total is below B_non, +1 to the layer
 * with the largest share_l - budget_l that is below n_l (ties: lower layer);
 * while above, -1 to the layer with the smallest share_l - budget_l above its
 * floor (ties: higher layer).  The total equals B_non whenever
 * sum min(1, n_l) <= B_non <= sum n_l.
 *   counts [L, E] int32 (device), tuning [L, E] uint8 (device, 1 = tuning
 *   expert), budget [L] int32 (device, written).  1 <= L <= 1024.
 */
int moe_merge_budget(const int32_t* counts, const uint8_t* tuning, int L, int E,
                     float total_tokens, int B_non, double eps, int32_t* budget,
                     void* stream);

/* moe_cluster_experts: which non-tuning experts of each layer share a group
 * (Section 5.2), for all L layers in one call.
 *   Features: the parameters of expert (l, e) form one vector, W_gate, W_up and
 *   W_down row-major in that order (D = 3 I d values).  Over the layer's n_l
 *   non-tuning experts the vectors are centred on their mean; the features are
 *   the scores on the r leading principal components (U sqrt(lambda) of the
 *   centred n_l x n_l Gram matrix, eigenvalues descending, ties lower index;
 *   components past the rank score 0), scaled to unit length (a zero vector
 *   stays zero).  The Gram matrix accumulates the stored values' products in
 *   fp32 per 32768-parameter chunk and sums chunks in fp64; the
 *   eigen-decomposition (cyclic Jacobi) and all that follows are fp64.
 *   K-Means with cosine similarity: B_l = clamp(budget[l], 1, n_l) centroids
 *   per layer, seeded by farthest-first traversal under 1 - cos (first the
 *   expert with the largest score norm, then the unchosen expert farthest from
 *   its nearest seed; ties lower index).  Each pass assigns every expert to the
 *   most similar centroid of its own layer (ties: lower centroid), then sets
 *   each centroid to the mean of its members' unit features (an empty cluster
 *   keeps its centroid).  A layer stops at the first pass that changes none of
 *   its labels, or after max_iter passes.
 *   w_src   device array of 3*L*E device pointers, (gate, up, down) of expert
 *           (l, e) at 3*(l*E + e) + {0, 1, 2}; gate/up [I, d], down [d, I],
 *           16-byte aligned, in dtype (MOE_BF16 or MOE_F32).
 *   tuning  [L, E] uint8 (device), 1 = tuning expert (not clustered).
 *   budget  [L] int32 (device), e.g. from moe_merge_budget.
 *   labels  [L, E] int32 (device, written): cluster in [0, B_l) for non-tuning
 *           experts, -1 for tuning ones.
 *   features  optional [L, E, r] fp32 (device): the unit features, 0 for
 *           tuning experts.   iters  optional [L] int32: passes run.
 *   ws      device workspace of moe_cluster_workspace_size(L, E, d, I) bytes.
 * Limits: E <= 64, 1 <= r <= 32, I*d*element size a multiple of 16 bytes,
 * max_iter >= 1.
 */
size_t moe_cluster_workspace_size(int L, int E, int d, int I);
int moe_cluster_experts(const void* const* w_src, int dtype, int L, int E, int d, int I,
                        const uint8_t* tuning, const int32_t* budget, int r, int max_iter,
                        void* ws, size_t ws_bytes, int32_t* labels, float* features,
                        int32_t* iters, void* stream);

/* ------------------------------------------------------------ the layer ----
 * A layer's slots: routed slots 0..S_routed-1 (kept experts and merged
 * groups), then S_shared always-on shared experts (gate 1.0, every token).
 * All pointer members are DEVICE arrays of S_routed + S_shared device pointers;
 * the matrices they point to must be 16-byte aligned (read on the device only,
 * not checked).
 * Non-tuning (merged, frozen) slots have dw_* == NULL: they get dX but no dW
 * (Section 1 and Section 3: non-tuning experts are merged and frozen).
 *
 * Row spaces.  For T tokens and top-k, routed rows live at [0, T*k) of every
 * per-row buffer (X_perm, A_g, A_u, H, O, dO, dX_perm), slot s at
 * [offsets[s], offsets[s+1]); rows from offsets[S_routed] to T*k are unused.
 * Shared slot i owns rows [T*k + i*T, T*k + (i+1)*T), one per token.  So
 * per-row buffers have R_tot = T*(k + S_shared) rows.
 */
typedef struct moe_layer {
  int d;            /* hidden size */
  int I;            /* expert intermediate size */
  int dtype;        /* MOE_F32 or MOE_BF16: weights and activations */
  int S_routed;     /* routed slots */
  int S_shared;     /* shared experts */
  const void* const* w_gate;   /* [S] -> [I,d] */
  const void* const* w_up;     /* [S] -> [I,d] */
  const void* const* w_down;   /* [S] -> [d,I] */
  float* const* dw_gate;       /* [S] -> [I,d] fp32, NULL = frozen slot */
  float* const* dw_up;         /* [S] -> [I,d] fp32, NULL = frozen slot */
  float* const* dw_down;       /* [S] -> [d,I] fp32, NULL = frozen slot */
} moe_layer;

/* moe_permute: gate re-routing (Section 7) and the per-slot token subsets D^e
 * of Section 4.1 as contiguous buckets.
 *   slot[t,j] = expert_map[idx[t,j]]   (identity when expert_map is NULL)
 *   choices of one token that land on the same slot form one row whose gate
 *   is their sum (in j order); rows of a slot are ordered by token;
 *   offsets = exclusive prefix sum of the per-slot row counts.
 * Outputs: offsets[S_routed+1]; perm_token[T*k] (row -> token); perm_gate[T*k]
 * fp32; inv[T,k]: p for the choice that opened row p, -2-p for a choice folded
 * into row p; X_perm[T*k, d] with X_perm[p] = X[perm_token[p]].  Entries at or
 * beyond offsets[S_routed] are left untouched.  x_sq [T] fp32 (optional, NULL
 * = not written): ||X[t]||^2, the squares of X's elements summed in fp32 in a
 * fixed order, the per-token input norms the expert utility (Eq. 3,
 * moe_expert_utility) needs, formed while the rows are read anyway.  idx
 * values must be in [0, E) and expert_map values in [0, S_routed) (not checked
 * on the device; see moe_validate_routing and FLUXMOE_DEBUG_CHECKS).
 */
int moe_permute(const void* X, int dtype, const int32_t* idx, const float* gate,
                const int32_t* expert_map, int T, int d, int E, int k, int S_routed,
                int32_t* offsets, int32_t* perm_token, float* perm_gate,
                int32_t* inv, void* X_perm, void* ws, size_t ws_bytes, float* x_sq, void* stream);
size_t moe_permute_workspace_size(int T, int k, int S_routed);

/* moe_permute_noalloc: moe_permute for callers that cannot allocate device
 * memory or hand over a workspace (code under HIP graph capture, tight serving
 * loops, harnesses that forbid hipMalloc).  Same arguments, outputs and
 * errors as moe_permute, without (ws, ws_bytes): the count table lives in a
 * device array of the library, moe_permute_noalloc_max_bytes() bytes (1 MiB)
 * on each device it runs on, held until the process ends.  Calls whose table,
 * moe_permute_workspace_size(T, k, S_routed), exceeds that are rejected with
 * MOE_ERR_UNSUPPORTED before anything is enqueued (e.g. T <= 131072 tokens at
 * 512 slots, T <= 1048576 at 64).  Every call on a device shares the array:
 * calls that overlap on one device (several streams or threads) race and must
 * be serialised by the caller.  Calls no allocating routine; the first call on
 * a device looks the array's address up (hipGetSymbolAddress).  The debug
 * range check of FLUXMOE_DEBUG_CHECKS is not run by this variant.
 */
int moe_permute_noalloc(const void* X, int dtype, const int32_t* idx, const float* gate,
                        const int32_t* expert_map, int T, int d, int E, int k, int S_routed,
                        int32_t* offsets, int32_t* perm_token, float* perm_gate,
                        int32_t* inv, void* X_perm, float* x_sq, void* stream);
size_t moe_permute_noalloc_max_bytes(void);

/* moe_validate_routing: range check of moe_permute's index inputs, for
 * debugging a caller (the routing it hands over must name experts that exist
 * and slots that exist, Section 7's re-routing table included).  idx [T,k] and
 * expert_map [E] (or NULL = identity, which needs S_routed >= E) are HOST
 * arrays.  Returns MOE_OK, or MOE_ERR_ARG naming the first entry outside
 * [0, E) resp. [0, S_routed).  With the environment variable
 * FLUXMOE_DEBUG_CHECKS set (to anything but "0"), moe_permute itself copies
 * idx and expert_map to the host, waits for `stream`, and runs this check
 * before it enqueues anything (slow: debugging only).  The same switch makes
 * the later entry points check the maps they index memory through, the same
 * way, before they enqueue anything: inv (every entry decodes to a row in
 * [0, T*k)) in moe_unpermute, moe_unpermute_bwd and moe_permute_bwd; offsets
 * (0 first, non-decreasing, at most T*k) in moe_unpermute_bwd, the grouped
 * SwiGLU forward (both) and backward, and moe_expert_utility; perm_token
 * (tokens in [0, T) over the routed rows) in moe_expert_utility.  A failed
 * check returns MOE_ERR_ARG naming the map and the entry.  A checking call
 * synchronises the stream, so it cannot be captured into a HIP graph.
 */
int moe_validate_routing(const int32_t* idx, const int32_t* expert_map, int T, int E, int k, int S_routed);

/* moe_grouped_swiglu_fwd: every slot's SwiGLU expert FFN on its rows
 * (the experts of Section 2.1; tuning and frozen slots alike):
 *   A_g = X_s W_gate^T,  A_u = X_s W_up^T,  H = silu(A_g) * A_u,  O = H W_down^T
 * with silu(z) = z / (1 + exp(-z)).  Routed slots read X_perm rows
 * [offsets[s], offsets[s+1]); shared slots read X [T,d].
 * Outputs (per-row buffers of R_tot rows, `L->dtype`): A_g, A_u, H [R_tot, I]
 * (kept for the backward) and O [R_tot, d].
 */
int moe_grouped_swiglu_fwd(const moe_layer* L, const void* X, const void* X_perm,
                           const int32_t* offsets, int T, int k,
                           void* A_g, void* A_u, void* H, void* O,
                           void* ws, size_t ws_bytes, void* stream);
size_t moe_grouped_swiglu_fwd_workspace_size(const moe_layer* L, int T, int k);

/* moe_grouped_swiglu_fwd_q8: the forward of the quantised profiling model
 * (Section 4.1: a low-bit copy of the experts decides nothing but which
 * experts the next layers see).  Expert weights are int8 codes with one fp32
 * scale per row, W = diag(s) Q as moe_quantize_int8 writes them; activations
 * are bf16.  Per slot, with the scales applied to the fp32 products:
 *   H = silu(s_g * (X_s Q_gate^T)) * (s_u * (X_s Q_up^T)),  O = s_d * (H Q_down^T)
 * (s_* scale output columns).  The codes are widened exactly to bf16 inside the
 * GEMM; no dequantised copy of the weights is made.  Rows, offsets, X, X_perm,
 * H [R_tot, I] and O [R_tot, d] as in moe_grouped_swiglu_fwd (bf16); A_g and
 * A_u are not written.  Limits: d and I multiples of 16; the struct's tables
 * are DEVICE arrays of S_routed + S_shared device pointers:
 *   q_gate, q_up [S] -> [I,d] int8;  q_down [S] -> [d,I] int8;
 *   s_gate, s_up [S] -> [I] fp32;    s_down [S] -> [d] fp32.
 * The pointers in the tables are read on the device only: each code matrix
 * must be 16-byte aligned and each scale array 4-byte aligned (not checked).
 */
typedef struct moe_layer_q8 {
  int d;
  int I;
  int S_routed;
  int S_shared;
  const int8_t* const* q_gate;
  const int8_t* const* q_up;
  const int8_t* const* q_down;
  const float* const* s_gate;
  const float* const* s_up;
  const float* const* s_down;
} moe_layer_q8;
int moe_grouped_swiglu_fwd_q8(const moe_layer_q8* L, const void* X, const void* X_perm,
                              const int32_t* offsets, int T, int k, void* H, void* O,
                              void* ws, size_t ws_bytes, void* stream);
size_t moe_grouped_swiglu_fwd_q8_workspace_size(const moe_layer_q8* L, int T, int k);

/* moe_unpermute: the gate-weighted combine of the expert outputs, the output
 * of the MoE layer of Section 2.1 (each token's output is the sum of its
 * selected experts' outputs weighted by the gating network's gates; shared
 * experts add with gate 1):
 *   Y[t] = sum_{j: inv[t,j] >= 0} perm_gate[inv[t,j]] * O[inv[t,j]]
 *          + sum_{shared i} O[T*k + i*T + t]              (fp32 accumulation)
 * O [R_tot, d] and Y [T, d] in L->dtype.
 */
int moe_unpermute(const moe_layer* L, const void* O, const int32_t* inv,
                  const float* perm_gate, int T, int k, void* Y, void* stream);

/* moe_unpermute_bwd: backward of the combine of moe_unpermute (the MoE layer
 * output of Section 2.1) with the gates as constants: the experts are what is
 * fine-tuned (Sections 1 and 3), so the expert path's gradient holds the
 * routing fixed; dgate hands the gates' share to moe_route_bwd:
 *   dO[p] = perm_gate[p] * dY[perm_token[p]]  for routed rows p < offsets[S_routed]
 *   dO[T*k + i*T + t] = dY[t]                  for shared slot i
 *   dgate[t,j] = <dY[t], O[row of (t,j)]>      (optional, fp32, when dgate != NULL;
 *                folded choices read the row they were folded into)
 *   dy_sq[t] = ||dY[t]||^2                     (optional, fp32 [T], when dy_sq != NULL:
 *                the squares summed in fp32 in a fixed order; the per-token
 *                output-gradient norms of moe_expert_utility, Eq. 3)
 */
int moe_unpermute_bwd(const moe_layer* L, const void* dY, const void* O,
                      const int32_t* inv, const int32_t* offsets,
                      const float* perm_gate, int T, int k,
                      void* dO, float* dgate, float* dy_sq, void* stream);

/* moe_grouped_swiglu_bwd: backward of every slot's SwiGLU FFN.  Only tuning
 * experts are updated during local fine-tuning; non-tuning experts are merged
 * and frozen (Section 1; Section 3, the tuning / non-tuning roles), so weight
 * gradients are formed for tuning slots only, while every slot passes dX on to
 * earlier layers:
 *   dH   = dO W_down
 *   dA_u = dH * silu(A_g)
 *   dA_g = dH * A_u * s * (1 + A_g (1 - s)),  s = sigmoid(A_g)
 *   dX_s = dA_g W_gate + dA_u W_up                 -> dX_perm rows (all slots)
 *   tuning slots only (dw_* != NULL), sums over the slot's rows in fp32:
 *   dW_down = dO^T H,  dW_gate = dA_g^T X_s,  dW_up = dA_u^T X_s
 * accumulate_dw = 0 overwrites dW (a tuning slot with no rows gets zeros),
 * 1 adds to it.  Inputs are the forward's saved A_g, A_u, H and the combine
 * backward's dO; dX_perm [R_tot, d] in L->dtype.
 */
int moe_grouped_swiglu_bwd(const moe_layer* L, const void* X, const void* X_perm,
                           const int32_t* offsets, int T, int k,
                           const void* A_g, const void* A_u, const void* H,
                           const void* dO, void* dX_perm, int accumulate_dw,
                           void* ws, size_t ws_bytes, void* stream);
size_t moe_grouped_swiglu_bwd_workspace_size(const moe_layer* L, int T, int k);

/* moe_expert_utility: the utility of each slot's expert (Section 6.1, Eq. 3),
 * the quantity the expert role assignment ranks experts by.  Eq. 3's summand
 * is garbled in print; read as the squared norm of the per-token gradient:
 *   u[s] = |D_s| * sqrt((1/|D_s|) * sum_{r in D_s} ||g_r||^2),
 * D_s the slot's rows (its tokens; a token whose choices share the slot is one
 * row with the summed gate) and g_r the gradient of the slot's W_gate, W_up,
 * W_down from row r alone, three rank-one products, so
 *   ||g_r||^2 = ||dO_r||^2 ||h_r||^2 + (||dA_g,r||^2 + ||dA_u,r||^2) ||x_r||^2
 * with x_r = X[t] and dO_r = gate_r dY[t] for the row's token t (gate 1 on a
 * shared slot).  The sums of squares of dA_g, dA_u and h = silu(a_g) a_u over
 * each row are left in the workspace by moe_grouped_swiglu_bwd (its dH step,
 * h recomputed from the saved A_g, A_u); the per-token ||X[t]||^2 and
 * ||dY[t]||^2 come from moe_permute (x_sq) and moe_unpermute_bwd (dy_sq),
 * which form them as they read X and dY; this call combines them per row and
 * reduces per slot (per-row and per-token sums in fp32, per-slot sums in fp64,
 * fixed order); an empty slot gets 0.  Every slot gets a utility, frozen ones
 * included.  Call it after moe_grouped_swiglu_bwd on the same stream with that
 * call's workspace and the same layer, offsets, T and k; nothing else may use
 * the workspace in between.
 * x_sq, dy_sq [T] fp32; perm_token, perm_gate: moe_permute's maps (may be NULL
 * when S_routed == 0); utility [S] fp32.
 */
int moe_expert_utility(const moe_layer* L, const float* x_sq, const float* dy_sq,
                       const int32_t* perm_token, const float* perm_gate,
                       const int32_t* offsets, int T, int k, void* ws, size_t ws_bytes,
                       float* utility, void* stream);

/* moe_permute_bwd: gradient of moe_permute's gather of each token into the
 * buckets of the slots it is re-routed to (the token subsets D^e of
 * Section 4.1 after the gate re-routing of Section 7): every row a token
 * opened sends its gradient back to that token (a deterministic gather):
 *   dX[t] = sum_{j: inv[t,j] >= 0} dX_perm[inv[t,j]]
 *           + sum_{shared i} dX_perm[T*k + i*T + t]       (fp32 accumulation)
 */
int moe_permute_bwd(const moe_layer* L, const void* dX_perm, const int32_t* inv,
                    int T, int k, void* dX, void* stream);

#ifdef __cplusplus
}
#endif
#endif /* FLUXMOE_H */
