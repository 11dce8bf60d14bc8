/*
 * moe.h - C ABI of the MI355X (gfx950) MoE expert-layer library.
 *
 * The layer is the Mixture-of-Experts feed-forward block of
 * Mixture-of-Parallelisms (Sec. 2.1, "Mixture-of-Experts": a light router
 * sends every token to its top-k of E experts; Sec. 3.1: H = d model width,
 * I = f expert width, k routing degree, N = T tokens on the device; eq.
 * (peaks): the N k H routed activations and the N_r I expert intermediates),
 * on one GPU's expert-parallel share (Sec. 3.2, hybrid expert parallelism:
 * this device owns experts [expert_begin, expert_begin + num_local)).
 * Sec. 3.3 (LLEP) moves where token-expert products run, never which ones
 * run, so the calls below compute exactly the plain layer.
 *
 * Conventions shared by every call
 *  - bf16 values are raw IEEE bfloat16 bit patterns (moe_bf16); fp32->bf16 is
 *    round-to-nearest-even.  All arrays are dense and row-major.
 *  - Every pointer is DEVICE memory owned by the caller; the library
 *    allocates nothing (callers pass workspaces sized by the
 *    *_workspace_bytes queries) and keeps no reference after the call
 *    returns.  Every product runs on the library's own kernels.  Required
 *    pointers must be non-NULL and 16-byte aligned.
 *  - `stream` is a hipStream_t passed as void* (NULL = default stream).
 *    Calls only enqueue work and return; no call synchronises the device.
 *    Data-dependent sizes (M, the number of local assignments) stay on the
 *    device: kernels read them from expert_offsets[num_local].
 *  - Return value: MOE_OK or a negative moe_status.  Arguments are checked
 *    on the host before any HIP call; on MOE_ERR_INVALID_ARG or
 *    MOE_ERR_WORKSPACE nothing was enqueued and outputs are untouched.
 *    moe_last_error() returns a message for the calling thread's last error.
 *  - Outputs must not alias inputs (moe_route_bwd's dx, updated in place, is
 *    the one exception).  Results are bitwise deterministic run to run (no
 *    floating-point atomics).
 *  - cap >= T * min(k, num_local) is the row capacity of permuted buffers;
 *    rows [M, cap) of them are never read and are left unspecified.
 *  - Limits: 1 <= k <= MOE_MAX_K, k <= E <= MOE_MAX_E, T >= 0,
 *    T * k < 2^31, d, f and H multiples of 8 in [8, MOE_MAX_DIM] (the
 *    kernels address a tile's rows with 32-bit offsets).  Calls outside the
 *    limits return MOE_ERR_INVALID_ARG.
 *  - Device-side garbage (an expert id outside [0, E) in a caller-supplied
 *    topk_idx) is undefined behaviour.
 */
#ifndef MOE_MI355X_H
#define MOE_MI355X_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#define MOE_ABI_VERSION 1
#define MOE_MAX_K 16
#define MOE_MAX_E 1024
#define MOE_MAX_DIM 262144
#define MOE_LLEP_MAX_RANKS 64
#define MOE_LLEP_MAX_GRANULE 65536
#define MOE_PERMUTE_NOALLOC_MAX_BYTES 8388608

typedef uint16_t moe_bf16;

enum moe_status {
  MOE_OK = 0,
  MOE_ERR_INVALID_ARG = -1,
  MOE_ERR_UNSUPPORTED = -2,
  MOE_ERR_WORKSPACE = -3,
  MOE_ERR_HIP = -4
};

/* flags of moe_grouped_swiglu_bwd */
enum { MOE_BWD_DGRAD = 1, MOE_BWD_WGRAD = 2 };

int moe_abi_version(void);
const char* moe_status_string(int status);
const char* moe_last_error(void);

/* ------------------------------------------------------------------ router
 * Router scores and top-k selection (Sec. 2.1: each token goes to its top-k
 * experts; the router is a dense weight, Sec. 3.1 eq. (param-decomp)).
 *
 * logits[t][e] = fp32 fused-multiply-add chain over j = 0..d-1 ascending of
 *   float(x[t][j]) * w_router[j][e], started at +0.0f, then + router_bias[e]
 *   (one fp32 add; bias optional).  This order is fixed so that routing is
 *   reproducible bit for bit on any device.
 * topk_idx[t][i], i = 0..k-1: the k experts with the largest logits, taken in
 *   the total order (logit descending, expert index ascending); -0.0 and +0.0
 *   are equal.  Slot i holds the i-th in that order.
 * topk_gate[t][i]: renorm = 0 -> softmax over all E logits, evaluated at the
 *   chosen expert; renorm = 1 -> softmax over the k chosen logits.
 *
 * x [T][d] bf16; w_router [d][E] fp32; router_bias [E] fp32 or NULL;
 * topk_idx [T][k] int32; topk_gate [T][k] fp32; logits [T][E] fp32 or NULL.
 * When logits is NULL the workspace must hold moe_route_workspace_bytes().
 * Logits must be finite (NaN routing is unspecified).
 */
int moe_route_workspace_bytes(int64_t T, int E, size_t* bytes);
int moe_route(const moe_bf16* x, const float* w_router, const float* router_bias, int64_t T,
              int d, int E, int k, int renorm, int32_t* topk_idx, float* topk_gate,
              float* logits, void* workspace, size_t workspace_bytes, void* stream);

/* --------------------------------------------------------- router backward
 * Gradient of the router (a dense weight, Sec. 3.1 eq. (param-decomp)) from
 * the gate gradients that moe_combine_bwd returns.  With s = sum_i dgate[t][i]
 * gate[t][i] (i ascending), the logit gradient is
 *   renorm = 0: dlogits[t][e] = -p_e s + sum over slots i with topk_idx = e of
 *               dgate[t][i] gate[t][i], p = softmax of logits[t] over all E;
 *   renorm = 1: dlogits[t][topk_idx[t][i]] = gate[t][i] (dgate[t][i] - s),
 *               0 for experts not chosen.
 * Then, with fixed summation orders (bitwise reproducible):
 *   dw_router[j][e] = sum over t of float(x[t][j]) dlogits[t][e]   (overwritten)
 *   dbias[e]        = sum over t of dlogits[t][e]                  (optional)
 *   dx[t][j]        = bf16( [float(dx[t][j]) +] sum over e of
 *                     dlogits[t][e] w_router[j][e] )               (optional)
 * in fp32 on the vector ALUs (e ascending for dx) when T*d*E < 2^28, and
 * above that on the library's bf16 matrix-core kernel with each fp32
 * operand v taken as bf16(v) + bf16(v - bf16(v)) (relative error <= 2^-17,
 * fp32 accumulation; token chunks of dw_router summed in order).  dlogits
 * and dbias are fp32 in both.
 * dx_accumulate = 1 adds the router's share to the expert path's input
 * gradient already in dx (e.g. from the unit-weight moe_combine of dx_perm),
 * giving the whole layer's dx; dx is then read and written in place (the one
 * allowed alias).  dx_accumulate = 0 writes the router's share alone.
 *
 * x [T][d] bf16; w_router [d][E] fp32; logits [T][E] fp32 (as moe_route
 * wrote them); topk_idx, topk_gate, dgate [T][k]; dw_router [d][E] fp32;
 * dbias [E] fp32 or NULL; dx [T][d] bf16 or NULL; dlogits [T][E] fp32 or
 * NULL (then kept in the workspace).  The workspace must hold
 * moe_route_bwd_workspace_bytes(), less the T*E*4 bytes of dlogits (rounded
 * up to 256) when dlogits is given; it may be NULL when that leaves 0.
 * T = 0 is valid: dw_router and dbias become exact zeros.
 */
int moe_route_bwd_workspace_bytes(int64_t T, int d, int E, size_t* bytes);
int moe_route_bwd(const moe_bf16* x, const float* w_router, const float* logits,
                  const int32_t* topk_idx, const float* topk_gate, const float* dgate,
                  int64_t T, int d, int E, int k, int renorm, float* dw_router, float* dbias,
                  moe_bf16* dx, int dx_accumulate, float* dlogits, void* workspace,
                  size_t workspace_bytes, void* stream);

/* ------------------------------------------------------------- permutation
 * Group this device's token-expert assignments into contiguous per-expert
 * segments (the N_r routed rows of Sec. 3.1 eq. (peaks)).
 *
 * Assignment a = t*k + i is local when expert_begin <= topk_idx[t][i] <
 *   expert_begin + num_local; its local expert is e' = topk_idx - expert_begin.
 * expert_offsets [num_local+1]: exclusive prefix sum of the per-expert
 *   counts; expert_offsets[num_local] = M.
 * counts_global [E] (optional): count of every expert over all assignments.
 * Rows of segment e' hold that expert's assignments in ascending a (a stable
 *   counting sort): row_src[p] = a for p < M; dst[a] = p, or -1 if a is not
 *   local.  x_perm[p][:] = x[row_src[p] / k][:] (a bit copy).
 *
 * x [T][d] bf16; topk_idx [T][k] int32; row_src [cap] int32; dst [T*k] int32;
 * x_perm [cap][d] bf16; workspace of moe_permute_workspace_bytes().
 * T = 0 is valid: offsets become zero.
 */
int moe_permute_workspace_bytes(int64_t T, int E, int k, int num_local, size_t* bytes);
int moe_permute(const moe_bf16* x, const int32_t* topk_idx, int64_t T, int d, int E, int k,
                int expert_begin, int num_local, int32_t* expert_offsets,
                int32_t* counts_global, int32_t* row_src, int32_t* dst, moe_bf16* x_perm,
                void* workspace, size_t workspace_bytes, void* stream);

/* moe_permute_noalloc: moe_permute for callers that cannot allocate device
 * memory or pass a workspace (code under HIP graph capture, tight serving
 * loops, harnesses that forbid hipMalloc).  Same arguments, results and
 * errors as moe_permute, minus the workspace: the call uses a static device
 * array of MOE_PERMUTE_NOALLOC_MAX_BYTES (8 MiB) that the library holds on
 * every GPU it runs on until the process ends, and calls no hipMalloc or
 * hipFree.  Sizes whose moe_permute_workspace_bytes() exceed that limit
 * (about T*k/4096 * (2*num_local + E) * 4 bytes; e.g. T*k = 2^19 with
 * E = 128 needs 0.2 MiB) return MOE_ERR_UNSUPPORTED.  Every call on one GPU
 * shares that GPU's array and leaves its contents behind: calls that
 * overlap on one GPU (different streams, or concurrent host threads)
 * race, so callers keep them ordered on one stream.
 */
int moe_permute_noalloc(const moe_bf16* x, const int32_t* topk_idx, int64_t T, int d, int E,
                        int k, int expert_begin, int num_local, int32_t* expert_offsets,
                        int32_t* counts_global, int32_t* row_src, int32_t* dst,
                        moe_bf16* x_perm, void* stream);

/* ----------------------------------------------------- grouped SwiGLU FFN
 * Expert feed-forward on the permuted rows (Sec. 3.1: Theta_exp = Theta(LEHI)
 * expert weights, N_r I intermediates).  For each local expert e and each row
 * p of its segment [expert_offsets[e], expert_offsets[e+1]):
 *   h_gate[p] = x_perm[p] W_gate[e],  h_up[p] = x_perm[p] W_up[e]
 *   a[p] = silu(h_gate[p]) * h_up[p],  silu(z) = z / (1 + exp(-z))
 *   y_perm[p] = a[p] W_down[e]
 * bf16 operands, fp32 accumulation, bf16 results (h_gate, h_up are saved for
 * the backward; a is computed from the rounded h_gate, h_up).  Experts with no
 * rows cost nothing; no padding to a capacity.
 *
 * w_gate, w_up [num_local][d][f]; w_down [num_local][f][d];
 * x_perm [cap][d]; h_gate, h_up [cap][f]; y_perm [cap][d]; all bf16.
 * expert_offsets [num_local+1] as produced by moe_permute.
 * Workspace: moe_grouped_swiglu_workspace_bytes(cap, num_local, d, f, 0).
 */
int moe_grouped_swiglu_workspace_bytes(int64_t cap, int num_local, int d, int f,
                                       unsigned flags, size_t* bytes);
int moe_grouped_swiglu_fwd(const moe_bf16* x_perm, const int32_t* expert_offsets, int num_local,
                           int64_t cap, int d, int f, const moe_bf16* w_gate,
                           const moe_bf16* w_up, const moe_bf16* w_down, moe_bf16* h_gate,
                           moe_bf16* h_up, moe_bf16* y_perm, void* workspace,
                           size_t workspace_bytes, void* stream);

/* Backward of the expert FFN, given dy_perm = dL/dy_perm:
 *   dA = dy_perm W_down[e]^T
 *   dh_gate = dA * h_up * silu'(h_gate),  silu'(z) = s (1 + z (1 - s)), s = sigmoid(z)
 *   dh_up = dA * silu(h_gate)
 * flags & MOE_BWD_DGRAD: dx_perm = dh_gate W_gate[e]^T + dh_up W_up[e]^T
 * flags & MOE_BWD_WGRAD: dw_gate[e] = x_perm_e^T dh_gate_e,
 *   dw_up[e] = x_perm_e^T dh_up_e, dw_down[e] = a_e^T dy_perm_e (sums over the
 *   rows of expert e); written (not accumulated) as bf16; an expert with no
 *   rows gets exact zeros.  dh_gate, dh_up and a are rounded to bf16.
 * dy_perm, x_perm [cap][d]; h_gate, h_up [cap][f]; dx_perm [cap][d];
 * dw_gate, dw_up [num_local][d][f]; dw_down [num_local][f][d]; all bf16.
 * Workspace: moe_grouped_swiglu_workspace_bytes(cap, num_local, d, f, flags).
 */
int moe_grouped_swiglu_bwd(const moe_bf16* dy_perm, const moe_bf16* x_perm,
                           const moe_bf16* h_gate, const moe_bf16* h_up,
                           const int32_t* expert_offsets, int num_local, int64_t cap, int d,
                           int f, const moe_bf16* w_gate, const moe_bf16* w_up,
                           const moe_bf16* w_down, moe_bf16* dx_perm, moe_bf16* dw_gate,
                           moe_bf16* dw_up, moe_bf16* dw_down, unsigned flags, void* workspace,
                           size_t workspace_bytes, void* stream);

/* ----------------------------------------------------------------- combine
 * Weighted combination of the expert outputs (Sec. 2.1):
 *   out[t] = sum over slots i = 0..k-1 ascending with dst[t*k+i] >= 0 of
 *            topk_gate[t][i] * y_perm[dst[t*k+i]]      (fp32 sum, bf16 result)
 * A token with no local slot gets 0.  topk_gate = NULL means weight 1; with
 * it this call is the backward of moe_permute (dx = sum of dx_perm rows).
 * y_perm [cap][d] bf16; dst [T*k] int32; topk_gate [T][k] fp32; out [T][d].
 */
int moe_combine(const moe_bf16* y_perm, const int32_t* dst, const float* topk_gate, int64_t T,
                int d, int k, moe_bf16* out, void* stream);

/* Backward of moe_combine, given dout = dL/dout:
 *   dy_perm[dst[t*k+i]] = topk_gate[t][i] * dout[t]          (bf16)
 *   dgate[t][i] = sum_j dout[t][j] * y_perm[dst[t*k+i]][j]   (fp32; 0 if not local)
 * dout [T][d] bf16; dy_perm [cap][d] bf16; dgate [T][k] fp32 or NULL.
 */
int moe_combine_bwd(const moe_bf16* dout, const moe_bf16* y_perm, const int32_t* dst,
                    const float* topk_gate, int64_t T, int d, int k, moe_bf16* dy_perm,
                    float* dgate, void* stream);

/* ---------------------------------------------- memory-efficient forward
 * The expert layer's forward over chunks of `chunk` tokens (the
 * memory-efficient variant of Sec. 3.3; its target is the O(N k H + N_r I)
 * transient of eq. (peaks): routed rows and expert intermediates exist for
 * one slice of the work at a time, while the next slice's row movement runs
 * beside the current slice's products).  For tokens [c*chunk, (c+1)*chunk)
 * it runs moe_permute, moe_grouped_swiglu_fwd and moe_combine (weighted by
 * topk_gate) into y, alternating chunks between `stream` and `stream2` with
 * two sets of transient buffers inside the workspace: the transient peak is
 * that of two chunks instead of all T tokens, and one chunk's permutation
 * and combine overlap the other chunk's grouped GEMMs.  Every row of y
 * depends on its own token only, so y is bit-identical to the unchunked
 * forward.  No backward state is kept (x_perm, h_gate, h_up are transient).
 *
 * x [T][d] bf16; topk_idx, topk_gate [T][k]; weights as for
 * moe_grouped_swiglu_fwd; y [T][d] bf16 (tokens with no local expert get 0).
 * workspace: moe_ffn_fwd_chunked_workspace_bytes(chunk, ...) bytes (it does
 * not depend on T).  `stream` is the caller's stream: the inputs must be
 * ready on it and the call's work is complete on it.  `stream2` may equal
 * `stream` (no overlap) or be another stream of the same device (made to
 * wait for `stream` first).  The library keeps one HIP event per device for
 * the two cross-stream waits.  The optional kernel profiler attributes the
 * two streams' interleaved kernels only approximately.
 */
int moe_ffn_fwd_chunked_workspace_bytes(int64_t chunk, int E, int k, int num_local, int d, int f,
                                        size_t* bytes);
int moe_ffn_fwd_chunked(const moe_bf16* x, const int32_t* topk_idx, const float* topk_gate,
                        int64_t T, int d, int E, int k, int expert_begin, int num_local, int f,
                        const moe_bf16* w_gate, const moe_bf16* w_up, const moe_bf16* w_down,
                        int64_t chunk, moe_bf16* y, void* workspace, size_t workspace_bytes,
                        void* stream, void* stream2);

/* Expert-range variant of the memory-efficient forward (Sec. 3.3, the same
 * target as moe_ffn_fwd_chunked).  The whole layer's permutation index
 * (moe_permute's offsets, row_src and dst, without gathering rows) is formed
 * once; the permuted rows [0, cap), cap = T * min(k, num_local), are then
 * taken in chunks of `chunk_rows` consecutive rows (consecutive experts, the
 * first and last possibly in part).  Each chunk's rows are gathered from x,
 * pass through moe_grouped_swiglu_fwd, and land in one y_perm of cap rows,
 * alternating chunks between `stream` and `stream2` with two sets of
 * buffers; a final moe_combine (weighted by topk_gate) forms y.  Token
 * chunks read every expert's weights once per chunk; here an expert's
 * weights are read by the one or two chunks its rows fall in, which is what
 * a layer bound by its weights needs.  The transient is y_perm (cap x d)
 * plus two chunks' rows, intermediates and activations, against all cap
 * rows of x_perm, h_gate, h_up, the activations and y_perm unchunked.  Every
 * y_perm row depends only on its own token and expert and the combine is
 * the unchunked one, so y is bit-identical to the unchunked forward.
 *
 * Arguments as for moe_ffn_fwd_chunked, with chunk_rows >= 1 in place of
 * chunk; workspace: moe_ffn_fwd_row_chunked_workspace_bytes(T, ...) bytes
 * (it grows with T: the index and y_perm cover the whole layer).
 */
int moe_ffn_fwd_row_chunked_workspace_bytes(int64_t T, int E, int k, int num_local, int d, int f,
                                            int64_t chunk_rows, size_t* bytes);
int moe_ffn_fwd_row_chunked(const moe_bf16* x, const int32_t* topk_idx, const float* topk_gate,
                            int64_t T, int d, int E, int k, int expert_begin, int num_local,
                            int f, const moe_bf16* w_gate, const moe_bf16* w_up,
                            const moe_bf16* w_down, int64_t chunk_rows, moe_bf16* y,
                            void* workspace, size_t workspace_bytes, void* stream,
                            void* stream2);

/* ------------------------------------------------------- vocabulary loss
 * Blockwise online loss of the vocabulary projection (Sec. 3.4, eq.
 * (voc-fwd-loss): Y = X W_voc, loss_n = Y[n][t_n] - log sum_v exp Y[n][v]),
 * on one device with the vocabulary walked in blocks of `vblock` columns
 * instead of split over ranks.  The logits are never stored: each block's
 * product reduces them in its epilogue (forward: a running max and sum of
 * exponentials per row, merged block by block; backward: the logit
 * gradient, the only per-block buffer, N x vblock bf16), and the loss and
 * its gradients are those of the dense projection up to rounding.
 *
 * x [N][H] bf16; w_voc [H][V] bf16; target [N] int32 in [0, V) (a target
 * outside [0, V) is undefined behaviour).  Logits are fp32 sums of bf16
 * products.  moe_vocab_loss_fwd writes loss [N] fp32 (the log-likelihood
 * of the target, <= 0) and lse [N] fp32 (log sum_v exp Y[n][v]), which the
 * backward takes back.  moe_vocab_loss_bwd, given dloss [N] fp32 =
 * dL/dloss, recomputes each block of logits and writes
 *   dx [N][H]  bf16 = sum_v G[n][v] W_voc[:, v]  (fp32 across blocks)
 *   dw_voc [H][V] bf16 = X^T G  (every column written; zeros when N = 0)
 * with G[n][v] = dloss_n ([v == t_n] - exp(Y[n][v] - lse_n)) rounded to
 * bf16 before the two products.  Limits: 0 <= N < 2^31, 1 <= V < 2^31, H a
 * multiple of 8, vblock a positive multiple of 8, N * vblock < 2^40.
 * workspace: moe_vocab_loss_workspace_bytes() bytes (serves both calls;
 * 2 N vblock bytes of logit gradients, up to 8 fp32 N x H slabs of dx
 * partial sums and N vblock / 8 bytes of per-64-column pairs; when V is not
 * a multiple of 8, also padded copies of one block of W and of dW).  It does
 * not depend on V otherwise.  All products run on the library's bf16
 * matrix-core kernel with fp32 accumulation.
 */
int moe_vocab_loss_workspace_bytes(int64_t N, int H, int64_t V, int64_t vblock, size_t* bytes);
int moe_vocab_loss_fwd(const moe_bf16* x, const moe_bf16* w_voc, const int32_t* target, int64_t N,
                       int H, int64_t V, int64_t vblock, float* loss, float* lse, void* workspace,
                       size_t workspace_bytes, void* stream);
int moe_vocab_loss_bwd(const moe_bf16* x, const moe_bf16* w_voc, const int32_t* target,
                       const float* lse, const float* dloss, int64_t N, int H, int64_t V,
                       int64_t vblock, moe_bf16* dx, moe_bf16* dw_voc, void* workspace,
                       size_t workspace_bytes, void* stream);

/* ------------------------------------------ least-loaded expert parallelism
 * Sec. 3.3 (recap of LLEP): the load of each rank is taken at every call
 * of the layer; a rank above its share hands some of its token-expert
 * products, together with the weights of those experts, to a rank below
 * it, which then computes them; the set of products does not change.  The
 * paper does not give the planning steps; this library's plan is:
 *   - load is counted in units of `granule` = g rows: g = 1 counts rows;
 *     g = the grouped GEMM's row-tile height (256) counts the tiles a
 *     rank's expert products run, since a window of w rows costs
 *     ceil(w / g) tiles however small w is;
 *   - E experts on E_p ranks, expert e at home on rank e / (E / E_p);
 *     u_e = ceil(counts[e] / g), U = sum u_e; capacity
 *     C = max(ceil(capacity / g), ceil(U / E_p)) units;
 *   - every rank keeps its own experts, ascending, while its load stays
 *     <= C units; the rest of an expert is its spill;
 *   - experts with spill, largest spill (in units) first (ties: lower
 *     index), hand it out in pieces of whole units, each to the rank with
 *     the fewest units (ties: lower rank) and as large as that rank's room
 *     below C; a piece of t units is t * g rows or what is left.
 * Expert e's assignments in the layer's row order (ascending t*k + i, the
 * order of moe_permute) are cut into consecutive windows: the home rank's
 * [0, keep) first, then the pieces in the order handed out.  Every window
 * but an expert's last is a whole number of units (no window splits a
 * tile); every rank's load is <= C units, so its largest tile count is the
 * least any plan can reach, ceil(U / E_p), when capacity = 0; a piece on a
 * rank other than the home is one shipment of that expert's weights.
 *
 * moe_llep_plan: counts [E] int32 (assignments per expert over all tokens,
 * e.g. moe_permute's counts_global) -> win_lo, win_hi [E_p][E] int32 (rank
 * r computes rows [win_lo[r][e], win_hi[r][e]) of expert e; empty windows
 * are [0, 0)), load [E_p] int32 (each rank's rows, at most C * g),
 * n_ship [1] int32.  One workgroup, all on the device (no host round trip
 * for the counts).  Limits: 1 <= E_p <= MOE_LLEP_MAX_RANKS, E a multiple
 * of E_p, capacity >= 0, 1 <= granule <= MOE_LLEP_MAX_GRANULE.
 *
 * moe_llep_dispatch: one rank's share of the layer under a plan.  Inputs:
 * x [T][d], topk_idx [T][k], and the permutation of ALL experts from
 * moe_permute(expert_begin = 0, num_local = E): offsets_all [E + 1] and
 * dst_all [T*k]; the plan (win_lo, win_hi, E_p) and the rank.  Outputs, in
 * the moe_permute layout over all E experts: offsets_r [E + 1] (expert e's
 * rows at [offsets_r[e], offsets_r[e + 1]), clamped to cap), row_src_r
 * [cap], dst_r [T*k] (-1 for assignments other ranks compute) and x_perm_r
 * [cap][d].  cap must be >= the rank's load (the plan's load output: at
 * most C * g rows, and never more than T*k); rows past cap are dropped.  The rank then
 * runs moe_grouped_swiglu_fwd/_bwd with num_local = E on these buffers (a
 * shipped expert's weights are read from the [E] weight arrays) and
 * moe_combine into its partial output; the partial outputs of all ranks
 * sum to the layer's output, and every y_perm row equals the one the whole
 * layer computes for that assignment.
 */
int moe_llep_plan(const int32_t* counts, int E, int E_p, int capacity, int granule,
                  int32_t* win_lo, int32_t* win_hi, int32_t* load, int32_t* n_ship, void* stream);
int moe_llep_dispatch(const moe_bf16* x, const int32_t* topk_idx, const int32_t* offsets_all,
                      const int32_t* dst_all, const int32_t* win_lo, const int32_t* win_hi,
                      int E_p, int rank, int64_t T, int d, int E, int k, int64_t cap,
                      int32_t* offsets_r, int32_t* row_src_r, int32_t* dst_r, moe_bf16* x_perm_r,
                      void* stream);

/* ------------------------------------------------------------- profiling
 * Optional per-kernel timing with HIP events recorded on the launch stream
 * around every kernel the library enqueues (for measurement only; off by
 * default).  moe_profile_query synchronises on the recorded events.
 */
int moe_profile_enable(int on);
int moe_profile_reset(void);
int moe_profile_num_kernels(void);
const char* moe_profile_kernel_name(int id);
int moe_profile_query(int id, double* total_ms, int64_t* launches);

#ifdef __cplusplus
}
#endif
#endif /* MOE_MI355X_H */
