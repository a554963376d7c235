/*
 * na.h -- C ABI of the fused neighborhood-attention (NA) library for MI355X
 * (gfx950).  Shared object: paper_2403_04690_amd/libna.so.
 *
 * Operation (Faster Neighborhood Attention, arXiv 2403.04690):
 *   Each query token of a rank-r token space (r = 1, 2, 3) attends to its
 *   k_a nearest same-group tokens along every axis a (Sec. 1, caption of Fig.
 *   "neighborhoodattention", Sec. 2).  The window is centred on the query
 *   where possible and shifted, never truncated, at borders, so each query has
 *   exactly prod_a k_a neighbours.  Dilation d_a splits axis a into the d_a
 *   sub-lattices x = g (mod d_a), each an independent non-dilated problem
 *   (Sec. 3.4).  Inside a group of n tokens, the window of position p starts
 *   at clamp(p - floor(k/2), 0, n - k).
 *   Causal masking per axis (Sec. 3.4; caption of Fig. "neighborhoodattention"):
 *   along a causal axis a query never attends to a token of larger
 *   coordinate; its window there is the k nearest same-group positions not
 *   after it, [max(0, p - k + 1), p], so the first k - 1 positions of each
 *   group have shorter windows (e.g. 3-D attention with causal time).
 *   The attention itself is Eq. 1 restricted to that neighbourhood, computed
 *   fused (Sec. 3.3, Fig. "fna-vis"): scores, mask, online softmax and the
 *   product with V in one kernel; no attention weights reach global memory.
 *
 * Conventions shared by every entry point:
 *   - q, k, v, out, dout, dq, dk, dv: contiguous [B, H, X_1 .. X_r, D] arrays
 *     of `dtype` in device memory, axis X_1 outermost (3-D is T, H, W).
 *   - logsumexp: contiguous [B, H, X_1 .. X_r] fp32 in device memory, natural
 *     log, scale included: lse = log sum_j exp(scale * q.k_j).
 *   - Every device pointer must be 16-byte aligned.
 *   - The caller owns all memory; the library never allocates or frees
 *     device memory and needs no workspace.  Its only global state is the
 *     tiling cache that na_tune (or tuning on first use) fills, guarded by a
 *     mutex, and the tune-on-first-use mode; every entry point is re-entrant.
 *   - Calls are asynchronous and stream-ordered on `stream` (a hipStream_t;
 *     NULL means the legacy default stream).  Problem validation is
 *     synchronous and happens before any launch: a non-NA_OK status means
 *     nothing was launched.  NA_ERR_HIP reports a failed launch.
 *   - causal: NULL (no causal axis) or rank int32 flags, outermost axis first;
 *     nonzero marks a causal axis.
 *   - B * H * N == 0 (empty batch or heads) is a no-op returning NA_OK.
 *   - Supported: rank 1..3, head_dim in {32, 64, 128}, any k_a >= 1 and
 *     d_a >= 1 with k_a * d_a <= X_a, fp32 / fp16 / bf16.  N * D must stay
 *     below 2^31 and B * H below 2^31, and a launch must stay below 2^32
 *     threads: nwg * 64 * (waves per workgroup) for the forward and
 *     (nwg + nwg rounded up to a multiple of 8) * 256 for the backward, nwg
 *     being the number of query tiles over every (batch, head, dilation
 *     group); for 1-D problems of at most 64 tokens per group that means
 *     B * H * prod(d) < 2^23.  Larger problems are rejected with NA_ERR_SHAPE
 *     before any launch (na_validate checks the heuristic tilings, the
 *     tiled entry points their own).
 */
#ifndef NA_H_
#define NA_H_

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

/* Same type as hipStream_t (struct ihipStream_t*). */
struct ihipStream_t;
typedef struct ihipStream_t* na_stream_t;

typedef enum { NA_FP32 = 0, NA_FP16 = 1, NA_BF16 = 2 } na_dtype;

typedef enum {
    NA_OK = 0,
    NA_ERR_NULL = 1,                  /* a required pointer is NULL */
    NA_ERR_RANK = 2,                  /* rank not in 1..3 */
    NA_ERR_SHAPE = 3,                 /* extent < 1, batch/heads < 0, or size limits exceeded */
    NA_ERR_KERNEL_SIZE = 4,           /* kernel_size[a] < 1 */
    NA_ERR_DILATION = 5,              /* dilation[a] < 1 */
    NA_ERR_WINDOW_EXCEEDS_EXTENT = 6, /* kernel_size[a] * dilation[a] > extents[a] */
    NA_ERR_HEAD_DIM = 7,              /* head_dim not in {32, 64, 128} */
    NA_ERR_DTYPE = 8,                 /* dtype not an na_dtype value */
    NA_ERR_ALIGNMENT = 9,             /* a device pointer is not 16-byte aligned */
    /* 10 is not used */
    NA_ERR_HIP = 11,                  /* a HIP launch or query failed */
    NA_ERR_SCALE = 12,                /* scale is not finite */
    NA_ERR_TILING = 13                /* an explicit tiling is not valid for the problem */
} na_status;

/*
 * How a launch cuts the problem into work (query tiles for the forward and
 * the dQ role, key tiles for the dK/dV role; multi-axis tiles as in the
 * paper's fused kernels, Sec. 3.3 and App. A):
 *   blocks_per_wave: 16-token blocks per wave, 1 or 2;
 *   wave_tile[a]:    tokens per wave along axis a (group coordinates), powers
 *                    of two whose product over the problem's axes is
 *                    16 * blocks_per_wave;
 *   waves[a]:        waves per workgroup along axis a, powers of two whose
 *                    product is 4 (8 is also allowed along the only axis of a
 *                    1-D forward of fp16 / bf16).
 * Entries for axes beyond the rank must be 1.  A workgroup tile is
 * wave_tile[a] * waves[a] tokens along axis a.
 */
typedef struct {
    int32_t blocks_per_wave;
    int32_t wave_tile[3];
    int32_t waves[3];
} na_tiling;

/* Human-readable text for a status code (static storage, never NULL). */
const char* na_status_string(na_status status);

/* Library version as major * 10000 + minor * 100 + patch. */
int na_version(void);

/*
 * Host-only check of the problem description used by every entry point
 * (rank, extents, kernel_size, dilation, causal, batch, heads, head_dim,
 * dtype, scale).  Touches no device and no pointer other than the arrays.
 * The paper leaves the legal parameters implicit: a window is never
 * truncated (Sec. 1-2, caption of Fig. "neighborhoodattention"), and a
 * dilated window lives in one sub-lattice of an axis (Sec. 3.4), so each axis
 * needs k_a * d_a <= X_a (NA_ERR_WINDOW_EXCEEDS_EXTENT otherwise); the
 * softmax scale of Eq. 1 must be finite.  Returns NA_OK or the status of
 * the first check that fails.
 */
na_status na_validate(int rank, const int64_t* extents, const int32_t* kernel_size,
                      const int32_t* dilation, const int32_t* causal, int64_t batch, int64_t heads,
                      int64_t head_dim, na_dtype dtype, float scale);

/*
 * Fused NA forward (Sec. 3.3): out = softmax(scale * q k^T restricted to each
 * query's neighbourhood) v, and logsumexp per query (kept for the backward,
 * which recomputes the probabilities from it instead of storing them).
 *   extents[rank], kernel_size[rank], dilation[rank], causal[rank] (or NULL):
 *   per axis, outermost first.
 *   scale: softmax scale (1/sqrt(head_dim) in Eq. 1; any finite value).
 */
na_status na_forward(int rank, const int64_t* extents, const int32_t* kernel_size,
                     const int32_t* dilation, const int32_t* causal, int64_t batch, int64_t heads,
                     int64_t head_dim, na_dtype dtype, float scale, const void* q, const void* k,
                     const void* v, void* out, float* logsumexp, na_stream_t stream);

/*
 * Fused NA backward: gradients of out with respect to q, k and v given
 * dout, from the saved out and logsumexp of na_forward on the same inputs.
 * Built from the operators of Sec. 3.1: dP = PN(dO, V), dA = P * (dP - Delta),
 * dQ = scale * NN(dA, K) over each query's neighbourhood, and dK = scale *
 * IN(dA, Q), dV = IN(P, dO) over each key's inverse neighbourhood.
 *   Delta = rowsum(dO * O) is formed inside the kernels, so no workspace is
 *   needed (for large 3-D problems a first launch writes -Delta into dq,
 *   which later launches of the same call read and then overwrite).  dq, dk,
 *   dv are fully overwritten and must not alias the inputs or each other.
 *   Deterministic: the same inputs give bit-identical gradients.
 */
na_status na_backward(int rank, const int64_t* extents, const int32_t* kernel_size,
                      const int32_t* dilation, const int32_t* causal, int64_t batch, int64_t heads,
                      int64_t head_dim, na_dtype dtype, float scale, const void* q, const void* k,
                      const void* v, const void* out, const float* logsumexp, const void* dout,
                      void* dq, void* dk, void* dv, na_stream_t stream);

/*
 * Tilings (see na_tiling).  The plain entry points above use the tiling
 * cached for the problem by na_tune, else a heuristic one.  The problem key
 * of the cache is (rank, extents, kernel_size, dilation, causal, batch * heads,
 * head_dim, dtype); the scale does not matter.
 *
 * na_candidate_tilings (host only): writes up to `max` of the candidate
 * tilings for the forward (forward != 0) or the backward of the problem, the
 * heuristic one first, and returns how many candidates there are in all (so
 * a return value above `max` means the list was cut; out may be NULL to count
 * them), or a negative na_status for an invalid problem.  na_tune times the
 * first NA_TUNE_DEFAULT_CANDIDATES of them, or all with NA_TUNE_THOROUGH.
 *
 * na_current_tiling (host only): the tiling na_forward (forward != 0) or
 * na_backward would use now for the problem.
 *
 * na_forward_tiled / na_backward_tiled: na_forward / na_backward with an
 * explicit tiling, which is validated first (NA_ERR_TILING, nothing launched).
 * Every valid tiling gives the same result up to summation order.
 *
 * na_tune (auto-tuner over the query-tile factorisations, App. A): after a
 * warm-up, times the candidate tilings of the forward and, separately, of the
 * backward (the first NA_TUNE_DEFAULT_CANDIDATES, or every one when flags has
 * NA_TUNE_THOROUGH), each over `repeats` launches (>= 1) after one warm-up
 * launch, then times the three fastest and the heuristic tiling again in five
 * interleaved rounds; the heuristic one is kept unless a finalist's median
 * beats it by more than 2 %.  Runs on
 * the caller's buffers, which end up holding the results of the chosen
 * tilings (out and logsumexp of the forward of q, k, v; dq, dk, dv of the
 * backward with dout).  Records the chosen forward and backward tilings in
 * the cache.  Synchronises `stream`; must not run concurrently with other
 * work on these buffers.  Unknown flags give NA_ERR_TILING.  Optional outputs
 * (NULL to skip): best_forward, best_backward, and times_ms[4] = {best
 * forward, best backward, heuristic forward, heuristic backward} in
 * milliseconds per launch.
 *
 * na_tune_clear: empties the cache, and drops every plan (below).
 *
 * Plans: na_forward and na_backward keep, per calling thread, the last few
 * problems they validated with the tiling and launch geometry chosen for each,
 * and launch a repeated problem from its plan (checking only the scale and the
 * pointers).  Recording a tuned tiling, na_tune_clear and na_set_autotune
 * retire every plan.  The forcing variables NA_WAVE_BLOCKS=1|2 (blocks per
 * wave), NA_FWD_WAVES=4|8 (1-D forward workgroup size) and NA_BWD_SPLIT=0|1
 * (backward form) are read when a plan is made: after changing one, call
 * na_tune_clear for it to take effect on problems already planned.
 *
 * na_set_autotune (tune on first use, App. A): mode 1 makes na_forward and
 * na_backward tune a problem whose tiling is not cached yet (forward and
 * backward each by its own timing, as na_tune does, with 3 launches per
 * candidate) on the call's own buffers, record the choice and return its
 * result; mode 2 does the same over every candidate (NA_TUNE_THOROUGH); 0
 * turns it off.  Such a first call synchronises its stream and takes as long
 * as timing every candidate; later calls on the problem run the cached
 * tiling.  A call on a stream that is being captured into a graph never
 * tunes.  The initial mode comes from the environment variable NA_AUTOTUNE
 * (0, 1 or 2; unset: 0).  na_autotune returns the mode in force.
 */
#define NA_TUNE_THOROUGH 1
#define NA_TUNE_DEFAULT_CANDIDATES 64
int na_candidate_tilings(int rank, const int64_t* extents, const int32_t* kernel_size,
                         const int32_t* dilation, int64_t batch, int64_t heads, int64_t head_dim,
                         na_dtype dtype, int forward, na_tiling* out, int max);
na_status na_current_tiling(int rank, const int64_t* extents, const int32_t* kernel_size,
                            const int32_t* dilation, const int32_t* causal, int64_t batch,
                            int64_t heads, int64_t head_dim, na_dtype dtype, int forward,
                            na_tiling* out);
na_status na_forward_tiled(int rank, const int64_t* extents, const int32_t* kernel_size,
                           const int32_t* dilation, const int32_t* causal, int64_t batch,
                           int64_t heads, int64_t head_dim, na_dtype dtype, float scale,
                           const na_tiling* tiling, const void* q, const void* k, const void* v,
                           void* out, float* logsumexp, na_stream_t stream);
na_status na_backward_tiled(int rank, const int64_t* extents, const int32_t* kernel_size,
                            const int32_t* dilation, const int32_t* causal, int64_t batch,
                            int64_t heads, int64_t head_dim, na_dtype dtype, float scale,
                            const na_tiling* tiling, const void* q, const void* k, const void* v,
                            const void* out, const float* logsumexp, const void* dout, void* dq,
                            void* dk, void* dv, na_stream_t stream);
na_status na_tune(int rank, const int64_t* extents, const int32_t* kernel_size,
                  const int32_t* dilation, const int32_t* causal, int64_t batch, int64_t heads,
                  int64_t head_dim, na_dtype dtype, float scale, const void* q, const void* k,
                  const void* v, void* out, float* logsumexp, const void* dout, void* dq, void* dk,
                  void* dv, int repeats, int flags, na_stream_t stream, na_tiling* best_forward,
                  na_tiling* best_backward, float* times_ms);
void na_tune_clear(void);
void na_set_autotune(int mode);
int na_autotune(void);

/*
 * Test hook: evaluates on the device, with the same index functions the
 * kernels use, the per-axis neighbourhood summary of the problem: the window
 * of each query coordinate (Sec. 1-2 and the caption of Fig.
 * "neighborhoodattention": k nearest same-group neighbours, shifted at
 * borders; Sec. 3.4: dilation groups and causal axes) and the inverse
 * neighbourhood of each key coordinate (the queries attending to it, which
 * the IN operator of Sec. 3.1 sums over).  Each output is a device int32
 * array of sum_a extents[a] entries, axis 0 first:
 *   start[x]  = first (smallest) neighbour coordinate of query coordinate x,
 *   inv_lo[j] = smallest query coordinate whose window contains key j,
 *   inv_hi[j] = largest query coordinate whose window contains key j.
 * Only the problem arguments are validated (batch, heads, head_dim and dtype
 * play no part).  Asynchronous on `stream`.
 */
na_status na_debug_windows(int rank, const int64_t* extents, const int32_t* kernel_size,
                           const int32_t* dilation, const int32_t* causal, int32_t* start,
                           int32_t* inv_lo, int32_t* inv_hi, na_stream_t stream);

/*
 * Unfused operators: the baseline the fused kernels are measured against.
 * The paper builds NA from separate operators (Sec. 3.1) that each read or
 * write the l-wide attention weights (l = prod_a kernel_size[a] per query) in
 * global memory; its naive and GEMM-based kernels (Sec. 3.1-3.2, Tables
 * "runtime_breakdown" and "runtime_breakdown_backward") work that way.  These
 * entry points are that design on this GPU, one launch per operator:
 *   forward   W = PN(q, k) * scale;  P = softmax(W);  out = NN(P, v)
 *   backward  dP = PN(dout, v);  dA = softmax_backward(P, dP);
 *             dq = NN(dA, k) * scale;  dk = IN(dA, q) * scale;  dv = IN(P, dout)
 * They give the same results as na_forward / na_backward up to rounding (the
 * weights are stored in the inputs' type), but move l-wide rows through
 * memory instead of keeping them in registers.
 *
 * Weights: contiguous [B, H, N, l] arrays of `dtype` (N = prod extents), row
 * i holding query i's neighbours in the row-major order of the per-axis
 * window offsets t_a (axis 0 outermost): entry e = sum_a t_a prod_{b>a} k_b
 * is the token whose coordinate along axis a is g_a + d_a (s_a + t_a), s_a
 * being the start of the query's window in its dilation group g_a.  Along a
 * causal axis the window of group position p has min(k_a, p + 1) positions;
 * entries of offsets beyond them are not neighbours (PN writes -inf, the
 * softmax 0, the others ignore them).  The caller allocates the weights
 * (B * H * N * l elements).
 *
 * Problem arguments and conventions as for na_forward (head_dim and dtype
 * describe a, b, out and the weights; scale multiplies the result of PN, NN
 * and IN).  All pointers 16-byte aligned; the weights are overwritten in
 * place by na_unfused_softmax (probabilities, and the natural-log logsumexp
 * per row in logsumexp [B, H, N] fp32) and by na_unfused_softmax_backward
 * (grad: in dP, out dA = P * (dP - sum_e P dP) per row).  Errors as for
 * na_forward; NA_ERR_SHAPE also when the weight tensor would exceed 2^62
 * elements or a row 2^31 - 1.
 *
 * na_unfused_pn:  weights[i, e] = scale * a_i . b_j(i,e)   (PN; a, b [B, H, N, D])
 * na_unfused_nn:  out_i = scale * sum_e weights[i, e] b_j(i,e)   (NN)
 * na_unfused_in:  out_j = scale * sum over the queries i whose window holds j
 *                 of weights[i, e(i, j)] b_i   (IN, the inverse neighbourhood)
 */
na_status na_unfused_pn(int rank, const int64_t* extents, const int32_t* kernel_size,
                        const int32_t* dilation, const int32_t* causal, int64_t batch,
                        int64_t heads, int64_t head_dim, na_dtype dtype, float scale,
                        const void* a, const void* b, void* weights, na_stream_t stream);
na_status na_unfused_softmax(int rank, const int64_t* extents, const int32_t* kernel_size,
                             const int32_t* dilation, const int32_t* causal, int64_t batch,
                             int64_t heads, int64_t head_dim, na_dtype dtype, void* weights,
                             float* logsumexp, na_stream_t stream);
na_status na_unfused_nn(int rank, const int64_t* extents, const int32_t* kernel_size,
                        const int32_t* dilation, const int32_t* causal, int64_t batch,
                        int64_t heads, int64_t head_dim, na_dtype dtype, float scale,
                        const void* weights, const void* b, void* out, na_stream_t stream);
na_status na_unfused_in(int rank, const int64_t* extents, const int32_t* kernel_size,
                        const int32_t* dilation, const int32_t* causal, int64_t batch,
                        int64_t heads, int64_t head_dim, na_dtype dtype, float scale,
                        const void* weights, const void* b, void* out, na_stream_t stream);
na_status na_unfused_softmax_backward(int rank, const int64_t* extents,
                                      const int32_t* kernel_size, const int32_t* dilation,
                                      const int32_t* causal, int64_t batch, int64_t heads,
                                      int64_t head_dim, na_dtype dtype, const void* probs,
                                      void* grad, na_stream_t stream);

#ifdef __cplusplus
}
#endif

#endif /* NA_H_ */
