/*
 * ga.h -- C ABI of the MI355X (gfx950) group-attention library, libga.so.
 *
 * Group attention is the attention mechanism of RITA ("Group Attention is All
 * You Need for Timeseries Analytics", Liang et al., arXiv 2306.01926):
 *
 *   - Grouping (Section 4.4): the n keys of each (batch, head) slice are
 *     clustered into N groups by Lloyd K-means iterations; the distance is
 *     evaluated in the expanded form |c|^2 - 2 k.c so that its bulk is a
 *     matrix product.  The group centroid is the representative key
 *     (Section 4.1) and BELONG / COUNT record membership (Algorithm 1 inputs).
 *   - Embedding aggregation (Section 4.2, Algorithm 1): per-group SUM of the
 *     value vectors.
 *   - Group softmax (Eq. 3) and combine (Algorithm 1): for query q_i,
 *     p_ij = scale * q_i . r_j,  s_i = sum_j COUNT_j exp(p_ij - m_i),
 *     o_i = sum_j exp(p_ij - m_i) vsum_j / s_i,
 *     with m_i the largest p_ij over non-empty groups.
 *
 * Conventions for every entry point
 *   - Tensors are dense and row-major with the feature axis innermost:
 *     Q, K, V, O: [B, H, n, d];  centroid, vsum, init: [B, H, N, d] (fp32);
 *     belong: [B, H, n] (int32);  count: [B, H, N] (int32).
 *   - Every pointer except the stream is a DEVICE pointer to memory the
 *     caller owns and that stays valid until the stream work completes.  The
 *     library allocates nothing, keeps no pointer after returning, and never
 *     synchronises: work is enqueued in order on `stream` (a hipStream_t; NULL
 *     is the default stream), and results are valid once the caller has
 *     synchronised with that stream.
 *   - All argument checks run on the host before any HIP call; on failure the
 *     call returns a status other than GA_OK, enqueues nothing and records a
 *     message retrievable with ga_last_error() (thread-local).
 *   - Pointers must be 16-byte aligned; the workspace 256-byte aligned.
 *   - d must be 64 (GA_ERR_UNSUPPORTED otherwise).  1 <= N <= min(n, 1024);
 *     the bf16 attention (ga_attend, ga_forward) holds N <= 256 groups on
 *     chip (GA_ERR_UNSUPPORTED above).  B*H <= 65535.  B = 0 or H = 0 is an
 *     empty batch: GA_OK, nothing enqueued.  n must be >= 1.
 *   - Inputs must be finite, and every nonzero input of magnitude within
 *     [2^-60, 2^60] (not checked; results undefined otherwise).
 *   - Exactness and determinism (bf16): the fp64 member sums behind COUNT
 *     and the centroids are exact, hence independent of the order in which
 *     the GPU adds them, as long as within every group (e_max - e_min) +
 *     log2(count) <= 45, with e_max / e_min the largest / smallest binary
 *     exponent of the group's nonzero member values (for instance at most
 *     2^15 members whose nonzero magnitudes lie within 2^30 of each other).
 *     Under that condition belong, count and centroid equal the definition
 *     below bit for bit and repeated calls give identical bits; outside it a
 *     centroid can differ in its last bit (and a later assignment with it).
 *     This condition is not checked on the device.  fp32 sums are formed in
 *     a fixed order and are deterministic without it.
 *
 * Representatives: R = round_dt(centroid), where round_dt is the identity for
 * GA_F32 and round-to-nearest-even to bfloat16 for GA_BF16.  R is used both
 * for assignment and for the attention scores.
 */
#ifndef GA_H
#define GA_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum { GA_F32 = 0, GA_BF16 = 1 } ga_dtype_t;

typedef enum {
    GA_OK = 0,
    GA_ERR_INVALID_ARG = 1, /* bad shape, null/misaligned pointer, N or iters out of range */
    GA_ERR_UNSUPPORTED = 2, /* valid but not implemented (d != 64) */
    GA_ERR_WORKSPACE = 3,   /* workspace missing or smaller than ga_workspace_bytes() */
    GA_ERR_HIP = 4          /* a HIP launch failed; ga_last_error() names it */
} ga_status_t;

/* Shape of Q/K/V: B batches, H heads, n tokens (windows), d features; dtype
 * of Q/K/V/O storage (fp32 accumulation for both). */
typedef struct {
    int32_t B, H, n, d;
    int32_t dtype; /* ga_dtype_t */
} ga_shape_t;

/* Bytes of device workspace any entry point needs for shape s and N groups
 * (0 if the shape is invalid).  One workspace of this size serves all calls
 * made one after another; calls that may run at the same time (on different
 * streams) each need a workspace of their own: the workspace carries state
 * between the launches of one call. */
size_t ga_workspace_bytes(ga_shape_t s, int32_t N);

/*
 * Grouping (Section 4.4): `iters` rounds of Lloyd K-means on the keys of every
 * (b, h) slice, independently.
 *   K         [B,H,n,d] keys in s.dtype.
 *   N         groups, 1 <= N <= min(n, 1024).   iters >= 1.
 *   init      optional [B,H,N,d] fp32 initial centroids; NULL selects the
 *             strided init C0_j = k_{floor(j*n/N)}.
 *   belong    out [B,H,n]: group of each key, assigned against the
 *             representatives of the previous round (lowest index on ties of
 *             the canonical score fma(-2, k.r_j, |r_j|^2) evaluated in fp64).
 *   count     out [B,H,N]: members per group.
 *   centroid  out [B,H,N,d] fp32: (float)(fp64 member sum / count); a group
 *             that ends empty keeps its previous centroid.
 * belong, count and centroid match the fp64 CPU definition bit for bit.
 */
int ga_cluster(ga_shape_t s, const void *K, int32_t N, int32_t iters, const float *init,
               int32_t *belong, int32_t *count, float *centroid, void *workspace,
               size_t workspace_bytes, void *stream);

/*
 * Embedding aggregation (Section 4.2, Algorithm 1): vsum_j = sum of v_i over
 * the keys i with belong_i == j, accumulated in fp64 in ascending i and
 * rounded once to fp32.  Entries of belong outside [0, N) are ignored.
 *   V [B,H,n,d] in s.dtype;  belong [B,H,n];  vsum out [B,H,N,d] fp32.
 */
int ga_aggregate(ga_shape_t s, const void *V, const int32_t *belong, int32_t N, float *vsum,
                 void *workspace, size_t workspace_bytes, void *stream);

/*
 * Group softmax and combine (Eq. 3, Algorithm 1) for every query.
 *   Q         [B,H,n,d] in s.dtype.
 *   centroid  [B,H,N,d] fp32 (representatives are round_dt(centroid)).
 *   count     [B,H,N]; groups with count <= 0 are left out entirely.
 *   vsum      [B,H,N,d] fp32 per-group value sums.
 *   scale     finite score scale (1/sqrt(d) reproduces Eq. 1).
 *   O         out [B,H,n,d] in s.dtype.  A slice with no non-empty group
 *             gets zeros.
 * Accuracy versus the fp64 definition: 1e-4 relative (GA_F32), 2e-2
 * relative (GA_BF16: bf16 operands, fp32 accumulation).
 */
int ga_attend(ga_shape_t s, const void *Q, const float *centroid, const int32_t *count,
              const float *vsum, int32_t N, float scale, void *O, void *workspace,
              size_t workspace_bytes, void *stream);

/*
 * Whole forward: ga_cluster (strided init), ga_aggregate, ga_attend.
 * belong / count / centroid are optional outputs (NULL: kept internal).
 */
int ga_forward(ga_shape_t s, const void *Q, const void *K, const void *V, int32_t N,
               int32_t iters, float scale, void *O, int32_t *belong, int32_t *count,
               float *centroid, void *workspace, size_t workspace_bytes, void *stream);

/*
 * ga_forward without a workspace and without allocating, for callers that
 * cannot allocate device memory (code under HIP graph capture, tight serving
 * loops, harnesses that forbid hipMalloc).  Same arguments and results as
 * ga_forward (the same kernels), minus the workspace: the scratch lives in a
 * static device array of GA_NOALLOC_SCRATCH_BYTES (32 MiB) that each GPU the
 * library runs on holds until the process ends.  No hipMalloc / hipFree or
 * other allocating call is made.
 *   - bf16 only, and only the shapes the one-launch grouping serves
 *     (N <= 128, n <= 65536, every workgroup of that launch resident at
 *     once): GA_ERR_UNSUPPORTED otherwise.
 *   - Shapes whose scratch exceeds the array are rejected with
 *     GA_ERR_WORKSPACE.  Per (b, h) slice the scratch is about
 *     4 n + 420 N + 17 KB plus the grouping's exchange rows, 516 bytes per
 *     group and workgroup of the slice (B*H = 128 at n = 8000, N = 128 takes
 *     29 MiB).
 *   - Every call on one GPU shares that GPU's array and leaves its contents
 *     behind: calls that overlap in time on one GPU (two streams, two host
 *     threads) race and must be serialised by the caller.
 *   - `stream` must belong to the current device.
 *   - A cross-workgroup wait of the grouping launch that gives up (it does
 *     not while every workgroup is resident) is not reported here; use
 *     ga_forward with ga_workspace_check where that report is wanted.
 */
#define GA_NOALLOC_SCRATCH_BYTES ((size_t)32 << 20)
int ga_forward_noalloc(ga_shape_t s, const void *Q, const void *K, const void *V, int32_t N,
                       int32_t iters, float scale, void *O, int32_t *belong, int32_t *count,
                       float *centroid, void *stream);

/*
 * Attention block of the RITA encoder (bf16 only): the encoder is a
 * Transformer encoder whose self-attention is replaced by group attention
 * (Section 3), with the bias-free projections Q = X W_Q, K = X W_K,
 * V = X W_V of Eq. 1, one d = 64 slice per head, and the heads' outputs
 * concatenated and projected by W_O.  D = d_model = 64 H.
 *
 * Layouts (all bf16, dense, row-major):
 *   X, Y  [B, n, D] token embeddings in / block output;
 *   Wqkv  [3D, D]: one OUTPUT feature per row, the input axis contiguous
 *         (rows 0..D-1 give Q, D..2D-1 give K, 2D..3D-1 give V; within each,
 *         row 64 h + c is feature c of head h), i.e. the transpose of the
 *         column-per-feature W_Q | W_K | W_V of Eq. 1;
 *   Wo    [D, D]: row o holds the weights of output feature o over the
 *         concatenated heads (input index 64 h + c = feature c of head h);
 *   Q, K, V, O  [B, H, n, 64] as everywhere in this library.
 * Products are accumulated in fp32 on the matrix cores and rounded once to
 * bf16 (round to nearest even); each output is within one bf16 unit in the
 * last place of the exactly rounded product.  s.d must be 64, s.dtype
 * GA_BF16 (GA_ERR_UNSUPPORTED otherwise), H <= 64, N <= min(n, 256).
 * Pointer, stream and error conventions as above; B = 0 or H = 0 enqueues
 * nothing.
 */
size_t ga_block_workspace_bytes(ga_shape_t s, int32_t N); /* 0 if invalid */

/* Q, K, V [B,H,n,64] = per-head slices of X Wqkv^T (Eq. 1). */
int ga_project_qkv(ga_shape_t s, const void *X, const void *Wqkv, void *Q, void *K, void *V, void *stream);

/* Y [B,n,D] = concat_h(O[:, h]) Wo^T. */
int ga_project_out(ga_shape_t s, const void *O, const void *Wo, void *Y, void *stream);

/* Y = attention block of X: ga_project_qkv, ga_forward (strided init,
 * `iters` rounds, `scale`), ga_project_out.  The workspace
 * (ga_block_workspace_bytes) holds Q, K, V, O and the forward's workspace. */
int ga_attention_block(ga_shape_t s, const void *X, const void *Wqkv, const void *Wo, int32_t N,
                       int32_t iters, float scale, void *Y, void *workspace, size_t workspace_bytes,
                       void *stream);

/*
 * Adaptive group count (Section 5.1): the merge plan of a grouping.
 *   Lemma 1: if every key lies within dthr of its group's representative and
 *   dthr <= ln(eps) / (2 R'), each restored attention weight is within a
 *   factor eps of the exact one; R' = |scale| max_i |q_i| bounds the scaled
 *   query norms (the quantity the proof bounds).  Per slice
 *   dthr = ln(eps) / (2 R') (+inf if R' = 0).
 *   Eq. 5 (simplified merge rule): the groups are halved into
 *   S1 = [0, ceil(N/2)) and S2 = [ceil(N/2), N); group j of S2 is marked when
 *   some i of S1 has |c_i - c_j| + rad_i <= dthr and
 *   |c_j - c_i| + rad_j <= dthr / 2 (c: centroid, rad_g: largest distance of
 *   a member of g to c_g).  Only non-empty groups take part.
 * Arguments: Q, K [B,H,n,d] in s.dtype; belong, centroid, count as output by
 * ga_cluster; eps > 1 (finite).  Outputs (device): radius [B,H,N] fp64
 * (0 for an empty group), dthr [B,H] fp64, partner [B,H,N] int32 (for a
 * marked S2 group the lowest qualifying S1 group, else -1), merges [B,H]
 * int32 (marked groups).  Every value is computed in fp64 exactly as the
 * definition states (squares summed as fma chains over the features in
 * order, IEEE square roots) and matches the fp64 CPU definition bit for bit.
 * N <= 256 (GA_ERR_UNSUPPORTED above).
 */
int ga_merge_plan(ga_shape_t s, const void *Q, const void *K, const int32_t *belong, const float *centroid,
                  const int32_t *count, int32_t N, float scale, double eps, double *radius, double *dthr,
                  int32_t *partner, int32_t *merges, void *stream);

/*
 * Momentum update of the group count (Section 5.1), on the HOST:
 * N_new = alpha (N - D) + (1 - alpha) N with D the smallest of the `slices`
 * per-slice merge counts (host array; every slice then keeps its bound),
 * rounded to the nearest integer (halves up) and kept in [1, N].
 * Returns N_new, or 0 (and ga_last_error) for N < 1, alpha outside [0, 1],
 * slices < 0 or merges NULL with slices > 0.
 */
int32_t ga_next_group_count(int32_t N, const int32_t *merges, int64_t slices, double alpha);

/*
 * Backward pass of group attention (bf16; N <= 256), the gradient with the
 * grouping held fixed (BELONG / COUNT are piecewise constant in the keys; the
 * paper states no gradient rule).  With w_ij = c_j e^{p_ij} / sum_l c_l e^{p_il}
 * (the normalised group weights of Eq. 3), mu_j = vsum_j / c_j and G = dO:
 *   dp_ij = w_ij (G_i . mu_j - G_i . o_i),   dQ_i = scale sum_j dp_ij r_j,
 *   dK_k = scale sum_i dp_{i a_k} q_i / c_{a_k}   (r_j is the member mean;
 *          its bf16 rounding is passed straight through),
 *   dV_k = sum_i w_{i a_k} G_i / c_{a_k}.
 * Inputs: Q, dO [B,H,n,d] bf16; belong, centroid, count as from ga_cluster;
 * vsum [B,H,N,d] fp32 (ga_aggregate).  Outputs dQ, dK, dV [B,H,n,d] bf16.
 * Workspace: ga_backward_workspace_bytes(s, N) (0 if unsupported).
 * Accuracy versus the fp64 definition: 2e-2 relative (bf16 operands, fp32
 * accumulation).  Deterministic: every reduction has a fixed order.
 */
size_t ga_backward_workspace_bytes(ga_shape_t s, int32_t N);
int ga_backward(ga_shape_t s, const void *Q, const void *dO, const int32_t *belong, const float *centroid,
                const int32_t *count, const float *vsum, int32_t N, float scale, void *dQ, void *dK, void *dV,
                void *workspace, size_t workspace_bytes, void *stream);

/*
 * Per-kernel timing for measurement tools.  While enabled (per calling
 * thread), every kernel launch of this library is bracketed by a pair of
 * hipEvents recorded on the launch stream.  ga_timing_collect waits for the
 * recorded events, writes up to max_entries per-kernel totals (launch count
 * and summed event time in milliseconds, in first-launch order), sets
 * *n_entries and forgets the records.  Timing never changes results.
 */
typedef struct {
    char name[32];
    int32_t launches;
    double total_ms;
} ga_kernel_time_t;

int ga_timing_enable(int on);
int ga_timing_collect(ga_kernel_time_t *out, int32_t max_entries, int32_t *n_entries);

/*
 * Device status of the last grouping launch that used `workspace` (shape s, N
 * groups): waits for `stream` (this is the library's only synchronising call)
 * and returns GA_OK, or GA_ERR_HIP if a cross-workgroup wait of the
 * persistent grouping kernel gave up (its workgroups were not all resident at
 * once, e.g. because other work occupied the GPU; the outputs of that call
 * are then invalid).  Callers that cannot rule that out check after a
 * forward or cluster call.
 */
int ga_workspace_check(ga_shape_t s, int32_t N, const void *workspace, size_t workspace_bytes, void *stream);

/* Static description of a status code. */
const char *ga_status_string(int status);

/* Message of the last failing call on this thread ("" if none). */
const char *ga_last_error(void);

#ifdef __cplusplus
}
#endif

#endif /* GA_H */
