/*
 * dpghost.h -- per-example gradient norms by ghost clipping, clip factors,
 * the clipped gradient sum and Gaussian noise for DP-SGD on decoder-only
 * transformers, on one AMD Instinct MI355X (gfx950).
 *
 * Method: El Mais, Chehab, Issa, Tajeddine, "Is Weight Tying Still Beneficial
 * for Decoder-Only LLMs in Private Settings Under DP-SGD?" (arXiv 2609.40335).
 * Section and equation numbers below refer to that paper.
 *
 * Conventions for every entry point
 *  - Tensor pointers are DEVICE pointers, row-major. A token-major matrix
 *    [B, T, w] with row stride ld (elements, ld >= w) holds token t of
 *    example b at row b*T + t. bf16 data is passed as its 16-bit patterns.
 *  - A matrix given with row stride ld > its width occupies ld elements in
 *    every row, the last one included (as a [rows, ld] buffer viewed to
 *    fewer columns does). When its rows are 16-byte aligned and ld is a
 *    whole number of 16-byte chunks, kernels may read, but never use, the
 *    elements between the width and the next 16-byte boundary of a row.
 *  - Outputs are fp32. Squared norms add across calls ("accumulate" = 1
 *    means +=, 0 means overwrite), which is eq. 6 / eq. 10.
 *  - `stream` is a hipStream_t (NULL = the default stream). Calls are
 *    asynchronous and stream-ordered; nothing synchronises the device.
 *  - Ownership: the caller allocates and owns every buffer. The library
 *    allocates no device memory. Entry points that need scratch take a
 *    caller-owned device `workspace` of at least the size returned by their
 *    *_workspace() function; its contents need no initialisation and are
 *    dead after the call's kernels finish. Two calls in flight at once must
 *    not share a workspace.
 *  - Operands are addressed with 32-bit byte offsets: every operand matrix
 *    (rows x row stride x element size) must span less than 4 GiB, else
 *    DP_EUNSUPPORTED.
 *  - Errors: arguments are validated on the host before any HIP call. A
 *    NULL required pointer, a non-positive size, a stride smaller than its
 *    row width, an unknown dtype or a too-small workspace returns DP_EINVAL;
 *    a size beyond a documented limit returns DP_EUNSUPPORTED; a failed
 *    kernel launch returns DP_EHIP. dp_last_error() describes the last
 *    failure on the calling thread. Exceptions never cross this interface.
 *  - Token ids outside [0, V) are a caller error; kernels never read or
 *    write out of bounds for them (they contribute nothing to cross terms or
 *    sums), but the results are then meaningless.
 *  - Thread safety: the functions keep no state between calls.
 */
#ifndef DPGHOST_H
#define DPGHOST_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#define DP_ABI_VERSION 3

/* Enumerations are int-sized in both languages. Compiled as C++ they have
 * int as their fixed underlying type, so that every int a C caller passes
 * (an unknown dtype, say, which the entry points reject) is a value of the
 * type: C++ leaves values outside an unfixed enumeration's range undefined. */
#ifdef __cplusplus
#define DP_INT_ENUM(tag) enum tag : int
#else
#define DP_INT_ENUM(tag) enum tag
#endif

typedef DP_INT_ENUM(dp_dtype_e) { DP_F32 = 0, DP_BF16 = 1 } dp_dtype_t;

typedef DP_INT_ENUM(dp_status_e) {
  DP_OK = 0,
  DP_EINVAL = 1,
  DP_EUNSUPPORTED = 2,
  DP_EHIP = 3
} dp_status_t;

/* How a linear layer's per-example norm is evaluated.
 * GRAM:   <A_i A_i^T, G_i G_i^T> from two T x T Grams (ghost clipping,
 *         Sec. "Ghost Clipping Mechanism").
 * DIRECT: ||A_i^T G_i||_F^2 from the per-example gradient, squared and
 *         summed in registers without storing it (the materialising form of
 *         "normal clipping", Sec. "Training Configurations").
 * AUTO:   DIRECT when T + 1 > R * 2 d_in d_out / (d_in + d_out), else GRAM,
 *         where 2 d_in d_out / (d_in + d_out) equates the two flop counts
 *         and R is the measured ratio of the Gram kernel's throughput to the
 *         direct kernel's on MI355X near the crossover (bf16, T = 384 .. 768):
 *         R = 0.49, or 0.38 when d_out > 4096 (G is then read in feature
 *         chunks, as for an output head). With it AUTO picked the faster
 *         kernel for every GPT-2 layer shape at T = 128, 256, 384, 512, 640,
 *         768 and 1024. */
typedef DP_INT_ENUM(dp_norm_algo_e) { DP_NORM_AUTO = 0, DP_NORM_GRAM = 1, DP_NORM_DIRECT = 2 } dp_norm_algo_t;

/* One linear layer y = x W with W [d_in, d_out]: activations A [B,T,d_in]
 * (row stride lda) entering it and output gradients G [B,T,d_out] (row
 * stride ldg) leaving it (Sec. "Ghost Clipping Mechanism", eq. 4). The
 * output head of a language model is the layer d -> V with A = the hidden
 * states H and G = the logit gradients. */
typedef struct {
  const void* A;
  int64_t lda;
  int32_t d_in;
  const void* G;
  int64_t ldg;
  int32_t d_out;
  int32_t algo; /* dp_norm_algo_t */
} dp_linear_t;

int dp_abi_version(void);
const char* dp_status_string(dp_status_t s);
const char* dp_last_error(void);

/* ---------------------------------------------------------------------
 * Linear-layer ghost norm (Sec. "Ghost Clipping Mechanism", eq. 4-6).
 * For every example b:
 *   norm2[b] (+)= sum over layers of ||A_b^T G_b||_F^2.
 * The grouped form evaluates many layers of one batch in one launch (all
 * share B, T and dtype). Limits: T <= 65536, d_in, d_out <= 2^31 - 1.
 * Workspace: dp_ghost_norm_linear_workspace() bytes (fp32 partials). The
 * size depends on the layer table, pointers included (their alignment picks
 * the kernel and so the number of partials): query it with the same table
 * the call gets; a smaller workspace is rejected with DP_EINVAL.
 * ------------------------------------------------------------------- */
size_t dp_ghost_norm_linear_workspace(const dp_linear_t* layers, int n_layers, int B, int T,
                                      dp_dtype_t dt);
dp_status_t dp_ghost_norm_linear_grouped(const dp_linear_t* layers, int n_layers, int B, int T,
                                         dp_dtype_t dt, float* norm2, int accumulate,
                                         void* workspace, size_t workspace_bytes, void* stream);
dp_status_t dp_ghost_norm_linear(const void* A, int64_t lda, const void* G, int64_t ldg, int B,
                                 int T, int d_in, int d_out, dp_dtype_t dt, int algo,
                                 float* norm2, int accumulate, void* workspace,
                                 size_t workspace_bytes, void* stream);

/* The grouped norm with the layers' bias vectors. A bias b_l adds
 * y_t = ... + b_l to layer l, so its per-example gradient is the sum over
 * the example's tokens of the layer's own output gradient,
 *   bias_grads[l][i, :] = sum_t G_l[i,t,:]      (fp32 [B, d_out], caller-owned)
 * and the flat norm (eq. 6) takes its square in like every other parameter:
 * norm2[i] (+)= sum_l ||A_l,i^T G_l,i||^2 + sum_l ||bias_grads[l][i,:]||^2.
 * bias_grads (host array of n_layers device pointers, or NULL for no biases)
 * holds NULL for a layer without bias. Where the layer's Gram launch already
 * streams G with every token row of an example in LDS (bf16, 16-byte rows,
 * T <= 256) the bias sums ride along in the same pass; other layers get them
 * from the vector kernel (a second pass over their G). Either way the result
 * equals dp_ghost_norm_linear_grouped plus dp_vector_grads_grouped over the
 * biases (X = NULL), up to fp32 summation order. The workspace is
 * dp_ghost_norm_linear_bias_workspace(...) bytes (only bias_grads[l] != NULL
 * matters to it). */
size_t dp_ghost_norm_linear_bias_workspace(const dp_linear_t* layers, float* const* bias_grads,
                                           int n_layers, int B, int T, dp_dtype_t dt);
dp_status_t dp_ghost_norm_linear_bias_grouped(const dp_linear_t* layers, float* const* bias_grads,
                                              int n_layers, int B, int T, dp_dtype_t dt,
                                              float* norm2, int accumulate, void* workspace,
                                              size_t workspace_bytes, void* stream);

/* For callers that cannot allocate device memory (code under HIP graph
 * capture, tight serving loops, harnesses that forbid hipMalloc): the same
 * operation as dp_ghost_norm_linear_bias_grouped, bit for bit, with the
 * partial sums in a static device scratch of DP_NOALLOC_SCRATCH_BYTES that
 * the library holds on each device from its load to the end of the process,
 * instead of a caller's workspace. It calls no allocating routine; the first
 * call on a device looks up that device's scratch address
 * (hipGetSymbolAddress) once. A call whose partials need more than the
 * scratch holds (dp_ghost_norm_linear_bias_workspace(...) bytes, so
 * B * (partials per example) * 4 rounded up) returns DP_EUNSUPPORTED before
 * any launch. Every call on one device shares that device's scratch: calls
 * that overlap on one device (other streams, other threads) race and must be
 * ordered by the caller; nothing in the scratch needs to start at zero (every
 * partial is written before it is read). */
#define DP_NOALLOC_SCRATCH_BYTES (8u << 20)
dp_status_t dp_ghost_norm_linear_bias_grouped_noalloc(const dp_linear_t* layers,
                                                      float* const* bias_grads, int n_layers,
                                                      int B, int T, dp_dtype_t dt, float* norm2,
                                                      int accumulate, void* stream);

/* ---------------------------------------------------------------------
 * Input-embedding ghost norm and token buckets (Sec. "Weight Tying in
 * Decoder-Only LLMs"; the embedding reads row ids[b,t] of E in R^{V x d}).
 * dE [B,T,d] (row stride lde) is the gradient w.r.t. the embedding output.
 *   norm2[b] (+)= sum_v || sum_{t: ids[b,t] = v} dE[b,t,:] ||^2
 *   seg_id[b,t]  = rank of ids[b,t] among the sorted distinct ids of b
 *   n_unique[b]  = number of distinct ids of b
 * seg_id and n_unique may be NULL. Exact (integer) outputs.
 * Limits: ceil(log2(V + 1)) + ceil(log2 T) <= 32 (a sort key holds an id
 * clamped to V and a position; T <= 65536 at V = 50257) and B*T < 2^31.
 * bf16 examples up to T = 128 whose rows are whole 16-byte units (d a
 * multiple of 8) take the pairwise form sum_{t,s: ids equal} <dE_t, dE_s>
 * (the same sum, in another rounding order) and rank ids by comparison.
 * Up to T = 4096 an example is sorted in LDS, longer ones by a radix sort
 * through the workspace; those need rows of whole 8-byte units (lde and d
 * times the element size multiples of 8, dE 8-byte aligned) whose T rows
 * span less than 4 GiB, and are refused with DP_EUNSUPPORTED otherwise.
 * ------------------------------------------------------------------- */
size_t dp_ghost_norm_embedding_workspace(int B, int T, int d);
dp_status_t dp_ghost_norm_embedding(const int32_t* ids, const void* dE, int64_t lde, int B, int T,
                                    int V, int d, dp_dtype_t dt, float* norm2, int accumulate,
                                    int32_t* seg_id, int32_t* n_unique, void* workspace,
                                    size_t workspace_bytes, void* stream);

/* ---------------------------------------------------------------------
 * Tied-embedding cross term (Sec. "Corrected Ghost Norm for Tied
 * Embeddings", eq. 11 and eq. 13): with W_out = E, the squared norm of the
 * tied gradient is ||g_in||^2 + ||g_out||^2 + 2 <g_in, g_out>. This computes
 *   cross_b = <g_in,b, g_out,b> = sum_{t,s} Gz[b,s,ids[b,t]] <dE[b,t], H[b,s]>
 * without forming either V x d gradient, and writes
 *   out[b] = (accumulate ? out[b] : 0) + scale * cross_b.
 * scale = 2, accumulate = 1 adds the correction straight into a norm2.
 * H [B,T,d] (ldh) are the hidden states entering the head; Gz [B,T,V]
 * (row stride ldz >= V) the logit gradients.
 * ------------------------------------------------------------------- */
size_t dp_tied_cross_term_workspace(int B, int T, int d);
dp_status_t dp_tied_cross_term(const int32_t* ids, const void* dE, int64_t lde, const void* H,
                               int64_t ldh, const void* Gz, int64_t ldz, int B, int T, int V,
                               int d, dp_dtype_t dt, float scale, float* out, int accumulate,
                               void* workspace, size_t workspace_bytes, void* stream);

/* ---------------------------------------------------------------------
 * Clip factors (eq. 2, eq. 7): c[b] = min(1, C / sqrt(norm2[b])), and 1
 * when norm2[b] <= 0. A squared norm that is not finite (inf from an
 * overflow, or NaN) gives c[b] = 0: min(1, C/inf) is 0, and NaN is read the
 * same way, so that no such example enters a sum unclipped (eq. 2). Every
 * clipped-sum entry point below leaves an example with c[b] = 0 out (it is
 * skipped, not multiplied by zero), so inf or NaN in its operands cannot
 * reach the outputs. C must be positive and finite.
 * ------------------------------------------------------------------- */
dp_status_t dp_clip_factors(const float* norm2, int B, float C, float* c, void* stream);

/* ---------------------------------------------------------------------
 * Scaled clip factors (eq. 2, eq. 7 and the 1/B of eq. 3):
 *   c_scaled[b] = scale * min(1, C / sqrt(norm2[b]))   (1 when norm2 <= 0,
 *                                                         0 when not finite)
 * evaluated in double and rounded once to fp32; c (may be NULL) receives
 * the unscaled factors of dp_clip_factors in the same launch. With scale =
 * 1/B these factors let an embedding-form clipped sum add its part of eq. 3
 * directly onto an output that already holds (S + sigma*C*z)/B (written by
 * dp_clipped_grad_sum_noised_grouped or dp_noise_fill), so the output is
 * written once. norm2, c and c_scaled are device arrays of B floats; scale
 * must be finite.
 * ------------------------------------------------------------------- */
dp_status_t dp_clip_factors_scaled(const float* norm2, int B, float C, float scale, float* c,
                                   float* c_scaled, void* stream);

/* The same from a squared norm held in two parts (terms computed on two
 * streams, say): norm2[b] = norm2_a[b] + norm2_b[b], added in fp32 as an
 * accumulating norm call would. Both are device arrays of B floats. */
dp_status_t dp_clip_factors_scaled2(const float* norm2_a, const float* norm2_b, int B, float C,
                                    float scale, float* c, float* c_scaled, void* stream);

/* ---------------------------------------------------------------------
 * Clipped gradient sum (the bracket of eq. 3 without noise): the gradient
 * of the loss reweighted by the clip factors, as one GEMM over the B*T
 * tokens (K = B*T) with token k of example b scaled by c[b]:
 *   out (+)= sum_b c[b] A_b^T G_b            [d_in, d_out]
 * (examples with c[b] = 0 are left out, whatever their rows hold)
 * or its transpose [d_out, d_in] when transpose_out = 1 (out is contiguous).
 * Embedding form: pass A = NULL and ids [B,T]; A_b is then onehot(ids_b)
 * with d_in = V, i.e. out[v,:] (+)= sum over tokens with id v of
 * c[b] G[b,t,:]. A tied matrix receives both the head and the embedding
 * parts in one buffer: call the head form, then the embedding form with
 * accumulate = 1.
 * Workspace: only the embedding form needs one,
 * dp_clipped_grad_sum_workspace(B, T, d_out, 1) bytes; limit for it:
 * ceil(log2(V + 1)) + ceil(log2(B*T)) <= 32 (a sort key holds an id
 * clamped to V and a token index; B*T <= 65536 at V = 50257). Up to 16384
 * tokens are sorted in one workgroup's LDS, more by a radix sort through
 * the workspace (same order, so the same result).
 * ------------------------------------------------------------------- */
size_t dp_clipped_grad_sum_workspace(int B, int T, int d_out, int with_ids);
dp_status_t dp_clipped_grad_sum(const void* A, int64_t lda, const void* G, int64_t ldg,
                                const int32_t* ids, const float* c, int B, int T, int d_in,
                                int d_out, dp_dtype_t dt, int transpose_out, float* out,
                                int accumulate, void* workspace, size_t workspace_bytes,
                                void* stream);
/* The embedding form in two calls, so that the part that does not touch
 * `out` can run while something else (the head's clipped-sum GEMM, say)
 * writes it. The embedding reads row ids[b,t] of E (Sec. "Weight Tying in
 * Decoder-Only LLMs"), so its share of the bracket of eq. 3 has one row per
 * id: row v of sum_b c[b] onehot(ids_b)^T G_b is the sum of c[b] G[b,t,:]
 * over the tokens with ids[b,t] = v.
 * dp_embedding_rows sorts the B*T tokens by id and writes one fp32 row per
 * distinct id (a run of equal ids) into the workspace, with the run list;
 * it reads G [B*T, ldg] (dt), ids [B,T] and c [B] (device) and touches
 * nothing else. Ids at or past V form one run that the add skips.
 * dp_embedding_rows_add then adds every run's row onto out[v,:] (out is
 * [V, d], or [d, V] with transpose_out; contiguous; always accumulated),
 * and must follow dp_embedding_rows on the same workspace with the same
 * B, T, V, d (same stream, or ordered by an event); on a workspace that call
 * has not filled, its result is undefined but its reads and writes stay
 * inside the workspace and out. Each row is added with
 * one fp32 addition, so the pair gives the same result, bit for bit, as the
 * embedding form of dp_clipped_grad_sum with accumulate = 1.
 * Workspace: dp_embedding_rows_workspace(B, T, d) bytes (B*T rows of d
 * floats plus the sort's buffers), owned by the caller and live from the
 * first call to the end of the second. Limits as for the embedding form. */
size_t dp_embedding_rows_workspace(int B, int T, int d);
dp_status_t dp_embedding_rows(const void* G, int64_t ldg, const int32_t* ids, const float* c,
                              int B, int T, int V, int d, dp_dtype_t dt, void* workspace,
                              size_t workspace_bytes, void* stream);
dp_status_t dp_embedding_rows_add(const void* workspace, size_t workspace_bytes, int B, int T,
                                  int V, int d, int transpose_out, float* out, void* stream);

/* Many linear layers in one launch; outs[l] is layer l's output. */
dp_status_t dp_clipped_grad_sum_grouped(const dp_linear_t* layers, float* const* outs,
                                        int n_layers, const float* c, int B, int T,
                                        dp_dtype_t dt, int transpose_out, int accumulate,
                                        void* stream);

/* ---------------------------------------------------------------------
 * Clipped sum and Gaussian mechanism in one pass (eq. 3): for each layer l
 *   outs[l] = (prior + sum_i c_i A_i^T G_i + sigma*C*z) / B_norm
 * where prior is outs[l]'s content if accumulate[l] != 0 (else 0), and z is
 * the standard normal that dp_add_noise(outs[l], rows*cols, sigma, C, B_norm,
 * seed, tensor_ids[l], step) would add to the same element: the element at
 * row r, column k of the output ([d_in, d_out], or [d_out, d_in] with
 * transpose_out) takes index r*cols + k of the tensor's Philox stream. The
 * result equals dp_clipped_grad_sum_grouped followed by dp_add_noise on each
 * output, without a second pass over the gradients. B_norm = 0: no
 * division. A tied matrix is noised once: either write the head's part here
 * (accumulate[l] = 0) and then add the embedding-form clipped sum with the
 * factors c/B_norm from dp_clip_factors_scaled (the matrix is written once),
 * or write the embedding part first and pass accumulate[l] = 1.
 * tensor_ids[l] and step must be < 2^32; accumulate may be NULL (all 0).
 * tensor_ids and accumulate are host arrays of n_layers entries.
 * ------------------------------------------------------------------- */
dp_status_t dp_clipped_grad_sum_noised_grouped(const dp_linear_t* layers, float* const* outs,
                                               const uint64_t* tensor_ids,
                                               const int32_t* accumulate, int n_layers,
                                               const float* c, int B, int T, dp_dtype_t dt,
                                               int transpose_out, float sigma, float C,
                                               int B_norm, uint64_t seed, uint64_t step,
                                               void* stream);

/* The same with a caller-owned workspace of at least
 * dp_clipped_grad_sum_noised_grouped_workspace(...) bytes (a NULL workspace
 * of 0 bytes gives the call above). Where a launch's last round of 256 x 256
 * output tiles would keep at most half of the compute units busy (bf16,
 * 16-byte rows, T a multiple of 32), each of its tiles is computed as 2-8
 * consecutive K ranges on separate compute units; the fp32 partial tiles go
 * to the workspace and are added in order before the prior and the noise, so
 * results differ from the call above by fp32 rounding only. The workspace
 * is dead after the call's kernels finish. */
size_t dp_clipped_grad_sum_noised_grouped_workspace(const dp_linear_t* layers, int n_layers,
                                                    int B, int T, dp_dtype_t dt,
                                                    int transpose_out);
dp_status_t dp_clipped_grad_sum_noised_grouped_ws(const dp_linear_t* layers, float* const* outs,
                                                  const uint64_t* tensor_ids,
                                                  const int32_t* accumulate, int n_layers,
                                                  const float* c, int B, int T, dp_dtype_t dt,
                                                  int transpose_out, float sigma, float C,
                                                  int B_norm, uint64_t seed, uint64_t step,
                                                  void* workspace, size_t workspace_bytes,
                                                  void* stream);

/* ---------------------------------------------------------------------
 * Per-example gradient store: the materialising ("normal clipping") form of
 * the clipped sum (Sec. "Training Configurations"; eq. 2-3), for the long
 * sequences where the direct norm is taken anyway (dp_norm_algo_t). The
 * direct norm forms every example's gradient A_b^T G_b tile by tile in
 * registers; dp_ghost_norm_linear_store also writes those fp32 tiles to the
 * store (B * tiles * 256 KB: 7.9 GB for GPT-2 small at B = 16), and
 * dp_clipped_grad_sum_noised_store then forms
 *   outs[l] = (prior + sum_b c_b (A_b^T G_b) + sigma*C*z) / B_norm
 * from the stored tiles, an HBM-bound weighted sum, instead of multiplying
 * the operands again. The result, noise included, is that of
 * dp_clipped_grad_sum_noised_grouped on the same arguments up to fp32
 * rounding order; an example with c_b = 0 is left out, as there.
 * Conditions: bf16, T a multiple of 32, every layer's A and G rows 16-byte
 * aligned (else DP_EUNSUPPORTED, and dp_grad_store_bytes returns 0).
 * dp_grad_store_bytes: the store size for this layer table (the tiles plus
 * B * tiles fp32 norm partials), 0 when the conditions fail.
 * dp_ghost_norm_linear_store: norm2[b] (+)= sum over layers of
 * ||A_b^T G_b||_F^2, every layer by the direct form whatever its algo field
 * (bit-identical to dp_ghost_norm_linear_grouped with DP_NORM_DIRECT), and
 * the tiles into the store.
 * dp_clipped_grad_sum_noised_store: outs, tensor_ids, accumulate and the
 * noise arguments as for dp_clipped_grad_sum_noised_grouped; the output
 * layout is chosen per layer: transpose_out[l] != 0 writes outs[l] as
 * [d_out, d_in] (transpose_out may be NULL: all [d_in, d_out]; a host array
 * of n_layers entries, like accumulate). layers must be the table the store
 * was written with (its pointers are not read again, only its shapes). store: device memory owned by the caller,
 * 16-byte aligned, at least dp_grad_store_bytes() bytes (the sum reads the
 * tiles only); it holds one step's tiles until the next store call.
 * ------------------------------------------------------------------- */
size_t dp_grad_store_bytes(const dp_linear_t* layers, int n_layers, int B, int T,
                           dp_dtype_t dt);
dp_status_t dp_ghost_norm_linear_store(const dp_linear_t* layers, int n_layers, int B, int T,
                                       dp_dtype_t dt, float* norm2, int accumulate, void* store,
                                       size_t store_bytes, void* stream);
dp_status_t dp_clipped_grad_sum_noised_store(const dp_linear_t* layers, float* const* outs,
                                             const uint64_t* tensor_ids,
                                             const int32_t* accumulate,
                                             const int32_t* transpose_out, int n_layers,
                                             const float* c, int B, int T, dp_dtype_t dt,
                                             float sigma, float C, int B_norm, uint64_t seed,
                                             uint64_t step, const void* store,
                                             size_t store_bytes, void* stream);

/* ---------------------------------------------------------------------
 * Gaussian mechanism (eq. 3): grad[j] = (grad[j] + sigma*C*z_j) / B_norm
 * (no division when B_norm = 0), in place, for j < n; the division is a
 * multiplication by 1/B_norm rounded to fp32 (within an ulp of dividing). z_j is a standard
 * normal from the counter-based Philox4x32-10 generator (Salmon et al.,
 * SC'11) and the Box-Muller transform: element j uses Philox block j/4 with
 * key (seed low word, seed high word) and counter (block low word, block
 * high word, tensor_id, step); the four outputs x become uniforms
 * (x + 1/2) 2^-32 and the pairs (0,1), (2,3) give r cos(2 pi u_odd),
 * r sin(2 pi u_odd) with r = sqrt(-2 ln u_even); element j takes output j%4.
 * The device evaluates the transform in fp32 on the hardware log2, sqrt,
 * sin and cos units (absolute error on z below 1e-4, tails included).
 * The same (seed, tensor_id, step) reproduces the same noise, so the
 * generator position is the only state to checkpoint. tensor_id and step
 * must be < 2^32. grad is fp32.
 * ------------------------------------------------------------------- */
dp_status_t dp_add_noise(float* grad, int64_t n, float sigma, float C, int B_norm, uint64_t seed,
                         uint64_t tensor_id, uint64_t step, void* stream);

/* Noise alone (eq. 3 with a zero sum): out[j] = sigma*C*z_j / B_norm with
 * the z_j of dp_add_noise for the same (seed, tensor_id, step), bit-identical
 * to dp_add_noise on zeros; out is written without being read. Arguments
 * and limits as for dp_add_noise. */
dp_status_t dp_noise_fill(float* out, int64_t n, float sigma, float C, int B_norm, uint64_t seed,
                          uint64_t tensor_id, uint64_t step, void* stream);

/* ---------------------------------------------------------------------
 * Vector parameters applied to every token: a linear layer's bias, a
 * LayerNorm gain or bias. The paper's parameter counts include them, and the
 * flat per-example norm (eq. 6) takes them in like every other parameter.
 * By the chain rule the per-example gradient of parameter v is
 *   g_v,i = sum_t X_v[i,t] * G_v[i,t]   (elementwise over the d_v features)
 * with X the LayerNorm's normalised input for a gain, and the plain sum
 * sum_t G_v[i,t] when X is NULL (a bias: y_t = ... + b; a LayerNorm bias).
 * G is the gradient w.r.t. the parameter's output (for a linear layer's bias,
 * the layer's own G). These gradients are d_v-vectors, so they are
 * materialised rather than recovered from a Gram product.
 * ------------------------------------------------------------------- */
typedef struct {
  const void* X;  /* [B*T rows, ldx] factor of a gain, or NULL (a bias) */
  int64_t ldx;    /* row stride of X, >= d (ignored when X is NULL) */
  const void* G;  /* [B*T rows, ldg] grads w.r.t. the parameter's output */
  int64_t ldg;    /* row stride of G, >= d */
  int32_t d;      /* features */
} dp_vector_t;

/* grads[v] (caller-owned fp32 [B, d_v], row stride d_v) receives g_v,i for
 * every example i; when norm2 is not NULL, norm2[i] (+)= sum_v ||g_v,i||^2.
 * Sums over tokens and features run in a fixed order (reproducible). The
 * workspace is at least dp_vector_grads_workspace(...) bytes. */
size_t dp_vector_grads_workspace(const dp_vector_t* params, int n, int B, int T, dp_dtype_t dt);
dp_status_t dp_vector_grads_grouped(const dp_vector_t* params, int n, int B, int T,
                                    dp_dtype_t dt, float* const* grads, float* norm2,
                                    int accumulate, void* workspace, size_t workspace_bytes,
                                    void* stream);

/* Clipped sums of materialised per-example gradients with the Gaussian
 * mechanism (eq. 3), for each parameter v:
 *   outs[v][f] = (prior + sum_i c_i grads[v][i*d[v] + f] + sigma*C*z_f) / B_norm
 * with prior = outs[v][f] if accumulate[v] != 0 (else 0), the sum over i in
 * order, and z_f the draw dp_add_noise(outs[v], d[v], sigma, C, B_norm, seed,
 * tensor_ids[v], step) would add to element f. sigma = 0 and B_norm = 0 give
 * the plain clipped sum. grads, d, outs, tensor_ids and accumulate are host
 * arrays of n entries (accumulate may be NULL: all 0). */
dp_status_t dp_vector_clipped_sum_noised_grouped(const float* const* grads, const int32_t* d,
                                                 int n, int B, const float* c,
                                                 float* const* outs, const uint64_t* tensor_ids,
                                                 const int32_t* accumulate, float sigma, float C,
                                                 int B_norm, uint64_t seed, uint64_t step,
                                                 void* stream);

/* ---------------------------------------------------------------------
 * Learned position table (n_pos rows of d features): token t of every
 * example adds row t to its input embedding, so the per-example gradient has
 * row t equal to that token's embedding-output grad dE[i,t] (t < T) and zero
 * rows below; an example's positions are distinct, so its squared norm is
 * sum_t ||dE[i,t]||^2 (contrast the token embedding, whose rows are keyed by
 * token id). dE is the same [B, T, d] buffer dp_ghost_norm_embedding reads.
 * norm2[i] (+)= sum_t ||dE[i,t]||^2; workspace >= the size returned.
 * ------------------------------------------------------------------- */
size_t dp_ghost_norm_positional_workspace(int B, int T, int d);
dp_status_t dp_ghost_norm_positional(const void* dE, int64_t lde, int B, int T, int d,
                                     dp_dtype_t dt, float* norm2, int accumulate,
                                     void* workspace, size_t workspace_bytes, void* stream);

/* The position table's clipped sum with the Gaussian mechanism (eq. 3):
 *   out[t, f] = (prior + [t < T] sum_i c_i dE[i,t,f] + sigma*C*z) / B_norm
 * for every row t < n_pos (out has row stride ldo >= d; T <= n_pos), the sum
 * over i in order, z the draw of element t*d + f of the table's stream
 * (tensor_id), as dp_add_noise on a contiguous [n_pos, d] table would add. */
dp_status_t dp_clipped_grad_sum_positional_noised(const void* dE, int64_t lde, const float* c,
                                                  int B, int T, int d, dp_dtype_t dt, float* out,
                                                  int n_pos, int64_t ldo, uint64_t tensor_id,
                                                  int accumulate, float sigma, float C,
                                                  int B_norm, uint64_t seed, uint64_t step,
                                                  void* stream);

#ifdef __cplusplus
}
#endif
#endif /* DPGHOST_H */
