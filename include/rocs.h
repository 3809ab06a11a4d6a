/*
 * rocs.h - C ABI of librocs, the MI355X (gfx950) IKBO inference hot path of
 * ROCS (Request-Oriented Compute Sharing, arXiv 2607.27744).
 *
 * In-Kernel Broadcast Optimization (IKBO, Section 4) keeps request-side and
 * candidate-side tensors at their natural batch sizes, R requests (B_r) and
 * N candidates (B_c), and resolves the candidate -> request map m inside the
 * consuming kernels instead of materialising a request-to-candidate
 * broadcast. Here m is given as CSR offsets:
 *
 *   cand_offsets[R + 1], int32, device memory:
 *     candidate n belongs to request r  iff  cand_offsets[r] <= n < cand_offsets[r+1]
 *   so the candidates of one request are contiguous (Section 4.2.1 and 4.3.1
 *   both rely on this ordering for cache locality).
 *
 * Conventions shared by every entry point
 *   - Tensor pointers are DEVICE pointers to contiguous row-major arrays owned
 *     by the caller. The library never allocates, frees or keeps them; it
 *     holds no pointer after a call returns.
 *   - `stream` is a hipStream_t passed as void* (NULL = the default stream).
 *     Work is enqueued asynchronously; nothing is synchronised. A fault in a
 *     kernel surfaces at the caller's next synchronisation.
 *   - Offsets arrays are trusted device data: offsets[0] == 0, non-decreasing,
 *     offsets[R] equal to the row count they index. They are not read on the
 *     host (that would need a synchronisation); malformed offsets give
 *     undefined results. rocs_validate_offsets() checks them when wanted.
 *   - Element types: ROCS_DTYPE_BF16 (bfloat16 storage, fp32 accumulation,
 *     results rounded to nearest-even) or ROCS_DTYPE_F32 (fp32 throughout).
 *     Inputs and outputs of one call share the dtype; bias and the linear
 *     workspace are always fp32.
 *   - Every call returns a rocs_status. On failure nothing has been enqueued,
 *     and rocs_last_error_message() (thread-local) explains the failure.
 *     R == 0 or N == 0 is a valid no-op (outputs that have no rows are not
 *     touched; request-side outputs are still produced where they exist).
 *   - Calls are reentrant; concurrent calls on different streams need
 *     separate workspaces.
 */
#ifndef ROCS_H
#define ROCS_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#define ROCS_ABI_VERSION 5

typedef enum rocs_status {
  ROCS_OK = 0,
  ROCS_ERR_INVALID_ARGUMENT = 1,   /* null pointer, bad size, bad enum, misalignment */
  ROCS_ERR_UNSUPPORTED = 2,        /* valid request this build cannot run */
  ROCS_ERR_WORKSPACE_TOO_SMALL = 3,
  ROCS_ERR_HIP = 4                 /* the HIP runtime refused a launch */
} rocs_status;

typedef enum rocs_dtype { ROCS_DTYPE_F32 = 0, ROCS_DTYPE_BF16 = 1 } rocs_dtype;

typedef enum rocs_activation { ROCS_ACT_NONE = 0, ROCS_ACT_RELU = 1 } rocs_activation;

int32_t rocs_abi_version(void);
const char* rocs_status_string(int32_t status);
/* Detail of the calling thread's last non-OK status ("" if none). */
const char* rocs_last_error_message(void);

/*
 * ---------------------------------------------------------------------------
 * rocs_ikbo_linear: the candidate-side output of a two-group GLM linear
 * (Eq. glm-linear with K = 2; Section 4.1 decomposition; Eq. broadcast_add;
 * fusion of the broadcast-add into the GEMM epilogue, Section 4.2.1).
 *
 *   out[n][d] = act( sum_k w_cand[d][k] * xc[n][k]
 *                  + sum_k w_req[d][k]  * x_req[m_n][k]   (= Z[m_n][d])
 *                  + bias[d] )
 *
 * where xc = x_cand, or, when x_cand_add is not NULL, the GLM pointwise
 * residual xc = round(x_cand + x_cand_add) computed elementwise in fp32 and
 * rounded to the input dtype (Eq. glm-elementwise) before the product.
 *
 * The request-side product Z = x_req . w_req^T ([R, d_out], fp32) is computed
 * once per request into the workspace, together with the expanded index map
 * m ([N] int32); the candidate GEMM adds Z[m_n] in its epilogue. No
 * candidate-batched copy of x_req or Z is ever formed.
 *
 *   x_req       [R, k_req]        request-side input; may be NULL iff k_req == 0
 *   k_req       >= 0; 0 makes this a plain linear (no request term)
 *   x_cand      [N, k_cand]       candidate-side input
 *   x_cand_add  [N, k_cand] or NULL
 *   k_cand      >= 1
 *   w_req       [d_out, k_req]    W_CR in the paper's [out, in] orientation
 *   w_cand      [d_out, k_cand]   W_CC
 *   bias        [d_out] fp32 or NULL (zero)
 *   cand_offsets [R + 1]          may be NULL iff k_req == 0
 *   out         [N, d_out]        must not overlap any input
 *   workspace   device memory of at least rocs_ikbo_linear_workspace_size()
 *               bytes, 256-byte aligned; may be NULL when that size is 0.
 *               Contents on entry are ignored; on return they are scratch.
 *
 * Fast path: bf16, k_req and k_cand multiples of 8, d_out a multiple of 4 and
 * every pointer 16-byte aligned. Other shapes take a slower general kernel
 * (the zero-padding transform of Section 4.2.4 restores the fast path).
 *
 * The request-side GEMM is a launch of its own; rocs_ikbo_linear_combined
 * runs it inside the candidate kernel instead (Section 4.2.3).
 *
 * Limits: every size below 2^31. Off the fast path the general kernels run
 * one thread per output element, so N * d_out must stay below 2^32
 * (ROCS_ERR_UNSUPPORTED otherwise).
 * ---------------------------------------------------------------------------
 */
size_t rocs_ikbo_linear_workspace_size(int64_t num_requests, int64_t num_cand,
                                       int64_t d_out, int64_t k_req);

int32_t rocs_ikbo_linear(const void* x_req, int64_t k_req,
                         const void* x_cand, const void* x_cand_add, int64_t k_cand,
                         const void* w_req, const void* w_cand, const float* bias,
                         const int32_t* cand_offsets,
                         int64_t num_requests, int64_t num_cand, int64_t d_out,
                         int32_t dtype, int32_t activation,
                         void* out, void* workspace, size_t workspace_bytes,
                         void* stream);

/*
 * ---------------------------------------------------------------------------
 * rocs_glm_linear: both outputs of a two-group GLM linear layer
 * (Eq. glm-linear with K = 2):
 *
 *   y_req[r]  = act( W_RR x_req[r] + b_req )                      [R, d_req]
 *   y_cand[n] = act( W_CR x_req[m_n] + W_CC xc[n] + b_cand )      [N, d_cand]
 *
 * (the masked block W_RC never exists). The request-side products W_RR x^R
 * and W_CR x^R come from one GEMM at batch size R over the stacked weight
 * [W_RR; W_CR] (Section 4.1); the candidate side is rocs_ikbo_linear.
 *
 *   w_rr [d_req, k_req], w_cr [d_cand, k_req], w_cc [d_cand, k_cand]
 *   b_req [d_req] fp32 or NULL; b_cand [d_cand] fp32 or NULL
 *   y_req [R, d_req] (required), y_cand [N, d_cand] (may be NULL iff N == 0)
 *   k_req >= 1, d_req >= 1; every other argument, the workspace
 *   (rocs_ikbo_linear_workspace_size(R, N, d_cand, k_req) bytes) and the
 *   errors as for rocs_ikbo_linear. N == 0 still produces y_req.
 * Fast path: that of rocs_ikbo_linear, plus d_req a multiple of 4, w_rr and
 * b_req 16-byte and y_req 8-byte aligned.
 * ---------------------------------------------------------------------------
 */
int32_t rocs_glm_linear(const void* x_req, int64_t k_req,
                        const void* x_cand, const void* x_cand_add, int64_t k_cand,
                        const void* w_rr, const void* w_cr, const void* w_cc,
                        const float* b_req, const float* b_cand, const int32_t* cand_offsets,
                        int64_t num_requests, int64_t num_cand, int64_t d_req, int64_t d_cand,
                        int32_t dtype, int32_t activation, void* y_req, void* y_cand,
                        void* workspace, size_t workspace_bytes, void* stream);

/*
 * ---------------------------------------------------------------------------
 * rocs_ikbo_linear_combined: the outputs of rocs_glm_linear (y_req optional)
 * from one launch: the combined request + candidate kernel of Section 4.2.3.
 * The streaming candidate kernel first computes the stacked request GEMM's
 * 16 x 16 tiles (request tiles in ascending order); each tile of the request
 * table Z publishes a completion flag with an agent-scope release, and a
 * workgroup waits for every flag (bounded: past the limit it computes the
 * missing tiles itself, with the same code and so the same values) while its
 * first candidate loads are in flight, then takes its candidate tiles in
 * descending order. The flags live in the workspace, tagged with a per-call
 * epoch, so nothing needs clearing between calls.
 *
 *   Arguments as for rocs_glm_linear, except that y_req may be NULL: then
 *   w_rr, b_req and d_req are ignored and only y_cand is produced (the
 *   rocs_ikbo_linear output, with w_cr and w_cc in the roles of w_req and
 *   w_cand). The workspace is rocs_ikbo_linear_workspace_size(R, N, d_cand,
 *   k_req) bytes, as for the separate launches.
 *
 * The results equal those of rocs_glm_linear / rocs_ikbo_linear bit for bit.
 * The combined kernel runs where the streaming candidate kernel does (bf16
 * fast path, k_cand a multiple of 64, no x_cand_add, k_req > 0, N > 0);
 * other calls run the separate launches. On MI355X the separate launches are
 * usually faster: the cross-XCD L2 write-back behind each release and the
 * invalidate behind each acquire cost more than the launch they save.
 * ---------------------------------------------------------------------------
 */
int32_t rocs_ikbo_linear_combined(const void* x_req, int64_t k_req,
                                  const void* x_cand, const void* x_cand_add, int64_t k_cand,
                                  const void* w_rr, const void* w_cr, const void* w_cc,
                                  const float* b_req, const float* b_cand,
                                  const int32_t* cand_offsets,
                                  int64_t num_requests, int64_t num_cand, int64_t d_req,
                                  int64_t d_cand, int32_t dtype, int32_t activation,
                                  void* y_req, void* y_cand,
                                  void* workspace, size_t workspace_bytes, void* stream);

/*
 * ---------------------------------------------------------------------------
 * rocs_ikbo_linear_noalloc: rocs_ikbo_linear for callers that cannot allocate
 * device memory (code under HIP graph capture, tight serving loops, hosts
 * that forbid allocation). It takes no workspace: the request table Z and the
 * index map live in a static scratch array of ROCS_NOALLOC_SCRATCH_BYTES
 * that the library holds on each device it runs on until the process ends.
 * The call itself allocates and frees nothing; the first call on a device
 * looks up that device's copy of the array (once).
 *
 *   Arguments, result, fast path and errors as for rocs_ikbo_linear, without
 *   workspace / workspace_bytes. The call needs
 *   rocs_ikbo_linear_workspace_size(R, N, d_out, k_req) <=
 *   ROCS_NOALLOC_SCRATCH_BYTES (for example R = 16, d_out = 1024 and up to
 *   about four million candidates); a larger call returns
 *   ROCS_ERR_WORKSPACE_TOO_SMALL before touching the device.
 *
 * All calls on one device share its scratch array, and a call leaves its own
 * contents there (nothing in it needs clearing: every call writes what it
 * reads). Calls that overlap in time on one device (concurrent streams,
 * threads) race on it and must be serialised by the caller.
 * ---------------------------------------------------------------------------
 */
#define ROCS_NOALLOC_SCRATCH_BYTES ((size_t)16 << 20)

int32_t rocs_ikbo_linear_noalloc(const void* x_req, int64_t k_req,
                                 const void* x_cand, const void* x_cand_add, int64_t k_cand,
                                 const void* w_req, const void* w_cand, const float* bias,
                                 const int32_t* cand_offsets,
                                 int64_t num_requests, int64_t num_cand, int64_t d_out,
                                 int32_t dtype, int32_t activation, void* out, void* stream);

/*
 * ---------------------------------------------------------------------------
 * rocs_ikbo_linear_mapped: rocs_ikbo_linear with the index map m given as a
 * per-candidate request id instead of CSR offsets (Section 4.1 defines m as
 * any map {0..B_c-1} -> {0..B_r-1}; candidates of one request need not be
 * contiguous or ordered).
 *
 *   cand_request_ids [N] int32, device memory: m_n for every candidate n,
 *                    each in [0, R). Trusted device data like the offsets: an
 *                    id outside [0, R) gives wrong rows for that candidate
 *                    (the kernels clamp it into range), never an access
 *                    outside the request-side product. May be NULL iff
 *                    k_req == 0.
 * Every other argument, the result, the workspace (at least
 * rocs_ikbo_linear_workspace_size() bytes) and the errors are those of
 * rocs_ikbo_linear. The request-side product is still formed once per
 * request. The candidate GEMM resolves m per row in its epilogue (a tile
 * whose rows share one request loads Z once), so it runs the kernel with a
 * per-row request lookup rather than the request-aligned streaming kernel.
 * ---------------------------------------------------------------------------
 */
int32_t rocs_ikbo_linear_mapped(const void* x_req, int64_t k_req,
                                const void* x_cand, const void* x_cand_add, int64_t k_cand,
                                const void* w_req, const void* w_cand, const float* bias,
                                const int32_t* cand_request_ids,
                                int64_t num_requests, int64_t num_cand, int64_t d_out,
                                int32_t dtype, int32_t activation,
                                void* out, void* workspace, size_t workspace_bytes,
                                void* stream);

/*
 * ---------------------------------------------------------------------------
 * rocs_dca_attention: candidate-side Deep Cross Attention
 * A^C = Attn(Q^C, S W_K, S W_V) (Section 3.2, Eq. dca-attention) with the
 * request-batched K/V consumed directly (Section 4.3.1): every candidate of
 * request r attends over r's history, which is read once per tile of that
 * request's candidates and shared by all of them; no per-candidate K/V copy.
 *
 * For candidate n with r = m_n, query token t and head h:
 *   s_j      = scale * <q[n][t][h][:], k[j][h][:]>   for kv_offsets[r] <= j < kv_offsets[r+1]
 *   out[n][t][h][:] = sum_j softmax(s)_j * v[j][h][:]   (no mask)
 * An empty history (L_r == 0) gives zeros.
 *
 *   q            [N, q_len, H, head_dim]
 *   k, v         history rows packed request after request; row j of k
 *                starts at k + j * kv_row_stride elements and holds
 *                [H, head_dim]; same for v. kv_row_stride == 0 means
 *                H * head_dim (dense [L_total, H, head_dim]). A larger stride
 *                lets k and v be column slices of one projection output.
 *   cand_offsets [R + 1]; kv_offsets [R + 1] (L_total = kv_offsets[R])
 *   q_len >= 1, num_heads >= 1, 1 <= head_dim <= 256
 *   softmax_scale  > 0, or <= 0 for 1/sqrt(head_dim)
 *   out          [N, q_len, H, head_dim], must not overlap any input
 *
 * Fast path (bf16 MFMA kernel): bf16, head_dim 64 or 128, H*head_dim and
 * kv_row_stride multiples of 8, pointers 16-byte aligned. Other cases run a
 * general kernel.
 *
 * Limits: N * q_len below 2^31 and num_heads below 2^16. The general kernel
 * runs one wave per query row and head, so it takes N * q_len below 2^26;
 * the fast path takes (R + N * q_len / 128) * num_heads below 2^24. Larger
 * calls return ROCS_ERR_UNSUPPORTED.
 * ---------------------------------------------------------------------------
 */
int32_t rocs_dca_attention(const void* q, const void* k, const void* v,
                           const int32_t* cand_offsets, const int32_t* kv_offsets,
                           int64_t num_requests, int64_t num_cand,
                           int32_t q_len, int32_t num_heads, int32_t head_dim,
                           int64_t kv_row_stride, float softmax_scale, int32_t dtype,
                           void* out, void* stream);

/*
 * ---------------------------------------------------------------------------
 * rocs_dca_attention_residual: rocs_dca_attention that also emits the
 * pointwise residual that feeds the next layer of stacked DCA (Section 3.2:
 * the next layer's query input is this layer's output plus the candidate
 * embedding; a pointwise operation, so GLM-compliant, Eq. glm-elementwise):
 *
 *   out_sum[n][t][h][e] = round(out[n][t][h][e] + residual[n][t][h][e])
 *
 * where out is first rounded to dtype (exactly the values written to out),
 * the sum is taken in fp32 and rounded to dtype (round to nearest even;
 * no rounding for fp32). The sum is formed in the attention's epilogue, so
 * the next projection reads one tensor instead of two.
 *
 *   residual  [N, q_len, H, head_dim], the layout of q (device memory)
 *   out_sum   [N, q_len, H, head_dim], must not overlap any input or out
 * Every other argument, the result and the errors are those of
 * rocs_dca_attention (the fast path also needs residual and out_sum 16-byte
 * aligned). An empty history gives out = 0 and out_sum = residual.
 * ---------------------------------------------------------------------------
 */
int32_t rocs_dca_attention_residual(const void* q, const void* k, const void* v,
                                    const int32_t* cand_offsets, const int32_t* kv_offsets,
                                    int64_t num_requests, int64_t num_cand,
                                    int32_t q_len, int32_t num_heads, int32_t head_dim,
                                    int64_t kv_row_stride, float softmax_scale, int32_t dtype,
                                    const void* residual, void* out, void* out_sum,
                                    void* stream);

/*
 * ---------------------------------------------------------------------------
 * rocs_dca_attention_ex: rocs_dca_attention with three options, any
 * combination of them:
 *
 * - fused query projection (w_q non-NULL): the candidate queries are the
 *   candidate side of the DCA query generator, a linear projection of the
 *   candidate's features (Section 3.2, Eq. dca-query), computed inside the
 *   attention kernel:
 *
 *     q[n][t][h][:] = round(x[n][t][:] W_q[h head_dim .. (h + 1) head_dim - 1][:]^T)
 *
 *   rounded to dtype exactly as a separate projection would store it; the
 *   queries never reach memory. `q` then holds x [N, q_len, d_in] (d_in >= 1)
 *   and w_q is [H * head_dim, d_in] (the paper's [out, in] orientation).
 *   With w_q NULL, q is the query [N, q_len, H, head_dim] and d_in is
 *   ignored.
 * - residual (non-NULL, with out_sum): out_sum = round(out + residual), as
 *   rocs_dca_attention_residual. residual may be x itself when d_in =
 *   H * head_dim (the stacked-DCA residual of the candidate embedding).
 * - plan (non-NULL): the tile order made by rocs_dca_attention_plan for
 *   these cand_offsets and kv_offsets, R, q_len and num_heads; plan_bytes >=
 *   rocs_dca_attention_plan_size(R) (else ROCS_ERR_WORKSPACE_TOO_SMALL),
 *   4-byte aligned, read only. The tiled kernel then takes its 128-row tiles
 *   longest history first. Results are bit-identical with or without it. A
 *   plan made for another R, q_len or num_heads is ignored (the built-in
 *   order runs); one made for other offsets of the same R gives wrong rows
 *   but never an access outside the arguments.
 *
 * out, out_sum and plan may not overlap x, w_q or each other
 * (ROCS_ERR_INVALID_ARGUMENT). Every other argument, the result and the
 * errors are those of rocs_dca_attention. Fast path: its conditions (with
 * the projection: head_dim 64, d_in 256 and w_q 16-byte aligned; each
 * workgroup projects its tile's query rows of one head on the matrix cores,
 * with the operand roles and k order of the streaming linear, so q matches
 * rocs_ikbo_linear's output bit for bit). Other shapes and fp32 run the
 * general kernel, which ignores the plan.
 * ---------------------------------------------------------------------------
 */
int32_t rocs_dca_attention_ex(const void* q, int64_t d_in, const void* w_q, const void* k,
                              const void* v, const int32_t* cand_offsets,
                              const int32_t* kv_offsets, const void* plan, size_t plan_bytes,
                              int64_t num_requests, int64_t num_cand, int32_t q_len,
                              int32_t num_heads, int32_t head_dim, int64_t kv_row_stride,
                              float softmax_scale, int32_t dtype, const void* residual,
                              void* out, void* out_sum, void* stream);

/*
 * ---------------------------------------------------------------------------
 * rocs_dca_attention_plan: the tile order of the tiled DCA kernel for one
 * batch (Section 4.3: candidates of one request share its K/V; the kernel's
 * time per tile grows with the request's history length). Written on
 * `stream` into plan (device memory, plan_bytes >=
 * rocs_dca_attention_plan_size(R), 4-byte aligned), from the device offsets
 * cand_offsets [R + 1] and kv_offsets [R + 1] (valid CSR offsets, as for
 * rocs_dca_attention), for q_len query tokens per candidate and num_heads
 * heads. Longest history first (histories of 2^20 - 1 rows or more count
 * as equal), ties by request index; all heads of one request next to each
 * other. Up to 4096 requests; beyond that the plan
 * records the kernel's built-in order. One plan serves every attention call
 * over the same offsets, q_len and num_heads (e.g. all DCA layers of a
 * batch). Errors: negative sizes, q_len or num_heads < 1, NULL pointers
 * (ROCS_ERR_INVALID_ARGUMENT); too small a plan (ROCS_ERR_WORKSPACE_TOO_SMALL);
 * (R + ceil(N q_len / 128)) num_heads >= 2^24 (ROCS_ERR_UNSUPPORTED).
 *
 * rocs_dca_attention_plan_size: bytes of the plan for R requests (0 for a
 * negative R or R >= 2^31).
 * ---------------------------------------------------------------------------
 */
size_t rocs_dca_attention_plan_size(int64_t num_requests);
int32_t rocs_dca_attention_plan(const int32_t* cand_offsets, const int32_t* kv_offsets,
                                int64_t num_requests, int64_t num_cand, int32_t q_len,
                                int32_t num_heads, void* plan, size_t plan_bytes,
                                void* stream);

/*
 * ---------------------------------------------------------------------------
 * rocs_dca_attention_mapped: rocs_dca_attention with the index map m given as
 * a per-candidate request id (Section 4.3.1: the kernel resolves m_i before
 * loading candidate i's K/V; here m need not keep a request's candidates
 * contiguous).
 *
 *   cand_request_ids [N] int32, device memory, each in [0, R) (trusted; an
 *                    id outside the range is clamped into it, so it gives
 *                    wrong rows, never an access outside kv_offsets).
 *   workspace        device memory of at least
 *                    rocs_dca_attention_mapped_workspace_size(R, N) bytes,
 *                    256-byte aligned (may be NULL when that size is 0 or the
 *                    general kernel runs). Contents on entry are ignored. On
 *                    return, when the tiled kernel ran, it holds the grouping
 *                    described below at offset 0: grp_off [R + 1] int32, then,
 *                    at the next 256-byte boundary, order [N] int32.
 * Every other argument, the result and the errors are those of
 * rocs_dca_attention.
 *
 * IKBO form on the fast path (the conditions of rocs_dca_attention): the
 * candidates are first grouped by request on the device, a stable counting
 * sort: order[p] lists request 0's candidates, then request 1's, ..., each
 * request's in their original order, and grp_off are the CSR offsets of that
 * order. The tiled kernel then runs on the grouped order, gathering query
 * rows and scattering output rows through `order`, so each request's K/V
 * is read once per tile of its candidates. This needs R <= 16384 and
 * R * ceil(N / G) <= 2^20 for a block size G of at least 4096 (the
 * workspace size is 0 otherwise). Other calls run the general kernel (one
 * wave per query row and head, history read through L2), which needs no
 * workspace.
 * ---------------------------------------------------------------------------
 */
size_t rocs_dca_attention_mapped_workspace_size(int64_t num_requests, int64_t num_cand);

int32_t rocs_dca_attention_mapped(const void* q, const void* k, const void* v,
                                  const int32_t* cand_request_ids, const int32_t* kv_offsets,
                                  int64_t num_requests, int64_t num_cand,
                                  int32_t q_len, int32_t num_heads, int32_t head_dim,
                                  int64_t kv_row_stride, float softmax_scale, int32_t dtype,
                                  void* out, void* workspace, size_t workspace_bytes,
                                  void* stream);

/*
 * ---------------------------------------------------------------------------
 * rocs_glm_interaction: the two-group GLM-masked factorization machine
 * (Eq. glm-fm, two-group form Eq. glm-fm-two-groups).
 *
 *   y_req[r]  = X^R_r (X^R_r)^T                      once per request,
 *               [F_r, F_r] flattened row-major        -> [R, F_r * F_r]
 *   y_cand[n] = [ X^C_n (X^R_{m_n})^T | X^C_n (X^C_n)^T ]  per candidate,
 *               [F_c, F_r + F_c] flattened row-major  -> [N, F_c * (F_r + F_c)]
 * The masked request-row/candidate-column block is structurally zero and is
 * not produced.
 *
 *   x_req  [R, f_req, emb_dim]     x_cand [N, f_cand, emb_dim]
 *   y_req  output or NULL (skip);  y_cand output or NULL (skip)
 *
 * Fast path (bf16 MFMA kernel): bf16, f_req a multiple of 16, f_cand in
 * {2, 4, 8, 16}, emb_dim a multiple of 32, pointers 16-byte aligned. Other
 * cases run a general kernel.
 * ---------------------------------------------------------------------------
 */
int32_t rocs_glm_interaction(const void* x_req, const void* x_cand,
                             const int32_t* cand_offsets,
                             int64_t num_requests, int64_t num_cand,
                             int32_t f_req, int32_t f_cand, int32_t emb_dim,
                             int32_t dtype, void* y_req, void* y_cand, void* stream);

/*
 * ---------------------------------------------------------------------------
 * rocs_ikbo_lcb: the two-group GLM linear compression block (Eq. glm-lcb,
 * Eq. glm-lcb-two-groups): the field (row) axis of embedding matrices is
 * mixed, block lower-triangularly.
 *
 *   y_req[r]  = W_RR X^R_r                      [o_req, emb]   once per request
 *   y_cand[n] = W_CR X^R_{m_n} + W_CC X^C_n     [o_cand, emb]  per candidate
 *
 * IKBO form (Section 4.1, 4.2): one launch at batch size R forms y_req and
 * Z_r = W_CR X^R_r (fp32, in the workspace) from the stacked weight
 * [W_RR; W_CR]; the candidate kernel adds Z_{m_n} to W_CC X^C_n in its
 * accumulators. No candidate-batched copy of X^R or Z is formed.
 *
 *   x_req   [R, f_req, emb_dim]       x_cand [N, f_cand, emb_dim]
 *   w_rr    [o_req, f_req] (ignored when o_req == 0 or y_req is NULL)
 *   w_cr    [o_cand, f_req]           w_cc   [o_cand, f_cand]
 *   cand_offsets [R + 1]
 *   y_req   [R, o_req, emb_dim] or NULL (request-side output skipped)
 *   y_cand  [N, o_cand, emb_dim]
 *   workspace  at least rocs_ikbo_lcb_workspace_size(R, o_cand, emb_dim) bytes,
 *              256-byte aligned; scratch on return.
 * No bias and no activation (the paper's LCB has neither); outputs do not
 * overlap inputs, each other or the workspace.
 *
 * Fast path (bf16 MFMA candidate kernel): bf16, f_cand in {16, 32, 64}, and
 * (emb_dim, o_cand) in {(128, 32), (64, 32), (64, 64)}, x_cand and y_cand
 * 16-byte, w_cc, x_req and y_req 8-byte aligned. Other cases run a general
 * kernel.
 * ---------------------------------------------------------------------------
 */
size_t rocs_ikbo_lcb_workspace_size(int64_t num_requests, int64_t o_cand, int64_t emb_dim);

int32_t rocs_ikbo_lcb(const void* x_req, const void* x_cand,
                      const void* w_rr, const void* w_cr, const void* w_cc,
                      const int32_t* cand_offsets, int64_t num_requests, int64_t num_cand,
                      int32_t f_req, int32_t f_cand, int32_t o_req, int32_t o_cand,
                      int32_t emb_dim, int32_t dtype, void* y_req, void* y_cand,
                      void* workspace, size_t workspace_bytes, void* stream);

/*
 * rocs_ikbo_lcb_mapped: rocs_ikbo_lcb with m given as a per-candidate request
 * id (cand_request_ids [N] int32, each in [0, R); an id outside the range is
 * clamped into it, never read out of bounds). Same kernels, same fast path.
 */
int32_t rocs_ikbo_lcb_mapped(const void* x_req, const void* x_cand,
                             const void* w_rr, const void* w_cr, const void* w_cc,
                             const int32_t* cand_request_ids, int64_t num_requests,
                             int64_t num_cand, int32_t f_req, int32_t f_cand, int32_t o_req,
                             int32_t o_cand, int32_t emb_dim, int32_t dtype, void* y_req,
                             void* y_cand, void* workspace, size_t workspace_bytes,
                             void* stream);

/*
 * ---------------------------------------------------------------------------
 * rocs_ikbo_mlp2: two stacked GLM linear layers on the candidate group, the
 * first with the request broadcast (Eq. glm-linear; a composition of
 * GLM-compliant layers stays compliant, Section 3.1):
 *
 *   H[n]   = act1(W1_CR x^R_{m_n} + W1_CC x^C_n + b1)     [d_hidden]
 *   out[n] = act2(W2 H[n] + b2)                           [d_out]
 *
 * H is rounded to the storage dtype before the second product (bf16: RNE),
 * the same rounding as two separate rocs_ikbo_linear calls. IKBO form: the
 * request table Zb = x_req W1_CR^T + b1 (fp32, workspace) is formed once per
 * request; the fused candidate kernel keeps H on chip (no HBM round trip).
 *
 *   x_req   [R, k_req] (k_req may be 0: no request term; then x_req, w1_req
 *           and cand_offsets are not read)
 *   x_cand  [N, k_cand]
 *   w1_req  [d_hidden, k_req]      w1_cand [d_hidden, k_cand]    b1 [d_hidden] or NULL
 *   w2      [d_out, d_hidden]      b2 [d_out] or NULL
 *   cand_offsets [R + 1] CSR (validate with rocs_validate_offsets if untrusted)
 *   activation1, activation2: ROCS_ACT_NONE or ROCS_ACT_RELU
 *   out     [N, d_out], not overlapping any input or the workspace
 *   workspace  at least rocs_ikbo_mlp2_workspace_size(R, N, k_req, k_cand,
 *              d_hidden, d_out, dtype) bytes, 256-byte aligned; scratch on
 *              return. The size covers Zb, and for shapes without the fused
 *              kernel also H [N, d_hidden] and the index map.
 *
 * Fused kernel: bf16, k_cand in {128, 256}, d_out in {128, 256}, d_hidden a
 * multiple of 64 up to 1024, k_req a multiple of 8; it needs every pointer
 * 16-byte aligned (ROCS_ERR_INVALID_ARGUMENT otherwise). Other shapes and
 * fp32 run two launches of the linear kernels with H in the workspace.
 * ---------------------------------------------------------------------------
 */
size_t rocs_ikbo_mlp2_workspace_size(int64_t num_requests, int64_t num_cand, int64_t k_req,
                                     int64_t k_cand, int64_t d_hidden, int64_t d_out,
                                     int32_t dtype);

int32_t rocs_ikbo_mlp2(const void* x_req, int64_t k_req, const void* x_cand, int64_t k_cand,
                       const void* w1_req, const void* w1_cand, const float* b1,
                       const void* w2, const float* b2, const int32_t* cand_offsets,
                       int64_t num_requests, int64_t num_cand, int64_t d_hidden,
                       int64_t d_out, int32_t dtype, int32_t activation1,
                       int32_t activation2, void* out, void* workspace,
                       size_t workspace_bytes, void* stream);

/*
 * ---------------------------------------------------------------------------
 * rocs_glm_fm_linear: a GLM FM interaction (Eq. glm-fm-two-groups, flattened
 * as in rocs_glm_interaction) feeding a GLM linear (Eq. glm-linear); the
 * composition stays GLM-compliant (Section 3.1):
 *
 *   Y^R_r  = X^R_r (X^R_r)^T                                     [f_req^2]
 *   Y^C_n  = [X^C_n (X^R_{m_n})^T | X^C_n (X^C_n)^T]              [f_cand (f_req + f_cand)]
 *   out[n] = act(W_CR Y^R_{m_n} + W_CC Y^C_n + bias)             [d_out]
 *
 * Y^R and Y^C are rounded to the storage dtype before the linear (bf16:
 * RNE), the same rounding as rocs_glm_interaction followed by
 * rocs_ikbo_linear. IKBO form: Y^R and Zb = W_CR Y^R + bias (fp32) are formed
 * once per request in the workspace; the fused candidate kernel computes Y^C
 * in registers as the linear's operand, so Y^C never reaches HBM.
 *
 *   x_req  [R, f_req, emb_dim]       x_cand [N, f_cand, emb_dim]
 *   cand_offsets [R + 1] CSR
 *   w_req  [d_out, f_req^2]          w_cand [d_out, f_cand (f_req + f_cand)]
 *   bias   [d_out] fp32 or NULL;     activation ROCS_ACT_NONE or ROCS_ACT_RELU
 *   out    [N, d_out], not overlapping any input or the workspace
 *   workspace  at least rocs_glm_fm_linear_workspace_size(R, N, f_req, f_cand,
 *              emb_dim, d_out, dtype) bytes, 256-byte aligned; on return it
 *              holds Y^R (bf16 or fp32 [R, f_req^2]) at offset 0, the rest is
 *              scratch. For shapes without the fused kernel it also holds Y^C.
 *
 * Fused kernel: bf16, f_req = 32, f_cand = 8, emb_dim = 128, d_out a multiple
 * of 64 up to 4096; it needs x_req, x_cand, w_req, w_cand, bias and out
 * 16-byte aligned (ROCS_ERR_INVALID_ARGUMENT otherwise). Other shapes and
 * fp32 run the interaction and linear kernels one after the other.
 * ---------------------------------------------------------------------------
 */
size_t rocs_glm_fm_linear_workspace_size(int64_t num_requests, int64_t num_cand, int32_t f_req,
                                         int32_t f_cand, int32_t emb_dim, int64_t d_out,
                                         int32_t dtype);

int32_t rocs_glm_fm_linear(const void* x_req, const void* x_cand, const int32_t* cand_offsets,
                           int64_t num_requests, int64_t num_cand, int32_t f_req,
                           int32_t f_cand, int32_t emb_dim, const void* w_req,
                           const void* w_cand, const float* bias, int64_t d_out, int32_t dtype,
                           int32_t activation, void* out, void* workspace,
                           size_t workspace_bytes, void* stream);

/*
 * ---------------------------------------------------------------------------
 * Index-map helpers (Section 4.1, m in {0..B_r-1}^{B_c}).
 *
 * rocs_request_ids: out_ids[n] = m_n for n < N, computed on the device by the
 * same routine the linear kernel uses (exposed so index handling can be
 * checked bit-exactly). out_ids is [N] int32.
 *
 * rocs_validate_offsets: copies offsets [count] to the host (synchronising
 * `stream`) and checks offsets[0] == 0, non-decreasing, offsets[count-1] ==
 * total. Returns ROCS_OK or ROCS_ERR_INVALID_ARGUMENT.
 * ---------------------------------------------------------------------------
 */
int32_t rocs_request_ids(const int32_t* cand_offsets, int64_t num_requests,
                         int64_t num_cand, int32_t* out_ids, void* stream);

int32_t rocs_validate_offsets(const int32_t* offsets, int64_t count, int64_t total,
                              void* stream);

#ifdef __cplusplus
}
#endif

#endif /* ROCS_H */
