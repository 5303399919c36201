/*
 * flashdiff.h - C ABI of the region-sparse DiT denoising step on MI355X (gfx950).
 *
 * The method is FlashDiff (arXiv 2607.12121): the latent is split into patches
 * ("regions"); a gate decides per denoising step which regions are refined; the
 * diffusion transformer runs only on the tokens of active regions, which attend
 * to every token of their request with keys/values of skipped tokens taken from
 * a per-block cache; skipped regions keep their latent (or advance with their
 * cached drift).  One step is, in order:
 *
 *   fd_region_score   -> per-region activity score          (Sec. 3.2)
 *   fd_select         -> gate, active mask, token index list (eq. gate-weight)
 *   fd_gather         -> active latent rows, bf16
 *   fd_embed          -> hidden rows
 *   fd_block_forward  -> one adaLN DiT block, L times        (Sec. 4 Backend)
 *   fd_final          -> velocity rows
 *   fd_scatter_update -> Euler update of the latent          (eq. sf-update)
 *
 * Regions come from fd_partition, run once per request on its saliency map
 * after the warm-up steps (Sec. 3.1): its token->region map is what
 * fd_plan_build takes.
 *
 * With the paper's own gate signal, fd_region_importance runs after the block
 * chosen to supply the self-attention, and its Delta replaces the region score
 * at the next step's fd_select (Sec. 3.2, refinement importance).
 *
 * Conventions for every entry point:
 *  - Pointers named in "device" are HIP device pointers; all other pointers are
 *    host pointers.  All device buffers are owned by the caller; the library
 *    allocates no device memory and keeps no pointer after a call returns.
 *  - Calls enqueue work on `stream` and return without synchronising.  Results
 *    are valid in stream order.  Arguments are validated before anything is
 *    enqueued: on a non-zero status nothing was enqueued.
 *  - bf16 values are passed as uint16_t bit patterns (round-to-nearest-even).
 *  - Matrices are row-major.  Weight matrices are [out][in]: y = x W^T + b.
 *  - The active row count M is produced on the device by fd_select and read by
 *    later calls from the device pointer `m`; the host never needs it.  Row
 *    buffers are sized for the plan's token count N (the largest M).
 *  - Errors: FD_OK = 0; otherwise a status below, with a message available from
 *    fd_last_error() (thread-local, valid until the next call on the thread).
 *    Device-side faults surface at the caller's next synchronisation.
 */
#ifndef FLASHDIFF_H_
#define FLASHDIFF_H_

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef struct ihipStream_t* fd_stream_t; /* a hipStream_t; NULL = default stream */

typedef enum fd_status {
  FD_OK = 0,
  FD_E_ARG = 1,          /* null pointer, negative or inconsistent size       */
  FD_E_SHAPE = 2,        /* dims do not fit the plan or a workspace too small */
  FD_E_UNSUPPORTED = 3,  /* a size the kernels do not implement              */
  FD_E_HIP = 4           /* a HIP runtime call failed                         */
} fd_status;

/* Skip modes of fd_scatter_update. */
enum { FD_SKIP_FREEZE = 0, FD_SKIP_REUSE_DRIFT = 1 };

/*
 * Region plan: the patch decomposition of a batch of B requests (Appendix
 * "Setup and Notation": disjoint patches covering the latent), numbered
 * request-major.  Built once per batch on the host with fd_plan_build, copied
 * to the device by the caller, then described by this struct.
 *   region_ptr    device int32 [R+1]  tokens of region r are
 *   region_tokens device int32 [N]    region_tokens[region_ptr[r] .. region_ptr[r+1]), ascending
 *   region_req    device int32 [R]    request of every region
 *   token_region  device int32 [N]    region of every token
 *   req_tok_off   device int32 [B+1]  tokens of request b are [req_tok_off[b], req_tok_off[b+1])
 *   req_reg_off   device int32 [B+1]  regions of request b are [req_reg_off[b], req_reg_off[b+1])
 * The scalars are host values.
 */
typedef struct fd_plan {
  int32_t n_tokens;             /* N */
  int32_t n_regions;            /* R */
  int32_t n_requests;           /* B */
  int32_t max_region_tokens;    /* largest region */
  int32_t max_request_tokens;   /* largest request */
  const int32_t* region_ptr;
  const int32_t* region_tokens;
  const int32_t* region_req;
  const int32_t* token_region;
  const int32_t* req_tok_off;
  const int32_t* req_reg_off;
} fd_plan;

/* Model dimensions.  D = H * dh.  Supported: dh in {16, 64, 128}; D % 64 == 0;
 * F % 64 == 0; C % 16 == 0 and C <= 256. */
typedef struct fd_dims {
  int32_t C;   /* latent channels per token */
  int32_t D;   /* hidden size               */
  int32_t H;   /* attention heads           */
  int32_t dh;  /* head dim                  */
  int32_t F;   /* MLP hidden size           */
} fd_dims;

/* One DiT block's parameters (device).  w_* bf16 [out][in], b_* fp32 [out]. */
typedef struct fd_block_weights {
  const uint16_t* w_qkv; const float* b_qkv;   /* [3D][D], [3D]: q | k | v, heads contiguous */
  const uint16_t* w_o;   const float* b_o;     /* [D][D]                                     */
  const uint16_t* w_1;   const float* b_1;     /* [F][D]                                     */
  const uint16_t* w_2;   const float* b_2;     /* [D][F]                                     */
  const uint16_t* w_ada; const float* b_ada;   /* [6D][D]: shift1|scale1|gate1|shift2|scale2|gate2 */
  const float* mod;      /* optional [B][6D]: this block's modulation from fd_adaln; when
                            non-null, w_ada, b_ada and cond are not read (may be null) */
} fd_block_weights;

/* Final layer (device): adaLN (shift | scale) [2D][D] and output projection [C][D]. */
typedef struct fd_final_weights {
  const uint16_t* w_ada; const float* b_ada;
  const uint16_t* w_out; const float* b_out;
} fd_final_weights;

/* Gate parameters (eq. gate-weight, eq. forced-reactivation). */
typedef struct fd_gate {
  double eta;        /* additive floor of the normalised weight, >= 0      */
  int32_t max_skip;  /* K: forced active after K consecutive skips; 0 = off */
} fd_gate;

const char* fd_last_error(void);
const char* fd_version(void);

/* ---------------------------------------------------------------- plan (host)
 * Builds the CSR region plan from a token->region map.  Host only, no HIP call.
 *   token_region  host int32 [N]    global region id of every token, 0 <= id < R
 *   req_tok_off   host int32 [B+1]  request token ranges, req_tok_off[0] = 0
 * Requirements: every region is non-empty and lies inside one request; the
 * region ids of request b form the contiguous range [req_reg_off[b], req_reg_off[b+1]).
 * Outputs (host, caller-allocated): region_ptr [R+1], region_tokens [N],
 * region_req [R], req_reg_off [B+1]; *max_region_tokens and *max_request_tokens.
 * Returns FD_E_ARG when a requirement fails (outputs then undefined).
 */
fd_status fd_plan_build(int32_t n_tokens, int32_t n_regions, int32_t n_requests,
                        const int32_t* token_region, const int32_t* req_tok_off,
                        int32_t* region_ptr, int32_t* region_tokens, int32_t* region_req,
                        int32_t* req_reg_off, int32_t* max_region_tokens,
                        int32_t* max_request_tokens);

/* ---------------------------------------------------------------- score
 * Activity of every region (Sec. 3.2 Patch Gate, change signal; the activity is
 * the mean squared step-to-step latent delta):
 *   score[r] = sum_{u in region r, c < C} d^2 / (|r| * C),  d = fl32(x_cur - x_prev)
 * with d^2 and the sum in fp64.
 *   x_cur, x_prev  device fp32 [N][C] (must not alias each other's rows differently)
 *   score          device fp64 [R]  (output)
 *   ws             device scratch of fd_region_score_ws_size bytes, 256-byte aligned
 */
size_t fd_region_score_ws_size(const fd_plan* plan, int32_t C);
fd_status fd_region_score(const fd_plan* plan, int32_t C, const float* x_cur, const float* x_prev,
                          double* score, void* ws, size_t ws_bytes, fd_stream_t stream);

/*
 * The same region score for callers that cannot allocate device memory (code
 * under HIP graph capture, tight serving loops, harnesses that forbid
 * allocation): the partial sums live in a scratch array built into the library
 * (1 MiB per GPU, held until the process ends), so no workspace is passed and
 * nothing is allocated.  Arguments, layout and result as fd_region_score.
 * FD_E_UNSUPPORTED (nothing enqueued) when fd_region_score_ws_size(plan, C)
 * exceeds 1 MiB.  Every call on a GPU shares that GPU's scratch: calls that
 * overlap on one GPU (concurrent streams or threads) race and must be ordered
 * by the caller.  A call writes every partial it reads, so nothing left by an
 * earlier call needs clearing.
 */
fd_status fd_region_score_noalloc(const fd_plan* plan, int32_t C, const float* x_cur, const float* x_prev,
                                  double* score, fd_stream_t stream);

/* ---------------------------------------------------------------- select
 * Patch Gate for every region, then the active-token index list:
 *  1. frozen change (eq. delta-i): s~[r] = prev_active[r] ? score[r] : s~[r]
 *  2. D_b = sum over request b of (s~ + eta)                  (eq. gate-weight),
 *     the binary64 terms added one at a time in ascending region order
 *  3. skip iff fl(s~[r] + eta) < fl(eps[b] * D_b) * (1 - 2^-40), or eps[b] = +inf:
 *     the division-free form of w_r < eps; the band keeps every exact-arithmetic
 *     tie (w_r = eps) active whatever way D_b rounds; a NaN score compares false,
 *     so it is active (and a NaN in D_b leaves its whole request active)
 *  4. forced active if max_skip > 0 and skip_run[r] >= max_skip (eq. forced-reactivation)
 *  5. skip_run[r] = active ? 0 : skip_run[r] + 1
 *  6. idx = ascending ids of tokens whose region is active; cu_q[b] = number of
 *     those before request b; *m = cu_q[B].
 *   score        device fp64 [R]   (input)
 *   eps          device fp64 [B]   (input, >= 0 or +inf)
 *   s_tilde      device fp64 [R]   (in/out)
 *   skip_run     device int32 [R]  (in/out)
 *   prev_active  device uint8 [R]  (input; may alias active)
 *   active       device uint8 [R]  (output, 0/1)
 *   idx          device int32 [N]  (output; entries >= *m untouched)
 *   cu_q         device int32 [B+1] (output)
 *   m            device int32 [1]  (output)
 * Supported: R <= 4096, B <= 1024.
 */
fd_status fd_select(const fd_plan* plan, const double* score, const double* eps, fd_gate gate,
                    double* s_tilde, int32_t* skip_run, const uint8_t* prev_active, uint8_t* active,
                    int32_t* idx, int32_t* cu_q, int32_t* m, fd_stream_t stream);

/* ---------------------------------------------------------------- gather
 * The restriction of the latent to the active patches (App. "Setup and
 * Notation": x^(i), the latent restricted to patch P_i; the update rule
 * evaluates the network only for i in the active set A_n; Sec. 4 Backend:
 * workers execute their assigned patches), as the network's bf16 input rows:
 * xa[i][c] = bf16(x_cur[idx[i]][c]) for i < *m (round to nearest even).
 *   x_cur device fp32 [N][C]; idx device int32 [N]; m device int32 [1];
 *   xa device bf16 [N][C] (rows >= *m untouched).
 */
fd_status fd_gather(const fd_plan* plan, int32_t C, const float* x_cur, const int32_t* idx,
                    const int32_t* m, uint16_t* xa, fd_stream_t stream);

/* ---------------------------------------------------------------- embed
 * Token embedding of the DiT backbone (Sec. 2.1: the served models are
 * Diffusion Transformers over latent tokens; the paper gives no block, this is
 * the standard DiT patch embedding with a learned position table), on the
 * active rows only:
 * h[i] = xa[i] W_e^T + b_e + pos[idx[i]] for i < *m (fp32 accumulate).
 *   xa device bf16 [N][C]; w_e device bf16 [D][C]; b_e device fp32 [D];
 *   pos device fp32 [N][D] (position table of every token); h device fp32 [N][D].
 */
fd_status fd_embed(const fd_plan* plan, const fd_dims* dims, const uint16_t* xa, const uint16_t* w_e,
                   const float* b_e, const float* pos, const int32_t* idx, const int32_t* m,
                   float* h, fd_stream_t stream);

/* ---------------------------------------------------------------- adaLN
 * The conditioning of the DiT blocks (Sec. 2.1 DiT backbone; standard adaLN
 * DiT block, which the paper does not spell out): modulation of n_blocks
 * stacked blocks in one pass over their weights:
 *   mod[l][b][j] = sum_k W[l][j][k] * SiLU(cond[b][k]) + bias[l][j],  j < n_out
 * (the adaLN conditioning of the DiT blocks; it depends on cond only, so the
 * modulation of every block of a step can be formed before the first block).
 *   w_ada  device bf16 [n_blocks][n_out][D] (D = dims->D), 16-byte aligned
 *   b_ada  device fp32 [n_blocks][n_out]
 *   cond   device fp32 [n_requests][D], 16-byte aligned
 *   mod    device fp32 [n_blocks][n_requests][n_out] (output)
 * Errors: FD_E_ARG for null or misaligned pointers or non-positive counts.
 */
fd_status fd_adaln(const fd_dims* dims, int32_t n_blocks, int32_t n_out, int32_t n_requests,
                   const uint16_t* w_ada, const float* b_ada, const float* cond, float* mod,
                   fd_stream_t stream);

/* ---------------------------------------------------------------- block
 * One adaLN DiT block on the active rows (Sec. 4 Backend: active patches run
 * with the K/V cache; Prop. "Stale-KV Perturbation"):
 *   (shift1, scale1, gate1, shift2, scale2, gate2) = SiLU(cond_b) W_ada^T + b_ada
 *   a   = bf16(LN(h) * (1 + scale1) + shift1)          LN: eps 1e-6, no affine
 *   q,k,v = a W_qkv^T + b_qkv; k, v are written (bf16) to k_cache/v_cache at
 *         rows idx[i] before attention
 *   o_i = softmax(q_i K_b^T / sqrt(dh)) V_b per head, over all tokens of the
 *         row's request b (rows of skipped tokens are the cached, stale ones)
 *   h  += gate1 * (o W_o^T + b_o)
 *   a   = bf16(LN(h) * (1 + scale2) + shift2)
 *   h  += gate2 * (GELU_tanh(a W_1^T + b_1) W_2^T + b_2)
 *   cond     device fp32 [B][D] (not read when w->mod is given)
 *   h        device fp32 [N][D], rows < *m updated in place
 *   idx, cu_q, m  from fd_select
 *   k_cache, v_cache  device bf16 [N][D] of this block (head h at columns h*dh..)
 *   ws       device scratch of fd_block_ws_size bytes, 256-byte aligned; after
 *            the call it holds this block's queries and per-query softmax
 *            normalisers, which fd_region_importance reads
 * Errors: FD_E_UNSUPPORTED for plans of more than 1024 requests (the limit of
 * fd_select as well), FD_E_SHAPE for dims that do not fit or a small workspace.
 */
size_t fd_block_ws_size(const fd_plan* plan, const fd_dims* dims);
fd_status fd_block_forward(const fd_plan* plan, const fd_dims* dims, const fd_block_weights* w,
                           const float* cond, float* h, const int32_t* idx, const int32_t* cu_q,
                           const int32_t* m, uint16_t* k_cache, uint16_t* v_cache, void* ws,
                           size_t ws_bytes, fd_stream_t stream);

/* ---------------------------------------------------------------- importance
 * The Patch Gate's own signal (Sec. 3.2, refinement importance, Alg. 1
 * PatchGate): for every active region i,
 *   R_i = |A_i|^-2 sum_{u,v in A_i} SA_uv,
 * SA the self-attention matrix of one block averaged over its H heads (SA_uv =
 * mean_h softmax over the tokens of u's request); then Delta_i = |R_i - Rbar_i|
 * and Rbar_i = R_i.  Skipped regions keep Rbar and Delta (their queries do not
 * run).  Passing Delta as `score` to the next step's fd_select gates on it.
 * Call right after fd_block_forward of the chosen block, with the workspace
 * that call used: it reads that call's queries and per-query softmax
 * normalisers from it, and the block's key cache as that call left it.
 *   block_ws, block_ws_bytes  device, the fd_block_forward workspace (not reused since)
 *   k_cache      device bf16 [N][D], the block's key cache
 *   idx, m       device, the active rows of fd_select
 *   active       device uint8 [R], this step's mask
 *   r_bar, delta device fp64 [R], updated in place (both 0 before the first step)
 *   importance   optional device fp64 [R]: R_i of active regions, NaN for skipped ones
 *   ws           device scratch of fd_importance_ws_size bytes, 256-byte aligned
 * FD_E_UNSUPPORTED when a region's key rows of one head exceed 156 KB of LDS.
 */
size_t fd_importance_ws_size(const fd_plan* plan, const fd_dims* dims);
fd_status fd_region_importance(const fd_plan* plan, const fd_dims* dims, const void* block_ws,
                               size_t block_ws_bytes, const uint16_t* k_cache, const int32_t* idx,
                               const int32_t* m, const uint8_t* active, double* r_bar, double* delta,
                               double* importance, void* ws, size_t ws_bytes, fd_stream_t stream);

/* ---------------------------------------------------------------- partition
 * Recursive load-aware patch partitioning (Sec. 3.1, Patch Partitioner; the
 * between-class variance of eq. otsu; the r_f allocation rule), run once per
 * request after the warm-up steps, before fd_plan_build.  For every request b
 * with n_b tokens and R_b regions, a node (initially all tokens, regions
 * [0, R_b)) is split into focus = {saliency >= theta} and context = the rest,
 * theta the distinct saliency value (all but the smallest) maximising
 *   sigma_B^2 = w_f w_c (mu_f - mu_c)^2,  w = class count / node count,
 * evaluated in fp64 from exact integer class counts and sums as
 * w_f * w_c * ((S_f / n_f - S_c / n_c)^2), ties to the smaller theta.  The focus
 * set gets the first r_f of the node's R regions, r_f the r in 1 .. R-1 nearest
 * to R n_f / (n_f + n_c) (ties to the smaller), clamped to
 * [max(1, R - n_c), min(R - 1, n_f)]; the context set gets the other R - r_f.
 * Nodes are split until each holds one region.  A node whose tokens share one
 * saliency value is cut into its R regions by token index: the token of rank k
 * (in index order) among its n tokens gets region first + floor(k R / n).
 *   n_requests   1 .. 64 requests per call
 *   req_tok_off  host int32 [B+1]  request token ranges, req_tok_off[0] = 0
 *   req_reg_off  host int32 [B+1]  request region ranges, req_reg_off[0] = 0
 *   saliency     device uint16 [N] integer saliency of every token (the
 *                request's quantised saliency map, any 16-bit values)
 *   token_region device int32 [N]  output: global region id of every token,
 *                req_reg_off[b] <= id < req_reg_off[b+1] for request b; the
 *                token_region input of fd_plan_build
 *   ws           device scratch of fd_partition_ws_size(N, B) bytes, 256-byte aligned
 * Requirements: 1 <= R_b <= n_b for every request (FD_E_ARG otherwise);
 * n_b <= 65535 and R_b <= 1024 (FD_E_UNSUPPORTED otherwise).  One workgroup
 * per request runs the whole recursion in one launch.
 */
size_t fd_partition_ws_size(int32_t n_tokens, int32_t n_requests);
fd_status fd_partition(int32_t n_requests, const int32_t* req_tok_off, const int32_t* req_reg_off,
                       const uint16_t* saliency, int32_t* token_region, void* ws, size_t ws_bytes,
                       fd_stream_t stream);

/* ---------------------------------------------------------------- final
 * The network output f_theta^(i)(x_n, t_n) of the active patches (App. "Setup
 * and Notation", FlashDiff update rule), through the standard DiT final layer:
 * v[i] = (LN(h_i) * (1 + scale) + shift) W_out^T + b_out, (shift, scale) =
 * SiLU(cond_b) W_ada^T + b_ada, for i < *m.  v device fp32 [N][C].
 * ws: device scratch of fd_block_ws_size bytes (the same size suffices).
 */
fd_status fd_final(const fd_plan* plan, const fd_dims* dims, const fd_final_weights* w,
                   const float* cond, const float* h, const int32_t* cu_q, const int32_t* m,
                   float* v, void* ws, size_t ws_bytes, fd_stream_t stream);

/* ---------------------------------------------------------------- update
 * Euler update of eq. sf-update on the fp32 latent x (in place), h_b = dt[b]:
 *   active token u = idx[i]:  x[u] = fl32(x[u] + fl32(dt_b * v[i])); vcache[u] = v[i]
 *   skipped token u:          FD_SKIP_FREEZE: untouched
 *                             FD_SKIP_REUSE_DRIFT: x[u] = fl32(x[u] + fl32(dt_b * vcache[u]))
 * No fused multiply-add is used.
 *   x device fp32 [N][C]; v device fp32 [N][C] (rows < *m); dt device fp32 [B];
 *   vcache device fp32 [N][C] (cached drift); active device uint8 [R] from fd_select.
 */
fd_status fd_scatter_update(const fd_plan* plan, int32_t C, float* x, const float* v,
                            const int32_t* idx, const int32_t* m, const float* dt, float* vcache,
                            const uint8_t* active, int32_t skip_mode, fd_stream_t stream);

/* ---------------------------------------------------------------- timing
 * Kernel timer for measurement: while armed for `kernel`, every launch of that
 * kernel records a pair of HIP events around it on its stream (up to
 * `capacity` launches).  The events carry no system-scope memory fence, so
 * arming the timer does not stall the stream around the timed kernel.
 * fd_timer_read synchronises on the recorded events and writes each launch's
 * duration in milliseconds; it returns the count.  The timer is the library's
 * only process-wide state (one per process, guarded by a mutex, measurement
 * only): while it is armed, the matching launches of every thread are timed.
 */
enum {
  FD_K_SCORE = 1, FD_K_SELECT, FD_K_GATHER, FD_K_EMBED, FD_K_ADALN, FD_K_LN,
  FD_K_GEMM_QKV, FD_K_ATTN, FD_K_GEMM_O, FD_K_GEMM_MLP1, FD_K_GEMM_MLP2,
  FD_K_FINAL, FD_K_SCATTER, FD_K_IMPORTANCE, FD_K_PARTITION
};
fd_status fd_timer_arm(int32_t kernel, int32_t capacity);
int32_t fd_timer_read(float* ms, int32_t capacity);
void fd_timer_disarm(void);

#ifdef __cplusplus
}
#endif
#endif /* FLASHDIFF_H_ */
