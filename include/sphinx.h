/*
 * sphinx.h -- C ABI of the selective partial-denoising step on AMD Instinct
 * MI355X (gfx950).
 *
 * The library implements the inner loop of Sphinx's inference algorithm
 * (Sphinx, arXiv 2511.18672, Alg. 1 "Sphinx Inference", partial-denoising
 * loop; Sec. 5.3 spatially selective refinement): a per-token uncertainty map
 * is thresholded into a binary mask, the selected latent tokens are
 * stream-compacted and gathered with noise injected at the frame's start step,
 * the transformer denoiser runs on the gathered tokens only, the DDIM update is
 * applied, and the result is scattered back while unselected tokens keep their
 * values.  Sampler, schedule and denoiser architecture are not fixed by the
 * paper; the library uses deterministic DDIM (eta = 0, eps-prediction), a
 * linear beta schedule 1e-4..2e-2 over 1000 steps and a DiT-style adaLN
 * transformer with joint attention over the selected tokens of each request.
 *
 * Conventions shared by every call
 * --------------------------------
 *  - Plain C types only.  Pointers marked "dev" are device (HBM) pointers,
 *    "host" are host pointers.  `stream` is a hipStream_t passed as void*
 *    (NULL = the default stream).  Every call only enqueues work on `stream`
 *    unless stated otherwise.
 *  - The caller owns every buffer.  No call allocates device memory; scratch
 *    space comes from a caller-provided workspace whose size a *_bytes query
 *    returns.  Device pointers must be 16-byte aligned.
 *  - Requests are concatenated.  Request r covers global tokens
 *    [tok_offset, tok_offset + frames*(h/2)*(w/2)) and global frames
 *    [frame_offset, frame_offset + frames); both offsets must equal the running
 *    sums over the preceding requests.  At most SPHINX_MAX_REQUESTS requests.
 *  - Token t of a request is t = f*(h/2)*(w/2) + y*(w/2) + x (patch 2x2).
 *    A token's 16 values are ordered c*4 + py*2 + px.  Latents come in one of
 *    two layouts (sphinx_layout), both 16*N elements with request r starting
 *    at element 16*tok_offset:
 *      SPHINX_LAYOUT_NCHW    per request [frames][4][h][w] (the VAE's layout);
 *      SPHINX_LAYOUT_TOKENS  [N][16]: token t's 16 values at 16*t, the layout
 *                            of an x_sel row, so gathering or scattering a
 *                            token moves one contiguous 64-byte row (f32).
 *  - Arguments are validated before any HIP call, so every error path is
 *    reachable without a GPU; an invalid call enqueues nothing.  No exception
 *    or abort crosses the ABI.  SPHINX_E_HIP reports a failed launch or copy.
 */
#ifndef SPHINX_H
#define SPHINX_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

/* The enumerations below are 32-bit values at the ABI.  In C++ they take
 * int32_t as their fixed underlying type, so every int32 a caller passes is a
 * representable value that the library can reject (out-of-range values return
 * SPHINX_E_INVALID or "unknown status"), never an undefined enum load. */
#ifdef __cplusplus
#define SPHINX_ENUM enum : int32_t
#else
#define SPHINX_ENUM enum
#endif

#define SPHINX_MAX_REQUESTS 64
#define SPHINX_TOKEN_DIM 16 /* 4 latent channels x 2 x 2 patch */
#define SPHINX_TEMB_DIM 256 /* sinusoidal timestep embedding width */
#define SPHINX_TRAIN_STEPS 1000

typedef SPHINX_ENUM {
  SPHINX_OK = 0,
  SPHINX_E_INVALID = 1,     /* null required pointer, bad size, misalignment, inconsistent offsets */
  SPHINX_E_UNSUPPORTED = 2, /* valid but not implemented (head_dim, dtype, sizes) */
  SPHINX_E_WORKSPACE = 3,   /* workspace too small */
  SPHINX_E_HIP = 4          /* a HIP launch or copy failed */
} sphinx_status;

typedef SPHINX_ENUM { SPHINX_F32 = 0, SPHINX_BF16 = 1 } sphinx_dtype;

typedef SPHINX_ENUM { SPHINX_LAYOUT_NCHW = 0, SPHINX_LAYOUT_TOKENS = 1 } sphinx_layout;

/* Attention of the denoiser blocks.  JOINT: every block attends over the
 * request's tokens.  FACTORISED (the spatial / temporal split of the paper's
 * video denoisers, Sec. 4 and Sec. 5.2): even blocks attend within a frame,
 * odd blocks across the request's frames at the same (y, x) position.  A
 * factorised model supports at most SPHINX_MAX_REQUESTS frames in a call and
 * 64 frames per request (fp32 models: head_dim a multiple of 4).  Its spatial
 * blocks need the forwarded rows per frame on the host: a refine call on a
 * factorised model synchronizes its stream once to read them, and requires
 * idx in ascending order (as sphinx_select_mask produces). */
typedef SPHINX_ENUM { SPHINX_ATTN_JOINT = 0, SPHINX_ATTN_FACTORISED = 1 } sphinx_attention;

/* Timestep grids of frames with different start indices (Alg. 1 per-frame
 * start): SHARED walks one grid per request from the largest start and lets a
 * frame join when the grid reaches its start; PER_FRAME walks every frame's
 * own n-step grid from its own start, all frames active from the first step. */
typedef SPHINX_ENUM { SPHINX_GRID_SHARED = 0, SPHINX_GRID_PER_FRAME = 1 } sphinx_grid;

typedef struct {
  int32_t frames;       /* F >= 1 */
  int32_t h, w;         /* latent height and width, even, h/2 and w/2 <= 1024 */
  int32_t frame_offset; /* first global frame of the request */
  int64_t tok_offset;   /* first global token of the request */
} sphinx_request;

/* Denoiser description.  `weights` is a caller-owned device blob whose layout
 * sphinx_model_param() defines; it is only read. */
typedef struct {
  int32_t D;        /* hidden size, = heads * head_dim */
  int32_t heads;
  int32_t head_dim; /* 64 or 72 for bf16 models; up to 64 for f32 models */
  int32_t mlp;      /* MLP hidden size */
  int32_t L;        /* number of blocks */
  sphinx_dtype dtype; /* storage and GEMM-operand type of weights/activations */
  sphinx_attention attention; /* block attention pattern */
  const void* weights; /* dev */
} sphinx_model_desc;

/* Parameter tensors of the blob.  Matrices are row-major [out][in]
 * (y = x W^T + b).  The adaLN projections of all blocks and the final adaLN
 * projection are stored as one matrix COND_W [(6L+2)D][D]: rows
 * [6D*l, 6D*(l+1)) belong to block l and give (shift1, scale1, gate1, shift2,
 * scale2, gate2); the last 2D rows give the final (shift, scale). */
typedef SPHINX_ENUM {
  SPHINX_P_PE_W = 0,  /* [D][16]     patch embedding */
  SPHINX_P_PE_B,      /* [D] */
  SPHINX_P_T1_W,      /* [D][256]    timestep MLP, first layer */
  SPHINX_P_T1_B,      /* [D] */
  SPHINX_P_T2_W,      /* [D][D]      timestep MLP, second layer */
  SPHINX_P_T2_B,      /* [D] */
  SPHINX_P_COND_W,    /* [(6L+2)D][D] adaLN projections, all blocks + final */
  SPHINX_P_COND_B,    /* [(6L+2)D] */
  SPHINX_P_QKV_W,     /* per block [3D][D] */
  SPHINX_P_QKV_B,     /* per block [3D] */
  SPHINX_P_O_W,       /* per block [D][D] */
  SPHINX_P_O_B,       /* per block [D] */
  SPHINX_P_FC1_W,     /* per block [mlp][D] */
  SPHINX_P_FC1_B,     /* per block [mlp] */
  SPHINX_P_FC2_W,     /* per block [D][mlp] */
  SPHINX_P_FC2_B,     /* per block [D] */
  SPHINX_P_OUT_W,     /* [16][D]     final projection to the noise prediction */
  SPHINX_P_OUT_B,     /* [16] */
  SPHINX_P_COUNT
} sphinx_param;

/* Human-readable name of a status code (static string). */
const char* sphinx_status_string(sphinx_status s);

/* Total blob size in bytes for a model description (weights pointer ignored). */
sphinx_status sphinx_model_blob_bytes(const sphinx_model_desc* m, size_t* bytes);

/* Byte offset and element count of parameter `p` (of block `block` for the
 * per-block tensors, block ignored otherwise).  Every tensor starts on a
 * 256-byte boundary; elements have the model dtype. */
sphinx_status sphinx_model_param(const sphinx_model_desc* m, sphinx_param p, int32_t block,
                                 size_t* offset_bytes, size_t* count);

/* Schedule of step `step` (0-based) for all frames, computed on the host in
 * double precision (Alg. 1 partial-denoising loop with per-frame start steps).
 * Request r walks the timestep grid tau_i = floor((n-i)(s+1)/n) - 1,
 * i = 0..n (n = nsteps[r], s = the largest start index among its frames),
 * with alpha_bar(-1) = 1.  Frame f is active at step i iff tau_i <= s_f and
 * i < n; on its first active step it is newly active and add_noise applies
 * a = sqrt(abar(tau_i)), b = sqrt(1 - abar(tau_i)); otherwise a = 1, b = 0.
 * The DDIM coefficients of the step are c1 = sqrt(abar'/abar) and
 * c2 = sqrt(1-abar') - sqrt(abar'(1-abar)/abar) with abar = abar(tau_i),
 * abar' = abar(tau_{i+1}).  Outputs are host arrays [G] (G = total frames):
 * active/newly (0/1), tau (timestep fed to the denoiser), a, b, c1, c2.
 * Inactive frames get tau of their request's step (or -1 when the request has
 * finished), a = 1, b = 0, c1 = 1, c2 = 0.  Pure host code. */
sphinx_status sphinx_plan_step(const sphinx_request* reqs, int32_t R, const int32_t* s_start /*host[G]*/,
                               const int32_t* nsteps /*host[R]*/, int32_t step, uint8_t* active,
                               uint8_t* newly, int32_t* tau, float* a, float* b, float* c1, float* c2);

/* sphinx_plan_step with a choice of grid.  SPHINX_GRID_SHARED is
 * sphinx_plan_step.  SPHINX_GRID_PER_FRAME: frame f of a live request walks
 * tau_i = floor((n-i)(s_f+1)/n) - 1 from its own start s_f; it is active at
 * every step i < n, newly active at i = 0 (a = sqrt(abar(s_f)), b =
 * sqrt(1 - abar(s_f))), and its DDIM coefficients use its own tau_i, tau_{i+1}. */
sphinx_status sphinx_plan_step_grid(const sphinx_request* reqs, int32_t R, const int32_t* s_start,
                                    const int32_t* nsteps, int32_t step, sphinx_grid grid, uint8_t* active,
                                    uint8_t* newly, int32_t* tau, float* a, float* b, float* c1, float* c2);

/* Adaptive start steps (Sec. 5.1, Eq. 2 and the k-decision logic; Alg. 1
 * k <- K_c(r), k_min <- min(k)).  Pure host code, double precision.
 *   Frame f of request r (F frames) is target f+1 of F, at t = (f+1)/(F+1).
 *   Reference quality (Eq. 2): Q* = c0 + (c1 - c0) * (t^gamma if c1 >= c0,
 *   else 1 - (1-t)^gamma), with c0 = q_in[2r], c1 = q_in[2r+1] the quality
 *   scores of the request's two input views.
 *   Ratio r_f = q_reg[g] / Q*; start step k_f = table.k[i] with i the number
 *   of breakpoints table.ratio[] <= r_f, using table tables[cluster[r]].
 *   Outputs: k[g], the start index s[g] = round(1000 (S - k)/S) - 1 (half up;
 *   the t_start = 1 - k/S of the plan), nsteps[r] = S - min over the request's
 *   frames of k (the loop from k_min to S-1), and optionally ratio[g].
 * With s_start = s and these nsteps, sphinx_plan_step activates frame f at
 * loop step u = k_f (Alg. 1 A_u = 1[k <= u]) when 1000 is a multiple of S.
 * Requirements: gamma in (0, 1]; 1 <= S <= 1000; every table has 0..15
 * strictly increasing finite breakpoints and n+1 non-decreasing k in
 * [0, S-1]; cluster[r] in [0, n_tables); c0, c1 > 0 and q_reg >= 0 finite. */
#define SPHINX_KLOGIC_MAX 15
typedef struct {
  int32_t n;                          /* number of breakpoints */
  float ratio[SPHINX_KLOGIC_MAX];     /* breakpoints of the quality ratio */
  int32_t k[SPHINX_KLOGIC_MAX + 1];   /* start step below ratio[0], ..., at or above ratio[n-1] */
} sphinx_klogic;

sphinx_status sphinx_adaptive_start(const sphinx_request* reqs, int32_t R, const float* q_in /*host[2R]*/,
                                    const float* q_reg /*host[G]*/, float gamma, const sphinx_klogic* tables,
                                    int32_t n_tables, const int32_t* cluster /*host[R]*/, int32_t S,
                                    int32_t* k /*host[G]*/, int32_t* s_start /*host[G]*/,
                                    int32_t* nsteps /*host[R]*/, double* ratio /*host[G] or NULL*/);

/* Workspace bytes needed by sphinx_select_mask for N tokens. */
sphinx_status sphinx_select_workspace_bytes(int64_t N, size_t* bytes);

/* Selection mask and its stable compaction (Alg. 1 opacity mask
 * 1[O < tau_o] with u = -O; Sec. 5.3: only masked positions are forwarded).
 *   mask[t] = active[frame(t)] && (uncert[t] > thr[frame(t)])   (strict, NaN -> 0)
 *   idx[0..n_sel)  = the selected t in ascending order,
 *   cu_sel[r]      = number of selected tokens before request r, cu_sel[R] = n_sel.
 * uncert: dev float [N]; thr: dev float [G]; active: dev uint8 [G] or NULL (all
 * active); mask: dev uint8 [N] out; idx: dev int32 [N] out; cu_sel: dev int32
 * [R+1] out.  If cu_sel_host (host int32 [R+1]) is non-NULL the call copies
 * cu_sel back and synchronizes `stream` once (its only host synchronization).
 * Bit-exact and deterministic. */
sphinx_status sphinx_select_mask(const sphinx_request* reqs, int32_t R, const float* uncert, const float* thr,
                                 const uint8_t* active, uint8_t* mask, int32_t* idx, int32_t* cu_sel,
                                 int32_t* cu_sel_host, void* ws, size_t ws_bytes, void* stream);

/* sphinx_select_mask without a workspace argument, for callers that cannot
 * allocate device memory (code under HIP graph capture, tight serving loops,
 * harnesses that forbid allocation).  Same arguments, results and errors as
 * sphinx_select_mask, bit-identical outputs.  Its scratch (per-chunk counts
 * and offsets, 512 KB) is a static array of the library, one per GPU, held
 * until the process ends; the call allocates nothing.  N (all requests'
 * tokens) is limited to SPHINX_SELECT_STATIC_MAX_TOKENS; larger inputs return
 * SPHINX_E_UNSUPPORTED before any HIP call.  Calls on the same GPU share the
 * array: calls that overlap in time on one GPU (other streams, other threads)
 * race and must be serialised by the caller. */
#define SPHINX_SELECT_STATIC_MAX_TOKENS (1LL << 28)
sphinx_status sphinx_select_mask_static(const sphinx_request* reqs, int32_t R, const float* uncert,
                                        const float* thr, const uint8_t* active, uint8_t* mask, int32_t* idx,
                                        int32_t* cu_sel, int32_t* cu_sel_host, void* stream);

/* Gather with noise injection (Alg. 1 add_noise on the selected tokens).
 *   x_sel[j][k] = a[g] * z[k] + b[g] * eps[k]   for token idx[j] of frame g,
 * z and eps read from the latents `state` / `eps` (dtype f32 or bf16), both in
 * `layout`.  eps may be NULL: then the noise term is dropped.  a, b: dev float
 * [G]; idx: dev int32 [n_sel]; x_sel: dev float [n_sel][16] out.  n_sel = 0
 * is a no-op.  An idx[j] outside [0, N) leaves row j unwritten. */
sphinx_status sphinx_gather(const sphinx_request* reqs, int32_t R, sphinx_layout layout, const void* state,
                            sphinx_dtype state_dtype, const void* eps, sphinx_dtype eps_dtype, const int32_t* idx,
                            int32_t n_sel, const float* a, const float* b, float* x_sel, void* stream);

/* Workspace bytes of sphinx_refine_step for up to max_sel selected tokens. */
sphinx_status sphinx_refine_workspace_bytes(const sphinx_model_desc* m, const sphinx_request* reqs, int32_t R,
                                            int64_t max_sel, size_t* bytes);

/* One denoiser pass over the gathered tokens plus the DDIM update,
 * in place on x_sel (Alg. 1 D.partial_step on the masked tokens).
 *   eps_hat = Denoiser(x_sel, positions, tau);  x_sel <- c1[g] x_sel + c2[g] eps_hat
 * Attention is non-causal over the selected tokens of the same request:
 * rows [cu_sel_host[r], cu_sel_host[r+1]) form segment r.  idx: dev int32
 * [n_sel] (positions of the rows); tau: dev int32 [G] timestep per frame;
 * c1, c2: dev float [G]; x_sel: dev float [n_sel][16] in/out; cu_sel_host:
 * host int32 [R+1] with cu_sel_host[R] = n_sel.  n_sel = 0 is a no-op.
 * bf16 models compute GEMMs and attention with bf16 operands and fp32
 * accumulation; residual stream, statistics, softmax and the update are fp32.
 * SPHINX_E_UNSUPPORTED when n_sel * max(3 D, mlp) >= 2^31 (the activation
 * matrices are addressed with 32-bit element offsets). */
sphinx_status sphinx_refine_step(const sphinx_model_desc* m, const sphinx_request* reqs, int32_t R,
                                 const int32_t* idx, int32_t n_sel, const int32_t* cu_sel_host,
                                 const int32_t* tau, const float* c1, const float* c2, float* x_sel, void* ws,
                                 size_t ws_bytes, void* stream);

/* Varlen non-causal attention, the attention step of the denoiser blocks
 * (Alg. 1 D.partial_step on the masked tokens; joint attention over each
 * request's selected tokens), on its own.  Per segment i and head h:
 *   o[j] = sum_t 2^(q[j].k[t]) v[t] / sum_t 2^(q[j].k[t])
 * for query rows j in [cu_q[i], cu_q[i+1]) and key/value rows t in
 * [cu_kv[i], cu_kv[i+1]), head h using columns [h d, (h+1) d).  The softmax
 * is in base 2: q must already be multiplied by log2(e)/sqrt(d) (the layout
 * the denoiser's QKV projection writes), which makes this softmax(q k^T /
 * sqrt(d)) of the unscaled queries.
 *   dtype: SPHINX_BF16 (head_dim 64 or 72; P is rounded to bf16, accumulation
 *          fp32, o rounded to bf16) or SPHINX_F32 (head_dim <= 64).
 *   q: dev [rows][ldq] elements; k, v: dev [rows][ldkv]; o: dev, row j at
 *   element j * heads * head_dim (written for the query rows of the segments
 *   only).  cu_q, cu_kv: host int32 [nseg+1], non-decreasing from 0; empty
 *   segments are skipped; 1 <= nseg <= SPHINX_MAX_REQUESTS.  ldq, ldkv >=
 *   heads * head_dim and multiples of 8; pointers 16-byte aligned.  A segment
 *   with queries needs at least one key (SPHINX_E_INVALID otherwise). */
sphinx_status sphinx_varlen_attention(sphinx_dtype dtype, int32_t heads, int32_t head_dim, const void* q,
                                      int32_t ldq, const void* k, const void* v, int32_t ldkv, void* o,
                                      const int32_t* cu_q, const int32_t* cu_kv, int32_t nseg, void* stream);

/* Scatter and blend (Sec. 3 and 5.3: confident regions keep their values).
 *   z_out = z_in with token idx[j] replaced by x_sel[j]   (j < n_sel)
 * z_in == z_out scatters in place (dtype and layout must match); otherwise
 * z_in is first copied to z_out with dtype and layout conversion (bf16 outputs
 * round to nearest even), so n_sel = 0 converts between layouts and dtypes.
 * x_sel: dev float [n_sel][16]; z_in, z_out: dev latents of all requests in
 * the given layouts; the two buffers must not partially overlap.  An idx[j]
 * outside [0, N) is skipped. */
sphinx_status sphinx_scatter_blend(const sphinx_request* reqs, int32_t R, const float* x_sel, const int32_t* idx,
                                   int32_t n_sel, const void* z_in, sphinx_dtype in_dtype, sphinx_layout in_layout,
                                   void* z_out, sphinx_dtype out_dtype, sphinx_layout out_layout, void* stream);

/* ------------------------------------------------------------------------
 * Latent cache with periodic full steps (Sec. 5.2, temporally consistent
 * partial denoising; Alg. 1 full_step every T steps with store_temporal, and
 * partial_step that reads the cache).
 *
 * Every T-th step of a request (i mod T = 0, counting from its first step so
 * that the first step fills the cache) is a full step: every token of the
 * request is forwarded through the denoiser and every block's keys and values
 * are stored in the cache.  In the steps between, only the selected tokens
 * are forwarded; they store their fresh keys and values and attend over all
 * tokens of their request through the cache, so unselected tokens and
 * inactive frames take part as they were at the last full step.  The write
 * set (tokens whose state is updated) is the selection of sphinx_select_mask
 * in every step.  Tokens forwarded only as context enter as their clean
 * latent noised to the step's level, add_noise(z0, tau_i) (Alg. 1 resamples
 * inactive content from the clean latents); the state holds z0 there because
 * only write-set tokens are ever written.  The cache rows of a token hold the
 * keys and values last computed for it; when the selection only grows from
 * step to step (fixed thresholds, a growing active set) this equals "the last
 * full step" for every token not selected now.
 *
 * A step with the cache: sphinx_plan_step + sphinx_plan_cache (host);
 * sphinx_select_mask for the write set and, on a full step, a second
 * sphinx_select_mask with thr = -inf and active = forward_all for the
 * forwarded set; sphinx_gather_ctx; sphinx_refine_step_cached;
 * sphinx_scatter_masked.
 * ------------------------------------------------------------------------ */

/* Cache plan of step `step` for period T = `period` >= 1 (pure host code).
 * full: host uint8 [R], 1 iff request r is live at this step (step <
 * nsteps[r]) and step mod T = 0.  forward_all: host uint8 [G], full[r] of the
 * frame's request.  a_ctx, b_ctx: host float [G], the context coefficients
 * sqrt(abar(tau_i)), sqrt(1 - abar(tau_i)) of the request's current timestep
 * (1, 0 for a finished request), in double precision rounded to float;
 * with SPHINX_GRID_PER_FRAME the frame's own tau_i.  s_start and nsteps as for
 * sphinx_plan_step. */
sphinx_status sphinx_plan_cache(const sphinx_request* reqs, int32_t R, const int32_t* s_start,
                                const int32_t* nsteps, int32_t step, int32_t period, sphinx_grid grid,
                                uint8_t* full, uint8_t* forward_all, float* a_ctx, float* b_ctx);

/* Bytes of the latent cache: L blocks x N tokens x (key, value) x D elements
 * of the model dtype, laid out [L][N][2][D] (token t of block l at element
 * (l*N + t)*2D, its key first).  The caller owns and allocates it; rows that
 * no call has stored are read as whatever they hold. */
sphinx_status sphinx_kv_cache_bytes(const sphinx_model_desc* m, const sphinx_request* reqs, int32_t R,
                                    size_t* bytes);

/* Gather of the forwarded tokens (Alg. 1 add_noise; context tokens resampled
 * from the clean latents).  As sphinx_gather over idx[0..n), except that a
 * token t with wmask[t] == 0 (not in the write set) uses a_ctx[g], b_ctx[g]
 * instead of a[g], b[g].  wmask: dev uint8 [N] (the write-set mask of
 * sphinx_select_mask); a, b, a_ctx, b_ctx: dev float [G]. */
sphinx_status sphinx_gather_ctx(const sphinx_request* reqs, int32_t R, sphinx_layout layout, const void* state,
                                sphinx_dtype state_dtype, const void* eps, sphinx_dtype eps_dtype, const int32_t* idx,
                                int32_t n, const uint8_t* wmask, const float* a, const float* b, const float* a_ctx,
                                const float* b_ctx, float* x, void* stream);

/* sphinx_refine_step with the latent cache.  Rows x[0..n) are the forwarded
 * tokens idx[0..n) (ascending within each request), segment r being rows
 * [cu_host[r], cu_host[r+1]).  In every block the keys and values of the
 * forwarded rows are first stored at their token rows of the block's cache
 * slice, then each row attends over cache rows [tok_offset_r, tok_offset_r +
 * tokens_r) of its request.  kv_cache: dev, sphinx_kv_cache_bytes bytes,
 * 16-byte aligned, read and written.  Other arguments, workspace and errors as
 * sphinx_refine_step (n up to N; size the workspace for the largest n). */
sphinx_status sphinx_refine_step_cached(const sphinx_model_desc* m, const sphinx_request* reqs, int32_t R,
                                        const int32_t* idx, int32_t n, const int32_t* cu_host, const int32_t* tau,
                                        const float* c1, const float* c2, float* x, void* kv_cache, void* ws,
                                        size_t ws_bytes, void* stream);

/* In-place scatter of the write set only (Sec. 5.3: unselected tokens keep
 * their values): z token idx[j] <- x[j] for every j < n with wmask[idx[j]] =
 * 1; forwarded context rows are dropped.  z: dev latents in `layout`/`dtype`
 * (bf16 rounds to nearest even); wmask: dev uint8 [N]. */
sphinx_status sphinx_scatter_masked(const sphinx_request* reqs, int32_t R, const float* x, const int32_t* idx,
                                    int32_t n, const uint8_t* wmask, void* z, sphinx_dtype dtype,
                                    sphinx_layout layout, void* stream);

/* ------------------------------------------------------------------------
 * Mask front-end (Sec. 5.3 spatially selective refinement; Alg. 1
 * laplacian_var, otsu(norm(.)), the opacity mask 1[O < tau_o] and their
 * union): the token mask of every request from the regression output frames
 * and their opacity, integer-exact.
 *
 *   luma   Y = (77 R + 150 G + 29 B + 128) >> 8
 *   blur   L = 4-neighbour Laplacian of Y; V = 81 * sum(L^2) - (sum L)^2 over
 *          the 9 x 9 window (81^2 times the local variance of L); Wm = sum of
 *          V over the 5 x 5 box; per frame q = floor(255 (Wm - min) / (max -
 *          min)) (0 for a constant frame) and inv = 255 - q; Otsu's threshold
 *          t of inv over the frame (the t in 0..254 maximising the
 *          between-class variance, exact, smallest t on ties); blurry = inv > t.
 *          Every stencil reads its input with replicated borders.
 *   mask   pixel = (opacity < tau_o) | blurry; token (f, y, x) = OR over
 *          image pixels [16y, 16y+16) x [16x, 16x+16) of frame f (a latent
 *          pixel is 8 x 8 image pixels, a token 2 x 2 latent pixels).
 * ------------------------------------------------------------------------ */

/* Workspace bytes of sphinx_mask_frontend (about one byte per image pixel). */
sphinx_status sphinx_mask_frontend_workspace_bytes(const sphinx_request* reqs, int32_t R, size_t* bytes);

/* rgb: dev uint8, per request [frames][8h][8w][3] (interleaved RGB, rows of
 * the image), requests concatenated (request r starts at byte 768 *
 * tok_offset_r).  opacity: dev float, per request [frames][8h][8w], request r
 * at element 256 * tok_offset_r.  tau_o: opacity threshold (strict; 0.5 in
 * the paper; NaN selects nothing by opacity).  token_mask: dev uint8 [N] out
 * (0/1).  uncert: dev float [N] out or NULL; 1.0 where the token is masked,
 * else 0.0, so that sphinx_select_mask with thr = 0.5 selects exactly the
 * mask.  otsu_t: dev int32 [G] out or NULL (each frame's threshold).  Images
 * are limited to 2^26 pixels per frame (h * w <= 2^20).  Bit-exact and
 * deterministic. */
sphinx_status sphinx_mask_frontend(const sphinx_request* reqs, int32_t R, const uint8_t* rgb, const float* opacity,
                                   float tau_o, uint8_t* token_mask, float* uncert, int32_t* otsu_t, void* ws,
                                   size_t ws_bytes, void* stream);

#ifdef __cplusplus
}
#endif

#endif /* SPHINX_H */
