/*
 * featfix.h -- C ABI of libfeatfix.so, the MI355X (gfx950) implementation of the
 * FeatFix cached diffusion-transformer denoising step.
 *
 * The operations follow the paper's statement of the problem (FeatFix, Sec. 3):
 *   ff_block_exact     exact block output h_f = B_l(u; t, c)                    (Eq. 1)
 *   ff_cache_update    feature history refreshed at exact refreshes            (Eq. 2)
 *   ff_draft_forecast  order-K Taylor draft h_d = D(u) from that history       (Eq. 2)
 *   ff_verify_replace  same-input pair, rel-L1 audit, forwarding rule          (Eq. 3-5)
 *   ff_denoise_step    one denoising step over a fixed site set, with the
 *                      Verify / Exact-only / Vanilla controls and accounting   (Sec. 3.3)
 *
 * Conventions (all calls):
 *  - Every device buffer belongs to the caller (weights, latents, stream tensors, cache,
 *    workspace, audit).  The library never allocates or frees device memory and owns
 *    only the host objects ff_plan and ff_ctx.  Pointers must stay valid until the work
 *    queued on the stream has completed.
 *  - Layouts are row-major.  Weight matrices are [out, in].  Activations are [B, N, C]
 *    with N = n_txt + n_img rows per sample, text rows first.  The cache is
 *    [L][S][B*N*C], contiguous, in the model dtype.
 *  - "dtype" tensors are fp32 (FF_F32) or bf16 (FF_BF16) as the model descriptor says.
 *    Conditioning vectors, the latent, modulation and audit values are always fp32.
 *  - Every pointer passed as a device pointer must be 16-byte aligned.
 *  - All validation happens on the host before anything is launched; on error nothing
 *    is launched, outputs are untouched and ff_last_error() describes the problem.
 *    Asynchronous device faults surface at the caller's stream synchronisation (or as
 *    FF_E_HIP from a later call).  No C++ exception crosses the ABI.
 *  - Calls are re-entrant; use one ff_ctx per stream.  Calls that share a workspace or
 *    cache must be ordered on one stream.
 *  - All kernels are deterministic: the same inputs give bitwise identical outputs.
 */
#ifndef FEATFIX_H
#define FEATFIX_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#define FF_ABI_VERSION 3
#define FF_MAX_K 3          /* largest supported forecast order K */
#define FF_MAX_SLOTS 8      /* largest supported ring size S      */
#define FF_TEMB_DIM 256     /* sinusoidal time-embedding width    */

typedef int32_t ff_status;
enum {
  FF_OK = 0,
  FF_E_NULL = -1,        /* a required pointer is NULL                                */
  FF_E_SHAPE = -2,       /* inconsistent or unsupported sizes                         */
  FF_E_DTYPE = -3,       /* unknown dtype                                             */
  FF_E_RANGE = -4,       /* layer / step / slot / order / mode out of range           */
  FF_E_STATE = -5,       /* slot never written, draft before first refresh, step order */
  FF_E_WORKSPACE = -6,   /* workspace or cache buffer too small                      */
  FF_E_HIP = -7,         /* a HIP runtime call failed                                 */
  FF_E_UNSUPPORTED = -8  /* valid request the library does not implement           */
};

enum { FF_DIT = 0, FF_MMDIT_DOUBLE = 1, FF_MMDIT_SINGLE = 2 };          /* block kinds  */
enum { FF_F32 = 0, FF_BF16 = 1 };                                        /* dtypes       */
/* Modes (Sec. 3.3).  The last three are the matched-compute arms the paper weighs
 * whole-block forwarding against: forwarding the exact output on every part_stride-th
 * token (FF_TOKENS_PARTIAL) or channel (FF_CHANNELS_PARTIAL) only, and recomputing the
 * rest of the timestep exactly from the first paid site on (FF_RECOMPUTE). */
enum { FF_VANILLA = 0, FF_DRAFT = 1, FF_VERIFY = 2, FF_FEATFIX = 3, FF_EXACT_ONLY = 4,
       FF_TOKENS_PARTIAL = 5, FF_CHANNELS_PARTIAL = 6, FF_RECOMPUTE = 7 };
enum { FF_RESIDUAL = 0, FF_OUTPUT = 1 };                                 /* feature mode */
enum { FF_STEP_REFRESH = 0, FF_STEP_CACHED = 1 };                        /* step kinds   */
/* actions; FF_ACT_RECOMPUTE: the exact block without a history refresh */
enum { FF_ACT_EXACT = 0, FF_ACT_DRAFT = 1, FF_ACT_SITE = 2, FF_ACT_RECOMPUTE = 3 };
/* what ff_verify_replace writes: the draft (Verify), the exact output (FeatFix), or the
 * exact output on every stride-th token / channel of each sample and the draft elsewhere */
enum { FF_FWD_DRAFT = 0, FF_FWD_EXACT = 1, FF_FWD_TOKENS = 2, FF_FWD_CHANNELS = 3 };

/* HIP stream handle (the same type as hipStream_t); NULL is the default stream. */
typedef struct ihipStream_t* ff_stream_t;

/* Model shape.  Block kinds: FF_DIT (adaLN DiT block), FF_MMDIT_DOUBLE (separate text /
 * image weight sets, joint attention, per-head QK RMSNorm), FF_MMDIT_SINGLE (one weight
 * set, fused attention+MLP input projection).  FF_DIT requires n_txt == 0.
 * Requirements: C == H*d, d in [8, 128] and d % 8 == 0, C % 8 == 0, mlp_hidden % 8 == 0,
 * 1 <= B <= 32, lat_f % pt == lat_h % ph == lat_w % pw == 0,
 * n_img == (lat_f/pt)*(lat_h/ph)*(lat_w/pw), (pt*ph*pw*lat_c) % 8 == 0.
 * rope_axes: all 0 for no rotary embedding; otherwise even dims summing to d.  The MMDiT
 * blocks then rotate q and k after their RMSNorms: the head dims are split into chunks of
 * rope_axes[0..2] dims and in chunk a the pair (2i, 2i+1) of a row is turned by
 * pos_a * rope_theta^(-2i / rope_axes[a]), where pos = (0, 0, 0) for text rows and
 * (frame, row, column) of the patch in the (lat_f/pt, lat_h/ph, lat_w/pw) grid for image
 * rows (FLUX-style 3-axis ids).  rope_theta > 1 when enabled.
 * cfg_pairs: 0, or 1 for classifier-free guidance by batch doubling: B is even and rows
 * b < B/2 are the conditional samples, rows B/2 + b their unconditional twins (the caller
 * passes both conditionings in cond / txt); the latent x of ff_denoise_step then holds
 * B/2 samples, both rows of a pair read latent b, and the Euler step uses
 * v = v_u + cfg_scale * (v_c - v_u) (cfg_scale finite). */
typedef struct {
  int32_t n_layers;
  const int32_t* kinds;   /* host array [n_layers]; copied where it is kept */
  int32_t C, H, d, mlp_hidden;
  int32_t n_img, n_txt, B;
  int32_t lat_c, lat_f, lat_h, lat_w;
  int32_t pt, ph, pw;
  int32_t dtype;
  float ln_eps;           /* LayerNorm / RMSNorm epsilon */
  int32_t rope_axes[3];
  float rope_theta;
  int32_t cfg_pairs;
  float cfg_scale;
} ff_model_desc;

/* One stream's weights of one block (device pointers, model dtype, [out, in]).
 * FF_DIT and the two streams of FF_MMDIT_DOUBLE use:
 *   mod_w [6C, C], mod_b [6C]   -> shift1, scale1, gate1, shift2, scale2, gate2
 *   qkv_w [3C, C], qkv_b [3C]   -> columns s*C + h*d + e, s in {q, k, v}
 *   o_w [C, C], o_b [C];  fc1_w [M, C], fc1_b [M];  fc2_w [C, M], fc2_b [C]
 *   q_g [d], k_g [d]            -> QK RMSNorm gains (MMDiT only)
 * FF_MMDIT_SINGLE uses:
 *   mod_w [3C, C], mod_b [3C]   -> shift, scale, gate
 *   lin1_w [3C+M, C], lin1_b    -> q | k | v | mlp input
 *   lin2_w [C, C+M], lin2_b [C] -> applied to [attention | GELU(mlp input)]
 *   q_g [d], k_g [d] */
typedef struct {
  const void *mod_w, *mod_b;
  const void *qkv_w, *qkv_b;
  const void *o_w, *o_b;
  const void *fc1_w, *fc1_b;
  const void *fc2_w, *fc2_b;
  const void *lin1_w, *lin1_b;
  const void *lin2_w, *lin2_b;
  const void *q_g, *k_g;
} ff_stream_weights;

/* s[0]: the DiT / single-stream weights, or the text stream of a double block;
 * s[1]: the image stream of a double block (unused otherwise). */
typedef struct {
  ff_stream_weights s[2];
} ff_layer_weights;

/* Embedders and final layer (device pointers, model dtype), P = pt*ph*pw*lat_c:
 *   t1_w [C, 256], t1_b [C], t2_w [C, C], t2_b [C]   time-embedding MLP
 *   pe_w [C, P], pe_b [C]                             patch embedding
 *   fmod_w [2C, C], fmod_b [2C]                       final adaLN (shift, scale)
 *   f_w [P, C], f_b [P]                               final linear */
typedef struct {
  const void *t1_w, *t1_b, *t2_w, *t2_b;
  const void *pe_w, *pe_b;
  const void *fmod_w, *fmod_b, *f_w, *f_b;
} ff_global_weights;

/* Schedule: T steps, full refresh every R steps (steps i with i % R == 0), forecast
 * order K (0 <= K <= FF_MAX_K), ring of S slots (K+1 <= S <= FF_MAX_SLOTS), rel-L1
 * epsilon eps > 0, mode (FF_VANILLA .. FF_RECOMPUTE), feature_mode (FF_RESIDUAL caches
 * h - u and drafts u + F; FF_OUTPUT caches h and drafts F).
 * tau: 0 keeps that fixed schedule.  tau > 0 (finite; FF_VERIFY and FF_FEATFIX only)
 * makes the base policy adaptive, discrepancy-triggered in the manner of speculative
 * caching (the paper's base policies decide when to refresh, Sec. 3.1; its FLUX policy
 * has a threshold, Sec. 4): step 0 refreshes, and a later step i refreshes when
 * i - (the last refresh step) >= R, or when step i-1 was a cached step whose largest
 * paid-site discrepancy max_{l,b} d_b (Eq. 4) is not <= tau (a NaN counts as above).
 * The finite differences then use the actual refresh steps (Eq. 2).
 * part_stride (>= 1, FF_TOKENS_PARTIAL and FF_CHANNELS_PARTIAL; ignored otherwise): the
 * exact output is forwarded on the tokens (rows of the block, text rows included) or
 * channels whose index within a sample is a multiple of it. */
typedef struct {
  int32_t T, R, K, S;
  float eps;
  int32_t mode;
  int32_t feature_mode;
  float tau;
  int32_t part_stride;
} ff_sched_desc;

/* Separate accounting of full-refresh steps, paid exact-block checks and forwarded
 * corrections (Sec. 3.3, matched-compute controls and accounting); the partial arms
 * count their partly forwarded sites as forwarded, and n_recomputed counts the exact
 * blocks the recompute arm adds after its paid sites. */
typedef struct {
  int64_t n_full_refresh, n_paid_checks, n_forwarded, n_recomputed;
} ff_counts;

/* Kernel classes of the optional per-launch profiler (ff_ctx_profile). */
enum {
  FF_PROF_GEMM = 0,    /* dense contractions of the exact block, patch embed, final linear */
  FF_PROF_ATTN = 1,    /* softmax attention                                                 */
  FF_PROF_NORM = 2,    /* adaLN LayerNorm, QK RMSNorm                                       */
  FF_PROF_GEMV = 3,    /* modulation and time-embedding GEMVs                               */
  FF_PROF_DRAFT = 4,   /* Taylor draft                                                      */
  FF_PROF_VERIFY = 5,  /* fused verify + replace (+ its second reduction stage)             */
  FF_PROF_CACHE = 6,   /* history refresh                                                   */
  FF_PROF_OTHER = 7,   /* time embedding, patchify, text rows, unpatchify + Euler           */
  FF_PROF_NCLASS = 8
};

/* Per-class totals: launches, summed event-measured duration (ms), algorithmic FLOPs
 * (2*M*N*K per GEMM, 4*B*N^2*H*d per attention) and algorithmic HBM bytes (each
 * operand read once, each output written once). */
typedef struct {
  int64_t launches;
  double ms, flops, bytes;
} ff_prof_stat;

typedef struct ff_plan ff_plan;
typedef struct ff_ctx ff_ctx;

/* ABI version (FF_ABI_VERSION). */
int32_t ff_abi_version(void);

/* Message for the last failing ff_* call on this thread ("" if none).  Thread-local;
 * valid until the next ff_* call on the same thread. */
const char* ff_last_error(void);

/* ---------------------------------------------------------------- schedule (host only)
 * Builds the fixed schedule (Sec. 3.3: sites frozen before evaluation; Eq. 2: finite
 * differences estimated at exact refreshes).  site_mask is a host uint8 array [T*L],
 * step-major; bits on refresh steps are ignored and Draft mode ignores all bits.
 * Per step i: refresh iff mode == FF_VANILLA or i % R == 0; refresh ordinal
 * j = (#refreshes up to i) - 1; k_eff = min(K, j); refresh steps write slot j % S (none
 * in Vanilla); cached steps read slots (j - m) % S for m = 0..k_eff with coefficients
 * c_m such that F(i) = sum_m c_m * Delta_{j-m} equals the Taylor forecast of Eq. 2.
 * Per (i, l): EXACT on refresh steps, SITE where the mask is set in the paid modes
 * (Verify, FeatFix, Exact-only and the three arms), DRAFT otherwise; in FF_RECOMPUTE the
 * layers after a cached step's first SITE are RECOMPUTE.  With tau > 0 this is the
 * schedule of a run in which no discrepancy exceeds tau; the context realises the
 * actual one step by step (ff_ctx_step_kinds).  *out is owned by the caller
 * (ff_plan_destroy).
 * Errors: FF_E_NULL, FF_E_RANGE (T, R, K, S, mode, feature_mode, n_layers, eps, tau,
 * part_stride). */
ff_status ff_plan_build(const ff_sched_desc* s, int32_t n_layers, const uint8_t* site_mask,
                        ff_plan** out);
void ff_plan_destroy(ff_plan* p);

/* Copies the plan's decisions into host arrays (any may be NULL to skip it):
 * step_kind[T], refresh_ord[T], k_eff[T], read_slots[T*(K+1)] (-1 padded),
 * write_slot[T] (-1 if none), action[T*L], coeffs[T*(K+1)] (fp32, 0 padded), counts
 * (totals over the whole schedule).  Errors: FF_E_NULL if p is NULL. */
ff_status ff_plan_export(const ff_plan* p, int32_t* step_kind, int32_t* refresh_ord,
                         int32_t* k_eff, int32_t* read_slots, int32_t* write_slot,
                         int32_t* action, float* coeffs, ff_counts* counts);

/* ---------------------------------------------------------------- sizing
 * Bytes of a cache with n_slots ring slots per layer: L * n_slots * B*N*C * dtype size.
 * Bytes of workspace ff_denoise_step needs (ff_block_exact and ff_verify_replace need
 * no more than this).  Both return 0 for an invalid descriptor. */
size_t ff_cache_bytes(const ff_model_desc* m, int32_t n_slots);
size_t ff_workspace_bytes(const ff_model_desc* m);

/* ---------------------------------------------------------------- block operations
 * Exact block output (Eq. 1): h = B_layer(u; c_t) for the block kind m->kinds[layer].
 * c_t: device fp32 [B, C] conditioning (class/text vector plus time embedding);
 * u, h: device [B, N, C] dtype; h must not overlap u or ws.  ws: device workspace of
 * at least ff_workspace_bytes(m) bytes.  Deterministic (bitwise reproducible).
 * Errors: FF_E_NULL, FF_E_RANGE (layer), FF_E_SHAPE, FF_E_DTYPE, FF_E_WORKSPACE. */
ff_status ff_block_exact(const ff_model_desc* m, int32_t layer, const ff_layer_weights* w,
                         const float* c_t, const void* u, void* h, void* ws, size_t ws_bytes,
                         ff_stream_t stream);

/* Refresh of the feature history (Eq. 2, estimated at exact refreshes):
 * cache[layer][slot] <- h - u (FF_RESIDUAL, rounded to dtype) or h (FF_OUTPUT; u unused,
 * may be NULL).  cache holds n_slots slots per layer.
 * Errors: FF_E_NULL, FF_E_RANGE (layer, slot, n_slots, feature_mode), FF_E_SHAPE. */
ff_status ff_cache_update(const ff_model_desc* m, void* cache, int32_t n_slots, int32_t layer,
                          int32_t slot, const void* u, const void* h, int32_t feature_mode,
                          ff_stream_t stream);

/* Draft forecast (Eq. 2): h_d = u + sum_{m=0..k_eff} coeffs[m] * cache[layer][slots[m]]
 * (u == NULL selects FF_OUTPUT: h_d = sum_m coeffs[m] * cache[layer][slots[m]]).
 * slots and coeffs are host arrays [k_eff+1].  Sums in fp32, one rounding to dtype.
 * h_d may alias u exactly (in-place); no other overlap is allowed.
 * Errors: FF_E_NULL, FF_E_RANGE (layer, k_eff, slot, n_slots), FF_E_SHAPE. */
ff_status ff_draft_forecast(const ff_model_desc* m, const void* cache, int32_t n_slots,
                            int32_t layer, int32_t k_eff, const int32_t* slots,
                            const float* coeffs, const void* u, void* h_d, ff_stream_t stream);

/* Paid verification and forwarding (Eq. 3-5) in one pass over the site tensor:
 * rebuilds h_d = D(u) as ff_draft_forecast does (u == NULL for FF_OUTPUT), computes per
 * sample b the normalised relative-L1 discrepancy
 *     rel_l1[b] = sum|h_d - h_f| / (sum|h_f| + eps)       (Eq. 4; fp32, fixed-order sums)
 * and writes h_out by forward: FF_FWD_EXACT h_f (FeatFix: bit-identical copy of h_f),
 * FF_FWD_DRAFT h_d (Verify), FF_FWD_TOKENS / FF_FWD_CHANNELS h_f on the tokens (rows n of
 * each sample's N) / channels c with n or c a multiple of stride (>= 1) and h_d elsewhere
 * (the partial arms of Sec. 3.3; stride is ignored for the first two).  h_out may alias
 * u exactly; it must not overlap h_f.  rel_l1 is a device fp32 [B] array or NULL.  ws
 * holds the partial sums (at least ff_workspace_bytes(m)).
 * Errors: FF_E_NULL, FF_E_RANGE (forward, stride, ...), FF_E_SHAPE, FF_E_WORKSPACE. */
ff_status ff_verify_replace(const ff_model_desc* m, const void* cache, int32_t n_slots,
                            int32_t layer, int32_t k_eff, const int32_t* slots,
                            const float* coeffs, const void* u, const void* h_f, void* h_out,
                            int32_t forward, int32_t stride, float eps, float* rel_l1, void* ws,
                            size_t ws_bytes, ff_stream_t stream);

/* ---------------------------------------------------------------- no-allocation verify
 * For callers that cannot allocate device memory or hand over a workspace: code under HIP
 * graph capture, tight serving loops, harnesses that forbid hipMalloc.  The same operation
 * as ff_verify_replace (same kernels, bit-identical h_out and rel_l1) without the ws
 * argument: the partial sums of Eq. 4 (B * 2048 * 2 floats) live in a library-owned
 * device array of FF_NOALLOC_VERIFY_MAX_B * 2048 * 2 floats (256 KB) on each GPU the
 * library runs on, held from the first call on that GPU until the process ends.  Nothing
 * in it needs to start at zero (every call writes the partials it reads).  Calls that
 * overlap on one GPU (several streams or threads) share that array and race: order them
 * on one stream.  stream must belong to the current device.  Allocates nothing: no
 * hipMalloc, hipFree or allocating library routine.
 * Errors: as ff_verify_replace; FF_E_WORKSPACE if m->B > FF_NOALLOC_VERIFY_MAX_B; FF_E_HIP
 * if the array's device address cannot be obtained. */
#define FF_NOALLOC_VERIFY_MAX_B 16
ff_status ff_verify_replace_noalloc(const ff_model_desc* m, const void* cache, int32_t n_slots,
                                    int32_t layer, int32_t k_eff, const int32_t* slots,
                                    const float* coeffs, const void* u, const void* h_f,
                                    void* h_out, int32_t forward, int32_t stride, float eps,
                                    float* rel_l1, ff_stream_t stream);

/* ---------------------------------------------------------------- step executor
 * A context binds a model, its weights (layer_w is a host array [n_layers]; the device
 * pointers inside are kept, the host arrays are copied), a plan (copied), a cache of at
 * least ff_cache_bytes(m, plan S) bytes (a Vanilla plan never touches it: cache may then
 * be NULL with cache_bytes 0) and a workspace of at least ff_workspace_bytes(m) bytes.
 * *out is owned by the caller (ff_ctx_destroy).
 * Errors: FF_E_NULL, FF_E_SHAPE, FF_E_DTYPE, FF_E_WORKSPACE, FF_E_RANGE. */
ff_status ff_ctx_create(const ff_model_desc* m, const ff_layer_weights* layer_w,
                        const ff_global_weights* g, const ff_plan* p, void* cache,
                        size_t cache_bytes, void* ws, size_t ws_bytes, ff_ctx** out);
void ff_ctx_destroy(ff_ctx* c);

/* Rewinds the context to step 0, forgets the cache history and zeroes the counts. */
ff_status ff_ctx_reset(ff_ctx* c);

/* Counts of the steps executed since creation / the last reset. */
ff_status ff_get_counts(const ff_ctx* c, ff_counts* out);

/* Realised kind of each step since creation / the last reset: kinds[i] = FF_STEP_REFRESH
 * or FF_STEP_CACHED for steps already run, -1 for the others (host array [T]).  With
 * tau == 0 it follows the plan; with tau > 0 it records the adaptive decisions.
 * Errors: FF_E_NULL. */
ff_status ff_ctx_step_kinds(const ff_ctx* c, int32_t* kinds);

/* One denoising step i = step (must be the context's next step, 0..T-1 in order):
 *   c_t = cond + TimeMLP(sinusoid(1000 t_i)), t_i = 1 - i/T
 *   X = [txt ; PatchEmbed(patchify(x))]
 *   for each layer l, by the plan's action:
 *     EXACT: X <- B_l(X); refresh the history of l (not in Vanilla)
 *     DRAFT: X <- D_l(X)
 *     SITE : h_f = B_l(X); audit and forward per mode (FeatFix / Exact-only / recompute:
 *            h_f, Verify: the draft, the partial arms: h_f on every part_stride-th
 *            token or channel); Exact-only skips the draft and the audit
 *     RECOMPUTE: X <- B_l(X) without a history refresh
 *   v = unpatchify(FinalLayer(X_img)); x <- x + (t_{i+1} - t_i) v
 * x: device fp32 latent [B, lat_c, lat_f, lat_h, lat_w] ([B/2, ...] with cfg_pairs),
 * updated in place.
 * cond: device fp32 [B, C].  txt: device dtype [B, n_txt, C] (NULL iff n_txt == 0).
 * audit: device fp32 [T*L*B] or NULL; entry (i*L + l)*B + b receives rel_l1 at paid
 * checks (other entries are not written).
 * With tau > 0 the step's kind is decided here (ff_sched_desc): a step that follows a
 * checked cached step first waits on the host for that step's discrepancies (queued
 * on the same stream as a small device-to-host copy), so the host blocks until the
 * previous step has finished on the device.
 * Errors: FF_E_NULL, FF_E_STATE (step out of order), FF_E_HIP. */
ff_status ff_denoise_step(ff_ctx* c, int32_t step, float* x, const float* cond,
                          const void* txt, float* audit, ff_stream_t stream);

/* ---------------------------------------------------------------- history sums
 * Eq. 2's draft is linear in the feature history.  A run of consecutive drafted layers
 * l0..l1-1 of a cached step (residual features) therefore moves the stream by
 * sum_m c_m * P_m, where P_m is the sum over the run's layers of the history slot the
 * m-th term reads.  That sum changes only when a refresh rewrites the slot.
 * ff_hist_sum_bytes(m, p): bytes of fp32 sums for plan p: runs * S * B*N*C * 4, where
 * runs counts the distinct maximal runs of two or more drafted layers over the plan's
 * cached steps (with tau > 0, over every step that may be cached).  Returns 0 when
 * there is no such run, with output features, in Vanilla, or on an invalid descriptor.
 * ff_ctx_hist_sums(c, buf, bytes): with buf set, each refresh step of c forms the sums
 * of the slot it wrote (one fp32 pass per run, in layer order), and each such run of a
 * cached step is applied in one pass from them:
 *   X <- round(X + sum_m c_m P_m), one rounding to the model dtype per run.
 * Without sums, the stream is rounded after every drafted layer.  The two agree to the
 * model dtype's rounding; in bf16 this is not bit for bit.  While a trace buffer is set,
 * runs are applied layer by layer.  buf is the caller's device memory, 16-byte aligned.
 * It must stay untouched while c uses it.  buf NULL turns the sums off at any time.
 * Errors: FF_E_NULL (c); FF_E_UNSUPPORTED (output features, Vanilla, or no run of two
 * drafted layers); FF_E_STATE (enabling after step 0 before ff_ctx_reset: the sums of
 * earlier refreshes are missing); FF_E_WORKSPACE (bytes); FF_E_SHAPE (alignment). */
size_t ff_hist_sum_bytes(const ff_model_desc* m, const ff_plan* p);
ff_status ff_ctx_hist_sums(ff_ctx* c, void* buf, size_t bytes);

/* ---------------------------------------------------------------- conditioning cache
 * The conditioning c_t = c + TimeMLP(phi(1000 t_i)) and the adaLN modulation of every
 * exact block (Eq. 1) depend on the class / text vector and the step only, never on the
 * latent.  ff_cond_cache_bytes(m, p): bytes of the cache for plan p (0 on an invalid
 * descriptor).  ff_ctx_cond_cache(c, buf, bytes): with buf set, step 0 of c forms the
 * conditioning of the whole schedule into buf from the cond it is given: the time
 * embedding and MLP of all T steps, SiLU(c_t), the modulation vectors of every layer at
 * the steps where the plan may run it exact (every step for layers that are sites of a
 * cached step, that run exact at a cached step, or when tau > 0; the refresh steps
 * otherwise), and the final layer's modulation of every step, as one GEMM per weight set
 * (bf16: SiLU(c_t) as the same bf16 hi + lo parts the per-step GEMVs use).  Later steps
 * read them and launch no conditioning work.  Every step must then pass the same cond
 * pointer as step 0, holding the same values (a different pointer is FF_E_STATE).  The
 * vectors agree with the per-step ones to fp32 rounding (other summation order), not bit
 * for bit.  buf is the caller's device memory, 256-byte aligned, untouched by the caller
 * while c uses it; buf NULL turns the cache off at any time.
 * Errors: FF_E_NULL (c); FF_E_STATE (enabling after step 0 before ff_ctx_reset);
 * FF_E_WORKSPACE (bytes); FF_E_SHAPE (alignment). */
size_t ff_cond_cache_bytes(const ff_model_desc* m, const ff_plan* p);
ff_status ff_ctx_cond_cache(ff_ctx* c, void* buf, size_t bytes);

/* ---------------------------------------------------------------- diagnostics
 * Per-layer feature traces for mechanism studies on synthetic weights (the paper tracks
 * the downstream relative-L1 error of corrected runs against Vanilla per layer and stage,
 * Sec. 4).  ff_ctx_trace(c, buf, bytes): while buf is set, every ff_denoise_step copies the
 * stream after each layer l (the [B, N, C] block output, text rows included) to
 * buf + l * B*N*C*dtype-size, so after a step buf holds that step's L layer outputs; runs
 * of drafted layers are then applied layer by layer (same values).  bytes must be at least
 * L * B*N*C * dtype size; buf NULL stops tracing.  buf is device memory of the caller.
 * Errors: FF_E_NULL (c), FF_E_WORKSPACE (bytes), FF_E_SHAPE (alignment). */
ff_status ff_ctx_trace(ff_ctx* c, void* buf, size_t bytes);

/* rel[b] = sum|a - b| / (sum|b| + eps) over sample b's N*C elements of two [B, N, C]
 * dtype tensors (Eq. 4's form, with b as the reference; fp32, fixed-order sums, as the
 * audit), rel a device fp32 [B] array.  ws: at least ff_workspace_bytes(m) bytes.
 * Errors: FF_E_NULL, FF_E_RANGE (eps), FF_E_SHAPE, FF_E_WORKSPACE. */
ff_status ff_rel_l1(const ff_model_desc* m, const void* a, const void* b, float eps, float* rel, void* ws,
                    size_t ws_bytes, ff_stream_t stream);

/* ---------------------------------------------------------------- profiling
 * Optional tracing of a context's launches (Sec. 4 reports latency per arm; this
 * attributes it to kernels).  While enabled, ff_denoise_step brackets every kernel
 * launch with a pair of HIP events recorded on the caller's stream; the events are
 * created on first use and kept by the context.  ff_ctx_profile(c, 1) enables and clears,
 * (c, 0) disables.  ff_ctx_profile_read waits for the recorded events, fills
 * out[FF_PROF_NCLASS] and clears the record.  Errors: FF_E_NULL, FF_E_HIP. */
ff_status ff_ctx_profile(ff_ctx* c, int32_t enable);
ff_status ff_ctx_profile_read(ff_ctx* c, ff_prof_stat* out);

#ifdef __cplusplus
}
#endif
#endif /* FEATFIX_H */
