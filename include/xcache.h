/*
 * xcache.h -- C ABI of the MI355X (gfx950) X-Cache cached chunk forward.
 *
 * The library runs the causal multi-block DiT forward of one few-step
 * generation chunk under X-Cache's cross-chunk block cache:
 *
 *   - rollout structure (Section 2.1, Eq. 1-2): generation n, denoising step
 *     t in [0, S), blocks b in [0, B); x_{t,b} = x_{t,b-1} + f_b(x_{t,b-1}; c_t);
 *     after the S steps one extra KV-update pass on the clean latent writes the
 *     chunk's keys/values into a rolling FIFO cache;
 *   - per-(t, b) residual cache and additive reuse (Section 2.2, Eq. 3-4);
 *   - fingerprint of each block input: a 3-D grid subsample per view group,
 *     a per-camera token-mean global channel and the chunk's action vector
 *     (Section 2.3.1-2.3.2);
 *   - dual-metric gate: min-cosine over all fingerprint entries, max token
 *     deviation over the spatial group entries, skip iff both pass
 *     (Section 2.3.3-2.3.5, Eq. 5-7);
 *   - adaptive per-(t, b) cosine threshold from an EMA (Section 2.4, Eq. 8-9);
 *   - safety mechanisms (Section 2.5): step-0 protection, front/back anchor
 *     blocks, KV-update protection (always on), maximum staleness.
 *
 * Conventions for every entry point:
 *   - Device pointers are HIP device addresses on the device that was current
 *     at xc_init; host pointers are ordinary CPU memory.  The caller owns every
 *     buffer it passes; the library owns everything it allocates.
 *   - All arguments are validated before anything is enqueued; a call that
 *     returns an error has changed no state, with the exception of
 *     XC_ERR_HIP, which is sticky: the handle must then be destroyed.
 *   - Work is enqueued on the stream bound at xc_init and the call returns
 *     without synchronising, except xc_stats and xc_kernel_times, which
 *     synchronise that stream.
 *   - A handle is not thread-safe; calls on one handle must be serialised.
 *   - No C++ exception crosses this ABI.
 */
#ifndef XCACHE_H
#define XCACHE_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum xc_status {
  XC_OK = 0,
  XC_ERR_INVALID_ARG = 1,  /* a pointer, size or configuration field is invalid */
  XC_ERR_STATE = 2,        /* call not allowed in the handle's current state     */
  XC_ERR_OOM = 3,          /* device or host allocation failed                  */
  XC_ERR_HIP = 4,          /* a HIP runtime call failed (sticky)                 */
  XC_ERR_UNSUPPORTED = 5   /* valid request this build does not implement        */
} xc_status;

/* model dtype: the residual stream is always float32; XC_BF16 stores weights,
 * activations, the KV cache and cached residuals in bf16 and runs the
 * contractions on bf16 matrix cores with float32 accumulation. */
enum { XC_F32 = 0, XC_BF16 = 1 };
enum { XC_STEP0_OFF = 0, XC_STEP0_FORCE = 1, XC_STEP0_STRICT = 2 };
enum { XC_FP_GRID3D = 0, XC_FP_LINSPACE1D = 1 };
/* When the cached fingerprint of (t, b) is replaced by the current one
   (Section 2.5 says the fingerprint cache stays refreshed; the paper does not
   say whether a skipped evaluation refreshes it). */
enum { XC_FP_REFRESH_EVERY = 0, XC_FP_REFRESH_ON_COMPUTE = 1 };
/* xc_forward_chunk flags */
enum { XC_FORCE_FULL = 1u };
/* per-block decision codes reported by xc_stats for the last denoising pass */
enum { XC_DEC_COMPUTE = 0, XC_DEC_SKIP = 1, XC_DEC_FORCED = 2, XC_DEC_NONE = 255 };

#define XC_MAX_GROUPS 8
#define XC_MAX_COND 512   /* temb_dim + action_dim */
#define XC_MAX_ACTION 64

/* Cameras sharing one latent grid (a view group, Section 2.3.1). */
typedef struct xc_view_group {
  int32_t views;   /* cameras stacked along V                         */
  int32_t frames;  /* latent frames per chunk (F)                      */
  int32_t height;  /* latent rows (H)                                  */
  int32_t width;   /* latent columns (W)                               */
} xc_view_group;

/* Model shape.  Tokens L = sum over groups of views*frames*height*width,
 * camera-major, each camera's (f, h, w) grid row-major.
 * Constraints: hidden == n_heads * head_dim; temb_dim even;
 * temb_dim + action_dim <= XC_MAX_COND; action_dim <= XC_MAX_ACTION;
 * XC_BF16 additionally needs head_dim in {64, 128} and hidden, mlp_hidden
 * multiples of 128.  Size limits of this build (32-bit kernel offsets;
 * XC_ERR_UNSUPPORTED beyond them): kv_window * L <= 2^24 keys and
 * ceil(L / 32) * 2 * hidden * 4 < 2^31.  Block internals: LayerNorm without affine (eps 1e-6),
 * six-way adaLN modulation from W_ada SiLU(c) + b_ada with
 * c = [sinusoidal temb(timestep); action], QK RMSNorm (eps 1e-6) with gains,
 * softmax attention over the rolling cache (no mask), tanh-GELU MLP.
 * Optional WAN-style extensions (the paper's model is built on WAN 2.2,
 * Section 3.1, and injects text / object / lane conditions through
 * cross-attention, Sections 2.1 and 2.3.2):
 *   rope = 1: 3-D rotary embedding of the self-attention q and k after their
 *     RMSNorm (so the cache holds rotated keys): head pairs (2j, 2j+1) rotate
 *     by p * rope_theta^(-2i/d_a); the first d - 4 floor(d/6) dimensions follow
 *     the frame position n*F + f (absolute across chunks, n the generation),
 *     the next 2 floor(d/6) the row h, the last 2 floor(d/6) the column w of
 *     the token in its camera's grid.  Needs head_dim even,
 *     rope_theta > 1, and every grid dimension < 1024.
 *   cond_len > 0: a cross-attention layer between the self-attention and the
 *     MLP: x1 += Wo_c softmax(q_c k_c^T / sqrt(d)) v_c + bo_c with
 *     q_c = RMSNorm(Wq_c (LN(x1) * ln3_w + ln3_b) + bq_c) * gq_c and
 *     k_c = RMSNorm(Wk_c cond + bk_c) * gk_c, v_c = Wv_c cond + bv_c over the
 *     condition tokens set by xc_set_condition (at most cond_len <= 4096).
 * Fields left zero select the plain block. */
typedef struct xc_model_config {
  int32_t n_blocks;    /* B                                                */
  int32_t hidden;      /* C                                                */
  int32_t n_heads;     /* H                                                */
  int32_t head_dim;    /* d                                                */
  int32_t mlp_hidden;  /* D_m                                              */
  int32_t temb_dim;    /* D_t                                              */
  int32_t action_dim;  /* A                                                */
  int32_t dtype;       /* XC_F32 or XC_BF16                                */
  int32_t n_steps;     /* S denoising steps per chunk                      */
  int32_t kv_window;   /* chunks visible to attention, current included    */
  int32_t n_groups;    /* 1..XC_MAX_GROUPS                                 */
  xc_view_group groups[XC_MAX_GROUPS];
  int32_t rope;        /* 0: none; 1: 3-D rotary embedding (see above)     */
  float rope_theta;    /* rotary base (10000 in WAN); ignored if rope == 0 */
  int32_t cond_len;    /* cross-attention condition capacity; 0: none      */
} xc_model_config;

/* Gate hyper-parameters; names and defaults follow Table 1. */
typedef struct xc_gate_config {
  int32_t enabled;        /* 0: plain DiT, no fingerprints, no cache          */
  int32_t fp_budget;      /* K tokens per camera fingerprint (32)             */
  int32_t warmup;         /* W >= 1 generations computed in full (1)          */
  int32_t front_anchors;  /* F_n always-computed leading blocks (1)           */
  int32_t back_anchors;   /* B_n always-computed trailing blocks (0)          */
  int32_t adaptive;       /* 1: EMA threshold (Eq. 8-9); 0: tau_cos_fixed     */
  float tau_floor;        /* quality floor (0.97)                             */
  float margin;           /* m (0.02)                                         */
  float alpha;            /* EMA coefficient in [0, 1] (0.3)                  */
  float tau_cos_fixed;    /* cosine threshold when adaptive == 0              */
  float tau_dev;          /* deviation threshold (2.0); +inf allowed          */
  float eps;              /* epsilon of Eq. 6 (1e-6)                          */
  int32_t max_stale;      /* M consecutive skips allowed, 0 = off             */
  int32_t step0_mode;     /* XC_STEP0_OFF / _FORCE / _STRICT                  */
  float tau_strict0;      /* strict step-0 threshold (0.999)                  */
  int32_t kv_protect;     /* must be 1: KV-update passes are never gated      */
  int32_t fp_mode;        /* XC_FP_GRID3D or XC_FP_LINSPACE1D                 */
  int32_t fp_refresh;     /* XC_FP_REFRESH_EVERY: at every evaluation (0);    */
                          /* XC_FP_REFRESH_ON_COMPUTE: only when computed     */
} xc_gate_config;

typedef struct xc_stats_t {
  int64_t generations;        /* completed KV-update passes (n)                  */
  int64_t evals_post_warmup;  /* B per denoising pass with n >= W                */
  int64_t gated_evals;        /* (t, b) gate tests actually evaluated            */
  int64_t skips;              /* block evaluations that reused a residual        */
  int64_t kv_block_evals;     /* B per KV-update pass                            */
  int32_t last_step;          /* t of the last pass, S for KV-update, -1 none    */
} xc_stats_t;

typedef struct xc_handle xc_handle;

/* Human-readable name of a status code (static string, never NULL). */
const char* xc_status_string(xc_status s);

/* Create a handle (Section 2.1 state: weights, rolling KV cache, residual and
 * fingerprint caches, EMA and staleness tables).
 *   model, gate     : host structs, copied.
 *   weights_host    : host float32 blob, per block in this order, row-major
 *                     [out, in]: W_ada [6C, D_t+A], b_ada [6C], Wq [C, C], bq,
 *                     Wk [C, C], bk, Wv [C, C], bv, Wo [C, C], bo,
 *                     W1 [D_m, C], b1, W2 [C, D_m], b2, gq [d], gk [d],
 *                     and with cond_len > 0 then ln3_w [C], ln3_b [C],
 *                     Wq_c [C, C], bq_c, Wk_c [C, C], bk_c, Wv_c [C, C], bv_c,
 *                     Wo_c [C, C], bo_c, gq_c [d], gk_c [d];
 *                     blocks concatenated.  Copied (Linear weights converted
 *                     to bf16 for XC_BF16) before return; the caller may free
 *                     it.
 *   weights_bytes   : must equal 4 * the blob's element count.
 *   hip_stream      : hipStream_t all work is enqueued on (NULL = default).
 *   out             : receives the handle.
 * Errors: XC_ERR_INVALID_ARG (NULL pointers, bad shape or gate field, size
 * mismatch), XC_ERR_UNSUPPORTED (kv_protect == 0, unsupported head_dim,
 * a shape past the size limits above),
 * XC_ERR_OOM, XC_ERR_HIP.  Synchronises the stream once (weight upload). */
xc_status xc_init(const xc_model_config* model, const xc_gate_config* gate,
                  const float* weights_host, size_t weights_bytes, void* hip_stream,
                  xc_handle** out);

/* One denoising pass (step t) of the current generation n (Eq. 1) under the
 * cross-chunk gate (Eq. 3-9, Section 2.5).
 *   step        : t in [0, S).
 *   timestep    : the diffusion timestep fed to the sinusoidal embedding.
 *   action_host : host float32 [action_dim], the chunk's action vector.
 *   x_in        : device float32 [L, C], the latent entering block 0.
 *   x_out       : device float32 [L, C], receives the last block's output;
 *                 may alias x_in.
 *   flags       : XC_FORCE_FULL computes every block but still refreshes the
 *                 fingerprint and residual caches (KV-update generation
 *                 protection, Section 2.5 item 3).
 * The current chunk's keys/values of each computed block are written into
 * this generation's cache slot and attended together with the kept past
 * chunks; they are replaced by the clean ones at xc_kv_update.
 * Decisions stay on the device; nothing is copied back.
 * Errors (nothing is enqueued and no state changes): XC_ERR_INVALID_ARG
 * (NULL pointer, step out of range, unknown flag, non-finite timestep or
 * action), XC_ERR_STATE (the action differs bitwise from the one this
 * generation's first pass used: one chunk has one action, Section 2.3.2; or
 * a cross-attention model has no condition yet), XC_ERR_HIP (sticky). */
xc_status xc_forward_chunk(xc_handle* h, int32_t step, float timestep, const float* action_host,
                           const void* x_in, void* x_out, uint32_t flags);

/* Bytes of the static device array that xc_forward_chunk_noalloc uses as its
 * scratch (one copy per GPU the library runs on, held until the process
 * ends). */
#define XC_NOALLOC_SCRATCH_BYTES (64u << 20)

/* xc_forward_chunk for callers that cannot allocate device memory (code under
 * HIP graph capture, tight serving loops, harnesses that forbid hipMalloc):
 * the same pass with the same arguments, state and errors, but the kernels'
 * per-pass scratch -- the gate's per-workgroup partial records and the
 * attention's key-split partials -- lives in a static device array of
 * XC_NOALLOC_SCRATCH_BYTES instead of the handle's buffers.  The call
 * allocates nothing (no hipMalloc, no events: xc_profile records none of its
 * launches).  The attention splits its keys over workgroups only as far as
 * the partials fit in what the records leave of the array (possibly not at
 * all), so its output may differ from xc_forward_chunk's by rounding.
 * Every handle on one GPU shares that GPU's array, and the array keeps the
 * last call's contents (each pass writes every value it reads): passes of
 * this entry point that overlap on one GPU (different handles on streams
 * that run concurrently) race.  Errors as xc_forward_chunk, plus
 * XC_ERR_UNSUPPORTED when the gate's records alone exceed the array and
 * XC_ERR_STATE when the array's device address could not be obtained at
 * xc_init. */
xc_status xc_forward_chunk_noalloc(xc_handle* h, int32_t step, float timestep, const float* action_host,
                                   const void* x_in, void* x_out, uint32_t flags);

/* The KV-update pass (Section 2.1; protection of Section 2.5 item 3): every
 * block computed in full on the clean latent, its keys/values committed to
 * the generation's slot of the rolling cache (the oldest chunk is evicted once
 * kv_window - 1 past chunks are kept), the action remembered for the next
 * generation's action channel, then n <- n + 1.  Never gated.
 *   x_clean : device float32 [L, C].
 *   x_out   : device float32 [L, C], or NULL when the pass's output is not
 *             needed: the last block then stops after its key/value
 *             projection (its attention and MLP feed nothing else).
 * Errors as xc_forward_chunk: the action must be the one this generation's
 * denoising passes used (XC_ERR_STATE otherwise); xc_reset and a completed
 * xc_kv_update release it. */
xc_status xc_kv_update(xc_handle* h, float timestep, const float* action_host,
                       const void* x_clean, void* x_out);

/* Condition tokens of the cross-attention layer (models with cond_len > 0;
 * the text / object / lane embeddings of Sections 2.1 and 2.3.2).
 *   cond_host : host float32 [n_tokens, C], row-major; copied before return.
 *   n_tokens  : 1 <= n_tokens <= cond_len.
 * Computes every block's cross-attention keys and values of these tokens
 * (bf16 models round the tokens to bf16 first); later passes attend to them
 * until the next call.  Must be called before the first xc_forward_chunk or
 * xc_kv_update of such a model (XC_ERR_STATE otherwise) and may be called
 * again between any two passes; xc_reset keeps it.  The gate does not see
 * the condition (the paper leaves condition changes to step-0 protection,
 * the anchor blocks and the cascade through block inputs, Section 2.5).
 * Errors: XC_ERR_INVALID_ARG (NULL, n_tokens out of range, non-finite
 * values), XC_ERR_STATE (model has no cross-attention), XC_ERR_HIP.
 * Synchronises the stream once (the upload). */
xc_status xc_set_condition(xc_handle* h, const float* cond_host, int32_t n_tokens);

/* Caches readable with xc_read_cache. */
enum { XC_CACHE_RESIDUAL = 0, XC_CACHE_KEYS = 1, XC_CACHE_VALUES = 2 };

/* Copies one of the handle's caches, as float32, into a caller device buffer
 * (enqueued on the bound stream; does not synchronise).  For bf16 models the
 * values are the stored bf16 numbers.
 *   XC_CACHE_RESIDUAL : the cached residual r_hat of (t = step, b = block),
 *                       Eq. 3, [L][C]; unspecified until (t, b) has computed
 *                       once.
 *   XC_CACHE_KEYS     : block b's rolling key cache (Section 2.1) as
 *                       [H][kv_window * L][d]: keys after the QK RMSNorm (and
 *                       the rotation with rope = 1); rows [s L, (s + 1) L)
 *                       hold the latest generation n with n mod kv_window ==
 *                       s -- the current generation's slot holds its latest
 *                       pass's keys until xc_kv_update writes the clean ones.
 *                       step is ignored.
 *   XC_CACHE_VALUES   : block b's value cache, same layout.
 *   out_dev    : device float32 buffer of out_floats elements, which must be
 *                the tensor's element count.
 * Errors: XC_ERR_INVALID_ARG (NULL, kind / step / block out of range, size
 * mismatch), XC_ERR_STATE (the residual of a block the gate never evaluates),
 * XC_ERR_HIP (sticky). */
xc_status xc_read_cache(xc_handle* h, int32_t kind, int32_t step, int32_t block, void* out_dev,
                        size_t out_floats);

/* Synchronise the stream and copy out counters and per-(t, b) state.
 * Every array pointer may be NULL.  skip_counts: int32 [S * B] (t-major);
 * last_decision: uint8 [B] for the last denoising pass (XC_DEC_*;
 * XC_DEC_NONE before any); last_cos, last_dev, last_tau: float [B] (NaN where
 * the gate was not evaluated); ema: float [S * B] (NaN where unset). */
xc_status xc_stats(xc_handle* h, xc_stats_t* stats, int32_t* skip_counts, uint8_t* last_decision,
                   float* last_cos, float* last_dev, float* last_tau, float* ema);

/* Start a new rollout: clears the KV cache, residual/fingerprint caches, EMA,
 * staleness and counters; keeps the weights. */
xc_status xc_reset(xc_handle* h);

/* Release everything the handle owns (synchronises its stream).  NULL is a
 * no-op. */
xc_status xc_destroy(xc_handle* h);

/* Sampler helper for the rollout driver: out = a*x + b*y over n float32
 * device elements (out may alias x or y). */
xc_status xc_axpby(xc_handle* h, float a, const void* x, float b, const void* y, void* out, size_t n);

/* Host-only (no HIP call): the token rows the fingerprint samples, per view
 * group in order, camera by camera (Section 2.3.1).  Writes up to cap int32
 * global row indices into rows (may be NULL) and the total into *n_rows. */
xc_status xc_fingerprint_rows(const xc_model_config* model, const xc_gate_config* gate,
                              int32_t* rows, size_t cap, size_t* n_rows);

/* Kernel timing: while enabled, every launch of the kernel kinds below is
 * bracketed by HIP events on the bound stream.  A gated evaluation is two
 * launches: XC_KERN_GATE reads the block input once, forms the fingerprint
 * and compares it with the cached one; XC_KERN_GATE_DECIDE takes the
 * decision.  The skip path (Eq. 4) runs inside the block's first LayerNorm
 * launch: for a block whose gate was evaluated that launch is counted as
 * XC_KERN_SKIP_ADD (it writes x + rhat when the block is skipped and the
 * LayerNorm otherwise); every other LayerNorm launch is XC_KERN_LN_MOD.  The
 * cross-attention layer's kernels are XC_KERN_CROSS_Q (its
 * LayerNorm and q projection), XC_KERN_CROSS_ATTENTION and XC_KERN_CROSS_O
 * (output projection and residual). */
enum {
  XC_KERN_ATTENTION = 0, XC_KERN_GEMM_QKV = 1, XC_KERN_GEMM_OPROJ = 2, XC_KERN_GEMM_UP = 3,
  XC_KERN_GEMM_DOWN = 4, XC_KERN_GATE = 5, XC_KERN_GATE_DECIDE = 6, XC_KERN_SKIP_ADD = 7, XC_KERN_LN_MOD = 8,
  XC_KERN_QK_NORM = 9, XC_KERN_ADALN = 10, XC_KERN_CROSS_Q = 11, XC_KERN_CROSS_ATTENTION = 12,
  XC_KERN_CROSS_O = 13, XC_KERN_COUNT = 14
};
xc_status xc_profile(xc_handle* h, int32_t enable);

/* Synchronise, then report launches and summed event time (ms) of one kernel
 * kind since profiling was enabled or last cleared; clear != 0 resets it. */
xc_status xc_kernel_times(xc_handle* h, int32_t kind, int64_t* launches, double* total_ms, int32_t clear);

/* Measurement aid, not a step of the method: the bf16 MFMA rate the chip
 * sustains on a loop whose operands stay in registers (no memory traffic),
 * i.e. the practical ceiling of the contractions above.  shape: 0 =
 * v_mfma_f32_32x32x16_bf16, 1 = v_mfma_f32_16x16x32_bf16 (four waves per
 * SIMD); 2-4 = 32x32x16 at the attention kernel's occupancy (one 512-thread
 * workgroup per CU) under its instruction mix, on independent data: 2 = one
 * 16-byte LDS operand read per MFMA, 3 = per 32 MFMAs the VALU work of one
 * 64-key softmax tile (max of 32 scores, 32 fused scale-and-subtract, 32
 * exp2, 16 bf16 pair conversions, 16 two-wide dot products), 4 = both.
 * random_operands != 0 fills the operands with random bf16 values of
 * magnitude 0.5 to 2, 0 with zeros: the power the matrix cores draw, and
 * with it the clock the chip holds, depends on the operand bits.  Runs on
 * stream (a hipStream_t; NULL is the null stream) on the current device: one
 * untimed launch, then the best of three timed ones (about 40 ms in all for
 * shapes 0 and 1, up to about 80 ms for the mixes); waits for them.
 * *tflops receives dense TFLOP/s (2 flops per multiply-add).
 * Errors: XC_ERR_INVALID_ARG (NULL tflops, unknown shape), XC_ERR_HIP. */
xc_status xc_mfma_rate(int32_t shape, int32_t random_operands, void* stream, double* tflops);

/* Measurement aid, not a step of the method: the rate of the global -> LDS
 * request stream (global_load_lds_dwordx4) that the GEMMs stage their
 * operands with, as a function of the row segment one request fetches.
 * 1008 workgroups (two per CU) each stream 24 KB stages of the rows of one
 * of 28 shared row blocks (33 MB in all, as the M-tiles of a GEMM share
 * their rows) through a 3-slot LDS ring two stages ahead, with no
 * arithmetic; each stage takes row_bytes (64, 128 or 256) of every one of
 * its 24 KB / row_bytes rows.  Allocates and frees the 33 MB source (zeros),
 * runs on stream (a hipStream_t; NULL is the null stream), three untimed
 * launches then the best of five timed ones, and waits for them;
 * *tbytes_per_s receives TB/s moved into LDS.
 * Errors: XC_ERR_INVALID_ARG (NULL output, other row_bytes), XC_ERR_OOM,
 * XC_ERR_HIP. */
xc_status xc_lds_dma_rate(int32_t row_bytes, void* stream, double* tbytes_per_s);

#ifdef __cplusplus
}
#endif
#endif /* XCACHE_H */
