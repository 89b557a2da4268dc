/*
 * vla.h -- C ABI of the MI355X (gfx950) flow-matching action-expert library.
 *
 * The library runs the action stage of the VLA inference pattern (paper,
 * Sec. 3.1 and Algorithm 1): a cached vision-language prefix is projected once
 * into a per-layer cross-attention K/V cache (Appendix A.2, item 3), and a
 * short action chunk is integrated over T solver steps by an action expert that
 * cross-attends to that cache; the chunk is then denormalised (Sec. 3.3 item iv).
 * A ternary-weight x int8-activation GEMM (Sec. 4.5, the W2A8 matmul of
 * BitVLA) is exported on its own.
 *
 * Conventions for every call:
 *  - Buffers are DEVICE pointers owned by the caller unless marked HOST.
 *  - Work is enqueued asynchronously on `stream` (a hipStream_t; NULL = the
 *    null stream); results are valid once the stream has synchronised.
 *  - Every argument is validated on the host before any work is enqueued.  On
 *    failure the call returns a non-zero vla_status, enqueues nothing, writes
 *    nothing, and vla_last_error() describes the failure.  Nothing throws.
 *  - Device pointers must be 16-byte aligned.
 *  - A model is not safe for concurrent calls; use one model per stream.
 */
#ifndef VLA_H_
#define VLA_H_

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
  VLA_OK = 0,
  VLA_E_ARG = 1,          /* null pointer, misaligned pointer, bad enum value */
  VLA_E_SHAPE = 2,        /* inconsistent or unsupported dimensions */
  VLA_E_UNSUPPORTED = 3,  /* valid request this build does not implement */
  VLA_E_NOMEM = 4,        /* device allocation failed */
  VLA_E_DEVICE = 5,       /* a HIP call or kernel launch failed, or an earlier call failed on the
                             device (see vla_model_check) */
  VLA_E_NONFINITE = 6     /* NaN/Inf in the output (VLA_CHECK_FINITE=1 only) */
} vla_status;

/* Weight element type of the dense matrices. */
typedef enum { VLA_W_F32 = 0, VLA_W_BF16 = 1, VLA_W_TERNARY = 2 } vla_wtype;

/* Sublayer pattern of each expert layer (execution order):
 *   SELF_CROSS     : self-attention, cross-attention, MLP
 *   JOINT          : joint attention (one softmax over [prefix ; chunk]), MLP
 *   ALT_CROSS_SELF : even layers cross-attention + MLP, odd layers self-attention + MLP
 *                    (SmolVLA's expert; the alternating DiT head of the GR00T series)
 *   CROSS          : cross-attention + MLP in every layer (Evo-1's cross-attention DiT
 *                    head); the action tokens interact only through the prefix */
typedef enum { VLA_PAT_SELF_CROSS = 0, VLA_PAT_JOINT = 1, VLA_PAT_ALT_CROSS_SELF = 2, VLA_PAT_CROSS = 3 } vla_pattern;

/* MLP form: GELU(u W1^T) W2^T, or act(u Wg^T) * (u Wu^T) then Wd, with act
 * GELU (tanh form) for GEGLU, SiLU for SWIGLU, relu^2 for RELU2GLU. */
typedef enum { VLA_MLP_GELU = 0, VLA_MLP_GEGLU = 1, VLA_MLP_SWIGLU = 2, VLA_MLP_RELU2GLU = 3 } vla_mlp;

typedef struct vla_config {
  int32_t n_layers;        /* L */
  int32_t d_model;         /* d (even) */
  int32_t n_heads;         /* H query heads */
  int32_t head_dim;        /* hd: 64, 128 or 256 (fp32 models: 64 or 128) */
  int32_t n_kv_heads;      /* G (H % G == 0); head i reads K/V head floor(i*G/H) */
  int32_t d_ff;            /* F (multiple of 16; of 64 for ternary models) */
  int32_t d_prefix;        /* d_p, width of the prefix hidden states */
  int32_t n_action;        /* n, action tokens per chunk */
  int32_t d_action;        /* A */
  int32_t d_state;         /* S, proprioceptive state width */
  int32_t pattern;         /* vla_pattern */
  int32_t mlp;             /* vla_mlp */
  int32_t wtype;           /* vla_wtype */
  int32_t head_regression; /* 1: single-pass regression head, no time input, n_steps must be 1 */
  float rms_eps;           /* adaRMS epsilon (e.g. 1e-6) */
} vla_config;

typedef struct vla_model vla_model; /* opaque */

/* Number of entries vla_model_create expects in its weight table. */
int32_t vla_weight_count(const vla_config* cfg);

/*
 * Create a model from a table of device pointers (copied into library-owned,
 * possibly re-tiled memory; the caller may free its buffers once this returns).
 * Synchronous.  Table order and shapes ([out][in] row-major, y = x W^T):
 *   globals: W_in [d][A], b_in [d], W_s [d][S], b_s [d], E_pos [n][d],
 *            then W_t1 [d][d], b_t1 [d], W_t2 [d][d], b_t2 [d], W_fm [2d][d], b_fm [2d]
 *            (regression head instead: mod_f [2d] fp32),
 *            then W_out [A][d], b_out [A];
 *   per layer: W_mod [3*n_sub*d][d], b_mod [3*n_sub*d] (regression: mod [3*n_sub*d] fp32),
 *            then per attention sublayer W_q [H*hd][d], W_k, W_v [G*hd][d] (self/joint),
 *            W_kc, W_vc [G*hd][d_p] (cross/joint), W_o [d][H*hd];
 *            per MLP W1 [F][d], W2 [d][F] (GELU) or W_g, W_u [F][d], W_d [d][F].
 * Dense matrices are fp32 (VLA_W_F32) or bf16 (VLA_W_BF16 and VLA_W_TERNARY);
 * biases and modulation tables are fp32.  With VLA_W_TERNARY every attention
 * and MLP matrix is packed 2-bit [N][K/4] bytes (code w+1 of w[n][4j+i] in bits
 * 2i..2i+1 of byte j) and is followed in the table by a device pointer to its
 * fp32 per-tensor scale.
 * n_sub = 3 (SELF_CROSS) or 2.  Errors: VLA_E_ARG, VLA_E_SHAPE, VLA_E_NOMEM, VLA_E_DEVICE.
 */
vla_status vla_model_create(const vla_config* cfg, const void* const* weights, int32_t n_weights,
                            vla_model** out);
void vla_model_destroy(vla_model* model);

/* Bytes of the cross-attention K/V cache for `batch` requests of `prefix_len`
 * prefix tokens: Lc * 2 * batch * G * prefix_len * hd * elem, with Lc the number
 * of layers that have a cross or joint sublayer and elem 4 (fp32 models) or 2.
 * Returns 0 on invalid arguments. */
size_t vla_kv_cache_bytes(const vla_model* model, int32_t batch, int32_t prefix_len);

/*
 * Project the prefix hidden states once into the cross-attention cache.
 * prefix_hidden: [batch][prefix_len][d_p], fp32 for fp32 models, bf16 otherwise.
 * kv_cache: [Lc][2][batch][G][prefix_len][hd] (K then V), same element type;
 * kv_cache_bytes must equal vla_kv_cache_bytes(model, batch, prefix_len).
 * The cache stays valid until the caller overwrites it (one denoising
 * integration, Appendix A.2 item 3).
 */
vla_status vla_prefix_kv_build(vla_model* model, const void* prefix_hidden, int32_t batch,
                               int32_t prefix_len, void* kv_cache, size_t kv_cache_bytes,
                               void* stream);

/*
 * vla_prefix_kv_build for callers that cannot allocate device memory (code
 * under HIP graph capture, tight serving loops, harnesses that forbid
 * hipMalloc): same arguments, same result, and it calls no hipMalloc, hipFree
 * or allocating library routine.  Its scratch (the W2A8 int8 codes and row
 * scales of the prefix rows; dense models use none) lives in a static device
 * array of 16 MiB per GPU, held until the process ends:
 * batch * prefix_len * (d_prefix + 4) bytes (plus alignment) must fit, else
 * VLA_E_UNSUPPORTED before any work is enqueued.  Every call on one GPU
 * shares that array, so calls that overlap on one GPU (other streams, other
 * threads) race; calls ordered on one stream do not.
 */
vla_status vla_prefix_kv_build_noalloc(vla_model* model, const void* prefix_hidden, int32_t batch,
                                       int32_t prefix_len, void* kv_cache, size_t kv_cache_bytes,
                                       void* stream);

/*
 * Integrate one action chunk per request (Algorithm 1, solver loop and
 * denormalisation).  For k = 0..n_steps-1 the expert evaluates the velocity v
 * at (a_k, tau_k) and a_{k+1} = a_k + (tau_{k+1} - tau_k) v; the regression
 * head (n_steps == 1) returns its output directly.  Finally
 * actions = a * act_std + act_mean.
 *   kv_cache   : as built by vla_prefix_kv_build for (batch, prefix_len)
 *   noise      : [batch][n][A] fp32 (a_0)
 *   state      : [batch][S] fp32
 *   t_schedule : HOST [n_steps+1] fp32, finite; copied before the call returns
 *   n_steps    : 1..64
 *   act_mean, act_std : [A] fp32 or NULL (identity)
 *   actions_out: [batch][n][A] fp32; may alias noise
 * Requests are independent; weights and the schedule are shared.
 * With the environment variable VLA_CHECK_FINITE=1 the call synchronises the
 * stream and returns VLA_E_DEVICE if the integration failed on the device,
 * else VLA_E_NONFINITE if any output is NaN or Inf.
 * Device-side failure: every barrier wait of the persistent step kernel (loop
 * mode 2) is bounded; if one times out, every workgroup leaves, that call's
 * actions_out is filled with NaN, and the failure is recorded in the model.
 * It is reported, once, as VLA_E_DEVICE by the first vla_denoise (before it
 * enqueues anything) or vla_model_check on the same model that runs after the
 * failed call has completed.  Each launch starts with a cleared record, so
 * one failure does not affect later calls.
 */
vla_status vla_denoise(vla_model* model, const void* kv_cache, size_t kv_cache_bytes, int32_t batch,
                       int32_t prefix_len, const float* noise, const float* state,
                       const float* t_schedule, int32_t n_steps, const float* act_mean,
                       const float* act_std, float* actions_out, void* stream);

/*
 * Synchronise `stream` and report a device-side failure of an earlier
 * vla_denoise on this model that has not been reported yet (VLA_E_DEVICE,
 * once; see vla_denoise), else VLA_OK.  Errors: VLA_E_ARG, VLA_E_DEVICE.
 */
vla_status vla_model_check(vla_model* model, void* stream);

/*
 * W2A8 GEMM (Sec. 4.5): acc[m][n] = sum_k x[m][k] * w[n][k], int32, exact.
 *   x        : [M][K] int8, row-major
 *   w_packed : [N][K/4] bytes in the 2-bit layout of vla_model_create
 *   acc_out  : [M][N] int32
 * K % 4 == 0, K <= 2^23 / 128 (so |acc| < 2^31 is guaranteed).  A code of 3 in
 * w_packed is undefined input.  M, N >= 0; M*N == 0 enqueues nothing.
 */
vla_status vla_ternary_gemm(const int8_t* x, const uint8_t* w_packed, int32_t M, int32_t N, int32_t K,
                            int32_t* acc_out, void* stream);

/* Options:
 *  VLA_OPT_LOOP_MODE: loop driver of vla_denoise, 0 = one launch per phase on
 *    the stream, 1 = the same launches captured once in a HIP graph and
 *    replayed, 2 (default) = one persistent kernel (every workgroup resident
 *    at once) for the whole step loop where the model and device support it
 *    (batch 1, bf16, joint attention,
 *    H % 8 == 0, the shape limits of the team layout, none of the causal,
 *    RoPE or state-token variants), else as 1.
 *  VLA_OPT_PROFILE: R in 1..1000 = time every launch of the following
 *    vla_denoise calls with HIP events (launch-per-phase driver; read with
 *    vla_profile_read).  Each launch runs R times back to back between its
 *    event pair and the reported time is the mean; with R > 1 the in-place
 *    updates repeat, so such a call is for timing only and its outputs are
 *    not the integration's.  0 = off.
 *  VLA_OPT_TRACE: 1 = the persistent kernel records a phase timeline (the
 *    100 MHz device clock before and after every barrier, one workgroup per
 *    team); 2 = every workgroup records its first 256 marks; read it with
 *    vla_test_persist_trace (vla_test.h).
 *  VLA_OPT_ATTN_SPLITS: work split of the attention launches of loop modes
 *    0 and 1: key splits (value % 100, 1..64) and head groups per K/V head
 *    (value / 100, 1..8); 0 in either part = automatic (default 0).
 *    Discards the model's cached plans.
 *  VLA_OPT_CAUSAL_SELF: architecture variant of the expert's attention
 *    (the paper leaves the action-token mask open; SmolVLA-style experts
 *    use a causal one): 1 = action token i attends only to action tokens
 *    0 .. i in self and joint attention, every prefix row stays visible;
 *    0 (default) = bidirectional.  Set it before the first vla_denoise that
 *    should use it; changing it discards the cached plans.  Causal models
 *    run on loop modes 0 and 1 (the persistent kernel is unmasked).
 *  VLA_OPT_ROPE_BASE: architecture variant (the paper's expert has no
 *    positions beyond the learned E_pos): value = base > 1 of a rotary
 *    position embedding (rotate-half form) on the queries and keys of self
 *    and joint attention; 0 (default) = none.  Action token i sits at
 *    position i in self attention and P + i in joint attention, whose cached
 *    prefix keys vla_prefix_kv_build rotates to positions 0 .. P-1 (build
 *    the cache after setting it).  Discards the cached plans; such models run
 *    on loop modes 0 and 1.
 *  VLA_OPT_STATE_TOKEN: architecture variant of the input embedding (the
 *    paper adds the projected state to every action token; pi0-style experts
 *    give it a token of its own): 1 = each request runs n + 1 token rows, row
 *    0 = s W_s^T + b_s and row 1 + i = a_i W_in^T + b_in + E_pos[i]; the
 *    state row takes part in attention (and is token 0 for the causal mask and
 *    RoPE) but yields no action, so actions_out keeps its [B, n, d_action]
 *    layout.  0 (default) = the paper's embedding.  Discards the cached plans;
 *    such models run on loop modes 0 and 1.
 *  VLA_OPT_PERSIST_SPIN_LIMIT: polls of one barrier wait of the persistent
 *    step kernel before it gives up (value >= 0; -1 = the default, 2^20
 *    polls, about 0.25 s).  For tests of the failure path: a small value makes waits time
 *    out, which every workgroup survives (see vla_denoise). */
enum { VLA_OPT_LOOP_MODE = 0, VLA_OPT_PROFILE = 1, VLA_OPT_TRACE = 2, VLA_OPT_ATTN_SPLITS = 3,
       VLA_OPT_CAUSAL_SELF = 4, VLA_OPT_ROPE_BASE = 5, VLA_OPT_STATE_TOKEN = 6,
       VLA_OPT_PERSIST_SPIN_LIMIT = 7 };
vla_status vla_model_set_option(vla_model* model, int32_t option, int32_t value);

/* One timed launch of a profiled vla_denoise call. */
enum { VLA_OP_GEMM = 0, VLA_OP_GEMM_GLU = 1, VLA_OP_ATTENTION = 2, VLA_OP_TERNARY = 3,
       VLA_OP_QUANTIZE = 4, VLA_OP_SMALL = 5, VLA_OP_ATTN_MERGE = 6, VLA_OP_PERSIST = 7 };
typedef struct vla_op_time {
  int32_t kind;   /* VLA_OP_* */
  int32_t M;      /* GEMM rows (tokens) / attention queries */
  int32_t N;      /* GEMM output columns / attention keys */
  int32_t K;      /* GEMM reduction length / attention head_dim */
  double bytes;   /* algorithmic bytes: weights + cached K/V read once, activations in and out */
  double flops;   /* algorithmic flops (integer ops for the W2A8 GEMM) */
  float ms;       /* mean duration of the launch (HIP events, see VLA_OPT_PROFILE) */
} vla_op_time;

/* Copy the launch timings of the model's last profiled vla_denoise call into
 * out[0 .. max_ops-1] (synchronising on its events).  Returns the number of
 * launches of that call, or -1 if nothing was profiled. */
int32_t vla_profile_read(vla_model* model, vla_op_time* out, int32_t max_ops);

/* ---- The prefix stage: backbone prefill --------------------------------------
 * The vision-language backbone encodes the prefix tokens in one bidirectional
 * pass (Algorithm 1: h = VLM-Prefix(I, l, s); Sec. 3.1: the prefix stage is
 * compute-bound like LLM prefill), and its final-layer hidden states, taken
 * before the output projection, are the cross-attention source that
 * vla_prefix_kv_build projects (App. A.2 items 1 and 2: full hidden states, a
 * bidirectional mask so that every prefix token attends to every other).
 * The paper gives no layer equations; this library's layer is a pre-norm
 * transformer layer:
 *   x += W_o Attn(RMS(x)(1 + g_att))   (bidirectional, GQA, RoPE on q and k)
 *   x += MLP(RMS(x)(1 + g_mlp))        (vla_mlp forms, as in the expert)
 * and the output is RMS(x)(1 + g_f), RMS(x) = x / sqrt(mean(x^2) + rms_eps).
 * With VLA_W_TERNARY every projection is the W2A8 linear of vla_model_create
 * (per-token int8 activations, packed 2-bit weights, int8 matrix cores). */
typedef struct vla_backbone_config {
  int32_t n_layers;        /* L */
  int32_t d_model;         /* d (multiple of 8, of 64 for ternary; <= 4096) */
  int32_t n_heads;         /* H */
  int32_t head_dim;        /* 64, 128 or 256 */
  int32_t n_kv_heads;      /* G (H % G == 0, H / G <= 8) */
  int32_t d_ff;            /* F */
  int32_t mlp;             /* vla_mlp */
  int32_t wtype;           /* VLA_W_BF16 or VLA_W_TERNARY */
  float rope_base;         /* > 1: rotate-half RoPE of q and k, row p of a request at position p; 0: none */
  float rms_eps;
} vla_backbone_config;

typedef struct vla_backbone vla_backbone; /* opaque */

/* Entries vla_backbone_create expects, or -1 for an invalid config. */
int32_t vla_backbone_weight_count(const vla_backbone_config* cfg);

/*
 * Create a backbone from a table of device pointers (copied into library
 * memory; the caller may free its buffers once this returns).  Synchronous.
 * Order: g_f [d] fp32; then per layer g_att [d] fp32, W_q [H*hd][d],
 * W_k [G*hd][d], W_v [G*hd][d], W_o [d][H*hd], g_mlp [d] fp32, then
 * W1 [F][d], W2 [d][F] (GELU) or W_g, W_u [F][d], W_d [d][F].  Matrices are
 * bf16 [out][in], or with VLA_W_TERNARY packed 2-bit [N][K/4] each followed
 * by a pointer to its fp32 per-tensor scale (the layout of vla_model_create).
 * Errors: VLA_E_ARG, VLA_E_SHAPE, VLA_E_UNSUPPORTED, VLA_E_NOMEM, VLA_E_DEVICE.
 */
vla_status vla_backbone_create(const vla_backbone_config* cfg, const void* const* weights, int32_t n_weights,
                               vla_backbone** out);
void vla_backbone_destroy(vla_backbone* backbone);

/*
 * Prefill: embeds [batch][prefix_len][d] bf16 (the prefix token embeddings:
 * vision-encoder patches, text, state) -> hidden_out [batch][prefix_len][d]
 * bf16, the final-layer hidden states after the final norm, ready for
 * vla_prefix_kv_build of an expert with d_prefix = d.  Requests are
 * independent; rows of one request attend to each other bidirectionally.
 * The workspace for (batch, prefix_len) is allocated by the first call of
 * that shape and kept by the backbone.  batch * prefix_len <= 65536.
 * Errors: VLA_E_ARG, VLA_E_SHAPE, VLA_E_UNSUPPORTED, VLA_E_NOMEM, VLA_E_DEVICE.
 */
vla_status vla_prefix_prefill(vla_backbone* backbone, const void* embeds, int32_t batch, int32_t prefix_len,
                              void* hidden_out, void* stream);

/* Thread-local message for the last non-OK status of this thread. */
const char* vla_last_error(void);
const char* vla_status_string(int32_t status);

#ifdef __cplusplus
}
#endif
#endif /* VLA_H_ */
