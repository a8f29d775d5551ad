/*
 * luna.h -- C ABI of the LUNA attention forward pass on AMD Instinct MI355X (gfx950).
 *
 * LUNA ("Learning Kernels for Linear Attention") replaces the softmax kernel by a
 * learned positive-definite kernel k(x, y) = phi(x) . phi(y) and evaluates attention
 * in linear time through the kernelised form, eq. (9) of Section 3.1:
 *
 *     out = phi(Q) (phi(K)^T V) / phi(Q) (phi(K)^T 1)          (row by row)
 *
 * with the feature map of eq. (11) of Section 3.2, envelope h = 1 (Table 5, "no gate"):
 *
 *     phi(x) = (1/sqrt(M)) [ psi_l(w_i . x + b_i) ]_{i = 1..M, l = 1..L}  in R^{M*L}
 *
 * where every channel function psi_l is a scalar MLP 1 -> hidden -> 1 with ReLU
 * activation and (by default) a ReLU on its output (Listing 1, the
 * feature-map code).  The statistics S = phi(K)^T V and z = phi(K)^T 1 are the key-side
 * sufficient statistics of the runtime section (section 4).
 *
 * Conventions shared by every entry point:
 *  - Every data pointer is caller-owned DEVICE memory, row-major and contiguous.
 *    Q, K, V and out are [B, H, n, d]; the library never allocates or frees on a
 *    call, keeps no pointer after it returns and, apart from the static scratch of
 *    luna_attn_fwd_causal_noalloc, has no global mutable state, so calls on
 *    different streams may run concurrently if their workspaces differ.
 *  - `stream` is a hipStream_t (NULL = the null stream).  Work is enqueued on it
 *    asynchronously; LUNA_OK means "enqueued", not "finished".
 *  - All arguments are validated on the host before anything is launched.  A
 *    failed validation returns an error code and enqueues nothing;
 *    luna_last_error() then describes the reason (thread-local string).
 *  - Precision follows `dtype`: LUNA_F32 computes in fp32 throughout (fp32 matrix
 *    cores); LUNA_BF16 takes bf16 Q, K, V and W, multiplies bf16 operands on the
 *    matrix cores with fp32 accumulation, keeps S and z in fp32 (rounded to bf16
 *    as matrix-core operands) and writes bf16 output.  Its channel functions psi
 *    are evaluated in fp32 arithmetic from their exact piecewise-linear form with
 *    fp16 coefficients: on each segment psi = slope (u - a) + value, with a the
 *    segment's breakpoint (fp32) and the value at a, so that the coefficients'
 *    rounding costs at most 2^-11 (|slope (u - a)| + |value|) per element, against
 *    the 2^-8 |phi| of phi's rounding to a bf16 operand.  luna_featuremap and the
 *    streaming step use fp32 coefficients.
 *  - The denominator gets an additive eps: out = num / (den + eps).  With ReLU
 *    features a row can have den = 0; it then yields 0.
 *  - Every problem with d in {32, 64, 128}, L in {1, 2, 4, 8, 16} and M*L <= 256
 *    runs on the GPU.  The shapes below have fused attention kernels (Q, K and V
 *    read once, out written once); the others (one channel per projection with
 *    M = 128 or 256, fp32 at d = 128, ...) take a path of fp32 matrix-core GEMMs
 *    and scans over 64-token chunks (causal) or 512-token pieces (non-causal) with
 *    the features in the workspace: the same results to fp32 rounding, slower, and
 *    about 4 (2 M L + 2 (d + 1)) bytes of workspace per token and head plus
 *    4 M L (d + 1) per chunk or piece (and 16 KiB per causal chunk).
 *      non-causal, (dtype, d, L, M): (f32, 32, 8 or 2, <= 16), (f32, 64, 8, <= 16),
 *        (bf16, 32, 8, <= 16), (bf16, 64, 8, <= 32), (bf16, 64, 4, <= 16),
 *        (bf16, 64, 1, 49..64 or 113..128), (bf16, 128, 8, <= 16);
 *      causal: (f32, 32, 8 or 2, <= 16), (f32, 64, 8, <= 16), (bf16, 32, 8, <= 16),
 *        (bf16, 64, 8, <= 32), (bf16, 128, 8, <= 32).
 *    Other shapes return LUNA_ERR_UNSUPPORTED; there is no host fallback.
 */
#ifndef LUNA_H_
#define LUNA_H_

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum luna_status {
  LUNA_OK = 0,
  LUNA_ERR_INVALID_ARG = 1, /* null pointer, non-positive size, inconsistent parameters */
  LUNA_ERR_UNSUPPORTED = 2, /* valid problem that the built kernels do not cover */
  LUNA_ERR_WORKSPACE = 3,   /* ws_bytes smaller than luna_workspace_bytes() */
  LUNA_ERR_HIP = 4          /* a HIP runtime call or kernel launch failed */
} luna_status;

typedef enum luna_dtype { LUNA_F32 = 0, LUNA_BF16 = 1 } luna_dtype;

/* Operation codes for luna_workspace_bytes(). */
enum {
  LUNA_OP_FEATUREMAP = 0,
  LUNA_OP_ATTN = 1,
  LUNA_OP_ATTN_CAUSAL = 2,
  LUNA_OP_STATE = 3,       /* luna_attn_state */
  LUNA_OP_CAUSAL_STEP = 4, /* luna_attn_causal_step (n = m, the new tokens) */
  LUNA_OP_ATTN_BWD = 5,    /* luna_attn_bwd, causal = 0 */
  LUNA_OP_ATTN_CAUSAL_BWD = 6  /* luna_attn_bwd, causal = 1 */
};

/*
 * Feature-map parameters, eq. (11) of Section 3.2 and Listing 1 (the feature-map
 * code in the Implementation Details appendix).
 *   M       number of projections w_i (rows of W), 1 <= M <= 256
 *   L       channels per projection (outputs of the psi_l), 1 <= L <= 16; D = M*L <= 256
 *   hidden  width of each channel MLP, 1 <= hidden <= 64
 *   shared_channels 0: L separate MLPs 1 -> hidden -> 1 (Listing 1's default);
 *                   1: one MLP 1 -> hidden -> L whose first layer all channels share
 *   nonneg  1: ReLU on every MLP output, so phi >= 0 (Listing 1's default); 0: none
 *   per_head 0: one parameter set shared by all heads (Listing 1's default);
 *            1: H sets, stored head-major (leading dimension H on every array)
 * Arrays (device memory; P = per_head ? H : 1; C1 = shared_channels ? 1 : L):
 *   W     [P][M][d]        element type = the call's dtype (bf16 or fp32)
 *   b     [P][M]           fp32 projection bias (the Fig. 3 caption's u = w_i.x + b_i)
 *   fc1_w [P][C1][hidden]  fp32 first-layer weight (a_lk)
 *   fc1_b [P][C1][hidden]  fp32 first-layer bias   (c_lk)
 *   fc2_w [P][L][hidden]   fp32 second-layer weight (f_lk)
 *   fc2_b [P][L]           fp32 second-layer bias   (g_l)
 * Channel l computes psi_l(u) = relu(g_l + sum_k f_lk relu(a_lk u + c_lk)) (outer
 * relu only when nonneg).  The struct is read during the call only.
 */
typedef struct luna_phi_params {
  int32_t M, L, hidden;
  int32_t shared_channels;
  int32_t nonneg;
  int32_t per_head;
  const void* W;
  const float* b;
  const float* fc1_w;
  const float* fc1_b;
  const float* fc2_w;
  const float* fc2_b;
} luna_phi_params;

/*
 * Bytes of device workspace an operation needs (0 if the arguments are invalid or
 * unsupported).  op is LUNA_OP_*; dtype is the call's dtype (for LUNA_OP_FEATUREMAP
 * the input dtype); chunk is used by LUNA_OP_ATTN_CAUSAL only.  The workspace must
 * be 256-byte aligned.  The workspace holds
 * the exact piecewise-linear tables of the channel MLPs, built on the device at the
 * start of every call, plus partial statistics and counters for long sequences.  It
 * needs no initialisation; it must stay untouched by other work until the call's
 * kernels have finished.
 */
size_t luna_workspace_bytes(int32_t op, luna_dtype dtype, int64_t B, int64_t H, int64_t n,
                            int64_t d, const luna_phi_params* p, int32_t chunk);

/*
 * Feature map phi of eq. (11) of Section 3.2 applied to every row of X [B, H, n, d].
 * phi_out [B, H, n, M*L] receives feature i*L + l (channel index fastest) of each
 * row, in out_dtype.  X and W are in x_dtype.  d must be 32, 64 or 128.
 */
luna_status luna_featuremap(const void* X, luna_dtype x_dtype, int64_t B, int64_t H, int64_t n,
                            int64_t d, const luna_phi_params* p, void* phi_out, luna_dtype out_dtype,
                            void* ws, size_t ws_bytes, void* stream);

/*
 * Non-causal LUNA attention, eq. (9) of Section 3.1:
 *   S = phi(K)^T V, z = phi(K)^T 1 per (b, h);  out = phi(Q) S / (phi(Q) z + eps).
 * Q, K, V, out: [B, H, n, d] in dtype (value width d_v = d).  d in {32, 64, 128}.
 */
luna_status luna_attn_fwd(const void* Q, const void* K, const void* V, luna_dtype dtype,
                          int64_t B, int64_t H, int64_t n, int64_t d, const luna_phi_params* p,
                          float eps, void* out, void* ws, size_t ws_bytes, void* stream);

/*
 * Causal (streaming) LUNA attention: the prefix form of eq. (9) of Section 3.1,
 *   out_t = phi(q_t)^T S_t / (phi(q_t)^T z_t + eps),
 *   S_t = sum_{s <= t} phi(k_s) v_s^T,  z_t = sum_{s <= t} phi(k_s)   (diagonal included),
 * evaluated as a chunked scan: per chunk of `chunk` tokens a masked intra-chunk block
 * plus the carried state.  chunk must be 64.  Same layouts as luna_attn_fwd.
 */
luna_status luna_attn_fwd_causal(const void* Q, const void* K, const void* V, luna_dtype dtype,
                                 int64_t B, int64_t H, int64_t n, int64_t d,
                                 const luna_phi_params* p, int32_t chunk, float eps, void* out,
                                 void* ws, size_t ws_bytes, void* stream);

/*
 * luna_attn_fwd_causal without a workspace argument, for callers that cannot
 * allocate device memory: code under HIP graph capture, tight serving loops and
 * harnesses that forbid allocation.  It computes exactly what luna_attn_fwd_causal
 * computes (the same kernels) and allocates nothing: its workspace is a static
 * array of luna_noalloc_scratch_bytes() bytes (64 MiB) in the library's code object,
 * one per device, held from the library's load until the process ends, on the
 * calling thread's current device (which must be the stream's device).  Problems
 * whose workspace (luna_workspace_bytes with LUNA_OP_ATTN_CAUSAL) exceeds it return
 * LUNA_ERR_WORKSPACE before anything is enqueued.  Every call on a device shares that
 * device's array and needs nothing from an earlier call (every buffer in it is
 * written before it is read), but two calls whose kernels overlap in time on one
 * device -- on different streams, or from different threads -- race on it; order
 * them on one stream.
 */
luna_status luna_attn_fwd_causal_noalloc(const void* Q, const void* K, const void* V, luna_dtype dtype,
                                         int64_t B, int64_t H, int64_t n, int64_t d,
                                         const luna_phi_params* p, int32_t chunk, float eps, void* out,
                                         void* stream);

/* Size in bytes of the static scratch of luna_attn_fwd_causal_noalloc. */
size_t luna_noalloc_scratch_bytes(void);

/*
 * Causal state of a token sequence: the key-side statistics of the runtime section
 * (section 4), which are the prefix state of the streaming form of eq. (9) of
 * Section 3.1 after the sequence's last token,
 *   S = phi(K)^T V   [B, H, M*L, d]   and   z = phi(K)^T 1   [B, H, M*L],
 * fp32 (caller-owned device memory), feature index i*L + l as in luna_featuremap.
 * K, V: [B, H, n, d] in dtype.  accumulate 0: S and z are overwritten; 1: the sums
 * are added to what S and z hold, so that a sequence can be consumed in pieces.
 * The same (dtype, d, L, M) combinations as luna_attn_fwd are built.
 */
luna_status luna_attn_state(const void* K, const void* V, luna_dtype dtype, int64_t B, int64_t H, int64_t n,
                            int64_t d, const luna_phi_params* p, int32_t accumulate, float* S, float* z,
                            void* ws, size_t ws_bytes, void* stream);

/*
 * One streaming (recurrent) step of causal attention, the prefix form of eq. (9) of
 * Section 3.1 continued from the state (S, z) of the tokens before it (from
 * luna_attn_state, an earlier step, or zeros for an empty prefix), over m new tokens
 * per (b, h), in order:
 *   S += phi(k_t) v_t^T;  z += phi(k_t);  out_t = phi(q_t)^T S / (phi(q_t)^T z + eps).
 * S [B, H, M*L, d] and z [B, H, M*L] (fp32, feature i*L + l) are read and updated in
 * place; they must not alias Q, K, V, out or the workspace, and S must be 16-byte
 * aligned.  Q, K, V, out:
 * [B, H, m, d] in dtype.  The state is carried in fp32 throughout.  Steps of 16
 * tokens or more run per 16-token stage in the chunked form of the same prefix sums
 * (fp32 matrix products), shorter ones token by token; the two agree up to rounding.
 * Stepping a sequence from zeros gives what luna_attn_fwd_causal computes, up to
 * rounding.
 * tables_ready 0: the call builds the channel tables in the workspace, as every
 * other entry point does; 1: it uses the tables an earlier luna_attn_causal_step
 * left in the same workspace, enqueued before it on the same stream, with the same
 * parameters (same arrays, unchanged contents) -- for decode loops, where the table
 * build would otherwise cost as much as the step itself.  With tables_ready = 1 and
 * a workspace that holds no tables built that way the results are undefined (the
 * kernels clamp what they read from it, so the call still ends and stays inside its
 * buffers).  The call also keeps a copy of z in the workspace for the duration of
 * its kernels.
 * The same (d, L, M) combinations as luna_featuremap are built.
 */
luna_status luna_attn_causal_step(const void* Q, const void* K, const void* V, luna_dtype dtype, int64_t B,
                                  int64_t H, int64_t m, int64_t d, const luna_phi_params* p, float eps,
                                  int32_t tables_ready, float* S, float* z, void* out, void* ws, size_t ws_bytes,
                                  void* stream);

/*
 * Gradients of the feature-map parameters (fp32 device memory, shaped like the
 * parameter arrays of luna_phi_params: W [P][M][d] (fp32 whatever the call's dtype),
 * b [P][M], fc1_w and fc1_b [P][C1][hidden], fc2_w [P][L][hidden], fc2_b [P][L]).
 */
typedef struct luna_phi_grads {
  float* W;
  float* b;
  float* fc1_w;
  float* fc1_b;
  float* fc2_w;
  float* fc2_b;
} luna_phi_grads;

/*
 * Backward pass of luna_attn_fwd (causal = 0) or luna_attn_fwd_causal (causal = 1),
 * for training the feature map end to end (section 5.1) and the fine-tuning of
 * converted models (section 5.2): for a loss L with dO = dL/dout [B, H, n, d], writes
 *   dQ, dK, dV = dL/dQ, dL/dK, dL/dV   [B, H, n, d] in dtype (overwritten), and, if
 *   grads is not NULL, the gradients of every feature-map parameter (overwritten),
 * by the chain rule through out = phi(Q) S / (phi(Q) z + eps) (eq. (9) of Section 3.1,
 * prefix states for the causal form) and phi of eq. (11) of Section 3.2 (Listing 1's
 * channel MLPs, ReLU'(0) = 0).  Q, K, V, dO: [B, H, n, d] in dtype; same parameters and
 * eps as the forward call.  All arithmetic is fp32 (the features are recomputed; the
 * channel functions through their exact piecewise-linear form, whose slopes give
 * dpsi/du).  Supported: d in {32, 64, 128}, L in {1, 2, 4, 8, 16}, M*L <= 256 and
 * H <= 65535.  The workspace (LUNA_OP_ATTN_BWD / LUNA_OP_ATTN_CAUSAL_BWD in
 * luna_workspace_bytes) holds the features, the per-chunk states and the partial
 * parameter sums: about 4 (2 M L + 3 (d + 1)) bytes per token and head, plus
 * 2 x 4 M L (d + 1) per chunk of 64 tokens for the causal form.
 */
luna_status luna_attn_bwd(const void* Q, const void* K, const void* V, const void* dO, luna_dtype dtype,
                          int64_t B, int64_t H, int64_t n, int64_t d, const luna_phi_params* p,
                          int32_t causal, float eps, void* dQ, void* dK, void* dV,
                          const luna_phi_grads* grads, void* ws, size_t ws_bytes, void* stream);

/*
 * Attention distillation, the first stage of the conversion recipe (Implementation
 * Details appendix: every pretrained weight frozen, the feature map trained so that
 * LUNA's attention distribution matches the teacher's softmax attention, eq. (1) of
 * Section 2).  Per query row t, over the keys s that t sees (all, or s <= t when
 * causal = 1; n_t of them):
 *   teacher  A_ts = softmax_s(q_t . k_s / sqrt(d))
 *   student  Ahat_ts = (P_ts + eps/n_t) / (den_t + eps), P = phi(Q) phi(K)^T,
 *            den_t = sum_s P_ts: LUNA's weights of eq. (9) of Section 3.1, smoothed
 *            into an exact distribution (a key with P_ts = 0 keeps a finite loss)
 *   row_loss[b][h][t] = -sum_s A_ts log Ahat_ts  (fp32, device memory, [B][H][n];
 *            the soft cross-entropy: KL(A_t || Ahat_t) plus the teacher's entropy)
 * and, if grads is not NULL, the gradients of the mean of row_loss over the B H n rows
 * with respect to every feature-map parameter (overwritten; the teacher is a fixed
 * target, Q and K get no gradient).  phi is eq. (11) of Section 3.2 (Listing 1's
 * channel MLPs) with the parameters p; eps >= 0 (with eps = 0 a visible key with
 * P_ts = 0 gives an infinite loss).  Q, K: [B, H, n, d] in dtype.  Nothing of size
 * n x n is stored: the work is quadratic in n, the memory linear.  bf16 calls take the
 * features and the products in bf16 with fp32 accumulation; fp32 calls compute in fp32.
 * Supported: d in {32, 64, 128}; D = M L in {64, 128, 256} (bf16) or {64, 128} (fp32);
 * the feature-map and, for grads, the backward pass's limits on (d, L, M).
 */
size_t luna_distill_workspace_bytes(luna_dtype dtype, int64_t B, int64_t H, int64_t n, int64_t d,
                                    const luna_phi_params* p, int32_t param_grads);
luna_status luna_distill(const void* Q, const void* K, luna_dtype dtype, int64_t B, int64_t H, int64_t n, int64_t d,
                         const luna_phi_params* p, int32_t causal, float eps, float* row_loss,
                         const luna_phi_grads* grads, void* ws, size_t ws_bytes, void* stream);

/*
 * Feature-map variants.  The map of eq. (11) of Section 3.2 is a template, phi(x) =
 * h(x)/sqrt(M) [psi_l(w_i . x + b_i)]; fixing h and psi by hand gives the random-feature
 * maps of Section 3.1, and the kernel ablation of Section 5.4 (Table 5) changes its
 * form.  Every variant uses the projection u = W x + b of `base` (W, b, M, per_head):
 *   LUNA_PHI_RFF_COS     sqrt(2/M) cos(u_i)                       D = M
 *   LUNA_PHI_RFF_SINCOS  (1/sqrt(M)) (sin u_i, cos u_i)           D = 2M, feature 2i + l
 *   LUNA_PHI_PERFORMER   (1/sqrt(M)) exp(u_i - |x|^2/(2 sqrt(d))) D = M (psi = exp, h(x) =
 *                        exp(-|x|^2/(2 sqrt d)); with w_i = omega_i / d^(1/4), omega_i ~
 *                        N(0, I), phi(x).phi(y) estimates exp(x.y / sqrt(d)))
 *   LUNA_PHI_MLP         the channel MLPs of `base` (L, hidden, shared_channels, nonneg,
 *                        fc*) with the hidden activation `act` (relu, gelu in its erf
 *                        form, silu, tanh), evaluated directly, then optionally:
 *                        env_w [P][L][d], env_b [P][L] (fp32): a tokenwise envelope
 *                        sigmoid(env_w x + env_b) in [0,1]^L multiplying channel l of
 *                        every projection (Table 5's envelope-gated map);
 *                        ch_rms = 1: Listing 1's channel RMS normalisation over the whole
 *                        call, y_l *= min(target / (rms_l + 1e-6), 1), rms_l = sqrt(mean
 *                        over every (batch, head, token, projection) of y_l^2 + 1e-6)
 *                        (a two-pass map; non-causal use only, as it pools all tokens);
 *                        bank [P][L] (fp32): Table 5's Bank+Coef map, feature i =
 *                        (1/sqrt(M)) sum_l bank_l y_l(u_i), D = M;
 *                        otherwise D = M L, feature i L + l.  Order: psi, envelope,
 *                        channel RMS, bank sum, 1/sqrt(M).
 * The variants compute in fp32 from the call's input (no piecewise-linear tables).
 * Limits: M <= 256, D <= 512; for LUNA_PHI_MLP L <= 16 and hidden <= 64.  The other
 * kinds take no envelope, bank or channel RMS (LUNA_ERR_INVALID_ARG).
 */
typedef enum luna_phi_kind {
  LUNA_PHI_MLP = 0,
  LUNA_PHI_RFF_COS = 1,
  LUNA_PHI_RFF_SINCOS = 2,
  LUNA_PHI_PERFORMER = 3
} luna_phi_kind;

typedef enum luna_act { LUNA_ACT_RELU = 0, LUNA_ACT_GELU = 1, LUNA_ACT_SILU = 2, LUNA_ACT_TANH = 3 } luna_act;

typedef struct luna_phi_variant {
  int32_t kind;                /* luna_phi_kind */
  int32_t act;                 /* luna_act (LUNA_PHI_MLP) */
  const luna_phi_params* base; /* projection (and, for LUNA_PHI_MLP, the channel MLPs) */
  const float* env_w;          /* optional envelope [P][L][d] (both or neither) */
  const float* env_b;          /* [P][L] */
  const float* bank;           /* optional Bank+Coef coefficients [P][L] */
  int32_t ch_rms;              /* 0 or 1 */
  float ch_rms_target;         /* > 0 (Listing 1's default is 0.1) */
} luna_phi_variant;

/* Features per row of a variant (D), or -1 when the description is invalid. */
int64_t luna_phi_variant_features(const luna_phi_variant* v);

/* Workspace of luna_featuremap_variant: 0 bytes without channel RMS; with it, about
 * 4 B H n M L bytes (y of every row in fp32, kept between the two passes) plus 256 KiB.
 * 0 also on invalid arguments: check the call's status. */
size_t luna_featuremap_variant_workspace_bytes(luna_dtype x_dtype, int64_t B, int64_t H, int64_t n, int64_t d,
                                               const luna_phi_variant* v);

/* The variant map of every row of X [B, H, n, d] (x_dtype) into phi_out [B, H, n, D]
 * (out_dtype).  W is in x_dtype; every other parameter is fp32.  d in {32, 64, 128}. */
luna_status luna_featuremap_variant(const void* X, luna_dtype x_dtype, int64_t B, int64_t H, int64_t n,
                                    int64_t d, const luna_phi_variant* v, void* phi_out, luna_dtype out_dtype,
                                    void* ws, size_t ws_bytes, void* stream);

/* Workspace of luna_attn_fwd_features. */
size_t luna_attn_features_workspace_bytes(luna_dtype phi_dtype, luna_dtype dtype, int64_t B, int64_t H, int64_t n,
                                          int64_t d, int64_t D, int32_t causal, int32_t chunk);

/*
 * Kernel attention, eq. (9) of Section 3.1, for given features: phiQ, phiK [B, H, n, D]
 * in phi_dtype (any feature map: a variant, luna_featuremap's output, ...), V and out
 * [B, H, n, d] in dtype; out = phiQ S / (phiQ z + eps) with S, z over every token, or
 * (causal = 1) over the prefix s <= t, evaluated as the chunked scan with chunk 64.
 * Features may be signed: the denominator is then the caller's concern.  Runs on the
 * fp32 GEMM path (bf16 features widened to fp32), or, for causal bf16 calls with
 * (d, D) = (128, 256) or (64, 128), on the causal scan kernel reading the bf16 features.
 * 1 <= d <= 256, 1 <= D <= 512.
 */
luna_status luna_attn_fwd_features(const void* phiQ, const void* phiK, luna_dtype phi_dtype, const void* V,
                                   luna_dtype dtype, int64_t B, int64_t H, int64_t n, int64_t d, int64_t D,
                                   int32_t causal, int32_t chunk, float eps, void* out, void* ws, size_t ws_bytes,
                                   void* stream);

/* Static description of a status code. */
const char* luna_status_string(luna_status s);

/* Detail of the last error returned on the calling thread ("" if none). */
const char* luna_last_error(void);

#ifdef __cplusplus
}
#endif

#endif /* LUNA_H_ */
