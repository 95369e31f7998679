/*
 * l4d.h -- C ABI of the MI355X (gfx950) Llama layer-shard training library.
 *
 * The library computes one GPU's share of a Llama decoder-layer training step
 * (forward and backward) at the shard shapes a 4D-parallel configuration
 * (DP x TP x PP x CP) assigns to it, the tensor-parallel LM head with
 * vocabulary-parallel cross-entropy, and the closed-form per-GPU memory
 * estimate of arXiv 2411.06465 (Fujii, Watanabe, Yokota), Sec. 3.
 *
 * Conventions shared by every entry point
 *  - Every function returns an int status: L4D_OK, or an error code with a
 *    message readable through l4d_last_error() (thread-local).  Nothing is
 *    launched when a call returns L4D_EINVAL or L4D_ENOMEM.
 *  - Device pointers are plain HIP device addresses owned by the caller.  The
 *    library never allocates device memory: it sub-allocates from an arena
 *    the caller creates over memory it owns.
 *  - Work is enqueued on the caller's HIP stream (hipStream_t passed as
 *    void*, NULL = the null stream); no call synchronizes the device.  An
 *    arena must only be used from one stream at a time.
 *  - bf16 = IEEE-style bfloat16 stored as 16-bit words; f32 = float.
 *  - Activations are token-major: [b][tokens][features], row-major.
 *    Weights are [out_features][in_features], row-major (y = x W^T).
 *  - Shard symbols (the paper's Table 1): h hidden, a heads, k kv-heads,
 *    h_ffn FFN width, s sequence, b micro-batch, t TP size, c CP size;
 *    d_h = h/a, a_t = a/t, k_t = k/t, f_t = h_ffn/t, s_c = s/c local tokens,
 *    s_sp = s_c/t sequence-parallel rows.
 */
#ifndef L4D_H
#define L4D_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

enum {
  L4D_OK = 0,
  L4D_EINVAL = 1,  /* bad shape, divisibility, NULL pointer or rank */
  L4D_ENOMEM = 2,  /* the arena cannot hold the request */
  L4D_EDEVICE = 3  /* a HIP call failed (message carries hipGetErrorString) */
};

/* Message of the last failing call on this thread ("" if none). */
const char* l4d_last_error(void);

/* ------------------------------------------------------------------------
 * Model and parallel layout
 * ---------------------------------------------------------------------- */

/* Global model dimensions (not divided by TP). */
typedef struct {
  int64_t hidden;      /* h */
  int64_t n_heads;     /* a */
  int64_t n_kv_heads;  /* k, grouped-query attention group g = a/k */
  int64_t ffn;         /* h_ffn */
  int64_t n_layers;    /* L */
  int64_t vocab;       /* v */
  float rms_eps;       /* RMSNorm epsilon */
  float rope_base;     /* RoPE base (theta) */
} l4d_model;

/* The 4D layout and this GPU's place in it. */
typedef struct {
  int64_t seq;          /* s, global sequence length */
  int64_t micro_batch;  /* b */
  int64_t tp, cp, pp, dp;
  int64_t tp_rank;      /* owns heads [r*a_t, (r+1)*a_t), SP rows [r*s_sp, (r+1)*s_sp) */
  int64_t cp_rank;      /* owns sequence chunks r and 2c-1-r of 2c equal chunks */
} l4d_parallel;

/* ------------------------------------------------------------------------
 * Memory estimate -- Sec. 3, Eqs. 1-18 (host only, touches no device)
 * ---------------------------------------------------------------------- */

typedef struct {
  uint64_t params_per_gpu;       /* Psi of the first pipeline stage of one TP rank:
                                    2hv/t + h + L*ell if p == 1, hv/t + (L/p)*ell else,
                                    ell = 2h^2(1+k/a)/t + 3h*h_ffn/t + 2h (Eqs. 1-3, 6, 7) */
  uint64_t weight_bytes;         /* 2 Psi, bf16 weights (Sec. 3.1) */
  uint64_t grad_bytes;           /* 4 Psi, fp32 gradients */
  uint64_t optim_bytes;          /* 12 Psi / (d c): fp32 master, momentum, variance sharded
                                    over data- and context-parallel ranks (Eqs. 5, 10) */
  uint64_t act_bytes_per_layer;  /* sbh(12 + 4k/a + 8h_ffn/h)/(tc) (Eqs. 12, 15, 17) */
  uint64_t act_bytes;            /* Eq. 17: first stage, L layers + 8sbhp + [p=1] 4sbh(1+v/h), /(tc) */
  uint64_t total_bytes;          /* Eq. 18: weight + grad + optim + act */
  uint32_t inexact;              /* 1 if a term was fractional and rounded up */
} l4d_mem;

/* Returns L4D_EINVAL unless a%k == 0, a%t == 0, k%t == 0, h%a == 0,
 * h_ffn%t == 0, v%t == 0, s%c == 0, L%p == 0, all sizes > 0 and
 * tp*cp*pp*dp is the GPU count implied by dp >= 1.  Exact integer arithmetic. */
int mem_estimate(const l4d_model* model, const l4d_parallel* par, l4d_mem* out);

/* Fit of an estimate in the device memory (Sec. 4.1): the paper
 * finds that a configuration whose estimated total is at most 80% of the GPU
 * memory trains (temporary buffers and fragmentation fit in the rest), one
 * above 100% runs out of memory, and one in between may go either way.
 *   est: a filled l4d_mem (its total_bytes is used);
 *   device_bytes: the GPU memory in bytes (the paper's 40 GB and 94 GB read as
 *   40 and 94 GiB);  *fit: one of the values below.
 * L4D_EINVAL for NULL pointers or device_bytes == 0.  Host only. */
enum { L4D_FITS = 0, L4D_NEAR_LIMIT = 1, L4D_OOM = 2 };
int mem_fit(const l4d_mem* est, uint64_t device_bytes, int* fit);

/* ------------------------------------------------------------------------
 * Arena and activation stash (Sec. 3.2)
 *
 * An arena manages [dev_base, dev_base + capacity) of caller-owned device
 * memory.  The layer forward reserves in it exactly the tensors Sec. 3.2 says
 * a layer keeps for its backward (the "stash"), plus a transient workspace
 * released before the call returns.  The stash lives until the matching
 * backward (or l4d_stash_release) returns it.  The arena is host
 * bookkeeping only; it never reads or writes the device memory.
 * ---------------------------------------------------------------------- */

typedef struct l4d_arena l4d_arena;
typedef struct l4d_stash l4d_stash;

int l4d_arena_create(void* dev_base, uint64_t capacity, l4d_arena** out);
int l4d_arena_destroy(l4d_arena* arena);            /* L4D_EINVAL while stashes are live */
int l4d_arena_stats(const l4d_arena* arena, uint64_t* in_use, uint64_t* peak, uint64_t* capacity);

/* Stashed tensors of one layer call.  Shapes (bf16):
 *   X, XN1, H1, XN2 : [b][s_sp][h]         (norm inputs and outputs, own SP rows)
 *   Q, CTX          : [b][s_c][a_t*d_h]    (post-RoPE queries, attention output)
 *   K, V            : [b][s_c][k_t*d_h]    (post-RoPE keys, values)
 *   GATE, UP, ACT, PROD : [b][s_c][f_t]    (SwiGLU: G, U, silu(G), silu(G)*U)
 * and the auxiliary attention log-sum-exp LSE: f32 [b][a_t][s_c], which
 * FlashAttention keeps but Sec. 3.2 counts as zero. */
enum {
  L4D_STASH_X = 0, L4D_STASH_XN1, L4D_STASH_Q, L4D_STASH_K, L4D_STASH_V, L4D_STASH_CTX,
  L4D_STASH_H1, L4D_STASH_XN2, L4D_STASH_GATE, L4D_STASH_UP, L4D_STASH_ACT, L4D_STASH_PROD,
  L4D_STASH_LSE, L4D_STASH_COUNT
};

/* Reserve a layer stash without launching anything (the forward does this
 * itself; exposed for accounting).  L4D_ENOMEM if it does not fit. */
int l4d_stash_reserve(l4d_arena* arena, const l4d_model* model, const l4d_parallel* par,
                      l4d_stash** out);
/* formula_bytes: sum of the 12 bf16 stash tensors, equal to Eq. 12 / (tc)
 * (LM-head stash: x, xn and the softmax, the LM-head term / (tc); embedding
 * stash: the int64 ids).  aux_bytes: the LSE buffer (0 for the ends).
 * padding_bytes: alignment gaps inside the arena. */
int l4d_stash_bytes(const l4d_stash* stash, uint64_t* formula_bytes, uint64_t* aux_bytes,
                    uint64_t* padding_bytes);
/* Device address and byte size of one stashed tensor (L4D_STASH_* for a layer
 * stash, L4D_HEAD_* / L4D_EMB_* for the stashes of the model's ends). */
int l4d_stash_tensor(const l4d_stash* stash, int which, void** ptr, uint64_t* bytes);
/* Return a stash to its arena without running the backward. */
int l4d_stash_release(l4d_arena* arena, l4d_stash* stash);

/* Transient workspace the forward / backward / LM head take from the arena
 * on top of the stash (so that callers can size an arena). */
int l4d_layer_workspace_bytes(const l4d_model* model, const l4d_parallel* par,
                              uint64_t* fwd_bytes, uint64_t* bwd_bytes);
/* Workspace lm_head_xent takes from the arena: the bf16 logits, plus an fp32
 * n_tokens x hidden buffer when vocab_shard is at least 1024 and not a multiple
 * of 128 (d_hidden is then summed in fp32 over two kernels). */
int l4d_lm_head_workspace_bytes(int64_t n_tokens, int64_t hidden, int64_t vocab_shard,
                                uint64_t* bytes);

/* ------------------------------------------------------------------------
 * Llama decoder layer, one (TP rank, CP rank) shard
 *
 *   xn1 = RMSNorm(x; g1)   [Q|K|V] = xn1 W_qkv^T, RoPE on Q and K
 *   ctx = causal GQA softmax(Q K^T / sqrt(d_h)) V        (FlashAttention)
 *   h1  = x + ctx W_o^T    xn2 = RMSNorm(h1; g2)
 *   [G|U] = xn2 W_gu^T     y = h1 + (silu(G) * U) W_down^T
 * Sec. 3 (architecture, Eqs. 1-2 for the weight shapes, GQA g = a/k),
 * Sec. 3.2 (activations kept: Eqs. 11-12), Sec. 3.2.1 (TP with sequence
 * parallelism), Sec. 2.1 and 3.2.3 (context parallelism).
 * RoPE pairs (i, i+d_h/2) with angle pos * base^(-2i/d_h) at the global
 * position; RMSNorm y = g * x / sqrt(mean(x^2) + eps).
 * ---------------------------------------------------------------------- */

/* This rank's weight shard, bf16. */
typedef struct {
  const void* norm1;    /* [h] */
  const void* qkv;      /* [(a_t + 2 k_t) d_h][h]: q-heads, then k-heads, then v-heads */
  const void* o;        /* [h][a_t d_h] */
  const void* norm2;    /* [h] */
  const void* gate_up;  /* [2 f_t][h]: gate rows then up rows */
  const void* down;     /* [h][f_t] */
} l4d_layer_weights;

/* Weight-gradient accumulators, f32, same shapes; the backward ADDS into them. */
typedef struct {
  float* norm1;
  float* qkv;
  float* o;
  float* norm2;
  float* gate_up;
  float* down;
} l4d_layer_grads;

/* What the collectives of the other ranks would deliver to this rank.
 * All bf16.  "gather" inputs are required when t > 1 (resp. c > 1);
 * "receipt" inputs may be NULL, meaning the peers contribute zero. */
typedef struct {
  const void* remote_k;      /* c>1, required: [b][s - s_c][k_t][d_h], post-RoPE keys of the other
                                CP ranks' chunks, in increasing global order */
  const void* remote_v;      /* c>1, required: same shape, values */
  const void* sp_peer_xn1;   /* t>1, required: [b][(t-1) s_sp][h] peers' norm-1 outputs (all-gather),
                                in rank order without this rank */
  const void* sp_peer_xn2;   /* t>1, required: same, norm-2 outputs */
  const void* sp_peer_o;     /* t>1, receipt: [b][s_sp][h] sum of peers' O-projection partial rows
                                for this rank's rows (reduce-scatter) */
  const void* sp_peer_ffn;   /* t>1, receipt: same for the down projection */
  const void* sp_peer_dy;    /* t>1, required: [b][(t-1) s_sp][h] peers' output gradients */
  const void* sp_peer_dh1;   /* t>1, required: same, peers' gradients at h1 */
  const void* sp_peer_dxn2;  /* t>1, receipt: [b][s_sp][h] peers' partial d(xn2) for own rows */
  const void* sp_peer_dxn1;  /* t>1, receipt: same for d(xn1) */
  const void* cp_peer_dk;    /* c>1, receipt: [b][s_c][k_t][d_h] other CP ranks' dK for local keys
                                (w.r.t. post-RoPE keys) */
  const void* cp_peer_dv;    /* c>1, receipt: same for dV */
} l4d_peer_inputs;

/* What this rank's reduce-scatters would send, bf16 [b][(t-1) s_sp][h] in
 * rank order without this rank.  Any member may be NULL: the rows are then
 * written to workspace and dropped. */
typedef struct {
  void* o_partial;     /* O-projection partial rows of the peers (forward) */
  void* ffn_partial;   /* down-projection partial rows (forward) */
  void* dxn2_partial;  /* gate/up input-gradient partial rows (backward) */
  void* dxn1_partial;  /* QKV input-gradient partial rows (backward) */
} l4d_peer_outputs;

/* Forward.  x, y: bf16 [b][s_sp][h] (own SP rows).  Reserves the stash in
 * `arena` and returns it in *stash_out (consumed by llama_layer_bwd).
 * peers may be NULL when t == c == 1; sends may be NULL. */
int llama_layer_fwd(const l4d_model* model, const l4d_parallel* par, const l4d_layer_weights* w,
                    const void* x, const l4d_peer_inputs* peers, const l4d_peer_outputs* sends,
                    void* y, l4d_arena* arena, l4d_stash** stash_out, void* hip_stream);

/* Backward.  dy, dx: bf16 [b][s_sp][h].  Adds the weight gradients into dw
 * (every member required).  d_remote_k / d_remote_v: bf16 [b][s - s_c][k_t][d_h],
 * this rank's dK/dV for the remote keys, required iff c > 1.  Consumes the
 * stash (returned to the arena when the call returns; the device work is
 * stream-ordered). */
int llama_layer_bwd(const l4d_model* model, const l4d_parallel* par, const l4d_layer_weights* w,
                    const l4d_peer_inputs* peers, const l4d_peer_outputs* sends, l4d_stash* stash,
                    const void* dy, void* dx, const l4d_layer_grads* dw, void* d_remote_k,
                    void* d_remote_v, l4d_arena* arena, void* hip_stream);

/* ------------------------------------------------------------------------
 * LM head + vocabulary-parallel cross-entropy (Sec. 3, LM head of Sec. 3.2)
 *
 * logits = hidden W_lm^T stored bf16 [N][v_t];  LSE_i = logaddexp(local LSE,
 * peer_lse_i) in f32;  loss_i = LSE_i - z_i where z_i is the target's logit
 * (from this shard when vocab_start <= target < vocab_start + v_t, else
 * peer_target_logit_i);  dlogits = (softmax - onehot) * grad_scale (bf16);
 * d_hidden = dlogits W_lm (bf16, overwritten);  d_w_lm += dlogits^T hidden.
 *   hidden: bf16 [N][h];  w_lm: bf16 [v_t][h] rows [vocab_start, +v_t) of the head;
 *   targets: int64 [N] device array of global ids in [0, v);
 *   peer_lse, peer_target_logit: f32 [N] device arrays, NULL iff t == 1;
 *   loss: f32 [N];  d_hidden: bf16 [N][h];  d_w_lm: f32 [v_t][h].
 * The logits live in arena workspace for the duration of the call.
 * ---------------------------------------------------------------------- */
int lm_head_xent(int64_t n_tokens, int64_t hidden, int64_t vocab_shard, int64_t vocab_start,
                 const void* hidden_states, const void* w_lm, const int64_t* targets,
                 const float* peer_lse, const float* peer_target_logit, float grad_scale,
                 float* loss, void* d_hidden, float* d_w_lm, l4d_arena* arena, void* hip_stream);

/* lm_head_xent without an arena, for callers that cannot allocate device
 * memory (code under HIP graph capture, tight serving loops, harnesses that
 * forbid hipMalloc).  Same arguments, layouts, results and errors as
 * lm_head_xent, minus the arena: the logits (and, for a vocabulary shard with
 * a ragged tail, the fp32 sum of d_hidden) live in a 64 MiB array of device
 * memory that the library holds per GPU, i.e. n_tokens * vocab_shard * 2
 * bytes, rounded up to 256, plus n_tokens * hidden * 4 for a ragged shard,
 * must fit in 67,108,864 bytes (e.g. 1024 tokens of a 32000-wide shard);
 * larger problems return L4D_EINVAL before anything is launched.  The call
 * itself allocates nothing (the first call on a device looks up that
 * device's array once).  Every call on one GPU uses the same array: calls
 * that overlap on one device (concurrent streams, or threads) race and give
 * wrong results; calls ordered on one stream are safe. */
int lm_head_xent_noalloc(int64_t n_tokens, int64_t hidden, int64_t vocab_shard, int64_t vocab_start,
                         const void* hidden_states, const void* w_lm, const int64_t* targets,
                         const float* peer_lse, const float* peer_target_logit, float grad_scale,
                         float* loss, void* d_hidden, float* d_w_lm, void* hip_stream);

/* ------------------------------------------------------------------------
 * The ends of the model (Sec. 3.2: the embedding and LM-head activation terms)
 *
 * Vocabulary-parallel embedding.  Rank tp_rank holds rows [v0, v0 + v_t) of
 * the table, v_t = v/t, v0 = tp_rank v_t.  For each of its CP chunk's b*s_c
 * tokens it produces the table row when the id is in range and zeros
 * otherwise; the TP reduce-scatter (sequence parallelism) is explicit:
 *   ids: int64 [b][s_c] device array of global ids in [0, v);
 *   w_emb: bf16 [v_t][h];  receipt: bf16 [b][s_sp][h], the sum of the peers'
 *   partial rows for this rank's rows (NULL = zero);  send: bf16
 *   [b][(t-1) s_sp][h], this rank's partial rows for the peers in rank order
 *   (NULL iff t == 1);  x_out: bf16 [b][s_sp][h], the own rows.
 * The stash keeps the int64 ids (8 b s_c bytes, slot L4D_EMB_IDS): the
 * backward needs nothing else.  The embedding term printed in Sec. 3.2,
 * 8sbhp/(tc), counts 8sbh bytes per micro-batch: h/t times these.
 * embedding_bwd adds, for every token whose id is in range, the all-gathered
 * output gradient (own rows dx: bf16 [b][s_sp][h]; peer rows peer_dx: bf16
 * [b][(t-1) s_sp][h], NULL iff t == 1) into d_w_emb: f32 [v_t][h], with fp32
 * atomic adds (tokens sharing an id add in no fixed order).  It releases the
 * stash.
 *
 * LM-head block: xn = RMSNorm(x; w_norm) on the own rows, all-gathered,
 * logits = xn W_lm^T in FP32 over the vocabulary shard, cross-entropy with
 * the other shards' statistics as inputs (as lm_head_xent), the FP32 softmax
 * kept for the backward.  The stash holds exactly the LM-head term of
 * Sec. 3.2 divided by tc: x and xn (bf16 [b][s_sp][h] each: "2sbh for the
 * output RMSNorm" and "2sbh for the output linear layer") and the softmax
 * (f32 [b*s_c][v_t]: "4sbv"), i.e. 4 s_c b h (1 + v/h) / t bytes.
 *   x: bf16 [b][s_sp][h], the last layer's output (own rows);
 *   w_norm: bf16 [h];  w_lm: bf16 [v_t][h];  targets: int64 [b*s_c];
 *   peer_xn: bf16 [b][(t-1) s_sp][h], the peers' normed rows (NULL iff t == 1);
 *   peer_lse, peer_target_logit: f32 [b*s_c] (NULL iff t == 1);  loss: f32 [b*s_c].
 * lm_head_bwd takes the same weights, targets and peer_xn (the re-gather),
 *   peer_dxn: bf16 [b][s_sp][h], the peers' partial d(xn) for the own rows
 *   (NULL = zero);  dxn_send: bf16 [b][(t-1) s_sp][h] or NULL (then dropped);
 *   dx: bf16 [b][s_sp][h];  d_w_norm: f32 [h] (+=);  d_w_lm: f32 [v_t][h] (+=);
 * with dlogits = (softmax - onehot) * grad_scale, and releases the stash.
 * Requirements: v % t == 0, (v/t) % 8 == 0, h % 8 == 0.
 * ---------------------------------------------------------------------- */
enum { L4D_EMB_IDS = 0, L4D_EMB_COUNT };
enum { L4D_HEAD_X = 0, L4D_HEAD_XN, L4D_HEAD_PROBS, L4D_HEAD_COUNT };

int embedding_fwd(const l4d_model* model, const l4d_parallel* par, const int64_t* ids, const void* w_emb,
                  const void* receipt, void* send, void* x_out, l4d_arena* arena, l4d_stash** stash_out,
                  void* hip_stream);
int embedding_bwd(const l4d_model* model, const l4d_parallel* par, l4d_stash* stash, const void* dx,
                  const void* peer_dx, float* d_w_emb, l4d_arena* arena, void* hip_stream);
int lm_head_fwd(const l4d_model* model, const l4d_parallel* par, const void* x, const void* w_norm,
                const void* w_lm, const int64_t* targets, const void* peer_xn, const float* peer_lse,
                const float* peer_target_logit, float* loss, l4d_arena* arena, l4d_stash** stash_out,
                void* hip_stream);
int lm_head_bwd(const l4d_model* model, const l4d_parallel* par, const void* w_norm, const void* w_lm,
                const int64_t* targets, const void* peer_xn, const void* peer_dxn, void* dxn_send,
                float grad_scale, l4d_stash* stash, void* dx, float* d_w_norm, float* d_w_lm, l4d_arena* arena,
                void* hip_stream);

/* ------------------------------------------------------------------------
 * Optimizer step over one shard of the model states (Sec. 3.1, Eqs. 4-5, 10)
 *
 * Each GPU holds 2 bytes (bf16 weight) and 4 bytes (fp32 gradient) per
 * parameter, plus 12 bytes of optimizer state (fp32 master weight, momentum,
 * variance) for the 1/(d c) of its parameters that it owns under the
 * distributed optimizer.  l4d_adam_step updates such a shard of n parameters
 * in one pass, with the bias-corrected Adam step and decoupled weight decay:
 *   g = grad * grad_scale [* *grad_scale_dev]
 *   m = beta1 m + (1 - beta1) g;   v = beta2 v + (1 - beta2) g^2
 *   master -= lr (m / (1 - beta1^step)) / (sqrt(v / (1 - beta2^step)) + eps)
 *             + lr weight_decay master
 *   weight = bf16(master), rounded to nearest even;  grad = 0 if zero_grad.
 * Arithmetic is fp32; the step-dependent constants are formed in double.
 *   grad, master, m, v: fp32 [n] device arrays, 16-byte aligned;
 *   weight: bf16 [n] device array, 8-byte aligned (the shard's slice of the
 *   full weight, which the data-parallel all-gather then distributes);
 *   the five arrays must not overlap; all are owned by the caller.
 * L4D_EINVAL for n < 0 or n > 2^33, a NULL or misaligned array, overlapping arrays,
 * step < 1, beta1 or beta2 outside [0, 1), eps < 0, or a non-finite lr,
 * weight decay or scale.  n == 0 launches nothing.
 * ---------------------------------------------------------------------- */
typedef struct {
  float lr;
  float beta1, beta2;
  float eps;
  float weight_decay;            /* decoupled: 0 gives plain Adam */
  float grad_scale;              /* multiplies the gradient (1 = none) */
  const float* grad_scale_dev;   /* optional device scalar multiplied in as well
                                    (e.g. a clipping factor computed on the GPU) */
  int64_t step;                  /* 1 for the first step */
  int32_t zero_grad;             /* != 0: clear grad after reading it */
} l4d_adam;

int l4d_adam_step(const l4d_adam* hp, int64_t n, float* grad, float* master, float* m, float* v,
                  void* weight, void* hip_stream);

/* ------------------------------------------------------------------------
 * Kernel timing (HIP events around every launch, on the launch stream)
 * ---------------------------------------------------------------------- */

/* on != 0: record a start/stop event pair around each kernel launch. */
int l4d_profile_enable(int on);
/* Restrict the timing to the launches labelled `name` (NULL or "": all
 * launches).  Each timed launch adds its event pair to the stream. */
int l4d_profile_only(const char* name);
/* Synchronize the recorded events and return, for the kernel `name`, the
 * number of timed launches and the summed duration in milliseconds.  With
 * name == NULL, the totals over all kernels. */
int l4d_profile_read(const char* name, int64_t* launches, double* total_ms);
/* Newline-separated "name launches total_ms" lines into buf (truncated to
 * buf_len); returns the needed length through *needed. */
int l4d_profile_dump(char* buf, uint64_t buf_len, uint64_t* needed);
/* The labels of the timed launches since the last reset, newline-separated,
 * in launch order (e.g. to label the dispatches of an external kernel trace);
 * same buffer convention as l4d_profile_dump. */
int l4d_profile_order(char* buf, uint64_t buf_len, uint64_t* needed);
int l4d_profile_reset(void);

#ifdef __cplusplus
}
#endif

#endif /* L4D_H */
