/*
 * mebp.h — C ABI of the MeBP checkpointed LoRA training step on AMD Instinct MI355X
 * (gfx950).
 *
 * MeBP (memory-efficient backpropagation, Sec. 3 and Algorithm 1 of the paper) trains
 * LoRA adapters of a decoder-only transformer with gradient checkpointing at every block
 * boundary. The forward loop stores only the block-boundary activations ("checkpoints");
 * the backward loop walks the blocks in reverse, decompresses each block's int4 base
 * weights just before use, recomputes the block's forward from its checkpoint, and
 * backpropagates into the LoRA A/B gradients and the block-input gradient (the backward
 * graph B_i(x, dE/dy, w) -> (dE/dx, dE/dw) of Sec. 3). Blocks are every transformer
 * layer plus the final linear layer and the cross-entropy loss (Sec. 4.2), the last two
 * fused into one call here.
 *
 * Conventions shared by every entry point:
 *  - Tensor arguments are DEVICE pointers owned by the caller; structs are host memory
 *    read during the call only. Nothing is allocated by the library: all scratch lives in
 *    the caller's workspace `ws` of at least mebp_workspace_bytes() bytes.
 *  - Activations are fp32, token-major: row n = b*T + t of a [B*T][hidden] matrix.
 *    Attention columns are head-major (column h*head_dim + e).
 *  - Compressed base weights (Sec. 3, 4-bit symmetric INT4 of every non-LoRA parameter
 *    incl. the embedding): per projection `q4` uint8 [out][in/2] (two's-complement
 *    nibbles, element 2j of a row in the low nibble of byte j) and `scale` raw fp16 bits
 *    [out][ceil(in/group)]; dequantised value W[o][i] = q[o][i] * scale[o][i/group].
 *    The last group of a row may be shorter than `group`.
 *  - LoRA: y = x W^T + (alpha/rank) (x A^T) B^T with A fp32 [rank][in], B fp32 [out][rank].
 *  - Every call validates all arguments first. On error it enqueues nothing, records a
 *    message for mebp_last_error() and returns a negative mebp_status. On success it
 *    enqueues work on `stream` and returns MEBP_OK without synchronising; outputs are
 *    valid once the stream reaches that point. Calls on one stream are ordered; two calls
 *    sharing one workspace must not run concurrently.
 *  - Results are deterministic: the same inputs give bit-identical outputs (no atomics
 *    in any reduction).
 */
#ifndef MEBP_H
#define MEBP_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

/* A hipStream_t passed as an opaque pointer; NULL selects the null stream. */
typedef void* mebp_stream_t;

typedef enum {
  MEBP_OK = 0,
  MEBP_EINVAL = -1,       /* null pointer, negative size, inconsistent config            */
  MEBP_EUNSUPPORTED = -2, /* valid but unsupported shape (head_dim, rank, alignment)     */
  MEBP_EWORKSPACE = -3,   /* ws_bytes smaller than mebp_workspace_bytes()                */
  MEBP_EHIP = -4          /* a HIP runtime call or kernel launch failed                  */
} mebp_status;

/* Projection indices used by every per-projection array. */
enum { MEBP_Q = 0, MEBP_K = 1, MEBP_V = 2, MEBP_O = 3, MEBP_GATE = 4, MEBP_UP = 5, MEBP_DOWN = 6,
       MEBP_NPROJ = 7 };

typedef struct {
  int32_t n_layers;      /* L >= 1                                                        */
  int32_t hidden;        /* d, multiple of 32                                             */
  int32_t n_heads;       /* Hq                                                            */
  int32_t n_kv_heads;    /* Hkv, divides Hq (grouped-query attention, consecutive heads)  */
  int32_t head_dim;      /* 64, 128 or 256                                                */
  int32_t ffn;           /* F, multiple of 16                                             */
  int32_t vocab;         /* V, multiple of 32; 0 when no LM head is used                  */
  int32_t act;           /* 0 = SwiGLU (SiLU gate), 1 = GeGLU (tanh-approximated GELU)    */
  float rms_eps;         /* RMSNorm epsilon                                               */
  float rope_theta_global; /* RoPE base of global layers                                  */
  float rope_theta_local;  /* RoPE base of sliding-window layers                          */
  int32_t window;        /* sliding window W of local layers: key j visible to query i    */
                         /* iff i-W < j <= i; 0 = no window                               */
  int32_t global_every;  /* 0: every layer global; k > 0: layer l global iff (l+1)%k == 0 */
  int32_t group;         /* int4 scale group along the input dim; must be 32              */
  int32_t lora_rank;     /* r: 8 or 16                                                    */
  float lora_alpha;      /* LoRA scale s = alpha / r                                      */
  uint32_t lora_mask;    /* bit p set: projection p carries a LoRA adapter                */
  uint32_t arch;         /* architecture details beyond the shapes (MEBP_ARCH_* bits); 0 =  */
                         /* the plain pre-norm block                                      */
} mebp_config;

/* mebp_config.arch bits (Sec. 4 trains Qwen2.5 and Gemma3 models; these are the parts of
 * their blocks beyond a plain pre-norm Llama-style block). The extra frozen weights are
 * fp32 vectors in mebp_layer_base.                                                      */
enum {
  MEBP_ARCH_QKV_BIAS = 1,     /* Qwen2.5: q, k, v projections add a bias                   */
  MEBP_ARCH_QK_NORM = 2,      /* Gemma3: RMSNorm over each head of q and of k, before RoPE */
  MEBP_ARCH_SANDWICH = 4,     /* Gemma3: RMSNorm on the attention output and on the MLP    */
                              /* output before each residual add                          */
  MEBP_ARCH_EMBED_SCALE = 8   /* Gemma3: embedding output times sqrt(hidden) (the tied LM  */
                              /* head uses the table unscaled)                            */
};

typedef struct {
  const uint8_t* q4;        /* [out][in/2]                                                */
  const uint16_t* scale;    /* [out][ceil(in/group)] fp16 bits                            */
} mebp_q4;

typedef struct {
  mebp_q4 w[MEBP_NPROJ];    /* q [Hq*dh][d], k,v [Hkv*dh][d], o [d][Hq*dh],               */
                            /* gate,up [F][d], down [d][F]                                */
  const float* norm_attn;   /* [d] fp32 RMSNorm weight before attention (frozen)          */
  const float* norm_mlp;    /* [d] fp32 RMSNorm weight before the MLP (frozen)            */
  const float* bias[3];     /* MEBP_ARCH_QKV_BIAS: q [Hq*dh], k, v [Hkv*dh]; else unused  */
  const float* q_norm;      /* MEBP_ARCH_QK_NORM: [dh] weights of the q and k head norms  */
  const float* k_norm;
  const float* post_attn_norm; /* MEBP_ARCH_SANDWICH: [d] weights of the norms on the    */
  const float* post_mlp_norm;  /* attention output and on the MLP output                  */
} mebp_layer_base;

typedef struct {
  const float* A[MEBP_NPROJ]; /* [r][in]; NULL where the projection is not adapted        */
  const float* B[MEBP_NPROJ]; /* [out][r]                                                 */
} mebp_layer_lora;

typedef struct {
  float* dA[MEBP_NPROJ];    /* [r][in], overwritten (not accumulated); NULL if not adapted */
  float* dB[MEBP_NPROJ];    /* [out][r]                                                   */
} mebp_layer_lora_grad;

/* Bytes of workspace every entry point below needs for this config and batch shape
 * (B sequences of T tokens). Pure host computation; returns 0 for an invalid config. */
size_t mebp_workspace_bytes(const mebp_config* cfg, int32_t B, int32_t T);

/* forward_i of Algorithm 1 for transformer layer `layer` (Sec. 3, "Runtime
 * implementation"): x_out = F(x_in) with the int4 weights decompressed inside the GEMMs.
 *   x_in  [B*T][d] fp32 checkpoint of the layer input (read only)
 *   x_out [B*T][d] fp32 checkpoint of the layer output (written; must not alias x_in)   */
int mebp_layer_forward_ckpt(const mebp_config* cfg, int32_t layer, const mebp_layer_base* base,
                            const mebp_layer_lora* lora, const float* x_in, float* x_out,
                            int32_t B, int32_t T, void* ws, size_t ws_bytes, mebp_stream_t stream);

/* backward_i of Algorithm 1 (Sec. 3 backward graph B_i(x, dE/dy, w) -> (dE/dx, dE/dw)):
 * recomputes the layer forward from its checkpoint and backpropagates.
 *   x_ckpt [B*T][d] fp32 layer input checkpoint
 *   dy     [B*T][d] fp32 gradient of the loss w.r.t. the layer output
 *   dx     [B*T][d] fp32 gradient w.r.t. the layer input, or NULL to skip it; may alias dy
 *   grads  LoRA gradients of the adapted projections (overwritten)                       */
int mebp_layer_recompute_backward(const mebp_config* cfg, int32_t layer, const mebp_layer_base* base,
                                  const mebp_layer_lora* lora, const float* x_ckpt, const float* dy,
                                  float* dx, const mebp_layer_lora_grad* grads, int32_t B, int32_t T,
                                  void* ws, size_t ws_bytes, mebp_stream_t stream);

/* Final block (Sec. 4.2: the final linear layer and the cross-entropy loss layer):
 * RMSNorm, logits against the tied int4 embedding, next-token cross-entropy averaged over
 * the B*(T-1) positions that have a target (position T-1 of each sequence has none), and
 * the gradient w.r.t. the last checkpoint.
 *   emb        tied embedding [V][d/2] / [V][d/32]
 *   norm_final [d] fp32
 *   x_last     [B*T][d] fp32 output checkpoint of the last layer
 *   ids        [B][T] int32 token ids in [0, V)
 *   loss       one fp32 on the device (written)
 *   dx_last    [B*T][d] fp32 (written)                                                    */
int mebp_lm_head_ce_backward(const mebp_config* cfg, const mebp_q4* emb, const float* norm_final,
                             const float* x_last, const int32_t* ids, int32_t B, int32_t T,
                             float* loss, float* dx_last, void* ws, size_t ws_bytes,
                             mebp_stream_t stream);

/* Embedding lookup with decompression of the tied int4 table (Sec. 3: the embeddings are
 * INT4 too): x0[b*T+t][:] = E[ids[b][t]][:] in fp32.                                    */
int mebp_embed(const mebp_config* cfg, const mebp_q4* emb, const int32_t* ids, int32_t B, int32_t T,
               float* x0, mebp_stream_t stream);

/* Backpropagation(x) of Algorithm 1 for one batch of token ids: embedding, forward loop
 * storing every checkpoint, final block, reverse loop recomputing each layer.
 *   layers, lora, grads  host arrays of cfg->n_layers entries
 *   ckpt  [(L+1)][B*T][d] fp32 checkpoint storage (written; ckpt[l] is the input of layer l)
 *   loss  one fp32 on the device (written)
 *   dx0   [B*T][d] fp32 gradient w.r.t. the embedding output, or NULL to skip layer 0's
 *         input gradient (the embedding is frozen)                                       */
int mebp_train_step(const mebp_config* cfg, const mebp_q4* emb, const mebp_layer_base* layers,
                    const float* norm_final, const mebp_layer_lora* lora, const int32_t* ids,
                    int32_t B, int32_t T, float* ckpt, float* loss, const mebp_layer_lora_grad* grads,
                    float* dx0, void* ws, size_t ws_bytes, mebp_stream_t stream);

/* ---------------- optimizer step on the LoRA parameters ------------------------------
 * Sec. 3 ("Runtime implementation"): the gradient of a batch may be obtained by gradient
 * accumulation over smaller inputs, and only the LoRA weights, their gradients and the
 * optimizer state are kept for the optimizer; Sec. 4.1: the optimizer is AdamW.        */

typedef struct {
  float* A[MEBP_NPROJ];     /* [r][in] fp32, updated in place; NULL if not adapted      */
  float* B[MEBP_NPROJ];     /* [out][r]                                                 */
} mebp_layer_lora_state;    /* writable LoRA-shaped tensors: parameters or moments      */

typedef struct {
  float lr, beta1, beta2, eps, weight_decay;
  float grad_scale;         /* the gradients are multiplied by this first               */
  int32_t step;             /* t >= 1, the index of this update (bias corrections)      */
} mebp_adamw_hparams;

/* acc = (first ? 0 : acc) + scale * grads for every adapted LoRA tensor of every layer
 * (with scale = 1/k over k micro-batches of equal size: the gradient of their mean loss).
 *   grads, acc  host arrays of cfg->n_layers entries; device tensors 16-byte aligned;
 *               acc may alias grads. Enqueued on stream; returns < 0 on invalid input.  */
int mebp_lora_grad_accumulate(const mebp_config* cfg, const mebp_layer_lora_grad* grads,
                              const mebp_layer_lora_grad* acc, float scale, int32_t first,
                              mebp_stream_t stream);

/* One AdamW update (decoupled weight decay) of every adapted LoRA tensor of every layer,
 * elementwise in fp32:
 *   g = grad_scale * grad;  m = beta1 m + (1 - beta1) g;  v = beta2 v + (1 - beta2) g^2;
 *   p = p - lr (weight_decay p + (m / (1 - beta1^t)) / (sqrt(v / (1 - beta2^t)) + eps)).
 *   params, m, v  host arrays of cfg->n_layers entries, device tensors updated in place
 *                 (callers start with m = v = 0); grads: host array, tensors read only.
 * All device tensors 16-byte aligned and distinct. Requires 0 <= beta1, beta2 < 1,
 * eps >= 0, step >= 1 and finite values; returns < 0 and enqueues nothing otherwise.     */
int mebp_lora_adamw_step(const mebp_config* cfg, const mebp_layer_lora_state* params,
                         const mebp_layer_lora_grad* grads, const mebp_layer_lora_state* m,
                         const mebp_layer_lora_state* v, const mebp_adamw_hparams* hp,
                         mebp_stream_t stream);

/* Backpropagation(x) of Algorithm 1 with the checkpoints kept in host memory (Sec. 3,
 * "Runtime implementation": the checkpoints are memory-mapped during the forward pass
 * instead of being kept in memory). Same kernels, order and results as mebp_train_step,
 * bit for bit; only where the checkpoints live differs. Checkpoint x_i is computed into
 * device ring slot i % ring_slots, copied to ckpt_host[i] by a copy stream as soon as it is
 * written, and copied back into its slot ring_slots - 1 layers before the reverse loop
 * recomputes layer i (the last ring_slots checkpoints never leave the ring). Device memory
 * for checkpoints drops from (L+1) to ring_slots activations of [B*T][d] fp32.
 *   ckpt_host  [(L+1)][B*T][d] fp32 pinned host memory (hipHostMalloc; pageable memory is
 *              refused), written; complete when the stream reaches the end of the step
 *   ring       [ring_slots][B*T][d] fp32 device memory, 16-byte aligned (scratch)
 *   ring_slots 4 .. 16
 * Other arguments as mebp_train_step. Calls on one device share its copy stream and are
 * serialised on the host.                                                              */
int mebp_train_step_offload(const mebp_config* cfg, const mebp_q4* emb, const mebp_layer_base* layers,
                            const float* norm_final, const mebp_layer_lora* lora, const int32_t* ids, int32_t B,
                            int32_t T, float* ckpt_host, float* ring, int32_t ring_slots, float* loss,
                            const mebp_layer_lora_grad* grads, float* dx0, void* ws, size_t ws_bytes,
                            mebp_stream_t stream);

/* ---------------- entry point for callers that cannot allocate ----------------------
 * For callers that can neither allocate device memory nor hand over a workspace: code
 * under HIP graph capture, tight serving loops, harnesses that forbid hipMalloc.
 * mebp_layer_recompute_backward with its scratch in a buffer of MEBP_STATIC_SCRATCH_BYTES
 * that the library holds on every device it runs on (reserved with the library's code on
 * that device and kept until the process ends) instead of a caller workspace: same kernels,
 * same order, same results. The call allocates nothing; arguments as
 * mebp_layer_recompute_backward without ws / ws_bytes. The layer must fit:
 * mebp_workspace_bytes() of the same config with vocab = 0 must not exceed
 * MEBP_STATIC_SCRATCH_BYTES (a Qwen2.5-0.5B-shaped layer at 256 tokens does), else the
 * call returns MEBP_EWORKSPACE and enqueues nothing. Every call on a device shares that
 * device's buffer and leaves its contents behind (no result depends on them): calls that
 * overlap on one device, from two streams or two host threads, race and must be
 * serialised by the caller.                                                            */
#define MEBP_STATIC_SCRATCH_BYTES ((size_t)64 << 20)
int mebp_layer_recompute_backward_static(const mebp_config* cfg, int32_t layer, const mebp_layer_base* base,
                                         const mebp_layer_lora* lora, const float* x_ckpt, const float* dy,
                                         float* dx, const mebp_layer_lora_grad* grads, int32_t B, int32_t T,
                                         mebp_stream_t stream);

/* Message for the last non-zero status returned on the calling thread ("" if none). */
const char* mebp_last_error(void);

/* ---------------- test and diagnostic entry points ---------------------------------- */

/* Workspace guards, a debug mode (also on when MEBP_WS_GUARD=1 is in the environment when
 * the library loads). On, every workspace slot is followed by a guard region of at least
 * 256 bytes holding a known pattern, so mebp_workspace_bytes() returns more (size the
 * workspace with the mode already set; a workspace sized without it is refused with
 * MEBP_EWORKSPACE) and mebp_workspace_offset() moves. Every entry point that takes a
 * workspace (the static-scratch one included) then fills the guards before its first
 * kernel, checks them after its last one on the caller's stream and waits for that stream
 * (so a guarded call cannot be captured into a graph); an overwritten guard fails the call
 * with MEBP_EWORKSPACE, the message naming the slot. Results are those of the unguarded
 * call. mebp_set_workspace_guards returns the previous mode (0 off, 1 on); switch it only
 * while no call is in flight. mebp_workspace_guard_check checks the guards of a workspace
 * that a guarded call used, without filling them first: MEBP_OK, MEBP_EWORKSPACE (names
 * the slot), or MEBP_EINVAL when the mode is off or an argument is bad.                  */
int mebp_set_workspace_guards(int32_t on);
int mebp_workspace_guard_check(const mebp_config* cfg, int32_t B, int32_t T, void* ws, size_t ws_bytes,
                               mebp_stream_t stream);

/* Decompression alone (Algorithm 1, decompress): out_f32[r][c] = q*s exactly and/or
 * out_bf16[r][c] = bf16 bits of that value rounded to nearest even (either may be NULL).
 * cols must be a multiple of 8; group as in mebp_config.                                 */
int mebp_dequant_q4(const mebp_q4* w, int32_t rows, int32_t cols, int32_t group, float* out_f32,
                    uint16_t* out_bf16, mebp_stream_t stream);

/* One production dequant-GEMM kernel on caller operands (test aid for the bit-exact check of
 * the decompression fused into the products, Algorithm 1's LazyLoadAndDecompressWeights):
 * one split, no LoRA term, no residual, fp32 outputs.
 *   forward kinds (the layer projections and the LM-head logits):
 *     out[m][n] = sum_k X[m][k] * fp16_rne(W[n][k]),   X fp16 [M][n_in], out [M][n_out]
 *   transposed kinds (the input gradients and the LM head's dH):
 *     out[m][c] = sum_n G[m][n] * bf16_rne(W[n][c]),   G bf16 [M][n_out], out [M][n_in]
 * with W [n_out][n_in] the decompressed weight (int4 codes times fp16 scale per 32 inputs).
 * A one-hot X (or G) makes each output one decompressed weight in the kernel's operand
 * type, exactly. n_in and n_out multiples of 16, 1 <= M <= 65536, n_in, n_out <= 65536,
 * x and out 16-byte aligned; MEBP_EINVAL / MEBP_EUNSUPPORTED otherwise.                  */
enum {
  MEBP_TEST_GEMM_NT = 0,        /* forward, 128 x 128 tiles (few tokens)                  */
  MEBP_TEST_GEMM_NT_BIG128 = 1, /* forward, 256 x 128 tiles, weights staged in registers  */
  MEBP_TEST_GEMM_NT_BIG256 = 2, /* forward, 256 x 256 tiles, weights staged in registers  */
  MEBP_TEST_GEMM_NT_LDS = 3,    /* forward, 256 x 256 tiles, activations loaded into LDS  */
  MEBP_TEST_GEMM_TN = 4,        /* transposed, 128 x 128 tiles                            */
  MEBP_TEST_GEMM_TN_BIG = 5,    /* transposed, 256 x 128 tiles                            */
  MEBP_TEST_GEMM_NT_LDS_W16 = 6, /* MEBP_TEST_GEMM_NT_LDS on plain fp16 weights: w->q4      */
                                 /* points at W fp16 [n_out][n_in], w->scale is unused (the */
                                 /* same kernel without the decompression, to measure it)   */
  MEBP_TEST_GEMM_TN_BIG_W16 = 7  /* MEBP_TEST_GEMM_TN_BIG on plain bf16 weights, likewise   */
};
int mebp_test_gemm(int32_t kind, const mebp_q4* w, int32_t n_out, int32_t n_in, const void* x, int32_t M,
                   float* out, mebp_stream_t stream);

/* Byte offset inside the workspace of an intermediate kept by the last
 * mebp_layer_recompute_backward / mebp_layer_forward_ckpt on that workspace (for tests).
 * Returns (size_t)-1 for an unknown slot. Slots are listed by mebp_workspace_slot_name. */
size_t mebp_workspace_offset(const mebp_config* cfg, int32_t B, int32_t T, int32_t slot);
const char* mebp_workspace_slot_name(int32_t slot);

/* Diagnostic per-kernel timing. mebp_kernel_timing(1) creates a pool of HIP events
 * (no device memory is allocated) and from then on brackets every kernel launch of this
 * library with an event pair tagged by kernel name and algorithmic flops / bytes;
 * mebp_kernel_timing(0) stops and frees the pool. Records beyond the pool's capacity
 * (`capacity` launches) are not timed. mebp_kernel_timing_report synchronises on the
 * recorded events and writes a JSON array
 *   [{"kernel": name, "launches": n, "ms": total, "flops": total, "bytes": total}, ...]
 * into buf (truncated to len); it returns the length the full report needs including the
 * terminating NUL, or a negative mebp_status. Host-thread-unsafe; for benchmarks only.  */
int mebp_kernel_timing(int32_t enable, int32_t capacity);
int mebp_kernel_timing_report(char* buf, size_t len);

/* Measurement aid. From this call on, every launch of the kernel named `kernel` (a name
 * as it appears in the timing report) is issued `times` times back to back on its stream;
 * kernel = NULL or times <= 1 switches it off. Results are unchanged, since every kernel
 * that may be repeated computes its outputs from inputs it does not overwrite; the kernels
 * that update a buffer in place are refused with MEBP_EINVAL ("gemm_tn_act_bwd",
 * "splitk_finalize_actbwd", "rope_fwd", "qkv_post", "headnorm_bwd", "ce_chunk_stats",
 * "ce_probs", "ce_dh_accum", "ce_final", "lora_adamw", "lora_grad_accumulate"). With timing enabled, each burst of repeated launches is bracketed by one
 * event pair and reported as `times` launches, so the report's average is the kernel's
 * back-to-back in-stream duration. Host-thread-unsafe; for benchmarks only. */
int mebp_kernel_repeat(const char* kernel, int32_t times);

#ifdef __cplusplus
}
#endif
#endif /* MEBP_H */
