/*
 * axon.h - C ABI of the MI355X decoder forward pass (prefill + greedy decode).
 *
 * The library runs the inference hot path of the decoder-only Llama/Qwen-style
 * models that the Axon compiler emits and benchmarks (Results section,
 * Experimental Setup; Technical Supplement, "Python Overhead"): RMSNorm,
 * QKV/O projections with rotary positions, causal grouped-query attention over
 * a KV cache, and the SwiGLU MLP, followed by the final norm, the output head
 * and a greedy argmax.
 *
 * The calls follow the paper's framing of a model: a definition (here the
 * typed configuration struct, the analogue of the ``Config.dim @@hidden_size``
 * lookups of the built-in Config module) plus a flat, path-keyed weight map as
 * found in a safetensors checkpoint (Introduction; ``_param("layers.0.
 * self_attn.q_proj.weight")`` in the Python-overhead study).  As with the
 * paper's typechecker, every shape is checked before anything executes.
 *
 * Conventions for every call
 *   - Every int-returning call returns AXON_OK (0) or a negative axon_status;
 *     nothing aborts.  axon_last_error() returns a thread-local message for the
 *     last failing call on the calling thread.
 *   - All argument checks run on the host before any work is enqueued; a call
 *     that fails validation enqueues nothing and leaves the model unchanged.
 *   - GPU work is enqueued asynchronously on the caller's hipStream_t (passed as
 *     void*; NULL means the default stream).  Only axon_init_model
 *     synchronizes.  The caller must not use one model from two streams at once.
 *   - "device pointer" means memory allocated with hipMalloc (or by a framework
 *     on the same device); "host pointer" means ordinary CPU memory.
 */
#ifndef AXON_H
#define AXON_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef struct axon_model axon_model; /* opaque; owned by the library */

enum axon_status {
  AXON_OK = 0,
  AXON_E_INVALID = -1,  /* bad argument: NULL pointer, bad config value, bad count */
  AXON_E_SHAPE = -2,    /* a weight's shape does not match the configuration */
  AXON_E_MISSING = -3,  /* a required weight is absent, or an unknown/duplicate name is given */
  AXON_E_DTYPE = -4,    /* a weight's dtype differs from the model dtype */
  AXON_E_CAPACITY = -5, /* batch, sequence length, token count or page table beyond capacity */
  AXON_E_OOM = -6,      /* device allocation failed */
  AXON_E_HIP = -7       /* a HIP runtime call failed (message carries hipGetErrorString) */
};

enum axon_dtype { AXON_BF16 = 1, AXON_F32 = 2 };
/* Model family.  AXON_ARCH_LLAMA: RMSNorm, rotary positions, SwiGLU MLP
 * (Llama / Qwen / Mistral / DeepSeek-MoE layouts).  AXON_ARCH_GPT2: the GPT-2
 * definition of the Technical Supplement ("A Complete Model Definition"):
 * LayerNorm with bias, learned positions added to the token embedding, one
 * fused c_attn projection with bias, multi-head attention without rotation,
 * c_proj with bias, GELU (tanh form) MLP with biases, head tied to the token
 * embedding. */
enum axon_arch { AXON_ARCH_LLAMA = 0, AXON_ARCH_GPT2 = 1 };

/* Model definition and capacities.  Field meanings follow the HF config keys
 * that the generated code reads (hidden_size, num_hidden_layers, ...). */
typedef struct {
  int32_t hidden;         /* D; multiple of 64 */
  int32_t n_layers;       /* L >= 1 */
  int32_t n_heads;        /* H; a multiple of n_kv_heads */
  int32_t n_kv_heads;     /* KV; H / KV <= 16 and (H / KV) * head_dim <= 1536 */
  int32_t head_dim;       /* hd; 64 or 128 */
  int32_t intermediate;   /* I; multiple of 64 */
  int32_t vocab;          /* V >= 1 */
  float rms_eps;          /* RMSNorm epsilon (inside the square root), > 0 */
  double rope_theta;      /* RoPE base, > 1 */
  int32_t qkv_bias;       /* 1: q/k/v projections carry a bias (Qwen-style) */
  int32_t tie_embeddings; /* 1: the output head reuses model.embed_tokens.weight */
  int32_t dtype;          /* AXON_BF16 or AXON_F32 (weights, KV cache, activations) */
  int32_t max_batch;      /* sequence slots, 1..1024 */
  int32_t max_seq;        /* tokens per sequence (prompt + generated), >= 1 */
  int32_t max_tokens;     /* largest prefill token count per call; 0 = max_batch*max_seq */
  int32_t kv_page_size;   /* 0: contiguous cache; else tokens per page, a multiple of 16 */
  int32_t kv_num_pages;   /* page-pool size when kv_page_size > 0 */
  /* Mixture of experts (the MoE built-in's softmax top-k router and grouped
   * experts; Built-In Libraries, "Activations and specialized modules").
   * n_experts == 0: every layer has the dense MLP and the fields below are
   * ignored.  Otherwise layers first_moe_layer.. replace it by: probabilities
   * = softmax of the router logits over the n_experts; the top_k experts by
   * probability (ties to the lowest index) weighted by their probabilities
   * (divided by their sum when norm_topk_prob == 1); each expert a SwiGLU MLP
   * of moe_intermediate; plus, when n_shared_experts > 0, an always-active
   * SwiGLU MLP of n_shared_experts * moe_intermediate added unweighted.
   * Requires dtype AXON_BF16. */
  int32_t n_experts;        /* 0, or 2..256 routed experts */
  int32_t top_k;            /* experts per token, 1..min(n_experts, 8) */
  int32_t moe_intermediate; /* multiple of 64 */
  int32_t n_shared_experts; /* >= 0 */
  int32_t first_moe_layer;  /* 0..n_layers: the layers before it keep the dense MLP */
  int32_t norm_topk_prob;   /* 0 or 1 */
  /* Sliding-window attention (the masking built-in's window; Mistral-style):
   * a query at position p attends to keys max(0, p - W + 1) .. p.  The cache
   * still holds every position.  0: full causal attention. */
  int32_t sliding_window;   /* 0 or >= 1 */
  /* AXON_ARCH_LLAMA or AXON_ARCH_GPT2.  For GPT-2: n_kv_heads == n_heads,
   * qkv_bias == 1 and tie_embeddings == 1 (the definition's fixed choices),
   * rms_eps is the LayerNorm epsilon, rope_theta is ignored, dtype must be
   * AXON_BF16 and n_experts 0. */
  int32_t arch;
  int32_t max_positions;    /* GPT-2: rows of the learned position table; max_seq <= max_positions */
} axon_config;

/* One entry of the flat weight map.  Names follow the HF Llama/Qwen2 layout:
 *   model.embed_tokens.weight                 [V, D]
 *   model.layers.{i}.input_layernorm.weight   [D]
 *   model.layers.{i}.self_attn.q_proj.weight  [H*hd, D]   (.bias [H*hd] iff qkv_bias)
 *   model.layers.{i}.self_attn.k_proj.weight  [KV*hd, D]  (.bias [KV*hd] iff qkv_bias)
 *   model.layers.{i}.self_attn.v_proj.weight  [KV*hd, D]  (.bias [KV*hd] iff qkv_bias)
 *   model.layers.{i}.self_attn.o_proj.weight  [D, H*hd]
 *   model.layers.{i}.post_attention_layernorm.weight [D]
 *   model.layers.{i}.mlp.gate_proj.weight     [I, D]
 *   model.layers.{i}.mlp.up_proj.weight       [I, D]
 *   model.layers.{i}.mlp.down_proj.weight     [D, I]
 * and in a mixture-of-experts layer (i >= first_moe_layer) instead of the mlp.* above:
 *   model.layers.{i}.mlp.gate.weight          [n_experts, D]  (the router)
 *   model.layers.{i}.mlp.experts.{e}.gate_proj.weight / up_proj.weight  [moe_intermediate, D]
 *   model.layers.{i}.mlp.experts.{e}.down_proj.weight                   [D, moe_intermediate]
 *   model.layers.{i}.mlp.shared_experts.{gate,up,down}_proj.weight      (iff n_shared_experts > 0;
 *                                          intermediate n_shared_experts * moe_intermediate)
 *   model.norm.weight                         [D]
 *   lm_head.weight                            [V, D]  (present iff tie_embeddings == 0)
 * Linear weights are [out, in] row-major.  Every tensor is contiguous,
 * row-major, in the model dtype.  ``data`` is a host pointer if on_device == 0,
 * else a device pointer on the current device. */
typedef struct {
  const char* name;
  int32_t dtype;     /* AXON_BF16 or AXON_F32 */
  int32_t ndim;      /* 1 or 2 */
  int64_t shape[2];  /* shape[1] ignored when ndim == 1 */
  const void* data;
  int32_t on_device;
} axon_weight;

/* Validate the configuration and the weight map, allocate device memory on
 * the current HIP device, copy and repack the weights (the caller keeps
 * ownership of its buffers and may free them once the call returns), allocate
 * the KV cache (contiguous or a page pool) and the work buffers, and build the
 * rotary cos/sin table.  Synchronizes ``stream`` before returning.
 * On success *out receives the handle; on failure *out is set to NULL and no
 * device memory stays allocated. */
int axon_init_model(const axon_config* cfg, const axon_weight* weights, int32_t n_weights,
                    void* stream, axon_model** out);

/* Prefill: start ``batch`` fresh sequences in slots 0..batch-1 (every earlier
 * sequence is dropped) and run the forward pass over their prompts.  This is
 * the model's forward over a whole prompt with an empty cache: positions
 * start at the past length 0 (Built-In Libraries, "Positions and cache
 * management"), each layer is the pre-norm attention + gated-MLP block of the
 * complete model definition (Technical Supplement), attention is causal
 * grouped-query attention with scale 1/sqrt(head_dim) (Built-In Libraries,
 * "Attention and masking", "Tensor and math built-ins"), and the greedy token
 * is the argmax of the final logits that generate() takes (Results,
 * Measures).  The page table is given here, on the host, and kept by the
 * library for the decode steps that follow (so it can be validated without a
 * device-to-host copy); axon_step replaces rows of it later.
 *   d_tokens      device int32 [sum S_b], the prompts packed back to back;
 *   d_cu_seqlens  device int32 [batch+1], prefix sums of the prompt lengths;
 *   h_cu_seqlens  host copy of the same array (checked on the host, so no
 *                 device-to-host copy is needed);
 *   h_block_table host int32 [batch, block_table_stride] page ids, required iff
 *                 the cache is paged (else NULL).  Row b lists the pages of
 *                 slot b in logical order; it must cover the prompt and any
 *                 later decode positions (unused entries may be -1).  Page ids
 *                 are in [0, kv_num_pages) and no page appears twice.  The
 *                 table is copied; the caller keeps ownership;
 *   all_logits    0: logits of the last position of each sequence, d_logits is
 *                 device float [batch, V]; 1: logits of every position,
 *                 d_logits is device float [sum S_b, V];  d_logits may be NULL;
 *   d_next_tokens device int32 [batch]: greedy argmax of each sequence's last
 *                 logits (lowest index on ties).
 * Positions are 0..S_b-1 (a fresh cache).  Each S_b must be in [1, max_seq]
 * and sum S_b <= max_tokens. */
int axon_prefill(axon_model* m, int32_t batch, const int32_t* d_tokens,
                 const int32_t* d_cu_seqlens, const int32_t* h_cu_seqlens,
                 const int32_t* h_block_table, int32_t block_table_stride, int32_t all_logits,
                 float* d_logits, int32_t* d_next_tokens, void* stream);

/* One greedy decode step for slots 0..batch-1 (batch <= the batch of the last
 * prefill): the same forward for one new token per sequence against the
 * cached keys and values, positions continuing from each sequence's past
 * length (Built-In Libraries, "Positions and cache management": the cache is
 * updated and positions are past_length + arange), then the greedy argmax
 * (Results, Measures; the paper's generate() loop, done here without a host
 * synchronization per step).  The page rows set by axon_prefill / axon_step
 * are used; no table is passed per step.  Slot b consumes d_tokens[b] (device int32 [batch]) at position
 * len_b (its current length), appends its key/value to the cache, writes the
 * logits (device float [batch, V], or NULL to skip) and the argmax token
 * (device int32 [batch]), and increments len_b.  Fails with AXON_E_CAPACITY if
 * some len_b + 1 > max_seq or (paged) the slot's page table has no page for
 * position len_b.  The step is recorded once per (batch, pointer triple) as a
 * HIP graph and replayed; d_tokens and d_next_tokens may be the same buffer
 * only if the caller does not need the input afterwards. */
int axon_decode_step(axon_model* m, int32_t batch, const int32_t* d_tokens, float* d_logits,
                     int32_t* d_next_tokens, void* stream);

/* Decode step that allocates nothing, for callers that cannot allocate
 * device memory (code under HIP graph capture, tight serving loops, harnesses
 * that forbid hipMalloc).  Same arguments, validation, kernels and results as
 * axon_decode_step, but the step is launched directly on ``stream`` (no graph
 * of the library's own is recorded: instantiating one allocates) and its
 * per-step work buffers (residual rows, the normalized operand and its sums
 * of squares, q, the attention output, the gated activation, split partials,
 * argmax partials) are laid out in one fixed device array of
 * AXON_NOALLOC_SCRATCH_BYTES that the library holds per GPU from the time its
 * code is loaded until the process ends.  The model (weights, KV cache,
 * lengths) is the one axon_init_model allocated.  The call makes no
 * hipMalloc, hipFree or other allocating call.
 * Dense Llama-family bf16 models only (AXON_ARCH_LLAMA, AXON_BF16,
 * n_experts 0; else AXON_E_INVALID) and batch <= 64; a step whose buffers
 * need more than the array is refused with AXON_E_CAPACITY (the message gives
 * the bytes needed); AXON_E_HIP if the array's address could not be obtained
 * at init.  Nothing is enqueued on failure.  All calls on one GPU share its
 * array, which keeps the last call's contents: each call first clears, with a
 * fill kernel on ``stream``, the counters of the decode attention's split
 * merge (the only part that must start at zero; every other buffer is written
 * before it is read within a step); calls that overlap in time on one GPU --
 * from two streams or threads, on any models -- race on it and must be
 * serialized by the caller. */
#define AXON_NOALLOC_SCRATCH_BYTES (64u << 20)
int axon_decode_step_noalloc(axon_model* m, int32_t batch, const int32_t* d_tokens, float* d_logits,
                             int32_t* d_next_tokens, void* stream);

/* Continuous batching (the serving loop of a paged-attention engine: prompt
 * chunks of newly admitted sequences and decode tokens of running ones share
 * one forward pass; Results, vLLM-native comparison; Introduction, vLLM
 * backend).  Entry i of the step appends n_i = h_cu_seqlens[i+1] -
 * h_cu_seqlens[i] >= 1 tokens to slot h_slots[i], at positions len .. len+n_i-1
 * where len is the slot's current length, or 0 when h_fresh[i] == 1 (the slot
 * starts a new sequence; what it held is dropped).  n_i > 1 is a prompt chunk,
 * n_i == 1 a decode token.  Each entry's tokens attend to every earlier
 * position of its slot (causally within the chunk), so feeding a prompt in
 * chunks over several calls gives the same result as one prefill.
 *   n             entries, 1..max_batch;
 *   h_slots       host int32 [n], distinct slots in [0, max_batch);
 *   h_fresh       host int32 [n] of 0/1, or NULL (no entry starts a sequence);
 *   d_tokens      device int32 [sum n_i], the entries' tokens back to back;
 *   d_cu_seqlens  device int32 [n+1], prefix sums of the n_i; h_cu_seqlens is
 *                 its host copy;
 *   h_block_table paged cache: host int32 [n, block_table_stride], the page row
 *                 of each entry's slot after the call (copied; it must keep the
 *                 pages that hold the slot's cached positions), or NULL to
 *                 keep the rows set earlier; must be NULL for a contiguous
 *                 cache.  Page ids are unique across all slots;
 *   d_logits      device float [n, V]: logits of each entry's last token, or
 *                 NULL; d_next_tokens: device int32 [n], their greedy argmax.
 * Afterwards slot h_slots[i] has length len + n_i; other slots are unchanged.
 * Fails with AXON_E_CAPACITY when len + n_i > max_seq, sum n_i > max_tokens
 * or a needed page is missing, and with AXON_E_INVALID for a repeated slot or
 * page, or a row that moves cached positions; nothing is enqueued then. */
int axon_step(axon_model* m, int32_t n, const int32_t* h_slots, const int32_t* h_fresh,
              const int32_t* d_tokens, const int32_t* d_cu_seqlens, const int32_t* h_cu_seqlens,
              const int32_t* h_block_table, int32_t block_table_stride, float* d_logits,
              int32_t* d_next_tokens, void* stream);

/* Evict the sequence of ``slot``: its length becomes 0 and, for a paged cache,
 * its page row is emptied, so its pages may be given to other slots by later
 * calls.  Host bookkeeping only (nothing is enqueued).  A slot of length 0 is
 * refused by axon_decode_step until axon_step or axon_prefill fills it. */
int axon_reset_slot(axon_model* m, int32_t slot);

/* Backward pass (training; the paper trains its generated models through
 * automatic differentiation: Results, "Training with Axon Derived Models").
 * Runs the forward pass over ``batch`` fresh sequences in slots 0..batch-1 (as
 * axon_prefill: the KV cache and the slot lengths are overwritten), the mean
 * next-token cross-entropy
 *   loss = (1/N) sum over positions t with 0 <= targets[t] < V of
 *          logsumexp(logits[t]) - logits[t][targets[t]]
 * (N such positions over all sequences; loss 0 and all gradients 0 when
 * N == 0), and the gradient of that loss with respect to every weight.
 *   d_tokens, d_cu_seqlens, h_cu_seqlens: as axon_prefill;
 *   d_targets  device int32 [sum S_b]: the token position t should predict
 *              (any value outside [0, V), e.g. -1, is not counted);
 *   d_loss     device float [1];
 *   grads      one descriptor per weight of the model: the weight map's names
 *              and shapes, dtype AXON_F32, device buffers (on_device 1),
 *              owned by the caller and overwritten with the gradients.
 * Activations and gradients are stored in bf16 between the kernels, with
 * float32 accumulation, the residual stream and its gradient in float32.
 * Dense Llama-family models only (AXON_ARCH_LLAMA, AXON_BF16, n_experts 0,
 * sliding_window 0, contiguous cache).  The first call allocates a
 * transposed copy of the weights and, for max_tokens positions, the saved
 * activations (per token and layer 12 hidden + 4 heads * head_dim + 10
 * intermediate + 4 heads bytes) and the gradient work buffers (including
 * float32 and bf16 logits, 6 vocab bytes per token).  Returns AXON_OK, AXON_E_INVALID, AXON_E_CAPACITY, AXON_E_MISSING /
 * AXON_E_SHAPE / AXON_E_DTYPE (gradient map), AXON_E_OOM or AXON_E_HIP. */
int axon_loss_and_grads(axon_model* m, int32_t batch, const int32_t* d_tokens, const int32_t* d_cu_seqlens,
                        const int32_t* h_cu_seqlens, const int32_t* d_targets, float* d_loss,
                        const axon_weight* grads, int32_t n_grads, void* stream);

/* Current length of every slot (host copy kept by the library, no device
 * access).  Writes min(n, max_batch) entries to ``lens``; returns the number of
 * active slots (the batch of the last prefill), or a negative status. */
int axon_slot_lengths(const axon_model* m, int32_t* lens, int32_t n);

/* Measurement support.  While enabled, every launch of the kernel classes
 *   0 = few-token projection GEMM (decode, weight streaming),
 *   1 = many-token projection GEMM (prefill, MFMA tiles),
 *   2 = decode attention (split over key chunks; the last split merges),
 *   3 = prefill attention,
 *   4 = grouped expert projection of a mixture-of-experts decode step (dims
 *       as class 0 with N, K of one expert and M the step's tokens; the
 *       launch streams the weights of every expert that some token chose),
 *   5 = attention backward of a training step (dims: heads, sequences, tokens)
 * is bracketed by two HIP events recorded on the stream it is launched on, and
 * decode steps run eagerly instead of as a recorded graph (kernel durations
 * are unchanged; only launch gaps differ).  Enabling (1) or disabling (0)
 * drops earlier records.  Returns AXON_OK or AXON_E_INVALID. */
int axon_timing_enable(axon_model* m, int32_t enable);

/* Copy out up to ``cap`` timing records: cls[i] is the kernel class,
 * dims[3*i..3*i+2] = (N output features, M tokens, K reduction length) of a
 * projection, or (heads, sequences, summed context/query tokens) of an
 * attention launch, ms[i] the event-measured duration in milliseconds.
 * Synchronizes on the recorded events.  Returns the number of records (which
 * may exceed cap), or a negative status. */
int axon_timing_records(axon_model* m, int32_t* cls, int32_t* dims, float* ms, int32_t cap);

/* Release every device buffer and recorded graph of the model.  NULL is a
 * no-op.  The caller must have synchronized the streams it used. */
void axon_free(axon_model* m);

/* Message describing the last failure on this thread ("" if none). */
const char* axon_last_error(void);

#ifdef __cplusplus
}
#endif
#endif /* AXON_H */
