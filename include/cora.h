/* cora.h - C ABI of the MI355X (gfx950) CORA-Diff denoising-step library.
 *
 * One executed denoising step of blockwise masked-diffusion decoding (Section 3
 * of the CORA-Diff paper, "Diffusion Decoding Setup" and "Confidence-Oriented
 * Residual Acceptance"): a dense bidirectional Transformer pass over the whole
 * prompt+generation canvas, per-position top-1 token and confidence (Eq. 1),
 * the persistence counter (Eq. 2), the original low-confidence transfer rule,
 * the residual confidence-and-persistence gate (Eq. 3), the commit of both
 * sets (Eq. 4) and block termination once the active block holds no
 * unresolved position (Fig. 2; "From acceptance to runtime").
 *
 * Conventions
 *  - Every function returns cora_status (0 = CORA_OK, < 0 = error) and never
 *    throws (a failed host allocation inside the library is CORA_ERR_OOM, and a
 *    failed create frees whatever it had allocated).  On error, cora_last_error() returns a thread-local message.  A
 *    failed HIP call inside the library is reported through the status alone:
 *    HIP's last-error state is cleared before the function returns.
 *  - "d_" pointers are device pointers, "h_" pointers are host pointers.  All
 *    caller buffers stay owned by the caller.  The library owns the model
 *    weights and a fixed workspace, both allocated in cora_model_create; no
 *    other entry point allocates device memory.
 *  - bf16 values cross the ABI as raw uint16_t bit patterns.
 *  - Work is enqueued on the caller's HIP stream (`hip_stream`, a hipStream_t;
 *    NULL = the default stream) in stream order.  Only cora_block_decode and
 *    cora_model_copy_tensor wait on the host.
 *  - Every call on one model uses that model's single workspace (activations,
 *    logits or score partials, split-K partials, decode state of
 *    cora_block_decode).  Calls on one model must therefore not overlap: issue
 *    them from one host thread at a time and on one stream, or order the
 *    streams.  Different models are independent.
 *  - Shapes are validated up front; unsupported shapes return
 *    CORA_ERR_UNSUPPORTED, malformed arguments CORA_ERR_INVALID_ARG, HIP
 *    failures CORA_ERR_HIP (with hipGetErrorString text in cora_last_error()).
 */
#ifndef CORA_H
#define CORA_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
  CORA_OK = 0,
  CORA_ERR_INVALID_ARG = -1,
  CORA_ERR_UNSUPPORTED = -2,
  CORA_ERR_OOM = -3,
  CORA_ERR_HIP = -4,
  CORA_ERR_STATE = -5
} cora_status;

#define CORA_MAX_BLOCK_LEN 256

/* Backbone shape.  The paper keeps the backbone frozen and runs one dense pass
 * per executed step (Section 3, first paragraph); the pass is a pre-norm
 * bidirectional Transformer: RMSNorm, QKV projection (+ optional bias),
 * rotate-half RoPE on q and k at absolute positions 0..L-1, non-causal
 * softmax attention (grouped kv heads allowed), output projection, RMSNorm,
 * SwiGLU MLP, final RMSNorm and an untied LM head scaled by logit_scale.
 * Limits: head_dim in {64, 128}; n_heads % n_kv_heads == 0; d_model and
 * n_heads*head_dim multiples of 64; d_model <= 8192; vocab >= 2;
 * 0 <= mask_id < vocab. */
typedef struct {
  int32_t n_layers, d_model, n_heads, n_kv_heads, head_dim, ffn_dim, vocab, mask_id;
  int32_t qkv_bias; /* 0/1: bias on the q, k and v projections */
  float rms_eps, rope_theta, logit_scale;
  double init_std;  /* std of the seeded N(0, std) weights, e.g. 0.02 */
} cora_model_cfg;

/* Blockwise schedule: the generation region is split into blocks of
 * block_len positions decoded left to right, each with a fixed horizon of
 * steps_per_block executed steps (Section 3, "Diffusion Decoding Setup").
 * The transfer rule fixes k_s = floor(block_len / S) + [s < block_len mod S]
 * positions at block step s (a linear split of the block's masked positions).
 * 1 <= steps_per_block <= block_len <= CORA_MAX_BLOCK_LEN.
 * eos_enabled != 0 turns on the EOS-aware controller of the deployment runs
 * (Table 2): after a step's commits, the lowest committed eos_id in the
 * generation region cuts the canvas; unresolved positions after it are
 * resolved as eos_id (decision code 3 inside the active block), committed
 * tokens keep their value, the active block finishes its positions before the
 * EOS and the row then stops (block_idx = number of blocks).  eos_enabled = 0
 * (a zero-initialised struct) keeps the fixed horizon. */
typedef struct {
  int32_t block_len, steps_per_block;
  int32_t eos_enabled, eos_id;
} cora_sched_cfg;

/* Residual gate of Eq. (3): accept i iff c_i >= delta_p and m_i >= m_req,
 * both inclusive, on unresolved active-block positions the transfer rule did
 * not fix.  gate_enabled = 0 gives the original dense decoder (no position
 * accepted).  persist_scope (the counter of Eq. (2) in blockwise decoding):
 * 0 = BLOCK: previous top-1 and counters reset when a block becomes active
 * (its first executed step), only the active block is scored;
 * 1 = GLOBAL: every unresolved generation position is scored on every
 * executed pass and its counter runs across blocks without a reset, so a
 * block whose positions already persisted can end after one pass; transfer
 * and gate still act on the active block only.  Other values return
 * CORA_ERR_UNSUPPORTED. */
typedef struct {
  float delta_p;
  int32_t m_req, gate_enabled, persist_scope;
} cora_gate_cfg;

/* Decode state of a batch of independent rows, all device pointers, updated
 * in place.  B rows, canvas length L = prompt_len + gen_len, gen_len a
 * multiple of block_len, n_blocks = gen_len / block_len.
 *   tokens     int32 [B, L]   canvas x; mask_id where masked
 *   unresolved uint8 [B, L]   1 iff the position is in U
 *   prev_top1  int32 [B, L]   top-1 of the previous executed step, -1 = none
 *   persist    int32 [B, L]   persistence counter m (Eq. 2)
 *   block_idx  int32 [B]      active block; n_blocks once the row is finished
 *   step_idx   int32 [B]      executed steps so far in the active block
 *   top1, conf int32/float [B, n_rows]  Eq. (1) outputs of the scored rows
 *   decision   uint8 [B, block_len]     0 none, 1 fixed by the transfer
 *                                       rule, 2 accepted by the gate
 *   done       int32 [B]      1 iff the active block was resolved by this step
 *                             (or the row was already finished)
 *   passes     int32 [B, n_blocks] or NULL: executed passes per block,
 *                             incremented for every row still decoding */
typedef struct {
  int32_t *tokens;
  uint8_t *unresolved;
  int32_t *prev_top1;
  int32_t *persist;
  int32_t *block_idx;
  int32_t *step_idx;
  int32_t *top1;
  float *conf;
  uint8_t *decision;
  int32_t *done;
  int32_t *passes;
  int32_t B, prompt_len, gen_len;
} cora_state;

typedef struct cora_model cora_model;

/* Allocate weights and workspace for batches of up to max_batch rows of up to
 * max_seq positions, and fill every weight with the counter-based generator:
 * element e (row-major [out, in]) of tensor t is
 *   key = mix(seed); ctr = (t << 40) | e;
 *   h1 = mix(key + (2 ctr + 1) G), h2 = mix(key + (2 ctr + 2) G),
 *   u1 = ((h1 >> 11) + 1) 2^-53, u2 = (h2 >> 11) 2^-53,
 *   w  = bf16_rne(float_rne(init_std * sqrt(-2 ln u1) cos(2 pi u2)))
 * with mix the SplitMix64 finaliser and G = 0x9E3779B97F4A7C15.  Tensor ids:
 * 1 embedding [V, d], 2 LM head [V, d], and 100 + 16 l + j for layer l with
 * j = 0 wq, 1 wk, 2 wv, 3 wo, 4 wg, 5 wu, 6 wd, 7 bq, 8 bk, 9 bv.  Norm
 * weights are 1.  The LM head is also kept in a second, packed layout (the
 * order in which the few-row LM-head kernel streams it: 32-row groups of 1 KB
 * MFMA operand blocks), written once here: weight bytes include one more
 * V x d bf16 matrix.  Synchronous.  *out is set only on success.
 * CORA_ERR_UNSUPPORTED when an activation matrix of max_batch x max_seq rows
 * (fp32 residual rows, bf16 FFN or attention-head rows, max_seq rounded up to
 * 64) would exceed 2 GB: the kernels address one with 32-bit byte offsets.
 * CORA_ERR_OOM when the device allocation fails. */
cora_status cora_model_create(const cora_model_cfg *cfg, uint64_t seed, int32_t max_batch,
                              int32_t max_seq, void *hip_stream, cora_model **out);
cora_status cora_model_destroy(cora_model *model);

/* Dense forward pass over tokens [B, L] (int32, device) and the LM head on
 * canvas rows [row_begin, row_begin + n_rows) of every batch row: writes
 * bf16 logits [B, n_rows, V] (device, caller-allocated).  When
 * max_batch * n_rows <= 64 the few-row LM-head kernel runs, else the tiled
 * GEMM; both round (sum_k a_k w_k) * logit_scale to bf16 and differ only in
 * fp32 summation order.  Every kernel choice that sets a summation order is
 * made for max_batch rows, so a row's logits do not depend on B.  Parity
 * hook. */
cora_status cora_forward_logits(cora_model *model, const int32_t *d_tokens, int32_t B, int32_t L,
                                int32_t row_begin, int32_t n_rows, uint16_t *d_logits,
                                void *hip_stream);

/* One executed denoising step on every row of `state` that is still decoding:
 * dense pass, LM head on the active block rows of each batch row, then the
 * vocab/gate kernels (Eq. 1, Eq. 2, transfer rule, Eq. 3, Eq. 4, termination;
 * see cora_vocab_gate).  top1/conf are [B, block_len] (the active block's
 * rows) under the BLOCK scope and [B, gen_len] (the generation region, LM head
 * and row reduction in chunks of up to 256 rows) under GLOBAL.  Eq. (1) is
 * computed inside the LM-head pass and no logits are written: when max_batch
 * times the rows scored per batch row (per chunk) is at most 64, the pass
 * streams the packed weight copy (per-128-entry partial max / first arg max /
 * sum of exp), else each wavefront's logit columns are reduced in the tiled
 * GEMM's epilogue; the partials are merged in vocab order.  The top-1 is then
 * the same as cora_vocab_gate's on the logits cora_forward_logits writes for
 * those rows, at any B (the kernel choices are made for max_batch).
 * Only a vocabulary too small for the partials to fit the logits buffer takes
 * logits + row reduction.  Asynchronous. */
cora_status cora_denoise_step(cora_model *model, cora_state *state, const cora_sched_cfg *sched,
                              const cora_gate_cfg *gate, void *hip_stream);

/* The vocab/gate kernel alone on caller logits.  d_logits: bf16 [B, n_rows, V];
 * row r of batch row b scores canvas position row_begin + r, or, when
 * row_begin < 0, position lo_b + r where lo_b is the first position of b's
 * active block.  For every row: top-1 token (lowest id among equal maxima,
 * mask_id never predicted) and confidence c = 1 / sum_v exp(l_v - l_max)
 * (fp32).  Then, per batch row still decoding, on its active block: counters
 * reset at block step 0, persistence update on unresolved positions, the
 * k highest-confidence unresolved positions (ties: lower position) fixed
 * (k = k_transfer if >= 0, else the schedule's k_s), the gate on the rest,
 * commit of both sets, and the block/step advance once the block is empty.
 * A fixed row_begin must cover the whole generation region; the GLOBAL
 * persistence scope needs fixed rows (it updates every scored unresolved
 * position).  top1/conf receive [B, n_rows].  Two kernel launches on
 * hip_stream (row reduction, then the decision rules); calls on one state must
 * not overlap.  Asynchronous. */
cora_status cora_vocab_gate(const uint16_t *d_logits, int32_t n_rows, int32_t row_begin,
                            int32_t V, int32_t mask_id, cora_state *state, int32_t k_transfer,
                            const cora_sched_cfg *sched, const cora_gate_cfg *gate,
                            void *hip_stream);

/* For callers that cannot allocate device memory (code under HIP graph capture,
 * tight serving loops, harnesses that forbid allocation): cora_vocab_gate with
 * the same arguments, outputs and error behaviour, computed without any
 * allocation.  Each logits row's vocabulary is split into consecutive ranges,
 * one workgroup each (so few rows still fill the GPU); their partial (max,
 * sum of exp, lowest arg max) go to a fixed device array of the library of
 * CORA_VOCAB_GATE_NOALLOC_MAX_PARTIALS entries (12 bytes each, 3 MiB per GPU,
 * held until the process ends) and are merged in vocab order.  top1 equals
 * cora_vocab_gate's bit for bit; conf differs only in fp32 summation order,
 * so decisions agree except where a cut or threshold lies within that
 * rounding.  B * n_rows above CORA_VOCAB_GATE_NOALLOC_MAX_PARTIALS returns
 * CORA_ERR_UNSUPPORTED.  The array's address is looked up on the first call
 * on a device (the current device, which must own the stream and pointers).
 * Every call on one GPU shares that array: calls that overlap on one GPU
 * (other threads, other streams) race and must be ordered by the caller.
 * No hipMalloc, hipFree or other allocating routine is called, also not on
 * error paths.  Asynchronous. */
#define CORA_VOCAB_GATE_NOALLOC_MAX_PARTIALS 262144
cora_status cora_vocab_gate_noalloc(const uint16_t *d_logits, int32_t n_rows, int32_t row_begin,
                                    int32_t V, int32_t mask_id, cora_state *state,
                                    int32_t k_transfer, const cora_sched_cfg *sched,
                                    const cora_gate_cfg *gate, void *hip_stream);

/* Gated block decode of B prompts (d_prompt int32 [B, prompt_len], device):
 * the canvas starts as prompt + gen_len masks, rows decode independently and
 * each block ends once it holds no unresolved position, skipping its
 * remaining passes.  With batch-row compaction on (the default, see
 * cora_model_set_compaction) a row that has finished all its blocks leaves the
 * dense pass: its final tokens and passes are written out and later passes run
 * on the live rows only.  Writes the final canvas to d_out_tokens int32 [B, L]
 * (device) and the executed passes per block to h_passes int32
 * [B, gen_len / block_len] (host).  If h_total_passes is not NULL it receives
 * the number of dense passes launched (the batch runs while any row decodes).
 * Synchronous on return. */
cora_status cora_block_decode(cora_model *model, const int32_t *d_prompt, int32_t B,
                              int32_t prompt_len, int32_t gen_len, const cora_sched_cfg *sched,
                              const cora_gate_cfg *gate, int32_t *d_out_tokens, int32_t *h_passes,
                              int32_t *h_total_passes, void *hip_stream);

/* Copy weight tensor `tensor_id` (ids as in cora_model_create) to host memory
 * in its logical row-major [out, in] layout as bf16 bits (biases too).
 * `bytes` must equal the tensor's size.  Synchronous. */
cora_status cora_model_copy_tensor(cora_model *model, int32_t tensor_id, void *h_dst, size_t bytes);

/* Kernel timing: while enabled, every launch of the gate/up SwiGLU GEMM is
 * dispatched with a pair of HIP events (hipExtLaunchKernel) that the dispatch
 * stamps with the kernel's start and end on the launching stream.  Enabling
 * and disabling keep what was recorded, so timing can cover a sample of the
 * launches.  Reading waits for the recorded events, returns the summed event
 * time (ms) and the number of timed launches since the previous read, and
 * clears both. */
cora_status cora_model_set_timing(cora_model *model, int32_t enable);
cora_status cora_model_read_timing(cora_model *model, double *total_ms, int64_t *launches);

/* Batch-row compaction in cora_block_decode (rows decode independently, so
 * dropping finished rows from the dense pass changes no live row's inputs).
 * Every kernel choice that sets an output's summation order (split-K count,
 * attention key-range parts, LM-head kernel and vocab partial layout) is made
 * for max_batch rows, never for the live row count, so a row's tokens and
 * passes are bit-identical with compaction on or off and equal to a decode of
 * that row alone on the same model.  enable != 0 turns it on (default), 0 off. */
cora_status cora_model_set_compaction(cora_model *model, int32_t enable);

/* Device bytes the model holds (weights + workspace). */
cora_status cora_model_device_bytes(cora_model *model, size_t *weight_bytes, size_t *workspace_bytes);

const char *cora_last_error(void);

#ifdef __cplusplus
}
#endif

#endif /* CORA_H */
