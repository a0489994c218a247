/*
 * stage.h -- C ABI of the MI355X pipeline-stage forward pass.
 *
 * What a stage is. ShuntServe splits a decoder-only LLM into pipeline stages,
 * each a contiguous range of transformer layers placed on one device
 * (Sec. 2.3, "Uneven Layer Partitioning in PP"; Algorithm 1 adds one stage of
 * l - l' consecutive layers at a time). Stages exchange only hidden states of
 * B*S*H*E bytes (Sec. 4.1.2, Eq. 2). Per layer the work is the QKV
 * projection, attention, output projection, up-and-gate projection and down
 * projection of Table 2 (Sec. 4.1.1), with prefill compute-bound and decode
 * memory-bound (Sec. 2.3, "The Optimization Challenge"; Sec. 4.2.2). The
 * weights and the KV-cache space live in a store separate from the engine
 * and are referenced zero-copy (Sec. 5.2, "Shared Tensor Store"); this ABI
 * therefore only borrows device memory and never allocates it.
 *
 * A layer is the pre-norm Llama-3 / Qwen3 block of the models the paper
 * serves (Sec. 7): RMSNorm -> fused QKV projection -> (Qwen3: per-head q/k
 * RMSNorm) -> rotary embedding (rotate-half pairing, angle p*theta^(-2j/d))
 * -> causal grouped-query attention over a paged KV cache (query head h reads
 * kv head h / (n_q/n_kv), scale 1/sqrt(d)) -> output projection + residual
 * -> RMSNorm -> SwiGLU FFN (silu(x Wg^T) * (x Wu^T)) -> down projection +
 * residual.
 *
 * Conventions shared by every entry point:
 *  - Weights are applied as y = x W^T for W [N, K]. In row-major form w_qkv
 *    stacks the n_q*d query rows, then n_kv*d key rows, then n_kv*d value
 *    rows; w_gate_up stacks ffn gate rows then ffn up rows. The stage reads
 *    the four projection matrices in the layout stage_pack_weight() produces
 *    from that row-major form (bf16: MFMA-fragment-packed; f32: row-major
 *    unchanged); a weight store packs them once, when it loads them. Norm
 *    gains are [hidden]; q/k-norm gains are [head_dim]. All weights are stored
 *    in the mode dtype.
 *  - KV pool (one allocation for the stage's layers):
 *      [n_layers][num_blocks][n_kv][2][block_size * head_dim]
 *    in the mode dtype. Token p of a sequence with block table bt lives in
 *    block bt[p / block_size] at offset o = p % block_size. Plane 0 holds K,
 *    plane 1 holds V, both as whole 1 KB MFMA operand fragments, so that
 *    the attention kernels read a block's K and V from HBM in contiguous
 *    16-byte-per-lane loads:
 *      K[o][d] at (d / 32) * 512 + (o + 16 * ((d % 32) / 8)) * 8 + d % 8
 *      V[o][d] at (d / 32) * 512 + (d % 16 + 16 * (o / 4)) * 8 + ((d / 16) % 2) * 4 + o % 4
 *    Block ids index the same blocks in every layer of the stage. Slots a
 *    call has not written (past a sequence's length in its last block) are
 *    read but given zero weight; they must hold finite values (a pool
 *    zeroed when allocated, or finite data of earlier sequences), since an
 *    Inf or NaN times a zero weight is NaN. The block-table entries a call
 *    reads (the first ceil((ctx_lens[i] + q_lens[i]) / block_size) of row
 *    i) must lie in [0, num_blocks): the kernels read
 *    them on the device and do not check them, so an id outside that range
 *    is an out-of-bounds access of the pool. With the environment variable
 *    STAGE_DEBUG=1 set when a stage is created, every forward call first
 *    copies the tables it uses to the host (synchronising the stream) and
 *    rejects out-of-range ids with STAGE_ERR_INVALID_ARG before enqueuing
 *    anything: a debugging aid, not for serving.
 *  - hidden_in / hidden_out: [T, hidden] in the mode dtype, rows packed
 *    sequence by sequence in batch order (for stage_step_mixed: all prefill
 *    rows first, then the decode rows). hidden_out may alias hidden_in.
 *    Inside a call the residual stream is kept in fp32.
 *  - Every call only enqueues work on `stream` (a hipStream_t; NULL = the
 *    default stream) and returns; outputs are valid once the stream has
 *    reached that point. Host arrays may be reused as soon as the call
 *    returns.
 *  - Errors: host-side arguments are validated before anything is enqueued;
 *    on failure the call returns a non-zero stage_status, enqueues nothing
 *    and stage_last_error() describes the failure. Device faults surface at
 *    stream synchronisation as HIP errors. No entry point throws or aborts.
 *  - A stage_t is not thread-safe; distinct stages may be used from
 *    different threads.
 */
#ifndef STAGE_H_
#define STAGE_H_

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef struct stage stage_t; /* opaque */

typedef enum {
  STAGE_OK = 0,
  STAGE_ERR_INVALID_ARG = 1, /* null pointer, bad length, inconsistent batch */
  STAGE_ERR_UNSUPPORTED = 2, /* shape or dtype the library does not implement */
  STAGE_ERR_OUT_OF_MEMORY = 3, /* host allocation failed */
  STAGE_ERR_DEVICE = 4,      /* a HIP call failed (no device, launch error) */
  STAGE_ERR_CAPACITY = 5     /* batch exceeds max_tokens / max_seqs / table
                                capacity / max_position / workspace */
} stage_status;

typedef enum { STAGE_F32 = 0, STAGE_BF16 = 1 } stage_dtype;

/* Shape and constants of one decoder layer.
 * Supported: head_dim in {64, 128}; n_q_heads % n_kv_heads == 0 with group
 * size n_q/n_kv in {1, 2, 4, 8, 16}; block_size == 16; hidden % 128 == 0;
 * (n_q_heads * head_dim) % 128 == 0; ffn % 64 == 0. */
typedef struct {
  int32_t hidden;
  int32_t n_q_heads;
  int32_t n_kv_heads;
  int32_t head_dim;
  int32_t ffn;
  int32_t qk_norm;      /* 1: per-head RMSNorm of q and k (Qwen3), else 0 */
  int32_t block_size;   /* KV block size in tokens; must be 16 */
  float rms_eps;        /* epsilon of the two layer RMSNorms */
  float qk_rms_eps;     /* epsilon of the q/k RMSNorm */
  double rope_theta;    /* rotary base */
  int32_t max_position; /* positions are in [0, max_position) */
  stage_dtype dtype;    /* storage dtype of weights, KV and hidden states */
} stage_model_config;

/* Device pointers to one layer's weights (q_norm/k_norm may be NULL unless
 * qk_norm is set). The four projections w_qkv, w_o, w_gate_up and w_down
 * must be in the stage_pack_weight() layout (bf16 mode), not row-major:
 * the stage cannot tell the two apart, so row-major bf16 matrices give
 * wrong outputs without an error. Pack each matrix once, when it is loaded
 * (stage_pack_weight can write straight into store memory). In fp32 mode
 * the packed layout is the row-major one. Gains are plain arrays. */
typedef struct {
  const void* attn_norm; /* [hidden] */
  const void* w_qkv;     /* [(n_q + 2 n_kv) * head_dim, hidden] */
  const void* q_norm;    /* [head_dim] */
  const void* k_norm;    /* [head_dim] */
  const void* w_o;       /* [hidden, n_q * head_dim] */
  const void* ffn_norm;  /* [hidden] */
  const void* w_gate_up; /* [2 * ffn, hidden] */
  const void* w_down;    /* [hidden, ffn] */
} stage_layer_weights;

/* One request batch. q_lens/ctx_lens are HOST arrays; block_tables is a
 * DEVICE array. Sequence i contributes q_lens[i] consecutive rows to
 * hidden_in, at positions ctx_lens[i] .. ctx_lens[i] + q_lens[i] - 1; its
 * first ctx_lens[i] tokens must already be in the KV cache (written by
 * earlier calls), and the call writes the keys and values of the new ones. */
typedef struct {
  int32_t num_seqs;
  const int32_t* q_lens;        /* host [num_seqs], each >= 1 */
  const int32_t* ctx_lens;      /* host [num_seqs], each >= 0 */
  const int32_t* block_tables;  /* device [num_seqs][max_blocks_per_seq] */
  int32_t max_blocks_per_seq;
} stage_batch;

/* The four projection matrices of a layer. */
typedef enum {
  STAGE_W_QKV = 0,     /* [(n_q + 2 n_kv) * head_dim, hidden] */
  STAGE_W_O = 1,       /* [hidden, n_q * head_dim] */
  STAGE_W_GATE_UP = 2, /* [2 * ffn, hidden] */
  STAGE_W_DOWN = 3     /* [hidden, ffn] */
} stage_weight_kind;

/* Convert one row-major projection matrix (device memory, mode dtype) into
 * the layout the stage reads, writing dst (device memory of the same size;
 * must not overlap src). bf16: whole 16 x 32 MFMA operand fragments (1 KB,
 * lane-major) stored contiguously, rows grouped by 64 so that one group's
 * fragments for successive k are adjacent; for the gate-up weight each
 * 64-row group holds 32 gate rows followed by the 32 matching up rows. f32:
 * a plain copy. Enqueued on `stream`; the caller owns both buffers. Meant
 * for load time (a weight store), not the forward path. */
stage_status stage_pack_weight(const stage_model_config* cfg, stage_weight_kind kind,
                               const void* src, void* dst, void* stream);

/* Create a stage over layers [layer_begin, layer_end) of a model: the
 * contiguous layer range that the paper's placement assigns to one device
 * (Sec. 2.3, "Uneven Layer Partitioning in PP"; Algorithm 1 adds stages of
 * l - l' consecutive layers), over weights and KV space that a store owns
 * and the engine only references (Sec. 5.2, "Shared Tensor Store").
 *  layers:   host array of layer_end - layer_begin weight sets (device
 *            pointers, borrowed: they must outlive the stage).
 *  kv_pool:  device pointer to the KV pool (layout above), borrowed.
 *  num_blocks: blocks per layer in kv_pool.
 *  max_tokens: largest T of any call; max_seqs: largest number of sequences
 *            (prefill + decode) of any call. They size the workspace.
 * The stage keeps host-side state only (including a small pinned staging
 * buffer); device scratch memory is supplied by stage_bind_workspace.
 * Returns STAGE_ERR_DEVICE if no HIP device is usable. */
stage_status stage_create(const stage_model_config* cfg, int32_t layer_begin, int32_t layer_end,
                          const stage_layer_weights* layers, void* kv_pool, int32_t num_blocks,
                          int32_t max_tokens, int32_t max_seqs, stage_t** out);

/* Bytes of device workspace the stage needs (activations, metadata, decode
 * split partials, the rotary cos/sin table). */
size_t stage_workspace_bytes(const stage_t* st);

/* Bind caller-owned device memory of at least stage_workspace_bytes() bytes
 * (256-byte aligned). Synchronously uploads the rotary cos/sin table into
 * it; nothing else in it needs initialising. Must be called before the first
 * forward call; may be called again to move the workspace. */
stage_status stage_bind_workspace(stage_t* st, void* dev, size_t bytes);

/* Prefill (or chunked prefill / recomputation): every sequence has
 * q_lens >= 1 new tokens. One pass of the stage's layers over the batch's
 * rows: hidden states in, hidden states out for the next stage (Sec. 4.1.2,
 * Eq. 2 prices exactly this B*S*H*E transfer); the compute-bound phase of
 * Sec. 2.3 and Table 2's prefill rows. Rebuilding a migrated request's KV
 * cache is a chunked call of this kind (Sec. 5.1, "Output-Preserving Request
 * Migration"). */
stage_status stage_prefill(stage_t* st, const stage_batch* batch, const void* hidden_in,
                           void* hidden_out, void* stream);

/* Decode: every sequence has exactly one new token (q_lens[i] == 1): the
 * memory-bound phase of Sec. 2.3 and Table 2's decode rows, one token per
 * running request and step, hidden states in and out (Sec. 4.1.2, Eq. 2). */
stage_status stage_decode(stage_t* st, const stage_batch* batch, const void* hidden_in,
                          void* hidden_out, void* stream);

/* One continuous-batching step: a prefill batch (may be NULL or empty) and a
 * decode batch (may be NULL or empty) in one pass over the layers. Rows of
 * hidden_in: prefill rows first, then decode rows. A sequence must not
 * appear in both batches. This is the request mix of one engine step, whose
 * latency the paper's estimator sums over Table 2's operations (Sec. 4.1.1,
 * Eq. 1) and whose batch size the placement optimizer bounds by memory
 * (Sec. 4.2.2, "Batch Size Determination"). */
stage_status stage_step_mixed(stage_t* st, const stage_batch* prefill, const stage_batch* decode,
                              const void* hidden_in, void* hidden_out, void* stream);

/* Decode over the library's static scratch array instead of the bound
 * workspace: the same forward pass, kernels and results as stage_decode, for
 * callers that cannot allocate device memory (code under HIP graph capture,
 * tight serving loops, harnesses that forbid hipMalloc). This call allocates
 * nothing: no hipMalloc/hipFree, no events; stage_bind_workspace is not
 * needed for it.
 *  - The scratch is a file-scope device array of 128 MiB per GPU, held from
 *    the library's loading until the process ends (each GPU has its own).
 *    A stage whose stage_workspace_bytes() exceeds it gets
 *    STAGE_ERR_CAPACITY before anything is enqueued (a Llama-3.1-70B-shaped
 *    layer range with max_tokens = max_seqs = 128 and max_position = 8192
 *    fits).
 *  - Every call on a GPU, from any stage, shares that GPU's array, which
 *    keeps the last call's contents. Nothing in it must start at zero; the
 *    rotary table is copied in (from host memory, on `stream`) whenever the
 *    previous call on that GPU came from another stage. Calls that overlap
 *    on one GPU (concurrent streams or threads) race on the array and give
 *    wrong results; serialise them.
 *  - Validation and error codes are those of stage_decode; op timing is not
 *    applied to its launches. */
stage_status stage_decode_noalloc(stage_t* st, const stage_batch* batch, const void* hidden_in,
                                  void* hidden_out, void* stream);

/* Destroy a stage (does not free any borrowed memory). NULL is allowed. */
stage_status stage_destroy(stage_t* st);

/* Description of the last failure on this thread ("" if none). */
const char* stage_last_error(void);

/* Host-only check of a step against a configuration and the stage limits,
 * with exactly the checks (and return codes) the forward entry points apply
 * before enqueuing anything. Touches no device memory (block_tables is only
 * checked for NULL). Useful for admission control in a scheduler. */
stage_status stage_validate_step(const stage_model_config* cfg, int32_t max_tokens,
                                 int32_t max_seqs, const stage_batch* prefill,
                                 const stage_batch* decode);

/* ---- last stage: LM head ---------------------------------------------- */
/* Only the last stage of a pipeline turns hidden states into logits: the
 * model's final RMSNorm (gain final_norm, epsilon cfg.rms_eps) of each
 * selected row of its output, then the vocabulary projection
 * logits = norm(x) W_lm^T with W_lm [vocab, hidden] (Table 2, "Logits
 * Calculation"). A prefill step needs the last row of each sequence, a decode
 * step every row.
 *  final_norm: device [hidden] gain (mode dtype).
 *  w_lm:       device [vocab, hidden] in the stage_pack_lm_head() layout.
 *  hidden:     device [hidden_rows, hidden] (mode dtype, row-major), e.g. the
 *              hidden_out of the stage's last forward call.
 *  rows:       HOST [n_rows] indices into hidden, each in [0, hidden_rows);
 *              NULL selects rows 0 .. n_rows-1 (then n_rows <= hidden_rows).
 *  logits:     device float32 [n_rows, vocab], row-major, written.
 * n_rows <= max_tokens of the stage; bf16 needs vocab % 128 == 0
 * (STAGE_ERR_UNSUPPORTED otherwise); bad row indices give
 * STAGE_ERR_INVALID_ARG before anything is enqueued. Uses the stage's
 * workspace, so it is ordered with the stage's forward calls only on the
 * same stream. Timed as STAGE_OP_LM_HEAD. */
stage_status stage_lm_head(stage_t* st, const void* final_norm, const void* w_lm, int32_t vocab,
                           const void* hidden, int32_t hidden_rows, const int32_t* rows,
                           int32_t n_rows, float* logits, void* stream);

/* Convert a row-major [vocab, hidden] LM-head matrix (device, mode dtype)
 * into the layout stage_lm_head reads (the stage_pack_weight fragment
 * layout; f32: a copy). dst must not overlap src. Meant for load time. */
stage_status stage_pack_lm_head(const stage_model_config* cfg, int32_t vocab, const void* src,
                                void* dst, void* stream);

/* ---- shared tensor store ---------------------------------------------- */
/* The paper keeps model weights and KV-cache space in a store process that
 * loads them once and hands them to engine processes zero-copy, so that an
 * engine (re)starts without reloading anything (Sec. 5.2, "Shared Tensor
 * Store"; the same section overlaps the store's loading with engine start-up,
 * its concurrent initialization). These
 * calls are that hand-over on one GPU: the store allocates and exports, an
 * engine in another process attaches and passes the pointers it gets to
 * stage_create like any other device memory.
 *  - Each allocation is one device allocation below STAGE_STORE_MAX_BYTES,
 *    exported whole: a handle maps exactly one allocation from its base.
 *    Larger tensors are split by the caller (a layer's weights are several
 *    allocations, a KV pool can be one per layer range).
 *  - The store owns its allocations and must keep them alive (and not free
 *    them) while any engine is attached; engines only read weights and
 *    write the KV blocks their own block tables name. Nothing orders work
 *    between processes: callers synchronise (e.g. the store finishes
 *    writing before it publishes the handles).
 *  - Both processes need the same GPU, and the engine must be a process of
 *    its own (a handle cannot be opened in the process that exported it). */
#define STAGE_STORE_MAX_BYTES ((size_t)1 << 31)

/* An exported allocation: opaque bytes, safe to copy between processes
 * (e.g. hex-encoded through a pipe). */
typedef struct {
  unsigned char bytes[64];
} stage_ipc_handle;

/* Store side: allocate `bytes` (0 < bytes < STAGE_STORE_MAX_BYTES, else
 * STAGE_ERR_INVALID_ARG / STAGE_ERR_CAPACITY) of zero-filled device memory on
 * the current device and export it. *dev receives the pointer in this
 * process, *handle what another process attaches with. Synchronous. */
stage_status stage_store_alloc(size_t bytes, void** dev, stage_ipc_handle* handle);

/* Store side: free an allocation of stage_store_alloc (NULL is allowed).
 * Engines must have detached. */
stage_status stage_store_free(void* dev);

/* Copy `bytes` from src (device or host memory) into store memory dst,
 * enqueued on `stream`: how a store loads tensors that need no packing
 * (norm gains; packed projections are written by stage_pack_weight straight
 * into store memory). */
stage_status stage_store_write(void* dst, const void* src, size_t bytes, void* stream);

/* Engine side: map an exported allocation into this process; *dev receives
 * its address here (the base of the allocation). STAGE_ERR_DEVICE if the
 * handle cannot be opened (wrong GPU, store gone, same process). */
stage_status stage_store_attach(const stage_ipc_handle* handle, void** dev);

/* Engine side: unmap what stage_store_attach mapped (NULL is allowed).
 * Stages created over it must have been destroyed and their work finished. */
stage_status stage_store_detach(void* dev);

/* ---- measurement hooks ------------------------------------------------ */

/* Operation classes timed by the op-timing hook. */
typedef enum {
  STAGE_OP_NORM = 0,      /* RMSNorms, input/output conversion, SwiGLU */
  STAGE_OP_QKV = 1,       /* QKV projection */
  STAGE_OP_ROPE_KV = 2,   /* q/k norm + RoPE + KV write */
  STAGE_OP_ATTN = 3,      /* attention (prefill + decode + merge) */
  STAGE_OP_O = 4,         /* output projection + residual */
  STAGE_OP_GATE_UP = 5,   /* gate-up projection (+ SwiGLU when fused) */
  STAGE_OP_DOWN = 6,      /* down projection + residual */
  STAGE_OP_LM_HEAD = 7,   /* final norm + logits projection (stage_lm_head) */
  STAGE_OP_COUNT = 8
} stage_op;

/* Enable (1) or disable (0) HIP-event timing of each op class. While
 * enabled, every launch of the stage is bracketed by events on the call's
 * stream (adding a little overhead). The events are timing-only: recording
 * them makes no memory visible to the host or to other devices. */
stage_status stage_set_op_timing(stage_t* st, int32_t enable);

/* Synchronise the recorded events and return, per op class, the summed
 * milliseconds and the number of launches since timing was enabled or last
 * read; then reset the counters. ms and launches have STAGE_OP_COUNT
 * entries. */
stage_status stage_read_op_times(stage_t* st, double* ms, int64_t* launches);

/* Enqueue a plain streaming copy of `bytes` from device buffer src to device
 * buffer dst on `stream`: the known-size reference kernel against which
 * bandwidth and the hardware traffic counters (FETCH_SIZE, WRITE_SIZE) of
 * the stage kernels are calibrated. Not part of the forward pass. bytes and
 * both pointers must be multiples of 16 and the buffers must not overlap
 * (STAGE_ERR_INVALID_ARG otherwise). */
stage_status stage_copy_probe(const void* src, void* dst, size_t bytes, void* stream);

#ifdef __cplusplus
}
#endif

#endif /* STAGE_H_ */
