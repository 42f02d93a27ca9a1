/*
 * stage.h - C ABI of libstage: one pipeline stage's stateful decode/verify
 * forward on an AMD Instinct MI355X (gfx950).
 *
 * A stage is a contiguous block of Llama-style decoder layers (paper,
 * "Per-Stage Export Pipeline": each shard covers a contiguous layer range)
 * with symmetric INT4 group-quantized weights (Step 4 of that pipeline),
 * RMSNorm, rotary embeddings from a precomputed cos/sin table indexed by
 * caller position ids (Step 2 and "Stateful KV-Cached Inference"), and
 * scaled-dot-product attention over a per-request stateful KV cache.
 *
 * Two properties of the paper's shards are reproduced exactly:
 *  - the cache is reordered along the slot axis through beam_idx, as the
 *    Gather(ReadValue, beam_idx, axis=0) the shards insert ("Reaching
 *    Monolithic Parity: the beam_idx Gather Injection"); here the reorder is
 *    applied to a per-state index table and cache rows are read through it,
 *    never copied;
 *  - rejected speculative positions stay in the cache and are hidden by a 0
 *    in attention_mask ("Mask-Based Rewind"); new rows are appended at the
 *    next physical index and rotary uses the caller's (logical) position ids.
 *
 * Conventions
 *  - Every call returns STAGE_OK (0) or a negative STAGE_E_* code;
 *    stage_last_error() returns a thread-local message for the last failure.
 *  - Validation is synchronous and all-or-nothing: on any error nothing has
 *    been enqueued and no state (length, table, contents) has changed.
 *  - `stream` is a hipStream_t passed as void* (NULL = the null stream).
 *    Device work is stream-ordered and asynchronous; host metadata arrays are
 *    copied before the call returns and may be reused immediately.
 *  - Calls on one Stage (and on the KV states it allocated) must be made
 *    from one host thread at a time.  Their device work runs in call order
 *    even across streams: a call issued on a different stream than the
 *    previous call on the stage first makes its stream wait for that call's
 *    work (the workspace, metadata buffer and exchange flag numbers are per
 *    stage), so two forwards of one stage never overlap on the device.
 *  - stage_forward must not be captured into a HIP graph: each call takes
 *    its exchange flag numbers, metadata buffer slot and beam-table side from
 *    host state at call time, and a replayed capture would reuse stale ones.
 *  - Dtype codes: STAGE_DTYPE_F16 = IEEE half, STAGE_DTYPE_BF16 = bfloat16.
 */
#ifndef PAPER_2608_19147_STAGE_H
#define PAPER_2608_19147_STAGE_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#define STAGE_OK                0
#define STAGE_E_INVALID        -1   /* bad argument value (NULL, range, fully masked query row) */
#define STAGE_E_SHAPE          -2   /* shape mismatch (mask length, matrix dims) */
#define STAGE_E_CAPACITY       -3   /* KV capacity, row count or position table exceeded */
#define STAGE_E_OOM            -4   /* device or pinned allocation failed */
#define STAGE_E_HIP            -5   /* a HIP runtime call failed (message has the HIP error) */
#define STAGE_E_STATE_MISMATCH -6   /* KV state belongs to another stage, or used twice in one call */
#define STAGE_E_UNSUPPORTED    -7   /* configuration outside what the kernels implement */
#define STAGE_E_DEVICE         -8   /* a single-launch forward gave up waiting on another workgroup: its outputs are invalid */

#define STAGE_DTYPE_F16  1
#define STAGE_DTYPE_BF16 2

/* Most activation rows (sum over requests of slots x tokens) per forward. */
#define STAGE_MAX_ROWS 64

/* Model dimensions of the stage.  Requirements: head_dim in {64, 128};
 * n_q_heads a multiple of n_kv_heads; hidden and ffn multiples of 8;
 * group_size a multiple of 32 (the paper's shards use 128). */
typedef struct StageConfig {
    int32_t n_layers;
    int32_t hidden;          /* H */
    int32_t n_q_heads;       /* Hq */
    int32_t n_kv_heads;      /* Hkv; q head h reads kv head h / (Hq/Hkv) */
    int32_t head_dim;        /* D */
    int32_t ffn;             /* F (SwiGLU inner size) */
    int32_t group_size;      /* G: INT4 quantization group along K */
    float   rms_eps;
    int32_t act_dtype;       /* dtype of hidden_in / hidden_out / norm weights */
    int32_t kv_dtype;        /* dtype of cached K/V rows */
    double  rope_theta;      /* cos/sin(p * theta^(-2i/D)), rotate-half pairing (i, i+D/2) */
    int32_t max_positions;   /* size of the rotary table; positions must be < this */
    /* Optional host table [max_positions][D/2][2] fp32 (cos, sin); NULL =>
     * computed in fp64 from rope_theta and stored as fp32. */
    const float* rope_cos_sin;
} StageConfig;

/* One INT4 matrix W [n, k] (out = x W^T) in the canonical layout:
 *   q      : uint8 [n][ceil(k/2)], offset-binary nibbles u = code + 8
 *            (code in [-8, 7]); the low nibble holds the even k.
 *   scales : fp16 bits [n][ceil(k/G)]; W[r][c] = code * scale[r][c / G]
 *            (symmetric, no zero point; the last group of a ragged k has its
 *            own scale; fp16 subnormal scales are honoured exactly).
 * Host or device pointers, per the weights_on_device flag of stage_create. */
typedef struct QuantMatrix {
    const uint8_t*  q;
    const uint16_t* scales;
    int32_t n;
    int32_t k;
} QuantMatrix;

/* One decoder layer: pre-norm attention then pre-norm SwiGLU FFN.
 * wq [Hq*D, H], wk/wv [Hkv*D, H], wo [H, Hq*D], wg/wu [F, H], wd [H, F].
 * attn_norm / ffn_norm: [H] in act_dtype. */
typedef struct LayerWeights {
    const uint16_t* attn_norm;
    const uint16_t* ffn_norm;
    QuantMatrix wq, wk, wv, wo, wg, wu, wd;
} LayerWeights;

typedef struct Stage Stage;
typedef struct KVState KVState;

/* Create a stage: one shard of the paper's pipeline, a contiguous range of
 * decoder layers ("Per-Stage Export Pipeline", Steps 1-4: layer range, rotary
 * precomputation, stateful KV, INT4 group-128 weights).  Copies and repacks
 * every weight into library-owned device memory (the caller may free its
 * copies when the call returns), builds the rotary table and sizes the
 * workspace for STAGE_MAX_ROWS rows.
 * layers: host array of cfg->n_layers entries; weight pointers are host
 * pointers if weights_on_device == 0, device pointers otherwise.
 * Errors: INVALID/SHAPE/UNSUPPORTED for a bad config or matrix dims, OOM, HIP. */
int stage_create(const StageConfig* cfg, const LayerWeights* layers, int weights_on_device,
                 void* stream, Stage** out);
int stage_destroy(Stage* stage);

/* Allocate a KV state of n_slots slots x capacity rows for every layer and
 * kv head (the paper's per-request ReadValue/Assign state, "Stateful
 * KV-Cached Inference"; one per micro-batched request, "Multi-User
 * Throughput via Micro-Batching").  Starts with physical length P = 0 and
 * the identity beam table.  The state is bound to `stage`. */
int kv_state_alloc(Stage* stage, int n_slots, int capacity, KVState** out);
int kv_state_free(KVState* state);
/* P = 0 (contents are left in place and overwritten by later appends). */
int kv_state_reset(KVState* state);

/* Append n_tokens already-stored rows (K after rotary, V raw) for every
 * layer, slot and kv head at physical rows P..P+n-1 of each slot, then
 * P += n: the Concat -> Assign step of the paper's stateful KV ("Stateful
 * KV-Cached Inference"), used to seed a state with an existing cache.
 * k, v: [L][S][Hkv][n][D] in kv_dtype; host pointers if on_device == 0
 * (copied before return), else device pointers aligned to 16 bytes.
 * Errors: CAPACITY if P + n > capacity; INVALID for n < 1 or NULL. */
int kv_append(KVState* state, const void* k, const void* v, int n_tokens, int on_device, void* stream);

int kv_length(const KVState* state, int* length_out);

/* Copy rows [start, start+count) of one layer and slot as the slot sees them
 * (resolved through the beam table, i.e. the rows the paper's
 * Gather(ReadValue, beam_idx) would hold: "Reaching Monolithic Parity: the
 * beam_idx Gather Injection") to k_out, v_out: [Hkv][count][D] in
 * kv_dtype; host pointers if out_on_device == 0 (the call then synchronizes
 * the stream), device pointers otherwise.
 * Errors: INVALID if the range exceeds P or layer/slot is out of range. */
int kv_read(KVState* state, int layer, int slot, int start, int count,
            void* k_out, void* v_out, int out_on_device, void* stream);

/* Drop trailing rows: P = new_len (metadata only; 0 <= new_len <= P).  This is
 * the physical trim the paper replaces by masking ("The Trim Problem"); it is
 * provided for twins in tests and for fixed-length benchmarking. */
int kv_truncate(KVState* state, int new_len);

/* ------------------------------------------------------------------------
 * Compaction and serialization ("Mask-Based Rewind": masked positions stay in
 * the cache during generation and are removed when the state is serialized;
 * "Prefix Caching: KV Capture and Warm-Resume": a stage serializes its own
 * layers' KV state into a self-describing blob keeping only mask-valid rows,
 * and a restore either installs the whole state or changes nothing).
 *
 * keep_mask (all three calls): host uint8 [S][P] or NULL (keep every row).
 * Row j of slot b, as the slot sees it (through the beam table), is kept iff
 * keep_mask[b*P + j] != 0.  Slot b keeps n_b rows; the compacted length is
 * P' = max_b n_b.  Slot b's kept rows become its rows 0..n_b-1 in ascending
 * j; its rows n_b..P'-1 are zero (a slot shorter than P' must hide them with
 * a 0 in the next forward's attention_mask).  The beam table becomes the
 * identity.  slot_lengths (optional host int32 [S]) receives n_b.
 * ------------------------------------------------------------------------ */

/* Remove the rows keep_mask drops, in place: after the call P = P' and every
 * slot's rows are as described above.  One pass over the kept rows (each is
 * read once and written once); stream-ordered like a forward.
 * Errors: INVALID (NULL state), HIP; nothing changes on error. */
int kv_compact(KVState* state, const uint8_t* keep_mask, int32_t* slot_lengths, void* stream);

/* Blob layout (little endian): a StageKVBlobHeader, then int32
 * slot_length[n_slots], zero padding to header_bytes (a multiple of 256),
 * then K rows [n_layers][n_slots][n_kv_heads][length][head_dim] and V rows of
 * the same shape, in kv_dtype.  `fingerprint` identifies the stage that wrote
 * it (its StageConfig fields and norm weights); a restore into a stage with
 * another fingerprint is refused. */
#define STAGE_KV_BLOB_MAGIC   0x31505643564B5453ULL   /* "STKVCVP1" */
#define STAGE_KV_BLOB_VERSION 1
typedef struct StageKVBlobHeader {
    uint64_t magic;
    uint32_t version;
    uint32_t header_bytes;
    uint64_t fingerprint;
    int32_t  n_layers, n_slots, n_kv_heads, head_dim, kv_dtype, length;
} StageKVBlobHeader;

/* Bytes of the blob kv_capture writes for this state and keep_mask. */
int kv_capture_size(const KVState* state, const uint8_t* keep_mask, int64_t* bytes_out);

/* Serialize the kept rows of every layer, slot and kv head (the state itself
 * is unchanged).  blob: blob_bytes >= kv_capture_size bytes; a host pointer if
 * blob_on_device == 0 (the rows are gathered into a device staging buffer the
 * call allocates and frees, and the call synchronizes the stream), a device
 * pointer aligned to 16 bytes otherwise (gathered straight into the blob,
 * asynchronous).
 * Errors: INVALID (NULL), CAPACITY (blob too small), OOM, HIP. */
int kv_capture(KVState* state, const uint8_t* keep_mask, void* blob, int64_t blob_bytes, int blob_on_device,
               void* stream);

/* kv_capture into a host blob for callers that cannot allocate device
 * memory (serving loops that forbid hipMalloc, code next to a graph capture):
 * the same blob bytes as kv_capture with blob_on_device == 0, staged through
 * a fixed device array inside the library (STAGE_STATIC_SCRATCH_BYTES per
 * GPU, set up at the first stage_create on that GPU and held until the
 * process ends) instead of an allocated buffer.  The call allocates no device
 * or pinned memory.  Rows move a whole number of layers at a time: the kept
 * row lists (4 x S x P' bytes, rounded up to 256) plus one layer's kept K and
 * V rows (2 x S x n_kv_heads x P' x head_dim x 2 bytes) must fit the array,
 * else STAGE_E_CAPACITY before any work.  Synchronizes the stream.  Every
 * call on one GPU shares that GPU's array, which keeps the last call's
 * contents: calls that overlap on one GPU (other threads, other streams)
 * race and must be serialized by the caller.
 * Errors: INVALID (NULL), CAPACITY (blob too small, array too small), HIP. */
#define STAGE_STATIC_SCRATCH_BYTES (64u << 20)
int kv_capture_noalloc(KVState* state, const uint8_t* keep_mask, void* blob_host, int64_t blob_bytes, void* stream);

/* Install a captured state: P = the blob's length, rows as captured, identity
 * beam table; the state's previous contents are discarded.  The blob must come
 * from a stage with the same fingerprint, with the state's slot count, and fit
 * the state's capacity.  blob is a host pointer if blob_on_device == 0 (copied
 * through a staging buffer the call allocates; the call synchronizes the
 * stream), else a device pointer aligned to 16 bytes (its header is read back
 * synchronously).
 * slot_lengths (optional host int32 [S]) receives the captured n_b.
 * Errors: INVALID (NULL, bad magic or version), STATE_MISMATCH (another
 * stage's blob, other slot count), SHAPE (blob_bytes does not match the
 * header), CAPACITY, OOM, HIP; on error the state is unchanged. */
int kv_restore(KVState* state, const void* blob, int64_t blob_bytes, int blob_on_device, int32_t* slot_lengths,
               void* stream);

/* One request of a forward: `state` with S slots and physical length P,
 * each slot carrying n_tokens new tokens (1 = decode, K+1 = verify).
 *   positions      : host int32 [S * n_tokens], rotary position of each new
 *                    token; callers keep them at the logical length (number
 *                    of unmasked rows before it) so that masking equals trimming.
 *   beam_idx       : host int32 [S] or NULL.  Before this forward, slot b takes
 *                    the rows of slot beam_idx[b] (duplicates allowed); the
 *                    reorder persists in the state.  NULL or the identity
 *                    leaves the state as is.
 *   attention_mask : host uint8 [S * mask_len], mask_len must equal P + n_tokens;
 *                    0 hides that key column from every query of the slot;
 *                    query i also never sees physical rows after P + i.
 *   attention_mask_rows : optional host uint8 [S * n_tokens * mask_len], one
 *                    key mask per query row (the 4-D form [slot][query][key] of
 *                    "Continuous Batching on CPU, GPU, and NPU": block-diagonal
 *                    packed sequences, a shared prefix region, tree-shaped
 *                    drafts); NULL = none.  With it, query i of slot b sees
 *                    key j iff attention_mask (if given) keeps j, row i keeps j,
 *                    and j <= P + i (a query never sees a row appended after
 *                    it; tree drafts are given in an order where every node
 *                    follows its ancestors).  attention_mask may then be NULL.
 * Every query row must see at least one key (else STAGE_E_INVALID; a fully
 * masked softmax row has no value). */
typedef struct StageRequest {
    KVState*       state;
    int32_t        n_tokens;
    const int32_t* positions;
    const int32_t* beam_idx;
    const uint8_t* attention_mask;
    int32_t        mask_len;
    const uint8_t* attention_mask_rows;
} StageRequest;

/* The forward of the stage ("Stateful KV-Cached Inference": hidden states,
 * attention_mask, position ids and beam_idx in, hidden states out, KV state
 * kept inside) over n_req independent requests in one pass (micro-batching,
 * "Multi-User Throughput via Micro-Batching").  hidden_in / hidden_out: device [M][H] in act_dtype with
 * M = sum over requests of S * n_tokens, rows request-major, then slot, then
 * token.  They must not overlap.  Appends each request's new K/V rows and
 * advances its P by n_tokens once the work is enqueued.
 * Errors: INVALID (NULL, bad n, beam_idx out of range, fully masked row,
 * state repeated), SHAPE (mask_len != P + n), CAPACITY (P + n > capacity,
 * M > STAGE_MAX_ROWS, position >= max_positions), STATE_MISMATCH, HIP.  A
 * failure inside a single-launch forward is reported by stage_device_status. */
int stage_forward(Stage* stage, const StageRequest* reqs, int n_req,
                  const void* hidden_in, void* hidden_out, void* stream);

/* ------------------------------------------------------------------------
 * Prefill ("Stateful KV-Cached Inference": the prompt goes through the stage
 * in one call that fills the cache before decoding; "NPU Stages: Static,
 * Stateless Shards": a long prompt is processed in fixed-size chunks).
 * ------------------------------------------------------------------------ */

/* Most prompt rows of one stage_prefill call. */
#define STAGE_MAX_PREFILL 8192

/* n_tokens prompt rows of a one-slot state, appended after its P rows:
 * hidden_in / hidden_out device [n][H] in act_dtype (must not overlap);
 * positions host int32 [n] (rotary positions); past_mask host uint8 [P] or
 * NULL (0 hides that past row from every prompt row).  Prompt row i sees the
 * past rows the mask keeps and prompt rows 0..i.  The result equals
 * stage_forward of the same rows with that mask, up to rounding: the prompt
 * goes through the layers in passes of at most 2048 rows (the products take a
 * whole pass at once, the attention its 64-row chunks in one launch, every
 * RMSNorm input is normalized in full).  Afterwards P += n.  Allocates a
 * workspace for min(n, 2048) rows on first use (kept, grown when a longer
 * prompt comes).
 * Errors: INVALID (NULL, overlap), SHAPE (state with more than one slot),
 * CAPACITY (n outside [1, STAGE_MAX_PREFILL], P + n > capacity, position),
 * STATE_MISMATCH, UNSUPPORTED (group size other than 128), OOM, HIP. */
int stage_prefill(Stage* stage, KVState* state, int n_tokens, const int32_t* positions, const uint8_t* past_mask,
                  const void* hidden_in, void* hidden_out, void* stream);

/* ------------------------------------------------------------------------
 * Final-stage epilogue ("Top-1 Logits Compression": the last stage returns
 * the top-1 token and its probability instead of a full logits row; the last
 * stage of the pipeline owns the final norm and the LM head).
 * ------------------------------------------------------------------------ */

/* Attach the model's final RMSNorm weight (final_norm [H] in act_dtype) and
 * INT4 LM head (lm_head [vocab][H], the canonical QuantMatrix layout, group
 * size of the stage, which must be 128) to the stage.  Copies and repacks both
 * into library-owned memory; host pointers if weights_on_device == 0, else
 * device pointers.  Synchronizes the stream.  Once per stage.
 * Errors: INVALID (NULL), SHAPE (k != hidden), UNSUPPORTED (already attached,
 * group size), CAPACITY, OOM, HIP. */
int stage_head_attach(Stage* stage, const uint16_t* final_norm, const QuantMatrix* lm_head, int weights_on_device,
                      void* stream);

/* For each of the M rows of hidden (device [M][H] in act_dtype, e.g. the
 * stage's hidden_out): logits = RMSNorm(row) * final_norm, times lm_head^T
 * (fp32 accumulation), then on the device
 *   token_out[m] = argmax_j logits[m][j] (the smallest j among equal maxima),
 *   p_out[m]     = its softmax probability 1 / sum_j exp(logits[m][j] - max),
 *   logit_out[m] = the maximum (optional, NULL skips it),
 *   logits_out   = the full rows, fp32 [M][vocab] (optional, NULL skips the
 *                  write; test support).
 * All outputs are device pointers; 1 <= M <= STAGE_MAX_ROWS.  Stream-ordered
 * with the stage's other calls (it uses the stage's workspace).
 * Errors: INVALID (NULL, no head), CAPACITY (M), HIP. */
int stage_head_top1(Stage* stage, const void* hidden, int M, int32_t* token_out, float* p_out, float* logit_out,
                    float* logits_out, void* stream);

/* ------------------------------------------------------------------------
 * First-stage role ("Per-Stage Export Pipeline": the first shard also holds
 * the token embedding; in the "Overview" figure the stage-0 shard runs the
 * embeddings before its layers).  The lookup is a plain row gather.
 * ------------------------------------------------------------------------ */

/* Attach the token embedding table: table [vocab][H] of act_dtype bit
 * patterns (row t is token t's hidden vector), host memory if
 * weights_on_device == 0, else device memory.  Copied into library-owned
 * device memory as it is (no quantization).  Synchronizes the stream.  Once
 * per stage.
 * Errors: INVALID (NULL), SHAPE (vocab < 1), UNSUPPORTED (already attached),
 * CAPACITY (vocab * H above 2^36), OOM, HIP. */
int stage_embed_attach(Stage* stage, const uint16_t* table, int vocab, int weights_on_device, void* stream);

/* hidden_out[m] = table[ids[m]] for m < n, bit for bit: ids device int32 [n]
 * (e.g. the token_out of stage_head_top1 on the last stage), hidden_out device
 * [n][H] in act_dtype, ready as the hidden_in of stage_forward or
 * stage_prefill.  1 <= n <= STAGE_MAX_PREFILL.  Stream-ordered; the ids are
 * read on the device, so an id outside [0, vocab) cannot fail the call: its
 * row is written as zeros and the stage is flagged, and the next
 * stage_device_status returns STAGE_E_DEVICE.
 * Errors: INVALID (NULL, no table attached), CAPACITY (n), HIP. */
int stage_embed(Stage* stage, const int32_t* ids, int n, void* hidden_out, void* stream);

/* Test support: the dequantized weight matrix as the kernels decode it,
 * W[r][c] = code * scale exactly, written to out_host fp32 [n][k].
 * which: 0..6 = wq, wk, wv, wo, wg, wu, wd in the tiled layout of the
 * multi-kernel path; 8..14 = the same matrices in the row layout of the
 * persistent path (STAGE_E_UNSUPPORTED when the stage keeps none).
 * Synchronizes the device. */
int stage_debug_dequant(Stage* stage, int layer, int which, float* out_host);

/* Measurement support.  stage_profile_enable(stage, kernel_class) makes later
 * forwards bracket every launch of that kernel class with a pair of hipEvents
 * recorded on the launch stream (at most 65536 launches are recorded);
 * kernel_class: STAGE_KERNEL_QKV, _ATTN, _OPROJ, _GATEUP, _DOWN (kernels of the
 * multi-kernel path, which profiling of these classes selects), _PERSISTENT
 * (the single-launch forward, when the stage and row count allow it), or -1
 * to stop.
 * stage_profile_read synchronizes on the last recorded event, returns the number
 * of recorded launches and the sum of their durations in milliseconds, and
 * clears the record.  stage_profile_read_each does the same but writes each
 * launch's duration in milliseconds, in launch order, to ms_out host [capacity]
 * (launches beyond capacity are counted in *launches, not written). */
#define STAGE_KERNEL_QKV    0
#define STAGE_KERNEL_ATTN   1
#define STAGE_KERNEL_OPROJ  2
#define STAGE_KERNEL_GATEUP 3
#define STAGE_KERNEL_DOWN   4
#define STAGE_KERNEL_PERSISTENT 5
int stage_profile_enable(Stage* stage, int kernel_class);
int stage_profile_read(Stage* stage, int* launches, double* total_ms);
int stage_profile_read_each(Stage* stage, float* ms_out, int capacity, int* launches);

/* Test and measurement support: phase-boundary timestamps of the last
 * single-launch forward, recorded only when STAGE_PS_TRACE=1 was set in the
 * environment at stage_create.  out_host receives [workgroups][n_layers][32]
 * entries; *n_workgroups (if not NULL) receives the workgroup count of that
 * launch.  Times are readings of the 100 MHz device real-time counter.
 * Entries 0-9 are taken by each workgroup's control wave at: layer start
 * (q|k|v input staged), q|k|v rows done, q|k|v published, attention partials
 * done, split merge done, o rows done, residual published, gate|up rows done,
 * SwiGLU output published, down rows done.  Entries 10-15 are taken by its
 * first compute wave at the start and end of its attention, gate|up and down
 * work.  Entries 16-21 count the polling passes of the control wave's six
 * exchange waits of the layer (queries and new cache row, split partials,
 * attention output, residual after o, SwiGLU output, residual after down),
 * entries 22-27 are the times those waits ended, entries 28-30 the times the
 * first pass of the residual-after-o, residual-after-down and remaining waits
 * returned, entry 31 the time an attention workgroup published its split's
 * partial, entries 32-37 the times the first polling pass of each of the six
 * waits was issued (38, 39 unused).  n = capacity of out_host in entries.  Synchronizes the device. */
int stage_debug_phase_trace(Stage* stage, uint64_t* out_host, int n, int* n_workgroups);

/* Test support: attention record of one layer.  stage_debug_attn_arm(stage,
 * layer, max_keys) makes later forwards (which then take the per-layer
 * kernels) record, for that layer, the rotated query of every activation row
 * and query head, fp32 [M][Hq][head_dim] (before the 1/sqrt(head_dim) scale),
 * and the attention score q.k / sqrt(head_dim) of every key the row sees,
 * fp32 [M][Hq][max_keys] by key index j < max_keys (keys it does not see, and
 * j >= max_keys, are left NaN).  layer = -1 disarms.  UNSUPPORTED with the
 * vector attention (STAGE_ATTN_VECTOR=1).  stage_debug_attn_read synchronizes
 * the device and copies the last record to q_host [rows][Hq][head_dim] and
 * logits_host [rows][Hq][keys] (rows = M of that forward, keys = max_keys; the
 * caller sizes both for STAGE_MAX_ROWS rows). */
int stage_debug_attn_arm(Stage* stage, int layer, int max_keys);
int stage_debug_attn_read(Stage* stage, float* q_host, float* logits_host, int* rows, int* keys);

/* Outcome of the single-launch forwards enqueued so far.  Workgroups of that
 * launch wait on each other's published values; a wait that does not complete
 * within a bounded number of polls (a workgroup held off the device) gives up,
 * lets the launch finish, and flags the stage.  Synchronizes the device, then
 * returns STAGE_OK, or STAGE_E_DEVICE once per flagged stage (the flag is
 * cleared; an id outside the table met by stage_embed flags the stage the
 * same way).  Call it where the caller synchronizes anyway. */
int stage_device_status(Stage* stage);

/* Bytes of device memory the stage holds for weights (packed codes + scales +
 * norm weights), as stored. */
int64_t stage_weight_bytes(const Stage* stage);

const char* stage_last_error(void);

#ifdef __cplusplus
}
#endif

#endif /* PAPER_2608_19147_STAGE_H */
