/*
 * actionflow.h -- C ABI of the MI355X (gfx950) Cross-Request State Packed Forward.
 *
 * The library implements the hot path of ActionFlow (arXiv 2512.20276): one
 * Llama-style decoder forward over a packed Cross-Request State (Eq. (1)) in which
 * the prefill rows of the newest request and the single decode rows of up to K-1
 * in-flight requests share every projection GEMM, while each row attends only to
 * its own request's region of a Unified KV Ring Buffer (Sec. 3.2-3.3, Alg. 2).
 *
 * Conventions (apply to every call below)
 *  - Every call returns af_status: AF_OK (0) or a negative error.  af_last_error()
 *    returns a thread-local message describing the last failure of the calling thread.
 *  - "device" pointers are HIP device allocations (e.g. torch tensors' data_ptr());
 *    "host" pointers are ordinary CPU memory.  Tensors are dense and row-major.
 *  - hip_stream is a hipStream_t (NULL = the null stream).  Device work is queued
 *    asynchronously on it; argument checking happens on the host before any launch,
 *    and a call rejected there queues nothing and leaves every handle unchanged.
 *  - Element type of weights, activations and the ring: af_dtype (bf16 or fp32);
 *    accumulation is always fp32.
 *  - Handles are not thread-safe; one handle must not be used by two threads at once.
 *  - A weights object keeps one device copy of the step tables and one set of scratch
 *    activations, and a ring one set of device KV: use each weights object and each ring on
 *    a single stream (or order the streams yourself), since two calls in flight on different
 *    streams would overwrite each other's tables and activations.
 *  - Ownership: the ring and the weights object own the device memory they allocate;
 *    caller buffers are only borrowed for the duration of a call.
 */
#ifndef ACTIONFLOW_H
#define ACTIONFLOW_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum af_status {
  AF_OK = 0,
  AF_ERR_INVALID_ARG = -1,     /* malformed argument, inconsistent shapes or segment table */
  AF_ERR_OUT_OF_RANGE = -2,    /* a position or index beyond the configured maximum */
  AF_ERR_SLOT_BUSY = -3,       /* the next ring slot still belongs to an unreleased request */
  AF_ERR_UNKNOWN_REQUEST = -4, /* the request id owns no ring slot */
  AF_ERR_DEVICE = -5,          /* a HIP runtime call failed */
  AF_ERR_OOM = -6,             /* device or pinned-host allocation failed */
  AF_ERR_UNSUPPORTED = -7      /* shape or dtype the kernels do not implement */
} af_status;

typedef enum af_dtype { AF_F32 = 0, AF_BF16 = 1 } af_dtype;

/* Decoder shape (Sec. 3.1: a Llama-style decoder; MHA, RMSNorm, rotary positions,
 * SwiGLU MLP, no biases).  Requirements: n_kv_heads == n_heads, head_dim in {64, 128},
 * d_model == n_heads * head_dim, d_model % 32 == 0, d_ff % 16 == 0. */
typedef struct af_model_desc {
  int32_t n_layers, d_model, n_heads, n_kv_heads, head_dim, d_ff, vocab;
  float rms_eps, rope_theta;
  int32_t dtype; /* af_dtype */
} af_model_desc;

/* Unified KV Ring Buffer (Sec. 3.3): n_slots request slots of max_pos positions per
 * layer.  n_layers == 0 creates a bookkeeping-only ring (no device memory, no HIP
 * call), used to test the slot logic on machines without a GPU. */
typedef struct af_ring_desc {
  int32_t n_layers, n_slots, max_pos, n_kv_heads, head_dim;
  int32_t dtype; /* af_dtype */
} af_ring_desc;

/* One request's rows in a packed step (the per-stage sequence lengths L_s of Alg. 2).
 * Rows [q_start, q_start + q_len) of the packed state belong to request request_id,
 * whose KV lives in ring slot `slot`; the first row has absolute position pos0 inside
 * its request, so the segment's KV length after the step is pos0 + q_len.  A prefill
 * segment has pos0 == 0; the stage-s decode row of a request with prefill length L_P
 * has q_len == 1 and pos0 == L_P + s - 1. */
#define AF_SEG_EMIT 1 /* flags: produce logits and a greedy token for the segment's last row */
typedef struct af_segment {
  int32_t q_start, q_len, slot, pos0;
  int64_t request_id;
  int32_t flags;
  int32_t reserved; /* must be 0 */
} af_segment;

typedef struct af_ring af_ring;
typedef struct af_weights af_weights;

/* Message of the last failed call on this thread ("" if none).  Valid until the next call. */
const char* af_last_error(void);

/* ------------------------------------------------------------------ KV ring buffer */

/* Creates a ring; device storage [n_layers][2 (k,v)][n_slots][n_kv_heads][max_pos][head_dim]
 * of dtype is allocated and zero-filled on hip_stream (the call returns after the fill).
 * All slots start free; the first new request takes slot 0. */
af_status af_ring_create(const af_ring_desc* desc, void* hip_stream, af_ring** out);
af_status af_ring_destroy(af_ring* ring);

/* Frees every slot and returns the rotation head to slot 0 (device contents are kept). */
af_status af_ring_reset(af_ring* ring);

/* Reserves n_new positions for request_id and describes them in *out (q_start = 0,
 * flags = AF_SEG_EMIT; the caller sets q_start and flags when packing).  Sec. 3.3 keeps
 * every request in one region of the ring and moves the stages along between steps
 * (InPlaceKVShift); here that motion is an index rotation and no KV moves:
 *  - request_id resident: continuation, pos0 = current length of its slot;
 *  - otherwise: a new request takes the slot at the rotation head, which must be free
 *    (AF_ERR_SLOT_BUSY otherwise); the head advances by one modulo n_slots; pos0 = 0.
 * n_new <= 0 or request_id < 0 -> AF_ERR_INVALID_ARG; pos0 + n_new > max_pos ->
 * AF_ERR_OUT_OF_RANGE.  A failed call changes nothing. */
af_status af_ring_append(af_ring* ring, int64_t request_id, int32_t n_new, af_segment* out);

/* Frees request_id's slot (its length returns to 0) so the rotation can reuse it.
 * AF_ERR_UNKNOWN_REQUEST if the id owns no slot. */
af_status af_ring_release(af_ring* ring, int64_t request_id);

/* InPlaceKVShift as the paper's physical copy (Alg. 2, Sec. 3.3): the stage regions move
 * one stage along, so that stage s's request ends up in slot s + 1.  For s = n_stages - 2
 * down to 0, the request in slot s (if any) is moved to slot s + 1: its keys and values
 * (every layer, positions 0 .. len - 1) are copied on hip_stream and its bookkeeping moves
 * with it; slot 0 is left free and the rotation head is set to 0, so the next new request
 * takes slot 0.  Slot n_stages - 1 must be free when the call is made (the finished request
 * released; AF_ERR_SLOT_BUSY otherwise); slots >= n_stages are untouched.
 * 2 <= n_stages <= n_slots, else AF_ERR_INVALID_ARG.  The attention inputs are the same as
 * with the index rotation of af_ring_append; this is the variant that moves bytes.
 * A bookkeeping-only ring (n_layers = 0) moves only the bookkeeping.  A failed call
 * changes nothing. */
af_status af_ring_shift_stages(af_ring* ring, int32_t n_stages, void* hip_stream);

/* Copies the bookkeeping to host arrays: owners[n_slots] (request id, -1 = free),
 * lens[n_slots], *head (next slot a new request takes).  Any pointer may be NULL. */
af_status af_ring_state(const af_ring* ring, int64_t* owners, int32_t* lens, int32_t* head);

/* Writes n positions [pos0, pos0 + n) of one slot of one layer from device buffers
 * k, v laid out [n][n_kv_heads][head_dim] (rotated keys, as the forward stores them).
 * Test and pre-fill hook; does not touch the bookkeeping.  Asynchronous on hip_stream. */
af_status af_ring_write_kv(af_ring* ring, int32_t layer, int32_t slot, int32_t pos0, int32_t n,
                           const void* k, const void* v, void* hip_stream);

/* Reads the same region into device buffers k, v laid out [n][n_kv_heads][head_dim]. */
af_status af_ring_read_kv(af_ring* ring, int32_t layer, int32_t slot, int32_t pos0, int32_t n,
                          void* k, void* v, void* hip_stream);

/* Copies keys and values of positions [pos0, pos0 + n), all heads, from (src_layer, src_slot)
 * of ring src to (dst_layer, dst_slot) of ring dst, one kernel on hip_stream.  The rings must
 * agree in n_kv_heads, head_dim and dtype and hold the region (else AF_ERR_INVALID_ARG or
 * AF_ERR_OUT_OF_RANGE, nothing launched); a region onto itself is a no-op.  Bookkeeping is
 * not touched.  This is the per-request gather into a contiguous buffer (and the scatter
 * back) that a pipeline without the unified ring needs before every layer's attention
 * (Sec. 3.1, Sec. 3.3); the ring's own forward never calls it. */
af_status af_ring_copy_kv(const af_ring* src, int32_t src_layer, int32_t src_slot, af_ring* dst,
                          int32_t dst_layer, int32_t dst_slot, int32_t pos0, int32_t n, void* hip_stream);

/* ------------------------------------------------------------------ weights */

/* Number of tensors af_weights_create expects for n_layers layers: 3 + 9 * n_layers. */
int32_t af_weights_tensor_count(int32_t n_layers);

/* Copies the model into library-owned device memory, repacked for the kernels.
 * tensors[] are device pointers of dtype in HF [out, in] layout, in this order:
 *   embed [vocab, d_model], final_norm [d_model], lm_head [vocab, d_model], then per layer
 *   attn_norm [d], wq [d, d], wk [d, d], wv [d, d], wo [d, d], mlp_norm [d],
 *   w_gate [d_ff, d], w_up [d_ff, d], w_down [d, d_ff].
 * The caller may free its tensors once the call returns (it synchronizes hip_stream).
 * The object also owns the scratch activations of the forward, grown on demand. */
af_status af_weights_create(const af_model_desc* desc, const void* const* tensors, int32_t n_tensors,
                            void* hip_stream, af_weights** out);
af_status af_weights_destroy(af_weights* w);

/* ------------------------------------------------------------------ packed forward */

/* One packed step through every layer (Alg. 1 lines "Embed" to "ArgMax", Alg. 2 per layer).
 *  token_ids  device int32 [M]: a vocabulary id, or -1 to take row r of embeds;
 *  embeds     device [M, d_model] of dtype, or NULL when every id is >= 0;
 *  segs       host [n_seg]: must tile rows [0, M) exactly once, each in a distinct slot, and
 *             agree with the ring's bookkeeping (owner[slot] == request_id and
 *             len[slot] == pos0 + q_len, i.e. the rows were reserved with af_ring_append);
 *  out_hidden device [M, d_model] of dtype: residual stream after the last layer (before the
 *             final norm);
 *  out_logits device fp32 [n_emit, vocab] or NULL; out_tokens device int32 [n_emit] or NULL:
 *             final norm + LM head + greedy argmax (lowest index on ties) of the last row of
 *             every segment with AF_SEG_EMIT, in segment order.
 * Each row's key and value are written to ring[layer][slot][pos0 + i] before attention, so a
 * row attends to its request's keys 0..pos0 + i (causal inside the segment).  An id outside
 * [0, vocab) yields a zero embedding row and is counted by af_weights_device_errors. */
af_status af_packed_forward(af_weights* w, const int32_t* token_ids, const void* embeds, int32_t M,
                            const af_segment* segs, int32_t n_seg, af_ring* ring, void* out_hidden,
                            float* out_logits, int32_t* out_tokens, void* hip_stream);

/* One layer of Alg. 2 in place on hidden_inout (device [M, d_model] of dtype); same segment
 * rules as af_packed_forward.  Used for per-layer parity and single-layer timing. */
af_status af_packed_layer_forward(af_weights* w, int32_t layer, void* hidden_inout, int32_t M,
                                  const af_segment* segs, int32_t n_seg, af_ring* ring, void* hip_stream);

/* The same with the layer's keys and values in ring layer ring_layer (layer `layer` of the
 * weights): for a ring that holds one layer at a time, as the per-layer gather buffer of a
 * pipeline without the unified ring does.  ring_layer < 0 or >= the ring's layers is
 * AF_ERR_OUT_OF_RANGE / AF_ERR_INVALID_ARG. */
af_status af_packed_layer_forward_kv(af_weights* w, int32_t layer, void* hidden_inout, int32_t M,
                                     const af_segment* segs, int32_t n_seg, af_ring* ring, int32_t ring_layer,
                                     void* hip_stream);

/* Options of the forward (bit flags; default 0):
 *  AF_OPT_NO_SPLIT_K  never split a projection's K range over workgroups.  Every kernel then
 *                     computes a row exactly as it would with no other rows packed beside it
 *                     (bit-identical), at some cost in parallelism for small packed steps.  By
 *                     default, projections with too few output tiles to fill the GPU sum fp32
 *                     partials over K splits (deterministic, but in another order). */
#define AF_OPT_NO_SPLIT_K 1u
af_status af_weights_set_options(af_weights* w, uint32_t flags);

/* Copies and clears the device error counter (ids out of range) after synchronizing hip_stream. */
af_status af_weights_device_errors(af_weights* w, void* hip_stream, int32_t* count);

/* ------------------------------------------------------------------ forward without allocation
 * For callers that cannot allocate device memory during a step: code under HIP graph capture,
 * serving loops and harnesses that forbid hipMalloc.  Not a step of the paper's method.
 *
 * af_packed_forward_noalloc takes the arguments of af_packed_forward, follows the same rules and
 * returns the same results (bit for bit: the same kernels in the same order).  Every device
 * workspace of the step (normalized rows, queries, attention output, the MLP activation, split-K
 * partial sums, the step tables and the rotary table) is carved from one array of
 * AF_NOALLOC_SCRATCH_BYTES (64 MiB) that the library holds on each GPU it runs on, from the
 * first call there until the process ends.  The call allocates nothing: no hipMalloc, hipFree
 * or pinned host memory (the step tables are copied from pageable host memory with
 * hipMemcpyAsync on hip_stream).  The first call on a device looks up the array's address
 * there, so that device must be current, as for every call.
 *  - A step whose workspace would not fit (it grows with M, d_model, d_ff, the ring's max_pos
 *    and the number of emitting rows; the 7B-shape step of 282 packed rows needs about 42 MiB)
 *    is rejected with AF_ERR_OUT_OF_RANGE before any launch, the need and the limit in
 *    af_last_error().
 *  - Every call on one GPU shares that GPU's array, which keeps the last call's contents: calls
 *    that overlap on one GPU (two streams, two threads) race and corrupt each other's results;
 *    serialize them. */
#define AF_NOALLOC_SCRATCH_BYTES (64ull * 1024 * 1024)
af_status af_packed_forward_noalloc(af_weights* w, const int32_t* token_ids, const void* embeds, int32_t M,
                                    const af_segment* segs, int32_t n_seg, af_ring* ring, void* out_hidden,
                                    float* out_logits, int32_t* out_tokens, void* hip_stream);

/* ------------------------------------------------------------------ single steps of the path
 * Each runs one step of Alg. 2 / Alg. 1 on caller buffers with the same kernels the forward
 * uses.  They exist for per-step parity tests and timing; the segment rules above apply. */

/* Alg. 1 Embed: out [M, d] <- embed[id] or embeds[r]. */
af_status af_op_embed(af_weights* w, const int32_t* token_ids, const void* embeds, int32_t M, void* out,
                      void* hip_stream);

/* Alg. 2 Norm: y[r] = g * x[r] / sqrt(mean(x[r]^2) + eps), rows of length D, dtype elements. */
af_status af_op_rmsnorm(int32_t dtype, const void* x, const void* g, void* y, int32_t M, int32_t D, float eps,
                        void* hip_stream);

/* Plain projection y [M, N] = x [M, K] . w [N, K]^T (the GEMM core of every projection). */
af_status af_op_linear(int32_t dtype, const void* x, const void* w, void* y, int32_t M, int32_t N, int32_t K,
                       void* hip_stream);

/* Alg. 2 QKVProj + FusedRoPEAndWriteKV on normalized rows xn [M, d]: q_out [M, d] receives the
 * rotated queries; rotated keys and values go to the ring at each row's (slot, position). */
af_status af_op_qkv_rope_write(af_weights* w, int32_t layer, const void* xn, int32_t M, const af_segment* segs,
                               int32_t n_seg, af_ring* ring, void* q_out, void* hip_stream);

/* Alg. 2 VarlenAttention: o [M, d] from rotated queries q [M, d] and the ring (keys/values of
 * positions 0..pos0 + i of each row's slot must already be in place). */
af_status af_op_attention(af_ring* ring, int32_t layer, const void* q, int32_t M, const af_segment* segs,
                          int32_t n_seg, void* o, void* hip_stream);

/* Alg. 2 OutputProj + residual: hidden [M, d] += o [M, d] . wo^T (in place). */
af_status af_op_o_proj_residual(af_weights* w, int32_t layer, const void* o, void* hidden, int32_t M,
                                void* hip_stream);

/* Alg. 2 MLP, first half: act [M, d_ff] = SiLU(xn . w_gate^T) * (xn . w_up^T). */
af_status af_op_gate_up_swiglu(af_weights* w, int32_t layer, const void* xn, void* act, int32_t M,
                               void* hip_stream);

/* Alg. 2 MLP, second half: hidden [M, d] += act [M, d_ff] . w_down^T (in place). */
af_status af_op_down_residual(af_weights* w, int32_t layer, const void* act, void* hidden, int32_t M,
                              void* hip_stream);

/* Alg. 1 ArgMax(LMHead(Norm(.))) for the last row of each emitting segment of hidden [M, d]. */
af_status af_op_lm_head_argmax(af_weights* w, const void* hidden, int32_t M, const af_segment* segs,
                               int32_t n_seg, float* out_logits, int32_t* out_tokens, void* hip_stream);

/* ------------------------------------------------------------------ timing
 * Kernel classes for per-kernel timing with HIP events recorded on the launch stream. */
typedef enum af_kernel_class {
  AF_K_EMBED = 0, AF_K_RMSNORM, AF_K_GEMM_QKV, AF_K_ATTENTION, AF_K_GEMM_O, AF_K_GEMM_GATEUP,
  AF_K_GEMM_DOWN, AF_K_LM_HEAD, AF_K_ARGMAX, AF_K_COUNT
} af_kernel_class;

/* Starts recording a start/stop event pair around every launch of the classes in mask
 * (bit c = class c; 0 stops recording).  Clears previous totals. */
af_status af_timing_enable(af_weights* w, uint32_t mask);

/* Synchronizes the recorded events and returns, per class, the summed kernel milliseconds
 * and the number of launches (arrays of AF_K_COUNT entries; either may be NULL). */
af_status af_timing_read(af_weights* w, double* total_ms, int64_t* launches);

#ifdef __cplusplus
}
#endif

#endif /* ACTIONFLOW_H */
