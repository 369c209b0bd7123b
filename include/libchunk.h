/*
 * libchunk — one device's share of Piper's data-parallel training hot path
 * on an AMD Instinct MI355X (gfx950).
 *
 * Piper lowers a training program to a DAG of Chunk (compute) and Comm
 * (communication) nodes; each Chunk has an exec run on an assigned stream
 * for one pass, F (forward) or B (backward) (Piper Section 4.1, "IR" and
 * the PASS dimension). Split replicates Chunks per microbatch and Order
 * sequences them (Section 4.1, "Scheduling directives"). The worker keeps
 * forward activations until the matching backward consumes them and
 * accumulates gradients into one flat buffer per model-state bucket
 * (Section 4.3.2, "Memory management"); under ZeRO-1 each rank updates the
 * optimizer state of its own shard (Section 6.2).
 *
 * This library implements that share for one transformer-decoder pipeline
 * stage: Chunk F / Chunk B of every microbatch in an Order, fp32 gradient
 * accumulation into the stage's flat bucket, and a fused AdamW step with a
 * bf16 cast over a flat shard.
 *
 * Conventions shared by every entry point
 *   - C ABI, never throws. Every function returns an lc_status; a negative
 *     value means failure and lc_last_error() gives a message.
 *   - Argument, descriptor and Order errors are detected on the host before
 *     anything is enqueued: such a call has no side effects.
 *   - "device" pointers are HIP device allocations owned by the caller; the
 *     library allocates no device memory. Work is enqueued on `stream`
 *     (a hipStream_t; NULL is the default stream) and nothing synchronises
 *     the host: results are ready once the caller synchronises the stream.
 *     LC_ERR_HIP reports a failed launch; faults surface at that sync.
 *   - Device pointers must be 16-byte aligned (else LC_ERR_INVALID_ARG).
 *   - Sizes and offsets are 64-bit.
 *   - Thread-compatible: one lc_stage must not be used by two host threads
 *     at once.
 */
#ifndef LIBCHUNK_H
#define LIBCHUNK_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum lc_status {
  LC_OK = 0,
  LC_ERR_INVALID_ARG = -1,  /* bad pointer, size, alignment or descriptor field */
  LC_ERR_UNSUPPORTED = -2,  /* a valid shape the library does not implement     */
  LC_ERR_BAD_ORDER = -3,    /* an Order that breaks the Order rules below        */
  LC_ERR_STASH_FULL = -4,   /* more microbatches in flight than stash slots      */
  LC_ERR_STATE = -5,        /* F twice for one microbatch, or B without its F    */
  LC_ERR_WORKSPACE = -6,    /* workspace smaller than lc_workspace_bytes()       */
  LC_ERR_HIP = -7           /* a HIP runtime call or kernel launch failed        */
} lc_status;

/* Element types. A stage's compute_dtype is LC_FP32 or LC_BF16; LC_FP16
 * appears only in the per-tensor types of libchunk_ops.h (a bf16 stage keeps
 * its attention q, k, v in fp16, see lc_stage_desc). */
typedef enum lc_dtype { LC_FP32 = 0, LC_BF16 = 1, LC_FP16 = 2 } lc_dtype;

/* Piper's PASS dimension (Section 4.1): F = forward, B = full backward,
 * BI = backward for the inputs (dX only), BW = backward for the weights (the
 * parameter gradient only). BI and BW split B for schedules that defer the
 * weight-gradient work into pipeline bubbles (ZeroBubble). */
typedef enum lc_pass { LC_PASS_F = 0, LC_PASS_B = 1, LC_PASS_BI = 2, LC_PASS_BW = 3 } lc_pass;

/* One pipeline stage: n_layers pre-norm decoder layers. Every layer is
 *   n1 = RMSNorm(x; g1); q,k,v = n1 Wq^T, n1 Wk^T, n1 Wv^T; rotate-half RoPE
 *   on q and k (positions 0..seq_len-1 per sequence, angle p*base^(-2i/hd));
 *   o = causal softmax(q k^T / sqrt(hd)) v per head; h = x + o Wo^T;
 *   n2 = RMSNorm(h; g2); y = h + FFN(n2)
 * Qwen3-style variant: with qk_norm, q and k are RMS-normalised over each
 * head's head_dim values (gains qn, kn [head_dim], epsilon rms_eps) before
 * RoPE; with 0 < n_kv_heads < n_heads (grouped-query attention) k and v
 * have n_kv_heads heads (Wk, Wv are [n_kv_heads*head_dim, d]) and query
 * head h uses key/value head h / (n_heads / n_kv_heads).
 * with FFN the SwiGLU (silu(n2 W1^T) * (n2 W3^T)) W2^T when n_experts == 0,
 * else a top-k (k = 2) softmax-routed mixture of SwiGLU experts whose gate
 * weights are renormalised over the selected experts (ties pick the lower
 * expert index). Activations are token-major [micro_batch, seq_len,
 * d_model]; weights are [out, in] row-major.
 *
 * Precision of a bf16 stage: every matrix product takes bf16 operands (the
 * weights, the normalised activations, the attention output, the SwiGLU
 * output and every gradient operand) with fp32 accumulation; attention's
 * q, k, v and softmax probabilities use fp16 operands (values of bounded
 * range, three more mantissa bits, same matrix-core rate); the residual
 * stream between and inside layers, the SwiGLU gate/up values kept for the
 * backward, the residual-stream gradient and all norm inputs are fp32.
 * X, Y, dY and dX at the stage boundary are bf16. An fp32 stage computes
 * everything in fp32. */
typedef struct lc_stage_desc {
  int32_t n_layers;
  int32_t d_model;       /* == n_heads * head_dim */
  int32_t n_heads;
  int32_t head_dim;
  int32_t d_ff;          /* dense FFN width (ignored when n_experts > 0) */
  int32_t n_experts;     /* 0 = dense SwiGLU FFN */
  int32_t top_k;         /* experts per token (must be 2 when n_experts > 0) */
  int32_t d_ff_expert;   /* FFN width of each expert */
  int32_t seq_len;
  int32_t micro_batch;   /* sequences per microbatch */
  float rms_eps;         /* RMSNorm epsilon, inside the square root */
  float rope_base;       /* RoPE base (10000) */
  int32_t causal;        /* must be 1 */
  int32_t compute_dtype; /* lc_dtype of weights and activations; gradients
                            are always accumulated in fp32 */
  int32_t n_kv_heads;    /* key/value heads; 0 = n_heads; divides n_heads */
  int32_t qk_norm;       /* 1: per-head RMSNorm of q and k before RoPE */
} lc_stage_desc;

/* Tensor ids of the canonical flat layout (one bucket per stage). Per layer,
 * in this order: WQ [d,d], WK, WV [n_kv_heads*head_dim, d], WO [d,d]; G1
 * [d]; with qk_norm QN, KN [head_dim]; dense: W1 (gate) [f,d],
 * W3 (up) [f,d], W2 (down) [d,f]; MoE: WR (router) [E,d], then for each
 * expert e: W1 [fe,d], W3 [fe,d], W2 [d,fe]; finally G2 [d]. The gradient,
 * master, m and v buffers use the same layout. */
typedef enum lc_tensor_id {
  LC_T_WQ = 0, LC_T_WK = 1, LC_T_WV = 2, LC_T_WO = 3, LC_T_G1 = 4,
  LC_T_W1 = 5, LC_T_W3 = 6, LC_T_W2 = 7, LC_T_G2 = 8, LC_T_WR = 9,
  LC_T_QN = 10, LC_T_KN = 11
} lc_tensor_id;

/* Flag or-ed into an entry's pass: this entry and the next one form an
 * overlapped pair (a nested list of two filters in Piper's Order directive,
 * Section 4.1), which lc_run_order_overlap runs on two streams. */
enum { LC_ORDER_WITH_NEXT = 0x100 };

/* One Order entry: run pass `pass` (lc_pass, optionally | LC_ORDER_WITH_NEXT)
 * of microbatch `mb`. */
typedef struct lc_order_entry {
  int32_t mb;
  int32_t pass;
} lc_order_entry;

/* An Order over num_microbatches microbatches (Piper Section 4.1, Order).
 * Rules (checked by lc_order_validate and again by lc_run_order):
 *   - for each 0 <= mb < num_microbatches, (mb, F) appears exactly once,
 *     and so does either (mb, B) or the pair (mb, BI), (mb, BW); F(mb)
 *     precedes B(mb) or BI(mb), and BI(mb) precedes BW(mb);
 *   - the F entries are in increasing mb order, and so are the B and BI
 *     entries taken together (both hand dX to the upstream stage): a
 *     pipeline stage must consume microbatches in the order its neighbour
 *     produced them, and Piper rejects schedules that do not (Section
 *     4.3.2, "Communication management"). BW entries only add into the
 *     local gradient accumulator and may come in any order;
 *   - at most max_in_flight microbatches sit between their F and their B
 *     or BW, and at most max_w_pending between their BI and BW (else
 *     LC_ERR_STASH_FULL);
 *   - an overlapped pair (first entry flagged LC_ORDER_WITH_NEXT) holds two
 *     entries of different microbatches: F with B, BI or BW, or BI with BW
 *     (at most one of the two uses the backward's working buffers, at most
 *     one adds into the gradient). Both may run at once, so the rules above
 *     are checked with the pair's F (or its BI, beside a BW) first. */
typedef struct lc_order {
  int32_t num_microbatches;
  int32_t n_entries;
  const lc_order_entry *entries; /* host memory, n_entries long */
} lc_order;

/* One microbatch's activations, all device pointers, [micro_batch, seq_len,
 * d_model] in compute_dtype. `x` is read by F and again by B (or BI): it
 * must stay valid and unchanged until B (or BI) of this microbatch has been
 * enqueued and has run. F writes `y`; B and BI read `dy` and write `dx`; BW
 * reads none of them. Unused fields may be NULL (F needs x and y; B and BI
 * need dy and dx). */
typedef struct lc_microbatch_desc {
  int32_t mb;
  int32_t reserved;
  const void *x;
  void *y;
  const void *dy;
  void *dx;
} lc_microbatch_desc;

/* The stage's bucket: compute weights in the canonical layout and the fp32
 * gradient accumulator with the same layout. The caller zeroes `grad` (+0.0)
 * before the first backward of a step; every backward adds its microbatch's
 * gradient (no 1/M scaling). */
typedef struct lc_param_bufs {
  const void *w;   /* device, compute_dtype */
  float *grad;     /* device, fp32 */
} lc_param_bufs;

/* AdamW hyper-parameters for shard_adam_step. step >= 1 counts optimizer
 * steps (bias correction uses beta^step). */
typedef struct lc_adam_hparams {
  float lr;
  float beta1;
  float beta2;
  float eps;
  float weight_decay;
  int32_t reserved;
  int64_t step;
} lc_adam_hparams;

typedef struct lc_stage lc_stage; /* opaque, host memory */

/* ---------------------------------------------------------------- host-only
 * These make no HIP call and may be used without a GPU. */

/* Number of elements of the stage's flat bucket: the one flat parameter
 * (and gradient) buffer per bucket that Piper's workers keep (Section 4.3.2,
 * "Memory management"; Section 6.2 shards such buffers for ZeRO). Per
 * layer, in order: Wq, Wk, Wv, Wo, g1, then W1 (gate), W3 (up), W2 (down)
 * or, for a mixture of experts, Wr and each expert's W1, W3, W2, then g2
 * (q/k gains after g1 when qk_norm is set). LC_ERR_INVALID_ARG for a bad
 * descriptor. */
lc_status lc_param_count(const lc_stage_desc *desc, size_t *n_elems);

/* Offset (elements) and shape of tensor `tensor_id` of layer `layer`
 * (expert `expert` for MoE W1/W3/W2, else pass 0) in the flat bucket of
 * lc_param_count (Section 4.3.2, "Memory management"). shape[1] is 1 for
 * vectors. LC_ERR_INVALID_ARG for an index out of range. */
lc_status lc_param_offset(const lc_stage_desc *desc, int32_t layer, int32_t tensor_id,
                          int32_t expert, size_t *offset, int64_t shape[2]);

/* The 1F1B Order of stage s of a P-stage pipeline over M microbatches:
 * W = min(P-s-1, M) forwards, then M-W (forward, backward) pairs, then W
 * backwards. `out` holds `capacity` entries (needs 2M); *n receives 2M. */
lc_status lc_order_1f1b(int32_t M, int32_t P, int32_t s, lc_order_entry *out,
                        int32_t capacity, int32_t *n);

/* The 1F1B Order above with every steady-state (F, B) pair flagged as an
 * overlapped pair (none when W = 0: each pair would be one microbatch's F
 * and B). Needs 2M entries. */
lc_status lc_order_1f1b_overlap(int32_t M, int32_t P, int32_t s, lc_order_entry *out,
                                int32_t capacity, int32_t *n);

/* The 1F1B Order above with every B split into BI then BW: BW(j) is placed
 * right after BI(j + w_delay) (after the last BI when there is none), and
 * the BW entries keep microbatch order. w_delay = 0 gives BI(j) BW(j)
 * pairs; larger values defer weight passes, up to min(w_delay + 1, M) of
 * them pending at once. `out` holds `capacity` entries (needs 3M). */
lc_status lc_order_1f1b_split(int32_t M, int32_t P, int32_t s, int32_t w_delay,
                              lc_order_entry *out, int32_t capacity, int32_t *n);

/* lc_order_1f1b_split with every BI that is directly followed by the BW of
 * another microbatch flagged LC_ORDER_WITH_NEXT: the two run as an
 * overlapped pair (a weight pass beside the next microbatch's input pass,
 * Section 4.1's nested Order), each entry in at most one pair. Same
 * arguments and errors as lc_order_1f1b_split. */
lc_status lc_order_1f1b_split_overlap(int32_t M, int32_t P, int32_t s, int32_t w_delay,
                                      lc_order_entry *out, int32_t capacity, int32_t *n);

/* Checks an Order against the rules above for at most max_in_flight
 * stashed microbatches and max_w_pending pending weight passes. *peak and
 * *peak_w (nullable) receive the largest numbers of each seen. Returns
 * LC_OK, LC_ERR_BAD_ORDER or LC_ERR_STASH_FULL. */
lc_status lc_order_validate_split(const lc_order *order, int32_t max_in_flight,
                                  int32_t max_w_pending, int32_t *peak, int32_t *peak_w);

/* lc_order_validate_split with max_w_pending = max_in_flight (a microbatch
 * whose weight pass is pending still holds its stash slot, so this is no
 * extra bound). */
lc_status lc_order_validate(const lc_order *order, int32_t max_in_flight, int32_t *peak);

/* Device workspace a stage needs for max_in_flight stashed microbatches and
 * max_w_pending weight-pass slots (0 <= max_w_pending <= max_in_flight). The
 * caller allocates it once; the stage carves it into the buffers that
 * Piper's memory manager allocates per task and frees after their last
 * consumer (Section 4.3.2, "Memory management"), reused here in stream
 * order:
 * activation stash, weight-pass slots, backward scratch and RoPE table. A
 * weight-pass slot holds, per layer, the gradient operands of the weight
 * products ([T, d], [R, 2 f], [T, d], [T, d + 2 d_kv] in the compute dtype,
 * T = micro_batch * seq_len; R = T and f = d_ff for a dense FFN, R = 2T
 * routed rows and f = d_ff_expert for a mixture of experts, which also keeps
 * its routed dy rows [2T, d], router logit gradients [T, 2] fp32 and the
 * router gradient's fp32 partial sums) and the norms' fp32 gain-gradient
 * partial sums. */
lc_status lc_workspace_bytes_split(const lc_stage_desc *desc, int32_t max_in_flight,
                                   int32_t max_w_pending, size_t *bytes);

/* lc_workspace_bytes_split with no weight-pass slots. */
lc_status lc_workspace_bytes(const lc_stage_desc *desc, int32_t max_in_flight, size_t *bytes);

/* ---------------------------------------------------------------- stage
 * lc_stage_create validates the descriptor, carves the caller's workspace
 * (device, >= lc_workspace_bytes, 256-byte aligned) into stash slots and
 * scratch, and enqueues the upload of the RoPE cos/sin table on `stream`.
 * The handle owns host memory only; lc_stage_destroy frees it (synchronise
 * the stream first). */
lc_status lc_stage_create(const lc_stage_desc *desc, void *workspace, size_t ws_bytes,
                          int32_t max_in_flight, void *stream, lc_stage **out);

/* lc_stage_create with max_w_pending weight-pass slots (workspace >=
 * lc_workspace_bytes_split): the stage can then run chunk_backward_input /
 * chunk_backward_weight. lc_stage_create has none (LC_ERR_STASH_FULL on
 * the first chunk_backward_input). */
lc_status lc_stage_create_split(const lc_stage_desc *desc, void *workspace, size_t ws_bytes,
                                int32_t max_in_flight, int32_t max_w_pending, void *stream,
                                lc_stage **out);
lc_status lc_stage_destroy(lc_stage *stage);

/* Chunk F of one microbatch: Y = stage(X). Stashes the activations the
 * backward needs in a free slot (LC_ERR_STATE if this microbatch is already
 * stashed, LC_ERR_STASH_FULL if no slot is free). */
lc_status chunk_forward(lc_stage *stage, const lc_param_bufs *params,
                        const lc_microbatch_desc *mb, void *stream);

/* Chunk B of one microbatch: dX = (dY/dX)^T dY and grad += dL/dW for
 * L = sum(dY * Y), using the slot stashed by chunk_forward of the same mb
 * (LC_ERR_STATE if none), which is released afterwards. Gradients are added
 * to params->grad in fp32, one addition per element. */
lc_status chunk_backward(lc_stage *stage, const lc_param_bufs *params,
                         const lc_microbatch_desc *mb, void *stream);

/* Chunk BI of one microbatch: dX = (dY/dX)^T dY exactly as
 * chunk_backward computes it, without the parameter gradient. Reads dy now
 * (and x, for the first layer's norm); writes the weight products' gradient
 * operands and the norms' gain partial sums into a free weight-pass slot
 * (LC_ERR_STASH_FULL if none). The stash slot stays taken until BW.
 * LC_ERR_STATE if mb has no stashed forward or already ran BI. */
lc_status chunk_backward_input(lc_stage *stage, const lc_param_bufs *params,
                               const lc_microbatch_desc *mb, void *stream);

/* Chunk BW of one microbatch: grad += dL/dW from the operands BI left,
 * then releases the microbatch's weight-pass and stash slots. Only mb->mb
 * is read from the descriptor. Per element the addition is the one
 * chunk_backward makes, so BI + BW in the same microbatch order as the B
 * entries of an Order gives a bit-identical gradient. LC_ERR_STATE if mb
 * has no pending BI. */
lc_status chunk_backward_weight(lc_stage *stage, const lc_param_bufs *params,
                                const lc_microbatch_desc *mb, void *stream);

/* Runs a whole Order: validates it (no side effects on failure), then
 * enqueues chunk_forward / chunk_backward / chunk_backward_input /
 * chunk_backward_weight in entry order. mbs[i] describes microbatch i
 * (num_microbatches entries). Needs an empty stash (LC_ERR_STATE). If a
 * launch fails after some entries were enqueued, the stash is emptied again
 * before the error returns (the run's outputs are then undefined), so the
 * stage stays usable. */
lc_status lc_run_order(lc_stage *stage, const lc_param_bufs *params, const lc_order *order,
                       const lc_microbatch_desc *mbs, void *stream);

/* lc_run_order on two streams (Piper Section 4.3.2, worker scheduling loop
 * and stream management; the overlap of Section 4.1's nested Order): entries
 * outside pairs and the backward of each overlapped pair (B, or BI beside a
 * BW) run on `stream`, the pair's other entry on `aux_stream`. Within a pair
 * the entry with more downstream dependants in the Order is enqueued first
 * (F before B; BI before BW). A stream waits on the other's hipEvent only
 * where an entry depends on work last enqueued there: the same microbatch's
 * earlier pass, the stash or weight-pass slot it takes, the backward's
 * working buffers, or the gradient bucket. aux_stream first waits for all
 * work already enqueued on `stream`, and `stream` finally waits for
 * aux_stream, so the call behaves like one enqueue on `stream`. Outputs and
 * gradients are identical to lc_run_order's. aux_stream may equal stream
 * (pairs then run one after the other). The events are host resources of
 * the stage (created on first use, destroyed by lc_stage_destroy). */
lc_status lc_run_order_overlap(lc_stage *stage, const lc_param_bufs *params,
                               const lc_order *order, const lc_microbatch_desc *mbs,
                               void *stream, void *aux_stream);

/* ZeRO-2/3 buffers of one data-parallel rank, for lc_run_order_zero (Piper
 * Section 4.3.2 "Memory management": persistent shard buffers, temporary full
 * buffers for rematerialised state, a full gradient buffer per backward;
 * ZeRO-2 and ZeRO-3 of Section 6.2). One GPU has no collectives: the
 * reduce-scatter after each backward is this rank's share of it (its slice
 * of the full gradient added into its shard), and the all-gather before
 * each chunk concatenates weight shards that are all resident here. */
typedef struct lc_zero_bufs {
  int32_t level;        /* 2: gradients sharded; 3: gradients and weights */
  int32_t n_w_shards;   /* level 3: number of weight shards, 1..1024 */
  float *grad_shard;    /* persistent fp32 gradient shard: bucket elements
                           [shard_offset, shard_offset + shard_len) */
  size_t shard_offset;  /* multiple of 4 */
  size_t shard_len;
  float *grad_full;     /* temporary fp32 [n_params]: each B / BW's full
                           gradient, zeroed at its start, reduced at its end */
  const void *const *w_shards;  /* level 3: host array of n_w_shards device
                                   pointers (compute dtype), bucket order */
  const size_t *w_shard_lens;   /* level 3: host array, elements, summing to
                                   the bucket size */
  void *w_full;         /* level 3: temporary full weights (compute dtype),
                           rebuilt from the shards before every entry */
} lc_zero_bufs;

/* Runs an Order on one stream like lc_run_order, with ZeRO buffers: before
 * every entry (level 3) the weight shards are gathered into w_full and the
 * entry reads its weights there (else params->w); every B and BW zeroes
 * grad_full, adds its gradient there, then adds grad_full's slice
 * [shard_offset, shard_offset + shard_len) into grad_shard. params->grad is
 * ignored. grad_shard then holds, bit for bit, that slice of the gradient
 * lc_run_order accumulates (every addition into +0 is exact). Overlapped
 * pairs run one after the other. Device buffers 16-byte aligned;
 * LC_ERR_INVALID_ARG for a bad layout, before anything is enqueued: a slice
 * out of range, shard lengths that do not sum to the bucket, a grad_shard
 * that overlaps grad_full, or a weight shard that overlaps w_full anywhere
 * but at its own place there (a shard already at its place, an in-place
 * gather, is not copied). */
lc_status lc_run_order_zero(lc_stage *stage, const lc_param_bufs *params, const lc_zero_bufs *zero,
                            const lc_order *order, const lc_microbatch_desc *mbs, void *stream);

/* Routing of a mixture-of-experts stage: copies the two experts chosen for
 * every token of layer `layer` of microbatch `mb` (int32 [micro_batch *
 * seq_len, 2], the order of lc_moe_route's sel) into the caller's device
 * buffer `sel_out`. Valid between chunk_forward(mb) and chunk_backward(mb)
 * (LC_ERR_STATE otherwise); LC_ERR_INVALID_ARG for a dense stage or a layer
 * out of range. Enqueued on `stream`; for tests and monitoring (routing
 * statistics), not needed to train. */
lc_status lc_stage_moe_routing(lc_stage *stage, int32_t mb, int32_t layer, int32_t *sel_out,
                               void *stream);

/* Timing of the weight-gradient products (measurement support, not needed to
 * train). These are the products that form dW from the backward's output
 * gradients and the stashed activations, in Chunk B or in its weight half
 * (the BW pass of Section 4.1): G[W2], G[W1;W3], G[Wo], G[Wq;Wk;Wv]
 * and, in mixture-of-experts layers, the grouped expert products.
 *
 * lc_stage_timer_enable(stage, max_launches): creates 2 * max_launches HIP
 * events (host-side handles, no device buffers) and from then on brackets
 * the next max_launches such launches, in launch order, with a pair of
 * events recorded on the stream each is launched on; later launches run
 * untimed. Any earlier events are destroyed and the count restarts.
 * max_launches = 0 turns timing off. LC_ERR_INVALID_ARG for a null stage or
 * max_launches outside [0, 2^20]; LC_ERR_HIP if event creation fails.
 *
 * lc_stage_timer_read(stage, ms, flop, cap, n): waits for the first
 * min(cap, timed) stop events and writes, per timed launch i, its duration
 * ms[i] (milliseconds between its two events) and its algorithmic FLOP
 * flop[i] = 2 M N K; *n receives the number of launches timed since the last
 * read (which may exceed cap) and the count restarts, so the events are
 * reused. ms and flop are host arrays of cap entries. LC_ERR_INVALID_ARG for a
 * null stage or n, negative cap, or null arrays with cap > 0. Events still
 * pending in a stream must not be re-armed: read only after the launches
 * timed so far were enqueued, and enable again only after a read. */
lc_status lc_stage_timer_enable(lc_stage *stage, int32_t max_launches);
lc_status lc_stage_timer_read(lc_stage *stage, float *ms, double *flop, int32_t cap, int32_t *n);

/* ---------------------------------------------------------------- buffers */

/* accum[i] += g[i] for i < n, in fp32 (g is fp32 or bf16 per g_dtype); each
 * element is read and written exactly once. accum and g must not overlap. */
lc_status chunk_accumulate_grad(float *accum, const void *g, int32_t g_dtype, size_t n,
                                void *stream);

/* buf[i] = +0.0f for i < n (a kernel, so that it can be captured in a
 * graph). buf 16-byte aligned. */
lc_status lc_zero_fill_f32(float *buf, size_t n, void *stream);

/* AdamW over a flat shard of n elements (decoupled weight decay, bias
 * correction). With host scalars c_wd = 1 - lr*wd, step_size =
 * lr/(1-beta1^t) and bc2s = sqrt(1-beta2^t) (computed in double, rounded
 * once to float), every element does, one fp32 rounding per operation:
 *   p = p*c_wd; m = b1*m + (1-b1)*g; v = b2*v + (1-b2)*(g*g);
 *   p = p - step_size * (m / (sqrt(v)/bc2s + eps));
 *   out_bf16 = round-to-nearest-even(p)   (if out_bf16 != NULL)
 * grad is fp32 or bf16 per grad_dtype. master, m, v are updated in place. */
lc_status shard_adam_step(float *master, float *m, float *v, const void *grad,
                          int32_t grad_dtype, uint16_t *out_bf16, size_t n,
                          const lc_adam_hparams *hp, void *stream);

/* Message for the last non-OK status returned on this thread. */
const char *lc_last_error(void);

#ifdef __cplusplus
}
#endif

#endif /* LIBCHUNK_H */
