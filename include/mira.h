/*
 * mira.h - C ABI of the Mira per-layer MoE expert step on AMD Instinct MI355X
 * (gfx950).
 *
 * Paper: "Memory-Efficient MoE Inference Using Adaptive Caching and
 * Predictive Expert Staging" (Mira).  The library runs one MoE layer over
 * experts held in the paper's compressed expert format (section IV-B): router
 * top-k and combine weights (section II-A), a stable token-to-expert
 * permutation, the SwiGLU expert FFN fused with INT8 dequantization
 * (sections IV-A and IV-F), and the weighted combine.  Experts are found
 * through a slot table into a caller-owned pool of device slots, the HOT and
 * STAGE regions of the expert cache (section IV-C); slots are filled from
 * pinned host memory by asynchronous copies (sections IV-E, IV-F).  Predictor
 * heads score the experts of layer l+2 (section IV-E): a two-layer MLP and the
 * paper's MixtureHead.
 *
 * Conventions for every entry point:
 *  - Return 0 (MIRA_OK) on success or a negative mira_status.  A failing call
 *    launches nothing; mira_last_error() then describes the failure (a
 *    thread-local string owned by the library, valid until the next call on
 *    the same thread).  No C++ exception crosses this interface.
 *  - "device" pointers are HIP device allocations of the current device;
 *    "host" pointers are ordinary host memory.  The caller owns every buffer;
 *    the library never frees caller memory and allocates none on the forward
 *    path (it uses the caller's workspace).
 *  - Work is enqueued on the given HIP stream and is asynchronous: outputs are
 *    valid once the stream reaches the call.  Only the host path of
 *    mira_pack_experts runs synchronously.  Calls on distinct workspaces may
 *    run concurrently.
 *  - mira_moe_forward, mira_moe_route and mira_moe_experts only launch
 *    kernels (no allocation, copy, memset or host synchronisation), so they
 *    can be captured into a HIP graph and replayed; a replay recomputes
 *    everything from the buffers the captured call was given.
 *  - Tensors are dense and row-major; shapes are given in brackets.
 */
#ifndef MIRA_H_
#define MIRA_H_

#include <stddef.h>
#include <stdint.h>

#include <hip/hip_runtime_api.h>

#ifdef __cplusplus
extern "C" {
#endif

/* ---- status codes ------------------------------------------------------- */
typedef enum mira_status {
  MIRA_OK = 0,
  MIRA_ERR_ARG = -1,        /* null pointer, bad enum or flag, inconsistent argument */
  MIRA_ERR_SHAPE = -2,      /* unsupported or inconsistent sizes */
  MIRA_ERR_ALIGN = -3,      /* a pointer or stride breaks the stated alignment */
  MIRA_ERR_WORKSPACE = -4,  /* workspace missing or smaller than mira_workspace_bytes() */
  MIRA_ERR_HIP = -5,        /* a HIP runtime call failed; the message names it */
  MIRA_ERR_UNSUPPORTED = -6 /* valid request the library does not implement */
} mira_status;

/* ---- element types ------------------------------------------------------ */
typedef enum mira_dtype {
  MIRA_F32 = 0,  /* IEEE binary32 */
  MIRA_BF16 = 1  /* bfloat16 (upper half of a binary32) */
} mira_dtype;

/* ---- flags of mira_shape.flags ------------------------------------------ */
/* Combine weights are, by default, a softmax over the k selected router
 * logits (renormalised top-k).  With this flag: softmax over all E logits,
 * keeping the k selected probabilities. */
#define MIRA_FLAG_SOFTMAX_ALL 0x1u
/* Force the small-batch (decode) expert kernels; needs n_tokens <= MIRA_DECODE_MAX_TOKENS. */
#define MIRA_FLAG_FORCE_DECODE 0x2u
/* Force the grouped-GEMM (prefill) expert kernels for any n_tokens. */
#define MIRA_FLAG_FORCE_PREFILL 0x4u

/* Experts are in the INT4 variant format below (4-bit values, one fp16 scale
 * per row and group of 64 columns) instead of the paper's INT8 format.  INT4
 * layers run on the decode kernels only: n_tokens must satisfy the decode
 * limits and MIRA_FLAG_FORCE_PREFILL is rejected (MIRA_ERR_UNSUPPORTED).
 * mira_pack_experts reads this bit to choose the format it writes. */
#define MIRA_FLAG_INT4 0x8u

/* Without a FORCE flag, calls with n_tokens <= this use the decode kernels. */
#define MIRA_DECODE_MAX_TOKENS 16

/* Size limits of the library. */
#define MIRA_MAX_EXPERTS 256 /* n_experts + n_shared */
#define MIRA_MAX_TOPK 16

/* ---- packed expert format (section IV-B) --------------------------------
 * One blob per expert, little-endian, at offsets
 *   0       int8  gate [R][C]   (the matrix that goes through SiLU)
 *   R*C     int8  up   [R][C]   (the linear branch)
 *   2*R*C   int8  down [C][R]
 *   3*R*C   bf16  sigma[R]      (one scale per expert-hidden row r, shared by
 *                                gate row r, up row r and down column r)
 * zero-padded to a multiple of 256 bytes.  Each int8 matrix [rows][K] is
 * stored as tiles of 16 rows x 64 columns (1024 bytes), tile-rows in order and
 * column blocks in order inside a tile-row; inside a tile, the 16-byte run
 * number g*16 + i holds row i, columns 16g .. 16g+15.  So element (r, k) is at
 *   ((r/16)*(K/64) + k/64)*1024 + ((k%64)/16*16 + r%16)*16 + k%16.  The dequantized weights are
 * sigma[r] * q.  Pack computes, per row r,
 *   alpha_r = max(|gate[r,:]|_inf, |up[r,:]|_inf, |down[:,r]|_inf)  (exact),
 *   s_r     = fl32(max(alpha_r, eps) / 127),
 *   sigma_r = s_r rounded to bf16 (nearest, ties to even),
 *   q       = clamp(rint_even(fl32(w / sigma_r)), -127, 127),
 * with correctly rounded fp32 division; the integers are made against the
 * stored sigma_r. */

/* Size of one packed expert: 3*R*C + 2*R rounded up to a multiple of 256.
 * Returns 0 if hidden or ffn is not positive or the size overflows. */
size_t mira_packed_expert_bytes(int32_t hidden, int32_t ffn);

/* ---- INT4 variant of the packed expert (MIRA_FLAG_INT4) -----------------
 * The 4-bit, group-64, fp16-scale format (the paper keeps INT8, section IV-B,
 * and lists INT4 as a quality point, Table I).  hidden and ffn must be
 * multiples of 128.  Per matrix [rows][K] (gate [R][C], up [R][C], down
 * [C][R], each with its own scales) and per row and group of 64 consecutive
 * columns:
 *   alpha = max |w| over the group (exact),
 *   s     = fp16 of fl32(max(alpha, eps) / 7), round to nearest even; 2^-24
 *           if that rounds to zero, 65504 if it overflows,
 *   q     = clamp(rint_even(fl32(w / s)), -7, 7),  the weight is s * q.
 * A matrix occupies M(rows, K) = rows*K/2 + rows*(K/64)*2 bytes: a nibble
 * region of rows*K/2 bytes, then a scale region.
 * Nibbles: tiles of 16 rows x 128 columns (two groups) of 1024 bytes, tile-rows
 * in order and column pairs in order inside a tile-row.  Element (r, k) is in
 * the byte at
 *   ((r/16)*(K/128) + k/128)*1024 + ((k%64)/16*16 + r%16)*16
 *     + ((k/64)%2)*8 + ((k%16)/8)*4 + k%4,
 * in its high nibble if k%8 < 4 and in its low nibble otherwise, as the 4-bit
 * two's complement of q.  (So the 16-byte run g*16 + i of a tile holds row i,
 * columns 16g .. 16g+15 of the tile's first group in bytes 0..7 and of its
 * second group in bytes 8..15.)
 * Scales: the little-endian fp16 scale of row r and group k/64 is at
 *   rows*K/2 + ((r/16)*(K/64) + k/64)*32 + (r%16)*2
 * from the start of the matrix (by tile-row, then group, then the 16 rows).
 * The blob holds gate at offset 0, up at M(R, C) and down at 2*M(R, C), then
 * zero padding to a multiple of 256 bytes. */
size_t mira_packed_expert_bytes_int4(int32_t hidden, int32_t ffn);

/* Shape of one MoE layer. */
typedef struct mira_shape {
  int32_t hidden;    /* C: model hidden size; multiple of 64 */
  int32_t ffn;       /* R: expert hidden size; multiple of 64 */
  int32_t n_experts; /* E: routed experts, >= 1 */
  int32_t top_k;     /* k: experts per token, 1 <= k <= min(E, MIRA_MAX_TOPK) */
  int32_t n_shared;  /* S: shared experts applied to every token with weight 1, >= 0 */
  int32_t act_dtype; /* mira_dtype of x and of the router weights */
  uint32_t flags;    /* MIRA_FLAG_* */
  int32_t reserved;  /* must be 0 */
} mira_shape;

/* Offline packing of experts into the format above (section IV-B; the
 * paper converts all expert weights offline).
 *   w_gate, w_up: [n_experts][R][C]; w_down: [n_experts][C][R]; element type
 *     w_dtype (MIRA_F32 or MIRA_BF16; bf16 is widened exactly), finite values.
 *   packed: [n_experts][packed_stride] bytes; packed_stride is a multiple of
 *     256 and >= mira_packed_expert_bytes(C, R).  Padding bytes are zeroed.
 *   eps: the paper's small constant (positive, finite), e.g. 1e-8.
 *   on_device = 0: host pointers; runs on host threads and returns when done
 *     (stream ignored).  on_device = 1: device pointers; enqueued on stream.
 * Both paths produce identical bytes.  Only s->hidden, s->ffn and the
 * MIRA_FLAG_INT4 bit of s->flags are read; with that bit the experts are
 * written in the INT4 variant and packed_stride must be a multiple of 256 and
 * >= mira_packed_expert_bytes_int4(C, R). */
int mira_pack_experts(const mira_shape* s, int32_t n_experts, int32_t w_dtype,
                      const void* w_gate, const void* w_up, const void* w_down,
                      float eps, void* packed, uint64_t packed_stride,
                      int32_t on_device, hipStream_t stream);

/* Arguments of one MoE-layer call; all pointers are device pointers. */
typedef struct mira_moe_args {
  const void* x;             /* [T][C] act_dtype, 16-byte aligned */
  int32_t n_tokens;          /* T >= 0 (T = 0 is a no-op) */
  int32_t n_slots;           /* number of slots in slot_pool */
  const void* w_router;      /* [E][C] act_dtype, 16-byte aligned */
  const float* router_bias;  /* [E] fp32, or NULL for no bias */
  const int32_t* slot_table; /* [E+S]: slot holding each expert (routed
                                experts first, then shared), or -1 when the
                                expert is not resident */
  const void* slot_pool;     /* n_slots * slot_stride bytes of packed experts */
  uint64_t slot_stride;      /* multiple of 256, >= mira_packed_expert_bytes(C, R)
                                (mira_packed_expert_bytes_int4 with MIRA_FLAG_INT4) */
  float* out;                /* [T][C] fp32: sum_j w[t,j] * expert_{idx[t,j]}(x_t)
                                plus the shared experts' outputs */
  int32_t* topk_idx;         /* optional [T][k]: selected experts, best first */
  float* topk_weight;        /* optional [T][k]: their combine weights */
  float* logits;             /* optional [T][E]: fp32 router logits */
  int32_t* expert_counts;    /* optional [E+S]: tokens routed to each expert */
  int32_t* status;           /* optional single int32, set by the kernels:
                                bit 0 = a selected expert had slot -1 (its
                                contribution is missing from out),
                                bit 1 = a slot index was >= n_slots (ignored) */
  int32_t* expert_offsets;   /* optional [E+S+1]: start of each expert's group in
                                the permuted pair order (exclusive scan of counts) */
  int32_t* pair_order;       /* optional [T*k + S*T]: pair_order[pos] = pair at
                                position pos of the permuted order; routed pair
                                t*k+j, shared pair T*k + s*T + t; groups follow
                                expert order, pairs inside a group increase */
  void* workspace;           /* mira_workspace_bytes(s, max_tokens) bytes, 256-byte aligned */
  uint64_t workspace_bytes;
} mira_moe_args;

/* Bytes of workspace needed by calls with up to max_tokens tokens (both
 * paths): the pre-allocated working buffers of the expert step (section
 * IV-F allocates its working buffers once, outside the per-layer path).  They
 * hold the router logits, the routing and permutation, the activations'
 * operand forms and the intermediate H' and expert outputs; nothing in them
 * outlives a call.  Returns 0 for an invalid shape or a negative max_tokens. */
size_t mira_workspace_bytes(const mira_shape* s, int32_t max_tokens);

/* One MoE layer (section II-A; expert step of sections IV-A, IV-F):
 * router logits l = x Wg^T + b (fp32 accumulate), top-k (value descending,
 * lower index on ties), combine weights, stable grouping of (token, slot)
 * pairs by expert, SwiGLU expert FFN on the packed experts fetched through
 * slot_table, weighted combine into out.  Reads status-free inputs only;
 * writes out and the optional outputs.  Deterministic: repeated calls on the
 * same inputs give bit-identical results.
 * Arithmetic: with n_tokens <= MIRA_DECODE_MAX_TOKENS (or MIRA_FLAG_FORCE_DECODE)
 * the experts run on int8 matrix cores with the packed bytes as one operand
 * and the activations as fixed-point digits as the other, so the sums are
 * exact integers and the rounding is that of the fixed points: x at 2^-22 of
 * each token's maximum, H' at 2^-22 of the maximum of its 16-row tile for a
 * one-token call, of its 64-row block for 2 to 5 tokens, and 2^-14 of its
 * 64-row block above.  Otherwise (or with
 * MIRA_FLAG_FORCE_PREFILL) the int8 weights are widened exactly to bf16 for
 * bf16 matrix cores with fp32 accumulation and H' is held in bf16; with fp32
 * activations x and H' are each carried as a high and a low bf16 part and
 * both GEMMs run their contraction over both parts (twice the matrix work),
 * so the result is near fp32 rather than bf16 accuracy.  Both paths take the
 * same routing. */
int mira_moe_forward(const mira_shape* s, const mira_moe_args* a, hipStream_t stream);

/* The same call split in two so a runtime can fetch missing experts in
 * between: mira_moe_route runs the router, top-k and permutation (writing the
 * routing into the workspace and the optional outputs); mira_moe_experts then
 * runs the expert FFN and combine for that routing.  Both calls must get the
 * same shape, tokens and workspace; slot_table may change in between. */
int mira_moe_route(const mira_shape* s, const mira_moe_args* a, hipStream_t stream);
int mira_moe_experts(const mira_shape* s, const mira_moe_args* a, hipStream_t stream);

/* ---- the layer call without a workspace ----------------------------------
 * For callers that cannot allocate device memory (code under HIP graph
 * capture, tight serving loops, harnesses that forbid hipMalloc): the same
 * call as mira_moe_forward, with the library's own scratch array of
 * MIRA_NOALLOC_SCRATCH_BYTES per device in place of the workspace.  It makes
 * no allocation of any kind.  a->workspace must be NULL and
 * a->workspace_bytes 0; every other argument, output and check is that of
 * mira_moe_forward.  A call whose workspace need, mira_workspace_bytes(s,
 * n_tokens), exceeds the scratch size fails with MIRA_ERR_WORKSPACE before
 * any launch (16 MiB covers every decode call of up to 16 tokens at hidden
 * 4096 and ffn 14336, and prefill calls of up to 64 such tokens).  All calls
 * on one device share its scratch: calls that overlap in time on one device
 * (on different streams, or from different threads) race on it and give
 * undefined results; calls ordered on one stream are safe.  The scratch is
 * held until the process ends. */
#define MIRA_NOALLOC_SCRATCH_BYTES (16u << 20)
int mira_moe_forward_noalloc(const mira_shape* s, const mira_moe_args* a, hipStream_t stream);

/* ---- predictor head (section IV-E) -------------------------------------- */
typedef struct mira_pred_shape {
  int32_t hidden;      /* C; multiple of 64 */
  int32_t pred_hidden; /* P: hidden width of the MLP, >= 1 */
  int32_t n_out;       /* experts scored for layer l+2, 1..MIRA_MAX_EXPERTS */
  int32_t group;       /* token rows mean-pooled per evaluation, >= 1 */
  int32_t act_dtype;   /* mira_dtype of x */
  int32_t reserved;    /* must be 0 */
} mira_pred_shape;

/* Bytes of workspace mira_predict needs for n_tokens tokens. */
size_t mira_predict_workspace_bytes(const mira_pred_shape* p, int32_t n_tokens);

/* Scores of layer l+2's experts from layer l's hidden states:
 *   f_i = mean of rows [i*group, (i+1)*group) of x,
 *   z   = ReLU(W1 f_i + b1),  scores[i] = sigmoid(W2 z + b2),
 * fp32 accumulation.  x [T][C] (act_dtype), T a multiple of group;
 * w1 [P][C] bf16, 16-byte aligned; b1 [P] fp32 or NULL; w2 [n_out][P] bf16; b2 [n_out] fp32 or
 * NULL; scores [T/group][n_out] fp32.  All device pointers. */
int mira_predict(const mira_pred_shape* p, const void* x, int32_t n_tokens,
                 const void* w1, const float* b1, const void* w2, const float* b2,
                 float* scores, void* workspace, uint64_t workspace_bytes,
                 hipStream_t stream);

/* ---- MixtureHead predictor (section IV-E) ------------------------------- */
/* The paper's predictor head: an ActHead over the semantic context and the
 * router logits and a HistHead over the expert-selection history, each giving
 * logits over the experts of layer l+2, mixed by a contextual gate alpha.  The
 * paper names the parts, not their sizes; the widths below are parameters. */
typedef struct mira_mixture_shape {
  int32_t hidden;      /* C: multiple of 64 */
  int32_t n_src;       /* E: experts of the source layer l, 1..MIRA_MAX_EXPERTS */
  int32_t top_k;       /* k: columns of topk_idx, 1..MIRA_MAX_TOPK */
  int32_t hist_top;    /* m: most-loaded experts flagged in the top-m feature, 1..n_src */
  int32_t act_hidden;  /* Pa: hidden width of the ActHead, >= 1 */
  int32_t hist_hidden; /* Ph: hidden width of the HistHead, >= 1 */
  int32_t n_out;       /* N: experts of layer l+2, 1..MIRA_MAX_EXPERTS */
  int32_t group;       /* token rows per prediction, >= 1 */
  int32_t act_dtype;   /* mira_dtype of x */
  int32_t reserved;    /* must be 0 */
} mira_mixture_shape;

/* Weights of one MixtureHead, device pointers.  Matrices and gate vectors are
 * bf16, row-major; biases are fp32 and may be NULL (zero).  wah and gh must be
 * 16-byte aligned. */
typedef struct mira_mixture_weights {
  const void* wah;  /* [Pa][C]  ActHead layer 1, pooled hidden part */
  const void* wal;  /* [Pa][E]  ActHead layer 1, mean router-logit part */
  const float* ba1; /* [Pa] */
  const void* wa2;  /* [N][Pa]  ActHead output layer */
  const float* ba2; /* [N] */
  const void* whq;  /* [Ph][E]  HistHead layer 1, selection-histogram part */
  const void* whu;  /* [Ph][E]  HistHead layer 1, top-m indicator part */
  const float* bh1; /* [Ph] */
  const void* wh2;  /* [N][Ph]  HistHead output layer */
  const float* bh2; /* [N] */
  const void* gh;   /* [C]  gate weights on the pooled hidden */
  const void* gl;   /* [E]  ... on the mean router logits */
  const void* gq;   /* [E]  ... on the selection histogram */
  const void* gu;   /* [E]  ... on the top-m indicator */
  float bg;         /* gate bias */
  int32_t reserved; /* must be 0 */
} mira_mixture_weights;

/* Bytes of workspace mira_predict_mixture needs for n_tokens tokens. */
size_t mira_mixture_workspace_bytes(const mira_mixture_shape* p, int32_t n_tokens);

/* Distribution over layer l+2's experts for each group i of `group` token rows
 * of layer l (rows [i*group, (i+1)*group)):
 *   h = mean hidden row, l = mean router-logit row,
 *   q[e] = (pairs of the group routed to e) / (group * k),
 *   u[e] = 1 for the m experts with the most routed pairs (count descending,
 *          index ascending) whose count is positive, else 0,
 *   a = wa2 ReLU(wah h + wal l + ba1) + ba2        (ActHead logits)
 *   b = wh2 ReLU(whq q + whu u + bh1) + bh2        (HistHead logits)
 *   alpha = sigmoid(gh.h + gl.l + gq.q + gu.u + bg) (contextual gate)
 *   probs[i] = softmax(alpha a + (1 - alpha) b),
 * fp32 accumulation.  x [T][C] (act_dtype, 16-byte aligned); logits [T][E]
 * fp32 and topk_idx [T][k] as written by mira_moe_forward for layer l; entries
 * of topk_idx outside 0..E-1 are not counted.  probs [T/group][N] fp32;
 * alpha [T/group] fp32 or NULL.  T must be a multiple of group. */
int mira_predict_mixture(const mira_mixture_shape* p, const mira_mixture_weights* w,
                         const void* x, const float* logits, const int32_t* topk_idx,
                         int32_t n_tokens, float* probs, float* alpha, void* workspace,
                         uint64_t workspace_bytes, hipStream_t stream);

/* ---- expert staging (sections IV-C, IV-E, IV-F) ------------------------- */
/* Copy one packed expert from pinned host memory into slot `slot` of a slot
 * pool with hipMemcpyAsync on copy_stream, then record `done` (if not NULL)
 * on copy_stream.  bytes <= slot_stride; pinned_src must be page-locked host
 * memory.  The caller makes the compute stream wait on `done` before any
 * kernel reads the slot. */
int mira_stage_expert(void* slot_pool, uint64_t slot_stride, int32_t slot,
                      const void* pinned_src, uint64_t bytes,
                      hipStream_t copy_stream, hipEvent_t done);

/* Write slot_table[expert] = slot with a one-thread kernel on `stream`
 * (stream-ordered, so a later forward call on the stream sees it). */
int mira_set_slot(int32_t* slot_table, int32_t expert, int32_t slot, hipStream_t stream);

/* ---- expert cache runtime (sections IV-C, IV-D, IV-E, IV-F) --------------
 * The HOT and STAGE regions of the GPU expert cache over one slot pool shared
 * by the L layers of a model, the lookahead-2 prefetch controller driven by a
 * predictor head, demand fetches of missing experts, per-expert telemetry and
 * the bounded HOT rebalancer.  A decode step calls mira_stack_begin_step, then
 * mira_stack_layer for layers 0..L-1 in order, then mira_stack_end_step.
 *
 * One mira_stack_layer call, for layer l, on the stack's compute stream:
 *  1. mira_moe_route for layer l; the tokens routed to each expert are read
 *     back to the host (the call waits for that copy: the host decides which
 *     experts to fetch);
 *  2. each selected expert is served from its HOT slot, from a STAGE slot
 *     filled earlier (the compute stream waits for that copy's event only),
 *     or by a demand copy from its CPU-store blob into a free STAGE slot (a
 *     miss); the layer's slot-table row is written in stream order;
 *  3. mira_moe_experts for layer l;
 *  4. prefetch for layer l + lookahead: the head's stage_per_layer best
 *     experts (scores summed over the call's token groups, ties to the lower
 *     index; the head runs on a side stream right after step 1, beside the
 *     experts), or a given list.  An expert already in HOT or STAGE is a
 *     skipped prefetch ("cached"), an (expert, layer) pair already staged is
 *     not copied twice, a prefetch finding no free STAGE slot is declined;
 *  5. when the layer's telemetry window holds rb_interval tokens, the
 *     rebalancer swaps at most rb_max_swaps HOT experts for candidates (a
 *     candidate held in a STAGE slot is relabelled HOT, otherwise it is
 *     copied from the CPU store into the victim's slot).
 * A STAGE slot may be taken by a copy when it is free or its layer has passed
 * in the current step (oldest first); a demand copy may also take the oldest
 * prefetch for a later layer, never a slot of the current layer.  Small-VRAM
 * mode frees a layer's STAGE slots right after its experts ran; large-VRAM
 * mode keeps them (a later step may hit them) until a copy needs the slot.
 * Every copy runs on the stack's copy stream (default priority) and waits
 * only for the last kernel that read its slot.
 *
 * Memory: the caller owns the slot pool, the slot tables and every CPU-store
 * blob (page-locked host memory) and keeps them alive until
 * mira_stack_destroy; the stack allocates its streams, events and small
 * pinned and device buffers in mira_stack_create and nothing afterwards.  A
 * stack is used from one host thread at a time. */
typedef struct mira_stack mira_stack; /* opaque */

#define MIRA_VRAM_LARGE 0
#define MIRA_VRAM_SMALL 1

typedef struct mira_stack_config {
  int32_t n_layers;        /* L >= 1 */
  int32_t n_hot;           /* slots [0, n_hot) of the pool are HOT */
  int32_t n_stage;         /* slots [n_hot, n_hot + n_stage) are STAGE, >= 0 */
  int32_t max_tokens;      /* most tokens of one mira_stack_layer call, >= 1 */
  uint64_t slot_stride;    /* bytes between slots, a multiple of 256 */
  int32_t vram_mode;       /* MIRA_VRAM_LARGE or MIRA_VRAM_SMALL */
  int32_t lookahead;       /* the layer staged ahead is l + lookahead (the paper: 2), >= 1 */
  int32_t stage_per_layer; /* m: experts the head picks per staged layer, >= 1 */
  int32_t rb_interval;     /* tokens of a layer between rebalancing passes; 0 = no rebalancing */
  int32_t rb_max_swaps;    /* swaps per layer and pass */
  int32_t rb_probation;    /* consecutive windows with traffic before a promotion, >= 1 */
  int32_t rb_margin;       /* a candidate must beat the victim's window volume by this much */
  float rb_miss_weight;    /* candidate score = routed + miss_weight * CPU-served tokens */
} mira_stack_config;

/* Counters of the steps since the last mira_stack_end_step (times in ms). */
typedef struct mira_stack_stats {
  int64_t hot_hits, stage_hits, misses;          /* selected experts by where they were served */
  int64_t hot_tokens, stage_tokens, cpu_tokens;  /* routed (token, expert) pairs by tier */
  int64_t prefetches, prefetch_cached, prefetch_declined;
  int64_t swaps, promote_copies;                 /* rebalancing swaps; those that copied */
  int64_t h2d_bytes;                             /* bytes copied host -> device */
  int64_t cov_hits, cov_total;                   /* Coverage@m: routed pairs of a predicted layer
                                                    on its predicted experts / all its routed pairs */
  double copy_ms;                                /* summed durations of the copies */
  double stall_ms;                               /* time the compute stream waited for copies */
  double wall_ms;                                /* compute stream, begin to end of the steps */
} mira_stack_stats;

/* Predictor of layer l + lookahead used by one mira_stack_layer call. */
#define MIRA_HEAD_NONE 0    /* no prefetch */
#define MIRA_HEAD_MLP 1     /* mira_predict with mlp_shape and w1, b1, w2, b2 */
#define MIRA_HEAD_MIXTURE 2 /* mira_predict_mixture with mix_shape and mix (needs the layer's
                               logits and topk_idx outputs in the layer's args) */
#define MIRA_HEAD_GIVEN 3   /* stage exactly given[0..n_given) (host array), e.g. the true
                               experts of the target layer as an upper bound */
typedef struct mira_stack_head {
  int32_t kind;
  int32_t n_given;
  const int32_t* given;
  const mira_pred_shape* mlp_shape;
  const void* w1;
  const float* b1;
  const void* w2;
  const float* b2;
  const mira_mixture_shape* mix_shape;
  const mira_mixture_weights* mix;
  void* workspace; /* the head's device workspace and its size */
  uint64_t workspace_bytes;
} mira_stack_head;

/* One entry of the stack's event log (kinds below). */
#define MIRA_EV_HOT_HIT 0
#define MIRA_EV_STAGE_HIT 1
#define MIRA_EV_DEMAND 2       /* a miss: copy from the CPU store */
#define MIRA_EV_PREDICTED 3    /* the head chose (target, expert) */
#define MIRA_EV_PREFETCH 4     /* copy issued for (target, expert) */
#define MIRA_EV_PREFETCH_CACHED 5
#define MIRA_EV_PREFETCH_DECLINED 6
#define MIRA_EV_PREFETCH_DROPPED 7 /* a staged prefetch gave its slot to a demand copy */
#define MIRA_EV_SWAP_RELABEL 8     /* expert promoted to HOT from its STAGE slot */
#define MIRA_EV_SWAP_COPY 9        /* expert promoted to HOT by a copy into the victim's slot */
#define MIRA_EV_EVICT 10           /* expert evicted from HOT */
typedef struct mira_stack_event {
  int32_t kind;
  int32_t layer;  /* the layer being run when the event happened */
  int32_t target; /* the layer the expert belongs to */
  int32_t expert;
  int32_t slot;   /* -1 if none */
  int32_t reserved;
} mira_stack_event;

/* Create a stack over a caller-owned pool of n_hot + n_stage slots and the
 * device slot tables [L][E+S] (int32; written only by the stack).  s gives
 * the layers' shape (all layers share it).  compute is the stream every
 * layer runs on.  On success *out holds the stack. */
int mira_stack_create(const mira_stack_config* cfg, const mira_shape* s, void* slot_pool,
                      int32_t* slot_tables, hipStream_t compute, mira_stack** out);
int mira_stack_destroy(mira_stack* st);

/* The CPU-store blob of expert e of layer l: `bytes` (<= slot_stride) bytes
 * of page-locked host memory holding the packed expert. */
int mira_stack_set_host(mira_stack* st, int32_t layer, int32_t expert, const void* pinned,
                        uint64_t bytes);
/* Make HOT slot `slot` hold expert e of layer l.  The HOT slots are the
 * first n_hot slots of the pool until a rebalancing swap relabels a STAGE
 * slot HOT and the victim's slot STAGE; a slot that is not HOT at the call is
 * rejected (MIRA_ERR_ARG).  With copy = 1 the expert's CPU-store blob is
 * copied in (copy stream); with copy = 0 the caller has written the slot's
 * bytes already. */
int mira_stack_set_hot(mira_stack* st, int32_t layer, int32_t expert, int32_t slot, int32_t copy);

int mira_stack_begin_step(mira_stack* st);
/* Run layer l (see above).  a carries the layer's inputs, outputs and
 * workspace; its slot_table, slot_pool, n_slots and slot_stride are taken
 * from the stack, and a NULL expert_counts is replaced by the stack's own
 * buffer.  head (may be NULL = MIRA_HEAD_NONE) picks layer l + lookahead's
 * experts to stage.  An error after step 1 leaves part of the layer's work
 * queued (copies issued, counters updated): end the step, call
 * mira_stack_reset_stage and start a new step. */
int mira_stack_layer(mira_stack* st, int32_t layer, const mira_moe_args* a,
                     const mira_stack_head* head);
/* Wait for the step's work and add its counters (times included) to *stats
 * (may be NULL). */
int mira_stack_end_step(mira_stack* st, mira_stack_stats* stats);
/* Free every STAGE slot (waits for the stack's queued work first). */
int mira_stack_reset_stage(mira_stack* st);
/* Slot holding expert e of layer l as HOT (role 0) or STAGE (role 1), or -1. */
int32_t mira_stack_find(const mira_stack* st, int32_t layer, int32_t expert, int32_t role);
/* Move up to max_events logged events (oldest first) to events; *n_events
 * gets the count.  The log keeps the last 65536 events. */
int mira_stack_read_events(mira_stack* st, int32_t max_events, mira_stack_event* events,
                           int32_t* n_events);

/* The rebalancer's decision for one layer (section IV-D), as the stack runs
 * it, on the host: per expert the tokens routed in the current window and of
 * those served by a CPU copy, the token clock of its last use (-1 = never),
 * the routed volumes of up to 8 past windows (hist_len of them, oldest
 * first, in history[e*8 ...]) and whether it is HOT.  Victims: HOT experts
 * ordered by (routed, last_use, sum of history, index) ascending.
 * Candidates: non-HOT experts with routed > 0 whose last probation-1 windows
 * all had traffic, ordered by score routed + miss_weight * cpu descending,
 * then index.  The i-th victim and candidate swap while fewer than max_swaps
 * swaps are planned and score >= victim's routed + margin.  Writes
 * evict[i], promote[i] for i < *n_swaps. */
int mira_rebalance_plan(const mira_stack_config* cfg, int32_t n_experts, const int32_t* routed,
                        const int32_t* cpu, const int64_t* last_use, const int32_t* history,
                        const int32_t* hist_len, const uint8_t* is_hot, int32_t max_swaps_out,
                        int32_t* evict, int32_t* promote, int32_t* n_swaps);

/* ---- diagnostics -------------------------------------------------------- */
/* Description of the last failure on this thread ("" if none). */
const char* mira_last_error(void);

/* Library version string. */
const char* mira_version(void);

/* Kernel timing for measurement.  While enabled, every kernel the library
 * launches is bracketed by a pair of HIP events recorded on its stream;
 * mira_profile_read synchronises on them and reports, per kernel name, the
 * launch count and the summed duration in milliseconds, then clears the
 * records.  Names are library-owned strings. */
int mira_profile_enable(int32_t enable);
/* Restrict the timing to kernels of one name (NULL or "" = all kernels), so
 * that only the kernel under study carries event records. */
int mira_profile_select(const char* kernel_name);
int mira_profile_read(int32_t max_entries, const char** names, int32_t* counts,
                      double* total_ms, int32_t* n_entries);

#ifdef __cplusplus
}
#endif

#endif /* MIRA_H_ */
