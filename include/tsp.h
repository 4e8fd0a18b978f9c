/*
 * tsp.h -- C ABI of libtsp: the per-rank forward of a folded Tensor-and-Sequence
 * Parallel (TSP) transformer layer on one AMD Instinct MI355X (gfx950).
 *
 * Paper: "Folding Tensor and Sequence Parallelism for Memory-Efficient Transformer
 * Training & Inference" (arXiv 2604.26294).  A TSP group of D ranks shards both the
 * sequence and the layer weights over one device axis: rank p holds S/D tokens and,
 * over D steps, applies every weight shard to them.  The tokens of rank p are
 *   layout 0 (contiguous): positions [p*S_loc, (p+1)*S_loc), S_loc = S/D;
 *   layout 1 (zigzag, Algorithm 1 as printed): with S_c = S_loc/2, chunk p followed by
 *     chunk 2D-1-p, i.e. local row t < S_c at position p*S_c + t and local row
 *     t >= S_c at position (2D-1-p)*S_c + (t - S_c).
 * "The position of local row t" below means this mapping.
 *
 *   - Attention (Algorithm 1): for r = 0..D-1 the rank projects Q, K, V of its chunk
 *     with shard r, attends causally against the full-sequence K/V of shard r (the
 *     sequence-wise all-gather), and accumulates Flatten(A) W_O^(r)^T.
 *   - Gated MLP (Algorithm 2): for t = 0..D-1 the rank applies the shard that started
 *     on rank (p - t) mod D (ring order) and accumulates (SiLU(X W1^T) * X W3^T) W2.
 *   - Layer (Section 4 model: pre-norm residual block, norms left out):
 *     u = x + Attn(x), y = u + MLP(u).
 *
 * On one GPU the exchanges are modelled by resident buffers: every weight shard is
 * already in device memory (the broadcast / ring hand-off has happened), and the
 * K/V buffer holds the full sequence in sequence order (the all-gather, reordered).
 * Each attention call WRITES the K/V rows at its own tokens' positions for every shard
 * and READS the keys its queries can see: [0, (p+1)*S_loc) for layout 0,
 * [0, (2D-p)*S_c) for layout 1; the other ranks' rows are the caller's (see
 * tsp_kv_rank_fwd).
 *
 * Conventions shared by every entry point
 *   - All tensor arguments are DEVICE pointers to dense row-major arrays.  bf16
 *     values are passed as their 16-bit patterns (uint16_t).  fp32 is float.
 *   - Arrays of D shard pointers ("w_gate", "w_attn", ...) are HOST arrays whose
 *     elements are device pointers, one per shard, indexed by shard number.
 *   - Every device pointer must be 16-byte aligned.
 *   - The caller owns every buffer.  The library never allocates or frees device
 *     memory and keeps no state between calls (apart from the opt-in kernel timing
 *     records of tsp_profile_enable, the per-thread code of the last HIP failure and
 *     the fixed scratch array of tsp_layer_rank_fwd_noalloc); scratch space is the
 *     caller's workspace, sized by tsp_workspace_bytes (tsp_layer_rank_fwd_noalloc
 *     excepted).
 *   - Calls only enqueue work on `stream` (NULL = the default stream) and never
 *     synchronise.  Calls on different streams must use different workspaces and
 *     must not write the same outputs.
 *   - All validation happens on the host, before anything is enqueued; a call that
 *     returns an error has enqueued nothing.  TSP_ERR_HIP reports a failed launch
 *     (work enqueued before the failure may still run); tsp_last_hip_error names
 *     the HIP error.
 *   - Results are deterministic: no atomics, fixed reduction orders.
 *   - Supported: head_dim in {64, 128}; hidden, ffn/degree and head_dim multiples
 *     of 8; layout 0 or 1 (layout 1 needs S divisible by 2D, else TSP_ERR_SHAPE).
 *     Anything else valid returns TSP_ERR_UNSUPPORTED.
 */
#ifndef TSP_H
#define TSP_H

#include <stddef.h>
#include <stdint.h>

#include <hip/hip_runtime_api.h>

#ifdef __cplusplus
extern "C" {
#endif

#define TSP_ABI_VERSION 2

typedef enum tsp_status {
  TSP_OK = 0,
  TSP_ERR_NULL = 1,        /* a required pointer (shape, tensor, shard, workspace) is NULL */
  TSP_ERR_SHAPE = 2,       /* dimensions are non-positive or inconsistent (see below) */
  TSP_ERR_RANK = 3,        /* rank outside [0, degree) */
  TSP_ERR_ALIGN = 4,       /* a device pointer is not 16-byte aligned */
  TSP_ERR_WORKSPACE = 5,   /* ws_bytes is smaller than tsp_workspace_bytes() */
  TSP_ERR_UNSUPPORTED = 6, /* valid shape the kernels do not implement */
  TSP_ERR_HIP = 7          /* a kernel launch failed */
} tsp_status;

/* Problem statement of one rank (paper notation, Section 4 notation table).
 * Shape rules (TSP_ERR_SHAPE otherwise): batch >= 0, seq >= 0, every other size >= 1;
 * seq % degree == 0; hidden == n_heads * head_dim; n_heads % n_kv_heads == 0;
 * n_heads % degree == 0; n_kv_heads % degree == 0; ffn % degree == 0.
 * Size limit (TSP_ERR_UNSUPPORTED otherwise): the rank's widest per-token operand,
 * batch * seq / degree rows of max(hidden, ffn, G * (ffn / degree rounded up to 64))
 * bf16 values (G the forward grouping below), is smaller than 4 GiB. */
typedef struct tsp_shape {
  int32_t batch;        /* B: micro-batch */
  int32_t seq;          /* S: full sequence length; each rank holds S_loc = S / D tokens */
  int32_t hidden;       /* h: model width */
  int32_t ffn;          /* MLP intermediate width (the paper's F*h); shards hold ffn / D rows */
  int32_t n_heads;      /* n_h: query heads; shard r holds heads [r*n_h/D, (r+1)*n_h/D) */
  int32_t n_kv_heads;   /* n_kv: key/value heads (GQA ratio g = n_h / n_kv); query head i
                           reads kv head i / g */
  int32_t head_dim;     /* d */
  int32_t degree;       /* D: TSP degree (number of shards) */
  int32_t rank;         /* p: this rank */
  int32_t layout;       /* 0 = contiguous chunks, 1 = zigzag (see the top of this file) */
  float softmax_scale;  /* <= 0 selects 1/sqrt(head_dim) */
  int32_t group_steps;  /* forward shard steps per grouped launch, 0..TSP_GROUP_STEPS_MAX
                           (0 = TSP_GROUP_STEPS_MAX; values above D act as D; negative:
                           TSP_ERR_SHAPE, above the maximum: TSP_ERR_UNSUPPORTED) */
} tsp_shape;

/* Forward shard-step grouping.  tsp_mlp_rank_fwd, tsp_attn_rank_fwd and the layer calls
 * take their D shard steps in groups of G = min(group_steps, D) consecutive steps of
 * the schedule's order (the last group holds the remainder).  A group's products run as
 * one launch each: its gate+up (Q/K/V) products as one grouped launch, its down (output)
 * projection as ONE product whose contraction runs over the group's shards in order
 * (Y += [Hs_1 .. Hs_G] [W_down_1; ..; W_down_G]), and its attention over the group's
 * G n_h/D heads at once.  The result is the step-by-step sum up to fp32 rounding order.
 * In a streaming schedule G is the number of weight shards held at once; with every
 * shard resident (one GPU) the default takes all D steps together (D <= the maximum).
 * The backward calls take their steps one (or two) at a time and ignore it. */
#define TSP_GROUP_STEPS_MAX 8

/* Gated ring MLP of rank p (Algorithm 2):
 *   Y (+)= sum over t = 0..D-1, j = (p - t) mod D, of
 *          bf16( SiLU(X W_gate[j]^T) * (X W_up[j]^T) ) W_down[j]
 * with SiLU(z) = z * sigmoid(z), fp32 accumulation across shards in ring order, the
 * steps grouped as tsp_shape.group_steps says (the down projections of a group's
 * steps one product over its shards): the same sum up to fp32 rounding order.
 *   x_loc      [B, S_loc, h] bf16       the rank's tokens
 *   w_gate[j]  [ffn/D, h]   bf16       W1 shard j
 *   w_up[j]    [ffn/D, h]   bf16       W3 shard j
 *   w_down[j]  [ffn/D, h]   bf16       W2 shard j, applied untransposed
 *   y_loc      [B, S_loc, h] fp32      accumulate == 0: overwritten; != 0: added to
 *   ws         workspace of at least tsp_workspace_bytes(shape, TSP_OP_MLP) bytes */
tsp_status tsp_mlp_rank_fwd(const tsp_shape* shape, const uint16_t* x_loc,
                            const uint16_t* const* w_gate, const uint16_t* const* w_up,
                            const uint16_t* const* w_down, float* y_loc, int accumulate,
                            void* ws, size_t ws_bytes, hipStream_t stream);

/* Backward of tsp_mlp_rank_fwd on rank p.  The paper costs TSP's backward (Section 4:
 * it mirrors the forward weight movement, and each weight shard's partial gradients
 * are summed to the rank that owns the shard) without printing an algorithm; these
 * are the chain-rule gradients of Algorithm 2, shards visited in the same ring order.
 * For each j, with G = X W_gate[j]^T, U = X W_up[j]^T recomputed, s = SiLU(G),
 * s' = sigmoid(G) (1 + G (1 - sigmoid(G))), Hs = s * U:
 *   dHs = dY W_down[j]^T;   dG = dHs * U * s';   dU = dHs * s
 *   dX (+)= dG W_gate[j] + dU W_up[j]                     (fp32, ring order)
 *   dw_gate[j] (+)= dG^T X;  dw_up[j] (+)= dU^T X;  dw_down[j] (+)= Hs^T dY
 * The dw outputs are this rank's contributions; summing them over the D ranks (the
 * sum-to-owner reduction, a collective outside this single-GPU library) gives the
 * gradients of the shards.  dG, dU and Hs are rounded to bf16 for the matrix cores.
 *   x_loc, w_gate, w_up, w_down  as for tsp_mlp_rank_fwd
 *   dy_loc     [B, S_loc, h] bf16       gradient of the MLP output for these tokens
 *   dx_loc     [B, S_loc, h] fp32       accumulate == 0: overwritten; != 0: added to
 *   dw_gate[j], dw_up[j], dw_down[j]  [ffn/D, h] fp32 (host arrays of D device
 *              pointers)                 overwritten or added to, as dx_loc
 *   ws         workspace of at least tsp_workspace_bytes(shape, TSP_OP_MLP_BWD) bytes */
tsp_status tsp_mlp_rank_bwd(const tsp_shape* shape, const uint16_t* x_loc,
                            const uint16_t* dy_loc, const uint16_t* const* w_gate,
                            const uint16_t* const* w_up, const uint16_t* const* w_down,
                            float* dx_loc, int accumulate, float* const* dw_gate,
                            float* const* dw_up, float* const* dw_down, void* ws,
                            size_t ws_bytes, hipStream_t stream);

/* This rank's contribution to the sequence-wise K/V all-gather of every shard
 * (Algorithm 1, the local K and V projections, with ZigZagReorder folded into the
 * addresses): for r = 0..D-1 writes
 *   k_buf[b, pos(t), r*n_kv/D + j, :] = (x_loc[b, t] W_K^(r)^T) head j, bf16
 * with pos(t) the position of local row t, and the same for V.  Used to fill the K/V
 * rows of ranks other than the caller.
 *   x_loc      [B, S_loc, h] bf16
 *   w_attn[r]  packed shard r, [(2*n_h/D + 2*n_kv/D) * d, h] bf16: rows
 *              [W_Q^(r) ; W_K^(r) ; W_V^(r) ; W_O^(r)^T] (the packed broadcast buffer)
 *   k_buf, v_buf [B, S, n_kv, d] bf16   rows at this rank's positions written */
tsp_status tsp_kv_rank_fwd(const tsp_shape* shape, const uint16_t* x_loc,
                           const uint16_t* const* w_attn, uint16_t* k_buf, uint16_t* v_buf,
                           hipStream_t stream);

/* TSP attention of rank p (Algorithm 1): for r = 0..D-1,
 *   Q = X W_Q^(r)^T; K, V rows of this rank written into k_buf / v_buf;
 *   A = causal softmax(Q K^T * scale) V, where local query row t at position pos(t)
 *       sees keys j <= pos(t) (layout 1: the two CausalAttn calls of Algorithm 1, the
 *       first half of the rows against keys [0, s1 = (p+1)*S_c), the second against
 *       [0, s2 = (2D-p)*S_c));
 *   Y (+)= Flatten(A) W_O^(r)^T   (fp32, shards accumulated in order r = 0..D-1,
 *       grouped as tsp_shape.group_steps says: the output projections of a group's
 *       shards one product over them).
 * Q, K, V, the softmax probabilities and A are rounded to bf16 for the matrix cores.
 *   x_loc, w_attn as for tsp_kv_rank_fwd;  k_buf, v_buf [B, S, n_kv, d] bf16: this
 *   rank's rows are written; every other row its queries can see must already hold
 *   the other ranks' K/V; rows past the last visible key are never read.
 *   y_loc [B, S_loc, h] fp32, overwritten (accumulate == 0) or added to. */
tsp_status tsp_attn_rank_fwd(const tsp_shape* shape, const uint16_t* x_loc,
                             const uint16_t* const* w_attn, uint16_t* k_buf, uint16_t* v_buf,
                             float* y_loc, int accumulate, void* ws, size_t ws_bytes,
                             hipStream_t stream);

/* tsp_attn_rank_fwd that also keeps what the backward needs (training): the attention
 * output A of every shard and the log-sum-exp of every query's logits, so that
 * tsp_attn_rank_bwd_saved need not recompute them (the forward in Algorithm 1's order,
 * grouped as tsp_shape.group_steps says; results as tsp_attn_rank_fwd's).
 *   a_out    [B, S_loc, n_h, d] bf16   A of all shards side by side: shard r's heads at
 *                                     columns r*n_h/D*d ..; written
 *   lse_out  [B, n_h, S_loc] fp32      log2 of the softmax denominator of each query's
 *                                     base-2 logits (scale * log2(e) * q k, with q rounded
 *                                     to bf16 as the kernels use it); written
 * Other arguments as tsp_attn_rank_fwd (same workspace size, TSP_OP_ATTN). */
tsp_status tsp_attn_rank_fwd_train(const tsp_shape* shape, const uint16_t* x_loc,
                                   const uint16_t* const* w_attn, uint16_t* k_buf,
                                   uint16_t* v_buf, float* y_loc, int accumulate,
                                   uint16_t* a_out, float* lse_out, void* ws, size_t ws_bytes,
                                   hipStream_t stream);

/* Backward of tsp_attn_rank_fwd on rank p, first stage.  As for the MLP, the paper
 * costs the backward (Section 4) without printing it; these are the chain-rule
 * gradients of Algorithm 1.  The forward's K/V all-gather becomes a reduce-scatter of
 * the K/V gradients, so the backward has two stages: this one produces the rank's
 * contributions to the gradients of every shard's gathered K-hat / V-hat; their sum
 * over ranks, restricted to a rank's own rows (a collective outside this single-GPU
 * library), is the input of tsp_attn_kv_rank_bwd.  For r = 0..D-1:
 *   Q, A recomputed as in the forward (A with the log-sum-exp of every query's logits);
 *   dA = dY W_O^(r);   dw_attn[r] W_O^T block (+)= A^T dY;
 *   per head, with P the causal softmax weights, dP = dA V^T, dS = P * (dP - rowsum(dA * A)):
 *     dQ = scale dS K,   dK-hat (+)= scale dS^T Q,   dV-hat (+)= P^T dA;
 *   dX (+)= dQ W_Q^(r);   dw_attn[r] W_Q block (+)= dQ^T X.
 * Q, A, dA, dQ, P, dS are rounded to bf16 for the matrix cores.
 *   x_loc, w_attn        as for tsp_attn_rank_fwd
 *   dy_loc  [B, S_loc, h] bf16     gradient of the attention block output (Y)
 *   k_buf, v_buf [B, S, n_kv, d] bf16   the gathered K/V as the forward used them
 *                                       (read only; rows past the last visible key unread)
 *   dx_loc  [B, S_loc, h] fp32     the query path of dX: overwritten (accumulate == 0)
 *                                  or added to
 *   dw_attn[r] [(2*n_h/D + 2*n_kv/D) * d, h] fp32, the packed shard's layout (host array
 *              of D device pointers): the W_Q and W_O^T row blocks are overwritten or
 *              added to, as dx_loc; the W_K, W_V blocks are not touched
 *   dk_buf, dv_buf [B, S, n_kv, d] fp32   this rank's contributions for all S rows
 *              (zero where none of its queries sees the key), overwritten or added to
 *   ws      workspace of at least tsp_workspace_bytes(shape, TSP_OP_ATTN_BWD) bytes */
tsp_status tsp_attn_rank_bwd(const tsp_shape* shape, const uint16_t* x_loc,
                             const uint16_t* dy_loc, const uint16_t* const* w_attn,
                             const uint16_t* k_buf, const uint16_t* v_buf, float* dx_loc,
                             int accumulate, float* const* dw_attn, float* dk_buf,
                             float* dv_buf, void* ws, size_t ws_bytes, hipStream_t stream);

/* tsp_attn_rank_bwd with A and the log-sum-exp taken from tsp_attn_rank_fwd_train
 * (a_saved, lse_saved in its a_out / lse_out layouts, from the same inputs) instead of
 * recomputed: the same gradients (Q is still recomputed from x, with the forward's single
 * rounding), without the forward attention pass.  Workspace as tsp_attn_rank_bwd
 * (TSP_OP_ATTN_BWD); other arguments as there. */
tsp_status tsp_attn_rank_bwd_saved(const tsp_shape* shape, const uint16_t* x_loc,
                                   const uint16_t* dy_loc, const uint16_t* const* w_attn,
                                   const uint16_t* k_buf, const uint16_t* v_buf,
                                   const uint16_t* a_saved, const float* lse_saved,
                                   float* dx_loc, int accumulate, float* const* dw_attn,
                                   float* dk_buf, float* dv_buf, void* ws, size_t ws_bytes,
                                   hipStream_t stream);

/* Backward of the rank's K/V projections, second stage of the attention backward:
 * with dK, dV the reduce-scattered gradients of this rank's rows of every shard's
 * K-hat / V-hat (K = X W_K^(r)^T, V = X W_V^(r)^T on the rank's own rows), for r = 0..D-1:
 *   dX (+)= dK_r W_K^(r) + dV_r W_V^(r);
 *   dw_attn[r] W_K block (+)= dK_r^T X;   W_V block (+)= dV_r^T X.
 *   x_loc, w_attn      as for tsp_attn_rank_fwd
 *   dk_loc, dv_loc [B, S_loc, n_kv, d] bf16   rows in local order; columns of shard r's
 *                      kv heads r*n_kv/D .. are dK_r, dV_r
 *   dx_loc [B, S_loc, h] fp32   overwritten (accumulate == 0) or added to
 *   dw_attn[r]         as for tsp_attn_rank_bwd; only the W_K, W_V blocks are written
 *   ws      workspace of at least tsp_workspace_bytes(shape, TSP_OP_ATTN_KV_BWD) bytes */
tsp_status tsp_attn_kv_rank_bwd(const tsp_shape* shape, const uint16_t* x_loc,
                                const uint16_t* const* w_attn, const uint16_t* dk_loc,
                                const uint16_t* dv_loc, float* dx_loc, int accumulate,
                                float* const* dw_attn, void* ws, size_t ws_bytes,
                                hipStream_t stream);

/* One rank's layer forward: u = x + Attn(x); y = u + MLP(bf16(u)).
 * Arguments as above; y_loc [B, S_loc, h] fp32 is overwritten with y. */
tsp_status tsp_layer_rank_fwd(const tsp_shape* shape, const uint16_t* x_loc,
                              const uint16_t* const* w_attn, const uint16_t* const* w_gate,
                              const uint16_t* const* w_up, const uint16_t* const* w_down,
                              uint16_t* k_buf, uint16_t* v_buf, float* y_loc, void* ws,
                              size_t ws_bytes, hipStream_t stream);

/* Scratch size available to tsp_layer_rank_fwd_noalloc on each device (128 MiB). */
#define TSP_NOALLOC_SCRATCH_BYTES (128u << 20)

/* tsp_layer_rank_fwd for callers that cannot allocate device memory: code under HIP
 * graph capture, tight serving loops, harnesses that forbid allocation.  Same arguments
 * and results, minus the workspace: the scratch space comes from a fixed array of
 * TSP_NOALLOC_SCRATCH_BYTES per device, part of the library's device code (resident on
 * every device the library has run on, until the process ends), used on the calling
 * thread's current HIP device, which must be the device of `stream`.  The call neither
 * allocates nor frees anything.
 *   - A shape whose layer workspace (tsp_workspace_bytes(shape, TSP_OP_LAYER)) exceeds
 *     TSP_NOALLOC_SCRATCH_BYTES returns TSP_ERR_WORKSPACE before anything is enqueued
 *     (the 7B-class layer at S = 8192, D = 8 needs 94 MiB and fits; at S = 65536 it
 *     needs 240 MiB and does not).
 *   - All calls on one device share its array: calls that can overlap in time on one
 *     device (different streams, or different host threads without ordering) race on
 *     it and must not be made; calls ordered on one stream are fine.
 *   - The array keeps whatever the last call left; no call needs it cleared.
 *   - The first call on a device looks up the array's device address (no kernel). */
tsp_status tsp_layer_rank_fwd_noalloc(const tsp_shape* shape, const uint16_t* x_loc,
                                      const uint16_t* const* w_attn,
                                      const uint16_t* const* w_gate,
                                      const uint16_t* const* w_up,
                                      const uint16_t* const* w_down, uint16_t* k_buf,
                                      uint16_t* v_buf, float* y_loc, hipStream_t stream);

enum {
  TSP_OP_MLP = 0,
  TSP_OP_ATTN = 1,
  TSP_OP_LAYER = 2,
  TSP_OP_MLP_BWD = 3,
  TSP_OP_ATTN_BWD = 4,
  TSP_OP_ATTN_KV_BWD = 5
};

/* Workspace bytes the entry point `op` needs for `shape` (validated as above). */
tsp_status tsp_workspace_bytes(const tsp_shape* shape, int op, size_t* bytes);

/* Per-kernel timing for measurement (not for production use; process-wide state,
 * not thread-safe).  While enabled, every launch of the listed kernel classes is
 * bracketed by a pair of HIP events recorded on the launch stream.  Enabling
 * clears the previous records.  tsp_profile_read waits for the recorded events of
 * one class and returns the summed kernel time and the number of launches. */
enum {
  TSP_KERNEL_GATE_UP = 0, /* gate + up projections with fused SwiGLU (Algorithm 2) */
  TSP_KERNEL_DOWN = 1,    /* down projection + fp32 shard accumulate, two ring steps per
                             launch (Algorithm 2) */
  TSP_KERNEL_QKV = 2,     /* Q/K/V projections with K/V scatter (Algorithm 1) */
  TSP_KERNEL_ATTN = 3,    /* causal flash attention of one shard step (Algorithm 1) */
  TSP_KERNEL_OPROJ = 4,   /* output projection + fp32 shard accumulate, two shards per
                             launch (Algorithm 1) */
  TSP_KERNEL_BWD_GATE = 5, /* MLP backward: G, U, dHs products with the SwiGLU backward */
  TSP_KERNEL_BWD_DX = 6,   /* MLP backward: dX accumulate (dG and dU paths, one launch) */
  TSP_KERNEL_BWD_DW = 7,   /* MLP backward: the three weight-gradient products, one launch */
  TSP_KERNEL_ABWD_PROJ = 8,  /* attention backward: Q and dA = dY W_O products */
  TSP_KERNEL_ABWD_FWD = 9,   /* attention backward: forward recomputation with lse */
  TSP_KERNEL_ABWD_KV = 10,   /* attention backward: dK / dV (key-stationary) */
  TSP_KERNEL_ABWD_Q = 11,    /* attention backward: dQ (query-stationary) */
  TSP_KERNEL_ABWD_DX = 12,   /* attention backward: dX accumulate (both stages) */
  TSP_KERNEL_ABWD_DW = 13,   /* attention backward: weight-gradient products, two per launch */
  TSP_KERNEL_ABWD_AUX = 14,  /* attention backward: delta / scaled-Q prep, transposes */
  TSP_KERNEL_COUNT = 15
};
tsp_status tsp_profile_enable(int enable);
tsp_status tsp_profile_read(int kernel, double* total_ms, int64_t* launches);

/* Test hook for the failure path of the attention kernels' tile hand-over (the forward
 * of tsp_attn_rank_fwd and every entry point that runs it, and the dK/dV kernel of the
 * attention backward): their workgroups hand K/V (or query) tiles over through counters
 * in LDS, and each wait polls its counter at most a bounded number of times, so that a
 * broken hand-over cannot hang the GPU; a workgroup in which a wait gave up writes its
 * outputs as NaN (attention output and log-sum-exp, or dK / dV contributions).
 * polls > 0 caps every such wait at that many polls for launches enqueued after the
 * call (a cap of 1 makes the waits give up and the outputs NaN, which is what the tests
 * check); 0 restores the default of 4096.  Process-wide.  TSP_ERR_SHAPE for polls < 0. */
tsp_status tsp_test_set_attn_poll_limit(int32_t polls);

/* Static, human-readable name of a status code. */
const char* tsp_status_str(tsp_status status);

/* The hipError_t behind the most recent TSP_ERR_HIP returned on the calling thread
 * (0 = hipSuccess if no call on this thread has failed that way).  Kept per thread
 * until the next such failure; no other call resets it. */
int tsp_last_hip_error(void);

/* Static name of a HIP error code (as hipGetErrorName), e.g. for tsp_last_hip_error. */
const char* tsp_hip_error_string(int hip_error);

/* TSP_ABI_VERSION of the built library. */
int tsp_abi_version(void);

#ifdef __cplusplus
}
#endif

#endif /* TSP_H */
