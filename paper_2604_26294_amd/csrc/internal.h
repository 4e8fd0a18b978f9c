// Internal launchers of libtsp's gfx950 kernels (not part of the C ABI).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace tsp {

// Most operand pairs of one multi-part contraction, and most products of one grouped
// launch (launch_gemm_*_group).
constexpr int kGemmPartsMax = 8;
constexpr int kGemmGroupMax = 8;

// Parameters of the bf16 MFMA GEMM family: C[M, N] = A[M, K] * B, fp32 accumulation.
// B is [N, K] row-major ("NT", both operands contraction-contiguous) or [K, N]
// row-major ("NN").  The epilogue decides what C becomes.
struct GemmParams {
  const uint16_t* A;
  int lda;
  const uint16_t* B;
  int ldb;
  const uint16_t* B2;  // SwiGLU (both directions): the up-projection operand, layout of B
  int M, N, K;         // K: contraction length, a multiple of 64
  int Kb_rows;         // [K, N] operands: rows actually present (rows >= Kb_rows are clamped)
  // Multi-part contraction ([K, N] products only): with n_parts >= 2 the contraction
  // indices form n_parts consecutive ranges of k_part each (k_part a multiple of 64,
  // K = n_parts k_part); index k of range i = k / k_part reads column k - i k_part of
  // A_part[i] (row stride lda) and row k - i k_part of B_part[i] (row stride ldb, rows
  // >= Kb_rows clamped).  n_parts <= 1: one part, A and B.
  int n_parts;
  int k_part;
  const uint16_t* A_part[kGemmPartsMax];
  const uint16_t* B_part[kGemmPartsMax];

  // SwiGLU epilogue: H[m, n] = bf16( SiLU(C_gate) * C_up ) for n < N, and 0 for
  // N <= n < h_cols (the zero padding that lets the down projection contract over
  // h_cols), row stride ldh; h_cols == 0 means h_cols = ldh.
  uint16_t* H;
  int ldh;
  int h_cols;

  // SwiGLU backward (fused products G = A B^T, U = A B2^T and dHs = A2 B3^T, all NT
  // with the same K): with s = SiLU(G), s' its derivative,
  //   dG = dHs * U * s'  and  dU = dHs * s  -> H, H2 [M, ldh] bf16 (columns N..ldh zero),
  //   dG^T, dU^T and Hs^T = (s * U)^T       -> T0, T1, T2 [N, ldt] bf16, row n holding
  //   column n of the product for every m < M (columns M..ldt zero).
  const uint16_t* A2;
  const uint16_t* B3;
  uint16_t* H2;
  uint16_t* T0;
  uint16_t* T1;
  uint16_t* T2;
  int ldt;

  // Accumulate epilogue: Y[m, n] = base + C, base = bf16 R[m, n] if R, else Y[m, n]
  // if accumulate, else 0; optionally U[m, n] = bf16(Y[m, n]).
  float* Y;
  int ldy;
  int accumulate;
  const uint16_t* R;
  int ldr;
  uint16_t* U;
  int ldu;
  // Split contraction (accumulate products of launch_gemm_nn_acc): with k_splits > 1
  // the K/64 contraction steps are cut into k_splits consecutive ranges (range c: steps
  // [c nk / k_splits, (c + 1) nk / k_splits)), each written as an fp32 partial product to
  // part + c M N (row stride N); a second kernel then forms Y = base + the partials
  // summed in range order (and U), as above.  Set by launch_gemm_nn_acc.
  int k_splits;
  float* part;

  // Q/K/V epilogue: columns [0, nq) -> Q[m, n] = bf16(q_scale C[m, n]) (the factor
  // applied to the fp32 product, so Q is rounded once); [nq, nq+nkv) -> K buffer;
  // [nq+nkv, nq+2nkv) -> V buffer.  Row m = b*rows_per_batch + t lands at sequence
  // position kv_pos0 + t of batch b if t < kv_seg, else at kv_pos1 + (t - kv_seg)
  // (the zigzag layout's second chunk); column c of the K (or V) block lands at
  // element kv_col0 + c of that position's row.
  uint16_t* Q;
  int ldq;
  float q_scale;
  uint16_t* Kb;
  uint16_t* Vb;
  int nq, nkv;
  int rows_per_batch;
  long long kv_batch_stride;
  int kv_row_stride;
  long long kv_pos0;
  int kv_seg;
  long long kv_pos1;
  int kv_col0;
};

hipError_t launch_gemm_swiglu(const GemmParams& p, hipStream_t s);
// Up to kGemmGroupMax independent products of launch_gemm_swiglu's form in one launch
// (each must have M, N > 0; the tiles of product i follow those of the ones before it).
hipError_t launch_gemm_swiglu_group(const GemmParams* ps, int n, hipStream_t s);
hipError_t launch_gemm_swiglu_bwd(const GemmParams& p, hipStream_t s);
// The accumulate epilogue over [K, N] operands.  Products with fewer 256 x 256 output
// tiles than CUs split their contraction (gemm_nn_acc_splits ranges) through an fp32
// workspace `part` of at least splits * M * N floats (unused when splits == 1); without
// one (part == nullptr) they run unsplit on 128 x 128 tiles.
hipError_t launch_gemm_nn_acc(const GemmParams& p, float* part, hipStream_t s);
int gemm_nn_acc_splits(int M, int N, int K);
// The accumulate epilogue on 128 x 128 tiles, for products with few output tiles
// (the weight gradients: F/D x h outputs).
hipError_t launch_gemm_nn_acc_small(const GemmParams& p, hipStream_t s);
// Up to kGemmGroupMax independent products of launch_gemm_nn_acc_small's form in one
// launch (each must have M, N > 0).
hipError_t launch_gemm_nn_acc_small_group(const GemmParams* ps, int n, hipStream_t s);
hipError_t launch_gemm_qkv(const GemmParams& p, hipStream_t s);
// Up to kGemmGroupMax products of launch_gemm_qkv's form in one launch.
hipError_t launch_gemm_qkv_group(const GemmParams* ps, int n, hipStream_t s);

// Causal flash attention of one rank's queries for the heads of one shard.
//   Q [B, S_loc, H_s, d] bf16, the queries times softmax scale * log2(e) (rounded to
//   bf16 once, by the projection's epilogue), so that Q K^T are base-2 logits;
//   K/V buffers [B, S, n_kv, d] bf16 (heads
//   kv_head0 .. kv_head0 + H_s/g - 1 are this shard's);  O [B, S_loc, H_s, d] bf16.
//   Q and O rows may be wider than H_s d (a launch over some of the heads of a wider
//   buffer): token row t of Q starts ld elements after row t - 1, of O ld_o.
//   The local rows form n_seg segments of consecutive global positions: rows
//   [seg_row0[k], seg_row0[k] + seg_rows[k]) sit at positions seg_pos0[k] + (row -
//   seg_row0[k]) (one segment for contiguous chunks, two for a zigzag shard).  A query
//   at position t sees keys j <= t; keys at or beyond kv_len are never read.
struct AttnParams {
  const uint16_t* Q;
  const uint16_t* Kb;
  const uint16_t* Vb;
  uint16_t* O;
  int batch;
  int s_loc;
  int heads;        // H_s
  int group;        // g = n_h / n_kv
  int head_dim;     // d
  long long seq;    // S (K/V buffer rows per batch)
  int n_kv;         // kv heads in the buffer
  int kv_head0;     // first kv head of this shard
  int n_seg;        // 1 or 2
  int seg_row0[2];
  int seg_rows[2];
  int seg_pos0[2];
  int kv_len;       // number of readable keys: the last segment position + 1
  int ld;           // elements between consecutive token rows of Q (0: H_s d)
  int ld_o;         // ... and of O (0: as Q)
  // Key-range split (attn_split_count): each query tile's keys [0, n) are processed in
  // ranges [c split_len, (c + 1) split_len), c < n_split.  With n_split > 1 the ranges
  // write partial results -- part_o [n_split][part_rows][d] fp32 (unnormalised O) and
  // part_ml [n_split][part_rows][2] fp32 (reference, sum) with part_rows = B S_loc H_s
  // -- which a second kernel merges into O.
  int n_split;
  int split_len;
  // With n_split = 1: each workgroup takes two query tiles of one head, the i-th most
  // and the i-th fewest keys (equal work per workgroup).
  int pair_tiles;
  // Polls after which a wait of the forward's slot hand-over gives up (its query tile is
  // then written as NaN); set by launch_flash_attn from the process-wide test limit.
  int poll_limit;
  long long part_rows;
  float* part_o;
  float* part_ml;
  // Optional: the log-sum-exp of each query's base-2 logits (the products of the
  // scaled bf16 queries with the keys, as the kernel computes them), fp32
  // [B, lse_heads, S_loc] with this launch's heads at rows lse_head0 .. lse_head0 + H_s - 1
  // (lse_heads = 0: H_s rows from 0); written when non-null.
  float* lse;
  int lse_head0;
  int lse_heads;
};

// Workgroups the attention kernel aims to launch: one per CU of an MI355X.
constexpr int kAttnTargetWorkgroups = 256;
// Queries per attention workgroup (one query tile), and keys per tile step (key-range
// lengths are multiples of it).
constexpr int kAttnQueryTile = 256;
constexpr int kAttnKeyStep = 128;

// Number of key ranges (and their length, a multiple of the key tile, in *split_len)
// for one rank's attention (uses batch, heads and the segments of p): enough (query
// tile, head, batch, range) work items to fill the GPU.  Depends on the shape only, so
// workspace sizes are known up front.
int attn_split_count(const AttnParams& p, int* split_len);
// Estimated seconds of one attention launch over p's heads: with the split that
// attn_split_count chooses (pair = false), or with paired query tiles and no split.
double attn_launch_seconds(const AttnParams& p, bool pair);

// Process-wide cap on the polls of the forward attention's slot waits (0: the default);
// a test hook for that protocol's failure path.
void set_attn_poll_limit(int polls);
int attn_poll_limit();
hipError_t launch_flash_attn(const AttnParams& p, hipStream_t s);

// Backward of launch_flash_attn for one shard's heads (same segments and buffers).
//   Qs   [B, S_loc, H_s, d] bf16   the recomputed queries, scaled as for the forward
//                                  (bf16(softmax scale * log2(e) * q));
//   O    [B, S_loc, H_s, d] bf16   the recomputed attention output;
//   dO   [B, S_loc, H_s, d] bf16   its upstream gradient;
//   lse  [B, H_s, S_loc] fp32      base-2 log-sum-exp from the forward (AttnParams::lse).
// Writes delta = rowsum(dO * O) [B, H_s, S_loc],
// dQ [B, S_loc, H_s, d] bf16 (the gradient of the unscaled queries), and the
// contributions to the gradients of the gathered
// K / V: dK, dV [B, S, n_kv, d] fp32, columns of kv heads kv_head0 .. + H_s/g - 1, every
// one of the S rows (overwritten, or added to if accumulate).
struct AttnBwdParams {
  const uint16_t* Qs;
  const uint16_t* O;
  const uint16_t* dO;
  const uint16_t* Kb;
  const uint16_t* Vb;
  const float* lse;
  float* delta;
  uint16_t* dQ;
  float* dK;
  float* dV;
  int accumulate;
  int batch;
  int s_loc;
  int heads;
  int group;
  int head_dim;
  long long seq;
  int n_kv;
  int kv_head0;
  int n_seg;
  int seg_row0[2];
  int seg_rows[2];
  int seg_pos0[2];
  float scale;       // softmax scale
  // dQ key-range split (attn_bwd_dq_split): with dq_split > 1 each query tile's keys
  // [c dq_split_len, (c + 1) dq_split_len) write fp32 partials dq_part
  // [dq_split][B S_loc H_s][d], summed into dQ by a second kernel.
  int dq_split;
  int dq_split_len;
  float* dq_part;
  // Row strides and head placement of inputs that come from a wider buffer (a saved
  // forward): O's token rows o_ld elements apart (0: H_s d); lse rows of this launch's
  // heads at lse_head0 .. of [B, lse_heads, S_loc] (lse_heads = 0: H_s rows from 0).
  long long o_ld;
  int lse_head0;
  int lse_heads;
  // Polls after which a wait of the dK/dV kernel's slot hand-over gives up (its dK / dV
  // are then written as NaN); set by the launcher from the process-wide test limit.
  int poll_limit;
};

// Number of key ranges for the dQ kernel (and their length, a multiple of the key
// stage, in *split_len); depends on the shape only.
int attn_bwd_dq_split(const AttnBwdParams& p, int* split_len);

// The three kernels of the backward, in this order: delta; dK / dV; dQ.
hipError_t launch_attn_bwd_prep(const AttnBwdParams& p, hipStream_t s);
hipError_t launch_attn_bwd_dkdv(const AttnBwdParams& p, hipStream_t s);
hipError_t launch_attn_bwd_dq(const AttnBwdParams& p, hipStream_t s);

// out[n][m] = in[m][n] (bf16) for m < rows, n < cols, and 0 for rows <= m < ld_out
// (ld_out a multiple of 8; in rows 16-byte aligned).
hipError_t launch_transpose_bf16(const uint16_t* in, int ld_in, int rows, int cols,
                                 uint16_t* out, int ld_out, hipStream_t s);

}  // namespace tsp
