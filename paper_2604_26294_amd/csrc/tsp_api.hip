// Host side of the libtsp C ABI: argument validation, workspace planning and the
// per-rank shard loops of the paper's two schedules.  Every check runs before the
// first launch, so a call that returns an error has enqueued nothing.
#include <algorithm>
#include <math.h>
#include <stdint.h>

#include <mutex>
#include <vector>

#include "internal.h"
#include "tsp.h"

namespace {

using tsp::AttnParams;
using tsp::AttnBwdParams;
using tsp::GemmParams;

constexpr size_t kAlign = 256;

struct Dims {
  int B, S, h, F, nh, nkv, d, D, p;
  int s_loc;   // S / D
  int hs;      // query heads per shard
  int ks;      // kv heads per shard
  int g;       // GQA ratio
  int fs;      // MLP rows per shard
  int fs_pad;  // fs rounded up to a multiple of 64 (width of the gated product in the workspace)
  long long M; // B * S_loc tokens of this rank
  float scale;
  bool zz;     // zigzag layout: local rows = [chunk p; chunk 2D-1-p] of S/(2D) tokens each
  int s_c;     // S_loc / 2 (zigzag chunk length)
  int G;       // forward shard steps per grouped launch (1 .. min(D, kGroupMax))
};

// Most shard steps of one grouped launch (the number of operand pairs one product's
// multi-part contraction, and one grouped launch, can hold).
constexpr int kGroupMax = tsp::kGemmGroupMax < tsp::kGemmPartsMax ? tsp::kGemmGroupMax
                                                                  : tsp::kGemmPartsMax;

size_t align_up(size_t x) { return (x + kAlign - 1) / kAlign * kAlign; }

tsp_status check_shape(const tsp_shape* s, Dims* o) {
  if (!s) return TSP_ERR_NULL;
  if (s->batch < 0 || s->seq < 0 || s->hidden < 1 || s->ffn < 1 || s->n_heads < 1 ||
      s->n_kv_heads < 1 || s->head_dim < 1 || s->degree < 1)
    return TSP_ERR_SHAPE;
  if (s->rank < 0 || s->rank >= s->degree) return TSP_ERR_RANK;
  if (s->seq % s->degree != 0 || (long long)s->n_heads * s->head_dim != s->hidden ||
      s->n_heads % s->n_kv_heads != 0 || s->n_heads % s->degree != 0 ||
      s->n_kv_heads % s->degree != 0 || s->ffn % s->degree != 0)
    return TSP_ERR_SHAPE;
  if (s->layout != 0 && s->layout != 1) return TSP_ERR_UNSUPPORTED;
  if (s->layout == 1 && s->seq % (2 * s->degree) != 0) return TSP_ERR_SHAPE;
  if (s->head_dim != 64 && s->head_dim != 128) return TSP_ERR_UNSUPPORTED;
  if (s->group_steps < 0) return TSP_ERR_SHAPE;
  if (s->group_steps > kGroupMax) return TSP_ERR_UNSUPPORTED;
  if (s->hidden % 8 != 0 || (s->ffn / s->degree) % 8 != 0) return TSP_ERR_UNSUPPORTED;
  o->B = s->batch;
  o->S = s->seq;
  o->h = s->hidden;
  o->F = s->ffn;
  o->nh = s->n_heads;
  o->nkv = s->n_kv_heads;
  o->d = s->head_dim;
  o->D = s->degree;
  o->p = s->rank;
  o->s_loc = s->seq / s->degree;
  o->hs = s->n_heads / s->degree;
  o->ks = s->n_kv_heads / s->degree;
  o->g = s->n_heads / s->n_kv_heads;
  o->fs = s->ffn / s->degree;
  o->fs_pad = (o->fs + 63) / 64 * 64;
  o->M = (long long)o->B * o->s_loc;
  if (o->M > INT32_MAX / 2) return TSP_ERR_UNSUPPORTED;
  o->scale = s->softmax_scale > 0.f ? s->softmax_scale : 1.0f / sqrtf((float)s->head_dim);
  o->zz = s->layout == 1;
  o->s_c = o->s_loc / 2;
  o->G = s->group_steps > 0 ? s->group_steps : kGroupMax;
  if (o->G > o->D) o->G = o->D;
  // The GEMM operand loads address each operand with 32-bit byte offsets: the widest
  // per-token rows (x and Y [M, h]; the group's gated products [M, G (F/D rounded up to
  // 64)]; the backward's [M, F/D] and transposed [F/D, M] operands) must stay below 4 GiB.
  const long long width = std::max({(long long)o->h, (long long)o->G * o->fs_pad, (long long)o->F});
  if (o->M * width * 2 >= (1LL << 32)) return TSP_ERR_UNSUPPORTED;
  return TSP_OK;
}

// Forward workspace regions (each 256-byte aligned), for groups of G shard steps:
//   MLP:   Hs of the G ring steps of a group side by side, [M, G x (F/D rounded up to
//          64)] bf16 (zero-padded columns), then the down projection's fp32 partial
//          products when its contraction is split (short sequences)
//   ATTN:  Q and A of the G shard steps of a group, [M, G H_s d] bf16 each, then the
//          attention's key-range partials, then the output projection's partials
//   LAYER: u [M, h] bf16, then max(MLP, ATTN)
//
// A group's products run as one launch each: the gate+up (and Q/K/V) products of its
// G shards as one grouped launch, and the down (output) projection as one product over
// the G shards' operands (Y += [Hs_1 .. Hs_G] [W2_1; ..; W2_G] = sum of Hs_i W2_i), so Y
// is read and written once per group instead of once per step, and the attention of
// the group's G H_s heads as one launch.  The steps of a group are consecutive in the
// schedule's order and their operand pairs are laid out in that order along the
// contraction; the sum differs from the step-by-step one only in fp32 rounding order.
// In a streaming schedule G is the number of shards held at once; with every shard
// resident (one GPU), the default groups min(D, kGroupMax) steps.
constexpr int kPair = 2;  // the backward's weight and dX products of two steps at once
// fp32 partial products of a split down (output) projection over groups of n steps of
// k_step contraction columns each, for the group sizes that occur.
size_t split_part_bytes(const Dims& d, int k_step) {
  size_t most = 0;
  for (const int n : {d.G, d.D % d.G}) {
    if (n == 0) continue;
    const int splits = tsp::gemm_nn_acc_splits((int)d.M, d.h, n * k_step);
    const size_t b = splits > 1 ? (size_t)splits * d.M * d.h * 4 : 0;
    if (b > most) most = b;
  }
  return align_up(most);
}
size_t ws_mlp_hs(const Dims& d) { return align_up((size_t)d.M * d.G * d.fs_pad * 2); }
size_t ws_mlp(const Dims& d) { return ws_mlp_hs(d) + split_part_bytes(d, d.fs_pad); }
// Attention workspace: Q of the current shard and the attention output A (bf16
// [M, H_s d] each), then the key-range partials when the shard's attention is split.
// The rank's query rows as segments of consecutive global positions (Algorithm 1):
// contiguous chunks are one segment starting at p S_loc; a zigzag shard is chunk p
// (first s1 = (p+1) S_c keys) followed by chunk 2D-1-p (first s2 = (2D-p) S_c keys).
void attn_segments(const Dims& d, AttnParams* ap) {
  ap->batch = d.B;
  ap->s_loc = d.s_loc;
  ap->heads = d.hs;
  ap->head_dim = d.d;
  if (!d.zz) {
    ap->n_seg = 1;
    ap->seg_row0[0] = 0;
    ap->seg_rows[0] = d.s_loc;
    ap->seg_pos0[0] = d.p * d.s_loc;
    ap->kv_len = (d.p + 1) * d.s_loc;
  } else {
    ap->n_seg = 2;
    ap->seg_row0[0] = 0;
    ap->seg_rows[0] = d.s_c;
    ap->seg_pos0[0] = d.p * d.s_c;
    ap->seg_row0[1] = d.s_c;
    ap->seg_rows[1] = d.s_c;
    ap->seg_pos0[1] = (2 * d.D - 1 - d.p) * d.s_c;
    ap->kv_len = (2 * d.D - d.p) * d.s_c;
  }
}

// Key ranges of the forward attention over the n H_s heads of n shards.
int attn_group_split(const Dims& d, int n, int* split_len) {
  AttnParams ap = {};
  attn_segments(d, &ap);
  ap.heads = n * d.hs;
  return tsp::attn_split_count(ap, split_len);
}
// Key-range length covering every key of a launch in one range (paired tiles).
int attn_full_len(const AttnParams& ap) {
  const int keys = ap.seg_pos0[ap.n_seg - 1] + ap.seg_rows[ap.n_seg - 1];
  return (keys + tsp::kAttnKeyStep - 1) / tsp::kAttnKeyStep * tsp::kAttnKeyStep;
}
// How a group of n shards runs its attention: launches over `width` shards each (the
// last over the remainder), with paired query tiles or with key ranges.  A launch takes
// the fewest shards whose work items fill the GPU once: the workgroups on an XCD then
// start together and stream the same keys of the same head through its L2 (a launch of
// several rounds drifts out of step, as the query tiles' key counts differ, and re-reads
// K/V).  Pairing (tile i with tile n_qt - 1 - i: equal work per workgroup) halves the
// work items; whichever plan the dispatch simulation of the attention launches
// (tsp::attn_launch_seconds) prices lower for the whole group is taken.
struct AttnLaunchPlan {
  int width;
  bool pair;
};
AttnLaunchPlan attn_launch_plan(const Dims& d, int n) {
  AttnParams ap = {};
  attn_segments(d, &ap);
  long long tiles = 0;
  for (int k = 0; k < ap.n_seg; ++k)
    tiles += (ap.seg_rows[k] + tsp::kAttnQueryTile - 1) / tsp::kAttnQueryTile;
  auto width_for = [&](long long items_per_shard) {
    if (items_per_shard <= 0) return n;
    const long long need = (tsp::kAttnTargetWorkgroups + items_per_shard - 1) / items_per_shard;
    return (int)(need < n ? need : n);
  };
  auto group_seconds = [&](int width, bool pair) {
    double sec = 0.0;
    for (int i = 0; i < n; i += width) {
      AttnParams q = ap;
      q.heads = (n - i < width ? n - i : width) * d.hs;
      sec += tsp::attn_launch_seconds(q, pair);
    }
    return sec;
  };
  const AttnLaunchPlan plain = {width_for(tiles * d.hs * d.B), false};
  if (tiles < 2) return plain;
  const AttnLaunchPlan paired = {width_for((tiles + 1) / 2 * d.hs * d.B), true};
  return group_seconds(paired.width, true) < group_seconds(plain.width, false) ? paired : plain;
}
struct AttnWs {
  size_t q, a, po, pml, proj, total;  // byte offsets and total size
};
AttnWs attn_ws(const Dims& d) {
  AttnWs w;
  // Partials for the widest need among the attention launches that occur: groups of G
  // (and D mod G for a last, smaller group), each in launches of attn_shards_per_launch
  // shards (and a remainder).
  size_t part = 0;
  for (const int n : {d.G, d.D % d.G}) {
    if (n == 0) continue;
    const AttnLaunchPlan lp = attn_launch_plan(d, n);
    if (lp.pair) continue;  // no key ranges
    const int sub = lp.width;
    for (const int w : {sub, n % sub}) {
      if (w == 0) continue;
      int len = 0;
      const int ns = attn_group_split(d, w, &len);
      const size_t p = ns > 1 ? (size_t)ns * d.M * w * d.hs : 0;
      if (p > part) part = p;
    }
  }
  const size_t qa = align_up((size_t)d.M * d.G * d.hs * d.d * 2);
  w.q = 0;
  w.a = qa;
  w.po = 2 * qa;
  w.pml = w.po + align_up(part * d.d * 4);
  // The output projection's partials reuse the key-range partials' space: the combine
  // kernel has consumed those before the projection starts (same stream).
  w.proj = w.po;
  const size_t after_attn = w.pml + align_up(part * 2 * 4);
  const size_t after_proj = w.proj + split_part_bytes(d, d.hs * d.d);
  w.total = after_attn > after_proj ? after_attn : after_proj;
  return w;
}
size_t ws_attn(const Dims& d) { return attn_ws(d).total; }
// MLP backward workspace: dG, dU [M, F/D rounded up to 64] bf16 (the A operands of the
// dX products), then dG^T, dU^T, Hs^T [F/D, M rounded up to 64] bf16 (the A operands of
// the weight-gradient products, zero-padded past M) of two ring steps (one when D = 1):
// the weight gradients of steps 2i and 2i + 1 run as one grouped launch.
struct MlpBwdWs {
  size_t dg, du, dgt, dut, hst, tr_set, total;
  int m_pad;
};
MlpBwdWs mlp_bwd_ws(const Dims& d) {
  MlpBwdWs w;
  w.m_pad = (int)((d.M + 63) / 64 * 64);
  const size_t rm = align_up((size_t)d.M * d.fs_pad * 2), tr = align_up((size_t)d.fs * w.m_pad * 2);
  w.dg = 0;
  w.du = rm;
  w.dgt = 2 * rm;
  w.dut = 2 * rm + tr;
  w.hst = 2 * rm + 2 * tr;
  w.tr_set = 3 * tr;  // one step's three transposes; the second step's follow
  w.total = 2 * rm + (d.D > 1 ? 2 : 1) * 3 * tr;
  return w;
}
// Attention backward, first stage: Q (recomputed, then scaled in place), A, dA, and dQ of
// two shard steps [M, H_s d] bf16 (the dX products of shards 2i and 2i + 1 run as one); lse, delta [B, H_s, S_loc] fp32; A^T and dQ^T [H_s d, M rounded up
// to 64] bf16 (the A operands of the weight-gradient products, zero past M); then the
// forward recomputation's key-range partials, as for the forward, and the dQ kernel's
// key-range partials.
struct AttnBwdWs {
  size_t q, a, da, dq, dq2, lse, delta, at, dqt, po, pml, dqp, total;
  int m_pad, n_split, split_len, dq_split, dq_split_len;
};
AttnBwdWs attn_bwd_ws(const Dims& d) {
  AttnBwdWs w;
  AttnParams ap = {};
  attn_segments(d, &ap);
  w.n_split = tsp::attn_split_count(ap, &w.split_len);
  {
    AttnBwdParams bp = {};
    bp.batch = d.B;
    bp.heads = d.hs;
    bp.n_seg = ap.n_seg;
    for (int k = 0; k < 2; ++k) {
      bp.seg_rows[k] = ap.seg_rows[k];
      bp.seg_pos0[k] = ap.seg_pos0[k];
    }
    w.dq_split = tsp::attn_bwd_dq_split(bp, &w.dq_split_len);
  }
  w.m_pad = (int)((d.M + 63) / 64 * 64);
  const size_t rows = (size_t)d.M * d.hs;
  const size_t qa = align_up(rows * d.d * 2), f = align_up(rows * 4);
  const size_t tr = align_up((size_t)d.hs * d.d * w.m_pad * 2);
  const size_t part = w.n_split > 1 ? (size_t)w.n_split * rows : 0;
  w.q = 0;
  w.a = qa;
  w.da = 2 * qa;
  w.dq = 3 * qa;
  w.dq2 = 4 * qa;  // dQ of the odd shard of a pair (unused when D = 1)
  w.lse = (d.D > 1 ? 5 : 4) * qa;
  w.delta = w.lse + f;
  w.at = w.delta + f;
  w.dqt = w.at + tr;
  w.po = w.dqt + tr;
  w.pml = w.po + align_up(part * d.d * 4);
  w.dqp = w.pml + align_up(part * 2 * 4);
  const size_t dq_part = w.dq_split > 1 ? (size_t)w.dq_split * rows * d.d * 4 : 0;
  w.total = w.dqp + align_up(dq_part);
  return w;
}
// Attention backward, second stage: the transposed gradients of one shard's K and V
// rows, [K_s d, M rounded up to 64] bf16 each.
size_t ws_attn_kv_bwd(const Dims& d) {
  const size_t m_pad = (size_t)((d.M + 63) / 64 * 64);
  return 2 * align_up((size_t)d.ks * d.d * m_pad * 2);
}
size_t ws_layer(const Dims& d) {
  const size_t a = ws_mlp(d), b = ws_attn(d);
  return align_up((size_t)d.M * d.h * 2) + (a > b ? a : b);
}

bool aligned(const void* p) { return ((uintptr_t)p & 15u) == 0; }

tsp_status check_ptr(const void* p) {
  if (!p) return TSP_ERR_NULL;
  return aligned(p) ? TSP_OK : TSP_ERR_ALIGN;
}

template <typename T>
tsp_status check_shards(T* const* arr, int D) {
  if (!arr) return TSP_ERR_NULL;
  for (int i = 0; i < D; ++i) {
    const tsp_status st = check_ptr(arr[i]);
    if (st != TSP_OK) return st;
  }
  return TSP_OK;
}

#define TSP_TRY(expr)                          \
  do {                                         \
    const tsp_status st_ = (expr);             \
    if (st_ != TSP_OK) return st_;             \
  } while (0)

// HIP error code of the last TSP_ERR_HIP returned on this thread.
thread_local int g_last_hip_error = 0;

tsp_status hip_failed(hipError_t e) {
  g_last_hip_error = (int)e;
  return TSP_ERR_HIP;
}

#define TSP_HIP(expr)                                \
  do {                                               \
    const hipError_t e_ = (expr);                    \
    if (e_ != hipSuccess) return hip_failed(e_);     \
  } while (0)


// ----------------------------------------------------------------- kernel timing
struct KernelTimer {
  std::mutex mu;
  bool on = false;
  std::vector<hipEvent_t> start[TSP_KERNEL_COUNT], stop[TSP_KERNEL_COUNT];
  size_t used[TSP_KERNEL_COUNT] = {};
};
KernelTimer g_timer;

// Records the start event of launch `kind` on `st`; returns the slot or -1.
long timer_begin(int kind, hipStream_t st) {
  if (!g_timer.on) return -1;
  std::lock_guard<std::mutex> lock(g_timer.mu);
  const size_t i = g_timer.used[kind];
  if (i == g_timer.start[kind].size()) {
    hipEvent_t a, b;
    if (hipEventCreate(&a) != hipSuccess) return -1;
    if (hipEventCreate(&b) != hipSuccess) {
      (void)hipEventDestroy(a);
      return -1;
    }
    g_timer.start[kind].push_back(a);
    g_timer.stop[kind].push_back(b);
  }
  if (hipEventRecord(g_timer.start[kind][i], st) != hipSuccess) return -1;
  g_timer.used[kind] = i + 1;
  return (long)i;
}

void timer_end(int kind, long slot, hipStream_t st) {
  if (slot >= 0) (void)hipEventRecord(g_timer.stop[kind][slot], st);
}

#define TSP_LAUNCH(kind, st, expr)                    \
  do {                                                \
    const long slot_ = timer_begin((kind), (st));     \
    const hipError_t e_ = (expr);                     \
    if (e_ != hipSuccess) return hip_failed(e_);      \
    timer_end((kind), slot_, (st));                   \
  } while (0)

// ----------------------------------------------------------------- launch sequences

// Algorithm 2 on an already validated problem.  Ring step t uses shard (p - t) mod D;
// the steps run in groups of G consecutive ones (the last group may be smaller): the
// group's gate+up products as one grouped launch (Hs of its i-th step in columns
// [i F/D_pad, (i + 1) F/D_pad) of the workspace), then one down projection over the
// group's shards.
tsp_status run_mlp(const Dims& d, const uint16_t* x, const uint16_t* const* wg,
                   const uint16_t* const* wu, const uint16_t* const* wd, float* y,
                   int accumulate, char* ws, hipStream_t st) {
  uint16_t* hs_ws = reinterpret_cast<uint16_t*>(ws);
  float* part = reinterpret_cast<float*>(ws + ws_mlp_hs(d));
  for (int t0 = 0; t0 < d.D; t0 += d.G) {
    const int n = d.D - t0 < d.G ? d.D - t0 : d.G;
    GemmParams up[tsp::kGemmGroupMax] = {};
    GemmParams dn = {};
    for (int i = 0; i < n; ++i) {
      const int t = t0 + i, j = ((d.p - t) % d.D + d.D) % d.D;
      GemmParams& u = up[i];
      u.A = x;
      u.lda = d.h;
      u.B = wg[j];
      u.B2 = wu[j];
      u.ldb = d.h;
      u.M = (int)d.M;
      u.N = d.fs;
      u.K = d.h;
      u.H = hs_ws + (size_t)i * d.fs_pad;
      u.ldh = n * d.fs_pad;
      u.h_cols = d.fs_pad;
      dn.A_part[i] = u.H;
      dn.B_part[i] = wd[j];
    }
    TSP_LAUNCH(TSP_KERNEL_GATE_UP, st, tsp::launch_gemm_swiglu_group(up, n, st));
    dn.A = hs_ws;
    dn.lda = n * d.fs_pad;
    dn.B = dn.B_part[0];
    dn.ldb = d.h;
    dn.M = (int)d.M;
    dn.N = d.h;
    dn.K = n * d.fs_pad;  // padded columns of Hs are zero; W2 rows past fs are clamped
    dn.Kb_rows = d.fs;
    dn.n_parts = n;
    dn.k_part = d.fs_pad;
    dn.Y = y;
    dn.ldy = d.h;
    dn.accumulate = (t0 > 0 || accumulate) ? 1 : 0;
    TSP_LAUNCH(TSP_KERNEL_DOWN, st, tsp::launch_gemm_nn_acc(dn, part, st));
  }
  return TSP_OK;
}

// Two-part contraction [A0 A1] [B0; B1] (row strides lda, ldb; B rows >= kb_rows of each
// part clamped), each part k_part wide.
void set_two_parts(GemmParams* p, const uint16_t* a0, const uint16_t* b0, const uint16_t* a1,
                   const uint16_t* b1, int k_part) {
  p->A = a0;
  p->B = b0;
  p->A_part[0] = a0;
  p->B_part[0] = b0;
  p->A_part[1] = a1;
  p->B_part[1] = b1;
  p->n_parts = 2;
  p->k_part = k_part;
  p->K = 2 * k_part;
}

// Backward of run_mlp (same ring order).  Per shard: one fused GEMM for G, U, dHs and
// the SwiGLU backward, two accumulating products for dX, three for the weight
// gradients (each [F/D, h], contracting over the M tokens).
tsp_status run_mlp_bwd(const Dims& d, const uint16_t* x, const uint16_t* dy,
                       const uint16_t* const* wg, const uint16_t* const* wu,
                       const uint16_t* const* wd, float* dx, int accumulate,
                       float* const* dwg, float* const* dwu, float* const* dwd, char* ws,
                       hipStream_t st) {
  const MlpBwdWs w = mlp_bwd_ws(d);
  uint16_t* dg = reinterpret_cast<uint16_t*>(ws + w.dg);
  uint16_t* du = reinterpret_cast<uint16_t*>(ws + w.du);
  GemmParams dw[kPair * 3] = {};
  int n_dw = 0;
  for (int t = 0; t < d.D; ++t) {
    const int j = ((d.p - t) % d.D + d.D) % d.D;
    const size_t set = (size_t)(t % kPair) * w.tr_set;
    uint16_t* dgt = reinterpret_cast<uint16_t*>(ws + w.dgt + set);
    uint16_t* dut = reinterpret_cast<uint16_t*>(ws + w.dut + set);
    uint16_t* hst = reinterpret_cast<uint16_t*>(ws + w.hst + set);
    GemmParams g = {};
    g.A = x;
    g.A2 = dy;
    g.lda = d.h;
    g.B = wg[j];
    g.B2 = wu[j];
    g.B3 = wd[j];
    g.ldb = d.h;
    g.M = (int)d.M;
    g.N = d.fs;
    g.K = d.h;
    g.H = dg;
    g.H2 = du;
    g.ldh = d.fs_pad;
    g.T0 = dgt;
    g.T1 = dut;
    g.T2 = hst;
    g.ldt = w.m_pad;
    TSP_LAUNCH(TSP_KERNEL_BWD_GATE, st, tsp::launch_gemm_swiglu_bwd(g, st));

    // dX (+)= dG W_gate[j] + dU W_up[j] = [dG dU] [W_gate[j]; W_up[j]] in one product
    // ([M, F/D] x [F/D, h] twice; padded columns of dG, dU are zero).
    {
      GemmParams p = {};
      set_two_parts(&p, dg, wg[j], du, wu[j], d.fs_pad);
      p.lda = d.fs_pad;
      p.ldb = d.h;
      p.Kb_rows = d.fs;
      p.M = (int)d.M;
      p.N = d.h;
      p.Y = dx;
      p.ldy = d.h;
      p.accumulate = (t > 0 || accumulate) ? 1 : 0;
      TSP_LAUNCH(TSP_KERNEL_BWD_DX, st, tsp::launch_gemm_nn_acc(p, nullptr, st));
    }
    // dW (+)= (dG^T | dU^T | Hs^T) (X | X | dY): [F/D, M] x [M, h], padded rows are zero;
    // the three products of steps 2i and 2i + 1 in one launch (an odd last step alone).
    for (int k = 0; k < 3; ++k) {
      GemmParams& q = dw[n_dw++];
      q = GemmParams{};
      q.A = k == 0 ? dgt : (k == 1 ? dut : hst);
      q.lda = w.m_pad;
      q.B = k < 2 ? x : dy;
      q.ldb = d.h;
      q.M = d.fs;
      q.N = d.h;
      q.K = w.m_pad;
      q.Kb_rows = (int)d.M;
      q.Y = k == 0 ? dwg[j] : (k == 1 ? dwu[j] : dwd[j]);
      q.ldy = d.h;
      q.accumulate = accumulate ? 1 : 0;
    }
    if (t % kPair == 1 || t == d.D - 1) {
      TSP_LAUNCH(TSP_KERNEL_BWD_DW, st, tsp::launch_gemm_nn_acc_small_group(dw, n_dw, st));
      n_dw = 0;
    }
  }
  return TSP_OK;
}

constexpr float kLog2e = 1.4426950408889634f;

GemmParams qkv_params(const Dims& d, const uint16_t* x, const uint16_t* shard, int r,
                      uint16_t* q_ws, uint16_t* kb, uint16_t* vb, bool with_q) {
  GemmParams g = {};
  const int qd = d.hs * d.d, kd = d.ks * d.d;
  g.A = x;
  g.lda = d.h;
  g.B = with_q ? shard : shard + (size_t)qd * d.h;
  g.ldb = d.h;
  g.M = (int)d.M;
  g.N = (with_q ? qd : 0) + 2 * kd;
  g.K = d.h;
  g.Q = q_ws;
  g.ldq = qd;
  g.q_scale = d.scale * kLog2e;  // the attention kernels take base-2-logit queries
  g.Kb = kb;
  g.Vb = vb;
  g.nq = with_q ? qd : 0;
  g.nkv = kd;
  g.rows_per_batch = d.s_loc;
  g.kv_batch_stride = (long long)d.S * d.nkv * d.d;
  g.kv_row_stride = d.nkv * d.d;
  if (!d.zz) {
    g.kv_pos0 = (long long)d.p * d.s_loc;
    g.kv_seg = d.s_loc;
    g.kv_pos1 = 0;
  } else {  // ZigZagReorder folded into the write addresses
    g.kv_pos0 = (long long)d.p * d.s_c;
    g.kv_seg = d.s_c;
    g.kv_pos1 = (long long)(2 * d.D - 1 - d.p) * d.s_c;
  }
  g.kv_col0 = r * kd;
  return g;
}

// Algorithm 1 on a validated problem.  `residual` (bf16 [M, h]) initialises Y at the
// first output projection instead of zero / the old Y; `u_out` receives bf16(Y) after
// the last.  The shards run in groups of G consecutive ones (the last may be smaller):
// per group one grouped Q/K/V launch (Q of its i-th shard in columns [i H_s d,
// (i + 1) H_s d) of the workspace, i.e. [M, n H_s, d] for a group of n), one attention
// launch over the group's n H_s heads (kv heads r0 K_s .. (r0 + n) K_s - 1), and one
// output projection over the group's shards.
tsp_status run_attn(const Dims& d, const uint16_t* x, const uint16_t* const* wa,
                    uint16_t* kb, uint16_t* vb, float* y, int accumulate,
                    const uint16_t* residual, uint16_t* u_out, char* ws, hipStream_t st,
                    uint16_t* a_out = nullptr, float* lse_out = nullptr) {
  const int qd = d.hs * d.d, kd = d.ks * d.d;
  const size_t wo = (size_t)(qd + 2 * kd) * d.h;  // W_O^(r)^T block [H_s d, h] of a shard
  const AttnWs aw = attn_ws(d);
  uint16_t* q_ws = reinterpret_cast<uint16_t*>(ws + aw.q);
  for (int r0 = 0; r0 < d.D; r0 += d.G) {
    const int n = d.D - r0 < d.G ? d.D - r0 : d.G;
    // A of the group: the workspace ([M, n H_s d]), or the caller's [M, n_h d] buffer at
    // the group's columns (kept for the backward)
    uint16_t* a_ws = a_out ? a_out + (size_t)r0 * qd : reinterpret_cast<uint16_t*>(ws + aw.a);
    const int a_ld = a_out ? d.D * qd : n * qd;
    GemmParams g[tsp::kGemmGroupMax] = {};
    GemmParams o = {};
    for (int i = 0; i < n; ++i) {
      g[i] = qkv_params(d, x, wa[r0 + i], r0 + i, q_ws + (size_t)i * qd, kb, vb, true);
      g[i].ldq = n * qd;
      o.A_part[i] = a_ws + (size_t)i * qd;
      o.B_part[i] = wa[r0 + i] + wo;
    }
    TSP_LAUNCH(TSP_KERNEL_QKV, st, tsp::launch_gemm_qkv_group(g, n, st));

    // Attention over the group's heads, lp.width shards per launch (the columns of those
    // shards within the group's Q and A).
    const AttnLaunchPlan lp = attn_launch_plan(d, n);
    const int sub = lp.width;
    for (int i = 0; i < n; i += sub) {
      const int w = n - i < sub ? n - i : sub;
      AttnParams ap = {};
      ap.Q = q_ws + (size_t)i * qd;
      ap.Kb = kb;
      ap.Vb = vb;
      ap.O = a_ws + (size_t)i * qd;
      attn_segments(d, &ap);
      ap.heads = w * d.hs;
      ap.ld = n * qd;     // Q: the group's workspace rows
      ap.ld_o = a_ld;     // A: the workspace's, or the caller's wider rows
      ap.lse = lse_out;
      ap.lse_head0 = (r0 + i) * d.hs;
      ap.lse_heads = d.nh;
      ap.group = d.g;
      ap.head_dim = d.d;
      ap.seq = d.S;
      ap.n_kv = d.nkv;
      ap.kv_head0 = (r0 + i) * d.ks;
      ap.pair_tiles = lp.pair ? 1 : 0;
      if (lp.pair) {
        ap.n_split = 1;
        ap.split_len = attn_full_len(ap);
      } else {
        ap.n_split = attn_group_split(d, w, &ap.split_len);
      }
      ap.part_rows = (long long)d.M * ap.heads;
      ap.part_o = reinterpret_cast<float*>(ws + aw.po);
      ap.part_ml = reinterpret_cast<float*>(ws + aw.pml);
      TSP_LAUNCH(TSP_KERNEL_ATTN, st, tsp::launch_flash_attn(ap, st));
    }

    o.A = a_ws;
    o.lda = a_ld;
    o.B = o.B_part[0];
    o.ldb = d.h;
    o.M = (int)d.M;
    o.N = d.h;
    o.K = n * qd;
    o.Kb_rows = qd;
    o.n_parts = n;
    o.k_part = qd;
    o.Y = y;
    o.ldy = d.h;
    const bool first = r0 == 0, last = r0 + n == d.D;
    o.accumulate = (!first || accumulate) ? 1 : 0;
    if (first && residual) {
      o.R = residual;
      o.ldr = d.h;
    }
    if (last && u_out) {
      o.U = u_out;
      o.ldu = d.h;
    }
    TSP_LAUNCH(TSP_KERNEL_OPROJ, st,
               tsp::launch_gemm_nn_acc(o, reinterpret_cast<float*>(ws + aw.proj), st));
  }
  return TSP_OK;
}

// C[M, n] = f A[M, h] B[n, h]^T, bf16 out (the Q epilogue of the projection kernel with
// every column in the Q block).
GemmParams nt_params(const Dims& d, const uint16_t* a, const uint16_t* b, int n, uint16_t* out,
                     float f) {
  GemmParams g = {};
  g.q_scale = f;
  g.A = a;
  g.lda = d.h;
  g.B = b;
  g.ldb = d.h;
  g.M = (int)d.M;
  g.N = n;
  g.K = d.h;
  g.Q = out;
  g.ldq = n;
  g.nq = n;
  g.rows_per_batch = d.s_loc;
  return g;
}

// Backward of run_attn, first stage (see tsp_attn_rank_bwd).
tsp_status run_attn_bwd(const Dims& d, const uint16_t* x, const uint16_t* dy,
                        const uint16_t* const* wa, const uint16_t* kb, const uint16_t* vb,
                        float* dx, int accumulate, float* const* dw, float* dk, float* dv,
                        char* ws, hipStream_t st, const uint16_t* a_saved = nullptr,
                        const float* lse_saved = nullptr) {
  const int qd = d.hs * d.d, kd = d.ks * d.d;
  const AttnBwdWs w = attn_bwd_ws(d);
  uint16_t* q_ws = reinterpret_cast<uint16_t*>(ws + w.q);
  uint16_t* a_ws = reinterpret_cast<uint16_t*>(ws + w.a);
  uint16_t* da_ws = reinterpret_cast<uint16_t*>(ws + w.da);
  uint16_t* dq_buf[kPair] = {reinterpret_cast<uint16_t*>(ws + w.dq),
                             reinterpret_cast<uint16_t*>(ws + w.dq2)};
  uint16_t* at_ws = reinterpret_cast<uint16_t*>(ws + w.at);
  uint16_t* dqt_ws = reinterpret_cast<uint16_t*>(ws + w.dqt);
  float* lse = reinterpret_cast<float*>(ws + w.lse);
  float* delta = reinterpret_cast<float*>(ws + w.delta);
  for (int r = 0; r < d.D; ++r) {
    const uint16_t* wq = wa[r];
    const uint16_t* wo_t = wa[r] + (size_t)(qd + 2 * kd) * d.h;  // W_O^(r)^T [H_s d, h]
    uint16_t* dq_ws = dq_buf[r % kPair];
    // Q times scale * log2(e), as the attention kernels take it
    GemmParams g = nt_params(d, x, wq, qd, q_ws, d.scale * kLog2e);
    TSP_LAUNCH(TSP_KERNEL_ABWD_PROJ, st, tsp::launch_gemm_qkv(g, st));

    AttnParams ap = {};
    attn_segments(d, &ap);
    // A and the log-sum-exp: the forward's, kept by tsp_attn_rank_fwd_train (shard r's
    // columns of [M, n_h d] and rows of [B, n_h, S_loc]), or recomputed into the workspace
    const uint16_t* a_src = a_saved ? a_saved + (size_t)r * qd : a_ws;
    const int a_ld = a_saved ? d.nh * d.d : qd;
    if (!a_saved) {
      ap.Q = q_ws;
      ap.Kb = kb;
      ap.Vb = vb;
      ap.O = a_ws;
      ap.group = d.g;
      ap.head_dim = d.d;
      ap.seq = d.S;
      ap.n_kv = d.nkv;
      ap.kv_head0 = r * d.ks;
      ap.n_split = w.n_split;
      ap.split_len = w.split_len;
      ap.part_rows = (long long)d.M * d.hs;
      ap.part_o = reinterpret_cast<float*>(ws + w.po);
      ap.part_ml = reinterpret_cast<float*>(ws + w.pml);
      ap.lse = lse;
      TSP_LAUNCH(TSP_KERNEL_ABWD_FWD, st, tsp::launch_flash_attn(ap, st));
    }

    g = nt_params(d, dy, wo_t, qd, da_ws, 1.f);  // dA = dY W_O^(r)
    TSP_LAUNCH(TSP_KERNEL_ABWD_PROJ, st, tsp::launch_gemm_qkv(g, st));

    AttnBwdParams bp = {};
    bp.Qs = q_ws;
    bp.O = a_src;
    bp.o_ld = a_ld;
    bp.dO = da_ws;
    bp.Kb = kb;
    bp.Vb = vb;
    bp.lse = lse_saved ? lse_saved : lse;
    if (lse_saved) {
      bp.lse_head0 = r * d.hs;
      bp.lse_heads = d.nh;
    }
    bp.delta = delta;
    bp.dQ = dq_ws;
    bp.dK = dk;
    bp.dV = dv;
    bp.accumulate = accumulate ? 1 : 0;
    bp.batch = d.B;
    bp.s_loc = d.s_loc;
    bp.heads = d.hs;
    bp.group = d.g;
    bp.head_dim = d.d;
    bp.seq = d.S;
    bp.n_kv = d.nkv;
    bp.kv_head0 = r * d.ks;
    bp.n_seg = ap.n_seg;
    for (int k = 0; k < 2; ++k) {
      bp.seg_row0[k] = ap.seg_row0[k];
      bp.seg_rows[k] = ap.seg_rows[k];
      bp.seg_pos0[k] = ap.seg_pos0[k];
    }
    bp.scale = d.scale;
    bp.dq_split = w.dq_split;
    bp.dq_split_len = w.dq_split_len;
    bp.dq_part = reinterpret_cast<float*>(ws + w.dqp);
    TSP_LAUNCH(TSP_KERNEL_ABWD_AUX, st, tsp::launch_attn_bwd_prep(bp, st));
    TSP_LAUNCH(TSP_KERNEL_ABWD_KV, st, tsp::launch_attn_bwd_dkdv(bp, st));
    TSP_LAUNCH(TSP_KERNEL_ABWD_Q, st, tsp::launch_attn_bwd_dq(bp, st));

    // dX (+)= dQ W_Q^(r): [M, H_s d] x [H_s d, h], shards 2i and 2i + 1 as one product
    // ([dQ dQ'] [W_Q; W_Q']), an odd last shard alone.
    const bool second = r % kPair == 1;
    if (second || r == d.D - 1) {
      GemmParams p = {};
      p.A = dq_buf[0];
      p.lda = qd;
      p.B = second ? wa[r - 1] : wq;
      p.ldb = d.h;
      p.M = (int)d.M;
      p.N = d.h;
      p.K = qd;
      p.Kb_rows = qd;
      if (second) set_two_parts(&p, dq_buf[0], wa[r - 1], dq_buf[1], wq, qd);
      p.Y = dx;
      p.ldy = d.h;
      p.accumulate = (r >= kPair || accumulate) ? 1 : 0;
      TSP_LAUNCH(TSP_KERNEL_ABWD_DX, st, tsp::launch_gemm_nn_acc(p, nullptr, st));
    }

    TSP_LAUNCH(TSP_KERNEL_ABWD_AUX, st,
               tsp::launch_transpose_bf16(dq_ws, qd, (int)d.M, qd, dqt_ws, w.m_pad, st));
    TSP_LAUNCH(TSP_KERNEL_ABWD_AUX, st,
               tsp::launch_transpose_bf16(a_src, a_ld, (int)d.M, qd, at_ws, w.m_pad, st));
    // W_Q block (+)= dQ^T X;  W_O^T block (+)= A^T dY: [H_s d, M] x [M, h], one launch.
    GemmParams q[2] = {};
    for (int k = 0; k < 2; ++k) {
      q[k].A = k == 0 ? dqt_ws : at_ws;
      q[k].lda = w.m_pad;
      q[k].B = k == 0 ? x : dy;
      q[k].ldb = d.h;
      q[k].M = qd;
      q[k].N = d.h;
      q[k].K = w.m_pad;
      q[k].Kb_rows = (int)d.M;
      q[k].Y = dw[r] + (k == 0 ? (size_t)0 : (size_t)(qd + 2 * kd) * d.h);
      q[k].ldy = d.h;
      q[k].accumulate = accumulate ? 1 : 0;
    }
    TSP_LAUNCH(TSP_KERNEL_ABWD_DW, st, tsp::launch_gemm_nn_acc_small_group(q, 2, st));
  }
  return TSP_OK;
}

// Second stage (see tsp_attn_kv_rank_bwd).
tsp_status run_attn_kv_bwd(const Dims& d, const uint16_t* x, const uint16_t* const* wa,
                           const uint16_t* dkl, const uint16_t* dvl, float* dx, int accumulate,
                           float* const* dw, char* ws, hipStream_t st) {
  const int qd = d.hs * d.d, kd = d.ks * d.d, ld = d.nkv * d.d;
  const int m_pad = (int)((d.M + 63) / 64 * 64);
  uint16_t* t_ws = reinterpret_cast<uint16_t*>(ws);
  const size_t t_elems = align_up((size_t)kd * m_pad * 2) / 2;
  for (int r = 0; r < d.D; ++r) {
    const uint16_t* gk = dkl + (size_t)r * kd;  // [M, K_s d], row stride ld
    const uint16_t* gv = dvl + (size_t)r * kd;
    {
      GemmParams p = {};  // dX (+)= dK W_K^(r) + dV W_V^(r), one product over both
      set_two_parts(&p, gk, wa[r] + (size_t)qd * d.h, gv, wa[r] + (size_t)(qd + kd) * d.h, kd);
      p.lda = ld;
      p.ldb = d.h;
      p.Kb_rows = kd;
      p.M = (int)d.M;
      p.N = d.h;
      p.Y = dx;
      p.ldy = d.h;
      p.accumulate = (r > 0 || accumulate) ? 1 : 0;
      TSP_LAUNCH(TSP_KERNEL_ABWD_DX, st, tsp::launch_gemm_nn_acc(p, nullptr, st));
    }
    // W_K block (+)= dK^T X;  W_V block (+)= dV^T X: [K_s d, M] x [M, h], one launch.
    GemmParams q[2] = {};
    for (int k = 0; k < 2; ++k) {
      const uint16_t* g = k == 0 ? gk : gv;
      uint16_t* gt = t_ws + (size_t)k * t_elems;
      TSP_LAUNCH(TSP_KERNEL_ABWD_AUX, st,
                 tsp::launch_transpose_bf16(g, ld, (int)d.M, kd, gt, m_pad, st));
      q[k].A = gt;
      q[k].lda = m_pad;
      q[k].B = x;
      q[k].ldb = d.h;
      q[k].M = kd;
      q[k].N = d.h;
      q[k].K = m_pad;
      q[k].Kb_rows = (int)d.M;
      q[k].Y = dw[r] + (size_t)(qd + k * kd) * d.h;
      q[k].ldy = d.h;
      q[k].accumulate = accumulate ? 1 : 0;
    }
    TSP_LAUNCH(TSP_KERNEL_ABWD_DW, st, tsp::launch_gemm_nn_acc_small_group(q, 2, st));
  }
  return TSP_OK;
}

// ------------------------------------------------------------ allocation-free layer call
// Scratch space of tsp_layer_rank_fwd_noalloc: one fixed array per GPU, part of this
// file's device code object (the runtime places it in each device's memory when the
// code object is loaded there, and it stays until the process ends).  In host code the
// name `scratch` is only a stand-in; its device address comes from hipGetSymbolAddress,
// taken once per device with that device current, and only that address is used.
//
// Nothing in it needs clearing: every kernel writes each scratch element it later reads
// in the same call (Q, A, the gated product including its zero padding, bf16(u), the
// attention key-range partials, which every (range, query tile) workgroup writes even
// when none of its keys is visible, and the split projections' partial products, which
// every (range, output tile) workgroup writes in full).
static __device__ __align__(256) char scratch[TSP_NOALLOC_SCRATCH_BYTES];

constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
void* g_scratch_ptr[kMaxDevices] = {};

// Device address of the current device's scratch array.
tsp_status scratch_of_current_device(void** out) {
  int dev = 0;
  TSP_HIP(hipGetDevice(&dev));
  if (dev < 0 || dev >= kMaxDevices) return TSP_ERR_UNSUPPORTED;
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  if (!g_scratch_ptr[dev]) {
    void* ptr = nullptr;
    TSP_HIP(hipGetSymbolAddress(&ptr, HIP_SYMBOL(scratch)));
    if (!ptr) return TSP_ERR_HIP;
    g_scratch_ptr[dev] = ptr;
  }
  *out = g_scratch_ptr[dev];
  return TSP_OK;
}

tsp_status check_layer_args(const tsp_shape* shape, const uint16_t* x_loc,
                            const uint16_t* const* w_attn, const uint16_t* const* w_gate,
                            const uint16_t* const* w_up, const uint16_t* const* w_down,
                            uint16_t* k_buf, uint16_t* v_buf, float* y_loc, Dims* d) {
  TSP_TRY(check_shape(shape, d));
  TSP_TRY(check_ptr(x_loc));
  TSP_TRY(check_shards(w_attn, d->D));
  TSP_TRY(check_shards(w_gate, d->D));
  TSP_TRY(check_shards(w_up, d->D));
  TSP_TRY(check_shards(w_down, d->D));
  TSP_TRY(check_ptr(k_buf));
  TSP_TRY(check_ptr(v_buf));
  TSP_TRY(check_ptr(y_loc));
  return TSP_OK;
}

// The layer on a validated problem, with scratch space `ws` (at least ws_layer(d) bytes).
tsp_status run_layer(const Dims& d, const uint16_t* x_loc, const uint16_t* const* w_attn,
                     const uint16_t* const* w_gate, const uint16_t* const* w_up,
                     const uint16_t* const* w_down, uint16_t* k_buf, uint16_t* v_buf,
                     float* y_loc, char* ws, hipStream_t stream) {
  uint16_t* u_ws = reinterpret_cast<uint16_t*>(ws);
  char* rest = ws + align_up((size_t)d.M * d.h * 2);
  // u = x + Attn(x): Y starts from x at the first output projection; the last one also
  // writes bf16(u).
  TSP_TRY(run_attn(d, x_loc, w_attn, k_buf, v_buf, y_loc, 0, x_loc, u_ws, rest, stream));
  // y = u + MLP(bf16 u): the MLP accumulates onto Y, which holds u.
  return run_mlp(d, u_ws, w_gate, w_up, w_down, y_loc, 1, rest, stream);
}

}  // namespace

extern "C" {

tsp_status tsp_workspace_bytes(const tsp_shape* shape, int op, size_t* bytes) {
  Dims d;
  TSP_TRY(check_shape(shape, &d));
  if (!bytes) return TSP_ERR_NULL;
  switch (op) {
    case TSP_OP_MLP: *bytes = ws_mlp(d); return TSP_OK;
    case TSP_OP_ATTN: *bytes = ws_attn(d); return TSP_OK;
    case TSP_OP_LAYER: *bytes = ws_layer(d); return TSP_OK;
    case TSP_OP_MLP_BWD: *bytes = mlp_bwd_ws(d).total; return TSP_OK;
    case TSP_OP_ATTN_BWD: *bytes = attn_bwd_ws(d).total; return TSP_OK;
    case TSP_OP_ATTN_KV_BWD: *bytes = ws_attn_kv_bwd(d); return TSP_OK;
    default: return TSP_ERR_SHAPE;
  }
}

tsp_status tsp_mlp_rank_fwd(const tsp_shape* shape, const uint16_t* x_loc,
                            const uint16_t* const* w_gate, const uint16_t* const* w_up,
                            const uint16_t* const* w_down, float* y_loc, int accumulate,
                            void* ws, size_t ws_bytes, hipStream_t stream) {
  Dims d;
  TSP_TRY(check_shape(shape, &d));
  TSP_TRY(check_ptr(x_loc));
  TSP_TRY(check_ptr(y_loc));
  TSP_TRY(check_shards(w_gate, d.D));
  TSP_TRY(check_shards(w_up, d.D));
  TSP_TRY(check_shards(w_down, d.D));
  TSP_TRY(check_ptr(ws));
  if (ws_bytes < ws_mlp(d)) return TSP_ERR_WORKSPACE;
  if (d.M == 0) return TSP_OK;
  return run_mlp(d, x_loc, w_gate, w_up, w_down, y_loc, accumulate, static_cast<char*>(ws),
                 stream);
}

tsp_status tsp_mlp_rank_bwd(const tsp_shape* shape, const uint16_t* x_loc,
                            const uint16_t* dy_loc, const uint16_t* const* w_gate,
                            const uint16_t* const* w_up, const uint16_t* const* w_down,
                            float* dx_loc, int accumulate, float* const* dw_gate,
                            float* const* dw_up, float* const* dw_down, void* ws,
                            size_t ws_bytes, hipStream_t stream) {
  Dims d;
  TSP_TRY(check_shape(shape, &d));
  TSP_TRY(check_ptr(x_loc));
  TSP_TRY(check_ptr(dy_loc));
  TSP_TRY(check_ptr(dx_loc));
  TSP_TRY(check_shards(w_gate, d.D));
  TSP_TRY(check_shards(w_up, d.D));
  TSP_TRY(check_shards(w_down, d.D));
  TSP_TRY(check_shards(dw_gate, d.D));
  TSP_TRY(check_shards(dw_up, d.D));
  TSP_TRY(check_shards(dw_down, d.D));
  TSP_TRY(check_ptr(ws));
  if (ws_bytes < mlp_bwd_ws(d).total) return TSP_ERR_WORKSPACE;
  if (d.M == 0) return TSP_OK;
  return run_mlp_bwd(d, x_loc, dy_loc, w_gate, w_up, w_down, dx_loc, accumulate, dw_gate,
                     dw_up, dw_down, static_cast<char*>(ws), stream);
}

tsp_status tsp_kv_rank_fwd(const tsp_shape* shape, const uint16_t* x_loc,
                           const uint16_t* const* w_attn, uint16_t* k_buf, uint16_t* v_buf,
                           hipStream_t stream) {
  Dims d;
  TSP_TRY(check_shape(shape, &d));
  TSP_TRY(check_ptr(x_loc));
  TSP_TRY(check_shards(w_attn, d.D));
  TSP_TRY(check_ptr(k_buf));
  TSP_TRY(check_ptr(v_buf));
  if (d.M == 0) return TSP_OK;
  for (int r = 0; r < d.D; ++r) {
    GemmParams g = qkv_params(d, x_loc, w_attn[r], r, nullptr, k_buf, v_buf, false);
    TSP_LAUNCH(TSP_KERNEL_QKV, stream, tsp::launch_gemm_qkv(g, stream));
  }
  return TSP_OK;
}

tsp_status tsp_attn_rank_fwd(const tsp_shape* shape, const uint16_t* x_loc,
                             const uint16_t* const* w_attn, uint16_t* k_buf, uint16_t* v_buf,
                             float* y_loc, int accumulate, void* ws, size_t ws_bytes,
                             hipStream_t stream) {
  Dims d;
  TSP_TRY(check_shape(shape, &d));
  TSP_TRY(check_ptr(x_loc));
  TSP_TRY(check_shards(w_attn, d.D));
  TSP_TRY(check_ptr(k_buf));
  TSP_TRY(check_ptr(v_buf));
  TSP_TRY(check_ptr(y_loc));
  TSP_TRY(check_ptr(ws));
  if (ws_bytes < ws_attn(d)) return TSP_ERR_WORKSPACE;
  if (d.M == 0) return TSP_OK;
  return run_attn(d, x_loc, w_attn, k_buf, v_buf, y_loc, accumulate, nullptr, nullptr,
                  static_cast<char*>(ws), stream);
}

tsp_status tsp_attn_rank_fwd_train(const tsp_shape* shape, const uint16_t* x_loc,
                                   const uint16_t* const* w_attn, uint16_t* k_buf,
                                   uint16_t* v_buf, float* y_loc, int accumulate,
                                   uint16_t* a_out, float* lse_out, void* ws, size_t ws_bytes,
                                   hipStream_t stream) {
  Dims d;
  TSP_TRY(check_shape(shape, &d));
  TSP_TRY(check_ptr(x_loc));
  TSP_TRY(check_shards(w_attn, d.D));
  TSP_TRY(check_ptr(k_buf));
  TSP_TRY(check_ptr(v_buf));
  TSP_TRY(check_ptr(y_loc));
  TSP_TRY(check_ptr(a_out));
  TSP_TRY(check_ptr(lse_out));
  TSP_TRY(check_ptr(ws));
  if (ws_bytes < ws_attn(d)) return TSP_ERR_WORKSPACE;
  if (d.M == 0) return TSP_OK;
  return run_attn(d, x_loc, w_attn, k_buf, v_buf, y_loc, accumulate, nullptr, nullptr,
                  static_cast<char*>(ws), stream, a_out, lse_out);
}

tsp_status tsp_attn_rank_bwd(const tsp_shape* shape, const uint16_t* x_loc,
                             const uint16_t* dy_loc, const uint16_t* const* w_attn,
                             const uint16_t* k_buf, const uint16_t* v_buf, float* dx_loc,
                             int accumulate, float* const* dw_attn, float* dk_buf,
                             float* dv_buf, void* ws, size_t ws_bytes, hipStream_t stream) {
  Dims d;
  TSP_TRY(check_shape(shape, &d));
  TSP_TRY(check_ptr(x_loc));
  TSP_TRY(check_ptr(dy_loc));
  TSP_TRY(check_shards(w_attn, d.D));
  TSP_TRY(check_ptr(k_buf));
  TSP_TRY(check_ptr(v_buf));
  TSP_TRY(check_ptr(dx_loc));
  TSP_TRY(check_shards(dw_attn, d.D));
  TSP_TRY(check_ptr(dk_buf));
  TSP_TRY(check_ptr(dv_buf));
  TSP_TRY(check_ptr(ws));
  if (ws_bytes < attn_bwd_ws(d).total) return TSP_ERR_WORKSPACE;
  if (d.M == 0) return TSP_OK;
  return run_attn_bwd(d, x_loc, dy_loc, w_attn, k_buf, v_buf, dx_loc, accumulate, dw_attn,
                      dk_buf, dv_buf, static_cast<char*>(ws), stream);
}

tsp_status tsp_attn_rank_bwd_saved(const tsp_shape* shape, const uint16_t* x_loc,
                                   const uint16_t* dy_loc, const uint16_t* const* w_attn,
                                   const uint16_t* k_buf, const uint16_t* v_buf,
                                   const uint16_t* a_saved, const float* lse_saved,
                                   float* dx_loc, int accumulate, float* const* dw_attn,
                                   float* dk_buf, float* dv_buf, void* ws, size_t ws_bytes,
                                   hipStream_t stream) {
  Dims d;
  TSP_TRY(check_shape(shape, &d));
  TSP_TRY(check_ptr(x_loc));
  TSP_TRY(check_ptr(dy_loc));
  TSP_TRY(check_shards(w_attn, d.D));
  TSP_TRY(check_ptr(k_buf));
  TSP_TRY(check_ptr(v_buf));
  TSP_TRY(check_ptr(a_saved));
  TSP_TRY(check_ptr(lse_saved));
  TSP_TRY(check_ptr(dx_loc));
  TSP_TRY(check_shards(dw_attn, d.D));
  TSP_TRY(check_ptr(dk_buf));
  TSP_TRY(check_ptr(dv_buf));
  TSP_TRY(check_ptr(ws));
  if (ws_bytes < attn_bwd_ws(d).total) return TSP_ERR_WORKSPACE;
  if (d.M == 0) return TSP_OK;
  return run_attn_bwd(d, x_loc, dy_loc, w_attn, k_buf, v_buf, dx_loc, accumulate, dw_attn,
                      dk_buf, dv_buf, static_cast<char*>(ws), stream, a_saved, lse_saved);
}

tsp_status tsp_attn_kv_rank_bwd(const tsp_shape* shape, const uint16_t* x_loc,
                                const uint16_t* const* w_attn, const uint16_t* dk_loc,
                                const uint16_t* dv_loc, float* dx_loc, int accumulate,
                                float* const* dw_attn, void* ws, size_t ws_bytes,
                                hipStream_t stream) {
  Dims d;
  TSP_TRY(check_shape(shape, &d));
  TSP_TRY(check_ptr(x_loc));
  TSP_TRY(check_shards(w_attn, d.D));
  TSP_TRY(check_ptr(dk_loc));
  TSP_TRY(check_ptr(dv_loc));
  TSP_TRY(check_ptr(dx_loc));
  TSP_TRY(check_shards(dw_attn, d.D));
  TSP_TRY(check_ptr(ws));
  if (ws_bytes < ws_attn_kv_bwd(d)) return TSP_ERR_WORKSPACE;
  if (d.M == 0) return TSP_OK;
  return run_attn_kv_bwd(d, x_loc, w_attn, dk_loc, dv_loc, dx_loc, accumulate, dw_attn,
                         static_cast<char*>(ws), stream);
}

tsp_status tsp_layer_rank_fwd(const tsp_shape* shape, const uint16_t* x_loc,
                              const uint16_t* const* w_attn, const uint16_t* const* w_gate,
                              const uint16_t* const* w_up, const uint16_t* const* w_down,
                              uint16_t* k_buf, uint16_t* v_buf, float* y_loc, void* ws,
                              size_t ws_bytes, hipStream_t stream) {
  Dims d;
  TSP_TRY(check_layer_args(shape, x_loc, w_attn, w_gate, w_up, w_down, k_buf, v_buf, y_loc, &d));
  TSP_TRY(check_ptr(ws));
  if (ws_bytes < ws_layer(d)) return TSP_ERR_WORKSPACE;
  if (d.M == 0) return TSP_OK;
  return run_layer(d, x_loc, w_attn, w_gate, w_up, w_down, k_buf, v_buf, y_loc,
                   static_cast<char*>(ws), stream);
}

tsp_status tsp_layer_rank_fwd_noalloc(const tsp_shape* shape, const uint16_t* x_loc,
                                      const uint16_t* const* w_attn,
                                      const uint16_t* const* w_gate,
                                      const uint16_t* const* w_up,
                                      const uint16_t* const* w_down, uint16_t* k_buf,
                                      uint16_t* v_buf, float* y_loc, hipStream_t stream) {
  Dims d;
  TSP_TRY(check_layer_args(shape, x_loc, w_attn, w_gate, w_up, w_down, k_buf, v_buf, y_loc, &d));
  if (ws_layer(d) > (size_t)TSP_NOALLOC_SCRATCH_BYTES) return TSP_ERR_WORKSPACE;
  if (d.M == 0) return TSP_OK;
  void* ws = nullptr;
  TSP_TRY(scratch_of_current_device(&ws));
  return run_layer(d, x_loc, w_attn, w_gate, w_up, w_down, k_buf, v_buf, y_loc,
                   static_cast<char*>(ws), stream);
}

tsp_status tsp_test_set_attn_poll_limit(int32_t polls) {
  if (polls < 0) return TSP_ERR_SHAPE;
  tsp::set_attn_poll_limit(polls);
  return TSP_OK;
}

tsp_status tsp_profile_enable(int enable) {
  std::lock_guard<std::mutex> lock(g_timer.mu);
  g_timer.on = enable != 0;
  if (g_timer.on)
    for (int k = 0; k < TSP_KERNEL_COUNT; ++k) g_timer.used[k] = 0;
  return TSP_OK;
}

tsp_status tsp_profile_read(int kernel, double* total_ms, int64_t* launches) {
  if (!total_ms || !launches) return TSP_ERR_NULL;
  if (kernel < 0 || kernel >= TSP_KERNEL_COUNT) return TSP_ERR_SHAPE;
  std::lock_guard<std::mutex> lock(g_timer.mu);
  double sum = 0.0;
  for (size_t i = 0; i < g_timer.used[kernel]; ++i) {
    float ms = 0.f;
    if (hipEventSynchronize(g_timer.stop[kernel][i]) != hipSuccess ||
        hipEventElapsedTime(&ms, g_timer.start[kernel][i], g_timer.stop[kernel][i]) != hipSuccess)
      return TSP_ERR_HIP;
    sum += ms;
  }
  *total_ms = sum;
  *launches = (int64_t)g_timer.used[kernel];
  return TSP_OK;
}

const char* tsp_status_str(tsp_status status) {
  switch (status) {
    case TSP_OK: return "TSP_OK";
    case TSP_ERR_NULL: return "TSP_ERR_NULL: a required pointer is NULL";
    case TSP_ERR_SHAPE: return "TSP_ERR_SHAPE: inconsistent or non-divisible dimensions";
    case TSP_ERR_RANK: return "TSP_ERR_RANK: rank outside [0, degree)";
    case TSP_ERR_ALIGN: return "TSP_ERR_ALIGN: device pointer not 16-byte aligned";
    case TSP_ERR_WORKSPACE: return "TSP_ERR_WORKSPACE: workspace too small";
    case TSP_ERR_UNSUPPORTED: return "TSP_ERR_UNSUPPORTED: shape not implemented";
    case TSP_ERR_HIP: return "TSP_ERR_HIP: kernel launch failed";
    default: return "TSP_ERR_UNKNOWN";
  }
}

int tsp_abi_version(void) { return TSP_ABI_VERSION; }

int tsp_last_hip_error(void) { return g_last_hip_error; }

const char* tsp_hip_error_string(int hip_error) {
  return hipGetErrorName((hipError_t)hip_error);
}

}  // extern "C"
