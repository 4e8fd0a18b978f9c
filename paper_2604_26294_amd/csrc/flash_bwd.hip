// Backward of the causal flash attention of one TSP rank (gfx950, bf16 MFMA).
//
// For one shard's heads, given the rank's queries Q, the upstream gradient dO = dA of
// the attention output, the resident gathered K / V (sequence order), the base-2
// log-sum-exp of every query's logits (from the forward recomputation) and
// delta = rowsum(dO * O), the chain rule through O = P V, P = softmax(scale Q K^T)
// gives, with dP = dO V^T and dS = P * (dP - delta):
//   dV = P^T dO,  dK = scale dS^T Q   (contributions to every key of the prefix)
//   dQ = scale dS K.
// Two kernels share the work without atomics: one is key-stationary (a workgroup owns
// 128 keys of one kv head, keeps their K and V in registers and streams the queries of
// the g query heads that read them: dK, dV accumulate in registers and are written
// once), the other query-stationary (a workgroup owns 128 queries of one head and
// streams the keys: dQ accumulates in registers).  Both recompute the scores; only
// the query-stationary one needs dP's row sums, which delta already holds.
//
// The logits are formed exactly as the forward formed them, from the queries scaled by
// scale * log2(e) and rounded to bf16 once (Qs, written so by the projection), so that
// P = 2^(Qs K^T - lse) reproduces the forward's probabilities.  Since scale Q =
// Qs / log2(e) up to that rounding, dK = ln(2) dS^T Qs.
//
// MFMA layouts (32 x 32 x 16).  Key-stationary: S = Qs K^T and dP = dO V^T with the
// queries as rows (A operands read from LDS row by row, K and V fragments as B from
// registers); the accumulator then holds 16 queries of one key per lane, which is
// the B-operand layout of dV^T = dO^T P and dK^T = Qs^T dS (contraction over queries
// in the accumulator's row order), whose A operands dO^T and Qs^T come from the same
// LDS tiles through transpose reads.  Query-stationary: S^T = K Qs^T and
// dP^T = V dO^T with keys as rows (Qs and dO fragments in registers), so each lane
// holds 16 keys of one query, the B-operand layout of dQ^T = K^T dS^T, whose A
// operand K^T comes from the K tile through transpose reads.
//
// LDS tiles are rows of 16-byte chunks; the physical chunk is the logical chunk XOR
// f(row), with f chosen so that both read forms are bank-conflict free: 16 rows at one
// logical chunk (row reads) and 4 rows x 4 chunks (transpose reads of a 32-column
// block).
#include <math.h>

#include <type_traits>

#include "common.h"
#include "internal.h"
#include "lds_dma.h"

namespace tsp {
namespace {

constexpr int kBwdWaves = 4;
constexpr int kBwdThreads = kBwdWaves * kWave;
constexpr int kKvWaves = 8;
constexpr int kKvThreads = kKvWaves * kWave;
constexpr int kKvTile = 32 * kKvWaves;  // keys per key-stationary workgroup
constexpr int kQStage = 64;              // queries staged per step (key-stationary)
constexpr int kDqTile = 32 * kBwdWaves;  // queries per query-stationary workgroup
constexpr int kKStage = 64;              // keys staged per step (query-stationary)
constexpr float kLn2 = 0.69314718055994531f;

template <int N>
using IC = std::integral_constant<int, N>;

template <int D>
struct BwCfg {
  static constexpr int KCH = D / 8;             // 16-byte chunks per row
  static constexpr int RB = D * 2;              // row bytes
  static constexpr int RPW = 256 / RB;          // rows per 256-byte bank window
  static constexpr int KS = D / 16;             // contraction steps over d
  static constexpr int EB = D / 32;             // 32-row blocks of d
  static constexpr int T64 = 64 * RB;           // bytes of a 64-row tile
  static constexpr int RPD = kWave / KCH;       // rows one wave-wide LDS load fills
  static constexpr int DMA64 = 64 / (kBwdWaves * RPD);  // such loads per wave per tile
  static_assert(DMA64 * kBwdWaves * RPD == 64, "tile cover");
  // m = row / RPW indexes the row's bank window.  d = 128 (one row per window):
  // f = 4 (m mod 4) + (m / 4 mod 4), distinct over 16 consecutive rows, and distinct
  // in its upper two bits over 4 consecutive rows.  d = 64 (two rows per window, at
  // chunk offsets 0 and 8): f = 4 (m mod 2) + (m / 2 mod 4), distinct over 8
  // consecutive windows, and rows r, r + 2 (same half of a window) differ in bit 2.
  __device__ static int f(int row) {
    const int m = row / RPW;
    return D == 128 ? (((m & 3) << 2) | ((m >> 2) & 3)) : (((m & 1) << 2) | ((m >> 1) & 3));
  }
  // Byte offset of (row, column) in a tile (column a multiple of 4 for transpose reads).
  __device__ static int off(int row, int col) {
    return row * RB + 16 * ((col >> 3) ^ f(row)) + 2 * (col & 7);
  }
};

// One 64-row tile into LDS at `dst`.  Row r of the tile comes from base + min(r, last)
// rows of `row_bytes` each; rows past `last` repeat it (finite values that the caller
// masks).  Wave w's load i fills rows (WAVES i + w) RPD .. + RPD - 1.
template <int D, int WAVES = kBwdWaves>
__device__ __forceinline__ void load_tile64(const uint16_t* base, uint32_t row_bytes, int last,
                                            lds_char* dst, int wave, int lane) {
  using C = BwCfg<D>;
  const rsrc_t rsrc = make_rsrc(base);
  constexpr int N = 64 / (WAVES * C::RPD);  // loads per wave
  static_assert(N * WAVES * C::RPD == 64, "tile cover");
#pragma unroll
  for (int i = 0; i < N; ++i) {
    const int blk = i * WAVES + wave;
    const int r = blk * C::RPD + lane / C::KCH;
    const uint32_t rr = (uint32_t)min(r, last);
    const uint32_t voff = rr * row_bytes + 16u * (uint32_t)((lane % C::KCH) ^ C::f(r));
    dma16(rsrc, voff, 0u, dst + blk * (kWave * 16));
  }
}

// Lane layout of the transpose reads: source lane (t, group g) of a 16-lane group
// points at row 4 (g / 2) + t / 4 and column 16 (g % 2) + 4 (t % 4) of a 32-column
// block, so lane l receives column l % 32 of rows 4 (l / 32) + 0..3: the contraction
// slots 0-3 of the accumulator-ordered B operands; rows + 8 give slots 4-7.
__device__ __forceinline__ int tr_row(int lane) { return (((lane >> 4) >> 1) << 2) + ((lane & 15) >> 2); }
__device__ __forceinline__ int tr_col(int lane) { return 16 * ((lane >> 4) & 1) + 4 * (lane & 3); }

// ---------------------------------------------------------------------------------
// delta = rowsum(dO * O) per (query, head).  A group of D / 8 lanes handles one
// (row, head): 8 elements per lane, reduced across the group.
template <int D>
__global__ __launch_bounds__(256) void attn_bwd_prep_kernel(const AttnBwdParams P) {
  constexpr int G = D / 8;
  const long long idx = (long long)blockIdx.x * blockDim.x + threadIdx.x;
  const long long rh = idx / G;                    // (b S_loc + t) H_s + head
  const int part = (int)(idx % G);
  const long long n_rows = (long long)P.batch * P.s_loc * P.heads;
  const bool valid = rh < n_rows;
  const size_t e0 = (size_t)(valid ? rh : 0) * D + 8 * part;
  // O may sit in a wider buffer (token rows o_ld elements apart)
  const long long bt_o = (valid ? rh : 0) / P.heads;
  const size_t eo = P.o_ld > 0 ? (size_t)bt_o * P.o_ld + (size_t)((valid ? rh : 0) - bt_o * P.heads) * D +
                                     8 * part
                               : e0;
  float acc = 0.f;
  if (valid) {
    const u32x4 o = ld16(P.O + eo), g = ld16(P.dO + e0);
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      acc += bf16_bits_to_f32(o[e] & 0xffffu) * bf16_bits_to_f32(g[e] & 0xffffu);
      acc += bf16_bits_to_f32(o[e] >> 16) * bf16_bits_to_f32(g[e] >> 16);
    }
  }
#pragma unroll
  for (int m = 1; m < G; m <<= 1) acc += __shfl_xor(acc, m);
  if (valid && part == 0) {
    const long long bt = rh / P.heads, b = bt / P.s_loc;
    const int head = (int)(rh - bt * P.heads), t = (int)(bt - b * P.s_loc);
    P.delta[((size_t)b * P.heads + head) * P.s_loc + t] = acc;
  }
}

// Slot hand-over of the dK/dV kernel's query ring through counters in LDS (as in the
// forward kernel): "full" gains one per loader wavefront whose share of the slot's tile
// (and its lse / delta rows) is in LDS, "empty" one per wavefront done reading the slot.
// Waits poll with s_sleep and give up after a bounded number of polls; a wait that gave
// up flags the workgroup, whose dK / dV are then written as NaN.
typedef __attribute__((address_space(3))) int lds_int;
constexpr int kKvLoaders = kKvWaves / 2;  // the older wavefront of each SIMD loads
constexpr int kBwdSpinMax = 4096;
__device__ __forceinline__ void bwd_signal(lds_int* p) {
  if ((threadIdx.x & 63) == 0)
    asm volatile("ds_add_u32 %0, %1" ::"v"((uint32_t)(uintptr_t)p), "v"(1u) : "memory");
}
__device__ __forceinline__ int bwd_count(lds_int* p) {
  int v;
  asm volatile("ds_read_b32 %0, %1\n\ts_waitcnt lgkmcnt(0)"
               : "=v"(v) : "v"((uint32_t)(uintptr_t)p) : "memory");
  return __builtin_amdgcn_readfirstlane(v);
}
__device__ __forceinline__ void bwd_wait_ge(lds_int* p, int target, lds_int* flag, int polls) {
  for (int i = 0; i < polls; ++i) {
    if (bwd_count(p) >= target) return;
    __builtin_amdgcn_s_sleep(1);
  }
  bwd_signal(flag);
}

// ---------------------------------------------------------------------------------
// Key-stationary kernel: dK, dV of 256 keys of one kv head.
//
// Eight waves, two per SIMD (at most 256 registers each), so that one wave's vector
// and LDS phases overlap the other's matrix work; wave w owns keys 32 w .. 32 w + 31 of
// the tile.  Its K fragments stay in registers; the V rows (B operand of dP) are read
// from the workgroup's V tile, loaded into LDS once.  Query tiles of 64 rows of Qs and
// dO stream through a two-slot ring (handed over through the counters above, not a
// barrier per tile), unrolled by slot so that LDS addresses are registers plus
// immediates; each wave takes a tile in two 32-query blocks: S and dP (row reads), the
// probabilities and dS (vector ops), then dV^T and dK^T (transpose reads).
template <int D>
__global__ __launch_bounds__(kKvThreads) __attribute__((amdgpu_waves_per_eu(2, 2)))
void attn_bwd_dkdv_kernel(const AttnBwdParams P) {
  using C = BwCfg<D>;
  constexpr int T64 = C::T64;
  constexpr int VT = kKvTile * C::RB;  // the V tile
  constexpr int VO = 4 * T64 + 2 * 2 * kQStage * 4;  // its offset
  // [Qs slot 0][Qs slot 1][dO slot 0][dO slot 1][lse, delta slot 0][slot 1][V tile]
  // [slot counters]: the ring first, so that its offsets fit the 16-bit immediate of the
  // LDS reads.
  __shared__ __attribute__((aligned(1024))) char L[VO + VT + 64];
  lds_char* Ls = (lds_char*)L;
  float* Lf = reinterpret_cast<float*>(L + 4 * T64);

  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int l32 = lane & 31, hh = lane >> 5;
  const int kv_heads = P.heads / P.group;

  // Work item -> (batch, kv head, key tile), key tile fastest: an XCD's contiguous share
  // of work indices streams the same queries through its L2.  Key tiles alternate from
  // both ends of the sequence (early keys see the most queries), so that every XCD's
  // share holds as much light work as heavy.
  const int n_kt = (int)((P.seq + kKvTile - 1) / kKvTile);
  const int w = xcd_work_index(blockIdx.x, n_kt * kv_heads * P.batch);
  const int kj = w % n_kt;
  const int kt = (kj & 1) ? n_kt - 1 - (kj >> 1) : (kj >> 1);
  const int kvl = (w / n_kt) % kv_heads;
  const int b = w / n_kt / kv_heads;
  const int kvh = P.kv_head0 + kvl;
  const int k0 = kt * kKvTile;
  const int wk0 = k0 + 32 * wave;  // this wave's first key
  const int key = wk0 + l32;       // this lane's key (the accumulator column)

  // Keys at or past kv_len (the last query position + 1) are never read: their K
  // fragments are zero and their V rows repeat the last readable key; every query masks
  // them, so their dK, dV come out exactly zero.
  int kv_len = 0;
  for (int sg = 0; sg < P.n_seg; ++sg) kv_len = max(kv_len, P.seg_pos0[sg] + P.seg_rows[sg]);
  const size_t kv_stride = (size_t)P.n_kv * D;
  const uint16_t* kvbase = P.Kb + ((size_t)b * P.seq) * kv_stride + (size_t)kvh * D;
  const uint16_t* vvbase = P.Vb + ((size_t)b * P.seq) * kv_stride + (size_t)kvh * D;
  // V tile into LDS: keys k0 .. k0 + 255, rows past the last readable key repeating it
  // (a tile with no readable key has no query tile to visit either and loads nothing).
  const int v_last = min(kKvTile, kv_len - k0) - 1;
  if (v_last >= 0)
    for (int part = 0; part < kKvTile / 64; ++part)
      load_tile64<D, kKvWaves>(vvbase + (size_t)(k0 + 64 * part) * kv_stride,
                               2u * (uint32_t)kv_stride, max(v_last - 64 * part, 0),
                               Ls + VO + part * T64, wave, lane);
  // K fragments of this lane's key (B operand of S): d slots 16 s + 8 hh.
  const bool kread = key < kv_len;
  u32x4 kf[C::KS];
#pragma unroll
  for (int s = 0; s < C::KS; ++s)
    kf[s] = kread ? ld16(kvbase + (size_t)key * kv_stride + 16 * s + 8 * hh) : u32x4{0u, 0u, 0u, 0u};
  // Consume the K fragments here, before the loop: the compiler then waits for their
  // loads once, instead of at a point inside the loop where the same wait would also
  // cover the newest tile loads.
#pragma unroll
  for (int s = 0; s < C::KS; ++s) asm volatile("" ::"v"(kf[s]));

  // Query tiles of 64 rows that can see key k0 or later: per segment, tiles from tf.
  int tf[2] = {0, 0}, nv[2] = {0, 0};
  for (int sg = 0; sg < P.n_seg; ++sg) {
    const int nt = (P.seg_rows[sg] + kQStage - 1) / kQStage;
    const int num = k0 - P.seg_pos0[sg] - (kQStage - 1);
    tf[sg] = num <= 0 ? 0 : (num + kQStage - 1) / kQStage;
    nv[sg] = max(0, nt - tf[sg]);
  }
  const int per_head = nv[0] + nv[1];
  const int n_tiles = per_head * P.group;
  struct Tile {
    int head, seg, r0;
  };
  // Tiles in order: for each of the g query heads, the visible tiles of segment 0 then
  // segment 1.  A cursor (u = tile within the head, gi = head) walks them without
  // divisions.
  struct Cursor {
    int u, gi;
  };
  auto adv = [&](Cursor& c) __attribute__((always_inline)) {
    if (++c.u == per_head) {
      c.u = 0;
      ++c.gi;
    }
  };
  auto tile_at = [&](const Cursor& c) __attribute__((always_inline)) {
    Tile T;
    T.head = kvl * P.group + c.gi;
    T.seg = c.u < nv[0] ? 0 : 1;
    T.r0 = kQStage * (T.seg == 0 ? tf[0] + c.u : tf[1] + c.u - nv[0]);
    return T;
  };
  Cursor c_next{0, 0};
  const uint32_t q_row_bytes = 2u * (uint32_t)(P.heads * D);
  // Tile at the cursor into slot S: Qs and dO rows (LDS-destination loads) and, in the
  // first 16 lanes of each wave, lse / delta of rows 8 w .. 8 w + 7 into registers.
  // They are written to LDS negated; rows past the segment are clamped on load and get
  // -lse = -inf, -delta = 0 there (P = 0).
  // (loader wavefronts only: 16 rows each, lanes 0-15 lse, 16-31 delta)
  const int pr = 16 * wave + (lane & 15), pwhich = (lane >> 4) & 1;
  // (the array base is chosen from two scalar values, not by indexing the parameter
  // block per lane, which would load the pointer from memory)
  const float* const pbase = pwhich ? P.delta : P.lse;
  const int lse_rows = P.lse_heads > 0 ? P.lse_heads : P.heads;
  // lse / delta run two tiles ahead of the rows (pend[S] holds those of the next tile
  // to use slot S), with one unconditional load per wave per tile so that the number of
  // loads behind a tile's rows is the same in every wave.
  float pend[2] = {0.f, 0.f};
  int pend_last[2] = {0, 0};
  Cursor c_lse{0, 0};
  int lse_left = n_tiles;
  auto pend_load = [&](auto slot) __attribute__((always_inline)) {
    constexpr int S = decltype(slot)::value;
    const Tile T = tile_at(c_lse);
    if (--lse_left > 0) adv(c_lse);  // past the last tile: reload the last one
    const int last = P.seg_rows[T.seg] - 1 - T.r0;
    const size_t t_row = (size_t)P.seg_row0[T.seg] + T.r0 + min(pr, last);
    // delta: [B, H_s, S_loc]; lse: [B, lse_heads, S_loc] from row lse_head0
    const size_t li = pwhich ? ((size_t)b * P.heads + T.head) * P.s_loc + t_row
                             : ((size_t)b * lse_rows + P.lse_head0 + T.head) * P.s_loc + t_row;
    pend[S] = pbase[li];
    pend_last[S] = last;
  };
  auto issue = [&](auto slot) __attribute__((always_inline)) {
    constexpr int S = decltype(slot)::value;
    const Tile T = tile_at(c_next);
    adv(c_next);
    const size_t e0 = (((size_t)b * P.s_loc + P.seg_row0[T.seg] + T.r0) * P.heads + T.head) * D;
    const int last = P.seg_rows[T.seg] - 1 - T.r0;
#pragma unroll
    for (int v = 0; v < 2; ++v) {  // the loader's two shares
      load_tile64<D, kKvWaves>(P.Qs + e0, q_row_bytes, last, Ls + S * T64, wave + v * kKvLoaders,
                               lane);
      load_tile64<D, kKvWaves>(P.dO + e0, q_row_bytes, last, Ls + (2 + S) * T64,
                               wave + v * kKvLoaders, lane);
    }
  };

  // Per-lane LDS offsets (the swizzle of a row depends only on its index mod 16, which
  // the slot, block and k-step offsets preserve): row reads of k-step ks at
  // kad ^ (32 ks); transpose reads of column block eb at tra[eb] / trb[eb].
  const int kad = l32 * C::RB + 16 * (hh ^ C::f(l32));
  const int trr = tr_row(lane), trc = tr_col(lane);
  int tra[C::EB], trb[C::EB];
#pragma unroll
  for (int eb = 0; eb < C::EB; ++eb) {
    tra[eb] = C::off(trr, 32 * eb + trc);
    trb[eb] = C::off(trr + 8, 32 * eb + trc);
  }
  const lds_char* vrows = Ls + VO + 32 * wave * C::RB;  // this wave's 32 V rows

  f32x16 dkT[C::EB], dvT[C::EB];
#pragma unroll
  for (int eb = 0; eb < C::EB; ++eb)
#pragma unroll
    for (int e = 0; e < 16; ++e) dkT[eb][e] = dvT[eb][e] = 0.f;

  // Block HF of the tile in slot S, at position tpos: element 4 g + r of the score /
  // dP accumulators is query row 32 HF + 8 g + 4 hh + r, key `key`.
  auto block = [&](auto slot, auto half, int tpos, int rows_left) __attribute__((always_inline)) {
    constexpr int S = decltype(slot)::value, HF = decltype(half)::value;
    constexpr int QB = S * T64 + HF * 32 * C::RB;  // this block's Qs rows
    constexpr int OB = QB + 2 * T64;                    // and dO rows
    // The accumulators start at -lse and -delta of their query rows (held negated in
    // LDS), so that they end as S - lse and dP - delta.
    const float* nlse = Lf + S * 2 * kQStage + 32 * HF + 4 * hh;
    f32x16 s, dp;
#pragma unroll
    for (int g = 0; g < 4; ++g) {
      const f32x4 l4 = *reinterpret_cast<const f32x4*>(nlse + 8 * g);
      const f32x4 d4 = *reinterpret_cast<const f32x4*>(nlse + kQStage + 8 * g);
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        s[4 * g + r] = l4[r];
        dp[4 * g + r] = d4[r];
      }
    }
#pragma unroll
    for (int ks = 0; ks < C::KS; ++ks) {
      const int o = kad ^ (32 * ks);
      const u32x4 vf = lds_read16(vrows + o);
      s = mfma32(lds_read16(Ls + QB + o), kf[ks], s);
      dp = mfma32(lds_read16(Ls + OB + o), vf, dp);
      // (no operand prefetch across steps: registers are the limit here, and the other
      // wave of the SIMD covers the LDS latency)
      __builtin_amdgcn_sched_barrier(0);
    }
    // Causal mask, only in blocks that cross this wave's diagonal: scores of keys after
    // the query (rel > 8 g + r) become -inf, so P and dS are zero there.
    if (wk0 + 31 > tpos + 32 * HF) {
      const int rel = key - (tpos + 32 * HF + 4 * hh);
#pragma unroll
      for (int e = 0; e < 16; ++e) s[e] = rel > 8 * (e >> 2) + (e & 3) ? -INFINITY : s[e];
    }
    // P = 2^(S - lse), dS = P (dP - delta), packed to bf16 in the accumulator's row order
    // (the B operands below).
    u32x4 pf[2], df[2];
#pragma unroll
    for (int g = 0; g < 4; ++g) {
      float pv[4], dv[4];
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        pv[r] = __builtin_amdgcn_exp2f(s[4 * g + r]);
        dv[r] = pv[r] * dp[4 * g + r];
      }
      pf[g >> 1][2 * (g & 1)] = pack_bf16x2(pv[0], pv[1]);
      pf[g >> 1][2 * (g & 1) + 1] = pack_bf16x2(pv[2], pv[3]);
      df[g >> 1][2 * (g & 1)] = pack_bf16x2(dv[0], dv[1]);
      df[g >> 1][2 * (g & 1) + 1] = pack_bf16x2(dv[2], dv[3]);
    }
    // dV^T += dO^T P and dK^T += Qs^T dS; k-step s2 covers query rows 32 HF + 16 s2 + ..
#pragma unroll
    for (int s2 = 0; s2 < 2; ++s2)
#pragma unroll
      for (int eb = 0; eb < C::EB; ++eb) {
        const lds_char* bq = Ls + QB + 16 * s2 * C::RB;
        const u32x2 olo = lds_read_tr(bq + 2 * T64 + tra[eb]), ohi = lds_read_tr(bq + 2 * T64 + trb[eb]);
        dvT[eb] = mfma32(u32x4{olo[0], olo[1], ohi[0], ohi[1]}, pf[s2], dvT[eb]);
        const u32x2 qlo = lds_read_tr(bq + tra[eb]), qhi = lds_read_tr(bq + trb[eb]);
        dkT[eb] = mfma32(u32x4{qlo[0], qlo[1], qhi[0], qhi[1]}, df[s2], dkT[eb]);
        __builtin_amdgcn_sched_barrier(0);
      }
    (void)rows_left;
  };

  // One tile in slot S: the loaders put its lse / delta into LDS once their shares of
  // its rows have landed and count themselves in; every wavefront waits for all four.
  // Between its two blocks a loader starts the next tile into the other slot (once every
  // wavefront is done with the tile before in that slot) and the lse / delta two tiles
  // on; the older wavefront of a SIMD can so run up to about half a tile ahead of the
  // younger one instead of waiting for it every tile.
  lds_int* const ctr_full = reinterpret_cast<lds_int*>(Ls + VO + VT);
  lds_int* const ctr_empty = ctr_full + 2;
  lds_int* const ctr_gave_up = ctr_full + 4;
  const int polls = P.poll_limit > 0 ? P.poll_limit : kBwdSpinMax;
  const bool loader = wave < kKvLoaders;
  Cursor c_pos{0, 0};
  auto tile = [&](auto slot, int t) __attribute__((always_inline)) {
    constexpr int S = decltype(slot)::value;
    if (loader) {
      asm volatile("s_waitcnt vmcnt(1)" ::: "memory");  // all but tile t + 1's lse / delta
      if (lane < 32)
        Lf[S * 2 * kQStage + pwhich * kQStage + pr] =
            pr <= pend_last[S] ? -pend[S] : (pwhich ? 0.f : -INFINITY);
      bwd_signal(ctr_full + S);  // (LDS operations complete in order)
    }
    bwd_wait_ge(ctr_full + S, kKvLoaders * ((t >> 1) + 1), ctr_gave_up, polls);
    const Tile T = tile_at(c_pos);
    adv(c_pos);
    const int tpos = P.seg_pos0[T.seg] + T.r0;
    block(slot, IC<0>{}, tpos, 0);
    if (loader) {
      if (t + 1 < n_tiles) {
        if (t > 0)
          bwd_wait_ge(ctr_empty + (1 - S), kKvWaves * (((t - 1) >> 1) + 1), ctr_gave_up, polls);
        issue(IC<1 - S>{});
      }
      pend_load(IC<S>{});  // tile t + 2
    }
    if (T.r0 + 32 < P.seg_rows[T.seg]) block(slot, IC<1>{}, tpos, 0);
    bwd_signal(ctr_empty + S);
  };
  if (tid < 5) ctr_full[tid] = 0;
  asm volatile("s_waitcnt vmcnt(0)" ::: "memory");  // this wavefront's V rows
  __syncthreads();  // every V row in LDS; counters zero
  if (n_tiles > 0 && loader) {
    pend_load(IC<0>{});
    issue(IC<0>{});
    pend_load(IC<1>{});
  }
  for (int t = 0; t < n_tiles; t += 2) {
    tile(IC<0>{}, t);
    if (t + 1 < n_tiles) tile(IC<1>{}, t + 1);
  }
  __syncthreads();  // every wavefront is past its last wait
  if (bwd_count(ctr_gave_up) != 0) {
#pragma unroll
    for (int eb = 0; eb < C::EB; ++eb)
#pragma unroll
      for (int e = 0; e < 16; ++e) dkT[eb][e] = dvT[eb][e] = __builtin_nanf("");
  }

  // Accumulator element 4 g + r of block eb: d = 32 eb + 8 g + 4 hh + r, key = `key`.
  if (key < P.seq) {
    float* dkrow = P.dK + ((size_t)b * P.seq + key) * kv_stride + (size_t)kvh * D;
    float* dvrow = P.dV + ((size_t)b * P.seq + key) * kv_stride + (size_t)kvh * D;
#pragma unroll
    for (int eb = 0; eb < C::EB; ++eb)
#pragma unroll
      for (int g = 0; g < 4; ++g) {
        const int c = 32 * eb + 8 * g + 4 * hh;
        f32x4 k4{dkT[eb][4 * g] * kLn2, dkT[eb][4 * g + 1] * kLn2, dkT[eb][4 * g + 2] * kLn2,
                 dkT[eb][4 * g + 3] * kLn2};
        f32x4 v4{dvT[eb][4 * g], dvT[eb][4 * g + 1], dvT[eb][4 * g + 2], dvT[eb][4 * g + 3]};
        if (P.accumulate) {
          k4 += *reinterpret_cast<const f32x4*>(dkrow + c);
          v4 += *reinterpret_cast<const f32x4*>(dvrow + c);
        }
        *reinterpret_cast<f32x4*>(dkrow + c) = k4;
        *reinterpret_cast<f32x4*>(dvrow + c) = v4;
      }
  }
}

// ---------------------------------------------------------------------------------
// Query-stationary kernel: dQ of 128 queries of one head over one range of keys.
//
// Built for two waves per SIMD (at most 256 registers, 64 KB of LDS, two workgroups
// per CU): one wave's vector and LDS phases overlap the other's matrix work.  When the
// (query tile, head, batch) work items alone cannot fill the GPU twice over, each
// tile's keys are split into n_split ranges whose partial dQ (fp32) a second kernel
// sums; with n_split = 1 the workgroup writes bf16 dQ itself.  The K / V tiles go round
// a two-slot ring, unrolled by slot so that LDS addresses are registers plus
// immediates.
template <int D>
__global__ __launch_bounds__(kBwdThreads) __attribute__((amdgpu_waves_per_eu(2, 2)))
void attn_bwd_dq_kernel(const AttnBwdParams P) {
  using C = BwCfg<D>;
  constexpr int T64 = C::T64;
  // [K slot 0][K slot 1][V slot 0][V slot 1]
  __shared__ __attribute__((aligned(1024))) char L[4 * T64];
  lds_char* Ls = (lds_char*)L;

  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int l32 = lane & 31, hh = lane >> 5;

  // Work item -> (batch, head, key range, query tile), query tile fastest; last segment
  // and last tile (most keys) first.
  const int nt0 = (P.seg_rows[0] + kDqTile - 1) / kDqTile;
  const int nt1 = P.n_seg > 1 ? (P.seg_rows[1] + kDqTile - 1) / kDqTile : 0;
  const int n_qt = nt0 + nt1;
  const int w = xcd_work_index(blockIdx.x, n_qt * P.dq_split * P.heads * P.batch);
  const int order = w % n_qt;
  const int seg = order < nt1 ? 1 : 0;
  const int qt = seg == 1 ? nt1 - 1 - order : nt0 - 1 - (order - nt1);
  const int split = (w / n_qt) % P.dq_split;
  const int head = (w / n_qt / P.dq_split) % P.heads;
  const int b = w / n_qt / P.dq_split / P.heads;
  const int seg_rows = P.seg_rows[seg], row0 = P.seg_row0[seg], pos0 = P.seg_pos0[seg];
  const int kvh = P.kv_head0 + head / P.group;
  const int q0 = qt * kDqTile;

  const int qloc = q0 + 32 * wave + l32;  // this lane's query (accumulator column)
  const bool qvalid = qloc < seg_rows;
  const int qpos = pos0 + qloc;
  const bool wave_active = q0 + 32 * wave < seg_rows;
  const int wpos_min = pos0 + q0 + 32 * wave;
  const int wpos_max = pos0 + min(q0 + 32 * wave + 31, seg_rows - 1);
  const int n_keys = pos0 + min(q0 + kDqTile, seg_rows);  // keys this tile can see
  const int k_begin = split * P.dq_split_len;              // a multiple of kKStage
  const int k_end = min(k_begin + P.dq_split_len, n_keys);
  const int j0 = k_begin / kKStage;
  const int n_steps = k_end > k_begin ? (k_end - k_begin + kKStage - 1) / kKStage : 0;

  // Qs and dO fragments of this lane's query (B operands of S^T and dP^T); the score
  // and dP accumulators start from -lse and -delta.
  const size_t qrow = (((size_t)b * P.s_loc + row0 + (qvalid ? qloc : 0)) * P.heads + head) * D;
  u32x4 qf[C::KS], of[C::KS];
#pragma unroll
  for (int s = 0; s < C::KS; ++s) {
    qf[s] = ld16(P.Qs + qrow + 16 * s + 8 * hh);
    of[s] = ld16(P.dO + qrow + 16 * s + 8 * hh);
  }
  const size_t li = ((size_t)b * P.heads + head) * P.s_loc + row0 + (qvalid ? qloc : 0);
  const size_t li_lse = ((size_t)b * (P.lse_heads > 0 ? P.lse_heads : P.heads) + P.lse_head0 +
                         head) * P.s_loc + row0 + (qvalid ? qloc : 0);
  const float neg_lse = qvalid ? -P.lse[li_lse] : -INFINITY;  // invalid query: P = 0
  const float neg_del = qvalid ? -P.delta[li] : 0.f;
  // Consume these loads before the loop: the compiler then waits for them once, not at
  // a point inside the loop where the same wait would also cover the newest key tiles.
#pragma unroll
  for (int s = 0; s < C::KS; ++s) asm volatile("" ::"v"(qf[s]), "v"(of[s]));
  asm volatile("" ::"v"(neg_lse), "v"(neg_del));

  const size_t kv_stride = (size_t)P.n_kv * D;
  const uint32_t kv_row_bytes = 2u * (uint32_t)kv_stride;
  const uint16_t* kbase = P.Kb + (size_t)b * P.seq * kv_stride + (size_t)kvh * D;
  const uint16_t* vbase = P.Vb + (size_t)b * P.seq * kv_stride + (size_t)kvh * D;
  // Keys of stage j into slot j % 2; keys at or past k_end repeat the range's last key
  // (it either ends at a multiple of the stage or at n_keys, past every query here).
  auto issue = [&](int j) __attribute__((always_inline)) {
    const int key0 = j * kKStage, slot = (j - j0) & 1;
    const int last = k_end - 1 - key0;
    load_tile64<D>(kbase + (size_t)key0 * kv_stride, kv_row_bytes, last, Ls + slot * T64, wave, lane);
    load_tile64<D>(vbase + (size_t)key0 * kv_stride, kv_row_bytes, last, Ls + (2 + slot) * T64,
                   wave, lane);
  };

  f32x16 dqT[C::EB];
#pragma unroll
  for (int eb = 0; eb < C::EB; ++eb)
#pragma unroll
    for (int e = 0; e < 16; ++e) dqT[eb][e] = 0.f;

  // Per-lane LDS offsets: row reads of k-step ks at ka ^ (32 ks); transpose reads of
  // column block eb at tra[eb] (rows trr) and trb[eb] (rows trr + 8).
  const int ka = l32 * C::RB + 16 * (hh ^ C::f(l32));
  const int trr = tr_row(lane), trc = tr_col(lane);
  int tra[C::EB], trb[C::EB];
#pragma unroll
  for (int eb = 0; eb < C::EB; ++eb) {
    tra[eb] = C::off(trr, 32 * eb + trc);
    trb[eb] = C::off(trr + 8, 32 * eb + trc);
  }

  // One step: the 64 keys of stage j (slot SLOT) in two blocks of 32.
  auto step = [&](auto slot, int j) __attribute__((always_inline)) {
    constexpr int S = decltype(slot)::value;
    wait_dma();
    __syncthreads();  // stage j resident; every wave is done with stage j - 1
    if (j + 1 < j0 + n_steps) issue(j + 1);
    if (!wave_active) return;
#pragma unroll
    for (int kb = 0; kb < kKStage / 32; ++kb) {
      const int kbase0 = j * kKStage + 32 * kb;
      if (kbase0 > wpos_max) break;  // every key after every query
      constexpr int KO = S * T64;    // this slot's K tile; the V tile follows at 2 T64
      f32x16 s, dp;
#pragma unroll
      for (int e = 0; e < 16; ++e) {
        s[e] = neg_lse;
        dp[e] = neg_del;
      }
#pragma unroll
      for (int ks = 0; ks < C::KS; ++ks) {
        const int o = (ka ^ (32 * ks)) + 32 * kb * C::RB;
        s = mfma32(lds_read16(Ls + KO + o), qf[ks], s);
        dp = mfma32(lds_read16(Ls + KO + 2 * T64 + o), of[ks], dp);
      }
      // Element 4 g + r: key kbase0 + 8 g + 4 hh + r, this lane's query.
      float pv[16];
#pragma unroll
      for (int e = 0; e < 16; ++e) pv[e] = __builtin_amdgcn_exp2f(s[e]);
      if (kbase0 + 31 > wpos_min) {  // the block crosses this wave's diagonal
        const int rel = qpos - kbase0 - 4 * hh;  // key offset 8 g + r must be <= rel
#pragma unroll
        for (int e = 0; e < 16; ++e) pv[e] = 8 * (e >> 2) + (e & 3) > rel ? 0.f : pv[e];
      }
      u32x4 df[2];
#pragma unroll
      for (int h = 0; h < 2; ++h)
#pragma unroll
        for (int q = 0; q < 4; ++q)
          df[h][q] = pack_bf16x2(pv[8 * h + 2 * q] * dp[8 * h + 2 * q],
                                 pv[8 * h + 2 * q + 1] * dp[8 * h + 2 * q + 1]);
      // dQ^T += K^T dS^T; k-step s2 covers keys 32 kb + 16 s2 + ..
#pragma unroll
      for (int s2 = 0; s2 < 2; ++s2)
#pragma unroll
        for (int eb = 0; eb < C::EB; ++eb) {
          const int ro = (32 * kb + 16 * s2) * C::RB;
          const u32x2 lo = lds_read_tr(Ls + KO + ro + tra[eb]);
          const u32x2 hi = lds_read_tr(Ls + KO + ro + trb[eb]);
          dqT[eb] = mfma32(u32x4{lo[0], lo[1], hi[0], hi[1]}, df[s2], dqT[eb]);
        }
    }
  };

  if (n_steps > 0) issue(j0);
  for (int j = j0; j < j0 + n_steps; j += 2) {
    step(IC<0>{}, j);
    if (j + 1 < j0 + n_steps) step(IC<1>{}, j + 1);
  }

  if (!qvalid) return;
  // Element 4 g + r of block eb: d = 32 eb + 8 g + 4 hh + r of this lane's query.
  if (P.dq_split == 1) {
    uint16_t* dqrow = P.dQ + qrow;
#pragma unroll
    for (int eb = 0; eb < C::EB; ++eb)
#pragma unroll
      for (int g = 0; g < 4; ++g)
        *reinterpret_cast<u32x2*>(dqrow + 32 * eb + 8 * g + 4 * hh) =
            u32x2{pack_bf16x2(dqT[eb][4 * g] * P.scale, dqT[eb][4 * g + 1] * P.scale),
                  pack_bf16x2(dqT[eb][4 * g + 2] * P.scale, dqT[eb][4 * g + 3] * P.scale)};
  } else {
    const size_t rows = (size_t)P.batch * P.s_loc * P.heads;
    float* prow = P.dq_part + ((size_t)split * rows +
                               ((size_t)b * P.s_loc + row0 + qloc) * P.heads + head) * D;
#pragma unroll
    for (int eb = 0; eb < C::EB; ++eb)
#pragma unroll
      for (int g = 0; g < 4; ++g)
        *reinterpret_cast<f32x4*>(prow + 32 * eb + 8 * g + 4 * hh) =
            f32x4{dqT[eb][4 * g], dqT[eb][4 * g + 1], dqT[eb][4 * g + 2], dqT[eb][4 * g + 3]};
  }
}

// Sums the key-range partials of dQ: dQ = bf16(scale sum_c part_c), 4 columns a thread.
__global__ __launch_bounds__(256) void attn_bwd_dq_combine_kernel(const AttnBwdParams P) {
  const long long n4 = (long long)P.batch * P.s_loc * P.heads * P.head_dim / 4;
  const long long i = (long long)blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= n4) return;
  f32x4 acc = {0.f, 0.f, 0.f, 0.f};
  for (int c = 0; c < P.dq_split; ++c)
    acc += *reinterpret_cast<const f32x4*>(P.dq_part + ((size_t)c * n4 + i) * 4);
  *reinterpret_cast<u32x2*>(P.dQ + 4 * i) =
      u32x2{pack_bf16x2(acc[0] * P.scale, acc[1] * P.scale),
            pack_bf16x2(acc[2] * P.scale, acc[3] * P.scale)};
}

// ---------------------------------------------------------------------------------
// out[n][m] = in[m][n] for m < rows, n < cols; out[n][m] = 0 for rows <= m < ld_out.
// 64 x 64 tiles through LDS; 16-byte loads and stores.
__global__ __launch_bounds__(256) void transpose_bf16_kernel(const uint16_t* in, int ld_in,
                                                             int rows, int cols, uint16_t* out,
                                                             int ld_out) {
  __shared__ uint16_t T[64][64 + 2];
  const int m0 = blockIdx.x * 64, n0 = blockIdx.y * 64;
  const int tid = threadIdx.x;
#pragma unroll
  for (int k = 0; k < 2; ++k) {
    const int i = tid + 256 * k;          // 512 chunks of 8 elements
    const int r = i >> 3, c8 = (i & 7) * 8;
    const int m = m0 + r, n = n0 + c8;
    u32x4 v = {0u, 0u, 0u, 0u};
    if (m < rows) {
      if (n + 8 <= cols) {
        v = ld16(in + (size_t)m * ld_in + n);
      } else {
        for (int e = 0; e < 8; ++e)
          if (n + e < cols) {
            const uint32_t x = in[(size_t)m * ld_in + n + e];
            v[e >> 1] |= (e & 1) ? (x << 16) : x;
          }
      }
    }
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      T[r][c8 + 2 * e] = (uint16_t)(v[e] & 0xffffu);
      T[r][c8 + 2 * e + 1] = (uint16_t)(v[e] >> 16);
    }
  }
  __syncthreads();
#pragma unroll
  for (int k = 0; k < 2; ++k) {
    const int i = tid + 256 * k;
    const int nr = i >> 3, m8 = (i & 7) * 8;  // output row n0 + nr, columns m0 + m8 ..
    const int n = n0 + nr, m = m0 + m8;
    if (n >= cols || m >= ld_out) continue;
    u32x4 v;
#pragma unroll
    for (int e = 0; e < 4; ++e)
      v[e] = (uint32_t)T[m8 + 2 * e][nr] | ((uint32_t)T[m8 + 2 * e + 1][nr] << 16);
    st16(out + (size_t)n * ld_out + m, v);
  }
}

hipError_t check_bwd(const AttnBwdParams& p) {
  if (p.n_seg < 1 || p.n_seg > 2 || p.group < 1 || p.heads % p.group != 0 || p.seq < 1 ||
      p.seq > (1LL << 30) || (p.head_dim != 64 && p.head_dim != 128))
    return hipErrorInvalidValue;
  int rows = 0;
  for (int k = 0; k < p.n_seg; ++k) {
    if (p.seg_rows[k] < 1 || p.seg_row0[k] != rows || p.seg_pos0[k] < 0 ||
        (long long)p.seg_pos0[k] + p.seg_rows[k] > p.seq)
      return hipErrorInvalidValue;
    rows += p.seg_rows[k];
  }
  if (rows != p.s_loc || p.kv_head0 < 0 || p.kv_head0 + p.heads / p.group > p.n_kv)
    return hipErrorInvalidValue;
  // Byte offsets inside one staged tile must fit the 32-bit buffer offsets.
  if ((long long)kKStage * p.n_kv * p.head_dim * 2 >= (1LL << 31) ||
      (long long)kQStage * p.heads * p.head_dim * 2 >= (1LL << 31))
    return hipErrorInvalidValue;
  return hipSuccess;
}

bool bwd_empty(const AttnBwdParams& p) { return p.batch <= 0 || p.s_loc <= 0 || p.heads <= 0; }

}  // namespace

hipError_t launch_attn_bwd_prep(const AttnBwdParams& p, hipStream_t s) {
  if (bwd_empty(p)) return hipSuccess;
  const hipError_t e = check_bwd(p);
  if (e != hipSuccess) return e;
  void* args[] = {const_cast<AttnBwdParams*>(&p)};
  const long long threads = (long long)p.batch * p.s_loc * p.heads * (p.head_dim / 8);
  const void* fn = p.head_dim == 128 ? reinterpret_cast<const void*>(&attn_bwd_prep_kernel<128>)
                                     : reinterpret_cast<const void*>(&attn_bwd_prep_kernel<64>);
  return hipLaunchKernel(fn, dim3((unsigned)((threads + 255) / 256)), dim3(256), args, 0, s);
}

hipError_t launch_attn_bwd_dkdv(const AttnBwdParams& p_in, hipStream_t s) {
  if (bwd_empty(p_in)) return hipSuccess;
  const hipError_t e = check_bwd(p_in);
  if (e != hipSuccess) return e;
  AttnBwdParams p = p_in;
  p.poll_limit = attn_poll_limit();
  void* args[] = {&p};
  const int n_kt = (int)((p.seq + kKvTile - 1) / kKvTile);
  const void* fn = p.head_dim == 128 ? reinterpret_cast<const void*>(&attn_bwd_dkdv_kernel<128>)
                                     : reinterpret_cast<const void*>(&attn_bwd_dkdv_kernel<64>);
  return hipLaunchKernel(fn, dim3(n_kt * (p.heads / p.group) * p.batch), dim3(kKvThreads), args,
                         0, s);
}

hipError_t launch_attn_bwd_dq(const AttnBwdParams& p, hipStream_t s) {
  if (bwd_empty(p)) return hipSuccess;
  const hipError_t e = check_bwd(p);
  if (e != hipSuccess) return e;
  void* args[] = {const_cast<AttnBwdParams*>(&p)};
  int n_qt = 0, max_keys = 0;
  for (int k = 0; k < p.n_seg; ++k) {
    n_qt += (p.seg_rows[k] + kDqTile - 1) / kDqTile;
    max_keys = max(max_keys, p.seg_pos0[k] + p.seg_rows[k]);
  }
  if (p.dq_split < 1 || p.dq_split_len % kKStage != 0 ||
      (long long)p.dq_split * p.dq_split_len < max_keys || (p.dq_split > 1 && !p.dq_part))
    return hipErrorInvalidValue;
  const void* fn = p.head_dim == 128 ? reinterpret_cast<const void*>(&attn_bwd_dq_kernel<128>)
                                     : reinterpret_cast<const void*>(&attn_bwd_dq_kernel<64>);
  const hipError_t e2 = hipLaunchKernel(fn, dim3(n_qt * p.dq_split * p.heads * p.batch),
                                        dim3(kBwdThreads), args, 0, s);
  if (e2 != hipSuccess || p.dq_split == 1) return e2;
  const long long n4 = (long long)p.batch * p.s_loc * p.heads * p.head_dim / 4;
  return hipLaunchKernel(reinterpret_cast<const void*>(&attn_bwd_dq_combine_kernel),
                         dim3((unsigned)((n4 + 255) / 256)), dim3(256), args, 0, s);
}

int attn_bwd_dq_split(const AttnBwdParams& p, int* split_len) {
  // Enough (query tile, head, batch, key range) items for two workgroups per CU, each
  // range at least four key stages long.
  int n_qt = 0, max_keys = 1;
  for (int k = 0; k < p.n_seg; ++k) {
    n_qt += (p.seg_rows[k] + kDqTile - 1) / kDqTile;
    max_keys = max(max_keys, p.seg_pos0[k] + p.seg_rows[k]);
  }
  const long long items = (long long)n_qt * p.heads * p.batch;
  int n = 1;
  while (n < 4 && items * n < 2LL * kAttnTargetWorkgroups) ++n;
  auto len_of = [&](int c) {
    const int len = (max_keys + c - 1) / c;
    return (len + kKStage - 1) / kKStage * kKStage;
  };
  while (n > 1 && len_of(n) < 4 * kKStage) --n;
  if (split_len) *split_len = len_of(n);
  return n;
}

hipError_t launch_transpose_bf16(const uint16_t* in, int ld_in, int rows, int cols,
                                 uint16_t* out, int ld_out, hipStream_t s) {
  if (rows < 0 || cols <= 0 || ld_out < rows || ld_out % 8 != 0) return hipErrorInvalidValue;
  if (ld_out == 0) return hipSuccess;
  const dim3 grid((ld_out + 63) / 64, (cols + 63) / 64);
  void* args[] = {const_cast<uint16_t**>(&in), &ld_in, &rows, &cols, &out, &ld_out};
  return hipLaunchKernel(reinterpret_cast<const void*>(&transpose_bf16_kernel), grid, dim3(256),
                         args, 0, s);
}

}  // namespace tsp
