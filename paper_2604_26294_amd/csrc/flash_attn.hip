// Causal flash attention of one TSP rank's query chunk (gfx950, bf16 MFMA).
//
// Algorithm 1's CausalAttn calls: the rank's local queries form one segment of
// consecutive global positions (contiguous chunks: rank p's rows start at p S_loc) or
// two (the zigzag shard's chunks p and 2D-1-p, the two CausalAttn calls with bounds
// s1 and s2); a query at position t sees keys j <= t of the gathered K/V (held
// resident, in sequence order, in a [B, S, n_kv, d] buffer).  The softmax is computed
// online, one key tile at a time, so the (S_loc x S) score matrix never exists.
//
// Work split.  A workgroup owns 256 queries of one head (GQA: head i reads kv head
// i / g) and one contiguous range of keys; it has 8 wavefronts, two per SIMD, and
// wavefront w handles queries 32 w .. 32 w + 31 against every key of the range.  The
// K and V tiles staged in LDS are what each CU pulls through its load path, so the
// number of queries sharing a tile sets the load traffic per MFMA; 256 halves it
// against 128-query tiles.  When (query tiles x heads x batch) alone would leave CUs
// idle, each query tile's keys are split into n_split ranges handled by different
// workgroups, which write unnormalised partial results (O, reference, sum) that a
// second kernel combines; with n_split = 1 the workgroup writes bf16 O itself.  Key
// tiles beyond the last query's position are never loaded, and only tiles that cross
// a wavefront's diagonal are masked.
//
// Scores are computed transposed, S^T = K Q^T, with K as the MFMA A operand and Q
// (held in registers) as B.  The 32 x 32 accumulator then gives each lane 16 keys of
// ONE query (its partner lane l ^ 32 holds the other 16), so the row max needs one
// cross-lane exchange and the row sum none until the end.  The probabilities P^T
// feed O^T = V^T P^T directly as the B operand (contraction over keys).
//
// Schedule.  Per step every wavefront takes the 128-key tile j in two 64-key halves
// (scores, softmax, P V each), while tile j+1 of K and V streams into the other slot
// of the two-slot rings.  The first tile of a key range also forms each half's row
// maximum (the online softmax's reference); later tiles skip it unless a half's
// probabilities outgrow the reference (see the softmax state below): with two
// wavefronts per SIMD the kernel is bound by instruction issue, so the vector work
// per score is what sets its speed.  The slots are handed over through counters in
// LDS rather than a workgroup barrier per step: the older wavefront of each SIMD
// (the one the arbiter favours, which also issues the tile loads) may then run up to
// about half a step ahead of the younger one instead of waiting for it every step.
// (Variants that delay P V by a step so the two wavefronts of a SIMD alternate matrix
// and vector phases measured slower, as did deeper rings, loads spread across the
// step, and separate K and V counters that let the older wavefront run a whole step
// ahead.)
//
// Data movement.  K and V tiles go from HBM straight into LDS (buffer loads with an
// LDS destination, no register staging) in their natural [key][d] layout, 16-byte
// chunks XOR-swizzled by a function of the row chosen per tile kind so that its reads
// are bank-conflict free.  The V^T operand is read with the gfx950 LDS transpose read
// (ds_read_b64_tr_b16): in each 16-lane group, source lane s points at row
// kbase + s/4, columns base + 4 (s % 4), and lane t receives column base + t of rows
// kbase .. kbase+3 -- four consecutive keys of one head-dim column.  Because tile rows
// are aligned to the row size and the swizzle only touches the in-row offset, every
// LDS read address is (per-lane base XOR a constant) + an immediate offset.
#include <math.h>

#include <atomic>

#include <functional>
#include <mutex>
#include <queue>
#include <type_traits>
#include <vector>

#include "common.h"
#include "internal.h"
#include "lds_dma.h"

namespace tsp {
namespace {

constexpr int kThreads = 512;
constexpr int kWaves = kThreads / kWave;
constexpr int kQTile = 32 * kWaves;  // queries per workgroup
constexpr int kStepKeys = 128;       // keys staged per step
static_assert(kQTile == kAttnQueryTile && kStepKeys == kAttnKeyStep, "tile sizes");
constexpr int kHalfKeys = 64;        // keys per sub-step
constexpr float kRescaleLog2 = 8.f;  // lazy-rescale threshold (exp2 units)
// After a query's first key tile its reference is left in place while the row sum stays
// below this bound (which also catches an overflow to inf): the normalised result does not
// depend on the reference, only the range of the fp32 / bf16 values does.
constexpr float kSumLimit = 0x1p40f;

template <int D>
struct FaCfg {
  static constexpr int KCH = D / 8;                           // 16-byte chunks per key row
  static constexpr int ROW_BYTES = D * 2;
  static constexpr int TILE_BYTES = kStepKeys * ROW_BYTES;    // one K or V tile
  static constexpr int ROWS_PER_DMA = kWave / KCH;            // rows one wave instruction fills
  static constexpr int DMA_PER_LANE = kStepKeys / (kWaves * ROWS_PER_DMA);
  static constexpr int EB = D / 32;                           // 32-row blocks of O^T
  static constexpr int KS = D / 16;                           // contraction steps of S^T
  static constexpr int RPW = 256 / ROW_BYTES;                 // rows per 256-byte bank window
  static_assert(DMA_PER_LANE * kWaves * ROWS_PER_DMA == kStepKeys, "DMA cover");
  // Chunk swizzles (physical 16-byte chunk = logical chunk XOR f(row)).  LDS has 64
  // banks of 4 bytes, so a row's bank window position is (row mod RPW) and its chunk.
  // K tiles are read 16 rows x one chunk per 16 lanes (ds_read_b128): f_K gives those
  // rows distinct windows.  V tiles are read by 8-byte transpose reads, 4 rows x 4
  // chunks per half-wave: f_V moves each of the 4 rows to its own 64-byte block.
  __device__ static int fk(int row) { return (row / RPW) & (KCH - 1); }
  __device__ static int fv(int row) { return 4 * ((row / RPW) & (KCH / 4 - 1)); }
};

template <int N>
using IC = std::integral_constant<int, N>;

// x combined with the value of lane l ^ 32.  v_permlane32_swap exchanges the upper 32
// lanes of its first operand with the lower 32 lanes of its second, so with both
// holding x they become [x_lo, x_lo] and [x_hi, x_hi]; a VALU op, where a shuffle
// through LDS (ds_bpermute) would wait on every LDS read still in flight.  Written as
// asm: this compiler folds the builtin's second result away.
__device__ __forceinline__ void swap_halves(float& a, float& b) {
  asm volatile("s_nop 1\n\tv_permlane32_swap_b32 %0, %1\n\ts_nop 1" : "+v"(a), "+v"(b));
}
__device__ __forceinline__ float max_with_partner(float x) {
  float a = x, b = x;
  swap_halves(a, b);
  return fmaxf(a, b);
}
__device__ __forceinline__ float sum_with_partner(float x) {
  float a = x, b = x;
  swap_halves(a, b);
  return a + b;
}

// Per-slot synchronisation of the K/V ring through counters in LDS (instead of a
// workgroup barrier per step).  The counters only grow within a query tile: slot s's
// "full" count gains one per loader wavefront whose share of the slot's tile has landed,
// its "empty" count one per wavefront done reading the slot.  A wait spins on the count
// with s_sleep and gives up after kSpinMax polls, so an error in the protocol can never
// hang the kernel.  A wavefront remembers in a register whether one of its waits gave
// up and raises the query tile's flag once, after its last step; the tile's results are
// then written as NaN (a loud wrong result rather than a quiet one).  The spin loop has
// a compile-time bound and nothing but the poll in it: the pattern in which the
// workgroups of an XCD reuse each other's K/V tiles in L2 turned out to depend on that
// loop's code (a flag store inside it raised the launch's HBM fetch by half).
typedef __attribute__((address_space(3))) int lds_int;
constexpr int kSpinMax = 4096;
constexpr int kLoaders = kWaves / 2;  // the older wavefront of each SIMD loads the tiles
__device__ __forceinline__ void lds_signal(lds_int* p) {
  if ((threadIdx.x & 63) == 0)
    asm volatile("ds_add_u32 %0, %1" ::"v"((uint32_t)(uintptr_t)p), "v"(1u) : "memory");
}
__device__ __forceinline__ int lds_read_count(lds_int* p) {
  int v;
  asm volatile("ds_read_b32 %0, %1\n\ts_waitcnt lgkmcnt(0)"
               : "=v"(v) : "v"((uint32_t)(uintptr_t)p) : "memory");
  return __builtin_amdgcn_readfirstlane(v);
}
// True once the count at p reaches target; false after `polls` polls.
__device__ __forceinline__ bool lds_wait_ge(lds_int* p, int target, int polls) {
  for (int i = 0; i < polls; ++i) {
    if (lds_read_count(p) >= target) return true;
    __builtin_amdgcn_s_sleep(1);
  }
  return false;
}

// One query tile of the kernel: tile `order` in the kernel's tile order (see
// flash_fwd_kernel), key range `split`, query head `head` of batch entry `b`; K/V slots
// in Ls.  A wavefront may return while others still read the slots: the caller's next
// tile may refill them only after a barrier.  kPollArg: the slot waits give up after
// P.poll_limit polls instead of kSpinMax (the instantiation behind the test hook that
// caps the polls; every other launch uses the compile-time bound).
template <int D, bool LSE, bool kPollArg>
__device__ __forceinline__ void flash_tile(const AttnParams& P, lds_char* Ls, const int nt0,
                                           const int nt1, const int order, const int split,
                                           const int head, const int b) {
  using C = FaCfg<D>;
  constexpr int KCH = C::KCH, RB = C::ROW_BYTES, TB = C::TILE_BYTES;
  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int l32 = lane & 31, hh = lane >> 5;
  const int seg = order < nt1 ? 1 : 0;
  const int qt = seg == 1 ? nt1 - 1 - order : nt0 - 1 - (order - nt1);
  const int q0 = qt * kQTile;                    // first query of the tile, within its segment
  const int seg_rows = P.seg_rows[seg], row0 = P.seg_row0[seg], pos0 = P.seg_pos0[seg];
  const int kvh = P.kv_head0 + head / P.group;
  const size_t ld = P.ld > 0 ? (size_t)P.ld : (size_t)P.heads * D;  // Q / O token row stride

  const int qloc = q0 + 32 * wave + l32;         // within the segment
  const bool qvalid = qloc < seg_rows;
  const int qpos = pos0 + qloc;
  const int wq_first = q0 + 32 * wave;
  const bool wave_active = wq_first < seg_rows;
  const int wpos_min = pos0 + wq_first;
  const int wpos_max = pos0 + min(wq_first + 31, seg_rows - 1);
  const int n_keys = pos0 + min(q0 + kQTile, seg_rows);  // keys this tile can see
  const int k_begin = split * P.split_len;                   // a multiple of kStepKeys
  const int k_end = min(k_begin + P.split_len, n_keys);
  const int j0 = k_begin / kStepKeys;
  const int n_steps = k_end > k_begin ? (k_end - k_begin + kStepKeys - 1) / kStepKeys : 0;

  // Q fragments (the B operand of S^T): lane holds Q[qloc][16 ks + 8 hh .. +7].  Q
  // arrives multiplied by softmax scale * log2(e) (and rounded once), so the score
  // MFMAs produce base-2 logits directly.
  u32x4 qf[C::KS];
  {
    const uint16_t* qrow =
        P.Q + ((size_t)b * P.s_loc + row0 + (qvalid ? qloc : 0)) * ld + (size_t)head * D;
#pragma unroll
    for (int s = 0; s < C::KS; ++s)
      qf[s] = qvalid ? ld16(qrow + 16 * s + 8 * hh) : u32x4{0u, 0u, 0u, 0u};
    // Take the loads' wait here, before any tile load is issued: left to the compiler,
    // the wait lands inside the key loop (ahead of the first score MFMA of every step),
    // where vmcnt(0) would also wait for the next tile's loads.
#pragma unroll
    for (int s = 0; s < C::KS; ++s) asm volatile("" : "+v"(qf[s]));
  }
  const size_t kv_stride = (size_t)P.n_kv * D;  // elements between consecutive keys
  const uint16_t* kbase = P.Kb + (size_t)b * P.seq * kv_stride + (size_t)kvh * D;
  const uint16_t* vbase = P.Vb + (size_t)b * P.seq * kv_stride + (size_t)kvh * D;

  // DMA geometry: instruction i of wave w fills rows (i kWaves + w) ROWS_PER_DMA + lane / KCH,
  // physical chunk lane % KCH, with the logical chunk that the tile's swizzle puts there
  // (the swizzle depends on the row only through bits that are the same for every i).
  // A full tile's source is (scalar tile base) + (scalar i * row step) + (per-lane 32-bit
  // offset), so its loads need no vector arithmetic.
  // The loader wavefront w (w < kLoaders) issues the instructions of shares w and
  // w + kLoaders; share w + kLoaders's rows are kShareRows further on and have the same
  // swizzle (which depends on the row only through (row / RPW) mod KCH).
  constexpr int kRowStep = kWaves * C::ROWS_PER_DMA;  // rows between instructions
  constexpr int kShareRows = kLoaders * C::ROWS_PER_DMA;
  static_assert(kShareRows % (C::RPW * KCH) == 0, "shares w and w + kLoaders swizzle alike");
  const int dma_row0 = wave * C::ROWS_PER_DMA + lane / KCH;
  const int dma_col_k = 8 * ((lane % KCH) ^ C::fk(dma_row0));
  const int dma_col_v = 8 * ((lane % KCH) ^ C::fv(dma_row0));
  const uint32_t row_bytes = 2u * (uint32_t)kv_stride;
  const uint32_t dma_off_k = (uint32_t)dma_row0 * row_bytes + 2u * dma_col_k;
  const uint32_t dma_off_v = (uint32_t)dma_row0 * row_bytes + 2u * dma_col_v;
  const uint32_t dma_step = (uint32_t)kRowStep * row_bytes;
  // One 128-key tile from HBM into an LDS slot.  In the last tile of the key range,
  // rows at or past k_end are clamped to its last key: the range either ends at a
  // multiple of the tile size or at n_keys, and keys >= n_keys are past every query
  // of this workgroup, so those rows are always masked and merely need to be finite.
  auto dma_share = [&](const uint16_t* base, uint32_t lane_off, int col, int v, int tile,
                       int slot_off) __attribute__((always_inline)) {
    const int key0 = tile * kStepKeys;
    const rsrc_t rsrc = make_rsrc(base + (size_t)key0 * kv_stride);
    lds_char* dst = Ls + slot_off + (wave + v * kLoaders) * (kWave * 16);
    const uint32_t share_off = (uint32_t)(v * kShareRows) * row_bytes;
    if (key0 + kStepKeys <= k_end) {
#pragma unroll
      for (int i = 0; i < C::DMA_PER_LANE; ++i)
        dma16(rsrc, lane_off, share_off + i * dma_step, dst + i * kWaves * (kWave * 16));
    } else {
      const int last = k_end - 1 - key0;
#pragma unroll
      for (int i = 0; i < C::DMA_PER_LANE; ++i) {
        const uint32_t row = (uint32_t)min(dma_row0 + v * kShareRows + i * kRowStep, last);
        dma16(rsrc, row * row_bytes + 2u * col, 0u, dst + i * kWaves * (kWave * 16));
      }
    }
  };
  // K and V of tile `tile` into slot S: the calling loader's two shares.
  auto load_tile = [&](int tile, int S) __attribute__((always_inline)) {
#pragma unroll
    for (int v = 0; v < 2; ++v) {
      dma_share(kbase, dma_off_k, dma_col_k, v, tile, S * TB);
      dma_share(vbase, dma_off_v, dma_col_v, v, tile, (2 + S) * TB);
    }
  };
  lds_int* const ctr_full = reinterpret_cast<lds_int*>(Ls + 4 * TB);
  lds_int* const ctr_empty = ctr_full + 2;
  lds_int* const ctr_gave_up = ctr_full + 4;
  const int polls = kPollArg ? P.poll_limit : kSpinMax;
  bool gave_up = false;  // one of this wavefront's waits gave up (wave-uniform)
  const bool loader = wave < kLoaders;

  // LDS read addresses.  Slot offsets and block strides are compile-time immediates;
  // the per-lane parts below are computed once.
  //  K operand: row 64 h + 32 bb + l32, logical chunk 2 ks + hh  ->  byte
  //    (64 h + 32 bb) RB + (ka ^ 32 ks),  ka = l32 RB + 16 (hh ^ f_K(l32)).
  //  V^T operand (transpose reads): rows 64 h + 32 bb + 16 s2 + tr_row (+8 for elements
  //    4-7), columns 32 eb + tr_col  ->  byte (64 h + 32 bb + 16 s2) RB + (va or vb)[eb].
  int kad[C::KS];
  {
    const int ka = l32 * RB + 16 * (hh ^ C::fk(l32));
#pragma unroll
    for (int ks = 0; ks < C::KS; ++ks) kad[ks] = ka ^ (32 * ks);
  }
  const int tr_t = lane & 15, tr_g = lane >> 4;
  const int tr_row = ((tr_g >> 1) << 2) + (tr_t >> 2);     // 4 hh + t / 4
  const int tr_col = 16 * (tr_g & 1) + 4 * (tr_t & 3);     // within a 32-column block
  int va[C::EB], vb[C::EB];
  {
    const int cl = tr_col >> 3, half8 = 8 * ((tr_col >> 2) & 1);
    const int xa = C::fv(tr_row), xb = C::fv(tr_row + 8);
    const int base_a = tr_row * RB + 16 * (cl ^ xa) + half8;
    const int base_b = (tr_row + 8) * RB + 16 * (cl ^ xb) + half8;
#pragma unroll
    for (int eb = 0; eb < C::EB; ++eb) {
      va[eb] = 2 * TB + (base_a ^ (64 * eb));
      vb[eb] = 2 * TB + (base_b ^ (64 * eb));
    }
  }

  // Half h of tile j has keys this wavefront's queries can see.
  auto half_active = [&](int j, int h) __attribute__((always_inline)) {
    return wave_active && j * kStepKeys + kHalfKeys * h <= wpos_max;
  };

  // Online-softmax state of this lane's query (shared with its partner lane l ^ 32).
  // Scores are produced relative to the reference mref (the score MFMAs start from the
  // accumulator value -mref), so o = sum 2^(s - mref) v and l = sum 2^(s - mref); the
  // normalised result o / l does not depend on mref, which only has to keep the values
  // in range.  In the first key tile of the range (which holds the first key every query
  // of the range sees) mref is set from the row maximum: it moves to the first visible
  // score and whenever a score exceeds it by more than kRescaleLog2.  After that the row
  // maximum is not formed: while the row sum stays below kSumLimit (so every probability
  // since mref last moved is below it, and none overflowed) mref stays; a 64-key half
  // that takes the sum past it takes the first tile's path instead and is formed again.
  f32x16 o[C::EB];
#pragma unroll
  for (int eb = 0; eb < C::EB; ++eb)
#pragma unroll
    for (int e = 0; e < 16; ++e) o[eb][e] = 0.f;
  float mref = 0.f, l_run = 0.f;
  bool seen = false;
  f32x16 negm;
#pragma unroll
  for (int e = 0; e < 16; ++e) negm[e] = 0.f;
  f32x16 sc[2][2];  // scores of the two 64-key halves of a tile, 2 blocks of 32 keys each
  u32x4 pf[2][2][2];  // bf16 probabilities of the halves (B operands of P V)

  // S^T - mref of half H of the tile in slot SLOT: 2 blocks of 32 keys x 32 queries.
  // The K fragments are read two contraction steps ahead of their MFMAs, in the source
  // order itself: at this register count the compiler keeps the order it is given, and
  // an MFMA whose operand read was issued just before it waits out the LDS latency.
  auto scores = [&](auto slot, auto half) __attribute__((always_inline)) {
    constexpr int S = decltype(slot)::value, H = decltype(half)::value;
    auto kread = [&](int ks, int bb) __attribute__((always_inline)) {
      return lds_read16(Ls + kad[ks] + (S * TB + (kHalfKeys * H + 32 * bb) * RB));
    };
    u32x4 kf[2][2];
#pragma unroll
    for (int ks = 0; ks < 2; ++ks)
#pragma unroll
      for (int bb = 0; bb < 2; ++bb) kf[ks][bb] = kread(ks, bb);
#pragma unroll
    for (int ks = 0; ks < C::KS; ++ks)
#pragma unroll
      for (int bb = 0; bb < 2; ++bb) {
        sc[H][bb] = mfma32(kf[ks & 1][bb], qf[ks], ks == 0 ? negm : sc[H][bb]);
        if (ks + 2 < C::KS) kf[ks & 1][bb] = kread(ks + 2, bb);
      }
  };
  // Issue order for a block holding only score MFMAs: K fragments two contraction steps
  // ahead of their MFMAs, so the LDS latency hides behind the matrix work.
  auto order_scores = [&]() __attribute__((always_inline)) {
    __builtin_amdgcn_sched_group_barrier(0x100, 4, 0);  // LDS reads
#pragma unroll
    for (int i = 0; i < C::KS - 2; ++i) {
      __builtin_amdgcn_sched_group_barrier(0x008, 2, 0);  // MFMAs
      __builtin_amdgcn_sched_group_barrier(0x100, 2, 0);
    }
    __builtin_amdgcn_sched_group_barrier(0x008, 4, 0);
  };
  // Causal mask of half H (keys from kt0) where it crosses this wavefront's diagonal.
  auto mask = [&](auto half, int kt0) __attribute__((always_inline)) {
    constexpr int H = decltype(half)::value;
    if (kt0 + kHalfKeys - 1 > wpos_min) {
      const int rel = qpos - kt0 - 4 * hh;  // key offset in the half tile must be <= this
#pragma unroll
      for (int bb = 0; bb < 2; ++bb)
#pragma unroll
        for (int e = 0; e < 16; ++e) {
          const int kofs = 32 * bb + 8 * (e >> 2) + (e & 3);
          sc[H][bb][e] = kofs > rel ? -INFINITY : sc[H][bb][e];
        }
    }
  };
  auto rowmax = [&](auto half) __attribute__((always_inline)) {
    constexpr int H = decltype(half)::value;
    float mx = sc[H][0][0];
#pragma unroll
    for (int bb = 0; bb < 2; ++bb)
#pragma unroll
      for (int e = 0; e < 16; ++e) mx = fmaxf(mx, sc[H][bb][e]);
    return max_with_partner(mx);  // both lanes of a query decide alike
  };
  // Lazy reference update for half H with row max mx (relative to mref).  Must follow
  // every P V product already issued: it rescales o.
  // With shift_other, the other half's scores (already formed against the old
  // reference) move along.
  auto rescale = [&](auto half, float mx, bool shift_other = false)
                     __attribute__((always_inline)) {
    constexpr int H = decltype(half)::value;
    const bool visible = mx != -INFINITY;
    const bool move = mx > kRescaleLog2 || (!seen && visible);
    if (__any(move)) {
      const float shift = move ? mx : 0.f;  // new reference mref + shift
      const float alpha = move && seen ? __builtin_amdgcn_exp2f(-shift) : (move ? 0.f : 1.f);
      mref += shift;
      seen = seen || visible;
      l_run *= alpha;
#pragma unroll
      for (int eb = 0; eb < C::EB; ++eb)
#pragma unroll
        for (int e = 0; e < 16; ++e) o[eb][e] *= alpha;
#pragma unroll
      for (int bb = 0; bb < 2; ++bb)
#pragma unroll
        for (int e = 0; e < 16; ++e) sc[H][bb][e] -= shift;
      if (shift_other) {
#pragma unroll
        for (int bb = 0; bb < 2; ++bb)
#pragma unroll
          for (int e = 0; e < 16; ++e) sc[1 - H][bb][e] -= shift;
      }
#pragma unroll
      for (int e = 0; e < 16; ++e) negm[e] = -mref;
    }
  };
  // Probabilities of half H (bf16) and their row sum.
  auto probs = [&](auto half) __attribute__((always_inline)) {
    constexpr int H = decltype(half)::value;
    typedef __bf16 bf16x2_t __attribute__((ext_vector_type(2)));
    const bf16x2_t ones = {(__bf16)1.f, (__bf16)1.f};
#pragma unroll
    for (int bb = 0; bb < 2; ++bb)
#pragma unroll
      for (int s2 = 0; s2 < 2; ++s2)
#pragma unroll
        for (int q = 0; q < 4; ++q) {
          const uint32_t pk = pack_bf16x2(__builtin_amdgcn_exp2f(sc[H][bb][8 * s2 + 2 * q]),
                                          __builtin_amdgcn_exp2f(sc[H][bb][8 * s2 + 2 * q + 1]));
          pf[H][bb][s2][q] = pk;
          // The denominator sums the same bf16 probabilities the numerator uses.
          l_run = __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(bf16x2_t, pk), ones, l_run,
                                                  false);
        }
  };
  // O^T += V^T P^T for half H of the tile in slot SLOT.  k-step (bb, s2) covers keys
  // 32 bb + 16 s2 + [0, 16) of the half tile; lane half hh feeds keys 4 hh + 0..3
  // (elements 0-3) and 8 + 4 hh + 0..3 (4-7), matching the accumulator layout of the
  // scores.
  // MFMA i takes k-step i / EB (bb, s2) and column block i % EB; its V^T fragment is read
  // kPvAhead MFMAs ahead, in the source order (as for the scores).
  constexpr int kPvAhead = 3;
  auto pv = [&](auto slot, auto half) __attribute__((always_inline)) {
    constexpr int S = decltype(slot)::value, H = decltype(half)::value;
    constexpr int N = 4 * C::EB;
    auto vread = [&](int i) __attribute__((always_inline)) {
      const int kx = i / C::EB, eb = i % C::EB;
      const int imm = S * TB + (kHalfKeys * H + 32 * (kx >> 1) + 16 * (kx & 1)) * RB;
      const u32x2 lo = lds_read_tr(Ls + va[eb] + imm);
      const u32x2 hi = lds_read_tr(Ls + vb[eb] + imm);
      return u32x4{lo[0], lo[1], hi[0], hi[1]};
    };
    u32x4 vf[kPvAhead];
#pragma unroll
    for (int i = 0; i < kPvAhead; ++i) vf[i] = vread(i);
#pragma unroll
    for (int i = 0; i < N; ++i) {
      const int kx = i / C::EB, eb = i % C::EB;
      o[eb] = mfma32(vf[i % kPvAhead], pf[H][kx >> 1][kx & 1], o[eb]);
      if (i + kPvAhead < N) vf[i % kPvAhead] = vread(i + kPvAhead);
    }
  };
  // Issue order for a block holding the probabilities of a half and its P V product:
  // the V^T reads of k-step k+1 and the 16 vector ops that produce its probabilities
  // interleave with the MFMAs of k-step k.
  auto order_probs_pv = [&]() __attribute__((always_inline)) {
    __builtin_amdgcn_sched_group_barrier(0x100, 2 * C::EB, 1);  // LDS reads, k-step 0
    __builtin_amdgcn_sched_group_barrier(0x002, 16, 1);         // probabilities, k-step 0
#pragma unroll
    for (int k = 0; k < 4; ++k)
#pragma unroll
      for (int eb = 0; eb < C::EB; ++eb) {
        __builtin_amdgcn_sched_group_barrier(0x008, 1, 1);
        if (k < 3) {
          __builtin_amdgcn_sched_group_barrier(0x100, 2, 1);
          __builtin_amdgcn_sched_group_barrier(0x002, 16 / C::EB, 1);
        }
      }
  };
  // Both halves of tile j (slot SLOT), in an order that gives each vector phase an
  // independent matrix phase to overlap with:
  //   scores(0) | max(0) | rescale(0) | scores(1) + probs(0) | mask(1) |
  //   P V(0) + max(1) | rescale(1) | probs(1) + P V(1)
  auto both_halves_a = [&](auto slot, int j) __attribute__((always_inline)) {
    constexpr IC<0> h0{};
    constexpr IC<1> h1{};
    const int kt0 = j * kStepKeys, kt1 = kt0 + kHalfKeys;
    scores(slot, h0);
    order_scores();
    mask(h0, kt0);
    rescale(h0, rowmax(h0));
    scores(slot, h1);
    probs(h0);
    // 16 score MFMAs and their 16 K reads with the 64 vector ops of probs(0).
    __builtin_amdgcn_sched_group_barrier(0x100, 4, 2);
#pragma unroll
    for (int i = 0; i < C::KS; ++i) {
      __builtin_amdgcn_sched_group_barrier(0x008, 2, 2);
      if (i + 2 < C::KS) __builtin_amdgcn_sched_group_barrier(0x100, 2, 2);
      __builtin_amdgcn_sched_group_barrier(0x002, 64 / C::KS, 2);
    }
    // Keep probs(0) in this block: without a use here the compiler sinks it past the
    // mask branch, next to P V(0), where it has no independent MFMAs to overlap with.
#pragma unroll
    for (int bb = 0; bb < 2; ++bb)
#pragma unroll
      for (int s2 = 0; s2 < 2; ++s2) asm volatile("" ::"v"(pf[0][bb][s2]));
    asm volatile("" ::"v"(l_run));
    mask(h1, kt1);
  };
  auto both_halves_b = [&](auto slot) __attribute__((always_inline)) {
    constexpr IC<0> h0{};
    constexpr IC<1> h1{};
    pv(slot, h0);
    const float mx1 = rowmax(h1);
    // P V(0): its V^T reads run a k-step ahead; the row max of half 1 fills in.
    __builtin_amdgcn_sched_group_barrier(0x100, 2 * C::EB, 3);
#pragma unroll
    for (int k = 0; k < 4; ++k)
#pragma unroll
      for (int eb = 0; eb < C::EB; ++eb) {
        __builtin_amdgcn_sched_group_barrier(0x008, 1, 3);
        if (k < 3) __builtin_amdgcn_sched_group_barrier(0x100, 2, 3);
        __builtin_amdgcn_sched_group_barrier(0x002, 2, 3);
      }
    rescale(h1, mx1);
    probs(h1);
    pv(slot, h1);
    order_probs_pv();
  };
  // Probabilities of half H (bf16, into pf) added to the row sum, as probs does; the
  // sum before the half is kept in l_prev.
  float l_prev = 0.f;
  auto probs_run = [&](auto half) __attribute__((always_inline)) {
    l_prev = l_run;
    probs(half);
  };
  // The half's probabilities are final while the row sum stays below kSumLimit (then so
  // does every probability since the reference last moved, and none overflowed).
  // Otherwise the sum goes back to its value before the half, the half's scores are
  // formed again from the K tile (still in its slot), the reference moves as in the
  // first tile and the probabilities are formed again.  Recomputing the scores on this
  // rare path lets them die as soon as their probabilities exist: keeping them for it
  // would hold 32 more registers through the step, which is what the schedule of the
  // steady-state step has no room for.  Half 0 settles after half 1's scores were
  // formed: those move with the reference.
  auto settle = [&](auto slot, auto half, int kt) __attribute__((always_inline)) {
    constexpr int H = decltype(half)::value;
    if (__any(!(l_run < kSumLimit))) {
      l_run = l_prev;
      scores(slot, half);
      mask(half, kt);
      rescale(half, rowmax(half), H == 0);
      probs(half);
    }
  };
  // Both halves of tile j after the query's first tile: no row maximum unless settle
  // finds one needed.
  //   scores(0) | scores(1) + probs(0) | settle(0) | P V(0) + probs(1) | settle(1) | P V(1)
  auto both_halves_fast_a = [&](auto slot, int j) __attribute__((always_inline)) {
    constexpr IC<0> h0{};
    constexpr IC<1> h1{};
    const int kt0 = j * kStepKeys, kt1 = kt0 + kHalfKeys;
    scores(slot, h0);
    order_scores();
    mask(h0, kt0);
    scores(slot, h1);
    probs_run(h0);
    __builtin_amdgcn_sched_group_barrier(0x100, 4, 2);
#pragma unroll
    for (int i = 0; i < C::KS; ++i) {
      __builtin_amdgcn_sched_group_barrier(0x008, 2, 2);
      if (i + 2 < C::KS) __builtin_amdgcn_sched_group_barrier(0x100, 2, 2);
      __builtin_amdgcn_sched_group_barrier(0x002, 64 / C::KS, 2);
    }
    settle(slot, h0, kt0);
    mask(h1, kt1);
  };
  auto both_halves_fast_b = [&](auto slot, int j) __attribute__((always_inline)) {
    constexpr IC<0> h0{};
    constexpr IC<1> h1{};
    pv(slot, h0);
    probs_run(h1);
    __builtin_amdgcn_sched_group_barrier(0x100, 2 * C::EB, 3);
#pragma unroll
    for (int k = 0; k < 4; ++k)
#pragma unroll
      for (int eb = 0; eb < C::EB; ++eb) {
        __builtin_amdgcn_sched_group_barrier(0x008, 1, 3);
        if (k < 3) __builtin_amdgcn_sched_group_barrier(0x100, 2, 3);
        __builtin_amdgcn_sched_group_barrier(0x002, 64 / (4 * C::EB), 3);
      }
    settle(slot, h1, j * kStepKeys + kHalfKeys);
    pv(slot, h1);
    __builtin_amdgcn_sched_group_barrier(0x100, 2 * C::EB, 4);
#pragma unroll
    for (int k = 0; k < 4; ++k)
#pragma unroll
      for (int eb = 0; eb < C::EB; ++eb) {
        __builtin_amdgcn_sched_group_barrier(0x008, 1, 4);
        if (k < 3) __builtin_amdgcn_sched_group_barrier(0x100, 2, 4);
      }
  };
  // One step: tile j in slot SLOT.  The loaders' shares of tile j were issued during
  // step j - 1; tile j + 1 goes into the other slot in the middle of this step, once
  // every wavefront is done with tile j - 1 there.  The older wavefront of a SIMD can so
  // run up to about half a step ahead of the younger one instead of waiting for it at a
  // barrier every step.
  auto step = [&](auto slot, int j) __attribute__((always_inline)) {
    constexpr int S = decltype(slot)::value;
    const int use = (j - j0) >> 1;  // earlier tiles in this slot
    if (loader) {
      wait_dma();
      lds_signal(ctr_full + S);
    }
    gave_up |= !lds_wait_ge(ctr_full + S, kLoaders * (use + 1), polls);  // tile j resident
    // A half past every query of the wavefront (only in its last tile) is fully masked
    // and leaves the softmax state unchanged, so one code path serves every tile.
    const bool active = half_active(j, 0);
    if (active) {
      if (j == j0) both_halves_a(slot, j);
      else both_halves_fast_a(slot, j);
    }
    if (loader && j + 1 < j0 + n_steps) {
      if (j > j0)
        gave_up |= !lds_wait_ge(ctr_empty + (1 - S), kWaves * (((j - 1 - j0) >> 1) + 1), polls);
      load_tile(j + 1, 1 - S);
    }
    if (active) {
      if (j == j0) both_halves_b(slot);
      else both_halves_fast_b(slot, j);
    }
    lds_signal(ctr_empty + S);  // done with slot S (LDS operations complete in order)
  };

  if (tid < 5) ctr_full[tid] = 0;  // full[0..1], empty[0..1], gave-up flag
  __syncthreads();
  if (n_steps > 0 && loader) load_tile(j0, 0);
  if (n_steps > 0) step(IC<0>{}, j0);
  for (int t = 1; t < n_steps; t += 2) {
    step(IC<1>{}, j0 + t);
    if (t + 1 < n_steps) step(IC<0>{}, j0 + t + 1);
  }

  if (gave_up) lds_signal(ctr_gave_up);
  __syncthreads();  // every wavefront is past its last wait and has raised its flag
  if (lds_read_count(ctr_gave_up) != 0) {
    l_run = __builtin_nanf("");
    mref = __builtin_nanf("");
  }
  l_run = sum_with_partner(l_run);
  if (!qvalid) return;
  const size_t trow = (size_t)b * P.s_loc + row0 + qloc;  // token row
  const size_t row = trow * P.heads + head;                // (token, head) row of partials
  if (P.n_split == 1) {
    // Whole key range: normalise and write bf16 O (key 0 is visible to every query,
    // so l > 0).
    const float inv = 1.f / l_run;
    if constexpr (LSE) {
      if (hh == 0)
        P.lse[((size_t)b * (P.lse_heads > 0 ? P.lse_heads : P.heads) + P.lse_head0 + head) *
                  P.s_loc + row0 + qloc] =
            mref + __builtin_amdgcn_logf(l_run);
    }
    const size_t ld_o = P.ld_o > 0 ? (size_t)P.ld_o : ld;
    uint16_t* orow = P.O + trow * ld_o + (size_t)head * D;
#pragma unroll
    for (int eb = 0; eb < C::EB; ++eb)
#pragma unroll
      for (int g = 0; g < 4; ++g)
        *reinterpret_cast<u32x2*>(orow + 32 * eb + 8 * g + 4 * hh) =
            u32x2{pack_bf16x2(o[eb][4 * g] * inv, o[eb][4 * g + 1] * inv),
                  pack_bf16x2(o[eb][4 * g + 2] * inv, o[eb][4 * g + 3] * inv)};
  } else {
    // Partial result of this key range: unnormalised O, reference (base-2 logit units;
    // -inf if no key of the range is visible) and sum.
    const size_t prow = (size_t)split * P.part_rows + row;
    float* po = P.part_o + prow * D;
#pragma unroll
    for (int eb = 0; eb < C::EB; ++eb)
#pragma unroll
      for (int g = 0; g < 4; ++g)
        *reinterpret_cast<f32x4*>(po + 32 * eb + 8 * g + 4 * hh) =
            f32x4{o[eb][4 * g], o[eb][4 * g + 1], o[eb][4 * g + 2], o[eb][4 * g + 3]};
    if (hh == 0)
      *reinterpret_cast<float2*>(P.part_ml + 2 * prow) =
          float2{l_run > 0.f ? mref : -INFINITY, l_run};
  }
}


template <int D, bool LSE, bool kPollArg>
__global__ __launch_bounds__(kThreads) void flash_fwd_kernel(const AttnParams P) {
  using C = FaCfg<D>;
  // [K slot 0][K slot 1][V slot 0][V slot 1][slot counters]
  __shared__ __attribute__((aligned(1024))) char L[4 * C::TILE_BYTES + 64];
  lds_char* Ls = (lds_char*)L;
  // Work item -> (batch, head, key range, query tile), query tile fastest, so the
  // workgroups that share an XCD (contiguous work indices) stream the same keys of the
  // same head through that XCD's L2.  Query tiles run over the segments' rows, last
  // segment (latest positions, most keys) first and, within one, last tile first.  With
  // pair_tiles, work item i of a head takes tiles i and n_qt - 1 - i one after the other
  // (the most and the fewest keys, the second most and second fewest, ...), so that all
  // items cost about the same and the workgroups of a launch finish together.
  const int nt0 = (P.seg_rows[0] + kQTile - 1) / kQTile;
  const int nt1 = P.n_seg > 1 ? (P.seg_rows[1] + kQTile - 1) / kQTile : 0;
  const int n_qt = nt0 + nt1;
  const int n_items = P.pair_tiles ? (n_qt + 1) / 2 : n_qt;
  const int w = xcd_work_index(blockIdx.x, n_items * P.n_split * P.heads * P.batch);
  const int item = w % n_items;
  int rest = w / n_items;
  const int split = rest % P.n_split;
  rest /= P.n_split;
  const int head = rest % P.heads;
  const int b = rest / P.heads;
  flash_tile<D, LSE, kPollArg>(P, Ls, nt0, nt1, item, split, head, b);
  if (P.pair_tiles && n_qt - 1 - item != item) {
    __syncthreads();  // every wavefront is done with the first tile's K/V slots
    flash_tile<D, LSE, kPollArg>(P, Ls, nt0, nt1, n_qt - 1 - item, split, head, b);
  }
}

// Merges the n_split partial results of each (batch, query, head) row: with
// M = max_c m_c, O = sum_c 2^(m_c - M) O_c / sum_c 2^(m_c - M) l_c, written as bf16.
// One thread per 4 consecutive head-dim columns of a row.
template <int D, bool LSE>
__global__ __launch_bounds__(256) void attn_combine_kernel(const AttnParams P) {
  constexpr int TPR = D / 4;  // threads per row
  const long long idx = (long long)blockIdx.x * blockDim.x + threadIdx.x;
  const long long row = idx / TPR;
  const int c4 = (int)(idx % TPR);
  if (row >= P.part_rows) return;
  float m = -INFINITY;
  for (int c = 0; c < P.n_split; ++c) m = fmaxf(m, P.part_ml[2 * (c * P.part_rows + row)]);
  f32x4 acc = {0.f, 0.f, 0.f, 0.f};
  float l = 0.f;
  for (int c = 0; c < P.n_split; ++c) {
    const long long prow = c * P.part_rows + row;
    const float mc = P.part_ml[2 * prow];
    if (mc == -INFINITY) continue;  // no visible key in this range
    const float wgt = __builtin_amdgcn_exp2f(mc - m);
    l += wgt * P.part_ml[2 * prow + 1];
    acc += wgt * *reinterpret_cast<const f32x4*>(P.part_o + prow * D + 4 * c4);
  }
  const float inv = 1.f / l;
  if constexpr (LSE) {
    if (c4 == 0) {
      // row = (b S_loc + t) H_s + head  ->  the [B, H_s, S_loc] log-sum-exp layout
      const long long bt = row / P.heads, b = bt / P.s_loc;
      const int head = (int)(row - bt * P.heads), t = (int)(bt - b * P.s_loc);
      const int lh = P.lse_heads > 0 ? P.lse_heads : P.heads;
      P.lse[((size_t)b * lh + P.lse_head0 + head) * P.s_loc + t] = m + __builtin_amdgcn_logf(l);
    }
  }
  const long long ld = P.ld_o > 0 ? P.ld_o : (P.ld > 0 ? P.ld : (long long)P.heads * D);
  *reinterpret_cast<u32x2*>(P.O + (row / P.heads) * ld + (row % P.heads) * D + 4 * c4) =
      u32x2{pack_bf16x2(acc[0] * inv, acc[1] * inv), pack_bf16x2(acc[2] * inv, acc[3] * inv)};
}

}  // namespace

namespace {

// Makespan, in keys visited by one workgroup plus fixed costs, of dispatching `total`
// work items of costs cost(w) (w in the kernel's work order): each XCD takes its
// contiguous share of work indices and gives each next item to its first free CU.
template <class Cost>
long long dispatch_makespan(long long total, Cost cost) {
  constexpr int kCusPerXcd = kAttnTargetWorkgroups / kXcds;
  const long long q = total / kXcds, rem = total % kXcds;
  long long worst = 0;
  for (int x = 0; x < kXcds; ++x) {
    // finish times of the XCD's CUs; the earliest-free one takes the next item
    std::priority_queue<long long, std::vector<long long>, std::greater<long long>> finish(
        std::greater<long long>(), std::vector<long long>(kCusPerXcd, 0));
    const long long w0 = x * q + (x < rem ? x : rem), w1 = w0 + q + (x < rem ? 1 : 0);
    for (long long w = w0; w < w1; ++w) {
      const long long f = finish.top() + cost(w);
      finish.pop();
      finish.push(f);
    }
    while (!finish.empty()) {
      worst = max(worst, finish.top());
      finish.pop();
    }
  }
  return worst;
}

// The launch plan of a shape: key ranges (and their length) without pairing, and the
// estimated seconds of that plan and of paired tiles without ranges.
struct AttnPlan {
  int n_split, split_len;
  double sec_split, sec_pair;
};

AttnPlan attn_plan_uncached(const AttnParams& p) {
  constexpr long long kPieceCost = kStepKeys;      // setup and output write: ~one step
  constexpr long long kEmptyCost = kStepKeys / 8;  // a workgroup with no keys to visit
  // Keys of each query tile, in the kernel's order (last segment first, last tile first).
  constexpr int kMaxTiles = 1024;
  int tile_keys[kMaxTiles];
  int n_qt = 0, max_keys = 1;
  for (int k = p.n_seg - 1; k >= 0; --k) {
    const int nt = (p.seg_rows[k] + kQTile - 1) / kQTile;
    for (int t = nt - 1; t >= 0; --t) {
      const int keys = p.seg_pos0[k] + min((t + 1) * kQTile, p.seg_rows[k]);
      if (n_qt < kMaxTiles) tile_keys[n_qt] = keys;
      ++n_qt;
      max_keys = max(max_keys, keys);
    }
  }
  auto len_of = [&](int n) {
    const int len = (max_keys + n - 1) / n;
    return (len + kStepKeys - 1) / kStepKeys * kStepKeys;
  };
  const long long bh = (long long)p.batch * p.heads;
  AttnPlan plan = {1, len_of(1), 0.0, 0.0};
  if (bh <= 0 || n_qt > kMaxTiles) return plan;
  // Time per key of a workgroup: 4 kQTile d FLOPs (its Q K^T and P V rows) at the
  // fraction of one CU's bf16 MFMA peak (2516.6 / 256 TFLOP/s) this kernel reaches (0.50
  // measured at 7B, S = 65536: ~27 ns per key at d = 128).  Key-range partials move at
  // about half the HBM peak (8 TB/s).  Only the ratio of the two matters; the fraction is
  // refitted to the measured one whenever the kernel's speed changes.
  constexpr double kCuPeak = 2516.6e12 / 256, kPeakFraction = 0.50, kPartialBw = 4e12;
  const double t_key = 4.0 * kQTile * p.head_dim / (kPeakFraction * kCuPeak);
  const double rows = (double)bh * p.s_loc;
  // Key ranges: candidate counts 1..8, at least 4 key tiles per range; estimated time =
  // simulated makespan x t_key + the partials' traffic (written, read back, merged); the
  // smallest wins, ties going to fewer ranges.
  double best = -1.0;
  for (int n = 1; n <= 8; ++n) {
    const int len = len_of(n);
    if (n > 1 && len < 4 * kStepKeys) break;
    if ((max_keys + len - 1) / len != n) continue;  // same ranges as a smaller n
    const double traffic =
        n > 1 ? (2.0 * n * rows * (p.head_dim + 2) * 4 + rows * p.head_dim * 2) / kPartialBw : 0.0;
    const long long span = dispatch_makespan(bh * n_qt * n, [&](long long w) {
      const int t = (int)(w % n_qt), split = (int)((w / n_qt) % n);
      const long long keys =
          min(max((long long)tile_keys[t] - (long long)split * len, 0LL), (long long)len);
      return keys > 0 ? keys + kPieceCost : kEmptyCost;
    });
    const double sec = span * t_key + traffic;
    if (best < 0 || sec < best) {
      best = sec;
      plan.n_split = n;
      plan.split_len = len;
    }
  }
  plan.sec_split = best;
  // Paired tiles: item i takes tiles i and n_qt - 1 - i (one tile if they coincide).
  const int n_items = (n_qt + 1) / 2;
  const long long span = dispatch_makespan(bh * n_items, [&](long long w) {
    const int i = (int)(w % n_items), j = n_qt - 1 - i;
    return tile_keys[i] + kPieceCost + (j != i ? tile_keys[j] + kPieceCost : 0LL);
  });
  plan.sec_pair = span * t_key;
  return plan;
}

// Shapes already planned (the plan depends on these fields only); callers ask for the
// same shape several times per entry point call.
struct PlanKey {
  int batch, heads, head_dim, n_seg, seg_rows[2], seg_pos0[2];
  bool operator==(const PlanKey& o) const {
    return batch == o.batch && heads == o.heads && head_dim == o.head_dim && n_seg == o.n_seg &&
           seg_rows[0] == o.seg_rows[0] && seg_rows[1] == o.seg_rows[1] &&
           seg_pos0[0] == o.seg_pos0[0] && seg_pos0[1] == o.seg_pos0[1];
  }
};
std::mutex g_plan_mu;
std::vector<std::pair<PlanKey, AttnPlan>> g_plan_cache;
constexpr size_t kPlanCacheMax = 64;

AttnPlan attn_plan(const AttnParams& p) {
  PlanKey key = {p.batch, p.heads, p.head_dim, p.n_seg, {0, 0}, {0, 0}};
  for (int k = 0; k < p.n_seg && k < 2; ++k) {
    key.seg_rows[k] = p.seg_rows[k];
    key.seg_pos0[k] = p.seg_pos0[k];
  }
  {
    std::lock_guard<std::mutex> lock(g_plan_mu);
    for (const auto& c : g_plan_cache)
      if (c.first == key) return c.second;
  }
  const AttnPlan plan = attn_plan_uncached(p);
  std::lock_guard<std::mutex> lock(g_plan_mu);
  if (g_plan_cache.size() >= kPlanCacheMax) g_plan_cache.erase(g_plan_cache.begin());
  g_plan_cache.push_back({key, plan});
  return plan;
}

}  // namespace

int attn_split_count(const AttnParams& p, int* split_len) {
  const AttnPlan plan = attn_plan(p);
  if (split_len) *split_len = plan.split_len;
  return plan.n_split;
}

double attn_launch_seconds(const AttnParams& p, bool pair) {
  const AttnPlan plan = attn_plan(p);
  return pair ? plan.sec_pair : plan.sec_split;
}

static std::atomic<int> g_attn_poll_limit{0};
void set_attn_poll_limit(int polls) { g_attn_poll_limit.store(polls); }
int attn_poll_limit() { return g_attn_poll_limit.load(); }

hipError_t launch_flash_attn(const AttnParams& p_in, hipStream_t s) {
  AttnParams p = p_in;
  p.poll_limit = g_attn_poll_limit.load();
  if (p.batch <= 0 || p.s_loc <= 0 || p.heads <= 0) return hipSuccess;
  if (p.n_seg < 1 || p.n_seg > 2) return hipErrorInvalidValue;
  int n_qt = 0, rows = 0;
  for (int k = 0; k < p.n_seg; ++k) {
    const long long end = (long long)p.seg_pos0[k] + p.seg_rows[k];
    if (p.seg_rows[k] < 1 || p.seg_row0[k] != rows || p.seg_pos0[k] < 0 || end > p.kv_len ||
        (long long)p.n_split * p.split_len < end)
      return hipErrorInvalidValue;
    rows += p.seg_rows[k];
    n_qt += (p.seg_rows[k] + kQTile - 1) / kQTile;
  }
  if (p.ld != 0 && (p.ld < p.heads * p.head_dim || p.ld % 8 != 0)) return hipErrorInvalidValue;
  if (p.ld_o != 0 && (p.ld_o < p.heads * p.head_dim || p.ld_o % 8 != 0)) return hipErrorInvalidValue;
  if (p.pair_tiles && p.n_split != 1) return hipErrorInvalidValue;
  if (rows != p.s_loc || p.n_split < 1 || p.split_len <= 0 || p.split_len % kStepKeys != 0 ||
      (p.n_split > 1 && (!p.part_o || !p.part_ml)))
    return hipErrorInvalidValue;
  const int n_items = p.pair_tiles ? (n_qt + 1) / 2 : n_qt;
  const dim3 grid(n_items * p.n_split * p.heads * p.batch);
  const bool capped = p.poll_limit > 0;
  const void* fn;
  const void* combine;
  if (p.head_dim == 128) {
    fn = p.lse ? (capped ? reinterpret_cast<const void*>(&flash_fwd_kernel<128, true, true>)
                         : reinterpret_cast<const void*>(&flash_fwd_kernel<128, true, false>))
               : (capped ? reinterpret_cast<const void*>(&flash_fwd_kernel<128, false, true>)
                         : reinterpret_cast<const void*>(&flash_fwd_kernel<128, false, false>));
    combine = p.lse ? reinterpret_cast<const void*>(&attn_combine_kernel<128, true>)
                    : reinterpret_cast<const void*>(&attn_combine_kernel<128, false>);
  } else if (p.head_dim == 64) {
    fn = p.lse ? (capped ? reinterpret_cast<const void*>(&flash_fwd_kernel<64, true, true>)
                         : reinterpret_cast<const void*>(&flash_fwd_kernel<64, true, false>))
               : (capped ? reinterpret_cast<const void*>(&flash_fwd_kernel<64, false, true>)
                         : reinterpret_cast<const void*>(&flash_fwd_kernel<64, false, false>));
    combine = p.lse ? reinterpret_cast<const void*>(&attn_combine_kernel<64, true>)
                    : reinterpret_cast<const void*>(&attn_combine_kernel<64, false>);
  } else {
    return hipErrorInvalidValue;
  }
  // hipLaunchKernel returns the status of this launch only (not an earlier error).
  void* args[] = {&p};
  const hipError_t e = hipLaunchKernel(fn, grid, dim3(kThreads), args, 0, s);
  if (e != hipSuccess || p.n_split == 1) return e;
  const long long threads = p.part_rows * (long long)(p.head_dim / 4);
  return hipLaunchKernel(combine, dim3((unsigned)((threads + 255) / 256)), dim3(256), args, 0, s);
}

}  // namespace tsp
