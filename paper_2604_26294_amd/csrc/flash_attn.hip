// Causal flash attention of one TSP rank's query chunk (gfx950, bf16 MFMA).
//
// Algorithm 1's CausalAttn for contiguous chunks: local query t of rank p sits at
// global position q_pos0 + t (q_pos0 = p S_loc) and sees keys j <= q_pos0 + t of the
// gathered K/V (held resident in a [B, S, n_kv, d] buffer).  The softmax is computed
// online, one key tile at a time, so the (S_loc x S) score matrix never exists.
//
// Work split.  A workgroup owns 128 queries of one head (GQA: head i reads kv head
// i / g) and has 8 wavefronts, two per SIMD: wavefront w handles queries
// 32 (w % 4) .. +31 against key group w / 4, i.e. every 128-key tile staged in LDS is
// consumed as two 64-key halves.  Each group keeps its own running max / sum /
// output; the groups are merged once at the end.  Key tiles beyond the last query's
// position are never loaded, and only tiles that cross the diagonal are masked.
//
// Scores are computed transposed, S^T = K Q^T, with K as the MFMA A operand and Q
// (held in registers) as B.  The 32 x 32 accumulator then gives each lane 16 keys of
// ONE query (its partner lane l ^ 32 holds the other 16), so the row max needs one
// cross-lane exchange and the row sum none until the end.  The probabilities P^T
// feed O^T = V^T P^T directly as the B operand (contraction over keys).
//
// Schedule.  Per step every wavefront computes the scores of its half of tile j,
// the softmax and the P V product, while tiles j+1 of K and V stream into the other
// slot of their two-slot rings.  (Variants that delay P V by a step so the two
// wavefronts of a SIMD alternate matrix and vector phases measured slower.)
//
// Data movement.  K and V tiles go from HBM straight into LDS (global_load_lds, no
// register staging) in their natural [key][d] layout, 16-byte chunks XOR-swizzled by
// a function of the row chosen per tile kind so that its reads are bank-conflict free.  The V^T operand is read with the gfx950 LDS transpose
// read (ds_read_b64_tr_b16): in each 16-lane group, source lane s points at row
// kbase + s/4, columns base + 4 (s % 4), and lane t receives column base + t of rows
// kbase .. kbase+3 -- four consecutive keys of one head-dim column.  Because tile rows
// are aligned to the row size and the swizzle only touches the in-row offset, every
// LDS read address is (per-lane base XOR a constant) + an immediate offset.
#include <math.h>

#include <type_traits>

#include "common.h"
#include "internal.h"

namespace tsp {
namespace {

constexpr int kThreads = 512;
constexpr int kWaves = kThreads / kWave;
constexpr int kQTile = 128;          // queries per workgroup
constexpr int kStepKeys = 128;       // keys staged per step
constexpr int kGroupKeys = 64;       // keys per group per step
constexpr float kRescaleLog2 = 8.f;  // lazy-rescale threshold (exp2 units)

typedef short i16x4 __attribute__((ext_vector_type(4)));
typedef __attribute__((address_space(3))) char lds_char;

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

__device__ __forceinline__ void wait_dma() { asm volatile("s_waitcnt vmcnt(0)" ::: "memory"); }

// 16 bytes per lane from global memory straight into LDS at lds + 16 * lane: the
// buffer form, with the address = resource base (scalar) + soff (scalar) + voff (lane).
__device__ __forceinline__ void dma16(__amdgpu_buffer_rsrc_t rsrc, uint32_t voff, uint32_t soff,
                                      lds_char* lds) {
  __builtin_amdgcn_raw_ptr_buffer_load_lds(rsrc, (__attribute__((address_space(3))) void*)lds, 16,
                                           (int)voff, (int)soff, 0, 0);
}

// Raw buffer resource over [base, base + 4 GiB) (stride 0, no format conversion).
__device__ __forceinline__ __amdgpu_buffer_rsrc_t make_rsrc(const void* base) {
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(base), (short)0, 0xffffffff,
                                           0x00020000);
}

__device__ __forceinline__ u32x4 lds_read16(const lds_char* p) {
  return *reinterpret_cast<const __attribute__((address_space(3))) u32x4*>(p);
}

__device__ __forceinline__ u32x2 lds_read_tr(const lds_char* p) {
  return __builtin_bit_cast(
      u32x2, __builtin_amdgcn_ds_read_tr16_b64_v4i16((__attribute__((address_space(3))) i16x4*)p));
}

template <int N>
using IC = std::integral_constant<int, N>;

template <int D>
__global__ __launch_bounds__(kThreads) void flash_fwd_kernel(const AttnParams P) {
  using C = FaCfg<D>;
  constexpr int KCH = C::KCH, RB = C::ROW_BYTES, TB = C::TILE_BYTES;
  // [K slot 0][K slot 1][V slot 0][V slot 1]
  __shared__ __attribute__((aligned(1024))) char L[4 * TB];
  lds_char* Ls = (lds_char*)L;

  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int grp = wave >> 2, wq = wave & 3;
  const int l32 = lane & 31, hh = lane >> 5;

  const int n_qt = (P.s_loc + kQTile - 1) / kQTile;
  const int w = xcd_work_index(blockIdx.x, n_qt * P.heads * P.batch);
  const int b = w / (P.heads * n_qt);
  const int rem = w - b * (P.heads * n_qt);
  const int head = rem / n_qt;
  const int qt = n_qt - 1 - (rem - head * n_qt);  // longest query tiles first
  const int q0 = qt * kQTile;
  const int kvh = P.kv_head0 + head / P.group;

  const int qloc = q0 + 32 * wq + l32;
  const bool qvalid = qloc < P.s_loc;
  const int qpos = P.q_pos0 + qloc;
  const int wq_first = q0 + 32 * wq;
  const bool wave_active = wq_first < P.s_loc;
  const int wpos_min = P.q_pos0 + wq_first;
  const int wpos_max = P.q_pos0 + min(wq_first + 31, P.s_loc - 1);
  const int n_keys = P.q_pos0 + min(q0 + kQTile, P.s_loc);  // <= kv_len
  const int n_steps = (n_keys + kStepKeys - 1) / kStepKeys;

  // Q fragments (the B operand of S^T): lane holds Q[qloc][16 ks + 8 hh .. +7], scaled
  // by c = softmax scale * log2(e) and rounded to bf16 once, so that the score MFMAs
  // produce base-2 logits directly.
  u32x4 qf[C::KS];
  {
    const float c = P.scale_log2;
    const uint16_t* qrow = P.Q + (((size_t)b * P.s_loc + (qvalid ? qloc : 0)) * P.heads + head) * D;
#pragma unroll
    for (int s = 0; s < C::KS; ++s) {
      const u32x4 raw = qvalid ? ld16(qrow + 16 * s + 8 * hh) : u32x4{0u, 0u, 0u, 0u};
#pragma unroll
      for (int e = 0; e < 4; ++e)
        qf[s][e] = pack_bf16x2(bf16_bits_to_f32(raw[e] & 0xffffu) * c,
                               bf16_bits_to_f32(raw[e] >> 16) * c);
    }
  }
  const size_t kv_stride = (size_t)P.n_kv * D;  // elements between consecutive keys
  const uint16_t* kbase = P.Kb + (size_t)b * P.seq * kv_stride + (size_t)kvh * D;
  const uint16_t* vbase = P.Vb + (size_t)b * P.seq * kv_stride + (size_t)kvh * D;

  // DMA geometry: instruction i of wave w fills rows (i kWaves + w) ROWS_PER_DMA + lane / KCH,
  // physical chunk lane % KCH, with the logical chunk that the tile's swizzle puts there
  // (the swizzle depends on the row only through bits that are the same for every i).
  // A full tile's source is (scalar tile base) + (scalar i * row step) + (per-lane 32-bit
  // offset), so its loads need no vector arithmetic.
  constexpr int kRowStep = kWaves * C::ROWS_PER_DMA;  // rows between instructions
  const int dma_row0 = wave * C::ROWS_PER_DMA + lane / KCH;
  const int dma_col_k = 8 * ((lane % KCH) ^ C::fk(dma_row0));
  const int dma_col_v = 8 * ((lane % KCH) ^ C::fv(dma_row0));
  const uint32_t row_bytes = 2u * (uint32_t)kv_stride;
  const uint32_t dma_off_k = (uint32_t)dma_row0 * row_bytes + 2u * dma_col_k;
  const uint32_t dma_off_v = (uint32_t)dma_row0 * row_bytes + 2u * dma_col_v;
  const uint32_t dma_step = (uint32_t)kRowStep * row_bytes;
  // One 128-key tile from HBM into an LDS slot.  In the last tile, rows past the last
  // needed key are clamped to it: they are always masked (keys > every query position
  // of this workgroup) and stay finite, so the P V product never sees garbage.
  auto dma_tile = [&](const uint16_t* base, uint32_t lane_off, int col, int tile,
                      int slot_off) __attribute__((always_inline)) {
    const int key0 = tile * kStepKeys;
    const __amdgpu_buffer_rsrc_t rsrc = make_rsrc(base + (size_t)key0 * kv_stride);
    lds_char* dst = Ls + slot_off + wave * (kWave * 16);
    if (key0 + kStepKeys <= n_keys) {
#pragma unroll
      for (int i = 0; i < C::DMA_PER_LANE; ++i)
        dma16(rsrc, lane_off, i * dma_step, dst + i * kWaves * (kWave * 16));
    } else {
      const int last = n_keys - 1 - key0;
#pragma unroll
      for (int i = 0; i < C::DMA_PER_LANE; ++i) {
        const uint32_t row = (uint32_t)min(dma_row0 + i * kRowStep, last);
        dma16(rsrc, row * row_bytes + 2u * col, 0u, dst + i * kWaves * (kWave * 16));
      }
    }
  };

  // LDS read addresses.  Slot offsets and block strides are compile-time immediates;
  // the per-lane parts below are computed once.
  //  K operand: row 64 grp + 32 bb + l32, logical chunk 2 ks + hh  ->  byte
  //    (64 grp + 32 bb) RB + (ka ^ 32 ks),  ka = l32 RB + 16 (hh ^ f_K(l32)).
  //  V^T operand (transpose reads): rows 64 grp + 32 bb + 16 s2 + tr_row (+8 for elements
  //    4-7), columns 32 eb + tr_col  ->  byte (64 grp + 32 bb + 16 s2) RB + (va or vb)[eb].
  const int grp_rows = kGroupKeys * grp * RB;  // this group's half of a tile
  int kad[C::KS];
  {
    const int ka = l32 * RB + 16 * (hh ^ C::fk(l32));
#pragma unroll
    for (int ks = 0; ks < C::KS; ++ks) kad[ks] = grp_rows + (ka ^ (32 * ks));
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
      va[eb] = 2 * TB + grp_rows + (base_a ^ (64 * eb));
      vb[eb] = 2 * TB + grp_rows + (base_b ^ (64 * eb));
    }
  }

  auto tile_active = [&](int tile) __attribute__((always_inline)) {
    return wave_active && tile * kStepKeys + kGroupKeys * grp <= wpos_max;
  };

  // Online-softmax state of this lane's query (shared with its partner lane l ^ 32).
  // Scores are produced relative to the reference mref (the score MFMAs start from the
  // accumulator value -mref), so o = sum 2^(s - mref) v and l = sum 2^(s - mref).
  // mref follows the running maximum lazily: it moves only when a score exceeds it by
  // more than kRescaleLog2, or to the first visible score of the query; in between,
  // every probability is bounded by 2^kRescaleLog2 and numerator and denominator share
  // the stale reference, so the normalised result is unchanged.
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
  f32x16 sacc[2];   // scores of this group's 64 keys of one tile
  u32x4 pf[2][2];   // bf16 probabilities of one tile (B operands of P V)

  // S^T - mref of the tile in slot SLOT: 2 blocks of 32 keys x 32 queries.
  auto scores = [&](auto slot) __attribute__((always_inline)) {
    constexpr int S = decltype(slot)::value;
#pragma unroll
    for (int ks = 0; ks < C::KS; ++ks)
#pragma unroll
      for (int bb = 0; bb < 2; ++bb)
        sacc[bb] = mfma32(lds_read16(Ls + kad[ks] + (S * TB + 32 * bb * RB)), qf[ks],
                          ks == 0 ? negm : sacc[bb]);
    // Issue order: the K fragments run two contraction steps ahead of their MFMAs, so
    // the LDS latency hides behind the matrix work.
    __builtin_amdgcn_sched_group_barrier(0x100, 4, 0);  // LDS reads
#pragma unroll
    for (int i = 0; i < C::KS - 2; ++i) {
      __builtin_amdgcn_sched_group_barrier(0x008, 2, 0);  // MFMAs
      __builtin_amdgcn_sched_group_barrier(0x100, 2, 0);
    }
    __builtin_amdgcn_sched_group_barrier(0x008, 4, 0);
  };
  // Mask (if tile j crosses the diagonal), lazy reference update, probabilities.
  auto softmax = [&](int j) __attribute__((always_inline)) {
    const int kt0 = j * kStepKeys + kGroupKeys * grp;
    if (kt0 + kGroupKeys - 1 > wpos_min) {
      const int rel = qpos - kt0 - 4 * hh;  // key offset in the group tile must be <= this
#pragma unroll
      for (int bb = 0; bb < 2; ++bb)
#pragma unroll
        for (int e = 0; e < 16; ++e) {
          const int kofs = 32 * bb + 8 * (e >> 2) + (e & 3);
          sacc[bb][e] = kofs > rel ? -INFINITY : sacc[bb][e];
        }
    }
    float mx = sacc[0][0];
#pragma unroll
    for (int bb = 0; bb < 2; ++bb)
#pragma unroll
      for (int e = 0; e < 16; ++e) mx = fmaxf(mx, sacc[bb][e]);
    mx = fmaxf(mx, __shfl_xor(mx, 32));  // both lanes of a query decide alike
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
        for (int e = 0; e < 16; ++e) sacc[bb][e] -= shift;
#pragma unroll
      for (int e = 0; e < 16; ++e) negm[e] = -mref;
    }
    typedef __bf16 bf16x2_t __attribute__((ext_vector_type(2)));
    const bf16x2_t ones = {(__bf16)1.f, (__bf16)1.f};
#pragma unroll
    for (int bb = 0; bb < 2; ++bb)
#pragma unroll
      for (int s2 = 0; s2 < 2; ++s2)
#pragma unroll
        for (int q = 0; q < 4; ++q) {
          const uint32_t pk = pack_bf16x2(__builtin_amdgcn_exp2f(sacc[bb][8 * s2 + 2 * q]),
                                          __builtin_amdgcn_exp2f(sacc[bb][8 * s2 + 2 * q + 1]));
          pf[bb][s2][q] = pk;
          // The denominator sums the same bf16 probabilities the numerator uses.
          l_run = __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(bf16x2_t, pk), ones, l_run,
                                                  false);
        }
  };
  // O^T += V^T P^T for the tile in slot SLOT.  k-step (bb, s2) covers keys 32 bb + 16 s2 +
  // [0, 16) of the group tile; lane half hh feeds keys 4 hh + 0..3 (elements 0-3) and
  // 8 + 4 hh + 0..3 (4-7), matching the accumulator layout of the scores.
  auto pv = [&](auto slot) __attribute__((always_inline)) {
    constexpr int S = decltype(slot)::value;
#pragma unroll
    for (int bb = 0; bb < 2; ++bb)
#pragma unroll
      for (int s2 = 0; s2 < 2; ++s2) {
#pragma unroll
        for (int eb = 0; eb < C::EB; ++eb) {
          const int imm = S * TB + (32 * bb + 16 * s2) * RB;
          const u32x2 lo = lds_read_tr(Ls + va[eb] + imm);
          const u32x2 hi = lds_read_tr(Ls + vb[eb] + imm);
          o[eb] = mfma32(u32x4{lo[0], lo[1], hi[0], hi[1]}, pf[bb][s2], o[eb]);
        }
      }
    // Issue order (this block also holds the exponentials of the tile): the V^T reads
    // of k-step k+1 and the 16 vector ops that produce its probabilities interleave
    // with the MFMAs of k-step k, so vector and matrix pipes work at the same time.
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
  // One step: tile j (resident in slot SLOT once every wave's DMA has landed) is
  // consumed while tile j + 1 streams into the other slot.
  auto step = [&](auto slot, int j) __attribute__((always_inline)) {
    constexpr int S = decltype(slot)::value;
    wait_dma();
    __syncthreads();  // K and V tile j resident; every wave is past step j-1
    if (j + 1 < n_steps) {
      dma_tile(kbase, dma_off_k, dma_col_k, j + 1, (1 - S) * TB);
      dma_tile(vbase, dma_off_v, dma_col_v, j + 1, (3 - S) * TB);
    }
    if (tile_active(j)) {
      scores(slot);
      softmax(j);
      pv(slot);
    }
  };

  dma_tile(kbase, dma_off_k, dma_col_k, 0, 0);
  dma_tile(vbase, dma_off_v, dma_col_v, 0, 2 * TB);
  for (int j = 0; j < n_steps; j += 2) {
    step(IC<0>{}, j);
    if (j + 1 < n_steps) step(IC<1>{}, j + 1);
  }

  // Merge the two key groups: group 1 parks its state in LDS, group 0 combines.  A group
  // that saw no visible key has l = 0 and takes no part.
  l_run += __shfl_xor(l_run, 32);
  const float m_own = l_run > 0.f ? mref : -INFINITY;
  __syncthreads();
  float* F = reinterpret_cast<float*>(L);
  const int slot = wq * 64 + lane;
  if (grp == 1) {
    F[slot] = m_own;
    F[256 + slot] = l_run;
#pragma unroll
    for (int eb = 0; eb < C::EB; ++eb)
#pragma unroll
      for (int e = 0; e < 16; ++e) F[(2 + 16 * eb + e) * 256 + slot] = o[eb][e];
  }
  __syncthreads();
  if (grp == 0 && qvalid) {
    const float m1 = F[slot], l1 = F[256 + slot];
    const float m = fmaxf(m_own, m1);  // finite: key 0 is visible to every query
    const float a0 = __builtin_amdgcn_exp2f(m_own - m);
    const float a1 = __builtin_amdgcn_exp2f(m1 - m);
    const float inv = 1.f / (l_run * a0 + l1 * a1);
    uint16_t* orow = P.O + (((size_t)b * P.s_loc + qloc) * P.heads + head) * D;
#pragma unroll
    for (int eb = 0; eb < C::EB; ++eb)
#pragma unroll
      for (int g = 0; g < 4; ++g) {
        float v[4];
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          const int e = 4 * g + r;
          v[r] = (o[eb][e] * a0 + F[(2 + 16 * eb + e) * 256 + slot] * a1) * inv;
        }
        *reinterpret_cast<u32x2*>(orow + 32 * eb + 8 * g + 4 * hh) =
            u32x2{pack_bf16x2(v[0], v[1]), pack_bf16x2(v[2], v[3])};
      }
  }
}

}  // namespace

hipError_t launch_flash_attn(const AttnParams& p, hipStream_t s) {
  if (p.batch <= 0 || p.s_loc <= 0 || p.heads <= 0) return hipSuccess;
  const int n_qt = (p.s_loc + kQTile - 1) / kQTile;
  const dim3 grid(n_qt * p.heads * p.batch);
  const void* fn;
  if (p.head_dim == 128)
    fn = reinterpret_cast<const void*>(&flash_fwd_kernel<128>);
  else if (p.head_dim == 64)
    fn = reinterpret_cast<const void*>(&flash_fwd_kernel<64>);
  else
    return hipErrorInvalidValue;
  // hipLaunchKernel returns the status of this launch only (not an earlier error).
  void* args[] = {const_cast<AttnParams*>(&p)};
  return hipLaunchKernel(fn, grid, dim3(kThreads), args, 0, s);
}

}  // namespace tsp
