// bf16 MFMA GEMM family for the TSP shard products (gfx950).
//
//   gate+up+SwiGLU  Hs = bf16( SiLU(X W1^T) * (X W3^T) )          Algorithm 2, gate/up
//   down / O-proj   Y (+)= Hs W2   or   Y (+)= Flatten(A) W_O^T    Algorithm 2 / 1, "+="
//                   (optionally over two shards at once: the contraction then runs over
//                   [A A'] and [B; B'], two operand pairs held in separate buffers)
//   SwiGLU backward G = X W1^T, U = X W3^T, dHs = dY W2^T in one pass; dG, dU and the
//                   transposes of dG, dU, Hs for the weight-gradient products
//   Q/K/V proj      Q = X W_Q^T (times a factor, then rounded) -> workspace, K, V ->
//                   full-sequence buffers at the rows' sequence positions (zigzag
//                   reorder folded in)  Algorithm 1
//
// One workgroup = WGM x WGN wavefronts (8 by default: two per SIMD); each wavefront owns
// a (BM/WGM) x (BN/WGN) block of C as 32 x 32 MFMA tiles.  K advances in steps of 64.
// Operand panels go from HBM straight into LDS (buffer loads with an LDS destination, no
// register staging), in a ring of STAGES slots: while the MFMAs consume step k the loads
// fill the steps up to k + STAGES - 1.
//
// LDS layouts.  LDS has 64 banks of 4 bytes, so a byte address maps to bank window
// position (address mod 256).  A [M, K] and "NT" B [N, K] panels are rows of 64 bf16
// (128 bytes, eight 16-byte chunks); an MFMA operand is one 16-byte read, 16 lanes of
// which read 16 consecutive rows at one logical chunk, so the physical chunk is the
// logical one XOR ((row / 2) mod 8) and those 16 reads hit 16 distinct windows.
// "NN" B panels ([K, N] operands: W2 and W_O^(r)^T) keep their natural [64][BN] layout,
// chunk XOR 4 (row mod 4) so that the 4 rows x 64 bytes of a half-wave transpose read
// cover all 64 banks, and are read with the gfx950 LDS transpose read
// ds_read_b64_tr_b16: in each 16-lane group, source lane s points at row kbase + s/4,
// columns base + 4 (s % 4), and lane t receives column base + t of rows kbase..kbase+3,
// i.e. four consecutive contraction indices of one output column -- no transpose pass
// over HBM and no register shuffles.  Every LDS address is a per-lane base XOR a
// wave-uniform constant plus an immediate offset.
//
// Tails.  Rows or columns past M / N are clamped to the last valid one on load (finite
// values, results never stored).  K must be a multiple of 64: the gated product Hs is
// stored with its width padded to a multiple of 64 with zero columns (written by the
// SwiGLU epilogue), and the matching W2 rows past F/D are clamped, so padded terms
// contribute exact zeros.
#include <climits>
#include <type_traits>

#include "common.h"
#include "internal.h"
#include "lds_dma.h"

namespace tsp {
namespace {

constexpr int BK = 64;
enum { EPI_SWIGLU = 0, EPI_ACC = 1, EPI_QKV = 2, EPI_SWIGLU_BWD = 3 };

// Wait until at most N of this wavefront's operand loads are still in flight (loads
// complete in issue order).
template <int N>
__device__ __forceinline__ void wait_dma() {
  static_assert(N >= 0 && N < 64, "vmcnt range");
  asm volatile("s_waitcnt vmcnt(%0)" ::"n"(N) : "memory");
}

template <int BM, int BN, int WGM, int WGN, bool NN, int EPI, int STAGES>
struct Cfg {
  static constexpr int WAVES = WGM * WGN, THREADS = kWave * WAVES;
  static constexpr int WM = BM / WGM, WN = BN / WGN;
  static constexpr int TM = WM / 32, TN = WN / 32;
  static constexpr bool BWD = EPI == EPI_SWIGLU_BWD;
  static constexpr int NAP = BWD ? 2 : 1;                                  // A panels
  static constexpr int NBP = EPI == EPI_SWIGLU ? 2 : (BWD ? 3 : 1);        // B panels
  static constexpr int TNB = NBP * TN;
  static constexpr int NB = NBP * BN;                         // B rows of an NT panel
  static constexpr int A_BYTES = NAP * BM * BK * 2;
  static constexpr int B_BYTES = NB * BK * 2;                  // NT [NB][64] or NN [64][BN]
  static constexpr int STAGE = A_BYTES + B_BYTES;
  static constexpr int LDS_BYTES = STAGES * STAGE;
  // Operand load instructions one wavefront issues per stage.
  // [N, K]-operand tiles: only the first half of the wavefronts (one per SIMD) load, each
  // its own share of a stage and that of the other wavefront of its SIMD; [K, N] tiles:
  // every wavefront loads its share.
  static constexpr bool HALF_LOADERS = !NN;
  static constexpr int LOADS = (HALF_LOADERS ? 2 : 1) *
      (NAP * BM / 8 / WAVES + (NN ? BK * (BN * 2) / 1024 / WAVES : NB / 8 / WAVES));
  static_assert(STAGES >= 2 && LDS_BYTES <= 160 * 1024, "LDS ring");
  static_assert(LOADS * (STAGES - 2) < 64, "vmcnt range");
  static constexpr int NN_RB = BN * 2;                         // NN panel row bytes
  static_assert(!(NN && (EPI == EPI_SWIGLU || BWD)), "SwiGLU operands are [N, K]");
  static_assert(WM % 32 == 0 && WN % 32 == 0, "wave tile");
  static_assert((BM / 8) % WAVES == 0 && (NB / 8) % WAVES == 0, "NT DMA cover");
  static_assert(!NN || (BK * NN_RB / 1024) % WAVES == 0, "NN DMA cover");
};

// Output tile t of a tiles_m x tiles_n grid in the work order: blocks of kTileGroupM
// consecutive row tiles, column tiles in order within a block and the rows of a block
// fastest, so that the 32 consecutive tiles an XCD runs at a time span about as many row
// as column tiles and its L2 serves each operand panel to several of them.
constexpr int kTileGroupM = 4;
__device__ __forceinline__ void tile_coords(int t, int tiles_m, int tiles_n, int* tm, int* tn) {
  const int blk = t / (kTileGroupM * tiles_n), in = t - blk * kTileGroupM * tiles_n;
  const int rows = min(kTileGroupM, tiles_m - blk * kTileGroupM);
  *tm = blk * kTileGroupM + in % rows;
  *tn = in / rows;
}

// Chunk swizzles of the NT and NN panels (physical chunk = logical chunk XOR swz(row)).
__device__ __forceinline__ int nt_swz(int row) { return (row >> 1) & 7; }
__device__ __forceinline__ int nn_swz(int row) { return 4 * (row & 3); }

// Operand panels go HBM -> LDS through buffer loads with an LDS destination (lds_dma.h):
// address = resource base (the matrix) + scalar offset (the stage's K position) + a
// per-lane offset.  The per-lane offsets only depend on the tile and the lane, so they
// are formed once per tile and a stage is issued without vector arithmetic.  The byte
// extent of every operand must stay below 4 GiB (checked at launch).
//
// NT panel rows [row0, row0 + ROWS) x k [k0, k0 + 64) of a row-major [nrows, ld] matrix
// (128-byte LDS rows): instruction i of wave w fills rows 8 (i W + w) .. +7, lane l row
// 8 (i W + w) + l / 8, physical chunk l % 8 (logical chunk XOR nt_swz(row)); rows past
// nrows are clamped to the last one.  Stage offset: 2 k0 bytes.
template <int ROWS, int WAVES>
struct NtRows {
  static constexpr int NI = ROWS / 8 / WAVES;
  uint32_t off[NI];
  __device__ __forceinline__ void init(int ld, int row0, int nrows, int wave, int lane) {
    const int rsub = lane >> 3, pc = lane & 7;
#pragma unroll
    for (int i = 0; i < NI; ++i) {
      const int r = 8 * (i * WAVES + wave) + rsub;
      const uint32_t grow = (uint32_t)min(row0 + r, nrows - 1);
      off[i] = 2u * (grow * (uint32_t)ld + 8u * (uint32_t)(pc ^ nt_swz(r)));
    }
  }
  __device__ __forceinline__ void issue(lds_char* dst, const rsrc_t& rs, uint32_t k0,
                                        int wave) const {
#pragma unroll
    for (int i = 0; i < NI; ++i) dma16(rs, off[i], 2u * k0, dst + (i * WAVES + wave) * 1024);
  }
};

// NN panel: k rows [k0, k0 + 64) x n [n0, n0 + BN) of a row-major [krows, ld] matrix
// (natural layout, BN * 2-byte LDS rows, chunk XOR nn_swz(row)); instruction i of wave w
// fills rows RPI (i W + w) .. +RPI-1.  Columns past ncols are clamped (in the per-lane
// offsets) and rows past krows too (only in a stage that reaches past them).
template <int BN, int WAVES>
struct NnRows {
  static constexpr int CH = BN / 8, RPI = kWave / CH, NI = BK / RPI / WAVES;
  uint32_t off[NI];  // 2 (r ld + gn): row r of the stage, column gn
  int r0;            // this lane's row in instruction 0 (instruction i: r0 + i RPI W)
  __device__ __forceinline__ void init(int ld, int n0, int ncols, int wave, int lane) {
    const int rsub = lane / CH, pc = lane % CH;
    r0 = RPI * wave + rsub;
#pragma unroll
    for (int i = 0; i < NI; ++i) {
      const int r = r0 + i * RPI * WAVES;
      const uint32_t gn = (uint32_t)min(n0 + 8 * (pc ^ nn_swz(r)), ncols - 8);
      off[i] = 2u * ((uint32_t)r * (uint32_t)ld + gn);
    }
  }
  __device__ __forceinline__ void issue(lds_char* dst, const rsrc_t& rs, int k0, int krows,
                                        int ld, int wave) const {
    if (k0 + BK <= krows) {
      const uint32_t soff = 2u * (uint32_t)k0 * (uint32_t)ld;
#pragma unroll
      for (int i = 0; i < NI; ++i) dma16(rs, off[i], soff, dst + (i * WAVES + wave) * 1024);
    } else {
#pragma unroll
      for (int i = 0; i < NI; ++i) {
        const int r = r0 + i * RPI * WAVES;
        const int gk = min(k0 + r, krows - 1);
        const uint32_t voff = off[i] + 2u * (uint32_t)(gk - r) * (uint32_t)ld;
        dma16(rs, voff, 0u, dst + (i * WAVES + wave) * 1024);
      }
    }
  }
};

// Orders this wavefront's LDS writes before its later LDS reads (and those reads before
// its next writes) without a workgroup barrier: every wavefront stages its blocks in an
// LDS region of its own, and LDS operations of one wavefront complete in issue order, so
// only the compiler must be kept from moving them across each other.
__device__ __forceinline__ void wave_lds_sync() {
  __builtin_amdgcn_fence(__ATOMIC_SEQ_CST, "wavefront");
  __builtin_amdgcn_wave_barrier();
}

// Epilogue of one C tile (configuration C: WAVES, WM, WN, TM, TN, TNB, LDS_BYTES, BWD)
// from the accumulators of each wavefront, staged through the workgroup's LDS (free:
// every operand read has completed).
template <class C, int EPI>
__device__ __forceinline__ void gemm_epilogue(const GemmParams& P, f32x16 (&acc)[C::TM][C::TNB],
                                              char* L, const int wave, const int lane,
                                              const int m0, const int n0, const int wm,
                                              const int wn, const int split = 0) {
  constexpr int TM = C::TM, TN = C::TN;
  const int l32 = lane & 31, hh = lane >> 5;
  // Each wavefront stages one 32-row block of its C tile in LDS as fp32, then writes it
  // out in 4-column chunks: consecutive lanes cover consecutive columns, every global
  // access is 16 bytes (fp32) or 8 bytes (bf16), and all loads of a block are in flight
  // before the first store.
  constexpr int EST = C::WN + 4;  // staging row stride in floats
  constexpr int CPR = C::WN / 4;  // 4-column chunks per row
  constexpr int PER_LANE = 32 * CPR / kWave;
  static_assert(C::WAVES * 32 * EST * 4 <= C::LDS_BYTES, "epilogue staging fits");
  float* E = reinterpret_cast<float*>(L) + wave * 32 * EST;
  const int ncol0 = n0 + wn * C::WN;
  if constexpr (C::BWD) {
    // SwiGLU backward.  Per 32-row block: dG, dU and Hs replace G, U and dHs in the
    // accumulators, then each goes through LDS once: dG and dU to their row-major
    // outputs (4-column chunks, as the forward's Hs), and all three transposed (each
    // lane writes 8 consecutive rows of one column as one 16-byte vector).
#pragma unroll
    for (int i = 0; i < TM; ++i) {
#pragma unroll
      for (int j = 0; j < TN; ++j)
#pragma unroll
        for (int e = 0; e < 16; ++e) {
          const float g = acc[i][j][e], u = acc[i][j + TN][e], dh = acc[i][j + 2 * TN][e];
          const float sg = __builtin_amdgcn_rcpf(1.f + __expf(-g));
          const float sl = g * sg;
          acc[i][j][e] = dh * u * (sg * (1.f + g * (1.f - sg)));  // dG
          acc[i][j + TN][e] = dh * sl;                           // dU
          acc[i][j + 2 * TN][e] = sl * u;                        // Hs
        }
      const int mrow0 = m0 + wm * C::WM + 32 * i;
#pragma unroll
      for (int q = 0; q < 3; ++q) {
#pragma unroll
        for (int j = 0; j < TN; ++j)
#pragma unroll
          for (int e = 0; e < 16; ++e)
            E[(8 * (e >> 2) + 4 * hh + (e & 3)) * EST + 32 * j + l32] = acc[i][q * TN + j][e];
        wave_lds_sync();
        if (q < 2) {
          uint16_t* H = q == 0 ? P.H : P.H2;
#pragma unroll
          for (int r = 0; r < PER_LANE; ++r) {
            const int idx = r * kWave + lane, row = idx / CPR, c4 = idx % CPR;
            const int mm = mrow0 + row, nn = ncol0 + 4 * c4;
            if (mm >= P.M || nn >= P.ldh) continue;  // columns N..ldh: zero padding
            const f32x4 v = *reinterpret_cast<const f32x4*>(E + row * EST + 4 * c4);
            *reinterpret_cast<u32x2*>(H + (size_t)mm * P.ldh + nn) =
                nn < P.N ? u32x2{pack_bf16x2(v[0], v[1]), pack_bf16x2(v[2], v[3])}
                         : u32x2{0u, 0u};
          }
        }
        uint16_t* T = q == 0 ? P.T0 : (q == 1 ? P.T1 : P.T2);
        for (int k = lane; k < 4 * C::WN; k += kWave) {
          const int c = k % C::WN, r0 = 8 * (k / C::WN);
          const int nn = ncol0 + c, mm = mrow0 + r0;
          if (nn >= P.N || mm >= P.ldt) continue;  // rows M..ldt: zero padding
          uint32_t w[4];
#pragma unroll
          for (int e = 0; e < 4; ++e) {
            const float v0 = mm + 2 * e < P.M ? E[(r0 + 2 * e) * EST + c] : 0.f;
            const float v1 = mm + 2 * e + 1 < P.M ? E[(r0 + 2 * e + 1) * EST + c] : 0.f;
            w[e] = pack_bf16x2(v0, v1);
          }
          *reinterpret_cast<u32x4*>(T + (size_t)nn * P.ldt + mm) = u32x4{w[0], w[1], w[2], w[3]};
        }
        wave_lds_sync();
      }
    }
    return;
  }
#pragma unroll
  for (int i = 0; i < TM; ++i) {
#pragma unroll
    for (int j = 0; j < TN; ++j)
#pragma unroll
      for (int e = 0; e < 16; ++e) {
        float v = acc[i][j][e];
        if constexpr (EPI == EPI_SWIGLU)
          v = v * __builtin_amdgcn_rcpf(1.f + __expf(-v)) * acc[i][j + TN][e];
        E[(8 * (e >> 2) + 4 * hh + (e & 3)) * EST + 32 * j + l32] = v;
      }
    wave_lds_sync();
    const int mrow0 = m0 + wm * C::WM + 32 * i;
    // Q/K/V scatter: batch entry and token of the block's first row, once per block (a row
    // r of the block is then token t0 + r of entry b0, or of the next entry past its end).
    int b0 = 0, t0 = 0;
    if constexpr (EPI == EPI_QKV) {
      b0 = mrow0 / P.rows_per_batch;
      t0 = mrow0 - b0 * P.rows_per_batch;
    }
    f32x4 v[PER_LANE];
    int mm[PER_LANE], nn[PER_LANE];
    bool ok[PER_LANE];
#pragma unroll
    for (int q = 0; q < PER_LANE; ++q) {
      const int idx = q * kWave + lane, row = idx / CPR, c4 = idx % CPR;
      v[q] = *reinterpret_cast<const f32x4*>(E + row * EST + 4 * c4);
      mm[q] = mrow0 + row;
      nn[q] = ncol0 + 4 * c4;
      ok[q] = mm[q] < P.M && nn[q] < P.N;
    }
    if constexpr (EPI == EPI_ACC) {
      if (P.k_splits > 1) {  // a partial product of one contraction range
        float* dst = P.part + (size_t)split * P.M * P.N;
#pragma unroll
        for (int q = 0; q < PER_LANE; ++q)
          if (ok[q]) *reinterpret_cast<f32x4*>(dst + (size_t)mm[q] * P.N + nn[q]) = v[q];
        wave_lds_sync();
        continue;
      }
      // The base values of the block: every lane loads (chunks outside the product read
      // an in-range element instead and are not stored), so that all loads of the block
      // are issued before the first wait rather than one load and one wait per chunk.
      f32x4 base[PER_LANE];
      if (P.R) {
        u32x2 r[PER_LANE];
#pragma unroll
        for (int q = 0; q < PER_LANE; ++q)
          r[q] = *reinterpret_cast<const u32x2*>(P.R + (size_t)min(mm[q], P.M - 1) * P.ldr +
                                                 min(nn[q], P.N - 4));
#pragma unroll
        for (int q = 0; q < PER_LANE; ++q)
          base[q] = f32x4{bf16_bits_to_f32(r[q][0] & 0xffffu), bf16_bits_to_f32(r[q][0] >> 16),
                          bf16_bits_to_f32(r[q][1] & 0xffffu), bf16_bits_to_f32(r[q][1] >> 16)};
      } else if (P.accumulate) {
#pragma unroll
        for (int q = 0; q < PER_LANE; ++q)
          base[q] = *reinterpret_cast<const f32x4*>(P.Y + (size_t)min(mm[q], P.M - 1) * P.ldy +
                                                    min(nn[q], P.N - 4));
      } else {
#pragma unroll
        for (int q = 0; q < PER_LANE; ++q) base[q] = f32x4{0.f, 0.f, 0.f, 0.f};
      }
#pragma unroll
      for (int q = 0; q < PER_LANE; ++q) {
        if (!ok[q]) continue;
        const f32x4 out = v[q] + base[q];
        *reinterpret_cast<f32x4*>(P.Y + (size_t)mm[q] * P.ldy + nn[q]) = out;
        if (P.U)
          *reinterpret_cast<u32x2*>(P.U + (size_t)mm[q] * P.ldu + nn[q]) =
              u32x2{pack_bf16x2(out[0], out[1]), pack_bf16x2(out[2], out[3])};
      }
    } else {
#pragma unroll
      for (int q = 0; q < PER_LANE; ++q) {
        if constexpr (EPI == EPI_SWIGLU) {
          // Columns [N, h_cols) are the zero padding of the gated product.
          if (mm[q] >= P.M || nn[q] >= (P.h_cols > 0 ? P.h_cols : P.ldh)) continue;
          const u32x2 bits = nn[q] < P.N ? u32x2{pack_bf16x2(v[q][0], v[q][1]),
                                                 pack_bf16x2(v[q][2], v[q][3])}
                                         : u32x2{0u, 0u};
          *reinterpret_cast<u32x2*>(P.H + (size_t)mm[q] * P.ldh + nn[q]) = bits;
        } else {
          if (!ok[q]) continue;
          const int n = nn[q], m = mm[q];
          const float f = n < P.nq ? P.q_scale : 1.f;  // the Q block is scaled, then rounded
          const u32x2 bits{pack_bf16x2(f * v[q][0], f * v[q][1]),
                           pack_bf16x2(f * v[q][2], f * v[q][3])};
          uint16_t* dst;
          if (n < P.nq) {
            dst = P.Q + (size_t)m * P.ldq + n;
          } else {
            int b = b0, t = t0 + (m - mrow0);
            while (t >= P.rows_per_batch) {  // once at most when entries hold >= 32 rows
              t -= P.rows_per_batch;
              ++b;
            }
            const long long pos = t < P.kv_seg ? P.kv_pos0 + t : P.kv_pos1 + (t - P.kv_seg);
            const size_t row = (size_t)b * P.kv_batch_stride +
                               (size_t)pos * P.kv_row_stride + P.kv_col0;
            dst = n < P.nq + P.nkv ? P.Kb + row + (n - P.nq) : P.Vb + row + (n - P.nq - P.nkv);
          }
          *reinterpret_cast<u32x2*>(dst) = bits;
        }
      }
    }
    wave_lds_sync();
  }
}

// One output tile (work index w) of the product P.
template <int BM, int BN, int WGM, int WGN, bool NN, int EPI, int STAGES>
__device__ __forceinline__ void gemm_tile(const GemmParams& P, const int w) {
  using C = Cfg<BM, BN, WGM, WGN, NN, EPI, STAGES>;
  constexpr int TM = C::TM, TN = C::TN, TNB = C::TNB;
  __shared__ __attribute__((aligned(1024))) char L[C::LDS_BYTES];
  lds_char* Ls = (lds_char*)L;

  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int wm = wave / WGN, wn = wave % WGN;
  const int l32 = lane & 31, hh = lane >> 5;

  const int tiles_n = (P.N + BN - 1) / BN;
  // Work index -> (contraction range, output tile): ranges outermost.
  int split = 0, wt = w;
  if (EPI == EPI_ACC && P.k_splits > 1) {
    const int tiles = ((P.M + BM - 1) / BM) * tiles_n;
    split = w / tiles;
    wt = w - split * tiles;
  }
  int tm, tn;
  tile_coords(wt, (P.M + BM - 1) / BM, tiles_n, &tm, &tn);
  const int m0 = tm * BM, n0 = tn * BN;

  f32x16 acc[TM][TNB];
#pragma unroll
  for (int i = 0; i < TM; ++i)
#pragma unroll
    for (int j = 0; j < TNB; ++j)
#pragma unroll
      for (int e = 0; e < 16; ++e) acc[i][j][e] = 0.f;

  // The operand pairs of a multi-part contraction, read once into scalar registers (the
  // asm keeps them there: the per-stage choice is then a chain of scalar selects, not an
  // indexed access, which would put the parameters in scratch memory).
  const uint16_t* ap[kGemmPartsMax];
  const uint16_t* bp[kGemmPartsMax];
  int k_part = INT_MAX;
  if constexpr (NN) {
    const bool multi = P.n_parts > 1;
#pragma unroll
    for (int i = 0; i < kGemmPartsMax; ++i) {
      ap[i] = multi && i < P.n_parts ? P.A_part[i] : P.A;
      bp[i] = multi && i < P.n_parts ? P.B_part[i] : P.B;
      asm volatile("" : "+s"(ap[i]), "+s"(bp[i]));
    }
    if (multi) k_part = P.k_part;
    asm volatile("" : "+s"(k_part));
  }
  // Per-lane DMA offsets of this tile (A and A2 share rows and stride, as do the NT B
  // panels), and the operands' buffer resources.
  // With HALF_LOADERS only the first half of the wavefronts (one per SIMD: wavefronts are
  // placed on the SIMDs round-robin) issue loads, each its own share and that of
  // wavefront wave + W/2 (the other wavefront of its SIMD): a CU's load path takes a
  // stage's 64 KB at about 60 bytes per cycle, so a wavefront that issues loads stalls
  // for hundreds of cycles, and this way one wavefront of every SIMD never does and keeps
  // the matrix pipe fed meanwhile.
  constexpr int HW = C::WAVES / 2;
  const bool loader = !C::HALF_LOADERS || wave < HW;
  const int wave2 = wave + HW;
  NtRows<BM, C::WAVES> rows_a, rows_a_hi;
  rows_a.init(P.lda, m0, P.M, wave, lane);
  if constexpr (C::HALF_LOADERS) rows_a_hi.init(P.lda, m0, P.M, wave2, lane);
  NtRows<NN ? 8 * C::WAVES : BN, C::WAVES> rows_b, rows_b_hi;  // (unused for NN)
  NnRows<BN, C::WAVES> rows_nn, rows_nn_hi;                     // (unused for NT)
  if constexpr (NN) {
    rows_nn.init(P.ldb, n0, P.N, wave, lane);
    if constexpr (C::HALF_LOADERS) rows_nn_hi.init(P.ldb, n0, P.N, wave2, lane);
  } else {
    rows_b.init(P.ldb, n0, P.N, wave, lane);
    if constexpr (C::HALF_LOADERS) rows_b_hi.init(P.ldb, n0, P.N, wave2, lane);
  }
  const rsrc_t rs_a = make_rsrc(P.A);
  const rsrc_t rs_a2 = make_rsrc(C::BWD ? P.A2 : P.A);
  const rsrc_t rs_b = make_rsrc(P.B);
  const rsrc_t rs_b2 = make_rsrc(EPI == EPI_SWIGLU || C::BWD ? P.B2 : P.B);
  const rsrc_t rs_b3 = make_rsrc(C::BWD ? P.B3 : P.B);
  auto dma_stage = [&](int stage, int k0) __attribute__((always_inline)) {
    if (!loader) return;
    lds_char* S = Ls + stage * C::STAGE;
    if constexpr (NN) {
      // (k0 is uniform: the part is chosen per stage, from scalar values)
      const int part = k0 / k_part, kk = k0 - part * k_part;
      const uint16_t* a = ap[0];
      const uint16_t* b = bp[0];
#pragma unroll
      for (int i = 1; i < kGemmPartsMax; ++i) {
        a = part == i ? ap[i] : a;
        b = part == i ? bp[i] : b;
      }
      const rsrc_t ra = make_rsrc(a), rb = make_rsrc(b);
      rows_a.issue(S, ra, (uint32_t)kk, wave);
      if constexpr (C::HALF_LOADERS) rows_a_hi.issue(S, ra, (uint32_t)kk, wave2);
      rows_nn.issue(S + C::A_BYTES, rb, kk, P.Kb_rows, P.ldb, wave);
      if constexpr (C::HALF_LOADERS)
        rows_nn_hi.issue(S + C::A_BYTES, rb, kk, P.Kb_rows, P.ldb, wave2);
      return;
    }
    rows_a.issue(S, rs_a, (uint32_t)k0, wave);
    if constexpr (C::HALF_LOADERS) rows_a_hi.issue(S, rs_a, (uint32_t)k0, wave2);
    if constexpr (C::BWD) {
      rows_a.issue(S + BM * BK * 2, rs_a2, (uint32_t)k0, wave);
      if constexpr (C::HALF_LOADERS) rows_a_hi.issue(S + BM * BK * 2, rs_a2, (uint32_t)k0, wave2);
    }
    rows_b.issue(S + C::A_BYTES, rs_b, (uint32_t)k0, wave);
    if constexpr (C::HALF_LOADERS) rows_b_hi.issue(S + C::A_BYTES, rs_b, (uint32_t)k0, wave2);
    if constexpr (EPI == EPI_SWIGLU || C::BWD) {
      rows_b.issue(S + C::A_BYTES + BN * BK * 2, rs_b2, (uint32_t)k0, wave);
      if constexpr (C::HALF_LOADERS)
        rows_b_hi.issue(S + C::A_BYTES + BN * BK * 2, rs_b2, (uint32_t)k0, wave2);
    }
    if constexpr (C::BWD) {
      rows_b.issue(S + C::A_BYTES + 2 * BN * BK * 2, rs_b3, (uint32_t)k0, wave);
      if constexpr (C::HALF_LOADERS)
        rows_b_hi.issue(S + C::A_BYTES + 2 * BN * BK * 2, rs_b3, (uint32_t)k0, wave2);
    }
  };

  // Operand addressing (see the header): A / NT-B row R, chunk 2 s + hh ->
  //   R_base * 128 + (opa ^ 32 s),  opa = l32 * 128 + 16 (hh ^ nt_swz(l32)).
  const int opa = l32 * 128 + 16 * (hh ^ nt_swz(l32));
  // NN-B transpose reads for output column block j: rows 16 s + 8 hh + t/4 (+4), columns
  // wn WN + 32 j + 16 (g mod 2) + 4 (t mod 4)  ->  16 s NN_RB + (nb ^ 2 (wn WN + 32 j)).
  int nb_lo = 0, nb_hi = 0;
  if constexpr (NN) {
    const int t = lane & 15, g = lane >> 4;
    const int cl = 2 * (g & 1) + ((t & 3) >> 1), half8 = 8 * (t & 1);
    const int r_lo = 8 * (g >> 1) + (t >> 2), r_hi = r_lo + 4;
    nb_lo = r_lo * C::NN_RB + 16 * (cl ^ nn_swz(r_lo)) + half8;
    nb_hi = r_hi * C::NN_RB + 16 * (cl ^ nn_swz(r_hi)) + half8;
  }

  // STAGES-deep ring: stage k lives in slot k mod STAGES.  Step kt waits for stage kt
  // (the loads of up to STAGES - 2 later stages stay in flight), then refills the slot
  // that step kt - 1 read with stage kt + STAGES - 1.
  // Contraction steps [kb, kb + nk) (all of them unless the contraction is split); step
  // kb + kt lives in ring slot kt mod STAGES.
  int kb = 0, nk = P.K / BK;
  if (EPI == EPI_ACC && P.k_splits > 1) {
    const int all = nk;
    kb = split * all / P.k_splits;
    nk = (split + 1) * all / P.k_splits - kb;
  }
#pragma unroll
  for (int st = 0; st < STAGES - 1; ++st)
    if (st < nk) dma_stage(st, (kb + st) * BK);
  for (int kt = 0; kt < nk; ++kt) {
    const int ahead = min(STAGES - 2, nk - 1 - kt);  // later stages already issued
    if constexpr (STAGES >= 4) {
      if (ahead >= 2) wait_dma<C::LOADS * 2>();
      else if (ahead == 1) wait_dma<C::LOADS>();
      else wait_dma<0>();
    } else if constexpr (STAGES == 3) {
      if (ahead >= 1) wait_dma<C::LOADS>();
      else wait_dma<0>();
    } else {
      wait_dma<0>();
    }
    __syncthreads();  // stage kt resident; every wave is past step kt-1
    const lds_char* SA = Ls + (kt % STAGES) * C::STAGE;
    const lds_char* SB = SA + C::A_BYTES;
    // Operands of substep s into set s % 2.
    u32x4 a[2][TM], a2[2][TM], b[2][TNB];
    auto read_sub = [&](int s) __attribute__((always_inline)) {
      const int xo = opa ^ (32 * s), q = s & 1;
#pragma unroll
      for (int i = 0; i < TM; ++i) a[q][i] = lds_read16(SA + (wm * C::WM + 32 * i) * 128 + xo);
      if constexpr (C::BWD) {
#pragma unroll
        for (int i = 0; i < TM; ++i)
          a2[q][i] = lds_read16(SA + BM * BK * 2 + (wm * C::WM + 32 * i) * 128 + xo);
      }
#pragma unroll
      for (int j = 0; j < TNB; ++j) {
        if constexpr (NN) {
          const int cx = 2 * (wn * C::WN + 32 * j);
          const u32x2 lo = lds_read_tr(SB + 16 * s * C::NN_RB + (nb_lo ^ cx));
          const u32x2 hi = lds_read_tr(SB + 16 * s * C::NN_RB + (nb_hi ^ cx));
          b[q][j] = u32x4{lo[0], lo[1], hi[0], hi[1]};
        } else {
          const int brow = (j / TN) * BN + wn * C::WN + 32 * (j % TN);  // panel j / TN
          b[q][j] = lds_read16(SB + brow * 128 + xo);
        }
      }
    };
    // The first substep's operand reads go out before the refill, so their LDS latency
    // overlaps the issue of the next stage's loads.
    read_sub(0);
    if (kt + STAGES - 1 < nk)
      dma_stage((kt + STAGES - 1) % STAGES, (kb + kt + STAGES - 1) * BK);
#pragma unroll
    for (int s = 0; s < BK / 16; ++s) {
      if (s + 1 < BK / 16) read_sub(s + 1);
      const int q = s & 1;
#pragma unroll
      for (int i = 0; i < TM; ++i)
#pragma unroll
        for (int j = 0; j < TNB; ++j)
          acc[i][j] = mfma32(C::BWD && j >= 2 * TN ? a2[q][i] : a[q][i], b[q][j], acc[i][j]);
    }
    // Issue order: the operand reads of k-substep s+1 are spread between the MFMAs of
    // substep s (R / M per MFMA, one more for the first R mod M), so LDS latency hides
    // behind matrix work.
    {
      constexpr int R = C::NAP * TM + (NN ? 2 : 1) * TNB;  // LDS reads per substep
      constexpr int M = TM * TNB;                          // MFMAs per substep
      constexpr int RM = R / M;
      __builtin_amdgcn_sched_group_barrier(0x100, R, 0);
#pragma unroll
      for (int s = 0; s < BK / 16; ++s)
#pragma unroll
        for (int i = 0; i < M; ++i) {
          __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
          if (s + 1 < BK / 16) {
            if (i < R % M) __builtin_amdgcn_sched_group_barrier(0x100, RM + 1, 0);
            else if (RM > 0) __builtin_amdgcn_sched_group_barrier(0x100, RM, 0);
          }
        }
    }
  }
  __syncthreads();  // operand stages are free for the epilogue

  gemm_epilogue<C, EPI>(P, acc, L, wave, lane, m0, n0, wm, wn, split);
}

template <int BM, int BN, int WGM, int WGN, bool NN, int EPI, int STAGES>
__global__ __launch_bounds__(kWave * WGM * WGN) void gemm_kernel(const GemmParams P) {
  const int tiles = ((P.M + BM - 1) / BM) * ((P.N + BN - 1) / BN);
  const int items = EPI == EPI_ACC && P.k_splits > 1 ? tiles * P.k_splits : tiles;
  gemm_tile<BM, BN, WGM, WGN, NN, EPI, STAGES>(P, xcd_work_index(blockIdx.x, items));
}

// Y = base + sum of the k_splits partial products in range order (base and U as in the
// accumulate epilogue); 4 consecutive columns per thread.
__global__ __launch_bounds__(256) void splitk_reduce_kernel(const GemmParams P) {
  const int c4 = P.N / 4;
  const long long i = (long long)blockIdx.x * 256 + threadIdx.x;
  if (i >= (long long)P.M * c4) return;
  const int m = (int)(i / c4), n = 4 * (int)(i - (long long)m * c4);
  const size_t mn = (size_t)P.M * P.N, at = (size_t)m * P.N + n;
  f32x4 sum = *reinterpret_cast<const f32x4*>(P.part + at);
  for (int c = 1; c < P.k_splits; ++c) sum += *reinterpret_cast<const f32x4*>(P.part + c * mn + at);
  f32x4 base = f32x4{0.f, 0.f, 0.f, 0.f};
  if (P.R) {
    const u32x2 r = *reinterpret_cast<const u32x2*>(P.R + (size_t)m * P.ldr + n);
    base = f32x4{bf16_bits_to_f32(r[0] & 0xffffu), bf16_bits_to_f32(r[0] >> 16),
                 bf16_bits_to_f32(r[1] & 0xffffu), bf16_bits_to_f32(r[1] >> 16)};
  } else if (P.accumulate) {
    base = *reinterpret_cast<const f32x4*>(P.Y + (size_t)m * P.ldy + n);
  }
  const f32x4 out = sum + base;
  *reinterpret_cast<f32x4*>(P.Y + (size_t)m * P.ldy + n) = out;
  if (P.U)
    *reinterpret_cast<u32x2*>(P.U + (size_t)m * P.ldu + n) =
        u32x2{pack_bf16x2(out[0], out[1]), pack_bf16x2(out[2], out[3])};
}

// Up to kGemmGroupMax independent products of one configuration in one launch: the tiles of
// product i follow those of the products before it, so small products that would each
// leave CUs idle fill the chip together.
struct GemmGroup {
  GemmParams p[kGemmGroupMax];
  int n;
};
static_assert(sizeof(GemmGroup) <= 4096, "kernel argument size limit");
template <int BM, int BN, int WGM, int WGN, bool NN, int EPI, int STAGES>
__global__ __launch_bounds__(kWave * WGM * WGN) void gemm_group_kernel(const GemmGroup G) {
  int tiles[kGemmGroupMax], total = 0;
#pragma unroll
  for (int i = 0; i < kGemmGroupMax; ++i) {
    tiles[i] = i < G.n ? ((G.p[i].M + BM - 1) / BM) * ((G.p[i].N + BN - 1) / BN) : 0;
    total += tiles[i];
  }
  int w = xcd_work_index(blockIdx.x, total), i = 0;
  while (i + 1 < G.n && w >= tiles[i]) w -= tiles[i++];  // uniform per workgroup
  // A copy of the product's parameters: read through G.p[i] (an index into the kernel
  // arguments), the compiler reloads every field after each global store of the epilogue
  // (it cannot rule out aliasing), hundreds of serialized scalar loads per tile.
  const GemmParams P = G.p[i];
  gemm_tile<BM, BN, WGM, WGN, NN, EPI, STAGES>(P, w);
}

template <int BM, int BN, int WGM, int WGN, bool NN, int EPI, int STAGES>
hipError_t check_params(const GemmParams& p) {
  if (p.K <= 0 || p.K % BK != 0) return hipErrorInvalidValue;
  // The operand loads address each operand with 32-bit byte offsets from its base.
  constexpr long long kMaxBytes = 1LL << 32;
  const long long b_rows = NN ? (long long)p.Kb_rows : (long long)p.N;
  if ((long long)p.M * p.lda * 2 >= kMaxBytes || b_rows * p.ldb * 2 >= kMaxBytes)
    return hipErrorInvalidValue;
  if (p.k_splits > 1 && (EPI != EPI_ACC || !p.part || p.N % 4 != 0 || p.k_splits > p.K / BK))
    return hipErrorInvalidValue;
  if (p.n_parts > 1) {
    if (!NN || p.n_parts > kGemmPartsMax || p.k_part <= 0 || p.k_part % BK != 0 ||
        (long long)p.n_parts * p.k_part != p.K)
      return hipErrorInvalidValue;
    for (int i = 0; i < p.n_parts; ++i)
      if (!p.A_part[i] || !p.B_part[i]) return hipErrorInvalidValue;
  }
  return hipSuccess;
}

template <int BM, int BN, int WGM, int WGN, bool NN, int EPI, int STAGES>
hipError_t launch_group(const GemmParams* ps, int n, hipStream_t s) {
  using C = Cfg<BM, BN, WGM, WGN, NN, EPI, STAGES>;
  if (n < 1 || n > kGemmGroupMax) return hipErrorInvalidValue;
  GemmGroup g = {};
  long long total = 0;
  for (int i = 0; i < n; ++i) {
    const GemmParams& p = ps[i];
    if (p.M <= 0 || p.N <= 0) return hipErrorInvalidValue;
    const hipError_t e = check_params<BM, BN, WGM, WGN, NN, EPI, STAGES>(p);
    if (e != hipSuccess) return e;
    g.p[i] = p;
    total += (long long)((p.M + BM - 1) / BM) * ((p.N + BN - 1) / BN);
  }
  g.n = n;
  if (total > INT32_MAX) return hipErrorInvalidValue;
  void* args[] = {&g};
  return hipLaunchKernel(
      reinterpret_cast<const void*>(&gemm_group_kernel<BM, BN, WGM, WGN, NN, EPI, STAGES>),
      dim3((unsigned)total), dim3(C::THREADS), args, 0, s);
}

template <int BM, int BN, int WGM, int WGN, bool NN, int EPI, int STAGES>
hipError_t launch(const GemmParams& p, hipStream_t s) {
  using C = Cfg<BM, BN, WGM, WGN, NN, EPI, STAGES>;
  if (p.M <= 0 || p.N <= 0) return hipSuccess;
  const hipError_t e = check_params<BM, BN, WGM, WGN, NN, EPI, STAGES>(p);
  if (e != hipSuccess) return e;
  long long tiles = (long long)((p.M + BM - 1) / BM) * ((p.N + BN - 1) / BN);
  if (EPI == EPI_ACC && p.k_splits > 1) tiles *= p.k_splits;
  if (tiles > INT32_MAX) return hipErrorInvalidValue;
  // hipLaunchKernel returns the status of this launch only (not an earlier error).
  void* args[] = {const_cast<GemmParams*>(&p)};
  return hipLaunchKernel(reinterpret_cast<const void*>(&gemm_kernel<BM, BN, WGM, WGN, NN, EPI, STAGES>),
                         dim3((unsigned)tiles), dim3(C::THREADS), args, 0, s);
}

long long tiles_of(const GemmParams* ps, int n, int bm, int bn) {
  long long t = 0;
  for (int i = 0; i < n && i < kGemmGroupMax; ++i)
    t += (long long)((ps[i].M + bm - 1) / bm) * ((ps[i].N + bn - 1) / bn);
  return t;
}

}  // namespace

// Tile shapes are chosen for the grouped shard products of the 7B-class layer on 256
// CUs (one workgroup per CU).  Gate+up (M = S_loc, N = F/D = 1376 per shard, 8 shards
// per launch) takes 256 x 128 tiles (256 x 256 accumulators: gate and up) with a 2-slot
// ring when they make at least 4 rounds (S_loc = 8192: 2816 tiles), else 128 x 128 tiles
// with a 3-slot ring;
// Q/K/V (N = 3 d H_s = 1536 per shard) 256 x 256 tiles when they make two rounds or more
// (S_loc = 8192: 1536 tiles), else 256 x 192 (S_loc = 1024: 256 tiles, one per CU) or,
// below one tile per CU, 128 x 128; down / O-proj (N = h = 4096)
// 256 x 256 tiles (512 at S_loc = 8192), their contraction split when that makes fewer
// tiles than CUs.
constexpr long long kCus = 256;

hipError_t launch_gemm_swiglu(const GemmParams& p, hipStream_t s) {
  return launch_gemm_swiglu_group(&p, 1, s);
}

hipError_t launch_gemm_swiglu_group(const GemmParams* ps, int n, hipStream_t s) {
  if (tiles_of(ps, n, 256, 128) >= 4 * kCus) {
    if (n == 1) return launch<256, 128, 2, 4, false, EPI_SWIGLU, 2>(ps[0], s);
    return launch_group<256, 128, 2, 4, false, EPI_SWIGLU, 2>(ps, n, s);
  }
  if (n == 1) return launch<128, 128, 2, 4, false, EPI_SWIGLU, 3>(ps[0], s);
  return launch_group<128, 128, 2, 4, false, EPI_SWIGLU, 3>(ps, n, s);
}

// Below one 256 x 256 output tile per CU (short sequences: M = S_loc = 1024 and N = h =
// 4096 make 64) the contraction is split into ranges, enough (tile, range) items for
// every CU with at least 16 steps of 64 per range; the partial products go through an
// fp32 workspace and a reduction kernel that applies the epilogue.
int gemm_nn_acc_splits(int M, int N, int K) {
  const long long tiles = (long long)((M + 255) / 256) * ((N + 255) / 256);
  if (tiles <= 0 || tiles >= kCus || N % 4 != 0) return 1;
  int splits = (int)((kCus + tiles - 1) / tiles);
  const int max_splits = K / BK / 16;
  if (splits > max_splits) splits = max_splits;
  return splits > 1 ? splits : 1;
}

hipError_t launch_gemm_nn_acc(const GemmParams& p, float* part, hipStream_t s) {
  if (p.M <= 0 || p.N <= 0) return hipSuccess;
  const int splits = gemm_nn_acc_splits(p.M, p.N, p.K);
  if (splits == 1) {
    GemmParams q = p;
    q.k_splits = 1;
    return launch<256, 256, 2, 4, true, EPI_ACC, 2>(q, s);
  }
  if (!part) {  // no workspace: the whole contraction per tile, on 128 x 128 tiles
    GemmParams q = p;
    q.k_splits = 1;
    return launch<128, 128, 2, 4, true, EPI_ACC, 2>(q, s);
  }
  GemmParams q = p;
  q.k_splits = splits;
  q.part = part;
  hipError_t e = launch<256, 256, 2, 4, true, EPI_ACC, 2>(q, s);
  if (e != hipSuccess) return e;
  const long long threads = (long long)p.M * (p.N / 4);
  void* args[] = {&q};
  return hipLaunchKernel(reinterpret_cast<const void*>(&splitk_reduce_kernel),
                         dim3((unsigned)((threads + 255) / 256)), dim3(256), args, 0, s);
}

// SwiGLU backward (M = S_loc, N = F/D): 128 x 128 tiles with five 16 KB operand panels
// per K step (X, dY; W1, W3, W2), two slots = 160 KB.
hipError_t launch_gemm_swiglu_bwd(const GemmParams& p, hipStream_t s) {
  if (p.ldt % 8 != 0 || p.ldt < p.M) return hipErrorInvalidValue;
  return launch<128, 128, 2, 4, false, EPI_SWIGLU_BWD, 2>(p, s);
}

// Weight gradients (M = F/D, N = h, K = tokens): 128 x 128 tiles make 352 at the 7B
// shape where 256 x 256 would make 96.
hipError_t launch_gemm_nn_acc_small(const GemmParams& p, hipStream_t s) {
  return launch<128, 128, 2, 4, true, EPI_ACC, 2>(p, s);
}

// Several weight-gradient products in one launch (each with M = F/D or H_s d rows).
hipError_t launch_gemm_nn_acc_small_group(const GemmParams* ps, int n, hipStream_t s) {
  return launch_group<128, 128, 2, 4, true, EPI_ACC, 2>(ps, n, s);
}

// Projections with few output tiles (the backward's Q and dA products, N = H_s d; GQA
// shapes; short sequences) would leave CUs idle with 256 x 192 tiles: below one tile per
// CU they take 128 x 128 tiles.
hipError_t launch_gemm_qkv(const GemmParams& p, hipStream_t s) {
  if (p.M <= 0 || p.N <= 0) return hipSuccess;
  return launch_gemm_qkv_group(&p, 1, s);
}

hipError_t launch_gemm_qkv_group(const GemmParams* ps, int n, hipStream_t s) {
  if (tiles_of(ps, n, 256, 256) >= 2 * kCus) {
    if (n == 1) return launch<256, 256, 2, 4, false, EPI_QKV, 2>(ps[0], s);
    return launch_group<256, 256, 2, 4, false, EPI_QKV, 2>(ps, n, s);
  }
  if (tiles_of(ps, n, 256, 192) < kCus) {
    if (n == 1) return launch<128, 128, 2, 4, false, EPI_QKV, 2>(ps[0], s);
    return launch_group<128, 128, 2, 4, false, EPI_QKV, 2>(ps, n, s);
  }
  if (n == 1) return launch<256, 192, 4, 2, false, EPI_QKV, 2>(ps[0], s);
  return launch_group<256, 192, 4, 2, false, EPI_QKV, 2>(ps, n, s);
}

}  // namespace tsp
