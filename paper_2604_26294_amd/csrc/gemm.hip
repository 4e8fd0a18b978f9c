// bf16 MFMA GEMM family for the TSP shard products (gfx950).
//
//   gate+up+SwiGLU  Hs = bf16( SiLU(X W1^T) * (X W3^T) )          Algorithm 2, gate/up
//   down / O-proj   Y (+)= Hs W2   or   Y (+)= Flatten(A) W_O^T    Algorithm 2 / 1, "+="
//   Q/K/V proj      Q = X W_Q^T -> workspace, K, V -> full-sequence buffers  Algorithm 1
//
// One workgroup = 256 threads = 4 wavefronts in a 2 x 2 grid; each wavefront owns a
// (BM/2) x (BN/2) block of C as 32 x 32 MFMA tiles.  K advances in steps of 64: the
// next A/B panels are fetched into registers while the MFMAs consume the current
// panels from LDS (two LDS stages, one barrier per step).  Every panel is stored in
// LDS as rows of eight 16-byte chunks (64 bf16 of the contraction dimension) so each
// MFMA operand is one 16-byte LDS read.  Operands stored [K, N] (W2, W_O^T) are
// transposed on the way into LDS with an in-register 8 x 8 (or 4 x 8) block swap, so
// both operand layouts share one inner loop and no extra pass over HBM is made.
#include "common.h"
#include "internal.h"

namespace tsp {
namespace {

constexpr int BK = 64;
constexpr int kThreads = 256;
enum { EPI_SWIGLU = 0, EPI_ACC = 1, EPI_QKV = 2 };

__device__ __forceinline__ int swz8(int row, int chunk) {
  return chunk ^ ((row ^ (row >> 3)) & 7);
}

template <int BM, int BN, bool NN, int EPI>
struct Cfg {
  static constexpr int NB = EPI == EPI_SWIGLU ? 2 * BN : BN;  // B rows held in LDS
  static constexpr int WM = BM / 2, WN = BN / 2;
  static constexpr int TM = WM / 32, TN = WN / 32;
  static constexpr int TNB = EPI == EPI_SWIGLU ? 2 * TN : TN;
  static constexpr int A_LOADS = BM / 32;
  static constexpr int B_LOADS = NN ? BN / 32 : NB / 32;      // NN: KH rows of one block
  static constexpr int STAGE = (BM + NB) * 8;                 // 16-byte chunks per stage
  static_assert(!(NN && EPI == EPI_SWIGLU), "SwiGLU operands are [N, K]");
  static_assert(BM % 64 == 0 && BN % 64 == 0, "tile");
};

// Row-major [rows, K] panel rows row0 .. row0+ROWS-1, columns k0 .. k0+63.
template <int NLOAD>
__device__ __forceinline__ void load_panel(u32x4 (&r)[NLOAD], const uint16_t* __restrict__ base,
                                           int ld, int row0, int nrows, int k0, int K,
                                           int tid) {
  const int k = k0 + 8 * (tid & 7);
#pragma unroll
  for (int i = 0; i < NLOAD; ++i) {
    const int row = row0 + (tid >> 3) + 32 * i;
    r[i] = (row < nrows && k < K) ? ld16(base + (size_t)row * ld + k) : u32x4{0u, 0u, 0u, 0u};
  }
}

template <int NLOAD>
__device__ __forceinline__ void store_panel(u32x4* L, int lds_row0, const u32x4 (&r)[NLOAD],
                                            int tid) {
  const int c = tid & 7;
#pragma unroll
  for (int i = 0; i < NLOAD; ++i) {
    const int row = (tid >> 3) + 32 * i;
    L[(lds_row0 + row) * 8 + swz8(row, c)] = r[i];
  }
}

// Two rows of bf16 pairs -> one dword holding column `odd` of each row.
__device__ __forceinline__ uint32_t pick_col(uint32_t row_lo, uint32_t row_hi, int odd) {
  return odd ? ((row_lo >> 16) | (row_hi & 0xffff0000u)) : ((row_lo & 0xffffu) | (row_hi << 16));
}

template <int BM, int BN, bool NN, int EPI>
__global__ __launch_bounds__(kThreads) void gemm_kernel(const GemmParams P) {
  using C = Cfg<BM, BN, NN, EPI>;
  constexpr int TM = C::TM, TN = C::TN, TNB = C::TNB;
  __shared__ u32x4 L[2 * C::STAGE];

  const int tid = threadIdx.x;
  const int lane = tid & 63, wave = tid >> 6;
  const int wm = wave >> 1, wn = wave & 1;
  const int l32 = lane & 31, hh = lane >> 5;

  const int tiles_n = (P.N + BN - 1) / BN;
  const int tiles_m = (P.M + BM - 1) / BM;
  const int w = xcd_work_index(blockIdx.x, tiles_m * tiles_n);
  const int m0 = (w / tiles_n) * BM;
  const int n0 = (w % tiles_n) * BN;

  f32x16 acc[TM][TNB];
#pragma unroll
  for (int i = 0; i < TM; ++i)
#pragma unroll
    for (int j = 0; j < TNB; ++j)
#pragma unroll
      for (int e = 0; e < 16; ++e) acc[i][j][e] = 0.f;

  u32x4 ra[C::A_LOADS];
  u32x4 rb[C::B_LOADS];

  // NN operand: thread owns a KH x 8 block (KH contraction rows, 8 output columns).
  constexpr int KH = BN / 32;
  const int nn_nb = tid % (BN / 8), nn_kb = tid / (BN / 8);

  auto load = [&](int k0) {
    load_panel<C::A_LOADS>(ra, P.A, P.lda, m0, P.M, k0, P.K, tid);
    if constexpr (NN) {
      const int n = n0 + 8 * nn_nb;
#pragma unroll
      for (int rr = 0; rr < KH; ++rr) {
        const int k = k0 + KH * nn_kb + rr;
        rb[rr] = (k < P.K && n < P.N) ? ld16(P.B + (size_t)k * P.ldb + n) : u32x4{0u, 0u, 0u, 0u};
      }
    } else if constexpr (EPI == EPI_SWIGLU) {
      u32x4 g[BN / 32], u[BN / 32];
      load_panel<BN / 32>(g, P.B, P.ldb, n0, P.N, k0, P.K, tid);
      load_panel<BN / 32>(u, P.B2, P.ldb, n0, P.N, k0, P.K, tid);
#pragma unroll
      for (int i = 0; i < BN / 32; ++i) {
        rb[i] = g[i];
        rb[BN / 32 + i] = u[i];
      }
    } else {
      load_panel<C::B_LOADS>(rb, P.B, P.ldb, n0, P.N, k0, P.K, tid);
    }
  };

  auto store = [&](int stage) {
    u32x4* S = L + stage * C::STAGE;
    store_panel<C::A_LOADS>(S, 0, ra, tid);
    if constexpr (NN) {
#pragma unroll
      for (int c = 0; c < 8; ++c) {
        const int row = 8 * nn_nb + c;  // output column n within the tile
        if constexpr (KH == 8) {
          u32x4 o;
#pragma unroll
          for (int q = 0; q < 4; ++q) o[q] = pick_col(rb[2 * q][c >> 1], rb[2 * q + 1][c >> 1], c & 1);
          S[(BM + row) * 8 + swz8(row, nn_kb)] = o;
        } else {
          static_assert(KH == 4, "KH");
          u32x2 o;
#pragma unroll
          for (int q = 0; q < 2; ++q) o[q] = pick_col(rb[2 * q][c >> 1], rb[2 * q + 1][c >> 1], c & 1);
          reinterpret_cast<u32x2*>(S)[((BM + row) * 8 + swz8(row, nn_kb >> 1)) * 2 + (nn_kb & 1)] = o;
        }
      }
    } else {
      store_panel<C::B_LOADS>(S, BM, rb, tid);
    }
  };

  const int nk = (P.K + BK - 1) / BK;
  load(0);
  store(0);
  __syncthreads();

  for (int kt = 0; kt < nk; ++kt) {
    const int cur = kt & 1;
    if (kt + 1 < nk) load((kt + 1) * BK);
    const u32x4* S = L + cur * C::STAGE;
#pragma unroll
    for (int s = 0; s < BK / 16; ++s) {
      const int ch = 2 * s + hh;
      u32x4 a[TM], b[TNB];
#pragma unroll
      for (int i = 0; i < TM; ++i) {
        const int row = wm * C::WM + 32 * i + l32;
        a[i] = S[row * 8 + swz8(row, ch)];
      }
#pragma unroll
      for (int j = 0; j < TNB; ++j) {
        const int row = (j < TN ? wn * C::WN + 32 * j : BN + wn * C::WN + 32 * (j - TN)) + l32;
        b[j] = S[(BM + row) * 8 + swz8(row, ch)];
      }
#pragma unroll
      for (int i = 0; i < TM; ++i)
#pragma unroll
        for (int j = 0; j < TNB; ++j) acc[i][j] = mfma32(a[i], b[j], acc[i][j]);
    }
    if (kt + 1 < nk) store(cur ^ 1);
    __syncthreads();
  }

  // ---------------------------------------------------------------- epilogue
  // Each wavefront stages one 32-row block of its C tile in LDS as fp32 (the last
  // main-loop barrier has released the operand stages), then writes it out in
  // 4-column chunks: consecutive lanes cover consecutive columns, every global access
  // is 16 bytes (fp32) or 8 bytes (bf16), and all loads of a block are in flight
  // before the first store.
  constexpr int EST = C::WN + 4;          // staging row stride in floats
  constexpr int CPR = C::WN / 4;          // 4-column chunks per row
  constexpr int PER_LANE = 32 * CPR / kWave;
  float* E = reinterpret_cast<float*>(L) + wave * 32 * EST;
  const int ncol0 = n0 + wn * C::WN;
#pragma unroll
  for (int i = 0; i < TM; ++i) {
#pragma unroll
    for (int j = 0; j < TN; ++j)
#pragma unroll
      for (int e = 0; e < 16; ++e) {
        float v = acc[i][j][e];
        if constexpr (EPI == EPI_SWIGLU) v = v / (1.f + __expf(-v)) * acc[i][j + TN][e];
        E[(8 * (e >> 2) + 4 * hh + (e & 3)) * EST + 32 * j + l32] = v;
      }
    __syncthreads();
    const int mrow0 = m0 + wm * C::WM + 32 * i;
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
      f32x4 base[PER_LANE];
#pragma unroll
      for (int q = 0; q < PER_LANE; ++q) {
        base[q] = f32x4{0.f, 0.f, 0.f, 0.f};
        if (ok[q]) {
          if (P.R) {
            const u32x2 r = *reinterpret_cast<const u32x2*>(P.R + (size_t)mm[q] * P.ldr + nn[q]);
            base[q] = f32x4{bf16_bits_to_f32(r[0] & 0xffffu), bf16_bits_to_f32(r[0] >> 16),
                            bf16_bits_to_f32(r[1] & 0xffffu), bf16_bits_to_f32(r[1] >> 16)};
          } else if (P.accumulate) {
            base[q] = *reinterpret_cast<const f32x4*>(P.Y + (size_t)mm[q] * P.ldy + nn[q]);
          }
        }
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
        if (!ok[q]) continue;
        const u32x2 bits{pack_bf16x2(v[q][0], v[q][1]), pack_bf16x2(v[q][2], v[q][3])};
        uint16_t* dst;
        if constexpr (EPI == EPI_SWIGLU) {
          dst = P.H + (size_t)mm[q] * P.ldh + nn[q];
        } else {
          const int n = nn[q], m = mm[q];
          if (n < P.nq) {
            dst = P.Q + (size_t)m * P.ldq + n;
          } else {
            const int b = m / P.rows_per_batch, t = m - b * P.rows_per_batch;
            const size_t row = (size_t)b * P.kv_batch_stride +
                               (size_t)(P.kv_pos0 + t) * P.kv_row_stride + P.kv_col0;
            dst = n < P.nq + P.nkv ? P.Kb + row + (n - P.nq) : P.Vb + row + (n - P.nq - P.nkv);
          }
        }
        *reinterpret_cast<u32x2*>(dst) = bits;
      }
    }
    __syncthreads();
  }
}

template <int BM, int BN, bool NN, int EPI>
hipError_t launch(const GemmParams& p, hipStream_t s) {
  if (p.M <= 0 || p.N <= 0) return hipSuccess;
  const int tiles = ((p.M + BM - 1) / BM) * ((p.N + BN - 1) / BN);
  hipLaunchKernelGGL((gemm_kernel<BM, BN, NN, EPI>), dim3(tiles), dim3(kThreads), 0, s, p);
  return hipGetLastError();
}

}  // namespace

hipError_t launch_gemm_swiglu(const GemmParams& p, hipStream_t s) {
  return launch<256, 128, false, EPI_SWIGLU>(p, s);
}

hipError_t launch_gemm_nn_acc(const GemmParams& p, hipStream_t s) {
  return launch<256, 128, true, EPI_ACC>(p, s);
}

hipError_t launch_gemm_qkv(const GemmParams& p, hipStream_t s) {
  return launch<256, 128, false, EPI_QKV>(p, s);
}

}  // namespace tsp
