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

// Epilogues for one 32 x 32 accumulator tile: element e of lane (l32, hh) is
// C[mrow + 8 (e / 4) + (e % 4)][nblk + l32], where mrow already includes 4 hh.
__device__ __forceinline__ void epi_swiglu(const GemmParams& P, const f32x16& g, const f32x16& u,
                                           int mrow, int nblk, int l32) {
  const int n = nblk + l32;
  if (n >= P.N) return;
#pragma unroll
  for (int e = 0; e < 16; ++e) {
    const int m = mrow + 8 * (e >> 2) + (e & 3);
    if (m < P.M) {
      const float v = g[e];
      P.H[(size_t)m * P.ldh + n] = to_bf16_bits(v / (1.f + __expf(-v)) * u[e]);
    }
  }
}

__device__ __forceinline__ void epi_acc(const GemmParams& P, const f32x16& c, int mrow, int nblk,
                                        int l32) {
  const int n = nblk + l32;
  if (n >= P.N) return;
#pragma unroll
  for (int e = 0; e < 16; ++e) {
    const int m = mrow + 8 * (e >> 2) + (e & 3);
    if (m < P.M) {
      const size_t yi = (size_t)m * P.ldy + n;
      float out = c[e];
      if (P.R) out += bf16_bits_to_f32(P.R[(size_t)m * P.ldr + n]);
      else if (P.accumulate) out += P.Y[yi];
      P.Y[yi] = out;
      if (P.U) P.U[(size_t)m * P.ldu + n] = to_bf16_bits(out);
    }
  }
}

__device__ __forceinline__ void epi_qkv(const GemmParams& P, const f32x16& c, int mrow, int nblk,
                                        int l32) {
  const int n = nblk + l32;
  if (n >= P.N) return;
#pragma unroll
  for (int e = 0; e < 16; ++e) {
    const int m = mrow + 8 * (e >> 2) + (e & 3);
    if (m < P.M) {
      const uint16_t bits = to_bf16_bits(c[e]);
      if (nblk < P.nq) {
        P.Q[(size_t)m * P.ldq + n] = bits;
      } else {
        const int b = m / P.rows_per_batch, t = m - b * P.rows_per_batch;
        const size_t row = (size_t)b * P.kv_batch_stride +
                           (size_t)(P.kv_pos0 + t) * P.kv_row_stride + P.kv_col0;
        if (nblk < P.nq + P.nkv) P.Kb[row + (n - P.nq)] = bits;
        else P.Vb[row + (n - P.nq - P.nkv)] = bits;
      }
    }
  }
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

  // ---------------------------------------------------------------- epilogues
  const int mw = m0 + wm * C::WM + 4 * hh;
#pragma unroll
  for (int i = 0; i < TM; ++i) {
#pragma unroll
    for (int j = 0; j < TN; ++j) {
      const int nblk = n0 + wn * C::WN + 32 * j;
      if constexpr (EPI == EPI_SWIGLU) epi_swiglu(P, acc[i][j], acc[i][j + TN], mw + 32 * i, nblk, l32);
      else if constexpr (EPI == EPI_ACC) epi_acc(P, acc[i][j], mw + 32 * i, nblk, l32);
      else epi_qkv(P, acc[i][j], mw + 32 * i, nblk, l32);
    }
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
