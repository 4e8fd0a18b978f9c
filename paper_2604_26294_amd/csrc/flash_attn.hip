// Causal flash attention of one TSP rank's query chunk (gfx950, bf16 MFMA).
//
// Algorithm 1's CausalAttn for contiguous chunks: local query t of rank p sits at
// global position q_pos0 + t (q_pos0 = p S_loc) and sees keys j <= q_pos0 + t of the
// gathered K/V (held resident in a [B, S, n_kv, d] buffer).  The softmax is computed
// online, one key tile at a time, so the (S_loc x S) score matrix never exists.
//
// Work split.  A workgroup owns 128 queries of one head (GQA: head i reads kv head
// i / g) and has 8 wavefronts: wavefront w handles queries 32 (w % 4) .. +31 against
// key group w / 4, i.e. each step stages 128 keys in LDS and the two groups of four
// wavefronts consume its two 64-key halves.  Each group keeps its own running max /
// sum / output; the groups are merged once at the end.  Key tiles beyond the last
// query's position are never loaded; only tiles that cross the diagonal are masked.
//
// Layout trick.  Scores are computed transposed, S^T = K Q^T, with K as the MFMA A
// operand and Q (held in registers) as B.  The 32 x 32 accumulator then gives each
// lane 16 keys of ONE query (its partner lane l ^ 32 holds the other 16), so the
// row max needs one cross-lane exchange and the row sum none until the end.  The
// probabilities P^T feed the second product O^T = V^T P^T directly as the B operand
// (contraction over keys), which needs V^T in LDS: V tiles are transposed in
// registers on their way into LDS, with the keys of every 16-key group stored in the
// order the accumulator layout delivers them.
#include <math.h>

#include "common.h"
#include "internal.h"

namespace tsp {
namespace {

constexpr int kThreads = 512;
constexpr int kQTile = 128;
constexpr int kKTile = 64;           // keys per group per step
constexpr int kStepKeys = 2 * kKTile;

__device__ __forceinline__ int swz(int row, int chunk) {
  return chunk ^ ((row ^ (row >> 3)) & 7);
}

__device__ __forceinline__ uint32_t pick_col(uint32_t row_lo, uint32_t row_hi, int odd) {
  return odd ? ((row_lo >> 16) | (row_hi & 0xffff0000u)) : ((row_lo & 0xffffu) | (row_hi << 16));
}

template <int D>
struct FaCfg {
  static constexpr int KCH = D / 8;                      // 16-byte chunks per K row
  static constexpr int K_CHUNKS = kStepKeys * KCH;       // K region of one stage
  static constexpr int VT_CHUNKS = 2 * D * 8;            // 2 groups x D rows x 64 keys
  static constexpr int STAGE = K_CHUNKS + VT_CHUNKS;
  static constexpr int K_LOADS = K_CHUNKS / kThreads;
  static constexpr int V_BLOCKS = (kStepKeys / 4) * (D / 8);  // 4 keys x 8 columns each
  static constexpr int EB = D / 32;                      // 32-row blocks of O^T
  static constexpr int KS = D / 16;                      // contraction steps of S^T
  static_assert(V_BLOCKS <= kThreads, "V blocks");
};

template <int D>
__global__ __launch_bounds__(kThreads) void flash_fwd_kernel(const AttnParams P) {
  using C = FaCfg<D>;
  __shared__ u32x4 L[2 * C::STAGE];

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
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
  const long long qpos = P.q_pos0 + qloc;
  const int wq_first = q0 + 32 * wq;
  const bool wave_active = wq_first < P.s_loc;
  const long long wpos_min = P.q_pos0 + wq_first;
  const long long wpos_max = P.q_pos0 + min(wq_first + 31, P.s_loc - 1);
  const long long n_keys = P.q_pos0 + min(q0 + kQTile, P.s_loc);  // <= kv_len
  const int n_steps = (int)((n_keys + kStepKeys - 1) / kStepKeys);
  const float c = P.scale_log2;

  // Q fragments: the B operand of S^T; lane holds Q[qloc][16 s + 8 hh .. +7].
  u32x4 qf[C::KS];
  {
    const uint16_t* qrow = P.Q + (((size_t)b * P.s_loc + (qvalid ? qloc : 0)) * P.heads + head) * D;
#pragma unroll
    for (int s = 0; s < C::KS; ++s)
      qf[s] = qvalid ? ld16(qrow + 16 * s + 8 * hh) : u32x4{0u, 0u, 0u, 0u};
  }

  f32x16 o[C::EB];
#pragma unroll
  for (int eb = 0; eb < C::EB; ++eb)
#pragma unroll
    for (int e = 0; e < 16; ++e) o[eb][e] = 0.f;
  float m_run = -INFINITY, l_run = 0.f;

  const size_t kv_stride = (size_t)P.n_kv * D;
  const uint16_t* kbase = P.Kb + (size_t)b * P.seq * kv_stride + (size_t)kvh * D;
  const uint16_t* vbase = P.Vb + (size_t)b * P.seq * kv_stride + (size_t)kvh * D;

  u32x4 rk[C::K_LOADS];
  u32x4 rv[4];
  const int v_db = tid % (D / 8), v_kq = tid / (D / 8);

  auto load = [&](int step) {
    const long long key0 = (long long)step * kStepKeys;
#pragma unroll
    for (int i = 0; i < C::K_LOADS; ++i) {
      const long long gk = key0 + tid / C::KCH + (kThreads / C::KCH) * i;
      rk[i] = gk < n_keys ? ld16(kbase + gk * kv_stride + 8 * (tid % C::KCH)) : u32x4{0u, 0u, 0u, 0u};
    }
    if (tid < C::V_BLOCKS) {
#pragma unroll
      for (int rr = 0; rr < 4; ++rr) {
        const long long gk = key0 + 4 * v_kq + rr;
        rv[rr] = gk < n_keys ? ld16(vbase + gk * kv_stride + 8 * v_db) : u32x4{0u, 0u, 0u, 0u};
      }
    }
  };

  auto store = [&](int stage) {
    u32x4* S = L + stage * C::STAGE;
#pragma unroll
    for (int i = 0; i < C::K_LOADS; ++i) {
      const int key = tid / C::KCH + (kThreads / C::KCH) * i;
      S[key * C::KCH + swz(key, tid % C::KCH)] = rk[i];
    }
    if (tid < C::V_BLOCKS) {
      // Keys 4 v_kq .. +3 of the step -> group g2, 16-key group G, quad q inside it.
      // Within each 16-key group the quads are stored in the order 0, 2, 1, 3 so that
      // one 16-byte chunk holds the 8 keys a lane half feeds to one MFMA.
      const int g2 = v_kq >> 4;
      const int kk = 4 * (v_kq & 15);
      const int G = kk >> 4, q = (kk & 15) >> 2;
      const int qp = ((q & 1) << 1) | (q >> 1);
      const int chunk = 2 * G + (qp >> 1), half = qp & 1;
      u32x2* VT = reinterpret_cast<u32x2*>(S + C::K_CHUNKS + g2 * D * 8);
#pragma unroll
      for (int cc = 0; cc < 8; ++cc) {
        const int row = 8 * v_db + cc;  // head-dim index
        u32x2 val;
        val[0] = pick_col(rv[0][cc >> 1], rv[1][cc >> 1], cc & 1);
        val[1] = pick_col(rv[2][cc >> 1], rv[3][cc >> 1], cc & 1);
        VT[(row * 8 + swz(row, chunk)) * 2 + half] = val;
      }
    }
  };

  load(0);
  store(0);
  __syncthreads();

  for (int step = 0; step < n_steps; ++step) {
    const int cur = step & 1;
    if (step + 1 < n_steps) load(step + 1);

    const long long kt0 = (long long)step * kStepKeys + kKTile * grp;
    if (wave_active && kt0 <= wpos_max) {
      const u32x4* S = L + cur * C::STAGE;
      f32x16 sacc[2];
#pragma unroll
      for (int bb = 0; bb < 2; ++bb)
#pragma unroll
        for (int e = 0; e < 16; ++e) sacc[bb][e] = 0.f;
#pragma unroll
      for (int s = 0; s < C::KS; ++s) {
#pragma unroll
        for (int bb = 0; bb < 2; ++bb) {
          const int row = kKTile * grp + 32 * bb + l32;
          sacc[bb] = mfma32(S[row * C::KCH + swz(row, 2 * s + hh)], qf[s], sacc[bb]);
        }
      }
      if (kt0 + kKTile - 1 > wpos_min) {
#pragma unroll
        for (int bb = 0; bb < 2; ++bb)
#pragma unroll
          for (int e = 0; e < 16; ++e) {
            const long long key = kt0 + 32 * bb + 8 * (e >> 2) + 4 * hh + (e & 3);
            if (key > qpos) sacc[bb][e] = -INFINITY;
          }
      }
      float mx = sacc[0][0];
#pragma unroll
      for (int bb = 0; bb < 2; ++bb)
#pragma unroll
        for (int e = 0; e < 16; ++e) mx = fmaxf(mx, sacc[bb][e]);
      mx = fmaxf(mx, __shfl_xor(mx, 32));
      const float m_new = fmaxf(m_run, mx);
      const float m_use = m_new == -INFINITY ? 0.f : m_new;
      const float alpha = __builtin_amdgcn_exp2f((m_run - m_use) * c);
      const float mc = m_use * c;
      float lsum = 0.f;
#pragma unroll
      for (int bb = 0; bb < 2; ++bb)
#pragma unroll
        for (int e = 0; e < 16; ++e) {
          const float pv = __builtin_amdgcn_exp2f(fmaf(sacc[bb][e], c, -mc));
          sacc[bb][e] = pv;
          lsum += pv;
        }
      l_run = l_run * alpha + lsum;
      m_run = m_new;
#pragma unroll
      for (int eb = 0; eb < C::EB; ++eb)
#pragma unroll
        for (int e = 0; e < 16; ++e) o[eb][e] *= alpha;

      u32x4 pf[2][2];
#pragma unroll
      for (int bb = 0; bb < 2; ++bb)
#pragma unroll
        for (int s2 = 0; s2 < 2; ++s2)
#pragma unroll
          for (int q = 0; q < 4; ++q)
            pf[bb][s2][q] = pack_bf16x2(sacc[bb][8 * s2 + 2 * q], sacc[bb][8 * s2 + 2 * q + 1]);

      const u32x4* VT = S + C::K_CHUNKS + grp * D * 8;
#pragma unroll
      for (int eb = 0; eb < C::EB; ++eb) {
        const int row = 32 * eb + l32;
#pragma unroll
        for (int bb = 0; bb < 2; ++bb)
#pragma unroll
          for (int s2 = 0; s2 < 2; ++s2)
            o[eb] = mfma32(VT[row * 8 + swz(row, 4 * bb + 2 * s2 + hh)], pf[bb][s2], o[eb]);
      }
    }

    if (step + 1 < n_steps) store(cur ^ 1);
    __syncthreads();
  }

  // Merge the two key groups: group 1 parks its state in LDS, group 0 combines.
  l_run += __shfl_xor(l_run, 32);
  float* F = reinterpret_cast<float*>(L);
  const int slot = wq * 64 + lane;
  if (grp == 1) {
    F[slot] = m_run;
    F[256 + slot] = l_run;
#pragma unroll
    for (int eb = 0; eb < C::EB; ++eb)
#pragma unroll
      for (int e = 0; e < 16; ++e) F[(2 + 16 * eb + e) * 256 + slot] = o[eb][e];
  }
  __syncthreads();
  if (grp == 0 && qvalid) {
    const float m1 = F[slot], l1 = F[256 + slot];
    const float m = fmaxf(m_run, m1);
    const float mu = m == -INFINITY ? 0.f : m;
    const float a0 = __builtin_amdgcn_exp2f((m_run - mu) * c);
    const float a1 = __builtin_amdgcn_exp2f((m1 - mu) * c);
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
        u32x2 pk;
        pk[0] = pack_bf16x2(v[0], v[1]);
        pk[1] = pack_bf16x2(v[2], v[3]);
        *reinterpret_cast<u32x2*>(orow + 32 * eb + 8 * g + 4 * hh) = pk;
      }
  }
}

}  // namespace

hipError_t launch_flash_attn(const AttnParams& p, hipStream_t s) {
  if (p.batch <= 0 || p.s_loc <= 0 || p.heads <= 0) return hipSuccess;
  const int n_qt = (p.s_loc + kQTile - 1) / kQTile;
  const dim3 grid(n_qt * p.heads * p.batch);
  if (p.head_dim == 128)
    hipLaunchKernelGGL(flash_fwd_kernel<128>, grid, dim3(kThreads), 0, s, p);
  else if (p.head_dim == 64)
    hipLaunchKernelGGL(flash_fwd_kernel<64>, grid, dim3(kThreads), 0, s, p);
  else
    return hipErrorInvalidValue;
  return hipGetLastError();
}

}  // namespace tsp
