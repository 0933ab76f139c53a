// Grouped SwiGLU expert FFN (Table 3 "MoE update": FFN_e on the rows routed
// to expert e).  Two grouped GEMMs over the permuted rows:
//   gate/up : h[rows,F] = silu(x_perm W_g[e]^T) * (x_perm W_u[e]^T)   (SwiGLU
//             fused into the epilogue; both products share the A tile)
//   down    : y[rows,d] = h W_d[e]^T
// Every weight is [out,in] (K-contiguous), so both GEMMs are "NT".
//
// bf16 path: v_mfma_f32_32x32x16_bf16, fp32 accumulation, tiles staged through
// LDS with double buffering (global loads of stage s+1 overlap the MFMAs of
// stage s).  The MFMA computes D = W_tile * X_tile^T so each lane ends up with
// 4 consecutive output columns of one row (8-byte stores).  The expert and row
// range of a workgroup come from the device-side offsets: one wave-wide prefix
// sum over the per-expert tile counts, so no host sync is needed.
#include "foe_common.hpp"

namespace foe {
namespace {

// Find the (expert, first row, row end) of global M-tile `mt`.  Returns false
// if `mt` is past the last tile.  Offsets are clamped to [0, rows]; a
// decreasing bound gives an empty segment.  E <= 256 (4 experts per lane).
__device__ bool find_tile(const int32_t* __restrict__ offsets, int E, int rows, int BM, int mt,
                          int& e_out, int& row0, int& row_end) {
  const int lane = lane_id();
  int lo[4], hi[4], nt[4];
  int mine = 0;
#pragma unroll
  for (int u = 0; u < 4; ++u) {
    const int e = lane * 4 + u;
    lo[u] = hi[u] = nt[u] = 0;
    if (e < E) {
      int a = min(max(offsets[e], 0), rows);
      int b = min(max(offsets[e + 1], 0), rows);
      if (b < a) b = a;
      lo[u] = a;
      hi[u] = b;
      nt[u] = (b - a + BM - 1) / BM;
    }
    mine += nt[u];
  }
  int incl = mine;
#pragma unroll
  for (int off = 1; off < kWave; off <<= 1) {
    const int t = __shfl_up(incl, off);
    if (lane >= off) incl += t;
  }
  const int excl = incl - mine;
  const uint64_t bal = __ballot(mt >= excl && mt < incl);
  if (bal == 0) return false;
  const int src = __builtin_ctzll(bal);
  int e_sel = 0, r0 = 0, r1 = 0;
  int t = mt - excl;
#pragma unroll
  for (int u = 0; u < 4; ++u) {
    if (t >= 0 && t < nt[u]) {
      e_sel = lane * 4 + u;
      r0 = lo[u] + t * BM;
      r1 = hi[u];
    }
    t -= nt[u];
  }
  e_out = __builtin_amdgcn_readlane(e_sel, src);
  row0 = __builtin_amdgcn_readlane(r0, src);
  row_end = __builtin_amdgcn_readlane(r1, src);
  return true;
}

__device__ __forceinline__ float silu_f(float g) { return g / (1.0f + __expf(-g)); }

template <int BM, int BN, int BK, int WM, int WN, bool GATEUP>
struct GemmCfg {
  static constexpr int NTHR = WM * WN * kWave;
  static constexpr int WTM = BM / WM, WTN = BN / WN;
  static constexpr int SM = WTM / 32, SN = WTN / 32;
  static constexpr int NB = GATEUP ? 2 : 1;
  static constexpr int LDK = BK + 8;  // padded LDS row (elements)
  static constexpr int CPR = BK / 8;  // 16-byte chunks per tile row
  static constexpr int A_PER = BM * CPR / NTHR;
  static constexpr int B_PER = BN * CPR / NTHR;
  static constexpr int A_ELEMS = BM * LDK, B_ELEMS = BN * LDK;
  static constexpr int STAGE_ELEMS = A_ELEMS + NB * B_ELEMS;
  static_assert(WTM % 32 == 0 && WTN % 32 == 0, "wave tile must be a multiple of 32");
  static_assert(BK % 16 == 0, "BK multiple of 16");
  static_assert(BM * CPR % NTHR == 0 && BN * CPR % NTHR == 0, "even load split");
};

template <int BM, int BN, int BK, int WM, int WN, bool GATEUP>
__global__ __launch_bounds__(WM* WN* kWave) void grouped_gemm_bf16(
    const bf16* __restrict__ A, const int32_t* __restrict__ offsets, int E, int rows,
    const bf16* __restrict__ B0, const bf16* __restrict__ B1, int N, int K,
    bf16* __restrict__ out, int n_tiles_n) {
  using C = GemmCfg<BM, BN, BK, WM, WN, GATEUP>;
  __shared__ __align__(16) bf16 lds[2 * C::STAGE_ELEMS];

  const int mt = blockIdx.x / n_tiles_n;
  const int ntile = blockIdx.x % n_tiles_n;
  int e, row0, row_end;
  if (!find_tile(offsets, E, rows, BM, mt, e, row0, row_end)) return;
  const int n0 = ntile * BN;

  const int tid = threadIdx.x;
  const int lane = lane_id();
  const int wave = tid >> 6;
  const int wm = wave / WN, wn = wave % WN;

  const bf16* Bw[2];
  Bw[0] = B0 + (size_t)e * N * K;
  Bw[1] = GATEUP ? B1 + (size_t)e * N * K : nullptr;

  f32x16 acc[C::NB][C::SM][C::SN];
#pragma unroll
  for (int b = 0; b < C::NB; ++b)
#pragma unroll
    for (int i = 0; i < C::SM; ++i)
#pragma unroll
      for (int j = 0; j < C::SN; ++j)
#pragma unroll
        for (int v = 0; v < 16; ++v) acc[b][i][j][v] = 0.f;

  u32x4 ra[C::A_PER];
  u32x4 rb[C::NB][C::B_PER];

  auto gload = [&](int k0) {
#pragma unroll
    for (int i = 0; i < C::A_PER; ++i) {
      const int c = tid + i * C::NTHR;
      const int r = c / C::CPR, kc = c % C::CPR;
      const int gr = row0 + r, gk = k0 + kc * 8;
      ra[i] = (gr < row_end && gk < K)
                  ? *reinterpret_cast<const u32x4*>(A + (size_t)gr * K + gk)
                  : zero_u32x4();
    }
#pragma unroll
    for (int b = 0; b < C::NB; ++b)
#pragma unroll
      for (int i = 0; i < C::B_PER; ++i) {
        const int c = tid + i * C::NTHR;
        const int r = c / C::CPR, kc = c % C::CPR;
        const int gn = n0 + r, gk = k0 + kc * 8;
        rb[b][i] = (gn < N && gk < K)
                       ? *reinterpret_cast<const u32x4*>(Bw[b] + (size_t)gn * K + gk)
                       : zero_u32x4();
      }
  };
  auto lstore = [&](int buf) {
    bf16* sa = lds + buf * C::STAGE_ELEMS;
#pragma unroll
    for (int i = 0; i < C::A_PER; ++i) {
      const int c = tid + i * C::NTHR;
      const int r = c / C::CPR, kc = c % C::CPR;
      *reinterpret_cast<u32x4*>(sa + r * C::LDK + kc * 8) = ra[i];
    }
#pragma unroll
    for (int b = 0; b < C::NB; ++b) {
      bf16* sb = sa + C::A_ELEMS + b * C::B_ELEMS;
#pragma unroll
      for (int i = 0; i < C::B_PER; ++i) {
        const int c = tid + i * C::NTHR;
        const int r = c / C::CPR, kc = c % C::CPR;
        *reinterpret_cast<u32x4*>(sb + r * C::LDK + kc * 8) = rb[b][i];
      }
    }
  };

  const int nk = (K + BK - 1) / BK;
  gload(0);
  lstore(0);
  __syncthreads();

  const int lrow = lane & 31;
  const int lk = (lane >> 5) * 8;
  for (int kt = 0; kt < nk; ++kt) {
    const int buf = kt & 1;
    if (kt + 1 < nk) gload((kt + 1) * BK);
    const bf16* sa = lds + buf * C::STAGE_ELEMS;
#pragma unroll
    for (int kk = 0; kk < BK; kk += 16) {
      bf16x8 xa[C::SM];
#pragma unroll
      for (int i = 0; i < C::SM; ++i)
        xa[i] = *reinterpret_cast<const bf16x8*>(sa + (wm * C::WTM + i * 32 + lrow) * C::LDK + kk + lk);
#pragma unroll
      for (int b = 0; b < C::NB; ++b) {
        const bf16* sb = sa + C::A_ELEMS + b * C::B_ELEMS;
#pragma unroll
        for (int j = 0; j < C::SN; ++j) {
          const bf16x8 wf =
              *reinterpret_cast<const bf16x8*>(sb + (wn * C::WTN + j * 32 + lrow) * C::LDK + kk + lk);
#pragma unroll
          for (int i = 0; i < C::SM; ++i)
            acc[b][i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(wf, xa[i], acc[b][i][j], 0, 0, 0);
        }
      }
    }
    if (kt + 1 < nk) lstore(buf ^ 1);
    __syncthreads();
  }

  // epilogue: lane holds row m = .. + lane%32, columns n = .. + 8q + 4*(lane/32) + [0,4)
#pragma unroll
  for (int i = 0; i < C::SM; ++i) {
    const int m = row0 + wm * C::WTM + i * 32 + lrow;
    if (m >= row_end) continue;
#pragma unroll
    for (int j = 0; j < C::SN; ++j) {
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        const int n = n0 + wn * C::WTN + j * 32 + q * 8 + (lane >> 5) * 4;
        if (n >= N) continue;
        bf16x4 o;
#pragma unroll
        for (int v = 0; v < 4; ++v) {
          float val = acc[0][i][j][q * 4 + v];
          if constexpr (GATEUP) val = silu_f(val) * acc[C::NB - 1][i][j][q * 4 + v];
          o[v] = (bf16)val;
        }
        *reinterpret_cast<bf16x4*>(out + (size_t)m * N + n) = o;
      }
    }
  }
}

// ---- fp32 path: plain FMA kernels (small shapes) ---------------------------
__device__ int expert_of_row(const int32_t* __restrict__ offsets, int E, int rows, int row) {
  for (int e = 0; e < E; ++e) {
    int a = min(max(offsets[e], 0), rows);
    int b = min(max(offsets[e + 1], 0), rows);
    if (row >= a && row < b) return e;
  }
  return -1;
}

__global__ __launch_bounds__(256) void gateup_f32(const float* __restrict__ xp,
                                                  const int32_t* __restrict__ offsets, int E,
                                                  int rows, const float* __restrict__ wg,
                                                  const float* __restrict__ wu, int F, int d,
                                                  float* __restrict__ h) {
  const long long id = (long long)blockIdx.x * blockDim.x + threadIdx.x;
  if (id >= (long long)rows * F) return;
  const int row = (int)(id / F), n = (int)(id % F);
  const int e = expert_of_row(offsets, E, rows, row);
  if (e < 0) return;
  const float* xr = xp + (size_t)row * d;
  const float* g = wg + ((size_t)e * F + n) * d;
  const float* u = wu + ((size_t)e * F + n) * d;
  float ag = 0.f, au = 0.f;
  for (int i = 0; i < d; ++i) {
    ag = fmaf(xr[i], g[i], ag);
    au = fmaf(xr[i], u[i], au);
  }
  h[(size_t)row * F + n] = ag / (1.0f + expf(-ag)) * au;
}

__global__ __launch_bounds__(256) void down_f32(const float* __restrict__ h,
                                                const int32_t* __restrict__ offsets, int E,
                                                int rows, const float* __restrict__ wd, int d,
                                                int F, float* __restrict__ y) {
  const long long id = (long long)blockIdx.x * blockDim.x + threadIdx.x;
  if (id >= (long long)rows * d) return;
  const int row = (int)(id / d), c = (int)(id % d);
  const int e = expert_of_row(offsets, E, rows, row);
  if (e < 0) return;
  const float* hr = h + (size_t)row * F;
  const float* w = wd + ((size_t)e * d + c) * F;
  float acc = 0.f;
  for (int i = 0; i < F; ++i) acc = fmaf(hr[i], w[i], acc);
  y[(size_t)row * d + c] = acc;
}

template <int BM, int BN, int BK, int WM, int WN, bool GATEUP>
void launch_gemm(const bf16* A, const int32_t* offsets, int E, int rows, const bf16* B0,
                 const bf16* B1, int N, int K, bf16* out, hipStream_t s, const char* name) {
  const int ntn = ceil_div(N, BN);
  const int max_mt = ceil_div(rows, BM) + E;  // sum_e ceil(M_e/BM) <= rows/BM + E
  dim3 grid((unsigned)((long long)max_mt * ntn));
  ProfileScope ps(name, s);
  hipLaunchKernelGGL((grouped_gemm_bf16<BM, BN, BK, WM, WN, GATEUP>), grid, dim3(WM * WN * kWave),
                     0, s, A, offsets, E, rows, B0, B1, N, K, out, ntn);
}

}  // namespace

size_t ffn_scratch_bytes(foe_dtype dt, int rows, int F) {
  return align_up((size_t)rows * F * (dt == FOE_BF16 ? 2 : 4), 256);
}

hipError_t launch_expert_ffn(foe_dtype dt, int E, int d, int F, int rows, const void* x_perm,
                             const int32_t* offsets, const void* w_gate, const void* w_up,
                             const void* w_down, void* y_perm, void* scratch, hipStream_t s) {
  if (rows == 0) return hipSuccess;
  if (dt == FOE_F32) {
    float* h = reinterpret_cast<float*>(scratch);
    {
      ProfileScope ps("ffn_gateup_f32", s);
      hipLaunchKernelGGL(gateup_f32, dim3(ceil_div((long long)rows * F, 256)), dim3(256), 0, s,
                         reinterpret_cast<const float*>(x_perm), offsets, E, rows,
                         reinterpret_cast<const float*>(w_gate),
                         reinterpret_cast<const float*>(w_up), F, d, h);
    }
    {
      ProfileScope ps("ffn_down_f32", s);
      hipLaunchKernelGGL(down_f32, dim3(ceil_div((long long)rows * d, 256)), dim3(256), 0, s, h,
                         offsets, E, rows, reinterpret_cast<const float*>(w_down), d, F,
                         reinterpret_cast<float*>(y_perm));
    }
    return hipGetLastError();
  }
  const bf16* xp = reinterpret_cast<const bf16*>(x_perm);
  const bf16* wg = reinterpret_cast<const bf16*>(w_gate);
  const bf16* wu = reinterpret_cast<const bf16*>(w_up);
  const bf16* wd = reinterpret_cast<const bf16*>(w_down);
  bf16* h = reinterpret_cast<bf16*>(scratch);
  bf16* y = reinterpret_cast<bf16*>(y_perm);
  const bool small_m = rows < 64 * E;  // few rows per expert: weight-streaming bound
  if (small_m) {
    launch_gemm<32, 64, 64, 1, 2, true>(xp, offsets, E, rows, wg, wu, F, d, h, s, "ffn_gateup");
    launch_gemm<32, 64, 64, 1, 2, false>(h, offsets, E, rows, wd, nullptr, d, F, y, s, "ffn_down");
  } else {
    launch_gemm<128, 128, 32, 2, 2, true>(xp, offsets, E, rows, wg, wu, F, d, h, s, "ffn_gateup");
    launch_gemm<128, 128, 32, 2, 2, false>(h, offsets, E, rows, wd, nullptr, d, F, y, s, "ffn_down");
  }
  return hipGetLastError();
}

}  // namespace foe
