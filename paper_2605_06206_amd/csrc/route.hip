// Router scores + per-group top-k + softmax weights (Section 3.1, routing
// equation), fused in one kernel: the [T,E] scores never leave the chip.
//
// One workgroup = TG groups of 16 tokens, 4 or 8 waves.  The score tile
// S[16 tokens][E] of each group is a skinny GEMM x[16,d] * W_r[E,d]^T on MFMA
// (bf16: 16x16x32, fp32: 16x16x4) with K split across the waves (each issuing
// the loads of several K steps at once); the partial tiles are summed in LDS
// in a fixed order.  In the 16x16
// MFMA result layout each row of 16 lanes holds all 16 experts of one token
// (per accumulator register), so the top-k is k rounds of a (score desc, id
// asc) arg-max across a 16-lane row with DPP rotations.
#include "foe_common.hpp"

namespace foe {
namespace {

constexpr int kTok = 16;    // tokens per workgroup
#ifndef FOE_ROUTE_BATCH
#define FOE_ROUTE_BATCH 4
#endif
constexpr int kBatch = FOE_ROUTE_BATCH;  // K steps whose loads are issued together

// (v, e) beats (w, f): larger score, equal scores -> lower id
__device__ __forceinline__ bool beats(float v, int e, float w, int f) {
  return v > w || (v == w && e < f);
}

template <int SH>
__device__ __forceinline__ void argmax_step(float& bv, int& be) {
  float ov = __int_as_float(row_ror<SH>(__float_as_int(bv)));
  int oe = row_ror<SH>(be);
  if (beats(ov, oe, bv, be)) { bv = ov; be = oe; }
}

template <typename T> struct RouteMma;

// bf16: each MFMA step consumes 32 k; lane (r = l%16, q = l/16) supplies
// x[r][kc + 8q .. +8) and W_r[e][same k] (the same k map on both operands).
// One W_r fragment serves the TG token groups of the workgroup.
template <> struct RouteMma<bf16> {
  static constexpr int KSTEP = 32;
  template <int NT, int NW, int TG>
  __device__ static void run(const bf16* x, const bf16* w, int T, int d, int E, int t0,
                             int wave, int lane, f32x4 (&acc)[TG][NT]) {
    const int r = lane & 15, q = lane >> 4;
    const bf16* xrow[TG];
    bool tok_ok[TG];
#pragma unroll
    for (int g = 0; g < TG; ++g) {
      const int tok = t0 + g * 16 + r;
      tok_ok[g] = tok < T;
      xrow[g] = x + (size_t)(tok_ok[g] ? tok : 0) * d;
    }
    const int nsteps = (d + KSTEP - 1) / KSTEP;
    // wave w takes K-step groups w, w+NW, ... of kBatch steps each
    for (int c0 = wave * kBatch; c0 < nsteps; c0 += NW * kBatch) {
      u32x4 a[kBatch][TG], b[kBatch][NT];
#pragma unroll
      for (int u = 0; u < kBatch; ++u) {
        const int kb = (c0 + u) * KSTEP + q * 8;
        const bool k_ok = c0 + u < nsteps && kb < d;
#pragma unroll
        for (int nt = 0; nt < NT; ++nt) {
          const int e = nt * 16 + r;
          b[u][nt] = (e < E && k_ok) ? *reinterpret_cast<const u32x4*>(w + (size_t)e * d + kb)
                                     : zero_u32x4();
        }
#pragma unroll
        for (int g = 0; g < TG; ++g)
          a[u][g] = (tok_ok[g] && k_ok) ? *reinterpret_cast<const u32x4*>(xrow[g] + kb)
                                        : zero_u32x4();
      }
#pragma unroll
      for (int u = 0; u < kBatch; ++u)
#pragma unroll
        for (int g = 0; g < TG; ++g)
#pragma unroll
          for (int nt = 0; nt < NT; ++nt)
            acc[g][nt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(
                __builtin_bit_cast(bf16x8, a[u][g]), __builtin_bit_cast(bf16x8, b[u][nt]),
                acc[g][nt], 0, 0, 0);
    }
  }
};

// fp32: 16x16x4 MFMA; a lane loads 4 consecutive k and issues 4 MFMAs, the
// s-th using element s (k map kc + 4q + s on both operands).
template <> struct RouteMma<float> {
  static constexpr int KSTEP = 16;
  template <int NT, int NW, int TG>
  __device__ static void run(const float* x, const float* w, int T, int d, int E, int t0,
                             int wave, int lane, f32x4 (&acc)[TG][NT]) {
    const int r = lane & 15, q = lane >> 4;
    const int nsteps = (d + KSTEP - 1) / KSTEP;
    for (int c = wave; c < nsteps; c += NW) {
      const int kb = c * KSTEP + q * 4;
      const bool k_ok = kb < d;
#pragma unroll
      for (int g = 0; g < TG; ++g) {
        const int tok = t0 + g * 16 + r;
        const float* xrow = x + (size_t)(tok < T ? tok : 0) * d;
        f32x4 a = (tok < T && k_ok) ? *reinterpret_cast<const f32x4*>(xrow + kb)
                                    : f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int nt = 0; nt < NT; ++nt) {
          const int e = nt * 16 + r;
          f32x4 b = (e < E && k_ok) ? *reinterpret_cast<const f32x4*>(w + (size_t)e * d + kb)
                                    : f32x4{0.f, 0.f, 0.f, 0.f};
          acc[g][nt] = __builtin_amdgcn_mfma_f32_16x16x4f32(a[0], b[0], acc[g][nt], 0, 0, 0);
          acc[g][nt] = __builtin_amdgcn_mfma_f32_16x16x4f32(a[1], b[1], acc[g][nt], 0, 0, 0);
          acc[g][nt] = __builtin_amdgcn_mfma_f32_16x16x4f32(a[2], b[2], acc[g][nt], 0, 0, 0);
          acc[g][nt] = __builtin_amdgcn_mfma_f32_16x16x4f32(a[3], b[3], acc[g][nt], 0, 0, 0);
        }
      }
    }
  }
};

// A "unit" is accumulator register i of token group g: in the 16x16 MFMA
// layout it holds tokens g*16 + 4*(lane/16) + i (one per 16-lane row) and
// experts nt*16 + lane%16.  The 4*TG units are spread over the waves.
template <typename T, int NT, int NW, int TG>
__global__ __launch_bounds__(NW * 64) void route_kernel(const T* __restrict__ x,
                                                        const T* __restrict__ w,
                                                        const float* __restrict__ bias, int T_,
                                                        int d, int E, int k,
                                                        int32_t* __restrict__ topk_idx,
                                                        float* __restrict__ topk_w) {
  constexpr int UPW = (4 * TG + NW - 1) / NW;  // units per wave
  extern __shared__ __align__(16) unsigned char smem[];
  const int lane = lane_id();
  const int wave = threadIdx.x >> 6;
  const int t0 = blockIdx.x * kTok * TG;

  f32x4 acc[TG][NT];
#pragma unroll
  for (int g = 0; g < TG; ++g)
#pragma unroll
    for (int nt = 0; nt < NT; ++nt) acc[g][nt] = f32x4{0.f, 0.f, 0.f, 0.f};
  RouteMma<T>::template run<NT, NW, TG>(x, w, T_, d, E, t0, wave, lane, acc);

  // partial tiles of the NW waves -> LDS [wave][g][nt][lane] (f32x4)
  f32x4* part = reinterpret_cast<f32x4*>(smem);
#pragma unroll
  for (int g = 0; g < TG; ++g)
#pragma unroll
    for (int nt = 0; nt < NT; ++nt) part[((wave * TG + g) * NT + nt) * kWave + lane] = acc[g][nt];
  __syncthreads();

  // scores of this wave's units: sum of the NW partials in wave order, + bias
  const int col = lane & 15;
  float gl[UPW][NT];
#pragma unroll
  for (int u = 0; u < UPW; ++u) {
    const int unit = wave + u * NW;
    const int g = (unit >> 2) < TG ? (unit >> 2) : 0, i = unit & 3;
#pragma unroll
    for (int nt = 0; nt < NT; ++nt) {
      float s = 0.f;
      if (unit < 4 * TG) {
#pragma unroll
        for (int wv = 0; wv < NW; ++wv) s += part[((wv * TG + g) * NT + nt) * kWave + lane][i];
        const int e = nt * 16 + col;
        if (bias != nullptr && e < E) s += bias[e];
      }
      gl[u][nt] = s;
    }
  }
  __syncthreads();  // partial tiles are dead; LDS is reused for the selection

  // per wave: the k selections of its 4 rows (one token per 16-lane row)
  int* sel_e = reinterpret_cast<int*>(smem) + wave * 8 * k;
  float* sel_v = reinterpret_cast<float*>(sel_e + 4 * k);
  const int row = lane >> 4;
#pragma unroll
  for (int u = 0; u < UPW; ++u) {
    const int unit = wave + u * NW;
    if (unit >= 4 * TG) break;
    const int tok = t0 + (unit >> 2) * 16 + 4 * row + (unit & 3);
    unsigned taken = 0;  // bit nt: expert nt*16 + col already selected / absent
#pragma unroll
    for (int nt = 0; nt < NT; ++nt)
      if (nt * 16 + col >= E) taken |= 1u << nt;
    for (int s = 0; s < k; ++s) {
      float bv = -__builtin_inff();
      int be = 0x7fffffff;
#pragma unroll
      for (int nt = 0; nt < NT; ++nt) {
        const int e = nt * 16 + col;
        if (!((taken >> nt) & 1u) && beats(gl[u][nt], e, bv, be)) { bv = gl[u][nt]; be = e; }
      }
      argmax_step<8>(bv, be);
      argmax_step<4>(bv, be);
      argmax_step<2>(bv, be);
      argmax_step<1>(bv, be);
      if (be != 0x7fffffff && (be & 15) == col) taken |= 1u << (be >> 4);
      if (col == 0) {
        sel_e[row * k + s] = (be == 0x7fffffff) ? -1 : be;
        sel_v[row * k + s] = bv;
      }
    }
    // softmax over the selected scores (this wave's own rows; LDS operations
    // of one wave complete in order); lane col writes slots col, col+16, ...
    if (tok < T_) {
      const float m = sel_v[row * k];
      float z = 0.f;
      for (int s = 0; s < k; ++s) z += expf(sel_v[row * k + s] - m);
      const float inv = 1.0f / z;
      for (int s = col; s < k; s += 16) {
        topk_idx[(size_t)tok * k + s] = sel_e[row * k + s];
        topk_w[(size_t)tok * k + s] = expf(sel_v[row * k + s] - m) * inv;
      }
    }
  }
}

template <typename T, int NT, int NW, int TG>
hipError_t launch_nt(int T_, int d, int E, int k, const void* x, const void* w,
                     const float* bias, int32_t* idx, float* wt, hipStream_t s) {
  size_t lds_red = (size_t)NW * TG * NT * kWave * sizeof(f32x4);
  size_t lds_sel = (size_t)NW * 8 * k * 4;
  size_t lds = lds_red > lds_sel ? lds_red : lds_sel;
  dim3 grid(ceil_div(T_, kTok * TG));
  ProfileScope ps("route", s);
  hipLaunchKernelGGL((route_kernel<T, NT, NW, TG>), grid, dim3(NW * kWave), lds, s,
                     reinterpret_cast<const T*>(x), reinterpret_cast<const T*>(w), bias, T_, d,
                     E, k, idx, wt);
  return hipGetLastError();
}

// (token groups per workgroup, waves) for many tokens: token groups share each
// router-weight fragment (otherwise the weights are read once per 16 tokens,
// more bytes than x itself at E = 32); few tokens: 8 waves split K of one
// 16-token group (more loads in flight per token).  Large E: 4 waves.
template <int TG_, int NW_> struct RouteCfg {
  static constexpr int TG = TG_, NW = NW_;
};
#ifndef FOE_ROUTE_TG16
#define FOE_ROUTE_TG16 1, 8
#endif
#ifndef FOE_ROUTE_TG32
#define FOE_ROUTE_TG32 2, 8
#endif
template <typename T>
hipError_t launch_t(int T_, int d, int E, int k, const void* x, const void* w, const float* bias,
                    int32_t* idx, float* wt, hipStream_t s) {
  const bool many = T_ >= 2048;
  if (E <= 16)
    return many ? launch_nt<T, 1, RouteCfg<FOE_ROUTE_TG16>::NW, RouteCfg<FOE_ROUTE_TG16>::TG>(
                      T_, d, E, k, x, w, bias, idx, wt, s)
                : launch_nt<T, 1, 8, 1>(T_, d, E, k, x, w, bias, idx, wt, s);
  if (E <= 32)
    return many ? launch_nt<T, 2, RouteCfg<FOE_ROUTE_TG32>::NW, RouteCfg<FOE_ROUTE_TG32>::TG>(
                      T_, d, E, k, x, w, bias, idx, wt, s)
                : launch_nt<T, 2, 8, 1>(T_, d, E, k, x, w, bias, idx, wt, s);
  if (E <= 64) return launch_nt<T, 4, 8, 1>(T_, d, E, k, x, w, bias, idx, wt, s);
  if (E <= 128) return launch_nt<T, 8, 4, 1>(T_, d, E, k, x, w, bias, idx, wt, s);
  return launch_nt<T, 16, 4, 1>(T_, d, E, k, x, w, bias, idx, wt, s);
}

}  // namespace

hipError_t launch_route(foe_dtype dt, int T, int d, int E, int k, const void* x,
                        const void* w_router, const float* bias, int32_t* topk_idx,
                        float* topk_w, hipStream_t s) {
  if (T == 0) return hipSuccess;
  if (dt == FOE_BF16) return launch_t<bf16>(T, d, E, k, x, w_router, bias, topk_idx, topk_w, s);
  return launch_t<float>(T, d, E, k, x, w_router, bias, topk_idx, topk_w, s);
}

}  // namespace foe
