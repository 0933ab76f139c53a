// Weighted un-permute-combine (Table 3 "MoE update") and the local reduction
// of cluster partials (Table 3 "Cross-group avg."; Section 3.2).  Both are
// HBM-bound row streams with 128-bit loads and stores and fp32 accumulation
// in a fixed order: the step-wise combine takes one wave per token row, the
// block's combine one wave per (token, chunk of the row).
#include "foe_common.hpp"

#ifndef FOE_COMBINE_U
#define FOE_COMBINE_U 2
#endif

namespace foe {
namespace {

template <typename T>
__global__ __launch_bounds__(256) void combine_kernel(const T* __restrict__ y,
                                                      const int32_t* __restrict__ row_of,
                                                      const float* __restrict__ w,
                                                      const T* __restrict__ res, int T_, int d,
                                                      int k, T* __restrict__ out) {
  constexpr int EPV = Vec16<T>::N;
  constexpr int U = 4;  // row chunks per lane; two slots' gathers are in flight together
  const int lane = lane_id();
  const int tok = blockIdx.x * 4 + (threadIdx.x >> 6);
  if (tok >= T_) return;
  const int R = T_ * k;
  const int nvec = d / EPV;
  const int32_t* rows = row_of + (size_t)tok * k;
  const float* wts = w + (size_t)tok * k;
  for (int c0 = 0; c0 < nvec; c0 += U * kWave) {
    float acc[U][EPV];
#pragma unroll
    for (int u = 0; u < U; ++u)
#pragma unroll
      for (int v = 0; v < EPV; ++v) acc[u][v] = 0.f;
    Vec16<T> res_v[U];
    if (res != nullptr) {
#pragma unroll
      for (int u = 0; u < U; ++u) {
        const int c = c0 + u * kWave + lane;
        if (c < nvec) res_v[u] = load16_cached(res + (size_t)tok * d + (size_t)c * EPV);
      }
    }
    for (int j = 0; j < k; j += 2) {
      // slots j and j+1 (the second may be absent); summed in slot order
      const bool two = j + 1 < k;
      const int p0 = rows[j], p1 = two ? rows[j + 1] : -1;
      const float w0 = wts[j], w1 = two ? wts[j + 1] : 0.f;
      const bool ok0 = p0 >= 0 && p0 < R, ok1 = p1 >= 0 && p1 < R;
      Vec16<T> v0[U], v1[U];
#pragma unroll
      for (int u = 0; u < U; ++u) {
        const int c = c0 + u * kWave + lane;
        if (c < nvec && ok0) v0[u] = load16_cached(y + (size_t)p0 * d + (size_t)c * EPV);
        if (c < nvec && ok1) v1[u] = load16_cached(y + (size_t)p1 * d + (size_t)c * EPV);
      }
#pragma unroll
      for (int u = 0; u < U; ++u) {
        if (ok0) {
#pragma unroll
          for (int e = 0; e < EPV; ++e) acc[u][e] = fmaf(w0, to_f32(v0[u].v[e]), acc[u][e]);
        }
        if (ok1) {
#pragma unroll
          for (int e = 0; e < EPV; ++e) acc[u][e] = fmaf(w1, to_f32(v1[u].v[e]), acc[u][e]);
        }
      }
    }
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const int c = c0 + u * kWave + lane;
      if (c >= nvec) continue;
      Vec16<T> o;
      if (res != nullptr) {
#pragma unroll
        for (int e = 0; e < EPV; ++e) o.v[e] = from_f32<T>(to_f32(res_v[u].v[e]) + acc[u][e]);
      } else {
#pragma unroll
        for (int e = 0; e < EPV; ++e) o.v[e] = from_f32<T>(acc[u][e]);
      }
      store16(out + (size_t)tok * d + (size_t)c * EPV, o);
    }
  }
}

// Fused combine + local reduction of C co-resident clusters that share the
// input x:  out[i] = scale * sum_h (x[i] + sum_j w_h[i,j] * y[row_of_h[i*k+j]])
// with y holding the FFN rows of every cluster (row_of values index it
// directly).  Evaluated as scale * (C * x[i] + S) where S sums the weighted
// rows in the order (h = 0..C-1, j = 0..k-1) in fp32; the per-cluster partials
// never reach HBM.  Without row_of, y is indexed by pair (h*T*k + i*k + j) and
// a pair counts when its expert id in sel_all lies in [0, E).
template <typename T, int NB>
__global__ __launch_bounds__(256) void combine_clusters_kernel(
    const T* __restrict__ y, const int32_t* __restrict__ row_of_all,
    const int32_t* __restrict__ sel_all, int E, const float* __restrict__ w_all,
    const T* __restrict__ x, int C, int T_, int d, int k, int y_rows, float scale,
    T* __restrict__ out) {
  constexpr int EPV = Vec16<T>::N;
  constexpr int U = FOE_COMBINE_U;
  const int lane = lane_id();
  const size_t R = (size_t)T_ * k;
  const int nvec = d / EPV;
  // one wave per (token, chunk of U*64 vectors): many short waves keep a
  // small batch's few dependent loads in flight together
  const int nch = (nvec + U * kWave - 1) / (U * kWave);
  const int wid = blockIdx.x * 4 + (threadIdx.x >> 6);
  const int tok = wid / nch;
  if (tok >= T_) return;
  const float cx = (float)C;
  {
    const int c0 = (wid - tok * nch) * U * kWave;
    float acc[U][EPV];
#pragma unroll
    for (int u = 0; u < U; ++u)
#pragma unroll
      for (int e = 0; e < EPV; ++e) acc[u][e] = 0.f;
    // x does not depend on the routing: issue its loads first
    Vec16<T> xv[U];
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const int c = c0 + u * kWave + lane;
      if (c < nvec) xv[u] = load16(x + (size_t)tok * d + (size_t)c * EPV);
    }
    // the token's C*k (cluster, slot) pairs in the order (h, j), NB at a
    // time: the NB row indices first, then all their y loads, then the sums
    // in that order, so that NB rows are in flight together (NB = 4 from
    // four pairs per token: 8 clusters 61 -> 56 us, 4 slots 142 -> 135 us;
    // 8 and 16 were slower, the registers cutting the waves in flight)
    const int ck = C * k;
    const bool by_pair = row_of_all == nullptr;
    for (int q0 = 0; q0 < ck; q0 += NB) {
      int prow[NB];
      bool ok[NB];
      float wq[NB];
#pragma unroll
      for (int b = 0; b < NB; ++b) {
        const int q = q0 + b;
        const bool in = q < ck;
        const int h = in ? q / k : 0;
        const size_t pr = h * R + (size_t)tok * k + (q - h * k);  // pair (h, j)
        if (by_pair) {
          // the y row of every pair exists: its loads need not wait for the
          // expert ids, which only decide whether it counts
          prow[b] = in ? (int)pr : -1;
          const int e = in ? sel_all[pr] : -1;
          ok[b] = e >= 0 && e < E;
        } else {
          prow[b] = in ? row_of_all[pr] : -1;
          ok[b] = prow[b] >= 0 && prow[b] < y_rows;
        }
        wq[b] = in ? w_all[pr] : 0.f;
      }
      Vec16<T> v[NB][U];
#pragma unroll
      for (int b = 0; b < NB; ++b)
#pragma unroll
        for (int u = 0; u < U; ++u) {
          const int c = c0 + u * kWave + lane;
          if (c < nvec && (by_pair ? prow[b] >= 0 : ok[b]))
            v[b][u] = load16(y + (size_t)prow[b] * d + (size_t)c * EPV);
        }
#pragma unroll
      for (int b = 0; b < NB; ++b)
        if (ok[b]) {
#pragma unroll
          for (int u = 0; u < U; ++u)
#pragma unroll
            for (int e = 0; e < EPV; ++e)
              acc[u][e] = fmaf(wq[b], to_f32(v[b][u].v[e]), acc[u][e]);
        }
    }
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const int c = c0 + u * kWave + lane;
      if (c >= nvec) continue;
      Vec16<T> o;
#pragma unroll
      for (int e = 0; e < EPV; ++e)
        o.v[e] = from_f32<T>(scale * fmaf(cx, to_f32(xv[u].v[e]), acc[u][e]));
      store16(out + (size_t)tok * d + (size_t)c * EPV, o);
    }
  }
}

// out = scale * sum_h (res + P_h), h = 0..C-1 in order; one 16-byte vector per
// thread per grid-stride step.
template <typename T>
__global__ __launch_bounds__(256) void reduce_kernel(const T* __restrict__ P,
                                                     const T* __restrict__ res, float scale,
                                                     int C, long long nvec, long long plane,
                                                     T* __restrict__ out) {
  constexpr int EPV = Vec16<T>::N;
  for (long long i = (long long)blockIdx.x * blockDim.x + threadIdx.x; i < nvec;
       i += (long long)gridDim.x * blockDim.x) {
    float acc[EPV];
#pragma unroll
    for (int e = 0; e < EPV; ++e) acc[e] = 0.f;
    float r[EPV];
    if (res != nullptr) {
      Vec16<T> rv = load16_cached(res + i * EPV);
#pragma unroll
      for (int e = 0; e < EPV; ++e) r[e] = to_f32(rv.v[e]);
    }
    for (int h = 0; h < C; ++h) {
      Vec16<T> pv = load16_cached(P + (size_t)h * plane + i * EPV);
#pragma unroll
      for (int e = 0; e < EPV; ++e)
        acc[e] += (res != nullptr) ? (r[e] + to_f32(pv.v[e])) : to_f32(pv.v[e]);
    }
    Vec16<T> o;
#pragma unroll
    for (int e = 0; e < EPV; ++e) o.v[e] = from_f32<T>(scale * acc[e]);
    store16(out + i * EPV, o);
  }
}

}  // namespace

hipError_t launch_combine(foe_dtype dt, int T, int d, int k, const void* y_perm,
                          const int32_t* row_of, const float* topk_w, const void* residual,
                          void* out, hipStream_t s) {
  if (T == 0) return hipSuccess;
  dim3 grid(ceil_div(T, 4));
  ProfileScope ps("combine", s);
  if (dt == FOE_BF16)
    FOE_LAUNCH(combine_kernel<bf16>, grid, dim3(256), 0, s,
                       reinterpret_cast<const bf16*>(y_perm), row_of, topk_w,
                       reinterpret_cast<const bf16*>(residual), T, d, k,
                       reinterpret_cast<bf16*>(out));
  else
    FOE_LAUNCH(combine_kernel<float>, grid, dim3(256), 0, s,
                       reinterpret_cast<const float*>(y_perm), row_of, topk_w,
                       reinterpret_cast<const float*>(residual), T, d, k,
                       reinterpret_cast<float*>(out));
  return hipGetLastError();
}

hipError_t launch_combine_clusters(foe_dtype dt, int C, int T, int d, int k, const void* y,
                                   const int32_t* row_of_all, const float* w_all, const void* x,
                                   float scale, void* out, hipStream_t s, const int32_t* sel_all,
                                   int E) {
  if (T == 0) return hipSuccess;
  const int y_rows = C * T * k;
  const int nvec = d / (dt == FOE_BF16 ? 8 : 4);
  const long long nch = ceil_div(nvec, FOE_COMBINE_U * kWave);
  dim3 grid(ceil_div((long long)T * nch, 4));
  ProfileScope ps("combine", s);
  // rows loaded together: 2 (one round at two pairs per token), else 4
  const bool two = (long long)C * k <= 2;
  if (dt == FOE_BF16) {
    const bf16* yb = reinterpret_cast<const bf16*>(y);
    const bf16* xb = reinterpret_cast<const bf16*>(x);
    bf16* ob = reinterpret_cast<bf16*>(out);
    if (two)
      FOE_LAUNCH((combine_clusters_kernel<bf16, 2>), grid, dim3(256), 0, s, yb, row_of_all,
                 sel_all, E, w_all, xb, C, T, d, k, y_rows, scale, ob);
    else
      FOE_LAUNCH((combine_clusters_kernel<bf16, 4>), grid, dim3(256), 0, s, yb, row_of_all,
                 sel_all, E, w_all, xb, C, T, d, k, y_rows, scale, ob);
  } else {
    const float* yf = reinterpret_cast<const float*>(y);
    const float* xf = reinterpret_cast<const float*>(x);
    float* of = reinterpret_cast<float*>(out);
    if (two)
      FOE_LAUNCH((combine_clusters_kernel<float, 2>), grid, dim3(256), 0, s, yf, row_of_all,
                 sel_all, E, w_all, xf, C, T, d, k, y_rows, scale, of);
    else
      FOE_LAUNCH((combine_clusters_kernel<float, 4>), grid, dim3(256), 0, s, yf, row_of_all,
                 sel_all, E, w_all, xf, C, T, d, k, y_rows, scale, of);
  }
  return hipGetLastError();
}

hipError_t launch_reduce(foe_dtype dt, int C, int T, int d, const void* partials,
                         const void* residual, float scale, void* out, hipStream_t s) {
  if (T == 0) return hipSuccess;
  const long long plane = (long long)T * d;
  const long long nvec = plane / (dt == FOE_BF16 ? 8 : 4);
  const long long want = (nvec + 255) / 256;
  dim3 grid((unsigned)(want < 8192 ? want : 8192));
  ProfileScope ps("reduce", s);
  if (dt == FOE_BF16)
    FOE_LAUNCH(reduce_kernel<bf16>, grid, dim3(256), 0, s,
                       reinterpret_cast<const bf16*>(partials),
                       reinterpret_cast<const bf16*>(residual), scale, C, nvec, plane,
                       reinterpret_cast<bf16*>(out));
  else
    FOE_LAUNCH(reduce_kernel<float>, grid, dim3(256), 0, s,
                       reinterpret_cast<const float*>(partials),
                       reinterpret_cast<const float*>(residual), scale, C, nvec, plane,
                       reinterpret_cast<float*>(out));
  return hipGetLastError();
}

}  // namespace foe
