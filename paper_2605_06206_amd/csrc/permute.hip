// Expert histogram, prefix sum and stable permutation of (token, slot) pairs:
// the on-device form of the intra-group dispatch (Section 3.2).
//
//   hist    : per-block expert counts of a chunk of kChunk pairs (LDS atomics;
//             integer adds commute, so the counts are deterministic)
//   scan    : one workgroup; per expert the exclusive prefix over blocks, then
//             the exclusive prefix over experts -> offsets, block bases
//   rank    : each block re-walks its chunk in flat order; a wave-level
//             ballot/popcount gives each pair its rank among the earlier pairs
//             of the same expert, so the order is (expert asc, flat index asc)
//             whatever the atomics did
//   scatter : every token row of x is read once and written to its k
//             destination rows with 128-bit stores
#include "foe_common.hpp"

namespace foe {
namespace {

constexpr int kChunk = 1024;            // pairs per block
constexpr int kWavesP = 4;
constexpr int kPerWave = kChunk / kWavesP;  // 512 pairs per wave
constexpr int kMaxE = 256;

__global__ __launch_bounds__(256) void hist_kernel(const int32_t* __restrict__ idx, int R, int E,
                                                   int32_t* __restrict__ block_counts) {
  __shared__ int cnt[kMaxE];
  for (int e = threadIdx.x; e < E; e += blockDim.x) cnt[e] = 0;
  __syncthreads();
  const int base = blockIdx.x * kChunk;
  const int end = min(base + kChunk, R);
  for (int f = base + threadIdx.x; f < end; f += blockDim.x) {
    const int e = idx[f];
    if (e >= 0 && e < E) atomicAdd(&cnt[e], 1);
  }
  __syncthreads();
  for (int e = threadIdx.x; e < E; e += blockDim.x)
    block_counts[(size_t)blockIdx.x * E + e] = cnt[e];
}

// Block counts are staged in LDS with coalesced loads (when they fit), so the
// per-expert prefix over blocks reads LDS instead of a chain of dependent
// global loads.
constexpr int kScanStage = 8192;  // int32 entries of block counts staged in LDS

__global__ __launch_bounds__(256) void scan_kernel(const int32_t* __restrict__ block_counts,
                                                   int nblk, int E,
                                                   int32_t* __restrict__ counts,
                                                   int32_t* __restrict__ offsets,
                                                   int32_t* __restrict__ block_base, int row_base,
                                                   int write_end) {
  __shared__ int total[kMaxE + 1];
  __shared__ int staged[kScanStage];
  const int e = threadIdx.x;
  const int n = nblk * E;
  const bool stage = n <= kScanStage;
  if (stage)
    for (int i = threadIdx.x; i < n; i += blockDim.x) staged[i] = block_counts[i];
  __syncthreads();
  if (e < E) {
    int run = 0;
    for (int b = 0; b < nblk; ++b) {
      const int c = stage ? staged[b * E + e] : block_counts[(size_t)b * E + e];
      if (stage)
        staged[b * E + e] = run;
      else
        block_base[(size_t)b * E + e] = run;
      run += c;
    }
    total[e] = run;
  }
  __syncthreads();
  // exclusive prefix over experts (E <= 256)
  if (threadIdx.x == 0) {
    int run = 0;
    for (int i = 0; i < E; ++i) {
      const int c = total[i];
      total[i] = run;
      run += c;
    }
    total[E] = run;
  }
  __syncthreads();
  if (e < E) {
    const int off = total[e];
    offsets[e] = row_base + off;
    if (counts != nullptr) counts[e] = total[e + 1] - off;
  }
  if (e == 0 && write_end) offsets[E] = row_base + total[E];
  // block bases (coalesced stores)
  if (stage) {
    for (int i = threadIdx.x; i < n; i += blockDim.x) block_base[i] = staged[i] + total[i % E];
  } else if (e < E) {
    for (int b = 0; b < nblk; ++b) block_base[(size_t)b * E + e] += total[e];
  }
}

__global__ __launch_bounds__(256) void rank_kernel(const int32_t* __restrict__ idx, int R, int E,
                                                   const int32_t* __restrict__ block_base,
                                                   int32_t* __restrict__ sorted_src,
                                                   int32_t* __restrict__ row_of, int row_base) {
  __shared__ int wcnt[kWavesP][kMaxE];
  const int lane = lane_id();
  const int wave = threadIdx.x >> 6;
  for (int i = threadIdx.x; i < kWavesP * kMaxE; i += blockDim.x) (&wcnt[0][0])[i] = 0;
  __syncthreads();

  const int start = blockIdx.x * kChunk + wave * kPerWave;
  const int end = min(start + kPerWave, R);
  // 1) per-wave counts of its contiguous sub-range
  for (int f = start + lane; f < end; f += kWave) {
    const int e = idx[f];
    if (e >= 0 && e < E) atomicAdd(&wcnt[wave][e], 1);
  }
  __syncthreads();
  // 2) per-wave base = block base + counts of the earlier waves (in place)
  for (int e = threadIdx.x; e < E; e += blockDim.x) {
    int run = block_base[(size_t)blockIdx.x * E + e];
    for (int w = 0; w < kWavesP; ++w) {
      const int c = wcnt[w][e];
      wcnt[w][e] = run;
      run += c;
    }
  }
  __syncthreads();
  // 3) ranks in flat order, 64 pairs at a time
  const uint64_t lt_mask = (lane == 0) ? 0ull : (~0ull >> (64 - lane));
  for (int f0 = start; f0 < end; f0 += kWave) {
    const int f = f0 + lane;
    const bool valid = f < end;
    const int e = valid ? idx[f] : -1;
    const bool ok = valid && e >= 0 && e < E;
    if (valid && !ok) row_of[f] = -1;
    uint64_t remaining = __ballot(ok);
    while (remaining) {
      const int leader = __builtin_ctzll(remaining);
      const int v = __builtin_amdgcn_readlane(e, leader);
      const uint64_t m = __ballot(ok && e == v);
      const int base = wcnt[wave][v];
      if (ok && e == v) {
        const int p = base + __popcll(m & lt_mask);
        sorted_src[p] = f;
        row_of[f] = row_base + p;
      }
      if (lane == leader) wcnt[wave][v] = base + __popcll(m);
      remaining &= ~m;
    }
  }
}

// Small R: histogram, scan and stable ranks in one workgroup of 16 waves;
// workgroup h handles cluster h (ids idx + h*R, outputs at h*R / h*E, rows
// numbered from row_base = h*R).  Wave w owns the contiguous pairs
// [w*per, (w+1)*per); per-wave counts give every wave its base per expert,
// then each wave ranks its pairs in flat order with the same ballot walk as
// rank_kernel.  The last workgroup writes the final offset.
constexpr int kSmallWaves = 16;
constexpr int kSmallMaxR = 8192;

__global__ __launch_bounds__(kSmallWaves * 64) void index_small_kernel(
    const int32_t* __restrict__ idx_all, int R, int E, int32_t* __restrict__ counts_all,
    int32_t* __restrict__ offsets_all, int32_t* __restrict__ sorted_src_all,
    int32_t* __restrict__ row_of_all) {
  const int h = blockIdx.x;
  const int row_base = h * R;
  const int32_t* __restrict__ idx = idx_all + (size_t)h * R;
  int32_t* __restrict__ counts = counts_all != nullptr ? counts_all + (size_t)h * E : nullptr;
  int32_t* __restrict__ offsets = offsets_all + (size_t)h * E;
  int32_t* __restrict__ sorted_src = sorted_src_all + (size_t)h * R;
  int32_t* __restrict__ row_of = row_of_all + (size_t)h * R;
  __shared__ int wcnt[kSmallWaves][kMaxE];
  __shared__ int total[kMaxE + 1];
  const int lane = lane_id();
  const int wave = threadIdx.x >> 6;
  for (int i = threadIdx.x; i < kSmallWaves * kMaxE; i += blockDim.x) (&wcnt[0][0])[i] = 0;
  __syncthreads();
  const int per = (R + kSmallWaves * kWave - 1) / (kSmallWaves * kWave) * kWave;
  const int start = wave * per;
  const int end = min(start + per, R);
  for (int f = start + lane; f < end; f += kWave) {
    const int e = idx[f];
    if (e >= 0 && e < E) atomicAdd(&wcnt[wave][e], 1);
  }
  __syncthreads();
  if (threadIdx.x < E) {
    const int e = threadIdx.x;
    int run = 0;
    for (int w = 0; w < kSmallWaves; ++w) run += wcnt[w][e];
    total[e] = run;
  }
  __syncthreads();
  if (threadIdx.x == 0) {
    int run = 0;
    for (int i = 0; i < E; ++i) {
      const int c = total[i];
      total[i] = run;
      run += c;
    }
    total[E] = run;
  }
  __syncthreads();
  if (threadIdx.x < E) {
    const int e = threadIdx.x;
    int run = total[e];
    offsets[e] = row_base + run;
    if (counts != nullptr) counts[e] = total[e + 1] - run;
    for (int w = 0; w < kSmallWaves; ++w) {
      const int c = wcnt[w][e];
      wcnt[w][e] = run;
      run += c;
    }
  }
  if (threadIdx.x == 0 && h == (int)gridDim.x - 1) offsets[E] = row_base + total[E];
  __syncthreads();
  const uint64_t lt_mask = (lane == 0) ? 0ull : (~0ull >> (64 - lane));
  for (int f0 = start; f0 < end; f0 += kWave) {
    const int f = f0 + lane;
    const bool valid = f < end;
    const int e = valid ? idx[f] : -1;
    const bool ok = valid && e >= 0 && e < E;
    if (valid && !ok) row_of[f] = -1;
    uint64_t remaining = __ballot(ok);
    while (remaining) {
      const int leader = __builtin_ctzll(remaining);
      const int v = __builtin_amdgcn_readlane(e, leader);
      const uint64_t m = __ballot(ok && e == v);
      const int base = wcnt[wave][v];
      if (ok && e == v) {
        const int p = base + __popcll(m & lt_mask);
        sorted_src[p] = f;
        row_of[f] = row_base + p;
      }
      if (lane == leader) wcnt[wave][v] = base + __popcll(m);
      remaining &= ~m;
    }
  }
}

template <typename T>
__global__ __launch_bounds__(256) void scatter_rows_kernel(const T* __restrict__ x,
                                                           const int32_t* __restrict__ row_of,
                                                           int T_, int d, int k, int R,
                                                           T* __restrict__ x_perm) {
  constexpr int EPV = Vec16<T>::N;
  const int lane = lane_id();
  const int tok = blockIdx.x * 4 + (threadIdx.x >> 6);
  if (tok >= T_) return;
  const int nvec = d / EPV;
  const T* src = x + (size_t)tok * d;
  for (int c0 = 0; c0 < nvec; c0 += 4 * kWave) {
    Vec16<T> v[4];
#pragma unroll
    for (int u = 0; u < 4; ++u) {
      const int c = c0 + u * kWave + lane;
      if (c < nvec) v[u] = load16_cached(src + (size_t)c * EPV);
    }
    for (int j = 0; j < k; ++j) {
      const int p = row_of[(size_t)tok * k + j];
      if (p < 0 || p >= R) continue;
      T* dst = x_perm + (size_t)p * d;
#pragma unroll
      for (int u = 0; u < 4; ++u) {
        const int c = c0 + u * kWave + lane;
        if (c < nvec) store16(dst + (size_t)c * EPV, v[u]);
      }
    }
  }
}

__global__ void fill_i32_kernel(int32_t* p, int n, int32_t v) {
  const int i = blockIdx.x * blockDim.x + threadIdx.x;
  if (i < n) p[i] = v;
}

}  // namespace

int permute_blocks(int R) { return R > 0 ? ceil_div(R, kChunk) : 0; }

size_t permute_scratch_bytes(int T, int k, int E) {
  const size_t nblk = (size_t)permute_blocks(T * k);
  return 2 * nblk * (size_t)E * sizeof(int32_t);
}

hipError_t launch_fill_i32(int32_t* p, int n, int32_t v, hipStream_t s) {
  if (n <= 0) return hipSuccess;
  ProfileScope ps("fill_i32", s);
  hipLaunchKernelGGL(fill_i32_kernel, dim3(ceil_div(n, 256)), dim3(256), 0, s, p, n, v);
  return hipGetLastError();
}

hipError_t launch_index(int T, int E, int k, int C, const int32_t* topk_idx, int32_t* counts,
                        int32_t* offsets, int32_t* sorted_src, int32_t* row_of, void* scratch,
                        hipStream_t s) {
  const int R = T * k;
  if (R == 0) {
    hipError_t err = launch_fill_i32(offsets, C * E + 1, 0, s);
    if (err == hipSuccess && counts != nullptr) err = launch_fill_i32(counts, C * E, 0, s);
    return err;
  }
  if (R <= kSmallMaxR) {
    ProfileScope ps("permute_index", s);
    hipLaunchKernelGGL(index_small_kernel, dim3(C), dim3(kSmallWaves * kWave), 0, s, topk_idx, R,
                       E, counts, offsets, sorted_src, row_of);
    return hipGetLastError();
  }
  const int nblk = permute_blocks(R);
  int32_t* block_counts = reinterpret_cast<int32_t*>(scratch);
  int32_t* block_base = block_counts + (size_t)nblk * E;
  for (int h = 0; h < C; ++h) {
    const int32_t* idx_h = topk_idx + (size_t)h * R;
    {
      ProfileScope ps("permute_hist", s);
      hipLaunchKernelGGL(hist_kernel, dim3(nblk), dim3(256), 0, s, idx_h, R, E, block_counts);
    }
    {
      ProfileScope ps("permute_scan", s);
      hipLaunchKernelGGL(scan_kernel, dim3(1), dim3(256), 0, s, block_counts, nblk, E,
                         counts != nullptr ? counts + (size_t)h * E : nullptr,
                         offsets + (size_t)h * E, block_base, h * R, h == C - 1 ? 1 : 0);
    }
    {
      ProfileScope ps("permute_rank", s);
      hipLaunchKernelGGL(rank_kernel, dim3(nblk), dim3(256), 0, s, idx_h, R, E, block_base,
                         sorted_src + (size_t)h * R, row_of + (size_t)h * R, h * R);
    }
  }
  return hipGetLastError();
}

hipError_t launch_permute(foe_dtype dt, int T, int d, int E, int k, const int32_t* topk_idx,
                          const void* x, int32_t* counts, int32_t* offsets, int32_t* sorted_src,
                          int32_t* row_of, void* x_perm, void* scratch, hipStream_t s) {
  hipError_t err =
      launch_index(T, E, k, 1, topk_idx, counts, offsets, sorted_src, row_of, scratch, s);
  if (err != hipSuccess || T == 0) return err;
  const int R = T * k;
  ProfileScope ps("permute_scatter", s);
  dim3 grid(ceil_div(T, 4));
  if (dt == FOE_BF16)
    hipLaunchKernelGGL(scatter_rows_kernel<bf16>, grid, dim3(256), 0, s,
                       reinterpret_cast<const bf16*>(x), row_of, T, d, k, R,
                       reinterpret_cast<bf16*>(x_perm));
  else
    hipLaunchKernelGGL(scatter_rows_kernel<float>, grid, dim3(256), 0, s,
                       reinterpret_cast<const float*>(x), row_of, T, d, k, R,
                       reinterpret_cast<float*>(x_perm));
  return hipGetLastError();
}

}  // namespace foe
