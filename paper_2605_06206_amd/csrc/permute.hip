// Expert histogram, prefix sum and stable permutation of (token, slot) pairs:
// the on-device form of the intra-group dispatch (Section 3.2).
//
//   hist    : per-block expert counts of a chunk of kChunk pairs (LDS atomics;
//             integer adds commute, so the counts are deterministic)
//   rank    : one pair per thread.  A wave finds the lanes that share its
//             lane's expert with ceil(log2 E) ballots (one per bit of the
//             expert id), so a pair's rank among the earlier pairs of its
//             expert in the wave is a popcount.  Per-wave counts, the counts
//             of the earlier blocks and the per-expert totals give the base,
//             and the order is (expert asc, flat index asc) whatever the
//             atomics did.  The block counts are summed by every block, so
//             there is no separate scan launch; past kFoldMax block counts a
//             scan kernel writes the block bases instead.
//   scatter : every token row of x is read once and written to its k
//             destination rows with 128-bit stores
// All clusters of a block run in one grid (blockIdx.y = cluster).
#include "foe_common.hpp"

namespace foe {
namespace {

constexpr int kChunk = 1024;  // pairs per block, one per thread in rank
constexpr int kRankWaves = kChunk / kWave;
constexpr int kMaxE = 256;
constexpr int kFoldMax = 16384;  // block counts per cluster summed inside rank

// Lanes of the wave whose expert equals this lane's, among the lanes with ok:
// the AND over the id's bits of the ballot of that bit or of its complement.
// Valid when every expert id is below 2^nbits.
__device__ __forceinline__ uint64_t match_expert(int e, bool ok, int nbits) {
  uint64_t m = __ballot(ok);
  for (int b = 0; b < nbits; ++b) {
    const bool bit = (e >> b) & 1;
    const uint64_t bb = __ballot(ok && bit);
    m &= bit ? bb : ~bb;
  }
  return m;
}

__device__ __forceinline__ uint64_t lanes_below() {
  const int lane = lane_id();
  return lane == 0 ? 0ull : (~0ull >> (64 - lane));
}

// Exclusive prefix of total[0..E) in place, total[E] = the sum; run by one
// whole wave (E <= 256: four experts per lane).
__device__ __forceinline__ void wave_excl_scan_experts(int* total, int E) {
  const int lane = lane_id();
  int v[4];
  int sum = 0;
#pragma unroll
  for (int j = 0; j < 4; ++j) {
    const int i = lane * 4 + j;
    v[j] = i < E ? total[i] : 0;
    sum += v[j];
  }
  int incl = sum;
#pragma unroll
  for (int dlt = 1; dlt < kWave; dlt <<= 1) {
    const int t = __shfl_up(incl, dlt);
    if (lane >= dlt) incl += t;
  }
  int run = incl - sum;
#pragma unroll
  for (int j = 0; j < 4; ++j) {
    const int i = lane * 4 + j;
    if (i < E) total[i] = run;
    run += v[j];
  }
  if (lane == kWave - 1) total[E] = incl;
}

__global__ __launch_bounds__(256) void hist_kernel(const int32_t* __restrict__ idx_all, int R,
                                                   int E, int32_t* __restrict__ block_counts_all) {
  __shared__ int cnt[kMaxE];
  const int h = blockIdx.y;
  const int32_t* __restrict__ idx = idx_all + (size_t)h * R;
  for (int e = threadIdx.x; e < E; e += blockDim.x) cnt[e] = 0;
  __syncthreads();
  const int base = blockIdx.x * kChunk;
  const int end = min(base + kChunk, R);
  for (int f = base + threadIdx.x; f < end; f += blockDim.x) {
    const int e = idx[f];
    if (e >= 0 && e < E) atomicAdd(&cnt[e], 1);
  }
  __syncthreads();
  int32_t* __restrict__ bc = block_counts_all + ((size_t)h * gridDim.x + blockIdx.x) * E;
  for (int e = threadIdx.x; e < E; e += blockDim.x) bc[e] = cnt[e];
}

// Past kFoldMax block counts: one workgroup per cluster writes the block
// bases (expert offset + counts of the earlier blocks), offsets and counts.
__global__ __launch_bounds__(256) void scan_kernel(const int32_t* __restrict__ block_counts_all,
                                                   int nblk, int E, int R,
                                                   int32_t* __restrict__ counts_all,
                                                   int32_t* __restrict__ offsets_all,
                                                   int32_t* __restrict__ block_base_all) {
  __shared__ int total[kMaxE + 1];
  const int h = blockIdx.x;
  const int32_t* __restrict__ bc = block_counts_all + (size_t)h * nblk * E;
  int32_t* __restrict__ bb = block_base_all + (size_t)h * nblk * E;
  const int e = threadIdx.x;
  if (e < E) {
    int run = 0;
    for (int b = 0; b < nblk; ++b) {
      const int c = bc[(size_t)b * E + e];
      bb[(size_t)b * E + e] = run;
      run += c;
    }
    total[e] = run;
  }
  __syncthreads();
  if (threadIdx.x < kWave) wave_excl_scan_experts(total, E);
  __syncthreads();
  const int row_base = h * R;
  if (e < E) {
    const int off = total[e];
    offsets_all[(size_t)h * E + e] = row_base + off;
    if (counts_all != nullptr) counts_all[(size_t)h * E + e] = total[e + 1] - off;
    for (int b = 0; b < nblk; ++b) bb[(size_t)b * E + e] += off;
  }
  if (e == 0 && h == (int)gridDim.x - 1) offsets_all[(size_t)(h + 1) * E] = row_base + total[E];
}

template <bool FOLD>
__global__ __launch_bounds__(kChunk) void rank_kernel(
    const int32_t* __restrict__ idx_all, int R, int E, int nbits,
    const int32_t* __restrict__ block_counts_all, const int32_t* __restrict__ block_base_all,
    int32_t* __restrict__ counts_all, int32_t* __restrict__ offsets_all,
    int32_t* __restrict__ sorted_src_all, int32_t* __restrict__ row_of_all,
    int32_t* __restrict__ zero, int nzero, int ncb, int cb_pairs) {
  // counters of the next kernel, cleared on the way (one workgroup)
  if (blockIdx.x == 0 && blockIdx.y == 0)
    for (int i = threadIdx.x; i < nzero; i += blockDim.x) zero[i] = 0;
  __shared__ int wcnt[kRankWaves][kMaxE];
  __shared__ int total[kMaxE + 1];
  __shared__ int before[kMaxE];
  const int h = blockIdx.y;
  const int nblk = gridDim.x;
  const int row_base = h * R;
  const int32_t* __restrict__ idx = idx_all + (size_t)h * R;
  int32_t* __restrict__ sorted_src = sorted_src_all + (size_t)h * R;
  int32_t* __restrict__ row_of = row_of_all + (size_t)h * R;
  const int tid = threadIdx.x;
  const int wave = tid >> 6;
  for (int i = tid; i < kRankWaves * kMaxE; i += kChunk) (&wcnt[0][0])[i] = 0;
  if (FOLD && tid < E) total[tid] = before[tid] = 0;
  __syncthreads();

  const int f = blockIdx.x * kChunk + tid;
  const bool valid = f < R;
  const int e = valid ? idx[f] : -1;
  const bool ok = valid && e >= 0 && e < E;
  const uint64_t m = match_expert(e, ok, nbits);
  const int r = __popcll(m & lanes_below());
  if (ok && r == 0) wcnt[wave][e] = __popcll(m);

  if (FOLD) {
    // per-expert totals and counts of the pairs before this block, from the
    // ncb count blocks of cb_pairs pairs each (split over kChunk / E parts of
    // the count-block list); the pairs of a count block that straddles this
    // block's start are counted here directly
    const int32_t* __restrict__ bc = block_counts_all + (size_t)h * ncb * E;
    const int parts = kChunk / E;
    const int pe = tid % E, part = tid / E;
    const int start = blockIdx.x * kChunk;
    const int full = start / cb_pairs;  // count blocks wholly before this block
    if (part < parts) {
      // eight count blocks' loads in flight at a time (one at a time, their
      // latencies added up: 8 of them per thread at 256 count blocks and 32
      // experts; index pass 6.3 -> 5.1 us there)
      int all = 0, bef = 0;
      int b = part;
      for (; b + 7 * parts < ncb; b += 8 * parts) {
        int c[8];
#pragma unroll
        for (int u = 0; u < 8; ++u) c[u] = bc[(size_t)(b + u * parts) * E + pe];
#pragma unroll
        for (int u = 0; u < 8; ++u) {
          all += c[u];
          bef += b + u * parts < full ? c[u] : 0;
        }
      }
      for (; b < ncb; b += parts) {
        const int c = bc[(size_t)b * E + pe];
        all += c;
        bef += b < full ? c : 0;
      }
      atomicAdd(&total[pe], all);
      atomicAdd(&before[pe], bef);
    }
    for (int f2 = full * cb_pairs + tid; f2 < start; f2 += kChunk) {
      const int e2 = idx[f2];
      if (e2 >= 0 && e2 < E) atomicAdd(&before[e2], 1);
    }
    __syncthreads();
    if (tid < kWave) wave_excl_scan_experts(total, E);
  }
  __syncthreads();
  if (FOLD && blockIdx.x == 0) {
    if (tid < E) {
      offsets_all[(size_t)h * E + tid] = row_base + total[tid];
      if (counts_all != nullptr) counts_all[(size_t)h * E + tid] = total[tid + 1] - total[tid];
    }
    if (tid == 0 && h == (int)gridDim.y - 1) offsets_all[(size_t)(h + 1) * E] = row_base + total[E];
  }
  // per-wave base = expert offset + earlier blocks + earlier waves (in place)
  if (tid < E) {
    int run = FOLD ? total[tid] + before[tid]
                   : block_base_all[((size_t)h * nblk + blockIdx.x) * E + tid];
#pragma unroll
    for (int w = 0; w < kRankWaves; ++w) {
      const int c = wcnt[w][tid];
      wcnt[w][tid] = run;
      run += c;
    }
  }
  __syncthreads();
  if (ok) {
    const int p = wcnt[wave][e] + r;
    sorted_src[p] = f;
    row_of[f] = row_base + p;
  } else if (valid) {
    row_of[f] = -1;
  }
}

// Small R: histogram, prefix sum and stable ranks in one workgroup of 16
// waves per cluster.  Wave w owns the contiguous range [w*per, (w+1)*per);
// its per-chunk match masks give per-wave counts, then every wave ranks its
// pairs in flat order, 64 at a time.
constexpr int kSmallWaves = 16;
// up to this many pairs per cluster the one-workgroup pass beats the two
// launches of hist + rank (about 4 µs plus 1 µs per 1000 pairs against 8 µs)
constexpr int kSmallMaxR = 4096;

__global__ __launch_bounds__(kSmallWaves * 64) void index_small_kernel(
    const int32_t* __restrict__ idx_all, int R, int E, int nbits,
    int32_t* __restrict__ counts_all, int32_t* __restrict__ offsets_all,
    int32_t* __restrict__ sorted_src_all, int32_t* __restrict__ row_of_all,
    int32_t* __restrict__ zero, int nzero) {
  // counters of the next kernel, cleared on the way (one workgroup)
  if (blockIdx.x == 0)
    for (int i = threadIdx.x; i < nzero; i += blockDim.x) zero[i] = 0;
  const int h = blockIdx.x;
  const int row_base = h * R;
  const int32_t* __restrict__ idx = idx_all + (size_t)h * R;
  int32_t* __restrict__ sorted_src = sorted_src_all + (size_t)h * R;
  int32_t* __restrict__ row_of = row_of_all + (size_t)h * R;
  __shared__ int wcnt[kSmallWaves][kMaxE];
  __shared__ int total[kMaxE + 1];
  const int wave = threadIdx.x >> 6;
  for (int i = threadIdx.x; i < kSmallWaves * kMaxE; i += blockDim.x) (&wcnt[0][0])[i] = 0;
  __syncthreads();
  const int per = (R + kSmallWaves * kWave - 1) / (kSmallWaves * kWave) * kWave;
  const int start = wave * per;
  const int end = min(start + per, R);
  const uint64_t below = lanes_below();
  for (int f0 = start; f0 < end; f0 += kWave) {
    const int f = f0 + lane_id();
    const int e = f < end ? idx[f] : -1;
    const bool ok = e >= 0 && e < E;
    const uint64_t m = match_expert(e, ok, nbits);
    if (ok && __popcll(m & below) == 0) wcnt[wave][e] += __popcll(m);
  }
  __syncthreads();
  if (threadIdx.x < E) {
    int run = 0;
    for (int w = 0; w < kSmallWaves; ++w) run += wcnt[w][threadIdx.x];
    total[threadIdx.x] = run;
  }
  __syncthreads();
  if (threadIdx.x < kWave) wave_excl_scan_experts(total, E);
  __syncthreads();
  if (threadIdx.x < E) {
    const int ex = threadIdx.x;
    int run = total[ex];
    offsets_all[(size_t)h * E + ex] = row_base + run;
    if (counts_all != nullptr) counts_all[(size_t)h * E + ex] = total[ex + 1] - run;
    for (int w = 0; w < kSmallWaves; ++w) {
      const int c = wcnt[w][ex];
      wcnt[w][ex] = run;
      run += c;
    }
  }
  if (threadIdx.x == 0 && h == (int)gridDim.x - 1)
    offsets_all[(size_t)(h + 1) * E] = row_base + total[E];
  __syncthreads();
  for (int f0 = start; f0 < end; f0 += kWave) {
    const int f = f0 + lane_id();
    const bool valid = f < end;
    const int e = valid ? idx[f] : -1;
    const bool ok = valid && e >= 0 && e < E;
    const uint64_t m = match_expert(e, ok, nbits);
    const int r = __popcll(m & below);
    // every lane reads its base before the group's first lane advances it
    // (a wave's LDS operations complete in order)
    const int base = ok ? wcnt[wave][e] : 0;
    if (ok) {
      sorted_src[base + r] = f;
      row_of[f] = row_base + base + r;
      if (r == 0) wcnt[wave][e] = base + __popcll(m);
    } else if (valid) {
      row_of[f] = -1;
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

size_t permute_scratch_bytes(int T, int k, int E, int C) {
  const size_t nblk = (size_t)permute_blocks(T * k);
  return 2 * (size_t)C * nblk * (size_t)E * sizeof(int32_t);
}

hipError_t launch_fill_i32(int32_t* p, int n, int32_t v, hipStream_t s) {
  if (n <= 0) return hipSuccess;
  ProfileScope ps("fill_i32", s);
  FOE_LAUNCH(fill_i32_kernel, dim3(ceil_div(n, 256)), dim3(256), 0, s, p, n, v);
  return hipGetLastError();
}

bool index_takes_route_counts(int T, int E, int k, int ncb) {
  const long long R = (long long)T * k;
  return R > kSmallMaxR && (long long)ncb * E <= kFoldMax;
}

hipError_t launch_index(int T, int E, int k, int C, const int32_t* topk_idx, int32_t* counts,
                        int32_t* offsets, int32_t* sorted_src, int32_t* row_of, void* scratch,
                        hipStream_t s, int32_t* zero, int nzero, const int32_t* route_counts,
                        int tok_per_cb, int ncb) {
  const int R = T * k;
  if (R == 0) {
    hipError_t err = launch_fill_i32(offsets, C * E + 1, 0, s);
    if (err == hipSuccess && counts != nullptr) err = launch_fill_i32(counts, C * E, 0, s);
    if (err == hipSuccess && nzero > 0) err = launch_fill_i32(zero, nzero, 0, s);
    return err;
  }
  const int nbits = E <= 1 ? 0 : 32 - __builtin_clz((unsigned)(E - 1));
  if (R <= kSmallMaxR) {
    ProfileScope ps("permute_index", s);
    FOE_LAUNCH(index_small_kernel, dim3(C), dim3(kSmallWaves * kWave), 0, s, topk_idx, R,
                       E, nbits, counts, offsets, sorted_src, row_of, zero, nzero);
    return hipGetLastError();
  }
  const int nblk = permute_blocks(R);
  if (route_counts != nullptr && index_takes_route_counts(T, E, k, ncb)) {
    // the routing kernel counted the experts of its token blocks
    ProfileScope ps("permute_rank", s);
    FOE_LAUNCH(rank_kernel<true>, dim3(nblk, C), dim3(kChunk), 0, s, topk_idx, R, E, nbits,
               route_counts, nullptr, counts, offsets, sorted_src, row_of, zero, nzero, ncb,
               tok_per_cb * k);
    return hipGetLastError();
  }
  int32_t* block_counts = reinterpret_cast<int32_t*>(scratch);
  int32_t* block_base = block_counts + (size_t)C * nblk * E;
  {
    ProfileScope ps("permute_hist", s);
    FOE_LAUNCH(hist_kernel, dim3(nblk, C), dim3(256), 0, s, topk_idx, R, E, block_counts);
  }
  const bool fold = (size_t)nblk * E <= (size_t)kFoldMax;
  if (!fold) {
    ProfileScope ps("permute_scan", s);
    FOE_LAUNCH(scan_kernel, dim3(C), dim3(256), 0, s, block_counts, nblk, E, R, counts,
                       offsets, block_base);
  }
  {
    ProfileScope ps("permute_rank", s);
    if (fold)
      FOE_LAUNCH(rank_kernel<true>, dim3(nblk, C), dim3(kChunk), 0, s, topk_idx, R, E,
                         nbits, block_counts, block_base, counts, offsets, sorted_src, row_of,
                         zero, nzero, nblk, kChunk);
    else
      FOE_LAUNCH(rank_kernel<false>, dim3(nblk, C), dim3(kChunk), 0, s, topk_idx, R, E,
                         nbits, block_counts, block_base, counts, offsets, sorted_src, row_of,
                         zero, nzero, nblk, kChunk);
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
    FOE_LAUNCH(scatter_rows_kernel<bf16>, grid, dim3(256), 0, s,
                       reinterpret_cast<const bf16*>(x), row_of, T, d, k, R,
                       reinterpret_cast<bf16*>(x_perm));
  else
    FOE_LAUNCH(scatter_rows_kernel<float>, grid, dim3(256), 0, s,
                       reinterpret_cast<const float*>(x), row_of, T, d, k, R,
                       reinterpret_cast<float*>(x_perm));
  return hipGetLastError();
}

}  // namespace foe
