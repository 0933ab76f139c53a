// Grouped SwiGLU expert FFN (Table 3 "MoE update": FFN_e on the rows routed
// to expert e).  Two grouped GEMMs over the permuted rows:
//   gate/up : h[rows,F] = silu(A W_g[e]^T) * (A W_u[e]^T)   (SwiGLU fused into
//             the epilogue; both products share the A tile)
//   down    : y[rows,d] = h W_d[e]^T
// Every weight is [out,in] (K-contiguous), so both GEMMs are "NT".  Row r of A
// is either row r of a permuted copy (x_perm) or, with a gather list, row
// gather[r] / kdiv of the unpermuted input: then the permutation is folded
// into the operand loads and x_perm is never written.
//
// bf16, many rows per expert (MFMA-bound): 8 waves (2 per SIMD) on a 256-row
// tile, v_mfma_f32_32x32x16_bf16 with fp32 accumulation, operands staged
// through two LDS stages.  Loads use buffer resources whose range ends where
// the valid rows / K end, so ragged tiles read zeros without branches.  The
// MFMA computes D = W_tile * A_tile^T: each lane holds 4 consecutive output
// columns of one row.  The expert and row range of a workgroup come from the
// device-side offsets (one wave prefix sum over per-expert tile counts), so no
// host sync is needed.
//
// bf16, few rows per expert (decode, weight-streaming bound): see
// ffn_skinny_bf16.  fp32: plain FMA kernels (small shapes only).
#include "foe_common.hpp"

// (BM, BN per weight matrix, waves along M, waves along N) of the large-M
// kernel; (register staging sets, max waves per SIMD); (K-split waves, K
// chunks per load batch) of the weight-streaming kernel.
#ifndef FOE_PIPE_GU
#define FOE_PIPE_GU 256, 128, 2, 4
#endif
#ifndef FOE_PIPE_DN
#define FOE_PIPE_DN 256, 256, 2, 4
#endif
#ifndef FOE_PIPE_OPT
#define FOE_PIPE_OPT 1, 2
#endif
#ifndef FOE_SKINNY
#define FOE_SKINNY 4, 4
#endif

namespace foe {
namespace {

template <int W, int U> struct FirstOf { static constexpr int value = W; };

// Find the (expert, first row, row end) of global M-tile `mt`.  Returns false
// if `mt` is past the last tile.  Offsets are clamped to [0, rows]; a
// decreasing bound gives an empty segment.  Lane l counts the tiles of a
// contiguous range of experts; a wave prefix sum locates the lane holding
// `mt`, which walks its range again to find the expert.
__device__ bool find_tile(const int32_t* __restrict__ offsets, int E, int rows, int BM, int mt,
                          int& e_out, int& row0, int& row_end) {
  const int lane = lane_id();
  const int per = (E + kWave - 1) / kWave;
  const int e_begin = min(lane * per, E), e_end = min(e_begin + per, E);
  auto seg = [&](int e, int& a, int& b) {
    a = min(max(offsets[e], 0), rows);
    b = min(max(offsets[e + 1], 0), rows);
    if (b < a) b = a;
  };
  int mine = 0;
  for (int e = e_begin; e < e_end; ++e) {
    int a, b;
    seg(e, a, b);
    mine += (b - a + BM - 1) / BM;
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
  if (lane == src) {
    int t = mt - excl;
    for (int e = e_begin; e < e_end; ++e) {
      int a, b;
      seg(e, a, b);
      const int n = (b - a + BM - 1) / BM;
      if (t < n) {
        e_sel = e;
        r0 = a + t * BM;
        r1 = b;
        break;
      }
      t -= n;
    }
  }
  e_out = __builtin_amdgcn_readlane(e_sel, src);
  row0 = __builtin_amdgcn_readlane(r0, src);
  row_end = __builtin_amdgcn_readlane(r1, src);
  return true;
}

__device__ __forceinline__ float silu_f(float g) { return g / (1.0f + __expf(-g)); }

// Buffer resource over `nbytes` bytes from `base`: loads at offsets at or past
// `nbytes` return zeros, which handles ragged rows and K tails without branches.
__device__ __forceinline__ __amdgpu_buffer_rsrc_t make_rsrc(const void* base, uint32_t nbytes) {
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(base), (short)0, nbytes, 0x00020000);
}
__device__ __forceinline__ u32x4 buf_load16(__amdgpu_buffer_rsrc_t r, uint32_t off) {
  return __builtin_bit_cast(u32x4, __builtin_amdgcn_raw_buffer_load_b128(r, off, 0, 0));
}
// weight stream of the decode kernel: read once per call (cache policy AUX)
#ifndef FOE_WSTREAM_AUX
#define FOE_WSTREAM_AUX 0
#endif
__device__ __forceinline__ u32x4 buf_load16_stream(__amdgpu_buffer_rsrc_t r, uint32_t off) {
  return __builtin_bit_cast(u32x4, __builtin_amdgcn_raw_buffer_load_b128(r, off, 0, FOE_WSTREAM_AUX));
}
constexpr uint32_t kOob = 0x80000000u;  // past every buffer range used here: reads zeros

// Source row of operand row r: r itself, or gather[r] / kdiv (-1 if that row
// is outside [0, src_rows)).
__device__ __forceinline__ int src_row(const int32_t* __restrict__ gather, int kdiv, int r,
                                       int src_rows) {
  if (gather == nullptr) return r;
  const int g = gather[r];
  const int s = g >= 0 ? g / kdiv : -1;
  return s < src_rows ? s : -1;
}

// Workgroups are dealt round-robin to the 8 XCDs (each with its own L2).  The
// tile index is remapped so that each XCD walks a contiguous range of tiles:
// neighbouring tiles share their A rows (same M-tile) or their weight slice
// (same expert), and now meet in the same L2.
__device__ __forceinline__ int xcd_tile(int bid, int nblocks) {
  constexpr int kXcd = 8;
  const int per = (nblocks + kXcd - 1) / kXcd;
  return (bid % kXcd) * per + bid / kXcd;
}

// LDS-only workgroup barrier: waits for this wave's LDS operations and meets
// the other waves, but (unlike __syncthreads) does not drain outstanding
// global loads, so prefetches stay in flight across it.
__device__ __forceinline__ void lds_barrier() {
  asm volatile("s_waitcnt lgkmcnt(0)\n\ts_barrier" ::: "memory");
}

// Scheduling-group masks of __builtin_amdgcn_sched_group_barrier.
constexpr int kSchedMfma = 0x008, kSchedDsRead = 0x100, kSchedDsWrite = 0x200,
              kSchedVmemRead = 0x020;

// Ask the scheduler for the order  MFMA, LDS read, <share of X>, MFMA, ...
// over one k16 step: NM MFMAs, NR fragment reads and NX extra instructions of
// kind XMASK spread evenly after the reads.  A wave issues in order, so a
// burst of memory instructions would otherwise idle its MFMA pipe.
template <int I, int NM, int NR, int NX, int XMASK>
__device__ __forceinline__ void interleave() {
  if constexpr (I < NM) {
    __builtin_amdgcn_sched_group_barrier(kSchedMfma, 1, 0);
    if constexpr (I < NR) {
      __builtin_amdgcn_sched_group_barrier(kSchedDsRead, 1, 0);
      constexpr int per = (NX + NR - 1) / NR;
      constexpr int done = I * per;
      constexpr int n = (NX - done) < per ? (NX - done) : per;
      if constexpr (n > 0) __builtin_amdgcn_sched_group_barrier(XMASK, n, 0);
    }
    interleave<I + 1, NM, NR, NX, XMASK>();
  }
}

template <int BM, int BN, int BK, int WM, int WN, bool GATEUP>
struct GemmCfg {
  static constexpr int NTHR = WM * WN * kWave;
  static constexpr int WTM = BM / WM, WTN = BN / WN;
  static constexpr int SM = WTM / 32, SN = WTN / 32;
  static constexpr int NB = GATEUP ? 2 : 1;
  static constexpr int LDK = BK + 8;  // padded LDS row (elements): conflict-free 16-byte reads
  static constexpr int CPR = BK / 8;  // 16-byte chunks per tile row
  static constexpr int A_PER = BM * CPR / NTHR;
  static constexpr int B_PER = BN * CPR / NTHR;
  static constexpr int A_ELEMS = BM * LDK, B_ELEMS = BN * LDK;
  static constexpr int STAGE_ELEMS = A_ELEMS + NB * B_ELEMS;
  static_assert(WTM % 32 == 0 && WTN % 32 == 0, "wave tile must be a multiple of 32");
  static_assert(BK % 16 == 0, "BK multiple of 16");
  static_assert(BM * CPR % NTHR == 0 && BN * CPR % NTHR == 0, "even load split");
};

// Large-M grouped GEMM, BK = 64, two LDS stages.  Stage s is loaded into
// register set s % NSETS and written to LDS one iteration before its MFMAs.
// Per iteration (4 k16 steps):
//   ks0: read frags ks1; MFMA ks0; write the staged next stage to the other
//        LDS buffer
//   ks1: read frags ks2; MFMA ks1; issue the global loads of a later stage
//   ks2: read frags ks3; MFMA ks2; LDS barrier (next stage complete; nobody
//        reads this stage's buffer any more)
//   ks3: read frags ks0 of the next stage; MFMA ks3
// With a gather list, operand row r of A is row gather[r]/kdiv of A.
template <int BM, int BN, int WM, int WN, bool GATEUP, int NSETS, int MAXW>
__global__ __launch_bounds__(WM* WN* kWave) __attribute__((amdgpu_waves_per_eu(1, MAXW)))
void grouped_gemm_bf16(const bf16* __restrict__ A, const int32_t* __restrict__ gather, int kdiv,
                       int a_rows, const int32_t* __restrict__ offsets, int E, int rows,
                       const bf16* __restrict__ B0, const bf16* __restrict__ B1, int N, int K,
                       bf16* __restrict__ out, int n_tiles_n, int n_tiles) {
  constexpr int BK = 64;
  using C = GemmCfg<BM, BN, BK, WM, WN, GATEUP>;
  constexpr int NLD = C::A_PER + C::NB * C::B_PER;  // 16-byte loads per thread per stage
  // two arrays so the compiler can tell the stages apart (the stage index is
  // a compile-time constant in the unrolled loop)
  __shared__ __align__(16) bf16 lds0[C::STAGE_ELEMS];
  __shared__ __align__(16) bf16 lds1[C::STAGE_ELEMS];
  auto stage = [&](int b) -> bf16* { return b ? lds1 : lds0; };

  const int tile = xcd_tile(blockIdx.x, gridDim.x);
  if (tile >= n_tiles) return;
  const int mt = tile / n_tiles_n;
  const int ntile = tile % n_tiles_n;
  int e, row0, row_end;
  if (!find_tile(offsets, E, rows, BM, mt, e, row0, row_end)) return;
  const int n0 = ntile * BN;

  const int tid = threadIdx.x;
  const int lane = lane_id();
  const int wave = tid >> 6;
  const int wm = wave / WN, wn = wave % WN;

  // A: a per-tile buffer (rows row0.. of a permuted copy) or, when gathering,
  // the whole source with per-row offsets; weights: one buffer per slice
  const int n_valid = min(BN, N - n0);
  __amdgpu_buffer_rsrc_t rsrc[1 + C::NB];
  if (gather == nullptr)
    rsrc[0] = make_rsrc(A + (size_t)row0 * K, (uint32_t)min(BM, row_end - row0) * K * 2u);
  else
    rsrc[0] = make_rsrc(A, (uint32_t)a_rows * K * 2u);
  rsrc[1] = make_rsrc(B0 + ((size_t)e * N + n0) * K, (uint32_t)n_valid * K * 2u);
  if constexpr (GATEUP) rsrc[2] = make_rsrc(B1 + ((size_t)e * N + n0) * K, (uint32_t)n_valid * K * 2u);

  // chunk i of a stage: byte offset in the K-slab (kOob for rows that read
  // zeros), k of the chunk, LDS slot
  uint32_t g_off[NLD];
  int g_k[NLD], l_off[NLD];
#pragma unroll
  for (int i = 0; i < NLD; ++i) {
    const bool is_a = i < C::A_PER;
    const int j = is_a ? i : i - C::A_PER;
    const int c = tid + (is_a ? j : j % C::B_PER) * C::NTHR;
    const int r = c / C::CPR, kc = c % C::CPR;
    g_k[i] = kc * 8;
    if (is_a) {
      l_off[i] = r * C::LDK + kc * 8;
      if (gather == nullptr) {
        g_off[i] = (uint32_t)(r * K + kc * 8) * 2u;
      } else {
        const int s = (row0 + r < row_end) ? src_row(gather, kdiv, row0 + r, a_rows) : -1;
        g_off[i] = s < 0 ? kOob : ((uint32_t)s * K + kc * 8) * 2u;
      }
    } else {
      l_off[i] = C::A_ELEMS + (j / C::B_PER) * C::B_ELEMS + r * C::LDK + kc * 8;
      g_off[i] = (uint32_t)(r * K + kc * 8) * 2u;
    }
  }
  auto rsrc_of = [&](int i) {
    return i < C::A_PER ? rsrc[0] : rsrc[1 + (i - C::A_PER) / C::B_PER];
  };

  f32x16 acc[C::NB][C::SM][C::SN];
#pragma unroll
  for (int b = 0; b < C::NB; ++b)
#pragma unroll
    for (int i = 0; i < C::SM; ++i)
#pragma unroll
      for (int j = 0; j < C::SN; ++j)
#pragma unroll
        for (int v = 0; v < 16; ++v) acc[b][i][j][v] = 0.f;

  u32x4 stg[NSETS][NLD];
  auto gload = [&](int set, int k0) {
    const uint32_t kb = (uint32_t)k0 * 2u;
#pragma unroll
    for (int i = 0; i < NLD; ++i)
      stg[set][i] =
          buf_load16(rsrc_of(i), (k0 + g_k[i] < K && g_off[i] != kOob) ? g_off[i] + kb : kOob);
  };
  auto lstore = [&](int set, int buf) {
    bf16* sb = stage(buf);
#pragma unroll
    for (int i = 0; i < NLD; ++i) *reinterpret_cast<u32x4*>(sb + l_off[i]) = stg[set][i];
  };

  const int lrow = lane & 31;
  const int lk = (lane >> 5) * 8;
  const int xa_base = (wm * C::WTM + lrow) * C::LDK + lk;
  const int wf_base = C::A_ELEMS + (wn * C::WTN + lrow) * C::LDK + lk;
  bf16x8 xa[2][C::SM];
  bf16x8 wf[2][C::NB][C::SN];
  auto fload = [&](int buf, int ks, int slot) {
    const bf16* sa = stage(buf) + ks * 16;
#pragma unroll
    for (int i = 0; i < C::SM; ++i)
      xa[slot][i] = *reinterpret_cast<const bf16x8*>(sa + xa_base + i * 32 * C::LDK);
#pragma unroll
    for (int b = 0; b < C::NB; ++b)
#pragma unroll
      for (int j = 0; j < C::SN; ++j)
        wf[slot][b][j] =
            *reinterpret_cast<const bf16x8*>(sa + wf_base + b * C::B_ELEMS + j * 32 * C::LDK);
  };
  auto mfma = [&](int slot) {
#pragma unroll
    for (int b = 0; b < C::NB; ++b)
#pragma unroll
      for (int j = 0; j < C::SN; ++j)
#pragma unroll
        for (int i = 0; i < C::SM; ++i)
          acc[b][i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(wf[slot][b][j], xa[slot][i],
                                                                 acc[b][i][j], 0, 0, 0);
  };
  constexpr int NM = C::NB * C::SM * C::SN;  // MFMAs per k16 step
  constexpr int NR = C::SM + C::NB * C::SN;  // fragment reads per k16 step
  // at iteration kt the register set of stage kt+1 is written to LDS and then
  // refilled with stage kt+1+NSETS
  auto iteration = [&](int kt, int cur) {
    const int nxt = cur ^ 1;
    const int set = (kt + 1) % NSETS;
    fload(cur, 1, 1);
    mfma(0);
    lstore(set, nxt);
    interleave<0, NM, NR, NLD, kSchedDsWrite>();
    __builtin_amdgcn_sched_barrier(0);
    fload(cur, 2, 0);
    mfma(1);
    gload(set, (kt + 1 + NSETS) * BK);
    interleave<0, NM, NR, NLD, kSchedVmemRead>();
    __builtin_amdgcn_sched_barrier(0);
    fload(cur, 3, 1);
    mfma(0);
    interleave<0, NM, NR, 0, 0>();
    __builtin_amdgcn_sched_barrier(0);
    lds_barrier();
    fload(nxt, 0, 0);
    mfma(1);
    interleave<0, NM, NR, 0, 0>();
    __builtin_amdgcn_sched_barrier(0);
  };

  // K steps rounded up to an even count: steps past K read zeros
  const int nk = ((K + BK - 1) / BK + 1) & ~1;
#pragma unroll
  for (int st = 0; st < NSETS; ++st) gload(st, st * BK);
  lstore(0, 0);
  gload(0, NSETS * BK);
  lds_barrier();
  fload(0, 0, 0);
  for (int kt = 0; kt < nk; kt += 2) {
    iteration(kt, 0);
    iteration(kt + 1, 1);
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

// Few rows per expert (decode): the FFN is a weight stream.  A workgroup owns
// one expert and a slice of weight rows (16 gate + 16 up rows, or 32 down
// rows); its KW waves split K and read the weights with 128-bit buffer loads
// straight into the operands of v_mfma_f32_16x16x32_bf16 (D = W * A^T, 16
// weight rows x 16 rows of A per MFMA), so there is no LDS staging and each
// wave has U K chunks of loads in flight.  The KW partial tiles are summed in
// LDS in wave order.  Experts with more than 32 rows take several passes.
template <bool GATEUP, int KW, int U>
__global__ __launch_bounds__(KW * 64) void ffn_skinny_bf16(
    const bf16* __restrict__ A, const int32_t* __restrict__ gather, int kdiv, int a_rows,
    const int32_t* __restrict__ offsets, int E, int rows, const bf16* __restrict__ W0,
    const bf16* __restrict__ W1, int N, int K, bf16* __restrict__ out, int n_groups) {
  constexpr int NPB = GATEUP ? 16 : 32;  // output columns per workgroup
  __shared__ __align__(16) f32x4 red[KW][2][2][kWave];

  const int e = blockIdx.x / n_groups;
  const int n0 = (blockIdx.x % n_groups) * NPB;
  const int a = min(max(offsets[e], 0), rows);
  const int b = max(min(max(offsets[e + 1], 0), rows), a);
  if (b == a || e >= E) return;
  const int lane = lane_id();
  const int wave = threadIdx.x >> 6;
  const int r16 = lane & 15;
  const uint32_t kq = (uint32_t)(lane >> 4) * 8u;

  // weight tiles: tile 0 / tile 1 = gate / up rows n0.. (GATEUP) or rows n0.., n0+16..
  const int nv = min(NPB, N - n0);
  const __amdgpu_buffer_rsrc_t wr0 =
      make_rsrc(W0 + ((size_t)e * N + n0) * K, (uint32_t)nv * K * 2u);
  const __amdgpu_buffer_rsrc_t wr1 =
      GATEUP ? make_rsrc(W1 + ((size_t)e * N + n0) * K, (uint32_t)nv * K * 2u) : wr0;
  const uint32_t w_off0 = (uint32_t)r16 * K * 2u + kq * 2u;
  const uint32_t w_off1 = GATEUP ? w_off0 : (uint32_t)(r16 + 16) * K * 2u + kq * 2u;
  const __amdgpu_buffer_rsrc_t ar = make_rsrc(A, (uint32_t)a_rows * K * 2u);
  const int nchunks = (K + 31) / 32;

  for (int t0 = a; t0 < b; t0 += 32) {
    const int tv = min(32, b - t0);
    uint32_t a_off[2];
#pragma unroll
    for (int j = 0; j < 2; ++j) {
      const int t = j * 16 + r16;
      const int s = t < tv ? src_row(gather, kdiv, t0 + t, a_rows) : -1;
      a_off[j] = s < 0 ? kOob : (uint32_t)s * K * 2u + kq * 2u;
    }
    f32x4 acc[2][2];
#pragma unroll
    for (int i = 0; i < 2; ++i)
#pragma unroll
      for (int j = 0; j < 2; ++j) acc[i][j] = f32x4{0.f, 0.f, 0.f, 0.f};
    for (int c0 = wave * U; c0 < nchunks; c0 += KW * U) {
      u32x4 wa[U][2], xb[U][2];
#pragma unroll
      for (int u = 0; u < U; ++u) {
        const int c = c0 + u;
        const bool ok = c < nchunks && (uint32_t)c * 32u + kq < (uint32_t)K;
        const uint32_t kb = (uint32_t)c * 64u;
        wa[u][0] = buf_load16_stream(wr0, ok ? w_off0 + kb : kOob);
        wa[u][1] = buf_load16_stream(wr1, ok ? w_off1 + kb : kOob);
        xb[u][0] = buf_load16(ar, (ok && a_off[0] != kOob) ? a_off[0] + kb : kOob);
        xb[u][1] = buf_load16(ar, (ok && a_off[1] != kOob) ? a_off[1] + kb : kOob);
      }
#pragma unroll
      for (int u = 0; u < U; ++u)
#pragma unroll
        for (int i = 0; i < 2; ++i)
#pragma unroll
          for (int j = 0; j < 2; ++j)
            acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(
                __builtin_bit_cast(bf16x8, wa[u][i]), __builtin_bit_cast(bf16x8, xb[u][j]),
                acc[i][j], 0, 0, 0);
    }
#pragma unroll
    for (int i = 0; i < 2; ++i)
#pragma unroll
      for (int j = 0; j < 2; ++j) red[wave][i][j][lane] = acc[i][j];
    __syncthreads();
    if (wave == 0) {
#pragma unroll
      for (int i = 0; i < 2; ++i)
#pragma unroll
        for (int j = 0; j < 2; ++j) {
          f32x4 s4 = red[0][i][j][lane];
#pragma unroll
          for (int w = 1; w < KW; ++w) s4 += red[w][i][j][lane];
          acc[i][j] = s4;
        }
      // lane holds row j*16 + lane%16 of A and weight rows 4*(lane/16) + [0,4)
      const int nb = 4 * (lane >> 4);
#pragma unroll
      for (int j = 0; j < 2; ++j) {
        const int t = j * 16 + r16;
        if (t >= tv) continue;
        bf16* orow = out + (size_t)(t0 + t) * N + n0;
        if constexpr (GATEUP) {
          if (nb < nv) {
            bf16x4 o;
#pragma unroll
            for (int v = 0; v < 4; ++v) o[v] = (bf16)(silu_f(acc[0][j][v]) * acc[1][j][v]);
            *reinterpret_cast<bf16x4*>(orow + nb) = o;
          }
        } else {
#pragma unroll
          for (int i = 0; i < 2; ++i) {
            if (i * 16 + nb >= nv) continue;
            bf16x4 o;
#pragma unroll
            for (int v = 0; v < 4; ++v) o[v] = (bf16)acc[i][j][v];
            *reinterpret_cast<bf16x4*>(orow + i * 16 + nb) = o;
          }
        }
      }
    }
    __syncthreads();
  }
}

constexpr int kSkinnyWaves = FirstOf<FOE_SKINNY>::value;

// ---- fp32 path: plain FMA kernels (small shapes) ---------------------------
__device__ int expert_of_row(const int32_t* __restrict__ offsets, int E, int rows, int row) {
  for (int e = 0; e < E; ++e) {
    int a = min(max(offsets[e], 0), rows);
    int b = min(max(offsets[e + 1], 0), rows);
    if (row >= a && row < b) return e;
  }
  return -1;
}

__global__ __launch_bounds__(256) void gateup_f32(const float* __restrict__ A,
                                                  const int32_t* __restrict__ gather, int kdiv,
                                                  int a_rows, const int32_t* __restrict__ offsets,
                                                  int E, int rows, const float* __restrict__ wg,
                                                  const float* __restrict__ wu, int F, int d,
                                                  float* __restrict__ h) {
  const long long id = (long long)blockIdx.x * blockDim.x + threadIdx.x;
  if (id >= (long long)rows * F) return;
  const int row = (int)(id / F), n = (int)(id % F);
  const int e = expert_of_row(offsets, E, rows, row);
  if (e < 0) return;
  const int s = src_row(gather, kdiv, row, a_rows);
  const float* g = wg + ((size_t)e * F + n) * d;
  const float* u = wu + ((size_t)e * F + n) * d;
  float ag = 0.f, au = 0.f;
  if (s >= 0) {
    const float* xr = A + (size_t)s * d;
    for (int i = 0; i < d; ++i) {
      ag = fmaf(xr[i], g[i], ag);
      au = fmaf(xr[i], u[i], au);
    }
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

template <int BM, int BN, int WM, int WN, bool GATEUP, int NSETS, int MAXW>
void launch_gemm(const bf16* A, const int32_t* gather, int kdiv, int a_rows,
                 const int32_t* offsets, int E, int rows, const bf16* B0, const bf16* B1, int N,
                 int K, bf16* out, hipStream_t s, const char* name) {
  const int ntn = ceil_div(N, BN);
  const int max_mt = ceil_div(rows, BM) + E;  // sum_e ceil(M_e/BM) <= rows/BM + E
  const long long n_tiles = (long long)max_mt * ntn;
  dim3 grid((unsigned)((n_tiles + 7) / 8 * 8));
  ProfileScope ps(name, s);
  hipLaunchKernelGGL((grouped_gemm_bf16<BM, BN, WM, WN, GATEUP, NSETS, MAXW>), grid,
                     dim3(WM * WN * kWave), 0, s, A, gather, kdiv, a_rows, offsets, E, rows, B0,
                     B1, N, K, out, ntn, (int)n_tiles);
}

}  // namespace

size_t ffn_scratch_bytes(foe_dtype dt, int rows, int F) {
  return align_up((size_t)rows * F * (dt == FOE_BF16 ? 2 : 4), 256);
}

hipError_t launch_expert_ffn_ex(foe_dtype dt, int E, int d, int F, int rows, const void* A,
                                const int32_t* gather, int kdiv, int a_rows,
                                const int32_t* offsets, const void* w_gate, const void* w_up,
                                const void* w_down, void* y_perm, void* scratch, hipStream_t s) {
  if (rows == 0) return hipSuccess;
  if (dt == FOE_F32) {
    float* h = reinterpret_cast<float*>(scratch);
    {
      ProfileScope ps("ffn_gateup_f32", s);
      hipLaunchKernelGGL(gateup_f32, dim3(ceil_div((long long)rows * F, 256)), dim3(256), 0, s,
                         reinterpret_cast<const float*>(A), gather, kdiv, a_rows, offsets, E,
                         rows, reinterpret_cast<const float*>(w_gate),
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
  const bf16* xa = reinterpret_cast<const bf16*>(A);
  const bf16* wg = reinterpret_cast<const bf16*>(w_gate);
  const bf16* wu = reinterpret_cast<const bf16*>(w_up);
  const bf16* wd = reinterpret_cast<const bf16*>(w_down);
  bf16* h = reinterpret_cast<bf16*>(scratch);
  bf16* y = reinterpret_cast<bf16*>(y_perm);
  if (rows < 64 * E) {  // few rows per expert: weight-streaming bound
    {
      const int ng = ceil_div(F, 16);
      ProfileScope ps("ffn_gateup", s);
      hipLaunchKernelGGL((ffn_skinny_bf16<true, FOE_SKINNY>), dim3(E * ng),
                         dim3(kSkinnyWaves * kWave), 0, s, xa, gather, kdiv, a_rows, offsets, E,
                         rows, wg, wu, F, d, h, ng);
    }
    {
      const int ng = ceil_div(d, 32);
      ProfileScope ps("ffn_down", s);
      hipLaunchKernelGGL((ffn_skinny_bf16<false, FOE_SKINNY>), dim3(E * ng),
                         dim3(kSkinnyWaves * kWave), 0, s, h, nullptr, 1, rows, offsets, E, rows,
                         wd, nullptr, d, F, y, ng);
    }
  } else {
    launch_gemm<FOE_PIPE_GU, true, FOE_PIPE_OPT>(xa, gather, kdiv, a_rows, offsets, E, rows, wg,
                                                 wu, F, d, h, s, "ffn_gateup");
    launch_gemm<FOE_PIPE_DN, false, FOE_PIPE_OPT>(h, nullptr, 1, rows, offsets, E, rows, wd,
                                                  nullptr, d, F, y, s, "ffn_down");
  }
  return hipGetLastError();
}

hipError_t launch_expert_ffn(foe_dtype dt, int E, int d, int F, int rows, const void* x_perm,
                             const int32_t* offsets, const void* w_gate, const void* w_up,
                             const void* w_down, void* y_perm, void* scratch, hipStream_t s) {
  return launch_expert_ffn_ex(dt, E, d, F, rows, x_perm, nullptr, 1, rows, offsets, w_gate, w_up,
                              w_down, y_perm, scratch, s);
}

}  // namespace foe
