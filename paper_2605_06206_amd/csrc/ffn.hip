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
// ffn_stream_bf16.  fp32: plain FMA kernels (small shapes only).
#include <type_traits>

#include "lds_dma.hpp"

// LDS-DMA large-M kernel: (BM, BN, WM, WN, BK, LDS stages, waves that issue
// the DMA (0 = all), M-tile group of the tile order, persistent)
#ifndef FOE_DMA_GU
#define FOE_DMA_GU 256, 128, 2, 4, 64, 2, 4, 4, 1
#endif
#ifndef FOE_DMA_DN
#define FOE_DMA_DN 256, 256, 2, 4, 64, 2, 4, 4, 1
#endif
// plain grouped GEMM over a few wide segments (the q/k/v projection of the
// attention groups): as the down projection, tiles walked XCD by XCD
#ifndef FOE_DMA_SEG
#define FOE_DMA_SEG 256, 256, 2, 4, 64, 2, 4, 4, 2
#endif
// plain GEMM with the residual epilogue (few M rows: 128 x 256 tiles, or
// 128 x 128 when the larger tiles would leave compute units idle); one tile
// per CU walks all of K, so a third LDS stage keeps more loads in flight
#ifndef FOE_DMA_RES
#define FOE_DMA_RES 128, 256, 2, 4, 64, 3, 3, 4, 1
#endif
#ifndef FOE_DMA_RES_SMALL
#define FOE_DMA_RES_SMALL 128, 128, 2, 4, 64, 3, 4, 4, 1
#endif
// few rows per expert (decode): LDS-staged weight stream with NS stages, K
// walk rotated per workgroup, and (block decode form) pair lists built in the
// kernel
#ifndef FOE_FFN_SEL
#define FOE_FFN_SEL 1
#endif
#ifndef FOE_STREAM_ROT
#define FOE_STREAM_ROT 1
#endif
#ifndef FOE_STREAM_NS
#define FOE_STREAM_NS 3
#endif

namespace foe {
namespace {

// Most (token, slot) pairs per cluster for which the decode FFN builds each
// expert's pair list itself from the routing decisions.
constexpr int kSelMax = 2048;
constexpr int kScDevice = 16;  // buffer cache policy SC1: device-scope coherence
typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));

// Number of M-tiles of BM rows over all experts (segments clamped as in
// find_tile); every lane of the wave gets the total.
// Start of segment e: offsets[e] clamped to [0, rows], or e * (rows / E) when
// offsets is null (E segments of equal length, rows a multiple of E).
__device__ __forceinline__ int seg_start(const int32_t* __restrict__ offsets, int e, int E,
                                         int rows) {
  return offsets == nullptr ? e * (rows / E) : min(max(offsets[e], 0), rows);
}

__device__ int total_mtiles(const int32_t* __restrict__ offsets, int E, int rows, int BM) {
  const int lane = lane_id();
  int mine = 0;
  for (int e = lane; e < E; e += kWave) {
    const int a = seg_start(offsets, e, E, rows);
    const int b = seg_start(offsets, e + 1, E, rows);
    mine += b > a ? (b - a + BM - 1) / BM : 0;
  }
#pragma unroll
  for (int off = kWave / 2; off > 0; off >>= 1) mine += __shfl_xor(mine, off);
  return mine;
}

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
    a = seg_start(offsets, e, E, rows);
    b = seg_start(offsets, e + 1, E, rows);
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

// M-tile table of the fused FFN, held in LDS: entry i (expert, first row,
// row end) is the i-th M-tile of the launch's tile order.  Experts are taken
// in ascending order of their row counts (equal counts: lower id first), each
// expert's tiles in row order.  The least-loaded experts' tiles -- mostly
// partly filled, and reading weight slices that no other M-tile shares, so
// slower than full tiles -- then run first and their down tiles early, and the
// schedule ends on full tiles of the most-loaded experts (in a list-scheduling
// model fitted to measured tile times this is 7% shorter at the Zipf-skewed
// prefill load than id order, and the same for uniform loads).
// kTabMaxE experts at most (their scratch fits the stage buffers), kTileTab
// entries.
constexpr int kTileTab = 2048;
constexpr int kTabMaxE = 1024;

// Builds the table with every thread of the workgroup; `aux` is LDS scratch of
// 4 * kTabMaxE + 1 ints.  Returns the number of M-tiles (the same in every
// thread); the table is complete only if that is at most kTileTab and
// E <= kTabMaxE (otherwise nothing is written and -1 is returned).
template <int NTHR>
__device__ int build_tile_table(const int32_t* __restrict__ offsets, int E, int rows, int BM,
                                int* aux, int* tab) {
  if (E > kTabMaxE) return -1;
  int* cnt = aux;                  // rows of expert e
  int* seg = aux + kTabMaxE;       // first row of expert e
  int* pos = aux + 2 * kTabMaxE;   // expert at position p of the order
  int* first = aux + 3 * kTabMaxE; // first M-tile of position p (E + 1 entries)
  const int tid = threadIdx.x;
  for (int e = tid; e < E; e += NTHR) {
    const int a = seg_start(offsets, e, E, rows);
    const int b = max(seg_start(offsets, e + 1, E, rows), a);
    cnt[e] = b - a;
    seg[e] = a;
  }
  __syncthreads();
  for (int e = tid; e < E; e += NTHR) {
    const int c = cnt[e];
    int r = 0;
    for (int f = 0; f < E; ++f) {
      const int cf = cnt[f];
      r += (cf < c || (cf == c && f < e)) ? 1 : 0;
    }
    pos[r] = e;
  }
  __syncthreads();
  if (tid < kWave) {
    // wave prefix sum of the M-tiles over the positions (contiguous ranges
    // of `per` positions per lane)
    const int per = (E + kWave - 1) / kWave;
    const int p0 = min(tid * per, E), p1 = min(p0 + per, E);
    int mine = 0;
    for (int p = p0; p < p1; ++p) mine += (cnt[pos[p]] + BM - 1) / BM;
    int incl = mine;
#pragma unroll
    for (int off = 1; off < kWave; off <<= 1) {
      const int v = __shfl_up(incl, off);
      if (tid >= off) incl += v;
    }
    int run = incl - mine;
    for (int p = p0; p < p1; ++p) {
      first[p] = run;
      run += (cnt[pos[p]] + BM - 1) / BM;
    }
    if (tid == kWave - 1) first[E] = incl;
  }
  __syncthreads();
  const int m_tiles = first[E];
  if (m_tiles > kTileTab) return m_tiles;
  for (int mt = tid; mt < m_tiles; mt += NTHR) {
    // last position p with first[p] <= mt (positions of empty experts share
    // their successor's first tile, so the last such p is the non-empty one)
    int lo = 0, hi = E - 1;
    while (lo < hi) {
      const int mid = (lo + hi + 1) >> 1;
      if (first[mid] <= mt) lo = mid;
      else hi = mid - 1;
    }
    const int e = pos[lo];
    tab[3 * mt] = e;
    tab[3 * mt + 1] = seg[e] + (mt - first[lo]) * BM;
    tab[3 * mt + 2] = seg[e] + cnt[e];
  }
  __syncthreads();
  return m_tiles;
}

// silu(g) = g * sigmoid(g) with the hardware reciprocal (v_rcp_f32, about one
// ulp) instead of an IEEE division (a ten-instruction sequence); the product
// is rounded to bf16 afterwards, so the two differ far below that rounding.
// g -> -inf: exp overflows to inf and the reciprocal to 0, as the division.
__device__ __forceinline__ float silu_f(float g) {
  return g * __builtin_amdgcn_rcpf(1.0f + __expf(-g));
}


// Calls f(integral_constant<int, I>) for I = B .. N-1 (compile-time indices).
template <int B, int N, typename F>
__device__ __forceinline__ void static_for(F&& f) {
  if constexpr (B < N) {
    f(std::integral_constant<int, B>{});
    static_for<B + 1, N>(f);
  }
}

// Source row of operand row r: r itself, or gather[r] / kdiv (-1 if that row
// is outside [0, src_rows)).
__device__ __forceinline__ int src_row(const int32_t* __restrict__ gather, int kdiv, int r,
                                       int src_rows) {
  if (gather == nullptr) return r;
  const int g = gather[r];
  const int s = g >= 0 ? g / kdiv : -1;
  return s < src_rows ? s : -1;
}

// ---- LDS-DMA variant of the large-M grouped GEMM ---------------------------
// Operand tiles go from global memory straight into LDS with
// `buffer_load_dwordx4 ... lds`: each lane of a wave deposits 16 bytes at
// M0 + 16 * lane, so one instruction fills 1 KiB of LDS and the tile never
// passes through VGPRs (no ds_write, no staging registers).  The loads are
// issued from inline assembly so that their completion is tracked here with
// explicit vmcnt waits (the compiler does not see them; the kernel issues no
// other global loads inside the main loop and uses M0 nowhere else).
//
// LDS layout of a tile: rows of BK bf16 (no padding), the 16-byte chunk c of
// row r stored in slot c ^ swz(r).  A fragment read (32 rows, one chunk) then
// touches every bank group once per 16 lanes.  Since a DMA instruction
// writes 1 KiB contiguously, the swizzle is applied on the load side: the
// lane that lands in slot s of row r fetches chunk s ^ swz(r).

template <int BM, int BN, int WM, int WN, bool GATEUP, int BK, int NST, int PW>
struct DmaCfg {
  static constexpr int NW = WM * WN, NTHR = NW * kWave;
  static constexpr int NP = PW > 0 ? PW : NW;  // waves that issue the DMA
  static constexpr int WTM = BM / WM, WTN = BN / WN;
  static constexpr int SM = WTM / 32, SN = WTN / 32;
  static constexpr int NB = GATEUP ? 2 : 1;
  static constexpr int RB = BK * 2;        // bytes per tile row
  static constexpr int CPR = BK / 8;       // 16-byte chunks per row
  static constexpr int RPI = 1024 / RB;    // rows per DMA instruction
  static constexpr int A_INS = BM / RPI, B_INS = BN / RPI;  // DMA instructions per tile
  static constexpr int NLD = (A_INS + NB * B_INS) / NP;      // per issuing wave
  // the swizzle of a row depends on row & 15, so on instruction ii through
  // ii & (NVAR - 1)
  static constexpr int NVAR = RPI >= 16 ? 1 : 16 / RPI;
  static constexpr int A_BYTES = BM * RB, B_BYTES = BN * RB;
  static constexpr int STAGE = A_BYTES + NB * B_BYTES;
  static constexpr int KS = BK / 16;       // k16 steps per stage
  static_assert(WTM % 32 == 0 && WTN % 32 == 0, "wave tile must be a multiple of 32");
  static_assert(BM % RPI == 0 && BN % RPI == 0 && (A_INS + NB * B_INS) % NP == 0 && NP <= NW,
                "even DMA split");
  // with several issuing waves, the instructions of one wave stay inside one
  // tile and start at a multiple of NVAR (a single issuing wave maps every
  // instruction to its tile at compile time)
  static_assert(NP == 1 || (A_INS % NLD == 0 && B_INS % NLD == 0 && NLD % NVAR == 0),
                "one tile per issuing wave");
  static_assert(KS % 2 == 0, "fragment slots alternate within a stage");
  static_assert(NST >= 2 && NLD * (NST - 2) <= 63, "vmcnt range");
  static_assert(NST * STAGE <= 160 * 1024, "LDS capacity");
};

// Stage kt (K columns kt*BK ..) lives in LDS buffer kt % NST.  Iteration kt:
//   issue the DMA of stage kt+NST-1 into the buffer freed by stage kt-1;
//   k16 steps 0..KS-2 of stage kt (fragment reads one step ahead);
//   wait for stage kt+1 and meet the other waves;
//   read the first fragments of stage kt+1; k16 step KS-1 of stage kt.
// Only the first PW waves (one per SIMD when PW = 4) issue DMA instructions.
// The address unit of a CU takes a stage's instructions at a fixed rate, and
// a wave whose instruction finds its queue full stops issuing; when every
// wave loads, both waves of a SIMD stall together and its MFMA pipe idles.
// With producer waves, the other wave of each SIMD keeps issuing MFMAs.
// Residual epilogue of the plain (non gate/up) form: the output becomes
// scale * (acc + x), x an fp32 matrix of the output's shape.
struct GemmResid {
  const float* x = nullptr;
  float scale = 1.f;
};

// Operands of one grouped GEMM: A rows (direct, or gathered as gather[r] /
// kdiv from a_rows source rows), one or two [E, N, K] weight stacks, the
// output [rows, N] (out_bytes = its size, for device-scope stores) and the
// residual epilogue.
struct GemmArgs {
  const bf16* A;
  const int32_t* gather;
  int kdiv;
  int a_rows;
  const bf16* B0;
  const bf16* B1;
  int N;
  int K;
  bf16* out;
  uint32_t out_bytes;
  GemmResid res;
  // two-matrix tile shape (GATEUP) used for a plain product: B1 is ignored,
  // and the tile's two BN-row weight slices are rows ntile*2*BN .. +BN and
  // .. +2*BN of B0, stored side by side (no SwiGLU); the tile covers 2*BN
  // output columns
  bool halves;
};

// One BM x BN output tile of expert e (rows row0 .. row_end-1, N-tile ntile)
// over all of K, staged through the workgroup's LDS `smem`.  OUT_CPOL = 0
// stores the output tile through the caches as usual; otherwise the stores
// carry that cache policy (kScDevice: written through past the XCD's L2, so
// that other XCDs can read the tile once the stores have completed).  The
// two-slice form (GemmArgs::halves) always stores as usual, staged through LDS.
template <int BM, int BN, int WM, int WN, bool GATEUP, int BK, int NST, int PW, bool RESID,
          int OUT_CPOL>
__device__ __forceinline__ void gemm_tile(unsigned char* smem, const GemmArgs& g, const int e,
                                          const int row0, const int row_end, const int ntile,
                                          int32_t* signal = nullptr) {
  static_assert(!(RESID && GATEUP), "residual epilogue on the plain form only");
  using C = DmaCfg<BM, BN, WM, WN, GATEUP, BK, NST, PW>;
  constexpr int NLD = C::NLD;
  const bf16* __restrict__ A = g.A;
  const int32_t* __restrict__ gather = g.gather;
  const int kdiv = g.kdiv, a_rows = g.a_rows, N = g.N, K = g.K;
  const bf16* __restrict__ B0 = g.B0;
  const bf16* __restrict__ B1 = g.B1;
  bf16* __restrict__ out = g.out;
  const GemmResid& res = g.res;

  const int tid = threadIdx.x;
  const int lane = lane_id();
  const int wave = tid >> 6;
  const int wm = wave / WN, wn = wave % WN;
  const int wave_u = __builtin_amdgcn_readfirstlane(wave);
  {
    const int n0 = ntile * BN;

    const int n_valid = min(BN, N - n0);
    // operand ranges: A rows (a per-tile range, or the whole source when
    // gathering), then one weight slice per matrix
    const bf16* t_base[1 + C::NB];
    uint32_t t_bytes[1 + C::NB];
    t_base[0] = gather == nullptr ? A + (size_t)row0 * K : A;
    t_bytes[0] = gather == nullptr ? (uint32_t)min(BM, row_end - row0) * K * 2u
                                   : (uint32_t)a_rows * K * 2u;
    t_base[1] = B0 + ((size_t)e * N + n0) * K;
    t_bytes[1] = (uint32_t)n_valid * K * 2u;
    if constexpr (GATEUP) {
      t_base[2] = B1 + ((size_t)e * N + n0) * K;
      t_bytes[2] = t_bytes[1];
      if (g.halves) {
        // the two slices of a 2*BN-column tile of B0 (a slice past N is empty)
        const int h0 = ntile * 2 * BN, h1 = min(h0 + BN, N);
        t_base[1] = B0 + ((size_t)e * N + h0) * K;
        t_bytes[1] = (uint32_t)max(min(BN, N - h0), 0) * K * 2u;
        t_base[2] = B0 + ((size_t)e * N + h1) * K;
        t_bytes[2] = (uint32_t)max(min(BN, N - h1), 0) * K * 2u;
      }
    }

    // DMA instruction gq of a stage covers RPI rows (1 KiB) of the A tile
    // (gq < A_INS) or of a weight tile.  Lane l lands in row rl = l/CPR, slot
    // l%CPR of the instruction's rows and so fetches chunk (l%CPR) ^ swz(row);
    // the swizzle depends on the instruction only through its variant
    // ii & (NVAR-1), so each lane keeps NVAR chunk choices.  Gathered A rows
    // keep one source offset per A instruction.
    const int rl = lane / C::CPR, cl = lane % C::CPR;
    int chunk[C::NVAR];
    uint32_t lane_off[C::NVAR];
#pragma unroll
    for (int v = 0; v < C::NVAR; ++v) {
      chunk[v] = cl ^ swz<C::CPR>(v * C::RPI + rl);
      lane_off[v] = ((uint32_t)rl * K + chunk[v] * 8) * 2u;
    }
    constexpr int NV = C::NVAR;
    const uint32_t row_step = (uint32_t)C::RPI * K * 2u;  // bytes between instructions
    auto a_src = [&](int ii) {  // gathered source offset of A instruction ii
      const int r = ii * C::RPI + rl;
      const int s = (row0 + r < row_end) ? src_row(gather, kdiv, row0 + r, a_rows) : -1;
      return s < 0 ? kOob : ((uint32_t)s * K + chunk[ii & (NV - 1)] * 8) * 2u;
    };
    const uint32_t smem_base = lds_addr(smem);

    // Several issuing waves: wave p loads instructions p*NLD .. p*NLD+NLD-1,
    // all inside tile tw starting at its instruction ii0.
    // Share p goes to wave (p + 4) mod NP.  With eight issuing waves, waves
    // 0..3 (the older wave of each SIMD) take the weight shares and waves
    // 4..7 the A rows (measured 1% faster at the prefill load than the other
    // way round, the same elsewhere; results identical).  With four issuing
    // waves this is the identity; with three (the residual GEMM) each share
    // moves to the next wave.
#ifndef FOE_DMA_ROT
#define FOE_DMA_ROT 4
#endif
    const int p = C::NP > 1 ? (min(wave_u, C::NP - 1) + FOE_DMA_ROT) % C::NP : 0;
    const int tw = p * NLD < C::A_INS ? 0 : 1 + (p * NLD - C::A_INS) / C::B_INS;
    const int ii0 = tw == 0 ? p * NLD : (p * NLD - C::A_INS) % C::B_INS;
    const __amdgpu_buffer_rsrc_t rsrc_w =
        make_rsrc_u(tw == 0 ? t_base[0] : (tw == 1 ? t_base[1] : t_base[C::NB]),
                    tw == 0 ? t_bytes[0] : (tw == 1 ? t_bytes[1] : t_bytes[C::NB]));
    const uint32_t lds_w = (tw == 0 ? 0 : C::A_BYTES + (tw - 1) * C::B_BYTES) + ii0 * 1024;
    const bool gather_a = tw == 0 && gather != nullptr;
    // source byte offset of this lane's chunk in instruction q (K slab 0)
    uint32_t off_q[C::NP > 1 ? NLD : 1];
    if constexpr (C::NP > 1) {
#pragma unroll
      for (int q = 0; q < NLD; ++q)
        off_q[q] = gather_a ? a_src(ii0 + q)
                            : (uint32_t)(ii0 + q) * row_step + lane_off[q & (NV - 1)];
    }
    // A single issuing wave: instruction q is fixed at compile time.
    __amdgpu_buffer_rsrc_t rsrc_t[1 + C::NB];
    uint32_t a_off[C::NP == 1 ? C::A_INS : 1];
    if constexpr (C::NP == 1) {
#pragma unroll
      for (int t = 0; t <= C::NB; ++t) rsrc_t[t] = make_rsrc_u(t_base[t], t_bytes[t]);
#pragma unroll
      for (int ii = 0; ii < C::A_INS; ++ii)
        a_off[ii] = gather != nullptr ? a_src(ii) : (uint32_t)ii * row_step + lane_off[ii & (NV - 1)];
    }

    // DMA instruction q (of this issuing wave) of stage kt into LDS buffer
    // buf; stages past K read zeros
    const uint32_t lds_base = smem_base + lds_w;
    auto issue_one = [&](int kt, int buf, int q) {
      const int k0 = kt * BK;
      if constexpr (C::NP == 1) {
        const int tb = q < C::A_INS ? 0 : 1 + (q - C::A_INS) / C::B_INS;
        const int ii = q < C::A_INS ? q : (q - C::A_INS) % C::B_INS;
        const uint32_t off =
            tb == 0 ? a_off[ii] : (uint32_t)ii * row_step + lane_off[ii & (NV - 1)];
        const bool ok = k0 + chunk[ii & (NV - 1)] * 8 < K && off != kOob;
        dma16(rsrc_t[tb], ok ? off + (uint32_t)k0 * 2u : kOob, smem_base,
              buf * C::STAGE + (tb == 0 ? 0 : C::A_BYTES + (tb - 1) * C::B_BYTES) + ii * 1024);
      } else {
        const bool ok = k0 + chunk[q & (NV - 1)] * 8 < K && off_q[q] != kOob;
        dma16(rsrc_w, ok ? off_q[q] + (uint32_t)k0 * 2u : kOob, lds_base,
              buf * C::STAGE + q * 1024);
      }
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

    // fragment rows are congruent to lane%32 modulo 32, so one swizzle per lane
    const int lrow = lane & 31;
    const int sw = swz<C::CPR>(lrow) ^ (lane >> 5);
    int xo[C::KS];
#pragma unroll
    for (int ks = 0; ks < C::KS; ++ks) xo[ks] = ((2 * ks) ^ sw) * 16;
    const int a_row = (wm * C::WTM + lrow) * C::RB;
    const int b_row = C::A_BYTES + (wn * C::WTN + lrow) * C::RB;
    bf16x8 xa[2][C::SM];
    bf16x8 wf[2][C::NB][C::SN];
    auto fload = [&](int buf, int ks, int slot) {
      const unsigned char* sa = smem + buf * C::STAGE;
#pragma unroll
      for (int i = 0; i < C::SM; ++i)
        xa[slot][i] = *reinterpret_cast<const bf16x8*>(sa + a_row + xo[ks] + i * 32 * C::RB);
#pragma unroll
      for (int b = 0; b < C::NB; ++b)
#pragma unroll
        for (int j = 0; j < C::SN; ++j)
          wf[slot][b][j] = *reinterpret_cast<const bf16x8*>(sa + b_row + xo[ks] + b * C::B_BYTES +
                                                            j * 32 * C::RB);
    };
    constexpr int NM = C::NB * C::SM * C::SN;  // MFMAs per k16 step
    constexpr int NR = C::SM + C::NB * C::SN;  // fragment reads per k16 step
    constexpr int NT = NM > NR ? NM : NR;  // slots of a k16 step
    // Valid 32-row sub-tiles of this wave's WTM rows: a partly filled tile
    // (an expert's last rows) skips the MFMAs and A fragment reads of the
    // sub-tiles past row_end (a variant of the loop; full tiles run without
    // the checks).
    const int smv = min(max((row_end - row0 - wm * C::WTM + 31) / 32, 0), C::SM);
    const bool partial_tile = __builtin_amdgcn_readfirstlane(row_end - row0) < BM;
    // One k16 step in a fixed order: (in an issuing wave) the DMA
    // instructions [q0, q1) of stage dkt (buffer dbuf) spread evenly over the
    // MFMAs, each ahead of its MFMA so that it does not queue behind it for the
    // SIMD's matrix pipe (measured 1-2% faster than after it), then MFMA t of
    // fragment slot `slot`, then fragment read t of (rbuf, rks) into the other
    // slot (rks >= 0).  mode: bit 0 issuing wave, bit 1 partly filled tile.
    auto kstep = [&](auto mode, int slot, int rbuf, int rks, int dkt, int dbuf, int q0,
                     int q1) {
      constexpr bool producer = decltype(mode)::value & 1, part = decltype(mode)::value & 2;
      const unsigned char* sa = smem + rbuf * C::STAGE;
#pragma unroll
      for (int t = 0; t < NT; ++t) {
        if constexpr (producer) {
#pragma unroll
          for (int q = q0; q < q1; ++q)
            if ((q - q0) * NT / (q1 - q0) == t) issue_one(dkt, dbuf, q);
        }
        if (t < NM) {
          const int b = t / (C::SN * C::SM), j = (t / C::SM) % C::SN, i = t % C::SM;
          if (!part || i < smv)
            acc[b][i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(wf[slot][b][j], xa[slot][i],
                                                                   acc[b][i][j], 0, 0, 0);
        }
        if (rks >= 0 && t < NR) {
          if (t < C::SM) {
            if (!part || t < smv)
              xa[slot ^ 1][t] =
                  *reinterpret_cast<const bf16x8*>(sa + a_row + xo[rks] + t * 32 * C::RB);
          } else {
            const int u = t - C::SM, ub = u / C::SN, uj = u % C::SN;
            wf[slot ^ 1][ub][uj] = *reinterpret_cast<const bf16x8*>(
                sa + b_row + xo[rks] + ub * C::B_BYTES + uj * 32 * C::RB);
          }
        }
        __builtin_amdgcn_sched_barrier(0);
      }
    };

    // K steps rounded up to a multiple of NST: steps past K read zeros.
    // The DMA of stage kt+NST-1 is spread over the k16 steps of iteration kt:
    // with more than two stages it may use every step.  With two stages it
    // must be complete at this iteration's barrier, and (EARLY) its first QE
    // instructions already go out in the last k16 step of iteration kt-1:
    // that step follows the barrier after which no wave reads the buffer of
    // stage kt-1 any more, so the loads of a stage start one k16 step sooner
    // and have about half as long again to arrive (the stage waits at the
    // barrier were most of what separated the loop from the MFMA rate).
    // DS = steps carrying the rest, Q(s) = first instruction of step s,
    // BEFORE = instructions issued before the barrier.
    const int nk = ((K + BK - 1) / BK + NST - 1) / NST * NST;
    constexpr int KS = C::KS;
    constexpr bool EARLY = NST == 2 && KS >= 3;
#ifndef FOE_DMA_EARLY_Q  // eighths of a stage's instructions issued early
#define FOE_DMA_EARLY_Q 4
#endif
    constexpr int QE = EARLY ? NLD * FOE_DMA_EARLY_Q / 8 : 0;
    constexpr int DS = EARLY ? 1 : (NST == 2 ? (KS - 2 > 1 ? KS - 2 : 1) : KS);
    constexpr int BEFORE = NST == 2 ? NLD : (KS - 1) * NLD / KS;
    // loads allowed in flight at the barrier of iteration kt (stage kt+1
    // complete): the later stages' DMAs issued so far
    constexpr int VM_AT_BARRIER = NST == 2 ? 0 : (NST - 3) * NLD + BEFORE;
    static_assert(VM_AT_BARRIER <= 63, "vmcnt range");
    auto qof = [&](int st) { return st >= DS ? NLD : QE + st * (NLD - QE) / DS; };
    auto iteration = [&](auto mode, int kt, int b) {
      const int dkt = kt + NST - 1, dbuf = (b + NST - 1) % NST;
#pragma unroll
      for (int st = 0; st + 1 < KS; ++st)
        kstep(mode, st & 1, b, st + 1, dkt, dbuf, qof(st), qof(st + 1));
      vm_barrier<VM_AT_BARRIER>();
      if constexpr (EARLY)  // stage kt+2 into the buffer of stage kt
        kstep(mode, (KS - 1) & 1, (b + 1) % NST, 0, kt + 2, b, 0, QE);
      else
        kstep(mode, (KS - 1) & 1, (b + 1) % NST, 0, dkt, dbuf, qof(KS - 1), qof(KS));
    };
    // the K loop, specialised for issuing and non-issuing waves (both meet
    // the same barriers)
    auto k_loop = [&](auto mode) {
      if constexpr (decltype(mode)::value & 1) {
#pragma unroll
        for (int st = 0; st < NST - 1; ++st)
#pragma unroll
          for (int q = 0; q < NLD; ++q) issue_one(st, st, q);
        if constexpr (EARLY) {  // the early part of stage 1
#pragma unroll
          for (int q = 0; q < QE; ++q) issue_one(1, 1, q);
        }
      }
      vm_barrier<EARLY ? QE : NLD * (NST - 2)>();
      // `signal`: counted once every wave's earlier stores have completed
      // (the wait drains every earlier memory operation of the wave, and the
      // barrier meets all waves)
      if (signal != nullptr) {
        if constexpr (NST != 2 || EARLY) vm_barrier<0>();
        if (threadIdx.x == 0) atomicAdd(signal, 1);
      }
      fload(0, 0, 0);
      for (int kt = 0; kt < nk; kt += NST) {
#pragma unroll
        for (int u = 0; u < NST; ++u) iteration(mode, kt + u, u);
      }
      // the last DMAs (zeros past K) land before the buffers are reused
      vm_barrier<0>();
    };
    if (!partial_tile) {
      if (wave_u < C::NP)
        k_loop(std::integral_constant<int, 1>{});
      else
        k_loop(std::integral_constant<int, 0>{});
    } else {
      if (wave_u < C::NP)
        k_loop(std::integral_constant<int, 3>{});
      else
        k_loop(std::integral_constant<int, 2>{});
    }

    // Thread indices of the epilogue, taken afresh: address arithmetic on
    // the ones above would be hoisted before the K loop and kept live through
    // it, where the accumulators and fragments leave no registers for it, so
    // the compiler would spill it and reload each value behind a wait for
    // every outstanding store.
    const int tid_e = opaque_int((int)threadIdx.x);
    const int lane_e = tid_e & (kWave - 1);
    const int wm_e = (tid_e >> 6) / WN, wn_e = (tid_e >> 6) % WN;
    const int lrow_e = lane_e & 31;
    // epilogue: lane_e holds row m = .. + lane_e%32, columns n = .. + 8q + 4*(lane_e/32) + [0,4)
    [[maybe_unused]] const __amdgpu_buffer_rsrc_t out_rsrc = make_rsrc_u(out, g.out_bytes);
    if constexpr (RESID) {
      // the residual added to the accumulators, the loads of all of the
      // lane_e's outputs in flight together
      f32x4 xv[C::SM][C::SN][4];
#pragma unroll
      for (int i = 0; i < C::SM; ++i)
#pragma unroll
        for (int j = 0; j < C::SN; ++j)
#pragma unroll
          for (int q = 0; q < 4; ++q) {
            const int m = row0 + wm_e * C::WTM + i * 32 + lrow_e;
            const int n = n0 + wn_e * C::WTN + j * 32 + q * 8 + (lane_e >> 5) * 4;
            xv[i][j][q] = (m < row_end && n < N)
                              ? *reinterpret_cast<const f32x4*>(res.x + (size_t)m * N + n)
                              : f32x4{0.f, 0.f, 0.f, 0.f};
          }
#pragma unroll
      for (int i = 0; i < C::SM; ++i)
#pragma unroll
        for (int j = 0; j < C::SN; ++j)
#pragma unroll
          for (int q = 0; q < 4; ++q)
#pragma unroll
            for (int v = 0; v < 4; ++v) acc[0][i][j][q * 4 + v] += xv[i][j][q][v];
    }
    if constexpr (GATEUP && OUT_CPOL != 0) {
      if (!g.halves) {
        // Device-scope stores of whole lines: the SwiGLU tile goes to LDS
        // first (free after the K loop; 16-byte chunk c of tile row r at slot
        // c ^ (r & 15), so the writes of 16 rows at one chunk spread over the
        // banks), then every lane_e stores 16-byte chunks of whole rows (a wave
        // instruction covers 4 rows of 256 bytes), so the stores that pass
        // the L2 are full 128-byte lines rather than 16-byte pieces of 32.
        static_assert(BN == 128, "16 chunks per staged row");
        constexpr int ORB = BN * 2;
#pragma unroll
        for (int i = 0; i < C::SM; ++i) {
          const int rr = wm_e * C::WTM + i * 32 + lrow_e;
#pragma unroll
          for (int q = 0; q < 4; ++q) {
            const int ch = (wn_e * C::WTN + q * 8) / 8;
            bf16x4 o;
#pragma unroll
            for (int v = 0; v < 4; ++v)
              o[v] = (bf16)(silu_f(acc[0][i][0][q * 4 + v]) * acc[1][i][0][q * 4 + v]);
            *reinterpret_cast<bf16x4*>(smem + rr * ORB + ((ch ^ (rr & 15)) * 16) +
                                       (lane_e >> 5) * 8) = o;
          }
        }
        lds_barrier();
        constexpr int NCH = BM * (BN / 8);
        static_assert(NCH % C::NTHR == 0, "whole store rounds");
#pragma unroll
        for (int k = 0; k < NCH / C::NTHR; ++k) {
          const int c = tid_e + k * C::NTHR;
          const int rr = c / (BN / 8), ch = c % (BN / 8);
          const int m = row0 + rr, n = n0 + ch * 8;
          if (m < row_end && n < N) {
            const bf16x8 o =
                *reinterpret_cast<const bf16x8*>(smem + rr * ORB + ((ch ^ (rr & 15)) * 16));
            __builtin_amdgcn_raw_buffer_store_b128(__builtin_bit_cast(u32x4, o), out_rsrc,
                                                   (uint32_t)(((size_t)m * N + n) * 2), 0,
                                                   OUT_CPOL);
          }
        }
        return;
      }
    }
    if constexpr (GATEUP) {
      if (g.halves) {
        // The BM x 2*BN output tile (slice b at columns ntile*2*BN + b*BN + ..)
        // goes to LDS first (the stage buffers are free after the K loop;
        // 16-byte chunk c of tile row r at slot c ^ (r & 31)), then every lane_e
        // stores 16-byte chunks of whole rows, so a wave instruction writes 2
        // full rows (8 whole 128-byte lines) instead of 32 rows x 16 bytes.
        static_assert(C::SN == 1 && BN == 128, "32 chunks per staged row");
        constexpr int ORB = 2 * BN * 2;                 // bytes per staged row
        constexpr int RCH = 2 * BN / 8;                 // 16-byte chunks per row
        static_assert(BM * ORB <= NST * C::STAGE, "staged tile fits the stage buffers");
#pragma unroll
        for (int i = 0; i < C::SM; ++i) {
          const int rr = wm_e * C::WTM + i * 32 + lrow_e;
#pragma unroll
          for (int b = 0; b < 2; ++b)
#pragma unroll
            for (int q = 0; q < 4; ++q) {
              const int ch = b * (BN / 8) + (wn_e * C::WTN + q * 8) / 8;
              bf16x4 o;
#pragma unroll
              for (int v = 0; v < 4; ++v) o[v] = (bf16)acc[b][i][0][q * 4 + v];
              *reinterpret_cast<bf16x4*>(smem + rr * ORB + ((ch ^ (rr & 31)) * 16) +
                                         (lane_e >> 5) * 8) = o;
            }
        }
        lds_barrier();
        // thread tid_e stores chunk tid_e % RCH of rows tid_e / RCH + k * RPR
        constexpr int RPR = C::NTHR / RCH;  // rows per store round
        static_assert(C::NTHR % RCH == 0 && BM % (2 * RPR) == 0 && 32 % RPR == 0,
                      "store rounds");
        const int ch = tid_e % RCH, r0 = tid_e / RCH;
        const int n = ntile * 2 * BN + ch * 8;
        if (n < N) {
          // rows r0 + k*RPR take 32 / RPR values of r & 31, so as many LDS
          // slot offsets serve all rounds
          constexpr int NV = 32 / RPR;
          int slot[NV];
#pragma unroll
          for (int v = 0; v < NV; ++v) slot[v] = (ch ^ ((r0 + v * RPR) & 31)) * 16;
          const unsigned char* src = smem + r0 * ORB;
          bf16* dst = out + (size_t)(row0 + r0) * N + n;
          const int nr = row_end - row0 - r0;  // rows of this thread's column still valid
#pragma unroll
          for (int k = 0; k < BM / RPR; ++k) {
            if (k * RPR < nr)
              *reinterpret_cast<bf16x8*>(dst + (size_t)k * RPR * N) =
                  *reinterpret_cast<const bf16x8*>(src + k * RPR * ORB + slot[k % NV]);
          }
        }
        return;
      }
    }
#pragma unroll
    for (int i = 0; i < C::SM; ++i) {
      const int m = row0 + wm_e * C::WTM + i * 32 + lrow_e;
      if (m >= row_end) continue;
#pragma unroll
      for (int j = 0; j < C::SN; ++j) {
#pragma unroll
        for (int q = 0; q < 4; ++q) {
          const int n = n0 + wn_e * C::WTN + j * 32 + q * 8 + (lane_e >> 5) * 4;
          if (n >= N) continue;
          float val[4];
#pragma unroll
          for (int v = 0; v < 4; ++v) {
            val[v] = acc[0][i][j][q * 4 + v];
            if constexpr (GATEUP) val[v] = silu_f(val[v]) * acc[C::NB - 1][i][j][q * 4 + v];
          }
          if constexpr (RESID) {
#pragma unroll
            for (int v = 0; v < 4; ++v) val[v] *= res.scale;
          }
          bf16x4 o;
#pragma unroll
          for (int v = 0; v < 4; ++v) o[v] = (bf16)val[v];
          if constexpr (OUT_CPOL != 0)
            __builtin_amdgcn_raw_buffer_store_b64(__builtin_bit_cast(u32x2, o), out_rsrc,
                                                  (uint32_t)(((size_t)m * N + n) * 2), 0,
                                                  OUT_CPOL);
          else
            *reinterpret_cast<bf16x4*>(out + (size_t)m * N + n) = o;
        }
      }
    }
  }
}

// tile t -> (M-tile, N-tile) of m_tiles x ntn tiles: groups of GM M-tiles are
// walked N-tile by N-tile, so that a run of consecutive tiles shares A rows
// and weight slices
template <int GM>
__device__ __forceinline__ void tile_coords(int t, int ntn, int m_tiles, int& mt, int& nt) {
  if constexpr (GM <= 1) {
    mt = t / ntn;
    nt = t % ntn;
  } else {
    // the last group may hold fewer than GM M-tiles
    const int grp = t / (GM * ntn), i = t % (GM * ntn);
    const int g = min(GM, m_tiles - grp * GM);
    mt = grp * GM + i % g;
    nt = i / g;
  }
}

template <int BM, int BN, int WM, int WN, bool GATEUP, int BK, int NST, int PW, int GM,
          int PERSIST, bool RESID = false>
__global__ __launch_bounds__(WM* WN* kWave) __attribute__((amdgpu_waves_per_eu(1, 2)))
void grouped_gemm_dma(const bf16* __restrict__ A, const int32_t* __restrict__ gather, int kdiv,
                      int a_rows, const int32_t* __restrict__ offsets, int E, int rows,
                      const bf16* __restrict__ B0, const bf16* __restrict__ B1, int N, int K,
                      bf16* __restrict__ out, int n_tiles_n, int n_tiles, GemmResid res) {
  using C = DmaCfg<BM, BN, WM, WN, GATEUP, BK, NST, PW>;
  __shared__ __align__(1024) unsigned char smem[NST * C::STAGE];
  const GemmArgs g{A, gather, kdiv, a_rows, B0, B1, N, K, out, 0u, res, false};
  auto run_tile = [&](const int e, const int row0, const int row_end, const int ntile) {
    gemm_tile<BM, BN, WM, WN, GATEUP, BK, NST, PW, RESID, 0>(smem, g, e, row0, row_end, ntile);
  };

  // M-tiles that hold rows (persistent form: the tile list is split over
  // the XCDs by this count, not by the launch's upper bound)
  const int m_tiles = PERSIST ? __builtin_amdgcn_readfirstlane(total_mtiles(offsets, E, rows, BM))
                              : n_tiles / n_tiles_n;
  auto tile_coords = [&](int t, int& mt, int& nt) {
    foe::tile_coords<GM>(t, n_tiles_n, m_tiles, mt, nt);
  };
  auto run_t = [&](int t) {
    int mt, nt, e, row0, row_end;
    tile_coords(t, mt, nt);
    if (!find_tile(offsets, E, rows, BM, mt, e, row0, row_end)) return;
    vm_barrier<0>();  // the previous tile's LDS reads are done everywhere
    run_tile(e, row0, row_end, nt);
  };
  if constexpr (PERSIST == 2) {
    // one workgroup per CU, each XCD walks a contiguous eighth of the tile
    // order (workgroup b runs on XCD b % 8; the grid is a multiple of 8), so
    // the N-tiles of an M-tile and the M-tiles of a segment meet in that
    // XCD's own L2: for a few wide segments (one per XCD) every A row and
    // weight slice is fetched from memory once
    const int n_real = m_tiles * n_tiles_n;
    const int x = blockIdx.x % 8, per = gridDim.x / 8;
    const int chunk = (n_real + 7) / 8;
    const int t_end = min((x + 1) * chunk, n_real);
    for (int t = x * chunk + (int)blockIdx.x / 8; t < t_end; t += per) run_t(t);
  } else if constexpr (PERSIST == 1) {
    // one workgroup per CU, tiles dealt round-robin: the tiles running at any
    // moment are a window of consecutive tiles of the order above, spread
    // over all XCDs, and their shared A rows and weight slices meet in the
    // Infinity Cache that every XCD reads through (measured faster than
    // giving each XCD a contiguous range for its own L2 on the expert GEMMs)
    const int n_real = m_tiles * n_tiles_n;
    for (int t = blockIdx.x; t < n_real; t += gridDim.x) run_t(t);
  } else {
    const int tile = blockIdx.x;
    if (tile >= n_tiles) return;
    int mt, nt, e, row0, row_end;
    tile_coords(tile, mt, nt);
    if (!find_tile(offsets, E, rows, BM, mt, e, row0, row_end)) return;
    run_tile(e, row0, row_end, nt);
  }
}

// Both grouped GEMMs of the expert FFN in one persistent launch.  Work items
// are the gate/up tiles (SwiGLU epilogue, writing h) followed by the down
// tiles (reading h, writing y), numbered in that order; a workgroup's first
// item is its own index and the later ones come one at a time, in order, from
// a device-side counter, so the two GEMMs share one schedule: the
// CUs that finish their last gate/up tile go on to down tiles instead of
// idling through a partly filled last round, and there is no launch between
// the two.
//
// Both tile kinds run the one tile body of the gate/up form (BM rows x two
// BN-row weight slices): a down tile's two slices are consecutive BN-row
// blocks of W_d, stored side by side instead of through SwiGLU.
//
// A down tile of M-tile m needs every gate/up tile of m.  A gate/up tile
// writes its h rows with device-scope stores of whole lines (staged through
// LDS, past its XCD's L2) and is counted in ready[m] once they have completed:
// at the prologue of the workgroup's next gate/up tile, whose wait drains them
// anyway, or before the workgroup's first wait and at its end.  A down tile
// waits until ready[m] holds all of m's gate/up tiles before loading h.  The
// wait always ends: every gate/up tile a down tile waits for is the first
// item of a workgroup of the grid or was taken from the counter, in order,
// before the down tile, by a workgroup that is running it (or holds it as its
// next item behind a gate/up tile); gate/up tiles wait on nothing.  (The
// wait also gives up after a bounded number of polls, so the launch drains
// whatever happens; a give-up is counted in the give-up word of sync.)  No h
// row is read before it is complete, and with rows of whole 128-byte lines (F a
// multiple of 64, checked by the caller) no line is shared by two M-tiles, so
// no XCD's L2 can hold a stale copy of an h line (the L2s hold no h lines from
// earlier launches: each launch starts with them invalidated).
//
// sync: the work counters (one 128-byte line each), give-ups, then ready[m];
// zeroed before the launch (by the index pass).
constexpr int kReadyPollLimit = 1 << 20;  // about a second of polling

// waves of the fused FFN that issue the DMA: all 8 (each its share of a
// stage, ahead of its MFMAs) measured 2-5% faster than one per SIMD
#ifndef FOE_FUSED_PW
#define FOE_FUSED_PW 8
#endif
// M-tiles per group of the fused FFN's tile order (a group's gate/up tiles
// are walked N-tile by N-tile)
#ifndef FOE_FUSED_GM
#define FOE_FUSED_GM 4
#endif
// per-XCD work lists from this many groups of M-tiles (fewer groups leave the
// lists unbalanced, and the tail goes to taking items from other lists)
#ifndef FOE_FUSED_XCD_MIN_GROUPS
#define FOE_FUSED_XCD_MIN_GROUPS 32
#endif
constexpr int kLineInts = 32;  // one counter per 128-byte line

// Work lists of the fused FFN, one per XCD: list x holds the groups of GM
// M-tiles g = x, x+8, x+16, ... (all their gate/up tiles, then all their down
// tiles, in the tile order), so the 32 workgroups of one XCD work on the tiles
// of a few groups at a time and their A rows and weight slices meet in that
// XCD's L2.  A group's down tiles depend only on the same group's gate/up
// tiles, so every dependency stays inside one list.
struct FusedLists {
  int m_tiles, ntg, ntd, n_groups, gm;
  // groups of list x and M-tiles of its last group
  __device__ int groups(int x) const { return x < n_groups ? (n_groups - 1 - x) / 8 + 1 : 0; }
  __device__ int tiles(int x, int ntn) const {
    const int ng = groups(x);
    if (ng == 0) return 0;
    const int last = x + 8 * (ng - 1);
    return ((ng - 1) * gm + min(gm, m_tiles - last * gm)) * ntn;
  }
  __device__ int size(int x) const { return tiles(x, ntg) + tiles(x, ntd); }
  // global item (tile order: gate/up tiles, then down tiles) of item i of list
  // x, i < size(x)
  __device__ int item(int x, int i) const {
    const int ngu = tiles(x, ntg);
    if (i < ngu) return (x + 8 * (i / (gm * ntg))) * gm * ntg + i % (gm * ntg);
    i -= ngu;
    return m_tiles * ntg + (x + 8 * (i / (gm * ntd))) * gm * ntd + i % (gm * ntd);
  }
};

template <int BM, int BN, int WM, int WN, int BK, int NST, int PW, int GM>
__global__ __launch_bounds__(WM* WN* kWave) __attribute__((amdgpu_waves_per_eu(1, 2)))
void ffn_fused_dma(const bf16* __restrict__ A, const int32_t* __restrict__ gather, int kdiv,
                   int a_rows, const int32_t* __restrict__ offsets, int E, int rows,
                   const bf16* __restrict__ wg, const bf16* __restrict__ wu,
                   const bf16* __restrict__ wd, int d, int F, bf16* __restrict__ h,
                   bf16* __restrict__ y, int32_t* __restrict__ sync) {
  // one tile shape for both GEMMs: BM rows x (BN gate + BN up) columns, or
  // BM rows x 2*BN down columns read as two BN-row slices of W_d (the same
  // operand loads, LDS layout and MFMA sequence; only the epilogue differs)
  using C = DmaCfg<BM, BN, WM, WN, true, BK, NST, PW>;
  __shared__ __align__(1024) unsigned char smem[NST * C::STAGE];
  __shared__ int s_item[2];  // alternate slots: a slot is rewritten one barrier after it is read
  __shared__ int s_tab[3 * kTileTab];

  // the M-tile order: the table (scratch in the stage buffers, which no DMA
  // uses yet), or experts in id order through find_tile past its capacity
  static_assert(NST * C::STAGE >= (4 * kTabMaxE + 1) * 4, "table scratch fits");
  const int mt_tab = build_tile_table<C::NTHR>(offsets, E, rows, BM,
                                               reinterpret_cast<int*>(smem), s_tab);
  const bool tab_ok = mt_tab >= 0 && mt_tab <= kTileTab;
  const int m_tiles = tab_ok ? mt_tab
                             : __builtin_amdgcn_readfirstlane(total_mtiles(offsets, E, rows, BM));
  const int ntg = (F + BN - 1) / BN, ntd = (d + 2 * BN - 1) / (2 * BN);
  const int n_gu = m_tiles * ntg, n_all = n_gu + m_tiles * ntd;
  // sync: list counters (one line each), give-ups, then ready[m]
  int32_t* giveups = sync + 8 * kLineInts;
  int32_t* ready = sync + 9 * kLineInts;
  const FusedLists fl{m_tiles, ntg, ntd, (m_tiles + GM - 1) / GM, GM};

  // The first item of a workgroup is fixed (a workgroup that starts early
  // cannot take two first-round items); the next item is taken while the
  // current one runs (its value is needed only at the end), so items come
  // without a wait.  With many groups (xq) workgroup b (on XCD b % 8) works
  // through list b % 8 and then takes the remaining items of the other lists
  // (measured 2.7% faster at 270 and 290 M-tiles, 8% slower at 73);
  // otherwise all items form one list.  Items of a list are taken in order.
  // Deadlock-free: a workgroup blocked on a down tile holds no unstarted
  // gate/up item (its next item was taken after its current, down, item, and
  // a list's gate/up items come before its down items), and first items
  // belong to workgroups of the grid, which run to their end.
  const bool xq = fl.n_groups >= FOE_FUSED_XCD_MIN_GROUPS;
  const int nper = xq ? (int)gridDim.x / 8 : (int)gridDim.x;
  int list = xq ? (int)blockIdx.x % 8 : 0;  // thread 0's current list
  auto list_size = [&](int l) { return xq ? fl.size(l) : n_all; };
  auto list_item = [&](int l, int i) { return xq ? fl.item(l, i) : i; };
  // thread 0: the next item after index i of the current list (i from the
  // list's counter), or one taken from the other lists, or -1
  auto next_item = [&](int i) {
    if (i < list_size(list)) return list_item(list, i);
    for (int k = 1; xq && k < 8; ++k) {
      const int l = (list + k) % 8;
      const int j = nper + atomicAdd(&sync[l * kLineInts], 1);
      if (j < list_size(l)) {
        list = l;
        return list_item(l, j);
      }
    }
    return -1;
  };
  if (threadIdx.x == 0) {
    const int i0 = xq ? (int)blockIdx.x / 8 : (int)blockIdx.x;
    s_item[0] = i0 < list_size(list) ? list_item(list, i0)
                                     : next_item(nper + atomicAdd(&sync[list * kLineInts], 1));
  }
  lds_barrier();
  int t = s_item[0];
  int slot = 0;
  // M-tile of this workgroup's last gate/up tile, not yet counted in ready[]:
  // it is counted at the next gate/up tile's prologue (whose wait drains the
  // stores anyway) or flushed before a wait and at the end
  int pending = -1;
  auto flush = [&]() {
    if (pending >= 0) {
      asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
      __syncthreads();
      if (threadIdx.x == 0) atomicAdd(&ready[pending], 1);
      pending = -1;
    }
  };
  while (t >= 0 && t < n_all) {
    int next_i = 0;
    if (threadIdx.x == 0) next_i = nper + atomicAdd(&sync[list * kLineInts], 1);
    const bool gu = t < n_gu;
    int mt, nt, e, row0, row_end;
    if (gu)
      tile_coords<GM>(t, ntg, m_tiles, mt, nt);
    else
      tile_coords<GM>(t - n_gu, ntd, m_tiles, mt, nt);
    bool have;
    if (tab_ok) {
      e = s_tab[3 * mt];
      row0 = s_tab[3 * mt + 1];
      row_end = s_tab[3 * mt + 2];
      have = true;
    } else {
      have = find_tile(offsets, E, rows, BM, mt, e, row0, row_end);
    }
    if (have) {
      if (!gu) {
        flush();
        if (threadIdx.x == 0) {
          int polls = 0;
          while (__hip_atomic_load(&ready[mt], __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) <
                 ntg) {
            if (++polls >= kReadyPollLimit) {
              atomicAdd(giveups, 1);
              break;
            }
            __builtin_amdgcn_s_sleep(2);
          }
        }
        __syncthreads();
      }
      // h is stored past the XCD's L2 (other XCDs read it in this launch), y
      // as usual (the next kernel reads it)
      const GemmArgs g = gu ? GemmArgs{A, gather, kdiv, a_rows, wg, wu, F, d, h,
                                       (uint32_t)rows * F * 2u, GemmResid{}, false}
                            : GemmArgs{h, nullptr, 1, rows, wd, nullptr, d, F, y,
                                       (uint32_t)rows * d * 2u, GemmResid{}, true};
      gemm_tile<BM, BN, WM, WN, true, BK, NST, PW, false, kScDevice>(
          smem, g, e, row0, row_end, nt, gu && pending >= 0 ? &ready[pending] : nullptr);
      if (gu) pending = mt;
    }
    // the next item in LDS; this item's LDS use is done everywhere
    slot ^= 1;
    if (threadIdx.x == 0) s_item[slot] = next_item(next_i);
    lds_barrier();
    t = s_item[slot];
  }
  flush();
}

// Few rows per expert (decode), LDS-staged weight stream.  A workgroup of 4
// waves takes one expert and 4 consecutive weight tiles (each 16 gate + 16 up
// rows, or 32 down rows), one per wave, over all of K, for up to 32 rows of A
// (tokens) at a time.  Operands stream through a ring of NS LDS stages of
// 128 K columns: per stage each wave loads its weight tile with 8 LDS-DMA
// instructions and a quarter of the shared token tile with 2, each
// instruction covering 4 rows x 256 bytes (the access pattern that reads HBM
// fastest).  The 16-byte chunk c of row r of any tile sits in slot
// c ^ (r & 15), so the v_mfma_f32_16x16x32_bf16 fragment reads (16 rows, one
// chunk) are conflict-free.
//
// All loads of the loop are LDS DMA issued from inline assembly with explicit
// vmcnt waits, so NS-2 later stages stay in flight while a stage is used.

template <bool GATEUP, int NS, bool SEL>
__global__ __launch_bounds__(256) void ffn_stream_bf16(
    const bf16* __restrict__ A, const int32_t* __restrict__ gather, int kdiv, int a_rows,
    const int32_t* __restrict__ offsets, int E, int rows, const bf16* __restrict__ W0,
    const bf16* __restrict__ W1, int N, int K, bf16* __restrict__ out, int n_groups,
    int e_per_c, int r_sel, FusedCombine fc) {
  static_assert(NS >= 2 && NS <= 4, "2 to 4 stages");
  constexpr int WPB = 4;
  constexpr int NPW = GATEUP ? 16 : 32;  // output columns per wave
  constexpr int WB = 8192;                // weight bytes per stage and wave
  constexpr int XB = WPB * WB;            // offset of the token rows in a stage
  constexpr int SB = XB + 8192;           // bytes per stage
  constexpr int NI = 10;                  // DMA instructions per stage and wave
  constexpr int SELB = SEL ? kSelMax * 4 : 0;       // staged expert ids of the cluster
  constexpr int LSTB = SEL ? kSelMax * 4 + 64 : 0;  // pair list + wave counts
  static_assert(NS * SB + SELB + LSTB <= 160 * 1024, "LDS capacity");
  __shared__ __align__(1024) unsigned char smem[NS * SB + SELB + LSTB];

  const int lane = lane_id();
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);  // wave-uniform
  const int gpe = (n_groups + WPB - 1) / WPB;                           // workgroups per expert
  const int e = blockIdx.x / gpe;
  if (e >= E) return;
  const int n0 = ((blockIdx.x % gpe) * WPB + wave) * NPW;
  int off_a = 0, off_b = 0;
  if constexpr (!SEL) {
    off_a = offsets[e];  // scalar loads, waited on below
    off_b = offsets[e + 1];
  }
  // selection mode: expert e is expert le of cluster hc
  const int hc = SEL ? e / e_per_c : 0;
  const int le = SEL ? e - hc * e_per_c : 0;
  const uint32_t lds0 = lds_addr(smem);
  if constexpr (SEL) {
    // the cluster's r_sel expert ids go to LDS first (256 per wave instruction)
    const __amdgpu_buffer_rsrc_t sr =
        make_rsrc_u(gather + (size_t)hc * r_sel, (uint32_t)r_sel * 4u);
    for (int c = wave * 256; c < r_sel; c += WPB * 256)
      dma16(sr, (uint32_t)(c + 4 * lane) * 4u, lds0 + NS * SB + c * 4, 0);
  }

  // weight sources: instruction i < 4 reads tile rows 4i.. of W0, i >= 4 rows
  // 4(i-4).. of W1 (gate/up) or rows 4i.. of W0 (down); a wave past N reads
  // zeros (empty range)
  const int nv = max(min(NPW, N - n0), 0);
  const size_t wrow = (size_t)e * N + min(n0, N);
  const __amdgpu_buffer_rsrc_t wr0 = make_rsrc_u(W0 + wrow * K, (uint32_t)nv * K * 2u);
  const __amdgpu_buffer_rsrc_t wr1 =
      GATEUP ? make_rsrc_u(W1 + wrow * K, (uint32_t)nv * K * 2u) : wr0;
  const __amdgpu_buffer_rsrc_t ar = make_rsrc_u(A, (uint32_t)a_rows * K * 2u);
  // output rows of the folded combine (down, selection mode)
  const __amdgpu_buffer_rsrc_t yr = make_rsrc_u(out, (uint32_t)rows * N * 2u);
  const int lr = lane >> 4, lc = lane & 15;
  uint32_t wv[8];  // byte offset of this lane's weight chunk in instruction i (stage 0)
  int wk[8];       // its K column
#pragma unroll
  for (int i = 0; i < 8; ++i) {
    const int tr = (GATEUP ? (i & 3) : i) * 4 + lr;  // row inside the rsrc range
    const int q = lc ^ (tr & 15);                     // chunk of the 256-byte segment
    wk[i] = q * 8;
    wv[i] = ((uint32_t)tr * K + q * 8) * 2u;
  }
  const int nks = (K + 127) / 128;
  // Workgroups start their K walk at different chunks, so the reads in flight
  // at any moment are spread over all column offsets of the 4 KB-strided
  // weight rows (and so over the HBM channels) instead of one.
  const int rot = FOE_STREAM_ROT ? (int)(blockIdx.x % (unsigned)nks) : 0;
  auto chunk0 = [&](int kt) {
    const int kc = kt + rot;
    return (kc >= nks ? kc - nks : kc) * 128;
  };
  // fragment read offsets inside a stage: row R of a 16-row tile
  const int R = lane & 15, g = lane >> 4;
  const int rbase = (R >> 2) * 1024 + (R & 3) * 256;

  auto issue_w = [&](int kt, int s) {
    const int k0 = chunk0(kt);
#pragma unroll
    for (int i = 0; i < 8; ++i) {
      const uint32_t off = k0 + wk[i] < K ? wv[i] + (uint32_t)k0 * 2u : kOob;
      dma16(GATEUP && i >= 4 ? wr1 : wr0, off, lds0 + wave * WB, s * SB + i * 1024);
    }
  };
  // The weights of the first NS-1 stages do not depend on the token rows:
  // they go out before the segment bounds and gather indices are read.
#pragma unroll
  for (int s = 0; s < NS - 1; ++s)
    if (s < nks) issue_w(s, s);
  int a = 0, b = 0;
  const int* lst = reinterpret_cast<const int*>(smem + NS * SB + SELB);
  if constexpr (SEL) {
    // Pair list of this expert in ascending pair order (the stable order of
    // the dispatch): per 256-pair chunk, each wave ballots its matches and
    // the wave counts give the positions.  The weight DMAs stay in flight.
    if (nks >= NS - 1) vm_wait<8 * (NS - 1)>();
    else vm_wait<0>();
    lds_barrier();
    const int* sel = reinterpret_cast<const int*>(smem + NS * SB);
    int* lw = reinterpret_cast<int*>(smem + NS * SB + SELB);
    int* wc = lw + kSelMax;
    const uint64_t below = lane == 0 ? 0ull : (~0ull >> (64 - lane));
    int n = 0;
    for (int c0 = 0; c0 < r_sel; c0 += WPB * 64) {
      const int f = c0 + (int)threadIdx.x;
      const bool ok = f < r_sel && sel[f] == le;
      const uint64_t m = __ballot(ok);
      if (lane == 0) wc[wave] = __popcll(m);
      lds_barrier();
      int pre = 0, tot = 0;
#pragma unroll
      for (int w = 0; w < WPB; ++w) {
        const int cw = wc[w];
        pre += w < wave ? cw : 0;
        tot += cw;
      }
      if (ok) lw[n + pre + __popcll(m & below)] = f;
      n += tot;
      lds_barrier();
    }
    b = n;
  } else {
    a = min(max(off_a, 0), rows);
    b = max(min(max(off_b, 0), rows), a);
  }
  if (b == a) {  // uniform over the workgroup; the DMAs land before LDS is released
    vm_wait<0>();
    return;
  }

  for (int t0 = a; t0 < b; t0 += 32) {
    const int tv = min(32, b - t0);
    if (t0 != a) {
#pragma unroll
      for (int s = 0; s < NS - 1; ++s)
        if (s < nks) issue_w(s, s);
    }
    // token instructions 2*wave and 2*wave+1 of this wave (rows 8*wave + 4u +
    // lane/16 of the pass); the wave's 8 gather indices are uniform loads
    uint32_t xv[2];
    int xk[2];
    if constexpr (SEL) {
#pragma unroll
      for (int u = 0; u < 2; ++u) {
        const int t = 8 * wave + 4 * u + lr;
        const int q = lc ^ (t & 15);
        int sr = -1;
        if (t < tv) {
          const int f = lst[t0 + t];
          sr = GATEUP ? f / kdiv : hc * r_sel + f;
          if (sr >= a_rows) sr = -1;
        }
        xk[u] = q * 8;
        xv[u] = sr < 0 ? kOob : ((uint32_t)sr * K + q * 8) * 2u;
      }
    } else {
      const int tw = 8 * wave;
      int gi[8];
#pragma unroll
      for (int j = 0; j < 8; ++j)
        gi[j] = (gather != nullptr && tw + j < tv) ? gather[t0 + tw + j] : t0 + tw + j;
#pragma unroll
      for (int u = 0; u < 2; ++u) {
        const int t = tw + 4 * u + lr;
        const int q = lc ^ (t & 15);
        const int gsel = lr == 0 ? gi[4 * u] : lr == 1 ? gi[4 * u + 1] : lr == 2 ? gi[4 * u + 2]
                                                                                 : gi[4 * u + 3];
        int sr = -1;
        if (t < tv) {
          sr = gather == nullptr ? gsel : (gsel >= 0 ? gsel / kdiv : -1);
          if (sr >= a_rows) sr = -1;
        }
        xk[u] = q * 8;
        xv[u] = sr < 0 ? kOob : ((uint32_t)sr * K + q * 8) * 2u;
      }
    }
    auto issue_x = [&](int kt, int s) {
      const int k0 = chunk0(kt);
#pragma unroll
      for (int u = 0; u < 2; ++u) {
        const uint32_t off = (k0 + xk[u] < K && xv[u] != kOob) ? xv[u] + (uint32_t)k0 * 2u : kOob;
        dma16(ar, off, lds0 + wave * 2048, s * SB + XB + u * 1024);
      }
    };
#pragma unroll
    for (int s = 0; s < NS - 1; ++s)
      if (s < nks) issue_x(s, s);
    f32x4 acc[2][2];
#pragma unroll
    for (int i = 0; i < 2; ++i)
#pragma unroll
      for (int j = 0; j < 2; ++j) acc[i][j] = f32x4{0.f, 0.f, 0.f, 0.f};

    // iteration kt: wait for this wave's part of stage kt, meet the other
    // waves (stage kt complete, stage kt-1 no longer read), issue stage
    // kt+NS-1 into the buffer of stage kt-1, use stage kt.  The pass starts
    // with the weights of stages 0..NS-2 and then their token rows, so stage
    // u < NS-1 still has 2*(NS-2-u) token and u*NI loop instructions behind it.
    auto body = [&](int kt, auto U, int s_next) {
      constexpr int u = decltype(U)::value;
      if (kt + NS - 2 >= nks) vm_wait<0>();
      else if (u < NS - 1 && kt == u) vm_wait<2 * (NS - 2 - u) + NI * u>();
      else vm_wait<NI * (NS - 2)>();
      lds_barrier();
      if (kt + NS - 1 < nks) {
        issue_w(kt + NS - 1, s_next);
        issue_x(kt + NS - 1, s_next);
      }
      const unsigned char* src = smem + u * SB + rbase;
#pragma unroll
      for (int c = 0; c < 4; ++c) {
        const int slot = ((c * 4 + g) ^ R) * 16;
        const bf16x8 w0 = *reinterpret_cast<const bf16x8*>(src + wave * WB + slot);
        const bf16x8 w1 = *reinterpret_cast<const bf16x8*>(src + wave * WB + 4096 + slot);
        const bf16x8 x0 = *reinterpret_cast<const bf16x8*>(src + XB + slot);
        const bf16x8 x1 = *reinterpret_cast<const bf16x8*>(src + XB + 4096 + slot);
        acc[0][0] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(w0, x0, acc[0][0], 0, 0, 0);
        acc[1][0] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(w1, x0, acc[1][0], 0, 0, 0);
        acc[0][1] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(w0, x1, acc[0][1], 0, 0, 0);
        acc[1][1] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(w1, x1, acc[1][1], 0, 0, 0);
      }
    };
    for (int kt0 = 0; kt0 < nks; kt0 += NS) {
      static_for<0, NS>([&](auto U) {
        constexpr int u = decltype(U)::value;
        const int kt = kt0 + u;
        if (kt < nks) body(kt, U, (u + NS - 1) % NS);
      });
    }
    // every wave is done with the ring before the next pass refills it
    asm volatile("s_waitcnt vmcnt(0) lgkmcnt(0)\n\ts_barrier" ::: "memory");

    // lane holds weight rows 4*(lane/16) + [0,4) of each tile for token lane%16 (+16)
    const int nb = 4 * g;
#pragma unroll
    for (int j = 0; j < 2; ++j) {
      const int t = j * 16 + R;
      if (t >= tv) continue;
      const int orow_i = SEL ? hc * r_sel + lst[t0 + t] : t0 + t;
      bf16* orow = out + (size_t)orow_i * N + n0;
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
          if (SEL && fc.out != nullptr)  // device-scope store: read back by other workgroups
            __builtin_amdgcn_raw_buffer_store_b64(
                __builtin_bit_cast(u32x2, o), yr,
                (uint32_t)(((size_t)orow_i * N + n0 + i * 16 + nb) * 2), 0, kScDevice);
          else
            *reinterpret_cast<bf16x4*>(orow + i * 16 + nb) = o;
        }
      }
    }
  }

  if constexpr (!GATEUP && SEL) {
    if (fc.out != nullptr) {
      // Combine folded in: this workgroup's y columns [cg*128, +128) of its
      // pairs are stored (device-scope stores, past the XCD's own L2, and
      // acknowledged once visible to every XCD); count one arrival per (token,
      // column group).  The workgroup that brings a count to C*k forms that
      // token's output columns from device-scope loads of the y rows, summing
      // the k rows of every cluster in the fixed order (h, j) exactly as the
      // combine kernel does.  Nothing waits on another workgroup.
      asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
      const int cg = blockIdx.x % gpe;
      int* done = reinterpret_cast<int*>(smem + NS * SB);  // staged ids are dead
      int* ndone = reinterpret_cast<int*>(smem + NS * SB + SELB) + kSelMax;
      if (threadIdx.x == 0) *ndone = 0;
      __syncthreads();
      const int need = fc.C * fc.k;
      for (int i = (int)threadIdx.x; i < b; i += WPB * 64) {
        const int t = lst[i] / fc.k;
        const int old = atomicAdd(&fc.cnt[(size_t)t * gpe + cg], 1);
        if (old == need - 1) done[atomicAdd(ndone, 1)] = t;
      }
      __syncthreads();
      const int nd = *ndone;
      if (nd > 0) {
        const int c0 = cg * 128;
        const int nvec = (min(128, N - c0) + 7) / 8;
        const float cx = (float)fc.C;
        for (int it = (int)threadIdx.x; it < nd * 16; it += WPB * 64) {
          const int v = it & 15;
          if (v >= nvec) continue;
          const int t = done[it >> 4];
          const int col = c0 + v * 8;
          float acc[8];
#pragma unroll
          for (int q = 0; q < 8; ++q) acc[q] = 0.f;
          for (int h = 0; h < fc.C; ++h) {
            for (int j = 0; j < fc.k; ++j) {
              const size_t p = (size_t)h * r_sel + (size_t)t * fc.k + j;
              const float wj = fc.w[p];
              const bf16x8 yv = __builtin_bit_cast(
                  bf16x8, __builtin_amdgcn_raw_buffer_load_b128(
                              yr, (uint32_t)((p * N + col) * 2), 0, kScDevice));
#pragma unroll
              for (int q = 0; q < 8; ++q) acc[q] = fmaf(wj, (float)yv[q], acc[q]);
            }
          }
          const bf16x8 xv = *reinterpret_cast<const bf16x8*>(fc.x + (size_t)t * N + col);
          bf16x8 o;
#pragma unroll
          for (int q = 0; q < 8; ++q) o[q] = (bf16)(fc.scale * fmaf(cx, (float)xv[q], acc[q]));
          *reinterpret_cast<bf16x8*>(fc.out + (size_t)t * N + col) = o;
        }
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

// compute units of the current device (one persistent workgroup each)
int device_cus() {
  int dev = 0, n = 0;
  if (hipGetDevice(&dev) != hipSuccess ||
      hipDeviceGetAttribute(&n, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess || n < 8)
    return 256;
  return n / 8 * 8;
}

template <int BM, int BN, int WM, int WN, int BK, int NST, int PW, int GM, int PERSIST, bool GATEUP,
          bool RESID = false>
void launch_gemm_dma(const bf16* A, const int32_t* gather, int kdiv, int a_rows,
                     const int32_t* offsets, int E, int rows, const bf16* B0, const bf16* B1,
                     int N, int K, bf16* out, hipStream_t s, const char* name,
                     GemmResid res = GemmResid{}) {
  const int ntn = ceil_div(N, BN);
  const int max_mt = ceil_div(rows, BM) + E;  // sum_e ceil(M_e/BM) <= rows/BM + E
  const long long n_tiles = (long long)max_mt * ntn;
  long long nb = (n_tiles + 7) / 8 * 8;
  if (PERSIST) {
    static const int cus = device_cus();
    nb = nb < cus ? nb : cus;
  }
  dim3 grid((unsigned)nb);
  ProfileScope ps(name, s);
  FOE_LAUNCH((grouped_gemm_dma<BM, BN, WM, WN, GATEUP, BK, NST, PW, GM, PERSIST, RESID>),
             grid, dim3(WM * WN * kWave), 0, s, A, gather, kdiv, a_rows, offsets, E, rows, B0, B1,
             N, K, out, ntn, (int)n_tiles, res);
}

template <int BM, int BN, int WM, int WN, int BK, int NST, int PW, int GM, int PERSIST>
struct DmaLaunch {
  template <bool GATEUP, bool RESID = false, typename... Args>
  static void run(Args... args) {
    launch_gemm_dma<BM, BN, WM, WN, BK, NST, PW, GM, PERSIST, GATEUP, RESID>(args...);
  }
};

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
      FOE_LAUNCH(gateup_f32, dim3(ceil_div((long long)rows * F, 256)), dim3(256), 0, s,
                         reinterpret_cast<const float*>(A), gather, kdiv, a_rows, offsets, E,
                         rows, reinterpret_cast<const float*>(w_gate),
                         reinterpret_cast<const float*>(w_up), F, d, h);
    }
    {
      ProfileScope ps("ffn_down_f32", s);
      FOE_LAUNCH(down_f32, dim3(ceil_div((long long)rows * d, 256)), dim3(256), 0, s, h,
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
      FOE_LAUNCH((ffn_stream_bf16<true, FOE_STREAM_NS, false>), dim3(E * ceil_div(ng, 4)),
                 dim3(256), 0, s, xa, gather, kdiv, a_rows, offsets, E, rows, wg, wu, F, d, h,
                 ng, 1, 0, FusedCombine{});
    }
    {
      const int ng = ceil_div(d, 32);
      ProfileScope ps("ffn_down", s);
      FOE_LAUNCH((ffn_stream_bf16<false, FOE_STREAM_NS, false>), dim3(E * ceil_div(ng, 4)),
                 dim3(256), 0, s, static_cast<const bf16*>(h), nullptr, 1, rows, offsets, E,
                 rows, wd, nullptr, d, F, y, ng, 1, 0, FusedCombine{});
    }
  } else {
    DmaLaunch<FOE_DMA_GU>::run<true>(xa, gather, kdiv, a_rows, offsets, E, rows, wg, wu, F, d, h,
                                     s, "ffn_gateup");
    DmaLaunch<FOE_DMA_DN>::run<false>(static_cast<const bf16*>(h), (const int32_t*)nullptr, 1,
                                      rows, offsets, E, rows, wd, (const bf16*)nullptr, d, F, y, s,
                                      "ffn_down");
  }
  return hipGetLastError();
}

size_t ffn_sync_ints(int E, int rows) { return (size_t)ceil_div(rows, 256) + E + 9 * kLineInts; }

hipError_t launch_expert_ffn_fused(int E, int d, int F, int rows, const void* A,
                                   const int32_t* gather, int kdiv, int a_rows,
                                   const int32_t* offsets, const void* w_gate, const void* w_up,
                                   const void* w_down, void* y, void* h, int32_t* sync,
                                   hipStream_t s) {
  if (rows == 0) return hipSuccess;
  static const int cus = device_cus();
  ProfileScope ps("ffn_fused", s);
  FOE_LAUNCH((ffn_fused_dma<256, 128, 2, 4, 64, 2, FOE_FUSED_PW, FOE_FUSED_GM>), dim3(cus),
             dim3(8 * kWave), 0, s,
             static_cast<const bf16*>(A), gather, kdiv, a_rows, offsets, E, rows,
             static_cast<const bf16*>(w_gate), static_cast<const bf16*>(w_up),
             static_cast<const bf16*>(w_down), d, F, static_cast<bf16*>(h),
             static_cast<bf16*>(y), sync);
  return hipGetLastError();
}

bool ffn_sel_ok(foe_dtype dt, int C, int E, int T, int k) {
  const long long R = (long long)T * k;
  return FOE_FFN_SEL && dt == FOE_BF16 && R > 0 && R <= kSelMax &&
         (long long)C * R < 64LL * C * E;
}

hipError_t launch_expert_ffn_sel(int C, int E, int d, int F, int T, int k, const void* x,
                                 const int32_t* topk_idx, const void* w_gate, const void* w_up,
                                 const void* w_down, void* y, void* scratch, hipStream_t s,
                                 const FusedCombine& fc) {
  const int R = T * k;
  const int rows = C * R;
  const bf16* xa = static_cast<const bf16*>(x);
  const bf16* wg = static_cast<const bf16*>(w_gate);
  const bf16* wu = static_cast<const bf16*>(w_up);
  const bf16* wd = static_cast<const bf16*>(w_down);
  bf16* h = static_cast<bf16*>(scratch);
  bf16* yo = static_cast<bf16*>(y);
  {
    const int ng = ceil_div(F, 16);
    ProfileScope ps("ffn_gateup", s);
    FOE_LAUNCH((ffn_stream_bf16<true, FOE_STREAM_NS, true>), dim3(C * E * ceil_div(ng, 4)),
                       dim3(256), 0, s, xa, topk_idx, k, T, nullptr, C * E, rows, wg, wu, F, d, h,
                       ng, E, R, FusedCombine{});
  }
  {
    const int ng = ceil_div(d, 32);
    ProfileScope ps("ffn_down", s);
    FOE_LAUNCH((ffn_stream_bf16<false, FOE_STREAM_NS, true>),
                       dim3(C * E * ceil_div(ng, 4)), dim3(256), 0, s,
                       static_cast<const bf16*>(h), topk_idx, 1, rows, nullptr, C * E, rows, wd,
                       nullptr, d, F, yo, ng, E, R, fc);
  }
  return hipGetLastError();
}

hipError_t launch_grouped_gemm(const void* A, const int32_t* offsets, int E, int rows,
                               const void* W, int N, int K, void* out, hipStream_t s,
                               const char* name) {
  if (rows == 0) return hipSuccess;
  DmaLaunch<FOE_DMA_SEG>::run<false>(static_cast<const bf16*>(A), (const int32_t*)nullptr, 1, rows,
                                    offsets, E, rows, static_cast<const bf16*>(W),
                                    (const bf16*)nullptr, N, K, static_cast<bf16*>(out), s, name);
  return hipGetLastError();
}

hipError_t launch_gemm_resid(const void* A, const int32_t* offsets, int rows, const void* W,
                             int N, int K, const float* x, float scale, void* out, hipStream_t s,
                             const char* name) {
  if (rows == 0) return hipSuccess;
  GemmResid res;
  res.x = x;
  res.scale = scale;
  static const int cus = device_cus();
  if ((long long)ceil_div(rows, 128) * ceil_div(N, 256) < cus)
    DmaLaunch<FOE_DMA_RES_SMALL>::run<false, true>(
        static_cast<const bf16*>(A), (const int32_t*)nullptr, 1, rows, offsets, 1, rows,
        static_cast<const bf16*>(W), (const bf16*)nullptr, N, K, static_cast<bf16*>(out), s, name,
        res);
  else
    DmaLaunch<FOE_DMA_RES>::run<false, true>(
        static_cast<const bf16*>(A), (const int32_t*)nullptr, 1, rows, offsets, 1, rows,
        static_cast<const bf16*>(W), (const bf16*)nullptr, N, K, static_cast<bf16*>(out), s, name,
        res);
  return hipGetLastError();
}

hipError_t launch_expert_ffn(foe_dtype dt, int E, int d, int F, int rows, const void* x_perm,
                             const int32_t* offsets, const void* w_gate, const void* w_up,
                             const void* w_down, void* y_perm, void* scratch, hipStream_t s) {
  return launch_expert_ffn_ex(dt, E, d, F, rows, x_perm, nullptr, 1, rows, offsets, w_gate, w_up,
                              w_down, y_perm, scratch, s);
}

}  // namespace foe
