// Router scores + per-group top-k + routing weights (Section 3.1, routing
// equation), fused in one kernel: the [T, G*E] scores never leave the chip.
//
// route_kernel: one workgroup = TG groups of 16 tokens, 4 or 8 waves.  The
// score tile S[16 tokens][G*E] of each token group is x[16,d] * W_r^T on
// MFMA (bf16: 16x16x32, fp32: 16x16x4) with K split across the waves (each
// issuing the loads of several K steps at once); the partial tiles are summed
// in LDS in a fixed order.  G router matrices of co-resident clusters are one
// score matrix, so x is read once for all of them.  In the 16x16 MFMA result
// layout each row of 16 lanes holds 16 score columns of one token (per
// accumulator register), so a group's top-k is k rounds of a (score desc, id
// asc) arg-max over the group's columns across a 16-lane row with DPP
// rotations.  route_stream_kernel (many tokens, one group, E <= 32) streams x
// and W_r through LDS with a wave per 16 tokens over all of K.
//
// Weights: the softmax over the k selected scores of the group, or (global
// gating) the softmax over all G*E scores of the token, not renormalised.
#include "lds_dma.hpp"

namespace foe {
namespace {

constexpr int kTok = 16;    // tokens per workgroup
constexpr int kMaxGE = 256;  // score columns of one routing pass
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

// Global softmax normaliser of one token whose score columns nt*16 + col (col
// = lane % 16) sit in the lanes of a 16-lane row: the row maximum m and
// z = sum over the valid columns (< ncol) of exp(g - m), both in every lane
// of the row (rotation reductions, a fixed order).
template <int NT>
__device__ __forceinline__ void row_softmax_norm(const float (&g)[NT], int col, int ncol,
                                                 float& m, float& z) {
  float mx = -__builtin_inff();
#pragma unroll
  for (int nt = 0; nt < NT; ++nt)
    if (nt * 16 + col < ncol) mx = fmaxf(mx, g[nt]);
  mx = fmaxf(mx, __int_as_float(row_ror<8>(__float_as_int(mx))));
  mx = fmaxf(mx, __int_as_float(row_ror<4>(__float_as_int(mx))));
  mx = fmaxf(mx, __int_as_float(row_ror<2>(__float_as_int(mx))));
  mx = fmaxf(mx, __int_as_float(row_ror<1>(__float_as_int(mx))));
  float sm = 0.f;
#pragma unroll
  for (int nt = 0; nt < NT; ++nt)
    if (nt * 16 + col < ncol) sm += expf(g[nt] - mx);
  sm += __int_as_float(row_ror<8>(__float_as_int(sm)));
  sm += __int_as_float(row_ror<4>(__float_as_int(sm)));
  sm += __int_as_float(row_ror<2>(__float_as_int(sm)));
  sm += __int_as_float(row_ror<1>(__float_as_int(sm)));
  m = mx;
  z = sm;
}

// Top-k of groups h0 .. h1-1 and the routing weights of one token whose G*E
// scores sit in a 16-lane row (column nt*16 + col in g[nt], bias included).
// After each arg-max round every lane of the row holds the selection, so the
// softmax normaliser is summed as the selections come (slot order), and lane
// col keeps slot col's id and score for the write (k <= 16).  For k > 16 the
// slots go through sel_e / sel_v, this row's scratch in LDS (a wave's LDS
// operations complete in order, so the row reads back what its lane col == 0
// wrote).  Group h writes topk_*[(h*T + tok)*k + s]; with `hist` (LDS,
// [G*E]) every selected id is also counted there.
template <int NT>
__device__ __forceinline__ void select_token(const float (&g)[NT], int col, int E, int G, int h0,
                                             int h1, int k, int gating, int tok, int T_,
                                             int* sel_e, float* sel_v,
                                             int32_t* __restrict__ topk_idx,
                                             float* __restrict__ topk_w, int* hist) {
  const int Et = G * E;
  const bool global = gating == FOE_GATE_GLOBAL;
  // global gating: softmax over all G*E scores of the token, not
  // renormalised over the selection
  float gm = 0.f, gz = 1.f;
  if (global) row_softmax_norm<NT>(g, col, Et, gm, gz);
  const bool in_regs = k <= 16;
  for (int h = h0; h < h1; ++h) {
    // bit nt: column nt*16 + col outside group h or already selected
    unsigned taken = 0;
#pragma unroll
    for (int nt = 0; nt < NT; ++nt) {
      const int e = nt * 16 + col;
      if (e < h * E || e >= (h + 1) * E) taken |= 1u << nt;
    }
    float m = gm, z = global ? gz : 0.f;
    int my_e = -1;
    float my_v = 0.f;
    for (int s = 0; s < k; ++s) {
      float bv = -__builtin_inff();
      int be = 0x7fffffff;
#pragma unroll
      for (int nt = 0; nt < NT; ++nt) {
        const int e = nt * 16 + col;
        if (!((taken >> nt) & 1u) && beats(g[nt], e, bv, be)) { bv = g[nt]; be = e; }
      }
      argmax_step<8>(bv, be);
      argmax_step<4>(bv, be);
      argmax_step<2>(bv, be);
      argmax_step<1>(bv, be);
      if (be != 0x7fffffff && (be & 15) == col) taken |= 1u << (be >> 4);
      const int id = (be == 0x7fffffff) ? -1 : be - h * E;
      if (!global) {
        if (s == 0) m = bv;
        z += __expf(bv - m);
      }
      if (in_regs) {
        if (s == col) {
          my_e = id;
          my_v = bv;
        }
      } else if (col == 0) {
        sel_e[s] = id;
        sel_v[s] = bv;
      }
    }
    // weights: slot s = exp(score_s - m) / z; lane col writes slots col,
    // col+16, ...
    if (tok < T_) {
      const float inv = __builtin_amdgcn_rcpf(z);
      const size_t o = ((size_t)h * T_ + tok) * k;
      for (int s = col; s < k; s += 16) {
        const int id = in_regs ? my_e : sel_e[s];
        const float v = in_regs ? my_v : sel_v[s];
        topk_idx[o + s] = id;
        topk_w[o + s] = __expf(v - m) * inv;
        if (hist != nullptr && id >= 0) atomicAdd(&hist[h * E + id], 1);
      }
    }
  }
}

// select_token for NB independent (token, group) entries at once: entry b
// is the token whose scores are g[b] (register index of the 16-lane rows)
// and its group hg[b] (-1: none).  k <= 16 (slots in registers).  The NB
// arg-max chains are independent, so their rotation steps interleave instead
// of running one after another; each entry's results are those of
// select_token.
template <int NT, int NB>
__device__ __forceinline__ void select_batch(const float (&g)[NB][NT], const int (&hg)[NB],
                                             const int (&tok)[NB], int col, int E, int G, int k,
                                             int gating, int T_, int32_t* __restrict__ topk_idx,
                                             float* __restrict__ topk_w, int* hist) {
  const bool global = gating == FOE_GATE_GLOBAL;
  unsigned taken[NB];
  float m[NB], z[NB], my_v[NB];
  int my_e[NB];
#pragma unroll
  for (int b = 0; b < NB; ++b) {
    // bit nt: column nt*16 + col outside the entry's group or already taken
    taken[b] = 0;
#pragma unroll
    for (int nt = 0; nt < NT; ++nt) {
      const int e = nt * 16 + col;
      if (hg[b] < 0 || e < hg[b] * E || e >= (hg[b] + 1) * E) taken[b] |= 1u << nt;
    }
    m[b] = 0.f;
    z[b] = 1.f;
    // global gating: softmax over all G*E scores of the token, not
    // renormalised over the selection
    if (global) row_softmax_norm<NT>(g[b], col, G * E, m[b], z[b]);
    else z[b] = 0.f;
    my_e[b] = -1;
    my_v[b] = 0.f;
  }
  for (int s = 0; s < k; ++s) {
    float bv[NB];
    int be[NB];
#pragma unroll
    for (int b = 0; b < NB; ++b) {
      bv[b] = -__builtin_inff();
      be[b] = 0x7fffffff;
#pragma unroll
      for (int nt = 0; nt < NT; ++nt) {
        const int e = nt * 16 + col;
        if (!((taken[b] >> nt) & 1u) && beats(g[b][nt], e, bv[b], be[b])) {
          bv[b] = g[b][nt];
          be[b] = e;
        }
      }
    }
#pragma unroll
    for (int b = 0; b < NB; ++b) argmax_step<8>(bv[b], be[b]);
#pragma unroll
    for (int b = 0; b < NB; ++b) argmax_step<4>(bv[b], be[b]);
#pragma unroll
    for (int b = 0; b < NB; ++b) argmax_step<2>(bv[b], be[b]);
#pragma unroll
    for (int b = 0; b < NB; ++b) argmax_step<1>(bv[b], be[b]);
#pragma unroll
    for (int b = 0; b < NB; ++b) {
      if (be[b] != 0x7fffffff && (be[b] & 15) == col) taken[b] |= 1u << (be[b] >> 4);
      if (!global) {
        if (s == 0) m[b] = bv[b];
        z[b] += __expf(bv[b] - m[b]);
      }
      if (s == col) {
        my_e[b] = (be[b] == 0x7fffffff) ? -1 : be[b] - hg[b] * E;
        my_v[b] = bv[b];
      }
    }
  }
  // weights: slot s = exp(score_s - m) / z, written by lane col = s
#pragma unroll
  for (int b = 0; b < NB; ++b) {
    if (hg[b] >= 0 && tok[b] < T_ && col < k) {
      const size_t o = ((size_t)hg[b] * T_ + tok[b]) * k + col;
      topk_idx[o] = my_e[b];
      topk_w[o] = __expf(my_v[b] - m[b]) * __builtin_amdgcn_rcpf(z[b]);
      if (hist != nullptr && my_e[b] >= 0) atomicAdd(&hist[hg[b] * E + my_e[b]], 1);
    }
  }
}

// Per-workgroup expert counts (the dispatch histogram, folded in): counts
// [C][gridDim.x][E] of the workgroup's tokens, cluster = blockIdx.y * G + h.
__device__ __forceinline__ void write_counts(const int* hist, int G, int E,
                                             int32_t* __restrict__ counts) {
  for (int i = threadIdx.x; i < G * E; i += blockDim.x) {
    const int h = i / E, e = i % E;
    const size_t c = (size_t)blockIdx.y * G + h;
    counts[(c * gridDim.x + blockIdx.x) * E + e] = hist[i];
  }
}

template <typename T> struct RouteMma;

// bf16: each MFMA step consumes 32 k; lane (r = l%16, q = l/16) supplies
// x[r][kc + 8q .. +8) and W_r[e][same k] (the same k map on both operands).
// One W_r fragment serves the TG token groups of the workgroup.
template <> struct RouteMma<bf16> {
  static constexpr int KSTEP = 32;
  template <int NT, int NW, int TG, int KB>
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
    // wave w takes K-step groups w, w+NW, ... of KB steps each
    for (int c0 = wave * KB; c0 < nsteps; c0 += NW * KB) {
      u32x4 a[KB][TG], b[KB][NT];
#pragma unroll
      for (int u = 0; u < KB; ++u) {
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
      for (int u = 0; u < KB; ++u)
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
  template <int NT, int NW, int TG, int KB>
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
template <typename T, int NT, int NW, int TG, int KB>
__global__ __launch_bounds__(NW * 64) void route_kernel(const T* __restrict__ x,
                                                        const T* __restrict__ w,
                                                        const float* __restrict__ bias, int T_,
                                                        int d, int E, int k, int G, int gating,
                                                        int32_t* __restrict__ topk_idx,
                                                        float* __restrict__ topk_w,
                                                        int32_t* __restrict__ zcnt, int zn,
                                                        int32_t* __restrict__ counts) {
  constexpr int UPW = (4 * TG + NW - 1) / NW;  // units per wave
  // waves beyond the 4*TG units share the units' groups: wave w takes unit
  // w % (4*TG) and part w / (4*TG) of its G groups
  constexpr int PARTS = NW > 4 * TG ? NW / (4 * TG) : 1;
  static_assert(PARTS == 1 || NW % (4 * TG) == 0, "whole parts");
  extern __shared__ __align__(16) unsigned char smem[];
  // expert counts (with `counts`): G*E ints after the partial-score and
  // selection area (the launch sizes the dynamic LDS for both)
  int* hist = reinterpret_cast<int*>(
      smem + max((size_t)NW * TG * NT * kWave * sizeof(f32x4), (size_t)NW * 8 * k * 4));
  if (counts != nullptr)
    for (int i = threadIdx.x; i < G * E; i += NW * kWave) hist[i] = 0;
  // cluster blockIdx.y: its router matrix, bias and output rows.  With G > 1
  // groups in one workgroup, the G router matrices [G][E][d] are one score
  // matrix of G*E columns and each group's top-k is taken over its own block
  // of E columns (the output of group h goes to topk_*[h][T][k]).
  w += (size_t)blockIdx.y * E * d;
  if (bias != nullptr) bias += (size_t)blockIdx.y * E;
  topk_idx += (size_t)blockIdx.y * T_ * k;
  topk_w += (size_t)blockIdx.y * T_ * k;
  const int lane = lane_id();
  const int wave = threadIdx.x >> 6;
  const int t0 = blockIdx.x * kTok * TG;
  // counters of later kernels of the same block call, per token of this tile
  if (zcnt != nullptr && blockIdx.y == 0)
    for (int i = threadIdx.x; i < kTok * TG * zn; i += NW * kWave)
      if (t0 + i / zn < T_) zcnt[(size_t)t0 * zn + i] = 0;

  f32x4 acc[TG][NT];
#pragma unroll
  for (int g = 0; g < TG; ++g)
#pragma unroll
    for (int nt = 0; nt < NT; ++nt) acc[g][nt] = f32x4{0.f, 0.f, 0.f, 0.f};
  const int Et = G * E;  // score columns
  RouteMma<T>::template run<NT, NW, TG, KB>(x, w, T_, d, Et, t0, wave, lane, acc);

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
  const int my_unit = PARTS > 1 ? wave % (4 * TG) : wave, gpart = PARTS > 1 ? wave / (4 * TG) : 0;
#pragma unroll
  for (int u = 0; u < UPW; ++u) {
    const int unit = my_unit + u * NW;
    const int g = (unit >> 2) < TG ? (unit >> 2) : 0, i = unit & 3;
#pragma unroll
    for (int nt = 0; nt < NT; ++nt) {
      float s = 0.f;
      if (unit < 4 * TG) {
#pragma unroll
        for (int wv = 0; wv < NW; ++wv) s += part[((wv * TG + g) * NT + nt) * kWave + lane][i];
        const int e = nt * 16 + col;
        if (bias != nullptr && e < Et) s += bias[e];
      }
      gl[u][nt] = s;
    }
  }
  __syncthreads();  // partial tiles are dead; LDS is reused for the selection

  // per wave: the k selections of its 4 rows (one token per 16-lane row)
  int* sel_e = reinterpret_cast<int*>(smem) + wave * 8 * k;
  float* sel_v = reinterpret_cast<float*>(sel_e + 4 * k);
  const int row = lane >> 4;
  const int h0 = gpart * G / PARTS, h1 = (gpart + 1) * G / PARTS;
#pragma unroll
  for (int u = 0; u < UPW; ++u) {
    const int unit = my_unit + u * NW;
    if (unit >= 4 * TG) break;
    const int tok = t0 + (unit >> 2) * 16 + 4 * row + (unit & 3);
    if (k <= 16 && h1 - h0 > 1) {
      // the unit's groups four at a time
      for (int h = h0; h < h1; h += 4) {
        float g4[4][NT];
        int hg[4], tk[4];
#pragma unroll
        for (int b = 0; b < 4; ++b) {
          hg[b] = h + b < h1 ? h + b : -1;
          tk[b] = tok;
#pragma unroll
          for (int nt = 0; nt < NT; ++nt) g4[b][nt] = gl[u][nt];
        }
        select_batch<NT, 4>(g4, hg, tk, col, E, G, k, gating, T_, topk_idx, topk_w,
                            counts != nullptr ? hist : nullptr);
      }
    } else {
      select_token<NT>(gl[u], col, E, G, h0, h1, k, gating, tok, T_, sel_e + row * k,
                       sel_v + row * k, topk_idx, topk_w, counts != nullptr ? hist : nullptr);
    }
  }
  if (counts != nullptr) {
    __syncthreads();
    write_counts(hist, G, E, counts);
  }
}

// Many tokens, bf16, G*E <= 64: a workgroup of WPB waves takes 16 tokens per
// wave over all of K, so no partial scores are exchanged.  x and the G*E
// router rows stream through a ring of NS LDS stages of 128 K columns with
// LDS-DMA loads of 4 rows x 256 bytes (each wave loads its own token rows and
// a share of the router rows, which all waves of the workgroup use), the
// 16-byte chunk c of row r stored in slot c ^ (r & 15).  Each wave then
// selects every group's top-k of its tokens from its own accumulators.
template <int NT, int NS, int WPB>
__global__ __launch_bounds__(WPB * 64) void route_stream_kernel(
    const bf16* __restrict__ x, const bf16* __restrict__ w, const float* __restrict__ bias,
    int T_, int d, int E, int G, int k, int gating, int32_t* __restrict__ topk_idx,
    float* __restrict__ topk_w, int32_t* __restrict__ counts) {
  constexpr int XB = WPB * 4096;          // token rows of a stage (16 rows x 256 B per wave)
  constexpr int SB = XB + NT * 4096;      // + router rows (16 rows x 256 B per score tile)
  constexpr int WI = NT * 4 / WPB;        // router DMA instructions per wave and stage
  constexpr int NI = 4 + WI;              // DMA instructions per wave and stage
  static_assert(NT * 4 % WPB == 0, "even split of the router rows");
  static_assert(NS >= 2 && NI * (NS - 2) <= 63, "vmcnt range");
  static_assert(NS * SB + WPB * 8 * 64 * 4 + kMaxGE * 4 <= 160 * 1024, "LDS capacity");
  __shared__ __align__(1024) unsigned char smem[NS * SB];
  __shared__ int sel_buf[WPB][8 * 64];  // per row of 16 lanes: k ids, k scores (k <= 64)
  __shared__ int hist[kMaxGE];
  const int Et = G * E;  // score columns
  for (int i = threadIdx.x; i < Et; i += WPB * kWave) hist[i] = 0;

  // cluster blockIdx.y (G == 1): its router matrix, bias and output rows
  w += (size_t)blockIdx.y * E * d;
  if (bias != nullptr) bias += (size_t)blockIdx.y * E;
  topk_idx += (size_t)blockIdx.y * T_ * k;
  topk_w += (size_t)blockIdx.y * T_ * k;
  const int lane = lane_id();
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int t0 = (blockIdx.x * WPB + wave) * 16;  // this wave's tokens
  // the bias of this lane's score columns, read before the K loop (read after
  // it, its latency would follow the loop)
  float bias_r[NT];
#pragma unroll
  for (int nt = 0; nt < NT; ++nt) {
    const int e = nt * 16 + (lane & 15);
    bias_r[nt] = (bias != nullptr && e < Et) ? bias[e] : 0.f;
  }
  const uint32_t lds0 = lds_addr(smem);
  const __amdgpu_buffer_rsrc_t xr = make_rsrc_u(x, (uint32_t)T_ * d * 2u);
  const __amdgpu_buffer_rsrc_t wr = make_rsrc_u(w, (uint32_t)Et * d * 2u);
  const int lr = lane >> 4, lc = lane & 15;
  // token instruction i (rows t0+4i..) and router instruction wave*WI + j
  uint32_t xv[4], wv[WI];
  int xk[4], wk[WI];
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const int r = 4 * i + lr;  // row in the 16-token tile
    const int q = lc ^ (r & 15);
    xk[i] = q * 8;
    xv[i] = t0 + r < T_ ? ((uint32_t)(t0 + r) * d + q * 8) * 2u : kOob;
  }
#pragma unroll
  for (int j = 0; j < WI; ++j) {
    const int e = 4 * (wave * WI + j) + lr;  // router row
    const int q = lc ^ (e & 15);
    wk[j] = q * 8;
    wv[j] = e < Et ? ((uint32_t)e * d + q * 8) * 2u : kOob;
  }
  const int nks = (d + 127) / 128;
  auto issue = [&](int kt, int s) {
    const int k0 = kt * 128;
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const uint32_t off = (k0 + xk[i] < d && xv[i] != kOob) ? xv[i] + (uint32_t)k0 * 2u : kOob;
      dma16(xr, off, lds0 + wave * 4096, s * SB + i * 1024);
    }
#pragma unroll
    for (int j = 0; j < WI; ++j) {
      const uint32_t off = (k0 + wk[j] < d && wv[j] != kOob) ? wv[j] + (uint32_t)k0 * 2u : kOob;
      dma16(wr, off, lds0 + wave * WI * 1024, s * SB + XB + j * 1024);
    }
  };
  const int R = lane & 15, g = lane >> 4;
  const int rbase = (R >> 2) * 1024 + (R & 3) * 256;
  f32x4 acc[NT];
#pragma unroll
  for (int nt = 0; nt < NT; ++nt) acc[nt] = f32x4{0.f, 0.f, 0.f, 0.f};
  auto body = [&](int kt, int s, int s_next) {
    if (kt + NS - 2 < nks) vm_wait<NI * (NS - 2)>();
    else vm_wait<0>();
    lds_barrier();
    if (kt + NS - 1 < nks) issue(kt + NS - 1, s_next);
    const unsigned char* src = smem + s * SB + rbase;
#pragma unroll
    for (int c = 0; c < 4; ++c) {
      const int slot = ((c * 4 + g) ^ R) * 16;
      const bf16x8 xa = *reinterpret_cast<const bf16x8*>(src + wave * 4096 + slot);
#pragma unroll
      for (int nt = 0; nt < NT; ++nt) {
        const bf16x8 wb = *reinterpret_cast<const bf16x8*>(src + XB + nt * 4096 + slot);
        acc[nt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(xa, wb, acc[nt], 0, 0, 0);
      }
    }
  };
#pragma unroll
  for (int s = 0; s < NS - 1; ++s)
    if (s < nks) issue(s, s);
  for (int kt0 = 0; kt0 < nks; kt0 += NS) {
#pragma unroll
    for (int u = 0; u < NS; ++u) {
      const int kt = kt0 + u;
      if (kt < nks) body(kt, u, (u + NS - 1) % NS);
    }
  }

  // accumulator register i holds token t0 + 4*(lane/16) + i (one per 16-lane
  // row) and score columns nt*16 + lane%16
  const int col = lane & 15, row = lane >> 4;
  int* sel_e = sel_buf[wave] + row * 2 * k;
  float* sel_v = reinterpret_cast<float*>(sel_e + k);
  float gl[4][NT];
  int tok[4];
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    tok[i] = t0 + 4 * row + i;
#pragma unroll
    for (int nt = 0; nt < NT; ++nt) gl[i][nt] = acc[nt][i] + bias_r[nt];
  }
  if (k <= 16) {
    for (int h = 0; h < G; ++h) {
      const int hg[4] = {h, h, h, h};
      select_batch<NT, 4>(gl, hg, tok, col, E, G, k, gating, T_, topk_idx, topk_w,
                          counts != nullptr ? hist : nullptr);
    }
  } else {
#pragma unroll
    for (int i = 0; i < 4; ++i)
      select_token<NT>(gl[i], col, E, G, 0, G, k, gating, tok[i], T_, sel_e, sel_v, topk_idx,
                       topk_w, counts != nullptr ? hist : nullptr);
  }
  if (counts != nullptr) {
    __syncthreads();
    write_counts(hist, G, E, counts);
  }
}

// C clusters as G groups of every workgroup (G = C) or one per grid row (G = 1)
template <typename T, int NT, int NW, int TG, int KB = kBatch>
hipError_t launch_nt(int C, int G, int T_, int d, int E, int k, int gating, const void* x,
                     const void* w, const float* bias, int32_t* idx, float* wt, hipStream_t s,
                     int32_t* zcnt, int zn, int32_t* counts) {
  size_t lds_red = (size_t)NW * TG * NT * kWave * sizeof(f32x4);
  size_t lds_sel = (size_t)NW * 8 * k * 4;
  size_t lds = (lds_red > lds_sel ? lds_red : lds_sel) + (counts != nullptr ? G * E * 4 : 0);
  dim3 grid(ceil_div(T_, kTok * TG), C / G);
  ProfileScope ps("route", s);
  FOE_LAUNCH((route_kernel<T, NT, NW, TG, KB>), grid, dim3(NW * kWave), lds, s,
             reinterpret_cast<const T*>(x), reinterpret_cast<const T*>(w), bias, T_, d, E, k, G,
             gating, idx, wt, zcnt, zn, counts);
  return hipGetLastError();
}

// (token groups per workgroup, waves) for many tokens: token groups share each
// router-weight fragment (otherwise the weights are read once per 16 tokens,
// more bytes than x itself at E = 32); few tokens: 8 waves split K of one
// 16-token group (more loads in flight per token).  Large E: 4 waves.
template <int TG_, int NW_> struct RouteCfg {
  static constexpr int TG = TG_, NW = NW_;
};
#ifndef FOE_ROUTE_STREAM
#define FOE_ROUTE_STREAM 1
#endif
// streaming kernel from this many tokens (two 16-token waves per CU or more)
#ifndef FOE_ROUTE_STREAM_MIN_T
#define FOE_ROUTE_STREAM_MIN_T 8192
#endif
// streaming kernel: waves per workgroup by token count (>= 16384, >= 8192,
// fewer) and LDS ring stages
#ifndef FOE_ROUTE_WPB_L
#define FOE_ROUTE_WPB_L 4
#endif
#ifndef FOE_ROUTE_WPB_M
#define FOE_ROUTE_WPB_M 2
#endif
#ifndef FOE_ROUTE_WPB_S
#define FOE_ROUTE_WPB_S 1
#endif
#ifndef FOE_ROUTE_NS
#define FOE_ROUTE_NS 4
#endif
#ifndef FOE_ROUTE_SMALL_NW
#define FOE_ROUTE_SMALL_NW 8
#endif
#ifndef FOE_ROUTE_TG16
#define FOE_ROUTE_TG16 1, 8
#endif
#ifndef FOE_ROUTE_TG32
#define FOE_ROUTE_TG32 2, 8
#endif
#ifndef FOE_ROUTE_TG64
#define FOE_ROUTE_TG64 1, 8
#endif

template <int NT, int WPB>
hipError_t launch_stream_nt(int C, int G, int T_, int d, int E, int k, int gating, const void* x,
                            const void* w, const float* bias, int32_t* idx, float* wt,
                            int32_t* counts, hipStream_t s) {
  // as many ring stages as the LDS holds, up to FOE_ROUTE_NS
  // (and as the vmcnt field can count: NI * (NS - 2) <= 63 loads in flight)
  constexpr int SB = (WPB + NT) * 4096;
  constexpr int NI = 4 + NT * 4 / WPB;
  constexpr int NS_FIT = (150 * 1024) / SB, NS_VM = 2 + 63 / NI;
  constexpr int NS_MAX = NS_FIT < NS_VM ? NS_FIT : NS_VM;
  constexpr int NS = NS_MAX < FOE_ROUTE_NS ? NS_MAX : FOE_ROUTE_NS;
  dim3 grid(ceil_div(T_, 16 * WPB), C / G);
  FOE_LAUNCH((route_stream_kernel<NT, NS, WPB>), grid, dim3(WPB * kWave), 0, s,
             reinterpret_cast<const bf16*>(x), reinterpret_cast<const bf16*>(w), bias, T_, d,
             E, G, k, gating, idx, wt, counts);
  return hipGetLastError();
}

template <int WPB>
hipError_t launch_stream(int C, int G, int T_, int d, int E, int k, int gating, const void* x,
                         const void* w, const float* bias, int32_t* idx, float* wt,
                         int32_t* counts, hipStream_t s) {
  ProfileScope ps("route", s);
  const int Et = G * E;
  if (Et <= 16)
    return launch_stream_nt<1, WPB>(C, G, T_, d, E, k, gating, x, w, bias, idx, wt, counts, s);
  if (Et <= 32)
    return launch_stream_nt<2, WPB>(C, G, T_, d, E, k, gating, x, w, bias, idx, wt, counts, s);
  return launch_stream_nt<4, WPB>(C, G, T_, d, E, k, gating, x, w, bias, idx, wt, counts, s);
}

template <typename T>
hipError_t launch_t(const RoutePlan& p, int C, int T_, int d, int E, int k, int gating,
                    const void* x, const void* w, const float* bias, int32_t* idx, float* wt,
                    hipStream_t s, int32_t* zcnt, int zn, int32_t* counts) {
  const int G = p.G;
  const int Et = G * E;
  if constexpr (sizeof(T) == 2) {
    if (p.stream) {
      if (p.wpb == 4)
        return launch_stream<4>(C, G, T_, d, E, k, gating, x, w, bias, idx, wt, counts, s);
      if (p.wpb == 2)
        return launch_stream<2>(C, G, T_, d, E, k, gating, x, w, bias, idx, wt, counts, s);
      return launch_stream<1>(C, G, T_, d, E, k, gating, x, w, bias, idx, wt, counts, s);
    }
  }
  const bool many = T_ >= 2048;
  if (Et <= 16)
    return many ? launch_nt<T, 1, RouteCfg<FOE_ROUTE_TG16>::NW, RouteCfg<FOE_ROUTE_TG16>::TG>(
                      C, G, T_, d, E, k, gating, x, w, bias, idx, wt, s, zcnt, zn, counts)
                : launch_nt<T, 1, FOE_ROUTE_SMALL_NW, 1>(C, G, T_, d, E, k, gating, x, w, bias,
                                                          idx, wt, s, zcnt, zn, counts);
  if (Et <= 32)
    return many ? launch_nt<T, 2, RouteCfg<FOE_ROUTE_TG32>::NW, RouteCfg<FOE_ROUTE_TG32>::TG>(
                      C, G, T_, d, E, k, gating, x, w, bias, idx, wt, s, zcnt, zn, counts)
                : launch_nt<T, 2, FOE_ROUTE_SMALL_NW, 1>(C, G, T_, d, E, k, gating, x, w, bias,
                                                          idx, wt, s, zcnt, zn, counts);
  if (Et <= 64)
    return many ? launch_nt<T, 4, RouteCfg<FOE_ROUTE_TG64>::NW, RouteCfg<FOE_ROUTE_TG64>::TG>(
                      C, G, T_, d, E, k, gating, x, w, bias, idx, wt, s, zcnt, zn, counts)
                : launch_nt<T, 4, 8, 1>(C, G, T_, d, E, k, gating, x, w, bias, idx, wt, s, zcnt,
                                        zn, counts);
  if (Et <= 128)
    return launch_nt<T, 8, 4, 1>(C, G, T_, d, E, k, gating, x, w, bias, idx, wt, s, zcnt, zn,
                                 counts);
  return launch_nt<T, 16, 4, 1>(C, G, T_, d, E, k, gating, x, w, bias, idx, wt, s, zcnt, zn,
                                counts);
}

}  // namespace

RoutePlan plan_route(foe_dtype dt, int C, int T, int d, int E, bool zero_counters) {
  RoutePlan p;
  // several clusters: one pass over x scores all C*E experts (the router
  // matrices are contiguous) and each cluster takes its top-k from its block
  p.G = (C > 1 && C * E <= 256) ? C : 1;
  const int Et = p.G * E;
  // buffer offsets are 32-bit: x must span less than 2 GiB
  p.stream = FOE_ROUTE_STREAM && dt == FOE_BF16 && !zero_counters &&
             T >= FOE_ROUTE_STREAM_MIN_T && Et <= 64 && (size_t)T * d * 2 < ((size_t)1 << 31);
  p.wpb = T >= 16384 ? FOE_ROUTE_WPB_L : T >= 8192 ? FOE_ROUTE_WPB_M : FOE_ROUTE_WPB_S;
  if (p.stream) {
    p.tok_per_blk = 16 * p.wpb;
  } else {
    const bool many = T >= 2048;
    int tg = 1;
    if (many && Et <= 16) tg = RouteCfg<FOE_ROUTE_TG16>::TG;
    else if (many && Et <= 32) tg = RouteCfg<FOE_ROUTE_TG32>::TG;
    else if (many && Et <= 64) tg = RouteCfg<FOE_ROUTE_TG64>::TG;
    p.tok_per_blk = kTok * tg;
  }
  p.nblk = ceil_div(T, p.tok_per_blk);
  return p;
}

hipError_t launch_route(foe_dtype dt, int C, int T, int d, int E, int k, int gating,
                        const void* x, const void* w_router, const float* bias,
                        int32_t* topk_idx, float* topk_w, hipStream_t s, int32_t* zero_cnt,
                        int zero_per_tok, int32_t* counts) {
  if (T == 0 || C == 0) return hipSuccess;
  const RoutePlan p = plan_route(dt, C, T, d, E, zero_cnt != nullptr);
  if (dt == FOE_BF16)
    return launch_t<bf16>(p, C, T, d, E, k, gating, x, w_router, bias, topk_idx, topk_w, s,
                          zero_cnt, zero_per_tok, counts);
  return launch_t<float>(p, C, T, d, E, k, gating, x, w_router, bias, topk_idx, topk_w, s,
                         zero_cnt, zero_per_tok, counts);
}

}  // namespace foe
