// Per-group attention that feeds the block (Table 3, FoE column, rows "Attn.
// residual" and "Cross-group avg."): every group h keeps its own
// representation x[h] and runs causal attention over it with its own KV head
// and nq query heads sharing it (grouped-query attention); the results are
// averaged over the groups:
//   r[h, i]    = x[h, i] + Attn_h(x[h, :])[i]
//   r_full[i]  = (1/H) sum_h r[h, i]
// Launches: the q/k/v projection of every group (one grouped GEMM with a
// segment per group), a preparation pass (rotary embedding of q and k in
// place, value head transposed), the attention (o as [S][H*nq*hd]) with the
// residual sum sum_h x[h] beside it on a side stream, and the output
// projection of all groups as one GEMM over K = H*nq*hd whose epilogue adds
// that sum and scales by 1/H, so the per-group outputs never reach memory.
// The kernels below describe their layouts.
#include <mutex>

#include "foe_common.hpp"
#include "lds_dma.hpp"

namespace foe {
namespace {

// head dimensions the kernels are built for: 128 (the 7B model) and 96 (the
// 1B model); a K tile row is 256 bytes either way (dims past hd read zeros)
constexpr int kHdMax = 128;
constexpr int kQB = 64;   // queries per workgroup and head
constexpr int kKB = 64;   // keys per block of the V^T layout (its zero padding)
// floor of the running maximum (log2 units): finite, and far below any score
constexpr float kMFloor = -1.0e30f;

// Attention inner step: fragment reads in flight ahead of the score and P V
// MFMAs, and vector instructions placed after each P V MFMA; FOE_ATT_SGB 0
// leaves the order to the compiler.
#ifndef FOE_ATT_KW
#define FOE_ATT_KW 4
#endif
#ifndef FOE_ATT_VPM
#define FOE_ATT_VPM 8
#endif
#ifndef FOE_ATT_SGB
#define FOE_ATT_SGB 1
#endif

// ---- preparation pass ----------------------------------------------------------
// One workgroup per (64-row block, group).  (1) Rotary embedding of the q and
// k heads in place: each angle (s / scale) * theta^(-2i/HD) is formed once,
// in double, reduced modulo 2*pi, and rotates the pair (i, i + HD/2) of every q
// head and of the k head (a thread takes 4 consecutive pairs of a row, 8-byte
// accesses).  (2) The value head
// transposed to vt[group][dim][key] (keys padded to s_pad with zeros), with
// the keys of each 16-key group stored in the order 0-3, 8-11, 4-7, 12-15
// (bits 2 and 3 swapped): that is the key order of the probabilities a lane
// holds as its B operand, so one 16-byte read gives its V^T operand.
__device__ __forceinline__ int vt_perm(int key) {
  return (key & ~12) | ((key & 4) << 1) | ((key & 8) >> 1);
}

template <int HD>
__global__ __launch_bounds__(256) void prep_kernel(bf16* __restrict__ qkv, bf16* __restrict__ vt,
                                                   int S, int s_pad, int nq, double theta,
                                                   double scale) {
  constexpr int CPR = HD / 8;  // 16-byte chunks of a head row
  constexpr int PPT = CPR / 4; // value pieces per thread (64 keys x CPR chunks)
  __shared__ double inv_freq[HD / 2];
  // V^T tile [HD dims][64 keys], 128-byte rows; 16-byte chunk cc of row dim
  // in slot cc ^ ((dim >> 3) & 7), so that the 2-byte writes of the 16 lanes
  // holding one key spread over 8 chunks
  __shared__ __align__(16) bf16 vtile[HD * kKB];
  const int tid = threadIdx.x;
  const int blk = blockIdx.x, grp = blockIdx.y;
  const size_t ld = (size_t)(nq + 2) * HD;
  bf16* base = qkv + (size_t)grp * S * ld;
  if (tid < HD / 2) inv_freq[tid] = pow(theta, -2.0 * tid / HD);

  // the value rows of the block: piece p = tid + 256 m is key p / CPR, dims
  // 8 (p % CPR) .. +8 (loads go out before the rotation work)
  bf16x8 vv[PPT];
#pragma unroll
  for (int m = 0; m < PPT; ++m) {
    const int p = tid + 256 * m;
    const int s = blk * kKB + p / CPR;
    vv[m] = s < S ? *reinterpret_cast<const bf16x8*>(base + (size_t)s * ld +
                                                     (size_t)(nq + 1) * HD + (p % CPR) * 8)
                  : bf16x8{};
  }
  __syncthreads();

  // rotary embedding: thread (row rs, pairs 4u .. 4u+3) for rows rs + 16 j;
  // 8-byte accesses, a wave covers 4 rows per instruction (threads with
  // 4u >= HD/2 have no pairs)
  const int u = tid & 15, rs = tid >> 4;
  constexpr double kTwoPi = 6.283185307179586476925286766559;
  for (int j = 0; j < kQB / 16 && 4 * u < HD / 2; ++j) {
    const int s = blk * kQB + rs + 16 * j;
    if (s >= S) break;
    float cs[4], sn[4];
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      double a = (double)s / scale * inv_freq[4 * u + e];
      a -= kTwoPi * floor(a / kTwoPi);
      sincosf((float)a, &sn[e], &cs[e]);
    }
    bf16* row = base + (size_t)s * ld + 4 * u;
    for (int h = 0; h <= nq; ++h) {
      bf16x4* lo = reinterpret_cast<bf16x4*>(row + (size_t)h * HD);
      bf16x4* hi = reinterpret_cast<bf16x4*>(row + (size_t)h * HD + HD / 2);
      const bf16x4 x1 = *lo, x2 = *hi;
      bf16x4 y1, y2;
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        const float a1 = (float)x1[e], a2 = (float)x2[e];
        y1[e] = (bf16)(a1 * cs[e] - a2 * sn[e]);
        y2[e] = (bf16)(a2 * cs[e] + a1 * sn[e]);
      }
      *lo = y1;
      *hi = y2;
    }
  }

  // V^T through LDS
#pragma unroll
  for (int m = 0; m < PPT; ++m) {
    const int p = tid + 256 * m;
    const int c = p % CPR;
    const int pk = vt_perm(p / CPR);
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      const int dim = c * 8 + e;
      vtile[dim * kKB + (((pk >> 3) ^ ((dim >> 3) & 7)) << 3) + (pk & 7)] = vv[m][e];
    }
  }
  __syncthreads();
  bf16* dst = vt + (size_t)grp * HD * s_pad + (size_t)blk * kKB;
#pragma unroll
  for (int m = 0; m < HD / 32; ++m) {  // HD rows x 8 chunks
    const int p = tid + 256 * m;
    const int dim = p >> 3, cc = p & 7;
    *reinterpret_cast<bf16x8*>(dst + (size_t)dim * s_pad + cc * 8) =
        *reinterpret_cast<const bf16x8*>(&vtile[dim * kKB + ((cc ^ ((dim >> 3) & 7)) << 3)]);
  }
}

// ---- attention ----------------------------------------------------------------
// Task: 64 queries of NH query heads of one group (the heads share the
// group's key/value head and so its LDS tiles).  A workgroup of 8 waves has
// NP parts of 2*NH waves; wave (part, head hh, query half qw) holds 32
// queries.  The parts split the task's key blocks (part p takes blocks p,
// p + NP, ...) and merge their partial softmax states through LDS at the end,
// so that every running workgroup keeps two waves on each SIMD however short
// its task: two heads per task use 2 parts of 64-key blocks, one head (nq
// odd) 4 parts of 32-key blocks.  Tasks are numbered longest first; with one
// workgroup per compute unit the dispatcher hands the next task to the first
// unit that frees up, which balances the causal walks.
// Each part streams its key blocks (KB keys) through its own 2-stage LDS
// rings filled by LDS-DMA:
//   K tile   [KB keys][128 dims], 256-byte rows, 16-byte chunk c in slot
//            c ^ (key & 15) (at HD = 96 the chunks past the head hold zeros);
//   V^T tile [HD dims][KB keys], 2 KB-byte rows, chunk c in slot c ^ swz(dim).
// Scores come out transposed, S^T = K Q^T (v_mfma_f32_32x32x16_bf16, A = K
// rows, B = Q^T held in registers): lane l holds 32 scores of query l%32, at
// keys 32t + 8(v/4) + 4(l/32) + v%4 of tile t.  Its 8 scores of key step u
// (16 keys) are directly the B operand of O^T += V^T P^T, whose A operand
// reads the V^T tile in the same key order (the permuted layout written by
// the preparation pass).
// Software pipeline: an iteration computes the scores of its block, then the
// P V product of the part's previous block while the softmax of the new block
// runs on the vector ALUs (independent instructions, interleaved); the K ring
// runs one block ahead, the V ring one block behind.
// Online softmax in base 2 with a lazily updated maximum: the running maximum
// m moves only when a block's maximum exceeds it by more than 8 (units of
// log2), so probabilities stay below 2^8 and the accumulators are rescaled
// only on those (wave-uniform) steps; the final O / l cancels m exactly.
// Masking (causal, and keys past S) runs only on the blocks that need it.
template <int NH, int HD, int NP>
__global__ __launch_bounds__(NP * NH * 128) __attribute__((amdgpu_waves_per_eu(2, 2))) void attn_fwd_kernel(
    const bf16* __restrict__ qkv, const bf16* __restrict__ vt, int S, int s_pad, int nq, int H,
    float c_log2, bf16* __restrict__ out) {
  constexpr int KB = 128 / NP;          // keys per block (64 with 2 parts, 32 with 4)
  constexpr int HW = 2 * NH;            // waves per part
  constexpr int KT = KB * kHdMax * 2;   // K tile bytes (256-byte rows)
  constexpr int VT = HD * KB * 2;       // V^T tile bytes (rows of 2 KB bytes)
  constexpr int VC = KB / 8;            // 16-byte chunks of a V^T row
  constexpr int NST = HD / 16;          // score k-steps (16 dims each)
  constexpr int NDT = HD / 32;          // output tiles (32 dims each)
  constexpr int NSC = KB / 32;          // score tiles per block (32 keys each)
  constexpr int NKS = KB / 16;          // P V key steps per block
  constexpr int PART = 2 * KT + 2 * VT; // LDS bytes per part
  constexpr int KI = KT / 1024 / HW;    // DMA instructions per wave and tile
  constexpr int VI = VT / 1024 / HW;
  static_assert(HD == 96 || HD == 128, "head dimension");
  static_assert((NP == 2 || NP == 4) && NP * NH * 2 == 8, "8 waves: 2 parts x 2 heads or 4 x 1");
  static_assert(KT % (1024 * HW) == 0 && VT % (1024 * HW) == 0, "DMA splits evenly over the waves");
  static_assert((NP - 1) * HW * 64 * (HD / 2 + 2) * 4 <= NP * PART, "merge buffers fit in the rings");
  __shared__ __align__(1024) unsigned char smem[NP * PART];

  const int tid = threadIdx.x;
  const int lane = lane_id();
  const int wave = tid >> 6;
  const int part = wave / HW;        // key blocks part, part + NP, ...
  const int hw = wave % HW;          // wave within its part
  const int hw_u = __builtin_amdgcn_readfirstlane(hw);
  const int part_u = __builtin_amdgcn_readfirstlane(part);
  const int nqb = (S + kQB - 1) / kQB;
  const int hgs = nq / NH;
  const int P = hgs * H;
  const int r = blockIdx.x;
  const int qb = nqb - 1 - r / P;    // longest walks first
  const int rest = r % P;
  const int grp = rest / hgs;
  const int head = (rest % hgs) * NH + (hw >> 1);
  const size_t ld = (size_t)(nq + 2) * HD;
  const bf16* gbase = qkv + (size_t)grp * S * ld;
  const int q0 = qb * kQB + (hw & 1) * 32;  // this wave's first query
  const int qi = lane & 31, hl = lane >> 5;
  const int q = q0 + qi;

  // Q^T fragments: query q, dims 16 st + 8 hl + [0, 8)
  bf16x8 qf[NST];
  {
    const bf16* qrow = gbase + (size_t)min(q, S - 1) * ld + (size_t)head * HD + hl * 8;
#pragma unroll
    for (int st = 0; st < NST; ++st) {
      qf[st] = *reinterpret_cast<const bf16x8*>(qrow + st * 16);
      if (q >= S) qf[st] = bf16x8{};
    }
  }
  // The fragments must have arrived before the loop: the compiler would
  // otherwise wait for them (vmcnt(0)) inside the loop, which also waits for
  // the LDS-DMA of the next block issued there.
#pragma unroll
  for (int st = 0; st < NST; ++st) asm volatile("" ::"v"(qf[st]));

  // DMA: K instruction g = hw*KI + i fills key rows 4g .. 4g+3 (lane ->
  // row 4g + lane/16, slot lane%16); V^T instruction g fills the 64 / VC dim
  // rows from g*64/VC (lane -> row g*64/VC + lane/VC, slot lane%VC).  Keys past S read zeros
  // (the K range ends at the group's last row; V^T is zero-padded).
  const __amdgpu_buffer_rsrc_t rk =
      make_rsrc_u(gbase + (size_t)nq * HD, (uint32_t)(((size_t)S * ld - (size_t)nq * HD) * 2));
  const __amdgpu_buffer_rsrc_t rv =
      make_rsrc_u(vt + (size_t)grp * HD * s_pad, (uint32_t)((size_t)HD * s_pad * 2));
  uint32_t koff[KI], voff[VI];
#pragma unroll
  for (int i = 0; i < KI; ++i) {
    const int row = 4 * (hw * KI + i) + (lane >> 4);
    const int chunk = (lane & 15) ^ (row & 15);
    // chunks past the head (HD < 128) read zeros and are never used
    koff[i] = chunk < HD / 8 ? (uint32_t)((size_t)row * ld * 2) + (uint32_t)(chunk << 4) : kOob;
  }
#pragma unroll
  for (int i = 0; i < VI; ++i) {
    const int row = (64 / VC) * (hw * VI + i) + lane / VC;
    voff[i] = (uint32_t)row * s_pad * 2u + (uint32_t)(((lane % VC) ^ swz<VC>(row)) << 4);
  }
  unsigned char* hs = smem + part * PART;  // this part's rings
  const uint32_t hbase = lds_addr(smem) + (uint32_t)part_u * PART;
  // the part's i-th block (key block NP i + part) -> K stage i&1 (bytes
  // [0, 2 KT)), V^T stage i&1 (bytes [2 KT, 2 KT + 2 VT))
  auto issue_k = [&](int i) {
    const uint32_t kstep = (uint32_t)(NP * i + part) * KB * (uint32_t)ld * 2u;
    const uint32_t lk = hbase + (uint32_t)(i & 1) * KT + (uint32_t)hw_u * KI * 1024;
#pragma unroll
    for (int j = 0; j < KI; ++j) dma16(rk, koff[j] + kstep, lk, j * 1024);
  };
  auto issue_v = [&](int i) {
    const uint32_t lv = hbase + 2 * KT + (uint32_t)(i & 1) * VT + (uint32_t)hw_u * VI * 1024;
    const uint32_t vstep = (uint32_t)(NP * i + part) * KB * 2u;
#pragma unroll
    for (int j = 0; j < VI; ++j) dma16(rv, voff[j] + vstep, lv, j * 1024);
  };
  auto pv = [&](f32x16* oacc, const bf16x8* pf, const unsigned char* vs) {
#pragma unroll
    for (int dt = 0; dt < NDT; ++dt) {
      const int row = dt * 32 + qi;
#pragma unroll
      for (int u = 0; u < NKS; ++u) {
        const bf16x8 vf = *reinterpret_cast<const bf16x8*>(vs + row * (KB * 2) +
                                                           (((u * 2 + hl) ^ swz<VC>(row)) << 4));
        oacc[dt] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(vf, pf[u], oacc[dt], 0, 0, 0);
      }
    }
  };

  f32x16 oacc[NDT];
#pragma unroll
  for (int t = 0; t < NDT; ++t)
#pragma unroll
    for (int v = 0; v < 16; ++v) oacc[t][v] = 0.f;
  // running maximum of query q, scaled (log2 units); it starts at a finite
  // floor so that a row whose keys in a block are all masked (possible in a
  // part's first block with 32-key blocks) gets p = 2^-inf = 0, not NaN
  float m_run = kMFloor;
  float l_run = 0.f;                // this lane's share of the running sum
  float alpha = 1.f;                // rescale owed to oacc before the next P V
  bool resc = false;                // (wave-uniform) some lane owes a rescale
  bf16x8 pf[NKS];                   // probabilities of the previous block (B operand)
#pragma unroll
  for (int u = 0; u < NKS; ++u) pf[u] = bf16x8{};
  // P V steps with P = 0 (the first iteration, and the last one of a part
  // left without a block) may read a V stage no DMA has filled: zero both
  // stages of every part so that they add exact zeros
  for (int i = tid; i < NP * 2 * (VT / 16); i += NP * NH * 128) {
    const int h = i / (2 * (VT / 16)), c = i % (2 * (VT / 16));
    *reinterpret_cast<u32x4*>(smem + h * PART + 2 * KT + c * 16) = u32x4{0u, 0u, 0u, 0u};
  }

  const int nkb = min((qb + 1) * (kQB / KB), (S + KB - 1) / KB);
  const int niter = (nkb + NP - 1) / NP;  // every part runs the same iterations
  if (part < nkb) issue_k(0);
  // One key block of a part, in two stretches of branch-free code (scheduling
  // regions) with the masking between them, on the blocks that reach the
  // causal diagonal or the end of the sequence (`masked`, wave-uniform):
  //   scores S^T = K Q^T, the K fragment reads KW ahead of the MFMAs and the
  //   first V^T reads behind them;
  //   O^T += V^T P^T of the previous block, each MFMA followed by one V^T read
  //   and a share of the softmax of this block (maximum, exponentials,
  //   packing, row sums), written to fresh registers that become P afterwards,
  //   so that the vector ALUs work while the MFMAs run.
  // (The masked and unmasked steps as two compiled copies, one region each,
  // needed 256 registers at HD = 128 and ran slower.)
  auto block_step = [&](bool masked, const unsigned char* ks, const unsigned char* vs,
                        int kbase) {
    constexpr int NS = NST * NSC;   // score MFMAs, st-major
    constexpr int NV = NKS * NDT;   // P V MFMAs, u-major
    constexpr int KW = FOE_ATT_KW;  // K fragment reads in flight
    constexpr int VW = KW;          // V^T fragment reads in flight
    static_assert(KW <= NS && VW <= NV, "reads in flight within one step");
    f32x16 sacc[NSC];
#pragma unroll
    for (int t = 0; t < NSC; ++t)
#pragma unroll
      for (int v = 0; v < 16; ++v) sacc[t][v] = 0.f;
    bf16x8 kf[NS];
    auto kread = [&](int j) {
      const int st = j / NSC, t = j % NSC, row = t * 32 + qi;
      kf[j] = *reinterpret_cast<const bf16x8*>(ks + row * 256 + (((st * 2 + hl) ^ (row & 15)) << 4));
    };
    bf16x8 vf[NV];
    auto vread = [&](int j) {
      const int u = j / NDT, dt = j % NDT, row = dt * 32 + qi;
      vf[j] = *reinterpret_cast<const bf16x8*>(vs + row * (KB * 2) +
                                               (((u * 2 + hl) ^ swz<VC>(row)) << 4));
    };
#pragma unroll
    for (int j = 0; j < KW; ++j) kread(j);
#pragma unroll
    for (int j = 0; j < NS; ++j) {
      if (j + KW < NS) kread(j + KW);
      else vread(j + KW - NS);
      sacc[j % NSC] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(kf[j], qf[j / NSC], sacc[j % NSC], 0, 0, 0);
    }
#if FOE_ATT_SGB
#pragma unroll
    for (int j = 0; j < KW; ++j) __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);  // DS read
#pragma unroll
    for (int j = 0; j < NS; ++j) {
      __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);  // MFMA
      __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);
    }
#endif
    if (masked) {
#pragma unroll
      for (int t = 0; t < NSC; ++t)
#pragma unroll
        for (int v = 0; v < 16; ++v) {
          const int key = kbase + t * 32 + (v >> 2) * 8 + hl * 4 + (v & 3);
          if (key > q || key >= S) sacc[t][v] = -__builtin_inff();
        }
    }
    // softmax of this block: maximum over the row's keys (the two lane halves
    // hold the two key halves of the same queries)
    float mx = sacc[0][0];
#pragma unroll
    for (int t = 0; t < NSC; ++t)
#pragma unroll
      for (int v = 0; v < 16; ++v) mx = fmaxf(mx, sacc[t][v]);
    {
      const auto sw = __builtin_amdgcn_permlane32_swap(__float_as_uint(mx), __float_as_uint(mx),
                                                       false, false);
      mx = fmaxf(__uint_as_float(sw[0]), __uint_as_float(sw[1]));
    }
    const float mxs = mx * c_log2;
    // a row with a visible key in the block has a finite mxs, far above the
    // floor, so the first such block always moves m; a row without one
    // (mxs = -inf) keeps m and gets p = 0
    const bool need = mxs > m_run + 8.f;
    const float m_new = need ? mxs : m_run;
    const float a_new = need ? __builtin_amdgcn_exp2f(m_run - m_new) : 1.f;
    bf16x8 pn[NKS];
    float ps = 0.f;
#pragma unroll
    for (int u = 0; u < NKS; ++u) {
      // P V MFMAs of key step u of the previous block
#pragma unroll
      for (int dt = 0; dt < NDT; ++dt) {
        const int j = u * NDT + dt;
        if (j + VW < NV) vread(j + VW);
        oacc[dt] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(vf[j], pf[u], oacc[dt], 0, 0, 0);
      }
      bf16x8 p8;
#pragma unroll
      for (int e = 0; e < 8; ++e)
        p8[e] = (bf16)__builtin_amdgcn_exp2f(fmaf(sacc[u >> 1][(u & 1) * 8 + e], c_log2, -m_new));
      pn[u] = p8;
#pragma unroll
      for (int e = 0; e < 8; e += 2)
        ps = __builtin_amdgcn_fdot2_f32_bf16(bf16x2{p8[e], p8[e + 1]},
                                             bf16x2{(bf16)1.f, (bf16)1.f}, ps, false);
    }
#pragma unroll
    for (int u = 0; u < NKS; ++u) pf[u] = pn[u];
#if FOE_ATT_SGB
    constexpr int VPM = FOE_ATT_VPM;
#pragma unroll
    for (int j = 0; j < NV; ++j) {
      __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
      if (j + VW < NV) __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);
      __builtin_amdgcn_sched_group_barrier(0x002, VPM, 0);  // VALU
    }
#endif
    resc = __builtin_amdgcn_ballot_w64(need) != 0;
    alpha = a_new;
    m_run = m_new;
    l_run = l_run * a_new + ps;
  };

  for (int it = 0; it < niter; ++it) {
    const int kb = NP * it + part;
    // K of this block and V of the previous one have landed for every wave,
    // and every wave is done with the previous iteration's stages
    vm_barrier<0>();
    if (kb + NP < nkb) issue_k(it + 1);
    if (kb < nkb) issue_v(it);
    const unsigned char* ks = hs + (it & 1) * KT;
    const unsigned char* vs = hs + 2 * KT + ((it + 1) & 1) * VT;  // previous block's V
    // the rescale owed by the previous block's softmax, before its P V
    if (resc) {
#pragma unroll
      for (int t = 0; t < NDT; ++t)
#pragma unroll
        for (int v = 0; v < 16; ++v) oacc[t][v] *= alpha;
    }
    if (kb >= nkb) {  // wave-uniform: this part has no block left
      pv(oacc, pf, vs);
      resc = false;
      alpha = 1.f;
#pragma unroll
      for (int u = 0; u < NKS; ++u) pf[u] = bf16x8{};
      continue;
    }
    const int kbase = kb * KB;
    const bool edge = kbase + KB - 1 > q0 || kbase + KB > S;  // wave-uniform
    block_step(edge, ks, vs, kbase);
  }
  // the last block's P V (P = 0 if the part's last iteration had no block)
  vm_barrier<0>();
  if (resc) {
#pragma unroll
    for (int t = 0; t < NDT; ++t)
#pragma unroll
      for (int v = 0; v < 16; ++v) oacc[t][v] *= alpha;
  }
  pv(oacc, pf, hs + 2 * KT + ((niter + 1) & 1) * VT);

  // merge: parts 1 .. NP-1 hand (m, l, O) to their partner wave of part 0
  // through LDS (the rings are free after this barrier); part 0 folds them
  // in part order
  float l = l_run + __shfl_xor(l_run, 32);
  __syncthreads();
  constexpr int MB = 64 * (HD / 2 + 2);  // floats per wave buffer
  if (part != 0) {
    float* mb = reinterpret_cast<float*>(smem) + (size_t)((part - 1) * HW + hw) * MB;
#pragma unroll
    for (int t = 0; t < NDT; ++t)
#pragma unroll
      for (int v = 0; v < 16; ++v) mb[(t * 16 + v) * 64 + lane] = oacc[t][v];
    mb[(HD / 2) * 64 + lane] = m_run;
    mb[(HD / 2 + 1) * 64 + lane] = l;
  }
  __syncthreads();
  if (part != 0) return;
#pragma unroll
  for (int pp = 1; pp < NP; ++pp) {
    const float* mb = reinterpret_cast<const float*>(smem) + (size_t)((pp - 1) * HW + hw) * MB;
    const float mo = mb[(HD / 2) * 64 + lane], lo = mb[(HD / 2 + 1) * 64 + lane];
    const float m = fmaxf(m_run, mo);
    // both maxima are at least the finite floor, so the factors are finite
    const float a0 = __builtin_amdgcn_exp2f(m_run - m);
    const float a1 = __builtin_amdgcn_exp2f(mo - m);
    l = l * a0 + lo * a1;
#pragma unroll
    for (int t = 0; t < NDT; ++t)
#pragma unroll
      for (int v = 0; v < 16; ++v) oacc[t][v] = oacc[t][v] * a0 + mb[(t * 16 + v) * 64 + lane] * a1;
    m_run = m;
  }

  // O[q][dim] = O^T / l; lane holds dims 32 dt + 8 g + 4 hl + [0, 4)
  if (q < S) {
    const float inv = 1.f / l;
    bf16* orow = out + ((size_t)q * H + grp) * ((size_t)nq * HD) + (size_t)head * HD;
#pragma unroll
    for (int dt = 0; dt < NDT; ++dt)
#pragma unroll
      for (int g = 0; g < 4; ++g) {
        bf16x4 o;
#pragma unroll
        for (int v = 0; v < 4; ++v) o[v] = (bf16)(oacc[dt][g * 4 + v] * inv);
        *reinterpret_cast<bf16x4*>(orow + dt * 32 + g * 8 + hl * 4) = o;
      }
  }
}

// ---- residual sum -------------------------------------------------------------
// xs = sum_h x[h] in fp32, h = 0..H-1 in order; 8 elements per thread and
// grid-stride step.  It runs on a side stream beside the attention (which
// reads little from HBM), so the output projection's epilogue reads one fp32
// plane instead of H bf16 planes.
__global__ __launch_bounds__(256) void xsum_kernel(const bf16* __restrict__ x, int H,
                                                   long long plane, float* __restrict__ xs) {
  const long long nvec = plane / 8;
  for (long long i = (long long)blockIdx.x * blockDim.x + threadIdx.x; i < nvec;
       i += (long long)gridDim.x * blockDim.x) {
    float acc[8];
#pragma unroll
    for (int e = 0; e < 8; ++e) acc[e] = 0.f;
#pragma unroll 4
    for (int h = 0; h < H; ++h) {
      const bf16x8 v = *reinterpret_cast<const bf16x8*>(x + (size_t)h * plane + i * 8);
#pragma unroll
      for (int e = 0; e < 8; ++e) acc[e] += (float)v[e];
    }
    *reinterpret_cast<f32x4*>(xs + i * 8) = f32x4{acc[0], acc[1], acc[2], acc[3]};
    *reinterpret_cast<f32x4*>(xs + i * 8 + 4) = f32x4{acc[4], acc[5], acc[6], acc[7]};
  }
}

// The side stream of the current device and the two events that fork it
// from the caller's stream and join it back (created on first use, default
// priority, kept until the process ends).  The fork / launch / join sequence
// runs under one lock, so concurrent calls cannot interleave their event
// records; under HIP-graph capture the fork and join become graph edges.
struct SideStream {
  hipStream_t s = nullptr;
  hipEvent_t fork = nullptr, join = nullptr;
};
std::mutex g_side_mu;

SideStream* side_stream_locked() {
  static SideStream sides[64];
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= 64) return nullptr;
  SideStream& sd = sides[dev];
  if (sd.s == nullptr) {
    hipStream_t st = nullptr;
    hipEvent_t f = nullptr, j = nullptr;
    if (hipStreamCreateWithFlags(&st, hipStreamNonBlocking) != hipSuccess) return nullptr;
    if (hipEventCreateWithFlags(&f, hipEventDisableTiming) != hipSuccess ||
        hipEventCreateWithFlags(&j, hipEventDisableTiming) != hipSuccess) {
      if (f != nullptr) (void)hipEventDestroy(f);
      (void)hipStreamDestroy(st);
      return nullptr;
    }
    sd.s = st;
    sd.fork = f;
    sd.join = j;
  }
  return &sd;
}

struct AttnWs {
  size_t qkv, vt, o, xs, total;
};

AttnWs attn_ws(int H, int S, int d, int nq, int hd) {
  AttnWs w{};
  const size_t rows = (size_t)H * S;
  size_t off = 0;
  auto take = [&](size_t& field, size_t bytes) {
    off = align_up(off, 256);
    field = off;
    off += bytes;
  };
  take(w.qkv, rows * (nq + 2) * hd * 2);
  take(w.vt, (size_t)H * hd * ceil_div(S, kKB) * kKB * 2);
  take(w.o, rows * nq * hd * 2);
  take(w.xs, (size_t)S * d * 4);
  w.total = align_up(off, 256);
  return w;
}

}  // namespace

size_t group_attention_scratch_bytes(int H, int S, int d, int nq, int hd) {
  return attn_ws(H, S, d, nq, hd).total;
}

hipError_t launch_group_attention(int H, int S, int d, int nq, int hd, float theta, float scale,
                                  const void* x, const void* w_qkv, const void* w_o, void* r_full,
                                  void* scratch, hipStream_t s) {
  if (S == 0) return hipSuccess;
  const AttnWs L = attn_ws(H, S, d, nq, hd);
  unsigned char* base = static_cast<unsigned char*>(scratch);
  bf16* qkv = reinterpret_cast<bf16*>(base + L.qkv);
  bf16* o = reinterpret_cast<bf16*>(base + L.o);
  const int rows = H * S;
  // one segment of S rows per group (equal segments: no offsets array)
  hipError_t e = launch_grouped_gemm(x, nullptr, H, rows, w_qkv, (nq + 2) * hd, d, qkv, s,
                                     "attn_qkv");
  if (e != hipSuccess) return e;
  bf16* vt = reinterpret_cast<bf16*>(base + L.vt);
  const int nqb = ceil_div(S, kQB);
  const int s_pad = nqb * kKB;
  {
    ProfileScope ps("attn_prep", s);
    if (hd == 96)
      FOE_LAUNCH(prep_kernel<96>, dim3(nqb, H), dim3(256), 0, s, qkv, vt, S, s_pad, nq,
                 (double)theta, (double)scale);
    else
      FOE_LAUNCH(prep_kernel<128>, dim3(nqb, H), dim3(256), 0, s, qkv, vt, S, s_pad, nq,
                 (double)theta, (double)scale);
  }
  // the residual sum on the side stream, beside the attention
  float* xs = reinterpret_cast<float*>(base + L.xs);
  const long long plane = (long long)S * d;
  std::unique_lock<std::mutex> lock(g_side_mu);
  SideStream* side = side_stream_locked();
  hipStream_t rs = s;
  if (side != nullptr && hipEventRecord(side->fork, s) == hipSuccess &&
      hipStreamWaitEvent(side->s, side->fork, 0) == hipSuccess)
    rs = side->s;
  {
    ProfileScope ps("attn_xsum", rs);
    const long long want = ceil_div(plane / 8, 256LL);
#ifndef FOE_XSUM_WG
#define FOE_XSUM_WG 256
#endif
    FOE_LAUNCH(xsum_kernel, dim3((unsigned)(want < FOE_XSUM_WG ? want : FOE_XSUM_WG)), dim3(256), 0,
               rs,
               static_cast<const bf16*>(x), H, plane, xs);
  }
  const bool joined = rs == s || (hipEventRecord(side->join, rs) == hipSuccess);
  {
    ProfileScope ps("attn_core", s);
    const float c_log2 = 1.4426950408889634f / sqrtf((float)hd);
    // two heads per task: two parts of 64-key blocks; one head: four parts
    // of 32-key blocks (8 waves either way)
    const dim3 g2(nqb * (nq / 2) * H), g1(nqb * nq * H);
    if (hd == 96) {
      if (nq % 2 == 0)
        FOE_LAUNCH((attn_fwd_kernel<2, 96, 2>), g2, dim3(512), 0, s, qkv, vt, S, s_pad, nq, H,
                   c_log2, o);
      else
        FOE_LAUNCH((attn_fwd_kernel<1, 96, 4>), g1, dim3(512), 0, s, qkv, vt, S, s_pad, nq, H,
                   c_log2, o);
    } else {
      if (nq % 2 == 0)
        FOE_LAUNCH((attn_fwd_kernel<2, 128, 2>), g2, dim3(512), 0, s, qkv, vt, S, s_pad, nq, H,
                   c_log2, o);
      else
        FOE_LAUNCH((attn_fwd_kernel<1, 128, 4>), g1, dim3(512), 0, s, qkv, vt, S, s_pad, nq, H,
                   c_log2, o);
    }
  }
  if (!joined) return hipErrorUnknown;
  if (rs != s && (e = hipStreamWaitEvent(s, side->join, 0)) != hipSuccess) return e;
  lock.unlock();
  // output projection of all groups at once (o is [S][H*nq*hd], w_o
  // [d][H*nq*hd]) with the residual average in its epilogue:
  // r_full = (o w_o^T + xs) / H
  e = launch_gemm_resid(o, nullptr, S, w_o, d, H * nq * hd, xs, 1.0f / H, r_full, s,
                        "attn_out");
  if (e != hipSuccess) return e;
  return hipGetLastError();
}

}  // namespace foe
