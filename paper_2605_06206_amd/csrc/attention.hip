// Per-group attention that feeds the block (Table 3, FoE column, rows "Attn.
// residual" and "Cross-group avg."): every group h keeps its own
// representation x[h] and runs causal attention over it with its own KV head
// and nq query heads sharing it (grouped-query attention); the results are
// averaged over the groups:
//   r[h, i]    = x[h, i] + Attn_h(x[h, :])[i]
//   r_full[i]  = (1/H) sum_h r[h, i]
// Five launches: the q/k/v projection of every group (one grouped GEMM with a
// segment per group), the rotary embedding of q and k in place, the
// attention, the output projection (grouped GEMM), and the residual average.
//
// Attention (head dim 128): a workgroup owns 64 queries of NH query heads of
// one group (4 waves per head, 16 queries per wave) and walks the key blocks
// of 64 up to its diagonal.  Per block the keys go to LDS as rows [key][dim]
// and the values transposed as rows [dim][key], both with XOR-swizzled
// 16/8-byte chunks; the next block is prefetched into registers meanwhile.  A
// wave computes the score tile transposed, S^T = K Q^T, on
// v_mfma_f32_16x16x32_bf16: lane l then holds 16 scores of query l%16, so the
// online softmax (exp2 form) needs only a reduction over the four lane groups
// and the probabilities are already laid out as the B operand of
// O^T += V^T P^T.  Keys of the MFMA K dimension follow the order the score
// registers come in; the transposed value tile is read in that same order.
#include "foe_common.hpp"

namespace foe {
namespace {

constexpr int kHd = 128;  // head dimension the attention kernel is built for
constexpr int kQB = 64;   // queries per workgroup and head
constexpr int kKB = 64;   // keys per block

// ---- rotary embedding -------------------------------------------------------
// One wave per (row, head) of the q and k heads; lane i rotates the pair
// (i, i + 64) by the angle (s / scale) * theta^(-2i/128).  The angle is formed
// and reduced modulo 2*pi in double, then sin/cos in float.
__global__ __launch_bounds__(256) void rope_kernel(bf16* __restrict__ qkv, int rows, int S,
                                                   int nq, double theta, double scale) {
  const int lane = lane_id();
  const long long wid = (long long)blockIdx.x * 4 + (threadIdx.x >> 6);
  const int nh = nq + 1;  // q heads and the k head
  if (wid >= (long long)rows * nh) return;
  const int row = (int)(wid / nh), head = (int)(wid % nh);
  const int s = row % S;
  const size_t ld = (size_t)(nq + 2) * kHd;
  bf16* v = qkv + (size_t)row * ld + (size_t)head * kHd;
  const double inv_freq = pow(theta, -2.0 * lane / kHd);
  double a = (double)s / scale * inv_freq;
  constexpr double kTwoPi = 6.283185307179586476925286766559;
  a -= kTwoPi * floor(a / kTwoPi);
  float sn, cs;
  sincosf((float)a, &sn, &cs);
  const float x1 = (float)v[lane], x2 = (float)v[lane + kHd / 2];
  v[lane] = (bf16)(x1 * cs - x2 * sn);
  v[lane + kHd / 2] = (bf16)(x2 * cs + x1 * sn);
}

// ---- attention ----------------------------------------------------------------
// K tile: key r, dims [8c, 8c+8) in 16-byte chunk c ^ (r & 15) of row r (256 B).
// V^T tile: dim r, keys [4c, 4c+4) in 8-byte chunk c ^ (r & 15) of row r (128 B).
__device__ __forceinline__ int k_off(int r, int c) { return r * 256 + ((c ^ (r & 15)) << 4); }
__device__ __forceinline__ int vt_off(int r, int key) {
  return r * 128 + ((((key >> 2) ^ (r & 15))) << 3) + ((key & 3) << 1);
}

template <int NH>
__global__ __launch_bounds__(NH * 256) void attn_kernel(const bf16* __restrict__ qkv, int S,
                                                        int nq, float scale_log2,
                                                        bf16* __restrict__ out) {
  __shared__ __align__(16) unsigned char ks[kKB * kHd * 2];
  __shared__ __align__(16) unsigned char vts[kHd * kKB * 2];
  const int tid = threadIdx.x;
  const int lane = lane_id();
  const int wave = tid >> 6;
  const int hw = wave & 3;   // wave within its head
  const int hh = wave >> 2;  // head within the workgroup
  const int nqb = (S + kQB - 1) / kQB;
  const int qb = nqb - 1 - (int)blockIdx.x;  // longest causal walks first
  const int head = blockIdx.y * NH + hh;
  const int grp = blockIdx.z;
  const size_t ld = (size_t)(nq + 2) * kHd;
  const bf16* base = qkv + (size_t)grp * S * ld;
  const int q0 = qb * kQB + hw * 16;  // this wave's first query
  const int qi = lane & 15, g = lane >> 4;
  const int qabs = q0 + qi;

  // Q fragments (B operand of S^T = K Q^T): query qi, dims kk*32 + 8g .. +8
  bf16x8 qf[4];
#pragma unroll
  for (int kk = 0; kk < 4; ++kk) {
    if (qabs < S && head < nq)
      qf[kk] = *reinterpret_cast<const bf16x8*>(base + (size_t)qabs * ld + (size_t)head * kHd +
                                                kk * 32 + 8 * g);
    else
      qf[kk] = bf16x8{};
  }

  f32x4 oacc[8];
#pragma unroll
  for (int t = 0; t < 8; ++t) oacc[t] = f32x4{0.f, 0.f, 0.f, 0.f};
  float m_run = -__builtin_inff();  // running max of this lane's query (log2 units)
  float l_run = 0.f;                // this lane's share of the running sum

  // block loads: 64 keys x 128 dims of K and of V, 16 bytes per piece; thread
  // t handles pieces t, t + NT, ... (key = piece / 16, dims (piece % 16) * 8)
  constexpr int NT = NH * 256;
  constexpr int NPC = kKB * kHd / 8 / NT;  // pieces of K (and of V) per thread
  bf16x8 kreg[NPC], vreg[NPC];
  auto load_block = [&](int kb) {
#pragma unroll
    for (int i = 0; i < NPC; ++i) {
      const int pc = tid + i * NT;
      const int key = kb * kKB + (pc >> 4), c = pc & 15;
      if (key < S) {
        const bf16* row = base + (size_t)key * ld + (size_t)nq * kHd;
        kreg[i] = *reinterpret_cast<const bf16x8*>(row + c * 8);
        vreg[i] = *reinterpret_cast<const bf16x8*>(row + kHd + c * 8);
      } else {
        kreg[i] = bf16x8{};
        vreg[i] = bf16x8{};
      }
    }
  };
  auto store_block = [&]() {
#pragma unroll
    for (int i = 0; i < NPC; ++i) {
      const int pc = tid + i * NT;
      const int key = pc >> 4, c = pc & 15;
      *reinterpret_cast<bf16x8*>(ks + k_off(key, c)) = kreg[i];
#pragma unroll
      for (int e = 0; e < 8; ++e)
        *reinterpret_cast<bf16*>(vts + vt_off(c * 8 + e, key)) = vreg[i][e];
    }
  };

  const int nkb = min(qb + 1, (S + kKB - 1) / kKB);
  load_block(0);
  for (int kb = 0; kb < nkb; ++kb) {
    __syncthreads();  // the previous block's tiles are no longer read
    store_block();
    __syncthreads();
    if (kb + 1 < nkb) load_block(kb + 1);

    // scores S^T[key][query]: lane holds keys kb*64 + 16j + 4g + v of query qi
    f32x4 sacc[4];
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      sacc[j] = f32x4{0.f, 0.f, 0.f, 0.f};
      const int kr = j * 16 + qi;  // key row of this lane's A fragment
#pragma unroll
      for (int kk = 0; kk < 4; ++kk) {
        const bf16x8 kf = *reinterpret_cast<const bf16x8*>(ks + k_off(kr, kk * 4 + g));
        sacc[j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(kf, qf[kk], sacc[j], 0, 0, 0);
      }
    }
    // mask (causal and past the sequence), scale, running max
    float mx = -__builtin_inff();
#pragma unroll
    for (int j = 0; j < 4; ++j)
#pragma unroll
      for (int v = 0; v < 4; ++v) {
        const int key = kb * kKB + j * 16 + 4 * g + v;
        const float sv = (key <= qabs && key < S) ? sacc[j][v] * scale_log2 : -__builtin_inff();
        sacc[j][v] = sv;
        mx = fmaxf(mx, sv);
      }
    mx = fmaxf(mx, __shfl_xor(mx, 16));
    mx = fmaxf(mx, __shfl_xor(mx, 32));
    const float m_new = fmaxf(m_run, mx);
    // a query with no visible key yet keeps m = -inf: scale 1, probabilities 0
    const bool live = m_new != -__builtin_inff();
    const float alpha = live ? exp2f(m_run - m_new) : 1.f;
    float psum = 0.f;
    bf16x8 pf[2];
#pragma unroll
    for (int j = 0; j < 4; ++j)
#pragma unroll
      for (int v = 0; v < 4; ++v) {
        const float p = live ? exp2f(sacc[j][v] - m_new) : 0.f;
        psum += p;
        pf[j >> 1][(j & 1) * 4 + v] = (bf16)p;
      }
    l_run = l_run * alpha + psum;
    m_run = m_new;
#pragma unroll
    for (int t = 0; t < 8; ++t)
#pragma unroll
      for (int v = 0; v < 4; ++v) oacc[t][v] *= alpha;
    // O^T[dim][query] += V^T[dim][keys] P^T[keys][query]; k-slot group g of
    // step s holds keys 32s + 4g + [0,4) and 32s + 16 + 4g + [0,4)
#pragma unroll
    for (int s2 = 0; s2 < 2; ++s2) {
#pragma unroll
      for (int t = 0; t < 8; ++t) {
        const int r = t * 16 + qi;  // dim row of this lane's A fragment
        const uint2 lo = *reinterpret_cast<const uint2*>(vts + vt_off(r, 32 * s2 + 4 * g));
        const uint2 hi = *reinterpret_cast<const uint2*>(vts + vt_off(r, 32 * s2 + 16 + 4 * g));
        const uint4 vv = uint4{lo.x, lo.y, hi.x, hi.y};
        oacc[t] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8, vv),
                                                          pf[s2], oacc[t], 0, 0, 0);
      }
    }
  }

  // O[query][dim] = O^T / l; lane holds dims 16t + 4g + [0,4) of query qi
  float l = l_run + __shfl_xor(l_run, 16);
  l += __shfl_xor(l, 32);
  if (qabs < S && head < nq) {
    const float inv = 1.f / l;
    bf16* orow = out + ((size_t)grp * S + qabs) * ((size_t)nq * kHd) + (size_t)head * kHd;
#pragma unroll
    for (int t = 0; t < 8; ++t) {
      bf16x4 o;
#pragma unroll
      for (int v = 0; v < 4; ++v) o[v] = (bf16)(oacc[t][v] * inv);
      *reinterpret_cast<bf16x4*>(orow + t * 16 + 4 * g) = o;
    }
  }
}

// ---- residual average ---------------------------------------------------------
// r_full = (1/H) sum_h (x[h] + a[h]) in fp32, h = 0..H-1 in order; 8 elements
// per thread per grid-stride step.
__global__ __launch_bounds__(256) void resid_avg_kernel(const bf16* __restrict__ x,
                                                        const bf16* __restrict__ a, int H,
                                                        long long plane, float inv_h,
                                                        bf16* __restrict__ out) {
  const long long nvec = plane / 8;
  for (long long i = (long long)blockIdx.x * blockDim.x + threadIdx.x; i < nvec;
       i += (long long)gridDim.x * blockDim.x) {
    float acc[8];
#pragma unroll
    for (int e = 0; e < 8; ++e) acc[e] = 0.f;
    for (int h = 0; h < H; ++h) {
      const bf16x8 xv = *reinterpret_cast<const bf16x8*>(x + (size_t)h * plane + i * 8);
      const bf16x8 av = *reinterpret_cast<const bf16x8*>(a + (size_t)h * plane + i * 8);
#pragma unroll
      for (int e = 0; e < 8; ++e) acc[e] += (float)xv[e] + (float)av[e];
    }
    bf16x8 o;
#pragma unroll
    for (int e = 0; e < 8; ++e) o[e] = (bf16)(acc[e] * inv_h);
    *reinterpret_cast<bf16x8*>(out + i * 8) = o;
  }
}

__global__ void iota_kernel(int32_t* p, int n, int step) {
  const int i = blockIdx.x * blockDim.x + threadIdx.x;
  if (i < n) p[i] = i * step;
}

struct AttnWs {
  size_t offsets, qkv, o, a, total;
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
  take(w.offsets, (size_t)(H + 1) * 4);
  take(w.qkv, rows * (nq + 2) * hd * 2);
  take(w.o, rows * nq * hd * 2);
  take(w.a, rows * d * 2);
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
  int32_t* offsets = reinterpret_cast<int32_t*>(base + L.offsets);
  bf16* qkv = reinterpret_cast<bf16*>(base + L.qkv);
  bf16* o = reinterpret_cast<bf16*>(base + L.o);
  bf16* a = reinterpret_cast<bf16*>(base + L.a);
  const int rows = H * S;
  {
    ProfileScope ps("attn_offsets", s);
    FOE_LAUNCH(iota_kernel, dim3(ceil_div(H + 1, 256)), dim3(256), 0, s, offsets, H + 1, S);
  }
  hipError_t e = launch_grouped_gemm(x, offsets, H, rows, w_qkv, (nq + 2) * hd, d, qkv, s,
                                     "attn_qkv");
  if (e != hipSuccess) return e;
  {
    ProfileScope ps("attn_rope", s);
    FOE_LAUNCH(rope_kernel, dim3(ceil_div((long long)rows * (nq + 1), 4)), dim3(256), 0, s, qkv,
               rows, S, nq, (double)theta, (double)scale);
  }
  {
    ProfileScope ps("attn_core", s);
    const float scale_log2 = 1.4426950408889634f / sqrtf((float)hd);
    const int nqb = ceil_div(S, kQB);
    if (nq % 2 == 0)
      FOE_LAUNCH(attn_kernel<2>, dim3(nqb, nq / 2, H), dim3(512), 0, s, qkv, S, nq, scale_log2,
                 o);
    else
      FOE_LAUNCH(attn_kernel<1>, dim3(nqb, nq, H), dim3(256), 0, s, qkv, S, nq, scale_log2, o);
  }
  e = launch_grouped_gemm(o, offsets, H, rows, w_o, d, nq * hd, a, s, "attn_out");
  if (e != hipSuccess) return e;
  {
    ProfileScope ps("attn_resid_avg", s);
    const long long plane = (long long)S * d;
    const long long nvec = plane / 8;
    const long long want = (nvec + 255) / 256;
    FOE_LAUNCH(resid_avg_kernel, dim3((unsigned)(want < 8192 ? want : 8192)), dim3(256), 0, s,
               static_cast<const bf16*>(x), a, H, plane, 1.0f / H, static_cast<bf16*>(r_full));
  }
  return hipGetLastError();
}

}  // namespace foe
