// Shared device/host helpers of the gfx950 per-cluster MoE block library.
#pragma once

#include <hip/hip_ext.h>
#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

#include "foe.h"

namespace foe {

typedef __bf16 bf16;
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x4 __attribute__((ext_vector_type(4)));
typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

constexpr int kWave = 64;

// ---- element conversion --------------------------------------------------
__device__ __forceinline__ float to_f32(float v) { return v; }
__device__ __forceinline__ float to_f32(bf16 v) { return (float)v; }
template <typename T> __device__ __forceinline__ T from_f32(float v);
template <> __device__ __forceinline__ float from_f32<float>(float v) { return v; }
// hardware v_cvt_pk_bf16_f32: round to nearest even
template <> __device__ __forceinline__ bf16 from_f32<bf16>(float v) { return (bf16)v; }

// A 16-byte vector of elements of type T (8 bf16 or 4 fp32).
template <typename T> struct Vec16 {
  static constexpr int N = 16 / sizeof(T);
  T v[N];
};

template <typename T>
__device__ __forceinline__ Vec16<T> load16(const T* p) {
  Vec16<T> r;
  *reinterpret_cast<u32x4*>(r.v) = __builtin_nontemporal_load(reinterpret_cast<const u32x4*>(p));
  return r;
}
template <typename T>
__device__ __forceinline__ Vec16<T> load16_cached(const T* p) {
  Vec16<T> r;
  *reinterpret_cast<u32x4*>(r.v) = *reinterpret_cast<const u32x4*>(p);
  return r;
}
template <typename T>
__device__ __forceinline__ void store16(T* p, const Vec16<T>& r) {
  *reinterpret_cast<u32x4*>(p) = *reinterpret_cast<const u32x4*>(r.v);
}
__device__ __forceinline__ u32x4 zero_u32x4() { return u32x4{0u, 0u, 0u, 0u}; }

// ---- wave helpers ----------------------------------------------------------
__device__ __forceinline__ int lane_id() { return threadIdx.x & (kWave - 1); }

// v unchanged, through an empty volatile asm: the compiler cannot move values
// derived from the result above this point (e.g. hoist them out of a loop).
__device__ __forceinline__ int opaque_int(int v) {
  asm volatile("" : "+v"(v));
  return v;
}

// Rotate a 32-bit value right by `sh` lanes inside each row of 16 lanes (DPP).
template <int SH>
__device__ __forceinline__ int row_ror(int v) {
  return __builtin_amdgcn_update_dpp(0, v, 0x120 + SH, 0xF, 0xF, false);
}

// ---- host side: launch bookkeeping ----------------------------------------
// Kernel timing hooks (see foe_profile_* in foe.h).  A ProfileScope names the
// one launch it encloses; while timing is on, `profile_begin` hands it a slot
// with an event pair and FOE_LAUNCH passes that pair to hipExtLaunchKernelGGL,
// which stamps the events with the dispatch's own start and end (the interval
// holds the kernel alone, not the launch latency before it).
int profile_begin(const char* name);
hipEvent_t profile_event(int slot, int stop);
int& profile_cur_slot();  // slot of this thread's innermost live scope, -1 none

struct ProfileScope {
  int slot, prev;
  ProfileScope(const char* name, hipStream_t)
      : slot(profile_begin(name)), prev(profile_cur_slot()) {
    profile_cur_slot() = slot;
  }
  ~ProfileScope() { profile_cur_slot() = prev; }
};

#define FOE_LAUNCH(kernel, grid, block, lds, stream, ...)                                     \
  hipExtLaunchKernelGGL(kernel, grid, block, lds, stream,                                   \
                        ::foe::profile_event(::foe::profile_cur_slot(), 0),                 \
                        ::foe::profile_event(::foe::profile_cur_slot(), 1), 0u, __VA_ARGS__)

inline int ceil_div(long long a, long long b) { return (int)((a + b - 1) / b); }
inline size_t align_up(size_t v, size_t a) { return (v + a - 1) / a * a; }

// ---- kernel launchers (one translation unit each) -------------------------
// C clusters in one grid: w_router [C][E][d], bias [C][E], outputs [C][T][k].
// zero_cnt != nullptr: the kernel also clears zero_cnt[T][zero_per_tok].
// gating: FOE_GATE_RENORM or FOE_GATE_GLOBAL (the global softmax needs every
// cluster's scores in one workgroup: C == 1 or C*E <= 256).
// counts != nullptr: the kernel also writes the expert counts of each of its
// workgroups' tokens, counts [C][nblk][E] (the dispatch histogram; nblk and
// the tokens per workgroup from plan_route; not with zero_cnt).
struct RoutePlan {
  int G = 1;            // clusters scored together in one workgroup
  bool stream = false;  // the streaming kernel
  int wpb = 1;          // its waves per workgroup
  int tok_per_blk = 16; // tokens per workgroup (count block)
  int nblk = 0;         // workgroups per cluster
};
RoutePlan plan_route(foe_dtype dt, int C, int T, int d, int E, bool zero_counters);
hipError_t launch_route(foe_dtype dt, int C, int T, int d, int E, int k, int gating,
                        const void* x, const void* w_router, const float* bias,
                        int32_t* topk_idx, float* topk_w, hipStream_t s,
                        int32_t* zero_cnt = nullptr, int zero_per_tok = 0,
                        int32_t* counts = nullptr);
// whether all C clusters' scores of a token are formed in one workgroup
inline bool route_one_pass(int C, int E) { return C == 1 || C * E <= 256; }

// permute scratch = 2 * C * nblk * E int32 (see permute_blocks())
int permute_blocks(int R);
size_t permute_scratch_bytes(int T, int k, int E, int C);
// histogram / scan / stable ranks of C clusters' ids (topk_idx [C,T,k]);
// offsets [C*E+1] and row_of values are global rows (cluster h starts at h*T*k)
// zero [nzero]: int32 counters of the kernel that follows, cleared on the way.
// route_counts [C][ncb][E]: expert counts of consecutive blocks of tok_per_cb
// tokens written by the routing kernel; when index_takes_route_counts() the
// pass uses them instead of a histogram launch of its own.
bool index_takes_route_counts(int T, int E, int k, int ncb);
hipError_t launch_index(int T, int E, int k, int C, const int32_t* topk_idx, int32_t* counts,
                        int32_t* offsets, int32_t* sorted_src, int32_t* row_of, void* scratch,
                        hipStream_t s, int32_t* zero = nullptr, int nzero = 0,
                        const int32_t* route_counts = nullptr, int tok_per_cb = 0,
                        int ncb = 0);
hipError_t launch_permute(foe_dtype dt, int T, int d, int E, int k, const int32_t* topk_idx,
                          const void* x, int32_t* counts, int32_t* offsets, int32_t* sorted_src,
                          int32_t* row_of, void* x_perm, void* scratch, hipStream_t s);

size_t ffn_scratch_bytes(foe_dtype dt, int rows, int F);
hipError_t launch_expert_ffn(foe_dtype dt, int E, int d, int F, int rows, const void* x_perm,
                             const int32_t* offsets, const void* w_gate, const void* w_up,
                             const void* w_down, void* y_perm, void* scratch, hipStream_t s);

// bf16 grouped GEMM out[r] = A[r] W[e]^T for the rows r of segment e
// (offsets [E+1]); W [E, N, K], A [rows, K], out [rows, N] (the down-projection
// kernel of the expert FFN)
// (offsets == nullptr: E segments of rows / E rows each)
hipError_t launch_grouped_gemm(const void* A, const int32_t* offsets, int E, int rows,
                               const void* W, int N, int K, void* out, hipStream_t s,
                               const char* name);
// out[m][n] = scale * (sum_k A[m][k] W[n][k] + x[m*N + n]) (A, W, out bf16; x
// fp32; fp32 sums; one segment of `rows` rows: offsets = {0, rows} or null)
hipError_t launch_gemm_resid(const void* A, const int32_t* offsets, int rows, const void* W,
                             int N, int K, const float* x, float scale, void* out, hipStream_t s,
                             const char* name);
// per-group attention of Table 3 (attention.hip): r_full [S, d] from x [H, S, d]
size_t group_attention_scratch_bytes(int H, int S, int d, int nq, int hd);
hipError_t launch_group_attention(int H, int S, int d, int nq, int hd, float theta, float scale,
                                  const void* x, const void* w_qkv, const void* w_o, void* r_full,
                                  void* scratch, hipStream_t s);

// bf16 expert FFN with both grouped GEMMs in one persistent launch (many rows
// per expert): h [rows, F] is its intermediate, sync [ffn_sync_ints(E, rows)]
// int32 counters that must be zero when it starts.  Operand rows as in
// launch_expert_ffn_ex.
size_t ffn_sync_ints(int E, int rows);
hipError_t launch_expert_ffn_fused(int E, int d, int F, int rows, const void* A,
                                   const int32_t* gather, int kdiv, int a_rows,
                                   const int32_t* offsets, const void* w_gate, const void* w_up,
                                   const void* w_down, void* y, void* h, int32_t* sync,
                                   hipStream_t s);
// expert FFN whose operand row r is row gather[r]/kdiv of A (a_rows rows);
// gather == nullptr: row r of A
hipError_t launch_expert_ffn_ex(foe_dtype dt, int E, int d, int F, int rows, const void* A,
                                const int32_t* gather, int kdiv, int a_rows,
                                const int32_t* offsets, const void* w_gate, const void* w_up,
                                const void* w_down, void* y_perm, void* scratch, hipStream_t s);
// The block's combine folded into the decode down kernel: w = topk_w [C][T*k],
// x and out [T][d], cnt = [T][ceil(d/128)] arrival counters that must be zero
// when the down kernel starts (the route kernel of the same call clears them).
// out == nullptr: not folded.
struct FusedCombine {
  const float* w = nullptr;
  const bf16* x = nullptr;
  bf16* out = nullptr;
  int32_t* cnt = nullptr;
  float scale = 1.f;
  int C = 0, k = 0;
};

// Decode form of the block's FFN (bf16, few pairs per expert): every
// workgroup lists its expert's pairs from the routing decisions topk_idx
// [C][T*k] itself (no dispatch index pass); the intermediate rows and the
// output rows y [C*T*k][d] are indexed by pair.  ffn_sel_ok() tells whether
// the shape takes this form.
bool ffn_sel_ok(foe_dtype dt, int C, int E, int T, int k);
hipError_t launch_expert_ffn_sel(int C, int E, int d, int F, int T, int k, const void* x,
                                 const int32_t* topk_idx, const void* w_gate, const void* w_up,
                                 const void* w_down, void* y, void* scratch, hipStream_t s,
                                 const FusedCombine& fc);
// row_of_all == nullptr: y row of pair p of cluster h is h*T*k + p, skipped
// when the expert id sel_all[h*T*k + p] is outside [0, E)
hipError_t launch_combine_clusters(foe_dtype dt, int C, int T, int d, int k, const void* y,
                                   const int32_t* row_of_all, const float* w_all, const void* x,
                                   float scale, void* out, hipStream_t s,
                                   const int32_t* sel_all = nullptr, int E = 0);
hipError_t launch_combine(foe_dtype dt, int T, int d, int k, const void* y_perm,
                          const int32_t* row_of, const float* topk_w, const void* residual,
                          void* out, hipStream_t s);
hipError_t launch_reduce(foe_dtype dt, int C, int T, int d, const void* partials,
                         const void* residual, float scale, void* out, hipStream_t s);
hipError_t launch_fill_i32(int32_t* p, int n, int32_t v, hipStream_t s);

}  // namespace foe
