// C ABI of the per-cluster MoE block library (declarations and contracts in
// include/foe.h).  Host code only: argument checks, workspace carving, the
// launch sequence of the block and the kernel-timing registry.
#include <limits.h>

#include <mutex>
#include <string>
#include <vector>

#include "foe_common.hpp"

// both grouped GEMMs of the block's expert FFN in one persistent launch
#ifndef FOE_FFN_FUSED
#define FOE_FFN_FUSED 1
#endif

namespace foe {
namespace {

thread_local std::string g_err;

int fail(int code, const std::string& msg) {
  g_err = msg;
  return code;
}

int hip_fail(hipError_t e, const char* where) {
  return fail(FOE_ERR_HIP, std::string(where) + ": " + hipGetErrorString(e));
}

bool aligned16(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }
bool aligned4(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 3u) == 0; }
size_t esize(foe_dtype dt) { return dt == FOE_BF16 ? 2 : 4; }

// ---- argument checks --------------------------------------------------------
struct Check {
  std::string err;
  void need(bool ok, const char* msg) {
    if (!ok && err.empty()) err = msg;
  }
  void tensor(const void* p, bool required, const char* name) {
    if (!err.empty()) return;
    if (p == nullptr) {
      if (required) err = std::string(name) + " is NULL";
    } else if (!aligned16(p)) {
      err = std::string(name) + " is not 16-byte aligned";
    }
  }
  void small(const void* p, bool required, const char* name) {
    if (!err.empty()) return;
    if (p == nullptr) {
      if (required) err = std::string(name) + " is NULL";
    } else if (!aligned4(p)) {
      err = std::string(name) + " is not 4-byte aligned";
    }
  }
};

void check_dtype(Check& c, foe_dtype dt) {
  c.need(dt == FOE_F32 || dt == FOE_BF16, "dt must be FOE_F32 or FOE_BF16");
}
void check_dim8(Check& c, int v, const char* msg) { c.need(v >= 8 && v % 8 == 0, msg); }
void check_route_shape(Check& c, int T, int E, int k) {
  c.need(T >= 0, "T must be >= 0");
  c.need(E >= 1 && E <= 256, "E must be in [1, 256]");
  c.need(k >= 1 && k <= E, "k must be in [1, E]");
  c.need((long long)T * (k < 1 ? 1 : k) <= INT_MAX, "T*k must fit in int32");
}

// 16-byte operand loads address their buffers with 32-bit byte offsets below
// 2^31 (larger offsets mean "read zeros"), which bounds the bf16 tensors that
// are read that way.
constexpr long long kMaxOperandBytes = (1ll << 31) - 64;
bool operand_fits(long long rows, long long cols, size_t el) {
  return rows * cols * (long long)el <= kMaxOperandBytes;
}

// ---- workspace layout of foe_cluster_block ---------------------------------
// All C clusters are processed together: routing of cluster h fills slice h of
// topk_idx / topk_w [C,T,k]; one index pass numbers the permuted rows of all
// clusters consecutively (cluster h from h*T*k); one grouped FFN runs over the
// C*E experts reading x through sorted_src; one kernel combines and reduces.
struct BlockWs {
  size_t topk_idx, topk_w, counts, offsets, sorted_src, row_of, y, perm, ffn, cnt, sync, rcnt,
      total;
};

BlockWs block_ws(foe_dtype dt, int C, int T, int d, int E, int k, int F) {
  BlockWs w{};
  const size_t R = (size_t)T * k, CR = (size_t)C * R, CE = (size_t)C * E, s = esize(dt);
  size_t off = 0;
  auto take = [&](size_t& field, size_t bytes) {
    off = align_up(off, 256);
    field = off;
    off += bytes;
  };
  take(w.topk_idx, CR * 4);
  take(w.topk_w, CR * 4);
  take(w.counts, CE * 4);
  take(w.offsets, (CE + 1) * 4);
  take(w.sorted_src, CR * 4);
  take(w.row_of, CR * 4);
  take(w.y, CR * d * s);
  take(w.perm, permute_scratch_bytes(T, k, E, C));
  take(w.ffn, ffn_scratch_bytes(dt, (int)CR, F));
  take(w.cnt, (size_t)T * ceil_div(d, 128) * 4);  // folded-combine arrival counters
  take(w.sync, ffn_sync_ints(C * E, (int)CR) * 4);  // fused FFN work and ready counters
  take(w.rcnt, (size_t)C * ceil_div(T, 16) * E * 4);  // expert counts of the routing blocks
  w.total = align_up(off, 256);
  return w;
}

// ---- kernel timing registry -------------------------------------------------
struct ProfRec {
  std::string name;
  int ev;
};
std::mutex g_prof_mu;
bool g_prof_on = false;
std::vector<hipEvent_t> g_events;  // pairs (2*ev, 2*ev+1), reused across resets
size_t g_events_used = 0;
std::vector<ProfRec> g_recs;

}  // namespace

int profile_begin(const char* name) {
  std::lock_guard<std::mutex> lock(g_prof_mu);
  if (!g_prof_on) return -1;
  if (g_events_used * 2 + 2 > g_events.size()) {
    hipEvent_t a, b;
    if (hipEventCreate(&a) != hipSuccess) return -1;
    if (hipEventCreate(&b) != hipSuccess) {
      (void)hipEventDestroy(a);
      return -1;
    }
    g_events.push_back(a);
    g_events.push_back(b);
  }
  const int ev = (int)g_events_used++;
  g_recs.push_back({name, ev});
  return ev;
}

hipEvent_t profile_event(int slot, int stop) {
  if (slot < 0) return nullptr;
  std::lock_guard<std::mutex> lock(g_prof_mu);
  return g_events[2 * slot + (stop ? 1 : 0)];
}

int& profile_cur_slot() {
  static thread_local int slot = -1;
  return slot;
}

}  // namespace foe

// ---- scratch of the entry point that allocates nothing ---------------------
// One copy per GPU the library runs on, held until the process ends.  Host
// code never uses the array's name as an address: the device address of each
// GPU's copy comes from hipGetSymbolAddress, taken once per device with that
// device current.
constexpr size_t kNoAllocScratchBytes = (size_t)128 << 20;
static __device__ __align__(256) unsigned char scratch[kNoAllocScratchBytes];

namespace foe {
namespace {
std::mutex g_scratch_mu;
std::vector<void*> g_scratch_ptr;  // per device ordinal; null until first taken

// Device address of the current device's scratch array.
int noalloc_scratch(void** out) {
  int dev = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return hip_fail(e, "foe_cluster_block_noalloc/hipGetDevice");
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  if ((size_t)dev >= g_scratch_ptr.size()) g_scratch_ptr.resize((size_t)dev + 1, nullptr);
  if (g_scratch_ptr[dev] == nullptr) {
    void* p = nullptr;
    e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess) return hip_fail(e, "foe_cluster_block_noalloc/hipGetSymbolAddress");
    if (p == nullptr) return fail(FOE_ERR_HIP, "foe_cluster_block_noalloc: no scratch address");
    g_scratch_ptr[dev] = p;
  }
  *out = g_scratch_ptr[dev];
  return FOE_OK;
}
}  // namespace
}  // namespace foe

using namespace foe;

extern "C" {

const char* foe_last_error(void) { return g_err.c_str(); }

size_t foe_workspace_bytes(const char* op, foe_dtype dt, int C, int T, int d, int E, int k,
                           int F) {
  if (op == nullptr) {
    g_err = "op is NULL";
    return SIZE_MAX;
  }
  const std::string o(op);
  Check c;
  check_dtype(c, dt);
  if (o == "route" || o == "combine" || o == "reduce") {
    if (!c.err.empty()) return (g_err = c.err, SIZE_MAX);
    return 0;
  }
  if (o == "permute") {
    check_route_shape(c, T, E, k);
    if (!c.err.empty()) return (g_err = c.err, SIZE_MAX);
    return permute_scratch_bytes(T, k, E, 1);
  }
  if (o == "expert_ffn") {
    c.need(T >= 0 && k >= 1 && (long long)T * k <= INT_MAX, "rows = T*k must be in [0, 2^31)");
    check_dim8(c, F, "F must be a positive multiple of 8");
    if (!c.err.empty()) return (g_err = c.err, SIZE_MAX);
    return ffn_scratch_bytes(dt, T * k, F);
  }
  if (o == "cluster_block") {
    check_route_shape(c, T, E, k);
    c.need(C >= 1 && C <= 64, "C must be in [1, 64]");
    c.need((long long)C * T * (k < 1 ? 1 : k) <= INT_MAX, "C*T*k must fit in int32");
    check_dim8(c, d, "d must be a positive multiple of 8");
    check_dim8(c, F, "F must be a positive multiple of 8");
    if (!c.err.empty()) return (g_err = c.err, SIZE_MAX);
    return block_ws(dt, C, T, d, E, k, F).total;
  }
  g_err = "unknown op '" + o + "'";
  return SIZE_MAX;
}

int foe_route_ex(foe_dtype dt, int G, int T, int d, int E, int k, foe_gating gating,
                 const void* x, const void* w_router, const float* bias, int32_t* topk_idx,
                 float* topk_w, void* stream) {
  Check c;
  check_dtype(c, dt);
  c.need(G >= 1 && G <= 64, "G must be in [1, 64]");
  check_route_shape(c, T, E, k);
  c.need((long long)G * T * (k < 1 ? 1 : k) <= INT_MAX, "G*T*k must fit in int32");
  check_dim8(c, d, "d must be a positive multiple of 8");
  c.need(gating == FOE_GATE_RENORM || gating == FOE_GATE_GLOBAL,
         "gating must be FOE_GATE_RENORM or FOE_GATE_GLOBAL");
  const bool any = T > 0;
  c.tensor(x, any, "x");
  c.tensor(w_router, any, "w_router");
  c.small(bias, false, "bias");
  c.small(topk_idx, any, "topk_idx");
  c.small(topk_w, any, "topk_w");
  if (!c.err.empty()) return fail(FOE_ERR_INVALID, "foe_route_ex: " + c.err);
  if (!route_one_pass(G, E))
    return fail(FOE_ERR_UNSUPPORTED, "foe_route_ex: G > 1 needs G*E <= 256");
  hipError_t e = launch_route(dt, G, T, d, E, k, gating, x, w_router, bias, topk_idx, topk_w,
                              reinterpret_cast<hipStream_t>(stream));
  if (e != hipSuccess) return hip_fail(e, "foe_route_ex");
  return FOE_OK;
}

int foe_route(foe_dtype dt, int T, int d, int E, int k, const void* x, const void* w_router,
              const float* bias, int32_t* topk_idx, float* topk_w, void* stream) {
  Check c;
  check_dtype(c, dt);
  check_route_shape(c, T, E, k);
  check_dim8(c, d, "d must be a positive multiple of 8");
  const bool any = T > 0;
  c.tensor(x, any, "x");
  c.tensor(w_router, any, "w_router");
  c.small(bias, false, "bias");
  c.small(topk_idx, any, "topk_idx");
  c.small(topk_w, any, "topk_w");
  if (!c.err.empty()) return fail(FOE_ERR_INVALID, "foe_route: " + c.err);
  hipError_t e = launch_route(dt, 1, T, d, E, k, FOE_GATE_RENORM, x, w_router, bias, topk_idx,
                              topk_w, reinterpret_cast<hipStream_t>(stream));
  if (e != hipSuccess) return hip_fail(e, "foe_route");
  return FOE_OK;
}

int foe_permute(foe_dtype dt, int T, int d, int E, int k, const int32_t* topk_idx, const void* x,
                int32_t* expert_counts, int32_t* expert_offsets, int32_t* sorted_src,
                int32_t* row_of, void* x_perm, void* ws, size_t ws_bytes, void* stream) {
  Check c;
  check_dtype(c, dt);
  check_route_shape(c, T, E, k);
  check_dim8(c, d, "d must be a positive multiple of 8");
  const bool any = T > 0;
  c.small(topk_idx, any, "topk_idx");
  c.tensor(x, any, "x");
  c.small(expert_counts, false, "expert_counts");
  c.small(expert_offsets, true, "expert_offsets");
  c.small(sorted_src, any, "sorted_src");
  c.small(row_of, any, "row_of");
  c.tensor(x_perm, any, "x_perm");
  if (!c.err.empty()) return fail(FOE_ERR_INVALID, "foe_permute: " + c.err);
  const size_t need = permute_scratch_bytes(T, k, E, 1);
  if (need > 0 && (ws == nullptr || !aligned16(ws)))
    return fail(FOE_ERR_INVALID, "foe_permute: ws is NULL or not 16-byte aligned");
  if (ws_bytes < need)
    return fail(FOE_ERR_WORKSPACE, "foe_permute: workspace needs " + std::to_string(need) +
                                       " bytes, got " + std::to_string(ws_bytes));
  hipError_t e = launch_permute(dt, T, d, E, k, topk_idx, x, expert_counts, expert_offsets,
                                sorted_src, row_of, x_perm, ws,
                                reinterpret_cast<hipStream_t>(stream));
  if (e != hipSuccess) return hip_fail(e, "foe_permute");
  return FOE_OK;
}

int foe_expert_ffn(foe_dtype dt, int E, int d, int F, int rows, const void* x_perm,
                   const int32_t* expert_offsets, const void* w_gate, const void* w_up,
                   const void* w_down, void* y_perm, void* ws, size_t ws_bytes, void* stream) {
  Check c;
  check_dtype(c, dt);
  c.need(E >= 1 && E <= 256, "E must be in [1, 256]");
  c.need(rows >= 0, "rows must be >= 0");
  check_dim8(c, d, "d must be a positive multiple of 8");
  check_dim8(c, F, "F must be a positive multiple of 8");
  const bool any = rows > 0;
  c.tensor(x_perm, any, "x_perm");
  c.small(expert_offsets, any, "expert_offsets");
  c.tensor(w_gate, any, "w_gate");
  c.tensor(w_up, any, "w_up");
  c.tensor(w_down, any, "w_down");
  c.tensor(y_perm, any, "y_perm");
  if (!c.err.empty()) return fail(FOE_ERR_INVALID, "foe_expert_ffn: " + c.err);
  if (dt == FOE_BF16 && !(operand_fits(rows, d, 2) && operand_fits(rows, F, 2)))
    return fail(FOE_ERR_UNSUPPORTED, "foe_expert_ffn: rows*d and rows*F must stay below 2^30 bf16 elements");
  const size_t need = any ? ffn_scratch_bytes(dt, rows, F) : 0;
  if (need > 0 && (ws == nullptr || !aligned16(ws)))
    return fail(FOE_ERR_INVALID, "foe_expert_ffn: ws is NULL or not 16-byte aligned");
  if (ws_bytes < need)
    return fail(FOE_ERR_WORKSPACE, "foe_expert_ffn: workspace needs " + std::to_string(need) +
                                       " bytes, got " + std::to_string(ws_bytes));
  hipError_t e = launch_expert_ffn(dt, E, d, F, rows, x_perm, expert_offsets, w_gate, w_up,
                                   w_down, y_perm, ws, reinterpret_cast<hipStream_t>(stream));
  if (e != hipSuccess) return hip_fail(e, "foe_expert_ffn");
  return FOE_OK;
}

int foe_combine(foe_dtype dt, int T, int d, int k, const void* y_perm, const int32_t* row_of,
                const float* topk_w, const void* residual, void* out, void* stream) {
  Check c;
  check_dtype(c, dt);
  c.need(T >= 0, "T must be >= 0");
  c.need(k >= 1 && k <= 256, "k must be in [1, 256]");
  c.need((long long)T * (k < 1 ? 1 : k) <= INT_MAX, "T*k must fit in int32");
  check_dim8(c, d, "d must be a positive multiple of 8");
  const bool any = T > 0;
  c.tensor(y_perm, any, "y_perm");
  c.small(row_of, any, "row_of");
  c.small(topk_w, any, "topk_w");
  c.tensor(residual, false, "residual");
  c.tensor(out, any, "out");
  if (!c.err.empty()) return fail(FOE_ERR_INVALID, "foe_combine: " + c.err);
  hipError_t e = launch_combine(dt, T, d, k, y_perm, row_of, topk_w, residual, out,
                                reinterpret_cast<hipStream_t>(stream));
  if (e != hipSuccess) return hip_fail(e, "foe_combine");
  return FOE_OK;
}

int foe_reduce(foe_dtype dt, int C, int T, int d, const void* partials, const void* residual,
               float scale, void* out, void* stream) {
  Check c;
  check_dtype(c, dt);
  c.need(C >= 1 && C <= 64, "C must be in [1, 64]");
  c.need(T >= 0, "T must be >= 0");
  check_dim8(c, d, "d must be a positive multiple of 8");
  const bool any = T > 0;
  c.tensor(partials, any, "partials");
  c.tensor(residual, false, "residual");
  c.tensor(out, any, "out");
  if (!c.err.empty()) return fail(FOE_ERR_INVALID, "foe_reduce: " + c.err);
  hipError_t e = launch_reduce(dt, C, T, d, partials, residual, scale, out,
                               reinterpret_cast<hipStream_t>(stream));
  if (e != hipSuccess) return hip_fail(e, "foe_reduce");
  return FOE_OK;
}

int foe_cluster_block(foe_dtype dt, int C, int T, int d, int E, int k, int F, const void* x,
                      const void* w_router, const float* bias, const void* w_gate,
                      const void* w_up, const void* w_down, float reduce_scale, void* out,
                      void* ws, size_t ws_bytes, void* stream) {
  return foe_cluster_block_ex(dt, C, T, d, E, k, F, FOE_GATE_RENORM, x, w_router, bias, w_gate,
                              w_up, w_down, reduce_scale, out, ws, ws_bytes, stream);
}

}  // extern "C"

namespace foe {
namespace {
// Argument checks of the whole block (every pointer and size; nothing is
// enqueued).  Returns FOE_OK or the status to report, with the message set.
int check_block_args(const char* who, foe_dtype dt, int C, int T, int d, int E, int k, int F,
                     foe_gating gating, const void* x, const void* w_router, const float* bias,
                     const void* w_gate, const void* w_up, const void* w_down, const void* out) {
  Check c;
  c.need(gating == FOE_GATE_RENORM || gating == FOE_GATE_GLOBAL,
         "gating must be FOE_GATE_RENORM or FOE_GATE_GLOBAL");
  check_dtype(c, dt);
  c.need(C >= 1 && C <= 64, "C must be in [1, 64]");
  check_route_shape(c, T, E, k);
  c.need((long long)C * T * (k < 1 ? 1 : k) <= INT_MAX, "C*T*k must fit in int32");
  check_dim8(c, d, "d must be a positive multiple of 8");
  check_dim8(c, F, "F must be a positive multiple of 8");
  const bool any = T > 0;
  c.tensor(x, any, "x");
  c.tensor(w_router, any, "w_router");
  c.small(bias, false, "bias");
  c.tensor(w_gate, any, "w_gate");
  c.tensor(w_up, any, "w_up");
  c.tensor(w_down, any, "w_down");
  c.tensor(out, any, "out");
  if (!c.err.empty()) return fail(FOE_ERR_INVALID, std::string(who) + ": " + c.err);
  if (gating == FOE_GATE_GLOBAL && !route_one_pass(C, E))
    return fail(FOE_ERR_UNSUPPORTED,
                std::string(who) + ": global gating needs C == 1 or C*E <= 256");
  const long long CR = (long long)C * T * k;
  if (any && dt == FOE_BF16 &&
      !(operand_fits(T, d, 2) && operand_fits(CR, F, 2) && operand_fits(CR, d, 2)))
    return fail(FOE_ERR_UNSUPPORTED, std::string(who) +
                                         ": T*d, C*T*k*F and C*T*k*d must stay below 2^30 "
                                         "bf16 elements");
  return FOE_OK;
}
}  // namespace
}  // namespace foe

extern "C" {

int foe_cluster_block_ex(foe_dtype dt, int C, int T, int d, int E, int k, int F,
                         foe_gating gating, const void* x, const void* w_router,
                         const float* bias, const void* w_gate, const void* w_up,
                         const void* w_down, float reduce_scale, void* out, void* ws,
                         size_t ws_bytes, void* stream) {
  const int rc = check_block_args("foe_cluster_block", dt, C, T, d, E, k, F, gating, x, w_router,
                                  bias, w_gate, w_up, w_down, out);
  if (rc != FOE_OK) return rc;
  if (T == 0) return FOE_OK;
  const long long CR = (long long)C * T * k;
  const BlockWs L = block_ws(dt, C, T, d, E, k, F);
  if (ws == nullptr || !aligned16(ws))
    return fail(FOE_ERR_INVALID, "foe_cluster_block: ws is NULL or not 16-byte aligned");
  if (ws_bytes < L.total)
    return fail(FOE_ERR_WORKSPACE, "foe_cluster_block: workspace needs " +
                                       std::to_string(L.total) + " bytes, got " +
                                       std::to_string(ws_bytes));

  hipStream_t s = reinterpret_cast<hipStream_t>(stream);
  unsigned char* base = reinterpret_cast<unsigned char*>(ws);
  int32_t* topk_idx = reinterpret_cast<int32_t*>(base + L.topk_idx);
  float* topk_w = reinterpret_cast<float*>(base + L.topk_w);
  int32_t* counts = reinterpret_cast<int32_t*>(base + L.counts);
  int32_t* offsets = reinterpret_cast<int32_t*>(base + L.offsets);
  int32_t* sorted_src = reinterpret_cast<int32_t*>(base + L.sorted_src);
  int32_t* row_of = reinterpret_cast<int32_t*>(base + L.row_of);
  void* y = base + L.y;
  void* perm_ws = base + L.perm;
  void* ffn_ws = base + L.ffn;

  // 1. routing of every cluster in one grid (Section 3.1: one score vector,
  //    per-group top-k); with many pairs it also counts the experts of its
  //    token blocks, the histogram of the dispatch
  const bool sel = ffn_sel_ok(dt, C, E, T, k);
  const RoutePlan rp = plan_route(dt, C, T, d, E, sel);
  int32_t* rcnt = reinterpret_cast<int32_t*>(base + L.rcnt);
  const bool use_rc = !sel && index_takes_route_counts(T, E, k, rp.nblk);
  hipError_t e = launch_route(dt, C, T, d, E, k, gating, x, w_router, bias, topk_idx, topk_w, s,
                              sel ? reinterpret_cast<int32_t*>(base + L.cnt) : nullptr,
                              ceil_div(d, 128), use_rc ? rcnt : nullptr);
  if (e != hipSuccess) return hip_fail(e, "foe_cluster_block/route");
  if (sel) {
    // few pairs per expert: the FFN workgroups list their expert's pairs from
    // the routing decisions themselves (the dispatch in its stable order,
    // without an index pass), y is indexed by pair, and the down kernel also
    // forms the combine (its arrival counters were cleared by the route
    // kernel above; every token has C*k valid pairs since k <= E)
    FusedCombine fc;
    fc.w = topk_w;
    fc.x = static_cast<const bf16*>(x);
    fc.out = static_cast<bf16*>(out);
    fc.cnt = reinterpret_cast<int32_t*>(base + L.cnt);
    fc.scale = reduce_scale;
    fc.C = C;
    fc.k = k;
    e = launch_expert_ffn_sel(C, E, d, F, T, k, x, topk_idx, w_gate, w_up, w_down, y, ffn_ws, s,
                              fc);
    if (e != hipSuccess) return hip_fail(e, "foe_cluster_block/expert_ffn");
    return FOE_OK;
  }
  // many rows per expert (bf16): both grouped GEMMs in one persistent launch,
  // whose counters the index pass clears.  Its h rows must be whole 128-byte
  // cache lines (F a multiple of 64), so that no line holds rows of two
  // M-tiles: a down tile then never caches part of a row that another tile is
  // still writing.
  const bool fused = FOE_FFN_FUSED && dt == FOE_BF16 && CR >= 64LL * C * E && F % 64 == 0;
  int32_t* sync = reinterpret_cast<int32_t*>(base + L.sync);
  const int nsync = fused ? (int)ffn_sync_ints(C * E, (int)CR) : 0;
  // 2. dispatch: expert histogram, prefix sum and stable ranks of all clusters
  e = launch_index(T, E, k, C, topk_idx, counts, offsets, sorted_src, row_of, perm_ws, s, sync,
                   nsync, use_rc ? rcnt : nullptr, rp.tok_per_blk, rp.nblk);
  if (e != hipSuccess) return hip_fail(e, "foe_cluster_block/index");
  // 3. one grouped SwiGLU FFN over the C*E experts (weights are [C*E, ...]),
  //    reading the rows of x through sorted_src
  if (fused)
    e = launch_expert_ffn_fused(C * E, d, F, (int)CR, x, sorted_src, k, T, offsets, w_gate, w_up,
                                w_down, y, ffn_ws, sync, s);
  else
    e = launch_expert_ffn_ex(dt, C * E, d, F, (int)CR, x, sorted_src, k, T, offsets, w_gate,
                             w_up, w_down, y, ffn_ws, s);
  if (e != hipSuccess) return hip_fail(e, "foe_cluster_block/expert_ffn");
  // 4. weighted combine of every cluster and the local cross-cluster reduction
  e = launch_combine_clusters(dt, C, T, d, k, y, row_of, topk_w, x, reduce_scale, out, s);
  if (e != hipSuccess) return hip_fail(e, "foe_cluster_block/combine");
  return FOE_OK;
}

int foe_cluster_block_noalloc(foe_dtype dt, int C, int T, int d, int E, int k, int F,
                              const void* x, const void* w_router, const float* bias,
                              const void* w_gate, const void* w_up, const void* w_down,
                              float reduce_scale, void* out, void* stream) {
  const int rc = check_block_args("foe_cluster_block_noalloc", dt, C, T, d, E, k, F,
                                  FOE_GATE_RENORM, x, w_router, bias, w_gate, w_up, w_down, out);
  if (rc != FOE_OK) return rc;
  const size_t need = block_ws(dt, C, T, d, E, k, F).total;
  if (need > kNoAllocScratchBytes)
    return fail(FOE_ERR_UNSUPPORTED,
                "foe_cluster_block_noalloc: these sizes need " + std::to_string(need) +
                    " bytes of scratch; the entry point holds at most " +
                    std::to_string(kNoAllocScratchBytes) + " (use foe_cluster_block)");
  if (T == 0) return FOE_OK;
  void* ws = nullptr;
  const int rs = noalloc_scratch(&ws);
  if (rs != FOE_OK) return rs;
  return foe_cluster_block_ex(dt, C, T, d, E, k, F, FOE_GATE_RENORM, x, w_router, bias, w_gate,
                              w_up, w_down, reduce_scale, out, ws, kNoAllocScratchBytes, stream);
}

size_t foe_group_attention_workspace_bytes(int H, int S, int d, int nq, int hd) {
  Check c;
  c.need(H >= 1 && H <= 64, "H must be in [1, 64]");
  c.need(S >= 0, "S must be >= 0");
  check_dim8(c, d, "d must be a positive multiple of 8");
  c.need(nq >= 1 && nq <= 64, "nq must be in [1, 64]");
  c.need(hd == 96 || hd == 128, "hd must be 96 or 128");
  if (!c.err.empty()) return (g_err = c.err, SIZE_MAX);
  return group_attention_scratch_bytes(H, S, d, nq, hd);
}

int foe_group_attention(foe_dtype dt, int H, int S, int d, int nq, int hd, float theta,
                        float scale, const void* x, const void* w_qkv, const void* w_o,
                        void* r_full, void* ws, size_t ws_bytes, void* stream) {
  Check c;
  check_dtype(c, dt);
  c.need(H >= 1 && H <= 64, "H must be in [1, 64]");
  c.need(S >= 0, "S must be >= 0");
  check_dim8(c, d, "d must be a positive multiple of 8");
  c.need(nq >= 1 && nq <= 64, "nq must be in [1, 64]");
  c.need(theta > 0.f && scale > 0.f, "theta and scale must be > 0");
  const bool any = S > 0;
  c.tensor(x, any, "x");
  c.tensor(w_qkv, any, "w_qkv");
  c.tensor(w_o, any, "w_o");
  c.tensor(r_full, any, "r_full");
  if (!c.err.empty()) return fail(FOE_ERR_INVALID, "foe_group_attention: " + c.err);
  if (dt != FOE_BF16 || (hd != 96 && hd != 128))
    return fail(FOE_ERR_UNSUPPORTED, "foe_group_attention: bf16 with hd = 96 or 128 only");
  const long long rows = (long long)H * S;
  if (!(operand_fits(rows, d, 2) && operand_fits(rows, (long long)(nq + 2) * hd, 2)))
    return fail(FOE_ERR_UNSUPPORTED,
                "foe_group_attention: H*S*d and H*S*(nq+2)*hd must stay below 2^30");
  if (!any) return FOE_OK;
  const size_t need = group_attention_scratch_bytes(H, S, d, nq, hd);
  if (ws == nullptr || !aligned16(ws))
    return fail(FOE_ERR_INVALID, "foe_group_attention: ws is NULL or not 16-byte aligned");
  if (ws_bytes < need)
    return fail(FOE_ERR_WORKSPACE, "foe_group_attention: workspace needs " +
                                       std::to_string(need) + " bytes, got " +
                                       std::to_string(ws_bytes));
  hipError_t e = launch_group_attention(H, S, d, nq, hd, theta, scale, x, w_qkv, w_o, r_full, ws,
                                        reinterpret_cast<hipStream_t>(stream));
  if (e != hipSuccess) return hip_fail(e, "foe_group_attention");
  return FOE_OK;
}

int foe_profile_enable(int on) {
  std::lock_guard<std::mutex> lock(g_prof_mu);
  g_prof_on = on != 0;
  return FOE_OK;
}

int foe_profile_reset(void) {
  std::lock_guard<std::mutex> lock(g_prof_mu);
  g_recs.clear();
  g_events_used = 0;
  return FOE_OK;
}

int foe_profile_kernel(const char* name, int* launches, double* total_ms) {
  if (name == nullptr || launches == nullptr || total_ms == nullptr)
    return fail(FOE_ERR_INVALID, "foe_profile_kernel: NULL argument");
  std::lock_guard<std::mutex> lock(g_prof_mu);
  int n = 0;
  double ms = 0.0;
  for (const ProfRec& r : g_recs) {
    if (r.name != name) continue;
    hipEvent_t a = g_events[2 * r.ev], b = g_events[2 * r.ev + 1];
    hipError_t e = hipEventSynchronize(b);
    if (e != hipSuccess) return hip_fail(e, "foe_profile_kernel");
    float t = 0.f;
    e = hipEventElapsedTime(&t, a, b);
    if (e != hipSuccess) return hip_fail(e, "foe_profile_kernel");
    ms += t;
    ++n;
  }
  if (n == 0) return fail(FOE_ERR_INVALID, std::string("no recorded launch of ") + name);
  *launches = n;
  *total_ms = ms;
  return FOE_OK;
}

int foe_profile_names(char* buf, size_t len) {
  std::lock_guard<std::mutex> lock(g_prof_mu);
  std::string all;
  for (const ProfRec& r : g_recs) {
    const std::string key = "," + r.name + ",";
    if (("," + all + ",").find(key) != std::string::npos) continue;
    if (!all.empty()) all += ",";
    all += r.name;
  }
  if (buf != nullptr && len > 0) {
    const size_t n = all.size() < len - 1 ? all.size() : len - 1;
    all.copy(buf, n);
    buf[n] = '\0';
  }
  return (int)all.size() + 1;
}

}  // extern "C"
