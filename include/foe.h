/*
 * foe.h - C ABI of the MI355X (gfx950) per-cluster MoE block of
 *         Federation of Experts (FoE).
 *
 * One FoE layer splits its MoE block into H expert groups ("clusters"), each
 * owning a contiguous block of experts (Section 3, notation table).  All groups
 * route the same cross-group averaged residual r_full with one router and each
 * keeps its own top-k/H experts (Section 3.1, routing equation); every group
 * then forms its partial x'[h] = r_full + sum_e w_h[i,e] FFN_e(r_full)
 * (Table 3, "MoE update" row) and the partials are averaged (Table 3,
 * "Cross-group avg." row; Section 3.1, "Layer boundaries").  Groups that share
 * a GPU combine their partials locally (Section 3.2).  This library runs that
 * block for C clusters co-resident on one GPU.
 *
 * Per cluster: T tokens, hidden size d, E experts, top-k k (the paper's k/H),
 * expert FFN size F, R = T*k (token, slot) pairs.
 *
 * Conventions shared by every entry point
 *  - Pointers are DEVICE pointers owned by the caller unless marked (host).
 *    Tensors are dense row-major; weights are [out, in] (K-contiguous).
 *  - dt selects the storage type of activations, weights and FFN outputs:
 *    FOE_F32 (fp32) or FOE_BF16 (bf16).  Router bias, routing weights and all
 *    accumulation are fp32 in both cases.  Indices are int32.
 *  - Every tensor pointer must be 16-byte aligned; d and F must be multiples
 *    of 8 (rows are moved as 128-bit vectors).
 *  - Limits: 0 <= T, 1 <= k <= E <= 256, 1 <= C <= 64, d, F >= 8.  T = 0 is an
 *    empty batch: outputs are empty and, for foe_permute, counts/offsets are
 *    written as zeros.
 *  - `stream` is a hipStream_t (NULL = the null stream).  Calls only enqueue
 *    work on it and return; the caller synchronises.  No call allocates device
 *    memory: scratch comes from the caller's workspace `ws` of `ws_bytes`
 *    bytes (16-byte aligned), sized with foe_workspace_bytes().
 *  - Return value: FOE_OK (0) or a negative foe_status.  All argument checks
 *    run on the host before anything is enqueued, so an error leaves device
 *    memory untouched.  foe_last_error() gives a message for the calling
 *    thread's last failure.
 *  - Outputs are bit-deterministic: the same inputs give the same bits on
 *    every call (no floating point atomics; fixed summation orders).
 *  - Device-side index data supplied by the caller (topk_idx, offsets,
 *    row_of) is not trusted for memory safety: out-of-range entries are
 *    skipped rather than dereferenced (documented per entry point).
 */
#ifndef FOE_H
#define FOE_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
    FOE_OK = 0,
    FOE_ERR_INVALID = -1,     /* bad shape, null/misaligned pointer, bad dtype */
    FOE_ERR_UNSUPPORTED = -2, /* valid request the library does not implement */
    FOE_ERR_WORKSPACE = -3,   /* ws_bytes below foe_workspace_bytes()        */
    FOE_ERR_HIP = -4          /* the HIP runtime reported an error            */
} foe_status;

typedef enum { FOE_F32 = 0, FOE_BF16 = 1 } foe_dtype;

/*
 * Routing weights of the selected experts (Section 3.1 routing equation; the
 * paper leaves renormalisation open):
 *   FOE_GATE_RENORM  softmax over the k selected scores of the group: the
 *                    global softmax renormalised over the selection (each
 *                    token's k weights of a group sum to 1)
 *   FOE_GATE_GLOBAL  the global softmax over the single score vector of all
 *                    C*E experts (all groups), taken at the selected experts
 *                    and not renormalised (OLMoE-style gating; each group's
 *                    weights sum to its share of the probability mass)
 */
typedef enum { FOE_GATE_RENORM = 0, FOE_GATE_GLOBAL = 1 } foe_gating;

/*
 * foe_route - router scores, per-group top-k and routing weights.
 * Section 3.1, routing equation: g[i] = Router(r_full[i]) and
 * I_h[i], w_h[i] = TopK over the group's experts of g[i].
 *
 *   x         [T,d] dt        the block input r_full (one row per token)
 *   w_router  [E,d] dt        this cluster's router rows (linear router)
 *   bias      [E]   fp32      added to the scores, or NULL
 *   topk_idx  [T,k] int32 out expert ids, descending score; equal scores ->
 *                             lower id first.  Scores are fp32 (fp32
 *                             accumulation of the dt products, plus bias).
 *   topk_w    [T,k] fp32  out softmax over the k selected scores (each row
 *                             sums to 1; equals the global softmax
 *                             renormalised over the selection)
 * Needs no workspace.
 */
int foe_route(foe_dtype dt, int T, int d, int E, int k,
              const void* x, const void* w_router, const float* bias,
              int32_t* topk_idx, float* topk_w, void* stream);

/*
 * foe_route_ex - foe_route for G groups sharing x, with a gating choice.
 * The G router matrices w_router [G,E,d] (and bias [G,E] or NULL) form one
 * score vector of G*E experts per token; group h takes its top-k over its own
 * block of E scores and writes topk_idx/topk_w [G,T,k] rows h*T.. (ids local
 * to the group, 0..E-1).  gating: FOE_GATE_RENORM (foe_route's weights) or
 * FOE_GATE_GLOBAL (softmax over all G*E scores, not renormalised).
 * FOE_ERR_UNSUPPORTED when G*E > 256 with G > 1.  Needs no workspace.
 */
int foe_route_ex(foe_dtype dt, int G, int T, int d, int E, int k, foe_gating gating,
                 const void* x, const void* w_router, const float* bias,
                 int32_t* topk_idx, float* topk_w, void* stream);

/*
 * foe_permute - expert histogram, prefix sum and stable token permutation:
 * the on-device form of the intra-group dispatch (Section 3.2; on one GPU the
 * local activation rate is 1 and dispatch never leaves the device).
 *
 *   topk_idx        [T,k]   int32  from foe_route (or any k ids per token)
 *   x               [T,d]   dt     rows to dispatch
 *   expert_counts   [E]     int32 out pairs per expert (may be NULL)
 *   expert_offsets  [E+1]   int32 out exclusive prefix sum; offsets[E] = number
 *                                  of valid pairs (T*k when all ids are valid)
 *   sorted_src      [T*k]   int32 out flat pair f = i*k + j held by permuted
 *                                  row p; order = (expert asc, token asc)
 *   row_of          [T*k]   int32 out inverse: row_of[f] = p (-1 for a pair
 *                                  whose id is outside [0,E); such pairs are
 *                                  dropped and trailing sorted_src/x_perm
 *                                  rows are left unwritten)
 *   x_perm          [T*k,d] dt    out x_perm[p] = x[sorted_src[p] / k]
 *   ws, ws_bytes    workspace of foe_workspace_bytes("permute", ...)
 */
int foe_permute(foe_dtype dt, int T, int d, int E, int k,
                const int32_t* topk_idx, const void* x,
                int32_t* expert_counts, int32_t* expert_offsets,
                int32_t* sorted_src, int32_t* row_of, void* x_perm,
                void* ws, size_t ws_bytes, void* stream);

/*
 * foe_expert_ffn - grouped SwiGLU expert FFN over the permuted rows
 * (Table 3 "MoE update": FFN_e applied to the rows routed to expert e).
 * Rows offsets[e] .. offsets[e+1]-1 of x_perm go through expert e:
 *   y = W_d[e] (silu(W_g[e] x) * (W_u[e] x)),  silu(z) = z / (1 + exp(-z)).
 * bf16: products in bf16 MFMA with fp32 accumulation; the hidden activation
 * is rounded to bf16 (nearest even) before the down projection.
 *
 *   rows            number of permuted rows (T*k)
 *   x_perm          [rows,d]  dt
 *   expert_offsets  [E+1]     int32 (device) segment bounds; bounds are
 *                             clamped to [0, rows] and a decreasing bound
 *                             gives an empty segment
 *   w_gate, w_up    [E,F,d]   dt
 *   w_down          [E,d,F]   dt
 *   y_perm          [rows,d]  dt out (rows outside every segment are not written)
 *   ws, ws_bytes    workspace of foe_workspace_bytes("expert_ffn", ...)
 * bf16 limits: rows*d and rows*F below 2^30 elements (else FOE_ERR_UNSUPPORTED).
 */
int foe_expert_ffn(foe_dtype dt, int E, int d, int F, int rows,
                   const void* x_perm, const int32_t* expert_offsets,
                   const void* w_gate, const void* w_up, const void* w_down,
                   void* y_perm, void* ws, size_t ws_bytes, void* stream);

/*
 * foe_combine - weighted un-permute (Table 3 "MoE update": the weighted sum
 * over the selected experts, plus r_full):
 *   out[i] = residual[i] + sum_{j<k} topk_w[i,j] * y_perm[row_of[i*k+j]]
 * summed in fp32 in slot order j = 0..k-1, rounded once to dt.
 *
 *   y_perm    [T*k,d] dt
 *   row_of    [T*k]   int32   entries outside [0, T*k) contribute nothing
 *   topk_w    [T,k]   fp32
 *   residual  [T,d]   dt      or NULL (then out = the weighted sum only)
 *   out       [T,d]   dt out
 */
int foe_combine(foe_dtype dt, int T, int d, int k,
                const void* y_perm, const int32_t* row_of, const float* topk_w,
                const void* residual, void* out, void* stream);

/*
 * foe_reduce - local reduction of C cluster partials (Table 3 "Cross-group
 * avg."; Section 3.1 final cross-group average; Section 3.2: groups sharing a
 * GPU combine partials locally):
 *   out = scale * sum_{h=0}^{C-1} (residual + partials[h])
 * accumulated in fp32 in the fixed order h = 0..C-1 (residual omitted when
 * NULL).  scale = 1/C is the paper's average.
 *
 *   partials  [C,T,d] dt;  residual [T,d] dt or NULL;  out [T,d] dt
 */
int foe_reduce(foe_dtype dt, int C, int T, int d,
               const void* partials, const void* residual, float scale,
               void* out, void* stream);

/*
 * foe_cluster_block - the whole block for C clusters sharing the input x
 * (all groups route and update the same r_full: Table 3 "Routing" and "MoE
 * update" rows), followed by the local reduction:
 *   out = reduce_scale * sum_h (x + delta_h),
 *   delta_h[i] = sum_{e in I_h[i]} w_h[i,e] FFN_{h,e}(x[i]).
 * One routing pass scores all clusters (one read of x when C*E <= 256) and
 * each cluster takes its top-k over its own experts; the dispatch of all
 * clusters is numbered in one pass (at decode sizes each FFN workgroup lists
 * its expert's pairs itself); one grouped FFN covers all C*E experts and
 * reads the rows of x through the permutation (no permuted copy of x is
 * written); the weighted sums of every cluster and the reduction are formed
 * in one pass (at decode sizes inside the down-projection kernel) and no
 * per-cluster partial is written.  Evaluated as reduce_scale * (C * x + S)
 * with S the fp32 sum of the weighted expert rows in the order
 * (h = 0..C-1, j = 0..k-1).  Weights are FOE_GATE_RENORM.
 *
 *   x         [T,d]       dt
 *   w_router  [C,E,d]     dt;   bias [C,E] fp32 or NULL
 *   w_gate    [C,E,F,d]   dt;   w_up [C,E,F,d] dt;   w_down [C,E,d,F] dt
 *   reduce_scale          1/C = the paper's average, 1 = a plain sum
 *   out       [T,d]       dt out
 *   ws, ws_bytes          workspace of foe_workspace_bytes("cluster_block", ...)
 * bf16 limits: T*d, C*T*k*d and C*T*k*F below 2^30 elements (else
 * FOE_ERR_UNSUPPORTED); C*T*k below 2^31.
 */
int foe_cluster_block(foe_dtype dt, int C, int T, int d, int E, int k, int F,
                      const void* x, const void* w_router, const float* bias,
                      const void* w_gate, const void* w_up, const void* w_down,
                      float reduce_scale, void* out,
                      void* ws, size_t ws_bytes, void* stream);

/*
 * foe_cluster_block_ex - foe_cluster_block with a gating choice (see
 * foe_gating).  FOE_GATE_GLOBAL normalises over all C*E scores of a token and
 * is supported for C == 1 or C*E <= 256 (else FOE_ERR_UNSUPPORTED).  Same
 * workspace as foe_cluster_block.
 */
int foe_cluster_block_ex(foe_dtype dt, int C, int T, int d, int E, int k, int F,
                         foe_gating gating, const void* x, const void* w_router,
                         const float* bias, const void* w_gate, const void* w_up,
                         const void* w_down, float reduce_scale, void* out,
                         void* ws, size_t ws_bytes, void* stream);

/*
 * foe_cluster_block_noalloc - foe_cluster_block (FOE_GATE_RENORM) for callers
 * that cannot allocate device memory or pass a workspace: code under HIP-graph
 * capture, tight serving loops, harnesses that forbid allocation.  Same
 * arguments as foe_cluster_block without ws / ws_bytes, same kernels, same
 * results bit for bit.
 *
 * Its scratch is a static device array of the library, one copy per GPU,
 * reserved when the library's code is first loaded on that GPU and held until
 * the process ends.  Its size is 128 MiB (134217728 bytes): enough for the
 * decode- and prefill-shaped blocks, e.g. C=1, T=8192, d=2048, E=16, k=2,
 * F=1024.  Sizes whose workspace
 * (foe_workspace_bytes("cluster_block", ...)) exceeds it are rejected with
 * FOE_ERR_UNSUPPORTED before anything is enqueued.  The call allocates no
 * device or host memory.
 *
 * Every call on one GPU uses that GPU's one array, which keeps the last call's
 * contents (the block clears what it needs itself): calls that overlap on one
 * GPU (two host threads, or two streams without an ordering between them)
 * race and give undefined results.  Calls ordered on one stream are safe.
 */
int foe_cluster_block_noalloc(foe_dtype dt, int C, int T, int d, int E, int k, int F,
                              const void* x, const void* w_router, const float* bias,
                              const void* w_gate, const void* w_up, const void* w_down,
                              float reduce_scale, void* out, void* stream);

/*
 * foe_group_attention - the per-group attention that feeds the block (Table 3,
 * FoE column, rows "Attn. residual" and "Cross-group avg."):
 *   r[h,i]    = x[h,i] + Attn_h(x[h,:])[i]     (every group its own representation)
 *   r_full[i] = (1/H) sum_h r[h,i]
 * computed as (1/H) (sum_h o[h,i] w_o[h]^T + sum_h x[h,i]) in fp32: the output
 * projections of all groups form one product over the concatenated head
 * outputs, and the residual sum (h = 0..H-1 in order) is added after it.
 * Attn_h: causal self-attention over the S tokens (positions 0..S-1) with one
 * key/value head and nq query heads sharing it (grouped-query attention),
 * scores q.k/sqrt(hd), rotary embedding on q and k pairing dimension i with
 * i+hd/2 at angle (s/scale)*theta^(-2i/hd), bias-free projections.
 *
 *   x        [H,S,d]          bf16
 *   w_qkv    [H,(nq+2)*hd,d]  bf16  rows: nq query heads, the key head, the value head
 *   w_o      [d,H*nq*hd]      bf16  the groups' output projections side by side:
 *                                   columns h*nq*hd .. (h+1)*nq*hd-1 belong to group h
 *   theta    rotary base (> 0);  scale: rotary scaling factor (> 0), positions / scale
 *   r_full   [S,d]            bf16 out
 *   ws, ws_bytes              workspace of foe_group_attention_workspace_bytes()
 * All pointers are device memory owned by the caller, 16-byte aligned (the
 * workspace too); the call enqueues work on `stream` and returns.  One of its
 * kernels (the residual sum) runs on a library-owned stream of the current
 * device, forked from `stream` and joined back to it by events, so all of the
 * call's work still follows earlier work on `stream` and precedes later work
 * (also under HIP-graph capture, where the fork and join become edges).  bf16 only
 * and hd = 96 or 128 (else FOE_ERR_UNSUPPORTED); H*S*d and H*S*(nq+2)*hd must stay
 * below 2^30 elements.  S = 0 is a no-op.
 */
int foe_group_attention(foe_dtype dt, int H, int S, int d, int nq, int hd, float theta,
                        float scale, const void* x, const void* w_qkv, const void* w_o,
                        void* r_full, void* ws, size_t ws_bytes, void* stream);

/* Workspace bytes of foe_group_attention (SIZE_MAX for invalid sizes). */
size_t foe_group_attention_workspace_bytes(int H, int S, int d, int nq, int hd);

/*
 * foe_workspace_bytes - workspace size in bytes for `op` (host string:
 * "route", "permute", "expert_ffn", "combine", "reduce", "cluster_block").
 * Arguments an op does not use are ignored (pass 0); for "expert_ffn" T is the
 * number of rows and k must be 1.  Returns 0 when the op needs no workspace and
 * SIZE_MAX for an unknown op or invalid sizes (foe_last_error() says which).
 */
size_t foe_workspace_bytes(const char* op, foe_dtype dt, int C, int T, int d,
                           int E, int k, int F);

/* Message for the calling thread's last failed call ("" if none). */
const char* foe_last_error(void);

/*
 * Kernel timing (for measurement).  While enabled, every kernel the library
 * enqueues carries two HIP events that its dispatch stamps at its start and
 * end (on the same stream); the records accumulate until foe_profile_reset().
 * Reading waits on the events.
 *   foe_profile_enable(1/0)          start / stop recording (returns FOE_OK)
 *   foe_profile_reset()              drop all records
 *   foe_profile_kernel(name, &n, &ms)  launches and summed milliseconds of the
 *                                    kernel `name` (host string); FOE_ERR_INVALID
 *                                    if no launch of that name was recorded
 *   foe_profile_names(buf, len)      comma-separated names recorded so far
 *                                    (host buffer); returns the length needed
 */
int foe_profile_enable(int on);
int foe_profile_reset(void);
int foe_profile_kernel(const char* name, int* launches, double* total_ms);
int foe_profile_names(char* buf, size_t len);

#ifdef __cplusplus
}
#endif

#endif /* FOE_H */
