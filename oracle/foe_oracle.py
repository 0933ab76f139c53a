"""Plain CPU oracle of the Federation-of-Experts per-cluster MoE block.

TEST INFRASTRUCTURE ONLY.  This module is the checker that the HIP path is
compared against.  Only the test suite, ``__graft_entry__.smoke()`` and the
``cpu_baseline`` leg of ``bench.py`` may import it; the product path never does.
It shares no code with the HIP library or its Python binding.

What the block computes (one cluster, i.e. one expert group ``h`` of the paper):

* Section 3.1, routing equation: one router produces a score vector ``g[i]``
  over the group's experts and the group keeps its top-``k/H`` experts
  ``I_h[i]`` with weights ``w_h[i]``.  Here ``k`` is the per-cluster top-k.
* Table 3 (FoE column, "MoE update" row): ``x'[h,i] = r_full[i] +
  sum_{e in I_h[i]} w_h[i,e] FFN_e(r_full[i])``.
* Table 3 ("Cross-group avg." row) and Section 3.1 "Layer boundaries": the
  group partials are averaged, ``(1/H) sum_h``; Section 3.2 states that groups
  sharing one GPU combine their partials locally.

Readings where the paper is silent:

* the router is a linear map ``W_r [E,d]`` with an optional bias ``[E]``;
* selection is decided on fp32 scores, descending, equal scores -> lower id;
* the weights are the softmax over the selected scores (global softmax
  renormalised over the top-k; the partition function cancels); the other
  reading, the global softmax over all groups' scores without
  renormalisation, is ``gate_weights_global``;
* ``FFN_e`` is SwiGLU without biases: ``W_d (silu(W_g x) * (W_u x))``;
* dropless: every (token, slot) pair is processed;
* dispatch order is (expert ascending, token ascending) = stable counting sort.

All floating point work is fp64.  The only fp32 step is the selection decision,
where both this oracle and the kernels compare fp32 router scores.
"""

from __future__ import annotations

import numpy as np

__all__ = [
    "router_logits",
    "topk_select",
    "gate_weights",
    "gate_weights_global",
    "route",
    "expert_histogram",
    "permutation",
    "gather_rows",
    "silu",
    "swiglu_ffn",
    "expert_ffn",
    "combine",
    "reduce_partials",
    "cluster_delta",
    "cluster_block",
    "moe_update_tokens",
]


def _f64(a):
    return np.asarray(a, dtype=np.float64)


# ---------------------------------------------------------------------------
# Routing (Section 3.1, routing equation; Table 3 "Routing" row)
# ---------------------------------------------------------------------------

def router_logits(x, w_router, bias=None):
    """Router scores ``g[i] = Router(r_full[i])`` of Section 3.1.

    ``x`` [T,d], ``w_router`` [E,d] (output x input), ``bias`` [E] or None.
    Returns fp64 [T,E]: ``g[i,e] = sum_j x[i,j] W_r[e,j] + b[e]``.
    """
    g = _f64(x) @ _f64(w_router).T
    if bias is not None:
        g = g + _f64(bias)[None, :]
    return g


def topk_select(logits, k):
    """Per-group ``TopK`` of the Section 3.1 routing equation.

    The decision is taken on the scores rounded to fp32 (the precision the
    scores are computed in on the device).  Order: descending score, equal
    scores -> lower expert id first.

    Returns ``idx`` [T,k] int64, ``margin`` [T] (fp32 score of the k-th minus
    the (k+1)-th choice, +inf when k == E) and ``min_gap`` [T] (smallest gap
    between adjacent selected scores, +inf when k == 1).
    """
    g32 = np.asarray(logits).astype(np.float32)
    T, E = g32.shape
    if not 1 <= k <= E:
        raise ValueError("need 1 <= k <= E")
    # a stable sort of the negated scores keeps lower ids first among equals
    order = np.argsort(-g32, axis=1, kind="stable")
    idx = order[:, :k].astype(np.int64)
    srt = np.take_along_axis(g32, order, axis=1).astype(np.float64)
    if k < E:
        margin = srt[:, k - 1] - srt[:, k]
    else:
        margin = np.full(T, np.inf)
    if k > 1:
        min_gap = np.min(srt[:, : k - 1] - srt[:, 1:k], axis=1)
    else:
        min_gap = np.full(T, np.inf)
    return idx, margin, min_gap


def gate_weights(logits, idx):
    """Routing weights ``w_h[i]`` of Section 3.1 (softmax over the selected scores).

    ``w[i,j] = exp(g[i,idx[i,j]] - m_i) / sum_j' exp(g[i,idx[i,j']] - m_i)``
    with ``m_i`` the largest selected score; fp64.
    """
    gsel = np.take_along_axis(_f64(logits), np.asarray(idx), axis=1)
    z = np.exp(gsel - gsel.max(axis=1, keepdims=True))
    return z / z.sum(axis=1, keepdims=True)


def gate_weights_global(group_logits, group_idx):
    """Routing weights with the global softmax of Section 3.1, not renormalised.

    The paper's routers give one score vector per token over the experts of
    all groups; here the G groups' score blocks ``group_logits[h]`` [T,E]
    together form that vector.  The weight of a selected expert ``e`` of group
    ``h`` is its probability under the softmax of the whole vector:
    ``exp(g_h[i,e] - m_i) / sum_{h',e'} exp(g_h'[i,e'] - m_i)`` with ``m_i``
    the largest score of token ``i`` over all groups (any ``m_i`` gives the same
    value; it only keeps ``exp`` in range).  fp64.  Returns one [T,k] array per
    group.
    """
    gl = [_f64(g) for g in group_logits]
    m = np.max(np.stack([g.max(axis=1) for g in gl]), axis=0)[:, None]
    z = np.zeros_like(m)
    for g in gl:
        z = z + np.exp(g - m).sum(axis=1, keepdims=True)
    return [np.exp(np.take_along_axis(g, np.asarray(ix), axis=1) - m) / z
            for g, ix in zip(gl, group_idx)]


def route(x, w_router, bias, k):
    """Router scores, top-k selection and weights for one cluster.

    Returns a dict with ``logits`` (fp64), ``idx``, ``w``, ``margin``, ``min_gap``.
    """
    g = router_logits(x, w_router, bias)
    idx, margin, min_gap = topk_select(g, k)
    return {"logits": g, "idx": idx, "w": gate_weights(g, idx),
            "margin": margin, "min_gap": min_gap}


# ---------------------------------------------------------------------------
# Local dispatch: histogram, prefix sum and stable permutation.  On one GPU the
# intra-group dispatch all-to-all of Section 3.2 (local activation rate 1)
# reduces to this on-device rearrangement of (token, slot) pairs.
# ---------------------------------------------------------------------------

def expert_histogram(idx, E):
    """``counts[e]`` = number of (token, slot) pairs routed to ``e``; ``offsets``
    = exclusive prefix sum with ``offsets[E] = T*k``."""
    counts = np.bincount(np.asarray(idx).ravel(), minlength=E).astype(np.int64)
    offsets = np.zeros(E + 1, dtype=np.int64)
    offsets[1:] = np.cumsum(counts)
    return counts, offsets


def permutation(idx):
    """Stable counting-sort order of the flat pairs ``f = i*k + j`` by expert.

    ``sorted_src[p]`` is the flat pair at permuted row ``p``; ``row_of`` is the
    inverse (``row_of[sorted_src[p]] = p``).
    """
    flat = np.asarray(idx).ravel()
    sorted_src = np.argsort(flat, kind="stable").astype(np.int64)
    row_of = np.empty_like(sorted_src)
    row_of[sorted_src] = np.arange(flat.size, dtype=np.int64)
    return sorted_src, row_of


def gather_rows(x, sorted_src, k):
    """``x_perm[p] = x[sorted_src[p] // k]`` (a pure copy)."""
    return np.asarray(x)[np.asarray(sorted_src) // k]


# ---------------------------------------------------------------------------
# Expert FFN (Table 3 "MoE update" row, FFN_e; SwiGLU per the OLMoE-style model
# of the model-specification appendix)
# ---------------------------------------------------------------------------

def silu(z):
    """``silu(z) = z * sigmoid(z)``."""
    z = _f64(z)
    with np.errstate(over="ignore"):
        return z / (1.0 + np.exp(-z))


def swiglu_ffn(xr, w_gate, w_up, w_down):
    """``FFN_e(x) = W_d (silu(W_g x) * (W_u x))`` on rows of ``xr``; fp64.

    ``w_gate``, ``w_up`` [F,d]; ``w_down`` [d,F].
    """
    xr = _f64(xr)
    a = xr @ _f64(w_gate).T
    u = xr @ _f64(w_up).T
    return (silu(a) * u) @ _f64(w_down).T


def expert_ffn(x_perm, offsets, w_gate, w_up, w_down):
    """Grouped FFN: rows ``offsets[e]:offsets[e+1]`` of ``x_perm`` use expert ``e``."""
    x_perm = _f64(x_perm)
    y = np.zeros((x_perm.shape[0], np.asarray(w_down).shape[1]), dtype=np.float64)
    E = len(offsets) - 1
    for e in range(E):
        lo, hi = int(offsets[e]), int(offsets[e + 1])
        if hi > lo:
            y[lo:hi] = swiglu_ffn(x_perm[lo:hi], w_gate[e], w_up[e], w_down[e])
    return y


# ---------------------------------------------------------------------------
# Combine and reduction
# ---------------------------------------------------------------------------

def combine(y_perm, row_of, w, residual=None):
    """Weighted un-permute: ``delta[i] = sum_j w[i,j] y[row_of[i*k+j]]``.

    Returns ``residual + delta`` (Table 3 "MoE update": the update includes
    ``r_full``) or ``delta`` when ``residual`` is None.
    """
    w = _f64(w)
    T, k = w.shape
    y = _f64(y_perm)[np.asarray(row_of)].reshape(T, k, -1)
    delta = np.einsum("tj,tjd->td", w, y)
    return delta if residual is None else _f64(residual) + delta


def reduce_partials(partials, scale, residual=None):
    """Local cross-cluster reduction (Table 3 "Cross-group avg."; Section 3.1
    last-layer average; Section 3.2 local combining of co-resident groups).

    ``out = scale * sum_h (residual + P_h)`` (``residual`` omitted when None).
    ``scale = 1/C`` is the paper's average.
    """
    P = _f64(partials)
    acc = np.zeros(P.shape[1:], dtype=np.float64)
    for h in range(P.shape[0]):
        acc += P[h] if residual is None else _f64(residual) + P[h]
    return scale * acc


def cluster_delta(x, cl, k, r=None):
    """One cluster's pipeline: route, histogram, permute, grouped FFN, combine.

    ``cl`` holds ``w_router`` [E,d], ``bias`` [E] or None, ``w_gate``/``w_up``
    [E,F,d], ``w_down`` [E,d,F].  ``r`` is the cluster's routing (a ``route``
    dict, possibly with other weights) or None to route here.  Returns a dict
    with every intermediate and ``delta`` = the MoE sum of Table 3 without the
    residual.
    """
    E = np.asarray(cl["w_router"]).shape[0]
    if r is None:
        r = route(x, cl["w_router"], cl.get("bias"), k)
    counts, offsets = expert_histogram(r["idx"], E)
    sorted_src, row_of = permutation(r["idx"])
    x_perm = gather_rows(x, sorted_src, k)
    y = expert_ffn(x_perm, offsets, cl["w_gate"], cl["w_up"], cl["w_down"])
    delta = combine(y, row_of, r["w"])
    r.update(counts=counts, offsets=offsets, sorted_src=sorted_src,
             row_of=row_of, x_perm=x_perm, y=y, delta=delta)
    return r


def cluster_block(x, clusters, k, reduce_scale=None, gating="renorm"):
    """C co-resident clusters sharing the input ``x`` (the paper's ``r_full``).

    ``P_h = x + delta_h`` is the group partial ``x'[h]`` of Table 3 and
    ``out = reduce_scale * sum_h P_h`` (default ``1/C``, the average).
    ``gating`` = "renorm" (``gate_weights``) or "global"
    (``gate_weights_global`` over all clusters' scores).
    Returns ``(out, per_cluster_results)``.
    """
    C = len(clusters)
    if reduce_scale is None:
        reduce_scale = 1.0 / C
    routes = [route(x, cl["w_router"], cl.get("bias"), k) for cl in clusters]
    if gating == "global":
        ws = gate_weights_global([r["logits"] for r in routes], [r["idx"] for r in routes])
        for r, w in zip(routes, ws):
            r["w"] = w
    elif gating != "renorm":
        raise ValueError("gating must be 'renorm' or 'global'")
    res = [cluster_delta(x, cl, k, r) for cl, r in zip(clusters, routes)]
    partials = np.stack([r["delta"] for r in res])
    return reduce_partials(partials, reduce_scale, residual=x), res


def moe_update_tokens(x_rows, cl, k):
    """Table 3 "MoE update" written per token, without any permutation.

    For each row ``x_i``: ``sum_{e in I[i]} w[i,e] FFN_e(x_i)`` (the delta).
    Used on sampled tokens of large workloads and as an independent second
    formulation of the permuted pipeline.  Returns ``(delta, route_dict)``.
    """
    x_rows = _f64(x_rows)
    r = route(x_rows, cl["w_router"], cl.get("bias"), k)
    out = np.zeros_like(x_rows)
    for t in range(x_rows.shape[0]):
        for j in range(k):
            e = int(r["idx"][t, j])
            out[t] += r["w"][t, j] * swiglu_ffn(x_rows[t:t + 1], cl["w_gate"][e],
                                                cl["w_up"][e], cl["w_down"][e])[0]
    return out, r
