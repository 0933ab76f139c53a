"""Checks shared by the block parity tests (GPU) and their CPU self-tests.

The block output is ``out = s * sum_h (x + delta_h) = s*C*x + s*sum_h delta_h``.
The residual part ``s*C*x`` (N(0,1) rows) dominates ``out``, so a bound on
``out`` alone admits large errors in the MoE update.  Every block comparison
therefore also bounds the update part ``out - s*C*x`` relative to its own
largest value.  That part is recovered from a stored output, which is rounded
once to the storage type (8 significant bits for bf16, 24 for fp32: at most
``2^-8 |out|`` resp. ``2^-24 |out|`` per element), so only the error beyond
that rounding is counted.

Routing near-ties: a token whose oracle fp32 margin between the k-th and
(k+1)-th score is below ``EXEMPT`` may be routed either way.  For such tokens
the oracle adopts the device's expert ids (its weights then follow from the
oracle's own scores at those ids), so every row of the output is compared.
"""

import numpy as np

import oracle

EXEMPT = 1e-5
TOL = {"bf16": 2e-2, "f32": 1e-4}
ROUND = {"bf16": 2.0 ** -8, "f32": 2.0 ** -24}


def rel_err(got, ref):
    ref = np.asarray(ref, np.float64)
    den = np.max(np.abs(ref)) if ref.size else 0.0
    if ref.size == 0:
        return 0.0
    return float(np.max(np.abs(np.asarray(got, np.float64) - ref)) / (den if den > 0 else 1.0))


def update_part_err(got, ref, base, dt):
    """Error of the update part ``ref - base`` beyond the output rounding,
    relative to the largest value of that part."""
    got = np.asarray(got, np.float64)
    ref = np.asarray(ref, np.float64)
    excess = np.maximum(np.abs(got - ref) - ROUND[dt] * np.abs(ref), 0.0)
    den = np.max(np.abs(ref - base)) if ref.size else 0.0
    if ref.size == 0:
        return 0.0
    return float(np.max(excess) / (den if den > 0 else 1e-30))


def oracle_routes(x, clusters, k):
    return [oracle.route(x, cl["w_router"], cl.get("bias"), k) for cl in clusters]


def exempt_mask(routes):
    m = np.zeros(routes[0]["idx"].shape[0], dtype=bool)
    for r in routes:
        m |= r["margin"] < EXEMPT
    return m


def oracle_block(x, clusters, k, reduce_scale=None, gating="renorm", routes=None,
                 device_idx=None):
    """The oracle's block output with near-tie tokens routed as the device
    routed them.  ``device_idx`` ([C,T,k] ids, or None when no token is
    exempt) supplies those tokens' ids.  Returns ``(out, routes, n_adopted)``."""
    C = len(clusters)
    scale = 1.0 / C if reduce_scale is None else reduce_scale
    if routes is None:
        routes = oracle_routes(x, clusters, k)
    adopted = 0
    for h, r in enumerate(routes):
        ex = r["margin"] < EXEMPT
        if ex.any():
            if device_idx is None:
                raise ValueError("exempt tokens need the device's ids")
            r["idx"] = r["idx"].copy()
            r["idx"][ex] = np.asarray(device_idx[h])[ex]
            r["w"] = oracle.gate_weights(r["logits"], r["idx"])
            adopted += int(ex.sum())
    if gating == "global":
        ws = oracle.gate_weights_global([r["logits"] for r in routes], [r["idx"] for r in routes])
        for r, w in zip(routes, ws):
            r["w"] = w
    elif gating != "renorm":
        raise ValueError(gating)
    res = [oracle.cluster_delta(x, cl, k, r) for cl, r in zip(clusters, routes)]
    out = oracle.reduce_partials(np.stack([r["delta"] for r in res]), scale, residual=x)
    return out, res, adopted


def block_errors(got, ref, x, C, reduce_scale, dt):
    """(error of out, error of the update part) of a block output."""
    scale = 1.0 / C if reduce_scale is None else reduce_scale
    base = scale * C * np.asarray(x, np.float64)
    return rel_err(got, ref), update_part_err(got, ref, base, dt)
