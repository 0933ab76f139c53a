"""Seeded synthetic inputs for the per-cluster MoE block.

This module only draws random inputs and rounds them to the storage precision.
It holds none of the block's arithmetic, so the CPU oracle and the HIP path can
both consume what it produces without sharing any of the method's code.

Workload shapes follow the per-group share of the paper's 7B model
(model-specification appendix: d=2048, E/H=8 experts per group, expert FFN
multiplier 1/2), plus the decode / prefill / large variants used to measure the
block.  The paper's own data (trained weights, LongBench prompts) is not
available; N(0,1) activations and N(0, sigma) weights stand in for it.
"""

from __future__ import annotations

import numpy as np

# name -> shape and draw parameters
CONFIGS = {
    "tiny_fp32": dict(dtype="f32", C=1, T=64, d=128, E=4, k=2, F=256,
                      sigma=0.02, seed=0, bias=None),
    "decode_bf16": dict(dtype="bf16", C=1, T=128, d=2048, E=16, k=2, F=1024,
                        sigma=0.02, seed=1, bias=None),
    "prefill_zipf_bf16": dict(dtype="bf16", C=1, T=8192, d=2048, E=16, k=2, F=1024,
                              sigma=0.02, seed=2, bias="zipf1.2"),
    "large_bf16": dict(dtype="bf16", C=1, T=16384, d=4096, E=32, k=4, F=1536,
                       sigma=0.015, seed=3, bias=None),
    "layer_share_bf16": dict(dtype="bf16", C=8, T=4096, d=2048, E=8, k=2, F=1024,
                             sigma=0.02, seed=4, bias=None),
}

CONFIG_ORDER = ["tiny_fp32", "decode_bf16", "prefill_zipf_bf16", "large_bf16",
                "layer_share_bf16"]


def round_to_bf16(a):
    """Round fp32 values to the nearest bf16 value (ties to even); returns fp32.

    NaN/Inf are not expected in the synthetic draws and are not special-cased.
    """
    a = np.ascontiguousarray(a, dtype=np.float32)
    out = np.empty_like(a)
    src = a.reshape(-1).view(np.uint32)
    dst = out.reshape(-1).view(np.uint32)
    step = 1 << 24
    for lo in range(0, src.size, step):
        b = src[lo:lo + step].copy()
        b += np.uint32(0x7FFF) + ((b >> np.uint32(16)) & np.uint32(1))
        b &= np.uint32(0xFFFF0000)
        dst[lo:lo + step] = b
    return out


def bf16_bits(a):
    """Upper 16 bits of fp32 values that are exactly bf16 (as int16 for upload)."""
    a = np.ascontiguousarray(a, dtype=np.float32)
    return (a.view(np.uint32) >> np.uint32(16)).astype(np.uint16).view(np.int16)


def _normal(rng, shape, sigma):
    return rng.standard_normal(shape, dtype=np.float32) * np.float32(sigma)


def zipf_bias(E, s):
    """Per-expert router bias ``b[e] = -s * ln(e + 1)``: the log of the
    unnormalised Zipf(s) pmf over expert ids (rank = id + 1)."""
    return (-s * np.log(np.arange(1, E + 1, dtype=np.float64))).astype(np.float32)


def make_cluster_weights(E, d, F, sigma, seed, h, dtype, bias=None):
    """Router and expert weights of cluster ``h``; drawn from
    ``default_rng([seed, h])`` in the order W_r, W_g, W_u, W_d."""
    rng = np.random.default_rng([seed, h])
    cl = {
        "w_router": _normal(rng, (E, d), sigma),
        "w_gate": _normal(rng, (E, F, d), sigma),
        "w_up": _normal(rng, (E, F, d), sigma),
        "w_down": _normal(rng, (E, d, F), sigma),
        "bias": None,
    }
    if dtype == "bf16":
        for key in ("w_router", "w_gate", "w_up", "w_down"):
            cl[key] = round_to_bf16(cl[key])
    if bias is not None:
        if not bias.startswith("zipf"):
            raise ValueError(bias)
        cl["bias"] = zipf_bias(E, float(bias[4:]))
    return cl


def make_block_inputs(cfg, T=None, weight_set=0):
    """Inputs of one block invocation for a config (name or dict).

    ``x ~ N(0,1) [T,d]`` from ``default_rng(seed + 7919*weight_set)``; cluster
    ``h`` weights from ``default_rng([seed + 7919*weight_set, h])``.  ``T`` may be overridden (the
    first ``T`` rows of the same draw are not kept: a fresh draw of that size).
    bf16 configs round every tensor to bf16.  Returns a dict with ``cfg``,
    ``x`` (fp32 array) and ``clusters`` (list of weight dicts).
    """
    if isinstance(cfg, str):
        cfg = dict(CONFIGS[cfg], name=cfg)
    else:
        cfg = dict(cfg)
    if T is not None:
        cfg["T"] = T
    wseed = cfg["seed"] + 7919 * weight_set
    rng = np.random.default_rng(wseed)
    x = rng.standard_normal((cfg["T"], cfg["d"]), dtype=np.float32)
    if cfg["dtype"] == "bf16":
        x = round_to_bf16(x)
    clusters = [make_cluster_weights(cfg["E"], cfg["d"], cfg["F"], cfg["sigma"],
                                     wseed, h, cfg["dtype"], cfg.get("bias"))
                for h in range(cfg["C"])]
    return {"cfg": cfg, "x": x, "clusters": clusters}


# ---------------------------------------------------------------------------
# Per-group attention that feeds the block (H groups, one KV head each)
# ---------------------------------------------------------------------------

# shapes of the paper's 7B model per group: 16 query / 8 KV heads over H = 8
# groups (nq = 2 query heads share each group's KV head), head dim 128, RoPE
# base 500000 with scaling factor 16; S tokens of one prefill chunk
ATTN_CONFIGS = {
    "attn_tiny_bf16": dict(H=2, S=200, d=256, nq=2, hd=128, theta=500000.0, scale=16.0,
                           sigma=0.05, seed=6),
    "attn_share_bf16": dict(H=8, S=4096, d=2048, nq=2, hd=128, theta=500000.0, scale=16.0,
                            sigma=0.02, seed=5),
    "attn_small_bf16": dict(H=8, S=4096, d=768, nq=1, hd=96, theta=500000.0, scale=16.0,
                            sigma=0.035, seed=7),
}


def make_attention_inputs(cfg, weight_set=0):
    """Inputs of one per-group attention pass for a config (name or dict).

    ``x ~ N(0,1) [H,S,d]`` (one representation per group) from
    ``default_rng(seed + 7919*weight_set)``; group ``h``'s ``w_qkv``
    [(nq+2)*hd, d] and ``w_o`` [d, nq*hd] ~ N(0, sigma) from
    ``default_rng([seed + 7919*weight_set, 100 + h])``.  Every tensor is
    rounded to bf16.  Returns a dict with ``cfg``, ``x`` and ``groups``.
    """
    if isinstance(cfg, str):
        cfg = dict(ATTN_CONFIGS[cfg], name=cfg)
    else:
        cfg = dict(cfg)
    wseed = cfg["seed"] + 7919 * weight_set
    rng = np.random.default_rng(wseed)
    H, S, d, nq, hd = cfg["H"], cfg["S"], cfg["d"], cfg["nq"], cfg["hd"]
    x = round_to_bf16(rng.standard_normal((H, S, d), dtype=np.float32))
    groups = []
    for h in range(H):
        g = np.random.default_rng([wseed, 100 + h])
        groups.append({"w_qkv": round_to_bf16(_normal(g, ((nq + 2) * hd, d), cfg["sigma"])),
                       "w_o": round_to_bf16(_normal(g, (d, nq * hd), cfg["sigma"]))})
    return {"cfg": cfg, "x": x, "groups": groups}


# ---------------------------------------------------------------------------
# Inputs for exercising one step on its own (decoupled from upstream steps)
# ---------------------------------------------------------------------------

def make_topk_idx(T, E, k, seed, skew=0.0, dead_experts=()):
    """Random routing decisions: ``k`` distinct experts per token, int32 [T,k].

    Experts are drawn without replacement with probabilities proportional to
    ``(e+1)^-skew``; experts listed in ``dead_experts`` are never drawn.
    """
    rng = np.random.default_rng(seed)
    logp = -skew * np.log(np.arange(1, E + 1, dtype=np.float64))
    logp = np.broadcast_to(logp, (T, E)).copy()
    if dead_experts:
        logp[:, list(dead_experts)] = -np.inf
    keys = logp + rng.gumbel(size=(T, E))
    order = np.argsort(-keys, axis=1, kind="stable")
    return np.ascontiguousarray(order[:, :k].astype(np.int32))


def make_offsets(R, E, seed, empty=()):
    """Random segment boundaries ``offsets[0]=0 <= ... <= offsets[E]=R`` (int32);
    experts listed in ``empty`` get zero rows."""
    rng = np.random.default_rng(seed)
    empty = set(empty)
    live = [e for e in range(E) if e not in empty]
    if not live:
        if R:
            raise ValueError("R > 0 rows need at least one live expert")
        return np.zeros(E + 1, dtype=np.int32)
    # bounds[m] is where the m-th live expert's segment starts
    cuts = np.sort(rng.integers(0, R + 1, size=len(live) - 1))
    bounds = np.concatenate([[0], cuts, [R]])
    off = np.zeros(E + 1, dtype=np.int64)
    n_live_before = 0
    for e in range(E):
        off[e] = bounds[n_live_before]
        if e not in empty:
            n_live_before += 1
    off[E] = R
    return off.astype(np.int32)


def make_ffn_inputs(R, E, d, F, seed, sigma=0.02, dtype="bf16", empty=()):
    """``x_perm ~ N(0,1) [R,d]``, segment offsets and expert weights."""
    rng = np.random.default_rng([seed, 11])
    x_perm = rng.standard_normal((R, d), dtype=np.float32)
    w = {
        "w_gate": _normal(rng, (E, F, d), sigma),
        "w_up": _normal(rng, (E, F, d), sigma),
        "w_down": _normal(rng, (E, d, F), sigma),
    }
    if dtype == "bf16":
        x_perm = round_to_bf16(x_perm)
        w = {key: round_to_bf16(v) for key, v in w.items()}
    return {"x_perm": x_perm, "offsets": make_offsets(R, E, seed, empty), **w}


def make_combine_inputs(T, k, d, seed, dtype="bf16"):
    """``y_perm ~ N(0, 0.25) [T*k,d]``, a random bijection ``row_of``, positive
    weights ``topk_w [T,k]`` and a residual ``N(0,1) [T,d]``."""
    rng = np.random.default_rng([seed, 23])
    y = rng.standard_normal((T * k, d), dtype=np.float32) * np.float32(0.25)
    res = rng.standard_normal((T, d), dtype=np.float32)
    row_of = rng.permutation(T * k).astype(np.int32)
    w = rng.uniform(0.05, 1.0, size=(T, k)).astype(np.float32)
    if dtype == "bf16":
        y = round_to_bf16(y)
        res = round_to_bf16(res)
    return {"y_perm": y, "row_of": row_of, "topk_w": w, "residual": res}
