"""Plain CPU oracle of the per-group attention that feeds the FoE block.

TEST INFRASTRUCTURE ONLY.  Only the test suite, ``__graft_entry__.smoke()`` and
the ``cpu_baseline`` leg of ``bench.py`` may import it; the product path never
does.  It shares no code with the HIP library or its Python binding.

What it computes (Table 3, FoE column, first two rows; Section 3.1):

* "Attn. residual": every expert group ``h`` keeps its own representation
  ``x[h]`` and runs its own attention over it, with the group's share of the
  heads: ``r[h, i] = x[h, i] + Attn_h(x[h, :])[i]``;
* "Cross-group avg.": ``r_full[i] = (1/H) sum_h r[h, i]`` (the input of the
  routing and of the MoE update).

Each group owns one KV head (the paper ties the groups to the KV heads) and
``nq`` query heads that share it (grouped-query attention).  Readings where
the paper is silent:

* ``Attn_h`` is causal self-attention over the S tokens of the sequence at
  positions 0..S-1, scores ``q.k / sqrt(hd)``, softmax over the keys up to and
  including the query's own position;
* the projections are bias-free: ``[q_1..q_nq, k, v] = x W_qkv^T`` and the
  output is ``o W_o^T`` with ``o`` the heads side by side;
* rotary position embedding on q and k, pairing dimension ``i`` with
  ``i + hd/2``, angle ``(s / scale) * theta^(-2i/hd)`` at position ``s``
  (``scale`` is the RoPE scaling factor read as linear position
  interpolation);
* no normalisation inside (a pre-norm, if any, precedes the given ``x``).

All arithmetic is fp64.
"""

from __future__ import annotations

import numpy as np

__all__ = ["rope_angles", "apply_rope", "group_attention", "group_attention_rows",
           "attention_block"]


def _f64(a):
    return np.asarray(a, dtype=np.float64)


def rope_angles(S, hd, theta, scale=1.0):
    """``cos`` and ``sin`` [S, hd/2] of the rotary angles
    ``(s / scale) * theta^(-2i/hd)`` for positions ``s`` and pairs ``i``."""
    i = np.arange(hd // 2, dtype=np.float64)
    inv_freq = float(theta) ** (-2.0 * i / hd)
    pos = np.arange(S, dtype=np.float64) / float(scale)
    ang = pos[:, None] * inv_freq[None, :]
    return np.cos(ang), np.sin(ang)


def apply_rope(v, cos, sin):
    """Rotate the pairs (i, i + hd/2) of the rows of ``v`` [S, hd] by the
    angles whose cosines and sines are ``cos``, ``sin`` [S, hd/2]."""
    v = _f64(v)
    h = v.shape[-1] // 2
    a, b = v[..., :h], v[..., h:]
    return np.concatenate([a * cos - b * sin, b * cos + a * sin], axis=-1)


def group_attention(xh, w_qkv, w_o, nq, hd, theta, scale=1.0):
    """``Attn_h(x[h, :])`` for one group: [S, d] -> [S, d].

    ``w_qkv`` [(nq+2)*hd, d] holds the rows of the nq query heads, then the key
    head, then the value head; ``w_o`` [d, nq*hd].  Returns ``(out, parts)``
    with the intermediate q, k (after the rotation), v and o.
    """
    xh = _f64(xh)
    S = xh.shape[0]
    qkv = xh @ _f64(w_qkv).T
    q = qkv[:, : nq * hd].reshape(S, nq, hd)
    k = qkv[:, nq * hd:(nq + 1) * hd]
    v = qkv[:, (nq + 1) * hd:(nq + 2) * hd]
    cos, sin = rope_angles(S, hd, theta, scale)
    q = np.stack([apply_rope(q[:, j], cos, sin) for j in range(nq)], axis=1)
    k = apply_rope(k, cos, sin)
    o = np.zeros((S, nq, hd))
    scores_mask = np.tril(np.ones((S, S), dtype=bool))  # key <= query
    for j in range(nq):
        s = (q[:, j] @ k.T) / np.sqrt(hd)
        s = np.where(scores_mask, s, -np.inf)
        s = s - s.max(axis=1, keepdims=True)
        p = np.exp(s)
        p = p / p.sum(axis=1, keepdims=True)
        o[:, j] = p @ v
    o = o.reshape(S, nq * hd)
    return o @ _f64(w_o).T, {"q": q, "k": k, "v": v, "o": o}


def group_attention_rows(xh, w_qkv, w_o, nq, hd, theta, scale, rows):
    """``Attn_h(x[h, :])`` at the positions ``rows`` only (the same definition
    as ``group_attention``; keys and values are formed for every position up
    to the last requested one).  Returns [len(rows), d]."""
    xh = _f64(xh)
    rows = np.asarray(rows)
    last = int(rows.max()) + 1
    w_qkv = _f64(w_qkv)
    kv = xh[:last] @ w_qkv[nq * hd:].T
    cos, sin = rope_angles(last, hd, theta, scale)
    k = apply_rope(kv[:, :hd], cos, sin)
    v = kv[:, hd:]
    q_all = xh[rows] @ w_qkv[: nq * hd].T
    out = np.zeros((len(rows), nq * hd))
    for n, s in enumerate(rows):
        for j in range(nq):
            q = apply_rope(q_all[n:n + 1, j * hd:(j + 1) * hd], cos[s:s + 1], sin[s:s + 1])[0]
            sc = (k[: s + 1] @ q) / np.sqrt(hd)
            p = np.exp(sc - sc.max())
            out[n, j * hd:(j + 1) * hd] = (p / p.sum()) @ v[: s + 1]
    return out @ _f64(w_o).T


def attention_block(x, groups, nq, hd, theta, scale=1.0):
    """Table 3's first two FoE rows for H groups: ``x`` [H, S, d] ->
    ``r_full`` [S, d] = (1/H) sum_h (x[h] + Attn_h(x[h])).

    ``groups[h]`` holds ``w_qkv`` and ``w_o``.  Returns ``(r_full, deltas)``
    with ``deltas[h]`` = Attn_h(x[h]).
    """
    x = _f64(x)
    H = x.shape[0]
    deltas = [group_attention(x[h], g["w_qkv"], g["w_o"], nq, hd, theta, scale)[0]
              for h, g in enumerate(groups)]
    r = np.zeros_like(x[0])
    for h in range(H):
        r = r + (x[h] + deltas[h])
    return r / H, deltas
