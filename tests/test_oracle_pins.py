"""Pins of the CPU oracle against facts fixed by the paper and the mathematics.

None of these re-types the oracle's own formula: each checks it against brute
force, a closed form, a library routine, an invariant the method guarantees,
or an independent formulation of the block (dense, un-permuted).
"""

import itertools
import json
import math
import os

import numpy as np
import pytest
import scipy.special
import torch

import oracle
from paper_2605_06206_amd import synth

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def _bruteforce_topk(g, k):
    """Top-k by enumeration: the unique k-subset S such that every member beats
    every non-member under (larger score, then lower id); slot order by the
    same comparison using Python tuple ordering."""
    E = len(g)
    beats = lambda a, b: (g[a] > g[b]) or (g[a] == g[b] and a < b)  # noqa: E731
    found = []
    for S in itertools.combinations(range(E), k):
        rest = [o for o in range(E) if o not in S]
        if all(beats(s, o) for s in S for o in rest):
            found.append(S)
    assert len(found) == 1
    return sorted(found[0], key=lambda e: (-g[e], e))


@pytest.mark.parametrize("E,k", [(4, 1), (4, 2), (5, 3), (6, 6), (7, 2)])
def test_topk_bruteforce_random(E, k):
    rng = np.random.default_rng(E * 10 + k)
    g = rng.standard_normal((64, E)).astype(np.float32)
    idx, margin, _ = oracle.topk_select(g, k)
    for t in range(64):
        assert list(idx[t]) == _bruteforce_topk([float(v) for v in g[t]], k)
    if k < E:
        srt = np.sort(g, axis=1)[:, ::-1]
        assert np.allclose(margin, srt[:, k - 1] - srt[:, k])
    else:
        assert np.all(np.isinf(margin))


@pytest.mark.parametrize("E,k", [(4, 2), (6, 3), (8, 1)])
def test_topk_integer_ties_max_sum(E, k):
    """With heavy exact ties the selected set is the max-sum subset and, among
    max-sum subsets, the lexicographically smallest id set (lower ids win)."""
    rng = np.random.default_rng(99 + E)
    g = rng.integers(-2, 3, size=(200, E)).astype(np.float32)
    idx, margin, _ = oracle.topk_select(g, k)
    for t in range(200):
        best = max(itertools.combinations(range(E), k),
                   key=lambda S: (sum(g[t, list(S)]), [-e for e in S]))
        assert sorted(idx[t]) == list(best)
        # slot order: non-increasing scores, equal scores by ascending id
        vals = [g[t, e] for e in idx[t]]
        for a in range(k - 1):
            assert vals[a] > vals[a + 1] or (vals[a] == vals[a + 1] and idx[t, a] < idx[t, a + 1])
    assert np.any(margin == 0)  # ties at the boundary do occur here


def _bruteforce_gaps(g32_row, k):
    """Margin and smallest adjacent gap among the top k, by sorting the fp32
    scores of one token with Python's ``sorted`` on (score desc, id asc)."""
    vals = [float(v) for v in g32_row]
    order = sorted(range(len(vals)), key=lambda e: (-vals[e], e))
    top = [vals[e] for e in order[:k]]
    margin = vals[order[k - 1]] - vals[order[k]] if k < len(vals) else math.inf
    gaps = [top[a] - top[a + 1] for a in range(k - 1)]
    return margin, (min(gaps) if gaps else math.inf)


@pytest.mark.parametrize("E,k,kind", [(8, 1, "normal"), (8, 3, "normal"), (16, 2, "normal"),
                                      (6, 6, "normal"), (8, 4, "ties"), (5, 1, "ties"),
                                      (7, 3, "near")])
def test_margin_and_min_gap_bruteforce(E, k, kind):
    """``margin`` and ``min_gap`` (which decide where ids and slot order are
    compared) against a per-token sort; exact ties give a zero gap, k = 1 no
    gap, k = E no margin."""
    rng = np.random.default_rng([E, k, len(kind)])
    if kind == "ties":
        g = rng.integers(-2, 3, size=(300, E)).astype(np.float64)
    elif kind == "near":
        # pairs of scores a few fp32 ulps apart, and pairs equal in fp32 but
        # not in fp64
        g = rng.standard_normal((300, E))
        g[:, 1] = np.nextafter(np.float32(g[:, 0]), np.float32(np.inf)).astype(np.float64)
        g[:100, 2] = g[:100, 0] + 1e-12
    else:
        g = rng.standard_normal((300, E))
    _, margin, min_gap = oracle.topk_select(g, k)
    g32 = g.astype(np.float32)
    for t in range(g.shape[0]):
        m, mg = _bruteforce_gaps(g32[t], k)
        assert margin[t] == m and min_gap[t] == mg, t
    if kind == "ties" and k > 1:
        assert np.any(min_gap == 0.0)
    if k == 1:
        assert np.all(np.isinf(min_gap))
    if k == E:
        assert np.all(np.isinf(margin))


@pytest.mark.parametrize("name", ["decode_bf16", "prefill_zipf_bf16", "layer_share_bf16"])
def test_slot_order_check_is_not_vacuous(name):
    """On the seeded workloads nearly every token has all adjacent top-k gaps
    and its k/(k+1) margin above the 1e-5 exemption, so the slot-order and id
    comparisons cover nearly all tokens (first 2048 tokens, every cluster)."""
    inp = synth.make_block_inputs(name, T=2048)
    for cl in inp["clusters"]:
        r = oracle.route(inp["x"], cl["w_router"], cl["bias"], inp["cfg"]["k"])
        assert np.mean(r["min_gap"] >= 1e-5) > 0.99
        assert np.mean(r["margin"] >= 1e-5) > 0.99


def test_topk_decided_in_fp32():
    """Scores that differ only below fp32 resolution are a tie -> lower id."""
    g = np.array([[1.0, 1.0 + 1e-12, 0.0], [0.5, 0.5 - 1e-13, 0.7]])
    idx, margin, _ = oracle.topk_select(g, 1)
    assert idx[:, 0].tolist() == [0, 2]
    assert margin[0] == 0.0


def test_router_logits_bruteforce():
    rng = np.random.default_rng(5)
    x = rng.standard_normal((3, 5))
    w = rng.standard_normal((4, 5))
    b = rng.standard_normal(4)
    g = oracle.router_logits(x, w, b)
    for i in range(3):
        for e in range(4):
            assert math.isclose(g[i, e], math.fsum(x[i, j] * w[e, j] for j in range(5)) + b[e],
                                rel_tol=1e-13, abs_tol=1e-13)


def test_gate_weights_invariants():
    rng = np.random.default_rng(7)
    g = rng.standard_normal((500, 16)) * 2.0
    for k in (1, 2, 5, 16):
        idx, _, _ = oracle.topk_select(g, k)
        w = oracle.gate_weights(g, idx)
        # rows sum to one
        assert np.max(np.abs(w.sum(axis=1) - 1.0)) <= 1e-12
        # non-increasing along the slots (slots are in descending score order)
        assert np.all(np.diff(w, axis=1) <= 1e-15)
        # unchanged when a constant is added to every score
        w2 = oracle.gate_weights(g + 123.25, idx)
        assert np.max(np.abs(w - w2)) <= 1e-12
        # equals the global softmax over all experts renormalised over the top-k
        p = scipy.special.softmax(g, axis=1)
        psel = np.take_along_axis(p, idx, axis=1)
        assert np.max(np.abs(w - psel / psel.sum(axis=1, keepdims=True))) <= 1e-12
        if k == 1:
            assert np.all(w == 1.0)
        if k == 16:
            # k = E: the weights are the plain softmax in descending order
            assert np.max(np.abs(w - np.sort(p, axis=1)[:, ::-1])) <= 1e-12


def test_global_gate_weights_pins():
    """Global-softmax gating (not renormalised) against the library softmax of
    the concatenated score vector, and the identities that tie it to the
    renormalised weights."""
    rng = np.random.default_rng(17)
    G, T, E = 3, 200, 8
    gl = [rng.standard_normal((T, E)) * 1.5 for _ in range(G)]
    for k in (1, 2, E):
        idx = [oracle.topk_select(g, k)[0] for g in gl]
        ws = oracle.gate_weights_global(gl, idx)
        p = scipy.special.softmax(np.concatenate(gl, axis=1), axis=1)
        for h in range(G):
            ref = np.take_along_axis(p, idx[h] + h * E, axis=1)
            assert np.max(np.abs(ws[h] - ref)) <= 1e-14
            # renormalising a group's weights gives the renormalised gating
            r = ws[h] / ws[h].sum(axis=1, keepdims=True)
            assert np.max(np.abs(r - oracle.gate_weights(gl[h], idx[h]))) <= 1e-12
        total = sum(w.sum(axis=1) for w in ws)
        assert np.all(total <= 1.0 + 1e-12)
        if k == E:
            assert np.max(np.abs(total - 1.0)) <= 1e-12
        # unchanged when a constant is added to every score of every group
        for a, b in zip(ws, oracle.gate_weights_global([g - 40.0 for g in gl], idx)):
            assert np.max(np.abs(a - b)) <= 1e-12
    # one group and k = E: the global softmax is the renormalised softmax
    idx = oracle.topk_select(gl[0], E)[0]
    assert np.max(np.abs(oracle.gate_weights_global([gl[0]], [idx])[0]
                         - oracle.gate_weights(gl[0], idx))) <= 1e-12


def test_global_gating_block_special_cases():
    """The block with global gating: one cluster with k = E equals the
    renormalised block; with C clusters each delta is scaled by the cluster's
    share of the probability mass relative to the renormalised one."""
    rng = np.random.default_rng(23)
    x = rng.standard_normal((12, 8)).astype(np.float32)
    cl = _small_cluster(4, 8, 12, seed=23)
    a, _ = oracle.cluster_block(x, [cl], 4, reduce_scale=1.0, gating="global")
    b, _ = oracle.cluster_block(x, [cl], 4, reduce_scale=1.0)
    assert np.max(np.abs(a - b)) <= 1e-12
    # k = 1 in every cluster: delta_h = p_h(selected) * FFN(x) for the top expert
    cls = [_small_cluster(4, 8, 12, seed=30 + h) for h in range(2)]
    out, res = oracle.cluster_block(x, cls, 1, reduce_scale=1.0, gating="global")
    g = np.concatenate([oracle.router_logits(x, c["w_router"]) for c in cls], axis=1)
    p = scipy.special.softmax(g, axis=1)
    ref = 2 * x.astype(np.float64)
    for h, c in enumerate(cls):
        e = res[h]["idx"][:, 0]
        for i in range(x.shape[0]):
            f = oracle.swiglu_ffn(x[i:i + 1], c["w_gate"][e[i]], c["w_up"][e[i]], c["w_down"][e[i]])
            ref[i] += p[i, h * 4 + e[i]] * f[0]
    assert np.max(np.abs(out - ref)) <= 1e-12


def test_histogram_bruteforce():
    idx = synth.make_topk_idx(37, 6, 3, seed=1, skew=1.0, dead_experts=(4,))
    counts, offsets = oracle.expert_histogram(idx, 6)
    for e in range(6):
        n = sum(1 for i in range(37) for j in range(3) if idx[i, j] == e)
        assert counts[e] == n
    assert counts[4] == 0
    assert offsets[0] == 0 and offsets[-1] == 37 * 3
    assert np.all(np.diff(offsets) == counts)


def test_permutation_bruteforce():
    T, E, k = 41, 7, 3
    idx = synth.make_topk_idx(T, E, k, seed=2, skew=1.2, dead_experts=(1,))
    sorted_src, row_of = oracle.permutation(idx)
    expect = [i * k + j for e in range(E) for i in range(T) for j in range(k) if idx[i, j] == e]
    assert sorted_src.tolist() == expect
    assert sorted(sorted_src.tolist()) == list(range(T * k))  # bijection
    assert np.all(row_of[sorted_src] == np.arange(T * k))  # inverse
    counts, offsets = oracle.expert_histogram(idx, E)
    flat = idx.ravel()
    for e in range(E):
        seg = sorted_src[offsets[e]:offsets[e + 1]]
        assert np.all(flat[seg] == e)
        assert np.all(np.diff(seg // k) > 0)  # tokens ascend inside a segment
    x = np.random.default_rng(0).standard_normal((T, 5))
    xp = oracle.gather_rows(x, sorted_src, k)
    for p in range(T * k):
        assert np.array_equal(xp[p], x[sorted_src[p] // k])


def test_silu_textbook():
    z = np.linspace(-30, 30, 1001)
    assert np.max(np.abs(oracle.silu(z) - z * scipy.special.expit(z))) <= 1e-13
    assert oracle.silu(np.array([0.0]))[0] == 0.0
    assert abs(oracle.silu(np.array([-800.0]))[0]) == 0.0


def _torch_swiglu(x, wg, wu, wd):
    x, wg, wu, wd = (torch.as_tensor(np.asarray(a, np.float64)) for a in (x, wg, wu, wd))
    return (torch.nn.functional.silu(x @ wg.T) * (x @ wu.T)) @ wd.T


def _small_cluster(E, d, F, seed, sigma=0.3):
    return synth.make_cluster_weights(E, d, F, sigma, seed, 0, "f32")


def test_E1_k1_is_dense_swiglu():
    """E=1, k=1: every token goes to the only expert with weight 1, so the block
    is x + the dense SwiGLU FFN (checked against torch's silu and matmul)."""
    rng = np.random.default_rng(3)
    x = rng.standard_normal((33, 16)).astype(np.float32)
    cl = _small_cluster(1, 16, 24, seed=3)
    out, res = oracle.cluster_block(x, [cl], k=1, reduce_scale=1.0)
    ref = x + _torch_swiglu(x, cl["w_gate"][0], cl["w_up"][0], cl["w_down"][0]).numpy()
    assert np.max(np.abs(out - ref)) <= 1e-12
    assert np.all(res[0]["w"] == 1.0)


def test_k_equals_E_dense_softmax_mixture():
    """k=E: the block is the dense softmax-weighted mixture of all experts,
    computed here without any top-k, permutation or combine."""
    rng = np.random.default_rng(4)
    T, d, E, F = 29, 12, 5, 20
    x = rng.standard_normal((T, d)).astype(np.float32)
    cl = _small_cluster(E, d, F, seed=4)
    cl["bias"] = rng.standard_normal(E).astype(np.float32)
    out, _ = oracle.cluster_block(x, [cl], k=E, reduce_scale=1.0)
    xt = torch.as_tensor(x, dtype=torch.float64)
    g = xt @ torch.as_tensor(cl["w_router"], dtype=torch.float64).T + torch.as_tensor(cl["bias"], dtype=torch.float64)
    p = torch.softmax(g, dim=1)
    ref = xt.clone()
    for e in range(E):
        ref += p[:, e:e + 1] * _torch_swiglu(x, cl["w_gate"][e], cl["w_up"][e], cl["w_down"][e])
    assert np.max(np.abs(out - ref.numpy())) <= 1e-12


def test_pipeline_matches_dense_masked_formulation():
    """General k < E: the permuted pipeline equals a dense formulation that runs
    every expert on every token and masks with a brute-force top-k."""
    rng = np.random.default_rng(6)
    T, d, E, F, k = 23, 10, 6, 14, 2
    x = rng.standard_normal((T, d)).astype(np.float32)
    cl = _small_cluster(E, d, F, seed=6)
    r = oracle.cluster_delta(x, cl, k)
    g = x.astype(np.float64) @ cl["w_router"].astype(np.float64).T
    ys = [_torch_swiglu(x, cl["w_gate"][e], cl["w_up"][e], cl["w_down"][e]).numpy() for e in range(E)]
    for t in range(T):
        sel = _bruteforce_topk([float(v) for v in g[t].astype(np.float32)], k)
        assert list(r["idx"][t]) == sel
        z = np.exp(g[t, sel] - g[t, sel].max())
        w = z / z.sum()
        ref = sum(w[j] * ys[sel[j]][t] for j in range(k))
        assert np.max(np.abs(r["delta"][t] - ref)) <= 1e-12
    # the per-token (un-permuted) formula of the oracle agrees as well
    delta_tok, _ = oracle.moe_update_tokens(x, cl, k)
    assert np.max(np.abs(delta_tok - r["delta"])) <= 1e-12


def test_down_projection_scaling_is_linear():
    rng = np.random.default_rng(8)
    x = rng.standard_normal((17, 8)).astype(np.float32)
    cl = _small_cluster(4, 8, 12, seed=8)
    d1 = oracle.cluster_delta(x, cl, 2)["delta"]
    cl2 = dict(cl, w_down=cl["w_down"].astype(np.float64) * 2.5)
    d2 = oracle.cluster_delta(x, cl2, 2)["delta"]
    assert np.max(np.abs(d2 - 2.5 * d1)) <= 1e-12


def test_token_permutation_equivariance():
    rng = np.random.default_rng(9)
    x = rng.standard_normal((19, 8)).astype(np.float32)
    cl = _small_cluster(5, 8, 12, seed=9)
    perm = rng.permutation(19)
    out, _ = oracle.cluster_block(x, [cl], 2)
    out_p, _ = oracle.cluster_block(x[perm], [cl], 2)
    assert np.max(np.abs(out_p - out[perm])) <= 1e-12


def test_combine_special_cases():
    rng = np.random.default_rng(10)
    T, d = 9, 6
    y = rng.standard_normal((T, d))
    res = rng.standard_normal((T, d))
    # k = 1, weight 1, identity permutation: out = res + y
    out = oracle.combine(y, np.arange(T), np.ones((T, 1)), residual=res)
    assert np.max(np.abs(out - (res + y))) == 0.0
    # k = 2 with a swap permutation: brute force sum
    k = 2
    y2 = rng.standard_normal((T * k, d))
    row_of = rng.permutation(T * k)
    w = rng.uniform(size=(T, k))
    delta = oracle.combine(y2, row_of, w)
    for i in range(T):
        ref = w[i, 0] * y2[row_of[i * k]] + w[i, 1] * y2[row_of[i * k + 1]]
        assert np.max(np.abs(delta[i] - ref)) <= 1e-14


def test_reduce_identical_clusters_is_one_cluster():
    """C identical clusters averaged (scale 1/C) give one cluster's x'[h]."""
    rng = np.random.default_rng(11)
    x = rng.standard_normal((15, 8)).astype(np.float32)
    cl = _small_cluster(4, 8, 12, seed=11)
    one, _ = oracle.cluster_block(x, [cl], 2, reduce_scale=1.0)
    four, _ = oracle.cluster_block(x, [cl] * 4, 2)
    assert np.max(np.abs(four - one)) <= 1e-12
    # literal sum (scale 1) of C partials is C times the average
    s4, _ = oracle.cluster_block(x, [cl] * 4, 2, reduce_scale=1.0)
    assert np.max(np.abs(s4 - 4 * one)) <= 1e-11
    # average of different clusters = x + mean of their deltas
    cls = [_small_cluster(4, 8, 12, seed=20 + h) for h in range(3)]
    avg, res = oracle.cluster_block(x, cls, 2)
    ref = x + sum(r["delta"] for r in res) / 3.0
    assert np.max(np.abs(avg - ref)) <= 1e-12
    # plain scaled sum of partials without a residual
    P = rng.standard_normal((3, 4, 5))
    assert np.max(np.abs(oracle.reduce_partials(P, 0.5) - 0.5 * (P[0] + P[1] + P[2]))) <= 1e-15


def test_every_cluster_processes_T_times_k_pairs():
    """Section 4.5: every group receives the same number of tokens; each
    cluster processes exactly T*k (token, slot) pairs whatever the skew."""
    inp = synth.make_block_inputs("tiny_fp32")
    cl = dict(inp["clusters"][0], bias=synth.zipf_bias(4, 3.0))
    r = oracle.cluster_delta(inp["x"], cl, 2)
    assert r["counts"].sum() == 64 * 2
    assert r["offsets"][-1] == 64 * 2
    assert r["counts"].max() > r["counts"].min()  # skewed, still T*k in total


def _eval_expr(s):
    env = {"sigmoid": lambda z: 1.0 / (1.0 + math.exp(-z)), "exp": math.exp}
    return float(eval(s, {"__builtins__": {}}, env))  # noqa: S307 (fixture of our own)


def test_golden_closed_form_cases():
    with open(os.path.join(GOLDEN, "closed_form_block.json")) as f:
        cases = json.load(f)["cases"]
    for case in cases:
        x = np.array(case["x"], dtype=np.float64)
        cls = []
        for c in case["clusters"]:
            cls.append({key: (None if c[key] is None else np.array(c[key], dtype=np.float64))
                        for key in ("w_router", "bias", "w_gate", "w_up", "w_down")})
        out, res = oracle.cluster_block(x, cls, case["k"], case["reduce_scale"])
        for h, r in enumerate(res):
            assert r["idx"].tolist() == case["expect_idx"][h], case["name"]
            ew = np.array([[_eval_expr(s) for s in row] for row in case["expect_w"][h]])
            assert np.max(np.abs(r["w"] - ew)) <= 1e-14, case["name"]
        expect = np.array([[_eval_expr(s) for s in row] for row in case["expect_out"]])
        assert np.max(np.abs(out - expect)) <= 1e-13, case["name"]


def test_config_inputs_are_seeded_and_bf16():
    a = synth.make_block_inputs("decode_bf16")
    b = synth.make_block_inputs("decode_bf16")
    assert np.array_equal(a["x"], b["x"])
    assert np.array_equal(a["clusters"][0]["w_down"], b["clusters"][0]["w_down"])
    # bf16 configs hold bf16-representable values (low 16 bits zero)
    assert np.all((a["x"].view(np.uint32) & 0xFFFF) == 0)
    c = synth.make_block_inputs("decode_bf16", weight_set=1)
    assert not np.array_equal(a["clusters"][0]["w_gate"], c["clusters"][0]["w_gate"])
