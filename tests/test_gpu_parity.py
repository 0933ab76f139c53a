"""GPU parity: every entry point of libfoe.so against the CPU oracle on the same
seeded inputs.

Bars: integer outputs (expert ids, counts, offsets, permutation) bit-exact;
floating point per tensor max|err| / max|ref| <= 2e-2 (bf16) or 1e-4 (fp32).
Routing: a token whose fp32 k-th/(k+1)-th score margin (oracle) is below 1e-5
is exempt from id bit-exactness (both choices are correct); it must still pick
a valid top-k.  Slot order is compared where every adjacent gap among the top
k is >= 1e-5.  Whole-block outputs are compared on every row: the oracle
adopts the device's ids for exempt tokens, and both the output and its update
part (output minus the residual part) are bounded (tests/block_check.py).
"""

import functools
import sys

import numpy as np
import pytest
import torch

import block_check as bc
import oracle
from paper_2605_06206_amd import foe, synth

pytestmark = pytest.mark.gpu

TOL = bc.TOL
EXEMPT = bc.EXEMPT
DEV = "cuda:0"


@pytest.fixture(autouse=True, scope="module")
def _need_gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    foe.lib()  # fail loudly if the HIP library is missing


def say(*a):
    print("[gpu-case]", *a, file=sys.stderr, flush=True)


def to_dev(a, dtype):
    a = np.ascontiguousarray(a)
    if a.dtype in (np.int32, np.int64):
        return torch.from_numpy(a.astype(np.int32)).to(DEV)
    if dtype == "bf16":
        return torch.from_numpy(synth.bf16_bits(a)).to(DEV).view(torch.bfloat16)
    return torch.from_numpy(a.astype(np.float32)).to(DEV)


def host(t):
    if t.dtype == torch.bfloat16:
        return t.float().cpu().numpy().astype(np.float64)
    return t.cpu().numpy()


rel_err = bc.rel_err


@functools.lru_cache(maxsize=2)
def cfg_inputs(name):
    return synth.make_block_inputs(name)


def stacked(inp):
    dt = inp["cfg"]["dtype"]
    cls = inp["clusters"]
    w = {key: to_dev(np.stack([c[key] for c in cls]), dt)
         for key in ("w_router", "w_gate", "w_up", "w_down")}
    w["bias"] = (to_dev(np.stack([c["bias"] for c in cls]), "f32")
                 if cls[0]["bias"] is not None else None)
    return w


def check_route(gidx, gw, ref, tol, g64=None, sums_to_one=True):
    """Compare GPU routing with the oracle's; returns the exempt mask."""
    gidx = np.asarray(gidx).astype(np.int64)
    gw = np.asarray(gw, np.float64)
    exempt = ref["margin"] < EXEMPT
    ne = ~exempt
    assert np.array_equal(np.sort(gidx[ne], 1), np.sort(ref["idx"][ne], 1)), "top-k sets differ"
    ordered = ne & (ref["min_gap"] >= EXEMPT)
    assert np.array_equal(gidx[ordered], ref["idx"][ordered]), "slot order differs"
    # weights, aligned by expert id
    o_g = np.argsort(gidx[ne], 1)
    o_r = np.argsort(ref["idx"][ne], 1)
    wg = np.take_along_axis(gw[ne], o_g, 1)
    wr = np.take_along_axis(ref["w"][ne], o_r, 1)
    assert rel_err(wg, wr) <= tol, rel_err(wg, wr)
    if sums_to_one:  # renormalised gating: rows of weights sum to one
        assert np.max(np.abs(gw.sum(1) - 1.0)) <= 1e-5
    # exempt tokens still pick a valid top-k of the oracle scores
    g32 = ref["logits"].astype(np.float32).astype(np.float64)
    k = gidx.shape[1]
    for t in np.nonzero(exempt)[0]:
        kth = np.sort(g32[t])[::-1][k - 1]
        assert len(set(gidx[t])) == k
        assert np.all(g32[t, gidx[t]] >= kth - EXEMPT)
    return exempt


# ---------------------------------------------------------------------------
# route
# ---------------------------------------------------------------------------

@pytest.mark.parametrize("name", synth.CONFIG_ORDER)
def test_route_parity_configs(name):
    inp = cfg_inputs(name)
    cfg = inp["cfg"]
    dt = cfg["dtype"]
    x = to_dev(inp["x"], dt)
    for h, cl in enumerate(inp["clusters"][:2]):
        say("route", name, "cluster", h, "T", cfg["T"], "d", cfg["d"], "E", cfg["E"], "k", cfg["k"])
        bias = to_dev(cl["bias"], "f32") if cl["bias"] is not None else None
        gidx, gw = foe.route(x, to_dev(cl["w_router"], dt), bias, cfg["k"])
        torch.cuda.synchronize()
        ref = oracle.route(inp["x"], cl["w_router"], cl["bias"], cfg["k"])
        exempt = check_route(host(gidx), host(gw), ref, TOL[dt])
        say("route", name, "cluster", h, "exempt tokens", int(exempt.sum()))


@pytest.mark.parametrize("T,d,E,k,dt", [
    (1, 64, 4, 1, "bf16"), (50, 136, 5, 3, "bf16"), (333, 64, 33, 5, "bf16"),
    (77, 256, 256, 8, "bf16"), (40, 32, 16, 16, "f32"), (129, 8, 2, 2, "f32"),
    (300, 512, 64, 64, "bf16"),
    # many-token streaming path: ragged token tails, K tail, partial expert tile
    (8195, 136, 20, 3, "bf16"), (16389, 520, 32, 4, "bf16"), (9000, 264, 9, 2, "bf16"),
])
def test_route_parity_shapes(T, d, E, k, dt):
    """Ragged token tails, K tails (d not a multiple of 32), E not a multiple
    of 16, E = 256, k = E."""
    say("route shapes", T, d, E, k, dt)
    rng = np.random.default_rng(T * 7 + E)
    xs = rng.standard_normal((T, d)).astype(np.float32)
    wr = (rng.standard_normal((E, d)) * 0.05).astype(np.float32)
    bias = (rng.standard_normal(E) * 0.1).astype(np.float32)
    if dt == "bf16":
        xs, wr = synth.round_to_bf16(xs), synth.round_to_bf16(wr)
    gidx, gw = foe.route(to_dev(xs, dt), to_dev(wr, dt), to_dev(bias, "f32"), k)
    ref = oracle.route(xs, wr, bias, k)
    check_route(host(gidx), host(gw), ref, TOL[dt])


@pytest.mark.parametrize("G,T,d,E,k,dt", [
    (1, 300, 256, 16, 2, "bf16"),   # one group
    (1, 8200, 136, 20, 3, "bf16"),  # many-token streaming path
    (1, 40, 32, 16, 16, "f32"),     # k = E: the softmax itself
    (4, 200, 128, 12, 2, "bf16"),   # four groups in one score matrix
    (3, 64, 64, 10, 3, "f32"),      # groups straddle the 16-column score tiles
])
def test_route_global_gating(G, T, d, E, k, dt):
    """Global softmax over all G*E scores, not renormalised (foe_route_ex)."""
    say("route global gating", G, T, d, E, k, dt)
    rng = np.random.default_rng(T + 31 * G + E)
    xs = rng.standard_normal((T, d)).astype(np.float32)
    wr = (rng.standard_normal((G, E, d)) * 0.05).astype(np.float32)
    bias = (rng.standard_normal((G, E)) * 0.1).astype(np.float32)
    if dt == "bf16":
        xs, wr = synth.round_to_bf16(xs), synth.round_to_bf16(wr)
    w_dev = to_dev(wr if G > 1 else wr[0], dt)
    b_dev = to_dev(bias if G > 1 else bias[0], "f32")
    gidx, gw = foe.route(to_dev(xs, dt), w_dev, b_dev, k, gating="global")
    gidx, gw = host(gidx).reshape(G, T, k), host(gw).reshape(G, T, k)
    refs = [oracle.route(xs, wr[h], bias[h], k) for h in range(G)]
    gws = oracle.gate_weights_global([r["logits"] for r in refs], [r["idx"] for r in refs])
    for h in range(G):
        check_route(gidx[h], gw[h], dict(refs[h], w=gws[h]), TOL[dt], sums_to_one=False)
    total = gw.astype(np.float64).sum(axis=(0, 2))
    assert np.all(total <= 1.0 + 1e-5)
    if k == E and G == 1:
        assert np.max(np.abs(total - 1.0)) <= 1e-5


@pytest.mark.parametrize("G,T,d,E,k,gating", [
    (8, 4096, 2048, 8, 2, "renorm"),    # the layer-share shape: 64 score columns, one pass
    (3, 4100, 136, 20, 3, "renorm"),    # ragged tokens and K, groups straddle score tiles
    (2, 9000, 264, 16, 4, "global"),    # two waves per workgroup
    (4, 16400, 128, 16, 2, "renorm"),   # four waves per workgroup, ragged last block
    (5, 4096, 64, 12, 12, "renorm"),    # k = E inside every group
])
def test_route_grouped_streaming(G, T, d, E, k, gating):
    """Several clusters scored in one pass over x by the streaming kernel
    (G*E <= 64 score columns, T >= 4096), each taking its top-k over its own
    block of E columns."""
    say("route grouped streaming", G, T, d, E, k, gating)
    rng = np.random.default_rng([G, T, E])
    xs = synth.round_to_bf16(rng.standard_normal((T, d)).astype(np.float32))
    wr = synth.round_to_bf16((rng.standard_normal((G, E, d)) * 0.05).astype(np.float32))
    bias = (rng.standard_normal((G, E)) * 0.1).astype(np.float32)
    gidx, gw = foe.route(to_dev(xs, "bf16"), to_dev(wr, "bf16"), to_dev(bias, "f32"), k,
                         gating=gating)
    gidx, gw = host(gidx).reshape(G, T, k), host(gw).reshape(G, T, k)
    refs = [oracle.route(xs, wr[h], bias[h], k) for h in range(G)]
    if gating == "global":
        ws = oracle.gate_weights_global([r["logits"] for r in refs], [r["idx"] for r in refs])
        refs = [dict(r, w=w) for r, w in zip(refs, ws)]
    for h in range(G):
        check_route(gidx[h], gw[h], refs[h], TOL["bf16"], sums_to_one=gating == "renorm")


@pytest.mark.parametrize("k", [1, 3])
def test_route_exact_ties_pick_lower_id(k):
    """Duplicate router rows give bit-identical scores on both sides: the
    lower expert id must win, bit-exact, even at the k/(k+1) boundary."""
    say("route ties k", k)
    rng = np.random.default_rng(31)
    T, d, E = 200, 128, 16
    xs = synth.round_to_bf16(rng.standard_normal((T, d)).astype(np.float32))
    wr = rng.standard_normal((E, d)).astype(np.float32) * 0.02
    wr[9] = wr[3] = wr[3] * 8.0  # a strong pair of twins: usually on top
    wr[12] = wr[5]
    wr = synth.round_to_bf16(wr)
    gidx, _ = foe.route(to_dev(xs, "bf16"), to_dev(wr, "bf16"), None, k)
    gidx = host(gidx)
    ref = oracle.route(xs, wr, None, k)
    assert np.array_equal(gidx, ref["idx"])
    has3 = np.any(gidx == 3, axis=1)
    has9 = np.any(gidx == 9, axis=1)
    assert np.all(has3 | ~has9)  # 9 is never chosen without its lower twin 3
    if k == 1:
        assert np.sum(gidx[:, 0] == 3) > 0 and not np.any(gidx[:, 0] == 9)


# ---------------------------------------------------------------------------
# permute
# ---------------------------------------------------------------------------

@pytest.mark.parametrize("T,d,E,k,skew,dead,dt", [
    (37, 64, 7, 3, 1.2, (1,), "bf16"),
    (3000, 128, 16, 2, 1.2, (), "bf16"),
    (16384, 4096, 32, 4, 0.0, (), "bf16"),
    (8192, 2048, 16, 2, 1.2, (), "bf16"),
    (1025, 32, 256, 8, 0.5, (0, 255), "f32"),
    (5, 16, 4, 4, 0.0, (), "f32"),
    (8800, 16, 256, 8, 0.8, (3,), "f32"),   # block counts past the in-rank sum
    (9000, 16, 1, 1, 0.0, (), "f32"),       # E = 1 on the multi-block path
])
def test_permute_parity(T, d, E, k, skew, dead, dt):
    say("permute", T, d, E, k, skew, dead, dt)
    idx = synth.make_topk_idx(T, E, k, seed=T + E, skew=skew, dead_experts=dead)
    rng = np.random.default_rng(T)
    xs = rng.standard_normal((T, d)).astype(np.float32)
    if dt == "bf16":
        xs = synth.round_to_bf16(xs)
    xd = to_dev(xs, dt)
    got = foe.permute(to_dev(idx, None), xd, E)
    torch.cuda.synchronize()
    counts, offsets = oracle.expert_histogram(idx, E)
    sorted_src, row_of = oracle.permutation(idx)
    assert np.array_equal(host(got["counts"]), counts)
    assert np.array_equal(host(got["offsets"]), offsets)
    assert np.array_equal(host(got["sorted_src"]), sorted_src)
    assert np.array_equal(host(got["row_of"]), row_of)
    # x_perm is a pure copy: bit-exact, checked on the device
    ref_rows = torch.from_numpy(sorted_src // k).to(DEV)
    assert torch.equal(got["x_perm"], xd[ref_rows])


@pytest.mark.parametrize("T", [300, 6000])
def test_permute_drops_invalid_ids(T):
    say("permute invalid ids", T)
    d, E, k = 64, 8, 2
    idx = synth.make_topk_idx(T, E, k, seed=5)
    idx[10, 1] = -1
    idx[200, 0] = E
    xs = np.random.default_rng(1).standard_normal((T, d)).astype(np.float32)
    got = foe.permute(to_dev(idx, None), to_dev(xs, "f32"), E)
    valid = (idx >= 0) & (idx < E)
    counts = np.bincount(idx[valid], minlength=E)
    assert np.array_equal(host(got["counts"]), counts)
    off = host(got["offsets"])
    assert off[-1] == T * k - 2
    row_of = host(got["row_of"])
    assert row_of[10 * k + 1] == -1 and row_of[200 * k] == -1
    flat = idx.ravel()
    keep = np.nonzero(valid.ravel())[0]
    order = keep[np.argsort(flat[keep], kind="stable")]
    assert np.array_equal(host(got["sorted_src"])[: T * k - 2], order)


def test_permute_empty_batch():
    say("permute T=0")
    got = foe.permute(torch.empty((0, 2), dtype=torch.int32, device=DEV),
                      torch.empty((0, 64), dtype=torch.bfloat16, device=DEV), 6)
    assert np.all(host(got["offsets"]) == 0) and np.all(host(got["counts"]) == 0)


# ---------------------------------------------------------------------------
# expert FFN
# ---------------------------------------------------------------------------

@pytest.mark.parametrize("R,E,d,F,empty,dt", [
    (300, 5, 128, 192, (2,), "bf16"),      # few rows per expert (weight-streaming tiles)
    (3000, 5, 256, 384, (0,), "bf16"),     # large-tile path, ragged row tails
    (777, 3, 136, 72, (), "bf16"),         # K and N tails (not multiples of the tiles)
    (256, 16, 2048, 1024, (), "bf16"),     # decode-shaped
    (4100, 7, 512, 520, (6,), "bf16"),
    (128, 4, 128, 256, (), "f32"),
    (90, 3, 40, 24, (1,), "f32"),
])
def test_expert_ffn_parity(R, E, d, F, empty, dt):
    say("expert_ffn", R, E, d, F, empty, dt)
    inp = synth.make_ffn_inputs(R, E, d, F, seed=R + d, dtype=dt, empty=empty)
    y = foe.expert_ffn(to_dev(inp["x_perm"], dt), to_dev(inp["offsets"], None),
                       to_dev(inp["w_gate"], dt), to_dev(inp["w_up"], dt),
                       to_dev(inp["w_down"], dt))
    torch.cuda.synchronize()
    ref = oracle.expert_ffn(inp["x_perm"], inp["offsets"], inp["w_gate"], inp["w_up"], inp["w_down"])
    err = rel_err(host(y), ref)
    say("expert_ffn rel err", err)
    assert err <= TOL[dt]


def test_expert_ffn_prefill_size():
    """Full prefill size (rows 16384, d 2048, F 1024, 16 experts, skewed, one
    empty expert), every row against the oracle."""
    R, E, d, F = 16384, 16, 2048, 1024
    say("expert_ffn prefill size", R, E, d, F)
    inp = synth.make_ffn_inputs(R, E, d, F, seed=3, empty=(4,))
    y = host(foe.expert_ffn(to_dev(inp["x_perm"], "bf16"), to_dev(inp["offsets"], None),
                            to_dev(inp["w_gate"], "bf16"), to_dev(inp["w_up"], "bf16"),
                            to_dev(inp["w_down"], "bf16")))
    say("expert_ffn prefill size: device done")
    ref = oracle.expert_ffn(inp["x_perm"], inp["offsets"], inp["w_gate"], inp["w_up"],
                            inp["w_down"])
    err = rel_err(y, ref)
    # per expert as well: a small expert's rows are a small part of max|ref|
    off = inp["offsets"]
    per = [rel_err(y[off[e]:off[e + 1]], ref[off[e]:off[e + 1]])
           for e in range(E) if off[e + 1] > off[e]]
    say("expert_ffn prefill size rel err", err, "worst expert", max(per))
    assert err <= 2e-2 and max(per) <= 2e-2


# ---------------------------------------------------------------------------
# combine / reduce
# ---------------------------------------------------------------------------

@pytest.mark.parametrize("T,k,d,dt", [(37, 3, 64, "bf16"), (4096, 2, 2048, "bf16"),
                                      (1000, 4, 136, "f32"), (64, 2, 128, "f32")])
def test_combine_parity(T, k, d, dt):
    say("combine", T, k, d, dt)
    inp = synth.make_combine_inputs(T, k, d, seed=T, dtype=dt)
    y, row_of, w = to_dev(inp["y_perm"], dt), to_dev(inp["row_of"], None), to_dev(inp["topk_w"], "f32")
    delta = foe.combine(y, row_of, w)
    out = foe.combine(y, row_of, w, residual=to_dev(inp["residual"], dt))
    ref_d = oracle.combine(inp["y_perm"], inp["row_of"], inp["topk_w"])
    ref_o = oracle.combine(inp["y_perm"], inp["row_of"], inp["topk_w"], inp["residual"])
    assert rel_err(host(delta), ref_d) <= TOL[dt]
    assert rel_err(host(out), ref_o) <= TOL[dt]


@pytest.mark.parametrize("C,T,d,scale,with_res,dt", [
    (8, 4096, 2048, 0.125, True, "bf16"), (3, 100, 64, 1.0, False, "bf16"),
    (1, 33, 8, 0.5, True, "f32"), (5, 64, 128, 0.2, False, "f32")])
def test_reduce_parity(C, T, d, scale, with_res, dt):
    say("reduce", C, T, d, scale, with_res, dt)
    rng = np.random.default_rng(C * T)
    P = (rng.standard_normal((C, T, d)) * 0.3).astype(np.float32)
    res = rng.standard_normal((T, d)).astype(np.float32)
    if dt == "bf16":
        P, res = synth.round_to_bf16(P), synth.round_to_bf16(res)
    out = foe.reduce(to_dev(P, dt), scale, residual=to_dev(res, dt) if with_res else None)
    ref = oracle.reduce_partials(P, scale, res if with_res else None)
    assert rel_err(host(out), ref) <= TOL[dt]


# ---------------------------------------------------------------------------
# whole block
# ---------------------------------------------------------------------------

def _block_gpu(inp, reduce_scale=None, gating="renorm"):
    cfg = inp["cfg"]
    w = stacked(inp)
    out = foe.cluster_block(to_dev(inp["x"], cfg["dtype"]), w["w_router"], w["bias"], w["w_gate"],
                            w["w_up"], w["w_down"], cfg["k"], reduce_scale=reduce_scale,
                            gating=gating)
    torch.cuda.synchronize()
    return host(out)


def _device_idx(inp):
    """The device's expert ids [C,T,k] for the block's inputs (the routing
    kernels the block runs, called through foe_route / foe_route_ex)."""
    cfg = inp["cfg"]
    C, E, k = cfg["C"], cfg["E"], cfg["k"]
    w = stacked(inp)
    x = to_dev(inp["x"], cfg["dtype"])
    bias = w["bias"]
    if C > 1 and C * E <= 256:
        idx, _ = foe.route(x, w["w_router"], bias, k)
        return host(idx).reshape(C, cfg["T"], k)
    out = []
    for h in range(C):
        idx, _ = foe.route(x, w["w_router"][h], None if bias is None else bias[h], k)
        out.append(host(idx))
    return np.stack(out)


def _check_block(inp, got, reduce_scale=None, gating="renorm", label=""):
    """Every row of the block output against the oracle (exempt tokens routed
    as the device routed them): the output and its update part."""
    cfg = inp["cfg"]
    C, k, dt = cfg["C"], cfg["k"], cfg["dtype"]
    routes = bc.oracle_routes(inp["x"], inp["clusters"], k)
    dev_idx = _device_idx(inp) if bc.exempt_mask(routes).any() else None
    ref, _, adopted = bc.oracle_block(inp["x"], inp["clusters"], k, reduce_scale, gating,
                                      routes=routes, device_idx=dev_idx)
    assert np.all(np.isfinite(got))
    e_out, e_upd = bc.block_errors(got, ref, inp["x"], C, reduce_scale, dt)
    say("block", label, f"rel err out {e_out:.3e} update part {e_upd:.3e} adopted ids", adopted)
    assert e_out <= TOL[dt] and e_upd <= TOL[dt]


@pytest.mark.parametrize("name", ["tiny_fp32", "decode_bf16"])
def test_block_parity_full(name):
    inp = cfg_inputs(name)
    say("block full", name)
    _check_block(inp, _block_gpu(inp), label=name)


@pytest.mark.parametrize("name", ["prefill_zipf_bf16", "large_bf16", "layer_share_bf16"])
def test_block_parity_large_configs(name):
    """The three large workloads at full size, every token row."""
    inp = cfg_inputs(name)
    cfg = inp["cfg"]
    say("block full size", name, "T", cfg["T"], "C", cfg["C"])
    got = _block_gpu(inp)
    say("block full size", name, "device done")
    _check_block(inp, got, label=name)


@pytest.mark.parametrize("T,d,E,k,F,C,scale,dt,bias", [
    (1000, 256, 8, 2, 384, 1, None, "bf16", None),   # large tiles, ragged tails
    (100, 256, 16, 2, 128, 1, None, "bf16", None),   # small-row tiles
    (50, 64, 4, 4, 64, 1, None, "bf16", None),       # k = E (dense mixture)
    (33, 32, 1, 1, 48, 1, None, "f32", None),        # E = 1, k = 1
    (1, 64, 8, 2, 64, 3, 1.0, "bf16", None),         # one token, literal sum of 3
    (257, 128, 8, 2, 128, 2, None, "bf16", "zipf4"),  # extreme skew: empty experts
    (130, 64, 4, 2, 64, 2, 0.5, "f32", None),
    (200, 64, 100, 3, 64, 3, None, "bf16", None),    # 300 experts in one grouped FFN
    (600, 128, 64, 2, 128, 4, None, "bf16", None),    # 256 experts, large-tile path
    (5000, 64, 8, 2, 64, 2, None, "bf16", None),      # two clusters, multi-block dispatch
    (40, 136, 6, 2, 200, 2, None, "bf16", None),      # decode form, d and F off the tile widths
    (70, 64, 10, 3, 64, 3, None, "bf16", "zipf1.2"),  # cluster blocks straddle 16-column tiles
    (4500, 64, 10, 3, 128, 2, None, "bf16", None),    # routing counts in 48-pair blocks
    (8300, 72, 16, 2, 64, 1, None, "bf16", "zipf1.2"),  # two-wave routing blocks, ragged
    (40000, 64, 4, 2, 64, 1, None, "bf16", None),     # 79 tile groups: per-XCD work lists
    (30000, 128, 6, 2, 128, 2, None, "bf16", "zipf1.2"),  # per-XCD lists, two clusters, skew
])
def test_block_parity_shapes(T, d, E, k, F, C, scale, dt, bias):
    say("block shapes", T, d, E, k, F, C, scale, dt, bias)
    cfg = dict(dtype=dt, C=C, T=T, d=d, E=E, k=k, F=F, sigma=0.05, seed=T + d, bias=bias)
    inp = synth.make_block_inputs(cfg)
    _check_block(inp, _block_gpu(inp, scale), scale)


def _random_block_case(i):
    """Shape i of a fixed pseudo-random set: dtype, clusters, tokens, widths,
    experts, top-k, router bias and reduction scale all drawn."""
    rng = np.random.default_rng([77, i])
    dt = "f32" if rng.random() < 0.3 else "bf16"
    C = int(rng.integers(1, 5))
    T = int(rng.integers(1, 700 if dt == "bf16" else 200))
    d = int(rng.integers(1, 49 if dt == "bf16" else 17)) * 8
    E = int(rng.integers(1, 33))
    k = int(rng.integers(1, min(E, 4) + 1))
    F = int(rng.integers(1, 41 if dt == "bf16" else 17)) * 8
    bias = "zipf1.2" if rng.random() < 0.5 else None
    scale = None if rng.random() < 0.5 else float(rng.choice([0.5, 1.0]))
    return dict(dtype=dt, C=C, T=T, d=d, E=E, k=k, F=F, sigma=0.05, seed=2000 + i,
                bias=bias), scale


@pytest.mark.parametrize("i", range(12))
def test_block_parity_random_shapes(i):
    cfg, scale = _random_block_case(i)
    say("block random shape", i, cfg, scale)
    inp = synth.make_block_inputs(cfg)
    _check_block(inp, _block_gpu(inp, scale), scale)


@pytest.mark.parametrize("T,d,E,k,F,C", [
    (128, 256, 16, 2, 128, 1),  # decode form, one cluster
    (96, 128, 8, 2, 64, 3),     # three clusters, one score matrix
    (600, 128, 8, 2, 128, 2),   # many pairs per expert: dispatch pass and grouped GEMM
])
def test_block_global_gating(T, d, E, k, F, C):
    say("block global gating", T, d, E, k, F, C)
    cfg = dict(dtype="bf16", C=C, T=T, d=d, E=E, k=k, F=F, sigma=0.05, seed=T + d + C, bias=None)
    inp = synth.make_block_inputs(cfg)
    _check_block(inp, _block_gpu(inp, gating="global"), gating="global")


def test_block_is_deterministic():
    inp = cfg_inputs("decode_bf16")
    say("block determinism")
    a = _block_gpu(inp)
    b = _block_gpu(inp)
    assert np.array_equal(a, b)


def test_block_reused_workspace_new_inputs():
    """Decode-sized block, two clusters, one workspace: first filled with 0xFF
    bytes (garbage counters and rows), then used for input set A and then for
    a different set B.  B must match the oracle, and match B run on a fresh
    workspace bit for bit (no value of the earlier call leaks in)."""
    say("block reused workspace")
    outs = {}
    base = dict(dtype="bf16", C=2, T=96, d=256, E=8, k=2, F=128, sigma=0.05, bias=None)
    need = foe.workspace_bytes("cluster_block", foe.BF16, 2, 96, 256, 8, 2, 128)
    ws = torch.full((need,), 255, dtype=torch.uint8, device=DEV)
    for tag, seed in (("A", 11), ("B", 12)):
        inp = synth.make_block_inputs(dict(base, seed=seed))
        w = stacked(inp)
        out = foe.cluster_block(to_dev(inp["x"], "bf16"), w["w_router"], w["bias"], w["w_gate"],
                                w["w_up"], w["w_down"], 2, ws=ws)
        torch.cuda.synchronize()
        outs[tag] = (host(out), inp)
    got, inp = outs["B"]
    _check_block(inp, got)
    assert np.array_equal(got, _block_gpu(inp))


def test_pipeline_properties_at_prefill_size():
    """Properties that hold at any size, on the real prefill configuration:
    every permuted row holds its expert's token, segments ascend, the counts
    sum to T*k, and combine(y = x_perm) with unit weights gives k * x."""
    inp = cfg_inputs("prefill_zipf_bf16")
    cfg = inp["cfg"]
    T, k, E = cfg["T"], cfg["k"], cfg["E"]
    say("properties prefill")
    cl = inp["clusters"][0]
    x = to_dev(inp["x"], "bf16")
    idx, w = foe.route(x, to_dev(cl["w_router"], "bf16"), to_dev(cl["bias"], "f32"), k)
    p = foe.permute(idx, x, E)
    counts = host(p["counts"])
    assert counts.sum() == T * k and counts.max() > 4 * np.median(counts)  # Zipf skew
    src = host(p["sorted_src"]).astype(np.int64)
    assert np.array_equal(np.sort(src), np.arange(T * k))
    flat = host(idx).ravel()
    off = host(p["offsets"])
    for e in range(E):
        seg = src[off[e]:off[e + 1]]
        assert np.all(flat[seg] == e) and np.all(np.diff(seg) > 0)
    ones = torch.ones((T, k), dtype=torch.float32, device=DEV)
    back = foe.combine(p["x_perm"], p["row_of"], ones)
    assert torch.equal(back.float(), (x.float() * k).bfloat16().float())


def test_block_graph_replay_matches_eager():
    """The block captured in a HIP graph: every replay (with eager work and
    synchronisations in between) equals the eager result bit for bit."""
    inp = cfg_inputs("decode_bf16")
    cfg = inp["cfg"]
    say("block graph replay")
    w = stacked(inp)
    x = to_dev(inp["x"], "bf16")
    C, T, d, E, k, F = cfg["C"], cfg["T"], cfg["d"], cfg["E"], cfg["k"], cfg["F"]
    ws = torch.empty(foe.workspace_bytes("cluster_block", foe.BF16, C, T, d, E, k, F),
                     dtype=torch.uint8, device=DEV)
    out = torch.empty((T, d), dtype=torch.bfloat16, device=DEV)
    eager = foe.cluster_block(x, w["w_router"], w["bias"], w["w_gate"], w["w_up"], w["w_down"], k,
                              ws=ws).clone()
    g = torch.cuda.CUDAGraph()
    side = torch.cuda.Stream()
    with torch.cuda.graph(g, stream=side):
        foe.cluster_block(x, w["w_router"], w["bias"], w["w_gate"], w["w_up"], w["w_down"], k,
                          out=out, ws=ws, stream=side)
    for rep in range(4):
        out.fill_(0)
        ws.fill_(7)  # scribble over the workspace between replays
        g.replay()
        torch.cuda.synchronize()
        assert torch.equal(out, eager), rep
        # unrelated eager work in between
        foe.route(x, w["w_router"][0], None, k)
        torch.cuda.synchronize()
