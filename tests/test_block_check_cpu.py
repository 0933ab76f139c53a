"""CPU checks of the block comparison itself: mistakes planted in the oracle's
result must fail it, the exact result rounded to the storage type must pass.

The planted mistakes are of the size that a bug in one cluster's update would
cause at the layer-share shape (C = 8 clusters averaged), where the update is
small next to the residual."""

import numpy as np
import pytest

import block_check as bc
from paper_2605_06206_amd import synth


@pytest.fixture(scope="module")
def share8():
    """The 8-cluster layer-share workload on its first 512 tokens."""
    inp = synth.make_block_inputs("layer_share_bf16", T=512)
    k = inp["cfg"]["k"]
    out, res, adopted = bc.oracle_block(inp["x"], inp["clusters"], k)
    assert adopted == 0
    return inp, out, res


def _stored(v):
    return synth.round_to_bf16(np.asarray(v, np.float32)).astype(np.float64)


def test_exact_result_rounded_to_bf16_passes(share8):
    inp, ref, _ = share8
    e_out, e_upd = bc.block_errors(_stored(ref), ref, inp["x"], 8, None, "bf16")
    assert e_out <= 2.0 ** -8 and e_upd == 0.0


@pytest.mark.parametrize("factor", [0.0, 0.5])
def test_one_cluster_update_wrong_fails(share8, factor):
    """One cluster's update zeroed (0.0) or halved (0.5).  Halving moves out by
    little next to the residual, so the out bound alone lets it through; the
    update-part bound does not."""
    inp, ref, res = share8
    bad = ref + (factor - 1.0) * res[3]["delta"] / 8.0
    e_out, e_upd = bc.block_errors(_stored(bad), ref, inp["x"], 8, None, "bf16")
    assert e_upd > bc.TOL["bf16"]
    if factor == 0.5:
        assert e_out < bc.TOL["bf16"]


def test_small_relative_error_in_all_updates_fails(share8):
    """A 3% scale error of every cluster's update (e.g. a wrong routing
    weight normalisation) stays inside the out bound but not the update one."""
    inp, ref, _ = share8
    x = inp["x"].astype(np.float64)
    bad = x + 1.03 * (ref - x)
    e_out, e_upd = bc.block_errors(_stored(bad), ref, inp["x"], 8, None, "bf16")
    assert e_out < bc.TOL["bf16"] < e_upd


def test_near_tie_tokens_take_the_device_ids():
    """A token exactly on a k/(k+1) tie is routed as the device routed it, and
    the oracle's weights follow its own scores at those ids."""
    rng = np.random.default_rng(4)
    T, d, E, k, F = 6, 16, 4, 1, 8
    x = rng.standard_normal((T, d))
    cl = {"w_router": rng.standard_normal((E, d)) * 0.3, "bias": None,
          "w_gate": rng.standard_normal((E, F, d)) * 0.3,
          "w_up": rng.standard_normal((E, F, d)) * 0.3,
          "w_down": rng.standard_normal((E, d, F)) * 0.3}
    cl["w_router"][2] = cl["w_router"][1]  # experts 1 and 2 always tie
    routes = bc.oracle_routes(x, [cl], k)
    ex = routes[0]["margin"] < bc.EXEMPT
    top = routes[0]["idx"][:, 0]
    assert np.array_equal(ex, (top == 1))  # exempt exactly where 1 (tying 2) wins
    assert ex.any()
    dev = routes[0]["idx"].copy()
    dev[ex] = 2
    with pytest.raises(ValueError):
        bc.oracle_block(x, [cl], k, routes=bc.oracle_routes(x, [cl], k))
    out, res, adopted = bc.oracle_block(x, [cl], k, device_idx=[dev])
    assert adopted == int(ex.sum())
    assert np.array_equal(res[0]["idx"][:, 0], dev[:, 0])
    # identical router rows and expert 2's own FFN: the adopted token's update
    # is expert 2's FFN with weight 1
    t = int(np.nonzero(ex)[0][0])
    import oracle
    want = x[t] + oracle.swiglu_ffn(x[t:t + 1], cl["w_gate"][2], cl["w_up"][2], cl["w_down"][2])[0]
    assert np.max(np.abs(out[t] - want)) <= 1e-12
