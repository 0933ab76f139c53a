"""foe_cluster_block_noalloc (no workspace argument; the library's per-GPU
scratch array) against foe_cluster_block on the same inputs, through the C
ABI: two calls in a row, the second with a smaller input, each bit-identical
to the workspace entry point (both run the same kernels)."""

import sys

import numpy as np
import pytest
import torch

from paper_2605_06206_amd import foe, synth

pytestmark = pytest.mark.gpu
DEV = "cuda:0"


def say(*a):
    print("[no-alloc]", *a, file=sys.stderr, flush=True)


def _inputs(cfg):
    inp = synth.make_block_inputs(cfg)

    def up(a):
        return torch.from_numpy(synth.bf16_bits(a)).to(DEV).view(torch.bfloat16)

    cls = inp["clusters"]
    w = {key: up(np.stack([c[key] for c in cls])) for key in ("w_router", "w_gate", "w_up",
                                                              "w_down")}
    w["bias"] = (torch.from_numpy(np.stack([c["bias"] for c in cls])).to(DEV)
                 if cls[0]["bias"] is not None else None)
    return up(inp["x"]), w


@pytest.fixture(autouse=True, scope="module")
def _need_gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    foe.lib()


def test_noalloc_matches_workspace_entry_point_on_two_calls():
    # first the prefill-shaped block (Zipf skew, index pass and grouped GEMM
    # path), then a smaller decode-shaped one with two clusters (the path in
    # which the FFN lists its experts' pairs and the down kernel combines)
    cases = [("prefill_zipf_bf16 C=1 T=8192", "prefill_zipf_bf16"),
             ("decode C=2 T=96", dict(dtype="bf16", C=2, T=96, d=2048, E=8, k=2, F=1024,
                                      sigma=0.02, seed=41, bias=None))]
    k = 2
    runs = []
    for label, case in cases:
        x, w = _inputs(case)
        C, E, F = w["w_gate"].shape[0], w["w_gate"].shape[1], w["w_gate"].shape[2]
        T, d = x.shape
        need = foe.workspace_bytes("cluster_block", foe.BF16, C, T, d, E, k, F)
        say(label, "workspace bytes", need, "of", foe.NOALLOC_SCRATCH_BYTES)
        assert need <= foe.NOALLOC_SCRATCH_BYTES
        ref = foe.cluster_block(x, w["w_router"], w["bias"], w["w_gate"], w["w_up"], w["w_down"],
                                k)
        runs.append((label, x, w, ref))
    torch.cuda.synchronize()
    # the two calls of the entry point in a row: the second finds the first's
    # contents in the scratch array
    outs = []
    for label, x, w, _ in runs:
        say(label, "no-alloc call")
        outs.append(foe.cluster_block_noalloc(x, w["w_router"], w["bias"], w["w_gate"], w["w_up"],
                                              w["w_down"], k))
    torch.cuda.synchronize()
    for (label, _, _, ref), got in zip(runs, outs):
        assert torch.isfinite(got.float()).all(), label
        assert torch.equal(got, ref), label
        say(label, "bit-identical to foe_cluster_block")
