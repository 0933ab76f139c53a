"""C-ABI checks that need no GPU: the library loads, exports every symbol the
header declares, and rejects bad arguments on the host before enqueuing work
(no call here reaches a kernel launch)."""

import ctypes
import os
import re

import pytest

from paper_2605_06206_amd import foe

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "foe.h")
SIZE_MAX = ctypes.c_size_t(-1).value

# fake, 16-byte aligned addresses: never dereferenced because every call below
# fails validation (or is a documented no-op) before anything is enqueued
P = 0x10000
P2 = 0x20000


@pytest.fixture(scope="module")
def L():
    if not os.path.exists(foe.LIB_PATH):
        from paper_2605_06206_amd import build
        build.build()
    return foe.lib()


def declared_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(foe_[a-z_]+)\s*\(", text)))


def test_header_declares_the_block_entry_points():
    names = declared_functions()
    for n in ("foe_route", "foe_permute", "foe_expert_ffn", "foe_combine", "foe_cluster_block",
              "foe_reduce", "foe_workspace_bytes", "foe_last_error"):
        assert n in names


def test_library_exports_every_declared_symbol(L):
    for name in declared_functions():
        assert hasattr(L, name), name
        assert name in foe._SIGNATURES, f"binding lacks {name}"


def test_exported_symbols_are_plain_c(root_dir):
    import subprocess
    if not os.path.exists(foe.LIB_PATH):
        pytest.skip("library not built")
    out = subprocess.run(["nm", "-D", "--defined-only", foe.LIB_PATH], capture_output=True,
                         text=True).stdout
    exported = {ln.split()[-1] for ln in out.splitlines() if " T " in ln}
    for name in declared_functions():
        assert name in exported, name


BF16, F32 = foe.BF16, foe.F32
INV, WS = foe.FOE_ERR_INVALID, foe.FOE_ERR_WORKSPACE


@pytest.mark.parametrize("args,msg", [
    ((7, 16, 64, 4, 2, P, P, None, P, P, None), "dt"),
    ((BF16, 16, 60, 4, 2, P, P, None, P, P, None), "d must"),
    ((BF16, 16, 64, 4, 0, P, P, None, P, P, None), "k must"),
    ((BF16, 16, 64, 4, 5, P, P, None, P, P, None), "k must"),
    ((BF16, 16, 64, 300, 2, P, P, None, P, P, None), "E must"),
    ((BF16, -1, 64, 4, 2, P, P, None, P, P, None), "T must"),
    ((BF16, 16, 64, 4, 2, None, P, None, P, P, None), "x is NULL"),
    ((BF16, 16, 64, 4, 2, P + 8, P, None, P, P, None), "x is not 16-byte aligned"),
    ((BF16, 16, 64, 4, 2, P, P, P + 2, P, P, None), "bias is not 4-byte aligned"),
    ((BF16, 16, 64, 4, 2, P, P, None, None, P, None), "topk_idx is NULL"),
])
def test_route_rejects(L, args, msg):
    assert L.foe_route(*args) == INV
    assert msg in foe.last_error()


def test_route_empty_batch_is_a_noop(L):
    assert L.foe_route(BF16, 0, 64, 4, 2, None, None, None, None, None, None) == foe.FOE_OK


def test_route_ex_rejects(L):
    base = [BF16, 2, 16, 64, 4, 2, foe.GATE_GLOBAL, P, P, None, P, P, None]
    bad = list(base)
    bad[6] = 2
    assert L.foe_route_ex(*bad) == INV and "gating must" in foe.last_error()
    bad = list(base)
    bad[1] = 0
    assert L.foe_route_ex(*bad) == INV and "G must" in foe.last_error()
    big = list(base)
    big[1], big[4] = 3, 100  # 300 score columns across groups
    assert L.foe_route_ex(*big) == foe.FOE_ERR_UNSUPPORTED
    assert L.foe_route_ex(BF16, 2, 0, 64, 4, 2, foe.GATE_RENORM, None, None, None, None, None,
                          None) == foe.FOE_OK


def test_cluster_block_ex_rejects(L):
    need = L.foe_workspace_bytes(b"cluster_block", BF16, 2, 64, 64, 200, 2, 64)
    args = [BF16, 2, 64, 64, 200, 2, 64, foe.GATE_GLOBAL, P, P, None, P, P, P,
            ctypes.c_float(0.5), P, P2, need, None]
    assert L.foe_cluster_block_ex(*args) == foe.FOE_ERR_UNSUPPORTED
    assert "global gating" in foe.last_error()
    bad = list(args)
    bad[7] = 5
    assert L.foe_cluster_block_ex(*bad) == INV and "gating must" in foe.last_error()


def test_group_attention_rejects(L):
    n = L.foe_group_attention_workspace_bytes(8, 4096, 2048, 2, 128)
    assert 0 < n < SIZE_MAX
    assert L.foe_group_attention_workspace_bytes(8, 4096, 2048, 2, 64) == SIZE_MAX
    assert "hd must be 96 or 128" in foe.last_error()
    assert 0 < L.foe_group_attention_workspace_bytes(8, 4096, 2048, 1, 96) < SIZE_MAX
    f = ctypes.c_float
    ok = [BF16, 2, 64, 64, 2, 128, f(500000.0), f(16.0), P, P, P, P]
    bad = list(ok)
    bad[5] = 64
    assert L.foe_group_attention(*bad, P2, n, None) == foe.FOE_ERR_UNSUPPORTED
    bad = list(ok)
    bad[0] = F32
    assert L.foe_group_attention(*bad, P2, n, None) == foe.FOE_ERR_UNSUPPORTED
    bad = list(ok)
    bad[1] = 0
    assert L.foe_group_attention(*bad, P2, n, None) == INV and "H must" in foe.last_error()
    bad = list(ok)
    bad[6] = f(0.0)
    assert L.foe_group_attention(*bad, P2, n, None) == INV and "theta" in foe.last_error()
    bad = list(ok)
    bad[8] = None
    assert L.foe_group_attention(*bad, P2, n, None) == INV and "x is NULL" in foe.last_error()
    need = L.foe_group_attention_workspace_bytes(2, 64, 64, 2, 128)
    assert L.foe_group_attention(*ok, P2, need - 256, None) == WS
    assert L.foe_group_attention(BF16, 2, 0, 64, 2, 128, f(500000.0), f(16.0), None, None, None,
                                 None, None, 0, None) == foe.FOE_OK


def test_permute_rejects(L):
    need = L.foe_workspace_bytes(b"permute", BF16, 1, 4096, 64, 8, 2, 0)
    assert 0 < need < SIZE_MAX
    base = (BF16, 4096, 64, 8, 2, P, P, None, P, P, P, P)
    assert L.foe_permute(*base, P2, need - 4, None) == WS
    assert "workspace needs" in foe.last_error()
    assert L.foe_permute(*base, None, need, None) == INV
    assert L.foe_permute(BF16, 4096, 64, 8, 2, P, P, None, None, P, P, P, P2, need, None) == INV
    assert "expert_offsets is NULL" in foe.last_error()
    assert L.foe_permute(BF16, 4096, 64, 8, 9, P, P, None, P, P, P, P, P2, need, None) == INV


def test_expert_ffn_rejects(L):
    need = L.foe_workspace_bytes(b"expert_ffn", BF16, 1, 512, 64, 8, 1, 128)
    assert need >= 512 * 128 * 2
    ok = (BF16, 8, 64, 128, 512, P, P, P, P, P, P)
    assert L.foe_expert_ffn(*ok, P2, need - 1, None) == WS
    assert L.foe_expert_ffn(BF16, 8, 64, 100, 512, P, P, P, P, P, P, P2, need, None) == INV
    assert "F must" in foe.last_error()
    assert L.foe_expert_ffn(BF16, 0, 64, 128, 512, P, P, P, P, P, P, P2, need, None) == INV
    assert L.foe_expert_ffn(BF16, 8, 64, 128, 512, P, P, None, P, P, P, P2, need, None) == INV
    # zero rows: nothing to do, no workspace needed
    assert L.foe_expert_ffn(BF16, 8, 64, 128, 0, None, None, None, None, None, None, None, 0,
                            None) == foe.FOE_OK


def test_combine_and_reduce_reject(L):
    assert L.foe_combine(BF16, 16, 64, 0, P, P, P, None, P, None) == INV
    assert L.foe_combine(BF16, 16, 64, 2, P, P, P, P + 4, P, None) == INV
    assert "residual" in foe.last_error()
    assert L.foe_combine(BF16, 0, 64, 2, None, None, None, None, None, None) == foe.FOE_OK
    assert L.foe_reduce(BF16, 0, 16, 64, P, None, ctypes.c_float(1.0), P, None) == INV
    assert L.foe_reduce(BF16, 65, 16, 64, P, None, ctypes.c_float(1.0), P, None) == INV
    assert L.foe_reduce(F32, 2, 16, 64, None, None, ctypes.c_float(1.0), P, None) == INV
    assert L.foe_reduce(F32, 2, 0, 64, None, None, ctypes.c_float(1.0), None, None) == foe.FOE_OK


def test_cluster_block_rejects(L):
    need = L.foe_workspace_bytes(b"cluster_block", BF16, 8, 4096, 2048, 8, 2, 1024)
    assert 0 < need < SIZE_MAX
    args = [BF16, 8, 4096, 2048, 8, 2, 1024, P, P, None, P, P, P, ctypes.c_float(0.125), P]
    assert L.foe_cluster_block(*args, P2, need - 256, None) == WS
    bad_c = list(args)
    bad_c[1] = 0
    assert L.foe_cluster_block(*bad_c, P2, need, None) == INV
    bad_k = list(args)
    bad_k[5] = 9
    assert L.foe_cluster_block(*bad_k, P2, need, None) == INV
    assert L.foe_cluster_block(BF16, 8, 0, 2048, 8, 2, 1024, None, None, None, None, None, None,
                               ctypes.c_float(0.125), None, None, 0, None) == foe.FOE_OK


def test_cluster_block_noalloc_rejects_on_the_host(L):
    """Sizes past the scratch array and bad arguments are refused before any
    device call (these run without a GPU)."""
    f = ctypes.c_float(0.125)
    cap = foe.NOALLOC_SCRATCH_BYTES
    # the prefill-shaped block fits, the large one does not
    assert L.foe_workspace_bytes(b"cluster_block", BF16, 1, 8192, 2048, 16, 2, 1024) <= cap
    assert L.foe_workspace_bytes(b"cluster_block", BF16, 1, 16384, 4096, 32, 4, 1536) > cap
    big = [BF16, 1, 16384, 4096, 32, 4, 1536, P, P, None, P, P, P, f, P, None]
    assert L.foe_cluster_block_noalloc(*big) == foe.FOE_ERR_UNSUPPORTED
    assert "bytes of scratch" in foe.last_error() and str(cap) in foe.last_error()
    bad = [BF16, 1, 128, 2048, 16, 2, 1024, None, P, None, P, P, P, f, P, None]
    assert L.foe_cluster_block_noalloc(*bad) == INV and "x is NULL" in foe.last_error()
    bad = [BF16, 1, 128, 2048, 16, 17, 1024, P, P, None, P, P, P, f, P, None]
    assert L.foe_cluster_block_noalloc(*bad) == INV and "k must" in foe.last_error()
    assert L.foe_cluster_block_noalloc(BF16, 1, 0, 2048, 16, 2, 1024, None, None, None, None,
                                       None, None, f, None, None) == foe.FOE_OK


def test_workspace_bytes(L):
    for op in (b"route", b"combine", b"reduce"):
        assert L.foe_workspace_bytes(op, BF16, 1, 128, 64, 4, 2, 64) == 0
    assert L.foe_workspace_bytes(b"unknown", BF16, 1, 1, 8, 1, 1, 8) == SIZE_MAX
    assert "unknown op" in foe.last_error()
    assert L.foe_workspace_bytes(None, BF16, 1, 1, 8, 1, 1, 8) == SIZE_MAX
    assert L.foe_workspace_bytes(b"cluster_block", BF16, 1, 128, 2048, 16, 17, 1024) == SIZE_MAX
    small = L.foe_workspace_bytes(b"cluster_block", BF16, 1, 128, 2048, 16, 2, 1024)
    big = L.foe_workspace_bytes(b"cluster_block", BF16, 1, 8192, 2048, 16, 2, 1024)
    more_c = L.foe_workspace_bytes(b"cluster_block", BF16, 8, 8192, 2048, 16, 2, 1024)
    assert 0 < small < big < more_c
    # the FFN output rows and the hidden layer of every (token, slot) dominate
    R = 8192 * 2
    assert big >= R * 2048 * 2 + R * 1024 * 2
    assert more_c >= 8 * (R * 2048 * 2 + R * 1024 * 2)


def test_profile_api_without_records(L):
    assert L.foe_profile_reset() == foe.FOE_OK
    n = ctypes.c_int(0)
    ms = ctypes.c_double(0)
    assert L.foe_profile_kernel(b"route", ctypes.byref(n), ctypes.byref(ms)) == INV
    assert foe.profile_names() == []
