"""The C ABI on the host: the library loads, exports every function the
header declares, sizes workspaces, and rejects invalid arguments before it
touches the GPU (these calls enqueue nothing, so they run without one)."""
import ctypes
import os
import re

import pytest

import paper_2608_06411_amd as mp
from paper_2608_06411_amd import binding as bd


@pytest.fixture(scope="module")
def L():
    if not os.path.exists(bd.LIB_PATH):
        pytest.fail("libmap.so is not built (run python -m paper_2608_06411_amd.build)")
    return bd.lib()


def test_header_declarations_are_exported(L, repo_root):
    header = open(os.path.join(repo_root, "include", "map.h")).read()
    declared = set(re.findall(r"\b(map_[a-z_]+)\s*\(", header))
    assert declared == set(bd.EXPORTS)
    for name in declared:
        assert hasattr(L, name)


def test_status_strings_and_version(L):
    assert L.map_status_string(0) == b"ok"
    assert b"workspace" in L.map_status_string(3)
    assert L.map_status_string(99) == b"unknown status"
    assert L.map_version() >= 100


def _fake_weights(D=64, D_h=32, d_p=16):
    w = bd.map_weights()
    for i, n in enumerate(("w1_v", "b1_v", "w2_v", "b2_v", "w_k", "w1_t", "b1_t", "w2_t", "b2_t", "w_q")):
        setattr(w, n, 0x1000 * (i + 1))
    w.D, w.D_h, w.d_p, w.rope_theta = D, D_h, d_p, 10000.0
    return w


def test_workspace_sizes(L):
    w = _fake_weights()
    assert L.map_score_workspace(bd.MAP_BF16, 2, 100, 10, ctypes.byref(w)) > 0
    assert L.map_select_workspace(2, 100, 10) >= 2 * 10 * 100 * 4
    assert L.map_similarity_workspace(bd.MAP_F32, 1, 100, 64) >= 400
    assert L.map_prune_workspace(bd.MAP_BF16, 1, 100, 5, ctypes.byref(w), 10) >= 100 * 100 * 4
    # invalid sizes give 0
    assert L.map_select_workspace(1, 10, 11) == 0
    assert L.map_select_workspace(1, 10, 0) == 0
    assert L.map_select_workspace(0, 10, 1) == 0
    assert L.map_select_workspace(bd.MAP_MAX_BATCH + 1, 10, 1) == 0
    assert L.map_select_workspace(1, bd.MAP_MAX_N + 1, 1) == 0
    assert L.map_similarity_workspace(bd.MAP_F32, 1, 100, 60) == 0
    bad = _fake_weights(d_p=130)
    assert L.map_score_workspace(bd.MAP_F32, 1, 100, 5, ctypes.byref(_fake_weights(d_p=6))) == 0
    assert L.map_score_workspace(bd.MAP_F32, 1, 100, 5, ctypes.byref(bad)) == 0
    bad = _fake_weights(D=60)
    assert L.map_prune_workspace(bd.MAP_F32, 1, 100, 5, ctypes.byref(bad), 10) == 0
    bad = _fake_weights()
    bad.w_q = None
    assert L.map_score_workspace(bd.MAP_F32, 1, 100, 5, ctypes.byref(bad)) == 0


P = ctypes.c_void_p


def _select(L, B=1, N=100, K=10, K0=5, tau=1e-2, p=1, S=1, n=1, idx=1, ws=None, nbytes=0):
    sp = bd.map_select_params(K, K0, tau)
    return L.map_select(B, N, P(p), P(S), P(n), sp, P(idx), None, None, ws, nbytes, None)


def test_select_argument_checks(L):
    assert _select(L, K=101) == bd.MAP_ERR_INVALID_ARG
    assert _select(L, K=0) == bd.MAP_ERR_INVALID_ARG
    assert _select(L, K0=11) == bd.MAP_ERR_INVALID_ARG
    assert _select(L, K0=-1) == bd.MAP_ERR_INVALID_ARG
    assert _select(L, tau=float("nan")) == bd.MAP_ERR_INVALID_ARG
    assert _select(L, tau=-1.0) == bd.MAP_ERR_INVALID_ARG
    assert _select(L, p=0) == bd.MAP_ERR_INVALID_ARG
    assert _select(L, idx=0) == bd.MAP_ERR_INVALID_ARG
    assert _select(L, B=0) == bd.MAP_ERR_INVALID_ARG
    assert _select(L, N=bd.MAP_MAX_N + 1, K=5) == bd.MAP_ERR_INVALID_ARG
    # valid request, missing / misaligned / short workspace
    need = L.map_select_workspace(1, 100, 10)
    assert _select(L) == bd.MAP_ERR_WORKSPACE
    assert _select(L, ws=P(0x10010), nbytes=need) == bd.MAP_ERR_WORKSPACE
    assert _select(L, ws=P(0x10000), nbytes=need - 1) == bd.MAP_ERR_WORKSPACE


def test_score_and_prune_argument_checks(L):
    w = _fake_weights()
    offs = (ctypes.c_int32 * 3)(0, 4, 9)
    args = [ctypes.byref(w), bd.MAP_BF16, 2, 100, P(1), P(1), P(1), P(1)]
    assert L.map_score(*args, offs, P(1), None, 0, None) == bd.MAP_ERR_WORKSPACE
    for bad in [(0, 4, 4), (1, 4, 9), (0, 9, 4)]:        # empty question, wrong start, decreasing
        o = (ctypes.c_int32 * 3)(*bad)
        assert L.map_score(*args, o, P(1), None, 0, None) == bd.MAP_ERR_INVALID_ARG
    assert L.map_score(*args, None, P(1), None, 0, None) == bd.MAP_ERR_INVALID_ARG
    assert L.map_score(ctypes.byref(w), 7, 2, 100, P(1), P(1), P(1), P(1), offs, P(1), None, 0,
                       None) == bd.MAP_ERR_INVALID_ARG
    sp = bd.map_select_params(10, 5, 1e-2)
    pr = [ctypes.byref(w), bd.MAP_BF16, 2, 100, P(1), P(1), P(1), P(1), offs, sp]
    assert L.map_prune(*pr, P(1), P(1), P(1), None, None, None, None, 0, None) == bd.MAP_ERR_WORKSPACE
    assert L.map_prune(*pr, P(1), None, P(1), None, None, None, None, 0, None) == bd.MAP_ERR_INVALID_ARG
    sp_bad = bd.map_select_params(101, 5, 1e-2)
    pr[-1] = sp_bad
    assert L.map_prune(*pr, P(1), P(1), P(1), None, None, None, None, 0, None) == bd.MAP_ERR_INVALID_ARG


def test_similarity_argument_checks(L):
    assert L.map_similarity(bd.MAP_F32, 1, 10, 12, P(1), P(1), P(1), None, 0, None) == bd.MAP_ERR_INVALID_ARG
    assert L.map_similarity(bd.MAP_F32, 1, 10, 16, P(1), None, P(1), None, 0, None) == bd.MAP_ERR_INVALID_ARG
    assert L.map_similarity(bd.MAP_F32, 1, 10, 16, P(1), P(1), P(1), None, 0, None) == bd.MAP_ERR_WORKSPACE


def test_timing_registry_without_launches(L):
    mp.timing_reset()
    mp.timing_enable(True)
    assert mp.timing_read() == {}
    mp.timing_enable(False)
