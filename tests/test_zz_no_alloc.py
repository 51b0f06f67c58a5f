"""map_prune_noalloc: map_prune with its workspace in the library's static
device buffer, for callers that cannot allocate.  Called through the C ABI
and checked bit for bit against map_prune on the same inputs (the same
kernels run on the same values), on two calls in a row, the second with a
smaller input; a call whose workspace would exceed the buffer is refused
with MAP_ERR_TOO_LARGE and enqueues nothing."""
import ctypes

import numpy as np
import pytest
import torch

import paper_2608_06411_amd as mp
from paper_2608_06411_amd import binding as bd
from workloads import get_config, make_inputs

from gpu_util import announce, dev_inputs, device

pytestmark = pytest.mark.gpu


def _noalloc(d, t_off, K, K0, tau, dev):
    V = d["V"]
    B, N, D = V.shape
    o = {"idx": torch.full((B, K), -7, dtype=torch.int32, device=dev),
         "V_out": torch.zeros(B, K, D, dtype=V.dtype, device=dev),
         "pos_out": torch.full((B, K), -7, dtype=torch.int32, device=dev),
         "p": torch.zeros(B, N, dtype=torch.float32, device=dev),
         "order": torch.full((B, K), -7, dtype=torch.int32, device=dev),
         "gain": torch.zeros(B, K, dtype=torch.float32, device=dev)}
    offs = (ctypes.c_int32 * len(t_off))(*[int(x) for x in t_off])
    w = d["w"].struct()
    st = bd.lib().map_prune_noalloc(
        ctypes.byref(w), bd._dtype_code(V), B, N, bd._ptr(V), bd._ptr(d["pos_v"]), bd._ptr(d["T"]),
        bd._ptr(d["pos_t"]), offs, bd.map_select_params(K, K0, tau), bd._ptr(o["idx"]), bd._ptr(o["V_out"]),
        bd._ptr(o["pos_out"]), bd._ptr(o["p"]), bd._ptr(o["order"]), bd._ptr(o["gain"]), bd._stream(dev))
    return st, o


def test_prune_noalloc_matches_prune_on_two_calls():
    dev = device()
    shapes = [("llava_next", {}), ("sweep", {"B": 2, "N": 640, "M": (16, 48), "K": 64, "K0": 32})]
    for name, over in shapes:  # the second call is smaller than the first
        cfg = get_config(name, **over)
        announce(f"map_prune_noalloc {name} B={cfg.B} N={cfg.N} K={cfg.K}")
        x = make_inputs(cfg)
        d = dev_inputs(x, dev)
        st, got = _noalloc(d, x["t_off"], cfg.K, cfg.K0, cfg.tau, dev)
        assert st == bd.MAP_OK, bd.lib().map_status_string(st)
        torch.cuda.synchronize()
        ref = mp.map_prune(d["w"], d["V"], d["pos_v"], d["T"], d["pos_t"], x["t_off"], cfg.K, cfg.K0, cfg.tau)
        torch.cuda.synchronize()
        for k in ("p", "idx", "order", "gain", "pos_out", "V_out"):
            assert torch.equal(got[k], ref[k]), (name, k)
        idx = got["idx"].cpu().numpy()
        for b in range(cfg.B):
            assert np.array_equal(idx[b], np.sort(got["order"].cpu().numpy()[b]))


def test_prune_noalloc_refuses_more_than_its_buffer():
    dev = device()
    cfg = get_config("sweep", B=2, N=2880, M=(64, 64), K=160, K0=80)   # about 124 MiB of workspace
    x = make_inputs(cfg)
    d = dev_inputs(x, dev)
    need = bd.lib().map_prune_workspace(bd.MAP_BF16, cfg.B, cfg.N, int(x["t_off"][-1]),
                                        ctypes.byref(d["w"].struct()), cfg.K)
    assert need > bd.MAP_PRUNE_NOALLOC_MAX_BYTES
    st, o = _noalloc(d, x["t_off"], cfg.K, cfg.K0, cfg.tau, dev)
    torch.cuda.synchronize()
    assert st == bd.MAP_ERR_TOO_LARGE
    assert int(o["idx"].min()) == -7 and int(o["idx"].max()) == -7   # nothing was written
