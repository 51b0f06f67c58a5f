"""map_assemble on the GPU: the pruned image's kept rows and its question
rows packed for the language model, byte-exact against oracle.assemble fed
the same inputs (map_prune's kept rows and positions, the question rows), and
map_prune_assemble, which writes the same layout from the selection's gather."""
import numpy as np
import pytest
import torch

import oracle
from workloads import get_config, make_inputs

from gpu_util import announce, dev_inputs, device

pytestmark = pytest.mark.gpu


def _bits(t):
    if t.dtype == torch.bfloat16:
        return t.view(torch.int16).cpu().numpy().view(np.uint16)
    return t.cpu().numpy()


@pytest.mark.parametrize("name,over", [
    ("tiny", {}),
    ("sweep", {"B": 3, "N": 600, "M": (16, 90), "K": 64, "K0": 32}),
])
def test_assemble_after_prune(name, over):
    from paper_2608_06411_amd import map_assemble, map_prune
    cfg = get_config(name, **over)
    announce(f"assemble {name} {over}")
    x = make_inputs(cfg)
    d = dev_inputs(x, device())
    o = map_prune(d["w"], d["V"], d["pos_v"], d["T"], d["pos_t"], x["t_off"], cfg.K, cfg.K0, cfg.tau)
    X, pos = map_assemble(o["V_out"], o["pos_out"], d["T"], d["pos_t"], x["t_off"])
    torch.cuda.synchronize()
    V_out, pos_out, idx = _bits(o["V_out"]), o["pos_out"].cpu().numpy(), o["idx"].cpu().numpy()
    want_X, want_pos = oracle.assemble(V_out, pos_out, x["T_store"], x["pos_t"], x["t_off"])
    got_X = _bits(X)
    assert got_X.shape == want_X.shape and pos.shape == want_pos.shape
    np.testing.assert_array_equal(got_X, want_X)
    np.testing.assert_array_equal(pos.cpu().numpy(), want_pos)
    # the kept rows are the image's own rows at the kept indices, in original order
    for b in range(cfg.B):
        start = b * cfg.K + int(x["t_off"][b])
        np.testing.assert_array_equal(got_X[start:start + cfg.K], x["V_store"][b][idx[b]])
        np.testing.assert_array_equal(pos.cpu().numpy()[start:start + cfg.K], x["pos_v"][b][idx[b]])


@pytest.mark.parametrize("name,over,subset", [
    ("tiny", {}, 0),                                                        # float32: full path, gathered by the selection
    ("sweep", {"B": 3, "N": 600, "M": (16, 90), "K": 64, "K0": 32}, 0),     # subset path, certified images
    ("sweep", {"B": 2, "N": 960, "M": (16, 64), "K": 96, "K0": 48}, 96),    # a subset too small: full selection behind it
    ("sweep", {"B": 2, "N": 700, "M": (16, 128), "K": 320, "K0": 160}, -1),  # a large K on the full path
    ("sweep", {"B": 2, "N": 600, "M": (100, 130), "K": 8, "K0": 4}, -1),    # more question rows than kept rows
])
def test_prune_assemble_fused(name, over, subset):
    """map_prune_assemble writes the layer-0 input in the same launches that
    select and gather: byte-exact against oracle.assemble of map_prune's own
    kept rows (same indices), and against map_assemble."""
    from paper_2608_06411_amd import map_assemble, map_prune, map_prune_assemble, set_subset_tokens
    cfg = get_config(name, **over)
    announce(f"fused assembly {name} {over} subset={subset}")
    x = make_inputs(cfg)
    d = dev_inputs(x, device())
    set_subset_tokens(subset)
    try:
        f = map_prune_assemble(d["w"], d["V"], d["pos_v"], d["T"], d["pos_t"], x["t_off"], cfg.K, cfg.K0, cfg.tau)
        o = map_prune(d["w"], d["V"], d["pos_v"], d["T"], d["pos_t"], x["t_off"], cfg.K, cfg.K0, cfg.tau)
    finally:
        set_subset_tokens(0)
    X2, pos2 = map_assemble(o["V_out"], o["pos_out"], d["T"], d["pos_t"], x["t_off"])
    torch.cuda.synchronize()
    for k in ("idx", "order", "gain", "p"):
        assert torch.equal(f[k], o[k]), k
    want_X, want_pos = oracle.assemble(_bits(o["V_out"]), o["pos_out"].cpu().numpy(), x["T_store"], x["pos_t"],
                                       x["t_off"])
    np.testing.assert_array_equal(_bits(f["X"]), want_X)
    np.testing.assert_array_equal(f["pos_x"].cpu().numpy(), want_pos)
    np.testing.assert_array_equal(_bits(f["X"]), _bits(X2))
    np.testing.assert_array_equal(f["pos_x"].cpu().numpy(), pos2.cpu().numpy())
    idx = f["idx"].cpu().numpy()
    for b in range(cfg.B):
        start = b * cfg.K + int(x["t_off"][b])
        np.testing.assert_array_equal(_bits(f["X"])[start:start + cfg.K], x["V_store"][b][idx[b]])


def test_prune_assemble_large_k():
    """K = 1000 of 1024 tokens (the pool shrinks to fit the coefficient
    columns in LDS) with questions of up to 40 tokens: the layer-0 output
    matches map_prune + oracle.assemble."""
    import paper_2608_06411_amd as mp
    from workloads import PredictorShape
    cfg = get_config("sweep", B=2, N=1024, M=(8, 40), K=1000, K0=500, pred=PredictorShape(D=256, D_h=64, d_p=32))
    announce("fused assembly, K = 1000")
    x = make_inputs(cfg)
    d = dev_inputs(x, device())
    f = mp.map_prune_assemble(d["w"], d["V"], d["pos_v"], d["T"], d["pos_t"], x["t_off"], cfg.K, cfg.K0, cfg.tau)
    o = mp.map_prune(d["w"], d["V"], d["pos_v"], d["T"], d["pos_t"], x["t_off"], cfg.K, cfg.K0, cfg.tau)
    torch.cuda.synchronize()
    assert torch.equal(f["idx"], o["idx"])
    want_X, want_pos = oracle.assemble(_bits(o["V_out"]), o["pos_out"].cpu().numpy(), x["T_store"], x["pos_t"],
                                       x["t_off"])
    np.testing.assert_array_equal(_bits(f["X"]), want_X)
    np.testing.assert_array_equal(f["pos_x"].cpu().numpy(), want_pos)
