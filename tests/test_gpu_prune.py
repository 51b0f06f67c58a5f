"""map_prune (score + similarity + selection + gather) on the GPU.

* p_hat against the oracle's Eq. (3): 1e-5 relative in float32, 2e-2 in bf16.
* The selection, replayed on the oracle with the GPU's own p_hat (exactly as
  float64): every pick is the oracle's, except below a 1e-4 decisive gap.
* The gather: kept rows and positions byte-exact, indices ascending.
* The candidate subset (bf16): automatic, off, and one so small that the
  certificate rejects its picks and the images are selected again in full;
  every mode meets the same bar.
"""
import numpy as np
import pytest
import torch

import oracle
from workloads import get_config, make_inputs

from gpu_util import announce, dev_inputs, device, oracle_weights

pytestmark = pytest.mark.gpu


def _prune(x, K, K0, tau):
    from paper_2608_06411_amd import map_prune
    dev = device()
    d = dev_inputs(x, dev)
    o = map_prune(d["w"], d["V"], d["pos_v"], d["T"], d["pos_t"], x["t_off"], K, K0, tau)
    torch.cuda.synchronize()
    out = {k: v.cpu() for k, v in o.items()}
    out["V_store_out"] = (out["V_out"].view(torch.int16).numpy().view(np.uint16)
                          if x["cfg"].dtype == "bf16" else out["V_out"].numpy())
    return out


def _check(x, out, K, K0, tau, rtol):
    cfg = x["cfg"]
    p_ref = oracle.predicted_attention_batch(x["V_f32"], x["T_f32"], x["t_off"], x["pos_v"],
                                             x["pos_t"], oracle_weights(x), cfg.pred.rope_theta)
    p = out["p"].numpy().astype(np.float64)
    np.testing.assert_allclose(p, p_ref, rtol=rtol, atol=0)
    idx, order, gain = out["idx"].numpy(), out["order"].numpy(), out["gain"].numpy()
    for b in range(cfg.B):
        rep = oracle.replay_check(p[b], x["V_f32"][b], K, K0, tau, order[b], gain[b])
        assert rep.ok, f"image {b}: {rep.failure}"
        assert rep.max_gain_rel_err < 1e-3
        np.testing.assert_array_equal(idx[b], np.sort(order[b]))
        np.testing.assert_array_equal(out["V_store_out"][b], x["V_store"][b][idx[b]])
        np.testing.assert_array_equal(out["pos_out"].numpy()[b], x["pos_v"][b][idx[b]])
    return rep


@pytest.mark.parametrize("name,over,rtol", [
    ("tiny", {}, 1e-5),
    ("sweep", {"B": 3, "N": 500, "M": (16, 128), "K": 64, "K0": 32}, 2e-2),
    ("sweep", {"B": 2, "N": 700, "M": (16, 128), "K": 320, "K0": 160}, 2e-2),
])
def test_prune_matches_oracle(name, over, rtol):
    cfg = get_config(name, **over)
    announce(f"prune {name} {over}")
    x = make_inputs(cfg)
    out = _prune(x, cfg.K, cfg.K0, cfg.tau)
    _check(x, out, cfg.K, cfg.K0, cfg.tau, rtol)


def test_prune_llava_next_full_size():
    """The headline workload: 2880 tokens x 4096, keep 160 (K0 = 80), bf16."""
    cfg = get_config("llava_next")
    announce("prune llava_next full size")
    x = make_inputs(cfg)
    out = _prune(x, cfg.K, cfg.K0, cfg.tau)
    rep = _check(x, out, cfg.K, cfg.K0, cfg.tau, 2e-2)
    print(f"[llava_next] exact picks {rep.exact}/{rep.steps}, near ties {rep.near_ties}, "
          f"min decisive gap {rep.min_gap:.3g}, max gain rel err {rep.max_gain_rel_err:.3g}")


def test_prune_top_k_mode():
    cfg = get_config("tiny", K=48, K0=48)
    x = make_inputs(cfg)
    out = _prune(x, 48, 48, cfg.tau)
    p = out["p"].numpy()[0].astype(np.float64)
    want = np.sort(np.lexsort((np.arange(cfg.N), -p))[:48])
    np.testing.assert_array_equal(out["idx"].numpy()[0], want)


def test_prune_is_deterministic():
    cfg = get_config("sweep", B=2, N=600, M=(20, 60), K=96, K0=48)
    x = make_inputs(cfg)
    a, b = _prune(x, 96, 48, cfg.tau), _prune(x, 96, 48, cfg.tau)
    for k in ("p", "idx", "order", "gain", "pos_out"):
        np.testing.assert_array_equal(a[k].numpy(), b[k].numpy())
    np.testing.assert_array_equal(a["V_store_out"], b["V_store_out"])


@pytest.mark.parametrize("mode", ["auto", "off", "K", "half"])
def test_prune_subset_modes(mode):
    from paper_2608_06411_amd import set_subset_tokens
    cfg = get_config("sweep", B=2, N=960, M=(16, 64), K=96, K0=48)
    announce(f"prune subset mode {mode}")
    x = make_inputs(cfg)
    set_subset_tokens({"auto": 0, "off": -1, "K": cfg.K, "half": cfg.N // 2}[mode])
    try:
        out = _prune(x, cfg.K, cfg.K0, cfg.tau)
    finally:
        set_subset_tokens(0)
    _check(x, out, cfg.K, cfg.K0, cfg.tau, 2e-2)


@pytest.mark.parametrize("K,K0,n", [(96, 0, 0), (64, 64, 0), (64, 64, 64), (100, 37, 101)])
def test_prune_subset_edges(K, K0, n):
    """The subset with no R0 (K0 = 0), with R0 alone (K0 = K: plain top-K),
    with R0 filling the whole subset (R0's candidates may overflow it: the
    full selection decides), and with an odd K0 and subset size."""
    from paper_2608_06411_amd import set_subset_tokens
    cfg = get_config("sweep", B=2, N=1000, M=(16, 64), K=K, K0=K0)
    announce(f"prune subset edges K={K} K0={K0} n={n}")
    x = make_inputs(cfg)
    set_subset_tokens(n)
    try:
        out = _prune(x, K, K0, cfg.tau)
    finally:
        set_subset_tokens(0)
    _check(x, out, K, K0, cfg.tau, 2e-2)


def test_prune_subset_multiframe_image():
    """D = 3584 (seven K ranges of 512) and a subset too small for the
    eight-frame image's picks: the full selection behind it decides."""
    cfg = get_config("multiframe", B=1)
    announce("prune multiframe B=1")
    x = make_inputs(cfg)
    out = _prune(x, cfg.K, cfg.K0, cfg.tau)
    _check(x, out, cfg.K, cfg.K0, cfg.tau, 2e-2)
