"""map_prune at the workloads' own shapes, and the selection split into
several persistent launches.

* Batched retention sweep: 16 images of 2880 tokens x 4096 (bf16), question
  lengths uniform in [16, 128], K in {64, 160, 320, 640} with K0 = K/2, the
  candidate subset automatic and off.  Every image: p_hat within 2e-2 of the
  oracle's Eq. (3), indices distinct and ascending, the gather byte-exact.
  The selection is replayed on the oracle (Eq. (4), float64, explicit
  Gram-Schmidt) for every image at K <= 160 and for two images per call at
  K = 320 and 640, where one replay costs N D K^2 flops; with the subset off,
  each image whose order differs from the subset run's is replayed too.
  K = 640 is where the pipelined selection no longer fits in LDS and the
  unpipelined variant runs at full N; with the subset off, 16 images of 45
  workgroups exceed what the device holds at once and the selection runs
  as several launches.
* Multi-frame images: 8 images of 4608 tokens x 3584, K = 256.
* The multi-launch path at small sizes: at most one or two images per
  launch must give the same bits as one launch, and replay on the oracle.
* The selection status word reads 0 after a completed call.
* A peaked predictor (weights N(0, 0.03^2): p_hat spans a factor of about
  40) at the LLaVA-NeXT shape, where the 2e-2 bf16 bar is tight against the
  signal (a 10 % logit-scale error moves p_hat by more than that; see
  test_oracle_predictor).

The oracle's replays run in threads (one BLAS thread each) across images.
"""
import os
from concurrent.futures import ThreadPoolExecutor

import numpy as np
import pytest
import torch
from threadpoolctl import threadpool_limits

import oracle
from workloads import PredictorShape, get_config, make_inputs

from gpu_util import announce, dev_inputs, device, oracle_weights

pytestmark = pytest.mark.gpu

CPUS = max(1, min(16, os.cpu_count() or 1))  # the host share of one GPU
WORKERS = CPUS


def _p_ref(x):
    cfg = x["cfg"]
    return oracle.predicted_attention_batch(x["V_f32"], x["T_f32"], x["t_off"], x["pos_v"], x["pos_t"],
                                            oracle_weights(x), cfg.pred.rope_theta)


def _prune(x, d, K, K0, tau, subset=0, per_launch=0, ws_out=None):
    import paper_2608_06411_amd as mp
    mp.set_subset_tokens(subset)
    mp.set_select_images_per_launch(per_launch)
    try:
        ws = mp.PruneWorkspace(d["w"], d["V"], x["t_off"], K)
        o = mp.map_prune(d["w"], d["V"], d["pos_v"], d["T"], d["pos_t"], x["t_off"], K, K0, tau, workspace=ws)
        torch.cuda.synchronize()
        status = mp.selection_status(ws.buf)
    finally:
        mp.set_subset_tokens(0)
        mp.set_select_images_per_launch(0)
    out = {k: v.cpu() for k, v in o.items()}
    out["V_store_out"] = (out["V_out"].view(torch.int16).numpy().view(np.uint16)
                          if x["cfg"].dtype == "bf16" else out["V_out"].numpy())
    out["status"] = status
    return out


def _check_structure(x, out, K, p_ref, rtol):
    """Every image: p_hat, distinct ascending indices, byte-exact gather."""
    cfg = x["cfg"]
    assert out["status"] == 0
    p = out["p"].numpy().astype(np.float64)
    np.testing.assert_allclose(p, p_ref, rtol=rtol, atol=0)
    idx, order = out["idx"].numpy(), out["order"].numpy()
    for b in range(cfg.B):
        assert np.unique(order[b]).size == K and order[b].min() >= 0 and order[b].max() < cfg.N, b
        np.testing.assert_array_equal(idx[b], np.sort(order[b]))
        np.testing.assert_array_equal(out["V_store_out"][b], x["V_store"][b][idx[b]])
        np.testing.assert_array_equal(out["pos_out"].numpy()[b], x["pos_v"][b][idx[b]])


def _replay(x, out, K, K0, tau, images, threads=WORKERS):
    """Replays the GPU's order of each listed image on the oracle, with the
    GPU's own p_hat (exact in float64); images run in parallel threads."""
    if not images:
        return []
    p = out["p"].numpy().astype(np.float64)
    order, gain = out["order"].numpy(), out["gain"].numpy()

    def one(b):
        rep = oracle.replay_check(p[b], x["V_f32"][b], K, K0, tau, order[b], gain[b])
        print(f"[replay] image {b} K={K}: ok={rep.ok} near ties {rep.near_ties}", flush=True)
        return b, rep

    blas = max(1, CPUS // max(1, min(threads, len(images))))
    with threadpool_limits(limits=blas, user_api="blas"), ThreadPoolExecutor(min(threads, len(images))) as ex:
        reps = list(ex.map(one, images))
    for b, rep in reps:
        assert rep.ok, f"image {b}: {rep.failure}"
        assert rep.max_gain_rel_err < 1e-3, (b, rep.max_gain_rel_err)
    return reps


@pytest.fixture(scope="module")
def sweep():
    cfg = get_config("sweep")
    announce(f"sweep inputs B={cfg.B} N={cfg.N} D={cfg.pred.D} M={cfg.M}")
    x = make_inputs(cfg)
    dev = device()
    with threadpool_limits(limits=max(1, CPUS // 4), user_api="blas"), ThreadPoolExecutor(4) as ex:
        rows = list(ex.map(lambda b: oracle.predicted_attention(
            x["V_f32"][b], x["T_f32"][x["t_off"][b]:x["t_off"][b + 1]], x["pos_v"][b],
            x["pos_t"][x["t_off"][b]:x["t_off"][b + 1]], oracle_weights(x), cfg.pred.rope_theta), range(cfg.B)))
    return x, dev_inputs(x, dev), np.stack(rows)


@pytest.mark.timeout(900)
@pytest.mark.parametrize("K", [64, 160, 320, 640])
def test_sweep_retention_budgets(sweep, K):
    x, d, p_ref = sweep
    cfg = x["cfg"]
    K0, tau = K // 2, cfg.tau
    # past K = N / 12 the automatic rule takes the full path at once; a
    # subset of N / 3 forced there still runs the subset, which flags the
    # images it cannot certify for the full selection behind it
    subset = 0 if 12 * K <= cfg.N else cfg.N // 3
    announce(f"sweep B={cfg.B} K={K} subset {subset or 'auto'}")
    auto = _prune(x, d, K, K0, tau, subset=subset)
    _check_structure(x, auto, K, p_ref, 2e-2)
    replayed = list(range(cfg.B)) if K <= 160 else [0, cfg.B - 1]
    reps = _replay(x, auto, K, K0, tau, replayed)
    near = sum(r.near_ties for _, r in reps)
    announce(f"sweep K={K} subset off")
    off = _prune(x, d, K, K0, tau, subset=-1)
    _check_structure(x, off, K, p_ref, 2e-2)
    np.testing.assert_array_equal(off["p"].numpy(), auto["p"].numpy())
    differ = [b for b in range(cfg.B) if not np.array_equal(off["order"].numpy()[b], auto["order"].numpy()[b])]
    _replay(x, off, K, K0, tau, [b for b in differ if b not in replayed] + ([] if differ else [1]))
    print(f"[sweep K={K}] replayed {len(replayed)} images ({near} near ties); "
          f"subset off differs on images {differ}")


@pytest.mark.timeout(900)
def test_multiframe_batch():
    cfg = get_config("multiframe")
    announce(f"multiframe B={cfg.B} N={cfg.N} D={cfg.pred.D} K={cfg.K}")
    x = make_inputs(cfg)
    d = dev_inputs(x, device())
    out = _prune(x, d, cfg.K, cfg.K0, cfg.tau)
    with threadpool_limits(limits=max(1, CPUS // 4), user_api="blas"), ThreadPoolExecutor(4) as ex:
        rows = list(ex.map(lambda b: oracle.predicted_attention(
            x["V_f32"][b], x["T_f32"][x["t_off"][b]:x["t_off"][b + 1]], x["pos_v"][b],
            x["pos_t"][x["t_off"][b]:x["t_off"][b + 1]], oracle_weights(x), cfg.pred.rope_theta), range(cfg.B)))
    _check_structure(x, out, cfg.K, np.stack(rows), 2e-2)
    _replay(x, out, cfg.K, cfg.K0, cfg.tau, list(range(cfg.B)))


@pytest.mark.parametrize("subset,per_launch", [(-1, 1), (-1, 2), (0, 1)])
def test_selection_split_into_launches(subset, per_launch):
    """At most `per_launch` images per persistent selection launch: the same
    bits as one launch, and every image replays on the oracle."""
    cfg = get_config("sweep", B=3, N=640, M=(16, 64), K=96, K0=48)
    announce(f"selection split subset={subset} per_launch={per_launch}")
    x = make_inputs(cfg)
    d = dev_inputs(x, device())
    one = _prune(x, d, cfg.K, cfg.K0, cfg.tau, subset=subset)
    split = _prune(x, d, cfg.K, cfg.K0, cfg.tau, subset=subset, per_launch=per_launch)
    for k in ("p", "idx", "order", "gain", "pos_out"):
        np.testing.assert_array_equal(split[k].numpy(), one[k].numpy())
    np.testing.assert_array_equal(split["V_store_out"], one["V_store_out"])
    _check_structure(x, split, cfg.K, _p_ref(x), 2e-2)
    _replay(x, split, cfg.K, cfg.K0, cfg.tau, list(range(cfg.B)))


def test_map_select_split_into_launches():
    import paper_2608_06411_amd as mp
    from workloads import peaked_scores
    cfg = get_config("sweep", B=4, N=500, M=(16, 16), K=80, K0=40, pred=PredictorShape(D=256, D_h=64, d_p=32))
    announce("map_select split into launches")
    x = make_inputs(cfg, with_weights=False)
    dev = device()
    V = torch.from_numpy(x["V_store"].view(np.int16)).to(dev).view(torch.bfloat16)
    S, n = mp.map_similarity(V)
    p = torch.from_numpy(peaked_scores(cfg.B, cfg.N)).to(dev)
    ref = [t.cpu() for t in mp.map_select(p, S, n, cfg.K, cfg.K0, cfg.tau)]
    mp.set_select_images_per_launch(1)
    try:
        got = [t.cpu() for t in mp.map_select(p, S, n, cfg.K, cfg.K0, cfg.tau)]
    finally:
        mp.set_select_images_per_launch(0)
    for a, b in zip(got, ref):
        assert torch.equal(a, b)
    for b in range(cfg.B):
        rep = oracle.replay_check(p[b].cpu().numpy().astype(np.float64), x["V_f32"][b], cfg.K, cfg.K0, cfg.tau,
                                  got[1][b].numpy())
        assert rep.ok, rep.failure


def test_similarity_norms_only():
    import paper_2608_06411_amd as mp
    cfg = get_config("tiny", N=300, pred=PredictorShape(D=512))
    x = make_inputs(cfg, with_weights=False)
    V = torch.from_numpy(x["V_store"]).to(device())
    S, n = mp.map_similarity(V, norms_only=True)
    torch.cuda.synchronize()
    assert S is None
    np.testing.assert_allclose(n.cpu().numpy(), oracle.row_norms(x["V_f32"][0])[None], rtol=2e-6)


def test_peaked_predictor_llava_next_shape():
    """The LLaVA-NeXT shape with a peaked predictor: p_hat to 2e-2 (bf16)
    where the bar discriminates, and the selection replayed."""
    cfg = get_config("llava_next", pred=PredictorShape(weight_std=0.03))
    announce("peaked predictor at the LLaVA-NeXT shape")
    x = make_inputs(cfg)
    d = dev_inputs(x, device())
    out = _prune(x, d, cfg.K, cfg.K0, cfg.tau)
    p_ref = _p_ref(x)
    assert p_ref.max() / p_ref.min() > 10.0  # the signal spans more than the bar
    _check_structure(x, out, cfg.K, p_ref, 2e-2)
    _replay(x, out, cfg.K, cfg.K0, cfg.tau, [0])
