"""map_train_step on the GPU against the training-step oracle (the KL
divergence from the teacher to p_hat and its chain-rule gradient, float64).

Bar.  p_hat as for map_score (1e-5 relative in float32, 2e-2 in bf16); each
image's loss to the same relative bound; each parameter's gradient in the
relative Frobenius norm, ||g - g_ref|| / ||g_ref||, within 1e-4 in float32
(float32 sums over up to a few thousand tokens, the erf approximation's
1.5e-7, and p_hat's own 1e-5) and 2e-2 in bf16, where the stored operands --
hidden states, GELU'(a), the gradients of the projections' inputs and of the
pre-activations, each rounded to bf16 (relative 2^-9) -- and the bf16 p_hat
(about 1e-3) chain through three products.  The teacher rows are Dirichlet(1)
draws, far from p_hat, so no cancellation in p* / p_hat - 1 magnifies those
errors.  The cosine between each GPU gradient and the oracle's must also
exceed 0.9995 (bf16) or 1 - 1e-8 (float32).
"""
import numpy as np
import pytest
import torch

import oracle
from workloads import PredictorShape, get_config, make_inputs

from gpu_util import announce, dev_inputs, device, oracle_weights

pytestmark = pytest.mark.gpu

NAMES = ("w1_v", "b1_v", "w2_v", "b2_v", "w_k", "w1_t", "b1_t", "w2_t", "b2_t", "w_q")


def _teacher(B, N, seed=5):
    rng = np.random.default_rng(seed)
    return rng.dirichlet(np.ones(N), size=B).astype(np.float32)


def _run(x, p_star):
    from paper_2608_06411_amd import map_train_step
    dev = device()
    d = dev_inputs(x, dev)
    loss, p, g = map_train_step(d["w"], d["V"], d["pos_v"], d["T"], d["pos_t"], x["t_off"],
                                torch.from_numpy(p_star).to(dev))
    torch.cuda.synchronize()
    return loss.cpu().numpy().astype(np.float64), p.cpu().numpy().astype(np.float64), \
        {k: v.cpu().numpy().astype(np.float64) for k, v in g.items()}


def _check(x, p_star, rtol_p, rtol_g, min_cos):
    cfg = x["cfg"]
    loss, p, g = _run(x, p_star)
    ref = oracle.train_step(x["V_f32"], x["T_f32"], x["t_off"], x["pos_v"], x["pos_t"], oracle_weights(x),
                            p_star.astype(np.float64), cfg.pred.rope_theta)
    np.testing.assert_allclose(p, ref.p_hat, rtol=rtol_p, atol=0)
    np.testing.assert_allclose(loss, ref.image_loss, rtol=rtol_p, atol=0)
    report = {}
    for k in NAMES:
        want = ref.grads[k]
        err = np.linalg.norm(g[k] - want) / np.linalg.norm(want)
        cos = float(np.sum(g[k] * want) / (np.linalg.norm(g[k]) * np.linalg.norm(want)))
        report[k] = (err, cos)
        assert err <= rtol_g, (k, err)
        assert cos >= min_cos, (k, cos)
    print("[train] " + ", ".join(f"{k} {e:.2e}" for k, (e, _) in report.items()), flush=True)
    return report


CASES = {
    "small_f32": ("sweep", {"B": 2, "N": 200, "M": (5, 40), "dtype": "f32",
                            "pred": PredictorShape(D=256, D_h=64, d_p=32)}, 1e-5, 1e-4, 1 - 1e-8),
    "small_bf16": ("sweep", {"B": 3, "N": 333, "M": (1, 70),
                             "pred": PredictorShape(D=512, D_h=136, d_p=64)}, 2e-2, 2e-2, 0.9995),
    "tiny_f32": ("tiny", {}, 1e-5, 1e-4, 1 - 1e-8),
}


@pytest.mark.parametrize("case", sorted(CASES))
def test_train_step_matches_oracle(case):
    name, over, rtol_p, rtol_g, min_cos = CASES[case]
    cfg = get_config(name, **over)
    announce(f"train {case}: B={cfg.B} N={cfg.N} M={cfg.M} {cfg.dtype} {cfg.pred}")
    x = make_inputs(cfg)
    _check(x, _teacher(cfg.B, cfg.N), rtol_p, rtol_g, min_cos)


def test_train_step_llava_next_full_size():
    """LLaVA-NeXT-7B's shape: 2880 visual tokens x 4096, a 64-token question,
    D_h = 1024, d_p = 128, bf16."""
    cfg = get_config("llava_next")
    announce("train llava_next full size")
    x = make_inputs(cfg)
    _check(x, _teacher(cfg.B, cfg.N, seed=9), 2e-2, 2e-2, 0.9995)


def test_train_step_teacher_from_map_teacher():
    """The teacher the paper distils: map_teacher's QCTS distribution from
    synthetic attention over the same 576 visual tokens, then one step."""
    import paper_2608_06411_amd as mp
    from workloads import make_attention
    cfg = get_config("sweep", B=1, N=576, M=(24, 24), dtype="f32", pred=PredictorShape(D=256, D_h=64, d_p=32))
    announce("train with map_teacher's teacher")
    x = make_inputs(cfg)
    dev = device()
    A_f, A_s = make_attention(8, 4, 24, 576, dtype="f32", seed=3)
    R_f, R_s = make_attention(8, 4, 6, 576, dtype="f32", seed=3, reference=True)
    t = mp.map_teacher(torch.from_numpy(A_s.reshape(-1)).to(dev), torch.from_numpy(R_s.reshape(-1)).to(dev),
                       [0, 24], 8, 4, 576, 6, n_top=1)
    torch.cuda.synchronize()
    p_star = t["teacher"].cpu().numpy()
    _check(x, p_star, 1e-5, 1e-4, 1 - 1e-8)


def test_train_step_is_deterministic():
    cfg = get_config("sweep", B=2, N=300, M=(8, 20), pred=PredictorShape(D=256, D_h=64, d_p=32))
    x = make_inputs(cfg)
    p_star = _teacher(cfg.B, cfg.N)
    a, b = _run(x, p_star), _run(x, p_star)
    np.testing.assert_array_equal(a[0], b[0])
    np.testing.assert_array_equal(a[1], b[1])
    for k in NAMES:
        np.testing.assert_array_equal(a[2][k], b[2][k])


def test_train_step_rejects_bad_arguments():
    from paper_2608_06411_amd import map_train_step
    cfg = get_config("sweep", B=1, N=64, M=(4, 4), pred=PredictorShape(D=64, D_h=32, d_p=12))
    x = make_inputs(cfg)
    d = dev_inputs(x, device())
    with pytest.raises(Exception):   # d_p % 8 != 0: refused before any launch
        map_train_step(d["w"], d["V"], d["pos_v"], d["T"], d["pos_t"], x["t_off"],
                       torch.full((1, 64), 1 / 64, device=d["V"].device))
    with pytest.raises(ValueError):  # a teacher of the wrong shape
        map_train_step(d["w"], d["V"], d["pos_v"], d["T"], d["pos_t"], x["t_off"],
                       torch.full((1, 63), 1 / 63, device=d["V"].device))
