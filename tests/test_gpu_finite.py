"""The finite check (map_set_finite_check): with it on, a call whose float
inputs hold an infinity or a NaN returns MAP_ERR_NONFINITE before it
enqueues any work, and a call on finite inputs gives the same bits as with
the check off.  Inputs with non-finite values are only ever handed to calls
with the check on (which then run nothing but the scan)."""
import numpy as np
import pytest
import torch

import paper_2608_06411_amd as mp
from paper_2608_06411_amd.binding import MAP_ERR_NONFINITE
from workloads import PredictorShape, get_config, make_inputs

from gpu_util import announce, dev_inputs, device

pytestmark = pytest.mark.gpu


@pytest.fixture
def finite_check():
    mp.set_finite_check(True)
    try:
        yield
    finally:
        mp.set_finite_check(False)


def _small():
    cfg = get_config("sweep", B=2, N=300, M=(8, 20), K=32, K0=16, pred=PredictorShape(D=256, D_h=128, d_p=32))
    x = make_inputs(cfg)
    return cfg, x, dev_inputs(x, device())


def _prune(cfg, x, d, **over):
    a = dict(d, **over)
    return mp.map_prune(a["w"], a["V"], a["pos_v"], a["T"], a["pos_t"], x["t_off"], cfg.K, cfg.K0, cfg.tau)


def _expect_nonfinite(fn):
    with pytest.raises(mp.MapError) as e:
        fn()
    assert e.value.status == MAP_ERR_NONFINITE, e.value


def test_finite_inputs_give_the_same_bits(finite_check):
    announce("finite check on clean inputs")
    cfg, x, d = _small()
    on = _prune(cfg, x, d)
    torch.cuda.synchronize()
    mp.set_finite_check(False)
    off = _prune(cfg, x, d)
    torch.cuda.synchronize()
    for k in ("idx", "pos_out", "order"):
        assert torch.equal(on[k], off[k])
    assert torch.equal(on["V_out"].view(torch.int16), off["V_out"].view(torch.int16))
    assert torch.equal(on["p"], off["p"])


@pytest.mark.parametrize("where", ["V", "T", "w2_t", "b1_v"])
@pytest.mark.parametrize("value", [float("nan"), float("inf"), float("-inf")])
def test_prune_reports_a_non_finite_input(finite_check, where, value):
    announce(f"finite check: {value} in {where}")
    cfg, x, d = _small()
    if where in ("V", "T"):
        t = d[where].clone()
        t.view(-1)[t.numel() // 3] = value
        _expect_nonfinite(lambda: _prune(cfg, x, d, **{where: t}))
    else:
        w = d["w"]
        t = getattr(w, where).clone()
        t.view(-1)[t.numel() - 1] = value
        kw = {n: getattr(w, n) for n in ("w1_v", "b1_v", "w2_v", "b2_v", "w_k", "w1_t", "b1_t", "w2_t", "b2_t", "w_q")}
        kw[where] = t
        _expect_nonfinite(lambda: _prune(cfg, x, d, w=mp.PredictorWeights(**kw, rope_theta=w.rope_theta)))


def test_select_and_similarity_report_non_finite_inputs(finite_check):
    announce("finite check: select and similarity")
    dev = device()
    cfg, x, d = _small()
    S, n = mp.map_similarity(d["V"])
    p = torch.full((cfg.B, cfg.N), 1.0 / cfg.N, device=dev)
    torch.cuda.synchronize()
    S_bad = S.clone()
    S_bad[1, 7, 9] = float("nan")
    _expect_nonfinite(lambda: mp.map_select(p, S_bad, n, cfg.K, cfg.K0, cfg.tau))
    p_bad = p.clone()
    p_bad[0, 3] = float("inf")
    _expect_nonfinite(lambda: mp.map_select(p_bad, S, n, cfg.K, cfg.K0, cfg.tau))
    # a bf16 buffer that is not 4-byte aligned (a view one element in) is
    # scanned value by value
    big = torch.zeros(cfg.B * cfg.N * 256 + 1, dtype=torch.bfloat16, device=dev)
    V_view = big[1:].view(cfg.B, cfg.N, 256)
    V_view.copy_(d["V"])
    V_view[1, 299, 255] = float("nan")
    _expect_nonfinite(lambda: mp.map_similarity(V_view))


def test_decoder_reports_a_non_finite_weight(finite_check):
    announce("finite check: decoder layer")
    dev = device()
    d, H, ff, R = 256, 2, 512, 40
    rng = np.random.default_rng(1)
    mk = lambda *s: torch.from_numpy((0.02 * rng.standard_normal(s)).astype(np.float32)).to(dev).to(torch.bfloat16)
    ones = lambda n: torch.ones(n, dtype=torch.bfloat16, device=dev)
    wts = dict(attn_norm=ones(d), w_qkv=mk(3 * d, d), w_o=mk(d, d), ffn_norm=ones(d), w_gate_up=mk(2 * ff, d),
               w_down=mk(d, ff))
    X = mk(R, d)
    pos = torch.arange(R, dtype=torch.int32, device=dev)
    Y_ok = mp.map_decoder_layer(mp.DecoderWeights(**wts, n_heads=H), X, pos, [0, R])
    torch.cuda.synchronize()
    assert torch.isfinite(Y_ok.float()).all()
    wts["w_down"] = wts["w_down"].clone()
    wts["w_down"][5, 7] = float("inf")
    _expect_nonfinite(lambda: mp.map_decoder_layer(mp.DecoderWeights(**wts, n_heads=H), X, pos, [0, R]))
