"""The seeded generators: determinism, bf16 rounding, duplicates, layout."""
import numpy as np

from workloads import bf16_bits_to_f32, f32_to_bf16_bits, get_config, make_inputs, peaked_scores


def test_bf16_round_to_nearest_even():
    x = np.array([1.0, 1.0 + 2.0 ** -8, 1.0 + 3 * 2.0 ** -8, -2.5, 1.0 + 2.0 ** -7], np.float32)
    bits = f32_to_bf16_bits(x)
    np.testing.assert_array_equal(bits, [0x3F80, 0x3F80, 0x3F82, 0xC020, 0x3F81])
    np.testing.assert_array_equal(bf16_bits_to_f32(bits)[[0, 3, 4]], [1.0, -2.5, 1.0 + 2.0 ** -7])


def test_deterministic_and_duplicates_exact():
    cfg = get_config("tiny", N=96, pred=get_config("tiny").pred.__class__(D=64, D_h=32, d_p=8))
    a, b = make_inputs(cfg), make_inputs(cfg)
    np.testing.assert_array_equal(a["V_store"], b["V_store"])
    np.testing.assert_array_equal(a["w1_v_store"], b["w1_v_store"])
    V = a["V_f32"][0]
    uniq = np.unique(V, axis=0).shape[0]
    assert uniq == 96 - int(np.floor(0.08 * 96))


def test_bf16_workload_layout_and_ragged_questions():
    from workloads import PredictorShape
    cfg = get_config("sweep", B=4, N=64, pred=PredictorShape(D=32, D_h=16, d_p=8))
    x = make_inputs(cfg)
    assert x["V_store"].dtype == np.uint16 and x["V_store"].shape == (4, 64, 32)
    np.testing.assert_array_equal(bf16_bits_to_f32(x["V_store"]), x["V_f32"])
    t_off = x["t_off"]
    assert t_off[0] == 0 and np.all(np.diff(t_off) >= 16) and np.all(np.diff(t_off) <= 128)
    assert x["T_store"].shape[0] == t_off[-1] == x["pos_t"].shape[0]
    np.testing.assert_array_equal(x["pos_t"][t_off[1]:t_off[2]], 64 + np.arange(t_off[2] - t_off[1]))


def test_multiframe_copies():
    from workloads import PredictorShape
    cfg = get_config("multiframe", B=1, N=8 * 40, pred=PredictorShape(D=16, D_h=8, d_p=4))
    V = make_inputs(cfg, with_weights=False)["V_f32"][0].reshape(8, 40, 16)
    same = np.all(V[1:] == V[:-1], axis=2)            # exact copies frame to frame
    np.testing.assert_array_equal(same.sum(axis=1), 40 - 28)


def test_peaked_scores_distribution():
    p = peaked_scores(3, 500)
    np.testing.assert_allclose(p.sum(axis=1), 1.0, rtol=1e-5)
    assert np.all(p > 0) and p.max() > 20.0 / 500
