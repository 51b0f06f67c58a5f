"""map_teacher on the GPU against the teacher-selection oracle (Eq. (1)-(2),
QCTS-n), on seeded synthetic attention.

Tolerances.  The GPU sums non-negative float32 values; along the deepest
chain a column sum adds ceil(H M / (4 S)) rows in one thread, then four
waves, then S slices, so with d that depth its relative error is at most
d * 2^-24, and p = a / sum(a) at most twice that plus the float32 rounding of
the output: rtol_p = (2 d + 1) * 2^-24.  D_JS changes by at most
rtol_p * (sum of p |log(p/m)| + q |log(q/m)|) <= rtol_p * 2 ln 2 + float64
rounding, so atol_js = 2 rtol_p.  The ranked layers must match the oracle's
except where two of the oracle's divergences lie within 2 atol_js of each
other; there the GPU's choice must still be one of them.
"""
import math

import numpy as np
import pytest
import torch

import oracle
from workloads import make_attention

from gpu_util import announce, device

pytestmark = pytest.mark.gpu


def _slices(B, L, N):
    wgs = 2 * B * L * ((N + 511) // 512)
    return min(16, max(1, -(-4096 // wgs)))


def _case(dtype, L, H, Ms, M_ref, N, zero_layer=None, same_layers=()):
    A_f, A_s, R_f, R_s = [], [], [], []
    for b, M in enumerate(Ms):
        af, a_s = make_attention(L, H, M, N, dtype=dtype, seed=40 + b, question=b)
        rf, r_s = make_attention(L, H, M_ref, N, dtype=dtype, seed=40 + b, reference=True)
        if zero_layer is not None:
            for x in (af, a_s, rf, r_s):
                x[zero_layer] = 0
        for l in same_layers:  # the reference question attends exactly like the question
            rf[l], r_s[l] = af[l], a_s[l]
        A_f.append(af), A_s.append(a_s), R_f.append(rf), R_s.append(r_s)
    return A_f, A_s, R_f, R_s


def _dev(stores, dtype, dev):
    flat = np.concatenate([s.reshape(-1) for s in stores])
    if dtype == "bf16":
        return torch.from_numpy(flat.view(np.int16)).to(dev).view(torch.bfloat16)
    return torch.from_numpy(np.ascontiguousarray(flat, dtype=np.float32)).to(dev)


def _run_and_check(dtype, L, H, Ms, M_ref, N, n_top, zero_layer=None, same_layers=()):
    from paper_2608_06411_amd import map_teacher
    announce(f"teacher {dtype} L={L} H={H} M={Ms} M_ref={M_ref} N={N} n_top={n_top}")
    A_f, A_s, R_f, R_s = _case(dtype, L, H, Ms, M_ref, N, zero_layer, same_layers)
    dev = device()
    m_off = np.concatenate([[0], np.cumsum(Ms)]).astype(np.int32)
    out = map_teacher(_dev(A_s, dtype, dev), _dev(R_s, dtype, dev), m_off, L, H, N, M_ref, n_top)
    torch.cuda.synchronize()
    got = {k: v.cpu().numpy() for k, v in out.items() if not k.startswith("_")}
    S = _slices(len(Ms), L, N)
    for b, M in enumerate(Ms):
        depth = max(-(-H * M // (4 * S)), -(-H * M_ref // (4 * S))) + 4 + S
        rtol = (2 * depth + 1) * 2.0 ** -24
        atol_js = 2 * rtol + 1e-12
        want = oracle.teacher_selection(A_f[b], R_f[b], n_top)
        np.testing.assert_allclose(got["p"][b], want.p, rtol=rtol, atol=0)
        np.testing.assert_allclose(got["p_ref"][b], want.p_ref, rtol=rtol, atol=0)
        np.testing.assert_allclose(got["js"][b], want.js, rtol=0, atol=atol_js)
        layers = got["layers"][b]
        ranked = sorted(range(L), key=lambda l: (-want.js[l], l))
        for k in range(n_top):
            if layers[k] != ranked[k]:
                assert abs(want.js[layers[k]] - want.js[ranked[k]]) <= 2 * atol_js, (b, k, layers, ranked)
        assert len(set(layers.tolist())) == n_top
        # the teacher is the mean of the chosen layers' distributions
        np.testing.assert_allclose(got["teacher"][b], want.p[layers].mean(axis=0), rtol=rtol, atol=0)
        np.testing.assert_allclose(got["teacher"][b].sum(), 1.0, rtol=1e-5)
    return got


@pytest.mark.parametrize("dtype,L,H,Ms,M_ref,N,n_top", [
    ("bf16", 6, 3, (5, 17), 4, 584, 3),      # two samples, ragged questions, a ragged column block
    ("f32", 5, 2, (7,), 3, 260, 1),
    ("bf16", 1, 1, (1, 2, 1), 1, 8, 1),      # one layer, one head, one-token questions, N = 8
    ("bf16", 7, 2, (9,), 5, 1024, 7),        # every layer in the teacher (QCTS-L)
    ("f32", 12, 4, (33, 2), 8, 4100, 4),
])
def test_teacher_matches_oracle(dtype, L, H, Ms, M_ref, N, n_top):
    _run_and_check(dtype, L, H, Ms, M_ref, N, n_top)


def test_teacher_zero_layer_is_uniform():
    got = _run_and_check("bf16", 8, 2, (3,), 2, 64, 2, zero_layer=2)
    np.testing.assert_array_equal(got["p"][0][2], np.full(64, np.float32(1 / 64)))
    assert got["js"][0][2] == 0.0


def test_teacher_identical_layers_tie_at_zero():
    """Two layers whose question and reference attention are identical have
    D_JS = 0 exactly on both sides; they rank last, the lower layer first
    (Eq. (2) with ties to the lower layer), after every positive divergence."""
    got = _run_and_check("bf16", 8, 2, (4,), 4, 256, 8, same_layers=(2, 5))
    assert got["js"][0][2] == 0.0 and got["js"][0][5] == 0.0
    assert got["layers"][0][-2:].tolist() == [2, 5]


def test_teacher_is_deterministic():
    from paper_2608_06411_amd import map_teacher
    announce("teacher determinism")
    dev = device()
    A_f, A_s, R_f, R_s = _case("bf16", 8, 4, (20,), 6, 576)
    A, R = _dev(A_s, "bf16", dev), _dev(R_s, "bf16", dev)
    o1 = {k: v.clone() for k, v in map_teacher(A, R, [0, 20], 8, 4, 576, 6, 2).items() if not k.startswith("_")}
    o2 = map_teacher(A, R, [0, 20], 8, 4, 576, 6, 2)
    for k, v in o1.items():
        assert torch.equal(v, o2[k]), k


def test_teacher_llava_next_full_size():
    """LLaVA-NeXT-7B's shape: 32 layers x 32 heads, 2880 visual tokens, a
    64-token question and an 8-token reference question, bf16 attention."""
    got = _run_and_check("bf16", 32, 32, (64,), 8, 2880, 4)
    print(f"[teacher llava_next] layers {got['layers'][0].tolist()} js {np.round(got['js'][0], 4).tolist()}")


def test_teacher_rejects_bad_arguments():
    from paper_2608_06411_amd import MapError, map_teacher
    dev = device()
    A = torch.zeros(2 * 2 * 3 * 12, dtype=torch.bfloat16, device=dev)   # N = 12: 24 bytes per row
    R = torch.zeros(2 * 2 * 1 * 12, dtype=torch.bfloat16, device=dev)
    with pytest.raises(MapError):
        map_teacher(A, R, [0, 3], 2, 2, 12, 1, 1)
    A = torch.zeros(2 * 2 * 3 * 16, dtype=torch.bfloat16, device=dev)
    R = torch.zeros(2 * 2 * 1 * 16, dtype=torch.bfloat16, device=dev)
    with pytest.raises((MapError, ValueError)):  # the binding refuses it before the library does
        map_teacher(A, R, [0, 3], 2, 2, 16, 1, 3)      # n_top > L
