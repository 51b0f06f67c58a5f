"""map_select on the GPU, replayed decision by decision against the oracle.

The GPU's own selection order is replayed on the oracle (float64, explicit
Gram-Schmidt on the raw embeddings, with the same p): every pick must be the
oracle's argmax given the GPU's prefix, except where the oracle's decisive
gap is below 1e-4 relative; the GPU's recorded gains must match the oracle's
scores to 1e-3 relative (float32 recurrence on a float32 cosine matrix)."""
import numpy as np
import pytest
import torch

import oracle
from workloads import bf16_bits_to_f32, f32_to_bf16_bits, peaked_scores

from gpu_util import announce, device, to_dev

pytestmark = pytest.mark.gpu

TAU = 1e-2


def _tokens(seed, B, N, D, dtype, dup=0.08, zero_rows=0, clusters=None):
    rng = np.random.default_rng(seed)
    C = clusters or max(2, N // 8)
    V = np.empty((B, N, D), np.float32)
    for b in range(B):
        cen = rng.standard_normal((C, D)).astype(np.float32)
        V[b] = cen[rng.integers(0, C, N)] + 0.3 * rng.standard_normal((N, D)).astype(np.float32)
        nd = int(dup * N)
        if nd:
            slots = rng.choice(N, nd, replace=False)
            keep = np.setdiff1d(np.arange(N), slots)
            V[b, slots] = V[b, keep[rng.integers(0, keep.size, nd)]]
        if zero_rows:
            V[b, rng.choice(N, zero_rows, replace=False)] = 0.0
    if dtype == "bf16":
        bits = f32_to_bf16_bits(V)
        return bf16_bits_to_f32(bits), bits
    return V, V


def _select(store, dtype, p, K, K0):
    from paper_2608_06411_amd import map_select, map_similarity
    dev = device()
    S, n = map_similarity(to_dev(store, dtype, dev))
    pt = torch.from_numpy(np.ascontiguousarray(p, np.float32)).to(dev)
    idx, order, gain = map_select(pt, S, n, K, K0, TAU)
    torch.cuda.synchronize()
    return idx.cpu().numpy(), order.cpu().numpy(), gain.cpu().numpy()


def _check(V, p, K, K0, idx, order, gain):
    for b in range(V.shape[0]):
        rep = oracle.replay_check(p[b].astype(np.float64), V[b], K, K0, TAU, order[b], gain[b])
        assert rep.ok, f"image {b}: {rep.failure}"
        assert rep.max_gain_rel_err < 1e-3, rep.max_gain_rel_err
        np.testing.assert_array_equal(idx[b], np.sort(order[b]))
        if K0 > 0:
            np.testing.assert_array_equal(gain[b][:K0], p[b][order[b][:K0]])


CASES = [
    # B, N, D, K, K0, dtype, scores, extra
    (1, 300, 64, 40, 20, "f32", "peaked", {}),
    (1, 300, 64, 40, 0, "f32", "peaked", {}),
    (1, 300, 64, 40, 40, "bf16", "peaked", {}),
    (2, 1000, 256, 160, 80, "bf16", "peaked", {}),
    (1, 1000, 256, 160, 80, "bf16", "flat", {}),
    (3, 257, 128, 100, 30, "f32", "flat", {"zero_rows": 5}),
    (1, 50, 8, 20, 5, "f32", "peaked", {}),            # D < K: rank runs out
    (1, 64, 32, 64, 10, "f32", "flat", {}),            # K = N
    (1, 17, 16, 1, 0, "f32", "peaked", {}),            # K = 1
    (1, 1, 16, 1, 1, "bf16", "flat", {}),              # N = 1
    (1, 600, 128, 500, 50, "bf16", "flat", {}),        # large K: small pool, many rounds
    (1, 5000, 64, 64, 32, "bf16", "peaked", {}),       # many workgroups per image
    (1, 9000, 64, 150, 100, "bf16", "flat", {}),       # more than 64 own tokens per workgroup
    (1, 2000, 256, 300, 200, "bf16", "peaked", {}),    # K0 beyond the one-pass R0: pool rounds
    (1, 1500, 64, 200, 128, "bf16", "peaked", {}),     # the largest one-pass R0 (eight pivot blocks)
]


@pytest.mark.parametrize("case", range(len(CASES)))
def test_select_replays_on_oracle(case):
    B, N, D, K, K0, dtype, scores, extra = CASES[case]
    announce(f"select B={B} N={N} D={D} K={K} K0={K0} {dtype} {scores} {extra}")
    V, store = _tokens(case, B, N, D, dtype, **extra)
    if scores == "peaked":
        p = peaked_scores(B, N, seed=case)
    else:
        rng = np.random.default_rng(100 + case)
        p = (1.0 + 0.05 * rng.standard_normal((B, N))).astype(np.float32)
        p /= p.sum(axis=1, keepdims=True)
    idx, order, gain = _select(store, dtype, p, K, K0)
    _check(V, p, K, K0, idx, order, gain)


def test_select_top_k_mode_is_exact():
    """K0 = K: the kept set is exactly the top K of p (ties to the lower index)."""
    V, store = _tokens(7, 1, 400, 32, "f32")
    p = peaked_scores(1, 400, seed=3)
    p[0, 10] = p[0, 11] = p[0].max()                  # an exact tie
    idx, order, _ = _select(store, "f32", p, 50, 50)
    want = np.lexsort((np.arange(400), -p[0].astype(np.float64)))[:50]
    np.testing.assert_array_equal(order[0], want)
    np.testing.assert_array_equal(idx[0], np.sort(want))


def test_select_is_deterministic():
    V, store = _tokens(8, 2, 900, 128, "bf16")
    p = peaked_scores(2, 900, seed=4)
    a = _select(store, "bf16", p, 120, 60)
    b = _select(store, "bf16", p, 120, 60)
    for x, y in zip(a, b):
        np.testing.assert_array_equal(x, y)


def test_select_r0_candidate_overflow():
    """p arranged so that very many keys reach the threads' K0-th largest
    maximum (token i is seen by thread i mod 256): R0 falls back to pool
    rounds and must still be the top K0 of p, placed in order."""
    N, K, K0 = 2560, 160, 128
    V, store = _tokens(11, 1, N, 64, "f32")
    i = np.arange(N)
    p = (1.0 + 1e-3 * (i % 256) + 1e-6 * (i // 256))[None, :]
    p = (p / p.sum()).astype(np.float32)
    idx, order, gain = _select(store, "f32", p, K, K0)
    want = np.lexsort((i, -p[0].astype(np.float64)))[:K0]
    np.testing.assert_array_equal(order[0][:K0], want)
    _check(V, p, K, K0, idx, order, gain)
