"""map_similarity on the GPU against the oracle's float64 cosine matrix.

Tolerance: inputs are exact in both dtypes and every product is exact in
float32, so the only error is float32 accumulation over D terms of size up to
|v_i||v_j|/D; for D <= 4096 that stays far below 1e-5 in a cosine."""
import numpy as np
import pytest
import torch

from oracle import cosine_similarity, row_norms
from workloads import bf16_bits_to_f32, f32_to_bf16_bits

from gpu_util import announce, device

pytestmark = pytest.mark.gpu


def _tokens(seed, B, N, D, dtype):
    rng = np.random.default_rng(seed)
    V = rng.standard_normal((B, N, D)).astype(np.float32)
    V[:, 1::7] = V[:, 0:1]               # exact duplicates
    if N > 3:
        V[:, 3] = 0.0                    # a zero row
    if dtype == "bf16":
        bits = f32_to_bf16_bits(V)
        return bf16_bits_to_f32(bits), bits
    return V, V


@pytest.mark.parametrize("dtype,B,N,D", [
    ("f32", 1, 576, 256), ("bf16", 2, 300, 512), ("bf16", 1, 1, 64), ("f32", 1, 130, 4096),
    ("bf16", 1, 257, 4096), ("bf16", 3, 129, 3584),
    # enough tiles for the 256 x 256 kernel (its last tile row and column
    # partial): the cosine epilogue's sub-tiles and their mirrors
    ("bf16", 2, 4500, 3584),
])
def test_similarity_matches_oracle(dtype, B, N, D):
    from paper_2608_06411_amd import map_similarity
    from gpu_util import to_dev
    dev = device()
    announce(f"similarity {dtype} B={B} N={N} D={D}")
    V, store = _tokens(B * 1000 + N, B, N, D, dtype)
    S, n = map_similarity(to_dev(store, dtype, dev))
    torch.cuda.synchronize()
    S, n = S.cpu().numpy(), n.cpu().numpy()
    for b in range(B):
        want = cosine_similarity(V[b])
        np.testing.assert_allclose(S[b], want, rtol=0, atol=1e-5)
        np.testing.assert_allclose(n[b], row_norms(V[b]), rtol=2e-6, atol=0)
        np.testing.assert_array_equal(S[b], S[b].T)       # mirrored tiles are bitwise symmetric
