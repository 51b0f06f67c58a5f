"""map_decoder_layer on the GPU against the decoder-layer oracle (float64),
on the same bf16 inputs and weights.

Bar.  The layer stores eight bf16 intermediates (the two RMSNorm outputs, q,
k and v, the attention output, the block residual, gate and up, their SwiGLU
product) and its output, each rounded to 2^-9 relative; the products sum
them in float32.  The layer's update Y - X must match the oracle's in the
relative Frobenius norm to 3e-2, and Y itself (dominated by the residual X)
to 1e-2; the cosine between the updates must exceed 0.999.  Cases: ragged
packed sequences at a small width (two heads), one sequence of the pruned
LLaVA-NeXT length (160 kept + 64 question tokens) at the 7B shape, and the
layer-0 input map_prune_assemble writes for a two-image batch.
"""
import numpy as np
import pytest
import torch

import oracle
from workloads import bf16_bits_to_f32, f32_to_bf16_bits

from gpu_util import announce, device

pytestmark = pytest.mark.gpu


def _weights(d, ff, seed, std=0.02):
    rng = np.random.default_rng(seed)
    shapes = {"attn_norm": (d,), "w_qkv": (3 * d, d), "w_o": (d, d), "ffn_norm": (d,), "w_gate_up": (2 * ff, d),
              "w_down": (d, ff)}
    out = {}
    for k, s in shapes.items():
        x = (1.0 + 0.1 * rng.standard_normal(s)) if "norm" in k else std * rng.standard_normal(s)
        out[k] = f32_to_bf16_bits(x.astype(np.float32))
    return out


def _dev(bits, dev):
    return torch.from_numpy(np.ascontiguousarray(bits).view(np.int16)).to(dev).view(torch.bfloat16)


def _run_and_check(X_bits, pos, seq_off, wb, n_heads, tag):
    import paper_2608_06411_amd as mp
    dev = device()
    d = X_bits.shape[1]
    w = mp.DecoderWeights(**{k: _dev(v, dev) for k, v in wb.items()}, n_heads=n_heads)
    Y = mp.map_decoder_layer(w, _dev(X_bits, dev), torch.from_numpy(np.asarray(pos, np.int32)).to(dev), seq_off)
    torch.cuda.synchronize()
    got = bf16_bits_to_f32(Y.view(torch.int16).cpu().numpy().view(np.uint16)).astype(np.float64)
    X = bf16_bits_to_f32(X_bits).astype(np.float64)
    want = oracle.decoder_layer(X, pos, seq_off, {k: bf16_bits_to_f32(v) for k, v in wb.items()}, n_heads)
    du, dw = got - X, want - X
    err_u = np.linalg.norm(du - dw) / np.linalg.norm(dw)
    err_y = np.linalg.norm(got - want) / np.linalg.norm(want)
    cos = float(np.sum(du * dw) / (np.linalg.norm(du) * np.linalg.norm(dw)))
    print(f"[decoder {tag}] update err {err_u:.2e}, output err {err_y:.2e}, cosine {cos:.6f}", flush=True)
    assert err_u <= 3e-2 and err_y <= 1e-2 and cos >= 0.999, (err_u, err_y, cos)
    return got


def test_decoder_small_ragged_sequences():
    d, H, ff = 256, 2, 512
    announce("decoder small ragged")
    rng = np.random.default_rng(3)
    seq_off = [0, 37, 140, 141, 300]          # one single-token sequence; blocks of 64 with tails
    R = seq_off[-1]
    X = f32_to_bf16_bits(rng.standard_normal((R, d)).astype(np.float32))
    pos = np.concatenate([np.sort(rng.choice(3000, seq_off[b + 1] - seq_off[b], replace=False))
                          for b in range(len(seq_off) - 1)]).astype(np.int32)
    _run_and_check(X, pos, seq_off, _weights(d, ff, 5, std=0.05), H, "small")


def test_decoder_7b_shape_pruned_length():
    """d 4096, 32 heads x 128, SwiGLU 11008: one sequence of 224 rows (the
    LLaVA-NeXT image pruned to 160 tokens, then a 64-token question)."""
    d, H, ff = 4096, 32, 11008
    announce("decoder 7B shape, 224 rows")
    rng = np.random.default_rng(4)
    X = f32_to_bf16_bits(rng.standard_normal((224, d)).astype(np.float32))
    pos = np.concatenate([np.sort(rng.choice(2880, 160, replace=False)), 2880 + np.arange(64)]).astype(np.int32)
    _run_and_check(X, pos, [0, 224], _weights(d, ff, 6), H, "7B 224")


def test_decoder_long_sequences_large_tiles():
    """Two sequences of 2944 and 1500 rows at d 1024 (8 heads), SwiGLU 2816:
    the QKV and gate/up products have enough tiles for the 256 x 256
    kernel (4444 rows: a ragged last tile row), the output and down
    products stay on 128 x 128 tiles."""
    d, H, ff = 1024, 8, 2816
    announce("decoder long sequences, 4444 rows at d 1024")
    rng = np.random.default_rng(8)
    seq_off = [0, 2944, 4444]
    X = f32_to_bf16_bits(rng.standard_normal((seq_off[-1], d)).astype(np.float32))
    pos = np.concatenate([np.arange(2944), np.arange(1500) * 2]).astype(np.int32)
    _run_and_check(X, pos, seq_off, _weights(d, ff, 9, std=0.03), H, "long")


def test_decoder_on_the_pruned_layer0_input():
    """map_prune_assemble's output for two images is the layer's input: the
    sequences are each image's kept rows then its question rows."""
    import paper_2608_06411_amd as mp
    from workloads import PredictorShape, get_config, make_inputs
    from gpu_util import dev_inputs
    cfg = get_config("sweep", B=2, N=600, M=(16, 40), K=64, K0=32, pred=PredictorShape(D=512, D_h=128, d_p=64))
    announce("decoder on map_prune_assemble's output")
    x = make_inputs(cfg)
    dev = device()
    di = dev_inputs(x, dev)
    f = mp.map_prune_assemble(di["w"], di["V"], di["pos_v"], di["T"], di["pos_t"], x["t_off"], cfg.K, cfg.K0, cfg.tau)
    torch.cuda.synchronize()
    seq_off = [b * cfg.K + int(x["t_off"][b]) for b in range(cfg.B + 1)]
    X_bits = f["X"].view(torch.int16).cpu().numpy().view(np.uint16)
    _run_and_check(X_bits, f["pos_x"].cpu().numpy(), seq_off, _weights(512, 768, 7, std=0.04), 4, "layer-0 input")
