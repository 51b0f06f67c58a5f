"""Seeded synthetic inputs: visual tokens, question tokens, positions and
predictor weights.

Recipe (one ``SeedSequence([seed, tag])`` stream per tensor):

* Visual tokens of one image: ``clusters`` centres c_j ~ N(0, I_D); each token
  picks a centre uniformly and adds sigma * N(0, I_D).  A fraction
  ``dup_frac`` of the slots (distinct, uniform) is then overwritten by exact
  copies of uniformly chosen non-overwritten slots, so the selection sees
  rank-deficient, redundant inputs.
* Multi-frame images: frame 0 is drawn as above; each later frame copies the
  previous one and adds N(0, frame_noise^2) noise to a random
  ``frame_move_frac`` of its slots (the rest are exact copies).
* Question tokens: N(0, 1), with per-image lengths uniform in [M_lo, M_hi],
  packed back to back (offsets ``t_off``).
* Positions: visual token n of an image sits at position n, question token m
  at N + m (the question follows the image in the LLM input).
* Predictor weights and biases: N(0, weight_std^2), drawn from a stream keyed
  by the predictor shape, so workloads of equal width share weights.
* bf16 workloads round every tensor to bf16 (round to nearest even) after the
  duplicates are made, so copies stay bit-identical.

Every array is returned twice: ``*_f32`` holds the exact stored values as
float32 (bf16 values are exactly representable), ``*_store`` the stored
representation (float32, or the bf16 bit patterns as uint16).
"""
import numpy as np

from .configs import PredictorShape, Workload

_TAG_V, _TAG_T, _TAG_M, _TAG_W = 11, 12, 13, 14


def f32_to_bf16_bits(x: np.ndarray) -> np.ndarray:
    """Round float32 values to bf16 (nearest, ties to even); return the bits."""
    u = np.ascontiguousarray(x, dtype=np.float32).view(np.uint32)
    bias = ((u >> 16) & np.uint32(1)) + np.uint32(0x7FFF)
    return ((u + bias) >> 16).astype(np.uint16)


def bf16_bits_to_f32(b: np.ndarray) -> np.ndarray:
    return (np.ascontiguousarray(b, dtype=np.uint16).astype(np.uint32) << 16).view(np.float32)


def _rng(seed: int, *tag: int) -> np.random.Generator:
    return np.random.Generator(np.random.PCG64(np.random.SeedSequence([seed, *tag])))


def _store(x: np.ndarray, dtype: str):
    if dtype == "bf16":
        bits = f32_to_bf16_bits(x)
        return bf16_bits_to_f32(bits), bits
    if dtype == "f32":
        x = np.ascontiguousarray(x, dtype=np.float32)
        return x, x
    raise ValueError(f"unknown dtype {dtype!r}")


def _mixture(rng, n, D, clusters, sigma, dup_frac):
    centres = rng.standard_normal((clusters, D), dtype=np.float32)
    assign = rng.integers(0, clusters, size=n)
    v = centres[assign] + np.float32(sigma) * rng.standard_normal((n, D), dtype=np.float32)
    n_dup = int(np.floor(dup_frac * n))
    if n_dup > 0:
        slots = rng.choice(n, size=n_dup, replace=False)
        keep = np.setdiff1d(np.arange(n), slots)
        src = keep[rng.integers(0, keep.size, size=n_dup)]
        v[slots] = v[src]
    return v


def make_visual_tokens(cfg: Workload, image: int) -> np.ndarray:
    """float32 visual tokens [N, D] of one image (before storage rounding)."""
    D = cfg.pred.D
    rng = _rng(cfg.seed, _TAG_V, image)
    if cfg.frames <= 1:
        return _mixture(rng, cfg.N, D, cfg.clusters, cfg.sigma, cfg.dup_frac)
    if cfg.N % cfg.frames:
        raise ValueError("N must be a multiple of frames")
    per = cfg.N // cfg.frames
    frames = [_mixture(rng, per, D, cfg.clusters, cfg.sigma, cfg.dup_frac)]
    n_move = int(round(cfg.frame_move_frac * per))
    for _ in range(1, cfg.frames):
        nxt = frames[-1].copy()
        moved = rng.choice(per, size=n_move, replace=False)
        nxt[moved] += np.float32(cfg.frame_noise) * rng.standard_normal((n_move, D), dtype=np.float32)
        frames.append(nxt)
    return np.concatenate(frames, axis=0)


def make_weights(pred: PredictorShape, dtype: str, seed: int = 1234) -> dict:
    """Predictor parameters in torch.nn.Linear layout (W[out][in])."""
    D, H, dp = pred.D, pred.D_h, pred.d_p
    shapes = {
        "w1_v": (H, D), "b1_v": (H,), "w2_v": (H, H), "b2_v": (H,), "w_k": (dp, H),
        "w1_t": (H, D), "b1_t": (H,), "w2_t": (H, H), "b2_t": (H,), "w_q": (dp, H),
    }
    out = {}
    for i, (name, shp) in enumerate(shapes.items()):
        rng = _rng(seed, _TAG_W, D, H, dp, i)
        w = np.float32(pred.weight_std) * rng.standard_normal(shp, dtype=np.float32)
        out[name + "_f32"], out[name + "_store"] = _store(w, dtype)
    return out


def make_inputs(cfg: Workload, *, with_weights: bool = True) -> dict:
    """All inputs of one call on workload ``cfg`` (see the module docstring)."""
    B, N, D = cfg.B, cfg.N, cfg.pred.D
    V = np.empty((B, N, D), dtype=np.float32)
    for b in range(B):
        V[b] = make_visual_tokens(cfg, b)
    lo, hi = cfg.M
    M = _rng(cfg.seed, _TAG_M).integers(lo, hi + 1, size=B) if hi > lo else np.full(B, lo)
    t_off = np.zeros(B + 1, dtype=np.int32)
    t_off[1:] = np.cumsum(M)
    T = _rng(cfg.seed, _TAG_T).standard_normal((int(t_off[-1]), D), dtype=np.float32)
    pos_v = np.broadcast_to(np.arange(N, dtype=np.int32), (B, N)).copy()
    pos_t = np.concatenate([N + np.arange(m, dtype=np.int32) for m in M]) if B else \
        np.zeros(0, np.int32)
    out = {"cfg": cfg, "t_off": t_off, "pos_v": pos_v, "pos_t": pos_t.astype(np.int32)}
    out["V_f32"], out["V_store"] = _store(V, cfg.dtype)
    out["T_f32"], out["T_store"] = _store(T, cfg.dtype)
    if with_weights:
        out.update(make_weights(cfg.pred, cfg.dtype))
    return out


def peaked_scores(B: int, N: int, alpha: float = 0.1, seed: int = 7) -> np.ndarray:
    """Importance distributions with large gaps: Dirichlet(alpha) per image,
    floored away from zero and renormalised, as float32 [B, N]."""
    rng = _rng(seed, 21, B, N)
    p = rng.dirichlet(np.full(N, alpha), size=B)
    p = np.maximum(p, 1e-12)
    p /= p.sum(axis=1, keepdims=True)
    return p.astype(np.float32)


_TAG_A = 15


def make_attention(L: int, H: int, M: int, N: int, *, dtype: str = "bf16", seed: int = 21, question: int = 0,
                   reference: bool = False, share: float = 0.5, focus_peak: float = 2.5, noise: float = 0.7):
    """Synthetic text-to-vision attention A [L][H][M][N] of one sample.

    Each row is a softmax over the N visual tokens scaled by ``share`` (the
    rest of the row's mass sits on the other tokens of the sequence).  Its
    logits are a per-layer image field g_l[n] ~ N(0, 1) shared by every
    question on the image, plus, for the input question (``reference`` False),
    beta_l * f[n] with a question field f ~ N(0, 1) keyed by ``question`` and
    a weight beta_l that peaks at ``focus_peak`` in the middle layers, plus
    per-(head, token) noise N(0, noise^2).  Returns (float32 values, stored
    array), stored as float32 or bf16 bit patterns.
    """
    g = _rng(seed, _TAG_A, 0).standard_normal((L, 1, 1, N)).astype(np.float32)
    z = g + noise * _rng(seed, _TAG_A, 1, question, int(reference)).standard_normal((L, H, M, N), dtype=np.float32)
    if not reference:
        f = _rng(seed, _TAG_A, 2, question).standard_normal(N).astype(np.float32)
        x = (np.arange(L, dtype=np.float32) + 0.5) / L
        beta = focus_peak * np.exp(-((x - 0.45) / 0.2) ** 2) * (1.0 + 0.3 * _rng(seed, _TAG_A, 3, question).random(L))
        z += beta.astype(np.float32)[:, None, None, None] * f[None, None, None, :]
    z -= z.max(axis=3, keepdims=True)
    np.exp(z, out=z)
    z *= np.float32(share) / z.sum(axis=3, keepdims=True)
    return _store(z, dtype)
