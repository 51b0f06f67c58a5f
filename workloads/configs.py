"""Workload definitions, shaped like the paper's settings.

Shapes follow the paper's evaluation backbones: 576 visual tokens per image
tile (LLaVA-1.5), 2880 = 5 x 576 for LLaVA-NeXT, 4096-wide LLM embeddings,
and the retention budgets of Tables 1-3 (64..640 kept tokens, 160 of 2880 =
5.56% as the headline).  The predictor's width is not given by the paper; the
reading used here (two-layer GELU MLPs of width 1024, a single 128-wide
query/key head, RoPE base 10^4) is stated with each field.
"""
from dataclasses import dataclass, field, replace
from typing import Optional, Tuple


@dataclass(frozen=True)
class PredictorShape:
    D: int = 4096          # LLM embedding width (feature width of v_n, t_m)
    D_h: int = 1024        # hidden width of f_V / f_T (unspecified by the paper)
    d_p: int = 128         # projection width d of W_Q / W_K in Eq. (3)
    rope_theta: float = 10000.0
    weight_std: float = 0.02


@dataclass(frozen=True)
class Workload:
    name: str
    B: int                      # images per call
    N: int                      # visual tokens per image
    M: Tuple[int, int]          # question length range [lo, hi] (lo == hi: fixed)
    K: int                      # tokens kept per image
    K0: int                     # size of the top-K0 initial retained set
    dtype: str                  # "f32" or "bf16" storage of V, T and weights
    clusters: int               # Gaussian-mixture components for V
    sigma: float = 0.3          # within-cluster standard deviation
    dup_frac: float = 0.0       # fraction of tokens overwritten by exact copies
    frames: int = 1             # temporally correlated frames (N = frames * tokens/frame)
    frame_noise: float = 0.1    # per-step noise std for moved tokens
    frame_move_frac: float = 0.7  # fraction of tokens that move between frames
    seed: int = 0
    tau: float = 1e-2           # rank-deficiency threshold on the unit residual
    pred: PredictorShape = field(default_factory=PredictorShape)

    def with_(self, **kw) -> "Workload":
        return replace(self, **kw)


CONFIGS = {
    # Tiny single image in fp32; the oracle finishes in seconds.
    "tiny": Workload("tiny", B=1, N=576, M=(32, 32), K=64, K0=32, dtype="f32",
                     clusters=64, dup_frac=0.08, seed=1),
    # LLaVA-NeXT-7B shape: 2880 visual tokens, 4096 wide, keep 160 (5.56%).
    "llava_next": Workload("llava_next", B=1, N=2880, M=(64, 64), K=160, K0=80,
                           dtype="bf16", clusters=256, dup_frac=0.08, seed=2),
    # Batched retention sweep; K is varied per run (64, 160, 320, 640).
    "sweep": Workload("sweep", B=16, N=2880, M=(16, 128), K=160, K0=80,
                      dtype="bf16", clusters=256, dup_frac=0.05, seed=3),
    # Multi-frame / high-res: 8 frames x 576 tokens, 3584 wide.
    "multiframe": Workload("multiframe", B=8, N=4608, M=(96, 96), K=256, K0=128,
                           dtype="bf16", clusters=512, dup_frac=0.0, frames=8,
                           seed=4, pred=PredictorShape(D=3584)),
}

SWEEP_K = (64, 160, 320, 640)


def get_config(name: str, **overrides) -> Workload:
    cfg = CONFIGS[name]
    if overrides:
        cfg = cfg.with_(**overrides)
    return cfg
