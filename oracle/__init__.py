"""CPU oracle for the MAP pruning hot path -- TEST INFRASTRUCTURE ONLY.

A plain, slow float64 implementation of what the paper's inference-time
pruning computes, written from the paper ("Learning to Predict Middle-Layer
Attention in MLLMs for Visual Token Pruning"):

* ``predictor``  -- the predicted attention p_hat of Eq. (3)
                    (section "Cross-Modal Attention Distillation");
* ``similarity`` -- row norms and the cosine similarity of the visual tokens;
* ``select``     -- top-K0 initial set, orthonormal basis, the greedy rule of
                    Eq. (4) and the restoration of the original order
                    (section "Inference-Time Token Pruning"), plus a replay
                    checker for another implementation's selection order;
* ``pipeline``   -- the three chained, with the gather of the kept tokens,
                    and the language model's layer-0 input after pruning;
* ``teacher``    -- teacher selection for predictor training: Eq. (1),
                    Eq. (2) and QCTS-n (section "Question Contrastive
                    Teacher Selection");
* ``decoder``    -- the language model's first layer (LLaMA decoder layer:
                    RMSNorm, RoPE attention with a causal mask, SwiGLU)
                    over the pruned input, the consumer of the pruning stage
                    (section "Inference-Time Token Pruning");
* ``train``      -- one predictor training step: the KL divergence from the
                    teacher distribution to p_hat and its gradient with
                    respect to every predictor parameter (section
                    "Cross-Modal Attention Distillation").

Only the test suite, the smoke entry point and the benchmark's CPU-baseline
leg may import this package.  The HIP product path never calls it, and it
shares no code, tables or helpers with that path.  Inputs arrive as arrays
(the seeded generators live in their own module); everything is computed in
float64 from the exact stored input values.
"""
from .predictor import gelu_erf, mlp, predicted_attention, predicted_attention_batch, rope
from .select import (SelectResult, greedy_select, replay_check, restore_order, top_k0)
from .similarity import cosine_entries, cosine_similarity, row_norms
from .pipeline import assemble, prune
from .teacher import TeacherResult, js_divergence, layer_distributions, teacher_selection
from .train import TrainStepResult, gelu_erf_grad, kl_divergence, train_step
from .decoder import decoder_layer

__all__ = [
    "decoder_layer",
    "TrainStepResult", "gelu_erf_grad", "kl_divergence", "train_step",
    "TeacherResult", "js_divergence", "layer_distributions", "teacher_selection",
    "assemble",
    "gelu_erf", "mlp", "rope", "predicted_attention", "predicted_attention_batch",
    "row_norms", "cosine_similarity", "cosine_entries", "top_k0", "greedy_select",
    "restore_order", "replay_check", "SelectResult", "prune",
]
