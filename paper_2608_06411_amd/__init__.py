"""MAP (Middle-layer Attention Prediction) visual-token pruning on MI355X.

The pruning stage of "Learning to Predict Middle-Layer Attention in MLLMs for
Visual Token Pruning" -- predictor scoring (Eq. (3)), cosine similarity of
the visual tokens, diversity-aware selection (Eq. (4)) and the gather of the
kept tokens -- as hand-written HIP kernels for gfx950 behind a C ABI
(include/map.h).  This package is the Python binding of that library.
"""
from .binding import (EXPORTS, MAP_BF16, MAP_F32, MapError, PredictorWeights, PruneWorkspace, TrainWorkspace, DecoderWeights, decoder_workspace, map_decoder_layer,
                      lib, map_assemble, map_prune, map_prune_assemble, map_score, map_train_step, map_select, map_similarity, map_teacher,
                      selection_status, set_finite_check, set_select_images_per_launch, set_subset_tokens,
                      timing_enable, timing_read, timing_reset)

__all__ = [
    "EXPORTS", "MAP_BF16", "MAP_F32", "MapError", "PredictorWeights", "PruneWorkspace", "lib",
    "TrainWorkspace", "map_train_step", "DecoderWeights", "decoder_workspace", "map_decoder_layer", "map_assemble", "map_prune", "map_prune_assemble", "map_score", "map_select", "map_similarity", "map_teacher", "selection_status",
    "set_finite_check", "set_select_images_per_launch", "set_subset_tokens", "timing_enable",
    "timing_read", "timing_reset",
]
