"""The layer-0 input after pruning (section "Inference-Time Token Pruning"):
oracle.assemble against a hand-written example."""
import numpy as np

import oracle


def test_assemble_hand_example():
    # two images, K = 2 kept rows each (already in original order), questions of 1 and 3 tokens
    V_out = np.array([[[1, 1], [2, 2]], [[3, 3], [4, 4]]], np.float32)
    pos_out = np.array([[5, 9], [0, 7]], np.int32)
    T = np.array([[10, 10], [20, 20], [21, 21], [22, 22]], np.float32)
    pos_t = np.array([16, 16, 17, 18], np.int32)
    X, pos = oracle.assemble(V_out, pos_out, T, pos_t, [0, 1, 4])
    np.testing.assert_array_equal(X, [[1, 1], [2, 2], [10, 10], [3, 3], [4, 4], [20, 20], [21, 21], [22, 22]])
    np.testing.assert_array_equal(pos, [5, 9, 16, 0, 7, 16, 17, 18])
