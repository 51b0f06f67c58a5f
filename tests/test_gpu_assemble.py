"""map_assemble on the GPU: the pruned image's kept rows and its question
rows packed for the language model, byte-exact against oracle.assemble fed
the same inputs (map_prune's kept rows and positions, the question rows)."""
import numpy as np
import pytest
import torch

import oracle
from workloads import get_config, make_inputs

from gpu_util import announce, dev_inputs, device

pytestmark = pytest.mark.gpu


def _bits(t):
    if t.dtype == torch.bfloat16:
        return t.view(torch.int16).cpu().numpy().view(np.uint16)
    return t.cpu().numpy()


@pytest.mark.parametrize("name,over", [
    ("tiny", {}),
    ("sweep", {"B": 3, "N": 600, "M": (16, 90), "K": 64, "K0": 32}),
])
def test_assemble_after_prune(name, over):
    from paper_2608_06411_amd import map_assemble, map_prune
    cfg = get_config(name, **over)
    announce(f"assemble {name} {over}")
    x = make_inputs(cfg)
    d = dev_inputs(x, device())
    o = map_prune(d["w"], d["V"], d["pos_v"], d["T"], d["pos_t"], x["t_off"], cfg.K, cfg.K0, cfg.tau)
    X, pos = map_assemble(o["V_out"], o["pos_out"], d["T"], d["pos_t"], x["t_off"])
    torch.cuda.synchronize()
    V_out, pos_out, idx = _bits(o["V_out"]), o["pos_out"].cpu().numpy(), o["idx"].cpu().numpy()
    want_X, want_pos = oracle.assemble(V_out, pos_out, x["T_store"], x["pos_t"], x["t_off"])
    got_X = _bits(X)
    assert got_X.shape == want_X.shape and pos.shape == want_pos.shape
    np.testing.assert_array_equal(got_X, want_X)
    np.testing.assert_array_equal(pos.cpu().numpy(), want_pos)
    # the kept rows are the image's own rows at the kept indices, in original order
    for b in range(cfg.B):
        start = b * cfg.K + int(x["t_off"][b])
        np.testing.assert_array_equal(got_X[start:start + cfg.K], x["V_store"][b][idx[b]])
        np.testing.assert_array_equal(pos.cpu().numpy()[start:start + cfg.K], x["pos_v"][b][idx[b]])
