"""Helpers shared by the GPU parity tests: moving seeded workloads to the
device and handing the same values to the oracle."""
import numpy as np
import pytest
import torch

import paper_2608_06411_amd as mp

WEIGHT_NAMES = ("w1_v", "b1_v", "w2_v", "b2_v", "w_k", "w1_t", "b1_t", "w2_t", "b2_t", "w_q")


def device():
    if not torch.cuda.is_available():
        pytest.skip("no GPU visible")
    mp.lib()  # fail loudly if the library is missing
    return torch.device("cuda:0")


def to_dev(store: np.ndarray, dtype: str, dev):
    if dtype == "bf16":
        return torch.from_numpy(np.ascontiguousarray(store).view(np.int16)).to(dev).view(torch.bfloat16)
    return torch.from_numpy(np.ascontiguousarray(store, dtype=np.float32)).to(dev)


def dev_weights(x: dict, dtype: str, dev, theta=10000.0) -> mp.PredictorWeights:
    return mp.PredictorWeights(**{n: to_dev(x[n + "_store"], dtype, dev) for n in WEIGHT_NAMES},
                               rope_theta=theta)


def oracle_weights(x: dict) -> dict:
    return {n: x[n + "_f32"] for n in WEIGHT_NAMES}


def dev_inputs(x: dict, dev):
    dt = x["cfg"].dtype
    return dict(V=to_dev(x["V_store"], dt, dev), T=to_dev(x["T_store"], dt, dev),
                pos_v=torch.from_numpy(x["pos_v"]).to(dev),
                pos_t=torch.from_numpy(x["pos_t"]).to(dev),
                w=dev_weights(x, dt, dev, x["cfg"].pred.rope_theta))


def announce(msg: str):
    print(f"[gpu case] {msg}", flush=True)
