"""Tensor ids of the input generator accept numpy integer indices (as the
oracle's selections are) and give the same tensors as Python ints."""
import numpy as np

import synth


def test_numpy_indices_give_the_same_tensors():
    w = synth.WORKLOADS["tiny"]
    for a, b in zip(synth.expert_host(w, np.int32(3), np.int32(15)), synth.expert_host(w, 3, 15)):
        assert np.array_equal(a, b)
    assert np.array_equal(synth.hidden_host(w, np.int64(0), np.int32(2), T=3), synth.hidden_host(w, 0, 2, T=3))
    assert synth.router_tid(np.int32(1), np.int32(2)) == synth.router_tid(1, 2)
