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


def test_layer_offset_selects_the_later_layers_of_the_model():
    """A workload with layer0 = j covers the model's layers j, j + 1, ...:
    its layer i has the weights, hidden states and Zipf bias of layer j + i
    of the whole model, and layer0 = 0 leaves every tensor as it was."""
    w = synth.WORKLOADS["tiny"].replace(zipf=1.1)
    tail = w.replace(L=2, layer0=2)
    for i in range(2):
        for kind in (synth.KIND_ROUTER_NATIVE, synth.KIND_ROUTER_TEMPORAL, synth.KIND_ROUTER_SPATIO):
            assert np.array_equal(synth.router_host(tail, kind, i), synth.router_host(w, kind, 2 + i))
        for a, b in zip(synth.expert_host(tail, i, 5), synth.expert_host(w, 2 + i, 5)):
            assert np.array_equal(a, b)
        assert np.array_equal(synth.hidden_host(tail, 0, i, T=4), synth.hidden_host(w, 0, 2 + i, T=4))
    assert np.array_equal(synth.zipf_bias(tail), synth.zipf_bias(w)[2:4])
    # a different layer really is a different tensor
    assert not np.array_equal(synth.router_host(tail, synth.KIND_ROUTER_NATIVE, 0),
                              synth.router_host(w, synth.KIND_ROUTER_NATIVE, 0))
