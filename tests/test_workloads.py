"""The synthetic workload recipe: sizes, prefix stability, mutant sampling."""
import numpy as np
import pytest

import workloads as W


def test_config_sizes():
    expect = {"mlp": (109386, 202, 4), "lenet5": (44426, 236, 6), "vgg": (2196810, 1162, 9),
              "resnet20": (269034, 698, 31), "resnet18w": (11266632, 5000, 31)}
    for cfg, (params, neurons, nodes) in expect.items():
        c = W.CONFIGS[cfg]
        m = W.make_model(c["graph"], c["dtype"], c["bias_std"])
        assert m.n_params() == params
        assert sum(m.nodes[i].c_out for i in m.weighted_nodes()) == neurons
        assert len(m.nodes) == nodes
        for i, n in enumerate(m.nodes):
            assert all(p < i for p in n.inputs)            # topological order


def test_prefix_stable_inputs_and_mutants():
    a = W.make_workload("lenet5", n_inputs=300, n_mutants=30)
    b = W.make_workload("lenet5", n_inputs=100, n_mutants=10)
    assert np.array_equal(a.inputs[:100], b.inputs)
    s = a.mutants.subset(10)
    for f in ("mutant_id", "op", "layer", "neuron", "partner"):
        assert np.array_equal(getattr(s, f), getattr(b.mutants, f))


@pytest.mark.parametrize("cfg,k", [("mlp", 1), ("lenet5", 2), ("resnet20", 7)])
def test_layer_first_sampling(cfg, k):
    wl = W.make_workload(cfg, n_inputs=1, n_mutants=200)
    mu = wl.mutants
    for m in range(mu.n_mutants):
        r = mu.records_of(m)
        assert r.size == k
        assert len(set(mu.op[r])) == 1                      # one operator per mutant
        first = mu.layer[r[0]]
        assert all(mu.layer[r] >= first)                    # the first record is the first layer
        pairs = set(zip(mu.layer[r].tolist(), mu.neuron[r].tolist()))
        assert len(pairs) == k                              # without replacement
        for i in r:
            node = wl.model.nodes[mu.layer[i]]
            assert 0 <= mu.neuron[i] < node.c_out
            if mu.op[i] == W.NS:
                assert mu.partner[i] != mu.neuron[i] and 0 <= mu.partner[i] < node.c_out
            if mu.op[i] == W.GF:
                assert mu.noise[i].shape == (node.fan_in,) and mu.noise[i].dtype == np.float32
    if cfg == "resnet20":
        names = {wl.model.nodes[l].name for l in mu.layer}
        assert "stem" not in names


def test_uniform_sampling_k_per_ratio():
    for ri, k in enumerate((1, 12, 58, 35)):
        wl = W.make_workload("vgg", n_inputs=1, n_mutants=5, ratio_index=ri)
        assert wl.mutants.n_records == 5 * k


def test_gf_noise_sigma():
    wl = W.make_workload("lenet5", n_inputs=1, n_mutants=400)
    mu = wl.mutants
    for l in wl.model.weighted_nodes():
        recs = [i for i in range(mu.n_records) if mu.op[i] == W.GF and mu.layer[i] == l]
        if len(recs) < 3:
            continue
        eps = np.concatenate([mu.noise[i] for i in recs]).astype(np.float64)
        sigma = 0.1 * wl.model.weights[l].astype(np.float64).std()
        assert abs(eps.std() / sigma - 1) < 0.25


def test_layer_first_draws_cap_at_the_neurons_left():
    """MobileNetV2 at 1% draws k = 46 neurons; a mutant whose first layer is
    near the output keeps every neuron at or after it instead."""
    wl = W.make_workload("mobilenetv2", n_inputs=1, n_mutants=300)
    m, mu = wl.model, wl.mutants
    k = max(1, int(0.01 * sum(m.nodes[i].c_out for i in m.weighted_nodes()) + 0.5))
    for mid in range(mu.n_mutants):
        r = mu.records_of(mid)
        first = int(mu.layer[r[0]])
        left = sum(m.nodes[l].c_out for l in m.weighted_nodes() if l >= first)
        assert len(r) == min(k, left)
        assert (mu.layer[r] >= first).all()
