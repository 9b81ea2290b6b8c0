"""The C-ABI library on the CPU: it loads, exports every declared symbol, and
its planner (planning-only contexts, no GPU) agrees with the oracle's
independent reading of Algorithm 1 (first mutated layer, boundary K,
clusters) and with the Lemma 4 ledger; invalid calls are rejected."""
import os
import re

import numpy as np
import pytest

import oracle as O
import workloads as W
from paper_2607_18582_amd import binding as B

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def _declared_functions():
    with open(os.path.join(ROOT, "include", "mure.h")) as f:
        src = f.read()
    return sorted(set(re.findall(r"\b(mure_[a-z_]+)\s*\(", src)))


def test_library_exports_every_declared_symbol():
    lib = B.load_library()
    declared = _declared_functions()
    assert set(declared) == set(B.EXPORTED)
    for name in declared:
        assert hasattr(lib, name), name
    assert lib.mure_version() == 6


def _plan_ctx(model):
    m = B.Mure(device=-1)
    m.load_model(model.nodes, model.in_hwc, model.dtype, model.weights, model.biases)
    return m


@pytest.mark.parametrize("cfg", ["mlp", "lenet5", "vgg", "resnet20", "resnet18w", "mobilenetv2", "lstm",
                                 "rnn_imdb"])
def test_planner_matches_oracle_boundaries_and_ledger(cfg):
    wl = W.make_workload(cfg, n_inputs=1, n_mutants=60)
    m = _plan_ctx(wl.model)
    m.apply(wl.mutants)
    om = O.OracleModel(wl.model)
    dg = O.get_dep_graph(om)
    groups = {}
    for mid in range(wl.mutants.n_mutants):
        mmi, grp, K = m.mutant_plan(mid)
        mu = sorted(set(wl.mutants.layer[wl.mutants.records_of(mid)].tolist()))
        assert mmi == mu[0]
        assert K == sorted(O.boundary(dg, mmi, len(om.nodes)))
        groups.setdefault(grp, set()).add(mmi)
    assert all(len(v) == 1 for v in groups.values())           # one mmi per cluster
    st = m.stats()
    assert st["n_groups"] == len(groups)
    cc = O.cluster_costs(om, wl.mutants)
    assert st["macs_vanilla"] == sum(c["vanilla"] for c in cc)
    assert st["macs_memoized"] == sum(c["memoized"] for c in cc)
    assert st["macs_vanilla"] - st["macs_memoized"] == sum((c["size"] - 1) * c["cost_prefix"] for c in cc)
    assert st["macs_executed"] <= st["macs_memoized"]
    m.close()


def test_vanilla_mode_starts_every_mutant_at_the_first_layer():
    wl = W.make_workload("resnet20", n_inputs=1, n_mutants=40)
    m = _plan_ctx(wl.model)
    m.set_option("vanilla", 1)
    m.apply(wl.mutants)
    assert {m.mutant_plan(i)[0] for i in range(40)} == {1}
    st = m.stats()
    assert st["n_groups"] == 1
    assert st["macs_memoized"] == st["macs_vanilla"]


def test_identity_mutants_have_no_plan():
    wl = W.make_workload("mlp", n_inputs=1, n_mutants=3)
    m = _plan_ctx(wl.model)
    mu = wl.mutants
    m.apply_mutants(5, mu.mutant_id, mu.op, mu.layer, mu.neuron, mu.partner, mu.noise)
    assert m.mutant_plan(4)[0] == -1 and m.mutant_plan(3)[0] == -1
    assert m.stats()["n_identity_mutants"] == 2


def test_records_without_a_permutation_list_are_accepted():
    # Mutants built field by field carry an empty perm list (no WS records)
    wl = W.make_workload("mlp", n_inputs=1, n_mutants=4)
    mu = wl.mutants
    bare = W.Mutants(mu.n_mutants, mu.mutant_id, mu.op, mu.layer, mu.neuron, mu.partner,
                     list(mu.noise))
    assert bare.perm == []
    m = _plan_ctx(wl.model)
    m.apply(bare)
    assert [m.mutant_plan(i)[0] for i in range(4)] == [
        int(mu.layer[mu.records_of(i)].min()) for i in range(4)]
    m.close()


def test_invalid_calls_are_rejected_atomically():
    wl = W.make_workload("lenet5", n_inputs=1, n_mutants=4)
    m = B.Mure(device=-1)
    mu = wl.mutants
    with pytest.raises(B.MureError) as e:                       # before load_model
        m.apply(mu)
    assert e.value.status == B.MURE_E_STATE
    model = wl.model
    m.load_model(model.nodes, model.in_hwc, model.dtype, model.weights, model.biases)
    m.apply(mu)
    before = [m.mutant_plan(i) for i in range(4)]
    bad_cases = [
        dict(layer=[0]),                     # the input has no neurons
        dict(neuron=[99]),                   # neuron out of range
        dict(op=[7]),                        # unknown operator
        dict(mutant_id=[9]),                 # mutant out of range
    ]
    for case in bad_cases:
        args = dict(mutant_id=[0], op=[1], layer=[1], neuron=[0], partner=[-1], noise=[None])
        args.update(case)
        with pytest.raises(B.MureError) as e:
            m.apply_mutants(4, **args)
        assert e.value.status == B.MURE_E_INVALID
    with pytest.raises(B.MureError):         # switch partner equal to the neuron
        m.apply_mutants(4, [0], [3], [1], [2], [2], [None])
    with pytest.raises(B.MureError):         # fuzz noise of the wrong length
        m.apply_mutants(4, [0], [0], [1], [2], [-1], [np.zeros(3, np.float32)])
    with pytest.raises(B.MureError):         # weight shuffle with a repeated index
        m.apply_mutants(4, [0], [4], [1], [2], [-1], [None], [np.zeros(25, np.int32)])
    with pytest.raises(B.MureError):         # weight shuffle of the wrong length
        m.apply_mutants(4, [0], [4], [1], [2], [-1], [None], [np.arange(5, dtype=np.int32)])
    assert [m.mutant_plan(i) for i in range(4)] == before     # nothing applied
    m.apply_mutants(4, [0], [4], [1], [2], [-1], [None], [np.arange(25, dtype=np.int32)[::-1].copy()])
    assert m.mutant_plan(0)[0] == 1
    with pytest.raises(B.MureError) as e:
        m.set_option("chunk_inputs", 100)
    assert e.value.status == B.MURE_E_INVALID


def test_planning_context_refuses_device_work():
    import ctypes as C
    wl = W.make_workload("mlp", n_inputs=1, n_mutants=2)
    m = _plan_ctx(wl.model)
    m.apply(wl.mutants)
    st = m.lib.mure_run_original(m.ctx, C.c_void_p(1), 1, None)
    assert st == B.MURE_E_UNSUPPORTED
    st = m.lib.mure_run_mutants(m.ctx, None, None, None)
    assert st == B.MURE_E_UNSUPPORTED


def test_model_validation():
    model = W.tiny_resnet()
    m = B.Mure(device=-1)
    nodes = [n for n in model.nodes]
    import copy
    bad = copy.deepcopy(nodes)
    bad[2].inputs = (5,)                     # reads a later node
    with pytest.raises(B.MureError):
        m.load_model(bad, model.in_hwc, "f32", model.weights, model.biases)
    bad = copy.deepcopy(nodes)
    bad[1].c_in = 3                          # wrong channel count
    with pytest.raises(B.MureError):
        m.load_model(bad, model.in_hwc, "f32", model.weights, model.biases)
    w = list(model.weights)
    w[1] = None                              # missing weights
    with pytest.raises(B.MureError):
        m.load_model(nodes, model.in_hwc, "f32", w, model.biases)
    m.load_model(nodes, model.in_hwc, "f32", model.weights, model.biases)


def test_depthwise_switch_recomputes_at_mmi():
    """A switch on a depthwise layer is not a channel exchange of the
    original's output (each filter meets the other channel's input), so the
    planner recomputes both channels there; on an ordinary convolution it
    remaps the cached output."""
    m = W.make_model("mobilenetv2", "bf16", 0.01)
    dw = next(i for i, n in enumerate(m.nodes) if n.kind == W.DWCONV)
    pw = next(i for i, n in enumerate(m.nodes) if n.kind == W.CONV2D and i > dw)
    ctx = _plan_ctx(m)
    z = np.zeros(0, np.int32)
    ctx.apply_mutants(2, np.array([0, 1], np.int32), np.array([W.NS, W.NS], np.int32),
                      np.array([dw, pw], np.int32), np.array([0, 0], np.int32),
                      np.array([1, 1], np.int32), [None, None])
    st = ctx.stats()
    per_dw = m.nodes[dw].out_hwc[0] * m.nodes[dw].out_hwc[1] * 9
    # algorithmic MACs at mmi: two depthwise channels for mutant 0, none for mutant 1
    after = lambda l: sum(O.node_macs(O.OracleModel(m))[l + 1:])
    assert st["macs_algorithmic"] == 2 * per_dw + after(dw) + after(pw)
    ctx.close()


def test_lstm_records_recompute_the_whole_layer():
    """Every record on an LSTM layer changes all of its units' trajectories
    (the recurrence), so even an effect block recomputes the layer, while an
    effect block on the embedding only remaps one feature."""
    m = W.make_model("lstm", "f32", 0.0)
    emb, l1 = 1, 2
    ctx = _plan_ctx(m)
    ctx.apply_mutants(2, np.array([0, 1], np.int32), np.array([W.NEB, W.NEB], np.int32),
                      np.array([l1, emb], np.int32), np.array([3, 3], np.int32),
                      np.array([-1, -1], np.int32), [None, None])
    macs = O.node_macs(O.OracleModel(m))
    st = ctx.stats()
    assert st["macs_algorithmic"] == sum(macs[l1:]) + sum(macs[emb + 1:])
    assert st["n_groups"] == 2
    ctx.close()


def test_sequence_layer_validation():
    m = W.make_model("lstm", "f32", 0.0)
    bad = list(m.nodes)
    bad[2] = W.Node(W.LSTM, (1,), 32, 24, out_hwc=(1, 40, 24), name="odd", seq=1)
    ctx = B.Mure(device=-1)
    with pytest.raises(B.MureError, match="units"):
        ctx.load_model(bad, m.in_hwc, "f32", m.weights, m.biases)
    ctx.close()


def test_record_parameter_packing():
    """Each record's noise/permutation entry is found at its address with its
    length; records without one get address 0 and length 0, and an empty
    entry gets length 0 (the library reads nothing there)."""
    import ctypes
    arrays = [np.array([1.5, -2.0], np.float32), None, np.arange(5, dtype=np.float64),
              np.zeros(0, np.float32), None, np.array([7.0], np.float32)]
    pool, addr, lens = B._pack(arrays, len(arrays), np.float32)
    assert all(p.dtype == np.float32 for p in pool) and sum(p.size for p in pool) == 8
    # an entry already float32 and contiguous is passed in place
    assert addr[0] == arrays[0].ctypes.data and addr[5] == arrays[5].ctypes.data
    assert lens.tolist() == [2, 0, 5, 0, 0, 1]
    assert addr[1] == 0 and addr[3] == 0 and addr[4] == 0
    for r, a in enumerate(arrays):
        if a is None or len(a) == 0:
            continue
        got = np.ctypeslib.as_array((ctypes.c_float * int(lens[r])).from_address(int(addr[r])))
        assert np.array_equal(got, a.astype(np.float32)), r
    pool, addr, lens = B._pack([None, None], 2, np.int32)
    assert not addr.any() and not lens.any()
    pool, addr, lens = B._pack(None, 3, np.int32)
    assert addr.shape == (3,) and not addr.any() and not lens.any()
    # a single non-empty entry (the itemgetter path for one index)
    arr = [None, np.array([3, 1, 2], np.int64)]
    pool, addr, lens = B._pack(arr, 2, np.int32)
    got = np.ctypeslib.as_array((ctypes.c_int32 * 3).from_address(int(addr[1])))
    assert got.tolist() == [3, 1, 2] and lens.tolist() == [0, 3]


def test_flatten_boundary_and_flatten_output_rejected():
    """A FLATTEN between a convolution and a dense layer is the boundary K of
    the mutants whose first mutated layer is that dense layer; a FLATTEN as
    the output node (a view, not logits) is refused."""
    b = W.configs._Builder((8, 8, 4))
    x = b.conv(0, 8, 3, pad=1, relu=True, pool=2, name="C1")
    f = b.flatten(x)
    b.dense(f, 10, False, "F")
    w, bb = W.configs._draw_weights(b.nodes, "f32", 0.1, seed=2)
    model = W.Model("flat", "f32", b.nodes, w, bb)
    mu = W.make_mutants(model, 20, 1, "layer_first", variant=1)
    m = _plan_ctx(model)
    m.apply(mu)
    plans = [m.mutant_plan(i) for i in range(mu.n_mutants)]
    assert any(p[0] == f + 1 and p[2] == [f] for p in plans)
    b2 = W.configs._Builder((1, 1, 16))
    x = b2.dense(0, 10, False, "F")
    b2.flatten(x)
    w2, bb2 = W.configs._draw_weights(b2.nodes, "f32", 0.1, seed=2)
    with pytest.raises(B.MureError) as e:
        _plan_ctx(W.Model("flat_out", "f32", b2.nodes, w2, bb2))
    assert e.value.status == B.MURE_E_INVALID and "FLATTEN" in e.value.message


def test_device_memory_cap_refuses_plans_with_nomem():
    """max_device_mb bounds the model plus the mutants' copy-on-write layers:
    resnet18w (22.5 MB of bf16 weights) with 40 mutants at 5% copies about
    40 x 22 MB; a 100 MB cap refuses the plan with MURE_E_NOMEM and keeps the
    previous mutants, a 2 GB cap accepts it."""
    wl = W.make_workload("resnet18w", n_inputs=1, n_mutants=40)
    m = _plan_ctx(wl.model)
    small = W.make_workload("resnet18w", n_inputs=1, n_mutants=1)
    m.apply(small.mutants)
    m.set_option("max_device_mb", 100)
    with pytest.raises(B.MureError) as e:
        m.apply(wl.mutants)
    assert e.value.status == B.MURE_E_NOMEM and "max_device_mb" in e.value.message
    assert m.stats()["n_mutants"] == 1                  # the earlier plan stands
    m.set_option("max_device_mb", 2048)
    m.apply(wl.mutants)
    assert m.stats()["n_mutants"] == 40
    with pytest.raises(B.MureError):
        m.set_option("max_device_mb", -1)
