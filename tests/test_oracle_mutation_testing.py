"""Pins for the oracle's operators, kill predicate, score and Algorithms 1-4.

* operators: hand-computed rows and output-layer closed forms (a switch swaps
  two logits exactly, an inverse negates one, a block zeroes one, a fuzz
  recomputes one from the penultimate activations);
* kill / killingLabels / MS: a hand-worked fixture (Section 5.2);
* Theorem 1 by brute force: Algorithms 1-4 (memoized) equal vanilla testing
  bit for bit on tiny sequential and residual networks, every neuron x every
  operator plus multi-neuron mutants;
* Lemma 1 and the boundary rule K (Section 4 vs Algorithm 1);
* invariants: identity mutants are never killed and reproduce the original's
  logits; a mutant's activations before its first mutated layer equal the
  original's;
* Lemma 4: vanilla - memoized = (|C| - 1) cost(P) per cluster.
"""
import itertools
import json
import os

import numpy as np
import pytest

import oracle as O
from oracle.memoized import mutated_layers
from oracle.vanilla import predicted
import workloads as W
from workloads.graph import Mutants, GF, NEB, NAI, NS, WS

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def _mutants(records, n_mutants=None):
    """records: list of (mutant, op, layer, neuron, partner, noise[, perm])."""
    if n_mutants is None:
        n_mutants = 1 + max(r[0] for r in records) if records else 0
    a = lambda k: np.array([r[k] for r in records], np.int32)
    return Mutants(n_mutants, a(0), a(1), a(2), a(3), a(4), [r[5] for r in records],
                   [r[6] if len(r) > 6 else None for r in records])


# ---------------------------------------------------------------- operators

def test_operators_on_a_dense_layer_by_hand():
    m = W.tiny_mlp()
    om = O.OracleModel(m)
    l = 1
    w0, b0 = om.weights[l].copy(), om.biases[l].copy()
    eps = np.linspace(-1, 1, 6).astype(np.float32)
    muts = _mutants([(0, GF, l, 2, -1, eps), (1, NEB, l, 3, -1, None),
                     (2, NAI, l, 4, -1, None), (3, NS, l, 0, 4, None)])
    Wg, Bg, _ = O.apply_records(om, muts, 0)
    assert np.array_equal(Wg[l][2], (w0[2] + eps).astype(np.float32))
    assert np.array_equal(np.delete(Wg[l], 2, 0), np.delete(w0, 2, 0)) and np.array_equal(Bg[l], b0)
    Wn, Bn, _ = O.apply_records(om, muts, 1)
    assert not Wn[l][3].any() and Bn[l][3] == 0 and Bn[l][2] == b0[2]
    Wa, Ba, _ = O.apply_records(om, muts, 2)
    assert np.array_equal(Wa[l][4], -w0[4]) and Ba[l][4] == -b0[4]
    Ws, Bs, _ = O.apply_records(om, muts, 3)
    assert np.array_equal(Ws[l][0], w0[4]) and np.array_equal(Ws[l][4], w0[0])
    assert Bs[l][0] == b0[4] and Bs[l][4] == b0[0]
    # the original is untouched
    assert np.array_equal(om.weights[l], w0) and np.array_equal(om.biases[l], b0)


def test_weight_shuffle_by_hand():
    om = O.OracleModel(W.tiny_mlp())
    w0 = om.weights[1].copy()
    perm = np.array([5, 0, 4, 1, 3, 2], np.int32)
    Wm, Bm, _ = O.apply_records(om, _mutants([(0, WS, 1, 2, -1, None, perm)]), 0)
    assert [Wm[1][2][k] for k in range(6)] == [w0[2][p] for p in perm]
    assert np.array_equal(np.delete(Wm[1], 2, 0), np.delete(w0, 2, 0))
    assert np.array_equal(Bm[1], om.biases[1])
    with pytest.raises(ValueError):                     # not a permutation
        O.apply_records(om, _mutants([(0, WS, 1, 2, -1, None, np.zeros(6, np.int32))]), 0)
    # the identity permutation is an identity mutation; a permutation followed
    # by its inverse too
    x = W.make_inputs(W.tiny_mlp(), 8, "uniform")
    inv = np.argsort(perm).astype(np.int32)
    muts = _mutants([(0, WS, 1, 2, -1, None, np.arange(6, dtype=np.int32)),
                     (1, WS, 1, 2, -1, None, perm), (1, WS, 1, 2, -1, None, inv)])
    van = O.run_vanilla(om, x, muts, keep_logits=[0, 1], accumulate="ordered")
    assert np.array_equal(van.mutant_logits[0], van.logits)
    assert np.array_equal(van.mutant_logits[1], van.logits)


def test_switch_chain_applies_in_record_order():
    om = O.OracleModel(W.tiny_mlp())
    w0 = om.weights[1].copy()
    muts = _mutants([(0, NS, 1, 0, 1, None), (0, NS, 1, 1, 2, None)])
    Wm, _, _ = O.apply_records(om, muts, 0)
    # (0 1) then (1 2): row0 <- w1, row1 <- w2, row2 <- w0
    assert np.array_equal(Wm[1][0], w0[1]) and np.array_equal(Wm[1][1], w0[2])
    assert np.array_equal(Wm[1][2], w0[0])


def test_gf_bf16_rounds_the_fuzzed_row():
    m = W.tiny_mlp("bf16")
    om = O.OracleModel(m)
    eps = np.full(6, 1e-3, np.float32)
    Wm, _, _ = O.apply_records(om, _mutants([(0, GF, 1, 0, -1, eps)]), 0)
    assert np.array_equal(Wm[1][0], O.rne_bf16(om.weights[1][0] + eps))
    assert np.array_equal(O.rne_bf16(Wm[1]), Wm[1])


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_output_layer_closed_forms(dtype):
    m = W.tiny_resnet(dtype)
    om = O.OracleModel(m)
    x = W.make_inputs(m, 16, "normal")
    out = om.out
    acts = O.forward_all(om, x, accumulate="ordered")
    z = acts[out].reshape(16, -1)
    h = acts[m.nodes[out].inputs[0]].reshape(16, -1).astype(np.float64)
    eps = np.arange(h.shape[1], dtype=np.float32) * np.float32(0.01)
    muts = _mutants([(0, NS, out, 0, 2, None), (1, NAI, out, 1, -1, None),
                     (2, NEB, out, 2, -1, None), (3, GF, out, 1, -1, eps)])
    zs = {k: O.forward(om, x, *O.apply_records(om, muts, k)[:2], accumulate="ordered")
          for k in range(4)}
    swapped = z.copy(); swapped[:, [0, 2]] = z[:, [2, 0]]
    assert np.array_equal(zs[0], swapped)
    neg = z.copy(); neg[:, 1] = -z[:, 1]
    assert np.array_equal(zs[1], neg)
    zero = z.copy(); zero[:, 2] = 0
    assert np.array_equal(zs[2], zero)
    wrow = (om.weights[out][1] + eps)
    if dtype == "bf16":
        wrow = O.rne_bf16(wrow)
    for n in range(16):
        acc = 0.0
        for c in range(h.shape[1]):
            acc += h[n, c] * float(wrow[c])
        assert zs[3][n, 1] == np.float32(acc + float(om.biases[out][1]))
        assert np.array_equal(np.delete(zs[3][n], 1), np.delete(z[n], 1))


# ---------------------------------------------------------------- kill / score

def test_kill_and_score_worked_example():
    with open(os.path.join(GOLDEN, "kill_score_worked_example.json")) as f:
        g = json.load(f)
    z = np.array(g["original_logits"], np.float32)
    zm = np.array(g["mutant_logits"], np.float32)
    pm = np.stack([predicted(q) for q in zm])
    for key in ("with_labels", "own_predictions"):
        case = g[key]
        label = np.array(case["labels"])
        if key == "own_predictions":
            assert np.array_equal(predicted(z), label)
        kill, killing, num, den, nl = O.kill_and_score(predicted(z), pm, label, 3)
        assert kill.astype(int).tolist() == case["kill"]
        assert [sorted(np.nonzero(k)[0].tolist()) for k in killing] == case["killing_labels"]
        assert (num, den, nl) == (case["ms_num"], case["ms_den"], case["n_labels"])
    own = g["own_predictions"]
    kill, *_ = O.kill_and_score(predicted(z), pm, np.array(own["labels"]), 3)
    assert O.pack_bits(kill)[:, 0].tolist() == own["kill_words"]
    assert int(kill.any(axis=1).sum()) == own["killed_mutants"]


def test_pack_bits_layout_and_padding():
    rng = np.random.default_rng(0)
    b = rng.random((3, 130)) < 0.5
    words = O.pack_bits(b)
    assert words.shape == (3, 3) and words.dtype == np.uint64
    for m in range(3):
        for x in range(130):
            assert bool((int(words[m, x >> 6]) >> (x & 63)) & 1) == b[m, x]
        assert int(words[m, 2]) >> 2 == 0          # padding bits are zero


def test_margins():
    z = np.array([[1, 3, 2], [5, 5, 0]], np.float32)
    assert O.margins(z).tolist() == [1.0, 0.0]


# ---------------------------------------------------------------- Theorem 1 by brute force

def _all_single_mutants(m: W.Model, seed=0):
    rng = np.random.default_rng(seed)
    recs = []
    mid = 0
    for l in m.weighted_nodes():
        node = m.nodes[l]
        for i in range(node.c_out):
            for op in (GF, NEB, NAI, NS, WS):
                part = -1
                if op == NS:
                    part = (i + 1 + int(rng.integers(node.c_out - 1))) % node.c_out
                eps = (rng.standard_normal(node.fan_in) * 0.1).astype(np.float32) if op == GF else None
                perm = rng.permutation(node.fan_in).astype(np.int32) if op == WS else None
                recs.append((mid, op, l, i, part, eps, perm))
                mid += 1
    # a few multi-neuron mutants across layers
    wn = m.weighted_nodes()
    for t in range(6):
        op = (GF, NEB, NAI, NS)[t % 4]
        for l in sorted(rng.choice(wn, size=2, replace=False)):
            node = m.nodes[l]
            i = int(rng.integers(node.c_out))
            part = (i + 1) % node.c_out if op == NS else -1
            eps = (rng.standard_normal(node.fan_in) * 0.1).astype(np.float32) if op == GF else None
            recs.append((mid, op, int(l), i, part, eps))
        mid += 1
    return _mutants(recs, mid + 1)          # the last mutant has no records (identity)


@pytest.mark.parametrize("builder", ["mlp", "lenet", "resnetA", "resnetP", "resnetA_bf16",
                                     "mobilenet", "mobilenet_bf16", "rnn"])
def test_soundness_memoized_equals_vanilla(builder):
    m = {"mlp": lambda: W.tiny_mlp(),
         "lenet": lambda: W.tiny_lenet(),
         "resnetA": lambda: W.tiny_resnet("f32", shortcut="optionA"),
         "resnetP": lambda: W.tiny_resnet("f32", shortcut="proj"),
         "resnetA_bf16": lambda: W.tiny_resnet("bf16", shortcut="optionA"),
         "mobilenet": lambda: W.tiny_mobilenet(),
         "mobilenet_bf16": lambda: W.tiny_mobilenet("bf16"),
         "rnn": lambda: W.tiny_rnn()}[builder]()
    om = O.OracleModel(m)
    x = W.make_inputs(m, 12, "tokens" if builder == "rnn" else "normal")
    muts = _all_single_mutants(m)
    memo = O.mure(om, x, muts)
    van = O.run_vanilla(om, x, muts, keep_logits=range(muts.n_mutants), accumulate="ordered")
    for mid in range(muts.n_mutants):
        assert np.array_equal(memo[mid], van.mutant_logits[mid]), mid
    pm = np.stack([predicted(memo[mid]) for mid in range(muts.n_mutants)])
    kill, killing, num, den, _ = O.kill_and_score(predicted(van.logits), pm, van.label, m.n_classes)
    assert np.array_equal(kill, van.kill)
    assert (num, den) == (van.ms_num, van.ms_den)          # mutation-score error 0
    assert van.kill.any()                                   # the test is not vacuous


# ---------------------------------------------------------------- Lemma 1 / K

def _edge_set(m):
    return {(p, v) for v, n in enumerate(m.nodes) for p in n.inputs}


@pytest.mark.parametrize("cfg", ["mlp", "lenet5", "vgg", "resnet20", "resnet18w", "mobilenetv2", "lstm"])
def test_dep_graph_and_boundary_definitions_agree(cfg):
    c = W.CONFIGS[cfg]
    m = W.make_model(c["graph"], c["dtype"], c["bias_std"])
    om = O.OracleModel(m)
    dg = O.get_dep_graph(om)
    E = _edge_set(m)
    for i in range(len(m.nodes)):                               # Lemma 1
        assert set(dg[i]) == {j for (j, v) in E if v == i}
    seen = {}
    for mmi in m.weighted_nodes():
        K = O.boundary(dg, mmi, len(m.nodes))
        K_sec4 = {p for (p, v) in E if v >= mmi and p < mmi}   # tau = node index
        assert K == K_sec4
        assert K not in seen, "two first-mutated layers share a boundary"
        seen[K] = mmi
        if c["graph"] in ("mlp", "lenet5", "vgg"):
            assert K == {mmi - 1}


def test_resnet_boundaries_have_two_tensors():
    m = W.make_model("resnet20", "bf16", 0.01)
    dg = O.get_dep_graph(O.OracleModel(m))
    names = {n.name: i for i, n in enumerate(m.nodes)}
    b = names["s1b1.b"]                                    # conv_b of an identity block
    assert O.boundary(dg, b, len(m.nodes)) == {names["s1b1.a"], names["s1b0.add"]}
    a = names["s1b1.a"]
    assert O.boundary(dg, a, len(m.nodes)) == {names["s1b0.add"]}


# ---------------------------------------------------------------- invariants

@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_identity_mutants_never_killed(dtype):
    m = W.tiny_resnet(dtype)
    om = O.OracleModel(m)
    x = W.make_inputs(m, 32, "normal")
    recs = [(0, GF, l, 0, -1, np.zeros(m.nodes[l].fan_in, np.float32)) for l in m.weighted_nodes()]
    recs = [(i, *r[1:]) for i, r in enumerate(recs)]
    n = len(recs)
    recs.append((n, NAI, m.weighted_nodes()[1], 1, -1, None))   # applied twice = identity
    recs.append((n, NAI, m.weighted_nodes()[1], 1, -1, None))
    muts = _mutants(recs, n + 2)                                 # mutant n+1 has no records
    van = O.run_vanilla(om, x, muts, keep_logits=range(n + 2), accumulate="ordered")
    assert not van.kill.any()
    for mid in range(n + 2):
        assert np.array_equal(van.mutant_logits[mid], van.logits)


def test_prefix_activations_equal_original():
    wl = W.make_workload("lenet5", n_inputs=8, n_mutants=40)
    om = O.OracleModel(wl.model)
    orig = O.forward_all(om, wl.inputs)
    for mid in range(wl.mutants.n_mutants):
        Wm, Bm, _ = O.apply_records(om, wl.mutants, mid)
        mmi = min(mutated_layers(wl.mutants, mid))
        acts = O.forward_all(om, wl.inputs, Wm, Bm)
        for v in range(mmi):
            assert np.array_equal(acts[v], orig[v])


# ---------------------------------------------------------------- Lemma 4 / Theorem 2

@pytest.mark.parametrize("cfg", ["mlp", "lenet5", "resnet20"])
def test_acceleration_closed_form(cfg):
    wl = W.make_workload(cfg, n_inputs=1, n_mutants=200)
    om = O.OracleModel(wl.model)
    macs = O.node_macs(om)
    total_v = total_m = 0
    for c in O.cluster_costs(om, wl.mutants):
        assert c["vanilla"] - c["memoized"] == (c["size"] - 1) * c["cost_prefix"]
        assert c["cost_prefix"] >= 0
        total_v += c["vanilla"]; total_m += c["memoized"]
    assert total_m < total_v                                # strict (Theorem 2)
    assert sum(macs) == {"mlp": 109184, "lenet5": 281640, "resnet20": 40551040}[cfg]


@pytest.mark.parametrize("builder", ["mlp", "lenet", "resnetA", "resnetP", "mobilenet", "rnn"])
def test_ledger_counts_the_macs_the_algorithms_perform(builder, monkeypatch):
    """cluster_costs (the Lemma 4 ledger) against the multiply-accumulates the
    oracle actually executes: every matrix product [R, K] x [K, C_out] of a
    layer function counts R K C_out, a depthwise layer n Ho Wo C kh kw.
    Algorithm 1 (memoized) executes cost(P) once per cluster plus every
    mutant from its mmi on; vanilla testing executes the whole network per
    mutant."""
    import oracle.layers as OL
    import oracle.memoized as OM
    m = {"mlp": lambda: W.tiny_mlp(), "lenet": lambda: W.tiny_lenet(),
         "resnetA": lambda: W.tiny_resnet("f32", shortcut="optionA"),
         "resnetP": lambda: W.tiny_resnet("f32", shortcut="proj"),
         "mobilenet": lambda: W.tiny_mobilenet(), "rnn": lambda: W.tiny_rnn()}[builder]()
    om = O.OracleModel(m)
    n = 5
    x = W.make_inputs(m, n, "tokens" if builder == "rnn" else "normal")
    muts = _all_single_mutants(m)
    muts = muts.subset(muts.n_mutants - 1)                 # drop the identity mutant
    count = [0]
    mm, ph = OL._matmul64, OL.phi

    def matmul(a64, w2, accumulate):
        count[0] += a64.shape[0] * a64.shape[1] * w2.shape[0]
        return mm(a64, w2, accumulate)

    def phi(model, v, ins, W_=None, b=None, accumulate="blas"):
        out = ph(model, v, ins, W_, b, accumulate)
        nd = model.nodes[v]
        if nd.kind == W.DWCONV:
            count[0] += out.size * nd.kh * nd.kw
        return out

    monkeypatch.setattr(OL, "_matmul64", matmul)
    monkeypatch.setattr(OL, "phi", phi)
    monkeypatch.setattr(OM, "phi", phi)
    cc = O.cluster_costs(om, muts)
    O.mure(om, x, muts)
    assert count[0] == n * sum(c["memoized"] for c in cc)
    count[0] = 0
    O.run_vanilla(om, x, muts, accumulate="ordered")
    full = sum(O.node_macs(om))
    assert count[0] == n * (sum(c["vanilla"] for c in cc) + full)   # + the original's forward
    assert sum(c["size"] for c in cc) == muts.n_mutants
