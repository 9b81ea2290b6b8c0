"""Pins for the oracle's rounding and layer functions (CPU only).

Each layer function is checked against something other than itself: torch's
float64 CPU operators (a different implementation of the textbook
definitions, in NCHW layout), pure-Python loops on tiny inputs, and
hand-computed cases."""
import json
import os

import numpy as np
import pytest
import torch
import torch.nn.functional as F

import oracle as O
from oracle.layers import phi
import workloads as W
from workloads.graph import Node, Model, CONV2D, DENSE, ADD, GAP, INPUT

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


# ---------------------------------------------------------------- bf16 RNE

def test_rne_bf16_matches_torch_conversion():
    rng = np.random.default_rng(0)
    x = np.concatenate([
        rng.standard_normal(100000).astype(np.float32) * 10.0 ** rng.integers(-30, 30, 100000),
        np.array([0.0, -0.0, np.inf, -np.inf, 3.4e38, -3.4e38, 1e-40, -1e-40], np.float32),
    ]).astype(np.float32)
    ref = torch.from_numpy(x).to(torch.bfloat16).to(torch.float32).numpy()
    got = O.rne_bf16(x)
    assert np.array_equal(got.view(np.uint32), ref.view(np.uint32))


def test_rne_bf16_ties_to_even():
    # low halves exactly 0x8000 are ties: round to the even kept pattern
    u = np.array([0x3F808000, 0x3F818000, 0x3F807FFF, 0x3F808001, 0x7F7F8000], np.uint32)
    got = O.rne_bf16(u.view(np.float32)).view(np.uint32)
    assert list(got) == [0x3F800000, 0x3F820000, 0x3F800000, 0x3F810000, 0x7F800000]
    assert np.isnan(O.rne_bf16(np.array([np.nan], np.float32)))[0]


# ---------------------------------------------------------------- helpers

def _model(nodes, dtype="f32", weights=None, biases=None):
    n = len(nodes)
    return O.OracleModel(Model("t", dtype, nodes, weights or [None] * n, biases or [None] * n))


def _conv_node(hwc, cout, k, s, p, relu, pool):
    h, w, c = hwc
    ho = (h + 2 * p - k) // s + 1
    wo = (w + 2 * p - k) // s + 1
    if pool:
        ho, wo = ho // 2, wo // 2
    return Node(CONV2D, (0,), c, cout, k, k, s, p, relu, pool, 0, (ho, wo, cout))


# ---------------------------------------------------------------- conv

@pytest.mark.parametrize("hwc,cout,k,s,p,relu,pool", [
    ((9, 9, 3), 5, 3, 1, 1, True, 0),
    ((12, 12, 6), 16, 5, 1, 0, True, 2),
    ((11, 10, 4), 8, 3, 2, 1, True, 0),
    ((8, 8, 4), 8, 1, 2, 0, False, 0),
    ((13, 13, 2), 3, 5, 1, 0, False, 2),
])
def test_conv_matches_torch_float64(hwc, cout, k, s, p, relu, pool):
    rng = np.random.default_rng(1)
    node = _conv_node(hwc, cout, k, s, p, relu, pool)
    Wt = rng.standard_normal((cout, k, k, hwc[2])).astype(np.float32)
    b = rng.standard_normal(cout).astype(np.float32)
    m = _model([Node(INPUT, (), out_hwc=hwc), node], weights=[None, Wt], biases=[None, b])
    x = rng.standard_normal((3,) + hwc).astype(np.float32)
    got = phi(m, 1, [x])
    xt = torch.from_numpy(x.astype(np.float64)).permute(0, 3, 1, 2)
    wt = torch.from_numpy(Wt.astype(np.float64)).permute(0, 3, 1, 2)
    ref = F.conv2d(xt, wt, torch.from_numpy(b.astype(np.float64)), stride=s, padding=p)
    ref = ref.float()
    if relu:
        ref = torch.relu(ref)
    if pool:
        ref = F.max_pool2d(ref, 2)
    ref = ref.permute(0, 2, 3, 1).numpy()
    assert got.shape == ref.shape == (3,) + node.out_hwc
    # torch adds the bias in float64 too: results agree to float32 rounding
    np.testing.assert_allclose(got, ref, rtol=1e-6, atol=1e-6)


def test_conv_brute_force_loops():
    rng = np.random.default_rng(2)
    hwc, cout, k, s, p = (5, 4, 2), 3, 3, 2, 1
    node = _conv_node(hwc, cout, k, s, p, False, 0)
    Wt = rng.standard_normal((cout, k, k, 2)).astype(np.float32)
    b = rng.standard_normal(cout).astype(np.float32)
    m = _model([Node(INPUT, (), out_hwc=hwc), node], weights=[None, Wt], biases=[None, b])
    x = rng.standard_normal((1,) + hwc).astype(np.float32)
    got = phi(m, 1, [x])
    ho, wo, _ = node.out_hwc
    for i in range(ho):
        for j in range(wo):
            for o in range(cout):
                acc = 0.0
                for dy in range(k):
                    for dx in range(k):
                        y, xx = i * s + dy - p, j * s + dx - p
                        if 0 <= y < hwc[0] and 0 <= xx < hwc[1]:
                            for c in range(2):
                                acc += float(x[0, y, xx, c]) * float(Wt[o, dy, dx, c])
                assert got[0, i, j, o] == np.float32(acc + float(b[o]))


# ---------------------------------------------------------------- dense / flatten order

def test_dense_reads_hwc_flatten_order():
    rng = np.random.default_rng(3)
    hwc = (2, 3, 4)
    node = Node(DENSE, (0,), 24, 5, relu=True, out_hwc=(1, 1, 5))
    Wt = rng.standard_normal((5, 24)).astype(np.float32)
    b = rng.standard_normal(5).astype(np.float32)
    m = _model([Node(INPUT, (), out_hwc=hwc), node], weights=[None, Wt], biases=[None, b])
    x = rng.standard_normal((2,) + hwc).astype(np.float32)
    got = phi(m, 1, [x]).reshape(2, 5)
    for n in range(2):
        for o in range(5):
            acc = sum(float(x[n, h, w, c]) * float(Wt[o, (h * 3 + w) * 4 + c])
                      for h in range(2) for w in range(3) for c in range(4))
            assert got[n, o] == max(np.float32(acc + float(b[o])), np.float32(0))
    ref = torch.relu(F.linear(torch.from_numpy(x.reshape(2, -1).astype(np.float64)),
                              torch.from_numpy(Wt.astype(np.float64)),
                              torch.from_numpy(b.astype(np.float64))).float()).numpy()
    np.testing.assert_allclose(got, ref, rtol=1e-6)


# ---------------------------------------------------------------- add / gap

def test_add_option_a_shortcut_hand_example():
    a = np.zeros((1, 2, 2, 4), np.float32)
    a[0, :, :, :] = np.arange(16, dtype=np.float32).reshape(2, 2, 4) - 8
    s = np.zeros((1, 4, 4, 2), np.float32)
    s[0, :, :, 0] = np.arange(16).reshape(4, 4)
    s[0, :, :, 1] = 100 + np.arange(16).reshape(4, 4)
    node = Node(ADD, (1, 2), 2, 4, relu=True, shortcut=1, out_hwc=(2, 2, 4))
    m = _model([Node(INPUT, (), out_hwc=(4, 4, 2))] * 3 + [node])
    got = phi(m, 3, [a, s])[0]
    # subsample rows/cols 0 and 2; one zero channel before, one after
    for i in range(2):
        for j in range(2):
            sub = [0.0, s[0, 2 * i, 2 * j, 0], s[0, 2 * i, 2 * j, 1], 0.0]
            for c in range(4):
                assert got[i, j, c] == max(a[0, i, j, c] + np.float32(sub[c]), 0)


def test_gap_matches_torch_mean_and_bf16_rounding():
    rng = np.random.default_rng(4)
    x = O.rne_bf16(rng.standard_normal((3, 8, 8, 5)).astype(np.float32))
    node = Node(GAP, (0,), 5, 5, out_hwc=(1, 1, 5))
    out = Node(DENSE, (1,), 5, 2, out_hwc=(1, 1, 2))
    m = _model([Node(INPUT, (), out_hwc=(8, 8, 5)), node, out], dtype="bf16")
    got = phi(m, 1, [x]).reshape(3, 5)
    ref = torch.from_numpy(x.astype(np.float64)).mean(dim=(1, 2)).float().to(torch.bfloat16).float()
    assert np.array_equal(got, ref.numpy())


# ---------------------------------------------------------------- rounding points

def test_bf16_rounding_points_every_node_but_logits():
    m = W.tiny_resnet("bf16")
    om = O.OracleModel(m)
    x = W.make_inputs(m, 4, "normal")
    acts = O.forward_all(om, x, accumulate="ordered")
    for v, a in acts.items():
        if v == om.out:
            continue
        assert np.array_equal(O.rne_bf16(a), a), f"node {v} not bf16-representable"
    logits = acts[om.out]
    assert not np.array_equal(O.rne_bf16(logits), logits)   # fp32 logits keep low bits


# ---------------------------------------------------------------- Table 1 pins the model builders

def test_table1_parameter_counts():
    with open(os.path.join(GOLDEN, "table1_param_counts.json")) as f:
        rows = json.load(f)["models"]
    for r in rows:
        m = W.make_model(r["graph"], "f32", 0.01, tuple(r["in_hwc"]), r["classes"])
        assert m.n_params() == r["params"], r["row"]
        # the oracle's layer functions produce the shapes the builder declares
        om = O.OracleModel(m)
        x = W.make_inputs(m, 2, "tokens" if any(n.kind == W.EMBED for n in m.nodes) else "uniform")
        acts = O.forward_all(om, x)
        for v, n in enumerate(m.nodes):
            assert acts[v].shape[1:] == tuple(n.out_hwc), (r["row"], v)


# ---------------------------------------------------------------- depthwise conv, ReLU6

def _dw_as_conv(m, v):
    """The depthwise node v as an ordinary CONV2D whose weights are zero off
    the channel diagonal: W_full[o, dy, dx, c] = W_dw[o, dy, dx] if c == o."""
    node = m.nodes[v]
    conv = W.Node(W.CONV2D, node.inputs, node.c_in, node.c_out, node.kh, node.kw, node.stride,
                  node.pad, node.relu, 0, 0, node.out_hwc, node.name)
    wd = O.OracleModel(m).weights[v].reshape(node.c_out, node.kh, node.kw)
    full = np.zeros((node.c_out, node.kh, node.kw, node.c_in), np.float32)
    for c in range(node.c_out):
        full[c, :, :, c] = wd[c]
    return conv, full


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_depthwise_equals_block_diagonal_conv(dtype):
    """A depthwise convolution is a convolution with a block-diagonal weight
    tensor; the oracle's two layer functions (tap loop vs im2col GEMM) agree."""
    m = W.tiny_mobilenet(dtype)
    om = O.OracleModel(m)
    x = W.make_inputs(m, 6, "normal")
    acts = O.forward_all(om, x)
    for v, node in enumerate(m.nodes):
        if node.kind != W.DWCONV:
            continue
        conv, full = _dw_as_conv(m, v)
        nodes = list(m.nodes)
        nodes[v] = conv
        cm = W.Model("dw_as_conv", dtype, nodes, list(m.weights), list(m.biases))
        com = O.OracleModel(cm)
        got = phi(com, v, [acts[node.inputs[0]]], W=full)
        np.testing.assert_allclose(got, acts[v], rtol=1e-6, atol=1e-7)
        assert node.stride in (1, 2)


def test_relu6_clamps_both_ends():
    b = W.configs._Builder((1, 1, 3))
    b.dense(0, 3, relu=2, name="d")
    nodes = b.nodes
    w = np.eye(3, dtype=np.float32) * np.float32(2.0)
    bias = np.array([0.0, -1.0, 1.0], np.float32)
    m = W.Model("relu6", "f32", nodes, [None, w], [None, bias])
    x = np.array([[[[-1.0, 1.0, 4.0]]], [[[0.25, 3.5, 2.5]]]], np.float32)
    z = phi(O.OracleModel(m), 1, [x]).reshape(2, 3)
    # 2x + b: (-2, 1, 9) -> (0, 1, 6); (0.5, 6, 6) -> (0.5, 6, 6)
    np.testing.assert_array_equal(z, np.array([[0, 1, 6], [0.5, 6, 6]], np.float32))


def test_mobilenetv2_shape_and_parameters():
    """Inverted residuals: identity ADD only at stride 1 with equal channels;
    the depthwise layers hold 9 weights per channel."""
    m = W.make_model("mobilenetv2", "bf16", 0.01)
    kinds = [n.kind for n in m.nodes]
    assert kinds.count(W.DWCONV) == sum(n for (_, _, n, _) in W.configs.MOBILENETV2_BLOCKS)
    for v, n in enumerate(m.nodes):
        if n.kind == W.DWCONV:
            assert m.weights[v].shape == (n.c_out, 3, 3) and n.fan_in == 9 and n.relu == 2
        if n.kind == W.ADD:
            a, s = (m.nodes[i] for i in n.inputs)
            assert a.out_hwc == s.out_hwc and n.relu == 0
    assert m.nodes[-1].out_hwc == (1, 1, 10)
    assert m.n_params() == 215210


# ---------------------------------------------------------------- embedding, LSTM

def test_embedding_and_lstm_match_torch():
    """The oracle's embedding lookup and LSTM recursion against torch's
    float64 reference modules with the same parameters (gate order input,
    forget, cell, output; one bias per gate)."""
    m = W.tiny_rnn()
    om = O.OracleModel(m)
    x = W.make_inputs(m, 6, "tokens")
    acts = O.forward_all(om, x)
    emb, l1, l2 = 1, 2, 3
    E = om.weights[emb].reshape(m.nodes[emb].c_out, m.nodes[emb].c_in)      # [D][V]
    tok = torch.from_numpy(x.reshape(6, -1).astype(np.int64))
    ref = F.embedding(tok, torch.from_numpy(E.T.astype(np.float64)))
    np.testing.assert_array_equal(acts[emb].reshape(6, -1, E.shape[0]), ref.numpy().astype(np.float32))
    for v in (l1, l2):
        node = m.nodes[v]
        d, hu = node.c_in, node.c_out
        Wr = om.weights[v].reshape(hu, 4, d + hu + 1).astype(np.float64)
        mod = torch.nn.LSTM(d, hu, batch_first=True).double()
        with torch.no_grad():
            mod.weight_ih_l0.copy_(torch.from_numpy(Wr[:, :, :d].transpose(1, 0, 2).reshape(4 * hu, d)))
            mod.weight_hh_l0.copy_(torch.from_numpy(Wr[:, :, d:d + hu].transpose(1, 0, 2).reshape(4 * hu, hu)))
            mod.bias_ih_l0.copy_(torch.from_numpy(Wr[:, :, -1].T.reshape(4 * hu)))
            mod.bias_hh_l0.zero_()
        inp = torch.from_numpy(acts[node.inputs[0]].reshape(6, -1, d).astype(np.float64))
        with torch.no_grad():
            y, _ = mod(inp)
        want = y.numpy() if node.seq else y.numpy()[:, -1:, :]
        np.testing.assert_allclose(acts[v].reshape(want.shape), want, rtol=2e-6, atol=2e-6)


def test_lstm_effect_block_silences_the_unit():
    """Zeroing a unit's incoming weights and gate biases gives i = f = o = 1/2
    and g = 0 at every step, so c and h stay exactly 0."""
    m = W.tiny_rnn()
    om = O.OracleModel(m)
    x = W.make_inputs(m, 5, "tokens")
    l1 = 2
    muts = W.Mutants(1, np.array([0], np.int32), np.array([W.NEB], np.int32), np.array([l1], np.int32),
                     np.array([1], np.int32), np.array([-1], np.int32), [None])
    Wm, Bm, _ = O.apply_records(om, muts, 0)
    acts = O.forward_all(om, x, Wm, Bm)
    assert np.all(acts[l1][..., 1] == 0)
    assert np.any(acts[l1][..., 0] != 0)
