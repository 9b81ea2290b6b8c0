"""The five synthetic workloads and two tiny test networks.

The paper's models and datasets (Table 1) are not available, so every workload
is synthetic: He-normal weights, i.i.d. inputs with the shape of the dataset
they stand in for (MNIST-like 28x28x1, CIFAR-like 32x32x3, a 64x64x3
200-class set), and mutation records drawn like the paper's neuron-level
mutators with a selection ratio (Section 3.1).  No dataset item is used.

Recipe (all draws with ``numpy.random.default_rng``):
  * weights: seed 0, in topological order, each weighted node draws its
    weight tensor (C order, ``[C_out][kh][kw][C_in]`` or ``[C_out][C_in]``)
    from N(0, 2/fan_in) in float64, then its bias (zero for the MLP,
    N(0, 0.01^2) otherwise); stored float32, or rounded to bfloat16 through
    float32 for the bf16 models;
  * inputs: seed 1, U[0,1) (fp32 models) or N(0,1) (bf16 models), NHWC;
  * mutants: seed [2, variant], mutant by mutant: one operator uniform over
    {GF, NEB, NAI, NS}, ``k`` neurons, then per neuron an NS partner (uniform
    over the other neurons of its layer) and GF noise N(0, sigma^2) with
    sigma = 0.1 * (population std of that layer's stored weights).

Every draw is sequential, so the first ``n`` inputs or mutants of a workload
do not depend on how many are drawn.
"""
from __future__ import annotations

import math
from typing import Dict, List, Optional, Sequence, Tuple

import numpy as np

from .graph import (INPUT, DENSE, CONV2D, ADD, GAP, FLATTEN, DWCONV, EMBED, LSTM, GF, NEB, NAI, NS,
                    WS, Node, Model, Mutants, Workload)


# --------------------------------------------------------------------------
# graph construction


class _Builder:
    def __init__(self, hwc: Tuple[int, int, int]):
        self.nodes: List[Node] = [Node(INPUT, (), out_hwc=tuple(hwc), name="input")]

    def conv(self, src, c_out, k, stride=1, pad=0, relu=True, pool=0, name=""):
        h, w, c = self.nodes[src].out_hwc
        ho = (h + 2 * pad - k) // stride + 1
        wo = (w + 2 * pad - k) // stride + 1
        if pool:
            ho, wo = ho // pool, wo // pool
        self.nodes.append(Node(CONV2D, (src,), c, c_out, k, k, stride, pad, int(relu),
                               pool, 0, (ho, wo, c_out), name))
        return len(self.nodes) - 1

    def dwconv(self, src, k, stride=1, pad=0, relu=2, name=""):
        h, w, c = self.nodes[src].out_hwc
        ho = (h + 2 * pad - k) // stride + 1
        wo = (w + 2 * pad - k) // stride + 1
        self.nodes.append(Node(DWCONV, (src,), c, c, k, k, stride, pad, int(relu),
                               0, 0, (ho, wo, c), name))
        return len(self.nodes) - 1

    def embed(self, src, vocab, dim, name=""):
        h, t, c = self.nodes[src].out_hwc
        assert h == 1 and c == 1, "an embedding reads a [1][T][1] token sequence"
        self.nodes.append(Node(EMBED, (src,), vocab, dim, out_hwc=(1, t, dim), name=name))
        return len(self.nodes) - 1

    def lstm(self, src, units, seq, name=""):
        h, t, c = self.nodes[src].out_hwc
        assert h == 1
        self.nodes.append(Node(LSTM, (src,), c, units, out_hwc=(1, t if seq else 1, units),
                               name=name, seq=int(seq)))
        return len(self.nodes) - 1

    def dense(self, src, c_out, relu=True, name=""):
        h, w, c = self.nodes[src].out_hwc
        self.nodes.append(Node(DENSE, (src,), h * w * c, c_out, 1, 1, 1, 0, int(relu),
                               0, 0, (1, 1, c_out), name))
        return len(self.nodes) - 1

    def add(self, a, skip, relu=True, shortcut=0, name=""):
        ha = self.nodes[a].out_hwc
        self.nodes.append(Node(ADD, (a, skip), self.nodes[skip].out_hwc[2], ha[2],
                               relu=int(relu), shortcut=shortcut, out_hwc=ha, name=name))
        return len(self.nodes) - 1

    def flatten(self, src, name="flatten"):
        h, w, c = self.nodes[src].out_hwc
        self.nodes.append(Node(FLATTEN, (src,), c, h * w * c, out_hwc=(1, 1, h * w * c), name=name))
        return len(self.nodes) - 1

    def gap(self, src, name="gap"):
        c = self.nodes[src].out_hwc[2]
        self.nodes.append(Node(GAP, (src,), c, c, out_hwc=(1, 1, c), name=name))
        return len(self.nodes) - 1


def _basic_block(b, src, c_out, stride, shortcut_kind, name):
    """conv3x3(s)+ReLU -> conv3x3 -> ADD(+ReLU) with the block input.

    shortcut_kind: "identity", "optionA" (subsample + zero-pad channels) or
    "proj" (1x1 stride-s conv placed before conv_a in topological order)."""
    skip = src
    if shortcut_kind == "proj":
        skip = b.conv(src, c_out, 1, stride=stride, pad=0, relu=False, name=name + ".proj")
    a = b.conv(src, c_out, 3, stride=stride, pad=1, relu=True, name=name + ".a")
    c = b.conv(a, c_out, 3, stride=1, pad=1, relu=False, name=name + ".b")
    return b.add(c, skip, relu=True, shortcut=1 if shortcut_kind == "optionA" else 0,
                 name=name + ".add")


def _inverted_residual(b, src, expand, c_out, stride, name):
    """MobileNetV2 block: 1x1 expansion (ReLU6, skipped when expand == 1), 3x3
    depthwise (stride s, ReLU6), 1x1 linear projection, and an identity ADD
    (no activation) when the stride is 1 and the channels agree."""
    c_in = b.nodes[src].out_hwc[2]
    x = src
    if expand != 1:
        x = b.conv(x, c_in * expand, 1, relu=2, name=name + ".expand")
    x = b.dwconv(x, 3, stride=stride, pad=1, relu=2, name=name + ".dw")
    x = b.conv(x, c_out, 1, relu=0, name=name + ".project")
    if stride == 1 and c_in == c_out:
        x = b.add(x, src, relu=0, name=name + ".add")
    return x


LSTM_VOCAB, LSTM_STEPS = 2000, 40
# the paper's RNN (Table 1): a 20,000-token vocabulary embedded in 128
# features, two 64-unit LSTM layers; sequences of 80 tokens
RNN_VOCAB, RNN_EMBED, RNN_UNITS, RNN_STEPS = 20000, 128, 64, 80


def lstm_bias_positions(node: Node) -> np.ndarray:
    """Positions of the four gate biases in an LSTM unit's weight row."""
    k = node.c_in + node.c_out + 1
    return np.arange(4) * k + (k - 1)


# MobileNetV2 for 32x32 inputs: (expansion t, channels c, repeats n, stride s)
MOBILENETV2_BLOCKS = ((1, 8, 1, 1), (6, 16, 2, 2), (6, 24, 3, 2), (6, 48, 3, 2), (6, 64, 2, 1))


def _graph(name: str, hwc=None, classes: int = 10) -> List[Node]:
    if name == "mlp":
        b = _Builder(hwc or (1, 1, 784))
        x = b.dense(0, 128, True, "L1")
        x = b.dense(x, 64, True, "L2")
        b.dense(x, classes, False, "L3")
    elif name == "fcnn":                     # the paper's 4-layer FCNN (Table 1)
        b = _Builder(hwc or (1, 1, 784))
        x = b.dense(0, 50, True, "D1")
        x = b.dense(x, 50, True, "D2")
        x = b.dense(x, 50, True, "D3")
        b.dense(x, classes, False, "D4")
    elif name == "lenet5":
        b = _Builder(hwc or (28, 28, 1))
        x = b.conv(0, 6, 5, relu=True, pool=2, name="C1")
        x = b.conv(x, 16, 5, relu=True, pool=2, name="C2")
        x = b.dense(x, 120, True, "F1")
        x = b.dense(x, 84, True, "F2")
        b.dense(x, classes, False, "F3")
    elif name == "vgg":
        b = _Builder((32, 32, 3))
        x = b.conv(0, 64, 3, pad=1, name="C1")
        x = b.conv(x, 64, 3, pad=1, pool=2, name="C2")
        x = b.conv(x, 128, 3, pad=1, name="C3")
        x = b.conv(x, 128, 3, pad=1, pool=2, name="C4")
        x = b.conv(x, 256, 3, pad=1, name="C5")
        x = b.conv(x, 256, 3, pad=1, pool=2, name="C6")
        x = b.dense(x, 256, True, "F1")
        b.dense(x, 10, False, "F2")
    elif name == "resnet20":
        b = _Builder((32, 32, 3))
        x = b.conv(0, 16, 3, pad=1, name="stem")
        for s, c in enumerate((16, 32, 64)):
            for k in range(3):
                first = (k == 0 and s > 0)
                x = _basic_block(b, x, c, 2 if first else 1,
                                 "optionA" if first else "identity", f"s{s}b{k}")
        x = b.gap(x)
        b.dense(x, classes, False, "fc")
    elif name == "resnet18w":
        b = _Builder((64, 64, 3))
        x = b.conv(0, 64, 3, pad=1, name="stem")
        for s, c in enumerate((64, 128, 256, 512)):
            for k in range(2):
                first = (k == 0 and s > 0)
                x = _basic_block(b, x, c, 2 if first else 1,
                                 "proj" if first else "identity", f"s{s}b{k}")
        x = b.gap(x)
        b.dense(x, 200 if classes == 10 else classes, False, "fc")
    elif name == "mobilenetv2":
        b = _Builder((32, 32, 3))
        x = b.conv(0, 16, 3, pad=1, relu=2, name="stem")
        for bi, (t, c, n, s) in enumerate(MOBILENETV2_BLOCKS):
            for r in range(n):
                x = _inverted_residual(b, x, t, c, s if r == 0 else 1, f"b{bi}.{r}")
        x = b.conv(x, 320, 1, relu=2, name="head")
        x = b.gap(x)
        b.dense(x, classes, False, "fc")
    elif name == "lstm":
        # embedding, two LSTM layers (the first returns its sequence), output
        # layer (the paper's RNN shape; softmax does not change the argmax)
        b = _Builder(hwc or (1, LSTM_STEPS, 1))
        x = b.embed(0, LSTM_VOCAB, 32, name="embed")
        x = b.lstm(x, 32, seq=1, name="lstm1")
        x = b.lstm(x, 32, seq=0, name="lstm2")
        b.dense(x, 2 if classes == 10 else classes, False, "out")
    elif name == "rnn":
        # Table 1's RNN: embedding 20,000 x 128, LSTM 64 (sequence), LSTM 64,
        # dense output (2 classes for IMDB, 90 for Reuters)
        b = _Builder(hwc or (1, RNN_STEPS, 1))
        x = b.embed(0, RNN_VOCAB, RNN_EMBED, name="embed")
        x = b.lstm(x, RNN_UNITS, seq=1, name="lstm1")
        x = b.lstm(x, RNN_UNITS, seq=0, name="lstm2")
        b.dense(x, 2 if classes == 10 else classes, False, "out")
    else:
        raise KeyError(name)
    return b.nodes


# --------------------------------------------------------------------------
# weights / inputs


def _to_bf16_bits(x64: np.ndarray) -> np.ndarray:
    """float64 draw -> float32 -> bfloat16 bit pattern (uint16), via torch's
    CPU conversion (data preparation only)."""
    import torch
    t = torch.from_numpy(np.ascontiguousarray(x64, dtype=np.float32))
    return t.to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16).copy()


def bf16_bits_to_f32(bits: np.ndarray) -> np.ndarray:
    return (bits.astype(np.uint32) << 16).view(np.float32)


def _draw_weights(nodes: List[Node], dtype: str, bias_std: float, seed: int = 0):
    rng = np.random.default_rng(seed)
    weights: List[Optional[np.ndarray]] = []
    biases: List[Optional[np.ndarray]] = []
    for n in nodes:
        if not n.weighted:
            weights.append(None)
            biases.append(None)
            continue
        if n.kind == CONV2D:
            shape = (n.c_out, n.kh, n.kw, n.c_in)
        elif n.kind == DWCONV:
            shape = (n.c_out, n.kh, n.kw)
        elif n.kind in (EMBED, LSTM):
            shape = (n.c_out, n.fan_in)
        else:
            shape = (n.c_out, n.c_in)
        if n.kind == EMBED:                       # unit-scale token vectors
            w64 = rng.standard_normal(shape)
        elif n.kind == LSTM:                      # N(0, 1/(D+H)); gate biases 0, forget gate 1
            w64 = rng.standard_normal(shape) * math.sqrt(1.0 / (n.c_in + n.c_out))
            pos = lstm_bias_positions(n)
            w64[:, pos] = 0.0
            w64[:, pos[1]] = 1.0
        else:
            w64 = rng.standard_normal(shape) * math.sqrt(2.0 / n.fan_in)
        weights.append(w64.astype(np.float32) if dtype == "f32" else _to_bf16_bits(w64))
        if bias_std > 0 and n.kind not in (EMBED, LSTM):
            biases.append((rng.standard_normal(n.c_out) * bias_std).astype(np.float32))
        else:
            biases.append(np.zeros(n.c_out, np.float32))
    return weights, biases


def make_inputs(model: Model, n: int, dist: str, seed: int = 1,
                chunk: int = 1024) -> np.ndarray:
    rng = np.random.default_rng(seed)
    h, w, c = model.in_hwc
    out = np.empty((n, h, w, c), np.float32 if model.dtype == "f32" else np.uint16)
    for s in range(0, n, chunk):
        e = min(n, s + chunk)
        if dist == "uniform":
            x = rng.random((e - s, h, w, c))
        elif dist == "tokens":                    # token ids, uniform over the vocabulary
            vocab = next(n.c_in for n in model.nodes if n.kind == EMBED)
            x = rng.integers(0, vocab, size=(e - s, h, w, c)).astype(np.float64)
        else:
            x = rng.standard_normal((e - s, h, w, c))
        out[s:e] = x.astype(np.float32) if model.dtype == "f32" else _to_bf16_bits(x)
    return out


# --------------------------------------------------------------------------
# mutants


def neuron_layers(model: Model) -> List[int]:
    """Weighted nodes, in topological order (every output channel is a neuron)."""
    return model.weighted_nodes()


def _layer_std(model: Model, li: int) -> float:
    w = model.weights[li]
    w64 = (bf16_bits_to_f32(w) if model.dtype == "bf16" else w).astype(np.float64)
    return float(w64.std())


def make_mutants(model: Model, n_mutants: int, k: int, mode: str,
                 candidates: Optional[Sequence[int]] = None,
                 variant: int = 0, ops: Sequence[int] = (GF, NEB, NAI, NS)) -> Mutants:
    """Draw ``n_mutants`` mutants of ``k`` neurons each.

    mode "layer_first": the first mutated layer is uniform over ``candidates``,
    the first neuron uniform in it, the other k-1 uniform (without
    replacement) over neurons of candidate layers at or after it.
    mode "uniform": k neurons uniform without replacement over all neurons of
    ``candidates``."""
    rng = np.random.default_rng([2, variant])
    cands = list(candidates) if candidates is not None else neuron_layers(model)
    pool_layer = np.concatenate([np.full(model.nodes[l].c_out, l, np.int64) for l in cands])
    pool_neuron = np.concatenate([np.arange(model.nodes[l].c_out, dtype=np.int64) for l in cands])
    sigma = {l: 0.1 * _layer_std(model, l) for l in cands}
    mid, opl, lay, neu, par, noise, perms = [], [], [], [], [], [], []
    for m in range(n_mutants):
        op = int(ops[int(rng.integers(len(ops)))])
        if mode == "layer_first":
            l0 = cands[int(rng.integers(len(cands)))]
            n0 = int(rng.integers(model.nodes[l0].c_out))
            rest = np.nonzero((pool_layer >= l0) & ~((pool_layer == l0) & (pool_neuron == n0)))[0]
            # (a first layer near the output may leave fewer than k-1 neurons)
            pick = rng.choice(rest.size, size=min(k - 1, rest.size), replace=False) if k > 1 else []
            sel = [(l0, n0)] + [(int(pool_layer[rest[i]]), int(pool_neuron[rest[i]])) for i in pick]
        elif mode == "uniform":
            pick = rng.choice(pool_layer.size, size=k, replace=False)
            sel = [(int(pool_layer[i]), int(pool_neuron[i])) for i in pick]
        else:
            raise ValueError(mode)
        for (l, i) in sel:
            c_out = model.nodes[l].c_out
            j = -1
            if op == NS:
                j = int(rng.integers(c_out - 1))
                j += int(j >= i)
            node = model.nodes[l]
            eps = None
            if op == GF:
                eps = (rng.standard_normal(node.fan_in) * sigma[l]).astype(np.float32)
                if node.kind == LSTM:             # the gate biases are kept
                    eps[lstm_bias_positions(node)] = 0.0
            perm = None
            if op == WS:
                perm = rng.permutation(node.fan_in).astype(np.int32)
                if node.kind == LSTM:             # shuffle the weights, keep the biases in place
                    pos = lstm_bias_positions(node)
                    keep = np.setdiff1d(np.arange(node.fan_in), pos)
                    perm = np.arange(node.fan_in, dtype=np.int32)
                    perm[keep] = keep[rng.permutation(keep.size)]
            mid.append(m); opl.append(op); lay.append(l); neu.append(i); par.append(j)
            noise.append(eps); perms.append(perm)
    a = lambda v: np.asarray(v, np.int32)
    return Mutants(n_mutants, a(mid), a(opl), a(lay), a(neu), a(par), noise, perms)


def _k(ratio: float, n_neurons: int) -> int:
    return max(1, int(math.floor(ratio * n_neurons + 0.5)))


# --------------------------------------------------------------------------
# the five workloads

CONFIGS: Dict[str, dict] = {
    "mlp": dict(graph="mlp", dtype="f32", bias_std=0.0, n_inputs=500, dist="uniform",
                n_mutants=100, ratio=None, k=1, mode="layer_first", variant=0,
                desc="MLP 784-128-64-10 fp32, 500 inputs U[0,1), 100 mutants of 1 neuron"),
    "lenet5": dict(graph="lenet5", dtype="f32", bias_std=0.01, n_inputs=10000, dist="uniform",
                   n_mutants=1000, ratio=0.01, mode="layer_first", variant=0,
                   desc="LeNet-5 28x28x1 fp32, 10,000 inputs U[0,1), 1,000 mutants at 1%"),
    # mutation ratios 0.1%, 1%, 3%, 5% (the sweep of the paper's RQ2)
    "vgg": dict(graph="vgg", dtype="bf16", bias_std=0.01, n_inputs=10000, dist="normal",
                n_mutants=2000, ratios=(0.001, 0.01, 0.05, 0.03), mode="uniform",
                desc="VGG-style 32x32x3 bf16, 10,000 inputs N(0,1), 2,000 mutants per ratio"),
    "resnet20": dict(graph="resnet20", dtype="bf16", bias_std=0.01, n_inputs=10000, dist="normal",
                     n_mutants=1000, ratio=0.01, mode="layer_first", variant=0,
                     desc="ResNet-20 32x32x3 bf16, 10,000 inputs N(0,1), 1,000 mutants, "
                          "first mutated layer uniform over 19 layers"),
    "mobilenetv2": dict(graph="mobilenetv2", dtype="bf16", bias_std=0.01, n_inputs=10000,
                        dist="normal", n_mutants=1000, ratio=0.01, mode="layer_first", variant=0,
                        desc="MobileNetV2 32x32x3 bf16 (inverted residuals, depthwise 3x3, ReLU6), "
                             "10,000 inputs N(0,1), 1,000 mutants at 1%, first mutated layer "
                             "uniform over the weighted layers"),
    "lstm": dict(graph="lstm", dtype="f32", bias_std=0.0, n_inputs=10000, dist="tokens",
                 n_mutants=1000, ratio=0.01, mode="layer_first", variant=0,
                 desc="RNN: embedding 2000x32, LSTM 32 (sequence), LSTM 32, dense 2, fp32, "
                      "40-token sequences uniform over the vocabulary, 10,000 inputs, "
                      "1,000 mutants at 1%"),
    "rnn_imdb": dict(graph="rnn", dtype="f32", bias_std=0.0, n_inputs=25000, dist="tokens",
                     n_mutants=1000, ratio=0.01, mode="layer_first", variant=0,
                     desc="RNN of Table 1 (IMDB): embedding 20,000x128, LSTM 64 (sequence), LSTM 64, "
                          "dense 2 (2,642,562 parameters), fp32, 80-token sequences uniform over the "
                          "vocabulary, 25,000 inputs, 1,000 mutants at 1%"),
    "resnet18w": dict(graph="resnet18w", dtype="bf16", bias_std=0.01, n_inputs=5000, dist="normal",
                      n_mutants=500, ratio=0.05, mode="uniform", variant=0,
                      desc="ResNet-18-style 64x64x3 bf16 FC200, 5,000 inputs N(0,1), "
                           "500 mutants at 5%"),
}

_MODEL_CACHE: Dict[str, Model] = {}


def make_model(graph: str, dtype: str, bias_std: float, hwc=None, classes: int = 10) -> Model:
    key = f"{graph}/{dtype}/{bias_std}/{hwc}/{classes}"
    if key not in _MODEL_CACHE:
        nodes = _graph(graph, hwc, classes)
        w, b = _draw_weights(nodes, dtype, bias_std, seed=0)
        _MODEL_CACHE[key] = Model(graph, dtype, nodes, w, b)
    return _MODEL_CACHE[key]


def _candidates(graph: str, model: Model) -> List[int]:
    wn = model.weighted_nodes()
    if graph == "resnet20":
        # the 18 block convs and the FC layer (the stem is not a candidate)
        return [i for i in wn if model.nodes[i].name != "stem"]
    return wn


def make_workload(cfg: str, n_inputs: Optional[int] = None, n_mutants: Optional[int] = None,
                  ratio_index: int = 1, ops: Sequence[int] = (GF, NEB, NAI, NS)) -> Workload:
    """Build workload ``cfg`` ("mlp".."resnet18w"); ``n_inputs``/``n_mutants``
    truncate it (prefix-stable); ``ratio_index`` picks vgg's ratio; ``ops``
    the operators drawn (the paper's fourth, weight shuffle, is WS)."""
    c = CONFIGS[cfg]
    model = make_model(c["graph"], c["dtype"], c["bias_std"])
    cands = _candidates(c["graph"], model)
    n_neurons = sum(model.nodes[i].c_out for i in model.weighted_nodes())
    if "ratios" in c:
        ratio = c["ratios"][ratio_index]
        variant = ratio_index
    else:
        ratio = c["ratio"]
        variant = c["variant"]
    k = c.get("k") or _k(ratio, n_neurons)
    ni = c["n_inputs"] if n_inputs is None else n_inputs
    nm = c["n_mutants"] if n_mutants is None else n_mutants
    x = make_inputs(model, ni, c["dist"])
    muts = make_mutants(model, nm, k, c["mode"], cands, variant=variant, ops=ops)
    name = cfg if "ratios" not in c else f"{cfg}_r{ratio:g}"
    return Workload(name, model, x, muts, c["desc"])


# --------------------------------------------------------------------------
# tiny networks for brute-force tests


def tiny_mlp(dtype: str = "f32", seed: int = 5) -> Model:
    """6-5-4-3 MLP."""
    b = _Builder((1, 1, 6))
    x = b.dense(0, 5, True, "h1")
    x = b.dense(x, 4, True, "h2")
    b.dense(x, 3, False, "out")
    w, bb = _draw_weights(b.nodes, dtype, 0.1, seed=seed)
    return Model("tiny_mlp", dtype, b.nodes, w, bb)


def tiny_resnet(dtype: str = "f32", seed: int = 6, shortcut: str = "optionA") -> Model:
    """6x6x2 input; stem 3x3 -> 4; one identity block; one stride-2 block
    (option A or projection); GAP; dense 3.  Boundaries with |K| = 2 occur."""
    b = _Builder((6, 6, 2))
    x = b.conv(0, 4, 3, pad=1, name="stem")
    x = _basic_block(b, x, 4, 1, "identity", "b0")
    x = _basic_block(b, x, 8, 2, shortcut, "b1")
    x = b.gap(x)
    b.dense(x, 3, False, "out")
    w, bb = _draw_weights(b.nodes, dtype, 0.1, seed=seed)
    return Model("tiny_resnet_" + shortcut, dtype, b.nodes, w, bb)


def tiny_lenet(dtype: str = "f32", seed: int = 7) -> Model:
    """10x10x1 input, conv3x3 valid 1->2 +pool, conv3x3 valid 2->3, dense 12->4 -> 3."""
    b = _Builder((10, 10, 1))
    x = b.conv(0, 2, 3, relu=True, pool=2, name="c1")
    x = b.conv(x, 3, 3, relu=True, pool=0, name="c2")
    x = b.dense(x, 4, True, "f1")
    b.dense(x, 3, False, "f2")
    w, bb = _draw_weights(b.nodes, dtype, 0.1, seed=seed)
    return Model("tiny_lenet", dtype, b.nodes, w, bb)


def tiny_mobilenet(dtype: str = "f32", seed: int = 8) -> Model:
    """6x6x3 input; stem 3x3 -> 4 (ReLU6); an inverted residual with identity
    ADD (expand 2, depthwise stride 1); one with stride 2 and no ADD; GAP;
    dense 3."""
    b = _Builder((6, 6, 3))
    x = b.conv(0, 4, 3, pad=1, relu=2, name="stem")
    x = _inverted_residual(b, x, 2, 4, 1, "r0")
    x = _inverted_residual(b, x, 2, 6, 2, "r1")
    x = b.gap(x)
    b.dense(x, 3, False, "out")
    w, bb = _draw_weights(b.nodes, dtype, 0.1, seed=seed)
    return Model("tiny_mobilenet", dtype, b.nodes, w, bb)


def tiny_rnn(dtype: str = "f32", seed: int = 9) -> Model:
    """Tokens [1][5][1] over a 7-word vocabulary; embedding 3; LSTM 4
    (sequence); LSTM 3 (last state); dense 3."""
    b = _Builder((1, 5, 1))
    x = b.embed(0, 7, 3, name="embed")
    x = b.lstm(x, 4, seq=1, name="lstm1")
    x = b.lstm(x, 3, seq=0, name="lstm2")
    b.dense(x, 3, False, "out")
    w, bb = _draw_weights(b.nodes, dtype, 0.1, seed=seed)
    return Model("tiny_rnn", dtype, b.nodes, w, bb)
