"""Layer functions Phi(v) and the activation recursion a_v (Section 4).

Semantics (the same on both sides of the parity check; see the design notes):
  * tensors are NHWC; a DENSE layer reads its input flattened in HWC order;
  * CONV2D: cross-correlation with stride s and zero padding p,
      acc[n,i,j,o] = sum_{dy,dx,c} x[n, i*s+dy-p, j*s+dx-p, c] * W[o,dy,dx,c],
    then t = fl32(acc + b[o]), optional activation, optional 2x2 stride-2
    max-pool (floor), then the node-output rounding;
  * DWCONV (depthwise): the same with each output channel reading only its
    own input channel,
      acc[n,i,j,c] = sum_{dy,dx} x[n, i*s+dy-p, j*s+dx-p, c] * W[c,dy,dx];
  * DENSE: t = fl32(sum_c x[n,c] * W[o,c] + b[o]), optional activation,
    rounding;
  * activation: ReLU max(t, 0) or ReLU6 min(max(t, 0), 6), in float32;
  * EMBED: out[n,0,t,d] = W[d, token], the token id being the input value;
  * LSTM (float32 models): for t = 0..T-1, with h = c = 0 at the start and
    each unit's row holding, per gate (input, forget, cell, output), its input
    weights, recurrent weights and bias,
      z_q = fl32(x_t . Wx_q + h . Wh_q + b_q)                (float64 sums),
      i, f, o = fl32(sigmoid(z)), g = fl32(tanh(z_g))        (float64, rounded),
      c = fl32(f*c + i*g),  h = fl32(o * fl32(tanh(c)));
    the output is every step's h, or the last one;
  * ADD: t = fl32(a + s) computed in float32, where s is the second input,
    for option A first subsampled s[:, ::2, ::2, :] and zero-padded in the
    channel dimension ((C_a - C_s)//2 zero channels before, the rest after);
    optional activation; rounding;
  * GAP: t = fl32(mean over H and W); rounding;
  * FLATTEN: a view.
  * Node-output rounding: bf16 models round every node output except the
    network output (the logits) to bfloat16 (round to nearest even); fp32
    models keep float32 everywhere.
The dot products are accumulated in float64 ("blas": numpy/BLAS, or
"ordered": a fixed sequential order over the reduction index, used where
bit-identity between two oracle evaluations is tested).
"""
from __future__ import annotations

from typing import Dict, List, Optional, Sequence

import numpy as np
from numpy.lib.stride_tricks import sliding_window_view

from workloads.graph import INPUT, DENSE, CONV2D, ADD, GAP, FLATTEN, DWCONV, EMBED, LSTM, Model
from .numerics import rne_bf16, bf16_bits_to_f32, to_f32


class OracleModel:
    """The oracle's view of a model: float32 weights (bf16 values widened)."""

    def __init__(self, model: Model):
        self.name = model.name
        self.nodes = model.nodes
        self.dtype = model.dtype
        bf = model.dtype == "bf16"
        self.weights = [None if w is None else
                        (bf16_bits_to_f32(w) if bf else np.asarray(w, np.float32))
                        for w in model.weights]
        self.biases = [None if b is None else np.asarray(b, np.float32) for b in model.biases]
        self.out = len(self.nodes) - 1

    def input_values(self, X: np.ndarray) -> np.ndarray:
        return bf16_bits_to_f32(X) if self.dtype == "bf16" else np.asarray(X, np.float32)


def _round_node(model: OracleModel, v: int, t32: np.ndarray) -> np.ndarray:
    if model.dtype == "bf16" and v != model.out:
        return rne_bf16(t32)
    return t32


def _act(t: np.ndarray, relu: int) -> np.ndarray:
    """The node's activation on float32 values: 1 ReLU, 2 ReLU6."""
    if relu:
        t = np.maximum(t, np.float32(0))
    if relu == 2:
        t = np.minimum(t, np.float32(6))
    return t


def _matmul64(a64: np.ndarray, w2: np.ndarray, accumulate: str) -> np.ndarray:
    """a64 [R, K] float64, w2 [C_out, K] -> [R, C_out] float64."""
    w64 = w2.astype(np.float64)
    if accumulate == "blas":
        return a64 @ w64.T
    acc = np.zeros((a64.shape[0], w64.shape[0]), np.float64)
    for k in range(a64.shape[1]):
        acc += a64[:, k:k + 1] * w64[None, :, k]
    return acc


def _im2col(x64: np.ndarray, kh: int, kw: int, s: int, p: int) -> np.ndarray:
    n, h, w, c = x64.shape
    xp = np.pad(x64, ((0, 0), (p, p), (p, p), (0, 0))) if p else x64
    win = sliding_window_view(xp, (kh, kw), axis=(1, 2))      # [n, H', W', c, kh, kw]
    win = win[:, ::s, ::s]
    ho, wo = win.shape[1], win.shape[2]
    cols = np.ascontiguousarray(win.transpose(0, 1, 2, 4, 5, 3))  # [n, ho, wo, kh, kw, c]
    return cols.reshape(n * ho * wo, kh * kw * c), ho, wo


def phi(model: OracleModel, v: int, ins: Sequence[np.ndarray], W=None, b=None,
        accumulate: str = "blas") -> np.ndarray:
    """Layer function of node v applied to its input activations ``ins``."""
    node = model.nodes[v]
    W = model.weights[v] if W is None else W
    b = model.biases[v] if b is None else b
    if node.kind == DENSE:
        x = ins[0]
        n = x.shape[0]
        acc = _matmul64(x.reshape(n, -1).astype(np.float64), W, accumulate)
        t = _act(to_f32(acc + b.astype(np.float64)[None, :]), node.relu)
        return _round_node(model, v, t.reshape(n, 1, 1, node.c_out))
    if node.kind == CONV2D:
        x = ins[0]
        n = x.shape[0]
        cols, ho, wo = _im2col(x.astype(np.float64), node.kh, node.kw, node.stride, node.pad)
        acc = _matmul64(cols, W.reshape(node.c_out, -1), accumulate)
        t = _act(to_f32(acc + b.astype(np.float64)[None, :]).reshape(n, ho, wo, node.c_out), node.relu)
        if node.maxpool:
            q = node.maxpool
            h2, w2 = ho // q, wo // q
            t = t[:, :h2 * q, :w2 * q].reshape(n, h2, q, w2, q, node.c_out).max(axis=(2, 4))
        return _round_node(model, v, np.ascontiguousarray(t))
    if node.kind == DWCONV:
        x = ins[0].astype(np.float64)
        n, h, w, c = x.shape
        p, st = node.pad, node.stride
        xp = np.pad(x, ((0, 0), (p, p), (p, p), (0, 0))) if p else x
        ho = (h + 2 * p - node.kh) // st + 1
        wo = (w + 2 * p - node.kw) // st + 1
        W64 = W.reshape(c, node.kh, node.kw).astype(np.float64)
        acc = np.zeros((n, ho, wo, c), np.float64)
        for dy in range(node.kh):                  # taps in (dy, dx) order
            for dx in range(node.kw):
                tap = xp[:, dy:dy + st * (ho - 1) + 1:st, dx:dx + st * (wo - 1) + 1:st, :]
                acc += tap * W64[None, None, None, :, dy, dx]
        t = _act(to_f32(acc + b.astype(np.float64)[None, None, None, :]), node.relu)
        return _round_node(model, v, np.ascontiguousarray(t))
    if node.kind == EMBED:
        x = ins[0]
        n, t = x.shape[0], x.shape[2]
        tok = x.reshape(n, t)
        ids = tok.astype(np.int64)
        if not np.array_equal(ids, tok) or ids.min() < 0 or ids.max() >= node.c_in:
            raise ValueError(f"node {v}: token ids must be integers in [0, {node.c_in})")
        out = np.asarray(W).reshape(node.c_out, node.c_in)[:, ids]         # [D, n, T]
        return _round_node(model, v, np.ascontiguousarray(out.transpose(1, 2, 0)).reshape(n, 1, t, node.c_out))
    if node.kind == LSTM:
        if model.dtype != "f32":
            raise ValueError("LSTM layers are defined for float32 models")
        x = ins[0]
        n, t, d = x.shape[0], x.shape[2], x.shape[3]
        hu = node.c_out
        Wr = np.asarray(W, np.float64).reshape(hu, 4, d + hu + 1)
        h = np.zeros((n, hu), np.float32)
        c = np.zeros((n, hu), np.float32)
        outs = []
        sig = lambda z: to_f32(1.0 / (1.0 + np.exp(-z.astype(np.float64))))
        th = lambda z: to_f32(np.tanh(z.astype(np.float64)))
        for step in range(t):
            a64 = np.concatenate([x[:, 0, step, :], h, np.ones((n, 1), np.float32)], axis=1).astype(np.float64)
            z = [to_f32(_matmul64(a64, Wr[:, q, :], accumulate)) for q in range(4)]
            i, f, g, o = sig(z[0]), sig(z[1]), th(z[2]), sig(z[3])
            c = to_f32(f.astype(np.float64) * c + i.astype(np.float64) * g)
            h = to_f32(o.astype(np.float64) * th(c))
            outs.append(h)
        y = np.stack(outs, axis=1) if node.seq else outs[-1][:, None, :]
        return y.reshape(n, 1, y.shape[1], hu)
    if node.kind == ADD:
        a, s = ins
        if node.shortcut == 1:
            s = s[:, ::2, ::2, :]
            extra = a.shape[3] - s.shape[3]
            before = extra // 2
            s = np.pad(s, ((0, 0), (0, 0), (0, 0), (before, extra - before)))
        t = _act(a.astype(np.float32) + s.astype(np.float32), node.relu)   # float32 addition
        return _round_node(model, v, t)
    if node.kind == GAP:
        x = ins[0]
        n, h, w, c = x.shape
        m = x.astype(np.float64).sum(axis=(1, 2)) * (1.0 / (h * w))
        return _round_node(model, v, to_f32(m).reshape(n, 1, 1, c))
    if node.kind == FLATTEN:
        x = ins[0]
        return x.reshape(x.shape[0], 1, 1, -1)
    raise ValueError(f"node {v}: kind {node.kind} has no layer function")


def forward_all(model: OracleModel, X: np.ndarray, weights=None, biases=None,
                accumulate: str = "blas", keep: Optional[Sequence[int]] = None,
                chunk: int = 256, last: Optional[int] = None) -> Dict[int, np.ndarray]:
    """Activations a_v(x) of every node (or of ``keep``) for all inputs.

    a_v(x) = x for the input node, Phi(v)(a_p(x) for p in Pred(v)) otherwise
    (Section 4).  ``weights``/``biases`` override per-node parameters (a
    mutant's Phi').  ``last``: compute the nodes up to that index only (every
    node of ``keep`` must be among them)."""
    xs = model.input_values(X)
    keep = set(range(len(model.nodes))) if keep is None else set(keep)
    n_run = len(model.nodes) if last is None else last + 1
    if any(v >= n_run for v in keep):
        raise ValueError("a kept node lies after the last computed node")
    parts: Dict[int, List[np.ndarray]] = {v: [] for v in keep}
    last_use = {}
    for v, node in enumerate(model.nodes):
        for p in node.inputs:
            last_use[p] = v
    for s in range(0, xs.shape[0], chunk):
        acts: Dict[int, np.ndarray] = {0: xs[s:s + chunk]}
        for v in range(1, n_run):
            node = model.nodes[v]
            W = weights[v] if weights is not None else None
            b = biases[v] if biases is not None else None
            acts[v] = phi(model, v, [acts[p] for p in node.inputs], W, b, accumulate)
            for p in node.inputs:           # drop activations nobody reads again
                if last_use.get(p) == v and p not in keep:
                    del acts[p]
        for v in keep:
            parts[v].append(acts[v])
    return {v: np.concatenate(p, axis=0) for v, p in parts.items()}


def forward(model: OracleModel, X: np.ndarray, weights=None, biases=None,
            accumulate: str = "blas", chunk: int = 256) -> np.ndarray:
    """M(x): the float32 logits [N, C] of the output node."""
    out = forward_all(model, X, weights, biases, accumulate, keep=[model.out], chunk=chunk)
    z = out[model.out].reshape(X.shape[0], -1)
    if not np.all(np.isfinite(z)):
        raise FloatingPointError("non-finite logits")
    return z
