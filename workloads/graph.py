"""Plain data containers for a model graph and a set of mutation records.

A model is a DAG given in topological order (Section 4: the order tau); node
``i`` lists the indices of the nodes it reads (the dependence graph of
Algorithm 2 stated explicitly), every index smaller than ``i``.  Node 0 is the
single input, the last node is the single output (logits).

Kinds: INPUT, DENSE, CONV2D (bias, optional activation and 2x2/2 max-pool
fused into the node), ADD (two inputs, optional activation, optional "option
A" shortcut: subsample the second input by 2 in H and W and zero-pad its
channels evenly), GAP (global average pool to 1x1xC), FLATTEN (a view, HWC
order), DWCONV (depthwise convolution: output channel c filters input channel
c only; C_in = C_out), EMBED (token embedding: input values are token ids,
output [1][T][D]), LSTM (a long short-term memory layer over the T steps of
its [1][T][D] input; output the whole sequence [1][T][H] or, with ``seq`` = 0,
the last hidden state [1][1][H]).

Activation (``relu``): 0 none, 1 ReLU, 2 ReLU6 (min(max(x, 0), 6)).

Weights: CONV2D ``[C_out][kh][kw][C_in]``; DWCONV ``[C][kh][kw]``; DENSE
``[C_out][C_in]`` where the C_in index runs over the flattened HWC input;
EMBED ``[D][V]`` (neuron d's incoming weights are its value for every token);
LSTM ``[H][4][D + H + 1]``: unit j's incoming weights are, for each gate in
the order input, forget, cell, output, its D input weights, its H recurrent
weights and the gate's bias (the node's own bias array is unused and zero).  fp32 models hold float32
arrays; bf16 models hold uint16 arrays of bfloat16 bit patterns.  Biases are
float32 ``[C_out]``.

Mutation records (one per mutated neuron, Section 3.1 and Section 4):
``op`` in {GF, NEB, NAI, NS, WS}; ``layer`` is a weighted node's index;
``neuron`` an output channel (a neuron of a conv layer is one filter, Section
2.1); ``partner`` the other neuron of a switch; GF records carry their noise,
``fan_in`` float32 values in the row order of ``W[neuron]``; WS records a
permutation of ``0..fan_in-1``.
"""
from __future__ import annotations

from dataclasses import dataclass, field
from typing import List, Optional, Tuple

import numpy as np

INPUT, DENSE, CONV2D, ADD, GAP, FLATTEN, DWCONV, EMBED, LSTM = 0, 1, 2, 3, 4, 5, 6, 7, 8
KIND_NAMES = {INPUT: "input", DENSE: "dense", CONV2D: "conv2d", ADD: "add",
              GAP: "gap", FLATTEN: "flatten", DWCONV: "dwconv", EMBED: "embed", LSTM: "lstm"}

# mutation operators (Section 3.1): Gaussian fuzzing, neuron effect block,
# neuron activation inverse, neuron switch, weight shuffle
GF, NEB, NAI, NS, WS = 0, 1, 2, 3, 4
OP_NAMES = {GF: "GF", NEB: "NEB", NAI: "NAI", NS: "NS", WS: "WS"}


@dataclass
class Node:
    kind: int
    inputs: Tuple[int, ...] = ()
    c_in: int = 0
    c_out: int = 0
    kh: int = 1
    kw: int = 1
    stride: int = 1
    pad: int = 0
    relu: int = 0             # 0 none, 1 ReLU, 2 ReLU6
    maxpool: int = 0          # 0 or 2
    shortcut: int = 0         # ADD only: 0 identity, 1 option A
    out_hwc: Tuple[int, int, int] = (0, 0, 0)
    name: str = ""
    seq: int = 0              # LSTM only: 1 = output every step, 0 = the last one

    @property
    def weighted(self) -> bool:
        return self.kind in (DENSE, CONV2D, DWCONV, EMBED, LSTM)

    @property
    def fan_in(self) -> int:
        if self.kind == DWCONV:
            return self.kh * self.kw
        if self.kind == LSTM:
            return 4 * (self.c_in + self.c_out + 1)
        return self.c_in * self.kh * self.kw


@dataclass
class Model:
    name: str
    dtype: str                      # "f32" or "bf16"
    nodes: List[Node]
    weights: List[Optional[np.ndarray]]
    biases: List[Optional[np.ndarray]]

    @property
    def in_hwc(self) -> Tuple[int, int, int]:
        return self.nodes[0].out_hwc

    @property
    def n_classes(self) -> int:
        return self.nodes[-1].out_hwc[2]

    def n_params(self) -> int:
        """Trainable parameters: every weight array, and the bias arrays of the
        kinds that use theirs (an embedding has none, an LSTM keeps its gate
        biases inside its weight rows)."""
        return int(sum(w.size for w in self.weights if w is not None)
                   + sum(b.size for b, n in zip(self.biases, self.nodes)
                         if b is not None and n.kind not in (EMBED, LSTM)))

    def weighted_nodes(self) -> List[int]:
        return [i for i, n in enumerate(self.nodes) if n.weighted]


@dataclass
class Mutants:
    n_mutants: int
    mutant_id: np.ndarray           # int32 [R]
    op: np.ndarray                  # int32 [R]
    layer: np.ndarray               # int32 [R]
    neuron: np.ndarray              # int32 [R]
    partner: np.ndarray             # int32 [R], -1 unless NS
    noise: List[Optional[np.ndarray]] = field(default_factory=list)  # per record (GF)
    perm: List[Optional[np.ndarray]] = field(default_factory=list)   # per record (WS)

    def perm_of(self, r: int):
        return self.perm[r] if self.perm else None

    @property
    def n_records(self) -> int:
        return int(self.mutant_id.size)

    def records_of(self, m: int) -> np.ndarray:
        return np.nonzero(self.mutant_id == m)[0]

    def subset(self, n: int) -> "Mutants":
        """The first ``n`` mutants (records keep their order)."""
        keep = np.nonzero(self.mutant_id < n)[0]
        return Mutants(n, self.mutant_id[keep].copy(), self.op[keep].copy(),
                       self.layer[keep].copy(), self.neuron[keep].copy(),
                       self.partner[keep].copy(), [self.noise[i] for i in keep],
                       [self.perm_of(i) for i in keep])

    def select(self, ids) -> "Mutants":
        """Mutants ``ids`` renumbered 0..len(ids)-1, records in their order."""
        ids = [int(i) for i in ids]
        rows = []
        for new, old in enumerate(ids):
            for r in self.records_of(old):
                rows.append((new, int(r)))
        idx = np.array([r for _, r in rows], dtype=np.int64)
        mid = np.array([n for n, _ in rows], dtype=np.int32)
        return Mutants(len(ids), mid, self.op[idx].copy(), self.layer[idx].copy(),
                       self.neuron[idx].copy(), self.partner[idx].copy(),
                       [self.noise[i] for i in idx], [self.perm_of(i) for i in idx])


@dataclass
class Workload:
    name: str
    model: Model
    inputs: np.ndarray              # [N][H][W][C], float32 or uint16 (bf16 bits)
    mutants: Mutants
    description: str = ""

    @property
    def n_inputs(self) -> int:
        return int(self.inputs.shape[0])
