"""The four neuron-level mutation operators (Section 3.1).

The paper takes GF, NAI, WS and NEB from DeepMutation without defining them;
the readings used here (shared with the GPU library's documentation):
  neuron i of a DENSE/CONV2D layer is output channel i (Section 2.1); its
  incoming weights are W[i] (all of C_in*kh*kw of them);
  GF  (Gaussian fuzzing)           W[i] <- round_dtype(fl32(W[i] + eps)), eps
                                   given (drawn by the workload generator),
                                   bias untouched;
  NEB (neuron effect block)        W[i] <- 0, b[i] <- 0  (the neuron outputs 0);
  NAI (neuron activation inverse)  W[i] <- -W[i], b[i] <- -b[i]  (the
                                   pre-activation is negated before ReLU);
  NS  (neuron switch)              W[i] <-> W[j], b[i] <-> b[j];
  WS  (weight shuffle)             W[i][k] <- W[i][perm[k]] for a given
                                   permutation of the incoming weights, bias
                                   untouched.
A mutant's records apply in array order.  Mutated layer functions Phi' are
therefore the original functions with changed parameters: the graph never
changes (Section 4).
"""
from __future__ import annotations

from typing import List, Optional, Tuple

import numpy as np

from workloads.graph import GF, NEB, NAI, NS, WS, Mutants
from .layers import OracleModel
from .numerics import rne_bf16


def apply_records(model: OracleModel, mutants: Mutants, m: int):
    """Return (weights, biases, mutated_layers) of mutant ``m``: per-node lists
    where mutated layers are copies, the rest alias the original."""
    W = list(model.weights)
    B = list(model.biases)
    copied = set()
    for r in mutants.records_of(m):
        l = int(mutants.layer[r]); i = int(mutants.neuron[r]); op = int(mutants.op[r])
        node = model.nodes[l]
        if not node.weighted:
            raise ValueError(f"record {r}: node {l} has no neurons")
        if not (0 <= i < node.c_out):
            raise ValueError(f"record {r}: neuron {i} out of range")
        if l not in copied:
            W[l] = W[l].copy(); B[l] = B[l].copy(); copied.add(l)
        w = W[l].reshape(node.c_out, -1)
        if op == GF:
            eps = np.asarray(mutants.noise[r], np.float32)
            if eps.size != w.shape[1]:
                raise ValueError(f"record {r}: noise length {eps.size} != fan-in {w.shape[1]}")
            t = w[i] + eps                                   # float32 addition
            w[i] = rne_bf16(t) if model.dtype == "bf16" else t
        elif op == NEB:
            w[i] = 0.0
            B[l][i] = 0.0
        elif op == NAI:
            w[i] = -w[i]
            B[l][i] = -B[l][i]
        elif op == NS:
            j = int(mutants.partner[r])
            if not (0 <= j < node.c_out) or j == i:
                raise ValueError(f"record {r}: bad switch partner {j}")
            w[[i, j]] = w[[j, i]]
            B[l][[i, j]] = B[l][[j, i]]
        elif op == WS:
            perm = np.asarray(mutants.perm_of(r), np.int64)
            if perm.size != w.shape[1] or not np.array_equal(np.sort(perm), np.arange(w.shape[1])):
                raise ValueError(f"record {r}: not a permutation of the fan-in")
            w[i] = w[i][perm]
        else:
            raise ValueError(f"record {r}: unknown operator {op}")
    return W, B, sorted(copied)
