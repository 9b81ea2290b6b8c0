"""Seeded synthetic workloads shaped like the paper's models (Section 5, Table 1).

This package only *draws data*: graph descriptors, He-normal weights, test
inputs and mutation records (with the Gaussian-fuzz noise already drawn).  It
holds none of the method's arithmetic (no layer functions, no operator
application, no kill or score logic), so both the CPU oracle and the GPU path
can consume it without sharing code.
"""
from .graph import (INPUT, DENSE, CONV2D, ADD, GAP, FLATTEN, DWCONV, EMBED, LSTM, KIND_NAMES,
                    GF, NEB, NAI, NS, WS, OP_NAMES, Node, Model, Mutants, Workload)
from .configs import (CONFIGS, make_workload, make_model, make_inputs,
                      make_mutants, neuron_layers, tiny_mlp, tiny_resnet,
                      tiny_lenet, tiny_mobilenet, tiny_rnn, lstm_bias_positions,
                      bf16_bits_to_f32)

__all__ = [
    "INPUT", "DENSE", "CONV2D", "ADD", "GAP", "FLATTEN", "DWCONV", "EMBED", "LSTM", "KIND_NAMES",
    "GF", "NEB", "NAI", "NS", "WS", "OP_NAMES", "Node", "Model", "Mutants", "Workload",
    "CONFIGS", "make_workload", "make_model", "make_inputs", "make_mutants",
    "neuron_layers", "tiny_mlp", "tiny_resnet", "tiny_lenet", "tiny_mobilenet", "tiny_rnn",
    "lstm_bias_positions",
    "bf16_bits_to_f32",
]
