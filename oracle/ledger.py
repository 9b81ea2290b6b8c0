"""The additive cost model of Section 4.2, counted in multiply-accumulates.

cost(v) per input = MACs of node v (CONV2D: pre-pool output pixels * C_out *
kh*kw*C_in; DWCONV: output pixels * C * kh*kw; DENSE: C_in*C_out; LSTM:
T * 4H * (D + H + 1); other kinds, the embedding lookup included, 0).  It is non-negative (C1),
additive over a prefix/suffix split (C2) and depends only on the layer shapes
(C3).  For a cluster C of mutants sharing mmi, the prefix P is every node
before mmi and the chopped mutant every node from mmi on, so
vanilla - memoized = (|C| - 1) * cost(P) (Lemma 4).
"""
from __future__ import annotations

from typing import Dict, List

from workloads.graph import CONV2D, DENSE, DWCONV, LSTM, Mutants
from .layers import OracleModel
from .memoized import boundary, get_dep_graph, mutated_layers


def node_macs(model: OracleModel) -> List[int]:
    out = []
    for v, n in enumerate(model.nodes):
        if n.kind in (CONV2D, DWCONV):
            h, w, _ = model.nodes[n.inputs[0]].out_hwc
            ho = (h + 2 * n.pad - n.kh) // n.stride + 1
            wo = (w + 2 * n.pad - n.kw) // n.stride + 1
            per_channel = n.kh * n.kw * (1 if n.kind == DWCONV else n.c_in)
            out.append(ho * wo * n.c_out * per_channel)
        elif n.kind == DENSE:
            out.append(n.c_in * n.c_out)
        elif n.kind == LSTM:
            steps = model.nodes[n.inputs[0]].out_hwc[1]
            out.append(steps * 4 * n.c_out * (n.c_in + n.c_out + 1))
        else:
            out.append(0)
    return out


def cluster_costs(model: OracleModel, mutants: Mutants) -> List[Dict]:
    """Per cluster: its boundary, size, mmi set, cost(P), and the per-input
    totals of vanilla and memoized testing."""
    macs = node_macs(model)
    dg = get_dep_graph(model)
    n = len(model.nodes)
    clusters: Dict[frozenset, List[int]] = {}
    mmis: Dict[frozenset, set] = {}
    for m in range(mutants.n_mutants):
        mu = mutated_layers(mutants, m)
        if not mu:
            continue
        K = boundary(dg, min(mu), n)
        clusters.setdefault(K, []).append(m)
        mmis.setdefault(K, set()).add(min(mu))
    full = sum(macs)
    out = []
    for K, ids in clusters.items():
        (mmi,) = mmis[K]                      # one mmi per boundary in these graphs
        cost_p = sum(macs[:mmi])
        suffix = sum(macs[mmi:])
        out.append(dict(K=sorted(K), mmi=mmi, size=len(ids), cost_prefix=cost_p,
                        vanilla=len(ids) * full, memoized=cost_p + len(ids) * suffix))
    return out
