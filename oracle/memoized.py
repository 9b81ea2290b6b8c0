"""Memoized mutation testing as the paper states it (Algorithms 1-4).

Used only by the CPU tests, to check Theorem 1 (the chopped mutant fed with
memo-table entries computes exactly what the full mutant computes) by brute
force against ``vanilla.run_vanilla``, and to pin the boundary rule that the
GPU library's planner implements independently.

Graph conventions: node 0 is the model input (so the memoization boundary of a
mutant whose first mutated layer is node 1 is {0}, the identity probe of
Algorithm 3); a node's inputs are read in the order its descriptor lists
them (an ADD's second input is its shortcut).
"""
from __future__ import annotations

from typing import Callable, Dict, FrozenSet, List, Sequence, Tuple

import numpy as np

from workloads.graph import Mutants
from .layers import OracleModel, forward_all, phi
from .mutate import apply_records


def get_dep_graph(model: OracleModel) -> Dict[int, Tuple[int, ...]]:
    """Algorithm 2: layer index -> the layers it receives inputs from.

    A purely sequential model maps i to (i-1,) and the first layer to nothing;
    otherwise each layer maps to the layers of its inbound nodes."""
    nodes = model.nodes
    sequential = all(n.inputs == (i - 1,) for i, n in enumerate(nodes) if i > 0)
    if sequential:
        return {i: ((i - 1,) if i > 0 else ()) for i in range(len(nodes))}
    return {i: tuple(n.inputs) for i, n in enumerate(nodes)}


def boundary(dg: Dict[int, Sequence[int]], mmi: int, n_layers: int) -> FrozenSet[int]:
    """Algorithm 1's memoization boundary: layers before ``mmi`` that some layer
    at or after ``mmi`` reads (equal to the set K of Section 4)."""
    return frozenset(j for li in range(mmi, n_layers) for j in dg[li] if j < mmi)


def mutated_layers(mutants: Mutants, m: int) -> List[int]:
    """mu(M'): the (zero-based) indices of the layers mutant m changes."""
    return sorted({int(mutants.layer[r]) for r in mutants.records_of(m)})


def instrument(model: OracleModel, probes: Sequence[int]) -> Callable[[np.ndarray], Dict[int, np.ndarray]]:
    """Algorithm 3: a model returning the original's activations at ``probes``.

    Its outputs are the probe tensors, so the layers after the last probe are
    not computed.  An empty probe list gives the identity on the input."""
    probes = sorted(probes)
    for p in probes:
        if not (0 <= p < len(model.nodes)):
            raise KeyError("Probe point not found")
    if not probes:
        return lambda X: {0: model.input_values(X)}
    return lambda X: forward_all(model, X, keep=probes, accumulate="ordered", last=probes[-1])


def chop_mutant(model: OracleModel, weights, biases, mmi: int,
                dg: Dict[int, Sequence[int]], K: FrozenSet[int]):
    """Algorithm 4: the mutant re-rooted at ``mmi``; it takes the memo-table
    tensors of the boundary layers K and runs layers mmi..L of the mutant."""
    L = len(model.nodes) - 1

    def chopped(MT: Dict[int, np.ndarray]) -> np.ndarray:
        fabricated = {k: MT[k] for k in K}          # one fabricated input per k in K
        past: Dict[int, np.ndarray] = {}
        for j in range(mmi, L + 1):
            layer_in = [fabricated[p] if p < mmi else past[p] for p in dg[j]]
            past[j] = phi(model, j, layer_in, weights[j], biases[j], accumulate="ordered")
        return past[L]

    return chopped


def mure(model: OracleModel, X: np.ndarray, mutants: Mutants) -> Dict[int, np.ndarray]:
    """Algorithm 1: every mutant's logits on X, computed with memoization.

    Mutants without records (identity mutants) are their original's output."""
    dg = get_dep_graph(model)
    n_layers = len(model.nodes)
    clusters: Dict[FrozenSet[int], List[int]] = {}
    res: Dict[int, np.ndarray] = {}
    identity: List[int] = []
    for mid in range(mutants.n_mutants):
        mu = mutated_layers(mutants, mid)
        if not mu:
            identity.append(mid)
            continue
        K = boundary(dg, min(mu), n_layers)
        clusters.setdefault(K, []).append(mid)
    for K, ids in clusters.items():
        MT = instrument(model, sorted(K))(X)
        for mid in ids:
            W, B, _ = apply_records(model, mutants, mid)
            mmi = min(mutated_layers(mutants, mid))
            out = chop_mutant(model, W, B, mmi, dg, K)(MT)
            res[mid] = out.reshape(out.shape[0], -1)
    if identity:
        z = forward_all(model, X, keep=[n_layers - 1], accumulate="ordered")[n_layers - 1]
        for mid in identity:
            res[mid] = z.reshape(z.shape[0], -1)
    return res
