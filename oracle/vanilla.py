"""Vanilla (exhaustive) mutation testing and the mutation score (Section 5.2).

Every mutant is evaluated from the raw input through every layer -- no
memoization -- which is the baseline the paper compares against and, by
Theorem 1, exactly what memoized testing computes.

Kill predicate: kill(mu, t) holds when the original's predicted label equals
label(t) and the mutant's predicted label differs from it.  predicted label =
argmax of the logits, lowest index on ties.  label(t) is the given label, or
(synthetic inputs have none) the original's prediction, which makes kill
equivalent to "the mutant's prediction differs from the original's".
killingLabels(mu) = { label(t) : kill(mu, t) };  L = { label(t) : t in T };
mutation score MS = sum_mu |killingLabels(mu)| / (|M| * |L|), kept as the
integer pair (numerator, denominator).

Ambiguous pairs: margin(z) = top1 - top2 of a logit row (float64); a pair
(m, x) is ambiguous when the original's margin at x or the mutant's margin is
below ``tau``; such pairs are reported, not compared.
"""
from __future__ import annotations

from dataclasses import dataclass, field
from typing import Dict, List, Optional, Sequence

import numpy as np

from workloads.graph import Mutants
from .layers import OracleModel, forward
from .mutate import apply_records


def predicted(z: np.ndarray) -> np.ndarray:
    """argmax over classes, the lowest index among equal maxima."""
    return np.argmax(z, axis=1).astype(np.int64)


def margins(z: np.ndarray) -> np.ndarray:
    """top-1 minus top-2 logit per row, in float64."""
    s = np.sort(z.astype(np.float64), axis=1)
    return s[:, -1] - s[:, -2]


def pack_bits(b: np.ndarray) -> np.ndarray:
    """bool [M][N] -> uint64 [M][ceil(N/64)]; bit (x & 63) of word x >> 6."""
    m, n = b.shape
    nw = (n + 63) // 64
    padded = np.zeros((m, nw * 64), np.uint64)
    padded[:, :n] = b
    shifts = np.arange(64, dtype=np.uint64)
    return (padded.reshape(m, nw, 64) << shifts).sum(axis=2, dtype=np.uint64)


def kill_and_score(pred_orig: np.ndarray, pred_mut: np.ndarray, label: np.ndarray,
                   n_classes: int):
    """kill matrix [M][N] (bool), killingLabels masks, MS numerator/denominator."""
    ok = pred_orig == label                                   # argmax m(t) = label(t)
    kill = ok[None, :] & (pred_mut != label[None, :])         # argmax mu(t) != label(t)
    M = pred_mut.shape[0]
    killing = np.zeros((M, n_classes), bool)
    for m in range(M):
        killing[m, np.unique(label[kill[m]])] = True
    n_labels = int(np.unique(label).size)
    num = int(killing.sum())
    den = int(M * n_labels)
    return kill, killing, num, den, n_labels


@dataclass
class VanillaResult:
    logits: np.ndarray                 # original z(x), float32 [N, C]
    label: np.ndarray                  # label(x)
    pred_mut: np.ndarray               # [M, N]
    margin_orig: np.ndarray            # [N]
    margin_mut: np.ndarray             # [M, N]
    kill: np.ndarray                   # bool [M, N]
    killing: np.ndarray                # bool [M, C]
    ms_num: int
    ms_den: int
    n_labels: int
    mutant_logits: Dict[int, np.ndarray] = field(default_factory=dict)

    @property
    def ms(self) -> float:
        return self.ms_num / self.ms_den if self.ms_den else 0.0

    @property
    def kills_per_mutant(self) -> np.ndarray:
        return self.kill.sum(axis=1).astype(np.int64)

    def ambiguous(self, tau: float = 1e-3) -> np.ndarray:
        return (self.margin_mut < tau) | (self.margin_orig[None, :] < tau)

    def kill_words(self) -> np.ndarray:
        return pack_bits(self.kill)


def run_vanilla(model: OracleModel, X: np.ndarray, mutants: Mutants,
                labels: Optional[np.ndarray] = None, keep_logits: Sequence[int] = (),
                mutant_ids: Optional[Sequence[int]] = None, accumulate: str = "blas",
                chunk: int = 256) -> VanillaResult:
    """Exhaustive mutation testing of ``mutants`` (or of ``mutant_ids`` only)."""
    z = forward(model, X, accumulate=accumulate, chunk=chunk)
    label = predicted(z) if labels is None else np.asarray(labels, np.int64)
    ids = list(range(mutants.n_mutants)) if mutant_ids is None else list(mutant_ids)
    N, C = z.shape
    pred_mut = np.empty((len(ids), N), np.int64)
    margin_mut = np.empty((len(ids), N), np.float64)
    keep = {}
    for row, m in enumerate(ids):
        W, B, _ = apply_records(model, mutants, m)
        zm = forward(model, X, W, B, accumulate=accumulate, chunk=chunk)
        pred_mut[row] = predicted(zm)
        margin_mut[row] = margins(zm)
        if m in keep_logits:
            keep[m] = zm
    kill, killing, num, den, nl = kill_and_score(predicted(z), pred_mut, label, C)
    return VanillaResult(z, label, pred_mut, margins(z), margin_mut, kill, killing,
                         num, den, nl, keep)
