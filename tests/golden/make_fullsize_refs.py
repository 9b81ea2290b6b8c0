"""Oracle references for the full-size GPU parity tests.

For each workload at its full size this runs the CPU oracle (vanilla
mutation testing, ``oracle/`` only) on a sample of (mutant, input) pairs and
stores what the GPU test compares against:

  mutants  at least ``per_group`` mutants of every first-mutated layer (the
           clusters of Algorithm 1), then further mutants drawn with a fixed
           seed until ``n_mut`` are chosen;
  inputs   ``n_spread`` inputs spread evenly over the whole set, the last one
           included (the ragged kill word), plus the ``n_small`` inputs whose
           original top-1/top-2 logit margin is smallest among the first
           ``screen`` inputs (the near-ties the bf16 path is most likely to
           flip).

Stored per workload (``fullsize_<name>.npz``): the chosen ids and inputs,
the oracle's kill bits, margins, labels and class count over the whole
sample, the original's and the chosen mutants' float32 logits, and keys that
tie the file to the oracle's source and to the workload (a hash of the
sampled inputs, weights and mutation records).  The GPU test refuses a file
whose keys do not match.

    python tests/golden/make_fullsize_refs.py [name ...]   # from the repo root
"""
from __future__ import annotations

import hashlib
import os
import sys
import time

import numpy as np

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(os.path.dirname(HERE))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

import oracle as O  # noqa: E402
import workloads as W  # noqa: E402

# name: (config, ratio index, mutants, spread inputs, smallest-margin inputs, screened prefix)
SAMPLES = {
    "resnet18w": ("resnet18w", 0, 6, 97, 32, 1024),
    "vgg_r0": ("vgg", 0, 16, 48, 16, 2048),
    "vgg_r1": ("vgg", 1, 16, 48, 16, 2048),
    "vgg_r2": ("vgg", 2, 16, 48, 16, 2048),
    "vgg_r3": ("vgg", 3, 16, 48, 16, 2048),
    "resnet20": ("resnet20", 1, 24, 48, 16, 2048),
    "lenet5": ("lenet5", 1, 24, 368, 32, 10000),
    "mobilenetv2": ("mobilenetv2", 1, 16, 48, 16, 2048),
    "lstm": ("lstm", 1, 24, 224, 32, 10000),
    "rnn_imdb": ("rnn_imdb", 1, 24, 96, 32, 4096),
}


def oracle_hash() -> str:
    """Hash of the oracle's code -- its syntax trees without docstrings, so
    that comments and docstrings do not count: references from another
    oracle are stale."""
    import ast

    h = hashlib.sha256()
    d = os.path.join(ROOT, "oracle")
    for f in sorted(os.listdir(d)):
        if f.endswith(".py"):
            with open(os.path.join(d, f)) as fh:
                tree = ast.parse(fh.read())
            for node in ast.walk(tree):
                body = getattr(node, "body", None)
                if isinstance(body, list) and body and isinstance(body[0], ast.Expr) and \
                        isinstance(getattr(body[0], "value", None), ast.Constant) and \
                        isinstance(body[0].value.value, str):
                    node.body = body[1:] or [ast.Pass()]
            h.update(f.encode())
            h.update(ast.dump(tree).encode())
    return h.hexdigest()[:16]


def workload_hash(wl: W.Workload, ids, xs) -> str:
    """Hash of what the sample depends on: its inputs, the weights and the
    chosen mutants' records."""
    h = hashlib.sha256()
    h.update(np.ascontiguousarray(wl.inputs[xs]).tobytes())
    for w, b in zip(wl.model.weights, wl.model.biases):
        if w is not None:
            h.update(np.ascontiguousarray(w).tobytes())
            h.update(np.ascontiguousarray(b).tobytes())
    sub = wl.mutants.select(ids)
    for a in (sub.mutant_id, sub.op, sub.layer, sub.neuron, sub.partner):
        h.update(np.ascontiguousarray(a).tobytes())
    for r in range(sub.n_records):
        if sub.noise[r] is not None:
            h.update(np.ascontiguousarray(sub.noise[r]).tobytes())
        p = sub.perm_of(r)
        if p is not None:
            h.update(np.ascontiguousarray(p).tobytes())
    return h.hexdigest()[:16]


def choose_mutants(wl: W.Workload, n_mut: int, per_group: int = 2, seed: int = 0):
    """per_group mutants of every first-mutated layer mmi = min over the
    mutant's records (identity mutants have none), then seeded extras."""
    groups = {}
    for m in range(wl.mutants.n_mutants):
        recs = wl.mutants.records_of(m)
        if len(recs):
            groups.setdefault(int(wl.mutants.layer[recs].min()), []).append(m)
    ids = []
    for _, ms in sorted(groups.items()):
        ids += ms[:per_group]
    rng = np.random.default_rng(seed)
    for m in rng.permutation(wl.mutants.n_mutants):
        if len(ids) >= n_mut:
            break
        if int(m) not in ids and len(wl.mutants.records_of(int(m))):
            ids.append(int(m))
    return sorted(set(ids))


def choose_inputs(wl: W.Workload, om, n_spread: int, n_small: int, screen: int):
    N = wl.n_inputs
    spread = np.unique(np.concatenate([np.linspace(0, N - 1, n_spread).astype(int), [N - 1]]))
    pre = min(screen, N)
    z = O.forward(om, wl.inputs[:pre], chunk=64)
    small = np.argsort(O.margins(z), kind="stable")[:n_small]
    return np.unique(np.concatenate([spread, small])).astype(np.int64)


def make(name: str) -> str:
    cfg, ri, n_mut, n_spread, n_small, screen = SAMPLES[name]
    t0 = time.time()
    wl = W.make_workload(cfg, ratio_index=ri)
    om = O.OracleModel(wl.model)
    ids = choose_mutants(wl, n_mut)
    xs = choose_inputs(wl, om, n_spread, n_small, screen)
    res = O.run_vanilla(om, wl.inputs[xs], wl.mutants.select(ids), keep_logits=range(len(ids)), chunk=32)
    out = os.path.join(HERE, f"fullsize_{name}.npz")
    np.savez_compressed(
        out, ids=np.array(ids, np.int64), xs=xs, kill=res.kill, label=res.label,
        margin_orig=res.margin_orig, margin_mut=res.margin_mut, n_labels=np.int64(res.n_labels),
        logits=res.logits.astype(np.float32),
        mutant_logits=np.stack([res.mutant_logits[j] for j in range(len(ids))]).astype(np.float32),
        oracle_hash=np.array(oracle_hash()), workload_hash=np.array(workload_hash(wl, ids, xs)),
        config=np.array(cfg), ratio_index=np.int64(ri), n_inputs=np.int64(wl.n_inputs),
        n_mutants=np.int64(wl.mutants.n_mutants))
    print(f"{name}: {len(ids)} mutants x {len(xs)} inputs, {time.time() - t0:.0f} s -> {out}", flush=True)
    return out


if __name__ == "__main__":
    for n in (sys.argv[1:] or list(SAMPLES)):
        make(n)
