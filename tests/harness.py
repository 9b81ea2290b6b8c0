"""Shared helpers of the parity tests: run a workload through the library on
the GPU, run it through the oracle on the CPU, and compare."""
from __future__ import annotations

import sys
import time

import numpy as np

import oracle as O
import workloads as W

TAU = 1e-3                                  # margin below which a pair is ambiguous
LOGIT_TOL = {"f32": 1e-4, "bf16": 2e-2}     # max |logit error| / S


def log(*a):
    print(*a, flush=True)
    sys.stdout.flush()


def device_inputs(wl: W.Workload):
    import torch
    x = wl.inputs
    if x.dtype == np.uint16:
        t = torch.from_numpy(x.view(np.int16).copy())
    else:
        t = torch.from_numpy(np.ascontiguousarray(x))
    return t.cuda()


def gpu_context(wl: W.Workload, **options):
    from paper_2607_18582_amd import Mure
    m = Mure(device=0)
    for k, v in options.items():
        m.set_option(k, v)
    md = wl.model
    m.load_model(md.nodes, md.in_hwc, md.dtype, md.weights, md.biases)
    m.apply(wl.mutants)
    return m


def run_gpu(wl: W.Workload, labels=None, **options):
    m = gpu_context(wl, **options)
    x = device_inputs(wl)
    m.run_original(x, labels)
    kb, kills, score = m.run_mutants()
    words = kb.cpu().numpy().view(np.uint64).copy()
    return m, words, kills, score


def unpack_words(words: np.ndarray, n: int) -> np.ndarray:
    bits = ((words[:, :, None] >> np.arange(64, dtype=np.uint64)) & np.uint64(1)).astype(bool)
    return bits.reshape(words.shape[0], -1)[:, :n]


def oracle_run(wl: W.Workload, labels=None, keep_logits=(), mutant_ids=None):
    t = time.time()
    om = O.OracleModel(wl.model)
    res = O.run_vanilla(om, wl.inputs, wl.mutants, labels=labels, keep_logits=keep_logits,
                        mutant_ids=mutant_ids, chunk=64)
    log(f"  oracle {wl.name}: {time.time() - t:.1f}s")
    return res


def sample_mutants(m, wl: W.Workload, per_group: int = 2, extra: int = 4, seed: int = 0):
    """Mutants covering every first-mutated layer (per_group each) plus a few random."""
    groups = {}
    for mid in range(wl.mutants.n_mutants):
        mmi, grp, _ = m.mutant_plan(mid)
        if mmi >= 0:
            groups.setdefault(grp, []).append(mid)
    ids = []
    for g, ms in sorted(groups.items()):
        ids += ms[:per_group]
    rng = np.random.default_rng(seed)
    ids += [int(i) for i in rng.choice(wl.mutants.n_mutants, size=min(extra, wl.mutants.n_mutants), replace=False)]
    return sorted(set(ids))


# One row per parity comparison, printed as a table at the end of the run
# (tests/conftest.py, pytest_terminal_summary).
RECORDS = []


def near_tie_band(dtype: str, S: float) -> float:
    """Margin below which a kill may legitimately differ beyond tau: the logit
    tolerance of the dtype times the logit scale S (an argmax can change
    only where a margin is within the logit error)."""
    return LOGIT_TOL[dtype] * S


def retained_score(kill: np.ndarray, label: np.ndarray, keep: np.ndarray, n_labels: int):
    """The mutation score over the retained pairs only: sum over mutants of
    |{label(x) : kill(m, x) and keep(m, x)}|, over |M| * |L|."""
    num = 0
    for m in range(kill.shape[0]):
        num += int(np.unique(label[kill[m] & keep[m]]).size)
    return num, int(kill.shape[0]) * int(n_labels)


def classify_pairs(gk, okill, margin_orig, margin_mut, dtype, S, tau=TAU):
    """A: an oracle margin below tau (reported, not compared).  A2: outside A,
    an oracle margin below the near-tie band tol * S (reported separately).
    Returns (A, A2, disagreements)."""
    amb = (margin_mut < tau) | (margin_orig[None, :] < tau)
    band = near_tie_band(dtype, S)
    amb2 = ~amb & ((margin_mut < band) | (margin_orig[None, :] < band))
    return amb, amb2, gk != okill


def record(name, dtype, gk, okill, amb, amb2, dis, err_over_s, gpu_label, oracle_label, n_labels,
           full_gpu=None, full_oracle=None):
    """Record one comparison and enforce the bar: no kill disagreement
    outside A and A2, and the score over the retained pairs identical."""
    keep = ~amb & ~amb2
    ms_g = retained_score(gk, gpu_label, keep, n_labels)
    ms_o = retained_score(okill, oracle_label, keep, n_labels)
    row = dict(name=name, dtype=dtype, pairs=int(gk.size), A=int(amb.sum()), A2=int(amb2.sum()),
               dis=int(dis.sum()), dis_A=int((dis & amb).sum()), dis_A2=int((dis & amb2).sum()),
               dis_out=int((dis & keep).sum()), err=err_over_s, ms_ret_gpu=ms_g, ms_ret_oracle=ms_o,
               ms_gpu=full_gpu, ms_oracle=full_oracle)
    RECORDS.append(row)
    log(f"  parity {name}: {row}")
    assert row["dis_out"] == 0, row
    assert ms_g == ms_o, row
    return row


def compare(res: "O.VanillaResult", words, kills, score, wl: W.Workload, tau: float = TAU,
            m=None, err_over_s=float("nan"), name=None, labels=None):
    """Kill bits against the oracle on every pair.  Pairs in A (an oracle
    margin below tau) and A2 (outside A, an oracle margin below tol * S) are
    reported; every other pair must agree, and the mutation score over those
    retained pairs must equal the oracle's.  The whole-matrix score must
    equal the oracle's whenever no pair disagrees.  Returns the row."""
    n = wl.n_inputs
    gk = unpack_words(words, n)
    S = float(np.abs(res.logits).max())
    amb, amb2, dis = classify_pairs(gk, res.kill, res.margin_orig, res.margin_mut, wl.model.dtype, S, tau)
    if labels is not None:
        gpu_label = np.asarray(labels, np.int64)
    else:
        gpu_label = m.get_logits(-1).cpu().numpy().argmax(axis=1) if m is not None else res.label
    row = record(name or wl.name, wl.model.dtype, gk, res.kill, amb, amb2, dis, err_over_s, gpu_label,
                 res.label, res.n_labels, (score["ms_num"], score["ms_den"]), (res.ms_num, res.ms_den))
    if n % 64:                                     # padding bits are zero
        assert not (words[:, -1] >> np.uint64(n % 64)).any()
    assert np.array_equal(kills, gk.sum(axis=1))   # counts consistent with the bits
    if not dis.any():
        assert (score["ms_num"], score["ms_den"]) == (res.ms_num, res.ms_den), (score, res.ms_num, res.ms_den)
        assert score["killed_mutants"] == int(res.kill.any(axis=1).sum())
    if np.array_equal(gpu_label, res.label):       # the same label set on both sides
        assert score["n_labels"] == res.n_labels
    assert score["nonfinite_logits"] == 0
    return row


def compare_logits(m, res: "O.VanillaResult", ids, dtype: str):
    tol = LOGIT_TOL[dtype]
    S = float(np.abs(res.logits).max())
    zo = m.get_logits(-1).cpu().numpy()
    worst = float(np.abs(zo - res.logits).max()) / S
    for mid in ids:
        z = m.get_logits(mid).cpu().numpy()
        e = float(np.abs(z - res.mutant_logits[mid]).max()) / S
        worst = max(worst, e)
        assert e <= tol, (mid, e, tol)
    assert worst <= tol
    return worst
