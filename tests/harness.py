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


def compare(res: "O.VanillaResult", words, kills, score, wl: W.Workload, tau: float = TAU,
            m=None):
    """Kill bits must agree with the oracle outside the ambiguous pairs
    (margin < tau).  For bf16 models every remaining disagreement must be a
    near-tie explained by the measured logit error of that very row (the GPU
    accumulates in float32, the oracle in float64, and a one-ulp bf16 rounding
    difference of an activation propagates): the oracle margin at the pair is
    at most twice the row's max |logit error|, and that error is within the
    bf16 logit tolerance.  The score must agree exactly whenever no pair
    disagrees.  Returns a summary dict."""
    n = wl.n_inputs
    gk = unpack_words(words, n)
    amb = res.ambiguous(tau)
    dis = gk != res.kill
    out = dict(pairs=int(gk.size), ambiguous=int(amb.sum()), disagree=int(dis.sum()),
               disagree_outside=int((dis & ~amb).sum()), unexplained=0)
    if out["disagree_outside"]:
        log(f"  kill disagreements outside margin {tau}: {out['disagree_outside']}")
        if wl.model.dtype == "f32" or m is None:
            raise AssertionError(out)
        out["unexplained"] = explain_near_ties(m, res, wl, np.argwhere(dis & ~amb))
        assert out["unexplained"] == 0, out
    if n % 64:                                     # padding bits are zero
        assert not (words[:, -1] >> np.uint64(n % 64)).any()
    assert np.array_equal(kills, gk.sum(axis=1))   # counts consistent with the bits
    if not dis.any():
        assert (score["ms_num"], score["ms_den"]) == (res.ms_num, res.ms_den), (score, res.ms_num, res.ms_den)
        assert score["killed_mutants"] == int(res.kill.any(axis=1).sum())
    assert score["n_labels"] == res.n_labels
    assert score["nonfinite_logits"] == 0
    return out


def explain_near_ties(m, res, wl, pairs) -> int:
    tol = LOGIT_TOL[wl.model.dtype]
    S = float(np.abs(res.logits).max())
    om = O.OracleModel(wl.model)
    zg_o = m.get_logits(-1).cpu().numpy()
    e_o = np.abs(zg_o - res.logits).max(axis=1)
    unexplained = 0
    for mid in sorted(set(int(p[0]) for p in pairs)):
        W_, B_, _ = O.apply_records(om, wl.mutants, mid)
        zo = O.forward(om, wl.inputs, W_, B_, chunk=64)
        zg = m.get_logits(mid).cpu().numpy()
        e_m = np.abs(zg - zo).max(axis=1)
        for (_, x) in [p for p in pairs if int(p[0]) == mid]:
            ok = (e_m[x] <= tol * S and e_o[x] <= tol * S and
                  (res.margin_mut[mid, x] <= 2 * e_m[x] or res.margin_orig[x] <= 2 * e_o[x]))
            log(f"  near-tie m={mid} x={x}: margin_mut={res.margin_mut[mid, x]:.4g} "
                f"margin_orig={res.margin_orig[x]:.4g} err_mut={e_m[x]:.3g} err_orig={e_o[x]:.3g} "
                f"(tol*S={tol * S:.3g}) {'explained' if ok else 'UNEXPLAINED'}")
            unexplained += (not ok)
    return unexplained


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
