"""GPU parity at the workloads' full sizes, in the launch configuration the
benchmark uses (default options: whole input set per chunk, 16 GB workspace).

The GPU runs the whole workload; the oracle recomputes a sample of (mutant,
input) pairs one by one -- mutants covering every first-mutated layer, inputs
spread over the whole set including the last (ragged) kill word -- and the
kill bits and logits of those pairs must match to the same bar as the small
parity tests.  Properties that hold at any size are checked on everything:
the kill counts are the popcounts of the kill words, padding bits are zero,
and the reported score equals the score of the GPU's own kill matrix."""
import numpy as np
import pytest

import oracle as O
import workloads as W
from harness import LOGIT_TOL, TAU, log, run_gpu, unpack_words, sample_mutants

pytestmark = pytest.mark.gpu


def _sampled_parity(cfg, ratio_index, n_mut, n_in):
    wl = W.make_workload(cfg, ratio_index=ratio_index)
    N, M = wl.n_inputs, wl.mutants.n_mutants
    log(f"[full] {wl.name} N={N} M={M}: GPU run")
    m, words, kills, score = run_gpu(wl)
    gk = unpack_words(words, N)
    # properties over the whole matrix
    assert np.array_equal(kills, gk.sum(axis=1))
    if N % 64:
        assert not (words[:, -1] >> np.uint64(N % 64)).any()
    z_orig = m.get_logits(-1).cpu().numpy()
    label = z_orig.argmax(axis=1)
    _, killing, num, den, nl = O.kill_and_score(label, np.zeros((1, N), np.int64), label, z_orig.shape[1])
    pm = np.where(gk, -1, label[None, :])               # any prediction != label where killed
    kill2, killing2, num2, den2, nl2 = O.kill_and_score(label, pm, label, z_orig.shape[1])
    assert np.array_equal(kill2, gk)
    assert (score["ms_num"], score["ms_den"], score["n_labels"]) == (num2, den2, nl2)
    # sampled pairs against the oracle
    ids = sample_mutants(m, wl, per_group=1, extra=2)[:n_mut]
    xs = np.unique(np.concatenate([np.linspace(0, N - 1, n_in).astype(int), [N - 1]]))
    sub = W.Workload(wl.name + "_sample", wl.model, wl.inputs[xs], wl.mutants.select(ids))
    res = O.run_vanilla(O.OracleModel(wl.model), sub.inputs, sub.mutants,
                        keep_logits=range(len(ids)), chunk=16)
    tol = LOGIT_TOL[wl.model.dtype]
    S = float(np.abs(res.logits).max())
    e_o = np.abs(z_orig[xs] - res.logits).max(axis=1)
    assert e_o.max() <= tol * S, (e_o.max(), tol * S)
    amb = res.ambiguous(TAU)
    gks = gk[ids][:, xs]
    bad = 0
    worst = float(e_o.max()) / S
    for j, mid in enumerate(ids):
        zg = m.get_logits(mid).cpu().numpy()[xs]
        e_m = np.abs(zg - res.mutant_logits[j]).max(axis=1)
        worst = max(worst, float(e_m.max()) / S)
        assert e_m.max() <= tol * S, (mid, e_m.max(), tol * S)
        for x in np.nonzero((gks[j] != res.kill[j]) & ~amb[j])[0]:
            explained = (wl.model.dtype == "bf16" and
                         (res.margin_mut[j, x] <= 2 * e_m[x] or res.margin_orig[x] <= 2 * e_o[x]))
            log(f"  pair m={mid} x={xs[x]}: margins {res.margin_mut[j, x]:.4g}/{res.margin_orig[x]:.4g} "
                f"errors {e_m[x]:.3g}/{e_o[x]:.3g} {'near-tie' if explained else 'MISMATCH'}")
            bad += not explained
    log(f"  sampled {len(ids)} mutants x {len(xs)} inputs: ambiguous {int(amb.sum())}, "
        f"max logit err/S {worst:.2e}, MS {score['ms_num']}/{score['ms_den']}")
    assert bad == 0


def test_lenet5_full_size():
    _sampled_parity("lenet5", 1, 24, 400)


def test_resnet20_full_size():
    _sampled_parity("resnet20", 1, 24, 48)


@pytest.mark.parametrize("ri", [0, 1, 2, 3])
def test_vgg_full_size(ri):
    _sampled_parity("vgg", ri, 8, 24)


def test_resnet18w_full_size():
    _sampled_parity("resnet18w", 0, 3, 10)


def test_mobilenetv2_full_size():
    _sampled_parity("mobilenetv2", 1, 16, 48)


def test_lstm_full_size():
    _sampled_parity("lstm", 1, 24, 256)
