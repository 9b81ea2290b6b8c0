"""GPU parity at the workloads' full sizes, in the launch configuration the
benchmark uses (default options: whole input set per chunk, the 64 GB workspace).

The GPU runs the whole workload.  The oracle's results for a sample of
(mutant, input) pairs -- at least two mutants of every first-mutated layer
plus seeded extras, inputs spread over the whole set (the last, ragged kill
word included) plus the inputs with the smallest original margins of a
screened prefix -- were computed on the CPU by
tests/golden/make_fullsize_refs.py, which calls only the oracle; the file is
tied to the oracle's sources and to the workload by two hashes, checked here.
On the sample the bar is the small tests' bar (tests/harness.py): logits
within the dtype's tolerance, no kill disagreement outside A and A2, the score
over the retained pairs identical.  Properties that hold at any size are
checked on the whole matrix: kill counts are popcounts, padding bits are
zero, and the reported score is the score of the GPU's own kill matrix."""
import importlib.util
import os

import numpy as np
import pytest

import oracle as O
import workloads as W
from harness import LOGIT_TOL, classify_pairs, log, record, run_gpu, unpack_words

pytestmark = pytest.mark.gpu

GOLDEN = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden")


def _refs_module():
    spec = importlib.util.spec_from_file_location("make_fullsize_refs", os.path.join(GOLDEN, "make_fullsize_refs.py"))
    mod = importlib.util.module_from_spec(spec)
    spec.loader.exec_module(mod)
    return mod


def _sampled_parity(name):
    ref = np.load(os.path.join(GOLDEN, f"fullsize_{name}.npz"), allow_pickle=False)
    mk = _refs_module()
    wl = W.make_workload(str(ref["config"]), ratio_index=int(ref["ratio_index"]))
    ids, xs = ref["ids"], ref["xs"]
    assert str(ref["oracle_hash"]) == mk.oracle_hash(), "oracle changed: rerun tests/golden/make_fullsize_refs.py"
    assert str(ref["workload_hash"]) == mk.workload_hash(wl, list(ids), xs), \
        "workload changed: rerun tests/golden/make_fullsize_refs.py"
    N, M = wl.n_inputs, wl.mutants.n_mutants
    log(f"[full] {wl.name} N={N} M={M}: GPU run; sample {len(ids)} mutants x {len(xs)} inputs")
    m, words, kills, score = run_gpu(wl)
    gk = unpack_words(words, N)
    # properties over the whole matrix
    assert np.array_equal(kills, gk.sum(axis=1))
    if N % 64:
        assert not (words[:, -1] >> np.uint64(N % 64)).any()
    z_orig = m.get_logits(-1).cpu().numpy()
    label = z_orig.argmax(axis=1)
    pm = np.where(gk, -1, label[None, :])               # any prediction != label where killed
    kill2, _, num2, den2, nl2 = O.kill_and_score(label, pm, label, z_orig.shape[1])
    assert np.array_equal(kill2, gk)
    assert (score["ms_num"], score["ms_den"], score["n_labels"]) == (num2, den2, nl2)
    # the sample against the oracle's references
    tol = LOGIT_TOL[wl.model.dtype]
    S = float(np.abs(ref["logits"]).max())
    e_o = np.abs(z_orig[xs] - ref["logits"]).max(axis=1)
    assert e_o.max() <= tol * S, (e_o.max(), tol * S)
    worst = float(e_o.max()) / S
    for j, mid in enumerate(ids):
        zg = m.get_logits(int(mid)).cpu().numpy()[xs]
        e_m = np.abs(zg - ref["mutant_logits"][j]).max()
        worst = max(worst, float(e_m) / S)
        assert e_m <= tol * S, (int(mid), e_m, tol * S)
    gks = gk[ids][:, xs]
    amb, amb2, dis = classify_pairs(gks, ref["kill"], ref["margin_orig"], ref["margin_mut"], wl.model.dtype, S)
    record(f"{wl.name} full {N}x{M}, sample", wl.model.dtype, gks, ref["kill"], amb, amb2, dis, worst,
           label[xs], ref["label"], int(ref["n_labels"]), (score["ms_num"], score["ms_den"]), None)


def test_lenet5_full_size():
    _sampled_parity("lenet5")


def test_resnet20_full_size():
    _sampled_parity("resnet20")


@pytest.mark.parametrize("name", ["vgg_r0", "vgg_r1", "vgg_r2", "vgg_r3"])
def test_vgg_full_size(name):
    _sampled_parity(name)


def test_resnet18w_full_size():
    _sampled_parity("resnet18w")


def test_mobilenetv2_full_size():
    _sampled_parity("mobilenetv2")


def test_lstm_full_size():
    _sampled_parity("lstm")


def test_rnn_imdb_full_size():
    _sampled_parity("rnn_imdb")
