"""The parity bar itself (tests/harness.py), on the CPU: which pairs fall in
A and A2, that a disagreement outside them fails, and the score over the
retained pairs."""
import numpy as np
import pytest

import harness as H


def _case():
    # 2 mutants x 4 inputs, labels 0..3, logit scale S = 10
    margin_orig = np.array([5.0, 5.0, 5e-4, 5.0])          # input 2: A
    margin_mut = np.array([[5.0, 0.1, 5.0, 5.0],           # (0, 1): A2 for bf16 (0.1 < 0.02 * 10)
                           [5.0, 5.0, 5.0, 5.0]])
    okill = np.array([[1, 0, 0, 1], [0, 1, 0, 0]], bool)
    label = np.arange(4)
    return margin_orig, margin_mut, okill, label


def test_classify_pairs_sets():
    mo, mm, ok, _ = _case()
    amb, amb2, dis = H.classify_pairs(ok.copy(), ok, mo, mm, "bf16", 10.0)
    assert amb.sum() == 2 and amb[:, 2].all()              # tau applies to the original's margin
    assert amb2.sum() == 1 and amb2[0, 1]
    assert not dis.any()
    # fp32: the band is 1e-4 * S = 1e-3, so (0, 1) is retained
    _, amb2f, _ = H.classify_pairs(ok.copy(), ok, mo, mm, "f32", 10.0)
    assert not amb2f.any()


def test_record_accepts_disagreements_in_a_and_a2_only():
    mo, mm, ok, label = _case()
    gk = ok.copy()
    gk[0, 1] = True                                        # in A2
    gk[1, 2] = True                                        # in A
    amb, amb2, dis = H.classify_pairs(gk, ok, mo, mm, "bf16", 10.0)
    row = H.record("t", "bf16", gk, ok, amb, amb2, dis, 1e-3, label, label, 4)
    assert (row["dis_A"], row["dis_A2"], row["dis_out"]) == (1, 1, 0)
    gk[1, 3] = True                                        # retained: must fail
    amb, amb2, dis = H.classify_pairs(gk, ok, mo, mm, "bf16", 10.0)
    with pytest.raises(AssertionError):
        H.record("t", "bf16", gk, ok, amb, amb2, dis, 1e-3, label, label, 4)
    del H.RECORDS[:]


def test_retained_score():
    kill = np.array([[1, 1, 0], [0, 0, 1]], bool)
    label = np.array([3, 3, 5])
    keep = np.ones_like(kill)
    assert H.retained_score(kill, label, keep, 2) == (2, 4)       # {3} and {5}
    keep[1, 2] = False
    assert H.retained_score(kill, label, keep, 2) == (1, 4)
