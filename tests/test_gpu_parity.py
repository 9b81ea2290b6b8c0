"""GPU parity: the library's kill bits, score and logits against the CPU oracle
(vanilla mutation testing) on the same seeded inputs.

Bar: logits within 1e-4*S (fp32) / 2e-2*S (bf16), where S is the largest
|logit| of the original; kill bits identical outside A (an oracle margin of
the original or the mutant below tau = 1e-3) and A2 (outside A, an oracle
margin below that logit tolerance times S); the mutation score over the
retained pairs identical to the oracle's; the whole score identical whenever
no pair disagrees.  Every comparison is a row of the table printed at the end
of the run."""
import numpy as np
import pytest

import oracle as O
import workloads as W
from harness import (log, run_gpu, oracle_run, compare, compare_logits, sample_mutants,
                     gpu_context, device_inputs, unpack_words)

pytestmark = pytest.mark.gpu


def _parity(wl, n_sample_logits=8, tau=1e-3, labels=None, name=None, **opts):
    log(f"[parity] {wl.name} N={wl.n_inputs} M={wl.mutants.n_mutants}")
    m, words, kills, score = run_gpu(wl, labels=labels, **opts)
    ids = sample_mutants(m, wl)[:max(n_sample_logits, 1) * 4]
    res = oracle_run(wl, labels=labels, keep_logits=ids)
    worst = compare_logits(m, res, ids, wl.model.dtype)
    compare(res, words, kills, score, wl, tau, m=m, err_over_s=worst, name=name, labels=labels)
    return m, res, words


def test_mlp_full():
    _parity(W.make_workload("mlp"))


def test_lenet5_ragged_inputs():
    _parity(W.make_workload("lenet5", n_inputs=1000, n_mutants=60))


def test_vgg_small_each_ratio():
    for ri in range(4):
        _parity(W.make_workload("vgg", n_inputs=130, n_mutants=24, ratio_index=ri))


def test_resnet20_small():
    _parity(W.make_workload("resnet20", n_inputs=66, n_mutants=24))


def test_resnet18w_small():
    _parity(W.make_workload("resnet18w", n_inputs=24, n_mutants=8))


def test_lstm_small():
    # embedding gathers, the LSTM recursion on MFMA, every operator
    _parity(W.make_workload("lstm", n_inputs=130, n_mutants=40,
                            ops=(W.GF, W.NEB, W.NAI, W.NS, W.WS)))


def test_rnn_imdb_small():
    # Table 1's RNN: 128-wide embedding, two 64-unit LSTMs (the wide LSTM kernel,
    # weights in registers), every operator
    _parity(W.make_workload("rnn_imdb", n_inputs=130, n_mutants=30,
                            ops=(W.GF, W.NEB, W.NAI, W.NS, W.WS)))


def test_mobilenetv2_small():
    # depthwise layers (full and channel-list kernels), ReLU6, inverted
    # residuals; weight shuffles included, switches on depthwise layers recompute
    _parity(W.make_workload("mobilenetv2", n_inputs=66, n_mutants=30,
                            ops=(W.GF, W.NEB, W.NAI, W.NS, W.WS)))


def test_ground_truth_labels_path():
    wl = W.make_workload("lenet5", n_inputs=300, n_mutants=30)
    labels = np.random.default_rng(9).integers(0, 10, wl.n_inputs).astype(np.int32)
    _parity(wl, labels=labels)


def test_chunking_does_not_change_results():
    wl = W.make_workload("lenet5", n_inputs=700, n_mutants=40)
    _, w0, k0, s0 = run_gpu(wl)
    _, w1, k1, s1 = run_gpu(wl, chunk_inputs=128, max_workspace_mb=1)
    assert np.array_equal(w0, w1) and np.array_equal(k0, k1) and s0 == s1


def test_repeat_is_deterministic():
    wl = W.make_workload("resnet20", n_inputs=64, n_mutants=12)
    m = gpu_context(wl)
    m.run_original(device_inputs(wl))
    a = m.run_mutants()
    b = m.run_mutants()
    assert np.array_equal(a[0].cpu().numpy(), b[0].cpu().numpy()) and a[2] == b[2]
    z1 = m.get_logits(3).cpu().numpy()
    z2 = m.get_logits(3).cpu().numpy()
    assert np.array_equal(z1, z2)


@pytest.mark.parametrize("cfg", ["lenet5", "resnet20", "mobilenetv2", "lstm", "rnn_imdb"])
def test_identity_mutants_bit_exact(cfg):
    """Zero-noise fuzz at every layer and a mutant without records reproduce
    the original's logits bit for bit and are never killed."""
    base = W.make_workload(cfg, n_inputs=130, n_mutants=1)
    md = base.model
    layers = md.weighted_nodes()
    recs = [(i, W.GF, l, i % md.nodes[l].c_out, -1, np.zeros(md.nodes[l].fan_in, np.float32))
            for i, l in enumerate(layers)]
    n = len(recs)
    a = lambda k: np.array([r[k] for r in recs], np.int32)
    muts = W.Mutants(n + 1, a(0), a(1), a(2), a(3), a(4), [r[5] for r in recs])
    wl = W.Workload(cfg + "_identity", md, base.inputs, muts)
    m, words, kills, score = run_gpu(wl)
    assert not words.any() and score["ms_num"] == 0
    z = m.get_logits(-1).cpu().numpy()
    for mid in range(n + 1):
        assert np.array_equal(m.get_logits(mid).cpu().numpy(), z), mid


def test_output_layer_closed_forms_on_gpu():
    """On the output layer a switch swaps two logits, an inverse negates one
    and a block zeroes one -- exactly, relative to the GPU's own original."""
    base = W.make_workload("vgg", n_inputs=64, n_mutants=1, ratio_index=0)
    md = base.model
    out = len(md.nodes) - 1
    muts = W.Mutants(3, np.array([0, 1, 2], np.int32), np.array([W.NS, W.NAI, W.NEB], np.int32),
                     np.array([out] * 3, np.int32), np.array([0, 1, 2], np.int32),
                     np.array([3, -1, -1], np.int32), [None, None, None])
    m, words, kills, score = run_gpu(W.Workload("closed", md, base.inputs, muts))
    z = m.get_logits(-1).cpu().numpy()
    sw = z.copy(); sw[:, [0, 3]] = z[:, [3, 0]]
    assert np.array_equal(m.get_logits(0).cpu().numpy(), sw)
    ng = z.copy(); ng[:, 1] = -z[:, 1]
    assert np.array_equal(m.get_logits(1).cpu().numpy(), ng)
    zr = z.copy(); zr[:, 2] = 0
    assert np.array_equal(m.get_logits(2).cpu().numpy(), zr)
    pred = z.argmax(1)
    for k, zz in enumerate((sw, ng, zr)):
        assert np.array_equal(unpack_words(words, 64)[k], zz.argmax(1) != pred)


def test_state_machine_errors():
    from paper_2607_18582_amd import MureError, MURE_E_STATE
    wl = W.make_workload("mlp", n_inputs=64, n_mutants=4)
    m = gpu_context(wl)
    with pytest.raises(MureError) as e:
        m.run_mutants()
    assert e.value.status == MURE_E_STATE
    m.run_original(device_inputs(wl))
    m.run_mutants()
    m.apply(wl.mutants)                      # invalidates the cache
    with pytest.raises(MureError) as e:
        m.run_mutants()
    assert e.value.status == MURE_E_STATE


def test_weight_shuffle_operator():
    """The paper's fourth mutator (weight shuffle) against the oracle."""
    for cfg, ni, nm in (("lenet5", 300, 40), ("resnet20", 66, 20)):
        _parity(W.make_workload(cfg, n_inputs=ni, n_mutants=nm,
                                ops=(W.GF, W.NEB, W.NAI, W.NS, W.WS)))


@pytest.mark.parametrize("cfg", ["lenet5", "vgg", "resnet20", "mobilenetv2", "lstm", "rnn_imdb", "resnet18w"])
def test_vanilla_mode_equals_memoized_bit_for_bit(cfg):
    """Theorem 1 on the GPU: running every mutant from the raw input gives
    exactly the memoized result -- kill bits, score and logits, bit for bit."""
    wl = W.make_workload(cfg, n_inputs=130, n_mutants=30, ops=(W.GF, W.NEB, W.NAI, W.NS, W.WS))
    m1, w1, k1, s1 = run_gpu(wl)
    m2, w2, k2, s2 = run_gpu(wl, vanilla=1)
    assert np.array_equal(w1, w2) and np.array_equal(k1, k2) and s1 == s2
    for mid in sample_mutants(m1, wl):
        assert np.array_equal(m1.get_logits(mid).cpu().numpy(), m2.get_logits(mid).cpu().numpy()), mid
    assert m2.stats()["n_groups"] == 1


@pytest.mark.parametrize("cfg", ["lenet5", "vgg", "resnet20"])
def test_vanilla_mode_against_the_oracle(cfg):
    """GPU vanilla mutation testing (every mutant from the raw input, the
    baseline of the paper's gain measure) against the oracle, to the same bar
    as the memoized path."""
    wl = W.make_workload(cfg, n_inputs=130, n_mutants=30, ops=(W.GF, W.NEB, W.NAI, W.NS, W.WS))
    m, _, _ = _parity(wl, name=f"{wl.name} vanilla", vanilla=1)
    assert m.stats()["n_groups"] == 1


def test_edge_cases_zero_mutants_identity_only_single_input():
    from paper_2607_18582_amd import MureError, MURE_E_INVALID
    wl = W.make_workload("lenet5", n_inputs=1, n_mutants=6)
    _parity(wl)                                             # one input: one ragged kill word
    # no mutants at all: an empty kill matrix and the score 0/0
    empty = W.Mutants(0, np.zeros(0, np.int32), np.zeros(0, np.int32), np.zeros(0, np.int32),
                      np.zeros(0, np.int32), np.zeros(0, np.int32), [])
    m, words, kills, score = run_gpu(W.Workload("none", wl.model, wl.inputs, empty))
    assert words.size == 0 and len(kills) == 0 and (score["ms_num"], score["ms_den"]) == (0, 0)
    # mutants without records (identity): never killed, the denominator still counts them
    ident = W.Mutants(3, np.zeros(0, np.int32), np.zeros(0, np.int32), np.zeros(0, np.int32),
                      np.zeros(0, np.int32), np.zeros(0, np.int32), [])
    wl3 = W.make_workload("lenet5", n_inputs=70, n_mutants=1)
    m, words, kills, score = run_gpu(W.Workload("identity", wl3.model, wl3.inputs, ident))
    assert not words.any() and score["ms_num"] == 0 and score["ms_den"] == 3 * score["n_labels"]
    assert m.stats()["n_groups"] == 0
    # an empty input set is rejected
    with pytest.raises(MureError) as e:
        m.run_original(device_inputs(wl3)[:0])
    assert e.value.status == MURE_E_INVALID


def test_largest_class_count():
    """512 classes (the library's maximum): the kill runs on its own kernel
    with an 8-word class mask; ground-truth labels spread over the classes."""
    b = W.configs._Builder((1, 1, 24))
    x = b.dense(0, 32, True, "h")
    b.dense(x, 512, False, "out")
    w, bb = W.configs._draw_weights(b.nodes, "f32", 0.1, seed=3)
    model = W.Model("mlp512", "f32", b.nodes, w, bb)
    x = W.make_inputs(model, 200, "uniform")
    mu = W.make_mutants(model, 24, 2, "layer_first", variant=5, ops=(W.GF, W.NEB, W.NAI, W.NS, W.WS))
    wl = W.Workload("mlp512", model, x, mu)
    _parity(wl)
    labels = np.random.default_rng(4).integers(0, 512, size=200).astype(np.int32)
    _parity(wl, labels=labels)


@pytest.mark.parametrize("cfg", ["lenet5", "resnet20"])
def test_fused_paths_equal_separate_kernels(cfg):
    """The ADD fused into a residual block's second convolution and the kill
    fused into the output layer give exactly the separate kernels' results."""
    wl = W.make_workload(cfg, n_inputs=130, n_mutants=30, ops=(W.GF, W.NEB, W.NAI, W.NS, W.WS))
    m1, w1, k1, s1 = run_gpu(wl)
    m2, w2, k2, s2 = run_gpu(wl, fused_paths=0)
    assert np.array_equal(w1, w2) and np.array_equal(k1, k2) and s1 == s2
    for mid in sample_mutants(m1, wl):
        assert np.array_equal(m1.get_logits(mid).cpu().numpy(), m2.get_logits(mid).cpu().numpy()), mid


@pytest.mark.parametrize("cfg", ["resnet18w", "vgg"])
def test_group_reads_equal_per_mutant_copies(cfg):
    """The halo kernel reading the first mutated node's output (and a fused
    identity shortcut) in 8-channel groups -- the cached groups shared, only
    each mutant's changed groups copied -- gives exactly the results of a full
    copy per mutant."""
    wl = W.make_workload(cfg, n_inputs=70 if cfg == "resnet18w" else 130, n_mutants=12,
                         ops=(W.GF, W.NEB, W.NAI, W.NS, W.WS))
    m1, w1, k1, s1 = run_gpu(wl)
    planes = m1.stats()["group_planes"]
    m2, w2, k2, s2 = run_gpu(wl, group_reads=0)
    assert planes > 0 and m2.stats()["group_planes"] == 0
    assert np.array_equal(w1, w2) and np.array_equal(k1, k2) and s1 == s2
    for mid in sample_mutants(m1, wl):
        assert np.array_equal(m1.get_logits(mid).cpu().numpy(), m2.get_logits(mid).cpu().numpy()), mid


def _fp32_cnn():
    """A small fp32 CNN whose convolutions take the LDS kernel's other
    instances and the fp32 im2col kernel:
      C1  20x20x1 -> 5x5 -> pool -> 8x8x16   LDS, C_in odd (4 consecutive k per MFMA)
      C2  1x1, 16 -> 32                      LDS, 32-column tiles, k pairs
      C3  1x1, 32 -> 48, pool -> 4x4x48      LDS, 64-column tiles, k pairs
      C4  3x3 pad 1, 48 -> 24                im2col (its images exceed the LDS budget)
    C1 and C2 feed LDS convolutions, so their clusters read mmi's output
    virtually."""
    b = W.configs._Builder((20, 20, 1))
    x = b.conv(0, 16, 5, relu=True, pool=2, name="C1")
    x = b.conv(x, 32, 1, relu=True, name="C2")
    x = b.conv(x, 48, 1, relu=True, pool=2, name="C3")
    x = b.conv(x, 24, 3, pad=1, relu=True, name="C4")
    x = b.dense(x, 20, True, "F1")
    b.dense(x, 10, False, "F2")
    w, bb = W.configs._draw_weights(b.nodes, "f32", 0.1, seed=7)
    model = W.Model("cnn_f32", "f32", b.nodes, w, bb)
    x = W.make_inputs(model, 150, "uniform")
    mu = W.make_mutants(model, 48, 2, "layer_first", variant=3, ops=(W.GF, W.NEB, W.NAI, W.NS, W.WS))
    return W.Workload("cnn_f32", model, x, mu)


def test_fp32_cnn_lds_instances_and_im2col():
    """Parity with the oracle on the fp32 CNN above, the kernel families it is
    meant to reach, and memoized equal to vanilla bit for bit."""
    wl = _fp32_cnn()
    m, _, _ = _parity(wl, kernel_timing=1)
    launches = m.stats()["kernel_launches"]
    assert launches[2] > 0 and launches[3] > 0, launches      # LDS and im2col families ran
    m1, w1, k1, s1 = run_gpu(wl)
    m2, w2, k2, s2 = run_gpu(wl, vanilla=1)
    assert np.array_equal(w1, w2) and np.array_equal(k1, k2) and s1 == s2
    for mid in sample_mutants(m1, wl):
        assert np.array_equal(m1.get_logits(mid).cpu().numpy(), m2.get_logits(mid).cpu().numpy()), mid


@pytest.mark.parametrize("shortcut", ["optionA", "proj"])
def test_fp32_tiny_resnet_unfused_adds(shortcut):
    """Parity on a small fp32 residual net whose mutants start at every
    convolution: a cluster whose first mutated node is a block's second
    convolution runs its ADD unfused (the 4-lane vector ADD on the identity
    block; the element ADD where option A's channel offset is not a whole
    vector), and memoized equals vanilla bit for bit."""
    model = W.tiny_resnet("f32", shortcut=shortcut)
    x = W.make_inputs(model, 300, "uniform")
    mu = W.make_mutants(model, 40, 1, "layer_first", variant=5, ops=(W.GF, W.NEB, W.NAI, W.NS, W.WS))
    wl = W.Workload("tiny_resnet_" + shortcut, model, x, mu)
    _parity(wl)
    m1, w1, k1, s1 = run_gpu(wl)
    m2, w2, k2, s2 = run_gpu(wl, vanilla=1)
    assert np.array_equal(w1, w2) and np.array_equal(k1, k2) and s1 == s2


def test_reapply_in_one_context_matches_fresh_contexts():
    """One context, three mutant sets in turn (larger, smaller with fewer
    inputs, the first again): each run equals a fresh context's bit for bit,
    so nothing left over from an earlier apply or input set leaks in."""
    a = W.make_workload("lenet5", n_inputs=300, n_mutants=40, ops=(W.GF, W.NEB, W.NAI, W.NS, W.WS))
    b = W.make_workload("lenet5", n_inputs=130, n_mutants=12, ops=(W.GF, W.NAI))
    fresh = {}
    for wl in (a, b):
        fm, fw, fk, fs = run_gpu(wl)
        fresh[wl.mutants.n_mutants] = (fw, fk, fs, [fm.get_logits(i).cpu().numpy() for i in (0, 5, -1)])
    m = gpu_context(a)
    for wl in (a, b, a):
        log(f"[reapply] M={wl.mutants.n_mutants} N={wl.n_inputs}")
        m.apply(wl.mutants)
        m.run_original(device_inputs(wl))
        kb, kills, score = m.run_mutants()
        fw, fk, fs, fz = fresh[wl.mutants.n_mutants]
        assert np.array_equal(kb.cpu().numpy().view(np.uint64), fw)
        assert np.array_equal(kills, fk) and score == fs
        for i, z in zip((0, 5, -1), fz):
            assert np.array_equal(m.get_logits(i).cpu().numpy(), z), i


def test_cached_flatten_node():
    """A FLATTEN view between a convolution and a dense layer, with every
    mutant's first mutated layer at the dense layer (so the FLATTEN is the
    memoization boundary and its output lives in the prefix cache), and with
    mutants on the convolution too, against the oracle."""
    for dtype in ("f32", "bf16"):
        b = W.configs._Builder((12, 12, 8))
        x = b.conv(0, 16, 3, pad=1, relu=True, pool=2, name="C1")
        f = b.flatten(x)
        x = b.dense(f, 40, True, "F1")
        b.dense(x, 10, False, "F2")
        w, bb = W.configs._draw_weights(b.nodes, dtype, 0.1, seed=11)
        model = W.Model(f"flat_{dtype}", dtype, b.nodes, w, bb)
        xin = W.make_inputs(model, 150, "uniform" if dtype == "f32" else "normal")
        mu = W.make_mutants(model, 30, 2, "layer_first", variant=7, ops=(W.GF, W.NEB, W.NAI, W.NS, W.WS))
        wl = W.Workload(f"flatten_{dtype}", model, xin, mu)
        m, _, _ = _parity(wl)
        assert any(m.mutant_plan(i)[0] == f + 1 for i in range(mu.n_mutants))   # mmi at the dense layer
        assert any(m.mutant_plan(i)[2] == [f] for i in range(mu.n_mutants))     # K = {the FLATTEN}


def test_binding_refuses_short_device_buffers():
    """The binding checks caller buffers against the shapes the library
    reports before a call that writes device memory."""
    import torch
    wl = W.make_workload("mlp", n_inputs=130, n_mutants=6)
    m = gpu_context(wl)
    m.run_original(device_inputs(wl))
    with pytest.raises(ValueError):
        m.run_mutants(torch.empty((6, 2), dtype=torch.int64, device="cuda:0"))       # needs 6 x 3 words
    with pytest.raises(ValueError):
        m.get_logits(0, out=torch.empty((130, 9), dtype=torch.float32, device="cuda:0"))
    kb, _, _ = m.run_mutants(torch.empty((6, 3), dtype=torch.int64, device="cuda:0"))
    assert kb.shape == (6, 3) and m.get_logits(0).shape == (130, 10)
