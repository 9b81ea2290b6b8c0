"""The allocation-free run_mutants entry point against mure_run_mutants.

mure_run_mutants_noalloc runs the same kernels with its chunk workspace and
per-mutant counters in the library's fixed device scratch array.  Two calls
in a row on one context -- the second after run_original over a smaller
input -- must each give the kill bits, kill counts and score of
mure_run_mutants on a separate context, bit for bit.  resnet18w's rows are
large enough that the scratch array forces chunks of fewer inputs and slots
than the default workspace, so the chunked path is the one compared."""
import numpy as np
import pytest

import workloads as W
from harness import device_inputs, gpu_context, log

pytestmark = pytest.mark.gpu


def _run(m, x, noalloc):
    m.run_original(x)
    kb, kills, score = m.run_mutants(noalloc=noalloc)
    return kb.cpu().numpy().copy(), kills.copy(), dict(score)


@pytest.mark.parametrize("cfg,n_in,n_mut,n_small", [("lenet5", 700, 40, 300),
                                                     ("resnet20", 200, 24, 70),
                                                     ("resnet18w", 200, 6, 90)])
def test_noalloc_equals_run_mutants(cfg, n_in, n_mut, n_small):
    wl = W.make_workload(cfg, n_inputs=n_in, n_mutants=n_mut)
    log(f"[noalloc] {cfg} N={n_in} then {n_small}, M={n_mut}")
    x = device_inputs(wl)
    ref = gpu_context(wl)
    na = gpu_context(wl)
    for n in (n_in, n_small):
        xs = x[:n].contiguous()
        r_bits, r_kills, r_score = _run(ref, xs, noalloc=False)
        a_bits, a_kills, a_score = _run(na, xs, noalloc=True)
        log(f"  N={n}: MS {a_score['ms_num']}/{a_score['ms_den']} (run_mutants "
            f"{r_score['ms_num']}/{r_score['ms_den']}), workspace of run_mutants "
            f"{ref.stats()['workspace_bytes'] >> 20} MiB")
        assert a_bits.shape == r_bits.shape == (n_mut, (n + 63) // 64)
        assert np.array_equal(a_bits, r_bits)
        assert np.array_equal(a_kills, r_kills)
        assert a_score == r_score
