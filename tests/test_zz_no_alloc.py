"""The allocation-free analysis (nsgcqt_analyse_noalloc) through the C ABI
against nsgcqt_analyse: the same kernels on the same inputs, so the results
must be bitwise identical. Two calls in a row on the library's device
array, the second with a smaller input; neither allocates."""
import gc

import numpy as np
import pytest

import workloads

torch = pytest.importorskip("torch")
from paper_2609_29119_amd import nsgcqt as nb  # noqa: E402

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    nb.lib()


def test_noalloc_analysis_matches_analyse():
    # 40 stress signals (28 MB of workspace), then one tiny signal (128 KB)
    for name, b in (("stress", 40), ("tiny", 1)):
        w = workloads.WORKLOADS[name]
        p = nb.Plan(*w.plan_args, batch=b)
        assert p.info.ws_analyse <= nb.NOALLOC_SCRATCH_BYTES
        x = torch.from_numpy(workloads.signals(w, batch=b)).cuda()
        ref = p.analyse(x)
        out = torch.full_like(ref, float("nan"))
        # no tensor of an earlier test may be freed inside the measured window
        gc.collect()
        gc.disable()
        try:
            torch.cuda.synchronize()
            torch.cuda.reset_peak_memory_stats()
            mem0 = torch.cuda.memory_allocated()
            p.analyse_noalloc(x, out)
            torch.cuda.synchronize()
            assert torch.cuda.max_memory_allocated() == mem0
        finally:
            gc.enable()
        assert np.array_equal(out.cpu().numpy().view(np.uint32), ref.cpu().numpy().view(np.uint32)), name


def test_noalloc_rejects_plans_beyond_its_array():
    w = workloads.WORKLOADS["stress"]
    p = nb.Plan(*w.plan_args, batch=w.batch)
    assert p.info.ws_analyse > nb.NOALLOC_SCRATCH_BYTES
    x = torch.zeros((w.batch, w.n_samples), dtype=torch.float32, device="cuda")
    out = torch.empty((w.batch, p.n_coeffs), dtype=torch.complex64, device="cuda")
    with pytest.raises(nb.NsgcqtError) as e:
        p.analyse_noalloc(x, out)
    assert e.value.status == nb.EWORKSPACE
