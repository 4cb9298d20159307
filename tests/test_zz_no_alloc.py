"""The allocation-free pruned recursion (rnnt_pruned_loss_noalloc) against
rnnt_pruned_loss with a caller workspace, through the C ABI: two calls in a
row on the same GPU (the scratch keeps the first call's contents), the
second with a smaller batch. The same kernels run on the same inputs, so the
results must be bitwise equal (which also meets the fp32 tolerances: loss
1e-5 relative, occupations 1e-4 absolute)."""
import numpy as np
import pytest
import torch

import paper_2206_13236_amd as P
from gpu_common import assert_close, dev_f32, dev_i32, host, make_dev_batch, run_step, say, sub_batch
from workloads import make_batch

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    assert torch.cuda.is_available(), "GPU tests need a ROCm device"
    P.lib()


def _band(b):
    """Band log-probs and bounds of batch b from the GPU's own pipeline."""
    out = run_step(b, b.wl.S)
    return out["px"].astype(np.float32), out["py"].astype(np.float32), out["ranges"]


@pytest.mark.parametrize("second", ["bpe_first_three", "tiny"])
def test_noalloc_pruned_loss_equals_the_workspace_entry(second):
    big = make_batch("bpe", seed=0)
    small = sub_batch(big, [0, 1, 2]) if second == "bpe_first_three" else make_batch("tiny", seed=0)
    for k, b in enumerate((big, small)):
        S = b.wl.S
        px, py, rg = _band(b)
        say(f"[noalloc] call {k + 1}: N={b.N} T={b.T} U={b.U} S={S}")
        batch = make_dev_batch(b)
        dpx, dpy, drg = dev_f32(px), dev_f32(py), dev_i32(rg)
        ref = P.rnnt_pruned_loss(batch, S, dpx, dpy, drg)
        f32 = dict(dtype=torch.float32, device=dpx.device)
        got = P.rnnt_pruned_loss_noalloc(batch, S, dpx, dpy, drg, px_occ=torch.empty(b.N, b.T, S, **f32),
                                         py_occ=torch.empty(b.N, b.T, S, **f32))
        torch.cuda.synchronize()
        for key in ("loss", "px_occ", "py_occ"):
            assert torch.equal(got[key], ref[key]), f"call {k + 1}: {key} differs"
        assert_close("loss", host(got["loss"]), host(ref["loss"]), rtol=1e-5)
        assert_close("px_occ", host(got["px_occ"]), host(ref["px_occ"]), atol=1e-4)
        assert np.all(np.isfinite(host(got["loss"])))
