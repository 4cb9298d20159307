"""Memory scaling of the whole step (the method's memory claim, Sec. 1 and
Sec. 3.2): at fixed N, T, S and V, the peak device memory of a training step
(inputs and outputs excluded) grows with U only through the lattice-sized
arrays of the simple loss (O(N T U)) and the lm-sized ones (O(N U V)), never
through an O(N T U V) tensor such as the unpruned [N, T, U+1, V] logits.
"""
import numpy as np
import pytest
import torch

import paper_2206_13236_amd as P
from gpu_common import dev_f32, dev_joiner, make_dev_batch, say
from workloads import make_batch

pytestmark = pytest.mark.gpu


def _step_peak(U):
    N, T, V, S, J = 8, 120, 500, 5, 256
    b = make_batch("bpe", seed=41, N=N, T_range=(T, T), U_range=(U, U), V=V, J=J, S=S)
    batch = make_dev_batch(b)
    args = (dev_f32(b.am), dev_f32(b.lm), dev_joiner(b.enc, False), dev_joiner(b.dec, False),
            dev_joiner(b.W, False), dev_joiner(b.bias, False))
    step = P.PrunedRnntLoss(S)
    step.step(batch, *args)  # allocates the outputs and workspaces it keeps
    torch.cuda.synchronize()
    base = torch.cuda.memory_allocated()
    torch.cuda.reset_peak_memory_stats()
    out = step.step(batch, *args)
    torch.cuda.synchronize()
    peak = torch.cuda.max_memory_allocated() - base
    kept = base - sum(t.numel() * t.element_size() for t in args)  # outputs + workspaces held by the module
    assert np.isfinite(out["pruned_loss"].cpu().numpy()).all()
    del step, out
    torch.cuda.empty_cache()
    return kept + peak, (N, T, V)


def test_peak_memory_grows_with_u_far_below_the_unpruned_logits():
    say("[memory] U sweep 16 / 64")
    m16, (N, T, V) = _step_peak(16)
    m64, _ = _step_peak(64)
    growth = m64 - m16
    unpruned_growth = N * T * (64 - 16) * V * 4  # [N, T, U+1, V] fp32 logits alone
    say(f"[memory] step memory U=16 {m16 / 1e6:.1f} MB, U=64 {m64 / 1e6:.1f} MB, "
        f"growth {growth / 1e6:.1f} MB vs {unpruned_growth / 1e6:.1f} MB for the unpruned logits")
    assert growth > 0
    assert growth < 0.25 * unpruned_growth
