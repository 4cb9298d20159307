"""GPU parity of the smoothed trivial joiner (Sec. 3.3.1) against the oracle:
log-probs, loss, occupations and the gradients w.r.t. am and lm, through
both simple-loss entry points and inside the fused training step."""
import numpy as np
import pytest
import torch

import oracle as O
import paper_2206_13236_amd as P
from gpu_common import assert_close, dev_f32, dev_joiner, host, make_dev_batch, ranges_valid, say
from workloads import make_batch

pytestmark = pytest.mark.gpu

WEIGHTS = [(0.25, 0.1), (0.0, 0.3), (0.4, 0.0), (0.5, 0.5)]


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    assert torch.cuda.is_available(), "GPU tests need a ROCm device"
    P.lib()


def _batch(seed):
    return make_batch("bpe", seed=seed, N=3, T_range=(30, 50), U_range=(4, 12), V=37, J=32, S=4)


@pytest.mark.parametrize("w", WEIGHTS, ids=[f"lm{a}_am{b}" for a, b in WEIGHTS])
def test_smoothed_simple_loss(w):
    a, bw = w
    b = _batch(seed=11)
    say(f"[smoothed] a_lm={a} a_ac={bw}")
    sc = np.array([0.5, 1.0, 2.0])
    ref = O.smoothed_simple_stage(b.am, b.lm, b.symbols, b.t_len, b.u_len, b.wl.blank, a, bw, scale=sc)
    batch = make_dev_batch(b)
    got = P.rnnt_simple_loss(batch, b.V, dev_f32(b.am), dev_f32(b.lm), dev_f32(sc), want_logprobs=True,
                             want_grads=True, lm_only_scale=a, am_only_scale=bw)
    torch.cuda.synchronize()
    assert_close("px", host(got["px"]), ref["px"], atol=5e-5)
    assert_close("py", host(got["py"]), ref["py"], atol=5e-5)
    assert_close("loss", host(got["loss"]), ref["loss"], rtol=1e-5)
    assert_close("px_occ", host(got["px_occ"]), ref["gx"], atol=1e-4)
    assert_close("py_occ", host(got["py_occ"]), ref["gy"], atol=1e-4)
    assert_close("am_grad", host(got["am_grad"]), ref["am_grad"], atol=1e-4)
    assert_close("lm_grad", host(got["lm_grad"]), ref["lm_grad"], atol=1e-4)


def test_smoothed_simple_loss_large_vocabulary():
    # V >= 2048: the contractions take 128 x 128 tiles (V = 2100: a ragged
    # last column tile)
    a, bw = 0.25, 0.1
    b = make_batch("bpe", seed=14, N=2, T_range=(100, 140), U_range=(20, 40), V=2100, J=32, S=4)
    say(f"[smoothed] V = {b.V}")
    sc = np.array([0.5, 2.0])
    ref = O.smoothed_simple_stage(b.am, b.lm, b.symbols, b.t_len, b.u_len, b.wl.blank, a, bw, scale=sc)
    batch = make_dev_batch(b)
    got = P.rnnt_simple_loss(batch, b.V, dev_f32(b.am), dev_f32(b.lm), dev_f32(sc), want_logprobs=True,
                             want_grads=True, lm_only_scale=a, am_only_scale=bw)
    torch.cuda.synchronize()
    assert_close("px", host(got["px"]), ref["px"], atol=5e-5)
    assert_close("py", host(got["py"]), ref["py"], atol=5e-5)
    assert_close("loss", host(got["loss"]), ref["loss"], rtol=1e-5)
    assert_close("px_occ", host(got["px_occ"]), ref["gx"], atol=1e-4)
    assert_close("py_occ", host(got["py_occ"]), ref["gy"], atol=1e-4)
    assert_close("am_grad", host(got["am_grad"]), ref["am_grad"], atol=1e-4)
    assert_close("lm_grad", host(got["lm_grad"]), ref["lm_grad"], atol=1e-4)


def test_smoothed_backward_entry_equals_the_direct_gradients():
    b = _batch(seed=12)
    say("[smoothed] split backward")
    batch = make_dev_batch(b)
    am, lm = dev_f32(b.am), dev_f32(b.lm)
    kw = dict(lm_only_scale=0.25, am_only_scale=0.1)
    direct = P.rnnt_simple_loss(batch, b.V, am, lm, want_grads=True, **kw)
    ws = torch.empty(P.simple_loss_workspace_size(b.N, b.T, b.U, b.V), dtype=torch.uint8, device=am.device)
    fwd = P.rnnt_simple_loss(batch, b.V, am, lm, workspace=ws, **kw)
    split = P.rnnt_simple_loss_backward(batch, b.V, am, lm, fwd["px_occ"], ws, **kw)
    torch.cuda.synchronize()
    assert torch.equal(direct["am_grad"], split["am_grad"])
    assert torch.equal(direct["lm_grad"], split["lm_grad"])


def test_smoothed_training_step():
    b = _batch(seed=13)
    S = b.wl.S
    a, bw = 0.25, 0.1
    say("[smoothed] fused step")
    s1 = O.smoothed_simple_stage(b.am, b.lm, b.symbols, b.t_len, b.u_len, b.wl.blank, a, bw,
                                 scale=np.full(b.N, 0.5))
    ranges = O.prune_ranges(s1["gx"], s1["gy"], b.t_len, b.u_len, S)
    st = O.pruned_stage(b.enc, b.dec, b.W, b.bias, ranges, b.symbols, b.t_len, b.u_len, b.wl.blank)
    batch = make_dev_batch(b)
    step = P.PrunedRnntLoss(S, simple_scale=0.5, lm_only_scale=a, am_only_scale=bw)
    out = step.step(batch, dev_f32(b.am), dev_f32(b.lm), dev_joiner(b.enc, False), dev_joiner(b.dec, False),
                    dev_joiner(b.W, False), dev_joiner(b.bias, False))
    torch.cuda.synchronize()
    assert_close("simple_loss", host(out["simple_loss"]), s1["loss"], rtol=1e-5)
    assert_close("am_grad", host(out["am_grad"]), s1["am_grad"], atol=1e-4)
    assert_close("lm_grad", host(out["lm_grad"]), s1["lm_grad"], atol=1e-4)
    got_r = out["ranges"].cpu().numpy()
    ranges_valid(got_r, b.t_len, b.u_len, S)
    from gpu_common import near_tie_utterances
    amb = near_tie_utterances(s1["gx"], s1["gy"], b.t_len, b.u_len, S)
    for n in range(b.N):
        if n in amb:
            continue
        assert np.array_equal(got_r[n], ranges[n])
        assert_close(f"pruned_loss[{n}]", host(out["pruned_loss"])[n], st["loss"][n], rtol=1e-5)
