"""The fused training entry (Sec. 3.3, Sec. 4): the two-stream step, the
warm-up switch, the split simple-loss backward and the autograd Function."""
import dataclasses

import numpy as np
import pytest
import torch

import oracle as O
import paper_2206_13236_amd as P
from gpu_common import (assert_close, check_step, dev_f32, dev_joiner, host, make_dev_batch, oracle_step,
                        run_step, say)
from workloads import make_batch

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    assert torch.cuda.is_available(), "GPU tests need a ROCm device"
    P.lib()


def _batch(seed=0, wl="bpe", **kw):
    kw = {"N": 3, "T_range": (40, 70), "U_range": (5, 20), "V": 37, "J": 64, "S": 5, **kw}
    return make_batch(wl, seed=seed, **kw)


def _dev(b, bf=False):
    return (dev_f32(b.am), dev_f32(b.lm), dev_joiner(b.enc, bf), dev_joiner(b.dec, bf), dev_joiner(b.W, bf),
            dev_joiner(b.bias, bf))


def test_simple_backward_entry_equals_the_direct_gradients():
    b = _batch(seed=1)
    say("[train] simple loss backward entry")
    batch = make_dev_batch(b)
    am, lm = dev_f32(b.am), dev_f32(b.lm)
    sc = dev_f32(np.array([0.5, 1.0, 2.0], np.float32))
    direct = P.rnnt_simple_loss(batch, b.V, am, lm, sc, want_grads=True)
    ws = torch.empty(P.simple_loss_workspace_size(b.N, b.T, b.U, b.V), dtype=torch.uint8, device=am.device)
    fwd = P.rnnt_simple_loss(batch, b.V, am, lm, sc, workspace=ws)
    split = P.rnnt_simple_loss_backward(batch, b.V, am, lm, fwd["px_occ"], ws, scale=sc)
    torch.cuda.synchronize()
    assert torch.equal(direct["loss"], fwd["loss"])
    assert torch.equal(direct["am_grad"], split["am_grad"])
    assert torch.equal(direct["lm_grad"], split["lm_grad"])


@pytest.mark.parametrize("bf", [False, True], ids=["f32", "bf16"])
def test_two_stream_step_equals_one_stream(bf):
    b = _batch(seed=2, wl="long" if bf else "bpe", V=72)
    say(f"[train] overlap vs sequential bf16={bf}")
    batch = make_dev_batch(b)
    args = _dev(b, bf)
    outs = []
    for overlap in (False, True):
        step = P.PrunedRnntLoss(b.wl.S, overlap=overlap)
        o = step.step(batch, *args)
        torch.cuda.synchronize()
        outs.append({k: v.clone() for k, v in o.items()})
    for k in outs[0]:
        assert torch.equal(outs[0][k], outs[1][k]), f"{k} differs between one and two streams"


def test_warmup_switch_skips_the_pruned_stages():
    b = _batch(seed=3)
    say("[train] warm-up (pruned scale 0)")
    batch = make_dev_batch(b)
    args = _dev(b)
    full = P.PrunedRnntLoss(b.wl.S).step(batch, *args)
    full = {k: v.clone() for k, v in full.items()}
    warm = P.PrunedRnntLoss(b.wl.S, pruned_scale=0.0).step(batch, *args)
    torch.cuda.synchronize()
    for k in ("simple_loss", "am_grad", "lm_grad", "simple_px_occ", "simple_py_occ"):
        assert torch.equal(full[k], warm[k]), k
    for k in ("pruned_loss", "enc_grad", "dec_grad", "W_grad", "bias_grad"):
        assert torch.count_nonzero(warm[k]) == 0, k
    assert "ranges" not in warm
    # the training loss is the scaled simple loss alone (formed by the library)
    assert torch.equal(warm["loss"], 0.5 * warm["simple_loss"])
    assert_close("total", host(warm["total"]), host(0.5 * warm["simple_loss"]).sum(), rtol=1e-6)


@pytest.mark.parametrize("reduction", ["sum", "mean"])
def test_autograd_function_against_the_oracle(reduction):
    b = make_batch("tiny", seed=4)
    S = b.wl.S
    say(f"[train] autograd reduction={reduction}")
    batch = make_dev_batch(b)
    am, lm, enc, dec, W, bias = (t.clone().requires_grad_(True) for t in _dev(b))
    loss = P.pruned_rnnt_loss(am, lm, enc, dec, W, bias, batch, S, simple_scale=0.5, reduction=reduction)
    (3.0 * loss).backward()
    torch.cuda.synchronize()
    ref = oracle_step(b, S)
    ref["st"] = O.pruned_stage(b.enc, b.dec, b.W, b.bias, ref["ranges"], b.symbols, b.t_len, b.u_len, b.wl.blank)
    total = 0.5 * ref["s1"]["loss"].sum() + ref["st"]["loss"].sum()
    k = 3.0 / (b.N if reduction == "mean" else 1)
    assert_close("loss", loss.item(), total / (b.N if reduction == "mean" else 1), rtol=1e-5)
    # the oracle's gradients are those of sum_n (0.5 simple_n + pruned_n)
    s1_grads = O.simple_stage(b.am, b.lm, b.symbols, b.t_len, b.u_len, b.wl.blank, scale=np.full(b.N, 0.5))
    assert_close("am.grad", host(am.grad), k * s1_grads["am_grad"], atol=k * 1e-4)
    assert_close("lm.grad", host(lm.grad), k * s1_grads["lm_grad"], atol=k * 1e-4)
    st = ref["st"]
    for t, key in ((enc, "enc_grad"), (dec, "dec_grad"), (W, "W_grad"), (bias, "bias_grad")):
        assert_close(f"{key}", host(t.grad), k * st[key], atol=k * 1e-4 * max(1.0, np.abs(st[key]).max()))
