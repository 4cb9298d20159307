"""The unpruned loss (the (N, T, U+1, V) joiner the method avoids) on the GPU
against the oracle: loss against the oracle's own full-joiner loss, and every
gradient against the oracle's joiner backward with the band covering the
whole lattice (all p_t = 0, S = U+1)."""
import numpy as np
import pytest
import torch

import oracle as O
import paper_2206_13236_amd as P
from gpu_common import assert_close, dev_f32, dev_joiner, grad_atol, host, loss_rtol, make_dev_batch, say
from workloads import make_batch

pytestmark = pytest.mark.gpu

CASES = {
    "tiny": dict(wl="tiny"),
    "small_f32": dict(wl="bpe", N=3, T_range=(20, 40), U_range=(3, 12), V=37, J=64),
    "small_bf16": dict(wl="long", N=2, T_range=(20, 30), U_range=(5, 10), V=72, J=64),
    "small_bf16_oddv": dict(wl="long", N=2, T_range=(20, 30), U_range=(5, 10), V=37, J=64),
}


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    assert torch.cuda.is_available(), "GPU tests need a ROCm device"
    P.lib()


@pytest.mark.parametrize("keep", [False, True], ids=["recompute", "stored_logits"])
@pytest.mark.parametrize("name", list(CASES))
def test_full_loss_against_oracle(name, keep):
    c = dict(CASES[name])
    b = make_batch(c.pop("wl"), seed=5, **c)
    bf = b.wl.joiner_dtype == "bf16"
    say(f"[full-loss] {name} keep_logits={keep}")
    sc = (0.5 + np.random.default_rng(3).random(b.N)).astype(np.float32)
    S = b.U + 1
    ranges = np.tile(np.arange(S, dtype=np.int32), (b.N, b.T, 1))
    st = O.pruned_stage(b.enc, b.dec, b.W, b.bias, ranges, b.symbols, b.t_len, b.u_len, b.wl.blank, scale=sc)
    full, _, _ = O.full_joiner_loss(b.enc, b.dec, b.W, b.bias, b.symbols, b.t_len, b.u_len, b.wl.blank)
    assert_close("oracle pruned(S=U+1) vs full", st["loss"], full, rtol=1e-12)
    batch = make_dev_batch(b)
    out = P.rnnt_full_loss(batch, dev_joiner(b.enc, bf), dev_joiner(b.dec, bf), dev_joiner(b.W, bf),
                           dev_joiner(b.bias, bf), scale=dev_f32(sc), keep_logits=keep)
    torch.cuda.synchronize()
    assert_close("loss", host(out["loss"]), full, rtol=loss_rtol(bf))
    for k in ("enc_grad", "dec_grad"):
        assert_close(k, host(out[k]), st[k], atol=grad_atol(st[k], bf))
    for k in ("W_grad", "bias_grad"):
        assert_close(k, host(out[k]), st[k], atol=grad_atol(st[k], bf, param=True))


def test_full_loss_equals_the_pruned_path_with_a_covering_band():
    b = make_batch("bpe", seed=6, N=3, T_range=(20, 40), U_range=(3, 12), V=37, J=64)
    S = b.U + 1
    say(f"[full-loss] vs pruned path, S = {S}")
    batch = make_dev_batch(b)
    args = (dev_joiner(b.enc, False), dev_joiner(b.dec, False), dev_joiner(b.W, False), dev_joiner(b.bias, False))
    full = P.rnnt_full_loss(batch, *args)
    ranges = torch.from_numpy(np.tile(np.arange(S, dtype=np.int32), (b.N, b.T, 1))).to(args[0].device)
    jo = P.rnnt_pruned_joiner(batch, S, *args, ranges)
    pl = P.rnnt_pruned_loss(batch, S, jo["px"], jo["py"], ranges)
    torch.cuda.synchronize()
    assert_close("loss", host(full["loss"]), host(pl["loss"]), rtol=1e-5)
