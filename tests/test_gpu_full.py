"""Parity at the full workload sizes, in the configuration the benchmark times
(PrunedRnntLoss.step: no [N, T, S, V] logits kept, the backward recomputes
them in chunks of rows).

- bpe and long (the two V=500, S=5 workloads): the oracle's whole pipeline on
  the whole batch, every output of every utterance compared (stage 4 and
  the bounds on the GPU's own occupations, see gpu_common.check_step).
- largev: the same on two sampled utterances of the full batch, and on those
  two as a batch of their own (so that dW and db are compared too), with the
  library's chunking and with chunks of 1,024 rows.
- stress: one full utterance as a batch of its own (two backward chunks),
  every output compared, in two tests (the oracle's simple stage, then its
  pruned stage: about a minute each); on the full batch the oracle checks
  sampled outputs one by one: the trivial joiner's log-probs on sampled
  frames, and the pruned joiner's on sampled frames of a full-size launch
  with fixed, valid bounds.

Every workload is also checked against properties that hold at any size:
flow conservation of both lattices' occupations, zero row sums of the
log-softmax backward, and valid bounds.
"""
import numpy as np
import pytest
import torch

import oracle as O
import paper_2206_13236_amd as P
from gpu_common import (assert_close, check_pruned_part, check_simple_part, check_step, dev_f32, dev_i32,
                        dev_joiner, host, make_dev_batch, oracle_step, own_bounds, ranges_valid, run_step, say,
                        sub_batch)
from workloads import make_batch

pytestmark = pytest.mark.gpu

_RUNS = {}


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    assert torch.cuda.is_available(), "GPU tests need a ROCm device"
    P.lib()
    yield
    _RUNS.clear()


def _run(name):
    if name not in _RUNS:
        _RUNS.clear()  # one full-size workload resident at a time
        b = make_batch(name, seed=0)
        say(f"[full] {name}: N={b.N} T={b.T} U={b.U} V={b.V} S={b.wl.S} J={b.wl.J} {b.wl.joiner_dtype}")
        _RUNS[name] = (b, run_step(b, b.wl.S))
        torch.cuda.empty_cache()
    return _RUNS[name]


@pytest.mark.parametrize("name", ["bpe", "long", "largev", "stress"])
def test_full_size_invariants(name):
    b, out = _run(name)
    S = b.wl.S
    ranges_valid(out["ranges"], b.t_len, b.u_len, S)
    for n in range(b.N):
        Tn, Un = int(b.t_len[n]), int(b.u_len[n])
        assert np.isfinite(out["simple_loss"][n]) and out["simple_loss"][n] > 0
        assert np.isfinite(out["pruned_loss"][n]) and out["pruned_loss"][n] > 0
        # every complete path crosses each frame through one blank edge and emits each token once
        gy, gx = out["simple_py_occ"][n], out["simple_px_occ"][n]
        assert_close(f"sum_u gy[{n}]", gy[:Tn, :Un + 1].sum(1), np.ones(Tn), atol=2e-4)
        if Un > 0:
            assert_close(f"sum_t gx[{n}]", gx[:Tn, :Un].sum(0), np.ones(Un), atol=2e-4)
        assert_close(f"band sum_s gy[{n}]", out["pruned_py_occ"][n, :Tn].sum(1), np.ones(Tn), atol=2e-4)
        # the log-softmax backward has zero row sums
        assert_close(f"am_grad rows[{n}]", out["am_grad"][n].sum(1), np.zeros(b.T), atol=2e-4)
        assert_close(f"lm_grad rows[{n}]", out["lm_grad"][n].sum(1), np.zeros(b.U + 1), atol=2e-4)
    assert abs(out["bias_grad"].sum()) <= 1e-4 * max(1.0, np.abs(out["bias_grad"]).max()) * np.sqrt(b.V)


@pytest.mark.parametrize("name", ["bpe", "long", "largev", "stress"])
def test_full_size_band_recursion_against_oracle(name):
    # both algorithms of the pruned recursion at the full size, on the GPU
    # joiner's own band log-probs and bounds (fp32, as the library takes them)
    b, out = _run(name)
    S = b.wl.S
    px, py, rg = out["px"].astype(np.float32), out["py"].astype(np.float32), out["ranges"]
    say(f"[full] {name}: oracle band recursion")
    loss_ref, gx_ref, gy_ref = O.pruned_loss(px.astype(np.float64), py.astype(np.float64), rg, b.t_len, b.u_len)
    batch = make_dev_batch(b)
    for alg in ("wavefront", "scan"):
        say(f"[full] {name}: band algorithm {alg}")
        r = P.rnnt_pruned_loss(batch, S, dev_f32(px), dev_f32(py), dev_i32(rg), algorithm=alg)
        torch.cuda.synchronize()
        assert_close(f"{alg} loss", host(r["loss"]), loss_ref, rtol=1e-5)
        assert_close(f"{alg} px_occ", host(r["px_occ"]), gx_ref, atol=1e-4)
        assert_close(f"{alg} py_occ", host(r["py_occ"]), gy_ref, atol=1e-4)


@pytest.mark.parametrize("name", ["bpe", "long"])
def test_full_size_whole_batch_against_oracle(name):
    b, out = _run(name)
    say(f"[full] {name}: oracle on all {b.N} utterances")
    amb = check_step(out, oracle_step(b, b.wl.S), b, b.wl.S)
    say(f"  near-tie utterances {sorted(amb)}")


def _largev_pick(b):
    return sorted({int(np.argmin(b.t_len)), int(np.argmax(b.u_len))})


def test_full_size_largev_sampled_utterances():
    b, out = _run("largev")
    idx = _largev_pick(b)
    say(f"[full] largev: oracle on utterances {idx}")
    check_step(out, oracle_step(b, b.wl.S, idx=idx), b, b.wl.S, whole_batch=False)


@pytest.mark.parametrize("chunk", [0, 1024])
def test_largev_two_utterances_as_a_batch(chunk):
    # V = 5000, J = 512, fp32: every output including dW and db; chunks of
    # 1,024 rows split the ~2,500 rows three ways (S = 5 does not divide 1,024,
    # so frames straddle chunk edges)
    full = make_batch("largev", seed=0)
    b = sub_batch(full, _largev_pick(full))
    say(f"[full] largev as a 2-utterance batch, backward chunk {chunk or 'default'}")
    out = run_step(b, b.wl.S, bwd_chunk_rows=chunk)
    check_step(out, oracle_step(b, b.wl.S), b, b.wl.S)


_STRESS1 = {}


def _stress_one():
    """Utterance 0 of the stress batch as a batch of its own (T = 970, U_n = 217,
    V = 8000, J = 768, S = 10, bf16 joiner): 9,700 padded rows, two backward
    chunks."""
    if not _STRESS1:
        _RUNS.clear()
        b = sub_batch(make_batch("stress", seed=0), [0])
        say(f"[full] stress utterance 0: T={b.t_len[0]} U={b.u_len[0]} V={b.V}")
        _STRESS1["b"] = b
        _STRESS1["out"] = run_step(b, b.wl.S)
        torch.cuda.empty_cache()
    return _STRESS1["b"], _STRESS1["out"]


def test_stress_utterance_simple_stage_against_oracle():
    b, out = _stress_one()
    say("[full] stress utterance 0: oracle simple stage (about a minute)")
    ref = oracle_step(b, b.wl.S)
    check_simple_part(out, ref, b, b.wl.S)
    _STRESS1["simple_loss"] = ref["s1"]["loss"]


def test_stress_utterance_pruned_stage_against_oracle():
    b, out = _stress_one()
    say("[full] stress utterance 0: oracle pruned stage on the GPU's bounds (about a minute)")
    idx = np.arange(b.N)
    r = own_bounds(out, b, b.wl.S, idx)
    assert np.array_equal(out["ranges"], r)
    check_pruned_part(out, b, b.wl.S, idx, r, simple_loss=_STRESS1.get("simple_loss"))


def _fixed_bounds(t_len, u_len, T, S):
    """A valid band independent of any occupation: p_t = floor(t P / (T_n - 1))."""
    N = len(t_len)
    r = np.tile(np.arange(S, dtype=np.int32), (N, T, 1))
    for n in range(N):
        Tn, Un = int(t_len[n]), int(u_len[n])
        P = max(0, Un - S + 1)
        t = np.arange(Tn)
        p = (t * P) // max(Tn - 1, 1)
        r[n, :Tn] = (p[:, None] + np.arange(S)[None, :]).astype(np.int32)
    return r


def test_full_size_stress_sampled_outputs():
    b = make_batch("stress", seed=0)
    S = b.wl.S
    _RUNS.clear()
    say(f"[full] stress sampled: N={b.N} T={b.T} U={b.U} V={b.V}")
    batch = make_dev_batch(b)
    rng = np.random.default_rng(123)
    picks = [(n, int(t)) for n in (0, b.N - 1) for t in rng.integers(0, b.t_len[n], size=3)]
    # trivial joiner log-probs (Eqs. (1)-(2), (5)-(6)) on sampled frames
    s = P.rnnt_simple_loss(batch, b.V, dev_f32(b.am), dev_f32(b.lm), want_logprobs=True)
    torch.cuda.synchronize()
    px, py = host(s["px"]), host(s["py"])
    del s
    for n, t in picks:
        Un = int(b.u_len[n])
        _, opx, opy = O.trivial_joiner_logprobs(b.am[n:n + 1, t:t + 1], b.lm[n:n + 1], b.symbols[n:n + 1],
                                                np.array([1]), np.array([Un]), b.wl.blank)
        assert_close(f"px[{n},{t}]", px[n, t, :Un + 1], opx[0, 0, :Un + 1], atol=5e-5)
        assert_close(f"py[{n},{t}]", py[n, t, :Un + 1], opy[0, 0, :Un + 1], atol=5e-5)
    # pruned joiner (full size, bf16 inputs) with fixed valid bounds, on sampled frames
    ranges = _fixed_bounds(b.t_len, b.u_len, b.T, S)
    ranges_valid(ranges, b.t_len, b.u_len, S)
    bf = True
    jo = P.rnnt_pruned_joiner(batch, S, dev_joiner(b.enc, bf), dev_joiner(b.dec, bf), dev_joiner(b.W, bf),
                              dev_joiner(b.bias, bf), dev_i32(ranges), keep_logits=True)
    torch.cuda.synchronize()
    jpx, jpy, jlse = host(jo["px"]), host(jo["py"]), host(jo["lse"])
    for n, t in picks:
        sl = (slice(n, n + 1), slice(t, t + 1))
        opx, opy, olse = O.pruned_joiner_logprobs(b.enc[sl], b.dec[n:n + 1], b.W, b.bias, ranges[sl],
                                                  b.symbols[n:n + 1], np.array([1]), b.u_len[n:n + 1],
                                                  b.wl.blank)
        assert_close(f"joiner px[{n},{t}]", jpx[n, t], opx[0, 0], atol=2e-2)
        assert_close(f"joiner py[{n},{t}]", jpy[n, t], opy[0, 0], atol=2e-2)
        assert_close(f"joiner lse[{n},{t}]", jlse[n, t], olse[0, 0], atol=2e-2, rtol=2e-2)
        lg = O.pruned_joiner_logits(b.enc[sl], b.dec[n:n + 1], b.W, b.bias, ranges[sl], np.array([1]),
                                    b.u_len[n:n + 1])
        present = ~np.isnan(lg[0, 0, :, 0])
        assert_close(f"logits[{n},{t}]", host(jo["logits"][n, t])[present], lg[0, 0][present], atol=2e-2)
