"""GPU edge cases against the oracle: empty and one-frame utterances, a band
that covers the whole lattice, a blank other than 0 (and a token equal to
blank), NaN in the padding, out-of-range lengths and symbols, an infeasible
band, S = 1 and the largest S, and U near the lattice limit.

Each case is a small batch whose oracle pipeline finishes in well under a
second; every batch still has ragged lengths and V not a multiple of the
tile width.
"""
import dataclasses

import numpy as np
import pytest
import torch

import oracle as O
import paper_2206_13236_amd as P
from gpu_common import (assert_close, check_step, dev_f32, dev_i32, host, make_dev_batch, oracle_step,
                        run_step, say)
from workloads import Workload, make_batch

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    assert torch.cuda.is_available(), "GPU tests need a ROCm device"
    P.lib()


def _small(seed=0, N=4, T_range=(12, 30), U_range=(3, 9), V=29, J=32, S=4, **wl_over):
    b = make_batch("bpe", seed=seed, N=N, T_range=T_range, U_range=U_range, V=V, J=J, S=S)
    if wl_over:
        b = dataclasses.replace(b, wl=Workload(**{**b.wl.__dict__, **wl_over}))
    return b


def _with_lengths(b, t_len=None, u_len=None):
    t = b.t_len.copy() if t_len is None else np.asarray(t_len, np.int32)
    u = b.u_len.copy() if u_len is None else np.asarray(u_len, np.int32)
    return dataclasses.replace(b, t_len=t, u_len=u)


def test_empty_transcripts():
    # U_n = 0 for some utterances: the lattice is one row, the loss the sum of blanks
    b = _with_lengths(_small(seed=1), u_len=[0, 5, 0, 3])
    say("[edge] U_n = 0")
    out = run_step(b, 4)
    check_step(out, oracle_step(b, 4), b, 4)


def test_all_transcripts_empty():
    b = _small(seed=2, U_range=(0, 0))
    assert b.U == 0
    say("[edge] U = 0 for the whole batch")
    out = run_step(b, 3)
    check_step(out, oracle_step(b, 3), b, 3)


def test_one_frame_utterances():
    # T_n = 1: one column; U_n <= (S-1) * T_n keeps the band feasible
    b = _with_lengths(_small(seed=3), t_len=[1, 17, 1, 9], u_len=[2, 7, 0, 4])
    say("[edge] T_n = 1")
    out = run_step(b, 4)
    check_step(out, oracle_step(b, 4), b, 4)


def test_band_covering_the_lattice_equals_the_full_loss():
    # S >= U+1: every p_t = 0 and the pruned loss is the unpruned loss (Sec. 3.2)
    b = _small(seed=4, U_range=(2, 5))
    S = b.U + 1
    say(f"[edge] S = U+1 = {S}")
    out = run_step(b, S)
    assert np.all(out["ranges"] == np.arange(S)[None, None, :])
    full, _, _ = O.full_joiner_loss(b.enc, b.dec, b.W, b.bias, b.symbols, b.t_len, b.u_len, b.wl.blank)
    assert_close("pruned_loss vs full loss", out["pruned_loss"], full, rtol=1e-5)
    check_step(out, oracle_step(b, S), b, S)


def test_blank_not_zero_and_token_equal_to_blank():
    b = _small(seed=5, blank=7)
    sym = b.symbols.copy()
    sym[0, 1] = 7  # a token equal to blank inside the transcript
    sym[2, 0] = 7
    b = dataclasses.replace(b, symbols=sym)
    say("[edge] blank = 7")
    out = run_step(b, 4)
    check_step(out, oracle_step(b, 4), b, 4)


def test_nan_in_padding_is_ignored():
    b = _small(seed=6)
    am, lm, enc, dec = b.am.copy(), b.lm.copy(), b.enc.copy(), b.dec.copy()
    for n in range(b.N):
        am[n, b.t_len[n]:] = np.nan
        lm[n, b.u_len[n] + 1:] = np.nan
        enc[n, b.t_len[n]:] = np.nan
        dec[n, b.u_len[n] + 1:] = np.nan
    poisoned = dataclasses.replace(b, am=am, lm=lm, enc=enc, dec=dec)
    say("[edge] NaN padding")
    out = run_step(poisoned, 4)
    for k in ("simple_loss", "pruned_loss", "enc_grad", "dec_grad", "W_grad", "bias_grad", "am_grad", "lm_grad"):
        assert np.all(np.isfinite(out[k])), f"{k} has non-finite values"
    check_step(out, oracle_step(b, 4), b, 4)
    # padding rows of the gradients are zero
    for n in range(b.N):
        assert np.all(out["am_grad"][n, b.t_len[n]:] == 0) and np.all(out["enc_grad"][n, b.t_len[n]:] == 0)
        assert np.all(out["lm_grad"][n, b.u_len[n] + 1:] == 0) and np.all(out["dec_grad"][n, b.u_len[n] + 1:] == 0)


def test_out_of_range_lengths_and_symbols_give_nan_for_that_utterance_only():
    b = _small(seed=7, N=5)
    t_len, u_len, sym = b.t_len.copy(), b.u_len.copy(), b.symbols.copy()
    t_len[1] = b.T + 3       # longer than the padded T
    u_len[2] = -1            # negative transcript length
    sym[3, 0] = b.V + 5      # symbol outside [0, V)
    bad = dataclasses.replace(b, t_len=t_len, u_len=u_len, symbols=sym)
    say("[edge] invalid lengths / symbols")
    out = run_step(bad, 4)
    for n in (1, 2, 3):
        assert np.isnan(out["simple_loss"][n]) and np.isnan(out["pruned_loss"][n]), f"utterance {n}"
    good = [0, 4]
    ref = oracle_step(b, 4, idx=good)
    check_step(out, ref, b, 4, whole_batch=False)


def test_infeasible_band_gives_inf_and_zero_joiner_gradients():
    # U_n > (S-1) T_n: no band admits a complete path
    b = _with_lengths(_small(seed=8, T_range=(10, 20), U_range=(6, 9)), t_len=[2, 15, 3, 12], u_len=[7, 8, 9, 6])
    S = 3
    say("[edge] infeasible band")
    out = run_step(b, S)
    ref = oracle_step(b, S)
    check_step(out, ref, b, S)
    infeasible = [n for n in range(b.N) if b.u_len[n] > (S - 1) * b.t_len[n]]
    assert infeasible == [0, 2]
    for n in infeasible:
        assert out["pruned_loss"][n] == np.inf and ref["st"]["loss"][n] == np.inf
        assert np.all(out["enc_grad"][n] == 0) and np.all(out["dec_grad"][n] == 0)


def test_s_equal_one():
    # S = 1: one node per frame, feasible only for U_n = 0
    b = _small(seed=9, U_range=(0, 0))
    say("[edge] S = 1")
    out = run_step(b, 1)
    check_step(out, oracle_step(b, 1), b, 1)


def test_largest_s():
    b = _small(seed=10, N=2, T_range=(20, 26), U_range=(30, 40), V=19, S=32)
    say("[edge] S = 32")
    out = run_step(b, 32)
    check_step(out, oracle_step(b, 32), b, 32)


def test_long_transcript_near_the_lattice_limit():
    # U close to the 1023-row limit: 16 lattice rows per lane in the wavefront
    b = _small(seed=11, N=2, T_range=(40, 48), U_range=(990, 1000), V=13, J=16, S=32)
    say(f"[edge] U = {b.U}")
    batch = make_dev_batch(b)
    sc = np.full(b.N, 0.5, np.float32)
    got = P.rnnt_simple_loss(batch, b.V, dev_f32(b.am), dev_f32(b.lm), dev_f32(sc), want_grads=True)
    torch.cuda.synchronize()
    s1 = O.simple_stage(b.am, b.lm, b.symbols, b.t_len, b.u_len, b.wl.blank, scale=sc)
    assert_close("loss", host(got["loss"]), s1["loss"], rtol=1e-5)
    assert_close("px_occ", host(got["px_occ"]), s1["gx"], atol=1e-4)
    assert_close("py_occ", host(got["py_occ"]), s1["gy"], atol=1e-4)
    assert_close("am_grad", host(got["am_grad"]), s1["am_grad"], atol=1e-4)
    assert_close("lm_grad", host(got["lm_grad"]), s1["lm_grad"], atol=1e-4)


@pytest.mark.parametrize("U_range,R", [((140, 150), 3), ((260, 300), 5), ((330, 370), 6), ((450, 500), 8),
                                       ((705, 760), 12)])
def test_simple_stage_at_every_lattice_width(U_range, R):
    # the recursion's wave holds R lattice rows per lane (the fewest that
    # hold U + 1 rows up to 6, then 8, 12, 16); ragged U inside each range
    b = _small(seed=13, N=3, T_range=(30, 40), U_range=U_range, V=11, J=16, S=8)
    need = -(-(b.U + 1) // 64)
    assert R == (need if need <= 6 else 8 if need <= 8 else 12 if need <= 12 else 16)
    say(f"[edge] simple stage, U = {b.U} ({R} rows per lane)")
    batch = make_dev_batch(b)
    sc = np.full(b.N, 0.5, np.float32)
    got = P.rnnt_simple_loss(batch, b.V, dev_f32(b.am), dev_f32(b.lm), dev_f32(sc), want_grads=True)
    torch.cuda.synchronize()
    s1 = O.simple_stage(b.am, b.lm, b.symbols, b.t_len, b.u_len, b.wl.blank, scale=sc)
    assert_close("loss", host(got["loss"]), s1["loss"], rtol=1e-5)
    assert_close("px_occ", host(got["px_occ"]), s1["gx"], atol=1e-4)
    assert_close("py_occ", host(got["py_occ"]), s1["gy"], atol=1e-4)
    assert_close("am_grad", host(got["am_grad"]), s1["am_grad"], atol=1e-4)
    assert_close("lm_grad", host(got["lm_grad"]), s1["lm_grad"], atol=1e-4)


def test_simple_stage_with_the_large_vocabulary_tiles():
    # V >= 2048: normaliser, d am and d lm take 128 x 128 tiles; ragged T, U
    # and V (2100 = 16 x 128 + 52), two tiles along T and along U + 1
    b = _small(seed=14, N=3, T_range=(130, 150), U_range=(128, 140), V=2100, J=16, S=8)
    say(f"[edge] simple stage, V = {b.V}, T = {b.T}, U = {b.U}")
    batch = make_dev_batch(b)
    sc = np.array([0.5, 1.0, 2.0], np.float32)
    got = P.rnnt_simple_loss(batch, b.V, dev_f32(b.am), dev_f32(b.lm), dev_f32(sc), want_grads=True)
    torch.cuda.synchronize()
    s1 = O.simple_stage(b.am, b.lm, b.symbols, b.t_len, b.u_len, b.wl.blank, scale=sc)
    assert_close("loss", host(got["loss"]), s1["loss"], rtol=1e-5)
    assert_close("px_occ", host(got["px_occ"]), s1["gx"], atol=1e-4)
    assert_close("py_occ", host(got["py_occ"]), s1["gy"], atol=1e-4)
    assert_close("am_grad", host(got["am_grad"]), s1["am_grad"], atol=1e-4)
    assert_close("lm_grad", host(got["lm_grad"]), s1["lm_grad"], atol=1e-4)


@pytest.mark.parametrize("cfg", [
    # T <= 32: one frame range, d lm finished in the kernel; V = 11: every
    # target in one column tile (more than one gather round of 32), scalar loads
    dict(seed=16, N=3, T_range=(20, 32), U_range=(90, 110), V=11),
    # 64 utterances x 8 column tiles: one frame range over several steps
    dict(seed=17, N=64, T_range=(40, 70), U_range=(20, 60), V=500),
    # a few workgroups: several frame ranges, partial sums finished by dlm_epi
    dict(seed=18, N=2, T_range=(90, 130), U_range=(40, 63), V=130),
    # the u extents the kernel is built for (64, 128, 192, 320) at and just
    # past each boundary; U + 1 = 321 takes the separate d am and d lm kernels
    dict(seed=19, N=3, T_range=(30, 50), U_range=(127, 127), V=70),
    dict(seed=20, N=3, T_range=(30, 50), U_range=(128, 128), V=70),
    dict(seed=21, N=2, T_range=(30, 40), U_range=(191, 192), V=70),
    dict(seed=22, N=2, T_range=(30, 40), U_range=(319, 319), V=70),
    dict(seed=23, N=2, T_range=(30, 40), U_range=(320, 320), V=70),
])
def test_simple_grads_fused_kernel_paths(cfg):
    # d am and d lm of the plain trivial joiner come from one kernel for
    # U + 1 <= 320; every branch of its launch and of its target lists
    c = dict(cfg)
    b = _small(seed=c.pop("seed"), J=16, S=4, **c)
    say(f"[edge] simple grads, N = {b.N}, T = {b.T}, U = {b.U}, V = {b.V}")
    batch = make_dev_batch(b)
    sc = (0.5 + np.random.default_rng(3).random(b.N)).astype(np.float32)
    got = P.rnnt_simple_loss(batch, b.V, dev_f32(b.am), dev_f32(b.lm), dev_f32(sc), want_grads=True)
    torch.cuda.synchronize()
    s1 = O.simple_stage(b.am, b.lm, b.symbols, b.t_len, b.u_len, b.wl.blank, scale=sc)
    assert_close("loss", host(got["loss"]), s1["loss"], rtol=1e-5)
    assert_close("am_grad", host(got["am_grad"]), s1["am_grad"], atol=1e-4)
    assert_close("lm_grad", host(got["lm_grad"]), s1["lm_grad"], atol=1e-4)


def test_step_with_the_wide_forward_tiles():
    # bf16 at V >= 2048: the joiner forward takes 256 x 256 tiles of 16
    # waves; ragged rows (M = S sum T_n is no multiple of 256) and columns
    # (2100 = 8 x 256 + 52); every output of the step against the oracle
    b = _small(seed=15, N=3, T_range=(40, 60), U_range=(10, 20), V=2100, J=64, S=5, joiner_dtype="bf16")
    say(f"[edge] step with the wide forward tiles, V = {b.V}, M = {5 * int(b.t_len.sum())}")
    out = run_step(b, 5)
    check_step(out, oracle_step(b, 5), b, 5)


@pytest.mark.parametrize("alg,chunk", [("wavefront", 0), ("scan", 0), ("scan", 1), ("scan", 2), ("scan", 7)])
def test_band_algorithms_on_a_mixed_batch(alg, chunk):
    # T_n = 1, U_n = 0, an infeasible utterance and ragged lengths in one
    # batch; bounds from the oracle's pruning of random occupations
    N, T, U, S = 6, 23, 9, 4
    rng = np.random.default_rng(21)
    t_len = np.array([1, 23, 5, 17, 2, 11], np.int32)
    u_len = np.array([0, 9, 3, 6, 7, 0], np.int32)
    gx = rng.random((N, T, U + 1))
    gy = rng.random((N, T, U + 1))
    ranges = O.prune_ranges(gx, gy, t_len, u_len, S)
    px = (-1.0 - np.abs(rng.standard_normal((N, T, S)))).astype(np.float32)
    py = (-1.0 - np.abs(rng.standard_normal((N, T, S)))).astype(np.float32)
    loss_ref, gx_ref, gy_ref = O.pruned_loss(px.astype(np.float64), py.astype(np.float64), ranges, t_len, u_len)
    assert loss_ref[4] == np.inf  # U_n = 7 > (S-1) T_n = 6
    b = dataclasses.replace(_small(seed=12, N=N, T_range=(T, T), U_range=(U, U), S=S), t_len=t_len, u_len=u_len)
    say(f"[edge] mixed batch, band algorithm {alg} chunk {chunk}")
    batch = make_dev_batch(b)
    r = P.rnnt_pruned_loss(batch, S, dev_f32(px), dev_f32(py), dev_i32(ranges), algorithm=alg, chunk=chunk)
    torch.cuda.synchronize()
    assert_close("loss", host(r["loss"]), loss_ref, rtol=1e-5)
    assert_close("px_occ", host(r["px_occ"]), gx_ref, atol=1e-4)
    assert_close("py_occ", host(r["py_occ"]), gy_ref, atol=1e-4)


@pytest.mark.parametrize("U_range", [(3, 9), (70, 90)])
def test_nan_inside_the_lattice_gives_nan_for_that_utterance_only(U_range):
    # a NaN logit at a node of the lattice (one row or more per lane of the
    # recursion's wave): that utterance's simple loss is NaN, the others
    # match the oracle on the clean batch
    b = _small(seed=31, N=4, T_range=(12, 30), U_range=U_range)
    am, lm = b.am.copy(), b.lm.copy()
    am[1, min(2, b.t_len[1] - 1), 3] = np.nan
    lm[2, b.u_len[2] // 2, 5] = np.nan
    say(f"[edge] NaN inside the lattice, U in {U_range}")
    batch = make_dev_batch(b)
    sc = np.full(b.N, 0.5, np.float32)
    got = P.rnnt_simple_loss(batch, b.V, dev_f32(am), dev_f32(lm), dev_f32(sc), want_grads=True)
    torch.cuda.synchronize()
    loss = host(got["loss"])
    assert np.isnan(loss[1]) and np.isnan(loss[2])
    good = [0, 3]
    s1 = O.simple_stage(b.am[good], b.lm[good], b.symbols[good], b.t_len[good], b.u_len[good], b.wl.blank,
                        scale=sc[good])
    assert_close("loss", loss[good], s1["loss"], rtol=1e-5)
    assert_close("px_occ", host(got["px_occ"])[good], s1["gx"], atol=1e-4)
    assert_close("py_occ", host(got["py_occ"])[good], s1["gy"], atol=1e-4)
    assert_close("am_grad", host(got["am_grad"])[good], s1["am_grad"], atol=1e-4)


@pytest.mark.parametrize("alg,chunk", [("wavefront", 0), ("scan", 0), ("scan", 3)])
def test_nan_inside_the_band_gives_nan_for_that_utterance_only(alg, chunk):
    N, T, U, S = 4, 19, 8, 4
    rng = np.random.default_rng(33)
    t_len = np.array([19, 14, 9, 17], np.int32)
    u_len = np.array([8, 5, 3, 6], np.int32)
    ranges = O.prune_ranges(rng.random((N, T, U + 1)), rng.random((N, T, U + 1)), t_len, u_len, S)
    px = (-1.0 - np.abs(rng.standard_normal((N, T, S)))).astype(np.float32)
    py = (-1.0 - np.abs(rng.standard_normal((N, T, S)))).astype(np.float32)
    loss_ref, gx_ref, gy_ref = O.pruned_loss(px.astype(np.float64), py.astype(np.float64), ranges, t_len, u_len)
    bad = px.copy()
    bad[1, 4, 1] = np.nan
    b = dataclasses.replace(_small(seed=13, N=N, T_range=(T, T), U_range=(U, U), S=S), t_len=t_len, u_len=u_len)
    say(f"[edge] NaN inside the band, algorithm {alg} chunk {chunk}")
    batch = make_dev_batch(b)
    r = P.rnnt_pruned_loss(batch, S, dev_f32(bad), dev_f32(py), dev_i32(ranges), algorithm=alg, chunk=chunk)
    torch.cuda.synchronize()
    loss = host(r["loss"])
    assert np.isnan(loss[1])
    good = [0, 2, 3]
    assert_close("loss", loss[good], loss_ref[good], rtol=1e-5)
    assert_close("px_occ", host(r["px_occ"])[good], gx_ref[good], atol=1e-4)
    assert_close("py_occ", host(r["py_occ"])[good], gy_ref[good], atol=1e-4)
