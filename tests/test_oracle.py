"""Pins for the CPU oracle (runs on CPU, no GPU).

Each check ties the oracle to something other than itself: closed forms of
the uniform lattice, brute-force enumeration of every monotone alignment,
invariants that follow from the lattice's structure, library routines for
single steps, central finite differences, and the worked example the paper
prints for the window score (Sec. 3.2.2, Eq. (7)).
"""
import itertools
import json
import math
import os

import numpy as np
import pytest

import oracle as O
from workloads import make_batch

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def _rand_lattice(rng, T, U, V=11):
    """px/py that are real log-probs of a random trivial joiner."""
    am = rng.standard_normal((1, T, V))
    lm = rng.standard_normal((1, U + 1, V))
    sym = rng.integers(1, V, size=(1, max(U, 1)))[:, :U]
    _, px, py = O.trivial_joiner_logprobs(am, lm, sym, [T], [U], 0)
    return px[0], py[0]


def _brute_force(px, py, T, U):
    """Enumerate every monotone path from (0,0) to (T-1,U) plus the final blank.

    Returns (L, gx, gy): log of the summed path probability and the expected
    number of uses of every vertical/horizontal edge.
    """
    nmov = T - 1 + U
    combos = list(itertools.combinations(range(nmov), U))
    combos = np.array(combos, dtype=np.int64).reshape(len(combos), U)
    P = combos.shape[0]
    up = np.zeros((P, nmov), dtype=bool)
    if U > 0:
        up[np.arange(P)[:, None], combos] = True
    u_before = np.cumsum(up, axis=1) - up
    t_before = np.arange(nmov)[None, :] - u_before
    edge = np.where(up, px[t_before, u_before], py[t_before, u_before])
    score = edge.sum(axis=1) + py[T - 1, U]
    finite = np.isfinite(score)
    m = score[finite].max()
    L = m + math.log(np.exp(score[finite] - m).sum())
    w = np.where(finite, np.exp(score - L), 0.0)
    gx = np.zeros((T, U + 1))
    gy = np.zeros((T, U + 1))
    ww = np.repeat(w[:, None], nmov, axis=1)
    np.add.at(gx, (t_before[up], u_before[up]), ww[up])
    np.add.at(gy, (t_before[~up], u_before[~up]), ww[~up])
    gy[T - 1, U] += w.sum()
    return L, gx, gy


# ---------------------------------------------------------------------------
# Closed forms of the uniform lattice (am = lm = 0  =>  px = py = -log V)
# ---------------------------------------------------------------------------

def test_uniform_lattice_closed_form_tiny_shape():
    T, U, V = 20, 5, 16
    am = np.zeros((1, T, V), np.float32)
    lm = np.zeros((1, U + 1, V), np.float32)
    sym = np.arange(1, U + 1, dtype=np.int32)[None, :]
    out = O.simple_stage(am, lm, sym, [T], [U], 0)
    # every (t,u) normaliser is log V
    np.testing.assert_allclose(out["Z"][0], math.log(V), rtol=0, atol=1e-12)
    # C(T-1+U, U) equally likely paths of T+U transitions of prob 1/V
    paths = math.comb(T - 1 + U, U)
    assert paths == 42504
    L = math.log(paths) - (T + U) * math.log(V)
    assert abs(-out["loss"][0] - L) < 1e-9
    # occupations are ratios of path counts
    tot = math.comb(T - 1 + U, U)
    for t in range(T - 1):
        for u in range(U + 1):
            gy = math.comb(t + u, u) * math.comb(T - 2 - t + U - u, U - u) / tot
            assert abs(out["gy"][0, t, u] - gy) < 1e-12
            if u < U:
                gx = math.comb(t + u, u) * math.comb(T - 2 - t + U - u, U - u - 1) / tot
                assert abs(out["gx"][0, t, u] - gx) < 1e-12


def test_uniform_lattice_general_values():
    # px == x, py == y everywhere: L = log C(T-1+U, U) + U x + T y
    for T, U, x, y in [(7, 3, -1.3, -0.4), (1, 4, -2.0, -0.1), (5, 0, -3.0, -0.7)]:
        px = np.full((T, U + 1), x)
        px[:, U] = -np.inf
        py = np.full((T, U + 1), y)
        r = O.lattice_forward_backward(px, py, T, U)
        L = math.log(math.comb(T - 1 + U, U)) + U * x + T * y
        assert abs(r["L"] - L) < 1e-10


# ---------------------------------------------------------------------------
# Brute force over every alignment
# ---------------------------------------------------------------------------

@pytest.mark.parametrize("T,U", [(1, 0), (1, 3), (4, 0), (3, 2), (6, 3), (20, 5)])
def test_recursion_matches_brute_force(T, U):
    rng = np.random.default_rng(100 + 7 * T + U)
    px, py = _rand_lattice(rng, T, U)
    r = O.lattice_forward_backward(px, py, T, U)
    L, gx, gy = _brute_force(px, py, T, U)
    assert abs(r["L"] - L) < 1e-9 * max(1.0, abs(L))
    np.testing.assert_allclose(r["gx"][:, :U], gx[:, :U], atol=1e-11)
    np.testing.assert_allclose(r["gy"], gy, atol=1e-11)


def test_pruned_recursion_matches_band_restricted_brute_force():
    # The -inf construction of Sec. 3.2: only paths that stay inside the band count.
    rng = np.random.default_rng(5)
    T, U, S = 9, 5, 3
    px, py = _rand_lattice(rng, T, U)
    p = np.array([0, 0, 1, 1, 2, 2, 3, 3, 3])
    ranges = (p[:, None] + np.arange(S)[None, :])[None].astype(np.int32)
    pxb = np.take_along_axis(px, ranges[0], axis=1)[None]
    pyb = np.take_along_axis(py, ranges[0], axis=1)[None]
    pxb[ranges > U - 1] = -np.inf
    loss, gxb, gyb = O.pruned_loss(pxb, pyb, ranges, [T], [U])
    mx = np.full((T, U + 1), -np.inf)
    my = np.full((T, U + 1), -np.inf)
    for t in range(T):
        for s in range(S):
            u = ranges[0, t, s]
            if u <= U:
                mx[t, u] = pxb[0, t, s]
                my[t, u] = pyb[0, t, s]
    L, gx, gy = _brute_force(mx, my, T, U)
    assert abs(-loss[0] - L) < 1e-9 * abs(L)
    for t in range(T):
        for s in range(S):
            u = ranges[0, t, s]
            assert abs(gyb[0, t, s] - gy[t, u]) < 1e-11
            if u < U:
                assert abs(gxb[0, t, s] - gx[t, u]) < 1e-11
    # the vertical edge out of the top of the band leads to a dead node
    assert np.all(gxb[0, :, S - 1] == 0.0)


# ---------------------------------------------------------------------------
# Structural invariants
# ---------------------------------------------------------------------------

def test_alpha_final_equals_beta_start_and_flow_conservation():
    rng = np.random.default_rng(11)
    for T, U in [(13, 4), (30, 9), (2, 7)]:
        px, py = _rand_lattice(rng, T, U)
        r = O.lattice_forward_backward(px, py, T, U)
        assert abs(r["L"] - r["beta"][0, 0]) < 1e-9 * abs(r["L"])
        # every path crosses each frame once and emits each symbol once
        np.testing.assert_allclose(r["gy"].sum(axis=1), 1.0, atol=1e-10)
        np.testing.assert_allclose(r["gx"][:, :U].sum(axis=0), 1.0, atol=1e-10)
        assert np.all(r["gx"] >= 0) and np.all(r["gx"] <= 1 + 1e-12)


def test_special_cases_U0_and_T1():
    rng = np.random.default_rng(3)
    px, py = _rand_lattice(rng, 8, 0)
    r = O.lattice_forward_backward(px, py, 8, 0)
    assert abs(r["L"] - py[:, 0].sum()) < 1e-10
    px, py = _rand_lattice(rng, 1, 6)
    r = O.lattice_forward_backward(px, py, 1, 6)
    assert abs(r["L"] - (px[0, :6].sum() + py[0, 6])) < 1e-10


# ---------------------------------------------------------------------------
# Trivial joiner: library checks of single steps, finite differences
# ---------------------------------------------------------------------------

def test_normalizer_matches_scipy_logsumexp():
    from scipy.special import logsumexp
    rng = np.random.default_rng(1)
    am = rng.standard_normal((2, 6, 9)) * 3
    lm = rng.standard_normal((2, 4, 9)) * 3
    Z = O.log_normalizer(am, lm, [6, 4], [3, 2])
    for n, (Tn, Un) in enumerate([(6, 3), (4, 2)]):
        ref = logsumexp(am[n, :Tn, None, :] + lm[n, None, :Un + 1, :], axis=-1)
        np.testing.assert_allclose(Z[n, :Tn, :Un + 1], ref, rtol=1e-13)


def test_trivial_joiner_rows_are_log_softmax():
    import torch
    rng = np.random.default_rng(2)
    am = rng.standard_normal((1, 5, 7))
    lm = rng.standard_normal((1, 4, 7))
    sym = np.array([[3, 0, 6]])  # a symbol equal to blank is allowed
    Z, px, py = O.trivial_joiner_logprobs(am, lm, sym, [5], [3], 0)
    ref = torch.log_softmax(torch.tensor(am[0, :, None, :] + lm[0, None, :, :]), dim=-1).numpy()
    for u in range(3):
        np.testing.assert_allclose(px[0, :, u], ref[:, u, sym[0, u]], rtol=1e-12)
    np.testing.assert_allclose(py[0], ref[:, :, 0], rtol=1e-12)
    assert np.all(np.isneginf(px[0, :, 3]))


def _total_simple_loss(am, lm, sym, tl, ul, sc):
    _, px, py = O.trivial_joiner_logprobs(am, lm, sym, tl, ul, 0)
    loss, _, _ = O.lattice_loss(px, py, tl, ul)
    return float((sc * loss).sum())


def test_trivial_joiner_grad_finite_difference():
    rng = np.random.default_rng(4)
    N, T, U, V = 2, 5, 3, 6
    am = rng.standard_normal((N, T, V))
    lm = rng.standard_normal((N, U + 1, V))
    sym = rng.integers(1, V, size=(N, U))
    sym[1, 1] = sym[1, 0]  # a repeated token
    tl, ul = np.array([5, 3]), np.array([3, 2])
    sc = np.array([0.7, 1.3])
    out = O.simple_stage(am, lm, sym, tl, ul, 0, scale=sc)
    eps = 1e-6
    for arr, g in ((am, out["am_grad"]), (lm, out["lm_grad"])):
        num = np.zeros_like(arr)
        for idx in np.ndindex(arr.shape):
            a0 = arr[idx]
            arr[idx] = a0 + eps
            fp = _total_simple_loss(am, lm, sym, tl, ul, sc)
            arr[idx] = a0 - eps
            fm = _total_simple_loss(am, lm, sym, tl, ul, sc)
            arr[idx] = a0
            num[idx] = (fp - fm) / (2 * eps)
        np.testing.assert_allclose(g, num, atol=2e-8, rtol=1e-6)
    # padding rows get no gradient; each log-softmax gradient sums to 0 over v
    assert np.all(out["am_grad"][1, 3:] == 0) and np.all(out["lm_grad"][1, 3:] == 0)
    np.testing.assert_allclose(out["am_grad"].sum(-1), 0, atol=1e-12)
    # the target column of lm row u collects exactly -sc * sum_t gx(t,u) = -sc
    n, u = 0, 1
    col = out["lm_grad"][n, u, sym[n, u]]
    P = np.exp(am[n, :5, None, :] + lm[n, None, :, :] - out["Z"][n, :5, :, None])
    expect = sc[n] * ((out["gx"][n, :5, u] + out["gy"][n, :5, u]) * P[:, u, sym[n, u]]).sum() - sc[n]
    assert abs(col - expect) < 1e-10


# ---------------------------------------------------------------------------
# Pruning bounds (Sec. 3.2.2)
# ---------------------------------------------------------------------------

def test_window_score_is_the_papers_eq7_example():
    with open(os.path.join(GOLDEN, "eq7_window_example.json")) as f:
        ex = json.load(f)
    rng = np.random.default_rng(9)
    T, U, S, p = 3, 9, ex["S"], ex["p"]
    gx = rng.random((T, U + 1)).astype(np.float32)
    gy = rng.random((T, U + 1)).astype(np.float32)
    sc = O.pruning_window_scores(gx, gy, T, U, S)
    for t in range(T):
        acc = np.float32(-gx[t, ex["subtracted_target_u"]])
        for u in ex["blank_terms_u"]:
            acc = np.float32(acc + gy[t, u])
        assert sc[t, p] == acc  # bit-exact, fp32, left to right
    # p = 0 has no subtracted arc
    assert sc[0, 0] == np.float32(np.float32(np.float32(np.float32(0) + gy[0, 0]) + gy[0, 1]) + gy[0, 2]) + gy[0, 3]


def test_window_score_identity():
    # score(t,p) = A_{t-1}(p) - A_t(p+S), A_t(p) = sum_{u>=p} gy(t,u)  (derived from flow conservation)
    rng = np.random.default_rng(21)
    T, U, S = 25, 12, 4
    px, py = _rand_lattice(rng, T, U)
    r = O.lattice_forward_backward(px, py, T, U)
    sc = O.pruning_window_scores(r["gx"], r["gy"], T, U, S)
    A = np.concatenate([np.cumsum(r["gy"][:, ::-1], axis=1)[:, ::-1], np.zeros((T, S + 1))], axis=1)
    for t in range(1, T):
        for p in range(U - S + 2):
            assert abs(sc[t, p] - (A[t - 1, p] - A[t, p + S])) < 2e-6


def test_adjustment_hand_example():
    # T=6, U=9, S=3 (P=7), worked by hand through the envelope clamp and the
    # MonotonicLowerBound procedure: clamp -> [0,2,1,3,7,7], suffix-min ->
    # [0,1,1,3,7,7], q=2t-p -> [0,1,3,3,1,3], suffix-min -> [0,1,1,1,1,3],
    # p=2t-q -> [0,1,3,5,7,7].
    p = O.adjust_pruning_bounds(np.array([0, 5, 1, 1, 9, 3]), 6, 9, 3)
    assert p.tolist() == [0, 1, 3, 5, 7, 7]
    assert O.monotonic_lower_bound(np.array([4, 2, 5, 3, 6])).tolist() == [2, 2, 3, 3, 6]


def test_ranges_invariants_random():
    rng = np.random.default_rng(31)
    for trial in range(40):
        T = int(rng.integers(1, 30))
        U = int(rng.integers(0, 25))
        S = int(rng.integers(2, 7))
        gx = rng.random((T, U + 1)).astype(np.float32)
        gy = rng.random((T, U + 1)).astype(np.float32)
        if trial % 5 == 0:
            gx[rng.random(gx.shape) < 0.1] = np.nan
        sc = O.pruning_window_scores(gx, gy, T, U, S)
        p = O.adjust_pruning_bounds(O.raw_pruning_bounds(sc), T, U, S)
        P = max(0, U - S + 1)
        assert np.all(p >= 0) and np.all(p <= P)
        assert np.all(np.diff(p) >= 0) and np.all(np.diff(p) < S)
        if U <= (S - 1) * T:  # a band exists (derived feasibility condition)
            assert p[0] == 0 and p[-1] == P
        if S >= U + 1:
            assert np.all(p == 0)


def test_argmax_ties_go_to_the_smallest_start_and_nan_never_wins():
    # Eq. (8) picks the window with the largest score; with this build's
    # reading, exact ties go to the smallest p and a NaN score never wins.
    sc = np.array([[0.2, 0.7, 0.7, 0.1],      # tie between p = 1 and p = 2
                   [0.5, 0.5, 0.5, 0.5],      # all tied
                   [np.nan, 0.3, np.nan, 0.3],  # NaN skipped, then the tie
                   [np.nan, np.nan, np.nan, np.nan],  # nothing wins: p = 0
                   [0.1, np.nan, 0.9, -np.inf]], dtype=np.float32)
    assert O.raw_pruning_bounds(sc).tolist() == [1, 0, 1, 0, 2]


def test_exact_fp32_window_tie_through_the_scores():
    # One frame of a T = 6, U = 4, S = 2 lattice (P = 3) whose blank
    # occupations make windows p = 0, 1, 2 score exactly 0.5 in fp32:
    # gy(2, .) = [1/4, 1/4, 1/4, 1/4, 0] and gx(2, .) = 0, so
    # score(p) = -0 + gy(p) + gy(p+1) = 1/2 for p <= 2 and 1/4 for p = 3.
    # Frame 2's envelope is [3 - (5 - 2), min(3, 2)] = [0, 2], so the raw
    # bound is not clamped; the smallest-p rule gives 0 (a largest-p rule 2).
    T, U, S = 6, 4, 2
    gx = np.zeros((T, U + 1), np.float32)
    gy = np.zeros((T, U + 1), np.float32)
    gy[2, :4] = 0.25
    sc = O.pruning_window_scores(gx, gy, T, U, S)
    assert sc[2].tolist() == [0.5, 0.5, 0.5, 0.25]
    assert O.raw_pruning_bounds(sc)[2] == 0
    # the same frame with every occupation NaN: no score wins, p = 0
    gy2 = gy.copy()
    gy2[2] = np.nan
    gx2 = gx.copy()
    gx2[2] = np.nan
    assert O.raw_pruning_bounds(O.pruning_window_scores(gx2, gy2, T, U, S))[2] == 0
    # every frame all-zero except frame 2: every other frame ties everywhere
    # and takes its smallest feasible start; the whole range set follows
    # from the envelope clamp and the adjustment: p = [0, 0, 0, 1, 2, 3]
    r = O.prune_ranges(gx[None], gy[None], [T], [U], S)
    assert r[0, :, 0].tolist() == [0, 0, 0, 1, 2, 3]


def test_ties_and_nan_frames_through_the_whole_bound_computation():
    # The GPU test of the bounds uses the same four utterances (T = 6, U = 4,
    # S = 2); the expected p_t were worked by hand through Eq. (8), the
    # envelope clamp and the adjustment.
    T, U, S = 6, 4, 2
    gx = np.zeros((4, T, U + 1), np.float32)
    gy = np.zeros((4, T, U + 1), np.float32)
    gy[:, 2, :4] = 0.25
    gy[1:3, 3, 3:] = 0.5
    gx[2, 3] = np.nan
    gy[2, 3] = np.nan
    gy[3, 2] = [0.0, 0.25, 0.25, 0.25, 0.25]
    r = O.prune_ranges(gx, gy, [T] * 4, [U] * 4, S)
    assert r[:, :, 0].tolist() == [[0, 0, 0, 1, 2, 3], [0, 0, 1, 2, 2, 3], [0, 0, 0, 1, 2, 3],
                                   [0, 0, 1, 1, 2, 3]]


def test_pruning_keeps_a_dominant_path():
    # One alignment carries (almost) all the mass: its occupations are ~1 and
    # the bounds must keep the whole path inside the band, so the pruned
    # recursion on the same log-probs loses no mass.
    T, U, S = 12, 8, 3
    path_u = [0, 1, 1, 2, 3, 3, 4, 6, 6, 7, 8, 8]  # u reached at the end of each frame
    px = np.full((T, U + 1), -60.0)
    py = np.full((T, U + 1), -60.0)
    px[:, U] = -np.inf
    u = 0
    for t in range(T):
        while u < path_u[t]:
            px[t, u] = 0.0
            u += 1
        py[t, u] = 0.0
    r = O.lattice_forward_backward(px, py, T, U)
    sc = O.pruning_window_scores(r["gx"], r["gy"], T, U, S)
    p = O.adjust_pruning_bounds(O.raw_pruning_bounds(sc), T, U, S)
    ranges = (p[:, None] + np.arange(S))[None].astype(np.int32)
    pxb = np.take_along_axis(px, np.minimum(ranges[0], U), axis=1)[None]
    pyb = np.take_along_axis(py, np.minimum(ranges[0], U), axis=1)[None]
    loss, _, _ = O.pruned_loss(pxb, pyb, ranges, [T], [U])
    assert abs(loss[0] + r["L"]) < 1e-9


# ---------------------------------------------------------------------------
# Pruned joiner and pruned loss
# ---------------------------------------------------------------------------

def test_pruned_equals_full_when_band_covers_lattice():
    b = make_batch("tiny", seed=0)
    S = b.U + 1
    ranges = np.tile(np.arange(S, dtype=np.int32), (b.N, b.T, 1))
    out = O.pruned_stage(b.enc, b.dec, b.W, b.bias, ranges, b.symbols, b.t_len, b.u_len, 0, grads=False)
    full, _, _ = O.full_joiner_loss(b.enc, b.dec, b.W, b.bias, b.symbols, b.t_len, b.u_len, 0)
    np.testing.assert_allclose(out["loss"], full, rtol=1e-12)
    # and so does a simple-stage range computation with S >= U+1
    s1 = O.simple_stage(b.am, b.lm, b.symbols, b.t_len, b.u_len, 0, grads=False)
    r2 = O.prune_ranges(s1["gx"], s1["gy"], b.t_len, b.u_len, S)
    assert np.array_equal(r2, ranges)


def test_pruned_joiner_logprobs_match_full_joiner_and_torch():
    import torch
    b = make_batch("tiny", seed=1)
    s1 = O.simple_stage(b.am, b.lm, b.symbols, b.t_len, b.u_len, 0, grads=False)
    ranges = O.prune_ranges(s1["gx"], s1["gy"], b.t_len, b.u_len, b.wl.S)
    px, py, lse = O.pruned_joiner_logprobs(b.enc, b.dec, b.W, b.bias, ranges, b.symbols,
                                           b.t_len, b.u_len, 0)
    fpx, fpy = O.full_joiner_logprobs(b.enc, b.dec, b.W, b.bias, b.symbols, b.t_len, b.u_len, 0)
    for n in range(b.N):
        for t in range(b.t_len[n]):
            for s in range(b.wl.S):
                u = ranges[n, t, s]
                if u <= b.u_len[n]:
                    assert abs(py[n, t, s] - fpy[n, t, u]) < 1e-12
                    assert (px[n, t, s] == fpx[n, t, u]) or abs(px[n, t, s] - fpx[n, t, u]) < 1e-12
    h = torch.tanh(torch.tensor(b.enc[0, 3], dtype=torch.float64) + torch.tensor(b.dec[0, ranges[0, 3, 1]], dtype=torch.float64))
    lg = h @ torch.tensor(b.W, dtype=torch.float64)
    ref = torch.log_softmax(lg, dim=-1)
    assert abs(py[0, 3, 1] - ref[0].item()) < 1e-12
    assert abs(lse[0, 3, 1] - torch.logsumexp(lg, dim=-1).item()) < 1e-12


def test_pruned_logits_special_cases():
    # W = I, bias = 0: the logits are the hidden activations tanh(enc + dec[p_t + s]) themselves
    rng = np.random.default_rng(11)
    N, T, U, J, S = 2, 5, 3, 6, 3
    enc = rng.standard_normal((N, T, J))
    dec = rng.standard_normal((N, U + 1, J))
    tl, ul = np.array([5, 3]), np.array([3, 2])
    ranges = np.zeros((N, T, S), np.int32)
    ranges[0] = (np.array([0, 0, 1, 1, 1])[:, None] + np.arange(S))
    ranges[1] = (np.array([0, 0, 0, 0, 0])[:, None] + np.arange(S))
    lg = O.pruned_joiner_logits(enc, dec, np.eye(J), np.zeros(J), ranges, tl, ul)
    for n in range(N):
        for t in range(T):
            for s in range(S):
                u = ranges[n, t, s]
                if t >= tl[n] or u > ul[n]:
                    assert np.all(np.isnan(lg[n, t, s]))
                else:
                    np.testing.assert_array_equal(lg[n, t, s], np.tanh(enc[n, t] + dec[n, u]))
    # dec = -enc broadcast: h = 0 and every present logit row is the bias
    dec2 = np.zeros((N, U + 1, J))
    enc2 = np.zeros((N, T, J))
    W = rng.standard_normal((J, 4))
    bias = rng.standard_normal(4)
    lg2 = O.pruned_joiner_logits(enc2, dec2, W, bias, ranges, tl, ul)
    ok = ~np.isnan(lg2[..., 0])
    np.testing.assert_array_equal(lg2[ok], np.broadcast_to(bias, lg2[ok].shape))
    # the log-softmax of the logits gives the joiner's px/py
    b = make_batch("tiny", seed=2)
    r = np.tile(np.arange(b.wl.S, dtype=np.int32), (b.N, b.T, 1))
    px, py, lse = O.pruned_joiner_logprobs(b.enc, b.dec, b.W, b.bias, r, b.symbols, b.t_len, b.u_len, 0)
    lg3 = O.pruned_joiner_logits(b.enc, b.dec, b.W, b.bias, r, b.t_len, b.u_len)
    from scipy.special import logsumexp
    np.testing.assert_allclose(logsumexp(lg3, axis=-1), lse, rtol=1e-13)
    np.testing.assert_allclose(lg3[..., 0] - lse, py, rtol=1e-13)


def _total_pruned_loss(enc, dec, W, bias, ranges, sym, tl, ul, sc):
    px, py, _ = O.pruned_joiner_logprobs(enc, dec, W, bias, ranges, sym, tl, ul, 0)
    loss, _, _ = O.pruned_loss(px, py, ranges, tl, ul)
    return float((sc * loss).sum())


def test_pruned_joiner_grad_finite_difference():
    rng = np.random.default_rng(6)
    N, T, U, V, J, S = 2, 6, 4, 7, 5, 3
    enc = rng.standard_normal((N, T, J))
    dec = rng.standard_normal((N, U + 1, J))
    W = rng.standard_normal((J, V)) / math.sqrt(J)
    bias = rng.standard_normal(V) * 0.1
    sym = rng.integers(1, V, size=(N, U))
    sym[0, 2] = 0  # a token equal to blank
    tl, ul = np.array([6, 4]), np.array([4, 3])
    sc = np.array([1.0, 0.5])
    ranges = np.zeros((N, T, S), np.int32)
    ranges[0] = (np.array([0, 0, 1, 1, 2, 2])[:, None] + np.arange(S))
    ranges[1] = (np.array([0, 1, 1, 1, 0, 0])[:, None] + np.arange(S))
    ranges[1, 4:] = np.arange(S)
    out = O.pruned_stage(enc, dec, W, bias, ranges, sym, tl, ul, 0, scale=sc, want_logits_grad=True)
    eps = 1e-6
    for arr, key in ((enc, "enc_grad"), (dec, "dec_grad"), (W, "W_grad"), (bias, "bias_grad")):
        num = np.zeros_like(arr)
        for idx in np.ndindex(arr.shape):
            a0 = arr[idx]
            arr[idx] = a0 + eps
            fp = _total_pruned_loss(enc, dec, W, bias, ranges, sym, tl, ul, sc)
            arr[idx] = a0 - eps
            fm = _total_pruned_loss(enc, dec, W, bias, ranges, sym, tl, ul, sc)
            arr[idx] = a0
            num[idx] = (fp - fm) / (2 * eps)
        np.testing.assert_allclose(out[key], num, atol=3e-8, rtol=1e-6)
    # d logits of every present slot sums to zero over v (log-softmax backward)
    np.testing.assert_allclose(out["logits_grad"].sum(-1), 0, atol=1e-12)


def test_infeasible_band_gives_infinite_loss_and_zero_occupation():
    # U > (S-1) T: no band admits a complete path
    T, U, S = 3, 7, 3
    rng = np.random.default_rng(8)
    px, py = _rand_lattice(rng, T, U)
    r = O.lattice_forward_backward(px, py, T, U)
    sc = O.pruning_window_scores(r["gx"], r["gy"], T, U, S)
    p = O.adjust_pruning_bounds(O.raw_pruning_bounds(sc), T, U, S)
    ranges = (p[:, None] + np.arange(S))[None].astype(np.int32)
    pxb = np.take_along_axis(px, np.minimum(ranges[0], U), axis=1)[None]
    pyb = np.take_along_axis(py, np.minimum(ranges[0], U), axis=1)[None]
    loss, gx, gy = O.pruned_loss(pxb, pyb, ranges, [T], [U])
    assert loss[0] == np.inf and np.all(gx == 0) and np.all(gy == 0)


# ---------------------------------------------------------------------------
# Sec. 3.3.1: the smoothed trivial joiner
# ---------------------------------------------------------------------------

def test_smoothed_joiner_reduces_to_the_trivial_joiner():
    b = make_batch("tiny", seed=7)
    px, py = O.smoothed_joiner_logprobs(b.am, b.lm, b.symbols, b.t_len, b.u_len, 0, 0.0, 0.0)
    _, tpx, tpy = O.trivial_joiner_logprobs(b.am, b.lm, b.symbols, b.t_len, b.u_len, 0)
    np.testing.assert_allclose(px, tpx, rtol=0, atol=1e-12)
    np.testing.assert_allclose(py, tpy, rtol=0, atol=1e-12)


def test_smoothed_joiner_special_cases():
    b = make_batch("tiny", seed=8)
    N, T, V = b.am.shape
    # acoustic only, with lm constant over v: the unigram prior is uniform and
    # L_acoustic is the trivial joiner with lm = 0
    lm0 = np.repeat(b.lm[:, :, :1], V, axis=2)
    px, py = O.smoothed_joiner_logprobs(b.am, lm0, b.symbols, b.t_len, b.u_len, 0, 0.0, 1.0)
    _, tpx, tpy = O.trivial_joiner_logprobs(b.am, np.zeros_like(b.lm), b.symbols, b.t_len, b.u_len, 0)
    np.testing.assert_allclose(px, tpx, atol=1e-12)
    np.testing.assert_allclose(py, tpy, atol=1e-12)
    # LM only: px(t,u) and py(t,u) do not depend on t or on am
    am2 = b.am + 3.0 * np.random.default_rng(0).standard_normal(b.am.shape).astype(np.float32)
    pa, pb = O.smoothed_joiner_logprobs(b.am, b.lm, b.symbols, b.t_len, b.u_len, 0, 1.0, 0.0)
    qa, qb = O.smoothed_joiner_logprobs(am2, b.lm, b.symbols, b.t_len, b.u_len, 0, 1.0, 0.0)
    np.testing.assert_allclose(pa, qa, atol=1e-12)
    np.testing.assert_allclose(pb, qb, atol=1e-12)
    for n in range(N):
        Tn = b.t_len[n]
        np.testing.assert_allclose(pb[n, :Tn], np.broadcast_to(pb[n, :1], pb[n, :Tn].shape), atol=1e-12)
    # every smoothed row is a mixture of log-softmaxes: for a = b = 1/2 at blank = 0
    # exp(py) is bounded by 1 and positive
    _, q = O.smoothed_joiner_logprobs(b.am, b.lm, b.symbols, b.t_len, b.u_len, 0, 0.5, 0.5)
    fin = np.isfinite(q)
    assert np.all(q[fin] < 0)


def test_smoothed_unigram_prior_is_the_log_of_the_mean_softmax():
    # Sec. 3.3.1: L_dec^avg(v) is the log of the mean over the utterance's
    # decoder rows of Softmax_v lm[u, v] (not the mean of the log-softmaxes).
    # V = 2, blank = 0, y_1 = 1; lm rows with softmaxes (1/4, 3/4) and
    # (1/2, 1/2): the prior is (log 3/8, log 5/8). With am = 0 the acoustic
    # joiner (a_ac = 1) is then exactly that prior: py = log 3/8 and
    # px = log 5/8 at every node. The mean of the log-softmaxes would give
    # softmax weights proportional to (1/8)^(1/2), (3/8)^(1/2) instead:
    # 0.366 / 0.634 rather than 0.375 / 0.625. A third lm row (padding,
    # u > U_n) must not enter the average.
    lm = np.array([[[0.0, math.log(3.0)], [0.0, 0.0], [5.0, -5.0]]])
    am = np.zeros((1, 3, 2))
    sym = np.array([[1, 1]])
    px, py = O.smoothed_joiner_logprobs(am, lm, sym, [3], [1], 0, 0.0, 1.0)
    np.testing.assert_allclose(py[0, :3, :2], math.log(3 / 8), rtol=0, atol=1e-14)
    np.testing.assert_allclose(px[0, :3, :1], math.log(5 / 8), rtol=0, atol=1e-14)
    # with a non-zero am the acoustic joiner is LogSoftmax_v(am + prior)
    am2 = np.array([[[0.3, -1.2], [2.0, 0.5], [0.0, 0.0]]])
    px2, py2 = O.smoothed_joiner_logprobs(am2, lm, sym, [3], [1], 0, 0.0, 1.0)
    for t in range(3):
        z0 = am2[0, t, 0] + math.log(3 / 8)
        z1 = am2[0, t, 1] + math.log(5 / 8)
        lse = math.log(math.exp(z0) + math.exp(z1))
        assert abs(py2[0, t, 0] - (z0 - lse)) < 1e-14
        assert abs(px2[0, t, 0] - (z1 - lse)) < 1e-14
    # LM only (a_lm = 1): px = log softmax(lm[u])[y_{u+1}] = log 3/4 at u = 0
    px3, py3 = O.smoothed_joiner_logprobs(am2, lm, sym, [3], [1], 0, 1.0, 0.0)
    np.testing.assert_allclose(px3[0, :3, 0], math.log(3 / 4), atol=1e-14)
    np.testing.assert_allclose(py3[0, :3, 0], math.log(1 / 4), atol=1e-14)
    np.testing.assert_allclose(py3[0, :3, 1], math.log(1 / 2), atol=1e-14)


def test_smoothed_simple_loss_finite_difference():
    rng = np.random.default_rng(9)
    N, T, U, V = 2, 5, 3, 6
    am = rng.standard_normal((N, T, V))
    lm = rng.standard_normal((N, U + 1, V))
    sym = rng.integers(1, V, size=(N, U))
    sym[1, 0] = 0  # a token equal to blank
    tl, ul = np.array([5, 4]), np.array([3, 2])
    sc = np.array([1.0, 0.7])
    a, bb = 0.25, 0.15
    out = O.smoothed_simple_stage(am, lm, sym, tl, ul, 0, a, bb, scale=sc)

    def total(am_, lm_):
        r = O.smoothed_simple_stage(am_, lm_, sym, tl, ul, 0, a, bb, grads=False)
        return float((sc * r["loss"]).sum())

    eps = 1e-6
    for arr, key in ((am, "am_grad"), (lm, "lm_grad")):
        num = np.zeros_like(arr)
        for idx in np.ndindex(arr.shape):
            a0 = arr[idx]
            arr[idx] = a0 + eps
            fp = total(am, lm)
            arr[idx] = a0 - eps
            fm = total(am, lm)
            arr[idx] = a0
            num[idx] = (fp - fm) / (2 * eps)
        np.testing.assert_allclose(out[key], num, atol=2e-8, rtol=1e-6)
