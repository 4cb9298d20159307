"""Plain fp64 CPU oracle for the pruned RNN-T loss.  TEST INFRASTRUCTURE ONLY.

This module restates the computations of "Pruned RNN-T for fast,
memory-efficient ASR training" (Kuang et al., arXiv 2206.13236) as directly
as possible:

* the lattice, its transition log-probs and the forward recursion
  (Sec. 2, Eqs. (1)-(4));
* the trivial joiner and its normaliser (Sec. 3.1, Eqs. (5)-(6)), computed as
  a plain log-sum-exp over the vocabulary, not as a matrix product;
* occupation counts, the locally optimal pruning bound and the consistency
  constraints (Sec. 3.2.2, Eqs. (7)-(10));
* the pruned lattice, where every entry outside p_t <= u < p_t + S is set to
  minus infinity before the same recursion runs (Sec. 3.2, Fig. 1(b));
* gradients by the chain rule through a log-softmax.

Arrays use the conventions of the C ABI: ``symbols[n, u]`` is y_{u+1}
(y_0 is the beginning-of-sentence blank, Sec. 2); ``px``/``py`` are
[N, T, U+1] with minus infinity outside the lattice; the loss of utterance n
is minus its total log-probability.

Readings where the paper is silent:
* y'(t, -1) in Eq. (8) is taken as 0 (the p = 0 window has no red arc);
* Eq. (8) is evaluated in fp32, left to right, and ties go to the smallest p;
  a NaN score never wins;
* window slots above U contribute 0 (they are absent from the lattice);
* before the adjustment the raw bound is clamped to the envelope
  [P - (S-1)(T-1-t), min(P, (S-1) t)], P = max(0, U-S+1), so that the band
  holds the start node at t = 0 and the final node at t = T-1;
* the adjustment is the MonotonicLowerBound procedure the paper's LaTeX source
  gives in a commented-out block of Sec. 3.2.2 (suffix minimum, reflection by
  (S-1) t, suffix minimum, reflection, max with 0);
* the full joiner is tanh(enc + dec) W + b, with enc and dec already
  projected to the joiner dimension (the paper does not print its form).
"""
from __future__ import annotations

import math
from typing import Optional

import numpy as np

NEG_INF = float("-inf")


# ---------------------------------------------------------------------------
# Sec. 2: LogAdd, the forward recursion, total log-probability
# ---------------------------------------------------------------------------

def log_add(a: float, b: float) -> float:
    """LogAdd(x, y) = log(e^x + e^y) (Sec. 2, Eq. (4)), on Python floats."""
    if a == NEG_INF:
        return b
    if b == NEG_INF:
        return a
    if a >= b:
        return a + math.log1p(math.exp(b - a))
    return b + math.log1p(math.exp(a - b))


def lattice_forward_backward(px, py, Tn: int, Un: int) -> dict:
    """Forward and backward passes over one utterance's T x (U+1) lattice.

    ``px[t][u]`` is y(t,u), the log-prob of the vertical transition leaving
    node (t,u) (it emits y_{u+1}); ``py[t][u]`` is the blank log-prob of the
    horizontal transition leaving (t,u) (Sec. 2, Eqs. (1)-(2), Fig. 1(a)).

    alpha follows Eq. (3): alpha(0,0) = 0 and
    alpha(t,u) = LogAdd(alpha(t-1,u) + py(t-1,u), alpha(t,u-1) + px(t,u-1)).
    The total log-prob is L = alpha(T-1,U) + py(T-1,U) (Sec. 2).

    beta(t,u) is the log-prob of every way to finish from node (t,u),
    including the final blank, so beta(T-1,U) = py(T-1,U) and beta(0,0) = L.

    The occupations are the derivatives of L with respect to px and py
    (Sec. 3.2.2): gx(t,u) = exp(alpha(t,u) + px(t,u) + beta(t,u+1) - L) and
    gy(t,u) = exp(alpha(t,u) + py(t,u) + beta(t+1,u) - L), where the final
    blank leads to beta(T,U) = 0. If L is -inf (no complete path) all
    occupations are 0.
    """
    Tn, Un = int(Tn), int(Un)
    X = np.asarray(px, dtype=np.float64)[:Tn, :Un + 1].tolist()
    Y = np.asarray(py, dtype=np.float64)[:Tn, :Un + 1].tolist()
    alpha = [[NEG_INF] * (Un + 1) for _ in range(Tn)]
    for t in range(Tn):
        at, am1 = alpha[t], (alpha[t - 1] if t > 0 else None)
        for u in range(Un + 1):
            if t == 0 and u == 0:
                at[0] = 0.0
                continue
            a = am1[u] + Y[t - 1][u] if t > 0 else NEG_INF
            b = at[u - 1] + X[t][u - 1] if u > 0 else NEG_INF
            at[u] = log_add(a, b)
    L = alpha[Tn - 1][Un] + Y[Tn - 1][Un]

    beta = [[NEG_INF] * (Un + 1) for _ in range(Tn)]
    beta[Tn - 1][Un] = Y[Tn - 1][Un]
    for t in range(Tn - 1, -1, -1):
        bt, bp1 = beta[t], (beta[t + 1] if t + 1 < Tn else None)
        for u in range(Un, -1, -1):
            if t == Tn - 1 and u == Un:
                continue
            a = Y[t][u] + bp1[u] if t + 1 < Tn else NEG_INF
            b = X[t][u] + bt[u + 1] if u < Un else NEG_INF
            bt[u] = log_add(a, b)

    gx = np.zeros((Tn, Un + 1))
    gy = np.zeros((Tn, Un + 1))
    if L != NEG_INF:
        for t in range(Tn):
            for u in range(Un + 1):
                if u < Un:
                    gx[t, u] = math.exp(alpha[t][u] + X[t][u] + beta[t][u + 1] - L) \
                        if not math.isnan(L) else math.nan
                if t + 1 < Tn:
                    nb = beta[t + 1][u]
                else:
                    nb = 0.0 if u == Un else NEG_INF
                gy[t, u] = math.exp(alpha[t][u] + Y[t][u] + nb - L) \
                    if not math.isnan(L) else math.nan
    return {"alpha": np.array(alpha), "beta": np.array(beta), "L": L, "gx": gx, "gy": gy}


def lattice_loss(px, py, t_len, u_len):
    """Per-utterance loss -L and occupations for a padded batch [N, T, U+1]."""
    px = np.asarray(px, np.float64)
    py = np.asarray(py, np.float64)
    N, T, U1 = py.shape
    loss = np.zeros(N)
    gx = np.zeros((N, T, U1))
    gy = np.zeros((N, T, U1))
    for n in range(N):
        Tn, Un = int(t_len[n]), int(u_len[n])
        r = lattice_forward_backward(px[n], py[n], Tn, Un)
        loss[n] = -r["L"]
        gx[n, :Tn, :Un + 1] = r["gx"]
        gy[n, :Tn, :Un + 1] = r["gy"]
    return loss, gx, gy


# ---------------------------------------------------------------------------
# Sec. 3.1: the trivial joiner
# ---------------------------------------------------------------------------

def log_normalizer(am, lm, t_len, u_len, t_chunk: int = 8):
    """L_normalizer(t,u) = log sum_v exp(L_enc(t,v) + L_dec(u,v)) (Sec. 3.1, Eq. (6)).

    Evaluated directly over v as a max-shifted sum of exponentials, in fp64.
    Returns [N, T, U+1] with 0 outside t < T_n, u <= U_n.
    """
    am = np.asarray(am, np.float64)
    lm = np.asarray(lm, np.float64)
    N, T, V = am.shape
    Z = np.zeros((N, T, lm.shape[1]))
    for n in range(N):
        Tn, Un = int(t_len[n]), int(u_len[n])
        for t0 in range(0, Tn, t_chunk):
            t1 = min(Tn, t0 + t_chunk)
            x = am[n, t0:t1, None, :] + lm[n, None, :Un + 1, :]
            m = x.max(axis=-1, keepdims=True)
            Z[n, t0:t1, :Un + 1] = (m + np.log(np.exp(x - m).sum(axis=-1, keepdims=True)))[..., 0]
    return Z


def trivial_joiner_logprobs(am, lm, symbols, t_len, u_len, blank: int = 0):
    """y(t,u) and blank(t,u) of the trivial joiner (Sec. 3.1 Eqs. (5)-(6) with Eqs. (1)-(2)).

    L_trivial(t,u,v) = am[t,v] + lm[u,v] - L_normalizer(t,u);
    px(t,u) = L_trivial(t,u,y_{u+1}) for u < U, py(t,u) = L_trivial(t,u,blank).
    Returns (Z, px, py), each [N, T, U+1] fp64, -inf outside the lattice.
    """
    am64 = np.asarray(am, np.float64)
    lm64 = np.asarray(lm, np.float64)
    N, T, V = am64.shape
    U1 = lm64.shape[1]
    Z = log_normalizer(am64, lm64, t_len, u_len)
    px = np.full((N, T, U1), NEG_INF)
    py = np.full((N, T, U1), NEG_INF)
    for n in range(N):
        Tn, Un = int(t_len[n]), int(u_len[n])
        y = np.asarray(symbols[n, :Un], np.int64)
        if Un > 0:
            px[n, :Tn, :Un] = am64[n, :Tn][:, y] + lm64[n, np.arange(Un), y][None, :] - Z[n, :Tn, :Un]
        py[n, :Tn, :Un + 1] = (am64[n, :Tn, blank][:, None] + lm64[n, :Un + 1, blank][None, :]
                               - Z[n, :Tn, :Un + 1])
    return Z, px, py


def trivial_joiner_grad(am, lm, symbols, t_len, u_len, blank, Z, gx, gy, scale=None,
                        t_chunk: int = 8):
    """Gradients of sum_n sc_n * loss_n w.r.t. am and lm through the trivial joiner.

    The loss is -L; dL/dpx = gx and dL/dpy = gy are the occupations of
    Sec. 3.2.2. px and py are entries of the log-softmax L_trivial of
    Sec. 3.1, so the chain rule runs through the log-softmax backward:
    for every (t,u), G(v) = dloss/dL_trivial(t,u,v) is -gx at v = y_{u+1} and
    -gy at v = blank; dloss/dlogit(v) = G(v) - P(t,u,v) * sum_v' G(v'), with
    P = exp(L_trivial). That logit is am[t,v] + lm[u,v], so d am[t] sums it
    over u and d lm[u] sums it over t.
    """
    am64 = np.asarray(am, np.float64)
    lm64 = np.asarray(lm, np.float64)
    N, T, V = am64.shape
    U1 = lm64.shape[1]
    sc = np.ones(N) if scale is None else np.asarray(scale, np.float64)
    d_am = np.zeros((N, T, V))
    d_lm = np.zeros((N, U1, V))
    for n in range(N):
        Tn, Un = int(t_len[n]), int(u_len[n])
        y = np.asarray(symbols[n, :Un], np.int64)
        for t0 in range(0, Tn, t_chunk):
            t1 = min(Tn, t0 + t_chunk)
            logp = am64[n, t0:t1, None, :] + lm64[n, None, :Un + 1, :] - Z[n, t0:t1, :Un + 1, None]
            P = np.exp(logp)
            G = np.zeros_like(P)
            if Un > 0:
                G[:, np.arange(Un), y] -= gx[n, t0:t1, :Un]
            G[:, :, blank] -= gy[n, t0:t1, :Un + 1]
            D = sc[n] * (G - P * G.sum(axis=-1, keepdims=True))
            d_am[n, t0:t1] += D.sum(axis=1)
            d_lm[n, :Un + 1] += D.sum(axis=0)
    return d_am, d_lm


def simple_stage(am, lm, symbols, t_len, u_len, blank=0, scale=None, grads=True) -> dict:
    """Stages 1-2: trivial-joiner log-probs, the full-lattice recursion and its gradients."""
    Z, px, py = trivial_joiner_logprobs(am, lm, symbols, t_len, u_len, blank)
    loss, gx, gy = lattice_loss(px, py, t_len, u_len)
    out = {"Z": Z, "px": px, "py": py, "loss": loss, "gx": gx, "gy": gy}
    if grads:
        out["am_grad"], out["lm_grad"] = trivial_joiner_grad(
            am, lm, symbols, t_len, u_len, blank, Z, gx, gy, scale)
    return out


# ---------------------------------------------------------------------------
# Sec. 3.3.1: the smoothed trivial joiner (small shapes: plain fp64 PyTorch)
# ---------------------------------------------------------------------------

def _smoothed_px_py(am_t, lm_t, symbols, t_len, u_len, blank, lm_only_scale, am_only_scale):
    """px, py of the smoothed joiner as fp64 torch tensors (differentiable).

    L_smoothed = (1 - a_lm - a_ac) L_trivial + a_lm L_lm + a_ac L_acoustic, with
      L_trivial(t,u,v)  = LogSoftmax_v(am[t,v] + lm[u,v])        (Eq. (5)),
      L_lm(u,v)         = LogSoftmax_v lm[u,v],
      L_dec^avg(v)      = log (1/(U+1)) sum_{u=0..U} Softmax_v lm[u,v],
      L_acoustic(t,v)   = LogSoftmax_v(am[t,v] + L_dec^avg(v)).
    Reading: the third term of the printed combination (a second L_lm) is
    L_acoustic, the only other joiner the section defines; L_dec^avg does not
    depend on u, and its average runs over the utterance's own U_n + 1 rows.
    """
    import torch
    N, T, _ = am_t.shape
    U1 = lm_t.shape[1]
    a, b = float(lm_only_scale), float(am_only_scale)
    out_x, out_y = [], []
    for n in range(N):
        Tn, Un = int(t_len[n]), int(u_len[n])
        amn, lmn = am_t[n, :Tn], lm_t[n, :Un + 1]
        triv = torch.log_softmax(amn[:, None, :] + lmn[None, :, :], dim=-1)     # [Tn, Un+1, V]
        llm = torch.log_softmax(lmn, dim=-1)                                     # [Un+1, V]
        lavg = torch.log(torch.softmax(lmn, dim=-1).mean(dim=0))                 # [V]
        lac = torch.log_softmax(amn + lavg[None, :], dim=-1)                     # [Tn, V]
        sm = (1.0 - a - b) * triv + a * llm[None, :, :] + b * lac[:, None, :]    # [Tn, Un+1, V]
        y = torch.as_tensor(np.asarray(symbols[n, :Un], np.int64))
        # -inf outside the lattice, assembled without in-place writes
        fx = torch.full((T, U1), NEG_INF, dtype=torch.float64)
        fy = torch.full((T, U1), NEG_INF, dtype=torch.float64)
        mx = torch.zeros((T, U1), dtype=torch.bool)
        my = torch.zeros((T, U1), dtype=torch.bool)
        mx[:Tn, :Un] = True
        my[:Tn, :Un + 1] = True
        if Un > 0:
            fx = fx.masked_scatter(mx, sm[:, torch.arange(Un), y].reshape(-1))
        fy = fy.masked_scatter(my, sm[:, :, blank].reshape(-1))
        out_x.append(fx)
        out_y.append(fy)
    return torch.stack(out_x), torch.stack(out_y)


def smoothed_joiner_logprobs(am, lm, symbols, t_len, u_len, blank=0, lm_only_scale=0.0,
                             am_only_scale=0.0):
    """px, py [N, T, U+1] (fp64 NumPy) of the smoothed trivial joiner (Sec. 3.3.1)."""
    import torch
    am_t = torch.as_tensor(np.asarray(am, np.float64))
    lm_t = torch.as_tensor(np.asarray(lm, np.float64))
    px, py = _smoothed_px_py(am_t, lm_t, symbols, t_len, u_len, blank, lm_only_scale, am_only_scale)
    return px.numpy(), py.numpy()


def smoothed_simple_stage(am, lm, symbols, t_len, u_len, blank=0, lm_only_scale=0.0, am_only_scale=0.0,
                          scale=None, grads=True) -> dict:
    """The simple loss with the smoothed joiner: recursion, occupations and the
    gradients of sum_n sc_n * loss_n w.r.t. am and lm. The loss is -L and
    dL/dpx = gx, dL/dpy = gy (Sec. 3.2.2), so the gradient is the
    vector-Jacobian product of px, py with -sc * gx, -sc * gy, taken by
    PyTorch's autograd in fp64 through the definitions above."""
    import torch
    am_t = torch.as_tensor(np.asarray(am, np.float64)).clone().requires_grad_(grads)
    lm_t = torch.as_tensor(np.asarray(lm, np.float64)).clone().requires_grad_(grads)
    px_t, py_t = _smoothed_px_py(am_t, lm_t, symbols, t_len, u_len, blank, lm_only_scale, am_only_scale)
    px, py = px_t.detach().numpy(), py_t.detach().numpy()
    loss, gx, gy = lattice_loss(px, py, t_len, u_len)
    out = {"px": px, "py": py, "loss": loss, "gx": gx, "gy": gy}
    if grads:
        N = px.shape[0]
        sc = torch.as_tensor(np.ones(N) if scale is None else np.asarray(scale, np.float64))
        wx = -sc[:, None, None] * torch.as_tensor(gx)
        wy = -sc[:, None, None] * torch.as_tensor(gy)
        # entries outside the lattice are -inf constants with zero weight
        fin_x, fin_y = torch.isfinite(px_t), torch.isfinite(py_t)
        obj = (torch.where(fin_x, px_t, torch.zeros_like(px_t)) * wx).sum() + \
              (torch.where(fin_y, py_t, torch.zeros_like(py_t)) * wy).sum()
        d_am, d_lm = torch.autograd.grad(obj, (am_t, lm_t), allow_unused=True)
        out["am_grad"] = np.zeros(am_t.shape) if d_am is None else d_am.numpy()
        out["lm_grad"] = np.zeros(lm_t.shape) if d_lm is None else d_lm.numpy()
    return out


# ---------------------------------------------------------------------------
# Sec. 3.2.2: locally optimal pruning bounds and the consistency constraints
# ---------------------------------------------------------------------------

def pruning_window_scores(gx, gy, Tn: int, Un: int, S: int) -> np.ndarray:
    """Scores of Eq. (8) for p = 0..P, P = max(0, U-S+1), in fp32.

    score(t,p) = -y'(t,p-1) + blank'(t,p) + ... + blank'(t,p+S-1), evaluated
    left to right in fp32 exactly as written (Eq. (7) is the p = 2, S = 4
    case). y'(t,-1) is read as 0 and slots above U contribute 0.
    """
    Tn, Un, S = int(Tn), int(Un), int(S)
    P = max(0, Un - S + 1)
    gx32 = np.asarray(gx, dtype=np.float32)[:Tn]
    gy32 = np.asarray(gy, dtype=np.float32)[:Tn]
    acc = np.zeros((Tn, P + 1), dtype=np.float32)
    if P > 0:
        acc[:, 1:] = -gx32[:, 0:P]
    p = np.arange(P + 1)
    zero = np.float32(0.0)
    for k in range(S):
        u = p + k
        term = np.where(u <= Un, gy32[:, np.minimum(u, Un)], zero).astype(np.float32)
        acc = np.add(acc, term, dtype=np.float32)
    return acc


def raw_pruning_bounds(scores: np.ndarray) -> np.ndarray:
    """Argmax of Eq. (8) per frame: the smallest p with the largest score.

    A NaN score never wins; a frame whose scores are all NaN gets 0.
    """
    s = np.where(np.isnan(scores), -np.inf, scores)
    return np.argmax(s, axis=1).astype(np.int64)


def monotonic_lower_bound(a: np.ndarray) -> np.ndarray:
    """b_i = min(a_i, a_{i+1}, ...): the largest sequence with b <= a and b_i <= b_{i+1}."""
    a = np.asarray(a)
    return np.minimum.accumulate(a[::-1])[::-1].copy()


def adjust_pruning_bounds(raw, Tn: int, Un: int, S: int) -> np.ndarray:
    """Enforce 0 <= p_t <= U-S+1, Eq. (9) p_t <= p_{t+1} and Eq. (10) p_{t+1} - p_t < S.

    Envelope clamp first (this build's reading: the band must contain the
    start node at t = 0 and the final node at t = T-1), then the
    MonotonicLowerBound procedure of the commented-out block in Sec. 3.2.2:
    suffix minimum, p <- (S-1) t - p, suffix minimum, p <- (S-1) t - p,
    p <- max(0, p).
    """
    Tn, Un, S = int(Tn), int(Un), int(S)
    P = max(0, Un - S + 1)
    t = np.arange(Tn, dtype=np.int64)
    lo = P - (S - 1) * (Tn - 1 - t)
    hi = np.minimum(P, (S - 1) * t)
    p = np.minimum(np.maximum(np.asarray(raw, np.int64), lo), hi)
    p = monotonic_lower_bound(p)
    p = (S - 1) * t - p
    p = monotonic_lower_bound(p)
    p = (S - 1) * t - p
    return np.maximum(0, p)


def prune_ranges(gx, gy, t_len, u_len, S: int) -> np.ndarray:
    """ranges[n, t, s] = p_t + s (Sec. 3.2); frames t >= T_n get ranges = s."""
    gx = np.asarray(gx)
    N, T = gx.shape[0], gx.shape[1]
    ranges = np.tile(np.arange(S, dtype=np.int32), (N, T, 1))
    for n in range(N):
        Tn, Un = int(t_len[n]), int(u_len[n])
        sc = pruning_window_scores(gx[n], gy[n], Tn, Un, S)
        p = adjust_pruning_bounds(raw_pruning_bounds(sc), Tn, Un, S)
        ranges[n, :Tn, :] = (p[:, None] + np.arange(S)[None, :]).astype(np.int32)
    return ranges


# ---------------------------------------------------------------------------
# Sec. 3.2: the full joiner on the pruned (t, u) pairs, and the pruned lattice
# ---------------------------------------------------------------------------

def joiner_hidden(enc_t, dec_u):
    """h = tanh(enc + dec): the non-linear part of the full joiner (fp64)."""
    return np.tanh(np.asarray(enc_t, np.float64) + np.asarray(dec_u, np.float64))


def _joiner_logits(enc, dec, W, bias, n, ts, us):
    h = joiner_hidden(enc[n, ts], dec[n, us])
    return h, h @ np.asarray(W, np.float64) + np.asarray(bias, np.float64)


def pruned_joiner_logits(enc, dec, W, bias, ranges, t_len, u_len):
    """The (N, T, S, V) pruned logits of Sec. 3.2: tanh(enc[t] + dec[u]) W + b at u = ranges[n,t,s].

    Absent slots (u > U_n) and frames t >= T_n are NaN.
    """
    N, T, S = ranges.shape
    V = np.asarray(W).shape[1]
    out = np.full((N, T, S, V), np.nan)
    for n in range(N):
        Tn, Un = int(t_len[n]), int(u_len[n])
        u = np.asarray(ranges[n, :Tn], np.int64)
        ts = np.repeat(np.arange(Tn)[:, None], S, axis=1)
        _, lg = _joiner_logits(enc, dec, W, bias, n, ts, np.minimum(u, Un))
        out[n, :Tn] = np.where((u <= Un)[..., None], lg, np.nan)
    return out


def pruned_joiner_logprobs(enc, dec, W, bias, ranges, symbols, t_len, u_len, blank=0,
                           t_chunk: int = 32):
    """Full joiner evaluated only at u = ranges[n,t,s] (Sec. 3.2, output (N,T,S,V)).

    logits = tanh(enc[t] + dec[u]) W + b; lse = log sum_v exp(logits);
    px = logits[y_{u+1}] - lse (u < U_n, else -inf); py = logits[blank] - lse.
    Slots with u > U_n, and frames t >= T_n, are absent: px = py = -inf, lse = 0.
    """
    N, T, S = ranges.shape
    px = np.full((N, T, S), NEG_INF)
    py = np.full((N, T, S), NEG_INF)
    lse = np.zeros((N, T, S))
    for n in range(N):
        Tn, Un = int(t_len[n]), int(u_len[n])
        for t0 in range(0, Tn, t_chunk):
            t1 = min(Tn, t0 + t_chunk)
            u = np.asarray(ranges[n, t0:t1], np.int64)
            ok = u <= Un
            uc = np.minimum(u, Un)
            ts = np.repeat(np.arange(t0, t1)[:, None], S, axis=1)
            _, lg = _joiner_logits(enc, dec, W, bias, n, ts, uc)
            m = lg.max(axis=-1, keepdims=True)
            l = (m + np.log(np.exp(lg - m).sum(axis=-1, keepdims=True)))[..., 0]
            b = lg[..., blank] - l
            yv = np.asarray(symbols[n], np.int64)
            tgt_ok = ok & (u < Un)
            ysym = yv[np.minimum(uc, max(Un - 1, 0))] if Un > 0 else np.zeros_like(uc)
            tg = np.take_along_axis(lg, ysym[..., None], axis=-1)[..., 0] - l
            px[n, t0:t1] = np.where(tgt_ok, tg, NEG_INF)
            py[n, t0:t1] = np.where(ok, b, NEG_INF)
            lse[n, t0:t1] = np.where(ok, l, 0.0)
    return px, py, lse


def pruned_loss(px_b, py_b, ranges, t_len, u_len):
    """The recursion of Eq. (3) on the pruned lattice (Sec. 3.2, Fig. 1(b)).

    Literally: scatter the band log-probs into T_n x (U_n+1) matrices that are
    -inf everywhere else, run the unpruned forward-backward, and gather the
    occupations back to the band. Returns (loss [N], gx_b, gy_b [N,T,S]).
    """
    N, T, S = ranges.shape
    loss = np.zeros(N)
    gx_b = np.zeros((N, T, S))
    gy_b = np.zeros((N, T, S))
    for n in range(N):
        Tn, Un = int(t_len[n]), int(u_len[n])
        X = np.full((Tn, Un + 1), NEG_INF)
        Y = np.full((Tn, Un + 1), NEG_INF)
        for t in range(Tn):
            for s in range(S):
                u = int(ranges[n, t, s])
                if u <= Un:
                    X[t, u] = px_b[n, t, s]
                    Y[t, u] = py_b[n, t, s]
        r = lattice_forward_backward(X, Y, Tn, Un)
        loss[n] = -r["L"]
        for t in range(Tn):
            for s in range(S):
                u = int(ranges[n, t, s])
                if u <= Un:
                    gx_b[n, t, s] = r["gx"][t, u]
                    gy_b[n, t, s] = r["gy"][t, u]
    return loss, gx_b, gy_b


def pruned_joiner_grad(enc, dec, W, bias, ranges, symbols, t_len, u_len, blank,
                       gx_b, gy_b, scale=None, want_logits_grad=False, t_chunk: int = 32):
    """Gradients of sum_n sc_n * pruned_loss_n w.r.t. enc, dec, W and bias.

    Chain rule through: the log-softmax over v (G = -gx at y_{u+1}, -gy at
    blank; dlogits = G - softmax * sum G), the projection logits = h W + b,
    tanh (dpre = dh * (1 - h^2)) and the sum enc[t] + dec[u]: d enc[t] sums
    over the S slots of frame t, d dec[u] over every (t, s) with p_t + s = u.
    """
    W64 = np.asarray(W, np.float64)
    N, T, S = ranges.shape
    J, V = W64.shape
    sc = np.ones(N) if scale is None else np.asarray(scale, np.float64)
    d_enc = np.zeros((N, T, J))
    d_dec = np.zeros((N, dec.shape[1], J))
    dW = np.zeros((J, V))
    db = np.zeros(V)
    dlog = np.zeros((N, T, S, V)) if want_logits_grad else None
    for n in range(N):
        Tn, Un = int(t_len[n]), int(u_len[n])
        yv = np.asarray(symbols[n], np.int64)
        for t0 in range(0, Tn, t_chunk):
            t1 = min(Tn, t0 + t_chunk)
            u = np.asarray(ranges[n, t0:t1], np.int64)
            ok = u <= Un
            uc = np.minimum(u, Un)
            ts = np.repeat(np.arange(t0, t1)[:, None], S, axis=1)
            h, lg = _joiner_logits(enc, dec, W, bias, n, ts, uc)
            m = lg.max(axis=-1, keepdims=True)
            P = np.exp(lg - m)
            P /= P.sum(axis=-1, keepdims=True)
            G = np.zeros_like(lg)
            gxs = np.where(ok & (u < Un), gx_b[n, t0:t1], 0.0)
            gys = np.where(ok, gy_b[n, t0:t1], 0.0)
            if Un > 0:
                ysym = yv[np.minimum(uc, Un - 1)]
                np.add.at(G, (np.arange(t1 - t0)[:, None], np.arange(S)[None, :], ysym), -gxs)
            G[..., blank] -= gys
            D = sc[n] * (G - P * G.sum(axis=-1, keepdims=True))
            D[~ok] = 0.0
            if dlog is not None:
                dlog[n, t0:t1] = D
            dW += np.einsum("tsj,tsv->jv", h, D)
            db += D.sum(axis=(0, 1))
            dh = D @ W64.T
            dpre = dh * (1.0 - h * h)
            dpre[~ok] = 0.0
            d_enc[n, t0:t1] += dpre.sum(axis=1)
            np.add.at(d_dec[n], uc.reshape(-1), dpre.reshape(-1, J))
    out = {"enc_grad": d_enc, "dec_grad": d_dec, "W_grad": dW, "bias_grad": db}
    if dlog is not None:
        out["logits_grad"] = dlog
    return out


def pruned_stage(enc, dec, W, bias, ranges, symbols, t_len, u_len, blank=0, scale=None,
                 grads=True, want_logits_grad=False) -> dict:
    """Stage 4: pruned joiner, pruned recursion and the joiner backward."""
    px, py, lse = pruned_joiner_logprobs(enc, dec, W, bias, ranges, symbols, t_len, u_len, blank)
    loss, gx, gy = pruned_loss(px, py, ranges, t_len, u_len)
    out = {"px": px, "py": py, "lse": lse, "loss": loss, "gx": gx, "gy": gy}
    if grads:
        out.update(pruned_joiner_grad(enc, dec, W, bias, ranges, symbols, t_len, u_len, blank,
                                      gx, gy, scale, want_logits_grad))
    return out


# ---------------------------------------------------------------------------
# Sec. 2: the unpruned loss with the same joiner (tiny shapes only)
# ---------------------------------------------------------------------------

def full_joiner_logprobs(enc, dec, W, bias, symbols, t_len, u_len, blank=0):
    """The (N, T, U+1, V) joiner the method avoids (Sec. 2), reduced to px and py."""
    N, T = enc.shape[0], enc.shape[1]
    U1 = dec.shape[1]
    px = np.full((N, T, U1), NEG_INF)
    py = np.full((N, T, U1), NEG_INF)
    for n in range(N):
        Tn, Un = int(t_len[n]), int(u_len[n])
        ts = np.repeat(np.arange(Tn)[:, None], Un + 1, axis=1)
        us = np.repeat(np.arange(Un + 1)[None, :], Tn, axis=0)
        _, lg = _joiner_logits(enc, dec, W, bias, n, ts, us)
        m = lg.max(axis=-1, keepdims=True)
        logp = lg - (m + np.log(np.exp(lg - m).sum(axis=-1, keepdims=True)))
        py[n, :Tn, :Un + 1] = logp[..., blank]
        if Un > 0:
            y = np.asarray(symbols[n, :Un], np.int64)
            px[n, :Tn, :Un] = logp[:, np.arange(Un), y]
    return px, py


def full_joiner_loss(enc, dec, W, bias, symbols, t_len, u_len, blank=0):
    px, py = full_joiner_logprobs(enc, dec, W, bias, symbols, t_len, u_len, blank)
    return lattice_loss(px, py, t_len, u_len)
