"""GPU parity: every stage of the HIP path against the CPU oracle.

Stage-wise checks feed both sides the same inputs (the oracle's own
intermediate results, rounded to the fp32 the ABI takes), so each kernel is
judged on its own; the end-to-end check runs the whole GPU path from am, lm,
enc, dec, W and compares final losses and gradients. Sizes are chosen so the
oracle finishes in seconds while every kernel still sees several tiles and
ragged tails (T, U, V and J not multiples of the tile sizes).
"""
import numpy as np
import pytest
import torch

import oracle as O
import paper_2206_13236_amd as P
from gpu_common import (DEV, assert_close, check_step, dev_f32, dev_i32, dev_joiner, grad_atol, host,
                        loss_rtol, make_dev_batch, oracle_step, run_step, say)
from workloads import make_batch

pytestmark = pytest.mark.gpu

CASES = {
    "tiny": dict(wl="tiny"),
    "small_f32": dict(wl="bpe", N=3, T_range=(40, 70), U_range=(5, 20), V=37, J=64, S=5),
    "small_bf16": dict(wl="long", N=3, T_range=(40, 70), U_range=(5, 20), V=72, J=64, S=4),
    # bf16 rows of odd length: element-wise W segments in the forward, the
    # zero-padded copy of W in dh
    "small_bf16_oddv": dict(wl="long", N=3, T_range=(30, 50), U_range=(4, 15), V=37, J=64, S=4),
    "bpe_sub": dict(wl="bpe", N=3),
    "long_sub": dict(wl="long", N=2),
}


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    assert torch.cuda.is_available(), "GPU tests need a ROCm device"
    P.lib()


def _case(name, seed=0):
    c = dict(CASES[name])
    wl = c.pop("wl")
    b = make_batch(wl, seed=seed, **c)
    return b


def _scale(N, seed=1):
    return (0.5 + np.random.default_rng(seed).random(N)).astype(np.float32)


_ORACLE_CACHE = {}


def _oracle(name):
    if name in _ORACLE_CACHE:
        return _ORACLE_CACHE[name]
    b = _case(name)
    S = b.wl.S
    sc = _scale(b.N)
    s1 = O.simple_stage(b.am, b.lm, b.symbols, b.t_len, b.u_len, b.wl.blank, scale=sc)
    gx32 = s1["gx"].astype(np.float32)
    gy32 = s1["gy"].astype(np.float32)
    ranges = O.prune_ranges(gx32, gy32, b.t_len, b.u_len, S)
    st = O.pruned_stage(b.enc, b.dec, b.W, b.bias, ranges, b.symbols, b.t_len, b.u_len, b.wl.blank,
                        scale=sc, want_logits_grad=(name == "tiny"))
    r = dict(b=b, S=S, sc=sc, s1=s1, gx32=gx32, gy32=gy32, ranges=ranges, st=st)
    _ORACLE_CACHE[name] = r
    return r


def _valid_mask_TU(b):
    m = np.zeros((b.N, b.T, b.U + 1), bool)
    for n in range(b.N):
        m[n, :b.t_len[n], :b.u_len[n] + 1] = True
    return m


@pytest.mark.parametrize("name", list(CASES))
def test_simple_stage(name):
    o = _oracle(name)
    b = o["b"]
    say(f"[simple] {name} N={b.N} T={b.T} U={b.U} V={b.V}")
    batch = make_dev_batch(b)
    out = P.rnnt_simple_loss(batch, b.V, dev_f32(b.am), dev_f32(b.lm), dev_f32(o["sc"]),
                             want_logprobs=True, want_grads=True)
    torch.cuda.synchronize()
    s1 = o["s1"]
    assert_close("loss", host(out["loss"]), s1["loss"], rtol=1e-5)
    assert_close("px", host(out["px"]), s1["px"], atol=5e-5)
    assert_close("py", host(out["py"]), s1["py"], atol=5e-5)
    assert_close("px_occ", host(out["px_occ"]), s1["gx"], atol=1e-4)
    assert_close("py_occ", host(out["py_occ"]), s1["gy"], atol=1e-4)
    assert_close("am_grad", host(out["am_grad"]), s1["am_grad"], atol=1e-4)
    assert_close("lm_grad", host(out["lm_grad"]), s1["lm_grad"], atol=1e-4)


@pytest.mark.parametrize("name", list(CASES))
def test_prune_ranges_bit_exact(name):
    o = _oracle(name)
    b = o["b"]
    say(f"[prune] {name}")
    batch = make_dev_batch(b)
    r = P.rnnt_prune_ranges(batch, o["S"], dev_f32(o["gx32"]), dev_f32(o["gy32"]))
    torch.cuda.synchronize()
    got = r.cpu().numpy()
    assert np.array_equal(got, o["ranges"]), f"{(got != o['ranges']).sum()} range entries differ"


def _tie_cases():
    """Occupations with exact fp32 window ties and an all-NaN frame (T = 6,
    U = 4, S = 2, so P = 3), and the bounds p_t worked out by hand through
    Eq. (8), the envelope clamp and the adjustment (ties to the smallest p,
    NaN never wins, an all-NaN frame takes 0)."""
    T, U, S = 6, 4, 2
    gx = np.zeros((4, T, U + 1), np.float32)
    gy = np.zeros((4, T, U + 1), np.float32)
    gy[:, 2, :4] = 0.25            # windows p = 0, 1, 2 of frame 2 all score 1/2
    gy[1:3, 3, 3:] = 0.5           # frame 3: window p = 3 scores 1
    gx[2, 3] = np.nan              # ... but utterance 2's frame 3 is all NaN
    gy[2, 3] = np.nan
    gy[3, 2] = [0.0, 0.25, 0.25, 0.25, 0.25]  # windows 1, 2, 3 tie at 1/2
    expect = [[0, 0, 0, 1, 2, 3], [0, 0, 1, 2, 2, 3], [0, 0, 0, 1, 2, 3], [0, 0, 1, 1, 2, 3]]
    return T, U, S, gx, gy, np.array(expect)


def test_prune_ranges_exact_ties_and_nan_frames():
    T, U, S, gx, gy, expect = _tie_cases()
    N = gx.shape[0]
    tl, ul = np.full(N, T, np.int32), np.full(N, U, np.int32)
    ref = O.prune_ranges(gx, gy, tl, ul, S)
    assert np.array_equal(ref[:, :, 0], expect)
    say("[prune] exact ties and all-NaN frames")
    batch = P.Batch(dev_i32(tl), dev_i32(ul), dev_i32(np.ones((N, U), np.int32)), T, U, 0)
    got = P.rnnt_prune_ranges(batch, S, dev_f32(gx), dev_f32(gy)).cpu().numpy()
    assert np.array_equal(got, ref), f"GPU bounds {got[:, :, 0].tolist()} vs {expect.tolist()}"


@pytest.mark.parametrize("name", list(CASES))
def test_pruned_joiner(name):
    o = _oracle(name)
    b = o["b"]
    bf = b.wl.joiner_dtype == "bf16"
    say(f"[joiner] {name} bf16={bf}")
    batch = make_dev_batch(b)
    out = P.rnnt_pruned_joiner(batch, o["S"], dev_joiner(b.enc, bf), dev_joiner(b.dec, bf), dev_joiner(b.W, bf),
                               dev_joiner(b.bias, bf), dev_i32(o["ranges"]), keep_logits=True)
    torch.cuda.synchronize()
    st = o["st"]
    tol = 2e-2 if bf else 5e-5
    assert_close("px", host(out["px"]), st["px"], atol=tol)
    assert_close("py", host(out["py"]), st["py"], atol=tol)
    assert_close("lse", host(out["lse"]), st["lse"], atol=tol, rtol=tol)
    # the stored logits at every present slot (absent slots are left untouched)
    ref = O.pruned_joiner_logits(b.enc, b.dec, b.W, b.bias, o["ranges"], b.t_len, b.u_len)
    present = ~np.isnan(ref[..., 0])
    assert_close("logits", host(out["logits"])[present], ref[present], atol=tol)


# the pruned recursion's algorithms: the library's choice, the wavefront, and
# the chunked scan with its default chunk and with chunks of 1, 3 and 32 frames
BAND_ALGS = [(None, 0), ("wavefront", 0), ("scan", 0), ("scan", 1), ("scan", 3), ("scan", 32)]


@pytest.mark.parametrize("alg,chunk", BAND_ALGS, ids=[f"{a}{c or ''}" for a, c in BAND_ALGS])
@pytest.mark.parametrize("name", list(CASES))
def test_pruned_loss(name, alg, chunk):
    o = _oracle(name)
    b = o["b"]
    say(f"[band] {name} algorithm={alg} chunk={chunk}")
    st = o["st"]
    # both sides take the same fp32 band log-probs
    px32, py32 = st["px"].astype(np.float32), st["py"].astype(np.float32)
    loss_ref, gx_ref, gy_ref = O.pruned_loss(px32.astype(np.float64), py32.astype(np.float64), o["ranges"],
                                             b.t_len, b.u_len)
    batch = make_dev_batch(b)
    out = P.rnnt_pruned_loss(batch, o["S"], dev_f32(px32), dev_f32(py32), dev_i32(o["ranges"]), algorithm=alg,
                             chunk=chunk)
    torch.cuda.synchronize()
    assert_close("loss", host(out["loss"]), loss_ref, rtol=1e-5)
    assert_close("px_occ", host(out["px_occ"]), gx_ref, atol=1e-4)
    assert_close("py_occ", host(out["py_occ"]), gy_ref, atol=1e-4)


def _joiner_backward(name, stored, chunk_rows=0, head=False):
    o = _oracle(name)
    b = o["b"]
    bf = b.wl.joiner_dtype == "bf16"
    say(f"[joiner-bwd] {name} bf16={bf} stored_logits={stored} chunk_rows={chunk_rows} head={head}")
    st = o["st"]
    lse32 = st["lse"].astype(np.float32)
    gx32, gy32 = st["gx"].astype(np.float32), st["gy"].astype(np.float32)
    ref = O.pruned_joiner_grad(b.enc, b.dec, b.W, b.bias, o["ranges"], b.symbols, b.t_len, b.u_len, b.wl.blank,
                               gx32.astype(np.float64), gy32.astype(np.float64), scale=o["sc"],
                               want_logits_grad=(name == "tiny"))
    batch = make_dev_batch(b)
    args = (dev_joiner(b.enc, bf), dev_joiner(b.dec, bf), dev_joiner(b.W, bf), dev_joiner(b.bias, bf))
    rng = dev_i32(o["ranges"])
    logits, lse = None, dev_f32(lse32)
    hd, C = None, 0
    if stored:
        # the backward streams the logits the forward kept, with the forward's own lse
        fw = P.rnnt_pruned_joiner(batch, o["S"], *args, rng, keep_logits=True)
        logits, lse = fw["logits"], fw["lse"]
    elif head:
        # the forward keeps the logits of the backward's first chunk only
        C = P.backward_chunk_rows(b.N, b.T, o["S"], b.wl.J, b.V, P._jdtype(args[2]), chunk_rows)
        hd = torch.empty(C, (b.V + 7) // 8 * 8, dtype=torch.float32, device=DEV)
        fw = P.rnnt_pruned_joiner(batch, o["S"], *args, rng, head=hd, head_rows=C)
        lse = fw["lse"]
    out = P.rnnt_pruned_joiner_backward(
        batch, o["S"], *args, rng, lse, dev_f32(gx32), dev_f32(gy32), scale=dev_f32(o["sc"]),
        want_logits_grad=(name == "tiny"), logits=logits, chunk_rows=chunk_rows, head=hd, head_rows=C)
    torch.cuda.synchronize()
    for k in ("enc_grad", "dec_grad"):
        assert_close(k, host(out[k]), ref[k], atol=grad_atol(ref[k], bf))
    for k in ("W_grad", "bias_grad"):
        assert_close(k, host(out[k]), ref[k], atol=grad_atol(ref[k], bf, param=True))
    if name == "tiny":
        assert_close("logits_grad", host(out["logits_grad"]), ref["logits_grad"], atol=1e-5)
    return out


@pytest.mark.parametrize("stored", [False, True], ids=["recompute", "stored_logits"])
@pytest.mark.parametrize("name", list(CASES))
def test_pruned_joiner_backward(name, stored):
    _joiner_backward(name, stored)


# chunks of rows that S does not divide (frames straddle chunk edges), three
# or more chunks per batch
CHUNKED = [("small_f32", 128), ("small_f32", 384), ("small_bf16", 128), ("small_bf16_oddv", 256), ("bpe_sub", 1024)]


@pytest.mark.parametrize("name,chunk", [("tiny", 0), ("small_f32", 128), ("small_bf16", 256),
                                        ("small_bf16_oddv", 128), ("bpe_sub", 0), ("long_sub", 1024)])
def test_pruned_joiner_backward_with_head(name, chunk):
    # the forward keeps the first chunk's logits, the backward streams that
    # chunk and recomputes the others; d enc and d dec are bitwise those of
    # the backward that recomputes every chunk
    _joiner_backward(name, False, chunk_rows=chunk, head=True)  # against the oracle
    # the same forward's lse for both backward calls, with and without the head
    o = _oracle(name)
    b = o["b"]
    bf = b.wl.joiner_dtype == "bf16"
    batch = make_dev_batch(b)
    args = (dev_joiner(b.enc, bf), dev_joiner(b.dec, bf), dev_joiner(b.W, bf), dev_joiner(b.bias, bf))
    rng = dev_i32(o["ranges"])
    C = P.backward_chunk_rows(b.N, b.T, o["S"], b.wl.J, b.V, P._jdtype(args[2]), chunk)
    hd = torch.empty(C, (b.V + 7) // 8 * 8, dtype=torch.float32, device=DEV)
    fw = P.rnnt_pruned_joiner(batch, o["S"], *args, rng, head=hd, head_rows=C)
    gx, gy = dev_f32(o["st"]["gx"].astype(np.float32)), dev_f32(o["st"]["gy"].astype(np.float32))
    with_head = P.rnnt_pruned_joiner_backward(batch, o["S"], *args, rng, fw["lse"], gx, gy, scale=dev_f32(o["sc"]),
                                              chunk_rows=chunk, head=hd, head_rows=C)
    without = P.rnnt_pruned_joiner_backward(batch, o["S"], *args, rng, fw["lse"], gx, gy, scale=dev_f32(o["sc"]),
                                            chunk_rows=chunk)
    torch.cuda.synchronize()
    for k in ("enc_grad", "dec_grad"):
        assert torch.equal(with_head[k], without[k]), f"{k} differs with the head"
    for k in ("W_grad", "bias_grad"):
        ref = host(without[k])
        assert_close(k, host(with_head[k]), ref, atol=1e-6 * max(1.0, np.abs(ref).max()))


@pytest.mark.parametrize("stored", [False, True], ids=["recompute", "stored_logits"])
@pytest.mark.parametrize("name,chunk", CHUNKED, ids=[f"{n}-{c}" for n, c in CHUNKED])
def test_pruned_joiner_backward_in_chunks(name, chunk, stored):
    b = _oracle(name)["b"]
    assert -(-b.N * b.T * _oracle(name)["S"] // chunk) >= 3, "the case must span at least three chunks"
    got = _joiner_backward(name, stored, chunk_rows=chunk)
    # d enc and d dec add their pieces in tile order whatever the chunking:
    # bitwise equal to the library's own chunk choice
    one = _joiner_backward(name, stored)
    for k in ("enc_grad", "dec_grad"):
        assert torch.equal(got[k], one[k]), f"{k} depends on the chunking"


@pytest.mark.parametrize("name", list(CASES))
def test_end_to_end(name):
    b = _case(name)
    S = b.wl.S
    say(f"[e2e] {name}")
    out = run_step(b, S)
    amb = check_step(out, oracle_step(b, S), b, S)
    say(f"  near-tie utterances {sorted(amb)}")


@pytest.mark.parametrize("name", ["small_f32", "small_bf16"])
def test_end_to_end_kept_logits(name):
    # the forward stores the [N, T, S, V] logits and the backward streams them
    b = _case(name)
    say(f"[e2e] {name} keep_logits=True")
    out = run_step(b, b.wl.S, keep_logits=True)
    check_step(out, oracle_step(b, b.wl.S), b, b.wl.S)


def test_end_to_end_small_chunks():
    # the training step with backward chunks of 128 rows (seven chunks)
    b = _case("small_f32")
    say("[e2e] small_f32 backward chunks of 128 rows")
    out = run_step(b, b.wl.S, bwd_chunk_rows=128)
    check_step(out, oracle_step(b, b.wl.S), b, b.wl.S)


def test_deterministic_repeat():
    b = _case("small_f32")
    say("[determinism] small_f32 x2")
    batch = make_dev_batch(b)
    args = (dev_f32(b.am), dev_f32(b.lm), dev_f32(b.enc), dev_f32(b.dec), dev_f32(b.W), dev_f32(b.bias))
    outs = []
    for _ in range(2):
        step = P.PrunedRnntLoss(b.wl.S)
        o = step.step(batch, *args)
        torch.cuda.synchronize()
        outs.append({k: v.clone() for k, v in o.items()})
    for k in outs[0]:
        assert torch.equal(outs[0][k], outs[1][k]), f"{k} differs between identical runs"
