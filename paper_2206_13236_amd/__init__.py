"""Pruned RNN-T loss (Kuang et al., arXiv 2206.13236) on MI355X (gfx950).

Every stage runs in the hand-written HIP kernels of ``librnnt_pruned.so``;
this package only marshals arguments through its C ABI (ctypes). PyTorch
provides device memory and the current stream. The functions named like the
C entry points (``rnnt_simple_loss`` ...) map one-to-one onto them; the
``PrunedRnntLoss`` helper chains the four stages the way the paper's training
step does (Sec. 3.3: loss = pruned + 0.5 * simple).
"""
from __future__ import annotations

import ctypes
from typing import Optional

import torch

from ._native import (RNNT_BF16, RNNT_EHIP, RNNT_EINVAL, RNNT_EUNSUPPORTED, RNNT_EWORKSPACE,  # noqa: F401
                      RNNT_F32, RNNT_FLAGS, RNNT_OK, RNNT_REDUCE_MEAN, RNNT_REDUCE_SUM, RnntBatch, RnntError,
                      check, lib)

__all__ = [
    "Batch", "RnntError", "rnnt_simple_loss", "rnnt_simple_loss_backward", "rnnt_prune_ranges",
    "rnnt_pruned_joiner", "pruned_rnnt_loss", "rnnt_full_loss", "full_loss_workspace_size",
    "rnnt_pruned_loss", "rnnt_pruned_joiner_backward", "simple_loss_workspace_size",
    "pruned_joiner_workspace_size", "pruned_loss_workspace_size", "BAND_ALGORITHMS",
    "pruned_joiner_backward_workspace_size", "PrunedRnntLoss", "RNNT_F32", "RNNT_BF16",
    "rnnt_combine_losses", "rnnt_validate_inputs", "RNNT_FLAGS", "rnnt_pruned_loss_noalloc",
    "backward_chunk_rows",
]


def _p(t: Optional[torch.Tensor]):
    return None if t is None else ctypes.c_void_p(t.data_ptr())


def _stream(stream) -> ctypes.c_void_p:
    if stream is None:
        stream = torch.cuda.current_stream()
    if isinstance(stream, torch.cuda.Stream):
        stream = stream.cuda_stream
    return ctypes.c_void_p(int(stream))


def _need(t: torch.Tensor, name: str, dtype: torch.dtype, shape: tuple):
    if not isinstance(t, torch.Tensor):
        raise TypeError(f"{name} must be a tensor")
    if t.device.type != "cuda":
        raise ValueError(f"{name} must be a device (cuda) tensor")
    if t.dtype != dtype:
        raise TypeError(f"{name} must be {dtype}, got {t.dtype}")
    if tuple(t.shape) != tuple(shape):
        raise ValueError(f"{name} must have shape {tuple(shape)}, got {tuple(t.shape)}")
    if not t.is_contiguous():
        raise ValueError(f"{name} must be contiguous")


def _ws(nbytes: int, device, workspace: Optional[torch.Tensor]) -> torch.Tensor:
    if workspace is not None:
        if workspace.numel() * workspace.element_size() < nbytes:
            raise ValueError(f"workspace has {workspace.numel()} bytes, {nbytes} needed")
        return workspace
    return torch.empty(max(nbytes, 1), dtype=torch.uint8, device=device)


def _jdtype(t: torch.Tensor) -> int:
    if t.dtype == torch.float32:
        return RNNT_F32
    if t.dtype == torch.bfloat16:
        return RNNT_BF16
    raise TypeError(f"joiner tensors must be float32 or bfloat16, got {t.dtype}")


class Batch:
    """Device description of a padded batch (the C ``rnnt_batch``).

    t_len [N], u_len [N] and symbols [N, U] are int32 device tensors;
    symbols[n, u] is y_{u+1}. T and U are the padded maxima.
    """

    def __init__(self, t_len: torch.Tensor, u_len: torch.Tensor, symbols: torch.Tensor,
                 T: int, U: int, blank: int = 0):
        N = int(t_len.shape[0])
        _need(t_len, "t_len", torch.int32, (N,))
        _need(u_len, "u_len", torch.int32, (N,))
        _need(symbols, "symbols", torch.int32, (N, U))
        self.t_len, self.u_len, self.symbols = t_len, u_len, symbols
        self.N, self.T, self.U, self.blank = N, int(T), int(U), int(blank)
        self.device = t_len.device
        self._c = RnntBatch(self.N, self.T, self.U, t_len.data_ptr(), u_len.data_ptr(),
                            symbols.data_ptr() if U > 0 else None, self.blank)

    @property
    def c(self):
        return ctypes.byref(self._c)


# --------------------------------------------------------------------------
# workspace queries
# --------------------------------------------------------------------------

def simple_loss_workspace_size(N, T, U, V) -> int:
    return int(lib().rnnt_simple_loss_workspace_size(N, T, U, V))


def pruned_joiner_workspace_size(N, T, S, J, V, dtype) -> int:
    return int(lib().rnnt_pruned_joiner_workspace_size(N, T, S, J, V, dtype))


def pruned_loss_workspace_size(N, T, U, S, algorithm=None, chunk=0) -> int:
    if algorithm is None:
        return int(lib().rnnt_pruned_loss_workspace_size(N, T, U, S))
    return int(lib().rnnt_pruned_loss_ex_workspace_size(N, T, U, S, BAND_ALGORITHMS[algorithm], chunk))


def pruned_joiner_backward_workspace_size(N, T, U, S, J, V, dtype, chunk_rows: int = 0) -> int:
    if chunk_rows == 0:
        return int(lib().rnnt_pruned_joiner_backward_workspace_size(N, T, U, S, J, V, dtype))
    return int(lib().rnnt_pruned_joiner_backward_ex_workspace_size(N, T, U, S, J, V, dtype, chunk_rows))


# --------------------------------------------------------------------------
# stage wrappers (same names and argument order as the C ABI)
# --------------------------------------------------------------------------

def rnnt_simple_loss(batch: Batch, V: int, am: torch.Tensor, lm: torch.Tensor,
                     scale: Optional[torch.Tensor] = None, loss=None, px_occ=None, py_occ=None,
                     px=None, py=None, am_grad=None, lm_grad=None, workspace=None, stream=None,
                     want_logprobs: bool = False, want_grads: bool = False, lm_only_scale: float = 0.0,
                     am_only_scale: float = 0.0) -> dict:
    N, T, U = batch.N, batch.T, batch.U
    dev = batch.device
    _need(am, "am", torch.float32, (N, T, V))
    _need(lm, "lm", torch.float32, (N, U + 1, V))
    f32 = dict(dtype=torch.float32, device=dev)
    loss = torch.empty(N, **f32) if loss is None else loss
    px_occ = torch.empty(N, T, U + 1, **f32) if px_occ is None else px_occ
    py_occ = torch.empty(N, T, U + 1, **f32) if py_occ is None else py_occ
    if want_logprobs and px is None:
        px, py = torch.empty(N, T, U + 1, **f32), torch.empty(N, T, U + 1, **f32)
    if want_grads and am_grad is None:
        am_grad, lm_grad = torch.empty(N, T, V, **f32), torch.empty(N, U + 1, V, **f32)
    if scale is not None:
        _need(scale, "scale", torch.float32, (N,))
    ws = _ws(simple_loss_workspace_size(N, T, U, V), dev, workspace)
    check(lib().rnnt_simple_loss(batch.c, V, _p(am), _p(lm), _p(scale), float(lm_only_scale),
                                 float(am_only_scale), _p(loss), _p(px_occ),
                                 _p(py_occ), _p(px), _p(py), _p(am_grad), _p(lm_grad), _p(ws),
                                 ws.numel(), _stream(stream)))
    return {"loss": loss, "px_occ": px_occ, "py_occ": py_occ, "px": px, "py": py,
            "am_grad": am_grad, "lm_grad": lm_grad}


def rnnt_simple_loss_backward(batch: Batch, V: int, am: torch.Tensor, lm: torch.Tensor, px_occ: torch.Tensor,
                              workspace: torch.Tensor, scale: Optional[torch.Tensor] = None, am_grad=None,
                              lm_grad=None, stream=None, lm_only_scale: float = 0.0,
                              am_only_scale: float = 0.0) -> dict:
    """d am, d lm from the state a preceding rnnt_simple_loss call left in ``workspace``."""
    N, T, U = batch.N, batch.T, batch.U
    dev = batch.device
    _need(am, "am", torch.float32, (N, T, V))
    _need(lm, "lm", torch.float32, (N, U + 1, V))
    _need(px_occ, "px_occ", torch.float32, (N, T, U + 1))
    if scale is not None:
        _need(scale, "scale", torch.float32, (N,))
    f32 = dict(dtype=torch.float32, device=dev)
    am_grad = torch.empty(N, T, V, **f32) if am_grad is None else am_grad
    lm_grad = torch.empty(N, U + 1, V, **f32) if lm_grad is None else lm_grad
    ws = _ws(simple_loss_workspace_size(N, T, U, V), dev, workspace)
    check(lib().rnnt_simple_loss_backward(batch.c, V, _p(am), _p(lm), _p(scale), float(lm_only_scale),
                                          float(am_only_scale), _p(px_occ), _p(am_grad),
                                          _p(lm_grad), _p(ws), ws.numel(), _stream(stream)))
    return {"am_grad": am_grad, "lm_grad": lm_grad}


def rnnt_prune_ranges(batch: Batch, S: int, px_occ: torch.Tensor, py_occ: torch.Tensor,
                      ranges: Optional[torch.Tensor] = None, stream=None) -> torch.Tensor:
    N, T, U = batch.N, batch.T, batch.U
    _need(px_occ, "px_occ", torch.float32, (N, T, U + 1))
    _need(py_occ, "py_occ", torch.float32, (N, T, U + 1))
    ranges = torch.empty(N, T, S, dtype=torch.int32, device=batch.device) if ranges is None else ranges
    check(lib().rnnt_prune_ranges(batch.c, S, _p(px_occ), _p(py_occ), _p(ranges), _stream(stream)))
    return ranges


def backward_chunk_rows(N, T, S, J, V, dtype, chunk_rows: int = 0) -> int:
    """Rows of the joiner backward's chunk (the head's rows)."""
    return int(lib().rnnt_pruned_joiner_backward_chunk_rows(N, T, S, J, V, dtype, chunk_rows))


def rnnt_pruned_joiner(batch: Batch, S: int, enc: torch.Tensor, dec: torch.Tensor, W: torch.Tensor,
                       bias: Optional[torch.Tensor], ranges: torch.Tensor, px=None, py=None, lse=None,
                       logits=None, workspace=None, stream=None, keep_logits: bool = False, head=None,
                       head_rows: int = 0) -> dict:
    """The pruned joiner; with ``head`` ([head_rows, ldl] fp32) it calls
    rnnt_pruned_joiner_ex, which also keeps the first chunk's logits there."""
    N, T, U = batch.N, batch.T, batch.U
    J, V = int(W.shape[0]), int(W.shape[1])
    dt = _jdtype(W)
    _need(enc, "enc", W.dtype, (N, T, J))
    _need(dec, "dec", W.dtype, (N, U + 1, J))
    if bias is not None:
        _need(bias, "bias", W.dtype, (V,))
    _need(ranges, "ranges", torch.int32, (N, T, S))
    f32 = dict(dtype=torch.float32, device=batch.device)
    px = torch.empty(N, T, S, **f32) if px is None else px
    py = torch.empty(N, T, S, **f32) if py is None else py
    lse = torch.empty(N, T, S, **f32) if lse is None else lse
    if keep_logits and logits is None:
        logits = torch.empty(N, T, S, V, **f32)
    if logits is not None:
        _need(logits, "logits", torch.float32, (N, T, S, V))
    ws = _ws(pruned_joiner_workspace_size(N, T, S, J, V, dt), batch.device, workspace)
    if head is None:
        check(lib().rnnt_pruned_joiner(batch.c, S, J, V, dt, _p(enc), _p(dec), _p(W), _p(bias), _p(ranges),
                                       _p(px), _p(py), _p(lse), _p(logits), _p(ws), ws.numel(), _stream(stream)))
    else:
        _need(head, "head", torch.float32, (head_rows, (V + 7) // 8 * 8))
        check(lib().rnnt_pruned_joiner_ex(batch.c, S, J, V, dt, _p(enc), _p(dec), _p(W), _p(bias), _p(ranges),
                                          _p(px), _p(py), _p(lse), _p(logits), _p(head), int(head_rows), _p(ws),
                                          ws.numel(), _stream(stream)))
    return {"px": px, "py": py, "lse": lse, "logits": logits}


# algorithms of the pruned recursion (rnnt_pruned_loss_ex)
BAND_ALGORITHMS = {"auto": 0, "wavefront": 1, "scan": 2}


def rnnt_pruned_loss(batch: Batch, S: int, px: torch.Tensor, py: torch.Tensor, ranges: torch.Tensor,
                     loss=None, px_occ=None, py_occ=None, workspace=None, stream=None,
                     want_occupations: bool = True, algorithm: str = None, chunk: int = 0) -> dict:
    """The pruned recursion; `algorithm` ("auto", "wavefront" or "scan") and
    `chunk` select rnnt_pruned_loss_ex, None calls rnnt_pruned_loss."""
    N, T = batch.N, batch.T
    _need(px, "px", torch.float32, (N, T, S))
    _need(py, "py", torch.float32, (N, T, S))
    _need(ranges, "ranges", torch.int32, (N, T, S))
    f32 = dict(dtype=torch.float32, device=batch.device)
    loss = torch.empty(N, **f32) if loss is None else loss
    if want_occupations and px_occ is None:
        px_occ, py_occ = torch.empty(N, T, S, **f32), torch.empty(N, T, S, **f32)
    ws = _ws(pruned_loss_workspace_size(N, T, batch.U, S, algorithm, chunk), batch.device, workspace)
    if algorithm is None:
        check(lib().rnnt_pruned_loss(batch.c, S, _p(px), _p(py), _p(ranges), _p(loss), _p(px_occ), _p(py_occ),
                                     _p(ws), ws.numel(), _stream(stream)))
    else:
        check(lib().rnnt_pruned_loss_ex(batch.c, S, BAND_ALGORITHMS[algorithm], chunk, _p(px), _p(py),
                                        _p(ranges), _p(loss), _p(px_occ), _p(py_occ), _p(ws), ws.numel(),
                                        _stream(stream)))
    return {"loss": loss, "px_occ": px_occ, "py_occ": py_occ}


def rnnt_pruned_loss_noalloc(batch: Batch, S: int, px: torch.Tensor, py: torch.Tensor, ranges: torch.Tensor,
                             loss=None, px_occ=None, py_occ=None, stream=None) -> dict:
    """rnnt_pruned_loss with its workspace in the library's static device
    scratch (no allocation in the call; overlapping calls on one GPU race)."""
    N, T = batch.N, batch.T
    _need(px, "px", torch.float32, (N, T, S))
    _need(py, "py", torch.float32, (N, T, S))
    _need(ranges, "ranges", torch.int32, (N, T, S))
    f32 = dict(dtype=torch.float32, device=batch.device)
    loss = torch.empty(N, **f32) if loss is None else loss
    check(lib().rnnt_pruned_loss_noalloc(batch.c, S, _p(px), _p(py), _p(ranges), _p(loss), _p(px_occ), _p(py_occ),
                                         _stream(stream)))
    return {"loss": loss, "px_occ": px_occ, "py_occ": py_occ}


def rnnt_pruned_joiner_backward(batch: Batch, S: int, enc, dec, W, bias, ranges, lse, px_occ, py_occ,
                                scale=None, enc_grad=None, dec_grad=None, W_grad=None, bias_grad=None,
                                logits_grad=None, workspace=None, stream=None, want_param_grads=True,
                                want_logits_grad=False, logits=None, chunk_rows: int = 0, head=None,
                                head_rows: int = 0) -> dict:
    """The joiner backward; chunk_rows != 0 (a multiple of 128) or a head
    (the first chunk's logits from rnnt_pruned_joiner with ``head``) selects
    rnnt_pruned_joiner_backward_ex."""
    N, T, U = batch.N, batch.T, batch.U
    J, V = int(W.shape[0]), int(W.shape[1])
    dt = _jdtype(W)
    _need(enc, "enc", W.dtype, (N, T, J))
    _need(dec, "dec", W.dtype, (N, U + 1, J))
    for name, t in (("lse", lse), ("px_occ", px_occ), ("py_occ", py_occ)):
        _need(t, name, torch.float32, (N, T, S))
    _need(ranges, "ranges", torch.int32, (N, T, S))
    if logits is not None:
        _need(logits, "logits", torch.float32, (N, T, S, V))
    f32 = dict(dtype=torch.float32, device=batch.device)
    enc_grad = torch.empty(N, T, J, **f32) if enc_grad is None else enc_grad
    dec_grad = torch.empty(N, U + 1, J, **f32) if dec_grad is None else dec_grad
    if want_param_grads and W_grad is None:
        W_grad, bias_grad = torch.empty(J, V, **f32), torch.empty(V, **f32)
    if want_logits_grad and logits_grad is None:
        logits_grad = torch.empty(N, T, S, V, **f32)
    ws = _ws(pruned_joiner_backward_workspace_size(N, T, U, S, J, V, dt, chunk_rows), batch.device, workspace)
    rest = (_p(enc), _p(dec), _p(W), _p(bias), _p(ranges), _p(lse), _p(logits), _p(px_occ), _p(py_occ), _p(scale),
            _p(enc_grad), _p(dec_grad), _p(W_grad), _p(bias_grad), _p(logits_grad), _p(ws), ws.numel(),
            _stream(stream))
    if chunk_rows == 0 and head is None:
        check(lib().rnnt_pruned_joiner_backward(batch.c, S, J, V, dt, *rest))
    else:
        if head is not None:
            _need(head, "head", torch.float32, (head_rows, (V + 7) // 8 * 8))
        check(lib().rnnt_pruned_joiner_backward_ex(batch.c, S, J, V, dt, int(chunk_rows), *rest[:7], _p(head),
                                                   int(head_rows), *rest[7:]))
    return {"enc_grad": enc_grad, "dec_grad": dec_grad, "W_grad": W_grad, "bias_grad": bias_grad,
            "logits_grad": logits_grad}


_REDUCTIONS = {"sum": RNNT_REDUCE_SUM, "mean": RNNT_REDUCE_MEAN}


def rnnt_combine_losses(simple_loss: Optional[torch.Tensor], pruned_loss: Optional[torch.Tensor],
                        simple_scale: float, pruned_scale: float, reduction: str = "sum", loss=None, total=None,
                        stream=None) -> dict:
    """The training loss of Sec. 3.3 per utterance and summed (or averaged), in the library."""
    ref = simple_loss if simple_loss is not None else pruned_loss
    N = int(ref.shape[0])
    for name, t in (("simple_loss", simple_loss), ("pruned_loss", pruned_loss)):
        if t is not None:
            _need(t, name, torch.float32, (N,))
    f32 = dict(dtype=torch.float32, device=ref.device)
    loss = torch.empty(N, **f32) if loss is None else loss
    total = torch.empty((), **f32) if total is None else total
    check(lib().rnnt_combine_losses(N, _p(simple_loss), _p(pruned_loss), float(simple_scale), float(pruned_scale),
                                    _REDUCTIONS[reduction], _p(loss), _p(total), _stream(stream)))
    return {"loss": loss, "total": total}


def rnnt_validate_inputs(batch: Batch, V: int, S: int = 0, am=None, lm=None, enc=None, dec=None, flags=None,
                         stream=None) -> dict:
    """Synchronous check of a batch (Sec. 2's problem statement; the band
    condition for S > 0). Returns the per-utterance flag tensor, the number of
    flagged utterances and, per flagged utterance, the names of its flags."""
    N, T, U = batch.N, batch.T, batch.U
    if am is not None:
        _need(am, "am", torch.float32, (N, T, V))
    if lm is not None:
        _need(lm, "lm", torch.float32, (N, U + 1, V))
    J, dt = 0, RNNT_F32
    if enc is not None or dec is not None:
        ref = enc if enc is not None else dec
        J, dt = int(ref.shape[-1]), _jdtype(ref)
        if enc is not None:
            _need(enc, "enc", ref.dtype, (N, T, J))
        if dec is not None:
            _need(dec, "dec", ref.dtype, (N, U + 1, J))
    flags = torch.empty(N, dtype=torch.int32, device=batch.device) if flags is None else flags
    n_bad = ctypes.c_int32(0)
    check(lib().rnnt_validate_inputs(batch.c, V, S, J, dt, _p(am), _p(lm), _p(enc), _p(dec), _p(flags),
                                     ctypes.byref(n_bad), _stream(stream)))
    fl = flags.cpu().tolist()
    bad = {n: [k for k, bit in RNNT_FLAGS.items() if f & bit] for n, f in enumerate(fl) if f}
    return {"flags": flags, "n_bad": int(n_bad.value), "bad": bad}


def full_loss_workspace_size(N, T, U, J, V, dtype) -> int:
    return int(lib().rnnt_full_loss_workspace_size(N, T, U, J, V, dtype))


def rnnt_full_loss(batch: Batch, enc, dec, W, bias=None, scale=None, keep_logits: bool = False, loss=None,
                   enc_grad=None, dec_grad=None, W_grad=None, bias_grad=None, logits=None, workspace=None,
                   stream=None) -> dict:
    """The unpruned RNN-T loss with the same joiner at every (t, u), and its gradients."""
    N, T, U = batch.N, batch.T, batch.U
    J, V = int(W.shape[0]), int(W.shape[1])
    dt = _jdtype(W)
    _need(enc, "enc", W.dtype, (N, T, J))
    _need(dec, "dec", W.dtype, (N, U + 1, J))
    if bias is not None:
        _need(bias, "bias", W.dtype, (V,))
    if scale is not None:
        _need(scale, "scale", torch.float32, (N,))
    f32 = dict(dtype=torch.float32, device=batch.device)
    loss = torch.empty(N, **f32) if loss is None else loss
    enc_grad = torch.empty(N, T, J, **f32) if enc_grad is None else enc_grad
    dec_grad = torch.empty(N, U + 1, J, **f32) if dec_grad is None else dec_grad
    W_grad = torch.empty(J, V, **f32) if W_grad is None else W_grad
    bias_grad = torch.empty(V, **f32) if bias_grad is None else bias_grad
    if keep_logits and logits is None:
        logits = torch.empty(N, T, U + 1, V, **f32)
    ws = _ws(full_loss_workspace_size(N, T, U, J, V, dt), batch.device, workspace)
    check(lib().rnnt_full_loss(batch.c, J, V, dt, _p(enc), _p(dec), _p(W), _p(bias), _p(scale), _p(loss),
                               _p(enc_grad), _p(dec_grad), _p(W_grad), _p(bias_grad), _p(logits), _p(ws),
                               ws.numel(), _stream(stream)))
    return {"loss": loss, "enc_grad": enc_grad, "dec_grad": dec_grad, "W_grad": W_grad, "bias_grad": bias_grad,
            "logits": logits}


class PrunedRnntLoss:
    """The paper's training loss on one batch: pruned_scale * pruned + simple_scale * simple (Sec. 3.3).

    Holds the intermediate tensors and two workspaces between calls, so that
    repeated steps on same-shaped batches allocate nothing new. ``step``
    enqueues the whole path on the caller's stream: the simple loss and its
    occupations, the pruning bounds, the pruned joiner, the pruned recursion
    and the joiner backward. The simple loss's own gradients (two
    contractions that only the caller needs) run on a second stream at the
    default priority, forked after the joiner forward so that they overlap
    the pruned recursion, which occupies a few workgroups per utterance; the
    combined loss follows them there once the pruned loss is final (beside
    the joiner backward), and the stream is joined back before ``step``
    returns (in stream order).

    With ``pruned_scale == 0`` (the warm-up of Sec. 4: the pruned part is
    disabled until the simple loss gives useful bounds) the pruned stages are
    skipped and their loss and gradients are zero.

    By default no [N, T, S, V] array is kept: the backward recomputes the
    logits in chunks of rows whose size does not depend on N or T. With
    ``keep_logits`` the pruned logits [N, T, S, V] are stored by the forward
    and streamed by the backward instead, in one chunk of all rows (one GEMM
    less, the logits' memory more). ``bwd_chunk_rows`` (a multiple of 128, 0 = the library's choice)
    sets the backward's chunk. With ``keep_head`` (default) the forward keeps
    the logits of the backward's first chunk only (at most 16,384 rows, a
    buffer whose size does not depend on N or T), so that the backward
    streams that chunk instead of recomputing it.

    ``step`` also returns the training loss per utterance (``loss``) and its
    sum or mean (``total``), formed by the library (rnnt_combine_losses).

    ``lm_only_scale`` and ``am_only_scale`` smooth the simple loss's joiner
    (Sec. 3.3.1); both 0 gives the plain trivial joiner.
    """

    def __init__(self, S: int, simple_scale: float = 0.5, pruned_scale: float = 1.0,
                 keep_logits: bool = False, overlap: bool = True, lm_only_scale: float = 0.0,
                 am_only_scale: float = 0.0, bwd_chunk_rows: int = 0, keep_head: bool = True):
        self.S = int(S)
        self.simple_scale = float(simple_scale)
        self.pruned_scale = float(pruned_scale)
        self.lm_only_scale = float(lm_only_scale)
        self.am_only_scale = float(am_only_scale)
        self.keep_logits = bool(keep_logits)
        self.overlap = bool(overlap)
        self.bwd_chunk_rows = int(bwd_chunk_rows)
        self.keep_head = bool(keep_head)
        self._cache = {}
        self._side = {}

    def _buf(self, key, shape, dtype, device):
        t = self._cache.get(key)
        if t is None or tuple(t.shape) != tuple(shape) or t.dtype != dtype or t.device != device:
            t = torch.empty(shape, dtype=dtype, device=device)
            self._cache[key] = t
        return t

    def _side_stream(self, device):
        key = device.index if device.index is not None else torch.cuda.current_device()
        if key not in self._side:
            self._side[key] = (torch.cuda.Stream(device=device), torch.cuda.Event(), torch.cuda.Event(),
                               torch.cuda.Event())
        return self._side[key]

    def step(self, batch: Batch, am, lm, enc, dec, W, bias=None, stream=None, out=None,
             reduction: str = "sum") -> dict:
        """Run one step; ``out`` optionally maps output names to caller-owned
        tensors; ``reduction`` ("sum" or "mean") is that of ``total``."""
        N, T, U, S = batch.N, batch.T, batch.U, self.S
        V = int(am.shape[2])
        J = int(W.shape[0])
        dev = batch.device
        dt = _jdtype(W)
        f32 = torch.float32
        out = {} if out is None else out
        main = torch.cuda.current_stream(dev) if stream is None else stream

        def o(key, shape, dtype=f32):
            t = out.get(key)
            return t if t is not None else self._buf(key, shape, dtype, dev)

        chunk = self.bwd_chunk_rows
        if self.keep_logits and chunk == 0:
            # the caller keeps all the logits anyway: one chunk of every row
            # (fewer, fuller launches) unless that breaks the 32-bit limit
            whole = (N * T * S + 127) // 128 * 128
            chunk = whole if backward_chunk_rows(N, T, S, J, V, dt, whole) else 0
        ws_s = self._buf("ws_simple", (simple_loss_workspace_size(N, T, U, V),), torch.uint8, dev)
        ws_p = self._buf("ws_pruned", (max(pruned_joiner_workspace_size(N, T, S, J, V, dt),
                                           pruned_loss_workspace_size(N, T, U, S),
                                           pruned_joiner_backward_workspace_size(N, T, U, S, J, V, dt, chunk)),),
                         torch.uint8, dev)
        ssc = self._buf("ssc", (N,), f32, dev)
        psc = self._buf("psc", (N,), f32, dev)
        if self._cache.get("scales") != (N, self.simple_scale, self.pruned_scale):
            with torch.cuda.stream(main):
                ssc.fill_(self.simple_scale)
                psc.fill_(self.pruned_scale)
            self._cache["scales"] = (N, self.simple_scale, self.pruned_scale)
        sim = rnnt_simple_loss(
            batch, V, am, lm, ssc, loss=o("simple_loss", (N,)),
            px_occ=o("simple_px_occ", (N, T, U + 1)), py_occ=o("simple_py_occ", (N, T, U + 1)),
            workspace=ws_s, stream=main, lm_only_scale=self.lm_only_scale, am_only_scale=self.am_only_scale)
        res = {"simple_loss": sim["loss"], "simple_px_occ": sim["px_occ"], "simple_py_occ": sim["py_occ"]}
        am_grad, lm_grad = o("am_grad", (N, T, V)), o("lm_grad", (N, U + 1, V))
        enc_grad, dec_grad = o("enc_grad", (N, T, J)), o("dec_grad", (N, U + 1, J))
        W_grad, bias_grad = o("W_grad", (J, V)), o("bias_grad", (V,))
        res.update(am_grad=am_grad, lm_grad=lm_grad, enc_grad=enc_grad, dec_grad=dec_grad, W_grad=W_grad,
                   bias_grad=bias_grad)

        def simple_backward(s):
            rnnt_simple_loss_backward(batch, V, am, lm, sim["px_occ"], ws_s, scale=ssc, am_grad=am_grad,
                                      lm_grad=lm_grad, stream=s, lm_only_scale=self.lm_only_scale,
                                      am_only_scale=self.am_only_scale)

        if self.pruned_scale == 0.0:
            # warm-up: the pruned part carries no weight and is not evaluated
            simple_backward(main)
            with torch.cuda.stream(main):
                pl = o("pruned_loss", (N,))
                for t in (pl, enc_grad, dec_grad, W_grad, bias_grad):
                    t.zero_()
            res["pruned_loss"] = pl
            res.update(rnnt_combine_losses(sim["loss"], None, self.simple_scale, 0.0, reduction,
                                           loss=o("loss", (N,)), total=o("total", ()), stream=main))
            return res

        ranges = rnnt_prune_ranges(batch, S, sim["px_occ"], sim["py_occ"], ranges=o("ranges", (N, T, S), torch.int32),
                                   stream=main)
        logits = o("logits", (N, T, S, V)) if self.keep_logits else None
        head, head_rows = None, 0
        if not self.keep_logits and self.keep_head:
            head_rows = backward_chunk_rows(N, T, S, J, V, dt, chunk)
            head = self._buf("head", (head_rows, (V + 7) // 8 * 8), f32, dev)
        jo = rnnt_pruned_joiner(batch, S, enc, dec, W, bias, ranges, px=o("px", (N, T, S)), py=o("py", (N, T, S)),
                                lse=o("lse", (N, T, S)), logits=logits, workspace=ws_p, stream=main, head=head,
                                head_rows=head_rows)
        if self.overlap:
            side, fork, join, lossev = self._side_stream(dev)
            fork.record(main)
            side.wait_event(fork)
            simple_backward(side)
        else:
            simple_backward(main)
        pl = rnnt_pruned_loss(batch, S, jo["px"], jo["py"], ranges, loss=o("pruned_loss", (N,)),
                              px_occ=o("pruned_px_occ", (N, T, S)), py_occ=o("pruned_py_occ", (N, T, S)),
                              workspace=ws_p, stream=main)
        if self.overlap:
            lossev.record(main)  # both losses are final here
        rnnt_pruned_joiner_backward(
            batch, S, enc, dec, W, bias, ranges, jo["lse"], pl["px_occ"], pl["py_occ"], scale=psc,
            enc_grad=enc_grad, dec_grad=dec_grad, W_grad=W_grad, bias_grad=bias_grad, workspace=ws_p,
            stream=main, logits=logits, chunk_rows=chunk, head=head, head_rows=head_rows)
        # the combined loss needs only the two losses: with the second stream
        # it runs there, beside the joiner backward, instead of after it
        if self.overlap:
            side.wait_event(lossev)
        res.update(rnnt_combine_losses(sim["loss"], pl["loss"], self.simple_scale, self.pruned_scale, reduction,
                                       loss=o("loss", (N,)), total=o("total", ()),
                                       stream=side if self.overlap else main))
        if self.overlap:
            join.record(side)
            main.wait_event(join)
        res.update(pruned_loss=pl["loss"], ranges=ranges, px=jo["px"], py=jo["py"], lse=jo["lse"],
                   pruned_px_occ=pl["px_occ"], pruned_py_occ=pl["py_occ"])
        return res


class _PrunedRnntFunction(torch.autograd.Function):
    """Forward computes the loss and every gradient at once (the kernels are
    fused forward-backward); backward scales the stored gradients."""

    @staticmethod
    def forward(ctx, am, lm, enc, dec, W, bias, module, batch, reduction):
        N, T, U, V, J = batch.N, batch.T, batch.U, int(am.shape[2]), int(W.shape[0])
        f32 = dict(dtype=torch.float32, device=am.device)
        fresh = {"am_grad": torch.empty(N, T, V, **f32), "lm_grad": torch.empty(N, U + 1, V, **f32),
                 "enc_grad": torch.empty(N, T, J, **f32), "dec_grad": torch.empty(N, U + 1, J, **f32),
                 "W_grad": torch.empty(J, V, **f32), "bias_grad": torch.empty(V, **f32)}
        fresh["total"] = torch.empty((), **f32)
        r = module.step(batch, am, lm, enc, dec, W, bias, out=fresh, reduction=reduction)
        loss = r["total"]
        ctx.reduction = reduction
        ctx.N = N
        ctx.has_bias = bias is not None
        ctx.dtypes = (enc.dtype, dec.dtype, W.dtype)
        ctx.save_for_backward(fresh["am_grad"], fresh["lm_grad"], fresh["enc_grad"], fresh["dec_grad"],
                              fresh["W_grad"], fresh["bias_grad"])
        return loss

    @staticmethod
    def backward(ctx, g):
        am_g, lm_g, enc_g, dec_g, W_g, b_g = ctx.saved_tensors
        if ctx.reduction == "mean":
            g = g / ctx.N
        ed, dd, wd = ctx.dtypes
        return (am_g * g, lm_g * g, (enc_g * g).to(ed), (dec_g * g).to(dd), (W_g * g).to(wd),
                (b_g * g).to(wd) if ctx.has_bias else None, None, None, None)


def pruned_rnnt_loss(am, lm, enc, dec, W, bias, batch: Batch, S: int, simple_scale: float = 0.5,
                     pruned_scale: float = 1.0, reduction: str = "sum", module: Optional[PrunedRnntLoss] = None,
                     lm_only_scale: float = 0.0, am_only_scale: float = 0.0):
    """Differentiable training loss: sum (or mean) over utterances of
    simple_scale * simple_loss + pruned_scale * pruned_loss (Sec. 3.3), the
    simple loss optionally with the smoothed joiner (Sec. 3.3.1)."""
    if reduction not in ("sum", "mean"):
        raise ValueError("reduction must be 'sum' or 'mean'")
    if module is None:
        module = PrunedRnntLoss(S, simple_scale=simple_scale, pruned_scale=pruned_scale,
                                lm_only_scale=lm_only_scale, am_only_scale=am_only_scale)
    return _PrunedRnntFunction.apply(am, lm, enc, dec, W, bias, module, batch, reduction)
