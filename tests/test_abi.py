"""Host-side checks of the C ABI (CPU only: no kernel is launched).

The library must load on a machine without a GPU, export every function the
header declares, answer the workspace queries, and reject bad arguments with
the documented status before any HIP call.
"""
import ctypes
import os
import re

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "rnnt_pruned.h")


@pytest.fixture(scope="module")
def L():
    from paper_2206_13236_amd import _native
    if not os.path.exists(_native.LIB_PATH):
        from paper_2206_13236_amd.build import build
        build()
    return _native.lib()


def _declared():
    src = open(HEADER).read()
    src = re.sub(r"/\*.*?\*/", "", src, flags=re.S)
    return sorted(set(re.findall(r"\b(rnnt_[a-z_]+)\s*\(", src)))


def test_header_declares_the_entry_points():
    names = _declared()
    for n in ("rnnt_simple_loss", "rnnt_prune_ranges", "rnnt_pruned_joiner", "rnnt_pruned_loss",
              "rnnt_pruned_joiner_backward", "rnnt_last_error", "rnnt_abi_version", "rnnt_validate_inputs",
              "rnnt_combine_losses", "rnnt_pruned_joiner_backward_ex"):
        assert n in names


def test_library_exports_every_declared_symbol(L):
    from paper_2206_13236_amd import _native
    missing = [n for n in _declared() if not hasattr(L, n)]
    assert not missing, f"not exported: {missing}"
    assert set(_declared()) == set(_native.SIGNATURES), "binding signatures out of sync with the header"
    assert L.rnnt_abi_version() == 8


def test_workspace_queries(L):
    from paper_2206_13236_amd import _native as N
    a = L.rnnt_simple_loss_workspace_size(16, 250, 60, 500)
    assert a > 0
    assert L.rnnt_simple_loss_workspace_size(16, 250, 60, 500) == a  # a pure function of the sizes
    assert L.rnnt_simple_loss_workspace_size(0, 250, 60, 500) == 0
    # bigger shapes need more
    assert L.rnnt_simple_loss_workspace_size(16, 250, 61, 500) >= a
    f = L.rnnt_pruned_joiner_workspace_size(16, 250, 5, 512, 500, N.RNNT_F32)
    assert f > 0
    b32 = L.rnnt_pruned_joiner_backward_workspace_size(16, 250, 60, 5, 512, 500, N.RNNT_F32)
    b16 = L.rnnt_pruned_joiner_backward_workspace_size(16, 250, 60, 5, 512, 500, N.RNNT_BF16)
    assert b32 > 0 and b16 > 0
    # wavefront: alpha and beta (fp64) over T+U diagonals of at least S slots
    wf = L.rnnt_pruned_loss_ex_workspace_size(16, 250, 60, 5, 1, 0)
    assert wf >= 2 * 16 * (250 + 60) * 5 * 8
    # scan with chunks of C frames: an S x S matrix per chunk (fp64), at least
    for C in (1, 8, 32):
        assert L.rnnt_pruned_loss_ex_workspace_size(16, 250, 60, 5, 2, C) >= 16 * (-(-250 // C)) * 25 * 8
    assert L.rnnt_pruned_loss_ex_workspace_size(16, 250, 60, 5, 2, 33) == 0    # chunk too long
    assert L.rnnt_pruned_loss_ex_workspace_size(16, 250, 60, 17, 2, 0) == 0    # S beyond the scan
    assert L.rnnt_pruned_loss_ex_workspace_size(16, 250, 60, 5, 3, 0) == 0     # no such algorithm
    # rnnt_pruned_loss: the automatic choice, the scan for S <= 16
    assert L.rnnt_pruned_loss_workspace_size(16, 250, 60, 5) == L.rnnt_pruned_loss_ex_workspace_size(
        16, 250, 60, 5, 2, 0)
    assert L.rnnt_pruned_loss_workspace_size(16, 250, 60, 20) == L.rnnt_pruned_loss_ex_workspace_size(
        16, 250, 60, 20, 1, 0)
    assert L.rnnt_pruned_loss_workspace_size(16, 250, 60, 0) == 0
    assert L.rnnt_full_loss_workspace_size(2, 20, 5, 32, 16, N.RNNT_F32) > 0


def _batch(N=2, T=10, U=3):
    from paper_2206_13236_amd._native import RnntBatch
    # fake device addresses: validation never dereferences them
    return RnntBatch(N, T, U, 0x1000, 0x2000, 0x3000, 0)


def _err(L):
    return L.rnnt_last_error().decode()


def test_validation_statuses(L):
    from paper_2206_13236_amd import _native as N
    b = _batch()
    pb = ctypes.byref(b)
    fake = ctypes.c_void_p(0x4000)
    # NULL batch
    assert L.rnnt_prune_ranges(None, 4, fake, fake, fake, None) == N.RNNT_EINVAL
    assert "NULL" in _err(L)
    # S out of range
    assert L.rnnt_prune_ranges(pb, 0, fake, fake, fake, None) == N.RNNT_EUNSUPPORTED
    assert L.rnnt_prune_ranges(pb, 33, fake, fake, fake, None) == N.RNNT_EUNSUPPORTED
    # missing required output
    assert L.rnnt_prune_ranges(pb, 4, fake, fake, None, None) == N.RNNT_EINVAL
    # simple loss: blank outside [0, V)
    b2 = _batch()
    b2.blank = 16
    assert L.rnnt_simple_loss(ctypes.byref(b2), 16, fake, fake, None, 0.0, 0.0, fake, fake, fake, None, None, None, None,
                              fake, 1 << 30, None) == N.RNNT_EINVAL
    # simple loss: workspace missing / too small / misaligned
    assert L.rnnt_simple_loss(pb, 16, fake, fake, None, 0.0, 0.0, fake, fake, fake, None, None, None, None,
                              None, 0, None) == N.RNNT_EWORKSPACE
    assert L.rnnt_simple_loss(pb, 16, fake, fake, None, 0.0, 0.0, fake, fake, fake, None, None, None, None,
                              fake, 16, None) == N.RNNT_EWORKSPACE
    assert L.rnnt_simple_loss(pb, 16, fake, fake, None, 0.0, 0.0, fake, fake, fake, None, None, None, None,
                              ctypes.c_void_p(0x4004), 1 << 30, None) == N.RNNT_EWORKSPACE
    # smoothing weights outside a_lm, a_ac >= 0, a_lm + a_ac <= 1
    for w in ((-0.1, 0.0), (0.0, -0.5), (0.7, 0.4)):
        assert L.rnnt_simple_loss(pb, 16, fake, fake, None, w[0], w[1], fake, fake, fake, None, None, None, None,
                                  fake, 1 << 30, None) == N.RNNT_EINVAL
    # px without py
    assert L.rnnt_simple_loss(pb, 16, fake, fake, None, 0.0, 0.0, fake, fake, fake, fake, None, None, None,
                              fake, 1 << 30, None) == N.RNNT_EINVAL
    # negative sizes
    bad = _batch(N=0)
    assert L.rnnt_pruned_loss(ctypes.byref(bad), 4, fake, fake, fake, fake, None, None, fake, 1 << 30,
                              None) == N.RNNT_EINVAL
    # pruned loss: unknown algorithm, scan beyond S = 16, chunk out of range
    assert L.rnnt_pruned_loss_ex(pb, 4, 3, 0, fake, fake, fake, fake, None, None, fake, 1 << 30,
                                 None) == N.RNNT_EINVAL
    assert L.rnnt_pruned_loss_ex(pb, 17, 2, 0, fake, fake, fake, fake, None, None, fake, 1 << 30,
                                 None) == N.RNNT_EUNSUPPORTED
    assert L.rnnt_pruned_loss_ex(pb, 4, 2, 33, fake, fake, fake, fake, None, None, fake, 1 << 30,
                                 None) == N.RNNT_EINVAL
    assert L.rnnt_pruned_loss_ex(pb, 4, 2, 0, fake, fake, fake, fake, None, None, fake, 8,
                                 None) == N.RNNT_EWORKSPACE
    # U beyond the lattice limit
    big = _batch(U=1024)
    assert L.rnnt_prune_ranges(ctypes.byref(big), 4, fake, fake, fake, None) == N.RNNT_EUNSUPPORTED
    # joiner: J not a multiple of 8, bad dtype
    assert L.rnnt_pruned_joiner(pb, 4, 12, 16, N.RNNT_F32, fake, fake, fake, None, fake, fake, fake, fake,
                                None, fake, 1 << 30, None) == N.RNNT_EUNSUPPORTED
    assert L.rnnt_pruned_joiner(pb, 4, 16, 16, 7, fake, fake, fake, None, fake, fake, fake, fake,
                                None, fake, 1 << 30, None) == N.RNNT_EINVAL
    # backward: enc_grad required
    assert L.rnnt_pruned_joiner_backward(pb, 4, 16, 16, N.RNNT_F32, fake, fake, fake, None, fake, fake, None,
                                         fake, fake, None, None, fake, None, None, None, fake, 1 << 30,
                                         None) == N.RNNT_EINVAL
    # a success clears the message; the last failure leaves one
    assert _err(L) != ""


def test_python_binding_checks_shapes_on_cpu():
    import torch
    import paper_2206_13236_amd as P
    with pytest.raises(ValueError):
        P.Batch(torch.zeros(2, dtype=torch.int32), torch.zeros(2, dtype=torch.int32),
                torch.zeros(2, 3, dtype=torch.int32), 10, 3)  # CPU tensors are rejected


def test_backward_chunk_memory_does_not_grow_with_the_batch(L):
    # The backward holds d(logits), h and the d dec pieces for one chunk of
    # rows whose size depends on J, V and the dtype only: ten times the
    # utterances add only per-row bookkeeping (row info, d enc pieces), far
    # below the V * 4 bytes per row that [N, T, S, V] logits would take.
    from paper_2206_13236_amd import _native as N
    shapes = {"bpe": (16, 248, 58, 5, 512, 500, N.RNNT_F32), "long": (32, 495, 100, 5, 512, 500, N.RNNT_BF16),
              "largev": (16, 298, 78, 5, 512, 5000, N.RNNT_F32), "stress": (8, 970, 298, 10, 768, 8000, N.RNNT_BF16)}
    for name, (n, t, u, s_, j, v, dt) in shapes.items():
        a = L.rnnt_pruned_joiner_backward_workspace_size(n, t, u, s_, j, v, dt)
        b = L.rnnt_pruned_joiner_backward_workspace_size(10 * n, t, u, s_, j, v, dt)
        per_row = (b - a) / (9 * n * t * s_)
        assert 0 < per_row < 16 + 8 * j / 64 + 8, (name, per_row)
    # the chunk override: a smaller chunk needs less workspace, an invalid one none
    big = L.rnnt_pruned_joiner_backward_ex_workspace_size(16, 248, 58, 5, 512, 500, N.RNNT_F32, 0)
    small = L.rnnt_pruned_joiner_backward_ex_workspace_size(16, 248, 58, 5, 512, 500, N.RNNT_F32, 256)
    assert 0 < small < big
    assert big == L.rnnt_pruned_joiner_backward_workspace_size(16, 248, 58, 5, 512, 500, N.RNNT_F32)
    assert L.rnnt_pruned_joiner_backward_ex_workspace_size(16, 248, 58, 5, 512, 500, N.RNNT_F32, 100) == 0
    assert L.rnnt_pruned_joiner_backward_ex_workspace_size(16, 248, 58, 5, 512, 500, N.RNNT_F32, -128) == 0


def test_sizes_beyond_32_bit_buffer_offsets_are_refused(L):
    # Chunk buffers are read through 32-bit buffer offsets: a vocabulary so
    # large that one 128-row tile of d(logits) reaches 2^31 bytes is refused
    # before any launch; so is an explicit chunk beyond that limit.
    from paper_2206_13236_amd import _native as N
    b = _batch(N=1, T=4, U=2)
    pb = ctypes.byref(b)
    fake = ctypes.c_void_p(0x4000)
    V = 5_000_000
    assert L.rnnt_pruned_joiner(pb, 2, 8, V, N.RNNT_F32, fake, fake, fake, None, fake, fake, fake, fake, None,
                                fake, 1 << 40, None) == N.RNNT_EUNSUPPORTED
    assert "too large" in _err(L)
    assert L.rnnt_pruned_joiner_backward(pb, 2, 8, V, N.RNNT_F32, fake, fake, fake, None, fake, fake, None,
                                         fake, fake, None, fake, fake, None, None, None, fake, 1 << 40,
                                         None) == N.RNNT_EUNSUPPORTED
    assert L.rnnt_full_loss(pb, 8, V, N.RNNT_F32, fake, fake, fake, None, None, fake, fake, fake, None, None,
                            None, fake, 1 << 40, None) == N.RNNT_EUNSUPPORTED
    # V = 500, J = 512: at most (2^31 - 1) / (512 * 4) rows, rounded down to 1,024
    args = (fake, fake, fake, None, fake, fake, None, None, 0, fake, fake, None, fake, fake, None, None, None, fake,
            1 << 40, None)
    assert L.rnnt_pruned_joiner_backward_ex(pb, 2, 512, 500, N.RNNT_F32, 1 << 20, *args) == N.RNNT_EUNSUPPORTED
    assert L.rnnt_pruned_joiner_backward_ex(pb, 2, 512, 500, N.RNNT_F32, 100, *args) == N.RNNT_EINVAL
    # the unpruned loss at the largest workload's shape (8 x 1000 x 301 rows of
    # J = 768) passes the size checks now that its row buffers are chunked:
    # only the (deliberately tiny) workspace is refused
    big = _batch(N=8, T=1000, U=300)
    assert L.rnnt_full_loss(ctypes.byref(big), 768, 8000, N.RNNT_BF16, fake, fake, fake, None, None, fake, fake,
                            fake, None, None, None, fake, 16, None) == N.RNNT_EWORKSPACE
    ws = L.rnnt_full_loss_workspace_size(8, 1000, 300, 768, 8000, N.RNNT_BF16)
    assert 0 < ws < 8 * 1000 * 301 * 768 * 4  # far below an [M, J] fp32 array


def test_combine_and_validate_statuses(L):
    from paper_2206_13236_amd import _native as N
    fake = ctypes.c_void_p(0x4000)
    # combine: N, reduction, scales, required inputs and outputs
    assert L.rnnt_combine_losses(0, fake, fake, 0.5, 1.0, 0, fake, fake, None) == N.RNNT_EINVAL
    assert L.rnnt_combine_losses(4, fake, fake, 0.5, 1.0, 2, fake, fake, None) == N.RNNT_EINVAL
    assert L.rnnt_combine_losses(4, fake, fake, -0.5, 1.0, 0, fake, fake, None) == N.RNNT_EINVAL
    assert L.rnnt_combine_losses(4, fake, None, 0.5, 1.0, 0, fake, fake, None) == N.RNNT_EINVAL
    assert L.rnnt_combine_losses(4, None, fake, 0.5, 1.0, 0, fake, fake, None) == N.RNNT_EINVAL
    assert L.rnnt_combine_losses(4, fake, fake, 0.5, 1.0, 0, None, None, None) == N.RNNT_EINVAL
    # validate: V, blank, S, J with enc, dtype, flags
    b = _batch()
    pb = ctypes.byref(b)
    n_bad = ctypes.c_int32()
    assert L.rnnt_validate_inputs(pb, 0, 4, 0, 0, None, None, None, None, fake, ctypes.byref(n_bad),
                                  None) == N.RNNT_EINVAL
    assert L.rnnt_validate_inputs(pb, 16, 33, 0, 0, None, None, None, None, fake, ctypes.byref(n_bad),
                                  None) == N.RNNT_EINVAL
    assert L.rnnt_validate_inputs(pb, 16, 4, 0, 0, None, None, fake, None, fake, ctypes.byref(n_bad),
                                  None) == N.RNNT_EINVAL
    assert L.rnnt_validate_inputs(pb, 16, 4, 32, 5, None, None, fake, None, fake, ctypes.byref(n_bad),
                                  None) == N.RNNT_EINVAL
    assert L.rnnt_validate_inputs(pb, 16, 4, 0, 0, None, None, None, None, None, ctypes.byref(n_bad),
                                  None) == N.RNNT_EINVAL
    b2 = _batch()
    b2.blank = 16
    assert L.rnnt_validate_inputs(ctypes.byref(b2), 16, 4, 0, 0, None, None, None, None, fake, None,
                                  None) == N.RNNT_EINVAL


def test_noalloc_entry_refuses_batches_beyond_its_scratch(L):
    # the allocation-free pruned recursion checks its workspace need against
    # the static scratch on the host, before any device call
    from paper_2206_13236_amd import _native as N
    fake = ctypes.c_void_p(0x4000)
    big = _batch(N=64, T=4096, U=0)
    need = L.rnnt_pruned_loss_workspace_size(64, 4096, 0, 16)
    assert need > N.RNNT_SCRATCH_BYTES
    assert L.rnnt_pruned_loss_noalloc(ctypes.byref(big), 16, fake, fake, fake, fake, None, None,
                                      None) == N.RNNT_EUNSUPPORTED
    assert "static scratch" in _err(L) and str(need) in _err(L)
    # argument checks as for rnnt_pruned_loss
    b = _batch()
    assert L.rnnt_pruned_loss_noalloc(ctypes.byref(b), 0, fake, fake, fake, fake, None, None,
                                      None) == N.RNNT_EUNSUPPORTED
    assert L.rnnt_pruned_loss_noalloc(ctypes.byref(b), 4, fake, fake, fake, None, None, None,
                                      None) == N.RNNT_EINVAL
    # the workloads' batches fit
    for n, t, u, s_ in ((16, 248, 58, 5), (32, 495, 100, 5), (8, 970, 298, 10)):
        assert 0 < L.rnnt_pruned_loss_workspace_size(n, t, u, s_) <= N.RNNT_SCRATCH_BYTES


def test_head_rows_must_match_the_backward_chunk(L):
    # the first chunk's logits kept by the forward are accepted by the
    # backward only with the row count of its own first chunk
    from paper_2206_13236_amd import _native as N
    b = _batch(N=16, T=248, U=58)
    pb = ctypes.byref(b)
    fake = ctypes.c_void_p(0x4000)
    C = L.rnnt_pruned_joiner_backward_chunk_rows(16, 248, 5, 512, 500, N.RNNT_F32, 0)
    assert C % 128 == 0 and 8192 <= C <= 16384
    assert L.rnnt_pruned_joiner_backward_chunk_rows(16, 248, 5, 512, 500, N.RNNT_F32, 1024) == 1024
    assert L.rnnt_pruned_joiner_backward_chunk_rows(16, 248, 5, 512, 500, N.RNNT_F32, 100) == 0
    args = lambda head_rows: (fake, fake, fake, None, fake, fake, None, fake, head_rows, fake, fake, None, fake,
                              fake, None, None, None, fake, 1 << 40, None)
    assert L.rnnt_pruned_joiner_backward_ex(pb, 5, 512, 500, N.RNNT_F32, 0, *args(C + 128)) == N.RNNT_EINVAL
    assert "head_rows" in _err(L)
    assert L.rnnt_pruned_joiner_ex(pb, 5, 512, 500, N.RNNT_F32, fake, fake, fake, None, fake, fake, fake, fake,
                                   None, fake, 100, fake, 1 << 40, None) == N.RNNT_EINVAL
