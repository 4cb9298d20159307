"""Host-side logic that needs no GPU: the benchmark's one-GPU contract and the
workspace rule of the pruned recursion's chunked scan."""
import os
import subprocess
import sys

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def test_more_than_one_gpu_exits_with_a_message():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"], capture_output=True,
                       text=True, timeout=120)
    assert r.returncode == 2
    assert "one GPU" in r.stderr and r.stdout == ""


def test_band_chunk_choice_and_workspace_track_the_scan_rule():
    # rnnt_pruned_loss's workspace at S <= 16 is the scan's, whose chunk
    # matrices grow as T / C for the chunk length C the library picks
    import paper_2206_13236_amd as P
    sizes = {T: P.pruned_loss_workspace_size(16, T, 60, 5) for T in (200, 256, 257, 640, 641)}
    assert sizes[200] > 0
    assert sizes[257] < sizes[256] * 257 / 256 * 0.75  # chunks of 16 from T = 257 on (8 below)
    assert sizes[641] < sizes[640] * 641 / 640 * 0.75  # chunks of 32 from T = 641 on
