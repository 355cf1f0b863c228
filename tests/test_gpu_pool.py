"""Cross-process KV-cache pool (paper Sec. 3, KV-cache sharing across
stages): a retrieval-side process encodes into a pool slot and exports the
pool's IPC handle to a file; a ranking-side process maps the pool and ranks
against the slot in place.  Both are fresh child processes; the consumer's
scores must equal an in-process encode + rank bit for bit."""
import os
import subprocess
import sys

import numpy as np
import pytest

from tests.gpu_util import GpuRun, say
from tests import pool_child

pytestmark = pytest.mark.gpu

CHILD = os.path.join(os.path.dirname(os.path.abspath(__file__)), "pool_child.py")


def test_pool_slot_shared_between_processes(tmp_path):
    say("[gpu] pool: producer and consumer child processes")
    procs = {r: subprocess.Popen([sys.executable, "-u", CHILD, r, str(tmp_path)],
                                 stdout=subprocess.PIPE, stderr=subprocess.STDOUT, text=True)
             for r in ("producer", "consumer")}
    outs = {}
    try:
        for r in ("consumer", "producer"):
            outs[r], _ = procs[r].communicate(timeout=240)
    finally:
        for p in procs.values():
            if p.poll() is None:
                p.kill()
                p.wait()
    for r in ("producer", "consumer"):
        say(f"[gpu] pool {r} (rc {procs[r].returncode}): {outs.get(r, '').strip()[-600:]}")
        assert procs[r].returncode == 0, f"{r} failed"
    got = np.load(tmp_path / "scores.npy")
    run = GpuRun(pool_child.inputs())
    run.encode()
    run.rank()
    ref = run.scores_np()[: got.size].astype(np.float32)
    assert np.all(np.isfinite(got))
    assert np.array_equal(got, ref), f"max |diff| {np.abs(got - ref).max():.3e}"
    say(f"[gpu] pool: {got.size} scores ranked in another process equal the in-process ones")
