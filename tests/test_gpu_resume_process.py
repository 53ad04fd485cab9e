"""Fresh-process resume (§3.5; Table "correctness", fresh-process resume): a
stage saved at an optimizer boundary by one process and imported by another
process, started afresh, continues bit for bit like a run that was never
interrupted: outputs, placed gradients and FP8 state of every step after the
save.  Each run is its own Python process on the same GPU, one after the
other."""
import os
import subprocess
import sys

import numpy as np
import pytest

pytestmark = pytest.mark.gpu

HERE = os.path.dirname(os.path.abspath(__file__))
WORKER = os.path.join(HERE, "resume_worker.py")


def _child(*args):
    r = subprocess.run([sys.executable, "-u", WORKER, *args], stdout=subprocess.PIPE, stderr=subprocess.STDOUT,
                       text=True, timeout=300)
    print(r.stdout[-2000:], flush=True)
    assert r.returncode == 0, r.stdout[-4000:]


@pytest.mark.timeout(900)
def test_resume_in_fresh_process_bitwise_equals_uninterrupted(tmp_path):
    from tests.gpu_util import dev
    dev()  # skips without a GPU
    full = tmp_path / "full.npz"
    ckpt = tmp_path / "ckpt.bin"
    resumed = tmp_path / "resumed.npz"
    _child("run", str(full))
    _child("save", str(ckpt))
    _child("resume", str(ckpt), str(resumed))
    a, b = np.load(full), np.load(resumed)
    assert sorted(a.files) == sorted(b.files) and len(a.files) > 0
    assert any(f.startswith("grad_7") for f in a.files)
    for f in a.files:
        np.testing.assert_array_equal(a[f].view(np.uint32) if a[f].dtype == np.float32 else a[f],
                                      b[f].view(np.uint32) if b[f].dtype == np.float32 else b[f], err_msg=f)
