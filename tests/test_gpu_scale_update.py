"""Scale-update kernel parity: the hand-computed rollover sequences and random
histories, bit-exact against the oracle."""
import math
import os

import numpy as np
import pytest

from oracle import fp8, scaling
from tests.gpu_util import dev, meta_buffer, meta_of, torch
from tests.libqe import need_lib

pytestmark = pytest.mark.gpu
GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def _parse(v):
    return float(v) if v in ("nan", "inf", "-inf") else float.fromhex(v)


def test_rollover_golden_on_gpu():
    qe = need_lib()
    d = dev()
    n = 0
    for line in open(os.path.join(GOLDEN, "scale_rollover.txt")):
        line = line.strip()
        if not line or line.startswith("#"):
            continue
        head, amaxes, scales = [p.strip() for p in line.split("|")]
        name, H, margin = head.split()
        H = int(H)
        mb = meta_buffer(H, d)
        m = meta_of(qe, mb, qe.E4M3 if name == "E4M3" else qe.E5M2, int(margin))
        for a, want in zip(amaxes.split(","), scales.split(",")):
            # record through the quantizer, exactly as an action does
            x = torch.tensor([[_parse(a)]], dtype=torch.float32, device=d)
            assert qe.qe_quantize_fp8(x, qe.F32, 1, 1, m) == "OK"
            assert qe.qe_amax_scale_update([m]) == "OK"
            torch.cuda.synchronize()
            assert mb[H].item() == _parse(want), (line, a)
            assert mb[H + 1].item() * mb[H].item() == 1.0
        n += 1
    assert n >= 5


@pytest.mark.parametrize("H", [1, 2, 16, 1000, 1024, 8192])
@pytest.mark.parametrize("fmt", ["E4M3", "E5M2"])
def test_random_histories(H, fmt):
    qe = need_lib()
    d = dev()
    rng = np.random.default_rng(H)
    hist = (rng.random(H) * np.exp2(rng.integers(-30, 30, H))).astype(np.float32)
    hist[rng.random(H) < 0.3] = 0
    for margin in (0, 2):
        s = scaling.DelayedScaler(fmt, H, margin)
        s.hist = hist.astype(np.float64).copy()
        mb = meta_buffer(H, d)
        mb[:H] = torch.from_numpy(hist).to(d)
        m = meta_of(qe, mb, qe.E4M3 if fmt == "E4M3" else qe.E5M2, margin)
        for _ in range(3):
            s.update()
            assert qe.qe_amax_scale_update([m]) == "OK"
            torch.cuda.synchronize()
            got = mb.cpu().numpy()
            np.testing.assert_array_equal(got[:H], s.hist.astype(np.float32))
            assert got[H] == s.scale and got[H + 1] == s.scale_inv


def test_many_roles_one_launch_and_token():
    qe = need_lib()
    d = dev()
    bufs, metas, oracles = [], [], []
    for i in range(8):
        H = 3 + i
        b = meta_buffer(H, d)
        b[0] = float(2.0 ** (i - 4) * 1.3)
        bufs.append(b)
        fmt = i % 2
        metas.append(meta_of(qe, b, fmt, i % 3))
        s = scaling.DelayedScaler("E4M3" if fmt == 0 else "E5M2", H, i % 3)
        s.hist[0] = float(np.float32(2.0 ** (i - 4) * 1.3))
        oracles.append(s)
    tok = torch.zeros(1, dtype=torch.int64, device=d)
    for _ in range(2):
        assert qe.qe_amax_scale_update(metas, device_token=tok) == "OK"
        for s in oracles:
            s.update()
    torch.cuda.synchronize()
    assert tok.item() == 2
    for b, s in zip(bufs, oracles):
        H = b.numel() - 2
        got = b.cpu().numpy()
        np.testing.assert_array_equal(got[:H], s.hist.astype(np.float32))
        assert got[H] == s.scale


def test_nan_and_subnormal_amax():
    qe = need_lib()
    d = dev()
    for a in (float("nan"), float("inf"), 0.0, 1e-40, 2.0 ** -149, 448.0):
        mb = meta_buffer(1, d, 4.0)
        mb[0] = a
        m = meta_of(qe, mb, qe.E4M3, 0)
        s = scaling.DelayedScaler("E4M3", 1, 0)
        s.scale, s.scale_inv = 4.0, 0.25
        s.hist[0] = float(np.float32(a))
        s.update()
        assert qe.qe_amax_scale_update([m]) == "OK"
        torch.cuda.synchronize()
        assert mb[1].item() == s.scale, a
        assert mb[0].item() == 0.0
