"""Helpers for GPU parity tests (marked gpu; run on an MI355X)."""
import numpy as np
import pytest

torch = pytest.importorskip("torch")


def dev():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    return torch.device("cuda:0")


def upload(t, device):
    """workloads.Tensor -> device tensor (float32, or int16 holding bf16 bits)."""
    if t.dtype == "bf16":
        return torch.from_numpy(np.ascontiguousarray(t.data).view(np.int16)).to(device)
    return torch.from_numpy(np.ascontiguousarray(t.data)).to(device)


def u8(n, device):
    return torch.zeros(max(int(n), 1), dtype=torch.uint8, device=device)


def meta_buffer(H, device, scale=1.0):
    """history[H] | scale | scale_inv in one float32 tensor."""
    b = torch.zeros(H + 2, dtype=torch.float32, device=device)
    b[H] = scale
    b[H + 1] = 1.0 / scale
    return b


def meta_of(qe, buf, fmt, margin=0, accum=None):
    """FP8Meta over a meta_buffer; `accum` (64 x 64 float32, zeroed) adds an amax accumulator."""
    H = buf.numel() - 2
    return qe.FP8Meta(buf.data_ptr(), buf.data_ptr() + 4 * H, buf.data_ptr() + 4 * (H + 1), H, margin, fmt, 0,
                      0 if accum is None else accum.data_ptr())


def accum_buffer(device):
    return torch.zeros(64 * 64, dtype=torch.float32, device=device)


def accum_value(accum):
    """Value of an amax accumulator: max over its 64 lines (NaN if any line holds NaN)."""
    lines = accum.cpu().numpy()[::64]
    return float(np.nan) if np.isnan(lines).any() else float(lines.max())


def rel_err(got, ref):
    got = np.asarray(got, dtype=np.float64)
    ref = np.asarray(ref, dtype=np.float64)
    den = np.max(np.abs(ref)) if ref.size else 0.0
    if den == 0.0:
        return float(np.max(np.abs(got))) if got.size else 0.0
    return float(np.max(np.abs(got - ref)) / den)


def dev_bytes(ptr_value, nbytes, device):
    """Copy nbytes at a raw device address into a numpy uint8 array."""
    out = torch.empty(nbytes, dtype=torch.uint8, device=device)
    if nbytes:
        import ctypes
        import os
        torch.cuda.synchronize()
        # the HIP runtime torch itself loaded (one runtime per process)
        hip = ctypes.CDLL(os.path.join(os.path.dirname(torch.__file__), "lib", "libamdhip64.so"))
        hip.hipMemcpy.argtypes = [ctypes.c_void_p, ctypes.c_void_p, ctypes.c_size_t, ctypes.c_int]
        rc = hip.hipMemcpy(ctypes.c_void_p(out.data_ptr()), ctypes.c_void_p(ptr_value), ctypes.c_size_t(nbytes), 3)
        assert rc == 0, rc
    return out.cpu().numpy()


def dev_f32(ptr_value, n, device):
    return dev_bytes(ptr_value, 4 * n, device).view(np.float32)
