"""Helpers shared by the GPU parity tests (tests only)."""
import numpy as np
import torch

ATOL, RTOL = 2e-3, 1e-2   # float parity bound: |gpu - ref| <= ATOL + RTOL |ref|


def dev_bf16(bits: np.ndarray) -> torch.Tensor:
    """uint16 bf16 bit patterns -> contiguous bf16 device tensor."""
    t = torch.from_numpy(np.ascontiguousarray(bits).view(np.int16)).to("cuda")
    return t.view(torch.bfloat16)


def host_bits(t: torch.Tensor) -> np.ndarray:
    return t.contiguous().view(torch.int16).cpu().numpy().view(np.uint16)


def image(cache) -> np.ndarray:
    torch.cuda.synchronize()
    return cache.storage.cpu().numpy()


def assert_close(gpu, ref, what="", atol=ATOL, rtol=RTOL):
    gpu = np.asarray(gpu, dtype=np.float64)
    ref = np.asarray(ref, dtype=np.float64)
    assert gpu.shape == ref.shape, (gpu.shape, ref.shape)
    err = np.abs(gpu - ref)
    bound = atol + rtol * np.abs(ref)
    bad = err > bound
    if bad.any():
        i = np.unravel_index(np.argmax(err - bound), err.shape)
        raise AssertionError(f"{what}: {bad.sum()} of {err.size} outside atol {atol} + rtol {rtol}; "
                             f"worst at {i}: gpu {gpu[i]!r} ref {ref[i]!r}; max abs err {err.max():.3e}")
    return float(err.max())

