"""Helpers shared by the GPU parity tests: moving seeded storage arrays to the
device and back, and the relative-error measure used against the oracle."""
import numpy as np
import torch

from paper_2307_04339_amd import synth

TORCH = {"f32": torch.float32, "f16": torch.float16, "bf16": torch.bfloat16}
RTOL = {"f32": 1e-4, "f16": 1e-2, "bf16": 1e-2}


def gpu_available():
    try:
        return torch.cuda.is_available()
    except Exception:
        return False


def to_dev(storage: np.ndarray, dtype: str) -> torch.Tensor:
    """Device tensor holding exactly the given storage bits."""
    if dtype == "bf16":
        t = torch.from_numpy(np.ascontiguousarray(storage).view(np.int16)).view(torch.bfloat16)
    else:
        t = torch.from_numpy(np.ascontiguousarray(storage))
    return t.cuda()


def rand(shape, dtype, seed, lo=-1.0, hi=1.0):
    """(device tensor, exact float64 copy) of a seeded U[lo, hi) tensor."""
    s, f = synth.storage_tensor(shape, dtype, seed, lo, hi)
    return to_dev(s, dtype), f


def ints(shape, dtype, seed, lo, hi):
    f = synth.integers(shape, lo, hi, seed)
    return to_dev(synth.to_storage(f, dtype), dtype), f


def f32_dev(a64):
    return torch.from_numpy(np.ascontiguousarray(a64, dtype=np.float32)).cuda()


def to_f64(t: torch.Tensor) -> np.ndarray:
    return t.detach().float().cpu().numpy().astype(np.float64)


def empty(shape, dtype):
    return torch.full(shape, float("nan"), dtype=TORCH[dtype], device="cuda")


def rel_err(g: np.ndarray, o: np.ndarray) -> float:
    """max_i |g_i - o_i| / max(|o_i|, rms(o)); rms over the whole tensor (1 if it is 0)."""
    g = np.asarray(g, dtype=np.float64).ravel()
    o = np.asarray(o, dtype=np.float64).ravel()
    rms = float(np.sqrt(np.mean(o * o))) if o.size else 1.0
    if rms == 0.0:
        rms = 1.0
    den = np.maximum(np.abs(o), rms)
    if not np.all(np.isfinite(g)):
        return float("inf")
    return float(np.max(np.abs(g - o) / den)) if o.size else 0.0


def bits(t: torch.Tensor) -> bytes:
    return t.detach().cpu().contiguous().view(torch.uint8).numpy().tobytes()
