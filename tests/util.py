"""Helpers shared by the tests: error metrics and host/device conversion."""
import numpy as np
import torch

# Tolerances, stated as the maximum over rows of ||gpu_row - ref_row||_2 / ||ref_row||_2
# (activations) and the Frobenius ratio ||gpu - ref||_F / ||ref||_F (weight gradients).
TOL = {"f32": 1e-5, "bf16": 2e-2}


def row_rel_err(got, ref) -> float:
    got = np.asarray(got, dtype=np.float64)
    ref = np.asarray(ref, dtype=np.float64)
    w = ref.shape[-1]
    g, r = got.reshape(-1, w), ref.reshape(-1, w)
    num = np.linalg.norm(g - r, axis=1)
    den = np.maximum(np.linalg.norm(r, axis=1), 1e-30)
    return float((num / den).max())


def fro_rel_err(got, ref) -> float:
    got = np.asarray(got, dtype=np.float64)
    ref = np.asarray(ref, dtype=np.float64)
    return float(np.linalg.norm(got - ref) / max(np.linalg.norm(ref), 1e-30))


def torch_dtype(name: str):
    return {"bf16": torch.bfloat16, "f32": torch.float32}[name]


def to_dev(a: np.ndarray, dtype: str, device="cuda") -> torch.Tensor:
    """Host float32 array (already exactly representable in `dtype`) -> device tensor."""
    t = torch.from_numpy(np.ascontiguousarray(a, dtype=np.float32))
    t = t.to(torch_dtype(dtype))
    # exactness: converting back must give the same numbers
    assert np.array_equal(t.to(torch.float32).numpy(), np.asarray(a, dtype=np.float32))
    return t.to(device)


def to_host(t: torch.Tensor) -> np.ndarray:
    return t.detach().to(torch.float32).cpu().numpy().astype(np.float64)
