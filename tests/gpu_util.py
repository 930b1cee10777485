"""Helpers shared by the GPU tests: move seeded inputs to the device, compare."""
import numpy as np
import torch

DEV = torch.device("cuda:0")


def to_dev(a, dtype: str):
    """numpy array of the workload module (bf16 bit patterns or float32) -> device tensor."""
    t = torch.from_numpy(np.ascontiguousarray(a))
    if dtype == "bf16":
        t = t.view(torch.bfloat16)
    return t.to(DEV)


def idx_dev(idx):
    return torch.from_numpy(np.ascontiguousarray(idx, dtype=np.int32)).to(DEV)


def rel(got, ref) -> float:
    got = np.asarray(got, dtype=np.float64)
    ref = np.asarray(ref, dtype=np.float64)
    return float(np.linalg.norm(got - ref) / max(np.linalg.norm(ref), 1e-300))


def host(t) -> np.ndarray:
    torch.cuda.synchronize()
    return t.detach().double().cpu().numpy()
