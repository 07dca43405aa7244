"""Helpers for the GPU parity tests: move seeded storage arrays to the GPU
and compare with the oracle."""
import numpy as np
import torch

from oracle.stmoe_oracle import decode_storage
from paper_2606_15453_amd import workload as W

DEV = "cuda:0"


def to_dev(a: np.ndarray) -> torch.Tensor:
    """Storage array (uint16 bf16 bits or float32) -> device tensor (bfloat16 or float32)."""
    a = np.ascontiguousarray(a)
    if a.dtype == np.uint16:
        return torch.from_numpy(a.view(np.int16)).to(DEV).view(torch.bfloat16)
    return torch.from_numpy(a.astype(np.float32)).to(DEV)


def i32(a) -> torch.Tensor:
    return torch.from_numpy(np.ascontiguousarray(a, dtype=np.int32)).to(DEV)


def rel_l2(got, ref) -> float:
    """Largest relative L2 error over the output rows (the last axis is the
    hidden dimension; every batch row must meet the bound on its own)."""
    got = np.asarray(got, np.float64)
    ref = np.asarray(ref, np.float64)
    H = ref.shape[-1]
    g, r = got.reshape(-1, H), ref.reshape(-1, H)
    err = np.linalg.norm(g - r, axis=1) / np.maximum(np.linalg.norm(r, axis=1), 1e-300)
    return float(err.max())


def storage_dtype(cfg):
    return 1 if cfg.dtype == "bf16" else 0


def blob_dev(cfg, l, e, shared=False) -> torch.Tensor:
    dt = torch.bfloat16 if cfg.dtype == "bf16" else torch.float32
    out = torch.empty(cfg.blob_elems, dtype=dt, device=DEV)
    W.expert_blob_torch(cfg, l, e, out, shared=shared)
    return out


def expert_f64(cfg, l, e, shared=False):
    return tuple(decode_storage(m) for m in W.expert_matrices(cfg, l, e, shared))


def ptr_array(ptrs) -> torch.Tensor:
    return torch.tensor([int(p) for p in ptrs], dtype=torch.int64, device=DEV)
