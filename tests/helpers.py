"""Test plumbing: move generated tensors into the oracle's terms and compare outputs."""
from __future__ import annotations

import numpy as np
import torch

from oracle import kvc_oracle as O


def to_np_storage(t: torch.Tensor) -> np.ndarray:
    """float32 tensors -> float32 arrays, bfloat16 tensors -> uint16 bit patterns (exact bytes)."""
    t = t.detach().to("cpu").contiguous()
    if t.dtype == torch.bfloat16:
        return t.view(torch.int16).numpy().view(np.uint16).copy()
    return t.numpy().copy()


def storage_name(t: torch.dtype) -> str:
    return "bf16" if t == torch.bfloat16 else "f32"


def oracle_cache(k_pools, v_pools, block_size: int, rope: "O.Rope | None" = None) -> O.Cache:
    dt = storage_name(k_pools[0].dtype)
    return O.Cache(dt, block_size, [to_np_storage(p) for p in k_pools], [to_np_storage(p) for p in v_pools], rope)


ROPE_STYLE_NAME = {1: "half", 2: "pairs"}


def rope_inv_freq(d: int, theta: float) -> np.ndarray:
    """Inverse frequencies theta^(-2i/d) of the standard rotary encoding (float64)."""
    return theta ** (-np.arange(0, d, 2, dtype=np.float64) / d)


def oracle_state(coef: torch.Tensor, basis: torch.Tensor, sigma=None) -> O.State:
    return O.State(to_np_storage(coef), to_np_storage(basis), None if sigma is None else to_np_storage(sigma),
                   storage_name(coef.dtype))


def table_np(tables, i):
    return None if tables is None else tables[i].to("cpu").numpy().astype(np.int64)


def rows_f64(stored: np.ndarray, dtype: str) -> np.ndarray:
    return O.to_f64(stored, dtype)


def max_rel_err_per_slice(got: np.ndarray, ref: np.ndarray, dtype: str) -> float:
    """max over slices of max|g - o| / max|o| (a slice = all rows of one unit)."""
    return O.max_relative_error(rows_f64(got, dtype), rows_f64(ref, dtype))
