"""Device placement of the seeded inputs (torch is used for memory only)."""
from __future__ import annotations

from typing import Dict, List, Sequence

import numpy as np

from .workload import MATRIX_NAMES

HEAD_MATRIX_NAMES = ("z_w", "t1_w", "t2_w", "in_w", "ada_w", "fc1_w", "fc2_w", "out_w")


def torch_dtype(dtype: str):
    import torch
    return {"f32": torch.float32, "bf16": torch.bfloat16}[dtype]


def to_device(a: np.ndarray, dtype: str, device="cuda"):
    """float32 host values (already exact in `dtype`) -> device tensor."""
    import torch
    t = torch.from_numpy(np.ascontiguousarray(a, dtype=np.float32))
    return t.to(device=device).to(torch_dtype(dtype)).contiguous()


def upload_blocks(blocks: Sequence[Dict[str, np.ndarray]], dtype: str, device="cuda") -> List[Dict[str, object]]:
    """Matrices in the storage dtype, LayerNorm parameters and biases fp32."""
    out = []
    for blk in blocks:
        out.append({k: to_device(v, dtype if k in MATRIX_NAMES else "f32", device) for k, v in blk.items()})
    return out


def upload_head(weights: Dict[str, np.ndarray], dtype: str, device="cuda") -> Dict[str, object]:
    """The diffusion head's matrices in the storage dtype, biases fp32."""
    return {k: to_device(v, dtype if k in HEAD_MATRIX_NAMES else "f32", device) for k, v in weights.items()}
