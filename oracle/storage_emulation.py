"""The oracle's cached step with the path's storage rounding applied.

TEST INFRASTRUCTURE ONLY, like the rest of this package: the product path
never imports it, and it imports nothing from the product.

Why it exists.  A pipeline that stores its matrix-product operands in
bfloat16 cannot meet an elementwise bar of 2e-2 + 1e-2 |y| against the fp64
oracle at every element of a 24-40 block stack: the rounding of those
operands alone moves some outputs further than that, and the deviation grows
with depth.  This module measures how far: it runs the oracle's own steps
(the same functions, in the same order, Sec. 3.2 / Eq. 3, 8, 9) in fp64, but
rounds every tensor at the points where the GPU path stores it:

* in the storage type (bfloat16 for the bf16 stacks): the LayerNorm outputs
  that feed the QKV product and fc1, the queries, keys and values, the
  attention output that feeds the output projection, the GELU output that
  feeds fc2;
* inside attention, the softmax probabilities that multiply the values are
  rounded to the storage type; their row sum is not;
* in fp32: the residual stream after each residual product, and the bias
  sum of each product that adds into it.

Products and sums are otherwise exact-in-fp64, so the figures this yields
are the error of the storage rounding alone, without any accumulation-order
or approximation error of a real kernel.  The GPU tests bound the path's
deviation from the oracle by a small multiple of these figures (stored in
tests/golden/ by the script that sits there).

For fp32 stacks only the fp32 roundings apply.
"""
from __future__ import annotations

import math
from typing import Dict

import numpy as np

from .mar_oracle import MarOracle, _split_qkv, gelu, layer_norm, linear, storage_round

__all__ = ["attention_stored", "block_rows_stored", "StorageEmulation"]


def attention_stored(q, k, v, dtype: str) -> np.ndarray:
    """Eq. (3) for one head with the probabilities that weight the values
    rounded to ``dtype`` (bf16 only; fp32 keeps them) and the normaliser
    summed from the unrounded ones."""
    q, k, v = (np.asarray(a, dtype=np.float64) for a in (q, k, v))
    logits = q @ k.T / math.sqrt(q.shape[-1])
    p = np.exp(logits - logits.max(axis=-1, keepdims=True))
    pw = storage_round(p, dtype) if dtype == "bf16" else p
    return (pw @ v) / p.sum(axis=-1, keepdims=True)


def block_rows_stored(m, rows, p: Dict[str, np.ndarray], n_heads: int, eps: float, dtype: str):
    """The oracle's block_rows with the stored tensors rounded (see the
    module docstring).  m holds the block input as stored (the fp32
    residual stream, or the step input in its storage type)."""
    m = np.asarray(m, dtype=np.float64)
    rows = np.asarray(rows, dtype=np.int64)
    S, D = m.shape
    dh = D // n_heads

    def st(a):  # the storage type
        return storage_round(a, dtype)

    def f32(a):
        return storage_round(a, "f32")

    (wq, bq), (wk, bk), (wv, bv) = _split_qkv(p, D)
    a = st(layer_norm(m, p["ln1_w"], p["ln1_b"], eps))
    q = st(linear(a[rows], wq, bq))
    k = st(linear(a, wk, bk))
    v = st(linear(a, wv, bv))
    o = np.empty((len(rows), D), dtype=np.float64)
    for h in range(n_heads):
        cols = slice(h * dh, (h + 1) * dh)
        o[:, cols] = attention_stored(q[:, cols], k[:, cols], v[:, cols], dtype)
    o = st(o)
    h1 = f32(m[rows] + f32(linear(o, p["proj_w"], p["proj_b"])))
    a2 = st(layer_norm(h1, p["ln2_w"], p["ln2_b"], eps))
    f = st(gelu(linear(a2, p["fc1_w"], p["fc1_b"])))
    out = f32(h1 + f32(linear(f, p["fc2_w"], p["fc2_b"])))
    return out, v


class StorageEmulation(MarOracle):
    """MarOracle whose blocks round at the path's storage points.  State,
    selection, scoring and the feature cache are the oracle's own."""

    def _block(self, m, rows, l: int):
        return block_rows_stored(m, rows, self.blocks[l], self.H, self.eps, self.dtype)

    def _values(self, x) -> np.ndarray:
        (_, _), (_, _), (wv, bv) = _split_qkv(self.blocks[0], self.D)
        a = storage_round(layer_norm(x, self.blocks[0]["ln1_w"], self.blocks[0]["ln1_b"], self.eps),
                          self.dtype)
        return linear(a, wv, bv)
