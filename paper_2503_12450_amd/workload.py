"""Seeded synthetic inputs for the cached MAR transformer step.

This module only draws numbers and lays them out; it holds none of the
method's arithmetic (no LayerNorm, attention, similarity, selection or
guidance).  The GPU path, the CPU oracle and the benchmark all take their
inputs from here, so both sides of every parity check consume identical
arrays.

Input recipe (stands in for the ImageNet 256x256 / KL-16 / MAR workloads of
the paper's Sec. 4.1, whose data and trained weights are not available):

* Weights: every matrix ~ N(0, 0.02); biases ~ N(0, 0.02); LayerNorm gain
  1 + N(0, 0.02) and shift N(0, 0.02).  Matrices are rounded to bfloat16 for
  the bf16 configurations (biases and LayerNorm parameters stay fp32).
* Sequence: 64 buffer/class rows followed by the image-token rows (256 for
  a 16x16 latent grid, 1024 for 32x32), as in Sec. 4.1.
* Condition tokens (Eq. 6): the conditional pathway carries a class vector
  c_b ~ N(0, 1) on the 64 buffer rows, the unconditional one carries zeros.
* Image rows: a shared mask vector m ~ N(0, 1) until the token is decoded,
  then P_z z_i with z_i ~ N(0, 1) in R^16 and P_z ~ N(0, 1/16); every row
  also gets a positional vector ~ N(0, 0.02).
* Decode order: a seeded permutation per image; the number of tokens still
  masked before step k of K is floor(T cos(pi/2 k/K)) (the MaskGIT/MAR
  cosine schedule; it only decides which rows change between steps).

Seeds: 0 weights, 1 inputs, 2 cache-fill noise, 3 decode order.  Every draw
uses numpy's counter-based Philox generator.
"""
from __future__ import annotations

import dataclasses
import math
from typing import Dict, List, Optional

import numpy as np

SEED_WEIGHTS = 0
SEED_INPUTS = 1
SEED_NOISE = 2
SEED_ORDER = 3

BUFFER_ROWS = 64
LATENT_DIM = 16

DTYPES = ("f32", "bf16")


@dataclasses.dataclass(frozen=True)
class MarDims:
    """Shape of one stack of identical bidirectional pre-LN blocks."""

    n_layers: int
    d_model: int
    n_heads: int
    d_mlp: int
    seq_len: int
    max_slots: int
    full_prefix: int  # P: blocks always computed on every row (paper: 3)
    dtype: str = "bf16"
    ln_eps: float = 1e-6
    # method options (Sec. 4.4 alternatives): what the similarity compares
    # ("values": the paper's choice, or "features"), and whether the
    # keys/values of the rows not computed are recomputed at block P
    score_source: str = "values"
    fresh_kv: bool = False

    @property
    def d_head(self) -> int:
        return self.d_model // self.n_heads


@dataclasses.dataclass(frozen=True)
class Workload:
    name: str
    dims: MarDims
    n_recompute: int
    images: int


def _n_round(ratio: float, seq: int) -> int:
    return int(math.floor(ratio * seq + 0.5))


# The five workloads: a single fp32 block, then MAR-B, -L, -H shaped stacks
# (Sec. 4.1 names the models; the widths/depths are the public MAR ones) and
# a high-resolution MAR-L.  Each pathway of classifier-free guidance is one
# sequence slot: slots [0, B) carry the condition, [B, 2B) the fake one.
WORKLOADS: Dict[str, Workload] = {
    "block-f32": Workload(
        "single pre-LN block, width 768, 12 heads, seq 320, 1x2 CFG, fp32",
        MarDims(1, 768, 12, 3072, 320, 2, 0, "f32"), _n_round(0.25, 320), 1),
    "mar-b": Workload(
        "MAR-B-shaped 12+12 blocks, width 768, 12 heads, seq 320, 32x2 CFG, bf16",
        MarDims(24, 768, 12, 3072, 320, 64, 3, "bf16"), _n_round(0.30, 320), 32),
    "mar-l": Workload(
        "MAR-L-shaped 16+16 blocks, width 1024, 16 heads, seq 320, 64x2 CFG, bf16",
        MarDims(32, 1024, 16, 4096, 320, 128, 3, "bf16"), 50, 64),
    "mar-h": Workload(
        "MAR-H-shaped 20+20 blocks, width 1280, 16 heads, seq 320, 128x2 CFG, bf16",
        MarDims(40, 1280, 16, 5120, 320, 256, 3, "bf16"), _n_round(0.10, 320), 128),
    "mar-l-hires": Workload(
        "MAR-L-shaped 16+16 blocks, width 1024, 16 heads, seq 1088 (64+32x32), 32x2 CFG, bf16",
        MarDims(32, 1024, 16, 4096, 1088, 64, 3, "bf16"), _n_round(0.20, 1088), 32),
}

MAR_H_SWEEP = tuple(_n_round(r, 320) for r in (0.10, 0.20, 0.30, 0.50))


def _gen(seed: int, stream: int = 0) -> np.random.Generator:
    bitgen = np.random.Philox(seed)
    if stream:
        bitgen = bitgen.jumped(stream)
    return np.random.Generator(bitgen)


def round_to_bf16(a: np.ndarray) -> np.ndarray:
    """Round float32 values to the nearest bfloat16 (ties to even).

    Returns float32 values that are exactly representable in bfloat16.
    NaN stays NaN; this is a storage conversion, nothing more.
    """
    a = np.ascontiguousarray(a, dtype=np.float32)
    u = a.view(np.uint32)
    # no finite value or infinity carries out of 32 bits here
    rounded = (u + np.uint32(0x7FFF) + ((u >> np.uint32(16)) & np.uint32(1))) & np.uint32(0xFFFF0000)
    out = rounded.view(np.float32)
    nan = np.isnan(a)
    if nan.any():
        out = out.copy()
        out[nan] = np.nan
    return out.reshape(a.shape)


def bf16_bits(a: np.ndarray) -> np.ndarray:
    """The upper 16 bits of float32 values already rounded to bfloat16."""
    a = np.ascontiguousarray(a, dtype=np.float32)
    return (a.view(np.uint32) >> 16).astype(np.uint16)


def bf16_from_bits(bits: np.ndarray) -> np.ndarray:
    return (np.asarray(bits, dtype=np.uint16).astype(np.uint32) << 16).view(np.float32)


def to_storage(a: np.ndarray, dtype: str) -> np.ndarray:
    """float32 copy of ``a`` holding exactly the values stored in ``dtype``."""
    if dtype == "bf16":
        return round_to_bf16(a)
    if dtype == "f32":
        return np.ascontiguousarray(a, dtype=np.float32)
    raise ValueError(f"unknown dtype {dtype!r}")


WEIGHT_NAMES = ("ln1_w", "ln1_b", "qkv_w", "qkv_b", "proj_w", "proj_b",
                "ln2_w", "ln2_b", "fc1_w", "fc1_b", "fc2_w", "fc2_b")
MATRIX_NAMES = ("qkv_w", "proj_w", "fc1_w", "fc2_w")


def block_weights(dims: MarDims, layer: int, seed: int = SEED_WEIGHTS,
                  std: float = 0.02) -> Dict[str, np.ndarray]:
    """Weights of one block, nn.Linear layout ([out, in], row-major).

    qkv_w stacks the query, key and value projections ([3D, D]); each layer
    draws from its own Philox stream so one layer can be made on its own.
    """
    D, F = dims.d_model, dims.d_mlp
    g = _gen(seed, 1 + layer)

    def n(*shape):
        return (g.standard_normal(shape, dtype=np.float32) * np.float32(std)).astype(np.float32)

    w = {
        "ln1_w": 1.0 + n(D), "ln1_b": n(D),
        "qkv_w": n(3 * D, D), "qkv_b": n(3 * D),
        "proj_w": n(D, D), "proj_b": n(D),
        "ln2_w": 1.0 + n(D), "ln2_b": n(D),
        "fc1_w": n(F, D), "fc1_b": n(F),
        "fc2_w": n(D, F), "fc2_b": n(D),
    }
    w = {k: np.ascontiguousarray(v, dtype=np.float32) for k, v in w.items()}
    for k in MATRIX_NAMES:
        w[k] = to_storage(w[k], dims.dtype)
    return w


def all_block_weights(dims: MarDims, seed: int = SEED_WEIGHTS) -> List[Dict[str, np.ndarray]]:
    return [block_weights(dims, l, seed) for l in range(dims.n_layers)]


def normal_rows(shape, seed: int, stream: int = 0, std: float = 1.0,
                dtype: str = "f32") -> np.ndarray:
    g = _gen(seed, stream)
    a = g.standard_normal(shape, dtype=np.float32) * np.float32(std)
    return to_storage(a, dtype)


def perturbed(a: np.ndarray, seed: int, std: float, dtype: str, stream: int = 0,
              rows: Optional[np.ndarray] = None) -> np.ndarray:
    """``a`` plus N(0, std^2) noise (on every row, or on the given rows of
    the second-to-last axis only), stored in ``dtype``."""
    g = _gen(seed, stream)
    noise = g.standard_normal(a.shape, dtype=np.float32) * np.float32(std)
    if rows is not None:
        keep = np.zeros(a.shape[-2], dtype=bool)
        keep[np.asarray(rows)] = True
        noise[..., ~keep, :] = 0.0
    return to_storage(a.astype(np.float32) + noise, dtype)


def random_index_sets(n_slots: int, seq: int, n: int, seed: int, stream: int = 0) -> np.ndarray:
    """n distinct token indices per slot, ascending, int32 [n_slots, n]."""
    g = _gen(seed, stream)
    out = np.empty((n_slots, n), dtype=np.int32)
    for b in range(n_slots):
        out[b] = np.sort(g.permutation(seq)[:n])
    return out


def changed_rows(base: np.ndarray, n: int, seed: int):
    """A copy of ``base`` [slots, S, D] in which n random rows per slot (the
    rows of random_index_sets(seed)) get N(0, 1) noise added (normal_rows,
    seed + 1); not yet rounded to a storage type.  Returns (copy, rows).
    A cached step on such an input has a well separated selection: the
    changed rows are far less similar than every other row."""
    rows = random_index_sets(base.shape[0], base.shape[1], n, seed=seed)
    noise = normal_rows(base.shape, seed=seed + 1)
    out = base.copy()
    for b in range(base.shape[0]):
        out[b, rows[b]] = base[b, rows[b]] + noise[b, rows[b]]
    return out, rows


# Full-size parity plan: workload -> recompute counts of the successive
# cached steps after one full step (each step's input from changed_rows with
# seed 100 + 10 k; then, for two-pathway workloads, one conditional-only
# step at the last count with seed 900)
FULLSIZE_PLANS = {
    "block-f32": (WORKLOADS["block-f32"].n_recompute,),
    "mar-b": (WORKLOADS["mar-b"].n_recompute,),
    # N = 50 (the 64-step setting), then N = 70 (the 32-step setting: about
    # 250 of 320 tokens skipped)
    "mar-l": (WORKLOADS["mar-l"].n_recompute, 70),
    "mar-h": MAR_H_SWEEP,
    "mar-l-hires": (WORKLOADS["mar-l-hires"].n_recompute,),
}
FULLSIZE_STEP_SEED = 100
FULLSIZE_COND_SEED = 900


# ---------------------------------------------------------------------------
# Masked-generation decode schedule inputs (Eq. 6 layout, cosine mask schedule)
# ---------------------------------------------------------------------------

def masked_counts(n_tokens: int, n_steps: int) -> np.ndarray:
    """Tokens still masked before each step k = 0..n_steps (last entry 0).

    floor(T cos(pi/2 k/K)) with at least one token decoded per step.
    """
    if n_tokens < n_steps:
        raise ValueError("need at least one token per decoding step")
    c = [n_tokens]
    for k in range(1, n_steps):
        m = int(math.floor(n_tokens * math.cos(math.pi / 2 * k / n_steps)))
        m = min(m, c[-1] - 1)       # decode at least one token this step
        m = max(m, n_steps - k)     # and leave one for every later step
        c.append(m)
    c.append(0)
    return np.asarray(c, dtype=np.int64)


@dataclasses.dataclass
class DecodeRecipe:
    """Small seeded factors from which every step's input is assembled."""

    dims: MarDims
    images: int
    n_steps: int
    cls: np.ndarray        # [images, D]   class vector of each image
    mask_vec: np.ndarray   # [D]           shared mask-token vector
    z: np.ndarray          # [images, T, 16] latent of each image token
    proj: np.ndarray       # [16, D]       latent-to-width projection
    pos: np.ndarray        # [S, D]        positional vectors
    order: np.ndarray      # [images, T]   decode order (token ids)
    counts: np.ndarray     # [n_steps + 1] tokens still masked before step k

    @property
    def image_tokens(self) -> int:
        return self.dims.seq_len - BUFFER_ROWS


def decode_recipe(dims: MarDims, images: int, n_steps: int = 64,
                  seed: int = SEED_INPUTS, order_seed: int = SEED_ORDER) -> DecodeRecipe:
    D, S = dims.d_model, dims.seq_len
    T = S - BUFFER_ROWS
    if T <= 0:
        raise ValueError("sequence must hold more than the 64 buffer rows")
    g = _gen(seed, 100)
    cls = g.standard_normal((images, D), dtype=np.float32)
    mask_vec = g.standard_normal(D, dtype=np.float32)
    z = g.standard_normal((images, T, LATENT_DIM), dtype=np.float32)
    proj = g.standard_normal((LATENT_DIM, D), dtype=np.float32) * np.float32(1.0 / 4.0)
    pos = g.standard_normal((S, D), dtype=np.float32) * np.float32(0.02)
    go = _gen(order_seed, 100)
    order = np.stack([go.permutation(T) for _ in range(images)]).astype(np.int64)
    return DecodeRecipe(dims, images, n_steps, cls, mask_vec, z, proj, pos, order,
                        masked_counts(T, n_steps))


def decoded_mask(recipe: DecodeRecipe, step: int) -> np.ndarray:
    """bool [images, T]: token already decoded before ``step``."""
    T = recipe.image_tokens
    n_dec = T - int(recipe.counts[step])
    mask = np.zeros((recipe.images, T), dtype=bool)
    rows = np.arange(recipe.images)[:, None]
    mask[rows, recipe.order[:, :n_dec]] = True
    return mask


def step_input(recipe: DecodeRecipe, step: int) -> np.ndarray:
    """x for decoding step ``step``: float32 [2*images, S, D] in storage
    precision; rows [0, B) are the conditional pathway, [B, 2B) the
    unconditional one (fake condition tokens are zero, Eq. 6)."""
    B, D = recipe.images, recipe.dims.d_model
    T = recipe.image_tokens
    dec = decoded_mask(recipe, step)
    img = np.where(dec[:, :, None], recipe.z @ recipe.proj, recipe.mask_vec[None, None, :])
    x = np.empty((2 * B, recipe.dims.seq_len, D), dtype=np.float32)
    x[:B, :BUFFER_ROWS] = recipe.cls[:, None, :]
    x[B:, :BUFFER_ROWS] = 0.0
    x[:B, BUFFER_ROWS:] = img
    x[B:, BUFFER_ROWS:] = img
    x += recipe.pos[None]
    del T
    return to_storage(x, recipe.dims.dtype)


def step_inputs_device(recipe: DecodeRecipe, steps, device="cuda"):
    """step_input() for several steps, assembled on the device with torch
    (same recipe; fp32 arithmetic, then the storage dtype).  Returns a list
    of [2B, S, D] tensors."""
    import torch

    dims = recipe.dims
    B, S, D = recipe.images, dims.seq_len, dims.d_model
    T = recipe.image_tokens
    tdt = {"f32": torch.float32, "bf16": torch.bfloat16}[dims.dtype]
    dev = lambda a: torch.from_numpy(np.ascontiguousarray(a)).to(device)  # noqa: E731
    zp = dev(recipe.z) @ dev(recipe.proj)                 # [B, T, D]
    mask_vec = dev(recipe.mask_vec)
    pos = dev(recipe.pos)
    cls = dev(recipe.cls)
    rank = torch.empty((B, T), dtype=torch.int64, device=device)
    order = dev(recipe.order)
    rank.scatter_(1, order, torch.arange(T, device=device).expand(B, T).contiguous())
    out = []
    for k in steps:
        n_dec = T - int(recipe.counts[k])
        dec = (rank < n_dec)[:, :, None]
        img = torch.where(dec, zp, mask_vec[None, None, :])
        x = torch.empty((2 * B, S, D), dtype=torch.float32, device=device)
        x[:B, :BUFFER_ROWS] = cls[:, None, :]
        x[B:, :BUFFER_ROWS] = 0.0
        x[:B, BUFFER_ROWS:] = img
        x[B:, BUFFER_ROWS:] = img
        x += pos[None]
        out.append(x.to(tdt).contiguous())
        del x, img, dec
    return out


# ---------------------------------------------------------------------------
# Per-token diffusion head (the denoiser MAR samples each token's latent with)
# ---------------------------------------------------------------------------

@dataclasses.dataclass(frozen=True)
class HeadDims:
    """Shape of the per-token diffusion head: a residual MLP of `depth`
    blocks and width `width`, conditioned by adaptive LayerNorm on the
    transformer's output row (cond_dim) and the diffusion time; it predicts
    the noise of a `token_dim`-dimensional latent.  `steps` sampling steps
    respace a `train_steps`-step linear noise schedule."""

    width: int
    depth: int
    cond_dim: int
    token_dim: int = LATENT_DIM
    steps: int = 100
    train_steps: int = 1000
    beta_start: float = 1e-4
    beta_end: float = 0.02
    freq_dim: int = 256
    max_rows: int = 4096
    dtype: str = "bf16"
    ln_eps: float = 1e-6

    @property
    def n_mod(self) -> int:
        """Modulation vectors per row: shift, scale, gate per block, and the
        final shift and scale."""
        return 3 * self.depth + 2


# Head sizes per model: chosen so that the head's FLOPs over one image (256
# tokens x 2 guidance pathways x 100 steps) reproduce the step-count
# independent constant of Table 1's baseline FLOPs within a few percent
# (checked in the tests).
HEADS = {
    "mar-b": HeadDims(width=1024, depth=6, cond_dim=768),
    "mar-l": HeadDims(width=1280, depth=8, cond_dim=1024),
    "mar-h": HeadDims(width=1536, depth=12, cond_dim=1280),
}

HEAD_WEIGHT_NAMES = ("z_w", "z_b", "t1_w", "t1_b", "t2_w", "t2_b", "in_w", "in_b", "ada_w", "ada_b",
                     "fc1_w", "fc1_b", "fc2_w", "fc2_b", "out_w", "out_b")


def head_weights(hd: HeadDims, seed: int = SEED_WEIGHTS, std: float = 0.02) -> Dict[str, np.ndarray]:
    """Random weights of the head, nn.Linear layout ([out, in]).  Per-block
    matrices are stacked on a leading axis: fc1_w, fc2_w [depth, w, w],
    fc1_b, fc2_b [depth, w]; ada_w [n_mod * w, w] holds the modulation
    products of every block and the final layer, block k's shift, scale and
    gate at rows (3k, 3k+1, 3k+2) * w, the final shift and scale last.
    Matrices are rounded to the storage type; biases stay fp32.  The input
    and output products (token_dim wide) use a larger scale so that the
    noise prediction is O(1)."""
    w, D, T = hd.width, hd.cond_dim, hd.token_dim
    g = _gen(seed, 1000)

    def n(*shape, s=std):
        return (g.standard_normal(shape, dtype=np.float32) * np.float32(s)).astype(np.float32)

    out = {
        "z_w": n(w, D), "z_b": n(w),
        "t1_w": n(w, hd.freq_dim, s=0.1), "t1_b": n(w),
        "t2_w": n(w, w), "t2_b": n(w),
        "in_w": n(w, T, s=0.25), "in_b": n(w),
        "ada_w": n(hd.n_mod * w, w), "ada_b": n(hd.n_mod * w),
        "fc1_w": n(hd.depth, w, w), "fc1_b": n(hd.depth, w),
        "fc2_w": n(hd.depth, w, w), "fc2_b": n(hd.depth, w),
        "out_w": n(T, w, s=1.0 / math.sqrt(w)), "out_b": n(T),
    }
    out = {k: np.ascontiguousarray(v, dtype=np.float32) for k, v in out.items()}
    for k in ("z_w", "t1_w", "t2_w", "in_w", "ada_w", "fc1_w", "fc2_w", "out_w"):
        out[k] = to_storage(out[k], hd.dtype)
    return out


def decoded_at(recipe: "DecodeRecipe", step: int) -> np.ndarray:
    """int64 [images, n]: the image tokens decoded at decoding step ``step``
    (the order's entries between the counts before and after it), the same
    number for every image."""
    T = recipe.image_tokens
    lo, hi = T - int(recipe.counts[step]), T - int(recipe.counts[step + 1])
    return np.sort(recipe.order[:, lo:hi], axis=1)
