"""Algorithmic work of the step (2 FLOPs per multiply-add; products and the
two attention contractions counted, LayerNorm / softmax / GELU not)."""
from __future__ import annotations


def gemm_flops_per_row(D: int, F: int) -> int:
    """QKV (3D x D), output projection (D x D), MLP (F x D and D x F)."""
    return 2 * (4 * D * D + 2 * F * D)


def block_flops(rows: int, D: int, F: int, queries: int, keys: int, seqs: int) -> int:
    """One block on `rows` rows; attention of `queries` rows per sequence
    against `keys` keys for `seqs` sequences (QK^T and PV)."""
    return rows * gemm_flops_per_row(D, F) + 4 * seqs * queries * keys * D


def step_flops(dims, n_slots: int, mode: str, n: int = 0) -> int:
    D, F, S, L, P = dims.d_model, dims.d_mlp, dims.seq_len, dims.n_layers, dims.full_prefix
    dense = block_flops(n_slots * S, D, F, S, S, n_slots)
    if mode == "full":
        return L * dense
    cached = block_flops(n_slots * n, D, F, n, S, n_slots)
    extra = 2 * n_slots * S * D * D if P == 0 else 0   # value rows of block 0 for scoring
    return P * dense + (L - P) * cached + extra


def gemm_launch_flops(M: int, N: int, K: int) -> int:
    return 2 * M * N * K


def gemm_launch_bytes(M: int, N: int, K: int, es: int, out_es: int, resid: bool = False) -> int:
    """Operands read once, output written once (+ residual read)."""
    return (M * K + N * K) * es + M * N * out_es + (M * N * 4 if resid else 0)


def head_flops_per_eval(hd) -> int:
    """One evaluation of the diffusion head for one row: the input product,
    the modulation product of every block and the final layer, the blocks'
    two products and the output product (the conditioning product and the
    time embedding run once per call and are not counted per evaluation)."""
    w, T = hd.width, hd.token_dim
    return 2 * (T * w + (3 * hd.depth + 2) * w * w + 2 * hd.depth * w * w + w * T)
