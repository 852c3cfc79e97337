"""Plain fp64 CPU oracle of LazyMAR's cached MAR transformer step.

TEST INFRASTRUCTURE ONLY.  Nothing on the product path imports this module:
only the tests, the smoke check and the benchmark's CPU-baseline leg do.  It
shares no code with the GPU library and imports nothing from it.

Everything is computed in float64 from the stored (float32 / bfloat16)
input values, one sequence at a time, in the order the paper states the
method.  The state is a *feature* cache (block outputs), as the paper writes
it in Sec. 3.2 (token cache, Eq. 9); the GPU library keeps a key/value cache
instead, so agreement between the two also checks that the forms match.

Readings of the paper taken here (the paper is silent or garbled on them):

* Eq. (8) writes arg max, while the text around it and Table 3's strategy V
  compute the tokens whose similarity is *low* and cache the most similar
  ones: the N least similar tokens are computed.
* The similarity is the cosine between this step's and the previous step's
  value rows (the self-attention value projection, bias included, all heads
  concatenated) of the last always-computed block (Sec. 4.4 "The position to
  calculate similarity"; the third block when three are always computed).
  With no always-computed block, the value rows of block 0 are formed from
  the step's input for scoring only.
* The value rows are scored as the path stores them (bfloat16 or float32);
  the products are exact in fp64 and each dot product is their exactly
  rounded fp64 sum, so the score does not depend on a summation order.  Zero norms: 1 when both rows are zero, else
  0.  A NaN score ranks as +inf (most similar).
* Ties go to the lower token index; selected indices are returned ascending.
* Table 3's strategy that caches the minimum-similarity tokens is taken as
  its exact opposite: the n *most* similar tokens are computed, ties to the
  lower index, a NaN score ranked last (never preferred).
* Option score_source = "features" (the alternative Sec. 4.4 weighs against
  the value matrix; Eq. (8) writes the features of the third layer): the
  similarity compares the output rows of block P-1 as the path stores its
  residual stream (float32), or the step input x when no block is always
  computed.
* Option fresh_kv (the reading the paper leaves open, taken the other way):
  at block P the rows that are not computed contribute keys/values formed
  from this step's block P-1 output instead of the cached ones; their
  outputs still come from the cache.
* Rows that are not computed keep the cached state of the previous block's
  output from the first cached block on, so their keys/values come from the
  cache (Eq. 9 applied from block P on).
* Classifier-free guidance mixes as u + s (c - u) (Eq. 7 is garbled in the
  text).  The condition cache stores C = u - c on a refresh and, on a reuse
  step, approximates u by c + C with c the conditional output of *that*
  step (Eq. 10; its reuse line carries the refresh step's superscript, read
  as the current step).
* Pre-LN blocks, LayerNorm eps from the dimensions, exact erf GELU, biases on
  every projection, attention scale 1/sqrt(d_head), no mask, no dropout.
"""
from __future__ import annotations

import math
from typing import Dict, List, Optional, Sequence

import numpy as np
from scipy.special import erf

__all__ = [
    "layer_norm", "gelu", "linear", "attention", "block_rows", "value_rows",
    "cosine_scores", "select_least_similar", "storage_round", "MarOracle",
    "cfg_store", "cfg_reuse", "guided",
]


def _f64(a) -> np.ndarray:
    return np.asarray(a, dtype=np.float64)


def layer_norm(x, w, b, eps: float) -> np.ndarray:
    """Row LayerNorm with biased variance (the block's LN1/LN2)."""
    x = _f64(x)
    mean = x.mean(axis=-1, keepdims=True)
    var = ((x - mean) ** 2).mean(axis=-1, keepdims=True)
    return (x - mean) / np.sqrt(var + eps) * _f64(w) + _f64(b)


def gelu(x) -> np.ndarray:
    """GELU in its exact form x * Phi(x)."""
    x = _f64(x)
    return 0.5 * x * (1.0 + erf(x / math.sqrt(2.0)))


def linear(x, w, b) -> np.ndarray:
    """x W^T + b with W in [out, in] layout."""
    return _f64(x) @ _f64(w).T + _f64(b)


def attention(q, k, v) -> np.ndarray:
    """Eq. (3): softmax(Q K^T / sqrt(d)) V for one head, no mask.

    q: [n_queries, d], k, v: [n_keys, d].  Rows of q may be any subset of the
    tokens; every query sees every key (bidirectional attention).
    """
    q, k, v = _f64(q), _f64(k), _f64(v)
    logits = q @ k.T / math.sqrt(q.shape[-1])
    logits = logits - logits.max(axis=-1, keepdims=True)
    p = np.exp(logits)
    p = p / p.sum(axis=-1, keepdims=True)
    return p @ v


def _split_qkv(p: Dict[str, np.ndarray], d_model: int):
    w, b = _f64(p["qkv_w"]), _f64(p["qkv_b"])
    D = d_model
    return (w[:D], b[:D]), (w[D:2 * D], b[D:2 * D]), (w[2 * D:], b[2 * D:])


def value_rows(m, p: Dict[str, np.ndarray], eps: float) -> np.ndarray:
    """Self-attention value rows LN1(m) W_v^T + b_v of every token."""
    m = _f64(m)
    _, _, (wv, bv) = _split_qkv(p, m.shape[-1])
    return linear(layer_norm(m, p["ln1_w"], p["ln1_b"], eps), wv, bv)


def block_rows(m, rows, p: Dict[str, np.ndarray], n_heads: int, eps: float):
    """One pre-LN bidirectional block evaluated for the token rows ``rows``.

    m is the block input of every token of one sequence [S, D].  Keys and
    values come from every row of m; queries, the output projection and the
    MLP are formed only for ``rows`` (Eq. 9: the computed set).  Returns the
    block output of those rows and the value rows of every token.
    """
    m = _f64(m)
    rows = np.asarray(rows, dtype=np.int64)
    S, D = m.shape
    dh = D // n_heads
    (wq, bq), (wk, bk), (wv, bv) = _split_qkv(p, D)
    a = layer_norm(m, p["ln1_w"], p["ln1_b"], eps)
    q = linear(a[rows], wq, bq)
    k = linear(a, wk, bk)
    v = linear(a, wv, bv)
    o = np.empty((len(rows), D), dtype=np.float64)
    for h in range(n_heads):
        cols = slice(h * dh, (h + 1) * dh)
        o[:, cols] = attention(q[:, cols], k[:, cols], v[:, cols])
    h1 = m[rows] + linear(o, p["proj_w"], p["proj_b"])
    f = gelu(linear(layer_norm(h1, p["ln2_w"], p["ln2_b"], eps), p["fc1_w"], p["fc1_b"]))
    out = h1 + linear(f, p["fc2_w"], p["fc2_b"])
    return out, v


def storage_round(a, dtype: str) -> np.ndarray:
    """Values as the path stores them: fp64 -> fp32 (-> bfloat16, ties to
    even), returned as fp64."""
    a32 = np.asarray(a, dtype=np.float32)
    if dtype == "f32":
        return a32.astype(np.float64)
    if dtype == "bf16":
        import torch
        t = torch.from_numpy(np.ascontiguousarray(a32)).to(torch.bfloat16)
        return t.to(torch.float64).numpy()
    raise ValueError(f"unknown dtype {dtype!r}")


def _exact_dot(a: np.ndarray, b: np.ndarray) -> np.ndarray:
    """Row dot products summed exactly and rounded once to fp64.

    The products of stored fp32/bf16 values are exact in fp64; math.fsum
    returns their exactly rounded sum, so the value does not depend on any
    summation order.
    """
    p = (a * b).reshape(-1, a.shape[-1])
    out = np.fromiter((math.fsum(row) for row in p.tolist()), dtype=np.float64, count=p.shape[0])
    return out.reshape(a.shape[:-1])


def cosine_scores(v, r) -> np.ndarray:
    """Eq. (8): S(x_i) = <v_i, r_i> / (||v_i|| ||r_i||) for every row i.

    v are this step's value rows, r the cached ones of the previous step.
    The three dot products are exactly rounded fp64 values; then
    s = dot / sqrt(|v|^2 |r|^2).  Zero norms: 1 if both rows are zero, else 0.
    """
    v, r = _f64(v), _f64(r)
    dot = _exact_dot(v, r)
    nv = _exact_dot(v, v)
    nr = _exact_dot(r, r)
    den = np.sqrt(nv * nr)
    with np.errstate(invalid="ignore", divide="ignore"):
        s = dot / den
    zero = den == 0.0
    s = np.where(zero, np.where((nv == 0.0) & (nr == 0.0), 1.0, 0.0), s)
    return s


def select_least_similar(s, n: int) -> np.ndarray:
    """I_compute of Eq. (8): the n tokens with the smallest similarity.

    Ties go to the lower token index (a stable sort); NaN ranks as +inf.
    The result is returned in ascending token order (int32).
    """
    s = np.array(s, dtype=np.float64)
    if not 0 <= n <= s.shape[-1]:
        raise ValueError("n out of range")
    s[np.isnan(s)] = np.inf
    order = np.argsort(s, kind="stable")
    return np.sort(order[:n]).astype(np.int32)


def select_most_similar(s, n: int) -> np.ndarray:
    """Table 3's strategy that caches the minimum-similarity tokens: the n
    tokens with the largest similarity are computed instead.

    Ties go to the lower token index; NaN ranks last.  Ascending order
    (int32).
    """
    s = np.array(s, dtype=np.float64)
    if not 0 <= n <= s.shape[-1]:
        raise ValueError("n out of range")
    key = -s
    key[np.isnan(key)] = np.inf
    order = np.argsort(key, kind="stable")
    return np.sort(order[:n]).astype(np.int32)


def cfg_store(y_cond, y_uncond, scale: float):
    """Refresh step of the condition cache (Eq. 10): returns (stored
    residual C = u - c, guided output u + s (c - u))."""
    c, u = _f64(y_cond), _f64(y_uncond)
    return u - c, guided(c, u, scale)


def cfg_reuse(y_cond, stored, scale: float):
    """Reuse step (Eq. 10): the unconditional output is approximated as
    u_hat = c + C from this step's conditional output and the stored
    residual; returns (u_hat, guided)."""
    c = _f64(y_cond)
    u_hat = c + _f64(stored)
    return u_hat, guided(c, u_hat, scale)


def guided(c, u, scale: float) -> np.ndarray:
    """Classifier-free guidance mix u + s (c - u)."""
    c, u = _f64(c), _f64(u)
    return u + scale * (c - u)


class MarOracle:
    """State and steps of the cached transformer for a set of sequence slots.

    Per slot b: the feature cache Hc[l] (output of block l for l = P-1..L-1,
    and the block-0 input when P = 0), the previous value rows used for
    scoring, and whether a full step has filled the cache.  Per CFG pair: the
    stored residual.
    """

    def __init__(self, dims, blocks: Sequence[Dict[str, np.ndarray]]):
        self.L = int(dims.n_layers)
        self.D = int(dims.d_model)
        self.H = int(dims.n_heads)
        self.S = int(dims.seq_len)
        self.P = int(dims.full_prefix)
        self.eps = float(dims.ln_eps)
        self.dtype = dims.dtype
        self.max_slots = int(dims.max_slots)
        if len(blocks) != self.L:
            raise ValueError("one weight dict per block expected")
        self.blocks = list(blocks)
        self.score_source = getattr(dims, "score_source", "values")
        self.fresh_kv = bool(getattr(dims, "fresh_kv", False))
        if self.score_source not in ("values", "features"):
            raise ValueError("score_source is 'values' or 'features'")
        self.hc: List[Optional[Dict[int, np.ndarray]]] = [None] * self.max_slots
        self.vref: List[Optional[np.ndarray]] = [None] * self.max_slots
        self.fref: List[Optional[np.ndarray]] = [None] * self.max_slots
        self.delta: Dict[int, np.ndarray] = {}

    # -- one sequence ------------------------------------------------------
    def _score_layer(self) -> int:
        return max(self.P - 1, 0)

    def _block(self, m, rows, l: int):
        """Block l on the rows ``rows`` of the block input m (one sequence)."""
        return block_rows(m, rows, self.blocks[l], self.H, self.eps)

    def _values(self, x) -> np.ndarray:
        """Value rows of block 0 formed from the step input (no always-computed
        block)."""
        return value_rows(x, self.blocks[0], self.eps)

    def full_slot(self, b: int, x) -> np.ndarray:
        """Full step (refresh / warm-up): every block on every row; fills the
        token cache of every cached block and the scoring reference."""
        h = _f64(x).reshape(self.S, self.D)
        rows = np.arange(self.S)
        hc: Dict[int, np.ndarray] = {}
        if self.P == 0:
            hc[-1] = h.copy()
            self.fref[b] = h.copy()
        for l in range(self.L):
            h, v = self._block(h, rows, l)
            if l == self._score_layer():
                self.vref[b] = storage_round(v, self.dtype)
            if l == self.P - 1:
                self.fref[b] = storage_round(h, "f32")
            if l >= self.P - 1:
                hc[l] = h.copy()
        self.hc[b] = hc
        return h

    def cached_slot(self, b: int, x, n: int, given: Optional[np.ndarray] = None, rule: str = "least"):
        """Cached step of one sequence (Sec. 3.2, Eq. 8 and 9).

        Blocks 0..P-1 run on every row; the value rows of block P-1 are scored
        against the previous step's; the n least similar rows (the n most
        similar with rule="most", Table 3; or the ``given`` rows) are
        computed through blocks P..L-1 and every other row is taken from the
        cache.  Returns (output rows of every token, the computed set, the
        scores).
        """
        if self.hc[b] is None:
            raise RuntimeError("cached step before a full step filled the cache")
        h = _f64(x).reshape(self.S, self.D)
        rows_all = np.arange(self.S)
        if self.P == 0:
            v = self._values(h)
        else:
            for l in range(self.P):
                h, v = self._block(h, rows_all, l)
        v = storage_round(v, self.dtype)
        if self.score_source == "features":
            feat = h.copy() if self.P == 0 else storage_round(h, "f32")
            scores = cosine_scores(feat, self.fref[b])
            self.fref[b] = feat
        else:
            scores = cosine_scores(v, self.vref[b])
        if given is None:
            if rule not in ("least", "most"):
                raise ValueError("rule is 'least' or 'most'")
            idx = select_least_similar(scores, n) if rule == "least" else select_most_similar(scores, n)
        else:
            idx = np.asarray(given, dtype=np.int32)
        self.vref[b] = v
        hc = self.hc[b]
        if self.fresh_kv:
            hc[self.P - 1] = h.copy()  # every row's block-P input (keys/values) from this step
        fresh = h[idx]
        for l in range(self.P, self.L):
            hc[l - 1][idx] = fresh
            fresh, _ = self._block(hc[l - 1], idx, l)
            hc[l][idx] = fresh
        return hc[self.L - 1].copy(), idx, scores

    # -- a range of slots ----------------------------------------------------
    def full(self, x, slot0: int = 0) -> np.ndarray:
        x = _f64(x)
        return np.stack([self.full_slot(slot0 + i, x[i]) for i in range(x.shape[0])])

    def cached(self, x, n: int, slot0: int = 0, given=None, rule: str = "least"):
        x = _f64(x)
        ys, idxs, ss = [], [], []
        for i in range(x.shape[0]):
            g = None if given is None else np.asarray(given)[i]
            y, idx, s = self.cached_slot(slot0 + i, x[i], n, g, rule)
            ys.append(y)
            idxs.append(idx)
            ss.append(s)
        return np.stack(ys), np.stack(idxs), np.stack(ss)

    def output(self, b: int) -> np.ndarray:
        return self.hc[b][self.L - 1].copy()

    def cfg(self, op: str, y_cond, y_uncond, scale: float, pair0: int = 0):
        """Condition cache: 'store' on a refresh (both pathways computed),
        'reuse' when only the conditional pathway was computed.  Returns
        (guided, unconditional output used)."""
        y_cond = _f64(y_cond)
        out_g, out_u = [], []
        for i in range(y_cond.shape[0]):
            if op == "store":
                d, g = cfg_store(y_cond[i], _f64(y_uncond)[i], scale)
                self.delta[pair0 + i] = d
                out_u.append(_f64(y_uncond)[i])
            elif op == "reuse":
                if pair0 + i not in self.delta:
                    raise RuntimeError("reuse before store")
                u, g = cfg_reuse(y_cond[i], self.delta[pair0 + i], scale)
                out_u.append(u)
            else:
                raise ValueError(op)
            out_g.append(g)
        return np.stack(out_g), np.stack(out_u)
