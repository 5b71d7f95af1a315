"""Window query recomputation (App. C.2) -- TEST INFRASTRUCTURE, NOT PRODUCT.

Only the tests, the smoke check and the benchmark's CPU-baseline leg may use
this module; the product's recompute pass is the library's own kernels
(include/kara_recompute.h) and shares nothing with it.

At a compression event the scoring queries of the window are not cached:
they are recomputed by one extra forward pass over the window's tokens that
forms only the query projections, attends causally to the K/V rows already
in the cache, and runs the feed-forward block (App. C.2).  Per triggered
sequence and layer, with h the residual stream of the |W| window tokens:

    x   = RMSNorm(h) * g_attn                      (each token over the hidden size)
    q   = RoPE(x W_q) at the tokens' positions     -> this layer's scoring queries
    o_w = softmax(q_w K[0 : p0+w+1]^T / sqrt(d)) V[0 : p0+w+1]
          for window token w at cache position p0 + w; query head hq reads
          KV head hq // G
    h  += concat_heads(o) W_o
    x'  = RMSNorm(h) * g_ffn
    h  += (silu(x' W_gate) * (x' W_up)) W_down

Readings where the paper only names the sub-steps:
* R-ARCH: the decoder architecture of the models the paper evaluates
  (Qwen3 / Llama-family): pre-norm RMSNorm (eps inside the square root),
  rotary embedding in the rotate-half form with base theta on the queries
  (cached keys already carry theirs), SwiGLU feed-forward, no biases.
* R-POS: a window token's rotary position is its logical position in the
  sequence, rope_pos0 + w, passed by the caller (after compressions the
  physical cache position p0 + w is smaller); the causal mask uses physical
  cache positions: token w sees cache rows [0, p0 + w].

Everything is fp64 numpy, one token and head at a time where the definition
is per token or per head; matrix products use numpy's matmul.
"""

from __future__ import annotations

import math

import numpy as np

from .kara_oracle import read_rows


def rms_norm(h: np.ndarray, g: np.ndarray, eps: float) -> np.ndarray:
    """h [T, D] -> h / sqrt(mean(h^2) + eps) * g."""
    h = np.asarray(h, dtype=np.float64)
    ms = (h * h).mean(axis=-1, keepdims=True)
    return h / np.sqrt(ms + eps) * np.asarray(g, dtype=np.float64)


def rope(x: np.ndarray, positions: np.ndarray, theta: float) -> np.ndarray:
    """Rotary embedding, rotate-half form: for i < d/2 the pair (x_i,
    x_{i+d/2}) is rotated by angle pos * theta^(-2i/d).  x [T, H, d]."""
    x = np.asarray(x, dtype=np.float64)
    d = x.shape[-1]
    half = d // 2
    inv_freq = theta ** (-np.arange(half, dtype=np.float64) * 2.0 / d)
    ang = np.asarray(positions, dtype=np.float64)[:, None] * inv_freq[None, :]        # [T, d/2]
    c, s = np.cos(ang)[:, None, :], np.sin(ang)[:, None, :]
    a, b = x[..., :half], x[..., half:]
    return np.concatenate([a * c - b * s, b * c + a * s], axis=-1)


def silu(x: np.ndarray) -> np.ndarray:
    x = np.asarray(x, dtype=np.float64)
    return x / (1.0 + np.exp(-x))


def causal_window_attention(q: np.ndarray, k_rows: np.ndarray, v_rows: np.ndarray, p0: int,
                            scale: float) -> np.ndarray:
    """q [W, Hq, d]; k_rows, v_rows [S, Hkv, d] with S >= p0 + W: the cache
    rows of the sequence in position order.  Window token w, at cache
    position p0 + w, attends to rows 0 .. p0 + w.  Returns [W, Hq, d]."""
    W, Hq, d = q.shape
    Hkv = k_rows.shape[1]
    G = Hq // Hkv
    out = np.zeros((W, Hq, d), dtype=np.float64)
    for w in range(W):
        n = p0 + w + 1
        for hq in range(Hq):
            h = hq // G
            logits = (k_rows[:n, h, :] @ q[w, hq, :]) * scale
            p = np.exp(logits - logits.max())
            p /= p.sum()
            out[w, hq, :] = p @ v_rows[:n, h, :]
    return out


def recompute_layer(h: np.ndarray, wt: dict, k_rows: np.ndarray, v_rows: np.ndarray, p0: int, rope_pos0: int,
                    dims: dict):
    """One layer of the recompute pass for one sequence.  h [W, D] (fp64);
    wt: w_q [D, Hq*d], w_o [Hq*d, D], w_gate / w_up [D, F], w_down [F, D],
    g_attn / g_ffn [D] (fp64).  Returns (q [W, Hq, d] after RoPE, h after the
    layer, attention output [W, Hq, d])."""
    W, D = h.shape
    Hq, d = dims["n_q_heads"], dims["head_dim"]
    x = rms_norm(h, wt["g_attn"], dims["rms_eps"])
    q = (x @ wt["w_q"]).reshape(W, Hq, d)
    q = rope(q, rope_pos0 + np.arange(W), dims["rope_theta"])
    o = causal_window_attention(q, k_rows, v_rows, p0, 1.0 / math.sqrt(d))
    h = h + o.reshape(W, Hq * d) @ wt["w_o"]
    x2 = rms_norm(h, wt["g_ffn"], dims["rms_eps"])
    h = h + (silu(x2 @ wt["w_gate"]) * (x2 @ wt["w_up"])) @ wt["w_down"]
    return q, h, o


def cache_rows(pool: np.ndarray, table_row: np.ndarray, count: int, block_size: int, to64) -> np.ndarray:
    """Rows 0 .. count-1 of every KV head of one sequence: [count, Hkv, d]."""
    pos = np.arange(count, dtype=np.int64)
    heads = [to64(read_rows(pool, table_row, pos, h, block_size)) for h in range(pool.shape[1])]
    return np.stack(heads, axis=1)


def recompute_sequence(h0: np.ndarray, weights: list, k_pools: list, v_pools: list, table_row, p0: int,
                       rope_pos0: int, dims: dict, to64):
    """The whole pass for one sequence over len(weights) layers.  Returns the
    per-layer queries [L, W, Hq, d], the per-layer residual streams entering
    each layer [L+1, W, D] and the attention outputs [L, W, Hq, d]."""
    W = h0.shape[0]
    h = np.asarray(h0, dtype=np.float64)
    qs, hs, os_ = [], [h], []
    for l, wt in enumerate(weights):
        kr = cache_rows(k_pools[l], table_row, p0 + W, dims["block_size"], to64)
        vr = cache_rows(v_pools[l], table_row, p0 + W, dims["block_size"], to64)
        q, h, o = recompute_layer(h, wt, kr, vr, p0, rope_pos0, dims)
        qs.append(q)
        hs.append(h)
        os_.append(o)
    return np.stack(qs), np.stack(hs), np.stack(os_)
