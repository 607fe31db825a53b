"""Plain fp64 definition of one Q-First decoder block at a decode step.

TEST INFRASTRUCTURE ONLY (see ``oracle/__init__.py``): only tests may use this module.

Paper: Q-First, arXiv:2608.15473.
  §2 (the decode protocol): u_j is the block's input, N1 the attention's normalisation, N2 the
      feed-forward's, M the feed-forward.  In the rewired block the query is projected from the
      input, q_j = W_q N1(u_j), and the key and value from the stream after the feed-forward,
      k_j = W_k N1(z_j), v_j = W_v N1(z_j), z_j = u_j + M(N2 u_j).
  §8 (the block algebra): the block is Q = (I + A_{x;z}) o (I + M) -- the feed-forward's residual
      update first, then attention scoring from x and loading values from z, added to z.  So the
      block's output is y_j = z_j + W_o attn_j.
  §2: attention at step j runs over the j-1 cached positions and the current one, s = q.k/sqrt(d).

Where the paper is silent the Qwen3 blocks it converts fix the form (readings):
  N1, N2 are RMS normalisations with a learned gain, x / sqrt(mean(x^2) + eps) * g, eps = 1e-6;
  M is the SwiGLU feed-forward W_down (silu(W_gate h) * W_up h), silu(x) = x sigmoid(x);
  query head h reads KV head floor(h / G) (grouped-query attention);
  the key reads z as §2 states it (in §8's A_{x;z} the scores come from x, which names the
  query's side; §8 also notes that where the key is read is free for the sweep);
  rotary position embeddings and Qwen3's per-head q/k normalisation are left out (they act on q
  and k elementwise and do not bear on which point of the stream each reads).

Weights are torch-layout [out, in] matrices: W x is ``x @ W.T``.  All arithmetic is float64 on
exact copies of the bf16 inputs.

Parity status: pinned by ``tests/test_oracle_block.py`` (torch's functional rms_norm / silu /
linear / scaled_dot_product_attention in float64 as independent library routines; the empty-cache
and zero-feed-forward special cases; step-by-step decode with appends equal to causal attention
over the whole sequence).
"""

from __future__ import annotations

import numpy as np

from .attention import attend, gather_rows

RMS_EPS = 1e-6


def round_bf16(x) -> np.ndarray:
    """Round to bfloat16 as a float32-computing kernel that stores bf16 does: the value is first
    the nearest float32, then the nearest bfloat16 (ties to even; the upper 16 bits of float32).
    NaN stays NaN.  Returned as float64."""
    f = np.asarray(x, dtype=np.float64).astype(np.float32)
    u = f.view(np.uint32).astype(np.uint64)
    lsb = (u >> 16) & 1
    r = ((u + 0x7FFF + lsb) >> 16) << 16
    out = r.astype(np.uint32).view(np.float32).astype(np.float64)
    return np.where(np.isnan(f), np.nan, out)


def rms_norm(x, g, eps: float = RMS_EPS) -> np.ndarray:
    """x / sqrt(mean(x^2) + eps) * g over the last axis."""
    x = np.asarray(x, dtype=np.float64)
    return x / np.sqrt(np.mean(x * x, axis=-1, keepdims=True) + eps) * np.asarray(g, np.float64)


def silu(x) -> np.ndarray:
    x = np.asarray(x, dtype=np.float64)
    return x / (1.0 + np.exp(-x))


def swiglu(gate, up) -> np.ndarray:
    """The feed-forward's activation: silu(gate) * up."""
    return silu(gate) * np.asarray(up, dtype=np.float64)


def feed_forward(h, w) -> np.ndarray:
    """M(h) = W_down (silu(W_gate h) * W_up h)."""
    return swiglu(h @ w["w_gate"].T, h @ w["w_up"].T) @ w["w_down"].T


def qfirst_block(u, w, k_cache, v_cache, block_table, ctx_lens, n_q_heads: int,
                 n_kv_heads: int, scale: float, page_size: int = 16, eps: float = RMS_EPS,
                 bf16_stores: bool = False):
    """One decode step of the Q-First block for every request.

    ``u`` [B, H]; ``w`` a dict of float64 arrays (w_q, w_k, w_v, w_o, w_gate, w_up, w_down, g1,
    g2); the cache holds ``ctx_lens[b]`` positions of request b (before this step's append).
    Returns a dict with q [B, Hq, D], k, v [B, Hkv, D], z [B, H], act [B, I] (the feed-forward's
    activation), attn [B, Hq, D] (attention over the cached positions and the current one),
    lse [B, Hq] and y [B, H].

    ``bf16_stores``: round q, act, z, k, v, attn and y to bfloat16 (round_bf16) where they are
    computed, as a pipeline does that keeps those seven tensors in bf16 between its steps; every
    other quantity (the normalisations, the products' sums, the softmax) stays exact.
    """
    rnd = round_bf16 if bf16_stores else (lambda a: np.asarray(a, dtype=np.float64))
    u = np.asarray(u, dtype=np.float64)
    B = u.shape[0]
    Hq, Hkv = n_q_heads, n_kv_heads
    G = Hq // Hkv
    q = rnd(rms_norm(u, w["g1"], eps) @ w["w_q"].T).reshape(B, Hq, -1)   # query from u
    h2 = rms_norm(u, w["g2"], eps)
    act = rnd(swiglu(h2 @ w["w_gate"].T, h2 @ w["w_up"].T))
    z = rnd(u + act @ w["w_down"].T)                                        # (I + M)
    hz = rms_norm(z, w["g1"], eps)
    k = rnd(hz @ w["w_k"].T).reshape(B, Hkv, -1)                            # key, value from z
    v = rnd(hz @ w["w_v"].T).reshape(B, Hkv, -1)
    D = q.shape[-1]
    attn = np.zeros((B, Hq, D))
    lse = np.zeros((B, Hq))
    for b in range(B):
        n = int(ctx_lens[b])
        row = block_table[b] if block_table is not None else None
        if row is None:
            max_pages = k_cache.shape[0] // B
            row = np.arange(b * max_pages, (b + 1) * max_pages)
        for h in range(Hq):
            g = h // G
            K = np.concatenate([gather_rows(k_cache, row, g, n, page_size), k[b, g][None]])
            V = np.concatenate([gather_rows(v_cache, row, g, n, page_size), v[b, g][None]])
            attn[b, h], lse[b, h] = attend(q[b, h], K, V, scale)
    attn = rnd(attn)
    y = rnd(z + attn.reshape(B, -1) @ w["w_o"].T)                           # (I + A) on z
    return dict(q=q, k=k, v=v, z=z, act=act, attn=attn, lse=lse, y=y)
