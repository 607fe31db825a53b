"""Pins of the fp64 Q-First block oracle (oracle/block.py) against things other than itself.

* torch's functional rms_norm / silu / linear / scaled_dot_product_attention (float64, CPU) as
  independent library routines for every primitive of the block;
* the special cases an empty cache (softmax over one position is 1, so attention is v_j) and a
  zero feed-forward (z = u) reduce the block to;
* a sequence decoded one step at a time, appending each step's key and value to the paged cache,
  equals causal attention over the whole sequence at once (§2: the cache plus the current token
  is the attention over j positions).
"""

import numpy as np
import pytest
import torch
import torch.nn.functional as F

import oracle
from oracle import block as oracle_block
from workloads import BlockShape, block_input, block_weights

SHAPE = BlockShape("tiny", hidden=64, inter=96, n_q_heads=4, n_kv_heads=2, layers=1)
D = 32
SCALE = D ** -0.5


def _weights(seed, shape=SHAPE):
    return {k: v.double().numpy() for k, v in block_weights(shape, seed, head_dim=D).items()}


def _t(x):
    return torch.from_numpy(np.ascontiguousarray(x))


def _cache(B, ctx, seed, spare=0, page=16, Hkv=SHAPE.n_kv_heads):
    """A paged cache with a permuted table; request b holds ctx[b] positions and has pages for
    ctx[b] + spare."""
    rng = np.random.default_rng(seed)
    ctx = np.asarray(ctx)
    pages = -(-(ctx + spare) // page)
    max_pages = max(1, int(pages.max()))
    num = max(1, int(pages.sum()))
    k = rng.standard_normal((num, Hkv, page, D))
    v = rng.standard_normal((num, Hkv, page, D))
    perm = rng.permutation(num)
    bt = np.full((B, max_pages), -1, dtype=np.int64)
    off = 0
    for b in range(B):
        bt[b, : pages[b]] = perm[off: off + pages[b]]
        off += pages[b]
    return k, v, bt, ctx.astype(np.int64)


def _torch_rows(cache, bt_row, g, n, page=16):
    """Rows 0..n-1 of KV head g by torch indexing (independent of the oracle's gather)."""
    pos = torch.arange(n)
    phys = torch.as_tensor(bt_row, dtype=torch.int64)[pos // page]
    return _t(cache)[phys, g, pos % page]


def _torch_block(u, w, k_cache, v_cache, bt, ctx, eps=oracle.RMS_EPS):
    """The rewired block of §2 written with torch's functional library routines."""
    Hq, Hkv = SHAPE.n_q_heads, SHAPE.n_kv_heads
    W = {k: _t(v) for k, v in w.items()}
    u = _t(u)
    B, H = u.shape
    q = F.linear(F.rms_norm(u, (H,), W["g1"], eps), W["w_q"]).view(B, Hq, D)
    h2 = F.rms_norm(u, (H,), W["g2"], eps)
    z = u + F.linear(F.silu(F.linear(h2, W["w_gate"])) * F.linear(h2, W["w_up"]), W["w_down"])
    hz = F.rms_norm(z, (H,), W["g1"], eps)
    k = F.linear(hz, W["w_k"]).view(B, Hkv, D)
    v = F.linear(hz, W["w_v"]).view(B, Hkv, D)
    outs = []
    for b in range(B):
        n = int(ctx[b])
        K = torch.stack([torch.cat([_torch_rows(k_cache, bt[b], g, n), k[b, g][None]])
                         for g in range(Hkv)])                      # [Hkv, n+1, D]
        V = torch.stack([torch.cat([_torch_rows(v_cache, bt[b], g, n), v[b, g][None]])
                         for g in range(Hkv)])
        o = F.scaled_dot_product_attention(q[b][:, None], K, V, scale=SCALE, enable_gqa=True)
        outs.append(o[:, 0])
    attn = torch.stack(outs)                                           # [B, Hq, D]
    y = z + F.linear(attn.reshape(B, -1), W["w_o"])
    return dict(q=q, k=k, v=v, z=z, attn=attn, y=y)


def test_rms_norm_and_silu_match_torch():
    rng = np.random.default_rng(1)
    x = rng.standard_normal((5, 64)) * np.array([1e-3, 1, 30, 1, 1])[:, None]
    g = rng.uniform(0.5, 1.5, 64)
    ref = F.rms_norm(_t(x), (64,), _t(g), oracle.RMS_EPS).numpy()
    np.testing.assert_allclose(oracle.rms_norm(x, g), ref, rtol=1e-13, atol=0)
    s = np.linspace(-60, 60, 2001)
    np.testing.assert_allclose(oracle.silu(s), F.silu(_t(s)).numpy(), rtol=1e-13, atol=1e-300)
    assert oracle.silu(np.array([0.0]))[0] == 0.0


def test_feed_forward_matches_torch():
    w = _weights(3)
    h = np.random.default_rng(2).standard_normal((3, SHAPE.hidden))
    W = {k: _t(v) for k, v in w.items()}
    ref = F.linear(F.silu(F.linear(_t(h), W["w_gate"])) * F.linear(_t(h), W["w_up"]),
                   W["w_down"]).numpy()
    np.testing.assert_allclose(oracle.feed_forward(h, w), ref, rtol=1e-12, atol=1e-13)


def test_block_matches_torch_functional_with_gqa():
    B, ctx = 3, [0, 5, 37]
    w = _weights(4)
    u = block_input(B, SHAPE.hidden, seed=5).double().numpy()
    k, v, bt, n = _cache(B, ctx, seed=6)
    got = oracle.qfirst_block(u, w, k, v, bt, n, SHAPE.n_q_heads, SHAPE.n_kv_heads, SCALE)
    ref = _torch_block(u, w, k, v, bt, n)
    for name in ("q", "k", "v", "z", "attn", "y"):
        np.testing.assert_allclose(got[name], ref[name].numpy(), rtol=1e-11, atol=1e-12,
                                   err_msg=name)


def test_empty_cache_and_zero_feed_forward():
    """No cached positions: attention is the current value; no feed-forward: z = u."""
    B = 2
    w = _weights(7)
    w["w_down"] = np.zeros_like(w["w_down"])
    u = block_input(B, SHAPE.hidden, seed=8).double().numpy()
    k, v, bt, n = _cache(B, [0, 0], seed=9, spare=1)
    got = oracle.qfirst_block(u, w, k, v, bt, n, SHAPE.n_q_heads, SHAPE.n_kv_heads, SCALE)
    np.testing.assert_array_equal(got["z"], u)
    G = SHAPE.n_q_heads // SHAPE.n_kv_heads
    np.testing.assert_allclose(got["attn"], np.repeat(got["v"], G, axis=1), rtol=4e-16, atol=0)
    np.testing.assert_allclose(got["y"], u + got["attn"].reshape(B, -1) @ w["w_o"].T, rtol=1e-14)


def test_query_reads_the_input_and_value_the_feed_forward_stream():
    """Changing only W_down moves k, v, z and y but not q (q reads u, §2)."""
    w = _weights(10)
    u = block_input(2, SHAPE.hidden, seed=11).double().numpy()
    k, v, bt, n = _cache(2, [20, 3], seed=12)
    a = oracle.qfirst_block(u, w, k, v, bt, n, SHAPE.n_q_heads, SHAPE.n_kv_heads, SCALE)
    w2 = dict(w, w_down=w["w_down"] * 1.5)
    b = oracle.qfirst_block(u, w2, k, v, bt, n, SHAPE.n_q_heads, SHAPE.n_kv_heads, SCALE)
    np.testing.assert_array_equal(a["q"], b["q"])
    for name in ("z", "k", "v", "y"):
        assert not np.allclose(a[name], b[name]), name


@pytest.mark.parametrize("T", [1, 19])
def test_stepwise_decode_equals_causal_attention_over_the_sequence(T):
    """Decode T steps, appending each step's (k, v) to the paged cache (oracle.append_kv): every
    step's output equals the same block applied to the whole sequence with causal attention."""
    Hq, Hkv, H = SHAPE.n_q_heads, SHAPE.n_kv_heads, SHAPE.hidden
    w = _weights(13)
    U = block_input(T, H, seed=14).double().numpy()                   # one request, T steps
    k, v, bt, n = _cache(1, [0], seed=15, spare=T)
    ys = []
    for t in range(T):
        r = oracle.qfirst_block(U[t][None], w, k, v, bt, n, Hq, Hkv, SCALE)
        ys.append(r["y"][0])
        k, v = oracle.append_kv(k, v, bt, n, r["k"], r["v"])
        n = n + 1
    W = {kk: _t(vv) for kk, vv in w.items()}
    Ut = _t(U)
    Q = F.linear(F.rms_norm(Ut, (H,), W["g1"], oracle.RMS_EPS), W["w_q"]).view(T, Hq, D)
    h2 = F.rms_norm(Ut, (H,), W["g2"], oracle.RMS_EPS)
    Z = Ut + F.linear(F.silu(F.linear(h2, W["w_gate"])) * F.linear(h2, W["w_up"]), W["w_down"])
    hz = F.rms_norm(Z, (H,), W["g1"], oracle.RMS_EPS)
    K = F.linear(hz, W["w_k"]).view(T, Hkv, D).transpose(0, 1)
    V = F.linear(hz, W["w_v"]).view(T, Hkv, D).transpose(0, 1)
    A = F.scaled_dot_product_attention(Q.transpose(0, 1), K, V, is_causal=True, scale=SCALE,
                                       enable_gqa=True)                # [Hq, T, D]
    Y = Z + F.linear(A.transpose(0, 1).reshape(T, -1), W["w_o"])
    np.testing.assert_allclose(np.stack(ys), Y.numpy(), rtol=1e-11, atol=1e-12)


def test_round_bf16_matches_torch_conversion():
    """The oracle's bf16 rounding (nearest float32, then nearest bf16, ties to even) against
    torch's float32 -> bfloat16 conversion, an independent library routine: random values over
    many binades, exact ties (the low 16 bits exactly 0x8000, both parities), subnormals, the
    largest finite values (which round to inf), infinities and NaN."""
    import torch
    rng = np.random.default_rng(11)
    vals = [rng.standard_normal(20000) * 10.0 ** rng.uniform(-40, 38, 20000)]
    base = rng.integers(0, 1 << 15, 4000, dtype=np.uint64) << np.uint64(16)
    ties = (base | np.uint64(0x8000)) | (rng.integers(0, 2, 4000, dtype=np.uint64) << np.uint64(31))
    vals.append(ties.astype(np.uint32).view(np.float32).astype(np.float64))
    vals.append(np.array([1e-40, -3e-45, 3.3895e38, -3.39e38, np.inf, -np.inf, 0.0, -0.0]))
    x = np.concatenate(vals)
    ref = torch.from_numpy(x.astype(np.float32)).to(torch.bfloat16).to(torch.float64).numpy()
    got = oracle_block.round_bf16(x)
    assert np.array_equal(got, ref, equal_nan=True)
    assert np.isnan(oracle_block.round_bf16(np.array([np.nan])))[0]


def test_block_with_bf16_stores_is_the_exact_block_rounded():
    """With bf16_stores the seven stored tensors are bf16 values, the rest of the block follows
    from them exactly, and the output stays within the rounding's reach of the exact block."""
    B, H, I, Hq, Hkv, D = 3, 64, 96, 4, 2, 16
    rng = np.random.default_rng(12)
    w = {"w_q": rng.standard_normal((Hq * D, H)) / 8, "w_k": rng.standard_normal((Hkv * D, H)) / 8,
         "w_v": rng.standard_normal((Hkv * D, H)) / 8, "w_o": rng.standard_normal((H, Hq * D)) / 8,
         "w_gate": rng.standard_normal((I, H)) / 8, "w_up": rng.standard_normal((I, H)) / 8,
         "w_down": rng.standard_normal((H, I)) / 10, "g1": rng.uniform(0.5, 1.5, H),
         "g2": rng.uniform(0.5, 1.5, H)}
    u = rng.standard_normal((B, H))
    kc = rng.standard_normal((6, Hkv, 16, D))
    vc = rng.standard_normal((6, Hkv, 16, D))
    bt = np.arange(6).reshape(3, 2)
    n = np.array([20, 0, 31])
    exact = oracle_block.qfirst_block(u, w, kc, vc, bt, n, Hq, Hkv, D ** -0.5)
    emu = oracle_block.qfirst_block(u, w, kc, vc, bt, n, Hq, Hkv, D ** -0.5, bf16_stores=True)
    for key in ("q", "act", "z", "k", "v", "attn", "y"):
        assert np.array_equal(oracle_block.round_bf16(emu[key]), emu[key]), key
    # the first stored tensors are the exact ones rounded (nothing upstream was rounded)
    assert np.array_equal(emu["q"], oracle_block.round_bf16(exact["q"]))
    assert np.array_equal(emu["act"], oracle_block.round_bf16(exact["act"]))
    rel = np.linalg.norm(emu["y"] - exact["y"]) / np.linalg.norm(exact["y"])
    assert 0 < rel < 2.0 ** -7
