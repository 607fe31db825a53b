"""GPU tests of the Q-First block stack with the sweep beside the feed-forward on two streams
(§2, §3 "across layers", §8), through the C ABI: the fused products (qf_linear), the sweep, the
merge with the current-token fold and the cache append.

* the fused products (qf_linear: RMS normalisation or SwiGLU prologue, residual epilogue) against
  the fp64 oracle, each output within the bf16 values around the exact result widened by the
  fp32 accumulation bound;
* the sweep and a product in one launch (qf_attn_decode_split_beside) give bitwise the results of
  the two separate calls;
* the three orders (serial, two streams, one shared launch) produce bitwise the same outputs and
  caches, eagerly and when the step is captured in a HIP graph and replayed (each replay checked,
  with eager work between);
* a whole block against the fp64 oracle of the block (oracle.qfirst_block), product by product:
  each of the seven bf16 tensors the GPU path stores (q, the feed-forward's activation, z, k, v,
  attn, y) is checked against the oracle fed the GPU's own bf16 inputs of that product, at the gate
  of the standalone products (the bf16 values around the exact result widened by the fp32
  accumulation bound) or of the attention (between the bf16 neighbours of O -/+ 1e-4 max|O|);
* a whole three-block step against the oracle that rounds those same seven tensors to bf16
  (qfirst_block with bf16_stores).  The two differ only where the GPU's fp32 sums and the
  oracle's exact ones fall on either side of a bf16 rounding boundary: the sums differ by at most
  ~(K/64 + 32) 2^-24 of their magnitude (~3e-6 here), so about one element in 700 of a tensor
  moves by one bf16 step (2^-8), ~1.5e-4 relative (L2) per stored tensor; 21 of them over three
  blocks add to ~7e-4.  Gate: 2e-3 relative (L2).  A query or key/value read from the wrong point
  of the stream, or the wrong residual, moves the output by 2e-2 ... 5e-1 (short contexts make the
  current token's key and value visible).
"""

import numpy as np
import pytest
import torch

import oracle
import paper_2608_15473_amd as qf
from paper_2608_15473_amd.stage import LayerCache, QFirstStack
from parity import bf16_neighbours, say
from workloads import SCALE, BlockShape, block_input, block_weights, make_case

pytestmark = pytest.mark.gpu

SHAPE = BlockShape("test", hidden=256, inter=512, n_q_heads=4, n_kv_heads=2, layers=3)
CTX = np.array([300, 2, 0])
SHARDS = [3, 1, 1]
SPARE = 8


def _build(gpu, L=SHAPE.layers, seed=500, ctx=CTX, shards=SHARDS):
    Hq, Hkv = SHAPE.n_q_heads, SHAPE.n_kv_heads
    layers, caches = [], []
    for l in range(L):
        layers.append({k: t.to(gpu) for k, t in block_weights(SHAPE, seed + l).items()})
        c = make_case(len(ctx), Hq, Hkv, np.asarray(ctx) + SPARE, shards, seed=seed + 100 + l,
                      device=gpu)
        c.ctx_lens -= SPARE
        caches.append(LayerCache(c.k_cache, c.v_cache, c.block_table, c.ctx_lens, c.n_shards))
    stack = QFirstStack(layers, caches, Hq, Hkv, max_shards=int(np.max(shards)), scale=SCALE)
    u = block_input(len(ctx), SHAPE.hidden, seed=seed + 999).to(gpu)
    return stack, u


def _state(stack):
    return [(c.k_cache.clone(), c.v_cache.clone(), c.ctx_lens.clone()) for c in stack.caches]


def _restore(stack, saved):
    for c, (k, v, n) in zip(stack.caches, saved):
        c.k_cache.copy_(k)
        c.v_cache.copy_(v)
        c.ctx_lens.copy_(n)


def _same_state(a, b):
    return all(torch.equal(x, y) for sa, sb in zip(a, b) for x, y in zip(sa, sb))


LINEAR_CASES = [  # (M, N, K, prologue, residual, split)
    (1, 2048, 1024, "rms_norm", False, None),     # W_q at Qwen3-0.6B
    (3, 6144, 1024, "rms_norm", False, None),     # W_gate|W_up
    (1, 1024, 3072, "swiglu", True, None),        # W_down + residual
    (5, 2560, 9728, "swiglu", True, None),        # W_down at Qwen3-4B
    (2, 1024, 2048, None, True, None),            # W_o + residual
    (4, 2048, 1024, "rms_norm", False, 1024),     # W_k|W_v into two buffers
    (7, 1001, 264, None, False, None),            # ragged: tail wavefront, partial chunk
    (8, 18, 4104, "rms_norm", True, 5),
    # 4-8 input rows: ragged tiles, residual, split
    (8, 1000, 1024, "rms_norm", True, None),
    (6, 2048, 3072, None, True, None),
    (4, 4096, 2560, "rms_norm", False, 2048),
    (5, 17, 96, "rms_norm", False, 9),
]


@pytest.mark.parametrize("M,N,K,pro,res,split", LINEAR_CASES)
def test_linear_matches_oracle(gpu, M, N, K, pro, res, split):
    """out = W . P(x) (+ residual): each output within the bf16 values around the exact result
    widened by the fp32 accumulation bound (K/64 + 32 roundings of 2^-24 on the absolute sum)."""
    gen = torch.Generator().manual_seed(M * 7919 + N * 31 + K)
    xk = 2 * K if pro == "swiglu" else K
    scales = torch.tensor([1.0, 1e-3, 30.0, 1.0, 3.0, 0.5, 1.0, 2.0])[:M, None]
    x = (torch.randn(M, xk, generator=gen) * scales).to(torch.bfloat16)
    w = (torch.randn(N, K, generator=gen) / K ** 0.5).to(torch.bfloat16)
    g = (torch.rand(K, generator=gen) + 0.5).to(torch.bfloat16)
    r = torch.randn(M, N, generator=gen).to(torch.bfloat16) if res else None
    say(f"[stage] linear M={M} N={N} K={K} prologue={pro} residual={res} split={split}")
    got = qf.linear(x.to(gpu), w.to(gpu), pro, g.to(gpu) if pro == "rms_norm" else None, 1e-6,
                    residual=None if r is None else r.to(gpu), split=split)
    torch.cuda.synchronize()
    got = torch.cat(got, 1) if split is not None else got
    xd, wd = x.double().numpy(), w.double().numpy()
    if pro == "rms_norm":
        px = oracle.rms_norm(xd, g.double().numpy(), 1e-6)
    elif pro == "swiglu":
        px = oracle.swiglu(xd[:, :K], xd[:, K:])
    else:
        px = xd
    ref = px @ wd.T
    bound = np.abs(px) @ np.abs(wd).T
    if r is not None:
        ref = ref + r.double().numpy()
        bound = bound + np.abs(r.double().numpy())
    delta = (K / 64 + 32) * 2.0 ** -24 * bound
    lo, _ = bf16_neighbours(ref - delta)
    _, hi = bf16_neighbours(ref + delta)
    out = got.double().cpu().numpy()
    ok = (out >= lo) & (out <= hi)
    assert ok.all(), (np.argwhere(~ok)[:4], out[~ok][:4], ref[~ok][:4])


@pytest.mark.parametrize("M,I,K", [(1, 3072, 1024), (3, 9728, 2560), (8, 24, 520),
                                   (8, 3072, 1024), (4, 52, 64)])
def test_linear_glu_output_matches_oracle(gpu, M, I, K):
    """Rows of W alternating gate and up, output silu(gate) * up from the fp32 sums: within the
    bf16 values around the exact activation widened by the accumulation bounds of both sums
    carried through silu (|silu'| <= 1.1) and the product."""
    gen = torch.Generator().manual_seed(M * 31 + I + K)
    x = (torch.randn(M, K, generator=gen) * 2).to(torch.bfloat16)
    wg = (torch.randn(I, K, generator=gen) / K ** 0.5).to(torch.bfloat16)
    wu = (torch.randn(I, K, generator=gen) / K ** 0.5).to(torch.bfloat16)
    g = (torch.rand(K, generator=gen) + 0.5).to(torch.bfloat16)
    w = torch.stack([wg, wu], 1).reshape(2 * I, K).contiguous()
    say(f"[stage] linear GLU M={M} I={I} K={K}")
    got = qf.linear(x.to(gpu), w.to(gpu), "rms_norm", g.to(gpu), 1e-6, glu_out=True)
    torch.cuda.synchronize()
    assert tuple(got.shape) == (M, I)
    px = oracle.rms_norm(x.double().numpy(), g.double().numpy(), 1e-6)
    G, U = px @ wg.double().numpy().T, px @ wu.double().numpy().T
    ref = oracle.swiglu(G, U)
    eps = (K / 64 + 32) * 2.0 ** -24
    dG = eps * (np.abs(px) @ np.abs(wg.double().numpy()).T)
    dU = eps * (np.abs(px) @ np.abs(wu.double().numpy()).T)
    delta = 1.1 * np.abs(U) * dG + np.abs(oracle.silu(G)) * dU + 1e-6 * np.abs(ref)
    lo, _ = bf16_neighbours(ref - delta)
    _, hi = bf16_neighbours(ref + delta)
    out = got.double().cpu().numpy()
    ok = (out >= lo) & (out <= hi)
    assert ok.all(), (np.argwhere(~ok)[:4], out[~ok][:4], ref[~ok][:4])


BESIDE_CASES = [  # (B, Hq, Hkv, ctx, shards, M, N, K, prologue, GLU output)
    (1, 16, 8, [4608], 8, 1, 6144, 1024, "rms_norm", False),       # chunked sweep (few units)
    (1, 16, 8, [4608], 32, 1, 6144, 1024, "rms_norm", True),       # the stage's shared launch
    (4, 32, 8, [900, 17, 3000, 0], 3, 4, 2056, 512, "rms_norm", False),
    (3, 8, 8, [300, 1, 77], 2, 8, 1001, 264, None, False),
    (3, 8, 8, [300, 1, 77], 2, 8, 1002, 264, None, True),
    (2, 64, 8, [5000, 40], [6, 1], 3, 1024, 3072, "swiglu", False),
    (2, 16, 4, [128, 2048], 64, 2, 520, 1024, "rms_norm", False),  # unchunked: many units
    (24, 16, 8, [3999], 4, 2, 1024, 1024, "rms_norm", False),      # the split call's deep buffers
]


@pytest.mark.parametrize("B,Hq,Hkv,ctx,shards,M,N,K,pro,glu", BESIDE_CASES)
def test_beside_equals_the_two_calls_bitwise(gpu, B, Hq, Hkv, ctx, shards, M, N, K, pro, glu):
    case = make_case(B, Hq, Hkv, ctx, shards, seed=800 + Hq + M, device=gpu)
    gen = torch.Generator(device=gpu).manual_seed(801 + N)
    x = torch.randn(M, 2 * K if pro == "swiglu" else K, generator=gen, device=gpu).to(torch.bfloat16)
    w = (torch.randn(N, K, generator=gen, device=gpu) / K ** 0.5).to(torch.bfloat16)
    g = (torch.rand(K, generator=gen, device=gpu) + 0.5).to(torch.bfloat16)
    res = torch.randn(M, N, generator=gen, device=gpu).to(torch.bfloat16)
    S = case.max_shards
    outs = []
    for together in (False, True):
        po = torch.full((B, S, Hq, 128), float("nan"), device=gpu)
        pl = torch.full((B, S, Hq), float("nan"), device=gpu)
        y = torch.full((M, N // 2 if glu else N), float("nan"), device=gpu).to(torch.bfloat16)
        lin = dict(x=x, w=w, prologue=pro, gain=g if pro == "rms_norm" else None,
                   residual=None if glu else res, out=y, glu_out=glu)
        say(f"[stage] beside B={B} G={Hq // Hkv} M={M} N={N} K={K} together={together}")
        sweep = (case.q, case.k_cache, case.v_cache, case.block_table, case.ctx_lens,
                 case.n_shards)
        if together:
            qf.attn_decode_split_beside(*sweep, lin, max_shards=S, scale=case.scale, part_out=po,
                                        part_lse=pl)
        else:
            qf.attn_decode_split(*sweep, max_shards=S, scale=case.scale, part_out=po, part_lse=pl)
            qf.linear(**lin)
        torch.cuda.synchronize()
        outs.append((po.view(torch.int32).clone(), pl.view(torch.int32).clone(),
                     y.view(torch.int16).clone()))
    for a, b in zip(*outs):
        assert torch.equal(a, b)


def test_all_modes_equal_the_serial_order_bitwise(gpu):
    stack, u = _build(gpu)
    saved = _state(stack)
    ys, states = {}, {}
    for mode in ("serial", "streams", "fused"):
        say(f"[stage] mode {mode}, eager, 2 steps")
        _restore(stack, saved)
        outs = [stack.step(u, mode=mode).clone() for _ in range(2)]
        torch.cuda.synchronize()
        ys[mode], states[mode] = outs, _state(stack)
    for mode in ("streams", "fused"):
        for a, b in zip(ys["serial"], ys[mode]):
            assert torch.equal(a, b), mode
        assert _same_state(states["serial"], states[mode]), mode
    assert int(stack.status.item()) == 0
    assert stack.caches[0].ctx_lens.tolist() == (CTX + 2).tolist()


def test_more_than_eight_requests_in_all_modes(gpu):
    """Ten requests: every product runs in blocks of 8 rows and only the first block of
    W_gate|W_up shares the sweep's launch; the three orders still agree bitwise."""
    ctx = [300, 2, 0, 45, 1000, 17, 64, 5, 129, 700]
    stack, u = _build(gpu, L=2, seed=650, ctx=ctx, shards=[3, 1, 1, 2, 4, 1, 1, 1, 2, 3])
    saved = _state(stack)
    ys, states = {}, {}
    for mode in ("serial", "streams", "fused"):
        say(f"[stage] ten requests, mode {mode}")
        _restore(stack, saved)
        ys[mode] = stack.step(u, mode=mode).clone()
        torch.cuda.synchronize()
        states[mode] = _state(stack)
    for mode in ("streams", "fused"):
        assert torch.equal(ys["serial"], ys[mode]), mode
        assert _same_state(states["serial"], states[mode]), mode
    assert torch.isfinite(ys["serial"].float()).all()


@pytest.mark.parametrize("mode", ["fused", "streams", "serial"])
def test_graph_replays_equal_eager(gpu, mode):
    stack, u = _build(gpu, seed=600)
    saved = _state(stack)
    y_eager = stack.step(u, mode=mode).clone()
    torch.cuda.synchronize()
    after = _state(stack)
    _restore(stack, saved)
    side = torch.cuda.Stream()                       # warm-up on a side stream, then capture
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):
        stack.step(u, mode=mode)
    torch.cuda.current_stream().wait_stream(side)
    torch.cuda.synchronize()
    say(f"[stage] capture mode={mode}")
    graph, y = stack.capture(u, mode=mode)
    other = "serial" if mode != "serial" else "fused"
    for r in range(3):
        _restore(stack, saved)
        torch.cuda.synchronize()
        graph.replay()
        torch.cuda.synchronize()
        say(f"[stage] replay {r}")
        assert torch.equal(y, y_eager), r
        assert _same_state(_state(stack), after), r
        stack.step(u, mode=other)                    # eager work between replays
        torch.cuda.synchronize()


def _host_cache(c):
    return (c.k_cache.double().cpu().numpy(), c.v_cache.double().cpu().numpy(),
            c.block_table.cpu().numpy(), c.ctx_lens.cpu().numpy())


def _rel(a, b):
    return float(np.linalg.norm(a - b) / np.linalg.norm(b))


def _np(t):
    return t.double().cpu().numpy()


def _product_gate(label, out, px, w, residual=None):
    """out = W . px (+ residual) stored in bf16: within the bf16 values around the exact result
    widened by the fp32 accumulation bound (K/64 + 32 roundings of 2^-24 on the absolute sum)."""
    K = px.shape[1]
    ref = px @ w.T
    bound = np.abs(px) @ np.abs(w).T
    if residual is not None:
        ref = ref + residual
        bound = bound + np.abs(residual)
    delta = (K / 64 + 32) * 2.0 ** -24 * bound
    lo, _ = bf16_neighbours(ref - delta)
    _, hi = bf16_neighbours(ref + delta)
    ok = (out >= lo) & (out <= hi)
    assert ok.all(), (label, np.argwhere(~ok)[:4], out[~ok][:4], ref[~ok][:4])


def _glu_gate(label, out, px, wg, wu):
    """silu(W_gate px) * (W_up px) stored in bf16, both sums in fp32 (the bound carried through
    silu, |silu'| <= 1.1, and the product)."""
    K = px.shape[1]
    G, U = px @ wg.T, px @ wu.T
    ref = oracle.swiglu(G, U)
    eps = (K / 64 + 32) * 2.0 ** -24
    delta = (1.1 * np.abs(U) * eps * (np.abs(px) @ np.abs(wg).T)
             + np.abs(oracle.silu(G)) * eps * (np.abs(px) @ np.abs(wu).T) + 1e-6 * np.abs(ref))
    lo, _ = bf16_neighbours(ref - delta)
    _, hi = bf16_neighbours(ref + delta)
    ok = (out >= lo) & (out <= hi)
    assert ok.all(), (label, np.argwhere(~ok)[:4], out[~ok][:4], ref[~ok][:4])


def test_step_matches_the_block_oracle(gpu):
    from oracle.attention import attend, gather_rows
    from parity import PART_REL
    stack, u = _build(gpu, seed=700)
    Hq, Hkv = SHAPE.n_q_heads, SHAPE.n_kv_heads
    G = Hq // Hkv
    host = [_host_cache(c) for c in stack.caches]
    w = [{k: t.double().cpu().numpy() for k, t in lw.items() if k not in ("w_gu", "w_kv")}
         for lw in stack.layers]
    u0 = _np(u)
    B = u0.shape[0]
    say("[stage] first block, product by product, on the GPU's own inputs")
    y0 = torch.empty_like(u)
    stack.block(0, u, y0, mode="fused")
    torch.cuda.synchronize()
    w0 = w[0]
    q, act, z = _np(stack.q).reshape(B, -1), _np(stack.act), _np(stack.z)
    k, v, attn = _np(stack.k), _np(stack.v), _np(stack.attn)
    _product_gate("q", q, oracle.rms_norm(u0, w0["g1"]), w0["w_q"])
    _glu_gate("act", act, oracle.rms_norm(u0, w0["g2"]), w0["w_gate"], w0["w_up"])
    _product_gate("z", z, act, w0["w_down"], residual=u0)
    hz = oracle.rms_norm(z, w0["g1"])
    _product_gate("k", k.reshape(B, -1), hz, w0["w_k"])
    _product_gate("v", v.reshape(B, -1), hz, w0["w_v"])
    kc, vc, bt, n = host[0]
    lse = stack.lse.cpu().numpy()
    for b in range(B):
        for h in range(Hq):
            g = h // G
            K = np.concatenate([gather_rows(kc, bt[b], g, int(n[b]), 16), k[b, g][None]])
            V = np.concatenate([gather_rows(vc, bt[b], g, int(n[b]), 16), v[b, g][None]])
            O, L = attend(q.reshape(B, Hq, -1)[b, h], K, V, SCALE)
            delta = PART_REL * float(np.max(np.abs(O)))
            lo, _ = bf16_neighbours(O - delta)
            _, hi = bf16_neighbours(O + delta)
            assert np.all((attn[b, h] >= lo) & (attn[b, h] <= hi)), (b, h)
            assert abs(lse[b, h] - L) <= 1e-5 * max(1.0, abs(L)), (b, h)
    _product_gate("y", _np(y0), attn.reshape(B, -1), w0["w_o"], residual=z)
    # the empty cache (request 2): attention is the current value exactly
    torch.testing.assert_close(stack.attn[2], stack.v[2].repeat_interleave(G, 0), rtol=0, atol=0)

    for c, (kk, vv, btt, nn) in zip(stack.caches, host):   # undo the append, run the whole step
        c.k_cache.copy_(torch.from_numpy(kk).to(torch.bfloat16))
        c.v_cache.copy_(torch.from_numpy(vv).to(torch.bfloat16))
        c.ctx_lens.copy_(torch.from_numpy(nn))
    say("[stage] whole step vs the oracle with the same seven bf16 stores")
    y = _np(stack.step(u, mode="fused"))
    x, x64 = u0, u0
    for l in range(SHAPE.layers):
        x = oracle.qfirst_block(x, w[l], *host[l], Hq, Hkv, SCALE, bf16_stores=True)["y"]
        x64 = oracle.qfirst_block(x64, w[l], *host[l], Hq, Hkv, SCALE)["y"]
    e = _rel(y, x)
    say(f"[stage] whole step: {e:.2e} relative (L2) from the bf16-store oracle, "
        f"{_rel(y, x64):.2e} from the exact one")
    assert e <= 2e-3, e
