"""Write-overrun checks: every output of every entry point is written inside its documented
extent and nowhere else.

Each output buffer (partials, slots, merged output and log-sum-exp, workspace, block products) is
carved out of a larger allocation whose margins before and after it hold a byte pattern; after the
call (and a synchronisation) both margins must still hold it.  The cache append must change the
appended position of each (request, KV head) and nothing else of the cache, and ctx_lens only
within the batch.  Shapes: short shards, sub-shard chunks with a workspace, long shards swept
largest first, a request with no positions, and more shard slots than shards."""

import numpy as np
import pytest
import torch

import paper_2608_15473_amd as qf
from parity import say
from workloads import make_case

pytestmark = pytest.mark.gpu

PAD = 4096          # bytes of margin on either side (keeps 16-byte alignment)
PATTERN = 0xA5


class Fenced:
    """A tensor of `shape` and `dtype` in the middle of a byte buffer with patterned margins."""

    def __init__(self, shape, dtype, device):
        n = int(np.prod(shape)) * torch.tensor([], dtype=dtype).element_size()
        self.raw = torch.full((n + 2 * PAD,), PATTERN, dtype=torch.uint8, device=device)
        self.n = n
        self.t = self.raw[PAD:PAD + n].view(dtype).view(shape)

    def intact(self):
        torch.cuda.synchronize()
        head = self.raw[:PAD]
        tail = self.raw[PAD + self.n:]
        return bool((head == PATTERN).all()) and bool((tail == PATTERN).all())


_SHAPES = {  # (batch, Hq, Hkv, ctx_lens, n_shards, max_shards)
    "short shards": (3, 16, 8, [1000, 37, 0], [5, 2, 3], 6),
    "chunked": (1, 32, 8, [40000], 3, 4),
    "long shards": (48, 16, 8, [4096 + 17 * k for k in range(48)], 2, 2),   # 768 units
}


@pytest.mark.parametrize("name", list(_SHAPES))
def test_sweep_and_merge_write_only_their_outputs(gpu, name):
    B, Hq, Hkv, ctx, S, smax = _SHAPES[name]
    case = make_case(B, Hq, Hkv, ctx, S, seed=990 + len(name), max_shards=smax, device=gpu)
    args = (case.q, case.k_cache, case.v_cache, case.block_table, case.ctx_lens, case.n_shards)
    D = 128
    desc = qf.make_desc(case.q, case.k_cache, case.block_table, smax, case.scale)
    need = qf.workspace_size(desc)
    C = qf.split_chunks(desc)
    say(f"[canary] {name}: chunks {C}, workspace {need} B")

    po, pl = Fenced((B, smax, Hq, D), torch.float32, gpu), Fenced((B, smax, Hq), torch.float32, gpu)
    ws = Fenced((max(need, 16),), torch.uint8, gpu)
    qf.attn_decode_split(*args, max_shards=smax, scale=case.scale, part_out=po.t, part_lse=pl.t,
                         workspace=ws.t if need else None)
    assert po.intact() and pl.intact() and ws.intact()

    out, lse = Fenced((B, Hq, D), torch.bfloat16, gpu), Fenced((B, Hq), torch.float32, gpu)
    qf.attn_combine(po.t, pl.t, out=out.t, lse=lse.t)
    assert out.intact() and lse.intact()

    so, sl = Fenced((B, smax * C, Hq, D), torch.float32, gpu), Fenced((B, smax * C, Hq),
                                                                      torch.float32, gpu)
    qf.attn_decode_split_unfolded(*args, max_shards=smax, scale=case.scale, slot_out=so.t,
                                  slot_lse=sl.t)
    assert so.intact() and sl.intact()

    o1, l1 = Fenced((B, Hq, D), torch.bfloat16, gpu), Fenced((B, Hq), torch.float32, gpu)
    dws = Fenced((max(qf.decode_workspace_size(desc), 16),), torch.uint8, gpu)
    cnt = Fenced((B * Hkv,), torch.int32, gpu)
    cnt.t.zero_()
    qf.attn_decode(*args, max_shards=smax, scale=case.scale, out=o1.t, lse=l1.t, workspace=dws.t,
                   counters=cnt.t)
    assert o1.intact() and l1.intact() and dws.intact() and cnt.intact()
    assert bool((cnt.t == 0).all())                        # counters left at zero

    o2, l2 = Fenced((B, Hq, D), torch.bfloat16, gpu), Fenced((B, Hq), torch.float32, gpu)
    qf.attn_decode_noalloc(*args, max_shards=smax, scale=case.scale, out=o2.t, lse=l2.t)
    assert o2.intact() and l2.intact()


def test_fold_and_append_write_only_the_appended_position(gpu):
    B, Hq, Hkv, D = 4, 16, 8, 128
    case = make_case(B, Hq, Hkv, [700 + 16, 1 + 16, 0 + 16, 33 + 16], [3, 1, 2, 4], seed=997,
                     max_shards=4, device=gpu)
    case.ctx_lens -= 16                                    # room for the appended position
    n0 = case.ctx_lens.clone()
    S = case.max_shards
    po, pl = qf.attn_decode_split(case.q, case.k_cache, case.v_cache, case.block_table,
                                  case.ctx_lens, case.n_shards, max_shards=S, scale=case.scale)
    gen = torch.Generator(device=gpu).manual_seed(998)
    k_new = torch.randn(B, Hkv, D, generator=gen, device=gpu).to(torch.bfloat16)
    v_new = torch.randn(B, Hkv, D, generator=gen, device=gpu).to(torch.bfloat16)
    k_before, v_before = case.k_cache.clone(), case.v_cache.clone()
    lens = Fenced((B,), torch.int32, gpu)
    lens.t.copy_(case.ctx_lens)
    status = Fenced((1,), torch.int32, gpu)
    status.t.zero_()
    out, lse = Fenced((B, Hq, D), torch.bfloat16, gpu), Fenced((B, Hq), torch.float32, gpu)
    say("[canary] fold + append")
    qf.attn_combine_current_append(po, pl, case.q, k_new, v_new, case.k_cache, case.v_cache,
                                   case.block_table, lens.t, scale=case.scale, out=out.t,
                                   lse=lse.t, status=status.t)
    assert out.intact() and lse.intact() and lens.intact() and status.intact()
    assert torch.equal(lens.t, n0 + 1) and int(status.t[0]) == 0
    # the cache: exactly the appended slot of every (request, KV head) changed
    changed = (case.k_cache != k_before).any(-1) | (case.v_cache != v_before).any(-1)
    expect = torch.zeros_like(changed)
    for b in range(B):
        n = int(n0[b])
        page = int(case.block_table[b, n // 16])
        expect[page, :, n % 16] = True
    assert torch.equal(changed & ~expect, torch.zeros_like(changed))
    for b in range(B):
        n = int(n0[b])
        page = int(case.block_table[b, n // 16])
        assert torch.equal(case.k_cache[page, :, n % 16], k_new[b])
        assert torch.equal(case.v_cache[page, :, n % 16], v_new[b])


@pytest.mark.parametrize("M,N,K,pro,split,glu", [(3, 1000, 264, "rms_norm", None, False),
                                                 (8, 520, 1024, "rms_norm", 200, False),
                                                 (5, 1002, 264, "rms_norm", None, True),
                                                 (2, 264, 520, "swiglu", None, False)])
def test_products_write_only_their_outputs(gpu, M, N, K, pro, split, glu):
    gen = torch.Generator(device=gpu).manual_seed(M * 1000 + N + K)
    xk = 2 * K if pro == "swiglu" else K
    x = torch.randn(M, xk, generator=gen, device=gpu).to(torch.bfloat16)
    w = (torch.randn(N, K, generator=gen, device=gpu) / K ** 0.5).to(torch.bfloat16)
    g = (torch.rand(K, generator=gen, device=gpu) + 0.5).to(torch.bfloat16)
    cols = N // 2 if glu else (split if split else N)
    out = Fenced((M, cols), torch.bfloat16, gpu)
    out_b = Fenced((M, N - split), torch.bfloat16, gpu) if split else None
    say(f"[canary] linear M={M} N={N} K={K} {pro} split={split} glu={glu}")
    qf.linear(x, w, pro, g if pro == "rms_norm" else None, 1e-6, out=out.t, split=split,
              out_b=None if out_b is None else out_b.t, glu_out=glu)
    assert out.intact() and (out_b is None or out_b.intact())
