"""GPU parity of ragged batches with long shards against the fp64 oracle.

Shapes with many (request, shard, KV head) units whose shards are long (128+ pages per shard at full
capacity) are swept longest shard first, one workgroup per unit: the split sweep ranks the
(request, shard) pairs by length and deals their units to the XCDs in its workspace before it
starts, the unfolded sweep (no workspace) takes them by shard index, descending.  Every output of every case is checked:
per-shard partials and the combined result, at every group size, including requests with no
positions, partial last pages, more shards than pages, very little work in all, one long request
next to many short ones, out-of-range device values, the unfolded sweep followed by the combine
(bitwise the ranked sweep's result), and the sweep sharing its launch with a product."""

import numpy as np
import pytest
import torch

import paper_2608_15473_amd as qf
from parity import check, oracle_ref, run_gpu, say
from workloads import make_case

pytestmark = pytest.mark.gpu


def _desc(case):
    return qf.make_desc(case.q, case.k_cache, case.block_table, case.max_shards, case.scale)


def _is_long_shard_shape(case):
    """128+ pages per shard at full capacity and at least one full set of resident workgroups'
    worth of units (no sub-shard chunks); the split sweep then takes its units in a ranked
    order, one int32 per workgroup index in its workspace."""
    B, S = case.q.shape[0], case.max_shards
    long = -(-case.block_table.shape[1] // S) >= 128
    desc = _desc(case)
    ranked = qf.workspace_size(desc) == 4 * (-(-B * S * case.k_cache.shape[1] // 8) * 8)
    return long and qf.split_chunks(desc) == 1 and ranked


def _ragged(batch, seed, n_max=40000):
    rng = np.random.default_rng(seed)
    n = np.rint(np.exp(rng.uniform(np.log(8), np.log(n_max), size=batch))).astype(int)
    n[[1, 7]] = 0                       # no positions
    n[2] = 1                            # one position
    n[3] = 16 * 37 + 5                  # partial last page
    S = np.maximum(1, -(-n // 4096))
    S[4] = 16                           # more shards than it has pages for some of them
    n[4] = 16 * 9 + 3
    return n, S


@pytest.mark.parametrize("G", [1, 2, 4, 8])
def test_long_shards_every_group_size(gpu, G):
    n, S = _ragged(48, 400 + G)
    case = make_case(48, 2 * G, 2, n, S, seed=400 + G, max_shards=16, max_pages=2560, device=gpu)
    assert _is_long_shard_shape(case), "the shape must be a long-shard, unchunked one"
    say(f"[long shards] G={G}: {int(n.sum())} positions")
    got = run_gpu(case)
    ref = oracle_ref(case)
    worst = check(case, got, ref, label=f"long shards G={G}")
    say(f"[long shards] G={G}: ok {worst}")
    assert np.all(got["part_lse"][[1, 7]] == -np.inf)
    for b in range(48):
        assert np.all(got["part_lse"][b, S[b]:] == -np.inf)


def test_long_shards_three_kv_heads(gpu):
    """A KV head count that is not a power of two (the dispatch order's unit arithmetic then
    divides instead of shifting), every output checked."""
    n, S = _ragged(48, 470)
    case = make_case(48, 6, 3, n, S, seed=470, max_shards=16, max_pages=2560, device=gpu)
    assert _is_long_shard_shape(case)
    say("[long shards] three KV heads")
    got = run_gpu(case)
    check(case, got, oracle_ref(case), label="long shards, 3 KV heads")


def test_long_shards_with_little_work(gpu):
    """Few pages in all (most units empty or of a few pages), and one request whose single shard
    is 100 times longer than the others."""
    n = np.full(64, 40)
    n[5] = 16 * 300 + 7                         # one shard of 301 pages
    S = np.ones(64, dtype=int)
    S[9] = 3
    case = make_case(64, 16, 8, n, S, seed=420, max_shards=4, max_pages=1024, device=gpu)
    assert _is_long_shard_shape(case)
    say("[long shards] little work")
    got = run_gpu(case)
    check(case, got, oracle_ref(case), label="long shards, little work")


def test_long_shards_poison_out_of_range_requests(gpu):
    n, S = _ragged(48, 430)
    case = make_case(48, 16, 2, n, S, seed=430, max_shards=16, max_pages=2560, device=gpu)
    assert _is_long_shard_shape(case)
    heavy = int(np.argmax(n))
    case.block_table[heavy, 5] = case.k_cache.shape[0] + 3     # entry past the pool
    case.ctx_lens[10] = 10**7                                  # past the table row
    case.n_shards[11] = 999                                    # more shards than slots
    case.ctx_lens[12] = -1
    say("[long shards] poisoned requests")
    got = run_gpu(case)
    for b in (heavy, 10, 11, 12):
        assert np.all(np.isnan(got["lse"][b])), b
    assert np.all(np.isnan(got["part_lse"][12]))
    good = [b for b in range(48) if b not in (heavy, 10, 11, 12)]
    pairs = [(b, h) for b in good[::5] for h in (0, 7)]
    ref = make_case(48, 16, 2, n, S, seed=430, max_shards=16, max_pages=2560, device=gpu)
    check(ref, got, oracle_ref(ref, pairs), pairs, label="long shards, poison/others")


def test_long_shards_unfolded_then_combine(gpu):
    """The unfolded sweep followed by the combine (no chunks here, so the slots are the shards)
    equals the split sweep followed by the combine bitwise, and the oracle's gates."""
    n, S = _ragged(48, 440)
    case = make_case(48, 32, 8, n, S, seed=440, max_shards=16, max_pages=2560, device=gpu)
    assert _is_long_shard_shape(case)
    C = qf.split_chunks(_desc(case))
    args = (case.q, case.k_cache, case.v_cache, case.block_table, case.ctx_lens, case.n_shards)
    so = torch.full((48, 16 * C, 32, 128), float("nan"), device=gpu)
    sl = torch.full((48, 16 * C, 32), float("nan"), device=gpu)
    qf.attn_decode_split_unfolded(*args, max_shards=16, scale=case.scale, slot_out=so,
                                  slot_lse=sl)
    out, lse = qf.attn_combine(so, sl)
    folded = run_gpu(case)
    torch.cuda.synchronize()
    say("[long shards] unfolded")
    assert not torch.isnan(sl).any()
    assert np.array_equal(lse.cpu().numpy(), folded["lse"])
    assert np.array_equal(out.view(torch.int16).cpu().numpy(), folded["out_bits"])
    got = dict(folded)
    got["out"], got["lse"] = out.float().cpu().numpy(), lse.cpu().numpy()
    got["out_bits"] = out.view(torch.int16).cpu().numpy()
    check(case, got, oracle_ref(case), label="long shards, unfolded")


def test_long_shards_are_deterministic(gpu):
    n, S = _ragged(48, 450)
    case = make_case(48, 16, 2, n, S, seed=450, max_shards=16, max_pages=2560, device=gpu)
    a, b = run_gpu(case), run_gpu(case)
    for key in ("part_out", "part_lse", "out_bits", "lse"):
        assert np.array_equal(a[key], b[key], equal_nan=True), key


def test_long_shards_beside_a_product_equal_the_two_calls_bitwise(gpu):
    """The sweep sharing one launch with a product (qf_attn_decode_split_beside, which ranks the
    shards like the split sweep) gives bitwise the split sweep's and the product's outputs."""
    n, S = _ragged(48, 460)
    case = make_case(48, 4, 2, n, S, seed=460, max_shards=16, max_pages=2560, device=gpu)
    assert _is_long_shard_shape(case)
    args = (case.q, case.k_cache, case.v_cache, case.block_table, case.ctx_lens, case.n_shards)
    gen = torch.Generator(device=gpu).manual_seed(461)
    M, N, K = 2, 1024, 1024
    x = torch.randn(M, K, generator=gen, device=gpu).to(torch.bfloat16)
    w = (torch.randn(N, K, generator=gen, device=gpu) / K ** 0.5).to(torch.bfloat16)
    g = (torch.rand(K, generator=gen, device=gpu) + 0.5).to(torch.bfloat16)
    outs = []
    for together in (False, True):
        po = torch.full((48, 16, 4, 128), float("nan"), device=gpu)
        pl = torch.full((48, 16, 4), float("nan"), device=gpu)
        y = torch.full((M, N), float("nan"), device=gpu).to(torch.bfloat16)
        lin = dict(x=x, w=w, prologue="rms_norm", gain=g, out=y)
        say(f"[long shards] beside, together={together}")
        if together:
            qf.attn_decode_split_beside(*args, lin, max_shards=16, scale=case.scale, part_out=po,
                                        part_lse=pl)
        else:
            qf.attn_decode_split(*args, max_shards=16, scale=case.scale, part_out=po, part_lse=pl)
            qf.linear(**lin)
        torch.cuda.synchronize()
        outs.append((po.view(torch.int32).clone(), pl.view(torch.int32).clone(),
                     y.view(torch.int16).clone()))
    for a, b in zip(*outs):
        assert torch.equal(a, b)
    assert not torch.isnan(outs[1][1].view(torch.float32)).any()


def test_long_shards_plan_replayed_from_a_graph(gpu):
    """The ordering kernel and the sweep and combine of a plan, captured in a HIP graph: every
    replay (with eager work on other buffers between replays) equals the eager call bitwise."""
    n, S = _ragged(48, 480)
    case = make_case(48, 16, 8, n, S, seed=480, max_shards=16, max_pages=2560, device=gpu)
    assert _is_long_shard_shape(case)
    args = (case.q, case.k_cache, case.v_cache, case.block_table, case.ctx_lens, case.n_shards)
    st = torch.cuda.Stream()                         # the plan's stream, captured below
    plan = qf.DecodeStepPlan(*args, max_shards=16, scale=case.scale, fold_chunks=False,
                             stream=st.cuda_stream)
    torch.cuda.synchronize()
    with torch.cuda.stream(st):
        out, lse = plan()
    torch.cuda.synchronize()
    eager = (out.view(torch.int16).clone(), lse.view(torch.int32).clone(),
             plan.part_lse.view(torch.int32).clone())
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph, stream=st):
        plan.split()
        plan.combine()
    other = make_case(4, 16, 8, [3000, 17, 0, 900], [2, 1, 1, 3], seed=481, device=gpu)
    for r in range(3):
        plan.out.fill_(float("nan"))
        plan.part_lse.fill_(float("nan"))
        graph.replay()
        torch.cuda.synchronize()
        say(f"[long shards] graph replay {r}")
        assert torch.equal(plan.out.view(torch.int16), eager[0])
        assert torch.equal(plan.lse.view(torch.int32), eager[1])
        assert torch.equal(plan.part_lse.view(torch.int32), eager[2])
        run_gpu(other)                                   # eager work between replays


def _shard_pages(n, S, s, max_pages, max_shards):
    """Pages of shard s of a request with n positions cut into S shards (the header's split
    rule; out-of-range values clamped as the kernels clamp them)."""
    n = min(max(int(n), 0), max_pages * 16)
    S = min(max(int(S), 1), max_shards)
    pages = -(-n // 16)
    per = -(-pages // S)
    return min((s + 1) * per, pages) - min(s * per, pages) if s < S else 0


def test_long_shards_dispatch_order(gpu):
    """The dispatch order the ordering kernel leaves in the workspace (white box): workgroup
    index i runs unit order[i] on XCD i % 8; every unit appears exactly once and the rest is -1;
    along each XCD's queue the live units come first, longest shard first (to the kernel's
    length buckets of 2^shift pages), then the empty ones; and the even XCDs get at least as many
    live units as the odd ones."""
    n, S = _ragged(48, 490)
    B, Hkv, smax, maxp = 48, 8, 16, 2560
    case = make_case(B, 16, Hkv, n, S, seed=490, max_shards=smax, max_pages=maxp, device=gpu)
    assert _is_long_shard_shape(case)
    desc = _desc(case)
    units = B * smax * Hkv
    ws = torch.empty(qf.workspace_size(desc), dtype=torch.uint8, device=gpu)
    qf.attn_decode_split(case.q, case.k_cache, case.v_cache, case.block_table, case.ctx_lens,
                         case.n_shards, max_shards=smax, scale=case.scale, workspace=ws)
    torch.cuda.synchronize()
    order = ws.view(torch.int32).cpu().numpy()
    say("[long shards] dispatch order")
    assert len(order) == -(-units // 8) * 8
    live_vals = order[order >= 0]
    assert np.all(order >= -1) and np.array_equal(np.sort(live_vals), np.arange(units))
    shift = 0
    while (maxp >> shift) >= 1024:
        shift += 1
    ctx = case.ctx_lens.cpu().numpy()
    ns = case.n_shards.cpu().numpy()

    def pages(u):                       # unit u = pair * Hkv + g, pair r: request r % B,
        r = u // Hkv                    # shard smax - 1 - r // B
        return _shard_pages(ctx[r % B], ns[r % B], smax - 1 - r // B, maxp, smax)

    live_per_xcd = []
    for x in range(8):
        q = [int(u) for u in order[x::8] if u >= 0]
        p = np.array([pages(u) for u in q])
        live = int(np.sum(p > 0))
        assert np.all(p[:live] > 0) and np.all(p[live:] == 0), x      # live units first
        assert np.all(np.diff(p[:live] >> shift) <= 0), x              # longest first
        live_per_xcd.append(live)
    assert sum(live_per_xcd) == sum(1 for u in range(units) if pages(u) > 0)
    assert min(live_per_xcd[0::2]) >= max(live_per_xcd[1::2]), live_per_xcd


@pytest.mark.parametrize("B", [256, 257])
def test_long_shards_at_the_ordering_limit(gpu, B):
    """8,192 (request, shard) pairs, the most the ordering kernel ranks (its LDS holds one int32
    per pair), and one request more, swept in the plain order: the workspace says which, and the
    sampled outputs meet the oracle's gates either way."""
    rng = np.random.default_rng(500 + B)
    n = np.rint(np.exp(rng.uniform(np.log(16), np.log(20000), size=B))).astype(int)
    n[:3] = [0, 1, 16 * 4096 // 2 + 7]
    S = np.maximum(1, -(-n // 4096))
    case = make_case(B, 4, 2, n, S, seed=500 + B, max_shards=32, max_pages=4096, device=gpu)
    desc = _desc(case)
    assert qf.split_chunks(desc) == 1
    ranked = qf.workspace_size(desc) > 0
    assert ranked == (B * 32 <= 8192)
    say(f"[long shards] {B} requests, {B * 32} pairs, ranked={ranked}")
    got = run_gpu(case)
    order = np.argsort(n)
    pairs = [(int(b), h) for b in (0, 1, 2, int(order[B // 2]), int(order[-1]), B - 1)
             for h in (0, 3)]
    check(case, got, oracle_ref(case, pairs), pairs, label=f"ordering limit B={B}")
    assert np.all(got["part_lse"][0] == -np.inf)
