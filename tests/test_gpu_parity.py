"""GPU parity: the HIP path (through the C ABI) against the fp64 oracle on the same seeded bytes.

Small cases run the oracle on every output; they span several pages per wavefront, ragged last
pages, empty shards and requests, every supported group size, the identity and permuted block
tables and the chunked (sub-shard) path.  Full-size cases run each registered workload's layer at
its real shape, in the launch configuration the bench times, and check sampled (request, head)
outputs one by one.
"""

import numpy as np
import pytest
import torch

import paper_2608_15473_amd as qf
import oracle
from parity import check, host_arrays, oracle_ref, run_gpu, say
from workloads import WORKLOADS, make_case, workload_case

pytestmark = pytest.mark.gpu


def _run(case, label, pairs=None):
    say(f"[parity] {label}: B,Hq,Hkv,D={case.shape} ctx={case.ctx_lens.tolist()[:8]} "
        f"S={case.n_shards.tolist()[:8]} S_max={case.max_shards}")
    got = run_gpu(case)
    ref = oracle_ref(case, pairs)
    worst = check(case, got, ref, pairs, label)
    say(f"[parity] {label}: ok {worst}")
    return got, ref


@pytest.mark.parametrize("G", [1, 2, 4, 8])
def test_group_sizes_ragged(gpu, G):
    case = make_case(3, 2 * G, 2, [1000, 37, 517], [5, 2, 3], seed=100 + G, device=gpu)
    _run(case, f"G={G} ragged")


@pytest.mark.parametrize("G", [1, 2, 4, 8])
def test_deep_buffers_ragged(gpu, G):
    """The deep-buffer sweep (short shards of 16+ pages, no sub-shard chunks: NBUF 5 at G <= 2,
    3 at G = 4) on ragged requests with partial last pages and shards of every length the split
    rule gives, every output checked."""
    rng = np.random.default_rng(190 + G)
    ctx = rng.integers(1, 3001, size=48)
    ctx[:4] = [3000, 16, 17, 255]
    shards = rng.integers(1, 9, size=48)
    case = make_case(48, 2 * G, 2, ctx, shards, seed=190 + G, max_shards=8, device=gpu)
    assert qf.workspace_size(qf.make_desc(case.q, case.k_cache, case.block_table,
                                          case.max_shards, case.scale)) == 0      # no chunks
    _run(case, f"deep buffers G={G}")


def test_empty_requests_and_more_shards_than_pages(gpu):
    case = make_case(4, 16, 8, [0, 16, 33, 100], [3, 4, 7, 1], seed=110, max_shards=8,
                     device=gpu)
    got, _ = _run(case, "empty/short")
    assert np.all(got["part_lse"][0] == -np.inf)
    assert np.all(got["out_bits"][0] == 0) and np.all(got["lse"][0] == -np.inf)
    # slots past S_b are -inf even though the buffers were NaN-poisoned before the call
    assert np.all(got["part_lse"][3, 1:] == -np.inf)


def test_identity_table(gpu):
    case = make_case(2, 16, 8, [700, 300], [3, 2], seed=120, table="identity", device=gpu)
    got = run_gpu(case)
    case_null = make_case(2, 16, 8, [700, 300], [3, 2], seed=120, table="identity", device=gpu)
    case_null.block_table = None
    got_null = run_gpu(case_null)
    for key in ("part_lse", "out_bits", "lse"):
        assert np.array_equal(got[key], got_null[key], equal_nan=True)
    ref = oracle_ref(case)
    check(case, got, ref, label="identity")


def test_chunked_path(gpu):
    """Few (request, KV head, shard) units and long shards: the sweep splits every shard into
    chunks and merges them before returning the per-shard pairs."""
    case = make_case(1, 8, 2, [20011], [3], seed=130, max_shards=3, device=gpu)
    desc = qf.make_desc(case.q, case.k_cache, case.block_table, case.max_shards, case.scale)
    assert qf.workspace_size(desc) > 0
    _run(case, "chunked")


def test_ragged_batch_long_shards(gpu):
    """A ragged batch whose shards are long enough (>= 128 pages at capacity) for the sweep to
    dispatch its units largest-shard-first; includes empty requests and partial last pages."""
    rng = np.random.default_rng(180)
    n = np.rint(np.exp(rng.uniform(np.log(16), np.log(8192), size=64))).astype(int)
    n[[3, 17]] = 0
    S = np.maximum(1, -(-n // 4096))
    case = make_case(64, 16, 8, n, S, seed=180, max_shards=4, max_pages=512, device=gpu)
    order = np.argsort(n)
    pairs = [(int(order[i]), h) for i, h in [(0, 0), (10, 5), (40, 9), (62, 14), (63, 15)]]
    got, ref = _run(case, "ragged long shards", pairs)
    assert np.all(got["part_lse"][[3, 17]] == -np.inf)


def test_physical_page_placement_is_bitwise_irrelevant(gpu):
    """The same logical cache stored contiguously or scattered over a permuted pool gives
    bitwise identical results."""
    a = make_case(2, 16, 8, [900, 555], [4, 3], seed=140, table="identity", device=gpu)
    b = make_case(2, 16, 8, [900, 555], [4, 3], seed=141, device=gpu)
    # move a's logical pages to b's physical placement
    bt = b.block_table.long()
    P = a.k_cache.shape[0] // 2
    k = torch.zeros_like(b.k_cache)
    v = torch.zeros_like(b.v_cache)
    for r in range(2):
        n_pg = -(-int(a.ctx_lens[r]) // 16)
        k[bt[r, :n_pg]] = a.k_cache[r * P: r * P + n_pg]
        v[bt[r, :n_pg]] = a.v_cache[r * P: r * P + n_pg]
    b.k_cache, b.v_cache, b.q = k, v, a.q
    ga, gb = run_gpu(a), run_gpu(b)
    for key in ("part_out", "part_lse", "out_bits", "lse"):
        assert np.array_equal(ga[key], gb[key], equal_nan=True), key


@pytest.mark.parametrize("G", [2, 4, 8])
def test_garbage_past_the_last_position_is_never_used(gpu, G):
    """The slots of a request's last page past its last position hold no position: NaN and Inf
    there (in K and in V) must leave every result bitwise as it is with finite values there, in
    the unchunked and chunked sweeps, both dispatch orders, and the one-launch decode."""
    shapes = [  # (batch, ctx_lens, n_shards, max_shards)
        (3, [1000, 37, 517], [5, 2, 3], None),          # short shards
        (1, [4607], 8, None),                           # chunked, one request
        (2, [70001, 9], [1, 1], None),                  # chunked, one long unit
        # 768 units of at least 128 pages at full capacity: the long-shard order, unchunked
        (24, [33001] + [997 * (k + 1) + 3 for k in range(23)], [16] + [1 + k % 4 for k in range(23)],
         16),
    ]
    for i, (B, ctx, S, smax) in enumerate(shapes):
        clean = make_case(B, 2 * G, 2, ctx, S, seed=300 + i, max_shards=smax, device=gpu)
        dirty = make_case(B, 2 * G, 2, ctx, S, seed=300 + i, max_shards=smax, device=gpu)
        bt = dirty.block_table.long()
        for b in range(B):
            n = int(dirty.ctx_lens[b])
            if n % 16 == 0:
                continue
            last = int(bt[b, n // 16])
            dirty.k_cache[last, :, n % 16:] = float("nan")
            dirty.v_cache[last, :, n % 16:] = float("nan")
            dirty.v_cache[last, :, 15] = float("inf")
            dirty.k_cache[last, 0, 15] = float("-inf")
        say(f"[parity] garbage past the last position: G={G} shape {i}")
        ga, gb = run_gpu(clean), run_gpu(dirty)
        for key in ("part_out", "part_lse", "out_bits", "lse"):
            assert np.array_equal(ga[key], gb[key], equal_nan=True), (i, key)
        args = lambda c: (c.q, c.k_cache, c.v_cache, c.block_table, c.ctx_lens, c.n_shards)
        o1, l1 = qf.attn_decode(*args(clean), max_shards=clean.max_shards, scale=clean.scale)
        o2, l2 = qf.attn_decode(*args(dirty), max_shards=dirty.max_shards, scale=dirty.scale)
        torch.cuda.synchronize()
        assert torch.equal(_bits(o1), _bits(o2)) and torch.equal(_bits(l1), _bits(l2)), i
        assert bool(torch.isfinite(l2).all()), i


def test_repeat_calls_are_deterministic(gpu):
    case = make_case(2, 32, 8, [3000, 1234], [6, 2], seed=150, device=gpu)
    g1, g2 = run_gpu(case), run_gpu(case)
    for key in ("part_out", "part_lse", "out_bits", "lse"):
        assert np.array_equal(g1[key], g2[key], equal_nan=True), key


@pytest.mark.parametrize("hq", [16, 32, 64], ids=["G2", "G4", "G8"])
def test_planted_large_logits_stay_finite(gpu, hq):
    """Logits near 85 over many positions: ln Z ~ 91 > ln(FLT_MAX), where a naive fp32 sum of
    exponentials overflows; every output must stay finite and match the oracle (both score paths:
    the VALU dot products at G = 2, the matrix cores at G = 4 and 8)."""
    case = make_case(1, hq, 8, [30000], [4], seed=160, planted=(400, 84.0, 86.0), device=gpu)
    got, ref = _run(case, f"planted ~85, {hq} query heads")
    assert np.all(np.isfinite(got["out"])) and np.all(np.isfinite(got["lse"]))
    assert np.all(ref["lse"] > 88.8)


@pytest.mark.parametrize("G", [2, 4, 8])
def test_nan_inputs_reach_exactly_the_heads_that_read_them(gpu, G):
    """A NaN is data, not masked (one reading of the paper's silence): a NaN query element poisons
    that head only; a NaN key element poisons every head of its KV group (through the score); a
    NaN value element poisons that dim of the group's outputs and leaves ln Z finite.  Every
    other output stays bitwise as in the clean run, and the NaN pattern is the oracle's."""
    ctx, S = [700, 300], [3, 2]
    clean = make_case(2, 2 * G, 2, ctx, S, seed=330 + G, device=gpu)
    base = run_gpu(clean)
    bt = clean.block_table.long()
    cases = {
        "q": lambda c: c.q.__setitem__((0, 1, 17), float("nan")),
        "k": lambda c: c.k_cache.__setitem__((int(bt[1, 5]), 1, 3, 40), float("nan")),
        "v": lambda c: c.v_cache.__setitem__((int(bt[0, 20]), 0, 9, 77), float("nan")),
    }
    for what, poison in cases.items():
        dirty = make_case(2, 2 * G, 2, ctx, S, seed=330 + G, device=gpu)
        poison(dirty)
        say(f"[parity] NaN in {what}, G={G}")
        got = run_gpu(dirty)
        a = host_arrays(dirty)
        ro, rl = oracle.decode_unsplit(a["q"], a["k"], a["v"], a["bt"], a["ctx"], dirty.scale)
        assert np.array_equal(np.isnan(got["out"]), np.isnan(ro)), what
        assert np.array_equal(np.isnan(got["lse"]), np.isnan(rl)), what
        hit = np.isnan(ro)
        assert hit.any(), what
        if what == "q":
            assert hit[0, 1].all() and hit.sum() == 128
        elif what == "k":
            assert hit[1, G:2 * G].all() and hit.sum() == 128 * G
        else:
            assert hit[0, :G, 77].all() and hit.sum() == G and np.isfinite(got["lse"]).all()
        keep = ~hit
        assert np.array_equal(got["out_bits"][keep], base["out_bits"][keep]), what
        keep_l = ~np.isnan(rl)
        assert np.array_equal(got["lse"][keep_l], base["lse"][keep_l]), what


def test_planted_secondary_reading(gpu):
    """The paper's number read the other way: ln Z ~ 85 with logits near 79."""
    case = make_case(1, 16, 8, [30000], [4], seed=161, planted=(400, 78.0, 80.0), device=gpu)
    got, ref = _run(case, "planted ~79")
    assert np.all(np.abs(ref["lse"] - 85.0) < 1.5)


def test_many_shard_slots_and_many_chunks(gpu):
    """Rows of more than 128 slots (the merge's 16-wavefront form): 256 shard slots merged by the
    combine, and one unit of a long cache cut into hundreds of chunks merged into its shard."""
    case = make_case(2, 16, 8, [3000, 70000], [150, 200], seed=175, max_shards=256, device=gpu)
    _run(case, "256 shard slots")
    one = make_case(1, 1, 1, [100000], 1, seed=176, device=gpu)     # one unit: ~780 chunks
    desc = qf.make_desc(one.q, one.k_cache, one.block_table, 1, one.scale)
    assert qf.workspace_size(desc) > 64 * (128 + 1) * 4
    _run(one, "one unit, many chunks")


def test_out_of_range_device_values_poison_lse(gpu):
    """Out-of-range context length, shard count or block-table entry: the kernel clamps (no
    out-of-bounds access) and the affected request's lse becomes NaN; other requests are exact."""
    case = make_case(3, 16, 8, [500, 500, 500], [2, 2, 2], seed=170, device=gpu)
    case.block_table[1, 3] = case.k_cache.shape[0] + 5        # entry past the pool
    case.ctx_lens[2] = 10**6                                  # longer than the table row
    got = run_gpu(case)
    assert np.all(np.isnan(got["lse"][1])) and np.all(np.isnan(got["lse"][2]))
    assert np.all(np.isnan(got["out"][1])) and np.all(np.isnan(got["out"][2]))
    ok = make_case(3, 16, 8, [500, 500, 500], [2, 2, 2], seed=170, device=gpu)
    ref = oracle_ref(ok, pairs=[(0, h) for h in range(16)])
    check(ok, got, ref, pairs=[(0, h) for h in range(16)], label="poison/request0")
    bad_s = make_case(2, 16, 8, [300, 300], [2, 99], seed=171, max_shards=4, device=gpu)
    g2 = run_gpu(bad_s)
    assert np.all(np.isnan(g2["lse"][1])) and np.all(np.isfinite(g2["lse"][0]))
    neg = make_case(2, 16, 8, [300, 40], [1, 1], seed=172, max_shards=3, device=gpu)
    neg.ctx_lens[1] = -5                       # out of range with nothing to read: empty units
    g3 = run_gpu(neg)
    assert np.all(np.isnan(g3["part_lse"][1]))                 # every slot of it, empty ones too
    assert np.all(np.isnan(g3["lse"][1])) and np.all(np.isfinite(g3["lse"][0]))
    assert np.all(g3["part_lse"][0, 1:] == -np.inf)            # a valid request's unused slots


def test_empty_batch(gpu):
    q = torch.zeros(0, 16, 128, dtype=torch.bfloat16, device=gpu)
    k = torch.zeros(1, 8, 16, 128, dtype=torch.bfloat16, device=gpu)
    po, pl = qf.attn_decode_split(q, k, k, None, torch.zeros(0, dtype=torch.int32, device=gpu), 1)
    out, lse = qf.attn_combine(po, pl)
    torch.cuda.synchronize()
    assert out.shape == (0, 16, 128)


def test_combine_selects_empty_slots_and_propagates_nan(gpu):
    B, S, Hq, D = 2, 6, 4, 128
    rng = np.random.default_rng(3)
    po = rng.standard_normal((B, S, Hq, D)).astype(np.float32)
    pl = (rng.standard_normal((B, S, Hq)) * 30 + 50).astype(np.float32)
    pl[0, 2:] = -np.inf
    po[0, 2:] = np.nan                        # garbage behind -inf: never read
    pl[1, :, 0] = -np.inf                     # a fully empty (request, head)
    pl[1, 3, 1] = np.nan                      # a NaN log partition poisons its head
    pl[1, :, 2] = [900.0, 899.0, -np.inf, 100.0, 901.0, -800.0]   # far beyond exp's range
    out, lse = qf.attn_combine(torch.from_numpy(po).to(gpu), torch.from_numpy(pl).to(gpu))
    torch.cuda.synchronize()
    out, lse = out.float().cpu().numpy(), lse.cpu().numpy()
    import oracle
    ro, rl = oracle.combine_max_shifted(np.where(np.isnan(po), 0, po).astype(np.float64),
                                        np.where(np.isnan(pl), -np.inf, pl).astype(np.float64))
    fo, fl = oracle.fold_combine(po.astype(np.float64), pl.astype(np.float64),
                                 rng=np.random.default_rng(0))
    from parity import PART_REL, bf16_neighbours
    for b, h in [(0, 0), (0, 1), (0, 3), (1, 2), (1, 3)]:
        assert abs(lse[b, h] - rl[b, h]) <= 1e-5 * max(1, abs(rl[b, h]))
        # the output gate of every parity test: between the bf16 neighbours of O -/+ 1e-4 max|O|
        O = fo[b, h]
        delta = PART_REL * float(np.max(np.abs(O)))
        lo, _ = bf16_neighbours(O - delta)
        _, hi = bf16_neighbours(O + delta)
        assert np.all((out[b, h] >= lo) & (out[b, h] <= hi)), (b, h)
        assert abs(fl[b, h] - rl[b, h]) < 1e-9 * max(1, abs(rl[b, h]))
    assert np.all(out[1, 0] == 0) and lse[1, 0] == -np.inf
    assert np.all(np.isnan(out[1, 1])) and np.isnan(lse[1, 1])


@pytest.mark.parametrize("live", [5, 16, 24])
def test_combine_bits_do_not_depend_on_appended_empty_slots(gpu, live):
    """Empty slots appended behind the live ones (ln Z = -inf, O garbage) change no bit of the
    merge as long as one round of 16 slots per wavefront covers the row: the workgroup grows from
    1 to 16 wavefronts with the slot count, every wavefront sums the same live slots, and empty
    ones add exact zeros."""
    B, Hq, D = 3, 8, 128
    rng = np.random.default_rng(40 + live)
    po = rng.standard_normal((B, live, Hq, D)).astype(np.float32)
    pl = (rng.standard_normal((B, live, Hq)) * 30 + 50).astype(np.float32)
    pl[1, ::3, 2] = -np.inf                   # some empty slots among the live ones
    ref_out, ref_lse = qf.attn_combine(torch.from_numpy(po).to(gpu), torch.from_numpy(pl).to(gpu))
    for total in sorted({live + 1, 32, 64, 128, 200, 256}):
        if total <= live:
            continue
        po2 = np.full((B, total, Hq, D), np.nan, dtype=np.float32)
        pl2 = np.full((B, total, Hq), -np.inf, dtype=np.float32)
        po2[:, :live], pl2[:, :live] = po, pl
        out, lse = qf.attn_combine(torch.from_numpy(po2).to(gpu), torch.from_numpy(pl2).to(gpu))
        torch.cuda.synchronize()
        assert torch.equal(out.view(torch.int16), ref_out.view(torch.int16)), total
        assert torch.equal(lse.view(torch.int32), ref_lse.view(torch.int32)), total


@pytest.mark.parametrize("slots", [40, 300])
def test_combine_at_the_query_head_limit(gpu, slots):
    """QF_MAX_Q_HEADS query heads, one round of slots (40) and two (300, past 16 wavefronts of 16):
    the merge of a head reads only that head's slots, so every head equals a combine of its own
    8-head slice, bitwise; and one head above the limit is refused before any launch."""
    B, Hq, D = 1, 4096, 128
    g = torch.Generator(device=gpu).manual_seed(300 + slots)
    po = torch.randn(B, slots, Hq, D, generator=g, device=gpu)
    pl = torch.randn(B, slots, Hq, generator=g, device=gpu) * 20 + 40
    pl[:, ::7, 2000:2100] = -float("inf")
    out, lse = qf.attn_combine(po, pl)
    for h0 in (0, 2048, 4088):
        o8, l8 = qf.attn_combine(po[:, :, h0:h0 + 8].contiguous(), pl[:, :, h0:h0 + 8].contiguous())
        torch.cuda.synchronize()
        assert torch.equal(out[:, h0:h0 + 8].view(torch.int16), o8.view(torch.int16)), h0
        assert torch.equal(lse[:, h0:h0 + 8].view(torch.int32), l8.view(torch.int32)), h0
    with pytest.raises(qf.QFError):
        qf.attn_combine(torch.zeros(1, 1, Hq + 1, D, device=gpu),
                        torch.zeros(1, 1, Hq + 1, device=gpu))


# ------------------------------------------------------------------------------------------------
# full-size workloads: one layer at its real shape, sampled outputs
# ------------------------------------------------------------------------------------------------
_SAMPLES = {
    "qwen3-0.6b_b1_n4608_s8": None,                                   # every output
    "qwen3-0.6b_b32_n32768_s64_l28": [(0, 0), (7, 5), (19, 11), (31, 15)],
    "qwen3-4b_b16_n36480_s32_l36": [(0, 0), (5, 13), (15, 31)],
    "qwen3-0.6b_b1_n1m_s16_l28_planted": [(0, 0), (0, 9)],
    "qwen3-4b_ragged_b64": "ragged",
    "qwen3-0.6b_b1_n131072_s2_l28_planted": [(0, 2), (0, 15)],
    "qwen3-32b_b16_n32768_s32_l64": [(0, 0), (6, 29), (15, 63)],
}


@pytest.mark.slow
@pytest.mark.parametrize("name", list(_SAMPLES))
def test_full_size_workload_layer(gpu, name):
    layer = 1 if WORKLOADS[name].layers > 1 else 0
    case = workload_case(name, layer=layer, device=gpu)
    pairs = _SAMPLES[name]
    if pairs == "ragged":
        n = case.ctx_lens.cpu().numpy()
        order = np.argsort(n)
        pairs = [(int(order[0]), 3), (int(order[32]), 17), (int(order[-1]), 30)]
    got, ref = _run(case, f"{name} layer {layer}", pairs)
    got_u = _bench_configuration(case, got, ref, pairs, f"{name} layer {layer}")
    if WORKLOADS[name].planted:
        for g in (got, got_u):
            assert np.all(np.isfinite(g["out"])) and np.all(np.isfinite(g["lse"]))
            assert np.all(g["lse"] > 88.0)
    del case
    torch.cuda.empty_cache()


def _bench_configuration(case, got, ref, pairs, label):
    """The launch configuration the bench times (DecodeStepPlan(fold_chunks=False): the sweep
    leaves sub-shard chunks as slots, one combine merges the max_shards * C of them), gated against
    the same oracle values as the split sweep and combine."""
    args = (case.q, case.k_cache, case.v_cache, case.block_table, case.ctx_lens, case.n_shards)
    plan = qf.DecodeStepPlan(*args, max_shards=case.max_shards, scale=case.scale,
                             fold_chunks=False)
    out, lse = plan()
    torch.cuda.synchronize()
    got_u = dict(got)
    got_u["out"], got_u["lse"] = out.float().cpu().numpy(), lse.cpu().numpy()
    got_u["out_bits"] = out.view(torch.int16).cpu().numpy()
    worst = check(case, got_u, ref, pairs, label + " (bench configuration)")
    say(f"[parity] {label} (bench configuration, {plan.part_lse.shape[1]} slots): ok {worst}")
    del plan
    return got_u


@pytest.mark.slow
@pytest.mark.parametrize("hq,hkv", [(64, 8), (32, 4)], ids=["G8_64q8kv", "G8_32q4kv"])
def test_eight_heads_per_kv_head_long_requests_sampled(gpu, hq, hkv):
    """Eight query heads per KV head (the matrix-core scores with 8-lane broadcasts) on long
    requests (chunked shards, the long-shard dispatch), sampled heads of every KV group; the
    short-shard dispatch at G = 8 is in the small cases above."""
    for B, n, S in [(4, 32768, 8), (1, 300000, 2)]:
        case = make_case(B, hq, hkv, [n] * B, S, seed=870 + hq + B, device=gpu)
        pairs = [(b, (5 * b + 8 * g + b % 8) % hq) for b in range(B) for g in range(hkv)]
        _run(case, f"G=8 {hq}q/{hkv}kv B={B} n={n} S={S}", pairs)
        del case
        torch.cuda.empty_cache()


@pytest.mark.slow
@pytest.mark.parametrize("name", ["qwen3-0.6b_b32_n32768_s64_l28", "qwen3-4b_b16_n36480_s32_l36",
                                  "qwen3-0.6b_b1_n1m_s16_l28_planted",
                                  "qwen3-0.6b_b1_n131072_s2_l28_planted",
                                  "qwen3-32b_b16_n32768_s32_l64"])
def test_full_size_every_layer_sampled(gpu, name):
    """Every layer of the multi-layer workloads, at its real shape: one (request, head) per layer,
    rotating through the batch and the heads."""
    w = WORKLOADS[name]
    for layer in range(w.layers):
        case = workload_case(name, layer=layer, device=gpu)
        B, Hq = case.shape[0], case.shape[1]
        pair = ((7 * layer + 3) % B, (5 * layer + 1) % Hq)
        got, ref = _run(case, f"{name} layer {layer}", [pair])
        got_u = _bench_configuration(case, got, ref, [pair], f"{name} layer {layer}")
        if w.planted:
            for g in (got, got_u):
                assert np.all(np.isfinite(g["out"])) and np.all(g["lse"] > 88.0)
        del case, got, got_u
        torch.cuda.empty_cache()


# ------------------------------------------------------------------------------------------------
# sweep and merge in one launch (qf_attn_decode): bitwise the two calls
# ------------------------------------------------------------------------------------------------
def _bits(t):
    return t.view(torch.int16 if t.dtype == torch.bfloat16 else torch.int32).clone()


def _one_launch_vs_two(case, workspace=None, counters=None):
    """Bitwise the two-launch result (which the oracle gates check) when the shape has no
    sub-shard chunks and at most 64 slots; otherwise the slots are grouped differently: within
    a few fp32 ulp (lse) and one bf16 step (out)."""
    args = (case.q, case.k_cache, case.v_cache, case.block_table, case.ctx_lens, case.n_shards)
    po, pl = qf.attn_decode_split(*args, max_shards=case.max_shards, scale=case.scale)
    out2, lse2 = qf.attn_combine(po, pl)
    out1, lse1 = qf.attn_decode(*args, max_shards=case.max_shards, scale=case.scale,
                                workspace=workspace, counters=counters)
    torch.cuda.synchronize()
    chunked = qf.split_chunks(qf.make_desc(case.q, case.k_cache, case.block_table,
                                           case.max_shards, case.scale)) > 1
    if not chunked and case.max_shards <= 64:
        assert torch.equal(_bits(out1), _bits(out2))
        assert torch.equal(_bits(lse1), _bits(lse2))
    else:
        a, b = lse1.double(), lse2.double()
        same = (a == b) | (torch.isnan(a) & torch.isnan(b))
        assert (same | ((a - b).abs() <= 8 * 2.0 ** -23 * b.abs())).all()
        d = (_bits(out1).int() - _bits(out2).int()).abs()       # adjacent bf16 at most
        assert int(d.max()) <= 1
    return out1, lse1


_UNFOLDED = {  # (batch, Hq, Hkv, ctx_lens, n_shards)
    "unchunked": (3, 16, 8, [1000, 37, 517], [5, 2, 3]),
    "chunked one request": (1, 16, 8, [4607], 8),
    "chunked long units": (2, 16, 8, [70001, 9], [1, 1]),
    "chunked G4": (1, 32, 8, [50000], 2),
    "chunked G8": (1, 64, 8, [40000], 2),
    "chunked empty shards": (3, 16, 8, [0, 16, 30000], [3, 4, 5]),
}


@pytest.mark.parametrize("name", list(_UNFOLDED))
def test_unfolded_sweep_then_combine(gpu, name):
    """The sweep with its sub-shard chunks left as slots (qf_attn_decode_split_unfolded), merged
    by one combine over S * C slots: the oracle's gates, and close to the folded sweep plus
    combine (bitwise when there are no chunks; otherwise the fp32 sums are grouped differently:
    lse within 8 fp32 ulp, out within one bf16 step or 1e-5 of its row's largest magnitude, since
    an element far below that can move by several of its own bf16 steps); empty chunks and the
    chunks of unused shard slots carry -inf; a plan with fold_chunks=False equals it."""
    B, hq, hkv, ctx, S = _UNFOLDED[name]
    case = make_case(B, hq, hkv, ctx, S, seed=880 + len(name), device=gpu)
    args = (case.q, case.k_cache, case.v_cache, case.block_table, case.ctx_lens, case.n_shards)
    C = qf.split_chunks(qf.make_desc(case.q, case.k_cache, case.block_table, case.max_shards,
                                     case.scale))
    assert (C > 1) == (name != "unchunked")
    so = torch.full((B, case.max_shards * C, hq, 128), float("nan"), device=gpu)
    sl = torch.full((B, case.max_shards * C, hq), float("nan"), device=gpu)
    qf.attn_decode_split_unfolded(*args, max_shards=case.max_shards, scale=case.scale,
                                  slot_out=so, slot_lse=sl)
    out_u, lse_u = qf.attn_combine(so, sl)
    plan = qf.DecodeStepPlan(*args, max_shards=case.max_shards, scale=case.scale,
                             fold_chunks=False)
    out_p, lse_p = plan()
    folded = run_gpu(case)
    torch.cuda.synchronize()
    say(f"[parity] unfolded sweep: {name}, {C} chunks per shard")
    assert torch.equal(_bits(out_p), _bits(out_u)) and torch.equal(_bits(lse_p), _bits(lse_u))
    lse_f = torch.from_numpy(folded["lse"]).to(gpu)
    bits_f = torch.from_numpy(folded["out_bits"]).to(gpu)
    if C == 1:
        assert torch.equal(_bits(lse_u), _bits(lse_f)) and torch.equal(_bits(out_u), bits_f)
    else:
        a, b = lse_u.double(), lse_f.double()
        same = (a == b) | (torch.isnan(a) & torch.isnan(b))
        assert (same | ((a - b).abs() <= 8 * 2.0 ** -23 * b.abs())).all()
        fo, uo = bits_f.view(torch.bfloat16).float(), out_u.float()
        row = fo.abs().amax(dim=-1, keepdim=True)
        assert ((uo - fo).abs() <= torch.maximum(fo.abs() * 2.0 ** -7, row * 1e-5)).all()
    # every slot written: -inf where a chunk or a shard slot holds no position
    lse_slots = sl.cpu().numpy()
    assert not np.isnan(lse_slots).any()
    n_sh = case.n_shards.cpu().numpy()
    for b in range(B):
        assert np.all(lse_slots[b, n_sh[b] * C:] == -np.inf)
        if int(case.ctx_lens[b]) == 0:
            assert np.all(lse_slots[b] == -np.inf)
    ref = oracle_ref(case)
    got = dict(folded)
    got["out"], got["lse"] = out_u.float().cpu().numpy(), lse_u.cpu().numpy()
    got["out_bits"] = _bits(out_u).cpu().numpy()
    check(case, got, ref, label=f"unfolded {name}")


_ONE_LAUNCH = {
    "G1": dict(batch=3, n_q_heads=2, n_kv_heads=2, ctx_lens=[1000, 37, 517], n_shards=[5, 2, 3]),
    "G2": dict(batch=3, n_q_heads=4, n_kv_heads=2, ctx_lens=[1000, 37, 517], n_shards=[5, 2, 3]),
    "G4": dict(batch=3, n_q_heads=8, n_kv_heads=2, ctx_lens=[1000, 37, 517], n_shards=[5, 2, 3]),
    "G8": dict(batch=3, n_q_heads=16, n_kv_heads=2, ctx_lens=[1000, 37, 517], n_shards=[5, 2, 3]),
    "chunked": dict(batch=1, n_q_heads=16, n_kv_heads=8, ctx_lens=[4608], n_shards=8),
    "empty": dict(batch=4, n_q_heads=16, n_kv_heads=8, ctx_lens=[0, 16, 33, 100],
                  n_shards=[3, 4, 7, 1], max_shards=8),
    "slots256": dict(batch=2, n_q_heads=16, n_kv_heads=8, ctx_lens=[3000, 70000],
                     n_shards=[150, 200], max_shards=256),
}


@pytest.mark.parametrize("name", list(_ONE_LAUNCH))
def test_one_launch_decode_equals_split_then_combine(gpu, name):
    kw = dict(_ONE_LAUNCH[name])
    case = make_case(kw.pop("batch"), kw.pop("n_q_heads"), kw.pop("n_kv_heads"),
                     kw.pop("ctx_lens"), kw.pop("n_shards"), seed=180, device=gpu, **kw)
    say(f"[parity] one launch vs two: {name}")
    out, lse = _one_launch_vs_two(case)
    ref = oracle_ref(case)
    check(case, run_gpu(case), ref, label=f"one launch {name}")


def test_one_launch_counters_are_left_at_zero_and_poison_propagates(gpu):
    """One workspace and one counter array across calls with different shapes (every call must
    leave the counters it used at zero, whatever the previous call wrote to the workspace),
    including a request whose device inputs are out of range."""
    cases = [make_case(3, 16, 8, [500, 500, 500], [2, 2, 2], seed=181, device=gpu),
             make_case(1, 16, 8, [4608], 8, seed=182, device=gpu),
             make_case(2, 32, 8, [900, 7000], [3, 9], seed=183, max_shards=16, device=gpu)]
    cases[0].ctx_lens[2] = 10 ** 6                           # out of range: NaN for request 2
    need = max(qf.decode_workspace_size(qf.make_desc(c.q, c.k_cache, c.block_table,
                                                     c.max_shards, c.scale)) for c in cases)
    ws = torch.empty(need, dtype=torch.uint8, device=gpu)
    counters = torch.zeros(64, dtype=torch.int32, device=gpu)
    for rep in range(2):
        for i, c in enumerate(cases):
            say(f"[parity] shared workspace and counters: call {rep}.{i}")
            out, lse = _one_launch_vs_two(c, workspace=ws, counters=counters)
            assert int(counters.abs().sum().item()) == 0
            if i == 0:
                assert torch.isnan(lse[2]).all() and torch.isfinite(lse[:2]).all()


@pytest.mark.slow
def test_one_launch_full_size_headline_layer(gpu):
    case = workload_case("qwen3-0.6b_b32_n32768_s64_l28", layer=3, device=gpu)
    say("[parity] one launch vs two: headline layer 3")
    _one_launch_vs_two(case)
    del case
    torch.cuda.empty_cache()


@pytest.mark.slow
def test_maximum_sizes(gpu):
    """The sweep's largest chunking (one unit of a 2^20-position cache: one chunk per resident
    workgroup, at most 1,024, merged into one shard) and a large grid (4,096 requests of short
    contexts: 32,768 units), on sampled pairs."""
    one = make_case(1, 1, 1, [1 << 20], 1, seed=190, device=gpu)
    desc = qf.make_desc(one.q, one.k_cache, one.block_table, 1, one.scale)
    ws = qf.workspace_size(desc)
    state = (128 + 1) * 4                                            # one chunk's (O, ln Z)
    assert ws % state == 0 and 256 <= ws // state <= 1024, ws
    _run(one, f"one unit, 2^20 positions, {ws // state} chunks")
    del one
    n = np.random.default_rng(191).integers(0, 64, size=4096)
    many = make_case(4096, 16, 8, n, 1, seed=192, device=gpu)
    pairs = [(0, 0), (1000, 7), (2047, 15), (4095, 3)] + [(int(b), 5) for b in np.where(n == 0)[0][:2]]
    _run(many, "4096 requests", pairs)
    del many
    torch.cuda.empty_cache()



@pytest.mark.parametrize("name,kw", [
    ("many units", dict(batch=3, ctx_lens=[1000, 37, 517], n_shards=[5, 2, 3])),
    ("chunked", dict(batch=1, ctx_lens=[4607], n_shards=8)),       # the plan owns a workspace
])
def test_decode_step_plan_equals_the_calls(gpu, name, kw):
    """DecodeStepPlan: bitwise the two calls, after other allocations have come and gone (the
    buffers it allocated are kept), and with its inputs changed in place between calls."""
    import gc
    case = make_case(kw["batch"], 16, 8, kw["ctx_lens"], kw["n_shards"], seed=330, device=gpu)
    args = (case.q, case.k_cache, case.v_cache, case.block_table, case.ctx_lens, case.n_shards)
    plan = qf.DecodeStepPlan(*args, max_shards=case.max_shards, scale=case.scale)
    gc.collect()
    junk = [torch.full((1 << 20,), float("nan"), device=gpu) for _ in range(8)]   # reuse bait
    say(f"[parity] decode-step plan: {name}")
    for _ in range(2):
        out1, lse1 = plan()
        out1, lse1 = out1.clone(), lse1.clone()
        po, pl = qf.attn_decode_split(*args, max_shards=case.max_shards, scale=case.scale)
        out2, lse2 = qf.attn_combine(po, pl)
        torch.cuda.synchronize()
        assert torch.equal(_bits(out1), _bits(out2)) and torch.equal(_bits(lse1), _bits(lse2))
        case.ctx_lens[0] -= 5                                       # in place: the plan sees it
        case.q.mul_(-1)
    del junk


def test_position_sharding_over_two_sweeps(gpu):
    """Position sharding as it would run over two devices (one GPU stands in for both): each
    sweep sees only its half of every request's pages (its own block-table rows and context
    length), the two sets of shard pairs are concatenated along the slot axis, and one combine
    merges them (§5: any partition, any order). Gated against the oracle's unsplit attention and
    within a few ulp of the one-sweep result."""
    from parity import LSE_REL, PART_REL, bf16_neighbours
    case = make_case(3, 16, 8, [5000, 3333, 17], [4, 3, 1], seed=340, device=gpu)
    B, Hq, Hkv, D = case.shape
    bt = case.block_table
    ctx = case.ctx_lens.long()
    pages = (ctx + 15) // 16
    cut = pages // 2                                   # first device: pages [0, cut)
    n1 = torch.minimum(cut * 16, ctx)
    parts = []
    for lo, n in ((torch.zeros_like(cut), n1), (cut, ctx - n1)):
        rows = torch.full_like(bt, -1)
        for b in range(B):
            m = int((n[b] + 15) // 16)
            rows[b, :m] = bt[b, int(lo[b]):int(lo[b]) + m]
        po, pl = qf.attn_decode_split(case.q, case.k_cache, case.v_cache, rows,
                                      n.to(torch.int32), 2, max_shards=2, scale=case.scale)
        parts.append((po, pl))
    po = torch.cat([parts[0][0], parts[1][0]], dim=1).contiguous()
    pl = torch.cat([parts[0][1], parts[1][1]], dim=1).contiguous()
    out2, lse2 = qf.attn_combine(po, pl)
    po1, pl1 = qf.attn_decode_split(case.q, case.k_cache, case.v_cache, case.block_table,
                                    case.ctx_lens, case.n_shards, max_shards=case.max_shards,
                                    scale=case.scale)
    out1, lse1 = qf.attn_combine(po1, pl1)
    torch.cuda.synchronize()
    say("[parity] position sharding over two sweeps")
    ref = oracle_ref(case)
    o2, l2 = out2.float().cpu().numpy(), lse2.cpu().numpy()
    for b in range(B):
        for h in range(Hq):
            O, L = ref["out"][b, h], ref["lse"][b, h]
            assert abs(l2[b, h] - L) <= LSE_REL * max(1.0, abs(L)), (b, h)
            delta = PART_REL * float(np.max(np.abs(O)))
            lo_, _ = bf16_neighbours(O - delta)
            _, hi_ = bf16_neighbours(O + delta)
            assert np.all((o2[b, h] >= lo_) & (o2[b, h] <= hi_)), (b, h)
    a, c = lse1.double(), lse2.double()
    assert ((a - c).abs() <= 8 * 2.0 ** -23 * a.abs()).all()
    assert int((_bits(out1).int() - _bits(out2).int()).abs().max()) <= 1
