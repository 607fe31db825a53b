"""Pins for the fp64 oracle, against facts that do not come from the oracle itself.

Each test names what fixes the expected value: a closed form, an invariant of softmax attention,
brute force with explicit loops and exactly rounded sums, a library routine that covers a special
case, or a number the paper prints (tests/golden/*.json, each entry with its citation).
"""

import json
import math
import os

import numpy as np
import pytest
import scipy.special
import torch

import oracle
from workloads import HEAD_DIM, PAGE, SCALE, make_case

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def _golden(name):
    with open(os.path.join(GOLDEN, name)) as f:
        return json.load(f)


def _bf16(rng, *shape, std=1.0):
    """Random values that are exactly representable in bf16, as float64."""
    x = torch.from_numpy(rng.standard_normal(shape) * std).to(torch.bfloat16)
    return x.double().numpy()


def _as_np(case):
    return dict(q=case.q.double().numpy(), k_cache=case.k_cache.float().numpy(),
                v_cache=case.v_cache.float().numpy(), block_table=case.block_table.numpy(),
                ctx_lens=case.ctx_lens.numpy(), n_shards=case.n_shards.numpy())


# ------------------------------------------------------------------------------------------------
# closed forms
# ------------------------------------------------------------------------------------------------
def test_identical_keys_give_mean_of_values():
    """Every key equal => every weight equal: O = mean(v_i) and ln Z = s + ln n."""
    rng = np.random.default_rng(1)
    n, D = 37, 16
    q, k = _bf16(rng, D), _bf16(rng, D)
    K = np.tile(k, (n, 1))
    V = _bf16(rng, n, D)
    O, lse = oracle.attend(q, K, V, 0.25)
    s = 0.25 * math.fsum(q[d] * k[d] for d in range(D))
    np.testing.assert_allclose(O, V.mean(axis=0), rtol=0, atol=1e-14)
    assert lse == pytest.approx(s + math.log(n), rel=0, abs=1e-13)


def test_one_entry_cache_puts_all_mass_there():
    """Appendix H: with one cached entry all attention mass is on it: O = v_0, ln Z = s_0."""
    rng = np.random.default_rng(2)
    q, k, v = _bf16(rng, 8), _bf16(rng, 1, 8), _bf16(rng, 1, 8)
    O, lse = oracle.attend(q, k, v, 0.5)
    np.testing.assert_array_equal(O, v[0])
    assert lse == pytest.approx(0.5 * math.fsum(q * k[0]), abs=1e-15)


def test_two_entry_cache_is_a_logistic():
    """Appendix A: two entries form a two-way softmax, a logistic in the score difference.
    Expected value from scipy's expit, a library logistic."""
    rng = np.random.default_rng(3)
    q, K, V = _bf16(rng, 8), _bf16(rng, 2, 8), _bf16(rng, 2, 8)
    s0 = 0.3 * math.fsum(q * K[0])
    s1 = 0.3 * math.fsum(q * K[1])
    O, lse = oracle.attend(q, K, V, 0.3)
    w1 = scipy.special.expit(s1 - s0)
    np.testing.assert_allclose(O, V[0] + w1 * (V[1] - V[0]), rtol=0, atol=1e-14)
    assert lse == pytest.approx(max(s0, s1) + math.log1p(math.exp(-abs(s0 - s1))), abs=1e-14)


def test_one_dominant_key_takes_its_value():
    """A key whose score exceeds every other by 60 nats carries weight 1 - O(e^-60)."""
    rng = np.random.default_rng(4)
    D = 8
    q = np.zeros(D); q[0] = 1.0
    K = _bf16(rng, 50, D) * 0.01
    K[17, 0] = 64.0
    V = _bf16(rng, 50, D)
    O, lse = oracle.attend(q, K, V, 1.0)
    np.testing.assert_allclose(O, V[17], rtol=0, atol=1e-20 + 60 * math.exp(-60))
    assert lse == pytest.approx(64.0, abs=1e-20 + 60 * math.exp(-60))


# ------------------------------------------------------------------------------------------------
# invariants
# ------------------------------------------------------------------------------------------------
def test_shift_invariance():
    """Appendix H: adding c to every score leaves O and moves ln Z by c.  The shift is made
    exactly: an extra coordinate with q = 1 and every key = c/scale."""
    rng = np.random.default_rng(5)
    n, D, scale, c = 300, 32, 0.125, 40.0
    q, K, V = _bf16(rng, D), _bf16(rng, n, D), _bf16(rng, n, D)
    O, lse = oracle.attend(q, K, V, scale)
    q2 = np.append(q, 1.0)
    K2 = np.hstack([K, np.full((n, 1), c / scale)])
    O2, lse2 = oracle.attend(q2, K2, V, scale)
    np.testing.assert_allclose(O2, O, rtol=1e-12, atol=1e-15)
    assert lse2 == pytest.approx(lse + c, rel=1e-14)


def test_convex_hull():
    """O is a convex combination of the values: every coordinate lies between their min and max."""
    rng = np.random.default_rng(6)
    for _ in range(20):
        n = int(rng.integers(1, 200))
        q, K, V = _bf16(rng, 16, std=3), _bf16(rng, n, 16, std=3), _bf16(rng, n, 16)
        O, _ = oracle.attend(q, K, V, 0.25)
        assert np.all(O >= V.min(axis=0) - 1e-12) and np.all(O <= V.max(axis=0) + 1e-12)


def test_position_permutation_invariance():
    rng = np.random.default_rng(7)
    q, K, V = _bf16(rng, 32), _bf16(rng, 500, 32), _bf16(rng, 500, 32)
    O, lse = oracle.attend(q, K, V, 0.2)
    p = rng.permutation(500)
    O2, lse2 = oracle.attend(q, K[p], V[p], 0.2)
    np.testing.assert_allclose(O2, O, rtol=1e-12, atol=1e-15)
    assert lse2 == pytest.approx(lse, rel=1e-14)


def test_shifted_and_unshifted_sums_agree():
    rng = np.random.default_rng(8)
    q, K, V = _bf16(rng, 64), _bf16(rng, 1000, 64), _bf16(rng, 1000, 64)
    O1, l1 = oracle.attend(q, K, V, SCALE)
    O2, l2 = oracle.attend_shifted(q, K, V, SCALE)
    np.testing.assert_allclose(O1, O2, rtol=1e-13, atol=1e-16)
    assert l1 == pytest.approx(l2, rel=1e-13)


def test_large_logits_stay_finite():
    """Scores beyond exp()'s float64 range (> 709) still give a finite (O, ln Z)."""
    rng = np.random.default_rng(9)
    q = np.zeros(4); q[0] = 1
    K = _bf16(rng, 20, 4); K[:, 0] = 800.0 + np.arange(20) * 0.5
    V = _bf16(rng, 20, 4)
    O, lse = oracle.attend(q, K, V, 1.0)
    assert np.all(np.isfinite(O)) and np.isfinite(lse)
    expect = 800.0 + 9.5 + math.log(math.fsum(math.exp(-0.5 * i) for i in range(20)))
    assert lse == pytest.approx(expect, rel=1e-14)


def test_nan_input_reaches_output():
    rng = np.random.default_rng(10)
    q, K, V = _bf16(rng, 8), _bf16(rng, 5, 8), _bf16(rng, 5, 8)
    V[2, 3] = np.nan
    O, lse = oracle.attend(q, K, V, 1.0)
    assert np.isnan(O[3]) and np.isfinite(lse)
    K[1, 0] = np.nan
    O, lse = oracle.attend(q, K, V, 1.0)
    assert np.isnan(lse) and np.all(np.isnan(O))


# ------------------------------------------------------------------------------------------------
# brute force: explicit loops, exactly rounded sums, explicit page walk
# ------------------------------------------------------------------------------------------------
def _brute(q, kc, vc, table, ctx, scale, P):
    B, Hq, D = q.shape
    Hkv = kc.shape[1]
    G = Hq // Hkv
    out = np.zeros((B, Hq, D))
    lse = np.full((B, Hq), -np.inf)
    for b in range(B):
        for h in range(Hq):
            g = h // G
            s, vs = [], []
            for i in range(int(ctx[b])):
                page = int(table[b][i // P])
                k = [float(kc[page, g, i % P, d]) for d in range(D)]
                vs.append([float(vc[page, g, i % P, d]) for d in range(D)])
                s.append(scale * math.fsum(float(q[b, h, d]) * k[d] for d in range(D)))
            if not s:
                continue
            e = [math.exp(x) for x in s]
            Z = math.fsum(e)
            out[b, h] = [math.fsum(e[i] * vs[i][d] for i in range(len(e))) / Z for d in range(D)]
            lse[b, h] = math.log(Z)
    return out, lse


@pytest.mark.parametrize("Hq,Hkv", [(4, 2), (4, 1), (2, 2)])
def test_brute_force_tiny_paged(Hq, Hkv):
    case = make_case(2, Hq, Hkv, [40, 23], [3, 2], seed=11 + Hq + Hkv, head_dim=8,
                     max_pages=4, spare_pages=3)
    a = _as_np(case)
    out_b, lse_b = _brute(a["q"], a["k_cache"], a["v_cache"], a["block_table"], a["ctx_lens"],
                          SCALE, PAGE)
    out, lse = oracle.decode_unsplit(a["q"], a["k_cache"], a["v_cache"], a["block_table"],
                                     a["ctx_lens"], SCALE)
    np.testing.assert_allclose(out, out_b, rtol=0, atol=1e-14)
    np.testing.assert_allclose(lse, lse_b, rtol=1e-14)
    po, pl = oracle.decode_split(a["q"], a["k_cache"], a["v_cache"], a["block_table"],
                                 a["ctx_lens"], a["n_shards"], SCALE, case.max_shards)
    fo, fl = oracle.fold_combine(po, pl, rng=np.random.default_rng(0))
    np.testing.assert_allclose(fo, out_b, rtol=0, atol=1e-14)
    np.testing.assert_allclose(fl, lse_b, rtol=1e-14)


def test_gqa_groups_are_contiguous_heads():
    """Query head h reads KV head h // G.  Distinct data per KV head makes the interleaved
    mapping (h % Hkv) produce a different answer, which brute force rules out."""
    case = make_case(1, 8, 2, [33], [1], seed=12, head_dim=8)
    a = _as_np(case)
    out, _ = oracle.decode_unsplit(a["q"], a["k_cache"], a["v_cache"], a["block_table"],
                                   a["ctx_lens"], SCALE)
    out_b, _ = _brute(a["q"], a["k_cache"], a["v_cache"], a["block_table"], a["ctx_lens"],
                      SCALE, PAGE)
    np.testing.assert_allclose(out, out_b, atol=1e-14)
    # the interleaved alternative would read KV head h % 2 for h = 1 (group 0 -> KV head 1)
    K1 = oracle.gather_rows(a["k_cache"], a["block_table"][0], 1, 33, PAGE)
    V1 = oracle.gather_rows(a["v_cache"], a["block_table"][0], 1, 33, PAGE)
    wrong, _ = oracle.attend(a["q"][0, 1], K1, V1, SCALE)
    assert np.max(np.abs(wrong - out[0, 1])) > 1e-3


# ------------------------------------------------------------------------------------------------
# library special case: the paper's own path (expanded K/V through stock attention)
# ------------------------------------------------------------------------------------------------
def test_matches_torch_sdpa_with_expanded_kv():
    """§2 ran the sweep through PyTorch's attention with K/V expanded to every query head; on the
    CPU in float64 that is an independent implementation of the same definition."""
    case = make_case(3, 8, 2, [100, 1, 257], [2, 1, 5], seed=13, head_dim=HEAD_DIM)
    a = _as_np(case)
    out, lse = oracle.decode_unsplit(a["q"], a["k_cache"], a["v_cache"], a["block_table"],
                                     a["ctx_lens"], SCALE)
    G = 4
    for b in range(3):
        n = int(a["ctx_lens"][b])
        pages = case.block_table[b, : -(-n // PAGE)].long()
        K = case.k_cache[pages].double().permute(1, 0, 2, 3).reshape(2, -1, HEAD_DIM)[:, :n]
        V = case.v_cache[pages].double().permute(1, 0, 2, 3).reshape(2, -1, HEAD_DIM)[:, :n]
        K = K.repeat_interleave(G, dim=0)
        V = V.repeat_interleave(G, dim=0)
        q = case.q[b].double()[:, None, :]
        ref = torch.nn.functional.scaled_dot_product_attention(q, K, V, scale=SCALE)[:, 0]
        np.testing.assert_allclose(out[b], ref.numpy(), rtol=1e-12, atol=1e-14)
        scores = (q @ K.transpose(1, 2))[:, 0] * SCALE
        np.testing.assert_allclose(lse[b], torch.logsumexp(scores, dim=-1).numpy(), rtol=1e-13)


# ------------------------------------------------------------------------------------------------
# split and merge (§5)
# ------------------------------------------------------------------------------------------------
def test_paper_random_four_way_splits():
    """§5: 200 random four-way splits (any partition, any order) agree with one sweep; the paper
    prints agreement to 1.4e-7, a bound the float64 oracle must meet by a wide margin."""
    g = _golden("paper_numerics.json")["random_split_agreement"]
    rng = np.random.default_rng(14)
    n, D = 600, 64
    q, K, V = _bf16(rng, D, std=2), _bf16(rng, n, D), _bf16(rng, n, D)
    O, lse = oracle.attend(q, K, V, SCALE)
    worst = 0.0
    for _ in range(g["trials"]):
        owner = rng.integers(0, g["ways"], size=n)            # non-contiguous, unbalanced
        parts = [oracle.attend(q, K[owner == w], V[owner == w], SCALE) for w in range(g["ways"])]
        order = rng.permutation(g["ways"])
        acc_O, acc_l = np.zeros(D), -np.inf
        for w in order:
            acc_O, acc_l = oracle.merge_pair(parts[w][0], parts[w][1], acc_O, acc_l)
        worst = max(worst, abs(acc_l - lse) / abs(lse),
                    np.linalg.norm(acc_O - O) / np.linalg.norm(O))
    assert worst <= g["agree_to"]
    assert worst < 1e-12


def test_merge_orientation_is_the_weighted_mean():
    """lerp(O_B, O_A, sigma(lnZ_A - lnZ_B)) must weight O_A by Z_A / (Z_A + Z_B)."""
    OA, OB = np.array([1.0, 0.0]), np.array([0.0, 1.0])
    O, l = oracle.merge_pair(OA, math.log(3.0), OB, math.log(1.0))
    np.testing.assert_allclose(O, [0.75, 0.25], atol=1e-15)
    assert l == pytest.approx(math.log(4.0), abs=1e-15)


def test_empty_shard_is_the_identity_and_is_never_read():
    """§5: an empty shard is ln Z = -inf with a vector that may be garbage."""
    junk = np.full(4, np.nan)
    OB = np.array([0.1, -0.2, 0.3, 0.4])
    O, l = oracle.merge_pair(junk, -np.inf, OB, 2.5)
    np.testing.assert_array_equal(O, OB); assert l == 2.5
    O, l = oracle.merge_pair(OB, 2.5, junk, -np.inf)
    np.testing.assert_array_equal(O, OB); assert l == 2.5
    part_out = np.full((1, 5, 1, 4), np.nan)
    part_lse = np.full((1, 5, 1), -np.inf)
    part_out[0, 3, 0] = OB; part_lse[0, 3, 0] = 2.5
    for fn in (lambda: oracle.fold_combine(part_out, part_lse, rng=np.random.default_rng(1)),
               lambda: oracle.combine_max_shifted(part_out, part_lse)):
        o, l = fn()
        np.testing.assert_array_equal(o[0, 0], OB); assert l[0, 0] == 2.5
    part_lse[0, 3, 0] = -np.inf
    for fn in (lambda: oracle.fold_combine(part_out, part_lse),
               lambda: oracle.combine_max_shifted(part_out, part_lse)):
        o, l = fn()
        assert np.all(o == 0) and l[0, 0] == -np.inf


def test_split_partials_merge_to_unsplit_any_order():
    case = make_case(3, 8, 4, [1000, 17, 0], [7, 4, 3], seed=15, head_dim=32, max_shards=9)
    a = _as_np(case)
    out, lse = oracle.decode_unsplit(a["q"], a["k_cache"], a["v_cache"], a["block_table"],
                                     a["ctx_lens"], SCALE)
    po, pl = oracle.decode_split(a["q"], a["k_cache"], a["v_cache"], a["block_table"],
                                 a["ctx_lens"], a["n_shards"], SCALE, 9)
    assert np.all(pl[0, 7:] == -np.inf) and np.all(pl[2] == -np.inf)
    po = np.where(np.isneginf(pl)[..., None], np.nan, po)     # garbage behind every -inf
    for fn in (lambda: oracle.fold_combine(po, pl, rng=np.random.default_rng(2)),
               lambda: oracle.fold_combine(po, pl, order=range(8, -1, -1)),
               lambda: oracle.combine_max_shifted(po, pl)):
        o, l = fn()
        np.testing.assert_allclose(o[:2], out[:2], rtol=1e-12, atol=1e-15)
        np.testing.assert_allclose(l[:2], lse[:2], rtol=1e-13)
        assert np.all(o[2] == 0) and np.all(l[2] == -np.inf)
    assert np.all(out[2] == 0) and np.all(lse[2] == -np.inf)


@pytest.mark.parametrize("n,S", [(0, 1), (0, 4), (1, 1), (1, 3), (16, 2), (17, 2), (80, 4),
                                 (81, 4), (5 * 16, 4), (1000, 64), (4608, 8), (36480, 32)])
def test_shard_ranges_partition_the_cache(n, S):
    r = oracle.shard_ranges(n, S, PAGE)
    assert len(r) == S
    pos = [i for lo, hi in r for i in range(lo, hi)]
    assert pos == list(range(n))                            # disjoint, ordered, covering
    pages = -(-n // PAGE)
    for lo, hi in r:
        if hi > lo:                                         # empty shards sit at the end, lo == n
            assert lo % PAGE == 0 and (hi % PAGE == 0 or hi == n)
        assert hi - lo <= -(-pages // S) * PAGE


# ------------------------------------------------------------------------------------------------
# the paper's numerical claims, in float32
# ------------------------------------------------------------------------------------------------
def test_sigmoid_form_finite_and_matches_library():
    """§2: 1/(1 + e^-x) is finite to +-800 and matches a library sigmoid on [-120, 120].  The
    paper reports bit-identity on its platform; numpy vs torch on this CPU differ by at most one
    float32 rounding."""
    g = _golden("paper_numerics.json")["sigmoid_form"]
    lo, hi = g["library_match_range"]
    x = np.linspace(lo, hi, g["library_match_points"], dtype=np.float32)
    with np.errstate(over="ignore"):
        ours = np.float32(1) / (np.float32(1) + np.exp(-x))
        lib = torch.sigmoid(torch.from_numpy(x)).numpy()
        assert np.max(np.abs(ours - lib)) <= 2.0 ** -23
        big = np.array([-g["finite_to"], g["finite_to"]], dtype=np.float32)
        assert np.all(np.isfinite(np.float32(1) / (np.float32(1) + np.exp(-big))))


def test_exp_form_weight_is_nan_past_89_in_float32():
    """§2: the exponential form e^a / (e^a + e^b) is NaN past 89 in single precision."""
    v = _golden("paper_numerics.json")["exp_form_nan_past"]["value"]
    with np.errstate(over="ignore", invalid="ignore"):
        at = np.float32(v)
        below = np.float32(v - 1)
        assert np.isnan(np.exp(at) / (np.exp(at) + np.exp(at)))
        assert np.exp(below) / (np.exp(below) + np.exp(below)) == np.float32(0.5)


def test_naive_logaddexp_overflows_at_100_in_float32():
    """Appendix E: log(e^a + e^b) overflows at a = b = 100; the stabilised form gives 100 + ln 2."""
    g = _golden("paper_numerics.json")["naive_logaddexp_overflow_at"]
    a, b = np.float32(g["a"]), np.float32(g["b"])
    with np.errstate(over="ignore"):
        assert np.isinf(np.log(np.exp(a) + np.exp(b)))
    o, l = oracle.merge_pair(np.zeros(1), float(a), np.zeros(1), float(b))
    assert l == pytest.approx(100.0 + math.log(2.0), abs=1e-13)


def test_merge_finite_for_log_partitions_far_apart():
    """The sigma form keeps the merge finite for ln Z differences out to +-800 and beyond."""
    OA, OB = np.array([1.0]), np.array([-1.0])
    for la, lb in [(900.0, 100.0), (100.0, 900.0), (1e4, 1e4), (-1e4, 50.0)]:
        O, l = oracle.merge_pair(OA, la, OB, lb)
        assert np.all(np.isfinite(O)) and np.isfinite(l)
        assert l == pytest.approx(np.logaddexp(la, lb))


# ------------------------------------------------------------------------------------------------
# the planted long-context construction and its overflow negative control
# ------------------------------------------------------------------------------------------------
def test_planted_logits_overflow_naive_float32_and_oracle_stays_finite():
    case = make_case(1, 4, 2, [6000], [4], seed=16, planted=(400, 84.0, 86.0))
    a = _as_np(case)
    po, pl = oracle.decode_split(a["q"], a["k_cache"], a["v_cache"], a["block_table"],
                                 a["ctx_lens"], a["n_shards"], SCALE, 4)
    out, lse = oracle.decode_unsplit(a["q"], a["k_cache"], a["v_cache"], a["block_table"],
                                     a["ctx_lens"], SCALE)
    assert np.all(np.isfinite(out)) and np.all(np.isfinite(lse))
    assert np.all(lse >= 88.8)                    # ln Z above ln(FLT_MAX) = 88.72
    for h in range(4):
        K = oracle.gather_rows(a["k_cache"], a["block_table"][0], h // 2, 6000, PAGE)
        s = SCALE * (K @ a["q"][0, h])
        assert 83.0 <= s.max() <= 87.0
        with np.errstate(over="ignore"):
            assert np.isinf(np.sum(np.exp(s.astype(np.float32)), dtype=np.float32))
    fo, fl = oracle.fold_combine(po, pl, rng=np.random.default_rng(3))
    np.testing.assert_allclose(fo, out, rtol=1e-11, atol=1e-14)
    np.testing.assert_allclose(fl, lse, rtol=1e-14)


# ------------------------------------------------------------------------------------------------
# the current token: fold and append (§2, Appendix A)
# ------------------------------------------------------------------------------------------------
def _with_current(case_np, k_new, v_new):
    """Attention over the cache plus the current token, by appending it and sweeping n + 1
    positions with the plain definition (an independent path to the fold)."""
    kc, vc = oracle.append_kv(case_np["k_cache"], case_np["v_cache"], case_np["block_table"],
                              case_np["ctx_lens"], k_new, v_new)
    return oracle.decode_unsplit(case_np["q"], kc, vc, case_np["block_table"],
                                 case_np["ctx_lens"] + 1, SCALE)


def test_fold_equals_attention_over_cache_plus_current():
    # pages are allocated for n + 1 positions; the cache then holds n of them
    case = make_case(3, 8, 2, [101, 2, 1], [3, 1, 1], seed=20, max_pages=8, head_dim=32)
    case.ctx_lens -= 1
    a = _as_np(case)
    rng = np.random.default_rng(21)
    k_new, v_new = _bf16(rng, 3, 2, 32), _bf16(rng, 3, 2, 32)
    O, lse = oracle.decode_unsplit(a["q"], a["k_cache"], a["v_cache"], a["block_table"],
                                   a["ctx_lens"], SCALE)
    fo, fl = oracle.fold_current(O, lse, a["q"], k_new, v_new, SCALE)
    ro, rl = _with_current(a, k_new, v_new)
    np.testing.assert_allclose(fo, ro, rtol=1e-12, atol=1e-14)
    np.testing.assert_allclose(fl, rl, rtol=1e-13)
    # empty cache (request 2): the result is the current token alone
    for h in range(8):
        np.testing.assert_array_equal(fo[2, h], v_new[2, h // 4])
        assert fl[2, h] == pytest.approx(SCALE * math.fsum(a["q"][2, h] * k_new[2, h // 4]))


@pytest.mark.parametrize("gap", [-120.0, -30.0, -9.7, 0.0, 9.7, 30.0, 120.0])
def test_fold_handles_either_sign_of_the_gap(gap):
    """Appendix E: s_jj may exceed lse_<j (short caches), so the fold must work for both signs.
    Expected weights from scipy's expit; the lse from the exactly rounded two-term sum."""
    rng = np.random.default_rng(22)
    D = 16
    O_prev = _bf16(rng, 1, 1, D)
    q = np.zeros((1, 1, D)); q[0, 0, 0] = 1.0
    lse_prev = np.array([[5.0]])
    k = np.zeros((1, 1, D)); k[0, 0, 0] = (5.0 + gap) / 0.25
    v = _bf16(rng, 1, 1, D)
    fo, fl = oracle.fold_current(O_prev, lse_prev, q, k, v, 0.25)
    w_cur = scipy.special.expit(gap)                       # weight of the current token
    np.testing.assert_allclose(fo[0, 0], (1 - w_cur) * O_prev[0, 0] + w_cur * v[0, 0],
                               rtol=1e-13, atol=1e-15)
    m = max(5.0, 5.0 + gap)
    assert fl[0, 0] == pytest.approx(m + math.log(math.fsum([math.exp(5.0 - m),
                                                             math.exp(5.0 + gap - m)])), rel=1e-14)


def test_append_writes_only_the_new_slot():
    case = make_case(2, 4, 2, [18, 32], [1, 1], seed=23, max_pages=4, head_dim=8)
    case.ctx_lens -= 1
    a = _as_np(case)
    rng = np.random.default_rng(24)
    k_new, v_new = _bf16(rng, 2, 2, 8), _bf16(rng, 2, 2, 8)
    kc, vc = oracle.append_kv(a["k_cache"], a["v_cache"], a["block_table"], a["ctx_lens"],
                              k_new, v_new)
    changed = np.argwhere(np.any(kc != a["k_cache"], axis=-1))
    want = {(int(a["block_table"][b, n // PAGE]), g, n % PAGE)
            for b, n in enumerate(a["ctx_lens"]) for g in range(2)}
    assert {tuple(map(int, x)) for x in changed} <= want
    for b, n in enumerate(a["ctx_lens"]):
        page = a["block_table"][b, n // PAGE]
        np.testing.assert_array_equal(kc[page, :, n % PAGE], k_new[b])
        np.testing.assert_array_equal(vc[page, :, n % PAGE], v_new[b])
    bad = a["block_table"].copy()
    bad[0, 1] = -1
    with pytest.raises(ValueError):
        oracle.append_kv(a["k_cache"], a["v_cache"], bad, a["ctx_lens"], k_new, v_new)
