"""The seeded generators and workload shapes, pinned to the paper's printed sizing."""

import json
import os

import numpy as np
import torch

import oracle
from workloads import (HEAD_DIM, PAGE, WORKLOADS, kv_bytes_per_position, make_case,
                       ragged_lengths, workload_case)

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def _golden():
    with open(os.path.join(GOLDEN, "paper_sizing.json")) as f:
        return json.load(f)


def test_kv_bytes_match_the_papers_sizing():
    """§3/§4: 4.1 KB per cached position per layer; 112 / 144 KB per token; 107 / 137 GB at 1M."""
    g = _golden()
    small = WORKLOADS["qwen3-0.6b_b32_n32768_s64_l28"]
    big = WORKLOADS["qwen3-4b_b16_n36480_s32_l36"]
    per_pos = kv_bytes_per_position(small.n_kv_heads)
    assert round(per_pos / 1000, 1) == g["kv_per_position_per_layer_kB"]["value"]
    assert kv_bytes_per_position(big.n_kv_heads) == per_pos
    assert per_pos * small.layers / 1024 == g["kv_per_token_KB"]["qwen3-0.6b"]
    assert per_pos * big.layers / 1024 == g["kv_per_token_KB"]["qwen3-4b"]
    assert round(per_pos * small.layers * 1e6 / 2**30) == g["kv_at_one_million_GB"]["qwen3-0.6b"]
    assert round(per_pos * big.layers * 1e6 / 2**30) == g["kv_at_one_million_GB"]["qwen3-4b"]


def test_crossover_contexts_match_the_ffn_bytes():
    """§3: at the crossover context one layer's KV bytes equal its FFN weight bytes (19 / 149 MB)."""
    g = _golden()
    per_pos = kv_bytes_per_position(8)
    for model in ("qwen3-0.6b", "qwen3-4b"):
        ffn = per_pos * g["crossover_positions"][model]
        assert round(ffn / 1e6) == g["ffn_MB"][model]
    assert WORKLOADS["qwen3-0.6b_b1_n4608_s8"].ctx == g["crossover_positions"]["qwen3-0.6b"]
    assert WORKLOADS["qwen3-4b_b16_n36480_s32_l36"].ctx == g["crossover_positions"]["qwen3-4b"]


def test_same_seed_same_bytes_and_different_layers_differ():
    a = make_case(2, 4, 2, [50, 70], [2, 3], seed=7)
    b = make_case(2, 4, 2, [50, 70], [2, 3], seed=7)
    c = make_case(2, 4, 2, [50, 70], [2, 3], seed=8)
    for x, y in [(a.q, b.q), (a.k_cache, b.k_cache), (a.v_cache, b.v_cache),
                 (a.block_table, b.block_table)]:
        assert torch.equal(x, y)
    assert not torch.equal(a.k_cache, c.k_cache)


def test_block_table_is_a_permutation_of_the_pool():
    case = make_case(3, 4, 2, [33, 0, 100], [1, 1, 4], seed=9)
    bt = case.block_table.numpy()
    pages = [3, 0, 7]
    used = np.concatenate([bt[b, :p] for b, p in enumerate(pages)])
    assert sorted(used.tolist()) == list(range(case.k_cache.shape[0]))
    for b, p in enumerate(pages):
        assert np.all(bt[b, p:] == -1)


def test_ragged_lengths_are_log_uniform_in_range():
    n = ragged_lengths()
    assert n.shape == (64,) and n.min() >= 512 and n.max() <= 131072
    assert np.array_equal(n, ragged_lengths())
    logn = np.log(n)
    assert abs(logn.mean() - (np.log(512) + np.log(131072)) / 2) < 0.6
    w = WORKLOADS["qwen3-4b_ragged_b64"]
    S = w.shard_counts()
    assert np.array_equal(S, np.maximum(1, -(-n // 4096))) and S.max() <= w.max_shards()


def test_small_workload_case_is_the_registered_shape():
    case = workload_case("qwen3-0.6b_b1_n4608_s8")
    assert case.q.shape == (1, 16, HEAD_DIM)
    assert case.k_cache.shape == (4608 // PAGE, 8, PAGE, HEAD_DIM)
    assert case.kv_bytes() == 18874368
    assert case.block_table.tolist() == [list(range(288))]


def test_planted_keys_reach_their_targets():
    case = make_case(1, 16, 8, [20000], [4], seed=4, planted=(400, 84.0, 86.0))
    q = case.q.double().numpy()
    kc = case.k_cache.float().numpy()
    for (b, g), (pos, t) in case.planted.items():
        K = oracle.gather_rows(kc, case.block_table[b].numpy(), g, 20000, PAGE)[pos]
        for h in (2 * g, 2 * g + 1):
            s = case.scale * (K @ q[b, h])
            assert np.max(np.abs(s - t)) < 0.5     # bf16 rounding of the key moves it a little


def test_one_gpu_share_of_the_long_request():
    """The per-GPU share of the 2^20-position request sharded by position over 8 GPUs: an eighth
    of its positions and of its planted keys, at the same model shape, two shards."""
    whole = WORKLOADS["qwen3-0.6b_b1_n1m_s16_l28_planted"]
    share = WORKLOADS["qwen3-0.6b_b1_n131072_s2_l28_planted"]
    assert share.ctx * 8 == whole.ctx and share.shards == 2
    assert (share.batch, share.n_q_heads, share.n_kv_heads, share.layers) == \
        (whole.batch, whole.n_q_heads, whole.n_kv_heads, whole.layers)
    assert share.planted and share.planted_count * 8 == whole.planted_count
    assert share.max_pages() * 8 == whole.max_pages()
