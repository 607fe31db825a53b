"""Seeded synthetic inputs for split-KV decode attention, shared by the tests and the bench.

This module only draws random numbers and lays them out; it holds none of the attention
arithmetic, so both the HIP path and the fp64 oracle can consume what it produces without sharing
any of the method's code.  Shapes follow the paper's Qwen3 sizing (Q-First, arXiv:2608.15473, §3
and §4 tables): 16 query / 8 KV heads at Qwen3-0.6B, 32 / 8 at Qwen3-4B, head_dim 128, bf16, i.e.
4,096 bytes of K+V per cached position per layer.

Draw order for one (workload, layer): a torch generator seeded with ``seed``, then Q, K, V
(i.i.d. N(0,1), bf16), then the physical-page permutation, then (planted workloads only) the
planted positions and their target logits.  The oracle receives the same bytes copied to the
host, so GPU and CPU generators never need to agree with each other.
"""

from __future__ import annotations

import dataclasses
import math

import numpy as np
import torch

HEAD_DIM = 128
PAGE = 16
SCALE = float(np.float32(1.0 / math.sqrt(HEAD_DIM)))  # the fp32 value every call passes


def kv_bytes_per_position(n_kv_heads: int, head_dim: int = HEAD_DIM, elem_bytes: int = 2) -> int:
    """K plus V bytes one cached position occupies in one layer (the sweep's bytes, §3)."""
    return 2 * n_kv_heads * head_dim * elem_bytes


# --------------------------------------------------------------------------------------------
# workload registry
# --------------------------------------------------------------------------------------------
@dataclasses.dataclass(frozen=True)
class Workload:
    name: str
    index: int                 # seeds are 1000 * index + layer
    batch: int
    n_q_heads: int
    n_kv_heads: int
    layers: int
    ctx: int | None            # uniform context, or None for ragged
    shards: int | None         # uniform shard count, or None for ceil(n / ragged_shard_len)
    table: str                 # "identity" | "perm"
    planted: bool = False
    planted_count: int = 400   # planted keys per (request, KV head)
    ragged_shard_len: int = 4096
    description: str = ""

    def lengths(self) -> np.ndarray:
        if self.ctx is not None:
            return np.full(self.batch, self.ctx, dtype=np.int64)
        return ragged_lengths(self.batch)

    def shard_counts(self, lengths=None) -> np.ndarray:
        if self.shards is not None:
            return np.full(self.batch, self.shards, dtype=np.int64)
        n = self.lengths() if lengths is None else np.asarray(lengths)
        return np.maximum(1, -(-n // self.ragged_shard_len))

    def max_shards(self) -> int:
        return int(self.shards) if self.shards is not None else 32

    def max_pages(self) -> int:
        if self.ctx is not None:
            return -(-self.ctx // PAGE)
        return -(-131072 // PAGE)


def ragged_lengths(batch: int = 64, seed: int = 5000, lo: int = 512, hi: int = 131072) -> np.ndarray:
    """Context lengths log-uniform in [lo, hi], rounded and clipped (numpy default_rng(seed))."""
    rng = np.random.default_rng(seed)
    n = np.rint(np.exp(rng.uniform(np.log(lo), np.log(hi), size=batch))).astype(np.int64)
    return np.clip(n, lo, hi)


WORKLOADS = {
    w.name: w
    for w in [
        Workload("qwen3-0.6b_b1_n4608_s8", 1, 1, 16, 8, 1, 4608, 8, "identity",
                 description="single layer, batch 1, context 4,608 (the 0.6B crossover), "
                             "contiguous KV, 8 shards"),
        Workload("qwen3-0.6b_b32_n32768_s64_l28", 2, 32, 16, 8, 28, 32768, 64, "perm",
                 description="28 layers, batch 32, context 32,768, paged KV with a random "
                             "block table, 64 shards"),
        Workload("qwen3-4b_b16_n36480_s32_l36", 3, 16, 32, 8, 36, 36480, 32, "perm",
                 description="36 layers, batch 16, context 36,480 (the 4B crossover), paged, "
                             "32 shards"),
        Workload("qwen3-0.6b_b1_n1m_s16_l28_planted", 4, 1, 16, 8, 28, 1 << 20, 16, "perm",
                 planted=True,
                 description="28 layers, batch 1, 2^20 positions, 16 shards of 65,536; 400 "
                             "planted keys per KV head with logits near 85"),
        Workload("qwen3-4b_ragged_b64", 5, 64, 32, 8, 1, None, None, "perm",
                 description="1 layer, 64 requests, contexts log-uniform in [512, 131072], "
                             "ceil(n/4096) shards each"),
        Workload("qwen3-32b_b16_n32768_s32_l64", 7, 16, 64, 8, 64, 32768, 32, "perm",
                 description="eight query heads per KV head (Qwen3-32B: 64 query / 8 KV heads), "
                             "64 layers, batch 16, context 32,768, paged, 32 shards"),
        Workload("qwen3-0.6b_b1_n131072_s2_l28_planted", 6, 1, 16, 8, 28, 1 << 17, 2, "perm",
                 planted=True, planted_count=50,
                 description="one GPU's share of the 2^20-position request sharded by position "
                             "over 8 GPUs: 28 layers, 131,072 positions, 2 shards, 50 planted "
                             "keys per KV head (the 400 of the whole request, spread evenly)"),
    ]
}


# --------------------------------------------------------------------------------------------
# one decode step's inputs
# --------------------------------------------------------------------------------------------
@dataclasses.dataclass
class Case:
    q: torch.Tensor            # bf16 [B, Hq, D]
    k_cache: torch.Tensor      # bf16 [num_pages, Hkv, P, D]
    v_cache: torch.Tensor      # bf16 [num_pages, Hkv, P, D]
    block_table: torch.Tensor  # int32 [B, max_pages]; unused entries -1
    ctx_lens: torch.Tensor     # int32 [B]
    n_shards: torch.Tensor     # int32 [B]
    max_shards: int
    scale: float = SCALE
    planted: dict | None = None  # kv head -> (positions, targets), planted cases only

    @property
    def shape(self):
        B, Hq, D = self.q.shape
        return B, Hq, self.k_cache.shape[1], D

    def kv_bytes(self) -> int:
        n = int(self.ctx_lens.to(torch.int64).sum())
        return n * kv_bytes_per_position(self.k_cache.shape[1], self.q.shape[2])


def make_case(batch: int, n_q_heads: int, n_kv_heads: int, ctx_lens, n_shards, *,
              seed: int, table: str = "perm", max_shards: int | None = None,
              max_pages: int | None = None, head_dim: int = HEAD_DIM, page: int = PAGE,
              planted: tuple[int, float, float] | None = None, spare_pages: int = 0,
              device="cpu") -> Case:
    """Draw one seeded decode step.

    ``ctx_lens`` / ``n_shards``: per-request ints (or one int broadcast).  ``table``: "identity"
    (request b owns pages b*max_pages ...) or "perm" (pages handed out from one random
    permutation of the pool, in request order).  ``planted=(count, lo, hi)`` plants ``count`` keys
    per KV head (and request) whose logits for every query head of the group are ~U(lo, hi).
    """
    ctx = np.broadcast_to(np.asarray(ctx_lens, dtype=np.int64), (batch,)).copy()
    shards = np.broadcast_to(np.asarray(n_shards, dtype=np.int64), (batch,)).copy()
    pages_b = -(-ctx // page)
    if max_pages is None:
        max_pages = max(1, int(pages_b.max()) if batch else 1)
    if max_shards is None:
        max_shards = max(1, int(shards.max()) if batch else 1)
    if table == "identity":
        num_pages = batch * max_pages
    else:
        num_pages = max(1, int(pages_b.sum()) + spare_pages)

    gen = torch.Generator(device=device)
    gen.manual_seed(seed)
    q = torch.randn(batch, n_q_heads, head_dim, generator=gen, device=device, dtype=torch.bfloat16)
    k = torch.randn(num_pages, n_kv_heads, page, head_dim, generator=gen, device=device,
                    dtype=torch.bfloat16)
    v = torch.randn(num_pages, n_kv_heads, page, head_dim, generator=gen, device=device,
                    dtype=torch.bfloat16)
    bt = torch.full((batch, max_pages), -1, dtype=torch.int32)
    if table == "identity":
        bt = torch.arange(batch * max_pages, dtype=torch.int32).reshape(batch, max_pages)
    else:
        perm = torch.randperm(num_pages, generator=gen, device=device).to(torch.int32).cpu()
        off = 0
        for b in range(batch):
            bt[b, : pages_b[b]] = perm[off: off + pages_b[b]]
            off += int(pages_b[b])
    case = Case(q=q, k_cache=k, v_cache=v, block_table=bt.to(device),
                ctx_lens=torch.as_tensor(ctx, dtype=torch.int32, device=device),
                n_shards=torch.as_tensor(shards, dtype=torch.int32, device=device),
                max_shards=int(max_shards))
    if planted is not None:
        _plant(case, gen, *planted)
    return case


def _plant(case: Case, gen: torch.Generator, count: int, lo: float, hi: float) -> None:
    """Plant ``count`` keys per (request, KV head) whose logits are ~U(lo, hi) for every query
    head of the group: k = (1/scale) Q^T (Q Q^T)^-1 t, the minimum-norm key reaching the targets
    t for all G queries at once, rounded to bf16.  The realised logits differ slightly after that
    rounding; checks recompute them from the stored bytes."""
    B, Hq, Hkv, D = case.shape
    G = Hq // Hkv
    dev = case.q.device
    bt = case.block_table.cpu()
    info = {}
    for b in range(B):
        n = int(case.ctx_lens[b])
        if n == 0:
            continue
        for g in range(Hkv):
            c = min(count, n)
            pos = torch.randperm(n, generator=gen, device=dev)[:c].cpu()
            t = (torch.rand(c, generator=gen, device=dev, dtype=torch.float64).cpu()
                 * (hi - lo) + lo)
            Q = case.q[b, g * G:(g + 1) * G].double().cpu()          # [G, D]
            coef = torch.linalg.solve(Q @ Q.T, t[None, :].expand(G, c))  # [G, c]
            keys = (Q.T @ coef).T / case.scale                        # [c, D]
            phys = bt[b, pos // PAGE].long()
            case.k_cache[phys.to(dev), g, (pos % PAGE).to(dev)] = keys.to(torch.bfloat16).to(dev)
            info[(b, g)] = (pos.numpy(), t.numpy())
    case.planted = info


def workload_case(name: str, layer: int = 0, device="cpu", **override) -> Case:
    """The full-size inputs of one layer of a registered workload."""
    w = WORKLOADS[name]
    lengths = w.lengths()
    kw = dict(seed=1000 * w.index + layer, table=w.table, max_shards=w.max_shards(),
              max_pages=w.max_pages(), device=device)
    if w.planted:
        kw["planted"] = (w.planted_count, 84.0, 86.0)
    kw.update(override)
    return make_case(w.batch, w.n_q_heads, w.n_kv_heads, lengths, w.shard_counts(lengths), **kw)


# --------------------------------------------------------------------------------------------
# Q-First decode blocks with synthetic weights (the [MLP || Attn] stage)
# --------------------------------------------------------------------------------------------
@dataclasses.dataclass(frozen=True)
class BlockShape:
    """Dense sizes of one decoder block (Qwen3 configurations; the byte table of the paper's §3 counts
    19 MB of feed-forward weights per layer at Qwen3-0.6B and 149 MB at Qwen3-4B)."""
    name: str
    hidden: int
    inter: int
    n_q_heads: int
    n_kv_heads: int
    layers: int

    def ffn_bytes(self) -> int:
        return 3 * self.hidden * self.inter * 2


BLOCKS = {
    b.name: b
    for b in [
        BlockShape("qwen3-0.6b", hidden=1024, inter=3072, n_q_heads=16, n_kv_heads=8, layers=28),
        BlockShape("qwen3-4b", hidden=2560, inter=9728, n_q_heads=32, n_kv_heads=8, layers=36),
    ]
}


@dataclasses.dataclass(frozen=True)
class StageWorkload:
    """A decode step of a stack of blocks at the context where the feed-forward's weight bytes
    equal the sweep's cache bytes (the crossover column of the byte table in the paper's §3)."""
    name: str
    index: int                 # seeds are 1000 * index + layer
    block: str
    batch: int
    ctx: int
    shards: int


STAGE_WORKLOADS = {
    w.name: w
    for w in [
        # One request fills the GPU only when cut finely, so the shards do what sub-shard chunks
        # would and the current-token fold merges them directly.  Measured (shared launch, one
        # MI355X): 24 shards beat 32 at Qwen3-0.6B and 128 beat 256 at Qwen3-4B by 4% a step
        # (fewer slots for the merge; 16 shards bring chunks and their merge launch back).
        StageWorkload("qwen3-0.6b_stage_b1_n4608", 11, "qwen3-0.6b", batch=1, ctx=4608, shards=24),
        StageWorkload("qwen3-4b_stage_b1_n36480", 12, "qwen3-4b", batch=1, ctx=36480, shards=128),
        # Eight requests (the products' row block): the sweep reads 8x the feed-forward's bytes.
        # 16 shards per request (measured: shared launch 2.02 ms per step with 8, 1.99 with 16,
        # 2.08 with 32).
        StageWorkload("qwen3-0.6b_stage_b8_n4608", 13, "qwen3-0.6b", batch=8, ctx=4608, shards=16),
    ]
}


def block_weights(shape: BlockShape, seed: int, head_dim: int = HEAD_DIM, device="cpu"):
    """Seeded bf16 weights of one block, torch layout [out, in].

    Draw order: W_q, W_k, W_v, W_o, W_gate, W_up, W_down (N(0, 1/fan_in), so activations stay
    O(1)), then the two norm gains g1, g2 (U(0.5, 1.5))."""
    H, I = shape.hidden, shape.inter
    qd, kd = shape.n_q_heads * head_dim, shape.n_kv_heads * head_dim
    gen = torch.Generator(device=device)
    gen.manual_seed(seed)

    def mat(rows, cols):
        w = torch.randn(rows, cols, generator=gen, device=device, dtype=torch.float32)
        return (w * (1.0 / math.sqrt(cols))).to(torch.bfloat16)

    w = {"w_q": mat(qd, H), "w_k": mat(kd, H), "w_v": mat(kd, H), "w_o": mat(H, qd),
         "w_gate": mat(I, H), "w_up": mat(I, H), "w_down": mat(H, I)}
    for g in ("g1", "g2"):
        w[g] = (torch.rand(H, generator=gen, device=device, dtype=torch.float32) + 0.5).to(
            torch.bfloat16)
    return w


def block_input(batch: int, hidden: int, seed: int, device="cpu") -> torch.Tensor:
    """The first block's input u, N(0, 1) bf16 [B, hidden]."""
    gen = torch.Generator(device=device)
    gen.manual_seed(seed)
    return torch.randn(batch, hidden, generator=gen, device=device, dtype=torch.bfloat16)
