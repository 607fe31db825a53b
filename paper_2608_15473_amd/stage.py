"""A stack of Q-First decoder blocks at one decode step, with the cache sweep on its own stream.

Q-First (arXiv:2608.15473): in the rewired block the query is projected from the block input u,
and the key and value from z = u + M(N2 u), the stream after the feed-forward (§2); the block is
(I + A_{x;z}) o (I + M) (§8), so its output is y = z + W_o attn.  The sweep needs the query alone
(§2), and neither it nor the feed-forward is downstream of the other (§3, "across layers"), so
the two may run at once.  On one GPU this module offers three orders of the same launches:

  mode="serial":   everything on one stream, in the order drawn below;
  mode="streams":  the sweep on a second HIP stream, forked after q and joined before the fold:

    main stream:       W_q N1(u) -> q --+--> SwiGLU(W_gate|W_up N2(u)) -> u + W_down(.) = z
                                        |     -> W_k|W_v N1(z) -> k, v --[join]--> merge + fold
                                        |                              + append -> z + W_o attn = y
    attention stream:                   +--> sweep of the layer's cache (split into shards) --^

  mode="fused":    the sweep and W_gate|W_up N2(u) in one launch whose workgroups take either
                   role (qf_attn_decode_split_beside), so the two share every CU.

Every step is one of the library's HIP kernels: the four products fused with the normalisation
or activation that feeds them and the residual add that follows (qf_linear), the sweep, and the merge
with the current-token fold and the cache append in one launch.  All three modes produce bitwise identical
outputs and caches.  Every buffer is allocated once, so a step can be captured in a HIP graph
(``capture``).
"""

from __future__ import annotations

import contextlib
import dataclasses

import torch

from . import binding as qf


@dataclasses.dataclass
class LayerCache:
    """One layer's paged KV cache (the layout of ``qf_attn_decode_split``)."""
    k_cache: torch.Tensor      # bf16 [num_pages, Hkv, P, D]
    v_cache: torch.Tensor      # bf16 [num_pages, Hkv, P, D]
    block_table: torch.Tensor  # int32 [B, max_pages]
    ctx_lens: torch.Tensor     # int32 [B], advanced by one per step
    n_shards: torch.Tensor     # int32 [B]


MODES = ("serial", "streams", "fused")
WEIGHT_NAMES = ("w_q", "w_k", "w_v", "w_o", "w_gate", "w_up", "w_down", "g1", "g2")


class QFirstStack:
    """Decode steps of ``len(layers)`` Q-First blocks for a batch of B requests.

    ``layers``: one dict per block of bf16 device tensors in torch layout [out, in]
    (``WEIGHT_NAMES``; g1, g2 are the N1, N2 gains); ``caches``: one ``LayerCache`` per block, with
    room for the positions the steps will append.
    """

    def __init__(self, layers, caches, n_q_heads: int, n_kv_heads: int, max_shards: int,
                 scale: float, eps: float = 1e-6):
        if len(layers) != len(caches) or not layers:
            raise ValueError("need one cache per layer and at least one layer")
        w0 = layers[0]
        self.device = w0["w_q"].device
        self.hidden = w0["w_q"].shape[1]
        self.inter = w0["w_gate"].shape[0]
        self.hq, self.hkv = n_q_heads, n_kv_heads
        self.d = w0["w_q"].shape[0] // n_q_heads
        self.max_shards, self.scale, self.eps = int(max_shards), float(scale), float(eps)
        self.layers = []
        for w in layers:
            missing = [n for n in WEIGHT_NAMES if n not in w]
            if missing:
                raise ValueError(f"missing weights {missing}")
            lw = dict(w)                                    # one product each for gate|up, k|v
            # gate and up rows interleaved, so the product's epilogue writes the activation
            lw["w_gu"] = torch.stack([w["w_gate"], w["w_up"]], 1).reshape(
                -1, w["w_gate"].shape[1]).contiguous()
            lw["w_kv"] = torch.cat([w["w_k"], w["w_v"]], 0).contiguous()
            self.layers.append(lw)
        self.caches = list(caches)
        self.B = int(caches[0].ctx_lens.shape[0])
        self.attn_stream = torch.cuda.Stream(self.device)    # default priority
        B, H, I, D = self.B, self.hidden, self.inter, self.d

        def buf(*shape, dtype=torch.bfloat16):
            return torch.empty(shape, dtype=dtype, device=self.device)

        self.z = buf(B, H)
        self.y = [buf(B, H), buf(B, H)]                       # ping-pong between layers
        self.q = buf(B, self.hq, D)
        self.k, self.v = buf(B, self.hkv, D), buf(B, self.hkv, D)
        self.act = buf(B, I)                                  # silu(gate) * up
        self.attn = buf(B, self.hq, D)
        self.lse = buf(B, self.hq, dtype=torch.float32)
        self.part_out = buf(B, self.max_shards, self.hq, D, dtype=torch.float32)
        self.part_lse = buf(B, self.max_shards, self.hq, dtype=torch.float32)
        self.status = torch.zeros(1, dtype=torch.int32, device=self.device)
        ws = max(qf.workspace_size(qf.make_desc(self.q, c.k_cache, c.block_table,
                                                self.max_shards, self.scale))
                 for c in self.caches)
        self.workspace = buf(max(ws, 1), dtype=torch.uint8) if ws else None
        # Optional: a callable name -> context manager wrapped around every launch of a block
        # (e.g. HIP events on the current stream, to time each kernel).
        self.recorder = None

    def _span(self, name: str):
        return contextlib.nullcontext() if self.recorder is None else self.recorder(name)

    # ----------------------------------------------------------------------------------------
    def _sweep(self, c: LayerCache) -> None:
        qf.attn_decode_split(self.q, c.k_cache, c.v_cache, c.block_table, c.ctx_lens,
                             c.n_shards, max_shards=self.max_shards, scale=self.scale,
                             part_out=self.part_out, part_lse=self.part_lse,
                             workspace=self.workspace)

    def _linear(self, x, w, out, prologue=None, gain=None, residual=None, out_b=None,
                glu_out=False):
        """qf_linear over the batch in blocks of at most 8 rows."""
        B, split = self.B, out.shape[-1] if out_b is not None else None
        for r in range(0, B, 8):
            e = min(B, r + 8)
            qf.linear(x[r:e], w, prologue, gain, self.eps,
                      residual=None if residual is None else residual[r:e], out=out[r:e],
                      split=split, out_b=None if out_b is None else out_b[r:e], glu_out=glu_out)

    def block(self, l: int, u: torch.Tensor, out: torch.Tensor, mode: str = "fused"):
        """One Q-First block: reads u [B, H], writes out [B, H], appends the layer's (k, v)."""
        if mode not in MODES:
            raise ValueError(f"mode must be one of {MODES}")
        w, c = self.layers[l], self.caches[l]
        B = self.B
        main = torch.cuda.current_stream(self.device)
        with self._span("W_q"):                                             # q reads u
            self._linear(u, w["w_q"], self.q.view(B, -1), "rms_norm", w["g1"])
        if mode == "fused":                                                  # sweep | W_gate|W_up
            head = min(B, 8)
            with self._span("sweep + W_gate,W_up"):
                qf.attn_decode_split_beside(
                    self.q, c.k_cache, c.v_cache, c.block_table, c.ctx_lens, c.n_shards,
                    dict(x=u[:head], w=w["w_gu"], prologue="rms_norm", gain=w["g2"], eps=self.eps,
                         out=self.act[:head], glu_out=True),
                    max_shards=self.max_shards, scale=self.scale, part_out=self.part_out,
                    part_lse=self.part_lse, workspace=self.workspace)
                if B > head:
                    self._linear(u[head:], w["w_gu"], self.act[head:], "rms_norm", w["g2"],
                                 glu_out=True)
        else:
            if mode == "streams":
                self.attn_stream.wait_stream(main)
                with torch.cuda.stream(self.attn_stream), self._span("sweep"):
                    self._sweep(c)
            else:
                with self._span("sweep"):
                    self._sweep(c)
            with self._span("W_gate,W_up"):                                  # the feed-forward
                self._linear(u, w["w_gu"], self.act, "rms_norm", w["g2"], glu_out=True)
        with self._span("W_down"):                                           # z = u + M(N2 u)
            self._linear(self.act, w["w_down"], self.z, residual=u)
        with self._span("W_k,W_v"):                                          # k, v read z
            self._linear(self.z, w["w_kv"], self.k.view(B, -1), "rms_norm", w["g1"],
                         out_b=self.v.view(B, -1))
        if mode == "streams":
            main.wait_stream(self.attn_stream)
        with self._span("merge, current-token fold + cache append"):    # one launch
            qf.attn_combine_current_append(self.part_out, self.part_lse, self.q, self.k, self.v,
                                           c.k_cache, c.v_cache, c.block_table, c.ctx_lens,
                                           scale=self.scale, out=self.attn, lse=self.lse,
                                           status=self.status)
        with self._span("W_o"):                                              # y = z + W_o attn
            self._linear(self.attn.view(B, -1), w["w_o"], out, residual=self.z)
        return out

    def step(self, u: torch.Tensor, mode: str = "fused") -> torch.Tensor:
        """One decode step through every block; returns the last block's output buffer."""
        if tuple(u.shape) != (self.B, self.hidden) or u.dtype != torch.bfloat16:
            raise ValueError(f"u must be bf16 [{self.B}, {self.hidden}]")
        x = u
        for l in range(len(self.layers)):
            x = self.block(l, x, self.y[l % 2], mode)
        return x

    def capture(self, u: torch.Tensor, mode: str = "fused"):
        """Capture one step in a HIP graph; returns (graph, output buffer).  Capturing runs
        nothing; each replay is one step (and appends one position per layer)."""
        graph = torch.cuda.CUDAGraph()
        with torch.cuda.graph(graph):
            y = self.step(u, mode)
        return graph, y
