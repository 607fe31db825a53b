"""Shared helpers of the GPU parity tests: run the HIP path through the C ABI, run the fp64 oracle
on the same bytes, and apply the gates.

Gates (floating point; derivation in the design doc):
  * combined output (bf16): the kernel rounds an fp32 value to nearest bf16; that fp32 value
    may differ from the exact O by the fp32 accumulation error, allowed up to
    delta = 1e-4 * max|O| per (request, head).  So out must lie between the bf16 value just below
    O - delta and the bf16 value just above O + delta.  The contract bound max|out - O| <= 2e-2
    is checked as well.
  * log-sum-exp (fp32), combined and per shard: |lse - LSE| <= 1e-5 * max(1, |LSE|).
  * per-shard O (fp32): max|O_s - O_s*| <= 1e-4 * max|O_s*| per (request, head).
  * empty shards: lse exactly -inf; all-empty requests: out exactly +0 and lse -inf.
"""

from __future__ import annotations

import sys
import time

import numpy as np
import torch

import oracle
import paper_2608_15473_amd as qf

LSE_REL = 1e-5
OUT_ABS = 2e-2
PART_REL = 1e-4


def say(msg: str) -> None:
    print(msg, flush=True)
    sys.stdout.flush()


def run_gpu(case, n_shards=None, poison_partials=True):
    """Sweep + merge on the GPU through the C ABI; returns numpy copies."""
    B, Hq, Hkv, D = case.shape
    S = case.max_shards
    po = torch.empty((B, S, Hq, D), dtype=torch.float32, device=case.q.device)
    pl = torch.empty((B, S, Hq), dtype=torch.float32, device=case.q.device)
    if poison_partials:   # unwritten (empty) slots must never be read by the merge
        po.fill_(float("nan"))
        pl.fill_(float("nan"))
    qf.attn_decode_split(case.q, case.k_cache, case.v_cache, case.block_table, case.ctx_lens,
                         case.n_shards if n_shards is None else n_shards, max_shards=S,
                         scale=case.scale, part_out=po, part_lse=pl)
    out, lse = qf.attn_combine(po, pl)
    torch.cuda.synchronize()
    return dict(part_out=po.cpu().numpy(), part_lse=pl.cpu().numpy(),
                out=out.float().cpu().numpy(), lse=lse.cpu().numpy(),
                out_bits=out.view(torch.int16).cpu().numpy())


def host_arrays(case, requests=None):
    """The case's bytes on the host as float arrays the oracle reads.  With ``requests`` only
    those requests' pages are copied, with a block table renumbered over the copied pages."""
    q = case.q.double().cpu().numpy()
    ctx = case.ctx_lens.cpu().numpy()
    S = case.n_shards.cpu().numpy()
    if requests is None:
        return dict(q=q, k=case.k_cache.float().cpu().numpy(), v=case.v_cache.float().cpu().numpy(),
                    bt=case.block_table.cpu().numpy(), ctx=ctx, S=S, sub=None)
    bt = case.block_table.cpu().numpy()
    pages, rows = [], {}
    for b in requests:
        npg = -(-int(ctx[b]) // 16)
        rows[b] = np.arange(len(pages), len(pages) + npg)
        pages.extend(bt[b, :npg].tolist())
    idx = torch.as_tensor(pages if pages else [0], dtype=torch.long, device=case.k_cache.device)
    k = case.k_cache.index_select(0, idx).float().cpu().numpy()
    v = case.v_cache.index_select(0, idx).float().cpu().numpy()
    sub_bt = np.zeros_like(bt)
    for b, r in rows.items():
        sub_bt[b, : len(r)] = r
    return dict(q=q, k=k, v=v, bt=sub_bt, ctx=ctx, S=S, sub=rows)


def oracle_ref(case, pairs=None):
    reqs = None if pairs is None else sorted({b for b, _ in pairs})
    a = host_arrays(case, reqs)
    t0 = time.perf_counter()
    po, pl = oracle.decode_split(a["q"], a["k"], a["v"], a["bt"], a["ctx"], a["S"], case.scale,
                                 case.max_shards, pairs=pairs)
    out, lse = oracle.decode_unsplit(a["q"], a["k"], a["v"], a["bt"], a["ctx"], case.scale,
                                     pairs=pairs)
    return dict(part_out=po, part_lse=pl, out=out, lse=lse, seconds=time.perf_counter() - t0)


def bf16_neighbours(x: np.ndarray):
    """The largest bf16 value <= x and the smallest >= x, for float64 x (equal when x is bf16).

    The float32 nearest to x is within one float32 ulp of x, so both neighbours are among the
    bf16 value that float32 truncates to and the bf16 values one step either side of it (or 0).
    """
    x = np.asarray(x, dtype=np.float64)
    b = (x.astype(np.float32).view(np.uint32) & np.uint32(0xFFFF0000)).astype(np.int64)
    cands = [np.zeros_like(x)]
    for step in (-0x10000, 0, 0x10000):
        c = b + step
        c = np.where((c >= 0) & (c <= 0xFFFFFFFF), c, b).astype(np.uint32)
        cands.append(c.view(np.float32).astype(np.float64))
    C = np.stack(cands)
    lo = np.max(np.where(C <= x, C, -np.inf), axis=0)
    hi = np.min(np.where(C >= x, C, np.inf), axis=0)
    return lo, hi


def check(case, got, ref, pairs=None, label=""):
    """Apply every gate; returns a dict of the worst errors."""
    B, Hq, Hkv, D = case.shape
    todo = pairs if pairs is not None else [(b, h) for b in range(B) for h in range(Hq)]
    worst = dict(out_abs=0.0, out_rel=0.0, lse_rel=0.0, part_rel=0.0, part_lse_rel=0.0)
    for b, h in todo:
        O, L = ref["out"][b, h], ref["lse"][b, h]
        o, l = got["out"][b, h], got["lse"][b, h]
        if L == -np.inf:
            assert l == -np.inf, (label, b, h, l)
            assert np.all(got["out_bits"][b, h] == 0), (label, b, h)
        else:
            assert np.isfinite(l), (label, b, h, l)
            rel = abs(l - L) / max(1.0, abs(L))
            assert rel <= LSE_REL, (label, b, h, l, L)
            worst["lse_rel"] = max(worst["lse_rel"], rel)
            delta = PART_REL * float(np.max(np.abs(O)))
            lo, _ = bf16_neighbours(O - delta)
            _, hi = bf16_neighbours(O + delta)
            ok = (o >= lo) & (o <= hi)
            assert ok.all(), (label, b, h, np.flatnonzero(~ok)[:5], o[~ok][:5], O[~ok][:5])
            worst["out_rel"] = max(worst["out_rel"],
                                   float(np.max(np.abs(o - O))) / float(np.max(np.abs(O))))
            err = float(np.max(np.abs(o - O)))
            assert err <= OUT_ABS
            worst["out_abs"] = max(worst["out_abs"], err)
        for s in range(case.max_shards):
            Ls = ref["part_lse"][b, s, h]
            ls = got["part_lse"][b, s, h]
            if Ls == -np.inf:
                assert ls == -np.inf, (label, b, s, h, ls)
                continue
            rel = abs(ls - Ls) / max(1.0, abs(Ls))
            assert rel <= LSE_REL, (label, b, s, h, ls, Ls)
            worst["part_lse_rel"] = max(worst["part_lse_rel"], rel)
            Os = ref["part_out"][b, s, h]
            d = float(np.max(np.abs(got["part_out"][b, s, h] - Os))) / float(np.max(np.abs(Os)))
            assert d <= PART_REL, (label, b, s, h, d)
            worst["part_rel"] = max(worst["part_rel"], d)
    return worst
