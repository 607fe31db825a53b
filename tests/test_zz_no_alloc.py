"""qf_attn_decode_noalloc: the one-launch decode in the library's fixed scratch array.

Called through the C ABI and compared with qf_attn_decode (the same kernels on a caller-supplied
workspace and counters), bitwise, and with the fp64 oracle at the parity gates, on several calls in
a row whose inputs shrink (each call must neither read what an earlier call left in the array nor
depend on it being clear).  Shapes beyond the array are refused on the host before anything is
enqueued."""

import ctypes
import math
import os

import numpy as np
import pytest

import paper_2608_15473_amd as qf
from paper_2608_15473_amd.binding import DecodeDesc, load_library

needs_lib = pytest.mark.skipif(not os.path.exists(qf.LIB_PATH), reason="libqfattn.so not built")


def _desc(**kw):
    base = dict(batch=2, n_q_heads=16, n_kv_heads=8, head_dim=128, page_size=16,
                max_pages_per_seq=64, num_pages=128, max_shards=4,
                softmax_scale=1 / math.sqrt(128))
    base.update(kw)
    return DecodeDesc(**base)


@needs_lib
@pytest.mark.parametrize("kw", [
    dict(batch=4096, n_q_heads=64, n_kv_heads=8, max_shards=64, max_pages_per_seq=4096,
         num_pages=1 << 20),                                  # partial states beyond the array
    dict(batch=10000, n_q_heads=8, n_kv_heads=8, max_shards=1, num_pages=1 << 21),  # counters
])
def test_shapes_beyond_the_scratch_are_refused_on_the_host(kw):
    lib = load_library()
    d = _desc(**kw)
    p = ctypes.c_void_p(256)   # never dereferenced: the size check comes before anything else
    rc = lib.qf_attn_decode_noalloc(ctypes.byref(d), p, p, p, p, p, p, p, p, None)
    assert rc == qf.QF_EINVAL
    assert "fixed scratch" in lib.qf_last_error().decode()


@needs_lib
def test_null_out_is_refused():
    lib = load_library()
    d = _desc()
    p = ctypes.c_void_p(256)
    rc = lib.qf_attn_decode_noalloc(ctypes.byref(d), p, p, p, p, p, p, None, p, None)
    assert rc == qf.QF_EINVAL


def _noalloc_via_abi(case, out, lse):
    """qf_attn_decode_noalloc called directly through ctypes on the case's tensors."""
    import torch
    lib = load_library()
    B, Hq, D = case.q.shape
    d = DecodeDesc(B, Hq, case.k_cache.shape[1], D, case.k_cache.shape[2],
                   case.block_table.shape[1], case.k_cache.shape[0], case.max_shards,
                   float(case.scale))
    vp = lambda t: ctypes.c_void_p(t.data_ptr())
    stream = torch.cuda.current_stream().cuda_stream
    rc = lib.qf_attn_decode_noalloc(ctypes.byref(d), vp(case.q), vp(case.k_cache),
                                    vp(case.v_cache), vp(case.block_table), vp(case.ctx_lens),
                                    vp(case.n_shards), vp(out), vp(lse), ctypes.c_void_p(stream))
    assert rc == qf.QF_OK, lib.qf_last_error().decode()


# Shrinking inputs: an unchunked batch, a chunked one (sub-shard chunks: partial states laid out
# differently), then a small chunked one; G = 2 (vector-ALU scores) and G = 4, 8 (matrix cores).
_CALLS = [
    dict(batch=16, hq=16, hkv=8, ctx=[2000, 4096, 1, 0] * 4, shards=[8, 8, 1, 3] * 4, seed=71),
    dict(batch=3, hq=32, hkv=8, ctx=[9000, 0, 3001], shards=[4, 2, 3], seed=72),
    dict(batch=2, hq=64, hkv=8, ctx=[2500, 700], shards=[3, 1], seed=73),
    dict(batch=1, hq=16, hkv=8, ctx=[777], shards=[2], seed=74),
]


@pytest.mark.gpu
def test_noalloc_equals_the_workspace_entry_point_on_calls_in_a_row(gpu):
    import torch

    import oracle
    from parity import OUT_ABS, LSE_REL, PART_REL, bf16_neighbours, say
    from workloads import make_case

    for i, c in enumerate(_CALLS):
        say(f"[noalloc] call {i}: batch {c['batch']}, Hq {c['hq']}, contexts {c['ctx'][:4]}")
        case = make_case(c["batch"], c["hq"], c["hkv"], c["ctx"], c["shards"], seed=c["seed"],
                         device=gpu)
        B, Hq, D = case.q.shape
        out = torch.full((B, Hq, D), float("nan"), dtype=torch.bfloat16, device=gpu)
        lse = torch.full((B, Hq), float("nan"), dtype=torch.float32, device=gpu)
        _noalloc_via_abi(case, out, lse)
        ref_o, ref_l = qf.attn_decode(case.q, case.k_cache, case.v_cache, case.block_table,
                                      case.ctx_lens, case.n_shards, max_shards=case.max_shards,
                                      scale=case.scale)
        torch.cuda.synchronize()
        # the existing entry point on the same inputs: bitwise the same
        assert torch.equal(out.view(torch.int16), ref_o.view(torch.int16)), i
        assert torch.equal(lse.view(torch.int32), ref_l.view(torch.int32)), i
        # and the oracle's gates
        O, L = oracle.decode_unsplit(case.q.double().cpu().numpy(),
                                     case.k_cache.float().cpu().numpy(),
                                     case.v_cache.float().cpu().numpy(),
                                     case.block_table.cpu().numpy(), case.ctx_lens.cpu().numpy(),
                                     case.scale)
        o = out.float().cpu().numpy()
        l = lse.cpu().numpy()
        bits = out.view(torch.int16).cpu().numpy()
        for b in range(B):
            for h in range(Hq):
                if L[b, h] == -np.inf:
                    assert l[b, h] == -np.inf and np.all(bits[b, h] == 0), (i, b, h)
                    continue
                assert abs(l[b, h] - L[b, h]) <= LSE_REL * max(1.0, abs(L[b, h])), (i, b, h)
                delta = PART_REL * float(np.max(np.abs(O[b, h])))
                lo, _ = bf16_neighbours(O[b, h] - delta)
                _, hi = bf16_neighbours(O[b, h] + delta)
                assert np.all((o[b, h] >= lo) & (o[b, h] <= hi)), (i, b, h)
                assert float(np.max(np.abs(o[b, h] - O[b, h]))) <= OUT_ABS


@pytest.mark.gpu
def test_noalloc_replayed_from_a_graph(gpu):
    """The callers the entry point is for include code under HIP graph capture: captured once
    (the counter-clearing kernel and the decode), replayed three times with eager calls of another
    shape on the same scratch array between the replays, every replay equals the eager call
    bitwise."""
    import torch

    from parity import say
    from workloads import make_case

    c = _CALLS[1]
    case = make_case(c["batch"], c["hq"], c["hkv"], c["ctx"], c["shards"], seed=c["seed"],
                     device=gpu)
    B, Hq, D = case.q.shape
    out = torch.empty((B, Hq, D), dtype=torch.bfloat16, device=gpu)
    lse = torch.empty((B, Hq), dtype=torch.float32, device=gpu)
    _noalloc_via_abi(case, out, lse)              # eager (and the scratch looked up on this GPU)
    torch.cuda.synchronize()
    eager = (out.view(torch.int16).clone(), lse.view(torch.int32).clone())
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph, stream=torch.cuda.Stream()):
        _noalloc_via_abi(case, out, lse)          # enqueued on the capturing stream
    d = _CALLS[3]
    other = make_case(d["batch"], d["hq"], d["hkv"], d["ctx"], d["shards"], seed=d["seed"],
                      device=gpu)
    o2 = torch.empty((1, 16, 128), dtype=torch.bfloat16, device=gpu)
    l2 = torch.empty((1, 16), dtype=torch.float32, device=gpu)
    for r in range(3):
        out.fill_(float("nan"))
        lse.fill_(float("nan"))
        graph.replay()
        torch.cuda.synchronize()
        say(f"[noalloc] graph replay {r}")
        assert torch.equal(out.view(torch.int16), eager[0]), r
        assert torch.equal(lse.view(torch.int32), eager[1]), r
        _noalloc_via_abi(other, o2, l2)           # eager use of the same array between replays
        torch.cuda.synchronize()
