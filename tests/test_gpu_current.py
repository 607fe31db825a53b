"""GPU parity for the current-token fold and the paged cache append (§2, Appendix A), through the
C ABI, against the fp64 oracle on the same seeded bytes."""

import numpy as np
import pytest
import torch

import oracle
import paper_2608_15473_amd as qf
from parity import LSE_REL, PART_REL, bf16_neighbours, host_arrays, say
from workloads import make_case

pytestmark = pytest.mark.gpu


def _allocated_case(gpu, B, Hq, Hkv, ctx, shards, seed, **kw):
    """A case whose pages hold n + 1 positions; the cache holds n (room for the new token)."""
    case = make_case(B, Hq, Hkv, np.asarray(ctx) + 1, shards, seed=seed, device=gpu, **kw)
    case.ctx_lens -= 1
    return case


def _new_token(case, seed):
    B, Hq, Hkv, D = case.shape
    gen = torch.Generator(device=case.q.device)
    gen.manual_seed(seed)
    k = torch.randn(B, Hkv, D, generator=gen, device=case.q.device, dtype=torch.bfloat16)
    v = torch.randn(B, Hkv, D, generator=gen, device=case.q.device, dtype=torch.bfloat16)
    return k, v


def _check_out(label, out, lse, ref_o, ref_l):
    for b in range(ref_o.shape[0]):
        for h in range(ref_o.shape[1]):
            L = ref_l[b, h]
            assert abs(lse[b, h] - L) <= LSE_REL * max(1.0, abs(L)), (label, b, h, lse[b, h], L)
            O = ref_o[b, h]
            delta = PART_REL * float(np.max(np.abs(O)))
            lo, _ = bf16_neighbours(O - delta)
            _, hi = bf16_neighbours(O + delta)
            ok = (out[b, h] >= lo) & (out[b, h] <= hi)
            assert ok.all(), (label, b, h, out[b, h][~ok][:4], O[~ok][:4])


def _fold_on_gpu(case, k_new, v_new):
    po, pl = qf.attn_decode_split(case.q, case.k_cache, case.v_cache, case.block_table,
                                  case.ctx_lens, case.n_shards, max_shards=case.max_shards,
                                  scale=case.scale)
    out, lse = qf.attn_combine_current(po, pl, case.q, k_new, v_new, scale=case.scale)
    torch.cuda.synchronize()
    return out.float().cpu().numpy(), lse.cpu().numpy()


def _fold_reference(case, k_new, v_new):
    a = host_arrays(case)
    O, L = oracle.decode_unsplit(a["q"], a["k"], a["v"], a["bt"], a["ctx"], case.scale)
    return oracle.fold_current(O, L, a["q"], k_new.double().cpu().numpy(),
                               v_new.double().cpu().numpy(), case.scale)


@pytest.mark.parametrize("Hq,Hkv", [(16, 8), (32, 8), (8, 8), (64, 8)])
def test_fold_current_matches_oracle(gpu, Hq, Hkv):
    case = _allocated_case(gpu, 4, Hq, Hkv, [700, 1, 0, 2100], [3, 1, 2, 5], seed=200 + Hq)
    k_new, v_new = _new_token(case, 201)
    say(f"[current] fold Hq={Hq} Hkv={Hkv}")
    out, lse = _fold_on_gpu(case, k_new, v_new)
    ref_o, ref_l = _fold_reference(case, k_new, v_new)
    _check_out("fold", out, lse, ref_o, ref_l)
    # empty cache (request 2): the current token alone
    G = Hq // Hkv
    for h in range(Hq):
        np.testing.assert_array_equal(out[2, h], v_new[2, h // G].float().cpu().numpy())


def test_fold_over_many_shard_slots(gpu):
    """The fold after a merge of 256 shard slots (the merge's 16-wavefront form)."""
    case = _allocated_case(gpu, 2, 32, 8, [36000, 900], [256, 40], seed=205, max_shards=256)
    k_new, v_new = _new_token(case, 206)
    say("[current] fold over 256 slots")
    out, lse = _fold_on_gpu(case, k_new, v_new)
    ref_o, ref_l = _fold_reference(case, k_new, v_new)
    _check_out("fold256", out, lse, ref_o, ref_l)


def test_fold_either_sign_of_the_gap(gpu):
    """s_jj - lse_<j from -120 to +120 nats (short caches put the current token on top)."""
    gaps = np.array([-120.0, -30.0, -9.7, -1.0, 0.0, 1.0, 9.7, 30.0, 120.0])
    B = len(gaps)
    case = _allocated_case(gpu, B, 4, 4, [1, 2, 5, 40, 300, 17, 1, 64, 3], 1, seed=210)
    a = host_arrays(case)
    O, L = oracle.decode_unsplit(a["q"], a["k"], a["v"], a["bt"], a["ctx"], case.scale)
    # k_new along q so that scale * q . k_new = L + gap (up to bf16 rounding of k_new)
    q = a["q"]
    k_new = np.zeros((B, 4, 128))
    for b in range(B):
        for g in range(4):
            target = L[b, g] + gaps[b]
            k_new[b, g] = q[b, g] * (target / case.scale / float(q[b, g] @ q[b, g]))
    k_t = torch.from_numpy(k_new).to(torch.bfloat16).to(gpu)
    _, v_t = _new_token(case, 211)
    out, lse = _fold_on_gpu(case, k_t, v_t)
    ref_o, ref_l = oracle.fold_current(O, L, q, k_t.double().cpu().numpy(),
                                       v_t.double().cpu().numpy(), case.scale)
    s_jj = np.einsum("bhd,bhd->bh", q, k_t.double().cpu().numpy()) * case.scale
    realised = s_jj - L
    assert realised.min() < -100 and realised.max() > 100
    _check_out("sign", out, lse, ref_o, ref_l)
    assert np.all(np.isfinite(out)) and np.all(np.isfinite(lse))


def test_append_writes_exactly_the_new_slot_and_advances(gpu):
    case = _allocated_case(gpu, 5, 16, 8, [0, 15, 16, 33, 200], 1, seed=220)
    k_new, v_new = _new_token(case, 221)
    a = host_arrays(case)
    ref_k, ref_v = oracle.append_kv(case.k_cache.view(torch.int16).cpu().numpy(),
                                    case.v_cache.view(torch.int16).cpu().numpy(), a["bt"],
                                    a["ctx"], k_new.view(torch.int16).cpu().numpy(),
                                    v_new.view(torch.int16).cpu().numpy())
    status = torch.zeros(1, dtype=torch.int32, device=gpu)
    qf.kv_append(case.k_cache, case.v_cache, case.block_table, case.ctx_lens, k_new, v_new,
                 advance=True, status=status)
    torch.cuda.synchronize()
    assert np.array_equal(case.k_cache.view(torch.int16).cpu().numpy(), ref_k)
    assert np.array_equal(case.v_cache.view(torch.int16).cpu().numpy(), ref_v)
    assert case.ctx_lens.tolist() == [1, 16, 17, 34, 201]
    assert int(status.item()) == 0


def test_append_past_capacity_is_skipped_and_flagged(gpu):
    case = make_case(2, 16, 8, [32, 20], 1, seed=230, max_pages=2, device=gpu)  # request 0 full
    k_before = case.k_cache.clone()
    k_new, v_new = _new_token(case, 231)
    status = torch.zeros(1, dtype=torch.int32, device=gpu)
    qf.kv_append(case.k_cache, case.v_cache, case.block_table, case.ctx_lens, k_new, v_new,
                 advance=True, status=status)
    torch.cuda.synchronize()
    assert int(status.item()) == 1
    assert case.ctx_lens.tolist() == [32, 21]
    changed = (case.k_cache != k_before).any(dim=(1, 2, 3)).nonzero().flatten().tolist()
    assert changed == [int(case.block_table[1, 1])]


def test_decode_step_then_append_is_consistent(gpu):
    """Fold with the current token, append it, and sweep n + 1 positions with the same query:
    the two paths reach the same attention (the fold is exact, §2)."""
    case = _allocated_case(gpu, 3, 16, 8, [1000, 5, 77], [4, 1, 2], seed=240)
    k_new, v_new = _new_token(case, 241)
    out_fold, lse_fold = _fold_on_gpu(case, k_new, v_new)
    qf.kv_append(case.k_cache, case.v_cache, case.block_table, case.ctx_lens, k_new, v_new)
    po, pl = qf.attn_decode_split(case.q, case.k_cache, case.v_cache, case.block_table,
                                  case.ctx_lens, case.n_shards, max_shards=case.max_shards,
                                  scale=case.scale)
    out2, lse2 = qf.attn_combine(po, pl)
    torch.cuda.synchronize()
    np.testing.assert_allclose(lse2.cpu().numpy(), lse_fold, rtol=2e-6)
    np.testing.assert_allclose(out2.float().cpu().numpy(), out_fold, atol=1e-2 * 0.05, rtol=1e-2)


@pytest.mark.parametrize("G", [1, 2, 4, 8])
def test_fold_and_append_in_one_launch_equal_the_two_calls(gpu, G):
    """qf_attn_combine_current_append: out, lse, both caches, ctx_lens and status bitwise those of
    qf_attn_combine_current followed by qf_kv_append (advance), for empty, partial-page,
    page-boundary and full requests (the full one is skipped and flagged), at every group size."""
    ctx = [0, 15, 16, 33, 47]
    a = _allocated_case(gpu, 5, 2 * G, 2, ctx, [1, 2, 1, 3, 2], seed=250 + G, max_pages=3)
    a.ctx_lens[4] = 48                           # request 4 is full: three pages of 16
    b = _allocated_case(gpu, 5, 2 * G, 2, ctx, [1, 2, 1, 3, 2], seed=250 + G, max_pages=3)
    b.ctx_lens[4] = 48
    k_new, v_new = _new_token(a, 260 + G)
    po, pl = qf.attn_decode_split(a.q, a.k_cache, a.v_cache, a.block_table, a.ctx_lens,
                                  a.n_shards, max_shards=a.max_shards, scale=a.scale)
    say(f"[current] fold + append in one launch: G={G}")
    sa = torch.zeros(1, dtype=torch.int32, device=gpu)
    sb = torch.zeros(1, dtype=torch.int32, device=gpu)
    out_a, lse_a = qf.attn_combine_current(po, pl, a.q, k_new, v_new, scale=a.scale)
    qf.kv_append(a.k_cache, a.v_cache, a.block_table, a.ctx_lens, k_new, v_new, advance=True,
                 status=sa)
    out_b, lse_b = qf.attn_combine_current_append(po, pl, b.q, k_new, v_new, b.k_cache, b.v_cache,
                                                  b.block_table, b.ctx_lens, scale=b.scale,
                                                  status=sb)
    torch.cuda.synchronize()
    assert torch.equal(out_a.view(torch.int16), out_b.view(torch.int16))
    assert torch.equal(lse_a.view(torch.int32), lse_b.view(torch.int32))
    assert torch.equal(a.k_cache.view(torch.int16), b.k_cache.view(torch.int16))
    assert torch.equal(a.v_cache.view(torch.int16), b.v_cache.view(torch.int16))
    assert a.ctx_lens.tolist() == b.ctx_lens.tolist() == [1, 16, 17, 34, 48]
    assert int(sa.item()) == int(sb.item()) == 1
