"""The C ABI without a GPU: the library loads, exports what include/qfattn.h declares, and rejects
bad arguments on the host with the documented codes before anything is launched."""

import ctypes
import math
import os
import re

import pytest

import paper_2608_15473_amd as qf
from paper_2608_15473_amd.binding import DecodeDesc, load_library

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "qfattn.h")

pytestmark = pytest.mark.skipif(not os.path.exists(qf.LIB_PATH),
                                reason="libqfattn.so not built (python -m paper_2608_15473_amd.build)")


def _declared():
    text = open(HEADER).read()
    return sorted(set(re.findall(r"^\s*(?:int|const char\*)\s+(qf_\w+)\s*\(", text, re.M)))


def test_every_declared_symbol_is_exported():
    lib = load_library()
    names = _declared()
    assert set(names) == set(qf.EXPORTED)
    for name in names:
        assert hasattr(lib, name), name


def test_version_and_error_codes_match_header():
    text = open(HEADER).read()
    assert load_library().qf_version() == int(re.search(r"#define QF_VERSION (\d+)", text).group(1))
    for name, val in [("QF_OK", qf.QF_OK), ("QF_EINVAL", qf.QF_EINVAL),
                      ("QF_EUNSUPPORTED", qf.QF_EUNSUPPORTED), ("QF_EALIGN", qf.QF_EALIGN),
                      ("QF_EHIP", qf.QF_EHIP)]:
        m = re.search(rf"#define {name} \(?(-?\d+)\)?", text)
        assert int(m.group(1)) == val


def _desc(**kw):
    base = dict(batch=2, n_q_heads=16, n_kv_heads=8, head_dim=128, page_size=16,
                max_pages_per_seq=64, num_pages=128, max_shards=4,
                softmax_scale=1 / math.sqrt(128))
    base.update(kw)
    return DecodeDesc(**base)


def _ws(desc):
    n = ctypes.c_size_t(0)
    rc = load_library().qf_attn_decode_split_workspace_size(ctypes.byref(desc), ctypes.byref(n))
    return rc, n.value


@pytest.mark.parametrize("kw,code", [
    (dict(batch=-1), qf.QF_EINVAL),
    (dict(n_q_heads=0), qf.QF_EINVAL),
    (dict(n_q_heads=8192, n_kv_heads=1024), qf.QF_EINVAL),     # above QF_MAX_Q_HEADS
    (dict(n_q_heads=12, n_kv_heads=8), qf.QF_EINVAL),
    (dict(n_q_heads=48, n_kv_heads=3), qf.QF_EUNSUPPORTED),
    (dict(n_q_heads=32, n_kv_heads=2), qf.QF_EUNSUPPORTED),
    (dict(head_dim=64), qf.QF_EUNSUPPORTED),
    (dict(page_size=32), qf.QF_EUNSUPPORTED),
    (dict(max_pages_per_seq=0), qf.QF_EINVAL),
    (dict(num_pages=0), qf.QF_EINVAL),
    (dict(max_shards=0), qf.QF_EINVAL),
    (dict(softmax_scale=float("nan")), qf.QF_EINVAL),
    (dict(max_pages_per_seq=1 << 28), qf.QF_EINVAL),
])
def test_bad_descriptor_is_rejected(kw, code):
    rc, _ = _ws(_desc(**kw))
    assert rc == code
    assert load_library().qf_last_error().decode() != ""
    # the sweep entry point rejects the same descriptor before any launch
    lib = load_library()
    d = _desc(**kw)
    p = ctypes.c_void_p(16)
    rc2 = lib.qf_attn_decode_split(ctypes.byref(d), p, p, p, p, p, p, p, p, p, 1 << 30, None)
    assert rc2 == code


def _order_bytes(d, chunks):
    """The header's rule for the dispatch order in the workspace: an unchunked shape whose shards
    are 128+ pages long at full capacity, with at most 8,192 (request, shard) pairs, keeps one
    int32 per workgroup index (the units rounded up to a multiple of 8)."""
    long = -(-d.max_pages_per_seq // d.max_shards) >= 128
    units = d.batch * d.max_shards * d.n_kv_heads
    ranked = chunks == 1 and long and d.batch * d.max_shards <= 8192
    return 4 * (-(-units // 8) * 8) if ranked else 0


def test_workspace_only_when_units_are_few_or_shards_are_ranked():
    rc, n = _ws(_desc(batch=32, max_shards=64, max_pages_per_seq=2048, num_pages=65536))
    assert rc == 0 and n == 0                              # short shards, many units
    rc, n = _ws(_desc(batch=1, max_shards=16, max_pages_per_seq=65536, num_pages=65536))
    assert rc == 0 and n > 0                               # chunk states
    assert n % 16 == 0
    rc, n = _ws(_desc(batch=48, max_shards=16, max_pages_per_seq=2560, num_pages=65536))
    assert rc == 0 and n == 48 * 16 * 8 * 4                # 160-page shards: the order only
    rc, n = _ws(_desc(batch=64, n_q_heads=32, max_shards=32, max_pages_per_seq=8192,
                      num_pages=140000))
    assert rc == 0 and n == 64 * 32 * 8 * 4                # the ragged 64-request batch
    rc, n = _ws(_desc(batch=3, n_q_heads=3, n_kv_heads=3, max_shards=87, max_pages_per_seq=20000,
                      num_pages=65536))
    assert rc == 0 and n == 784 * 4                        # 783 units, rounded up to 8
    rc, n = _ws(_desc(batch=8193, max_shards=1, max_pages_per_seq=128, num_pages=1 << 21))
    assert rc == 0 and n == 0                              # too many pairs to rank


def _chunks(**kw):
    d = _desc(**kw)
    rc, n = _ws(d)
    assert rc == 0
    per_chunk = d.batch * d.max_shards * d.n_q_heads * (128 + 1) * 4
    for c in range(0, 2049):                               # n = chunk states + dispatch order
        if n == c * per_chunk + _order_bytes(d, max(c, 1)):
            return c
    raise AssertionError(f"workspace of {n} bytes fits no chunk count")


# Sweep workgroups resident on one MI355X (256 CUs) per group size: what the library assumes
# without a device, and what a GPU test requires the device to report.
RESIDENT = {1: 1024, 2: 768, 4: 768, 8: 512}


def _one_unit_chunks(G):
    """Chunks of one (request, shard, KV head) unit of 2^20 positions: one per resident
    workgroup (the page cap, 5,461 at three pages per wavefront, and the 1,024 cap do not bind)."""
    return _chunks(batch=1, n_q_heads=G, n_kv_heads=1, max_shards=1, max_pages_per_seq=65536,
                   num_pages=65536)


def test_chunks_fill_one_set_of_resident_workgroups():
    """Without a GPU to ask, the library assumes the MI355X's resident sweep workgroups (768 at
    G = 2): the 1M-token shape's 128 units take 6 chunks (768 workgroups), whose states are
    B * S * C * Hq * (128 + 1) fp32; a wavefront keeps at least 3 pages (C <= pages / 12), and
    shapes with at least 768 units take none.  (On a GPU the count comes from its occupancy.)"""
    import torch
    if torch.cuda.is_available():
        pytest.skip("the resident-workgroup count is the device's own here")
    assert _chunks(batch=1, max_shards=16, max_pages_per_seq=65536, num_pages=65536) == 6
    assert _chunks(batch=1, max_shards=8, max_pages_per_seq=288, num_pages=288) == 3    # 36 pages
    assert _chunks(batch=3, max_shards=32, max_pages_per_seq=65536, num_pages=65536) == 0  # 768
    for G, resident in RESIDENT.items():
        assert _one_unit_chunks(G) == resident, G


@pytest.mark.gpu
def test_device_resident_workgroups_match_the_host_assumption():
    """The resident sweep workgroups the device reports (HIP occupancy of this build) are the ones
    the library assumes on a host without a GPU, so a workspace sized there fits here."""
    import torch
    assert torch.cuda.is_available()
    for G, resident in RESIDENT.items():
        assert _one_unit_chunks(G) == resident, G


def test_fold_and_append_rejects_before_launch():
    """qf_attn_combine_current_append validates its descriptor and pointers on the host."""
    lib = load_library()
    a = ctypes.c_void_p(4096)
    odd = ctypes.c_void_p(4096 + 2)
    fn = lib.qf_attn_combine_current_append

    def call(d, **over):
        args = dict(po=a, pl=a, q=a, kc=a, vc=a, out=a, lse=None, kk=a, vv=a, bt=a, ctx=a,
                    status=None)
        args.update(over)
        return fn(ctypes.byref(d), *args.values(), None)

    assert call(_desc(n_q_heads=12)) == qf.QF_EINVAL
    assert call(_desc(head_dim=64)) == qf.QF_EUNSUPPORTED
    assert call(_desc(), kk=None) == qf.QF_EINVAL
    assert call(_desc(), ctx=None) == qf.QF_EINVAL
    assert call(_desc(), po=ctypes.c_void_p(4096 + 4)) == qf.QF_EALIGN
    assert call(_desc(), vv=odd) == qf.QF_EALIGN
    assert call(_desc(num_pages=1), bt=None) == qf.QF_EINVAL       # identity map out of the pool
    assert call(_desc(batch=0)) == qf.QF_OK                        # nothing to do
    assert load_library().qf_last_error().decode() == ""


def test_null_and_misaligned_pointers_are_rejected_before_launch():
    lib = load_library()
    d = _desc()
    a = ctypes.c_void_p(4096)
    odd = ctypes.c_void_p(4096 + 8)
    args = [a, a, a, a, a, a, a, a]
    rc = lib.qf_attn_decode_split(ctypes.byref(d), None, *args[1:], None, 0, None)
    assert rc == qf.QF_EINVAL
    rc = lib.qf_attn_decode_split(ctypes.byref(d), odd, a, a, a, a, a, a, a, None, 0, None)
    assert rc == qf.QF_EALIGN
    rc = lib.qf_attn_decode_split(ctypes.byref(d), a, a, a, a, a, a, a, ctypes.c_void_p(4098),
                                  None, 0, None)
    assert rc == qf.QF_EALIGN
    # identity table with too small a pool
    rc = lib.qf_attn_decode_split(ctypes.byref(_desc(num_pages=100)), a, a, a, None, a, a, a, a,
                                  None, 0, None)
    assert rc == qf.QF_EINVAL
    # a shape that needs workspace, called without one
    d1 = _desc(batch=1, max_shards=16, max_pages_per_seq=65536, num_pages=65536)
    rc = lib.qf_attn_decode_split(ctypes.byref(d1), a, a, a, a, a, a, a, a, None, 0, None)
    assert rc == qf.QF_EINVAL and "workspace" in lib.qf_last_error().decode()


def test_combine_rejects_bad_arguments():
    lib = load_library()
    a = ctypes.c_void_p(4096)
    assert lib.qf_attn_combine(-1, 16, 128, 4, a, a, a, a, None) == qf.QF_EINVAL
    assert lib.qf_attn_combine(2, 0, 128, 4, a, a, a, a, None) == qf.QF_EINVAL
    assert lib.qf_attn_combine(2, 4097, 128, 4, a, a, a, a, None) == qf.QF_EINVAL
    assert lib.qf_attn_combine(2, 16, 64, 4, a, a, a, a, None) == qf.QF_EUNSUPPORTED
    assert lib.qf_attn_combine(2, 16, 128, 0, a, a, a, a, None) == qf.QF_EINVAL
    assert lib.qf_attn_combine(2, 16, 128, 4, None, a, a, a, None) == qf.QF_EINVAL
    assert lib.qf_attn_combine(2, 16, 128, 4, ctypes.c_void_p(4104), a, a, a, None) == qf.QF_EALIGN
    assert lib.qf_attn_combine(0, 16, 128, 4, None, None, None, None, None) == qf.QF_OK


def test_current_token_entry_points_reject_bad_arguments():
    lib = load_library()
    a = ctypes.c_void_p(4096)
    f = lib.qf_attn_combine_current
    assert f(-1, 16, 8, 128, 4, a, a, a, a, a, 0.1, a, a, None) == qf.QF_EINVAL
    assert f(2, 16, 6, 128, 4, a, a, a, a, a, 0.1, a, a, None) == qf.QF_EINVAL
    assert f(2, 8192, 1024, 128, 4, a, a, a, a, a, 0.1, a, a, None) == qf.QF_EINVAL
    assert f(2, 16, 8, 64, 4, a, a, a, a, a, 0.1, a, a, None) == qf.QF_EUNSUPPORTED
    assert f(2, 16, 8, 128, 4, a, a, None, a, a, 0.1, a, a, None) == qf.QF_EINVAL
    assert f(2, 16, 8, 128, 4, a, a, a, a, a, float("inf"), a, a, None) == qf.QF_EINVAL
    assert f(2, 16, 8, 128, 4, a, a, ctypes.c_void_p(4098), a, a, 0.1, a, a, None) == qf.QF_EALIGN
    assert f(0, 16, 8, 128, 4, None, None, None, None, None, 0.1, None, None, None) == qf.QF_OK
    g = lib.qf_kv_append
    d = _desc()
    assert g(ctypes.byref(_desc(head_dim=64)), a, a, a, a, a, a, 1, None, None) == qf.QF_EUNSUPPORTED
    assert g(ctypes.byref(d), None, a, a, a, a, a, 1, None, None) == qf.QF_EINVAL
    assert g(ctypes.byref(d), a, a, a, a, ctypes.c_void_p(4099), a, 1, None, None) == qf.QF_EALIGN
    assert g(ctypes.byref(_desc(num_pages=100)), a, a, None, a, a, a, 1, None, None) == qf.QF_EINVAL
    assert g(ctypes.byref(_desc(batch=0)), None, None, None, None, None, None, 1, None, None) == 0


def test_linear_rejects_bad_arguments():
    lib = load_library()
    a = ctypes.c_void_p(4096)
    f = lib.qf_linear
    P, R, S = qf.QF_LINEAR_PLAIN, qf.QF_LINEAR_RMS_NORM, qf.QF_LINEAR_SWIGLU
    assert f(-1, 64, 64, P, a, a, None, 0.0, None, a, 64, None, None) == qf.QF_EINVAL
    assert f(9, 64, 64, P, a, a, None, 0.0, None, a, 64, None, None) == qf.QF_EUNSUPPORTED
    assert f(2, 0, 64, P, a, a, None, 0.0, None, a, 1, None, None) == qf.QF_EINVAL
    assert f(2, 64, 4, P, a, a, None, 0.0, None, a, 64, None, None) == qf.QF_EINVAL
    assert f(2, 64, 60, P, a, a, None, 0.0, None, a, 64, None, None) == qf.QF_EUNSUPPORTED
    assert f(2, 64, 64, 7, a, a, None, 0.0, None, a, 64, None, None) == qf.QF_EINVAL
    assert f(2, 64, 64, P, a, a, None, 0.0, None, a, 0, None, None) == qf.QF_EINVAL
    assert f(2, 64, 64, P, a, a, None, 0.0, None, a, 65, None, None) == qf.QF_EINVAL
    assert f(2, 64, 64, R, a, a, a, -1.0, None, a, 64, None, None) == qf.QF_EINVAL
    assert f(2, 64, 64, R, a, a, a, float("nan"), None, a, 64, None, None) == qf.QF_EINVAL
    assert f(2, 64, 64, R, a, a, None, 1e-6, None, a, 64, None, None) == qf.QF_EINVAL
    assert f(2, 64, 64, P, a, a, None, 0.0, None, a, 32, None, None) == qf.QF_EINVAL
    assert f(2, 64, 64, P, None, a, None, 0.0, None, a, 64, None, None) == qf.QF_EINVAL
    assert f(2, 64, 64, S, a, ctypes.c_void_p(4104), None, 0.0, None, a, 64, None,
             None) == qf.QF_EALIGN
    assert f(2, 64, 64, P, a, a, None, 0.0, ctypes.c_void_p(4097), a, 64, None,
             None) == qf.QF_EALIGN
    assert f(0, 64, 64, P, None, None, None, 0.0, None, None, 64, None, None) == qf.QF_OK
    G = qf.QF_LINEAR_GLU_OUT
    assert f(2, 63, 64, R | G, a, a, a, 1e-6, None, a, 63, None, None) == qf.QF_EINVAL   # odd
    assert f(2, 64, 64, R | G, a, a, a, 1e-6, a, a, 64, None, None) == qf.QF_EINVAL     # residual
    assert f(2, 64, 64, R | G, a, a, a, 1e-6, None, a, 32, a, None) == qf.QF_EINVAL     # split
    assert f(2, 64, 64, S | G, a, a, None, 0.0, None, a, 64, None, None) == qf.QF_EINVAL  # swiglu in
    assert f(2, 64, 64, 4 | G, a, a, None, 0.0, None, a, 64, None, None) == qf.QF_EINVAL  # unknown


def test_beside_checks_both_calls_before_launching():
    lib = load_library()
    a = ctypes.c_void_p(4096)
    d = _desc()
    la = qf.LinearArgs(2, 64, 64, qf.QF_LINEAR_PLAIN, 4096, 4096, None, 0.0, None, 4096, 64, None)
    f = lib.qf_attn_decode_split_beside
    args = (a, a, a, a, a, a, a, a, a, 1 << 40)
    assert f(ctypes.byref(d), *args, None, None) == qf.QF_EINVAL
    assert f(ctypes.byref(_desc(head_dim=64)), *args, ctypes.byref(la), None) == qf.QF_EUNSUPPORTED
    bad = qf.LinearArgs(9, 64, 64, qf.QF_LINEAR_PLAIN, 4096, 4096, None, 0.0, None, 4096, 64, None)
    assert f(ctypes.byref(d), *args, ctypes.byref(bad), None) == qf.QF_EUNSUPPORTED
    nul = qf.LinearArgs(2, 64, 64, qf.QF_LINEAR_PLAIN, None, 4096, None, 0.0, None, 4096, 64, None)
    assert f(ctypes.byref(d), *args, ctypes.byref(nul), None) == qf.QF_EINVAL
    none = qf.LinearArgs(0, 64, 64, qf.QF_LINEAR_PLAIN, None, None, None, 0.0, None, None, 64, None)
    assert f(ctypes.byref(_desc(batch=0)), None, None, None, None, None, None, None, None, None, 0,
             ctypes.byref(none), None) == qf.QF_OK


def test_one_launch_decode_rejects_bad_arguments():
    lib = load_library()
    a = ctypes.c_void_p(4096)
    d = _desc()
    n = ctypes.c_size_t(0)
    assert lib.qf_attn_decode_workspace_size(ctypes.byref(d), None) == qf.QF_EINVAL
    assert lib.qf_attn_decode_workspace_size(ctypes.byref(d), ctypes.byref(n)) == qf.QF_OK
    assert n.value > 0
    f = lib.qf_attn_decode
    ws = n.value
    assert f(ctypes.byref(d), a, a, a, a, a, a, None, None, a, ws, a, 16, None) == qf.QF_EINVAL
    assert f(ctypes.byref(d), a, a, a, a, a, a, a, None, None, ws, a, 16, None) == qf.QF_EINVAL
    assert f(ctypes.byref(d), a, a, a, a, a, a, a, None, a, ws, None, 16, None) == qf.QF_EINVAL
    assert f(ctypes.byref(d), a, a, a, a, a, a, a, None, a, ws, a, 15, None) == qf.QF_EINVAL
    assert f(ctypes.byref(d), a, a, a, a, a, a, a, None, a, ws - 1, a, 16, None) == qf.QF_EINVAL
    assert f(ctypes.byref(d), a, a, a, a, a, a, a, None, ctypes.c_void_p(4100), ws, a, 16,
             None) == qf.QF_EALIGN
    assert f(ctypes.byref(d), a, a, a, a, a, a, a, None, a, ws, ctypes.c_void_p(4098), 16,
             None) == qf.QF_EALIGN
    assert f(ctypes.byref(_desc(head_dim=64)), a, a, a, a, a, a, a, None, a, ws, a, 16,
             None) == qf.QF_EUNSUPPORTED
    assert f(ctypes.byref(_desc(batch=0)), None, None, None, None, None, None, None, None, None,
             0, None, 0, None) == qf.QF_OK


def test_empty_batch_is_a_no_op():
    lib = load_library()
    d = _desc(batch=0)
    assert lib.qf_attn_decode_split(ctypes.byref(d), None, None, None, None, None, None, None,
                                    None, None, 0, None) == qf.QF_OK


def test_binding_refuses_cpu_tensors():
    import torch
    q = torch.zeros(1, 16, 128, dtype=torch.bfloat16)
    k = torch.zeros(4, 8, 16, 128, dtype=torch.bfloat16)
    with pytest.raises(qf.QFError):
        qf.attn_decode_split(q, k, k, None, torch.zeros(1, dtype=torch.int32), 1)


def test_chunk_count_agrees_with_the_workspace():
    """qf_attn_decode_split_chunks gives the chunk count behind the workspace size: the chunk
    states are B * S * C * Hq * (128 + 1) fp32 when C > 1 (none when C == 1), followed by the
    dispatch order of a ranked shape (B * S int32)."""
    lib = load_library()
    for kw in [dict(batch=1, max_shards=16, max_pages_per_seq=65536, num_pages=65536),
               dict(batch=1, max_shards=8, max_pages_per_seq=288, num_pages=288),
               dict(batch=3, max_shards=32, max_pages_per_seq=65536, num_pages=65536),
               dict(batch=1, n_q_heads=8, n_kv_heads=1, max_shards=1, max_pages_per_seq=65536,
                    num_pages=65536),
               dict(batch=2, max_shards=4)]:
        d = _desc(**kw)
        c = ctypes.c_int32(0)
        assert lib.qf_attn_decode_split_chunks(ctypes.byref(d), ctypes.byref(c)) == qf.QF_OK
        rc, n = _ws(d)
        assert rc == 0 and c.value >= 1
        per_chunk = d.batch * d.max_shards * d.n_q_heads * (128 + 1) * 4
        states = 0 if c.value == 1 else c.value * per_chunk
        assert n == states + _order_bytes(d, c.value), (kw, c.value, n)
    bad = _desc(n_q_heads=12, n_kv_heads=8)
    assert lib.qf_attn_decode_split_chunks(ctypes.byref(bad), ctypes.byref(c)) == qf.QF_EINVAL
    assert lib.qf_attn_decode_split_chunks(ctypes.byref(_desc()), None) == qf.QF_EINVAL


def test_unfolded_sweep_rejects_before_launch():
    """qf_attn_decode_split_unfolded validates the descriptor and its pointers on the host."""
    lib = load_library()
    a = ctypes.c_void_p(4096)
    fn = lib.qf_attn_decode_split_unfolded
    d = _desc()
    c = ctypes.c_int32(0)
    assert lib.qf_attn_decode_split_chunks(ctypes.byref(d), ctypes.byref(c)) == qf.QF_OK
    slots = d.max_shards * c.value
    assert fn(ctypes.byref(d), a, a, a, None, a, a, a, None, slots, None) == qf.QF_EINVAL
    assert fn(ctypes.byref(d), ctypes.c_void_p(4098), a, a, None, a, a, a, a, slots,
              None) == qf.QF_EALIGN
    # slot arrays sized for another chunk count (e.g. by max_shards alone on a chunked shape):
    # refused before anything is enqueued
    for wrong in (slots - 1, slots + 1, d.max_shards if c.value > 1 else 0):
        assert fn(ctypes.byref(d), a, a, a, None, a, a, a, a, wrong, None) == qf.QF_EINVAL
        assert "slots" in lib.qf_last_error().decode()
    chunked = _desc(batch=1, max_shards=16, max_pages_per_seq=65536, num_pages=65536)
    assert lib.qf_attn_decode_split_chunks(ctypes.byref(chunked), ctypes.byref(c)) == qf.QF_OK
    assert c.value > 1
    assert fn(ctypes.byref(chunked), a, a, a, None, a, a, a, a, 16, None) == qf.QF_EINVAL
    bad = _desc(head_dim=64)
    assert fn(ctypes.byref(bad), a, a, a, None, a, a, a, a, slots, None) == qf.QF_EUNSUPPORTED
    empty = _desc(batch=0)
    assert fn(ctypes.byref(empty), None, None, None, None, None, None, None, None, 0,
              None) == qf.QF_OK
