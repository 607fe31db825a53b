"""ctypes binding of libqfattn.so (include/qfattn.h): argument marshalling only.

Every step of the computation runs in the HIP kernels behind the C ABI; this module turns torch
tensors into device pointers, picks the caller's current HIP stream and raises on error codes.
There is no fallback: if the library is missing or the tensors are not on a GPU, calls raise.
"""

from __future__ import annotations

import ctypes
import os

import torch

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "lib", "libqfattn.so")

QF_OK, QF_EINVAL, QF_EUNSUPPORTED, QF_EALIGN, QF_EHIP = 0, -1, -2, -3, -4
EXPORTED = ("qf_attn_decode_split_workspace_size", "qf_attn_decode_split", "qf_attn_combine",
            "qf_attn_decode_split_chunks", "qf_attn_decode_split_unfolded",
            "qf_attn_decode_workspace_size", "qf_attn_decode", "qf_attn_decode_noalloc",
            "qf_attn_combine_current", "qf_attn_combine_current_append", "qf_kv_append",
            "qf_linear", "qf_attn_decode_split_beside",
            "qf_schedule_simulate", "qf_last_error", "qf_version")
QF_WIRING_QFIRST, QF_WIRING_COMPOSED = 0, 1
QF_LINEAR_PLAIN, QF_LINEAR_RMS_NORM, QF_LINEAR_SWIGLU, QF_LINEAR_GLU_OUT = 0, 1, 2, 16


class QFError(RuntimeError):
    def __init__(self, code: int, msg: str):
        super().__init__(f"qfattn error {code}: {msg}")
        self.code = code


class DecodeDesc(ctypes.Structure):
    _fields_ = [("batch", ctypes.c_int32), ("n_q_heads", ctypes.c_int32),
                ("n_kv_heads", ctypes.c_int32), ("head_dim", ctypes.c_int32),
                ("page_size", ctypes.c_int32), ("max_pages_per_seq", ctypes.c_int32),
                ("num_pages", ctypes.c_int32), ("max_shards", ctypes.c_int32),
                ("softmax_scale", ctypes.c_float)]


class LinearArgs(ctypes.Structure):
    _fields_ = [("rows", ctypes.c_int32), ("n_out", ctypes.c_int32), ("k", ctypes.c_int32),
                ("prologue", ctypes.c_int32), ("x", ctypes.c_void_p), ("w", ctypes.c_void_p),
                ("gain", ctypes.c_void_p), ("eps", ctypes.c_float), ("residual", ctypes.c_void_p),
                ("out", ctypes.c_void_p), ("n_split", ctypes.c_int32), ("out_b", ctypes.c_void_p)]


_lib = None


def load_library(path: str = LIB_PATH) -> ctypes.CDLL:
    """Load (once) and return the C library; raises if it has not been built."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(path):
        raise QFError(QF_EHIP, f"{path} not found: build it with "
                               "`python -m paper_2608_15473_amd.build`")
    lib = ctypes.CDLL(path)
    vp, i32, sz = ctypes.c_void_p, ctypes.c_int32, ctypes.c_size_t
    lib.qf_attn_decode_split_workspace_size.argtypes = [ctypes.POINTER(DecodeDesc),
                                                        ctypes.POINTER(sz)]
    lib.qf_attn_decode_split.argtypes = [ctypes.POINTER(DecodeDesc), vp, vp, vp, vp, vp, vp, vp,
                                         vp, vp, sz, vp]
    lib.qf_attn_combine.argtypes = [i32, i32, i32, i32, vp, vp, vp, vp, vp]
    lib.qf_attn_decode_split_chunks.argtypes = [ctypes.POINTER(DecodeDesc),
                                                ctypes.POINTER(ctypes.c_int32)]
    lib.qf_attn_decode_split_unfolded.argtypes = [ctypes.POINTER(DecodeDesc), vp, vp, vp, vp, vp,
                                                  vp, vp, vp, i32, vp]
    lib.qf_attn_decode_workspace_size.argtypes = [ctypes.POINTER(DecodeDesc), ctypes.POINTER(sz)]
    lib.qf_attn_decode.argtypes = [ctypes.POINTER(DecodeDesc), vp, vp, vp, vp, vp, vp, vp, vp, vp,
                                   sz, vp, ctypes.c_int64, vp]
    lib.qf_attn_decode_noalloc.argtypes = [ctypes.POINTER(DecodeDesc), vp, vp, vp, vp, vp, vp, vp,
                                           vp, vp]
    lib.qf_attn_combine_current.argtypes = [i32, i32, i32, i32, i32, vp, vp, vp, vp, vp,
                                            ctypes.c_float, vp, vp, vp]
    lib.qf_attn_combine_current_append.argtypes = [ctypes.POINTER(DecodeDesc), vp, vp, vp, vp, vp,
                                                   vp, vp, vp, vp, vp, vp, vp, vp]
    lib.qf_kv_append.argtypes = [ctypes.POINTER(DecodeDesc), vp, vp, vp, vp, vp, vp, i32, vp, vp]
    lib.qf_linear.argtypes = [i32, i32, i32, i32, vp, vp, vp, ctypes.c_float, vp, vp, i32, vp,
                              vp]
    lib.qf_attn_decode_split_beside.argtypes = [ctypes.POINTER(DecodeDesc), vp, vp, vp, vp, vp, vp,
                                                vp, vp, vp, sz, ctypes.POINTER(LinearArgs), vp]
    dp = ctypes.POINTER(ctypes.c_double)
    lib.qf_schedule_simulate.argtypes = [i32, dp, dp, i32, i32, ctypes.c_double, i32,
                                         ctypes.c_double, dp, dp, dp, dp, dp]
    lib.qf_last_error.restype = ctypes.c_char_p
    lib.qf_last_error.argtypes = []
    lib.qf_version.argtypes = []
    for name in ("qf_attn_decode_split_workspace_size", "qf_attn_decode_split",
                 "qf_attn_decode_split_chunks", "qf_attn_decode_split_unfolded",
                 "qf_attn_decode_workspace_size", "qf_attn_decode", "qf_attn_decode_noalloc",
                 "qf_attn_combine", "qf_attn_combine_current", "qf_attn_combine_current_append",
                 "qf_kv_append",
                 "qf_linear", "qf_attn_decode_split_beside", "qf_schedule_simulate", "qf_version"):
        getattr(lib, name).restype = ctypes.c_int
    _lib = lib
    return lib


def _check(rc: int) -> None:
    if rc != QF_OK:
        raise QFError(rc, load_library().qf_last_error().decode())


def _ptr(t):
    return None if t is None else ctypes.c_void_p(t.data_ptr())


def _require(t, name, dtype, dim=None):
    if not isinstance(t, torch.Tensor):
        raise TypeError(f"{name} must be a torch.Tensor")
    if t.device.type != "cuda":
        raise QFError(QF_EINVAL, f"{name} must be a GPU tensor (got {t.device})")
    if t.dtype != dtype:
        raise QFError(QF_EINVAL, f"{name} must be {dtype} (got {t.dtype})")
    if not t.is_contiguous():
        raise QFError(QF_EINVAL, f"{name} must be contiguous")
    if dim is not None and t.dim() != dim:
        raise QFError(QF_EINVAL, f"{name} must have {dim} dimensions (got {t.dim()})")


def make_desc(q, k_cache, block_table, max_shards, scale, num_pages=None, max_pages=None):
    B, Hq, D = q.shape
    P, Hkv = k_cache.shape[2], k_cache.shape[1]
    if max_pages is None:
        max_pages = block_table.shape[1] if block_table is not None else k_cache.shape[0] // max(B, 1)
    return DecodeDesc(B, Hq, Hkv, D, P, int(max_pages),
                      int(k_cache.shape[0] if num_pages is None else num_pages),
                      int(max_shards), float(scale))


def workspace_size(desc: DecodeDesc) -> int:
    n = ctypes.c_size_t(0)
    _check(load_library().qf_attn_decode_split_workspace_size(ctypes.byref(desc), ctypes.byref(n)))
    return n.value


def split_chunks(desc: DecodeDesc) -> int:
    """Sub-shard chunks per shard the sweep uses for this shape (qf_attn_decode_split_chunks)."""
    c = ctypes.c_int32(0)
    _check(load_library().qf_attn_decode_split_chunks(ctypes.byref(desc), ctypes.byref(c)))
    return c.value


def _split_call(q, k_cache, v_cache, block_table, ctx_lens, n_shards, max_shards, scale,
                part_out, part_lse, workspace, max_pages, unfolded=False):
    """Checks and allocations of qf_attn_decode_split (or, ``unfolded``, of
    qf_attn_decode_split_unfolded, whose slot arrays hold max_shards * chunks slots and which takes
    no workspace): returns (C arguments, descriptor, part_out, part_lse, workspace, n_shards), the
    last three as tensors the C arguments point into."""
    _require(q, "q", torch.bfloat16, 3)
    _require(k_cache, "k_cache", torch.bfloat16, 4)
    _require(v_cache, "v_cache", torch.bfloat16, 4)
    if v_cache.shape != k_cache.shape:
        raise QFError(QF_EINVAL, "k_cache and v_cache shapes differ")
    if block_table is not None:
        _require(block_table, "block_table", torch.int32, 2)
    _require(ctx_lens, "ctx_lens", torch.int32, 1)
    B = q.shape[0]
    if isinstance(n_shards, int):
        if max_shards is None:
            max_shards = n_shards
        n_shards = torch.full((B,), n_shards, dtype=torch.int32, device=q.device)
    _require(n_shards, "n_shards", torch.int32, 1)
    if max_shards is None:
        raise QFError(QF_EINVAL, "max_shards is required when n_shards is a tensor")
    if scale is None:
        scale = q.shape[-1] ** -0.5
    desc = make_desc(q, k_cache, block_table, max_shards, scale, max_pages=max_pages)
    Hq, D = q.shape[1], q.shape[2]
    slots = max_shards * (split_chunks(desc) if unfolded else 1)
    if part_out is None:
        part_out = torch.empty((B, slots, Hq, D), dtype=torch.float32, device=q.device)
    if part_lse is None:
        part_lse = torch.empty((B, slots, Hq), dtype=torch.float32, device=q.device)
    _require(part_out, "part_out", torch.float32)
    _require(part_lse, "part_lse", torch.float32)
    if tuple(part_out.shape) != (B, slots, Hq, D) or tuple(part_lse.shape) != (B, slots, Hq):
        raise QFError(QF_EINVAL, f"partial outputs must be [{B}, {slots}, {Hq}, {D}] and "
                                 f"[{B}, {slots}, {Hq}] (got {tuple(part_out.shape)} and "
                                 f"{tuple(part_lse.shape)})")
    head = (ctypes.byref(desc), _ptr(q), _ptr(k_cache), _ptr(v_cache), _ptr(block_table),
            _ptr(ctx_lens), _ptr(n_shards), _ptr(part_out), _ptr(part_lse))
    if unfolded:
        return head + (slots,), desc, part_out, part_lse, None, n_shards
    need = workspace_size(desc)
    if need and workspace is None:
        workspace = torch.empty(need, dtype=torch.uint8, device=q.device)
    ws_bytes = 0 if workspace is None else workspace.numel() * workspace.element_size()
    args = head + (_ptr(workspace), ws_bytes)
    return args, desc, part_out, part_lse, workspace, n_shards


def attn_decode_split(q, k_cache, v_cache, block_table, ctx_lens, n_shards, max_shards=None,
                      scale=None, part_out=None, part_lse=None, workspace=None,
                      max_pages=None):
    """The sweep split into position shards (qf_attn_decode_split).

    q bf16 [B, Hq, D]; k_cache / v_cache bf16 [num_pages, Hkv, P, D]; block_table int32
    [B, max_pages] or None (identity); ctx_lens int32 [B]; n_shards an int or int32 [B].
    Returns (part_out fp32 [B, S_max, Hq, D], part_lse fp32 [B, S_max, Hq]).
    """
    args, desc, part_out, part_lse, workspace, n_shards = _split_call(
        q, k_cache, v_cache, block_table, ctx_lens, n_shards, max_shards, scale, part_out,
        part_lse, workspace, max_pages)
    stream = torch.cuda.current_stream(q.device).cuda_stream
    _check(load_library().qf_attn_decode_split(*args, ctypes.c_void_p(stream)))
    return part_out, part_lse


def attn_decode_split_unfolded(q, k_cache, v_cache, block_table, ctx_lens, n_shards,
                               max_shards=None, scale=None, slot_out=None, slot_lse=None,
                               max_pages=None):
    """The sweep with its sub-shard chunks left as slots (qf_attn_decode_split_unfolded).

    Arguments as for ``attn_decode_split``.  Returns (slot_out fp32 [B, S_max * C, Hq, D],
    slot_lse fp32 [B, S_max * C, Hq]), C = the sweep's chunks per shard: slot s * C + c is chunk c
    of shard s.  ``attn_combine`` over them gives the merged attention with one launch fewer than
    ``attn_decode_split`` when C > 1.
    """
    args, desc, slot_out, slot_lse, _, n_shards = _split_call(
        q, k_cache, v_cache, block_table, ctx_lens, n_shards, max_shards, scale, slot_out,
        slot_lse, None, max_pages, unfolded=True)
    stream = torch.cuda.current_stream(q.device).cuda_stream
    _check(load_library().qf_attn_decode_split_unfolded(*args, ctypes.c_void_p(stream)))
    return slot_out, slot_lse


def attn_decode_split_beside(q, k_cache, v_cache, block_table, ctx_lens, n_shards, beside,
                             max_shards=None, scale=None, part_out=None, part_lse=None,
                             workspace=None, max_pages=None):
    """The sweep and one fused product in a single launch (qf_attn_decode_split_beside).

    The sweep's arguments are those of ``attn_decode_split``; ``beside`` is a dict of ``linear``'s
    keyword arguments (x, w, prologue, gain, eps, residual, out, split, out_b).  Returns
    (part_out, part_lse, the product's output(s)); bitwise the results of the two separate calls.
    """
    args, desc, part_out, part_lse, workspace, n_shards = _split_call(
        q, k_cache, v_cache, block_table, ctx_lens, n_shards, max_shards, scale, part_out,
        part_lse, workspace, max_pages)
    la, result = _linear_call(**beside)
    stream = torch.cuda.current_stream(q.device).cuda_stream
    _check(load_library().qf_attn_decode_split_beside(*args, ctypes.byref(la),
                                                      ctypes.c_void_p(stream)))
    return part_out, part_lse, result


def attn_combine(part_out, part_lse, out=None, lse=None, want_lse=True):
    """Merge every shard slot (qf_attn_combine): returns (out bf16 [B, Hq, D], lse fp32 [B, Hq])."""
    _require(part_out, "part_out", torch.float32, 4)
    _require(part_lse, "part_lse", torch.float32, 3)
    B, S, Hq, D = part_out.shape
    if tuple(part_lse.shape) != (B, S, Hq):
        raise QFError(QF_EINVAL, "part_lse shape does not match part_out")
    if out is None:
        out = torch.empty((B, Hq, D), dtype=torch.bfloat16, device=part_out.device)
    if lse is None and want_lse:
        lse = torch.empty((B, Hq), dtype=torch.float32, device=part_out.device)
    stream = torch.cuda.current_stream(part_out.device).cuda_stream
    _check(load_library().qf_attn_combine(B, Hq, D, S, _ptr(part_out), _ptr(part_lse), _ptr(out),
                                          _ptr(lse), ctypes.c_void_p(stream)))
    return out, lse


class DecodeStepPlan:
    """attn_decode_split then attn_combine on fixed buffers, checked and converted once.

    The arguments are those of ``attn_decode_split`` (plus ``out`` / ``lse`` of ``attn_combine``);
    every tensor, the workspace included, is allocated here when not given and kept by the plan.
    With ``fold_chunks=False`` and a chunked shape the sweep is ``attn_decode_split_unfolded`` (its
    sub-shard chunks stay slots of part_out / part_lse, [B, S_max * C, ...], and the combine merges
    them: one launch fewer); otherwise, C == 1 included, it is ``attn_decode_split`` and part_out /
    part_lse are the per-shard partials (with C == 1 the two calls give the same bits, and the
    split, having a workspace, also ranks a ragged batch's long shards by length).
    Calling the plan enqueues the two library calls on ``stream`` (default: the current stream at
    construction) with the pointers taken at construction, so the caller updates tensors in
    place (e.g. the query, the cache, ctx_lens) and never reallocates them; per call the host does
    two foreign calls and nothing else, which matters when the kernels take a few microseconds.
    Returns (out, lse).
    """

    def __init__(self, q, k_cache, v_cache, block_table, ctx_lens, n_shards, max_shards=None,
                 scale=None, part_out=None, part_lse=None, out=None, lse=None, workspace=None,
                 max_pages=None, stream=None, fold_chunks=True):
        args, desc, part_out, part_lse, workspace, n_shards = _split_call(
            q, k_cache, v_cache, block_table, ctx_lens, n_shards, max_shards, scale, part_out,
            part_lse, workspace, max_pages, unfolded=not fold_chunks)
        if not fold_chunks and split_chunks(desc) == 1:
            fold_chunks = True
            args, desc, part_out, part_lse, workspace, n_shards = _split_call(
                q, k_cache, v_cache, block_table, ctx_lens, n_shards, desc.max_shards,
                desc.softmax_scale, part_out, part_lse, workspace, max_pages)
        B, S, Hq, D = part_out.shape
        if out is None:
            out = torch.empty((B, Hq, D), dtype=torch.bfloat16, device=q.device)
        if lse is None:
            lse = torch.empty((B, Hq), dtype=torch.float32, device=q.device)
        _require(out, "out", torch.bfloat16, 3)
        _require(lse, "lse", torch.float32, 2)
        if tuple(out.shape) != (B, Hq, D) or tuple(lse.shape) != (B, Hq):
            raise QFError(QF_EINVAL, "out / lse shapes do not match the partials")
        if stream is None:
            stream = torch.cuda.current_stream(q.device).cuda_stream
        # keep every buffer (and the descriptor the first call points to) alive with the plan
        self._keep = (q, k_cache, v_cache, block_table, ctx_lens, n_shards, part_out, part_lse,
                      out, lse, workspace, desc)
        self._desc = desc
        lib = load_library()
        self._split = lib.qf_attn_decode_split if fold_chunks else lib.qf_attn_decode_split_unfolded
        self._combine = lib.qf_attn_combine
        self._split_args = args + (ctypes.c_void_p(stream),)
        self._combine_args = (B, Hq, D, S, _ptr(part_out), _ptr(part_lse), _ptr(out), _ptr(lse),
                              ctypes.c_void_p(stream))
        self.part_out, self.part_lse, self.out, self.lse = part_out, part_lse, out, lse

    def split(self):
        """Enqueue the sweep (qf_attn_decode_split, or its unfolded form) into part_out / part_lse."""
        rc = self._split(*self._split_args)
        if rc != QF_OK:
            raise QFError(rc, load_library().qf_last_error().decode())

    def combine(self):
        """Enqueue the merge of the partials (qf_attn_combine) into out / lse."""
        rc = self._combine(*self._combine_args)
        if rc != QF_OK:
            raise QFError(rc, load_library().qf_last_error().decode())

    def __call__(self):
        self.split()
        self.combine()
        return self.out, self.lse


def attn_combine_current(part_out, part_lse, q, k_cur, v_cur, scale=None, out=None, lse=None):
    """Merge the shard slots, then fold in the current token (qf_attn_combine_current):
    returns (out bf16 [B, Hq, D], lse fp32 [B, Hq]) = attention over cache + current token."""
    _require(part_out, "part_out", torch.float32, 4)
    _require(part_lse, "part_lse", torch.float32, 3)
    _require(q, "q", torch.bfloat16, 3)
    _require(k_cur, "k_cur", torch.bfloat16, 3)
    _require(v_cur, "v_cur", torch.bfloat16, 3)
    B, S, Hq, D = part_out.shape
    Hkv = k_cur.shape[1]
    if tuple(q.shape) != (B, Hq, D) or tuple(k_cur.shape) != (B, Hkv, D) or v_cur.shape != k_cur.shape:
        raise QFError(QF_EINVAL, "q / k_cur / v_cur shapes do not match the partials")
    if scale is None:
        scale = D ** -0.5
    if out is None:
        out = torch.empty((B, Hq, D), dtype=torch.bfloat16, device=part_out.device)
    if lse is None:
        lse = torch.empty((B, Hq), dtype=torch.float32, device=part_out.device)
    stream = torch.cuda.current_stream(part_out.device).cuda_stream
    _check(load_library().qf_attn_combine_current(
        B, Hq, Hkv, D, S, _ptr(part_out), _ptr(part_lse), _ptr(q), _ptr(k_cur), _ptr(v_cur),
        float(scale), _ptr(out), _ptr(lse), ctypes.c_void_p(stream)))
    return out, lse


def attn_combine_current_append(part_out, part_lse, q, k_cur, v_cur, k_cache, v_cache, block_table,
                                ctx_lens, scale=None, out=None, lse=None, status=None,
                                max_pages=None):
    """attn_combine_current, then kv_append of k_cur / v_cur with the context lengths advanced,
    in one launch (qf_attn_combine_current_append); returns (out, lse)."""
    _require(part_out, "part_out", torch.float32, 4)
    _require(part_lse, "part_lse", torch.float32, 3)
    _require(q, "q", torch.bfloat16, 3)
    _require(k_cur, "k_cur", torch.bfloat16, 3)
    _require(v_cur, "v_cur", torch.bfloat16, 3)
    _require(k_cache, "k_cache", torch.bfloat16, 4)
    _require(v_cache, "v_cache", torch.bfloat16, 4)
    _require(ctx_lens, "ctx_lens", torch.int32, 1)
    if block_table is not None:
        _require(block_table, "block_table", torch.int32, 2)
    if status is not None:
        _require(status, "status", torch.int32)
    B, S, Hq, D = part_out.shape
    Hkv, P = k_cache.shape[1], k_cache.shape[2]
    if (tuple(q.shape) != (B, Hq, D) or tuple(k_cur.shape) != (B, Hkv, D)
            or v_cur.shape != k_cur.shape or v_cache.shape != k_cache.shape
            or k_cache.shape[3] != D or ctx_lens.shape[0] != B):
        raise QFError(QF_EINVAL, "q / k_cur / v_cur / cache / ctx_lens shapes do not match the partials")
    if scale is None:
        scale = D ** -0.5
    if max_pages is None:
        max_pages = block_table.shape[1] if block_table is not None else k_cache.shape[0] // max(B, 1)
    if out is None:
        out = torch.empty((B, Hq, D), dtype=torch.bfloat16, device=part_out.device)
    if lse is None:
        lse = torch.empty((B, Hq), dtype=torch.float32, device=part_out.device)
    desc = DecodeDesc(B, Hq, Hkv, D, P, int(max_pages), int(k_cache.shape[0]), S, float(scale))
    stream = torch.cuda.current_stream(part_out.device).cuda_stream
    _check(load_library().qf_attn_combine_current_append(
        ctypes.byref(desc), _ptr(part_out), _ptr(part_lse), _ptr(q), _ptr(k_cur), _ptr(v_cur),
        _ptr(out), _ptr(lse), _ptr(k_cache), _ptr(v_cache), _ptr(block_table), _ptr(ctx_lens),
        _ptr(status), ctypes.c_void_p(stream)))
    return out, lse


def kv_append(k_cache, v_cache, block_table, ctx_lens, k_new, v_new, advance=True, status=None,
              max_pages=None):
    """Write each request's current key/value at position ctx_lens[b] (qf_kv_append); with
    ``advance`` the context lengths are incremented on the device after the write."""
    _require(k_cache, "k_cache", torch.bfloat16, 4)
    _require(v_cache, "v_cache", torch.bfloat16, 4)
    _require(ctx_lens, "ctx_lens", torch.int32, 1)
    _require(k_new, "k_new", torch.bfloat16, 3)
    _require(v_new, "v_new", torch.bfloat16, 3)
    if block_table is not None:
        _require(block_table, "block_table", torch.int32, 2)
    if status is not None:
        _require(status, "status", torch.int32)
    B = ctx_lens.shape[0]
    Hkv, P, D = k_cache.shape[1], k_cache.shape[2], k_cache.shape[3]
    if max_pages is None:
        max_pages = block_table.shape[1] if block_table is not None else k_cache.shape[0] // max(B, 1)
    desc = DecodeDesc(B, Hkv, Hkv, D, P, int(max_pages), int(k_cache.shape[0]), 1, 1.0)
    stream = torch.cuda.current_stream(k_cache.device).cuda_stream
    _check(load_library().qf_kv_append(ctypes.byref(desc), _ptr(k_cache), _ptr(v_cache),
                                       _ptr(block_table), _ptr(ctx_lens), _ptr(k_new),
                                       _ptr(v_new), 1 if advance else 0, _ptr(status),
                                       ctypes.c_void_p(stream)))


_PROLOGUES = {None: QF_LINEAR_PLAIN, "rms_norm": QF_LINEAR_RMS_NORM, "swiglu": QF_LINEAR_SWIGLU}


def _linear_call(x, w, prologue=None, gain=None, eps=1e-6, residual=None, out=None, split=None,
                 out_b=None, glu_out=False):
    """Checks and allocations of qf_linear: returns (LinearArgs, the output(s))."""
    if prologue not in _PROLOGUES:
        raise QFError(QF_EINVAL, f"unknown prologue {prologue!r}")
    _require(x, "x", torch.bfloat16, 2)
    _require(w, "w", torch.bfloat16, 2)
    M = x.shape[0]
    N, K = w.shape
    if x.shape[1] != (2 * K if prologue == "swiglu" else K):
        raise QFError(QF_EINVAL, f"x has {x.shape[1]} columns for a weight of {K} inputs")
    if gain is not None:
        _require(gain, "gain", torch.bfloat16, 1)
    if residual is not None:
        _require(residual, "residual", torch.bfloat16, 2)
        if tuple(residual.shape) != (M, N):
            raise QFError(QF_EINVAL, "residual must be [M, N]")
    n_split = N if split is None else int(split)
    if glu_out and (N % 2 or n_split != N or residual is not None or prologue == "swiglu"):
        raise QFError(QF_EINVAL, "glu_out needs an even N, no split, no residual, no swiglu input")
    cols = N // 2 if glu_out else n_split
    if out is None:
        out = torch.empty((M, cols), dtype=torch.bfloat16, device=x.device)
    if n_split < N and out_b is None:
        out_b = torch.empty((M, N - n_split), dtype=torch.bfloat16, device=x.device)
    _require(out, "out", torch.bfloat16)
    if out.numel() != M * cols:
        raise QFError(QF_EINVAL, f"out must hold [M, {cols}] elements")
    if out_b is not None:
        _require(out_b, "out_b", torch.bfloat16)
        if out_b.numel() != M * (N - n_split):
            raise QFError(QF_EINVAL, "out_b must hold [M, N - split] elements")
    code = _PROLOGUES[prologue] | (QF_LINEAR_GLU_OUT if glu_out else 0)
    la = LinearArgs(M, N, K, code, x.data_ptr(), w.data_ptr(),
                    None if gain is None else gain.data_ptr(), float(eps),
                    None if residual is None else residual.data_ptr(), out.data_ptr(), n_split,
                    None if out_b is None else out_b.data_ptr())
    return la, ((out, out_b) if n_split < N else out)


def linear(x, w, prologue=None, gain=None, eps=1e-6, residual=None, out=None, split=None,
           out_b=None, glu_out=False):
    """out = W . P(x) (+ residual) for up to 8 rows (qf_linear), all bf16.

    x [M, K] ([M, 2K] for "swiglu": gate, then up); w [N, K] (torch layout); prologue None,
    "rms_norm" (with ``gain`` [K]) or "swiglu".  With ``split`` the first ``split`` outputs go to
    ``out`` [M, split] and the rest to ``out_b`` [M, N - split].  With ``glu_out`` the rows of w
    alternate gate and up and the output is silu(gate) * up, [M, N / 2]."""
    la, result = _linear_call(x, w, prologue, gain, eps, residual, out, split, out_b, glu_out)
    stream = torch.cuda.current_stream(x.device).cuda_stream
    _check(load_library().qf_linear(la.rows, la.n_out, la.k, la.prologue, la.x, la.w, la.gain,
                                    la.eps, la.residual, la.out, la.n_split, la.out_b,
                                    ctypes.c_void_p(stream)))
    return result


def decode_workspace_size(desc: DecodeDesc) -> int:
    n = ctypes.c_size_t(0)
    _check(load_library().qf_attn_decode_workspace_size(ctypes.byref(desc), ctypes.byref(n)))
    return n.value


def attn_decode(q, k_cache, v_cache, block_table, ctx_lens, n_shards, max_shards=None,
                scale=None, out=None, lse=None, workspace=None, counters=None, max_pages=None,
                want_lse=True):
    """Sweep and merge in one launch (qf_attn_decode): returns (out bf16 [B, Hq, D],
    lse fp32 [B, Hq]), those of ``attn_combine(*attn_decode_split(...))`` (bitwise when the
    shape needs no sub-shard chunks and has at most 64 shard slots; otherwise the slots are
    grouped differently, which can move the last bits).

    ``workspace``: uint8 tensor of at least ``decode_workspace_size`` bytes (allocated when
    None); ``counters``: int32 tensor of at least B * Hkv entries, zero-filled before its first
    use (every call leaves it at zero; allocated zeroed when None)."""
    _require(q, "q", torch.bfloat16, 3)
    _require(k_cache, "k_cache", torch.bfloat16, 4)
    _require(v_cache, "v_cache", torch.bfloat16, 4)
    if v_cache.shape != k_cache.shape:
        raise QFError(QF_EINVAL, "k_cache and v_cache shapes differ")
    if block_table is not None:
        _require(block_table, "block_table", torch.int32, 2)
    _require(ctx_lens, "ctx_lens", torch.int32, 1)
    B, Hq, D = q.shape
    if isinstance(n_shards, int):
        if max_shards is None:
            max_shards = n_shards
        n_shards = torch.full((B,), n_shards, dtype=torch.int32, device=q.device)
    _require(n_shards, "n_shards", torch.int32, 1)
    if max_shards is None:
        raise QFError(QF_EINVAL, "max_shards is required when n_shards is a tensor")
    if scale is None:
        scale = D ** -0.5
    desc = make_desc(q, k_cache, block_table, max_shards, scale, max_pages=max_pages)
    if out is None:
        out = torch.empty((B, Hq, D), dtype=torch.bfloat16, device=q.device)
    if lse is None and want_lse:
        lse = torch.empty((B, Hq), dtype=torch.float32, device=q.device)
    _require(out, "out", torch.bfloat16)
    if workspace is None:
        workspace = torch.empty(max(decode_workspace_size(desc), 16), dtype=torch.uint8,
                                device=q.device)
    _require(workspace, "workspace", torch.uint8)
    if counters is None:
        counters = torch.zeros(B * k_cache.shape[1], dtype=torch.int32, device=q.device)
    _require(counters, "counters", torch.int32)
    stream = torch.cuda.current_stream(q.device).cuda_stream
    _check(load_library().qf_attn_decode(
        ctypes.byref(desc), _ptr(q), _ptr(k_cache), _ptr(v_cache), _ptr(block_table),
        _ptr(ctx_lens), _ptr(n_shards), _ptr(out), _ptr(lse), _ptr(workspace),
        workspace.numel(), _ptr(counters), counters.numel(), ctypes.c_void_p(stream)))
    return out, lse


def attn_decode_noalloc(q, k_cache, v_cache, block_table, ctx_lens, n_shards, max_shards=None,
                        scale=None, out=None, lse=None, max_pages=None, want_lse=True):
    """``attn_decode`` without a workspace or counters (qf_attn_decode_noalloc): the library works
    in its own fixed device array, so the call allocates nothing on the device (``out`` / ``lse``
    and an int ``n_shards`` are still made here when not given).  Calls that may overlap on one
    GPU race on that array.  Returns (out bf16 [B, Hq, D], lse fp32 [B, Hq])."""
    _require(q, "q", torch.bfloat16, 3)
    _require(k_cache, "k_cache", torch.bfloat16, 4)
    _require(v_cache, "v_cache", torch.bfloat16, 4)
    if v_cache.shape != k_cache.shape:
        raise QFError(QF_EINVAL, "k_cache and v_cache shapes differ")
    if block_table is not None:
        _require(block_table, "block_table", torch.int32, 2)
    _require(ctx_lens, "ctx_lens", torch.int32, 1)
    B, Hq, D = q.shape
    if isinstance(n_shards, int):
        if max_shards is None:
            max_shards = n_shards
        n_shards = torch.full((B,), n_shards, dtype=torch.int32, device=q.device)
    _require(n_shards, "n_shards", torch.int32, 1)
    if max_shards is None:
        raise QFError(QF_EINVAL, "max_shards is required when n_shards is a tensor")
    if scale is None:
        scale = D ** -0.5
    desc = make_desc(q, k_cache, block_table, max_shards, scale, max_pages=max_pages)
    if out is None:
        out = torch.empty((B, Hq, D), dtype=torch.bfloat16, device=q.device)
    if lse is None and want_lse:
        lse = torch.empty((B, Hq), dtype=torch.float32, device=q.device)
    _require(out, "out", torch.bfloat16)
    if out.numel() != B * Hq * D or (lse is not None and lse.numel() != B * Hq):
        raise QFError(QF_EINVAL, "out / lse sizes do not match q")
    stream = torch.cuda.current_stream(q.device).cuda_stream
    _check(load_library().qf_attn_decode_noalloc(
        ctypes.byref(desc), _ptr(q), _ptr(k_cache), _ptr(v_cache), _ptr(block_table),
        _ptr(ctx_lens), _ptr(n_shards), _ptr(out), _ptr(lse), ctypes.c_void_p(stream)))
    return out, lse


def schedule_simulate(arrival, attn_time, n_layers, wiring="qfirst", ffn_time=1.0, min_batch=2,
                      max_wait=float("inf")):
    """Host simulation of the layer-wise decode schedule (qf_schedule_simulate).

    Returns a dict of numpy float64 arrays: finish [R] (NaN = stranded), sweep_start, sweep_end,
    ffn_depart, ffn_return [R, n_layers] (NaN = never happened)."""
    import numpy as np

    arr = np.ascontiguousarray(arrival, dtype=np.float64)
    att = np.ascontiguousarray(attn_time, dtype=np.float64)
    R = arr.shape[0]
    if att.shape != (R,):
        raise QFError(QF_EINVAL, "arrival and attn_time must have the same length")
    w = {"qfirst": QF_WIRING_QFIRST, "composed": QF_WIRING_COMPOSED}[wiring]
    out = {k: np.full((R, n_layers) if k != "finish" else (R,), np.nan)
           for k in ("finish", "sweep_start", "sweep_end", "ffn_depart", "ffn_return")}
    dptr = lambda a: a.ctypes.data_as(ctypes.POINTER(ctypes.c_double))
    _check(load_library().qf_schedule_simulate(
        R, dptr(arr), dptr(att), int(n_layers), w, float(ffn_time), int(min_batch),
        float(max_wait), dptr(out["finish"]), dptr(out["sweep_start"]), dptr(out["sweep_end"]),
        dptr(out["ffn_depart"]), dptr(out["ffn_return"])))
    return out
