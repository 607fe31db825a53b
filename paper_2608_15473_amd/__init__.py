"""MI355X (gfx950) split-KV grouped-query decode attention with an LSE shard merge.

The computation is the cache-side sweep of the Q-First decode protocol (arXiv:2608.15473, §2 and
§5) with its merge, the current-token fold and cache append of the protocol (§2), the dense
products of a decoder block and the sweep sharing a launch with the feed-forward (§3), and a
simulation of the layer-wise decode schedule (Appendix D).  It all runs in hand-written HIP kernels
behind the C ABI of ``include/qfattn.h`` (``lib/libqfattn.so``); this package is the thin Python
binding over that library (``binding``) plus a stack of Q-First blocks built on it (``stage``).
"""

from .binding import (  # noqa: F401
    EXPORTED,
    LIB_PATH,
    QF_EALIGN,
    QF_EHIP,
    QF_EINVAL,
    QF_EUNSUPPORTED,
    QF_LINEAR_GLU_OUT,
    QF_LINEAR_PLAIN,
    QF_LINEAR_RMS_NORM,
    QF_LINEAR_SWIGLU,
    QF_OK,
    DecodeDesc,
    LinearArgs,
    QFError,
    attn_combine,
    attn_combine_current,
    attn_combine_current_append,
    attn_decode,
    attn_decode_noalloc,
    attn_decode_split,
    attn_decode_split_beside,
    attn_decode_split_unfolded,
    split_chunks,
    DecodeStepPlan,
    decode_workspace_size,
    kv_append,
    load_library,
    schedule_simulate,
    make_desc,
    linear,
    workspace_size,
)
