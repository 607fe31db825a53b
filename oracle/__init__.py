"""fp64 CPU oracle for split-KV decode attention over a paged grouped-query KV cache.

TEST INFRASTRUCTURE ONLY.  This package is the independent checker of the HIP path.  Only the
tests, ``__graft_entry__.smoke()`` and the ``cpu_baseline`` leg of ``bench.py`` may import or call
it; the product package never does, and this package imports nothing from the product.

What it computes follows the paper (Q-First, arXiv:2608.15473):

* §2 (the decode protocol): the cache-side device receives only the query and returns the
  attention vector over the cached positions together with its log-sum-exp.
* §5 (splitting the cache): for a set S of positions with scores s_i and values
  v_i, Z(S) = sum_i exp(s_i), W(S) = sum_i exp(s_i) v_i, O(S) = W(S)/Z(S); a shard returns
  (O, log Z); two shards merge by lerp / sigmoid / logaddexp; an empty shard is log Z = -inf
  and its vector is never read.
* §2 (score definition): s = q . k / sqrt(d); here the scale is passed in explicitly.
* §2 and §8 (the rewired block): the query reads the block input u, the key and value the
  post-feed-forward stream z = u + M(N2 u); the block's output is z + W_o attn (``block.py``).

Every function works in float64 on exact copies of the bf16 inputs.  Parity status of each
function is stated in its docstring; the pins live in ``tests/test_oracle_*.py``.
"""

from .attention import (  # noqa: F401
    shard_ranges,
    gather_rows,
    attend,
    attend_shifted,
    decode_split,
    decode_unsplit,
    merge_pair,
    fold_combine,
    combine_max_shifted,
    fold_current,
    append_kv,
)
from .block import (  # noqa: F401
    RMS_EPS,
    rms_norm,
    silu,
    swiglu,
    feed_forward,
    qfirst_block,
)
