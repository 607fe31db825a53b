// Host side of the C-ABI: argument validation, the chunking rule, launches on the caller's stream.
// Declarations and the full contract are in include/qfattn.h.
#include <math.h>
#include <stdarg.h>
#include <stdio.h>
#include <string.h>

#include <algorithm>

#include "qf_internal.h"
#include "qfattn.h"

namespace {

thread_local char g_error[512];

int fail(int code, const char* fmt, ...) {
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(g_error, sizeof g_error, fmt, ap);
  va_end(ap);
  return code;
}

bool aligned(const void* p, size_t a) { return ((uintptr_t)p % a) == 0; }

// Sub-shard chunks, only for shapes with fewer (request, shard, KV head) units than the sweep has
// resident workgroups: as many chunks as fill one full set of resident workgroups, never a partial
// second round (measured on the 1M-token shape, 128 units: 6 chunks beat 16 and 12).  The count
// depends on the descriptor and the device's occupancy for the kernel only, so a given shape on a
// given GPU always runs the same decomposition (and gives the same bits); with no device to ask
// (a host without a GPU sizing a workspace) it assumes the counts this build reaches on an MI355X
// (256 CUs; 4 workgroups per CU at G = 1, 3 at G = 2 and 4, 2 at G = 8), which a GPU test checks
// against the device.
int64_t fallback_resident(int group) {
  return group == 1 ? 1024 : group == 8 ? 512 : 768;
}
// ... and no more chunks than leave every wavefront at least this many pages: on the 4,608-position
// single layer (36 pages per shard) 3 pages per wavefront (3 chunks) beat 2 (4 chunks) by 2%,
// 1 (9 chunks) by 17%, and 4 (2 chunks) by 6%.
constexpr int64_t kMinPagesPerWave = 3;

int check_desc(const qf_decode_desc* d) {
  if (!d) return fail(QF_EINVAL, "desc is NULL");
  if (d->batch < 0) return fail(QF_EINVAL, "batch %d < 0", d->batch);
  if (d->n_q_heads < 1 || d->n_kv_heads < 1)
    return fail(QF_EINVAL, "n_q_heads %d / n_kv_heads %d must be >= 1", d->n_q_heads, d->n_kv_heads);
  if (d->n_q_heads > QF_MAX_Q_HEADS)
    return fail(QF_EINVAL, "n_q_heads %d > %d", d->n_q_heads, QF_MAX_Q_HEADS);
  if (d->n_q_heads % d->n_kv_heads != 0)
    return fail(QF_EINVAL, "n_q_heads %d is not a multiple of n_kv_heads %d", d->n_q_heads,
                d->n_kv_heads);
  const int G = d->n_q_heads / d->n_kv_heads;
  if (G != 1 && G != 2 && G != 4 && G != 8)
    return fail(QF_EUNSUPPORTED, "group size %d (n_q_heads / n_kv_heads) not in {1,2,4,8}", G);
  if (d->head_dim != qf::kHeadDim)
    return fail(QF_EUNSUPPORTED, "head_dim %d != %d", d->head_dim, qf::kHeadDim);
  if (d->page_size != qf::kPage)
    return fail(QF_EUNSUPPORTED, "page_size %d != %d", d->page_size, qf::kPage);
  if (d->max_pages_per_seq < 1) return fail(QF_EINVAL, "max_pages_per_seq %d < 1", d->max_pages_per_seq);
  if ((int64_t)d->max_pages_per_seq * qf::kPage > INT32_MAX)
    return fail(QF_EINVAL, "max_pages_per_seq %d too large", d->max_pages_per_seq);
  if (d->num_pages < 1) return fail(QF_EINVAL, "num_pages %d < 1", d->num_pages);
  if (d->max_shards < 1) return fail(QF_EINVAL, "max_shards %d < 1", d->max_shards);
  if (!isfinite(d->softmax_scale)) return fail(QF_EINVAL, "softmax_scale is not finite");
  return QF_OK;
}

int64_t choose_chunks(const qf_decode_desc* d) {
  const int64_t units = (int64_t)d->batch * d->n_kv_heads * d->max_shards;
  if (units <= 0) return 1;
  const int group = d->n_q_heads / d->n_kv_heads;
  int64_t slots = qf::split_resident_workgroups(group);
  if (slots <= 0) slots = fallback_resident(group);
  if (units >= slots) return 1;
  const int64_t est_pages = (d->max_pages_per_seq + d->max_shards - 1) / d->max_shards;
  int64_t c = slots / units;
  c = std::min(c, std::max<int64_t>(1, est_pages / (qf::kSplitWaves * kMinPagesPerWave)));
  return std::max<int64_t>(1, std::min<int64_t>(c, 1024));
}

// Long shards: long-lived workgroups, the dispatch order decides the tail (largest first).
// Short shards: short workgroups, prologue latency decides (keep a request on one XCD).
int sweep_order(const qf_decode_desc* d, int64_t chunks) {
  const int64_t shard_pages = (d->max_pages_per_seq + d->max_shards - 1) / d->max_shards / chunks;
  return shard_pages >= qf::kLongShardPages ? qf::kOrderByShardDesc : qf::kOrderByRequest;
}

// An unchunked long-shard sweep (of up to kRankMaxPairs (request, shard) pairs) takes its units in
// the order of rank_units_kernel, which it keeps in the workspace: one int32 per workgroup index.
bool ranks_units(const qf_decode_desc* d, int64_t chunks) {
  return chunks == 1 && sweep_order(d, chunks) == qf::kOrderByShardDesc &&
         (int64_t)d->batch * d->max_shards <= qf::kRankMaxPairs;
}
size_t unit_order_bytes(const qf_decode_desc* d, int64_t chunks) {
  if (!ranks_units(d, chunks)) return 0;
  const int64_t units = (int64_t)d->batch * d->max_shards * d->n_kv_heads;
  return (size_t)((units + 7) / 8 * 8) * sizeof(int32_t);
}

size_t chunk_state_bytes(const qf_decode_desc* d, int64_t chunks) {
  if (chunks <= 1) return 0;
  const size_t states = (size_t)d->batch * d->max_shards * chunks * d->n_q_heads;
  return states * qf::kHeadDim * sizeof(float) + states * sizeof(float);
}

// qf_attn_decode_split's workspace: the chunk states or the unit order (never both).
size_t workspace_bytes(const qf_decode_desc* d, int64_t chunks) {
  return chunk_state_bytes(d, chunks) + unit_order_bytes(d, chunks);
}

// Everything qf_attn_decode_split checks and derives before launching.
struct Split {
  bool noop = false;
  bool fold = true;  // chunks folded into their shards (qf_attn_decode_split) or left as slots
  int group = 1;
  int64_t chunks = 1;
  qf::SplitParams p{};
  qf::MergeParams chunk_merge{};
};

// fold: the chunks are folded into part_out / part_lse (chunk states in the workspace) or left
// as slots there; rank: the workspace holds the unit order of a ranked sweep.  The workspace is
// needed for whichever of the two applies.
int prepare_split(const qf_decode_desc* desc, const void* q, const void* k_cache,
                  const void* v_cache, const int32_t* block_table, const int32_t* ctx_lens,
                  const int32_t* n_shards, float* part_out, float* part_lse, void* workspace,
                  size_t workspace_size, Split* sp, bool fold = true, bool rank = true) {
  int rc = check_desc(desc);
  if (rc) return rc;
  const qf_decode_desc& d = *desc;
  if (d.batch == 0) {
    sp->noop = true;
    return QF_OK;
  }
  if (!q || !k_cache || !v_cache || !ctx_lens || !n_shards || !part_out || !part_lse)
    return fail(QF_EINVAL, "a required pointer is NULL");
  if (!aligned(q, 16) || !aligned(k_cache, 16) || !aligned(v_cache, 16) || !aligned(part_out, 16))
    return fail(QF_EALIGN, "q, k_cache, v_cache and part_out must be 16-byte aligned");
  if (!aligned(part_lse, 4) || !aligned(ctx_lens, 4) || !aligned(n_shards, 4) ||
      (block_table && !aligned(block_table, 4)))
    return fail(QF_EALIGN, "part_lse, ctx_lens, n_shards and block_table must be 4-byte aligned");
  if (!block_table && (int64_t)d.batch * d.max_pages_per_seq > d.num_pages)
    return fail(QF_EINVAL, "identity block table needs num_pages >= batch * max_pages_per_seq (%lld > %d)",
                (long long)d.batch * d.max_pages_per_seq, d.num_pages);

  const int64_t chunks = choose_chunks(&d);
  const size_t state_bytes = fold ? chunk_state_bytes(&d, chunks) : 0;
  const size_t need = state_bytes + (rank ? unit_order_bytes(&d, chunks) : 0);
  rank = need > state_bytes;
  if (need) {
    if (!workspace) return fail(QF_EINVAL, "this shape needs %zu bytes of workspace", need);
    if (workspace_size < need)
      return fail(QF_EINVAL, "workspace of %zu bytes < %zu needed", workspace_size, need);
    if (!aligned(workspace, 16)) return fail(QF_EALIGN, "workspace must be 16-byte aligned");
  }
  const int64_t units = (int64_t)d.batch * d.max_shards * chunks * d.n_kv_heads;
  if (units > (int64_t)INT32_MAX - 8) return fail(QF_EINVAL, "too many work units (%lld)", (long long)units);

  qf::SplitParams p{};
  p.q = static_cast<const uint16_t*>(q);
  p.k = static_cast<const uint16_t*>(k_cache);
  p.v = static_cast<const uint16_t*>(v_cache);
  p.block_table = block_table;
  p.ctx_lens = ctx_lens;
  p.n_shards = n_shards;
  const size_t states = (size_t)d.batch * d.max_shards * chunks * d.n_q_heads;
  if (chunks > 1 && fold) {
    p.out_o = static_cast<float*>(workspace);
    p.out_lse = static_cast<float*>(workspace) + states * qf::kHeadDim;
  } else {
    p.out_o = part_out;
    p.out_lse = part_lse;
  }
  p.batch = d.batch;
  p.hq = d.n_q_heads;
  p.hkv = d.n_kv_heads;
  p.max_pages = d.max_pages_per_seq;
  p.num_pages = d.num_pages;
  p.max_shards = d.max_shards;
  p.chunks = (int32_t)chunks;
  p.n_units = (int32_t)units;
  p.units_per_xcd = (int32_t)((units + 7) / 8);
  const int64_t shard_pages = (d.max_pages_per_seq + d.max_shards - 1) / d.max_shards / chunks;
  p.order = sweep_order(&d, chunks);
  p.unit_order = rank ? reinterpret_cast<int32_t*>(static_cast<char*>(workspace) + state_bytes)
                      : nullptr;
  p.rank_shift = 0;
  while ((d.max_pages_per_seq >> p.rank_shift) >= qf::kRankBuckets) ++p.rank_shift;
  // Deep buffers cost occupancy (two wavefronts per SIMD instead of three), so a chunked sweep,
  // whose chunk count fills exactly the resident workgroups of the two-buffer kernel, keeps two
  // buffers (deep ones would leave a second, partial round: -2% on the 131,072-position share).
  p.deep = p.order == qf::kOrderByRequest && shard_pages >= qf::kDeepMinPages && chunks == 1;
  p.scale_log2 = (float)((double)d.softmax_scale * 1.4426950408889634);

  sp->group = d.n_q_heads / d.n_kv_heads;
  sp->chunks = chunks;
  sp->fold = fold;
  sp->p = p;
  if (chunks > 1 && fold) {
    qf::MergeParams& m = sp->chunk_merge;
    m.in_o = p.out_o;
    m.in_lse = p.out_lse;
    m.out_o = part_out;
    m.out_lse = part_lse;
    m.rows = d.batch * d.max_shards;
    m.entries = (int32_t)chunks;
    m.hq = d.n_q_heads;
  }
  return QF_OK;
}

// Workspace of qf_attn_decode: the partial states of every (shard, chunk) slot.
size_t fused_workspace_bytes(const qf_decode_desc* d, int64_t chunks) {
  const size_t states = (size_t)d->batch * d->max_shards * chunks * d->n_q_heads;
  return states * (qf::kHeadDim + 1) * sizeof(float);
}

// After the sweep's launch: fold the chunks of each shard into the caller's per-shard partials.
int finish_split(const Split& sp, hipStream_t s) {
  if (sp.chunks <= 1 || !sp.fold) return QF_OK;
  const hipError_t e = qf::launch_merge(sp.chunk_merge, false, s);
  if (e != hipSuccess) return fail(QF_EHIP, "chunk merge launch: %s", hipGetErrorString(e));
  return QF_OK;
}

// Everything qf_linear checks and derives before launching.
int prepare_linear(const qf_linear_args* a, qf::LinearParams* out_p, bool* noop) {
  const int32_t rows = a->rows, n_out = a->n_out, k = a->k;
  const bool glu = (a->prologue & QF_LINEAR_GLU_OUT) != 0;
  const int32_t prologue = a->prologue & ~QF_LINEAR_GLU_OUT;
  const int32_t n_split = a->n_split;
  const void *x = a->x, *w = a->w, *gain = a->gain, *residual = a->residual;
  void *out = a->out, *out_b = a->out_b;
  const float eps = a->eps;
  if (rows < 0) return fail(QF_EINVAL, "rows must be >= 0 (got %d)", rows);
  if (rows > qf::kLinearMaxRows)
    return fail(QF_EUNSUPPORTED, "at most %d rows per call (got %d)", qf::kLinearMaxRows, rows);
  if (n_out < 1 || k < 8) return fail(QF_EINVAL, "need n_out >= 1 and k >= 8");
  if (k % 8) return fail(QF_EUNSUPPORTED, "k must be a multiple of 8 (got %d)", k);
  if (prologue != QF_LINEAR_PLAIN && prologue != QF_LINEAR_RMS_NORM &&
      prologue != QF_LINEAR_SWIGLU)
    return fail(QF_EINVAL, "unknown prologue %d", prologue);
  if (n_split < 1 || n_split > n_out)
    return fail(QF_EINVAL, "n_split must be in [1, n_out] (got %d)", n_split);
  if (glu && (prologue == QF_LINEAR_SWIGLU || n_out % 2 || n_split != n_out || a->residual))
    return fail(QF_EINVAL, "QF_LINEAR_GLU_OUT needs an even n_out, n_split == n_out, no residual "
                           "and no SwiGLU input");
  if (prologue == QF_LINEAR_RMS_NORM && !(eps >= 0.0f)) return fail(QF_EINVAL, "eps must be >= 0");
  if (rows == 0) {
    *noop = true;
    return QF_OK;
  }
  if (!x || !w || !out || (prologue == QF_LINEAR_RMS_NORM && !gain) ||
      (n_split < n_out && !out_b))
    return fail(QF_EINVAL, "a required pointer is NULL");
  if (!aligned(x, 16) || !aligned(w, 16) || (gain && !aligned(gain, 16)) ||
      !aligned(out, 2) || (out_b && !aligned(out_b, 2)) || (residual && !aligned(residual, 2)))
    return fail(QF_EALIGN, "x, w and gain must be 16-byte aligned, out and residual 2-byte");
  qf::LinearParams p{};
  p.x = static_cast<const uint16_t*>(x);
  p.w = static_cast<const uint16_t*>(w);
  p.gain = static_cast<const uint16_t*>(gain);
  p.residual = static_cast<const uint16_t*>(residual);
  p.out_a = static_cast<uint16_t*>(out);
  p.out_b = static_cast<uint16_t*>(out_b);
  p.M = rows;
  p.N = n_out;
  p.K = k;
  p.n_split = n_split;
  p.prologue = prologue == QF_LINEAR_RMS_NORM ? qf::kProRmsNorm
             : prologue == QF_LINEAR_SWIGLU   ? qf::kProSwiglu
                                              : qf::kProNone;
  p.eps = eps;
  p.glu = glu;
  *out_p = p;
  return QF_OK;
}

// The one-launch decode on a given workspace and counters (qf_attn_decode's body; defined below).
int decode_fused(const qf_decode_desc* desc, const void* q, const void* k_cache,
                 const void* v_cache, const int32_t* block_table, const int32_t* ctx_lens,
                 const int32_t* n_shards, void* out, float* lse, void* workspace,
                 size_t workspace_size, int32_t* counters, int64_t n_counters, void* stream,
                 bool fixed_scratch);

}  // namespace

extern "C" {

int qf_version(void) { return QF_VERSION; }

const char* qf_last_error(void) { return g_error; }

int qf_attn_decode_split_workspace_size(const qf_decode_desc* desc, size_t* bytes) {
  g_error[0] = 0;
  const int rc = check_desc(desc);
  if (rc) return rc;
  if (!bytes) return fail(QF_EINVAL, "bytes is NULL");
  *bytes = workspace_bytes(desc, choose_chunks(desc));
  return QF_OK;
}

int qf_attn_decode_split(const qf_decode_desc* desc, const void* q, const void* k_cache,
                         const void* v_cache, const int32_t* block_table,
                         const int32_t* ctx_lens, const int32_t* n_shards, float* part_out,
                         float* part_lse, void* workspace, size_t workspace_size, void* stream) {
  g_error[0] = 0;
  Split sp;
  const int rc = prepare_split(desc, q, k_cache, v_cache, block_table, ctx_lens, n_shards,
                               part_out, part_lse, workspace, workspace_size, &sp);
  if (rc || sp.noop) return rc;
  hipStream_t s = static_cast<hipStream_t>(stream);
  const hipError_t e = qf::launch_decode_split(sp.p, sp.group, s);
  if (e != hipSuccess) return fail(QF_EHIP, "decode_split launch: %s", hipGetErrorString(e));
  return finish_split(sp, s);
}

int qf_attn_decode_split_chunks(const qf_decode_desc* desc, int32_t* chunks) {
  g_error[0] = 0;
  const int rc = check_desc(desc);
  if (rc) return rc;
  if (!chunks) return fail(QF_EINVAL, "chunks is NULL");
  *chunks = (int32_t)choose_chunks(desc);
  return QF_OK;
}

int qf_attn_decode_split_unfolded(const qf_decode_desc* desc, const void* q, const void* k_cache,
                                  const void* v_cache, const int32_t* block_table,
                                  const int32_t* ctx_lens, const int32_t* n_shards,
                                  float* slot_out, float* slot_lse, int32_t n_slots,
                                  void* stream) {
  g_error[0] = 0;
  int rc = check_desc(desc);
  if (rc) return rc;
  if (desc->batch == 0) return QF_OK;
  // The slot count of the caller's arrays, checked against the one the sweep writes (it depends on
  // the device's resident workgroups, so a caller sizing by max_shards alone would be overrun).
  const int64_t want = (int64_t)desc->max_shards * choose_chunks(desc);
  if (want > (int64_t)INT32_MAX) return fail(QF_EINVAL, "max_shards * chunks exceeds int32");
  if (n_slots != want)
    return fail(QF_EINVAL,
                "the slot arrays hold %d slots per request; this shape needs %lld (max_shards x "
                "qf_attn_decode_split_chunks)",
                n_slots, (long long)want);
  Split sp;
  rc = prepare_split(desc, q, k_cache, v_cache, block_table, ctx_lens, n_shards, slot_out,
                     slot_lse, nullptr, 0, &sp, false, false);
  if (rc || sp.noop) return rc;
  hipStream_t s = static_cast<hipStream_t>(stream);
  const hipError_t e = qf::launch_decode_split(sp.p, sp.group, s);
  if (e != hipSuccess) return fail(QF_EHIP, "decode_split launch: %s", hipGetErrorString(e));
  return QF_OK;
}

int qf_attn_decode_workspace_size(const qf_decode_desc* desc, size_t* bytes) {
  g_error[0] = 0;
  if (!bytes) return fail(QF_EINVAL, "bytes is NULL");
  const int rc = check_desc(desc);
  if (rc) return rc;
  *bytes = fused_workspace_bytes(desc, choose_chunks(desc));
  return QF_OK;
}

int qf_attn_decode(const qf_decode_desc* desc, const void* q, const void* k_cache,
                   const void* v_cache, const int32_t* block_table, const int32_t* ctx_lens,
                   const int32_t* n_shards, void* out, float* lse, void* workspace,
                   size_t workspace_size, int32_t* counters, int64_t n_counters, void* stream) {
  g_error[0] = 0;
  return decode_fused(desc, q, k_cache, v_cache, block_table, ctx_lens, n_shards, out, lse,
                      workspace, workspace_size, counters, n_counters, stream, false);
}

int qf_attn_decode_noalloc(const qf_decode_desc* desc, const void* q, const void* k_cache,
                           const void* v_cache, const int32_t* block_table,
                           const int32_t* ctx_lens, const int32_t* n_shards, void* out,
                           float* lse, void* stream) {
  g_error[0] = 0;
  return decode_fused(desc, q, k_cache, v_cache, block_table, ctx_lens, n_shards, out, lse,
                      nullptr, 0, nullptr, 0, stream, true);
}

}  // extern "C"

namespace {

// fixed_scratch: workspace and counters are the library's own scratch array (decode_noalloc.hip),
// looked up and its counters cleared only once every argument has passed its checks, so that a
// refused call enqueues nothing.
int decode_fused(const qf_decode_desc* desc, const void* q, const void* k_cache,
                 const void* v_cache, const int32_t* block_table, const int32_t* ctx_lens,
                 const int32_t* n_shards, void* out, float* lse, void* workspace,
                 size_t workspace_size, int32_t* counters, int64_t n_counters, void* stream,
                 bool fixed_scratch) {
  int rc = check_desc(desc);
  if (rc) return rc;
  const qf_decode_desc& d = *desc;
  if (d.batch == 0) return QF_OK;
  const int64_t chunks = choose_chunks(&d);
  const size_t need = fused_workspace_bytes(&d, chunks);
  const int64_t groups = (int64_t)d.batch * d.n_kv_heads;
  if (fixed_scratch) {
    // Sizes first: a shape beyond the fixed scratch is refused before anything touches the GPU.
    const int64_t max_groups = (int64_t)(qf::kNoallocCounterBytes / sizeof(int32_t));
    if (need > qf::kNoallocStateBytes || groups > max_groups)
      return fail(QF_EINVAL,
                  "shape needs %zu bytes of partial states and %lld (request, KV head) counters; "
                  "the fixed scratch holds %zu bytes and %lld counters (qf_attn_decode takes a "
                  "workspace of any size)",
                  need, (long long)groups, qf::kNoallocStateBytes, (long long)max_groups);
    // Placeholders (aligned, never dereferenced) until the arguments have been checked.
    workspace = reinterpret_cast<void*>(uintptr_t(256));
    workspace_size = need;
    counters = reinterpret_cast<int32_t*>(uintptr_t(256));
    n_counters = groups;
    if (!out) return fail(QF_EINVAL, "out is required");
  } else if (!out || !workspace || !counters) {
    return fail(QF_EINVAL, "out, workspace and counters are required");
  }
  if (n_counters < groups)
    return fail(QF_EINVAL, "counters holds %lld entries < batch * n_kv_heads = %lld",
                (long long)n_counters, (long long)groups);
  if (!aligned(out, 4) || (lse && !aligned(lse, 4)) || !aligned(workspace, 16) ||
      !aligned(counters, 4))
    return fail(QF_EALIGN, "out, lse and counters must be 4-byte aligned, workspace 16-byte");
  if (workspace_size < need)
    return fail(QF_EINVAL, "workspace of %zu bytes < %zu needed", workspace_size, need);
  // The partial states live in the workspace, seen by the sweep as its per-slot outputs (with
  // chunks == 1 its direct outputs, otherwise its chunk states): one layout [B, S x C, Hq, .].
  const size_t n_states = (size_t)d.batch * d.max_shards * chunks * d.n_q_heads;
  float* states = static_cast<float*>(workspace);
  Split sp;
  rc = prepare_split(desc, q, k_cache, v_cache, block_table, ctx_lens, n_shards, states,
                     states + n_states * qf::kHeadDim, chunks > 1 ? workspace : nullptr,
                     chunks > 1 ? need : 0, &sp, true, false);
  if (rc || sp.noop) return rc;
  hipStream_t s = static_cast<hipStream_t>(stream);
  if (fixed_scratch) {
    void* base = nullptr;
    const hipError_t e = qf::noalloc_prepare((int32_t)groups, s, &counters, &base);
    if (e != hipSuccess) return fail(QF_EHIP, "scratch set-up: %s", hipGetErrorString(e));
    states = static_cast<float*>(base);
    sp.p.out_o = states;
    sp.p.out_lse = states + n_states * qf::kHeadDim;
  }
  const hipError_t e = qf::launch_decode_fused(sp.p, sp.group, counters, out, lse, s);
  if (e != hipSuccess) return fail(QF_EHIP, "decode launch: %s", hipGetErrorString(e));
  return QF_OK;
}

}  // namespace

extern "C" {

int qf_attn_combine(int32_t batch, int32_t n_q_heads, int32_t head_dim, int32_t max_shards,
                    const float* part_out, const float* part_lse, void* out, float* lse,
                    void* stream) {
  g_error[0] = 0;
  if (batch < 0) return fail(QF_EINVAL, "batch %d < 0", batch);
  if (n_q_heads < 1 || n_q_heads > QF_MAX_Q_HEADS)
    return fail(QF_EINVAL, "n_q_heads %d not in [1, %d]", n_q_heads, QF_MAX_Q_HEADS);
  if (max_shards < 1) return fail(QF_EINVAL, "max_shards %d < 1", max_shards);
  if (head_dim != qf::kHeadDim) return fail(QF_EUNSUPPORTED, "head_dim %d != %d", head_dim, qf::kHeadDim);
  if (batch == 0) return QF_OK;
  if (!part_out || !part_lse || !out) return fail(QF_EINVAL, "a required pointer is NULL");
  if (!aligned(part_out, 16)) return fail(QF_EALIGN, "part_out must be 16-byte aligned");
  if (!aligned(part_lse, 4) || !aligned(out, 4) || (lse && !aligned(lse, 4)))
    return fail(QF_EALIGN, "part_lse, out and lse must be 4-byte aligned");
  if ((int64_t)batch * n_q_heads > INT32_MAX) return fail(QF_EINVAL, "batch * n_q_heads too large");
  qf::MergeParams m{};
  m.in_o = part_out;
  m.in_lse = part_lse;
  m.out_o = out;
  m.out_lse = lse;
  m.rows = batch;
  m.entries = max_shards;
  m.hq = n_q_heads;
  const hipError_t e = qf::launch_merge(m, true, static_cast<hipStream_t>(stream));
  if (e != hipSuccess) return fail(QF_EHIP, "combine launch: %s", hipGetErrorString(e));
  return QF_OK;
}

int qf_attn_combine_current(int32_t batch, int32_t n_q_heads, int32_t n_kv_heads, int32_t head_dim,
                            int32_t max_shards, const float* part_out, const float* part_lse,
                            const void* q, const void* k_cur, const void* v_cur,
                            float softmax_scale, void* out, float* lse, void* stream) {
  g_error[0] = 0;
  if (batch < 0) return fail(QF_EINVAL, "batch %d < 0", batch);
  if (n_q_heads < 1 || n_kv_heads < 1)
    return fail(QF_EINVAL, "n_q_heads %d / n_kv_heads %d must be >= 1", n_q_heads, n_kv_heads);
  if (n_q_heads > QF_MAX_Q_HEADS)
    return fail(QF_EINVAL, "n_q_heads %d > %d", n_q_heads, QF_MAX_Q_HEADS);
  if (n_q_heads % n_kv_heads != 0)
    return fail(QF_EINVAL, "n_q_heads %d is not a multiple of n_kv_heads %d", n_q_heads, n_kv_heads);
  if (max_shards < 1) return fail(QF_EINVAL, "max_shards %d < 1", max_shards);
  if (head_dim != qf::kHeadDim) return fail(QF_EUNSUPPORTED, "head_dim %d != %d", head_dim, qf::kHeadDim);
  if (!isfinite(softmax_scale)) return fail(QF_EINVAL, "softmax_scale is not finite");
  if (batch == 0) return QF_OK;
  if (!part_out || !part_lse || !out || !q || !k_cur || !v_cur)
    return fail(QF_EINVAL, "a required pointer is NULL");
  if (!aligned(part_out, 16)) return fail(QF_EALIGN, "part_out must be 16-byte aligned");
  if (!aligned(part_lse, 4) || !aligned(out, 4) || (lse && !aligned(lse, 4)) || !aligned(q, 4) ||
      !aligned(k_cur, 4) || !aligned(v_cur, 4))
    return fail(QF_EALIGN, "part_lse, out, lse, q, k_cur and v_cur must be 4-byte aligned");
  if ((int64_t)batch * n_q_heads > INT32_MAX) return fail(QF_EINVAL, "batch * n_q_heads too large");
  qf::MergeParams m{};
  m.in_o = part_out;
  m.in_lse = part_lse;
  m.out_o = out;
  m.out_lse = lse;
  m.rows = batch;
  m.entries = max_shards;
  m.hq = n_q_heads;
  m.q = static_cast<const uint16_t*>(q);
  m.k_cur = static_cast<const uint16_t*>(k_cur);
  m.v_cur = static_cast<const uint16_t*>(v_cur);
  m.hkv = n_kv_heads;
  m.scale = softmax_scale;
  const hipError_t e = qf::launch_merge(m, true, static_cast<hipStream_t>(stream));
  if (e != hipSuccess) return fail(QF_EHIP, "combine launch: %s", hipGetErrorString(e));
  return QF_OK;
}

int qf_attn_combine_current_append(const qf_decode_desc* desc, const float* part_out,
                                   const float* part_lse, const void* q, const void* k_cur,
                                   const void* v_cur, void* out, float* lse, void* k_cache,
                                   void* v_cache, const int32_t* block_table, int32_t* ctx_lens,
                                   int32_t* status, void* stream) {
  g_error[0] = 0;
  const int rc = check_desc(desc);
  if (rc) return rc;
  const qf_decode_desc& d = *desc;
  if (d.batch == 0) return QF_OK;
  if (!part_out || !part_lse || !out || !q || !k_cur || !v_cur || !k_cache || !v_cache ||
      !ctx_lens)
    return fail(QF_EINVAL, "a required pointer is NULL");
  if (!aligned(part_out, 16)) return fail(QF_EALIGN, "part_out must be 16-byte aligned");
  if (!aligned(part_lse, 4) || !aligned(out, 4) || (lse && !aligned(lse, 4)) || !aligned(q, 4) ||
      !aligned(k_cur, 4) || !aligned(v_cur, 4) || !aligned(k_cache, 4) || !aligned(v_cache, 4) ||
      !aligned(ctx_lens, 4) || (block_table && !aligned(block_table, 4)) ||
      (status && !aligned(status, 4)))
    return fail(QF_EALIGN, "every pointer must be 4-byte aligned (part_out 16-byte)");
  if (!block_table && (int64_t)d.batch * d.max_pages_per_seq > d.num_pages)
    return fail(QF_EINVAL, "identity block table needs num_pages >= batch * max_pages_per_seq");
  if ((int64_t)d.batch * (d.n_q_heads + 1) > INT32_MAX)
    return fail(QF_EINVAL, "batch * (n_q_heads + 1) too large");
  qf::AppendParams a{};
  a.k = static_cast<uint16_t*>(k_cache);
  a.v = static_cast<uint16_t*>(v_cache);
  a.block_table = block_table;
  a.ctx_lens = ctx_lens;
  a.status = status;
  a.batch = d.batch;
  a.hkv = d.n_kv_heads;
  a.max_pages = d.max_pages_per_seq;
  a.num_pages = d.num_pages;
  a.advance = 1;
  qf::MergeParams m{};
  m.in_o = part_out;
  m.in_lse = part_lse;
  m.out_o = out;
  m.out_lse = lse;
  m.rows = d.batch;
  m.entries = d.max_shards;
  m.hq = d.n_q_heads;
  m.q = static_cast<const uint16_t*>(q);
  m.k_cur = static_cast<const uint16_t*>(k_cur);
  m.v_cur = static_cast<const uint16_t*>(v_cur);
  m.hkv = d.n_kv_heads;
  m.scale = d.softmax_scale;
  m.append = &a;
  const hipError_t e = qf::launch_merge(m, true, static_cast<hipStream_t>(stream));
  if (e != hipSuccess) return fail(QF_EHIP, "combine + append launch: %s", hipGetErrorString(e));
  return QF_OK;
}

int qf_kv_append(const qf_decode_desc* desc, void* k_cache, void* v_cache,
                 const int32_t* block_table, int32_t* ctx_lens, const void* k_new,
                 const void* v_new, int32_t advance, int32_t* status, void* stream) {
  g_error[0] = 0;
  const int rc = check_desc(desc);
  if (rc) return rc;
  const qf_decode_desc& d = *desc;
  if (d.batch == 0) return QF_OK;
  if (!k_cache || !v_cache || !ctx_lens || !k_new || !v_new)
    return fail(QF_EINVAL, "a required pointer is NULL");
  if (!aligned(k_cache, 4) || !aligned(v_cache, 4) || !aligned(k_new, 4) || !aligned(v_new, 4) ||
      !aligned(ctx_lens, 4) || (block_table && !aligned(block_table, 4)) ||
      (status && !aligned(status, 4)))
    return fail(QF_EALIGN, "cache, new-token, index and status pointers must be 4-byte aligned");
  if (!block_table && (int64_t)d.batch * d.max_pages_per_seq > d.num_pages)
    return fail(QF_EINVAL, "identity block table needs num_pages >= batch * max_pages_per_seq");
  qf::AppendParams p{};
  p.k = static_cast<uint16_t*>(k_cache);
  p.v = static_cast<uint16_t*>(v_cache);
  p.block_table = block_table;
  p.ctx_lens = ctx_lens;
  p.k_new = static_cast<const uint16_t*>(k_new);
  p.v_new = static_cast<const uint16_t*>(v_new);
  p.status = status;
  p.batch = d.batch;
  p.hkv = d.n_kv_heads;
  p.max_pages = d.max_pages_per_seq;
  p.num_pages = d.num_pages;
  p.advance = advance ? 1 : 0;
  const hipError_t e = qf::launch_kv_append(p, static_cast<hipStream_t>(stream));
  if (e != hipSuccess) return fail(QF_EHIP, "kv_append launch: %s", hipGetErrorString(e));
  return QF_OK;
}

int qf_linear(int32_t rows, int32_t n_out, int32_t k, int32_t prologue, const void* x,
              const void* w, const void* gain, float eps, const void* residual, void* out,
              int32_t n_split, void* out_b, void* stream) {
  g_error[0] = 0;
  const qf_linear_args a{rows, n_out, k, prologue, x, w, gain, eps, residual, out, n_split, out_b};
  qf::LinearParams p{};
  bool noop = false;
  const int rc = prepare_linear(&a, &p, &noop);
  if (rc || noop) return rc;
  const hipError_t e = qf::launch_linear(p, static_cast<hipStream_t>(stream));
  if (e != hipSuccess) return fail(QF_EHIP, "linear launch: %s", hipGetErrorString(e));
  return QF_OK;
}

int qf_attn_decode_split_beside(const qf_decode_desc* desc, const void* q, const void* k_cache,
                                const void* v_cache, const int32_t* block_table,
                                const int32_t* ctx_lens, const int32_t* n_shards,
                                float* part_out, float* part_lse, void* workspace,
                                size_t workspace_size, const qf_linear_args* beside,
                                void* stream) {
  g_error[0] = 0;
  if (!beside) return fail(QF_EINVAL, "beside is NULL");
  Split sp;
  int rc = prepare_split(desc, q, k_cache, v_cache, block_table, ctx_lens, n_shards, part_out,
                         part_lse, workspace, workspace_size, &sp);
  if (rc) return rc;
  qf::LinearParams lp{};
  bool lin_noop = false;
  rc = prepare_linear(beside, &lp, &lin_noop);
  if (rc) return rc;
  hipStream_t s = static_cast<hipStream_t>(stream);
  hipError_t e = hipSuccess;
  if (sp.noop && lin_noop) return QF_OK;
  if (sp.noop)
    e = qf::launch_linear(lp, s);
  else if (lin_noop)
    e = qf::launch_decode_split(sp.p, sp.group, s);
  else
    e = qf::launch_decode_split_beside(sp.p, sp.group, lp, s);
  if (e != hipSuccess) return fail(QF_EHIP, "decode_split_beside launch: %s", hipGetErrorString(e));
  return sp.noop ? QF_OK : finish_split(sp, s);
}

int qf_schedule_simulate(int32_t n_requests, const double* arrival, const double* attn_time,
                         int32_t n_layers, int32_t wiring, double ffn_time, int32_t min_batch,
                         double max_wait, double* finish, double* sweep_start, double* sweep_end,
                         double* ffn_depart, double* ffn_return) {
  g_error[0] = 0;
  if (n_requests < 0) return fail(QF_EINVAL, "n_requests %d < 0", n_requests);
  if (n_layers < 1) return fail(QF_EINVAL, "n_layers %d < 1", n_layers);
  if (min_batch < 1) return fail(QF_EINVAL, "min_batch %d < 1", min_batch);
  if (wiring != QF_WIRING_QFIRST && wiring != QF_WIRING_COMPOSED)
    return fail(QF_EINVAL, "wiring %d is neither QF_WIRING_QFIRST nor QF_WIRING_COMPOSED", wiring);
  if (!(ffn_time > 0.0) || !isfinite(ffn_time))
    return fail(QF_EINVAL, "ffn_time must be finite and > 0");
  if (!(max_wait >= 0.0)) return fail(QF_EINVAL, "max_wait must be >= 0 (INFINITY: no time-out)");
  if (n_requests == 0) return QF_OK;
  if (!arrival || !attn_time || !finish) return fail(QF_EINVAL, "a required pointer is NULL");
  for (int r = 0; r < n_requests; ++r)
    if (!isfinite(arrival[r]) || !isfinite(attn_time[r]) || attn_time[r] < 0.0)
      return fail(QF_EINVAL, "request %d: arrival and attention time must be finite, time >= 0", r);
  if ((int64_t)n_requests * n_layers > (int64_t)INT32_MAX)
    return fail(QF_EINVAL, "n_requests * n_layers too large");
  const int rc = qf::simulate_schedule(n_requests, arrival, attn_time, n_layers, wiring, ffn_time,
                                       min_batch, max_wait, finish, sweep_start, sweep_end,
                                       ffn_depart, ffn_return);
  if (rc) return fail(rc, "simulation failed (out of host memory, or no end within its bound on instants)");
  return QF_OK;
}

}  // extern "C"
