// C-ABI host layer: argument validation, workspace layout, launch sequencing and error mapping for
// the gfx950 paged-KV attention kernels.  The interface and its contract are documented in
// include/pearl_attn.h.

#include "../../include/pearl_attn.h"
#include "pearl_internal.h"

#include <hip/hip_runtime.h>

#include <algorithm>
#include <cmath>
#include <cstdarg>
#include <cstdio>
#include <cstdlib>
#include <cstring>

namespace pearl {
namespace {

thread_local char g_err[512] = "";
thread_local hipEvent_t g_ev_before = nullptr;
thread_local hipEvent_t g_ev_after = nullptr;

hipError_t record_before(hipStream_t s) { return g_ev_before ? hipEventRecord(g_ev_before, s) : hipSuccess; }
hipError_t record_after(hipStream_t s) { return g_ev_after ? hipEventRecord(g_ev_after, s) : hipSuccess; }

void set_err(const char* fmt, ...) {
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(g_err, sizeof(g_err), fmt, ap);
  va_end(ap);
}

pearl_status fail(pearl_status st, const char* fmt, ...) {
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(g_err, sizeof(g_err), fmt, ap);
  va_end(ap);
  return st;
}

size_t align256(size_t x) { return (x + 255) & ~size_t(255); }

bool aligned16(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15) == 0; }

int64_t cdiv(int64_t a, int64_t b) { return (a + b - 1) / b; }

bool debug_mode() {
  const char* e = std::getenv("PEARL_DEBUG");
  return e && e[0] && e[0] != '0';
}

// Shape checks shared by every entry point.
pearl_status check_shape(const pearl_kv_shape* s) {
  if (!s) return fail(PEARL_ERR_INVALID_ARG, "shape is NULL");
  if (s->num_q_heads <= 0 || s->num_kv_heads <= 0)
    return fail(PEARL_ERR_INVALID_ARG, "num_q_heads (%d) and num_kv_heads (%d) must be > 0", s->num_q_heads, s->num_kv_heads);
  if (s->num_q_heads % s->num_kv_heads != 0)
    return fail(PEARL_ERR_INVALID_ARG, "num_q_heads (%d) is not a multiple of num_kv_heads (%d)", s->num_q_heads, s->num_kv_heads);
  const int G = s->num_q_heads / s->num_kv_heads;
  if (G != 1 && G != 2 && G != 4 && G != 8)
    return fail(PEARL_ERR_UNSUPPORTED, "query heads per kv-head G=%d not in {1,2,4,8}", G);
  if (s->head_dim != 64 && s->head_dim != 128)
    return fail(PEARL_ERR_UNSUPPORTED, "head_dim %d not in {64,128}", s->head_dim);
  if (s->page_size != kPage) return fail(PEARL_ERR_UNSUPPORTED, "page_size %d != 16", s->page_size);
  if (s->num_pages <= 0) return fail(PEARL_ERR_INVALID_ARG, "num_pages (%d) must be > 0", s->num_pages);
  return PEARL_OK;
}

pearl_status check_seqs(const pearl_seq_desc* q, bool need_q_lens) {
  if (!q) return fail(PEARL_ERR_INVALID_ARG, "seqs is NULL");
  if (q->batch <= 0) return fail(PEARL_ERR_INVALID_ARG, "batch (%d) must be > 0", q->batch);
  if (!q->block_table) return fail(PEARL_ERR_INVALID_ARG, "block_table is NULL");
  if (!q->ctx_lens) return fail(PEARL_ERR_INVALID_ARG, "ctx_lens is NULL");
  if (q->bt_stride <= 0) return fail(PEARL_ERR_INVALID_ARG, "bt_stride (%d) must be > 0", q->bt_stride);
  if (q->total_q < 0 || q->max_q_len < 0 || q->max_kv_len < 0)
    return fail(PEARL_ERR_INVALID_ARG, "total_q, max_q_len and max_kv_len must be >= 0");
  if (need_q_lens && !q->cu_q_lens) return fail(PEARL_ERR_INVALID_ARG, "cu_q_lens is NULL");
  if (!q->cu_q_lens) {
    if (q->total_q != q->batch)
      return fail(PEARL_ERR_INVALID_ARG, "cu_q_lens is NULL (one token per sequence) but total_q (%d) != batch (%d)", q->total_q, q->batch);
    if (q->max_q_len < 1) return fail(PEARL_ERR_INVALID_ARG, "max_q_len (%d) < 1 with one token per sequence", q->max_q_len);
  }
  if (q->max_q_len > q->total_q) return fail(PEARL_ERR_INVALID_ARG, "max_q_len (%d) > total_q (%d)", q->max_q_len, q->total_q);
  if (q->max_q_len > q->max_kv_len && q->total_q > 0)
    return fail(PEARL_ERR_INVALID_ARG, "max_q_len (%d) > max_kv_len (%d)", q->max_q_len, q->max_kv_len);
  if ((int64_t)q->bt_stride * kPage < q->max_kv_len)
    return fail(PEARL_ERR_INVALID_ARG, "bt_stride (%d) pages cannot hold max_kv_len (%d) tokens", q->bt_stride, q->max_kv_len);
  if ((int64_t)q->batch * q->bt_stride > INT32_MAX)
    return fail(PEARL_ERR_INVALID_ARG, "block table too large");
  if (q->max_q_len > kMaxQLen) return fail(PEARL_ERR_UNSUPPORTED, "max_q_len (%d) > %d", q->max_q_len, kMaxQLen);
  if (q->max_kv_len > kMaxKvLen) return fail(PEARL_ERR_UNSUPPORTED, "max_kv_len (%d) > %d", q->max_kv_len, kMaxKvLen);
  return PEARL_OK;
}

struct Plan {
  PlanParams p;
  WsLayout lay;
};

Plan make_plan(const pearl_kv_shape* s, const pearl_seq_desc* q, int mode) {
  Plan pl;
  const int G = s->num_q_heads / s->num_kv_heads;
  const int pps = choose_pages_per_split(q->batch, s->num_kv_heads, q->max_kv_len, kPlanComputeUnits);
  pl.lay = workspace_layout(q->batch, q->total_q, q->max_kv_len, s->num_q_heads, s->num_kv_heads, s->head_dim, G, pps,
                            q->cu_q_lens != nullptr);
  PlanParams& p = pl.p;
  p.mode = mode;
  p.batch = q->batch;
  p.total_q = q->total_q;
  p.max_q_len = q->max_q_len;
  p.max_kv_len = q->max_kv_len;
  p.bt_stride = q->bt_stride;
  p.num_kv_heads = s->num_kv_heads;
  p.group = G;
  p.tokens_per_tile = kRowsPerTile / G;
  p.pages_per_split = pps;
  p.max_pre = pl.lay.max_pre;
  p.max_dec = pl.lay.max_dec;
  p.pre_slots = mode == kModeDecode ? 0 : pl.lay.pre_slots;
  p.pre_jobs_cap = mode == kModeDecode ? 0 : pl.lay.pre_jobs_cap;
  p.mixed_grid = mode == kModeMixed ? attention_grid(s->head_dim, 3) : 0;
  return pl;
}

// static_ws: use the library's static per-device workspace (pearl_attn_decode_static) instead of
// the caller's ws / ws_bytes; its address is looked up only after every host check has passed.
// k_new / v_new (decode only, both or neither): append the new tokens' K/V first, as
// pearl_kv_append would; decode planned in-kernel does it inside the attention kernel.
pearl_status run_attention(int mode, const pearl_kv_shape* s, const pearl_seq_desc* q, const void* qp,
                           const void* k_pool, const void* v_pool, float scale, void* out, float* lse,
                           void* ws, size_t ws_bytes, void* stream, bool static_ws = false,
                           const void* k_new = nullptr, const void* v_new = nullptr) {
  g_err[0] = 0;
  pearl_status st = check_shape(s);
  if (st != PEARL_OK) return st;
  st = check_seqs(q, mode == kModeMixed);
  if (st != PEARL_OK) return st;
  if (mode == kModeDecode && q->cu_q_lens)
    return fail(PEARL_ERR_INVALID_ARG, "pearl_attn_decode requires cu_q_lens == NULL (one token per sequence)");
  if (!qp || !k_pool || !v_pool || !out) return fail(PEARL_ERR_INVALID_ARG, "q, k_pool, v_pool and out must be non-NULL");
  if ((k_new == nullptr) != (v_new == nullptr)) return fail(PEARL_ERR_INVALID_ARG, "k_new and v_new must both be given");
  if (k_new && (!aligned16(k_new) || !aligned16(v_new)))
    return fail(PEARL_ERR_INVALID_ARG, "k_new and v_new must be 16-byte aligned");
  if (!ws && !static_ws) return fail(PEARL_ERR_WORKSPACE, "workspace is NULL");
  if (!aligned16(qp) || !aligned16(k_pool) || !aligned16(v_pool) || !aligned16(out))
    return fail(PEARL_ERR_INVALID_ARG, "q, k_pool, v_pool and out must be 16-byte aligned");
  if (!static_ws && (reinterpret_cast<uintptr_t>(ws) & 255) != 0)
    return fail(PEARL_ERR_WORKSPACE, "workspace must be 256-byte aligned");
  if (lse && (reinterpret_cast<uintptr_t>(lse) & 3) != 0) return fail(PEARL_ERR_INVALID_ARG, "lse must be 4-byte aligned");
  if (!(scale > 0.f) || !std::isfinite(scale)) return fail(PEARL_ERR_INVALID_ARG, "softmax_scale must be finite and > 0");
  const int64_t total_rows = (int64_t)q->total_q * s->num_q_heads * s->head_dim;
  if (total_rows > INT32_MAX * int64_t(8)) return fail(PEARL_ERR_UNSUPPORTED, "q/out too large");
  Plan pl = make_plan(s, q, mode);
  // the device keeps entry and item counts in int32
  if ((pl.lay.max_pre + pl.lay.max_dec) * (int64_t)s->num_kv_heads > INT32_MAX)
    return fail(PEARL_ERR_UNSUPPORTED, "work list bound (%lld entries x %d kv-heads) exceeds int32",
                (long long)(pl.lay.max_pre + pl.lay.max_dec), s->num_kv_heads);
  if (static_ws) {
    if (pl.lay.total > kStaticScratchBytes)
      return fail(PEARL_ERR_UNSUPPORTED, "this batch needs %zu bytes of workspace, above the static limit of %zu "
                  "bytes (use pearl_attn_decode with a caller workspace)", pl.lay.total, kStaticScratchBytes);
    hipError_t se = hipSuccess;
    ws = static_scratch(&se);
    if (!ws) return fail(PEARL_ERR_HIP, "static workspace address: %s", hipGetErrorString(se));
    ws_bytes = kStaticScratchBytes;
  }
  if (ws_bytes < pl.lay.total)
    return fail(PEARL_ERR_WORKSPACE, "workspace_bytes %zu < required %zu", ws_bytes, pl.lay.total);
  hipStream_t hs = reinterpret_cast<hipStream_t>(stream);
  char* w = static_cast<char*>(ws);
  // decode batches up to kDecPlanMaxSeqs are planned inside the attention kernel, which also
  // merges the splits; everything else is planned by plan_kernel and merged by the merge kernels
  const bool dec_in_kernel = mode == kModeDecode && q->batch <= kDecPlanMaxSeqs;
  hipError_t e = hipSuccess;
  if (k_new && !dec_in_kernel) {
    e = launch_kv_append(static_cast<const uint16_t*>(k_new), static_cast<const uint16_t*>(v_new),
                         static_cast<uint16_t*>(const_cast<void*>(k_pool)), static_cast<uint16_t*>(const_cast<void*>(v_pool)),
                         q->block_table, q->bt_stride, q->ctx_lens, nullptr, q->batch, 1, s->num_kv_heads, s->head_dim,
                         s->num_pages, q->total_q, hs);
    if (e != hipSuccess) return fail(PEARL_ERR_HIP, "kv_append launch: %s", hipGetErrorString(e));
  }
  if (!dec_in_kernel) {
    e = launch_plan(pl.p, q->ctx_lens, q->cu_q_lens, ws, pl.lay, hs);
    if (e != hipSuccess) return fail(PEARL_ERR_HIP, "plan launch: %s", hipGetErrorString(e));
  }
  AttnArgs a;
  a.q = static_cast<const uint16_t*>(qp);
  a.k_pool = static_cast<const uint16_t*>(k_pool);
  a.v_pool = static_cast<const uint16_t*>(v_pool);
  a.block_table = q->block_table;
  a.out = static_cast<uint16_t*>(out);
  a.lse = lse;
  a.ws_hdr = reinterpret_cast<int32_t*>(w + pl.lay.hdr);
  a.seqinfo = reinterpret_cast<const SeqInfo*>(w + pl.lay.seqinfo);
  a.split_base = reinterpret_cast<const int32_t*>(w + pl.lay.split_base);
  a.entries = reinterpret_cast<const int2*>(w + pl.lay.entries);
  a.part_o = reinterpret_cast<float*>(w + pl.lay.part_o);
  a.part_ml = reinterpret_cast<float*>(w + pl.lay.part_ml);
  a.pre_jobs = reinterpret_cast<const int4*>(w + pl.lay.pre_jobs);
  a.part_pre_o = reinterpret_cast<float*>(w + pl.lay.part_pre_o);
  a.part_pre_ml = reinterpret_cast<float*>(w + pl.lay.part_pre_ml);
  a.split_cnt = reinterpret_cast<int32_t*>(w + pl.lay.split_cnt);
  a.k_new = dec_in_kernel ? static_cast<const uint16_t*>(k_new) : nullptr;
  a.v_new = dec_in_kernel ? static_cast<const uint16_t*>(v_new) : nullptr;
  a.k_pool_w = static_cast<uint16_t*>(const_cast<void*>(k_pool));
  a.v_pool_w = static_cast<uint16_t*>(const_cast<void*>(v_pool));
  a.bt_stride = q->bt_stride;
  a.num_pages = s->num_pages;
  a.num_q_heads = s->num_q_heads;
  a.num_kv_heads = s->num_kv_heads;
  a.group = pl.p.group;
  a.tokens_per_tile = pl.p.tokens_per_tile;
  a.scale_log2 = scale * 1.4426950408889634f;
  const int64_t max_items = (pl.lay.max_pre + pl.lay.max_dec) * s->num_kv_heads;
  if (dec_in_kernel) {
    e = launch_decode_prologue(a, q->batch, hs);
    if (e != hipSuccess) return fail(PEARL_ERR_HIP, "decode prologue launch: %s", hipGetErrorString(e));
  }
  e = record_before(hs);
  if (e != hipSuccess) return fail(PEARL_ERR_HIP, "timing event: %s", hipGetErrorString(e));
  if (dec_in_kernel) {
    DecPlanArgs d;
    d.ctx_lens = q->ctx_lens;
    d.batch = q->batch;
    d.max_kv_len = q->max_kv_len;
    d.pps_min = pl.p.pages_per_split;
    d.max_dec = (int)pl.lay.max_dec;
    e = launch_decode(a, d, s->head_dim, pl.lay.max_dec * s->num_kv_heads, hs);
  } else {
    const int kinds = mode == kModePrefill ? 1 : (mode == kModeDecode ? 2 : 3);
    e = launch_attention(a, s->head_dim, kinds, max_items, (int)pl.lay.max_pre, hs);
  }
  if (e != hipSuccess) return fail(PEARL_ERR_HIP, "attention launch: %s", hipGetErrorString(e));
  e = record_after(hs);
  if (e != hipSuccess) return fail(PEARL_ERR_HIP, "timing event: %s", hipGetErrorString(e));
  if (!dec_in_kernel && mode != kModePrefill && pl.lay.max_dec > 0) {
    e = launch_merge(a, s->head_dim, q->batch, hs);
    if (e != hipSuccess) return fail(PEARL_ERR_HIP, "merge launch: %s", hipGetErrorString(e));
  }
  if (pl.p.pre_jobs_cap > 0) {
    e = launch_merge_prefill(a, s->head_dim, pl.p.pre_jobs_cap, hs);
    if (e != hipSuccess) return fail(PEARL_ERR_HIP, "prefill merge launch: %s", hipGetErrorString(e));
  }
  if (debug_mode()) {
    e = hipStreamSynchronize(hs);
    if (e != hipSuccess) return fail(PEARL_ERR_HIP, "PEARL_DEBUG sync: %s", hipGetErrorString(e));
    int32_t flag = 0;
    e = hipMemcpy(&flag, w + pl.lay.hdr + 4 * kHdrError, sizeof(flag), hipMemcpyDeviceToHost);
    if (e != hipSuccess) return fail(PEARL_ERR_HIP, "PEARL_DEBUG readback: %s", hipGetErrorString(e));
    if (flag == 1) return fail(PEARL_ERR_INVALID_ARG, "device lengths violate the host bounds (total_q/max_q_len/max_kv_len/bt_stride) or decode q_len != 1; nothing was computed");
    if (flag != 0) return fail(PEARL_ERR_INVALID_ARG, "work list exceeded its capacity; nothing was computed");
  }
  return PEARL_OK;
}

}  // namespace

void clear_error() { g_err[0] = 0; }

pearl_status set_error(pearl_status st, const char* fmt, ...) {
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(g_err, sizeof(g_err), fmt, ap);
  va_end(ap);
  return st;
}

int choose_pages_per_split(int batch, int num_kv_heads, int max_kv_len, int num_cu) {
  // The least pages per decode split, which sizes the workspace: about 16 decode items per
  // compute unit if every sequence were as long as the bound.  A split never holds fewer than 16
  // pages (two pages for each of the 8 waves), and its size is a multiple of 16 pages.  The
  // planner takes larger splits from the launch's actual pages (kDecItemsPerCU).
  const int64_t max_pages = std::max<int64_t>(1, cdiv(std::max(max_kv_len, 1), kPage));
  const int64_t target = std::max<int64_t>(1, (int64_t)num_cu * 16);
  int64_t pps = cdiv((int64_t)batch * num_kv_heads * max_pages, target);
  pps = std::max<int64_t>(pps, kMinPagesPerSplit);
  pps = cdiv(pps, 16) * 16;
  if (pps > kMaxPagesPerSplit) pps = kMaxPagesPerSplit;
  return (int)pps;
}

WsLayout workspace_layout(int batch, int total_q, int max_kv_len, int num_q_heads, int num_kv_heads,
                          int head_dim, int group, int pages_per_split, bool has_prefill) {
  WsLayout l;
  const int T = kRowsPerTile / group;
  // prefill tiles: sum_b ceil(n_b / T) <= total_q / T + batch, and <= total_q
  const int64_t tiles = std::min<int64_t>(total_q, total_q / T + batch);
  // split prefill items: every tile splits into at most ceil(max_kv_len / kMinSplitKeys) ranges,
  // and the planner keeps the split items of a launch within kMaxPreSplitItems
  l.pre_slots = 0;
  if (has_prefill && max_kv_len > kMinSplitKeys)
    l.pre_slots = std::min<int64_t>(kMaxPreSplitItems, (int64_t)num_kv_heads * tiles * cdiv(max_kv_len, kMinSplitKeys));
  l.pre_jobs_cap = l.pre_slots / num_kv_heads;
  l.max_pre = std::max<int64_t>(tiles, l.pre_jobs_cap);
  // decode entries: every sequence holds at most ceil(max_kv_len / 16) pages
  const int64_t max_pages = cdiv(std::max(max_kv_len, 1), kPage);
  l.max_dec = (int64_t)batch * cdiv(max_pages, pages_per_split);
  size_t off = 0;
  l.hdr = off; off = align256(off + sizeof(int32_t) * kHdrWords);
  l.seqinfo = off; off = align256(off + sizeof(SeqInfo) * (size_t)batch);
  l.split_base = off; off = align256(off + sizeof(int32_t) * (size_t)batch);
  l.entries = off; off = align256(off + sizeof(int2) * (size_t)(l.max_pre + l.max_dec));
  l.part_o = off; off = align256(off + sizeof(float) * (size_t)l.max_dec * num_q_heads * head_dim);
  l.part_ml = off; off = align256(off + sizeof(float) * 2 * (size_t)l.max_dec * num_q_heads);
  l.pre_jobs = off; off = align256(off + sizeof(int4) * (size_t)l.pre_jobs_cap);
  l.part_pre_o = off; off = align256(off + sizeof(float) * (size_t)l.pre_slots * kRowsPerTile * head_dim);
  l.part_pre_ml = off; off = align256(off + sizeof(float) * 2 * (size_t)l.pre_slots * kRowsPerTile);
  l.split_cnt = off; off = align256(off + sizeof(int32_t) * (size_t)batch * num_kv_heads);
  l.total = off;
  return l;
}

}  // namespace pearl

using namespace pearl;

extern "C" {

int pearl_abi_version(void) { return PEARL_ABI_VERSION; }

const char* pearl_status_str(pearl_status st) {
  switch (st) {
    case PEARL_OK: return "PEARL_OK";
    case PEARL_ERR_INVALID_ARG: return "PEARL_ERR_INVALID_ARG";
    case PEARL_ERR_UNSUPPORTED: return "PEARL_ERR_UNSUPPORTED";
    case PEARL_ERR_WORKSPACE: return "PEARL_ERR_WORKSPACE";
    case PEARL_ERR_HIP: return "PEARL_ERR_HIP";
  }
  return "PEARL_ERR_UNKNOWN";
}

const char* pearl_last_error(void) { return g_err; }

pearl_status pearl_kv_append(const pearl_kv_shape* shape, const pearl_seq_desc* seqs, const void* k_new,
                             const void* v_new, void* k_pool, void* v_pool, void* stream) {
  try {
    g_err[0] = 0;
    pearl_status st = check_shape(shape);
    if (st != PEARL_OK) return st;
    st = check_seqs(seqs, false);
    if (st != PEARL_OK) return st;
    if (seqs->total_q == 0) return PEARL_OK;
    if (!k_new || !v_new || !k_pool || !v_pool) return fail(PEARL_ERR_INVALID_ARG, "k_new, v_new, k_pool and v_pool must be non-NULL");
    if (!aligned16(k_new) || !aligned16(v_new) || !aligned16(k_pool) || !aligned16(v_pool))
      return fail(PEARL_ERR_INVALID_ARG, "k_new, v_new, k_pool and v_pool must be 16-byte aligned");
    hipError_t e = record_before(reinterpret_cast<hipStream_t>(stream));
    if (e != hipSuccess) return fail(PEARL_ERR_HIP, "timing event: %s", hipGetErrorString(e));
    e = launch_kv_append(static_cast<const uint16_t*>(k_new), static_cast<const uint16_t*>(v_new),
                                    static_cast<uint16_t*>(k_pool), static_cast<uint16_t*>(v_pool), seqs->block_table,
                                    seqs->bt_stride, seqs->ctx_lens, seqs->cu_q_lens, seqs->batch, seqs->max_q_len,
                                    shape->num_kv_heads, shape->head_dim, shape->num_pages, seqs->total_q,
                                    reinterpret_cast<hipStream_t>(stream));
    if (e != hipSuccess) return fail(PEARL_ERR_HIP, "kv_append launch: %s", hipGetErrorString(e));
    e = record_after(reinterpret_cast<hipStream_t>(stream));
    if (e != hipSuccess) return fail(PEARL_ERR_HIP, "timing event: %s", hipGetErrorString(e));
    return PEARL_OK;
  } catch (...) {
    return fail(PEARL_ERR_HIP, "unexpected exception in pearl_kv_append");
  }
}

pearl_status pearl_kv_pack(const pearl_kv_shape* shape, const pearl_seq_desc* seqs, const void* k_pool,
                           const void* v_pool, void* buf, void* stream) {
  try {
    g_err[0] = 0;
    pearl_status st = check_shape(shape);
    if (st != PEARL_OK) return st;
    st = check_seqs(seqs, false);
    if (st != PEARL_OK) return st;
    if (seqs->total_q == 0) return PEARL_OK;
    if (!k_pool || !v_pool || !buf) return fail(PEARL_ERR_INVALID_ARG, "k_pool, v_pool and buf must be non-NULL");
    if (!aligned16(k_pool) || !aligned16(v_pool) || !aligned16(buf))
      return fail(PEARL_ERR_INVALID_ARG, "k_pool, v_pool and buf must be 16-byte aligned");
    hipStream_t hs = reinterpret_cast<hipStream_t>(stream);
    uint16_t* k_rows = static_cast<uint16_t*>(buf);
    uint16_t* v_rows = k_rows + (size_t)seqs->total_q * shape->num_kv_heads * shape->head_dim;
    hipError_t e = record_before(hs);
    if (e != hipSuccess) return fail(PEARL_ERR_HIP, "timing event: %s", hipGetErrorString(e));
    e = launch_kv_pack(static_cast<const uint16_t*>(k_pool), static_cast<const uint16_t*>(v_pool), k_rows, v_rows,
                       seqs->block_table, seqs->bt_stride, seqs->ctx_lens, seqs->cu_q_lens, seqs->batch,
                       seqs->max_q_len, shape->num_kv_heads, shape->head_dim, shape->num_pages, seqs->total_q, hs);
    if (e != hipSuccess) return fail(PEARL_ERR_HIP, "kv_pack launch: %s", hipGetErrorString(e));
    e = record_after(hs);
    if (e != hipSuccess) return fail(PEARL_ERR_HIP, "timing event: %s", hipGetErrorString(e));
    return PEARL_OK;
  } catch (...) {
    return fail(PEARL_ERR_HIP, "unexpected exception in pearl_kv_pack");
  }
}

pearl_status pearl_kv_unpack(const pearl_kv_shape* shape, const pearl_seq_desc* seqs, const void* buf,
                             void* k_pool, void* v_pool, void* stream) {
  try {
    g_err[0] = 0;
    pearl_status st = check_shape(shape);
    if (st != PEARL_OK) return st;
    st = check_seqs(seqs, false);
    if (st != PEARL_OK) return st;
    if (seqs->total_q == 0) return PEARL_OK;
    if (!buf) return fail(PEARL_ERR_INVALID_ARG, "buf must be non-NULL");
    // the unpack is the append of the buffer's K half and V half
    const uint16_t* k_rows = static_cast<const uint16_t*>(buf);
    const uint16_t* v_rows = k_rows + (size_t)seqs->total_q * shape->num_kv_heads * shape->head_dim;
    return pearl_kv_append(shape, seqs, k_rows, v_rows, k_pool, v_pool, stream);
  } catch (...) {
    return fail(PEARL_ERR_HIP, "unexpected exception in pearl_kv_unpack");
  }
}

void pearl_set_kernel_events(void* before, void* after) {
  g_ev_before = reinterpret_cast<hipEvent_t>(before);
  g_ev_after = reinterpret_cast<hipEvent_t>(after);
}

size_t pearl_attn_workspace_bytes(const pearl_kv_shape* shape, const pearl_seq_desc* seqs) {
  try {
    g_err[0] = 0;
    if (check_shape(shape) != PEARL_OK) return 0;
    if (check_seqs(seqs, false) != PEARL_OK) return 0;
    const int G = shape->num_q_heads / shape->num_kv_heads;
    const int pps = choose_pages_per_split(seqs->batch, shape->num_kv_heads, seqs->max_kv_len, kPlanComputeUnits);
    return workspace_layout(seqs->batch, seqs->total_q, seqs->max_kv_len, shape->num_q_heads, shape->num_kv_heads,
                            shape->head_dim, G, pps, seqs->cu_q_lens != nullptr).total;
  } catch (...) {
    set_err("unexpected exception in pearl_attn_workspace_bytes");
    return 0;
  }
}

#define PEARL_ATTN_ENTRY(NAME, MODE)                                                                       \
  pearl_status NAME(const pearl_kv_shape* shape, const pearl_seq_desc* seqs, const void* q, const void* k_pool, \
                    const void* v_pool, float softmax_scale, void* out, float* lse, void* workspace,         \
                    size_t workspace_bytes, void* stream) {                                                \
    try {                                                                                                  \
      return run_attention(MODE, shape, seqs, q, k_pool, v_pool, softmax_scale, out, lse, workspace,      \
                           workspace_bytes, stream);                                                       \
    } catch (...) {                                                                                        \
      return fail(PEARL_ERR_HIP, "unexpected exception in " #NAME);                                         \
    }                                                                                                      \
  }

PEARL_ATTN_ENTRY(pearl_attn_prefill_append, kModePrefill)
PEARL_ATTN_ENTRY(pearl_attn_decode, kModeDecode)
PEARL_ATTN_ENTRY(pearl_attn_mixed, kModeMixed)

pearl_status pearl_attn_decode_append(const pearl_kv_shape* shape, const pearl_seq_desc* seqs, const void* q,
                                      const void* k_new, const void* v_new, void* k_pool, void* v_pool,
                                      float softmax_scale, void* out, float* lse, void* workspace,
                                      size_t workspace_bytes, void* stream) {
  try {
    if (!k_new || !v_new) {
      g_err[0] = 0;
      return fail(PEARL_ERR_INVALID_ARG, "k_new and v_new must be non-NULL");
    }
    return run_attention(kModeDecode, shape, seqs, q, k_pool, v_pool, softmax_scale, out, lse, workspace,
                         workspace_bytes, stream, false, k_new, v_new);
  } catch (...) {
    return fail(PEARL_ERR_HIP, "unexpected exception in pearl_attn_decode_append");
  }
}

size_t pearl_attn_decode_static_max_bytes(void) { return kStaticScratchBytes; }

pearl_status pearl_attn_decode_static(const pearl_kv_shape* shape, const pearl_seq_desc* seqs, const void* q,
                                      const void* k_pool, const void* v_pool, float softmax_scale, void* out,
                                      float* lse, void* stream) {
  try {
    return run_attention(kModeDecode, shape, seqs, q, k_pool, v_pool, softmax_scale, out, lse, nullptr, 0, stream,
                         /*static_ws=*/true);
  } catch (...) {
    return fail(PEARL_ERR_HIP, "unexpected exception in pearl_attn_decode_static");
  }
}

}  // extern "C"
