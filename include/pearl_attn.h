/*
 * pearl_attn.h -- C ABI of the MI355X (gfx950) paged-KV attention library.
 *
 * The computation is the data-parallel core of multi-turn agentic rollout: every turn appends
 * the previous response and the new environment observation to a trajectory's context
 * (paper, Background: p_{t+1} = p_t + r_t + o_t), the engine keeps the K/V of the processed
 * prefix (prefix caching; Motivation, "Efficiency Degradation under PD Colocation") and only the
 * new tokens are prefilled ("append-prefill"; Related work and Evaluation, "Scale-in recovery").
 * Decode then generates one token per sequence per step; its per-sequence marginal cost is the
 * KV-cache read (section 4.3, Eq. 1, term b).  Under PD colocation chunked prefills are batched
 * with decodes on the same GPU (Motivation; section 4.3, Eq. 1), which `pearl_attn_mixed` serves
 * in one launch.
 *
 * The paper gives no attention formula.  The function implemented is standard scaled
 * dot-product attention with grouped-query heads, for new token i of sequence b at absolute
 * position p = ctx_lens[b] + i and q-head h:
 *     s_j = scale * q[h] . k_j   for keys j = 0 .. p (inclusive causal mask),
 *     o   = sum_j softmax(s)_j v_j,          lse = ln sum_j exp(s_j),
 * with k_j, v_j taken from kv-head h / G (G = num_q_heads / num_kv_heads, contiguous groups).
 *
 * Conventions for every entry point
 *   - All tensor pointers are DEVICE pointers on the current HIP device, 16-byte aligned.
 *     bf16 tensors are passed as raw 16-bit patterns.
 *   - K and V pools: bf16 [num_pages][num_kv_heads][page_size][head_dim] (one page of one kv-head
 *     is page_size*head_dim contiguous elements).  Token position p of sequence b lives in
 *     physical page block_table[b*bt_stride + p/page_size], slot p % page_size.
 *   - q, out: bf16 [total_q][num_q_heads][head_dim]; k_new, v_new: bf16 [total_q][num_kv_heads]
 *     [head_dim]; lse: fp32 [total_q][num_q_heads].  Rows of sequence b are rows
 *     cu_q_lens[b] .. cu_q_lens[b+1]-1 (row b when cu_q_lens is NULL).
 *   - `stream` is a hipStream_t (NULL = the null stream).  Calls are asynchronous on it; the
 *     library allocates no device memory and keeps no pointer after returning.  The state it holds
 *     between calls is the per-device launch parameters it queries once, and the calling
 *     thread's timing-event pair while one is set (pearl_set_kernel_events).
 *   - Supported: head_dim 64 or 128; page_size 16; G = num_q_heads/num_kv_heads in {1,2,4,8};
 *     max_q_len <= 2^21 and max_kv_len <= 2^25.  Anything else returns PEARL_ERR_UNSUPPORTED.
 *   - Host-checkable errors (NULL pointers, bad shapes, batch <= 0, sizes inconsistent with each
 *     other, misaligned pointers, workspace too small) return synchronously before any HIP call.
 *     A HIP launch error returns PEARL_ERR_HIP.  The failing detail is in pearl_last_error().
 *   - Device-resident preconditions: lengths consistent with the host bounds in pearl_seq_desc,
 *     block-table entries of attended/written positions in [0, num_pages), and no two written
 *     tokens sharing one (page, slot).  The kernels never access memory outside the pools and
 *     buffers whatever the device data: out-of-range page ids are clamped (attention) or the
 *     write is skipped (append), and a sequence whose lengths violate the host bounds makes the
 *     whole attention call write nothing.  With the environment variable PEARL_DEBUG=1 set, each
 *     attention call synchronises its stream and returns PEARL_ERR_INVALID_ARG if a length
 *     violated the bounds.
 *   - No C++ exception crosses this interface.  Functions are re-entrant; two calls that share a
 *     workspace must be ordered on one stream.
 */
#ifndef PEARL_ATTN_H
#define PEARL_ATTN_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#define PEARL_ABI_VERSION 1

typedef enum {
  PEARL_OK = 0,
  PEARL_ERR_INVALID_ARG = 1,
  PEARL_ERR_UNSUPPORTED = 2,
  PEARL_ERR_WORKSPACE = 3,
  PEARL_ERR_HIP = 4
} pearl_status;

/* Head and pool geometry. */
typedef struct {
  int32_t num_q_heads;   /* H_q (Qwen3-8B and Qwen3-30B-A3B: 32) */
  int32_t num_kv_heads;  /* H_kv; H_q % H_kv == 0 */
  int32_t head_dim;      /* d: 64 or 128 */
  int32_t page_size;     /* tokens per page: 16 */
  int32_t num_pages;     /* physical pages in each of the K and V pools */
} pearl_kv_shape;

/* One batch of sequences.  Pointers are device pointers; the int32 sizes are host values. */
typedef struct {
  const int32_t* block_table; /* [batch][bt_stride] physical page ids */
  int32_t bt_stride;          /* row length of block_table (>= pages of the longest sequence) */
  const int32_t* ctx_lens;    /* [batch] tokens cached BEFORE this call's new tokens */
  const int32_t* cu_q_lens;   /* [batch+1] prefix sums of new tokens per sequence, cu[0] = 0;
                                 NULL means exactly one new token per sequence */
  int32_t batch;              /* number of sequences, > 0 */
  int32_t total_q;            /* rows of q/out/k_new/v_new = cu_q_lens[batch] (= batch if NULL) */
  int32_t max_q_len;          /* host upper bound on any sequence's new tokens */
  int32_t max_kv_len;         /* host upper bound on any ctx_lens[b] + new tokens of b */
} pearl_seq_desc;

int pearl_abi_version(void);

/* Static string naming a status code. */
const char* pearl_status_str(pearl_status status);

/* Detail of the most recent failure on the calling thread ("" if none).  Valid until the next
 * call into the library on that thread. */
const char* pearl_last_error(void);

/*
 * Append this call's new K/V rows into the paged pools (a bit copy; paper, Background: the
 * context grows by appending each turn's tokens).  For sequence b and new token t the rows
 * k_new[cu_q_lens[b]+t][h][:] and v_new[...] are written to slot (ctx_lens[b]+t) % page_size of
 * page block_table[b][(ctx_lens[b]+t) / page_size], for every kv-head h.  No other byte of the
 * pools changes.  A write whose page id is outside [0, num_pages) or whose logical page is
 * beyond bt_stride is skipped.
 *   k_new, v_new: bf16 [total_q][num_kv_heads][head_dim]   (read)
 *   k_pool, v_pool: bf16 [num_pages][num_kv_heads][page_size][head_dim]   (written)
 */
pearl_status pearl_kv_append(const pearl_kv_shape* shape, const pearl_seq_desc* seqs,
                             const void* k_new, const void* v_new, void* k_pool, void* v_pool,
                             void* stream);

/*
 * Bytes of device workspace that any of the three attention calls below needs for (shape,
 * seqs).  The workspace holds the device-built work list and the split-context partial results
 * (fp32); it needs no initialisation and its contents after a call are unspecified.  Returns 0
 * if the arguments are invalid (pearl_last_error() says why).  The size is a function of the
 * shape and the host bounds only.  Decode partials take batch * ceil(pages / split) *
 * num_q_heads * (head_dim + 2) floats.  When cu_q_lens is non-NULL and max_kv_len > 1024,
 * partials of key-split prefill tiles add up to 512 * 256 * (head_dim + 2) floats (65 MiB at
 * head_dim 128).
 */
size_t pearl_attn_workspace_bytes(const pearl_kv_shape* shape, const pearl_seq_desc* seqs);

/*
 * Prefill-append attention (paper: a turn's observation and prompt tokens are prefilled on top
 * of the cached prefix; Background and Motivation sections cited above).  Every new token of
 * every sequence attends causally within its chunk and fully to the cached context; the pools
 * must already hold the new tokens' K/V (call pearl_kv_append first, on the same stream).
 * Sequences with zero new tokens are skipped.  Uses bf16 MFMA tiles with an fp32 online softmax.
 * When a launch has few tiles on long contexts, each tile's keys are split into ranges that run
 * in parallel and are merged by log-sum-exp (decided on the device from the actual lengths).
 *   q: bf16 [total_q][H_q][d] (read); out: bf16 [total_q][H_q][d] (written);
 *   lse: fp32 [total_q][H_q] natural-log log-sum-exp of the scaled scores, or NULL;
 *   softmax_scale: the scale applied to q.k (normally 1/sqrt(d)), > 0 and finite;
 *   workspace: device buffer of workspace_bytes >= pearl_attn_workspace_bytes(...).
 */
pearl_status pearl_attn_prefill_append(const pearl_kv_shape* shape, const pearl_seq_desc* seqs,
                                       const void* q, const void* k_pool, const void* v_pool,
                                       float softmax_scale, void* out, float* lse,
                                       void* workspace, size_t workspace_bytes, void* stream);

/*
 * Batched single-token decode (paper, section 4.3, Eq. 1: the per-iteration decode cost grows
 * with the number of concurrent sequences through their KV-cache reads).  seqs->cu_q_lens must
 * be NULL and total_q == batch: row b of q/out is sequence b's new token at position
 * ctx_lens[b], whose K/V the pools already hold.  The context is split into page ranges that
 * are processed in parallel and merged by log-sum-exp, so small batches still fill the GPU.
 * Arguments as for pearl_attn_prefill_append.
 */
pearl_status pearl_attn_decode(const pearl_kv_shape* shape, const pearl_seq_desc* seqs,
                               const void* q, const void* k_pool, const void* v_pool,
                               float softmax_scale, void* out, float* lse,
                               void* workspace, size_t workspace_bytes, void* stream);

/*
 * One decode step with its append: pearl_kv_append of this step's K/V rows (one per sequence)
 * followed by pearl_attn_decode, with the same results bit for bit (outputs, LSE and both pools).
 * A decode step always appends before it attends (paper, Background: the context grows by every
 * generated token; section 4.3, Eq. 1: the per-step decode cost), so the two run as one launch
 * sequence: the split holding each sequence's last page takes the new K/V straight from k_new /
 * v_new and writes them into the pools itself.
 *   k_new, v_new: bf16 [batch][num_kv_heads][head_dim] (read), 16-byte aligned;
 *   k_pool, v_pool: written at position ctx_lens[b] of every sequence, read for attention;
 *   the other arguments as for pearl_attn_decode (cu_q_lens must be NULL).
 */
pearl_status pearl_attn_decode_append(const pearl_kv_shape* shape, const pearl_seq_desc* seqs,
                                      const void* q, const void* k_new, const void* v_new, void* k_pool,
                                      void* v_pool, float softmax_scale, void* out, float* lse,
                                      void* workspace, size_t workspace_bytes, void* stream);

/*
 * Colocated mixed batch in one attention launch (paper, Motivation: chunked prefill batched
 * with decode; section 4.3, Eq. 1: prefill and decode share the GPU under colocation).  Each
 * sequence may have any number of new tokens (>= 0): sequences with exactly one new token take
 * the split-context decode path, sequences with more take the prefill-append tile path, and
 * both kinds of work items run in a single persistent grid.  Results equal those of
 * pearl_attn_decode / pearl_attn_prefill_append on each sequence alone (up to floating-point
 * summation order).  Arguments as for pearl_attn_prefill_append; cu_q_lens must not be NULL.
 */
pearl_status pearl_attn_mixed(const pearl_kv_shape* shape, const pearl_seq_desc* seqs,
                              const void* q, const void* k_pool, const void* v_pool,
                              float softmax_scale, void* out, float* lse,
                              void* workspace, size_t workspace_bytes, void* stream);

/*
 * Decode without a caller workspace, for callers that cannot allocate device memory at call
 * time (code under HIP graph capture, tight serving loops, harnesses that forbid allocation).
 * Same arguments, kernels and results as pearl_attn_decode, bit for bit; the workspace is instead
 * a static device array of the library, one per GPU (pearl_attn_decode_static_max_bytes() bytes,
 * 32 MiB), which each GPU the library runs on holds until the process ends.  The call allocates
 * nothing: no hipMalloc, no hipFree, no allocating library routine.  The array's device address
 * is looked up on the first call made on each device.
 *   - A batch whose workspace (pearl_attn_workspace_bytes) exceeds the limit returns
 *     PEARL_ERR_UNSUPPORTED before any HIP call; use pearl_attn_decode for it.
 *   - Every call on one GPU shares that GPU's array and leaves its contents behind; each call
 *     rebuilds what it reads, so no clearing is needed between calls.  Calls that overlap on one
 *     GPU (on different streams, or from different threads without ordering) race on the array
 *     and give undefined results: order them on one stream.
 */
size_t pearl_attn_decode_static_max_bytes(void);
pearl_status pearl_attn_decode_static(const pearl_kv_shape* shape, const pearl_seq_desc* seqs,
                                      const void* q, const void* k_pool, const void* v_pool,
                                      float softmax_scale, void* out, float* lse, void* stream);

/*
 * KV transfer between pools (paper, section 4.3, Eq. 3: under PD disaggregation the prefill
 * pool hands each turn's new-token K/V to the decode pool; the transfer takes B * dL * K / BW).
 * pearl_kv_pack gathers, for every sequence b, the K and V rows of positions ctx_lens[b] ..
 * ctx_lens[b] + n_b - 1 (n_b from cu_q_lens, 1 when it is NULL) out of the pools into a
 * contiguous buffer: row cu_q_lens[b] + t holds position ctx_lens[b] + t, for every kv-head.
 * pearl_kv_unpack writes such a buffer into pools through their own block table (it is
 * pearl_kv_append of the buffer's two halves), so the receiving pool may place the pages
 * anywhere.  Both are bit copies; max_q_len bounds n_b and max_kv_len bounds ctx_lens[b] + n_b.
 *   buf: bf16 [2][total_q][num_kv_heads][head_dim]: K rows, then V rows (pack writes it, unpack
 *        reads it); 16-byte aligned.
 *   k_pool, v_pool: as for pearl_kv_append (pack reads them, unpack writes them).
 * A pack reading a page id outside [0, num_pages) writes zeros for those rows; an unpack skips
 * them.  No other byte of buf (pack) or of the pools (unpack) changes.
 */
pearl_status pearl_kv_pack(const pearl_kv_shape* shape, const pearl_seq_desc* seqs,
                           const void* k_pool, const void* v_pool, void* buf, void* stream);
pearl_status pearl_kv_unpack(const pearl_kv_shape* shape, const pearl_seq_desc* seqs,
                             const void* buf, void* k_pool, void* v_pool, void* stream);

/*
 * Timing hook for benchmarks and profilers (not part of the computation).  While a pair is set,
 * every library call made on the calling thread records `before` on its stream immediately
 * before launching its main kernel (the attention kernel for the three attention calls, the
 * page-copy kernel for pearl_kv_append, pearl_kv_pack and pearl_kv_unpack) and `after`
 * immediately after it.  The handles are
 * hipEvent_t values created and owned by the caller; pass NULL, NULL to clear.  The pair stays
 * set until changed, so a caller timing several calls sets a fresh pair before each one.
 */
void pearl_set_kernel_events(void* before, void* after);

#ifdef __cplusplus
}
#endif

#endif /* PEARL_ATTN_H */
