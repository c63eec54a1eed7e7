// gfx950 kernels that move K/V rows between paged pools and row-major buffers: kv_append (a
// turn's new tokens into their pages; paper, Background: the context grows by each turn's
// tokens) and the KV transfer pack/unpack between two pools (section 4.3, Eq. 3: under PD
// disaggregation the prefill pool hands the new tokens' K/V to the decode pool, the
// B * dL * K / BW term).
//
// One workgroup copies the rows of one (sequence, logical page): the token range
// [ctx_lens[b], ctx_lens[b] + n_b) cut at page boundaries.  Chunks are 16 bytes and are ordered
// (kv-head, slot, chunk) as in the pool, so pool accesses are contiguous page-head blocks
// (page_size * d * 2 bytes) and row-buffer accesses are contiguous rows of one kv-head.  Each
// thread has four chunks of K and four of V in flight before it stores any.

#include "pearl_internal.h"

namespace pearl {

typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));

constexpr int kCopyThreads = 256;
constexpr int kCopyUnroll = 4;

// kToPool: rows -> pool (append / unpack); otherwise pool -> rows (pack).  A page id outside
// [0, num_pages) is never dereferenced: an append skips those rows, a pack writes zeros.
template <bool kToPool>
__global__ __launch_bounds__(kCopyThreads) void kv_copy_kernel(
    u32x4* __restrict__ pool_k, u32x4* __restrict__ pool_v, u32x4* __restrict__ rows_k,
    u32x4* __restrict__ rows_v, const int32_t* __restrict__ bt, int bt_stride,
    const int32_t* __restrict__ ctx_lens, const int32_t* __restrict__ cu, int pages_per_seq,
    int num_kv_heads, int cpr, int num_pages, int total_q) {
  const int b = blockIdx.x / pages_per_seq;
  const int rel = blockIdx.x - b * pages_per_seq;
  const int q_start = cu ? cu[b] : b;
  const int ctx = ctx_lens[b];
  const int q_len = min(cu ? cu[b + 1] - q_start : 1, total_q - q_start);
  if (q_len <= 0 || q_start < 0 || ctx < 0) return;
  const int lp = ctx / kPage + rel;
  const int p0 = max(ctx, lp * kPage), p1 = min(ctx + q_len, (lp + 1) * kPage);
  if (p0 >= p1 || lp >= bt_stride) return;
  const int page = bt[(size_t)b * bt_stride + lp];
  const bool page_ok = page >= 0 && page < num_pages;
  if (kToPool && !page_ok) return;
  const int ns = p1 - p0, s0 = p0 - lp * kPage;
  const int per_head = ns * cpr;
  const int total = num_kv_heads * per_head;
  const size_t row0 = (size_t)(q_start + p0 - ctx);
  for (int base = 0; base < total; base += kCopyUnroll * kCopyThreads) {
    u32x4 k[kCopyUnroll], v[kCopyUnroll];
    size_t dst[kCopyUnroll];
    bool ok[kCopyUnroll];
#pragma unroll
    for (int u = 0; u < kCopyUnroll; ++u) {
      const int i = base + u * kCopyThreads + threadIdx.x;
      ok[u] = i < total;
      const int ii = ok[u] ? i : 0;
      const int h = ii / per_head;
      const int rem = ii - h * per_head;
      const int s = rem / cpr;
      const int c = rem - s * cpr;
      const size_t poff = (((size_t)(page_ok ? page : 0) * num_kv_heads + h) * kPage + s0 + s) * cpr + c;
      const size_t roff = ((row0 + s) * num_kv_heads + h) * cpr + c;
      if (kToPool) {
        k[u] = ok[u] ? rows_k[roff] : u32x4{0u, 0u, 0u, 0u};
        v[u] = ok[u] ? rows_v[roff] : u32x4{0u, 0u, 0u, 0u};
        dst[u] = poff;
      } else {
        k[u] = ok[u] && page_ok ? pool_k[poff] : u32x4{0u, 0u, 0u, 0u};
        v[u] = ok[u] && page_ok ? pool_v[poff] : u32x4{0u, 0u, 0u, 0u};
        dst[u] = roff;
      }
    }
#pragma unroll
    for (int u = 0; u < kCopyUnroll; ++u) {
      if (!ok[u]) continue;
      if (kToPool) {
        pool_k[dst[u]] = k[u];
        pool_v[dst[u]] = v[u];
      } else {
        rows_k[dst[u]] = k[u];
        rows_v[dst[u]] = v[u];
      }
    }
  }
}

namespace {
hipError_t launch_copy(bool to_pool, uint16_t* pool_k, uint16_t* pool_v, uint16_t* rows_k, uint16_t* rows_v,
                       const int32_t* block_table, int bt_stride, const int32_t* ctx_lens,
                       const int32_t* cu_q_lens, int batch, int max_q_len, int num_kv_heads, int head_dim,
                       int num_pages, int total_q, hipStream_t stream) {
  if (max_q_len <= 0 || batch <= 0 || total_q <= 0) return hipSuccess;
  // a range of n tokens starting anywhere touches at most ceil((n + 15) / 16) pages
  const int pages_per_seq = (max_q_len + 2 * kPage - 2) / kPage;
  const int64_t blocks = (int64_t)batch * pages_per_seq;
  if (blocks > INT32_MAX) return hipErrorInvalidValue;
  const dim3 grid((unsigned)blocks);
  auto* pk = reinterpret_cast<u32x4*>(pool_k);
  auto* pv = reinterpret_cast<u32x4*>(pool_v);
  auto* rk = reinterpret_cast<u32x4*>(rows_k);
  auto* rv = reinterpret_cast<u32x4*>(rows_v);
  if (to_pool)
    hipLaunchKernelGGL(kv_copy_kernel<true>, grid, dim3(kCopyThreads), 0, stream, pk, pv, rk, rv, block_table,
                       bt_stride, ctx_lens, cu_q_lens, pages_per_seq, num_kv_heads, head_dim / 8, num_pages, total_q);
  else
    hipLaunchKernelGGL(kv_copy_kernel<false>, grid, dim3(kCopyThreads), 0, stream, pk, pv, rk, rv, block_table,
                       bt_stride, ctx_lens, cu_q_lens, pages_per_seq, num_kv_heads, head_dim / 8, num_pages, total_q);
  return hipGetLastError();
}
}  // namespace

hipError_t launch_kv_append(const uint16_t* k_new, const uint16_t* v_new, uint16_t* k_pool,
                            uint16_t* v_pool, const int32_t* block_table, int bt_stride,
                            const int32_t* ctx_lens, const int32_t* cu_q_lens, int batch,
                            int max_q_len, int num_kv_heads, int head_dim, int num_pages,
                            int total_q, hipStream_t stream) {
  return launch_copy(true, k_pool, v_pool, const_cast<uint16_t*>(k_new), const_cast<uint16_t*>(v_new),
                     block_table, bt_stride, ctx_lens, cu_q_lens, batch, max_q_len, num_kv_heads, head_dim,
                     num_pages, total_q, stream);
}

hipError_t launch_kv_pack(const uint16_t* k_pool, const uint16_t* v_pool, uint16_t* k_rows, uint16_t* v_rows,
                          const int32_t* block_table, int bt_stride, const int32_t* ctx_lens,
                          const int32_t* cu_q_lens, int batch, int max_q_len, int num_kv_heads, int head_dim,
                          int num_pages, int total_q, hipStream_t stream) {
  return launch_copy(false, const_cast<uint16_t*>(k_pool), const_cast<uint16_t*>(v_pool), k_rows, v_rows,
                     block_table, bt_stride, ctx_lens, cu_q_lens, batch, max_q_len, num_kv_heads, head_dim,
                     num_pages, total_q, stream);
}

}  // namespace pearl
