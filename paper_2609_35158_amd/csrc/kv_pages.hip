// gfx950 kernels that move K/V rows between paged pools and row-major buffers: kv_append (a
// turn's new tokens into their pages; paper, Background: the context grows by each turn's
// tokens) and the KV transfer pack/unpack between two pools (section 4.3, Eq. 3: under PD
// disaggregation the prefill pool hands the new tokens' K/V to the decode pool, the
// B * dL * K / BW term).
//
// One workgroup copies the K and the V block of one kv-head of one (sequence, logical page): the
// token range [ctx_lens[b], ctx_lens[b] + n_b) cut at page boundaries gives up to 16 slots, and a
// page-head block is those slots' rows of one kv-head, contiguous in the pool (slots * d * 2
// bytes, 4 KiB for a full page at d = 128).  Its 16-byte chunks are ordered (slot, chunk), so the
// pool side is one contiguous run and the row side is runs of d * 2 bytes, num_kv_heads rows
// apart.  Each of the 128 threads holds at most four chunks (two of K, two of V at d = 128) in
// flight before storing.  Small workgroups with a few chunks each keep reads and writes
// interleaved across the chip over the whole copy.  Measured on a 70 MB turn hand-off and a
// 2.47 GB whole-context move against other shapes: one workgroup per tensor block (half the
// chunks per thread) was 2-3% slower on the unpacks and no faster on the packs; 2 or 4 kv-heads
// per workgroup were 7-13% slower on the turn; one workgroup per page with both tensors and all
// heads (64 KiB) made every workgroup read first and write afterwards in step with all others,
// 0.50 of the HBM peak on the turn.

#include "pearl_internal.h"

namespace pearl {

typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));

constexpr int kCopyThreads = 128;
constexpr int kCopyUnroll = 2;

// kToPool: rows -> pool (append / unpack); otherwise pool -> rows (pack).  A page id outside
// [0, num_pages) is never dereferenced: an append skips those rows, a pack writes zeros.
// blockIdx.x = (b * pages_per_seq + rel) * num_kv_heads + h.
template <bool kToPool>
__global__ __launch_bounds__(kCopyThreads) void kv_copy_kernel(
    u32x4* __restrict__ pool_k, u32x4* __restrict__ pool_v, u32x4* __restrict__ rows_k,
    u32x4* __restrict__ rows_v, const int32_t* __restrict__ bt, int bt_stride,
    const int32_t* __restrict__ ctx_lens, const int32_t* __restrict__ cu, int pages_per_seq,
    int num_kv_heads, int cpr, int num_pages, int total_q) {
  const int bh = blockIdx.x;
  const int item = bh / num_kv_heads;
  const int h = bh - item * num_kv_heads;
  const int b = item / pages_per_seq;
  const int rel = item - b * pages_per_seq;
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
  const int total = (p1 - p0) * cpr;
  const size_t pbase = (((size_t)(page_ok ? page : 0) * num_kv_heads + h) * kPage + (p0 - lp * kPage)) * cpr;
  const size_t row0 = (size_t)(q_start + p0 - ctx);
  for (int base = 0; base < total; base += kCopyUnroll * kCopyThreads) {
    u32x4 x[2 * kCopyUnroll];
    size_t dst[kCopyUnroll];
    bool ok[kCopyUnroll];
#pragma unroll
    for (int u = 0; u < kCopyUnroll; ++u) {
      const int i = base + u * kCopyThreads + threadIdx.x;
      ok[u] = i < total;
      const int ii = ok[u] ? i : 0;
      const int s = ii / cpr;
      const size_t poff = pbase + ii;
      const size_t roff = ((row0 + s) * num_kv_heads + h) * cpr + (ii - s * cpr);
      if (kToPool) {
        x[2 * u] = ok[u] ? rows_k[roff] : u32x4{0u, 0u, 0u, 0u};
        x[2 * u + 1] = ok[u] ? rows_v[roff] : u32x4{0u, 0u, 0u, 0u};
        dst[u] = poff;
      } else {
        // pool pages are read once here: a non-temporal load (measured 5.12 -> 5.48 TB/s on a
        // 2.47 GB pack; rows -> pool copies measured no gain from it, and non-temporal stores
        // were slower in every direction)
        x[2 * u] = ok[u] && page_ok ? __builtin_nontemporal_load(&pool_k[poff]) : u32x4{0u, 0u, 0u, 0u};
        x[2 * u + 1] = ok[u] && page_ok ? __builtin_nontemporal_load(&pool_v[poff]) : u32x4{0u, 0u, 0u, 0u};
        dst[u] = roff;
      }
    }
#pragma unroll
    for (int u = 0; u < kCopyUnroll; ++u) {
      if (!ok[u]) continue;
      if (kToPool) {
        pool_k[dst[u]] = x[2 * u];
        pool_v[dst[u]] = x[2 * u + 1];
      } else {
        rows_k[dst[u]] = x[2 * u];
        rows_v[dst[u]] = x[2 * u + 1];
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
  const int64_t blocks = (int64_t)batch * pages_per_seq * num_kv_heads;
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
