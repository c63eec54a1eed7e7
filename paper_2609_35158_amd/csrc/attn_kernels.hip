// gfx950 (MI355X) kernels for paged-KV GQA attention: the device-side work
// planner, the persistent attention kernel (prefill-append tiles on bf16 MFMA and split-context
// decode items in one grid), and the split merge.
//
// The computation: new tokens of each sequence attend causally within their chunk and fully to
// the cached context (paper, Background: context growth p_{t+1} = p_t + r_t + o_t; Motivation:
// prefix caching and chunked prefill batched with decode; section 4.3, Eq. 1: decode cost per
// sequence is its KV-cache read).  Scores are s_j = scale * q.k_j over keys j <= position; the
// softmax is evaluated online in base 2 (exp(x) = 2^(x log2 e)), fp32 state, bf16 operands.
// The row sum l accumulates the fp32 weights (so the LSE is accurate to fp32); the weights enter
// the P.V product rounded to bf16 (round to nearest even).
//
// MFMA lane layouts used below (gfx950, bf16, fp32 accumulate; lane l of a 64-lane wave):
//   32x32x16: A row l%32, k 8*(l/32)+e;  B col l%32, k 8*(l/32)+e;
//             D col l%32, row (r%4) + 8*(r/4) + 4*(l/32) for accumulator r = 0..15.
//   16x16x32: A row l%16, k 8*(l/16)+e;  B col l%16, k 8*(l/16)+e;
//             D col l%16, row 4*(l/16) + r for r = 0..3.
// The contraction index k may be any permutation of the reduced dimension as long as A and B
// use the same one; the P.V products below use that freedom so the probabilities feed the B
// operand straight from the score accumulators.
//
// LDS transpose read (ds_read_b64_tr_b16): inside each 16-lane group, lane j supplies the
// address of an 8-byte row; lane l receives element l%4 of the rows supplied by lanes l/4,
// l/4+4, l/4+8, l/4+12.  With lane j addressing V[kbase + j/4][dbase + 4*(j%4)] (V row-major,
// keys x dims), lane l receives V[kbase + i][dbase + l%16] for i = 0..3: four consecutive keys
// of one dim, i.e. a k-contiguous MFMA operand of V^T.

#include "pearl_internal.h"

#include <math.h>

#include <atomic>
#include <type_traits>
#include <mutex>

namespace pearl {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef short i16x4 __attribute__((ext_vector_type(4)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));
typedef unsigned int u32x2 __attribute__((ext_vector_type(2)));

#define LDS_AS __attribute__((address_space(3)))

constexpr float kLn2 = 0.69314718055994530942f;

__device__ __forceinline__ u32x4 ld16(const uint16_t* p) { return *reinterpret_cast<const u32x4*>(p); }
__device__ __forceinline__ bf16x8 as_bf16x8(u32x4 v) { return __builtin_bit_cast(bf16x8, v); }
__device__ __forceinline__ bf16x8 zero_bf16x8() { return as_bf16x8(u32x4{0u, 0u, 0u, 0u}); }

__device__ __forceinline__ float fexp2(float x) { return __builtin_amdgcn_exp2f(x); }

// The XCD this wave runs on (hardware register XCC_ID, bits 3:0), in [0, kNumXcd).
__device__ __forceinline__ int xcc_id() { return __builtin_amdgcn_s_getreg(20 | (0 << 6) | (3 << 11)) % kNumXcd; }
__device__ __forceinline__ float flog2(float x) { return __builtin_amdgcn_logf(x); }

__device__ __forceinline__ uint16_t bf16_bits(float x) { return __builtin_bit_cast(uint16_t, (__bf16)x); }

__device__ __forceinline__ i16x4 lds_read_tr(const char* base, int byte_off) {
  // generic -> LDS address-space cast (the pointer always points into __shared__ memory)
  LDS_AS i16x4* p = (LDS_AS i16x4*)((LDS_AS char*)(base) + byte_off);
  return __builtin_amdgcn_ds_read_tr16_b64_v4i16(p);
}

__device__ __forceinline__ bf16x8 concat_tr(i16x4 a, i16x4 b) {
  typedef short i16x8 __attribute__((ext_vector_type(8)));
  i16x8 v = {a[0], a[1], a[2], a[3], b[0], b[1], b[2], b[3]};
  return __builtin_bit_cast(bf16x8, v);
}

// Combine x with the value held by lane l ^ 32, using v_permlane32_swap (one VALU instruction,
// no LDS round trip).  With both operands x, the swap returns r0 = (x[l] for l < 32, x[l-32]
// otherwise) and r1 = (x[l+32] for l < 32, x[l] otherwise); both halves then combine the same
// two values in the same order, so the results are bit-identical across the pair.
__device__ __forceinline__ float xor32_max(float x) {
  const unsigned u = __builtin_bit_cast(unsigned, x);
  const auto r = __builtin_amdgcn_permlane32_swap(u, u, false, false);
  return fmaxf(__builtin_bit_cast(float, (unsigned)r[0]), __builtin_bit_cast(float, (unsigned)r[1]));
}

__device__ __forceinline__ float xor32_add(float x) {
  const unsigned u = __builtin_bit_cast(unsigned, x);
  const auto r = __builtin_amdgcn_permlane32_swap(u, u, false, false);
  return __builtin_bit_cast(float, (unsigned)r[0]) + __builtin_bit_cast(float, (unsigned)r[1]);
}

// The block table is read-only for the whole kernel; reading it through the constant address
// space lets the compiler use scalar loads (counted by lgkmcnt, not vmcnt) for these uniform reads.
typedef const __attribute__((address_space(4))) int32_t* ConstI32Ptr;

__device__ __forceinline__ int clamp_page(int p, int num_pages) {
  return p < 0 ? 0 : (p >= num_pages ? num_pages - 1 : p);
}

// The online softmax lets the running maximum m of a row lag the true maximum by up to kMaxLag
// (log2 units): weights 2^(s c - m) then stay below 2^kMaxLag, which bf16 and the fp32 sums hold
// as precisely as weights below 1.  A lane's 32 weights of a prefill stage summing to at most
// kMaxWeightSum guarantees that bound without finding the stage's maximum.
constexpr float kMaxLag = 8.0f;
constexpr float kMaxWeightSum = 256.0f;             // 2^kMaxLag

// LDS of the attention kernel beyond its separate arrays.  NW = waves per workgroup; kinds as
// in attn_kernel.
template <int D, int NW, int kKinds> struct Lds {
  // prefill stages travel by LDS-DMA into six stage buffers (three K, three V): separate arrays
  // in prefill-only kernels, carved from the region of the decode stages in the mixed kernel
  static constexpr int prefill_bytes = (kKinds == 3) ? 6 * kKeysPerStage * D * 2 : 0;
  static constexpr int decode_stage_bytes = NW * 2 * (2 * kPage * D * 2);   // per-wave K+V double buffer
  static constexpr int merge_bytes = NW * 8 * D * 4 + 2 * NW * 8 * 4;
  // decode-only kernels keep their stages in separate arrays; the mixed kernel carves them here
  static constexpr int decode_bytes = (kKinds == 3) ? decode_stage_bytes : 0;
  static constexpr int bytes0 = prefill_bytes > decode_bytes ? prefill_bytes : decode_bytes;
  static constexpr int bytes = bytes0 > 16 ? bytes0 : 16;
};

// ------------------------------------------------------------------------------------------------
// Planner: one workgroup validates the device-resident lengths against the host bounds and
// builds the work list (prefill q-tiles, then decode page-range splits), so no host sync is
// needed.  Writes the header, per-sequence records and entries; zeroes the work counter.
//
// Prefill tiles are split along the keys when the launch holds at most one tile item per compute
// unit and its longest tile would outlast the average work per unit.  Work is estimated in
// key-units: a prefill tile key (256 q-rows on MFMA) costs about 3/2 of a decode key (one K/V row
// read from HBM).  A split covers kKeysPerStage-aligned key ranges [s S, (s+1) S) of the tile,
// the last one running to the tile's end; splits start at or before the first key that only
// some rows of the tile see (key ctx + t0 + 1), so every row sees at least one key of every
// split.  S is at least kMinSplitKeys and at least the tile keys per unit, which keeps the split
// items of a launch under 2 * kPlanComputeUnits (the partial-slot capacity).
//
// Decode splits hold pps pages each (the last one of a sequence the rest): pps is sized from the
// launch's actual pages (about kDecItemsPerCU items per compute unit) but never below the host's
// bound, so the workspace always holds the splits.  They are ordered longest first: every full
// split, then the shorter last splits in kPartBuckets size classes, largest class first, so the
// last items a launch hands out are its shortest ones.
// ------------------------------------------------------------------------------------------------
constexpr int kPlanThreads = 256;
constexpr int kPartBuckets = 16;

// Size class of a short last split of `rest` pages (1 <= rest < pps); class 0 holds the longest.
// inv_pps = kPartBuckets / pps; the class only orders work, so rounding at a class edge is harmless.
__device__ __forceinline__ int part_bucket(int rest, float inv_pps) {
  return kPartBuckets - 1 - min(kPartBuckets - 1, (int)((float)(rest - 1) * inv_pps));
}

// Size class of an unsplit prefill tile whose first row sees `keys` keys (at most max_full;
// inv_keys = kPartBuckets / (max_full + 1)): the longest tiles are class 0.
__device__ __forceinline__ int tile_class(int keys, float inv_keys) {
  return kPartBuckets - 1 - min(kPartBuckets - 1, (int)((float)keys * inv_keys));
}

__device__ __forceinline__ int tile_splits(int ctx, int t0, int split_keys) {
  return split_keys > 0 ? (ctx + t0 + split_keys) / split_keys : 1;   // ceil((ctx + t0 + 1) / S)
}

__global__ __launch_bounds__(kPlanThreads) void plan_kernel(
    PlanParams p, const int32_t* __restrict__ ctx_lens, const int32_t* __restrict__ cu,
    int32_t* __restrict__ hdr, SeqInfo* __restrict__ seqinfo, int32_t* __restrict__ split_base,
    int2* __restrict__ entries, int4* __restrict__ pre_jobs) {
  __shared__ int s_err, s_tiles, s_max_full, s_split_keys, s_pre_first;
  __shared__ unsigned long long s_pre_keys, s_dec_keys;
  __shared__ int s_wave[4][kPlanThreads / 64];
  __shared__ int s_carry[4];
  __shared__ int s_n_full;                     // full decode splits of the launch
  __shared__ int s_pps;                        // pages per decode split
  __shared__ unsigned long long s_dec_pages;
  __shared__ int s_part_cnt[kPartBuckets];     // short last splits per size class, then fill counts
  __shared__ int s_part_off[kPartBuckets];     // first position of each size class after the full splits
  __shared__ int s_tile_cnt[kPartBuckets];     // unsplit prefill tiles per size class, then fill counts
  __shared__ int s_tile_off[kPartBuckets];     // first prefill entry of each size class
  const int tid = threadIdx.x;
  const int T = p.tokens_per_tile;
  if (tid == 0) {
    s_err = 0; s_tiles = 0; s_max_full = 0; s_pre_keys = 0; s_dec_keys = 0; s_n_full = 0; s_dec_pages = 0;
    s_carry[0] = s_carry[1] = s_carry[2] = s_carry[3] = 0;
  }
  if (tid < kPartBuckets) { s_part_cnt[tid] = 0; s_tile_cnt[tid] = 0; }
  if (tid < kHdrWords - kHdrZero) hdr[kHdrZero + tid] = 0;   // zero block read by decode items
  if (tid < kNumXcd) hdr[kHdrQueues + tid] = 0;
  __syncthreads();
  // pass 1: validate every sequence and total the work
  // sequence tid's lengths (first chunk), kept for the later passes
  int my_pages = 0, my_q_start = 0, my_q_len = 0, my_ctx = 0;
  {
    int tiles = 0, max_full = 0;
    unsigned long long pre_keys = 0, dec_keys = 0, dec_pages = 0;
    for (int b = tid; b < p.batch; b += kPlanThreads) {
      const int q_start = cu ? cu[b] : b;
      const int q_len = cu ? cu[b + 1] - q_start : 1;
      const int ctx = ctx_lens[b];
      if (b == tid) {
        my_q_start = q_start;
        my_q_len = q_len;
        my_ctx = ctx;
      }
      const long long kv = (long long)ctx + q_len;
      bool bad = q_len < 0 || ctx < 0 || q_start < 0 || q_len > p.max_q_len ||
                 (long long)q_start + q_len > p.total_q || kv > p.max_kv_len ||
                 (kv + kPage - 1) / kPage > p.bt_stride;
      if (p.mode == kModeDecode && q_len != 1) bad = true;
      if (bad) { atomicOr(&s_err, 1); continue; }
      if (q_len <= 0) continue;
      if (p.mode == kModeDecode || (p.mode == kModeMixed && q_len == 1)) {
        dec_keys += (unsigned long long)kv;
        const int pages = (int)((kv + kPage - 1) / kPage);
        dec_pages += (unsigned long long)pages;
        if (b == tid) my_pages = pages;
      } else {
        const int nt = (q_len + T - 1) / T;
        tiles += nt;
        // keys seen by every row of tile t: ctx + t T + 1
        pre_keys += (unsigned long long)nt * (ctx + 1) + (unsigned long long)T * nt * (nt - 1) / 2;
        max_full = max(max_full, ctx + (nt - 1) * T + 1);
      }
    }
    if (tiles) atomicAdd(&s_tiles, tiles);
    if (dec_pages) atomicAdd(&s_dec_pages, dec_pages);
    if (max_full) atomicMax(&s_max_full, max_full);
    if (pre_keys) atomicAdd(&s_pre_keys, pre_keys);
    if (dec_keys) atomicAdd(&s_dec_keys, dec_keys);
  }
  __syncthreads();
  if (s_err) {
    if (tid == 0) {
      hdr[kHdrCounter] = 0; hdr[kHdrNumPre] = 0; hdr[kHdrNumDec] = 0;
      hdr[kHdrError] = 1; hdr[kHdrNumItems] = 0; hdr[kHdrPreSplitKeys] = 0; hdr[kHdrNumPreJobs] = 0;
      hdr[kHdrPagesPerSplit] = p.pages_per_split;
    }
    return;
  }
  if (tid == 0) {
    long long S = 0;
    const long long H = p.num_kv_heads;
    if (p.pre_slots > 0 && s_tiles > 0 && (long long)s_tiles * H <= kPlanComputeUnits) {
      const long long pre_units = (long long)s_pre_keys * H;
      const long long work = pre_units + pre_units / 2 + (long long)s_dec_keys * H;
      const long long per_cu = (work + kPlanComputeUnits - 1) / kPlanComputeUnits;
      S = max((long long)kMinSplitKeys, (pre_units + kPlanComputeUnits - 1) / kPlanComputeUnits);
      S = max(S, (2 * per_cu + 2) / 3);
      S = (S + kKeysPerStage - 1) / kKeysPerStage * kKeysPerStage;
      if (S >= s_max_full) S = 0;            // no tile would split
    }
    s_split_keys = (int)S;
    // Mixed launches: how many workgroups take prefill items first (the others take decode items
    // first): 1.2 x prefill's share of the estimated work, in prefill and decode key-units
    // weighted 3 : 2 as above.  A prefill tile left for the end of a launch holds one workgroup
    // far longer than a decode split, so prefill gets more than its share.
    int pre_first = 0;
    if (p.mixed_grid > 0) {
      const long long pu = 3LL * (long long)s_pre_keys * H;
      const long long du = 2LL * (long long)s_dec_keys * H;
      pre_first = pu + du > 0 ? (int)min((long long)p.mixed_grid, (6LL * p.mixed_grid * pu) / (5 * (pu + du)))
                              : p.mixed_grid;
    }
    s_pre_first = pre_first;
    // Decode split size: about kDecItemsPerCU items per compute unit over the launch's actual
    // pages, a multiple of 16 pages, at least the host's bound and at most kMaxPagesPerSplit.
    // Splits of at least kDecLongSplitPages pages (16 pages per wave) while that still leaves
    // 2 items per compute unit: a wave's first page of an item waits unhidden, so short splits
    // pay it often.
    long long pps = p.pages_per_split;
    if (s_dec_pages > 0) {
      const long long units = (long long)s_dec_pages * H;
      const long long per = (long long)kPlanComputeUnits * kDecItemsPerCU;
      const long long want = (units + per - 1) / per;
      const long long two = (units + 2LL * kPlanComputeUnits - 1) / (2LL * kPlanComputeUnits);
      pps = max(pps, (want + 15) / 16 * 16);
      pps = max(pps, min((long long)kDecLongSplitPages, (two + 15) / 16 * 16));
      pps = min(pps, (long long)max(p.pages_per_split, kMaxPagesPerSplit));
    }
    s_pps = (int)pps;
  }
  __syncthreads();
  const int pps = s_pps;
  const float inv_pps = (float)kPartBuckets / (float)pps;
  const int S = s_split_keys;
  const float inv_keys = (float)kPartBuckets / (float)(s_max_full + 1);
  // pass 1b: full decode splits and the size classes of the short last splits; without key
  // splits, the size classes of the prefill tiles too
  {
    int n_full = 0;
    for (int b = tid; b < p.batch; b += kPlanThreads) {
      int pages = my_pages, q_len = my_q_len, ctx = my_ctx;
      bool dec = pages > 0;
      if (b != tid) {
        const int q_start = cu ? cu[b] : b;
        q_len = cu ? cu[b + 1] - q_start : 1;
        ctx = ctx_lens[b];
        dec = p.mode == kModeDecode || (p.mode == kModeMixed && q_len == 1);
        pages = dec ? (ctx + q_len + kPage - 1) / kPage : 0;
      }
      if (pages > 0) {
        const int rest = pages % pps;
        n_full += pages / pps;
        if (rest) atomicAdd(&s_part_cnt[part_bucket(rest, inv_pps)], 1);
      } else if (!dec && q_len > 0 && S == 0) {
        const int nt = (q_len + T - 1) / T;
        for (int t = 0; t < nt; ++t) atomicAdd(&s_tile_cnt[tile_class(ctx + t * T + 1, inv_keys)], 1);
      }
    }
    if (n_full) atomicAdd(&s_n_full, n_full);
  }
  __syncthreads();
  if (tid < kPartBuckets) {                   // size classes, largest first (decode: after the full splits)
    int off = s_n_full, toff = 0;
    for (int k = 0; k < tid; ++k) { off += s_part_cnt[k]; toff += s_tile_cnt[k]; }
    s_part_off[tid] = off;
    s_tile_off[tid] = toff;
  }
  __syncthreads();
  if (tid < kPartBuckets) { s_part_cnt[tid] = 0; s_tile_cnt[tid] = 0; }   // now the fill counts
  __syncthreads();
  // pass 2: per-sequence counts (prefill entries, decode splits, split tiles, full decode splits),
  // block-wide exclusive scans, then the entries: prefill tiles longest first (unsplit tiles by
  // size class across the launch; key-split tiles per sequence, last tile first, splits in
  // order); decode splits longest first (full splits, then size classes)
  for (int base = 0; base < p.batch; base += kPlanThreads) {
    const int b = base + tid;
    int cnt[4] = {0, 0, 0, 0};              // prefill entries, decode splits, split tiles, full decode splits
    int kind = kSeqNone, q_start = 0, q_len = 0, ctx = 0, nt = 0, rest = 0;
    if (b < p.batch) {
      q_start = base == 0 ? my_q_start : (cu ? cu[b] : b);
      q_len = base == 0 ? my_q_len : (cu ? cu[b + 1] - q_start : 1);
      ctx = base == 0 ? my_ctx : ctx_lens[b];
      if (q_len > 0) {
        const bool dec = p.mode == kModeDecode || (p.mode == kModeMixed && q_len == 1);
        if (dec) {
          const int pages = (ctx + q_len + kPage - 1) / kPage;
          kind = kSeqDecode;
          cnt[1] = (pages + pps - 1) / pps;
          cnt[3] = pages / pps;
          rest = pages - cnt[3] * pps;
        } else {
          kind = kSeqPrefill;
          nt = (q_len + T - 1) / T;
          for (int t = 0; t < nt; ++t) {
            const int ns = tile_splits(ctx, t * T, S);
            cnt[0] += ns;
            cnt[2] += ns > 1;
          }
        }
      }
    }
    // exclusive scan: wave-level inclusive scans by shuffles, then the totals of earlier waves
    const int lane = tid & 63, wv = tid >> 6;
    int incl[4] = {cnt[0], cnt[1], cnt[2], cnt[3]};
#pragma unroll
    for (int off = 1; off < 64; off <<= 1) {
#pragma unroll
      for (int c = 0; c < 4; ++c) {
        const int v = __shfl_up(incl[c], off);
        if (lane >= off) incl[c] += v;
      }
    }
    if (lane == 63) {
#pragma unroll
      for (int c = 0; c < 4; ++c) s_wave[c][wv] = incl[c];
    }
    __syncthreads();
    int excl[4];
#pragma unroll
    for (int c = 0; c < 4; ++c) {
      int before = s_carry[c];
      for (int k = 0; k < wv; ++k) before += s_wave[c][k];
      excl[c] = before + incl[c] - cnt[c];
    }
    if (b < p.batch) {
      seqinfo[b] = SeqInfo{q_start, q_len, ctx, kind | (cnt[1] << 4)};
      split_base[b] = excl[1];
      if (S == 0) {
        // unsplit tiles go longest first across the whole launch (by size class), so the last
        // tiles the persistent grid hands out are short ones from any sequence.  A sequence's
        // tiles of one class (a run of consecutive tiles) are claimed together and stay
        // adjacent, so the tiles that read the same K/V still run at about the same time.
        for (int t = nt - 1; t >= 0;) {
          const int k = tile_class(ctx + t * T + 1, inv_keys);
          int t_end = t;
          while (t_end > 0 && tile_class(ctx + (t_end - 1) * T + 1, inv_keys) == k) --t_end;
          int pos = s_tile_off[k] + atomicAdd(&s_tile_cnt[k], t - t_end + 1);
          for (; t >= t_end; --t, ++pos)
            if (pos < p.max_pre) entries[pos] = make_int2(b, t);
        }
      } else {
        // key-split tiles: each tile's splits stay contiguous (their partial slots follow the
        // entry index), last tile of the sequence first
        int e = excl[0], j = excl[2];
        for (int t = nt - 1; t >= 0; --t) {
          const int ns = tile_splits(ctx, t * T, S);
          if (ns > 1 && j < p.pre_jobs_cap) pre_jobs[j++] = make_int4(b, t, e, ns);
          for (int sp = 0; sp < ns; ++sp, ++e)
            if (e < p.max_pre) entries[e] = make_int2(b, t | (sp << 16));
        }
      }
      // full splits in sequence order; the short last split at its size class's next position
      // (claimed before the loop, so the wave issues the atomic once)
      int part_pos = 0;
      if (rest) {
        const int k = part_bucket(rest, inv_pps);
        part_pos = s_part_off[k] + atomicAdd(&s_part_cnt[k], 1);
      }
      for (int sp = 0; sp < cnt[1]; ++sp) {
        const int pos = sp < cnt[3] ? excl[3] + sp : part_pos;
        if (pos < p.max_dec) entries[p.max_pre + pos] = make_int2(b, sp);
      }
    }
    __syncthreads();
    if (tid == kPlanThreads - 1) {
#pragma unroll
      for (int c = 0; c < 4; ++c) s_carry[c] = excl[c] + cnt[c];
    }
    __syncthreads();
  }
  if (tid == 0) {
    const int n_pre = s_carry[0], n_dec = s_carry[1], n_jobs = s_carry[2];
    const bool over = n_pre > p.max_pre || n_dec > p.max_dec || n_jobs > p.pre_jobs_cap ||
                      (n_jobs > 0 && (long long)n_pre * p.num_kv_heads > p.pre_slots);
    hdr[kHdrCounter] = 0;
    hdr[kHdrPreFirstWG] = s_pre_first;
    hdr[kHdrNumPre] = over ? 0 : n_pre;
    hdr[kHdrNumDec] = over ? 0 : n_dec;
    hdr[kHdrError] = over ? 2 : 0;
    hdr[kHdrNumItems] = over ? 0 : (n_pre + n_dec) * p.num_kv_heads;
    hdr[kHdrPreSplitKeys] = S;
    hdr[kHdrNumPreJobs] = over ? 0 : n_jobs;
    hdr[kHdrPagesPerSplit] = pps;
  }
}

// 16 bytes per lane from global memory straight into LDS (lane l writes lds_base + 16 l), issued
// as inline assembly, which the compiler does not track: it then inserts no waits of its own for
// it (it would wait for every copy in flight before any LDS read), and the caller waits with
// explicit vmcnt counts.  The compiler's own vmcnt waits stay correct, because copies it does
// not know about can only make them wait longer.  The LDS base goes through M0, which the
// sequence saves and restores (the copy reads it at issue, one wait state after it is written).
// lds_base must be uniform across the wave.  kOnce: the load is marked non-temporal (nt), for
// bytes read once per launch.
template <bool kOnce = false>
__device__ __forceinline__ void lds_dma16_untracked(const void* g, const char* lds_base) {
  const unsigned lds = __builtin_amdgcn_readfirstlane((unsigned)(uintptr_t)((LDS_AS const char*)lds_base));
  unsigned saved;
  if constexpr (kOnce) {
    __asm__ volatile(
        "s_mov_b32 %0, m0\n\t"
        "s_mov_b32 m0, %2\n\t"
        "s_nop 0\n\t"
        "global_load_lds_dwordx4 %1, off nt\n\t"
        "s_mov_b32 m0, %0"
        : "=&s"(saved)
        : "v"(g), "s"(lds)
        : "memory");
  } else {
    __asm__ volatile(
        "s_mov_b32 %0, m0\n\t"
        "s_mov_b32 m0, %2\n\t"
        "s_nop 0\n\t"
        "global_load_lds_dwordx4 %1, off\n\t"
        "s_mov_b32 m0, %0"
        : "=&s"(saved)
        : "v"(g), "s"(lds)
        : "memory");
  }
}

// vmcnt(n) with the other counters left alone (gfx9 encoding: vmcnt in bits 3:0 and 15:14)
#define PEARL_VMCNT(n) (((n) & 15) | (((n) >> 4) << 14) | 0x0F70)
// lgkmcnt(0) with the other counters left alone
#define PEARL_LGKMCNT0 0xC07F

// A prefill stage staged by LDS-DMA: kKeysPerStage key rows of D bf16, unpadded.  The 16-byte
// chunk q of row r sits in slot q ^ swz(r), which keeps both operand read patterns free of bank
// conflicts on the 64 banks of 4 bytes: the row reads of the Q.K products (16 lanes read one chunk
// of 16 consecutive rows: swz is a permutation of the 16 rows' slots) and the transposing reads of
// the P.V products (32 lanes read 4 adjacent chunks of 4 consecutive rows: swz moves each of the 4
// rows to its own quarter of the 256 bank bytes).  Wave w copies rows [RPW w, RPW w + RPW) of the
// stage, RPI rows per 64-lane DMA instruction.
template <int D, int KEYS = kKeysPerStage> struct DmaTile {
  static_assert(D == 64 || D == 128, "head_dim");
  static constexpr int CPR = D / 8;                 // 16-byte chunks per row
  static constexpr int RB = D * 2;                  // bytes per row
  static constexpr int BYTES = KEYS * RB;
  static constexpr int RPI = 64 / CPR;              // rows per DMA instruction
  static constexpr int RPW = KEYS / kWaves;         // rows copied per wave
  static constexpr int NDMA = RPW / RPI;            // DMA instructions per wave and tensor
  static_assert(NDMA >= 1 && NDMA * RPI == RPW && kPage % RPW == 0, "DMA split");
  __device__ static __forceinline__ int swz(int r) {
    // d = 128: a row is all 64 banks, rows 4i..4i+3 get slot offsets 0, 4, 8, 12 (+ i);
    // d = 64: two rows share the banks, rows 4i..4i+3 get offsets 0, 0, 4, 4 (+ i)
    if constexpr (D == 128) return ((r & 3) << 2) | ((r >> 2) & 3);
    else return (((r >> 1) & 1) << 2) | ((r >> 2) & 3);
  }
};

// ------------------------------------------------------------------------------------------------
// Prefill-append work item: one (sequence, kv-head g, q-tile).  The tile holds 256 q-rows =
// tokens_per_tile tokens x G heads of the group (row rho -> token rho / G, head rho % G), so every
// staged K/V byte is shared by the whole group.  Wave w owns rows [32w, 32w+32).
//   S^T (keys x rows) = K . Q^T     (32x32x16 MFMA: A = K tile from LDS, B = Q^T in registers)
//   O^T (dims x rows) += V^T . P^T  (A = V^T via LDS transpose reads, B = P^T from S^T registers)
// Each lane owns one q-row (l%32) for both products, so the softmax row statistics are
// lane-local apart from one exchange with lane l^32, which holds the row's other keys.
// A split item (entry e, code = tile | split << 16) covers only its key range and writes the
// unnormalised (o~, m, l) of its rows to partial slot e * H_kv + g for the prefill merge.
//
// Schedule (prefill-only and mixed kernels): the matrix and vector work of the two waves on each
// SIMD overlap.  The 8 waves form two groups, waves 0-3 and waves 4-7 (the waves w and w + 4 share
// a SIMD), and the item runs in phases separated by workgroup barriers.  In each of its phases a
// wave does either
//   M(j): S(j) = K(j) Q^T and O += V(j-1)^T P(j-1)   (32 MFMAs at d = 128, no dependence between
//         the two products), or
//   V(j): the online softmax of S(j), giving P(j)    (exp, scale and sums on the vector ALU),
// alternating M(0) V(0) M(1) V(1) ... M(n); group B runs one phase behind group A.  In every phase
// one wave of each SIMD therefore issues MFMAs while the other runs its softmax, so the matrix core
// works through the vector phase of the other wave instead of waiting for it.
// Stages travel by LDS-DMA into three DmaTile buffers per tensor: K(j) into K buffer j % 3, V(j)
// into V buffer j % 3.  K(j) is
// read in phases 2j and 2j+1, V(j) in phases 2j+2 and 2j+3.  Each wave copies its rows of K(j+2)
// and V(j+1) (the pair j) in phases 2j and 2j+1, into buffers last read in phase 2j-1: half of the
// DMA instructions right after its MFMAs of M(j), the other half at the start of its adjacent
// softmax phase.  A DMA instruction holds its wave for tens of cycles before it is accepted, and
// longer when many queue at the compute unit at once: issued all together at a phase start they
// stalled every wave for hundreds of cycles; after the MFMAs they overlap the draining matrix
// pipeline, and at the start of a softmax phase they use the slack that phase has over an M phase.
// Before the barrier that ends phase 2j-1 every wave waits for its own copies of K(j) and V(j-1)
// (the copies issued since stay in flight).
// ------------------------------------------------------------------------------------------------
template <int D>
__device__ __forceinline__ void prefill_tile_pp(const AttnArgs& a, int e, int b, int code, int g, int split_keys,
                                                char* kb0, char* vb0) {
  constexpr int KB = D / 16;                        // 16-wide k blocks of the QK product
  constexpr int MB = D / 32;                        // 32-wide dim blocks of the PV product
  constexpr int SK = kKeysPerStage;                 // keys per stage
  constexpr int NST = SK / 32;                      // 32-key sub-tiles per stage
  static_assert(kKeysPerStage % SK == 0, "key splits stay stage-aligned");
  using DT = DmaTile<D, SK>;
  constexpr int RB = DT::RB;
  // buffer r of each tensor (r = stage % 3 is a compile-time constant wherever a buffer is used, so
  // every LDS address is a per-lane offset plus an immediate)
  auto kbuf = [&](int r) { return kb0 + r * DT::BYTES; };
  auto vbuf = [&](int r) { return vb0 + r * DT::BYTES; };

  const int lane = threadIdx.x & 63, half = lane >> 5;
  const int w = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);   // wave index (uniform)
  const int grp = w >> 2;                           // 0: waves 0-3, 1: waves 4-7 (one phase later)
  const SeqInfo si = a.seqinfo[b];
  const int G = a.group;
  const int tile = code & 0xffff, split = code >> 16;
  const int t0 = tile * a.tokens_per_tile;
  const int t_end = min(t0 + a.tokens_per_tile, si.q_len);
  const int ctx = si.ctx_len;
  const int kv_needed = ctx + t_end;
  const int rho = 32 * w + (lane & 31);
  const int tok = t0 + rho / G;
  const int hh = rho - (rho / G) * G;
  const int h = g * G + hh;
  const bool row_ok = tok < t_end;
  const int row_limit = ctx + tok;                  // last visible key of this row
  const int wave_min_limit = ctx + t0 + (32 * w) / G;
  const int H_q = a.num_q_heads, H_kv = a.num_kv_heads;
  const size_t head_stride = (size_t)kPage * D;     // elements per (page, kv-head) block
  const float c = a.scale_log2;

  bf16x8 qop[KB];
  {
    const uint16_t* qrow = a.q + ((size_t)(si.q_start + (row_ok ? tok : t0)) * H_q + h) * D + 8 * half;
#pragma unroll
    for (int kb = 0; kb < KB; ++kb) qop[kb] = row_ok ? as_bf16x8(ld16(qrow + 16 * kb)) : zero_bf16x8();
  }
  f32x16 oacc[MB];
#pragma unroll
  for (int mb = 0; mb < MB; ++mb)
#pragma unroll
    for (int r = 0; r < 16; ++r) oacc[mb][r] = 0.f;
  float m_run = -INFINITY, l_run = 0.f;

  const int n_steps = (kv_needed + SK - 1) / SK;
  const int n_split = tile_splits(ctx, t0, split_keys);
  const int step_begin = split * (split_keys / SK);
  const int step_end = split + 1 < n_split ? step_begin + split_keys / SK : n_steps;
  const int n = step_end - step_begin;              // stages of this item (>= 1)

  const ConstI32Ptr bt_c = (ConstI32Ptr)(a.block_table + (size_t)b * a.bt_stride);
  const int last_pidx = (kv_needed - 1) / kPage;
  const int gi = lane >> 4, jl = lane & 15;
  const int krow = 4 * (gi >> 1) + (jl >> 2);
  const int dcol = 16 * (gi & 1) + 4 * (jl & 3);
  int koff[KB], voff[2][MB], goff[DT::NDMA];
#pragma unroll
  for (int kb = 0; kb < KB; ++kb) koff[kb] = (lane & 31) * RB + (((2 * kb + half) ^ DT::swz(lane & 15)) << 4);
#pragma unroll
  for (int sec = 0; sec < 2; ++sec)
#pragma unroll
    for (int mb = 0; mb < MB; ++mb) {
      const int r = krow + 8 * sec;
      voff[sec][mb] = r * RB + ((((32 * mb + dcol) >> 3) ^ DT::swz(r)) << 4) + (jl & 1) * 8;
    }
#pragma unroll
  for (int i = 0; i < DT::NDMA; ++i) {
    const int r = DT::RPW * w + DT::RPI * i + lane / DT::CPR;
    goff[i] = (r % kPage) * RB + (((lane % DT::CPR) ^ DT::swz(r)) << 4);
  }
  // this wave's rows of the K (or V) tile of local stage j, by LDS-DMA; V rows past the last
  // needed key come from the workspace's zero block (K rows there are always masked)
  const char* zero_src = reinterpret_cast<const char*>(a.ws_hdr + kHdrZero);
  // block-table entry of this wave's rows of local stage j (a scalar load; clamped where used)
  auto page_of = [&](int j) {
    const int pidx = min(((step_begin + j) * SK + DT::RPW * w) / kPage, last_pidx);
    return bt_c[pidx];
  };
  // DMA instruction i of this wave's rows of local stage j
  auto dma_one = [&](int j, bool is_v, int entry, char* dst, int i) {
    const int step = step_begin + j;
    const int page = clamp_page(entry, a.num_pages);
    const size_t base = (((size_t)page * H_kv + g) * head_stride) * 2;
    const char* src = reinterpret_cast<const char*>(is_v ? a.v_pool : a.k_pool) + base;
    const int key = step * SK + DT::RPW * w + DT::RPI * i + lane / DT::CPR;
    const int row0 = DT::RPW * w + DT::RPI * i;
    lds_dma16_untracked(is_v && key >= kv_needed ? zero_src : src + goff[i], dst + row0 * RB);
  };
  auto dma = [&](int j, bool is_v, int entry, char* dst) {
#pragma unroll
    for (int i = 0; i < DT::NDMA; ++i) dma_one(j, is_v, entry, dst, i);
  };

  // block-table entries of the next copies: pid_k for K rows, pid_v for V rows (pid_n: the K
  // rows after those, read ahead by group B)
  int pid_v = 1 < n ? page_of(1) : 0, pid_k = 2 < n ? page_of(2) : 0, pid_n = 0;

  f32x16 s[NST];                                    // S^T of the stage between its M and V phases
  bf16x8 pop[NST][2];                               // P^T of the stage between its V and next M phases
  const f32x16 zero16 = {0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f};
#pragma unroll
  for (int st = 0; st < NST; ++st) s[st] = zero16;
#pragma unroll
  for (int st = 0; st < NST; ++st)
#pragma unroll
    for (int kk = 0; kk < 2; ++kk) pop[st][kk] = zero_bf16x8();

  // M(j): PV of stage j - 1 (if any), then QK of stage j (if any).  P(j - 1) dies before S(j) is
  // born, so the two share registers.  The phase is one wave's stream of MFMAs while the other
  // wave of its SIMD runs a softmax, so nothing else hides its LDS latency: the operands are read
  // kLead MFMAs ahead through a small ring, and a scheduling barrier after each step keeps that
  // order (the compiler would otherwise read each operand just before its MFMA).
  constexpr int NPV = 2 * NST * MB, NQK = NST * KB, kLead = 3;
  auto operand = [&](int i, const char* kb_, const char* vb_) -> bf16x8 {
    if (i < NPV) {                                  // V^T of (dim block, sub-tile, 16-key half)
      const int mb = i / (2 * NST), st = (i >> 1) % NST, kk = i & 1;
      const int vo = (32 * st + 16 * kk) * RB;
      return concat_tr(lds_read_tr(vb_, vo + voff[0][mb]), lds_read_tr(vb_, vo + voff[1][mb]));
    }
    const int q = i - NPV, st = q / KB, kb = q - (q / KB) * KB;   // K rows of (sub-tile, k block)
    return *reinterpret_cast<const bf16x8*>(kb_ + 32 * st * RB + koff[kb]);
  };
  auto mfma_slot = [&](int i, const bf16x8& op) {
    if (i < NPV) {
      const int mb = i / (2 * NST), st = (i >> 1) % NST, kk = i & 1;
      oacc[mb] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(op, pop[st][kk], oacc[mb], 0, 0, 0);
    } else {
      const int q = i - NPV, st = q / KB, kb = q - (q / KB) * KB;
      s[st] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(op, qop[kb], kb == 0 ? zero16 : s[st], 0, 0, 0);
    }
  };
  constexpr int NM = NPV + NQK;
  // One instruction stream for every M phase (no joins of differently allocated copies): M(0)
  // adds P = 0 times a zero-filled V buffer 2, and M(n) computes an S that no V phase reads.
  // R = j % 3: K(j) sits in K buffer R and V(j - 1) in V buffer (R + 2) % 3.
  // The first kLead operands (V^T reads) of an M phase are read at the end of the softmax phase
  // before it, so that their latency passes while the wave waits at the barrier.
  bf16x8 ring[kLead];
  auto prefetch = [&](auto r_c) {
    constexpr int R = decltype(r_c)::value;
#pragma unroll
    for (int d = 0; d < kLead; ++d) ring[d] = operand(d, kbuf(R), vbuf((R + 2) % 3));
  };
  auto phase_m = [&](auto r_c, bool prefetched) {
    constexpr int R = decltype(r_c)::value;
    const char* kb_ = kbuf(R);
    const char* vb_ = vbuf((R + 2) % 3);
    if (!prefetched) prefetch(r_c);
#pragma unroll
    for (int i = 0; i < NM; ++i) {
      const bf16x8 op = ring[i % kLead];
      if (i + kLead < NM) ring[i % kLead] = operand(i + kLead, kb_, vb_);
      mfma_slot(i, op);
      __builtin_amdgcn_sched_barrier(0);
    }
  };
  // The copies of stage j's pair: K(j + 2) into K buffer (R + 2) % 3 and V(j + 1) into V buffer
  // (R + 1) % 3 (R = j % 3).
  auto copy_k = [&](auto r_c, int j) {
    constexpr int R = decltype(r_c)::value;
#pragma unroll
    for (int i = 0; i < DT::NDMA; ++i)
      if (j + 2 < n) dma_one(j + 2, false, pid_k, kbuf((R + 2) % 3), i);
  };
  auto copy_v = [&](auto r_c, int j) {
    constexpr int R = decltype(r_c)::value;
#pragma unroll
    for (int i = 0; i < DT::NDMA; ++i)
      if (j + 1 < n) dma_one(j + 1, true, pid_v, vbuf((R + 1) % 3), i);
  };
  // V(j), 0 <= j < n: causal mask (only on stages that reach past some row's last visible key; the
  // empty asm keeps that a real branch), then the online softmax (base 2).  The weights are first
  // taken against the running maximum m without looking for this stage's maximum; that is exact
  // (any m gives the same softmax) as long as no weight exceeds 2^kMaxLag, which the lane's sum of
  // its 32 weights bounds.  Otherwise (the first stage of an item, where m is still -inf, or
  // scores jumping more than kMaxLag above m) the stage is redone with the row maximum, and m
  // moves to it only when it exceeds m by more than kMaxLag, so the O rescale is rare too.  A NaN
  // sum (a masked key against m = -inf) also takes the redo.
  auto phase_v = [&](int j) {
    const int k0 = (step_begin + j) * SK;
    if (k0 + SK - 1 > wave_min_limit) {
      __asm__ volatile("" ::);
#pragma unroll
      for (int st = 0; st < NST; ++st)
#pragma unroll
        for (int r = 0; r < 16; ++r) {
          const int key = k0 + 32 * st + (r & 3) + 8 * (r >> 2) + 4 * half;
          if (key > row_limit) s[st][r] = -INFINITY;
        }
    }
    float ps0 = 0.f, ps1 = 0.f;
#pragma unroll
    for (int st = 0; st < NST; ++st)
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const float pv = fexp2(__builtin_fmaf(s[st][r], c, -m_run));
        if (r & 1) ps1 += pv; else ps0 += pv;
        pop[st][r >> 3][r & 7] = (__bf16)pv;
      }
    float psum = ps0 + ps1;
    if (__ballot(!(psum <= kMaxWeightSum))) {
      __asm__ volatile("" ::);
      float mx = s[0][0];
#pragma unroll
      for (int r = 1; r < 16; ++r) mx = fmaxf(mx, s[0][r]);
#pragma unroll
      for (int st = 1; st < NST; ++st)
#pragma unroll
        for (int r = 0; r < 16; ++r) mx = fmaxf(mx, s[st][r]);
      mx = xor32_max(mx);
      const bool grow = mx * c > m_run + kMaxLag;
      const float m_new = grow ? mx * c : m_run;
      const float alpha = grow ? fexp2(m_run - m_new) : 1.0f;
      ps0 = ps1 = 0.f;
#pragma unroll
      for (int st = 0; st < NST; ++st)
#pragma unroll
        for (int r = 0; r < 16; ++r) {
          const float pv = fexp2(__builtin_fmaf(s[st][r], c, -m_new));
          if (r & 1) ps1 += pv; else ps0 += pv;
          pop[st][r >> 3][r & 7] = (__bf16)pv;
        }
      psum = ps0 + ps1;
      l_run *= alpha;
      if (__ballot(grow)) {
#pragma unroll
        for (int mb = 0; mb < MB; ++mb)
#pragma unroll
          for (int r = 0; r < 16; ++r) oacc[mb][r] *= alpha;
      }
      m_run = m_new;
    }
    l_run += psum;
  };
  // end of phase t: at t = 2i, wait for this wave's copies of V(i) and everything before it (K(i + 1)
  // among them), which M(i + 1) reads from phase 2i + 2 on and the softmax phase before it reads
  // ahead (the copy of K(i + 2), issued since, stays in flight); then drain the LDS reads and pass
  // the barrier without the release fence of __syncthreads (which would drain every copy)
  constexpr int P = DT::NDMA;                       // DMA instructions per tensor and stage
  auto end_phase = [&](int t) {
    if ((t & 1) == 0) {
      const int i = t >> 1;
      if (i + 2 < n) __builtin_amdgcn_s_waitcnt(PEARL_VMCNT(P));   // K(i + 2) stays in flight
      else __builtin_amdgcn_s_waitcnt(PEARL_VMCNT(0));
    }
    __builtin_amdgcn_s_waitcnt(PEARL_LGKMCNT0);
    __asm__ volatile("s_barrier" ::: "memory");
  };

  // prologue: K(0), V(0), K(1), and zeros into V buffer 2 (read by M(0), whose P is 0; V(2) is
  // copied there only with the pair 1); the first M phase needs K(0).  Block-table entries are
  // read in softmax phases, a phase or more before they are used: scalar loads share the LDS
  // reads' counter and complete out of order, so one in flight during an M phase would make
  // every operand wait drain the counter, and one used right away would stall the phase for a
  // memory round trip.  The end-of-phase drain completes them.
  {
    const int p0 = page_of(0);
    dma(0, false, p0, kbuf(0));
    dma(0, true, p0, vbuf(0));
  }
  if (1 < n) dma(1, false, pid_v, kbuf(1));
#pragma unroll
  for (int i = 0; i < DT::NDMA; ++i)
    lds_dma16_untracked(zero_src, vbuf(2) + (DT::RPW * w + DT::RPI * i) * RB);
  __builtin_amdgcn_s_waitcnt(PEARL_VMCNT(0));       // Q loads and the first copies (also this item's)
  __asm__ volatile("s_barrier" ::: "memory");
  using I0 = std::integral_constant<int, 0>;
  using I1 = std::integral_constant<int, 1>;
  using I2 = std::integral_constant<int, 2>;
  // Each group runs its own loop (the same barriers in the same number: 2n + 2), so the registers
  // of S and P are never live together on any path.  The loops are unrolled over the three buffers
  // and no phase is conditional inside them.
  if (grp == 0) {
    // phases 2j, 2j + 1 for j < n: M(j), V(j); then M(n) and an empty phase.  The K rows of the
    // pair follow the MFMAs of M(j), the V rows open V(j), and the block-table entry of the next K
    // rows is read during V(j).
    auto step = [&](auto r_c, int j, auto first_c) {
      constexpr int R = decltype(r_c)::value;
      phase_m(r_c, !decltype(first_c)::value);
      copy_k(r_c, j);
      end_phase(2 * j);
      copy_v(r_c, j);
      pid_v = pid_k;
      if (j + 3 < n) pid_k = page_of(j + 3);
      phase_v(j);
      prefetch(std::integral_constant<int, (R + 1) % 3>{});
      end_phase(2 * j + 1);
    };
    using F = std::false_type;
    step(I0{}, 0, std::true_type{});                // n >= 1
    int j = 1;
    for (; j + 3 <= n; j += 3) {
      step(I1{}, j, F{});
      step(I2{}, j + 1, F{});
      step(I0{}, j + 2, F{});
    }
    if (j < n) { step(I1{}, j, F{}); ++j; }
    if (j < n) { step(I2{}, j, F{}); ++j; }
    const int r = n % 3;                            // j == n
    if (r == 0) phase_m(I0{}, true); else if (r == 1) phase_m(I1{}, true); else phase_m(I2{}, true);
    end_phase(2 * n);
    end_phase(2 * n + 1);
  } else {
    // phases 0, 1: an empty phase, M(0); phases 2j, 2j + 1 for 1 <= j <= n: V(j - 1), M(j).  The
    // K rows of pair j open V(j - 1) (phase 0 for pair 0), the V rows follow the MFMAs of M(j),
    // and the block-table entry of the K rows after them is read during V(j - 1).
    auto pair_done = [&]() {
      pid_v = pid_k;
      pid_k = pid_n;
    };
    auto step = [&](auto r_c, int j) {
      copy_k(r_c, j);
      if (j + 3 < n) pid_n = page_of(j + 3);
      phase_v(j - 1);
      prefetch(r_c);
      end_phase(2 * j);
      phase_m(r_c, true);
      copy_v(r_c, j);
      pair_done();
      end_phase(2 * j + 1);
    };
    copy_k(I0{}, 0);
    if (3 < n) pid_n = page_of(3);
    end_phase(0);
    phase_m(I0{}, false);
    copy_v(I0{}, 0);
    pair_done();
    end_phase(1);
    int j = 1;
    for (; j + 3 <= n + 1; j += 3) {
      step(I1{}, j);
      step(I2{}, j + 1);
      step(I0{}, j + 2);
    }
    if (j <= n) { step(I1{}, j); ++j; }
    if (j <= n) { step(I2{}, j); ++j; }
  }

  // epilogue: combine the two half-row sums; a split item stores its fp32 partial state, a whole
  // item normalises and stores bf16 O and the fp32 LSE
  const float l_tot = xor32_add(l_run);
  if (row_ok && n_split > 1) {
    const size_t prow = (size_t)(e * H_kv + g) * kRowsPerTile + rho;
    float* po = a.part_pre_o + prow * D;
#pragma unroll
    for (int mb = 0; mb < MB; ++mb)
#pragma unroll
      for (int rq = 0; rq < 4; ++rq)
        *reinterpret_cast<f32x4*>(po + 32 * mb + 8 * rq + 4 * half) =
            f32x4{oacc[mb][4 * rq + 0], oacc[mb][4 * rq + 1], oacc[mb][4 * rq + 2], oacc[mb][4 * rq + 3]};
    if (half == 0) {
      a.part_pre_ml[2 * prow] = m_run;
      a.part_pre_ml[2 * prow + 1] = l_tot;
    }
  } else if (row_ok) {
    const float inv = 1.0f / l_tot;
    uint16_t* orow = a.out + ((size_t)(si.q_start + tok) * H_q + h) * D;
#pragma unroll
    for (int mb = 0; mb < MB; ++mb)
#pragma unroll
      for (int rq = 0; rq < 4; ++rq) {
        const int dim = 32 * mb + 8 * rq + 4 * half;
        u32x2 pk;
        pk[0] = (uint32_t)bf16_bits(oacc[mb][4 * rq + 0] * inv) | ((uint32_t)bf16_bits(oacc[mb][4 * rq + 1] * inv) << 16);
        pk[1] = (uint32_t)bf16_bits(oacc[mb][4 * rq + 2] * inv) | ((uint32_t)bf16_bits(oacc[mb][4 * rq + 3] * inv) << 16);
        *reinterpret_cast<u32x2*>(orow + dim) = pk;
      }
    if (half == 0 && a.lse) a.lse[(size_t)(si.q_start + tok) * H_q + h] = (m_run + flog2(l_tot)) * kLn2;
  }
}

// ------------------------------------------------------------------------------------------------
// Decode work item: one (sequence, kv-head g, split of pps pages; the planner chooses pps).  The
// G q-heads of the group are the 16 columns of the MFMA products (columns >= G are zero), so each
// K/V byte is loaded once for the whole group.  Wave w takes pages w, w+8, ... of the split:
//   S^T (16 keys x heads) = K_page . Q^T           (16x16x32 MFMA: A = K rows read from LDS)
//   O^T (dims x heads)   += V^T . P^T over 16 keys (16x16x16 MFMA: A = V^T read transposed from LDS)
// K and V travel HBM -> LDS by 16-byte LDS-DMA loads (no VGPRs, no LDS store instructions) into a
// per-wave double buffer, so the next page's loads are in flight while the current page is
// consumed.  Each DMA instruction moves whole key rows (1 KiB of consecutive bytes), marked
// non-temporal: every K/V byte is read once per launch, and such full-line reads marked that way
// reach a higher HBM rate than plain ones (K read straight into MFMA operand registers touched
// half of each 128-byte line per instruction, which the non-temporal mark made slower).  Every
// load is unconditional: addresses stay inside the split's own pages, and V rows of keys past the
// sequence end are fetched from a zeroed block of the workspace so they add nothing to P.V
// (their scores are masked to -inf).  The 8 waves' partial softmax states are merged through
// LDS; a sequence with one split writes its output directly, otherwise the (o~, m, l) partial
// goes to the workspace.
//
// Stage layout (per wave): the page's K rows, then its V rows, kPage rows x D/8 16-byte chunks
// each, unpadded.  Chunk c of K row r sits in slot c ^ kswz(r), so the 16 rows that one operand
// read covers fall in 16 different 16-byte bank groups; chunk c of V row r sits in slot
// c ^ vswz(r), which spreads the transposing reads over all LDS banks.
// ------------------------------------------------------------------------------------------------
template <int D> struct PageTile {
  static constexpr int CPR = D / 8;                 // 16-byte chunks per key row
  static constexpr int ROWB = D * 2;                // bytes per key row
  static constexpr int RPI = 64 / CPR;              // rows written by one 64-lane DMA instruction
  static constexpr int TBYTES = kPage * ROWB;       // one tensor of one page
  static constexpr int BYTES = 2 * TBYTES;          // K rows, then V rows
  static constexpr int NDMA = kPage / RPI;          // DMA instructions per tensor and page
  static constexpr int KB = D / 32;                 // 32-wide k blocks of the QK product
  static constexpr int MB = D / 16;                 // 16-wide dim blocks of the PV product
  __device__ static __forceinline__ int kswz(int r) {
    // d = 128: 16 slots per row, one per row of the page; d = 64: 8 slots per row and rows 2i,
    // 2i + 1 in opposite halves of the banks
    if constexpr (D == 128) return r & 15;
    else return (r >> 1) & 7;
  }
  __device__ static __forceinline__ int vswz(int r) {
    return (((r & 3) << 2) | (((r >> 2) & 1) << 1)) & (CPR - 1);
  }
  // byte offset of K row r, chunk c
  __device__ static __forceinline__ int koff(int r, int c) { return r * ROWB + ((c ^ kswz(r)) << 4); }
  // byte offset of (V row r, 4-element group starting at dim d0)
  __device__ static __forceinline__ int voff(int r, int d0) {
    return TBYTES + r * ROWB + (((d0 >> 3) ^ vswz(r)) << 4) + ((d0 >> 2) & 1) * 8;
  }
};


// The new token's K/V row of a fused append-and-decode: logical page `page`, slot `slot`, taken
// from the caller's k_new / v_new rows instead of the pool (page -1: none).
struct NewRow {
  int page, slot;
  const uint16_t* k;
  const uint16_t* v;
};

// Issues the copies of logical page p (physical page phys) of kv-head g into the stage at dst.
// kNew: the item may hold the new row (decode_kernel); otherwise nr is ignored.
template <int D, bool kNew>
__device__ __forceinline__ void decode_issue(const AttnArgs& a, int phys, int p, int g, int kv, char* dst,
                                             const NewRow& nr) {
  using PT = PageTile<D>;
  const int lane = threadIdx.x & 63;
  const size_t blk = ((size_t)phys * a.num_kv_heads + g) * (size_t)(kPage * D);
  const uint16_t* zero = reinterpret_cast<const uint16_t*>(a.ws_hdr + kHdrZero);
  const int slot = lane % PT::CPR;                  // chunk slot this lane fills
#pragma unroll
  for (int i = 0; i < PT::NDMA; ++i) {
    const int r = i * PT::RPI + lane / PT::CPR;     // key row of the page written by this lane
    const bool is_new = kNew && p == nr.page && r == nr.slot;
    const int ck = slot ^ PT::kswz(r);
    lds_dma16_untracked<true>(is_new ? nr.k + ck * 8 : a.k_pool + blk + r * D + ck * 8, dst + i * 1024);
  }
#pragma unroll
  for (int i = 0; i < PT::NDMA; ++i) {
    const int r = i * PT::RPI + lane / PT::CPR;
    const bool ok = p * kPage + r < kv;
    const bool is_new = kNew && p == nr.page && r == nr.slot;
    const int cv = slot ^ PT::vswz(r);
    const uint16_t* src = ok ? (is_new ? nr.v + cv * 8 : a.v_pool + blk + r * D + cv * 8) : zero;
    lds_dma16_untracked<true>(src, dst + PT::TBYTES + i * 1024);
  }
}

// Attends the G heads to logical page p staged at buf, updating the wave's online softmax state.
template <int D>
__device__ __forceinline__ void decode_consume(int p, int kv, const bf16x8* qop, f32x4* oacc, float& m_run,
                                               float& l_run, const float c, const char* buf) {
  using PT = PageTile<D>;
  const int lane = threadIdx.x & 63, gi = lane >> 4, j = lane & 15;
  // S^T: lane l holds head l % 16 of keys 4 gi .. 4 gi + 3; its K operand is row l % 16, dims of
  // chunk 4 kb + gi (the Q operand holds the same dims)
  f32x4 sc = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
  for (int kb = 0; kb < PT::KB; ++kb) {
    const bf16x8 kop = *reinterpret_cast<const bf16x8*>(buf + PT::koff(j, 4 * kb + gi));
    sc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(kop, qop[kb], sc, 0, 0, 0);
  }
  // mask keys past the end of the sequence (a select, so stray bit patterns never leak)
#pragma unroll
  for (int r = 0; r < 4; ++r) sc[r] = (p * kPage + 4 * gi + r < kv) ? sc[r] : -INFINITY;
  float mx = fmaxf(fmaxf(sc[0], sc[1]), fmaxf(sc[2], sc[3]));
  mx = fmaxf(mx, __shfl_xor(mx, 16));
  mx = fmaxf(mx, __shfl_xor(mx, 32));
  // the maximum only moves when this page exceeds it, and the O rescale is skipped when no lane
  // of the wave moved (decode is bound by HBM, so it keeps the exact maximum)
  const bool grow = mx * c > m_run;
  const float m_new = grow ? mx * c : m_run;
  const float alpha = grow ? fexp2(m_run - m_new) : 1.0f;
  i16x4 pop;
  float psum = 0.f;
#pragma unroll
  for (int r = 0; r < 4; ++r) {
    const float pr = fexp2(__builtin_fmaf(sc[r], c, -m_new));
    psum += pr;
    pop[r] = (short)bf16_bits(pr);
  }
  l_run = l_run * alpha + psum;
  if (__ballot(grow)) {
#pragma unroll
    for (int mb = 0; mb < PT::MB; ++mb) oacc[mb] *= alpha;
  }
  m_run = m_new;
  // O^T += V^T P^T: the transposing read gives lane l dim 16 mb + l % 16 of keys 4 gi .. 4 gi + 3,
  // the k index of the P^T operand that lane already holds
  const int r0 = 4 * gi + (j >> 2);
#pragma unroll
  for (int mb = 0; mb < PT::MB; ++mb) {
    const i16x4 v = lds_read_tr(buf, PT::voff(r0, 16 * mb + 4 * (j & 3)));
    oacc[mb] = __builtin_amdgcn_mfma_f32_16x16x16bf16_1k(v, pop, oacc[mb], 0, 0, 0);
  }
}


// Physical page of logical page p of the row, read with a scalar load from the block table.
__device__ __forceinline__ int page_id(ConstI32Ptr bt_row, int p, int num_pages) {
  return clamp_page(bt_row[p], num_pages);
}

// One decode work item as the kernels see it: sequence b (its new token is row q_row of q/out),
// kv attended keys, split `split` of n_splits (pps pages each), kv-head g; the partials of a
// multi-split sequence go to slots slot_base + split.
struct DecItem {
  int b, split, g, q_row, kv, n_splits, slot_base;
};

// Split merge inside the attention kernel.  Every split of a multi-split (sequence, kv-head) pair
// stores its partial (o~, m, l) with device-scope stores (written through to the level every XCD
// reads) and moves on.  One item later, once every thread of the workgroup has drained its memory
// operations (so those stores are acknowledged) and passed a barrier, one thread counts the split
// in with a device-scope atomic in split_cnt[b][g] (zeroed before the launch); the workgroup that
// brings the count to n_splits merges the pair (merge_in_kernel).  No release fence is issued: on
// this chip its L2 write-back costs far more than the merge launch it replaces, and deferring the
// count-in by one item keeps the store acknowledgements off the critical path.
//
// merge_in_kernel: wave w merges q-head w of the group (G <= NW) from the partials, read with
// device-scope loads (which do not hit stale cache lines):
//   o = sum_s 2^(m_s - m*) o~_s / sum_s 2^(m_s - m*) l_s,   lse = (m* + log2 l*) ln 2.
// Lane s holds split s's (m, l); every lane holds D/64 dims of o.  The first block of o~ loads is
// issued together with the (m, l) loads, so up to kMergeBlock splits cost one memory round trip.
constexpr int kMergeBlock = 8;

template <int D, int NW>
__device__ __forceinline__ void merge_in_kernel(const AttnArgs& a, const DecItem& it) {
  const int G = a.group, H_q = a.num_q_heads;
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  if (w >= G) return;
  constexpr int PER = D / 64;
  constexpr int U = kMergeBlock;
  const int hq = it.g * G + w;
  const size_t base = (size_t)it.slot_base;
  const int ns = it.n_splits;
  auto ld = [](const float* p) { return __hip_atomic_load(p, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT); };
  auto o_ptr = [&](int sp) { return a.part_o + ((base + sp) * H_q + hq) * D + lane * PER; };
  // (m, l) of the first 64 splits and o~ of the first U, all in flight together
  float m0 = -INFINITY, l0 = 0.f;
  if (lane < ns) {
    m0 = ld(&a.part_ml[2 * ((base + lane) * H_q + hq)]);
    l0 = ld(&a.part_ml[2 * ((base + lane) * H_q + hq) + 1]);
  }
  float v0[U][PER];
#pragma unroll
  for (int u = 0; u < U; ++u) {
    const float* po = o_ptr(min(u, ns - 1));      // past the end: reload the last split, weight 0
#pragma unroll
    for (int i = 0; i < PER; ++i) v0[u][i] = ld(po + i);
  }
  float M = m0;
  for (int s0 = 64; s0 < ns; s0 += 64)
    if (s0 + lane < ns) M = fmaxf(M, ld(&a.part_ml[2 * ((base + s0 + lane) * H_q + hq)]));
#pragma unroll
  for (int off = 32; off >= 1; off >>= 1) M = fmaxf(M, __shfl_xor(M, off));
  float acc[PER];
#pragma unroll
  for (int i = 0; i < PER; ++i) acc[i] = 0.f;
  float L = 0.f;
  for (int s0 = 0; s0 < ns; s0 += 64) {
    const int cnt = min(64, ns - s0);
    float f = 0.f;
    if (lane < cnt) {
      const size_t pidx = (base + s0 + lane) * H_q + hq;
      const float m = s0 == 0 ? m0 : ld(&a.part_ml[2 * pidx]);
      const float l = s0 == 0 ? l0 : ld(&a.part_ml[2 * pidx + 1]);
      f = fexp2(m - M);
      L += f * l;
    }
    for (int j = 0; j < cnt; j += U) {
      float v[U][PER], fj[U];
#pragma unroll
      for (int u = 0; u < U; ++u) {
        const int jj = min(j + u, cnt - 1);
        const float wgt = __shfl(f, jj);
        fj[u] = j + u < cnt ? wgt : 0.f;
        if (s0 == 0 && j == 0) {
#pragma unroll
          for (int i = 0; i < PER; ++i) v[u][i] = v0[u][i];
        } else {
          const float* po = o_ptr(s0 + jj);
#pragma unroll
          for (int i = 0; i < PER; ++i) v[u][i] = ld(po + i);
        }
      }
#pragma unroll
      for (int u = 0; u < U; ++u)
#pragma unroll
        for (int i = 0; i < PER; ++i) acc[i] += fj[u] * v[u][i];
    }
  }
#pragma unroll
  for (int off = 32; off >= 1; off >>= 1) L += __shfl_xor(L, off);
  const float inv = 1.0f / L;
  uint16_t* orow = a.out + ((size_t)it.q_row * H_q + hq) * D + lane * PER;
#pragma unroll
  for (int i = 0; i < PER; ++i) orow[i] = bf16_bits(acc[i] * inv);
  if (lane == 0 && a.lse) a.lse[(size_t)it.q_row * H_q + hq] = (M + flog2(L)) * kLn2;
}

// Counts a finished split in (thread 0; the caller has made its partial stores acknowledged and
// passed a barrier); returns 1 to the thread if this was the pair's last split.
__device__ __forceinline__ int count_split_in(const AttnArgs& a, const DecItem& it) {
  const int prev = __hip_atomic_fetch_add(&a.split_cnt[it.b * a.num_kv_heads + it.g], 1, __ATOMIC_RELAXED,
                                          __HIP_MEMORY_SCOPE_AGENT);
  return prev == it.n_splits - 1;
}

// One pipeline step: issue the next page's copies into s_next (when the wave has one: `more`,
// wave-uniform), then wait for the current page's and consume it from s_cur.  The copies are
// issued untracked, so the compiler adds no waits of its own for them (left to itself it drained
// every copy in flight in one of the loop's two unrolled steps); s_next was last read in the
// previous step, whose operand reads all completed before its MFMAs.
template <int D, bool kNew>
__device__ __forceinline__ void decode_step(const AttnArgs& a, int p_cur, int p_nxt, int phys_nxt, int g, int kv,
                                            char* __restrict__ s_next, const char* __restrict__ s_cur,
                                            const bf16x8* qop, f32x4* oacc, float& m_run, float& l_run,
                                            const NewRow& nr, bool more) {
  constexpr int PAGE_LOADS = 2 * PageTile<D>::NDMA;   // vector-memory ops per page
  // the current page has landed; the copies are invisible to the compiler, so the wait is also a
  // compiler barrier that keeps the stage reads below it
  if (more) {
    decode_issue<D, kNew>(a, phys_nxt, p_nxt, g, kv, s_next, nr);
    __asm__ volatile("s_waitcnt vmcnt(%0)" ::"n"(PAGE_LOADS) : "memory");
  } else {
    __asm__ volatile("s_waitcnt vmcnt(0)" ::: "memory");
  }
  decode_consume<D>(p_cur, kv, qop, oacc, m_run, l_run, a.scale_log2, s_cur);
}

// kMergeHere: a multi-split (sequence, kv-head) is merged inside the attention kernel by the split
// that finishes last (see the end of decode_split); otherwise merge_kernel runs after the launch.
// kMergeHere: `pend` is this workgroup's previous multi-split item, not yet counted in (b < 0:
// none); it is counted in (and merged if last) here, and becomes this item if it has splits.
// s_flag: an LDS word.
// before_end: called by every thread just before the item's closing barrier (decode_kernel
// decodes its next item there, so the claim's latency hides behind this item).
template <int D, int NW, bool kMergeHere, typename BeforeEnd>
__device__ __forceinline__ void decode_split(const AttnArgs& a, const DecItem& it, int pps, char* stageA,
                                             char* stageB, DecItem& pend, int* s_flag, BeforeEnd before_end) {
  constexpr int NT = NW * 64;
  using PT = PageTile<D>;
  constexpr int MB = PT::MB;
  constexpr int KB = PT::KB;
  const int lane = threadIdx.x & 63, w = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);   // wave index (uniform)
  const int gi = lane >> 4, hh = lane & 15;
  const int b = it.b, split = it.split, g = it.g;
  const int G = a.group, H_q = a.num_q_heads;
  const int kv = it.kv;
  const int n_pages = (kv + kPage - 1) / kPage;
  const int p_begin = split * pps;
  const int p_end = min(p_begin + pps, n_pages);
  const int n_pg = p_end - p_begin;                 // pages of this split (>= 1)
  const bool head_ok = hh < G;
  char* st0 = stageA + w * PT::BYTES;
  char* st1 = stageB + w * PT::BYTES;

  const ConstI32Ptr bt_row = (ConstI32Ptr)(a.block_table + (size_t)b * a.bt_stride);

  bf16x8 qop[KB];
  {
    const uint16_t* qrow = a.q + ((size_t)it.q_row * H_q + g * G + (head_ok ? hh : 0)) * D + 8 * gi;
#pragma unroll
    for (int kb = 0; kb < KB; ++kb) {
      const bf16x8 v = as_bf16x8(ld16(qrow + 32 * kb));
      qop[kb] = head_ok ? v : zero_bf16x8();
    }
  }
  // the page ids run one page ahead of the copies, which run one page ahead of the compute
  int cur = min(w, n_pg - 1);
  int ph_cur = page_id(bt_row, p_begin + cur, a.num_pages);
  // fused append (decode kernel with k_new): the split holding the sequence's last page takes the
  // new token's K/V from k_new / v_new; its last wave writes them into the pools once the item's
  // reads are done (a write whose page id is out of range is skipped, as pearl_kv_append does).
  // No other item reads that row.
  NewRow nr{-1, 0, a.k_pool, a.v_pool};            // no new row (valid pointers, never selected)
  if constexpr (kMergeHere) {
    if (a.k_new && split == it.n_splits - 1) {
      const size_t row = ((size_t)it.q_row * a.num_kv_heads + g) * D;
      nr = NewRow{(kv - 1) / kPage, (kv - 1) % kPage, a.k_new + row, a.v_new + row};
    }
  }
  if (w < n_pg) decode_issue<D, kMergeHere>(a, ph_cur, p_begin + cur, g, kv, st0, nr);
  f32x4 oacc[MB];
#pragma unroll
  for (int mb = 0; mb < MB; ++mb) oacc[mb] = f32x4{0.f, 0.f, 0.f, 0.f};
  float m_run = -INFINITY, l_run = 0.f;

  // page indices past the wave's last page are clamped to the split's last page; such a page id is
  // read but never copied
  int nxt = min(w + NW, n_pg - 1);
  int ph_nxt = page_id(bt_row, p_begin + nxt, a.num_pages);
  for (int pi = w; pi < n_pg; pi += 2 * NW) {
    const int pj = pi + NW;
    const int n2 = min(pj + NW, n_pg - 1);
    const int ph_n2 = page_id(bt_row, p_begin + n2, a.num_pages);
    decode_step<D, kMergeHere>(a, p_begin + cur, p_begin + nxt, ph_nxt, g, kv, st1, st0, qop, oacc, m_run,
                               l_run, nr, pj < n_pg);
    if (pj >= n_pg) break;
    const int n3 = min(pj + 2 * NW, n_pg - 1);
    const int ph_n3 = page_id(bt_row, p_begin + n3, a.num_pages);
    decode_step<D, kMergeHere>(a, p_begin + nxt, p_begin + n2, ph_n2, g, kv, st0, st1, qop, oacc, m_run,
                               l_run, nr, pj + NW < n_pg);
    cur = n2;
    nxt = n3;
    ph_nxt = ph_n3;
  }
  __asm__ volatile("s_waitcnt vmcnt(0)" ::: "memory");
  // the new row's bytes and page id are loaded now, to be stored once the LDS merge below has
  // waited for them
  const bool writer = kMergeHere && nr.page >= 0 && w == NW - 1 && lane < D / 8;
  u32x4 new_k = u32x4{0u, 0u, 0u, 0u}, new_v = new_k;
  int new_page = -1;
  if (writer) {
    new_k = ld16(nr.k + 8 * lane);
    new_v = ld16(nr.v + 8 * lane);
    new_page = bt_row[nr.page];
  }
  // each head's four lane groups hold different keys: sum their l
  l_run += __shfl_xor(l_run, 16);
  l_run += __shfl_xor(l_run, 32);

  // merge the waves' states through LDS
  __syncthreads();
  static_assert(Lds<D, NW, 2>::merge_bytes <= NW * PT::BYTES, "merge scratch fits in one set of stages");
  float* mo = reinterpret_cast<float*>(stageA);               // [wave][8 heads][D]
  float* mm = mo + NW * 8 * D;                            // [wave][8]
  float* ml = mm + NW * 8;                                // [wave][8]
  if (head_ok) {
#pragma unroll
    for (int mb = 0; mb < MB; ++mb)
      *reinterpret_cast<f32x4*>(mo + (w * 8 + hh) * D + 16 * mb + 4 * gi) = oacc[mb];
    if (gi == 0) { mm[w * 8 + hh] = m_run; ml[w * 8 + hh] = l_run; }
  }
  __syncthreads();
  const int n_splits = it.n_splits;
  // the previous item's partial stores: every thread drained its memory operations above
  // (vmcnt(0)) before the barrier, so they are acknowledged.  The count-in's result is used only
  // after the output loop, so its latency hides behind that loop.
  int last_in = 0;
  if constexpr (kMergeHere) {
    // the new row's loads have completed (the barriers above waited for them); saying so here lets
    // its stores below go out before the partial stores without any later wait reaching past them
    __builtin_amdgcn_s_waitcnt(PEARL_VMCNT(0));
    if (threadIdx.x == 0 && pend.b >= 0) last_in = count_split_in(a, pend);
    if (writer && new_page >= 0 && new_page < a.num_pages) {
      const size_t dst = (((size_t)new_page * a.num_kv_heads + g) * kPage + nr.slot) * D + 8 * lane;
      *reinterpret_cast<u32x4*>(a.k_pool_w + dst) = new_k;
      *reinterpret_cast<u32x4*>(a.v_pool_w + dst) = new_v;
    }
  }
  for (int t = threadIdx.x; t < G * D; t += NT) {
    const int head = t / D, dim = t - head * D;
    float M = -INFINITY;
#pragma unroll
    for (int ww = 0; ww < NW; ++ww) M = fmaxf(M, mm[ww * 8 + head]);
    float L = 0.f, o = 0.f;
#pragma unroll
    for (int ww = 0; ww < NW; ++ww) {
      const float f = fexp2(mm[ww * 8 + head] - M);
      L += f * ml[ww * 8 + head];
      o += f * mo[(ww * 8 + head) * D + dim];
    }
    const int hq = g * G + head;
    if (n_splits == 1) {
      a.out[((size_t)it.q_row * H_q + hq) * D + dim] = bf16_bits(o / L);
      if (dim == 0 && a.lse) a.lse[(size_t)it.q_row * H_q + hq] = (M + flog2(L)) * kLn2;
    } else {
      const size_t pidx = (size_t)(it.slot_base + split) * H_q + hq;
      if constexpr (kMergeHere) {
        // device-scope stores: written through to the level where every XCD reads them
        __hip_atomic_store(&a.part_o[pidx * D + dim], o, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        if (dim == 0) {
          __hip_atomic_store(&a.part_ml[2 * pidx], M, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
          __hip_atomic_store(&a.part_ml[2 * pidx + 1], L, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        }
      } else {
        a.part_o[pidx * D + dim] = o;
        if (dim == 0) { a.part_ml[2 * pidx] = M; a.part_ml[2 * pidx + 1] = L; }
      }
    }
  }
  before_end();
  if constexpr (kMergeHere) {
    if (threadIdx.x == 0) *s_flag = last_in;
    // the LDS scratch has been read (the next item's copies overwrite it) and s_flag written; the
    // stores just issued stay in flight (a plain barrier, without the release fence's vmcnt(0))
    __builtin_amdgcn_s_waitcnt(PEARL_LGKMCNT0);
    __asm__ volatile("s_barrier" ::: "memory");
    if (*s_flag) merge_in_kernel<D, NW>(a, pend);
    pend = n_splits > 1 ? it : DecItem{-1, 0, 0, 0, 0, 0, 0};
  } else {
    __syncthreads();
  }
}

// ------------------------------------------------------------------------------------------------
// Persistent attention kernel: workgroups pull items (entry x kv-head) from the planner's list
// with an atomic counter (the next item is claimed while the current one runs); prefill tiles
// come first (largest work), decode splits fill the tail.
// ------------------------------------------------------------------------------------------------
// kKinds: 1 = prefill tiles only, 2 = decode splits only, 3 = both (mixed batches).
template <int D, int kKinds> struct KernelCfg {
  static constexpr int NW = kWaves;
  static constexpr int NT = NW * 64;
};

template <int D, int kKinds>
__global__ __launch_bounds__((KernelCfg<D, kKinds>::NT)) void attn_kernel(AttnArgs a, int max_pre) {
  constexpr int NW = KernelCfg<D, kKinds>::NW;
  __shared__ __attribute__((aligned(16))) char smem[Lds<D, NW, kKinds>::bytes];
  // the two stages of the decode pipeline are separate objects so the LDS reads of one are
  // known not to alias the LDS-DMA writes still in flight into the other
  __shared__ __attribute__((aligned(16))) char stageA_[(kKinds == 2) ? NW * PageTile<D>::BYTES : 16];
  __shared__ __attribute__((aligned(16))) char stageB_[(kKinds == 2) ? NW * PageTile<D>::BYTES : 16];
  char* stageA = (kKinds == 2) ? stageA_ : smem;
  char* stageB = (kKinds == 2) ? stageB_ : smem + NW * PageTile<D>::BYTES;
  // prefill-only kernels: three K and three V stage buffers, each set contiguous
  constexpr int kDT = (kKinds == 1) ? DmaTile<D>::BYTES : 16;
  __shared__ __attribute__((aligned(16))) char pk[3 * kDT], pv[3 * kDT];
  __shared__ int s_item[2];
  const int n_items = a.ws_hdr[kHdrNumItems];
  const int n_pre = a.ws_hdr[kHdrNumPre];
  const int split_keys = a.ws_hdr[kHdrPreSplitKeys];
  const int pps = a.ws_hdr[kHdrPagesPerSplit];
  const int H_kv = a.num_kv_heads;
  // Items: prefill items [0, n_pre * H_kv), decode items after them.  Prefill items are handed
  // out by the per-XCD queues below, decode items by one counter.  In mixed launches workgroups
  // below kHdrPreFirstWG take prefill items first, the others decode items first, and each takes
  // the other kind once its own is exhausted, so both kinds run side by side.
  const int n_pre_items = n_pre * H_kv;
  const bool pre_first = (int)blockIdx.x < a.ws_hdr[kHdrPreFirstWG];
  // Prefill items: item i belongs to queue i % 8, and a workgroup takes the items of the queue of
  // the XCD it runs on, then those of the other queues in turn.  With 8 kv-heads the items of
  // one (sequence, kv-head) then share one XCD's L2 (with 4, two XCDs): every tile of a sequence
  // re-reads that head's whole context, which other XCDs would each fetch from memory again.  The
  // queues are balanced (the heads of a tile are equal work), and the turn to other queues
  // completes every item wherever the workgroups run.
  int queue = xcc_id(), queues_left = kNumXcd;      // thread 0's claim state
  auto claim_pre = [&](int limit) -> int {          // a prefill item below limit, or -1
    while (queues_left > 0) {
      const int c = atomicAdd(&a.ws_hdr[kHdrQueues + queue], 1);
      const int64_t i = queue + (int64_t)kNumXcd * c;
      if (i < limit) return (int)i;
      queue = (queue + 1) % kNumXcd;
      --queues_left;
    }
    return -1;
  };
  auto claim = [&]() -> int {
    if constexpr (kKinds == 1) {
      const int i = claim_pre(n_items);
      return i >= 0 ? i : n_items;
    } else if constexpr (kKinds == 2) {
      return atomicAdd(&a.ws_hdr[kHdrCounter], 1);
    } else {
      const int n_dec_items = n_items - n_pre_items;
      if (pre_first) {
        const int c = claim_pre(n_pre_items);
        if (c >= 0) return c;
        const int d = atomicAdd(&a.ws_hdr[kHdrCounter], 1);
        return d < n_dec_items ? n_pre_items + d : n_items;
      } else {
        const int d = atomicAdd(&a.ws_hdr[kHdrCounter], 1);
        if (d < n_dec_items) return n_pre_items + d;
        const int c = claim_pre(n_pre_items);
        return c >= 0 ? c : n_items;
      }
    }
  };
  if (threadIdx.x == 0) s_item[0] = claim();
  __syncthreads();
  int slot = 0;
  int item = s_item[0];
  while (item < n_items) {
    if (threadIdx.x == 0) s_item[slot ^ 1] = claim();
    const int e = item / H_kv;
    const int g = item - e * H_kv;
    if (e < n_pre) {
      if constexpr ((kKinds & 1) != 0) {
        static_assert(NW == kWaves, "prefill tiles use 8 waves");
        const int2 en = a.entries[e];
        if constexpr (kKinds == 1) {
          prefill_tile_pp<D>(a, e, en.x, en.y, g, split_keys, pk, pv);
        } else {
          // the mixed kernel's prefill stage buffers share its LDS region with the decode stages (a
          // workgroup runs one item at a time, and items are separated by a drained barrier)
          constexpr int B = DmaTile<D>::BYTES;
          static_assert(6 * B <= Lds<D, NW, kKinds>::bytes, "stage buffers fit the shared region");
          prefill_tile_pp<D>(a, e, en.x, en.y, g, split_keys, smem, smem + 3 * B);
        }
      }
    } else {
      if constexpr ((kKinds & 2) != 0) {
        const int2 en = a.entries[max_pre + (e - n_pre)];
        const SeqInfo si = a.seqinfo[en.x];
        const DecItem it{en.x, en.y, g, si.q_start, si.ctx_len + si.q_len, si.kind >> 4, a.split_base[en.x]};
        DecItem none{-1, 0, 0, 0, 0, 0, 0};
        decode_split<D, NW, false>(a, it, pps, stageA, stageB, none, nullptr, [] {});
      }
    }
    __syncthreads();
    slot ^= 1;
    item = s_item[slot];
  }
}

// ------------------------------------------------------------------------------------------------
// Decode-only batches of up to kDecPlanMaxSeqs sequences are planned inside the attention kernel:
// every workgroup reads the lengths and builds the same work list in LDS (the same split sizing
// and longest-first order as plan_kernel), so a decode call is one zeroing launch and this kernel,
// with the split merge done by the last split of each (sequence, kv-head) (merge_in_kernel).
// ------------------------------------------------------------------------------------------------
constexpr int kDecPlanChunks = kDecPlanMaxSeqs / kThreads;
static_assert(kDecPlanChunks * kThreads == kDecPlanMaxSeqs, "plan chunks");

struct DecPlanLds {
  int kv[kDecPlanMaxSeqs];                 // keys attended per sequence (context + the new token)
  int full_pre[kDecPlanMaxSeqs + 1];       // exclusive prefix sums of full splits
  int split_pre[kDecPlanMaxSeqs + 1];      // exclusive prefix sums of all splits (partial slot bases)
  int order[kDecPlanMaxSeqs];              // sequences with a short last split, longest class first
  int wsum[2][kWaves];
  int cls_cnt[kDecPlanChunks][kWaves][kPartBuckets];
  int cls_off[kDecPlanChunks][kWaves][kPartBuckets];   // first position of (chunk, wave, class) in order
  unsigned long long pages;
  int err, pps, n_full, n_items;
};

// Pages per decode split over `pages` pages of H kv-heads: about kDecItemsPerCU items per compute
// unit, a multiple of 16, at least the host's bound, at least kDecLongSplitPages while that leaves
// 2 items per compute unit, at most kMaxPagesPerSplit (the rule plan_kernel applies).
__device__ __forceinline__ int dec_split_pages(unsigned long long pages, int H, int pps_min) {
  long long pps = pps_min;
  if (pages > 0) {
    const long long units = (long long)pages * H;
    const long long per = (long long)kPlanComputeUnits * kDecItemsPerCU;
    const long long want = (units + per - 1) / per;
    const long long two = (units + 2LL * kPlanComputeUnits - 1) / (2LL * kPlanComputeUnits);
    pps = max(pps, (want + 15) / 16 * 16);
    pps = max(pps, min((long long)kDecLongSplitPages, (two + 15) / 16 * 16));
    pps = min(pps, (long long)max(pps_min, kMaxPagesPerSplit));
  }
  return (int)pps;
}

// Validates the lengths against the host bounds (any violation: no work, error 1) and builds the
// list; splits beyond the workspace's partial slots give no work and error 2.  Ends with a barrier.
// Sequences are taken kThreads at a time (chunks); a batch of at most kThreads sequences runs one.
__device__ __forceinline__ void decode_plan(const AttnArgs& a, const DecPlanArgs& d, DecPlanLds& P) {
  constexpr int C = kDecPlanChunks;
  const int tid = threadIdx.x, lane = tid & 63, wv = tid >> 6;
  const int B = d.batch, H = a.num_kv_heads;
  const int nch = (B + kThreads - 1) / kThreads;    // chunks holding sequences (<= C)
  if (tid == 0) { P.pages = 0; P.err = 0; }
  int pages[C];
  bool bad = false;
#pragma unroll
  for (int c = 0; c < C; ++c) {
    const int b = c * kThreads + tid;
    pages[c] = 0;
    if (b < B) {
      const int ctx = d.ctx_lens[b];
      const long long kv = (long long)ctx + 1;
      if (ctx < 0 || kv > d.max_kv_len || (kv + kPage - 1) / kPage > a.bt_stride) {
        bad = true;
      } else {
        pages[c] = (int)((kv + kPage - 1) / kPage);
        P.kv[b] = (int)kv;
      }
    }
  }
  unsigned long long wsum = 0;
#pragma unroll
  for (int c = 0; c < C; ++c) {
    unsigned sum = pages[c];                        // 64 sequences of < 2^21 pages
#pragma unroll
    for (int off = 32; off >= 1; off >>= 1) sum += __shfl_xor(sum, off);
    wsum += sum;
  }
  const bool wave_bad = __any(bad);
  __syncthreads();                                  // P.pages and P.err are initialised
  if (lane == 0) {
    atomicAdd(&P.pages, wsum);
    if (wave_bad) atomicOr(&P.err, 1);
  }
  __syncthreads();
  if (tid == 0) P.pps = dec_split_pages(P.pages, H, d.pps_min);
  __syncthreads();
  const int pps = P.pps;
  const int err = P.err;
  if (err) {
#pragma unroll
    for (int c = 0; c < C; ++c) pages[c] = 0;
  }
  const float inv_pps = (float)kPartBuckets / (float)pps;
  int cls[C], rank[C];
#pragma unroll
  for (int c = 0; c < C; ++c) { cls[c] = -1; rank[c] = 0; }
  int carry_f = 0, carry_s = 0;
#pragma unroll
  for (int c = 0; c < C; ++c) {
    if (c >= nch) break;                            // uniform
    const int b = c * kThreads + tid;
    const int nf = pages[c] / pps, rest = pages[c] - nf * pps;
    const int ns = nf + (rest > 0);
    cls[c] = rest > 0 ? part_bucket(rest, inv_pps) : -1;
    int incl_f = nf, incl_s = ns;
#pragma unroll
    for (int off = 1; off < 64; off <<= 1) {
      const int vf = __shfl_up(incl_f, off), vs = __shfl_up(incl_s, off);
      if (lane >= off) { incl_f += vf; incl_s += vs; }
    }
    if (lane == 63) { P.wsum[0][wv] = incl_f; P.wsum[1][wv] = incl_s; }
    // size classes of the short last splits: counts per (chunk, wave) and ranks inside the wave
#pragma unroll
    for (int k = 0; k < kPartBuckets; ++k) {
      const unsigned long long m = __ballot(cls[c] == k);
      if (lane == 0) P.cls_cnt[c][wv][k] = __popcll(m);
      if (cls[c] == k) rank[c] = __popcll(m & ((1ull << lane) - 1ull));
    }
    __syncthreads();
    int bf = carry_f, bs = carry_s, tf = 0, ts = 0;
#pragma unroll
    for (int w = 0; w < kWaves; ++w) {
      if (w < wv) { bf += P.wsum[0][w]; bs += P.wsum[1][w]; }
      tf += P.wsum[0][w];
      ts += P.wsum[1][w];
    }
    if (b < B) { P.full_pre[b] = bf + incl_f - nf; P.split_pre[b] = bs + incl_s - ns; }
    carry_f += tf;
    carry_s += ts;
    if (c + 1 < nch) __syncthreads();               // wsum is reused by the next chunk
  }
  if (wv == 0) {
    // positions of the short splits: classes largest first, and inside a class (chunk, wave)
    // order.  Lane l handles class l/4 and a quarter (4 consecutive (chunk, wave) entries) of it.
    constexpr int E = C * kWaves;                   // (chunk, wave) entries per class
    static_assert(E % 4 == 0, "quarters");
    const int k = lane >> 2, q = lane & 3;
    int cnt[E / 4], part = 0;
#pragma unroll
    for (int j = 0; j < E / 4; ++j) {
      const int e = q * (E / 4) + j, c = e / kWaves, w = e - c * kWaves;
      cnt[j] = c < nch ? P.cls_cnt[c][w][k] : 0;
      part += cnt[j];
    }
    int incl = part;
#pragma unroll
    for (int off = 1; off < 4; off <<= 1) {
      const int v = __shfl_up(incl, off, 4);
      if (q >= off) incl += v;
    }
    const int total = __shfl(incl, (lane & ~3) + 3);   // the class's short splits
    int t = q == 0 ? total : 0, cs = t;                 // inclusive scan of class totals over lanes
#pragma unroll
    for (int off = 1; off < 64; off <<= 1) {
      const int v = __shfl_up(cs, off);
      if (lane >= off) cs += v;
    }
    int run = cs - total + incl - part;                  // class start + quarter start
#pragma unroll
    for (int j = 0; j < E / 4; ++j) {
      const int e = q * (E / 4) + j, c = e / kWaves, w = e - c * kWaves;
      P.cls_off[c][w][k] = run;
      run += cnt[j];
    }
  }
  if (tid == 0) {
    P.full_pre[B] = carry_f;
    P.split_pre[B] = carry_s;
    P.n_full = carry_f;
    P.err = err ? 1 : (carry_s > d.max_dec ? 2 : 0);
    P.n_items = P.err ? 0 : carry_s * H;
  }
  __syncthreads();
#pragma unroll
  for (int c = 0; c < C; ++c) {
    const int b = c * kThreads + tid;
    if (b < B && cls[c] >= 0) P.order[P.cls_off[c][wv][cls[c]] + rank[c]] = b;
  }
  __syncthreads();
}

// The same plan for batches of at most 64 sequences, built by wave 0 alone with a lane per
// sequence: wave reductions, scans and ballots replace the LDS atomics and the barriers between
// the phases (measured: the 8-wave plan spends about 3 us after the lengths arrive; most of it in
// barriers).  The list is identical to decode_plan's.  Ends with a barrier.
__device__ __forceinline__ void decode_plan_small(const AttnArgs& a, const DecPlanArgs& d, DecPlanLds& P) {
  if (threadIdx.x < 64) {
    const int lane = threadIdx.x, B = d.batch, H = a.num_kv_heads;
    int pages = 0;
    bool bad = false;
    if (lane < B) {
      const int ctx = d.ctx_lens[lane];
      const long long kv = (long long)ctx + 1;
      if (ctx < 0 || kv > d.max_kv_len || (kv + kPage - 1) / kPage > a.bt_stride) {
        bad = true;
      } else {
        pages = (int)((kv + kPage - 1) / kPage);
        P.kv[lane] = (int)kv;
      }
    }
    const bool err = __any(bad);
    unsigned total = pages;                         // 64 sequences of < 2^21 pages
#pragma unroll
    for (int off = 32; off >= 1; off >>= 1) total += __shfl_xor(total, off);
    const int pps = dec_split_pages(total, H, d.pps_min);
    if (err) pages = 0;
    const int nf = pages / pps, rest = pages - nf * pps;
    const int ns = nf + (rest > 0);
    const int cls = rest > 0 ? part_bucket(rest, (float)kPartBuckets / (float)pps) : -1;
    int incl_f = nf, incl_s = ns;
#pragma unroll
    for (int off = 1; off < 64; off <<= 1) {
      const int vf = __shfl_up(incl_f, off), vs = __shfl_up(incl_s, off);
      if (lane >= off) { incl_f += vf; incl_s += vs; }
    }
    const int tot_f = __shfl(incl_f, 63), tot_s = __shfl(incl_s, 63);
    // position of a short split: the short splits of the classes before its own (class 0, the
    // longest, first), then those of its class in sequence order
    int pos = 0;
    const unsigned long long below = (1ull << lane) - 1ull;
#pragma unroll
    for (int k = 0; k < kPartBuckets; ++k) {
      const unsigned long long m = __ballot(cls == k);
      if (k < cls) pos += __popcll(m);
      if (k == cls) pos += __popcll(m & below);
    }
    if (lane < B) {
      P.full_pre[lane] = incl_f - nf;
      P.split_pre[lane] = incl_s - ns;
      if (cls >= 0) P.order[pos] = lane;
    }
    if (lane == 0) {
      P.full_pre[B] = tot_f;
      P.split_pre[B] = tot_s;
      P.n_full = tot_f;
      P.pps = pps;
      P.err = err ? 1 : (tot_s > d.max_dec ? 2 : 0);
      P.n_items = P.err ? 0 : tot_s * H;
    }
  }
  __syncthreads();
}

// Work item `item` of the in-kernel plan: entries are the full splits in sequence order, then the
// short last splits by size class; the kv-head runs fastest.
__device__ __forceinline__ DecItem decode_item(const DecPlanLds& P, int item, int H, int B) {
  const int e = item / H, g = item - e * H;
  int b, split;
  if (e < P.n_full) {
    int lo = 0, hi = B - 1;                         // the last sequence whose full splits start at or before e
    while (lo < hi) {
      const int mid = (lo + hi + 1) >> 1;
      if (P.full_pre[mid] <= e) lo = mid; else hi = mid - 1;
    }
    b = lo;
    split = e - P.full_pre[b];
  } else {
    b = P.order[e - P.n_full];
    split = P.full_pre[b + 1] - P.full_pre[b];
  }
  return DecItem{b, split, g, b, P.kv[b], P.split_pre[b + 1] - P.split_pre[b], P.split_pre[b]};
}

template <int D>
__global__ __launch_bounds__(kThreads) void decode_kernel(AttnArgs a, DecPlanArgs d) {
  constexpr int NW = kWaves;
  // separate objects, so the LDS reads of one are known not to alias the LDS-DMA into the other
  __shared__ __attribute__((aligned(16))) char stageA[NW * PageTile<D>::BYTES];
  __shared__ __attribute__((aligned(16))) char stageB[NW * PageTile<D>::BYTES];
  __shared__ DecPlanLds P;
  __shared__ DecItem s_it[2];
  __shared__ int s_flag;
  int first = 0;
  if (threadIdx.x == 0) first = atomicAdd(&a.ws_hdr[kHdrCounter], 1);   // in flight during the plan
  if (d.batch <= 64) decode_plan_small(a, d, P);
  else decode_plan(a, d, P);
  // the error flag shares a cache line with the work counter, so it is written only when set
  // (then no work follows); the prologue cleared it
  if (blockIdx.x == 0 && threadIdx.x == 0 && P.err) a.ws_hdr[kHdrError] = P.err;
  const int n_items = P.n_items, pps = P.pps, H = a.num_kv_heads, B = d.batch;
  const DecItem none{-1, 0, 0, 0, 0, 0, 0};
  if (threadIdx.x == 0) s_it[0] = first < n_items ? decode_item(P, first, H, B) : none;
  __syncthreads();
  int slot = 0;
  DecItem pend = none;                              // previous multi-split item, not yet counted in
  while (s_it[slot].b >= 0) {
    const DecItem it = s_it[slot];
    int nx = 0;
    if (threadIdx.x == 0) nx = atomicAdd(&a.ws_hdr[kHdrCounter], 1);   // used at the item's end
    decode_split<D, NW, true>(a, it, pps, stageA, stageB, pend, &s_flag, [&] {
      if (threadIdx.x == 0) s_it[slot ^ 1] = nx < n_items ? decode_item(P, nx, H, B) : none;
    });                                             // ends with a barrier
    slot ^= 1;
  }
  if (pend.b >= 0) {                                // the last item's count-in
    __builtin_amdgcn_s_waitcnt(PEARL_VMCNT(0));
    __syncthreads();
    if (threadIdx.x == 0) s_flag = count_split_in(a, pend);
    __syncthreads();
    if (s_flag) merge_in_kernel<D, NW>(a, pend);
  }
}

// Zeroes what the in-kernel decode plan needs zeroed: the workspace header (work counter, error
// flag, the zero block) and the split counters.  A kernel, not a memset, so it can be captured.
__global__ __launch_bounds__(256) void decode_prologue_kernel(int32_t* hdr, int32_t* split_cnt, int n_cnt) {
  for (int i = threadIdx.x; i < n_cnt; i += 256) split_cnt[i] = 0;
  if (threadIdx.x < kHdrWords) hdr[threadIdx.x] = 0;
}

// ------------------------------------------------------------------------------------------------
// Split merge: one wave per (sequence, q-head) with more than one split.  The maximum of the
// split maxima is found with a wavefront shuffle reduction; then
//   o = sum_s 2^(m_s - m*) o~_s / sum_s 2^(m_s - m*) l_s,   lse = (m* + log2 l*) ln 2.
// ------------------------------------------------------------------------------------------------
template <int D>
__global__ __launch_bounds__(256) void merge_kernel(AttnArgs a, int batch) {
  const int lane = threadIdx.x & 63;
  const int wid = blockIdx.x * 4 + (threadIdx.x >> 6);
  const int H_q = a.num_q_heads;
  if (wid >= batch * H_q) return;
  const int b = wid / H_q, h = wid - (wid / H_q) * H_q;
  // three independent reads (the record and base of a sequence the planner skipped are read but
  // not used)
  const int err = a.ws_hdr[kHdrError];
  const SeqInfo si = a.seqinfo[b];
  const size_t base = (size_t)a.split_base[b];
  const int ns = si.kind >> 4;
  if (err != 0 || (si.kind & 15) != kSeqDecode || ns <= 1) return;
  float M = -INFINITY;
  for (int s = lane; s < ns; s += 64) M = fmaxf(M, a.part_ml[2 * ((base + s) * H_q + h)]);
#pragma unroll
  for (int off = 32; off >= 1; off >>= 1) M = fmaxf(M, __shfl_xor(M, off));
  constexpr int PER = D / 64;
  constexpr int U = 8;                              // splits whose o~ loads are in flight together
  float acc[PER];
#pragma unroll
  for (int i = 0; i < PER; ++i) acc[i] = 0.f;
  float L = 0.f;
  for (int s0 = 0; s0 < ns; s0 += 64) {
    const int cnt = min(64, ns - s0);
    // lane j computes split s0 + j's weight 2^(m - M) and its share of the sum
    float f = 0.f;
    if (lane < cnt) {
      const size_t pidx = (base + s0 + lane) * H_q + h;
      f = fexp2(a.part_ml[2 * pidx] - M);
      L += f * a.part_ml[2 * pidx + 1];
    }
    for (int j = 0; j < cnt; j += U) {
      float v[U][PER], fj[U];
#pragma unroll
      for (int u = 0; u < U; ++u) {
        const int jj = min(j + u, cnt - 1);       // past the end: reload the last split, weight 0
        const float w = __shfl(f, jj);
        fj[u] = j + u < cnt ? w : 0.f;
        const size_t pidx = (base + s0 + jj) * H_q + h;
#pragma unroll
        for (int i = 0; i < PER; ++i) v[u][i] = a.part_o[pidx * D + lane * PER + i];
      }
#pragma unroll
      for (int u = 0; u < U; ++u)
#pragma unroll
        for (int i = 0; i < PER; ++i) acc[i] += fj[u] * v[u][i];
    }
  }
#pragma unroll
  for (int off = 32; off >= 1; off >>= 1) L += __shfl_xor(L, off);
  const float inv = 1.0f / L;
  uint16_t* orow = a.out + ((size_t)si.q_start * H_q + h) * D + lane * PER;
#pragma unroll
  for (int i = 0; i < PER; ++i) orow[i] = bf16_bits(acc[i] * inv);
  if (lane == 0 && a.lse) a.lse[(size_t)si.q_start * H_q + h] = (M + flog2(L)) * kLn2;
}

// ------------------------------------------------------------------------------------------------
// Merge of split prefill tiles: one wave per (job, kv-head, tile row), grid-stride over the jobs
// the planner recorded.  Same combination as the decode merge, over the tile's splits.
// ------------------------------------------------------------------------------------------------
constexpr int kMergeMaxBlocks = 4096;

template <int D>
__global__ __launch_bounds__(256) void merge_prefill_kernel(AttnArgs a) {
  if (a.ws_hdr[kHdrError] != 0) return;
  const int lane = threadIdx.x & 63;
  const int H_kv = a.num_kv_heads, H_q = a.num_q_heads, G = a.group, T = a.tokens_per_tile;
  const int total = a.ws_hdr[kHdrNumPreJobs] * H_kv * kRowsPerTile;
  constexpr int PER = D / 64;
  for (int r = blockIdx.x * 4 + (threadIdx.x >> 6); r < total; r += gridDim.x * 4) {
    const int rho = r % kRowsPerTile, jg = r / kRowsPerTile;
    const int g = jg % H_kv, j = jg / H_kv;
    const int4 job = a.pre_jobs[j];                  // (sequence, tile, first entry, splits)
    const SeqInfo si = a.seqinfo[job.x];
    const int tok = job.y * T + rho / G;
    if (tok >= si.q_len) continue;
    const int h = g * G + rho % G;
    const int ns = job.w;
    float M = -INFINITY;
    for (int sp = lane; sp < ns; sp += 64)
      M = fmaxf(M, a.part_pre_ml[2 * ((size_t)((job.z + sp) * H_kv + g) * kRowsPerTile + rho)]);
#pragma unroll
    for (int off = 32; off >= 1; off >>= 1) M = fmaxf(M, __shfl_xor(M, off));
    float acc[PER];
#pragma unroll
    for (int i = 0; i < PER; ++i) acc[i] = 0.f;
    float L = 0.f;
    for (int sp = 0; sp < ns; ++sp) {
      const size_t prow = (size_t)((job.z + sp) * H_kv + g) * kRowsPerTile + rho;
      const float f = fexp2(a.part_pre_ml[2 * prow] - M);
      L += f * a.part_pre_ml[2 * prow + 1];
#pragma unroll
      for (int i = 0; i < PER; ++i) acc[i] += f * a.part_pre_o[prow * D + lane * PER + i];
    }
    const float inv = 1.0f / L;
    const size_t orow = (size_t)(si.q_start + tok) * H_q + h;
#pragma unroll
    for (int i = 0; i < PER; ++i) a.out[orow * D + lane * PER + i] = bf16_bits(acc[i] * inv);
    if (lane == 0 && a.lse) a.lse[orow] = (M + flog2(L)) * kLn2;
  }
}

// ------------------------------------------------------------------------------------------------
// Device memory of the allocation-free decode entry point (pearl_attn_decode_static): the
// workspace of one call, one array per device for the life of the process.  Host code never uses
// the array's name as an address: the device address comes from hipGetSymbolAddress, taken once
// per device with that device current.
// ------------------------------------------------------------------------------------------------
static __device__ __align__(256) char scratch[kStaticScratchBytes];

// ------------------------------------------------------------------------------------------------
// host launchers
// ------------------------------------------------------------------------------------------------
namespace {
// Launch parameters per device (compute units, occupancy per kernel), queried on the first call
// that runs on the device.  Initialisation is guarded so concurrent first calls are safe.
struct DevCache {
  std::atomic<int> ready{0};
  int num_cu = 0;
  int occ[2][4] = {{0, 0, 0, 0}, {0, 0, 0, 0}};   // [D == 128][kinds]
  int occ_dec[2] = {0, 0};                        // decode_kernel, [D == 128]
  void* scratch = nullptr;                        // device address of this device's scratch array
  hipError_t scratch_err = hipSuccess;
};

template <int D, int K>
int occupancy_of() {
  int o = 1;
  if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&o, attn_kernel<D, K>, KernelCfg<D, K>::NT, 0) != hipSuccess || o < 1) o = 1;
  return o;
}

template <int D>
int occupancy_of_dec() {
  int o = 1;
  if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&o, decode_kernel<D>, kThreads, 0) != hipSuccess || o < 1) o = 1;
  return o;
}

void fill_cache(DevCache& c, int dev) {
  hipDeviceProp_t prop;
  int ncu = 256;
  if (hipGetDeviceProperties(&prop, dev) == hipSuccess && prop.multiProcessorCount > 0) ncu = prop.multiProcessorCount;
  c.occ[0][1] = occupancy_of<64, 1>(); c.occ[0][2] = occupancy_of<64, 2>(); c.occ[0][3] = occupancy_of<64, 3>();
  c.occ[1][1] = occupancy_of<128, 1>(); c.occ[1][2] = occupancy_of<128, 2>(); c.occ[1][3] = occupancy_of<128, 3>();
  c.occ_dec[0] = occupancy_of_dec<64>(); c.occ_dec[1] = occupancy_of_dec<128>();
  c.num_cu = ncu;
  void* p = nullptr;
  c.scratch_err = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
  c.scratch = c.scratch_err == hipSuccess ? p : nullptr;
}

constexpr int kCachedDevices = 64;
DevCache g_cache[kCachedDevices];
std::mutex g_cache_mutex;

const DevCache& dev_cache() {
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0) dev = 0;
  if (dev >= kCachedDevices) {                   // beyond the cache: query every time
    thread_local DevCache t;
    fill_cache(t, dev);
    return t;
  }
  DevCache& c = g_cache[dev];
  if (!c.ready.load(std::memory_order_acquire)) {
    std::lock_guard<std::mutex> lock(g_cache_mutex);
    if (!c.ready.load(std::memory_order_relaxed)) {
      fill_cache(c, dev);
      c.ready.store(1, std::memory_order_release);
    }
  }
  return c;
}
}  // namespace

int device_num_cu() { return dev_cache().num_cu; }

void* static_scratch(hipError_t* err) {
  const DevCache& c = dev_cache();
  if (err) *err = c.scratch_err;
  return c.scratch;
}

int attention_grid(int head_dim, int kinds) {
  const DevCache& c = dev_cache();
  return c.num_cu * c.occ[head_dim == 128 ? 1 : 0][kinds];
}

hipError_t launch_plan(const PlanParams& p, const int32_t* ctx_lens, const int32_t* cu_q_lens,
                       void* workspace, const WsLayout& lay, hipStream_t stream) {
  char* ws = static_cast<char*>(workspace);
  hipLaunchKernelGGL(plan_kernel, dim3(1), dim3(kPlanThreads), 0, stream, p, ctx_lens, cu_q_lens,
                     reinterpret_cast<int32_t*>(ws + lay.hdr), reinterpret_cast<SeqInfo*>(ws + lay.seqinfo),
                     reinterpret_cast<int32_t*>(ws + lay.split_base), reinterpret_cast<int2*>(ws + lay.entries),
                     reinterpret_cast<int4*>(ws + lay.pre_jobs));
  return hipGetLastError();
}

hipError_t launch_attention(const AttnArgs& a, int head_dim, int kinds, int64_t max_items, int max_pre,
                            hipStream_t stream) {
  if (max_items <= 0) return hipSuccess;
  if (kinds < 1 || kinds > 3) return hipErrorInvalidValue;
  const DevCache& c = dev_cache();
  const int occ = c.occ[head_dim == 128 ? 1 : 0][kinds];
  int64_t grid = (int64_t)c.num_cu * occ;
  if (grid > max_items) grid = max_items;
  const dim3 g((unsigned)grid);
  if (head_dim == 64) {
    if (kinds == 1) hipLaunchKernelGGL((attn_kernel<64, 1>), g, dim3(KernelCfg<64, 1>::NT), 0, stream, a, max_pre);
    else if (kinds == 2) hipLaunchKernelGGL((attn_kernel<64, 2>), g, dim3(KernelCfg<64, 2>::NT), 0, stream, a, max_pre);
    else hipLaunchKernelGGL((attn_kernel<64, 3>), g, dim3(KernelCfg<64, 3>::NT), 0, stream, a, max_pre);
  } else {
    if (kinds == 1) hipLaunchKernelGGL((attn_kernel<128, 1>), g, dim3(KernelCfg<128, 1>::NT), 0, stream, a, max_pre);
    else if (kinds == 2) hipLaunchKernelGGL((attn_kernel<128, 2>), g, dim3(KernelCfg<128, 2>::NT), 0, stream, a, max_pre);
    else hipLaunchKernelGGL((attn_kernel<128, 3>), g, dim3(KernelCfg<128, 3>::NT), 0, stream, a, max_pre);
  }
  return hipGetLastError();
}

hipError_t launch_decode_prologue(const AttnArgs& a, int batch, hipStream_t stream) {
  hipLaunchKernelGGL(decode_prologue_kernel, dim3(1), dim3(256), 0, stream, a.ws_hdr, a.split_cnt,
                     batch * a.num_kv_heads);
  return hipGetLastError();
}

hipError_t launch_decode(const AttnArgs& a, const DecPlanArgs& d, int head_dim, int64_t max_items,
                         hipStream_t stream) {
  if (max_items <= 0) return hipSuccess;
  const DevCache& c = dev_cache();
  int64_t grid = (int64_t)c.num_cu * c.occ_dec[head_dim == 128 ? 1 : 0];
  if (grid > max_items) grid = max_items;
  if (head_dim == 64)
    hipLaunchKernelGGL(decode_kernel<64>, dim3((unsigned)grid), dim3(kThreads), 0, stream, a, d);
  else
    hipLaunchKernelGGL(decode_kernel<128>, dim3((unsigned)grid), dim3(kThreads), 0, stream, a, d);
  return hipGetLastError();
}

hipError_t launch_merge(const AttnArgs& a, int head_dim, int batch, hipStream_t stream) {
  const int64_t waves = (int64_t)batch * a.num_q_heads;
  const unsigned grid = (unsigned)((waves + 3) / 4);
  if (grid == 0) return hipSuccess;
  if (head_dim == 64)
    hipLaunchKernelGGL(merge_kernel<64>, dim3(grid), dim3(256), 0, stream, a, batch);
  else
    hipLaunchKernelGGL(merge_kernel<128>, dim3(grid), dim3(256), 0, stream, a, batch);
  return hipGetLastError();
}

hipError_t launch_merge_prefill(const AttnArgs& a, int head_dim, int64_t jobs_cap, hipStream_t stream) {
  const int64_t waves = jobs_cap * a.num_kv_heads * kRowsPerTile;
  int64_t grid = (waves + 3) / 4;
  if (grid > kMergeMaxBlocks) grid = kMergeMaxBlocks;
  if (grid <= 0) return hipSuccess;
  if (head_dim == 64)
    hipLaunchKernelGGL(merge_prefill_kernel<64>, dim3((unsigned)grid), dim3(256), 0, stream, a);
  else
    hipLaunchKernelGGL(merge_prefill_kernel<128>, dim3((unsigned)grid), dim3(256), 0, stream, a);
  return hipGetLastError();
}

}  // namespace pearl
