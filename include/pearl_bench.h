/*
 * pearl_bench.h -- measurement tooling exported by the same library: HBM bandwidth probes and a
 * cache flush.  They compute nothing of the attention path.  A benchmark uses them to state a
 * kernel's time against the bandwidth this device actually reaches (besides its published
 * peak) and to start a timed launch with cold caches: reading a scratch buffer much larger than
 * the caches (1 GiB or more; the L2 caches hold 4 MiB per XCD and the memory-side Infinity Cache
 * 256 MiB) leaves none of the previously used data cached.  The flush reads rather than writes:
 * a written flush leaves dirty lines behind, and their write-back lands in the next kernel's
 * time (on this part a 1 GiB read right after a 1 GiB written flush runs about 25% slower).
 *
 * Conventions (as in pearl_attn.h): device pointers on the current HIP device, 16-byte aligned;
 * `bytes` a multiple of 16 (0 does nothing); asynchronous on `stream` (a hipStream_t, NULL = the
 * null stream); no allocation, no state kept.  Invalid arguments return PEARL_ERR_INVALID_ARG
 * before any HIP call, a size beyond 2^31 - 1 workgroups of 32 KiB returns
 * PEARL_ERR_UNSUPPORTED, a launch error PEARL_ERR_HIP; pearl_last_error() gives the detail.
 * These calls do not record the pearl_set_kernel_events pair.
 */
#ifndef PEARL_BENCH_H
#define PEARL_BENCH_H

#include <stddef.h>
#include <stdint.h>

#include "pearl_attn.h"

#ifdef __cplusplus
extern "C" {
#endif

/* dst[0 .. bytes) = src[0 .. bytes): reads `bytes` (non-temporal loads), writes `bytes`.  The
 * ranges must not overlap. */
pearl_status pearl_hbm_copy(const void* src, void* dst, size_t bytes, void* stream);

/* Reads src[0 .. bytes) and discards it.  `sink` is a caller-owned 16-byte device slot that the
 * kernel may overwrite (almost never does); it reads nothing else.  Over a buffer of 1 GiB or
 * more this is the cache flush. */
pearl_status pearl_hbm_read(const void* src, size_t bytes, void* sink, void* stream);

/* As pearl_hbm_read, with the loads marked non-temporal: the faster read mode of this part for
 * bytes read once, and not a cache flush (such lines are not kept in the caches). */
pearl_status pearl_hbm_read_nt(const void* src, size_t bytes, void* sink, void* stream);

/* Writes the 32-bit `pattern` over dst[0 .. bytes); reads nothing. */
pearl_status pearl_hbm_fill(void* dst, size_t bytes, uint32_t pattern, void* stream);

#ifdef __cplusplus
}
#endif

#endif /* PEARL_BENCH_H */
