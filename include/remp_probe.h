/*
 * remp_probe.h -- HBM access-pattern probes for gfx950 (measurement only).
 *
 * The KV migration reads and writes paged blocks of 4-64 KiB at scattered
 * places (a serving engine's block tables come from a free list).  These
 * probes measure what the memory system sustains for such patterns on its
 * own, so the migration's kernels can be placed against a practical ceiling
 * next to the 8 TB/s peak.  They live in their own library, libremp_probe.so,
 * and never run as part of a migration.
 */
#ifndef REMP_PROBE_H
#define REMP_PROBE_H

#include <stdint.h>
#include <hip/hip_runtime_api.h>

#ifdef __cplusplus
extern "C" {
#endif

#define REMP_PROBE_API __attribute__((visibility("default")))

/* Enqueue one probe launch on `stream`.  The chunk list has n_chunks entries;
 * entry i touches chunk src_idx[i] of src and chunk dst_idx[i] of dst
 * (chunk c is bytes [c * chunk_bytes, (c + 1) * chunk_bytes)); a NULL index
 * array means the identity.  mode 0 copies each source chunk to its
 * destination chunk, mode 1 only reads the source chunks (each lane folds
 * what it read into a value that a store to `sink`, threads * 16 bytes of
 * device memory, would write on a condition that practically never holds),
 * mode 2 only writes the destination chunks, mode 3 copies like mode 0 but
 * stores at device scope (written through the L2 instead of held there).
 * Other accesses are 16-byte non-temporal loads and stores.
 * chunk_bytes: a power of two >= 16.  threads: 256, 512 or 1024; unroll
 * (16-byte vectors in flight per lane): 1, 2, 4 or 8; chunks_per_wg >= 1;
 * ceil(n_chunks / chunks_per_wg) * threads below 2^32.
 * The caller guarantees that src, dst (device, 16-byte aligned) hold every
 * chunk the index arrays (device, n_chunks int32 each) name.  Returns 0, -1
 * for an invalid argument (nothing enqueued), -2 for a launch error. */
REMP_PROBE_API int32_t remp_probe_chunks(int32_t mode, const void* src, void* dst, void* sink, int64_t sink_bytes,
                                         int64_t n_chunks, int32_t chunk_bytes, const int32_t* src_idx,
                                         const int32_t* dst_idx, int32_t threads, int32_t unroll,
                                         int32_t chunks_per_wg, hipStream_t stream);

/* Enqueue a phased copy of `bytes` from src to dst (device, 16-byte aligned,
 * non-overlapping) on `stream`: a persistent grid of `grid` workgroups of
 * `threads` lanes copies consecutive batches of grid * threads * vecs 16-byte
 * vectors, each workgroup its own contiguous part of a batch, each lane `vecs`
 * vectors held in registers between its loads and its stores.  barriers 0: no
 * waits; 1: every workgroup waits, between the loads and the stores of each
 * batch, until all workgroups have completed the batch's loads, so the chip
 * reads and writes in separate phases; 2: also after the stores.  A wait ends
 * after at most wait_us microseconds (then it is counted as a time-out), so the
 * launch always completes; the waits never change the bytes copied.  sync: 8
 * bytes of device memory; the call zeroes it first, and after the launch
 * completes its second 32-bit word holds the number of timed-out waits.
 * threads: 256, 512 or 1024; vecs: 4, 8 or 16; bytes a multiple of the batch;
 * grid at most the number of workgroups the GPU holds at once, which is
 * returned in *max_resident (if not NULL) whenever threads, vecs and barriers
 * are valid, also when the call is refused (so a call with grid 0 queries it).
 * Returns 0, -1 for an invalid argument (nothing enqueued), -2 for a HIP
 * error. */
REMP_PROBE_API int32_t remp_probe_phased(const void* src, void* dst, void* sync, int64_t bytes, int32_t threads,
                                         int32_t vecs, int32_t barriers, int32_t grid, double wait_us,
                                         int32_t* max_resident, hipStream_t stream);

#ifdef __cplusplus
}
#endif

#endif /* REMP_PROBE_H */
