// Access-pattern probes for gfx950 HBM: chunk copies, reads and writes in any
// chunk order, to measure what the memory system sustains for the patterns the
// KV migration produces (contiguous, gathered and scattered 4-8 KiB pieces).
// Measurement infrastructure only: built into its own library
// (libremp_probe.so), never called by the migration.
#include <hip/hip_runtime.h>

#include <cstdint>

#include "remp_probe.h"

namespace {

typedef unsigned int V4 __attribute__((ext_vector_type(4)));

// 16-byte store at device scope: written through the XCD's L2 rather than held
// there as a dirty line.
__device__ __forceinline__ void store_device_scope(V4 v, V4* p) {
    asm volatile("global_store_dwordx4 %0, %1, off sc1" : : "v"(p), "v"(v) : "memory");
}

// One workgroup takes `cpw` consecutive entries of the chunk list; its lanes
// stride over the (chunk, 16-byte vector) space with UNROLL vectors in flight.
// Entry i moves chunk src_idx[i] of src to chunk dst_idx[i] of dst (identity
// when an index array is NULL).  MODE 0 copies, 1 only reads (each lane folds what
// it read into a register that a practically never taken store keeps alive), 2 only writes,
// 3 copies with device-scope stores.
template <int THREADS, int UNROLL, int MODE>
__global__ __launch_bounds__(THREADS) void chunk_probe(const char* __restrict__ src, char* __restrict__ dst,
                                                       V4* __restrict__ sink, int64_t n_chunks, uint32_t chunk_vecs,
                                                       uint32_t vec_shift, const int32_t* __restrict__ src_idx,
                                                       const int32_t* __restrict__ dst_idx, int32_t cpw) {
    const int64_t c0 = static_cast<int64_t>(blockIdx.x) * cpw;
    const int64_t nc = min(static_cast<int64_t>(cpw), n_chunks - c0);
    if (nc <= 0) return;
    const uint32_t total = static_cast<uint32_t>(nc) * chunk_vecs;
    const uint64_t chunk_bytes = static_cast<uint64_t>(chunk_vecs) * 16;
    V4 acc = {0u, 0u, 0u, 0u};
    for (uint32_t base = threadIdx.x; base < total; base += THREADS * UNROLL) {
        V4 r[UNROLL];
        uint64_t d[UNROLL];
        bool ok[UNROLL];
#pragma unroll
        for (int j = 0; j < UNROLL; ++j) {
            const uint32_t x = base + j * THREADS;
            ok[j] = x < total;
            d[j] = 0;
            if (ok[j]) {
                const int64_t c = c0 + (x >> vec_shift);
                const uint32_t v = x & (chunk_vecs - 1);
                const int64_t sc = src_idx ? src_idx[c] : c;
                const int64_t dc = dst_idx ? dst_idx[c] : c;
                d[j] = static_cast<uint64_t>(dc) * chunk_bytes + v * 16;
                if (MODE != 2)
                    r[j] = __builtin_nontemporal_load(
                        reinterpret_cast<const V4*>(src + static_cast<uint64_t>(sc) * chunk_bytes + v * 16));
                else
                    r[j] = V4{x, 1u, 2u, 3u};
            }
        }
#pragma unroll
        for (int j = 0; j < UNROLL; ++j) {
            if (!ok[j]) continue;
            if (MODE == 1) acc ^= r[j];
            else if (MODE == 3) store_device_scope(r[j], reinterpret_cast<V4*>(dst + d[j]));
            else __builtin_nontemporal_store(r[j], reinterpret_cast<V4*>(dst + d[j]));
        }
    }
    // keeps the loads of the read-only probe alive; the stored value is practically never reached
    if (MODE == 1 && acc.x == 0x9E3779B9u && acc.y == 0x7F4A7C15u && acc.z == 0x85EBCA6Bu) sink[threadIdx.x] = acc;
}

template <int THREADS, int UNROLL>
hipError_t launch_mode(int32_t mode, dim3 grid, const char* src, char* dst, V4* sink, int64_t n, uint32_t cv,
                       uint32_t sh, const int32_t* si, const int32_t* di, int32_t cpw, hipStream_t s) {
    if (mode == 0) hipLaunchKernelGGL((chunk_probe<THREADS, UNROLL, 0>), grid, dim3(THREADS), 0, s, src, dst, sink, n, cv, sh, si, di, cpw);
    else if (mode == 1) hipLaunchKernelGGL((chunk_probe<THREADS, UNROLL, 1>), grid, dim3(THREADS), 0, s, src, dst, sink, n, cv, sh, si, di, cpw);
    else if (mode == 2) hipLaunchKernelGGL((chunk_probe<THREADS, UNROLL, 2>), grid, dim3(THREADS), 0, s, src, dst, sink, n, cv, sh, si, di, cpw);
    else hipLaunchKernelGGL((chunk_probe<THREADS, UNROLL, 3>), grid, dim3(THREADS), 0, s, src, dst, sink, n, cv, sh, si, di, cpw);
    return hipGetLastError();
}

template <int THREADS>
hipError_t launch_unroll(int32_t unroll, int32_t mode, dim3 grid, const char* src, char* dst, V4* sink, int64_t n,
                         uint32_t cv, uint32_t sh, const int32_t* si, const int32_t* di, int32_t cpw, hipStream_t s) {
    switch (unroll) {
        case 1: return launch_mode<THREADS, 1>(mode, grid, src, dst, sink, n, cv, sh, si, di, cpw, s);
        case 2: return launch_mode<THREADS, 2>(mode, grid, src, dst, sink, n, cv, sh, si, di, cpw, s);
        case 4: return launch_mode<THREADS, 4>(mode, grid, src, dst, sink, n, cv, sh, si, di, cpw, s);
        default: return launch_mode<THREADS, 8>(mode, grid, src, dst, sink, n, cv, sh, si, di, cpw, s);
    }
}

// Grid-wide wait of the phased copy: every workgroup counts itself in at sync[0]
// once all its lanes' memory operations have completed, then waits until
// `target` arrivals are counted or `wait_ticks` of the constant-rate clock have
// passed (then it counts a time-out in sync[1] and goes on).  Nothing depends on
// the wait for correctness: each workgroup only moves its own vectors, so the
// wait only lines up the phases of the workgroups, and the time bound ends it
// even if some workgroups are not resident.
__device__ __forceinline__ void grid_wait(uint32_t* sync, uint32_t target, uint64_t wait_ticks) {
    __builtin_amdgcn_s_waitcnt(0);
    __syncthreads();
    if (threadIdx.x == 0) {
        __hip_atomic_fetch_add(&sync[0], 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        const uint64_t t0 = static_cast<uint64_t>(wall_clock64());
        while (__hip_atomic_load(&sync[0], __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) < target) {
            if (static_cast<uint64_t>(wall_clock64()) - t0 > wait_ticks) {
                __hip_atomic_fetch_add(&sync[1], 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
                break;
            }
            __builtin_amdgcn_s_sleep(1);
        }
    }
    __syncthreads();
}

// Phased copy: a persistent grid copies `cycles` consecutive batches of
// gridDim.x * THREADS * VECS 16-byte vectors; in each batch workgroup w takes
// its own contiguous THREADS * VECS vectors, each lane VECS of them held in
// registers between its loads and its stores.  BARRIERS 0: no waits (the same
// copy without phases); 1: a grid-wide wait between the loads and the stores of
// every batch, so that the whole chip reads, then writes; 2: a second wait after
// the stores.
template <int THREADS, int VECS, int BARRIERS>
__global__ __launch_bounds__(THREADS) void phased_copy(const V4* __restrict__ src, V4* __restrict__ dst,
                                                       uint32_t* __restrict__ sync, int32_t cycles,
                                                       uint64_t wait_ticks) {
    const uint32_t g = gridDim.x;
    uint32_t waits = 0;
    for (int32_t c = 0; c < cycles; ++c) {
        const uint64_t base = (static_cast<uint64_t>(c) * g + blockIdx.x) * (THREADS * VECS) + threadIdx.x;
        V4 r[VECS];
#pragma unroll
        for (int j = 0; j < VECS; ++j) r[j] = __builtin_nontemporal_load(src + base + j * THREADS);
        if (BARRIERS > 0) grid_wait(sync, ++waits * g, wait_ticks);
#pragma unroll
        for (int j = 0; j < VECS; ++j) __builtin_nontemporal_store(r[j], dst + base + j * THREADS);
        if (BARRIERS > 1) grid_wait(sync, ++waits * g, wait_ticks);
    }
}

__global__ void zero_words(uint32_t* p, int32_t n) {
    if (static_cast<int32_t>(threadIdx.x) < n) p[threadIdx.x] = 0;
}

// Workgroups of phased_copy<THREADS, VECS, barriers> the GPU holds at once.
template <int THREADS, int VECS>
hipError_t resident_b(int32_t barriers, int32_t* out) {
    const void* fn = barriers == 0   ? reinterpret_cast<const void*>(phased_copy<THREADS, VECS, 0>)
                     : barriers == 1 ? reinterpret_cast<const void*>(phased_copy<THREADS, VECS, 1>)
                                     : reinterpret_cast<const void*>(phased_copy<THREADS, VECS, 2>);
    int per_cu = 0, dev = 0, cus = 0;
    hipError_t e = hipOccupancyMaxActiveBlocksPerMultiprocessor(&per_cu, fn, THREADS, 0);
    if (e != hipSuccess) return e;
    if ((e = hipGetDevice(&dev)) != hipSuccess) return e;
    if ((e = hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev)) != hipSuccess) return e;
    *out = per_cu * cus;
    return hipSuccess;
}

template <int THREADS>
hipError_t resident_v(int32_t vecs, int32_t barriers, int32_t* out) {
    switch (vecs) {
        case 4: return resident_b<THREADS, 4>(barriers, out);
        case 8: return resident_b<THREADS, 8>(barriers, out);
        default: return resident_b<THREADS, 16>(barriers, out);
    }
}

template <int THREADS, int VECS>
hipError_t launch_phased_b(int32_t barriers, int32_t grid, const V4* src, V4* dst, uint32_t* sync, int32_t cycles,
                           uint64_t ticks, hipStream_t s) {
    hipLaunchKernelGGL(zero_words, dim3(1), dim3(64), 0, s, sync, 2);
    if (barriers == 0)
        hipLaunchKernelGGL((phased_copy<THREADS, VECS, 0>), dim3(grid), dim3(THREADS), 0, s, src, dst, sync, cycles, ticks);
    else if (barriers == 1)
        hipLaunchKernelGGL((phased_copy<THREADS, VECS, 1>), dim3(grid), dim3(THREADS), 0, s, src, dst, sync, cycles, ticks);
    else
        hipLaunchKernelGGL((phased_copy<THREADS, VECS, 2>), dim3(grid), dim3(THREADS), 0, s, src, dst, sync, cycles, ticks);
    return hipGetLastError();
}

template <int THREADS>
hipError_t launch_phased_v(int32_t vecs, int32_t barriers, int32_t grid, const V4* src, V4* dst, uint32_t* sync,
                           int32_t cycles, uint64_t ticks, hipStream_t s) {
    switch (vecs) {
        case 4: return launch_phased_b<THREADS, 4>(barriers, grid, src, dst, sync, cycles, ticks, s);
        case 8: return launch_phased_b<THREADS, 8>(barriers, grid, src, dst, sync, cycles, ticks, s);
        default: return launch_phased_b<THREADS, 16>(barriers, grid, src, dst, sync, cycles, ticks, s);
    }
}

}  // namespace

extern "C" {

int32_t remp_probe_chunks(int32_t mode, const void* src, void* dst, void* sink, int64_t sink_bytes,
                          int64_t n_chunks, int32_t chunk_bytes, const int32_t* src_idx, const int32_t* dst_idx,
                          int32_t threads, int32_t unroll, int32_t chunks_per_wg, hipStream_t stream) {
    if (mode < 0 || mode > 3) return -1;
    if (n_chunks <= 0 || chunk_bytes < 16 || (chunk_bytes & (chunk_bytes - 1)) != 0) return -1;
    if (threads != 256 && threads != 512 && threads != 1024) return -1;
    if (unroll != 1 && unroll != 2 && unroll != 4 && unroll != 8) return -1;
    if (chunks_per_wg < 1) return -1;
    const uint32_t cv = static_cast<uint32_t>(chunk_bytes / 16);
    uint32_t sh = 0;
    while ((1u << sh) < cv) ++sh;
    if (static_cast<uint64_t>(chunks_per_wg) * cv + static_cast<uint64_t>(threads) * unroll >= (uint64_t(1) << 31))
        return -1;
    const int64_t grid = (n_chunks + chunks_per_wg - 1) / chunks_per_wg;
    if (grid * threads >= (int64_t(1) << 32)) return -1;   // work-items of a dispatch are counted in 32 bits
    if (mode != 2 && !src) return -1;
    if (mode != 1 && !dst) return -1;
    if (mode == 1 && (!sink || sink_bytes < static_cast<int64_t>(threads) * 16)) return -1;
    const dim3 g(static_cast<uint32_t>(grid));
    const char* s = static_cast<const char*>(src);
    char* d = static_cast<char*>(dst);
    V4* k = static_cast<V4*>(sink);
    hipError_t e;
    if (threads == 256) e = launch_unroll<256>(unroll, mode, g, s, d, k, n_chunks, cv, sh, src_idx, dst_idx, chunks_per_wg, stream);
    else if (threads == 512) e = launch_unroll<512>(unroll, mode, g, s, d, k, n_chunks, cv, sh, src_idx, dst_idx, chunks_per_wg, stream);
    else e = launch_unroll<1024>(unroll, mode, g, s, d, k, n_chunks, cv, sh, src_idx, dst_idx, chunks_per_wg, stream);
    return e == hipSuccess ? 0 : -2;
}

int32_t remp_probe_phased(const void* src, void* dst, void* sync, int64_t bytes, int32_t threads, int32_t vecs,
                          int32_t barriers, int32_t grid, double wait_us, int32_t* max_resident, hipStream_t stream) {
    int32_t resident = 0;
    if (max_resident) *max_resident = 0;
    if (threads != 256 && threads != 512 && threads != 1024) return -1;
    if (vecs != 4 && vecs != 8 && vecs != 16) return -1;
    if (barriers < 0 || barriers > 2) return -1;
    const hipError_t re = threads == 256   ? resident_v<256>(vecs, barriers, &resident)
                          : threads == 512 ? resident_v<512>(vecs, barriers, &resident)
                                           : resident_v<1024>(vecs, barriers, &resident);
    if (re != hipSuccess) return -2;
    if (max_resident) *max_resident = resident;
    if (!src || !dst || !sync || bytes <= 0 || grid < 1 || grid > resident) return -1;
    if (!(wait_us > 0.0) || wait_us > 1.0e6) return -1;
    if ((reinterpret_cast<uintptr_t>(src) | reinterpret_cast<uintptr_t>(dst)) % 16 || reinterpret_cast<uintptr_t>(sync) % 4)
        return -1;
    const int64_t batch = static_cast<int64_t>(grid) * threads * vecs * 16;
    if (bytes % batch) return -1;
    const int64_t cycles = bytes / batch;
    if (cycles * 2 * grid >= (int64_t(1) << 31)) return -1;
    int dev = 0, khz = 0;
    if (hipGetDevice(&dev) != hipSuccess || hipDeviceGetAttribute(&khz, hipDeviceAttributeWallClockRate, dev) != hipSuccess ||
        khz <= 0)
        return -2;
    const uint64_t ticks = static_cast<uint64_t>(wait_us * khz / 1000.0) + 1;
    const V4* s = static_cast<const V4*>(src);
    V4* d = static_cast<V4*>(dst);
    uint32_t* y = static_cast<uint32_t*>(sync);
    const int32_t cyc = static_cast<int32_t>(cycles);
    hipError_t e;
    if (threads == 256) e = launch_phased_v<256>(vecs, barriers, grid, s, d, y, cyc, ticks, stream);
    else if (threads == 512) e = launch_phased_v<512>(vecs, barriers, grid, s, d, y, cyc, ticks, stream);
    else e = launch_phased_v<1024>(vecs, barriers, grid, s, d, y, cyc, ticks, stream);
    return e == hipSuccess ? 0 : -2;
}

}  // extern "C"
