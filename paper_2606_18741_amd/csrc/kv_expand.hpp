// Block-table expansion into per-block descriptors, and the bucket sort of the new
// descriptors by physical block.
// Included by migrate.hip only (one translation unit holds every kernel).
#pragma once

#include <hip/hip_runtime.h>

#include <cstdint>

#include "kv_device.hpp"

namespace remp {

// ---------------------------------------------------------------------------
// expansion: block tables -> one descriptor per live block
// ---------------------------------------------------------------------------

// Bucket of a physical block for the descriptor sort of the new tables (see
// below): nb buckets spread evenly over [0, num_blocks).
constexpr int kDescsPerBucket = 4;   // buckets = ceil(live blocks / 4): order kept at ~4-block granularity

__device__ __forceinline__ uint32_t block_bucket(int32_t block, int64_t num_blocks, uint32_t nb) {
    const int64_t b = static_cast<int64_t>(block > 0 ? block : 0) * nb / num_blocks;
    return static_cast<uint32_t>(b < nb ? b : nb - 1);
}

// Exclusive prefix sums of tokens and of blocks per sequence (one workgroup,
// wave64 shuffle scans combined through LDS, carried across chunks of 1024).
__global__ __launch_bounds__(kScanThreads) void expand_scan(const int32_t* __restrict__ lens, int32_t S,
                                                           int32_t bs, int32_t reset_flag, int32_t* __restrict__ flag,
                                                           int32_t* __restrict__ tok_off,
                                                           int32_t* __restrict__ blk_off,
                                                           int32_t* __restrict__ bucket, uint32_t nb) {
    __shared__ int64_t wave_tok[kScanThreads / 64];
    __shared__ int64_t wave_blk[kScanThreads / 64];
    __shared__ int64_t carry[2];
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    if (tid == 0) {
        carry[0] = 0;
        carry[1] = 0;
        if (reset_flag) *flag = 0;
    }
    if (bucket)   // counters of the descriptor sort, filled by expand_emit
        for (uint32_t i = tid; i < nb; i += kScanThreads) bucket[i] = 0;
    __syncthreads();
    bool bad = false;
    for (int32_t base = 0; base < S; base += kScanThreads) {
        const int32_t s = base + tid;
        int64_t n = s < S ? lens[s] : 0;
        if (n < 0) {
            n = 0;
            bad = true;
        }
        const int64_t nb = (n + bs - 1) / bs;
        int64_t it = n, ib = nb;
#pragma unroll
        for (int d = 1; d < 64; d <<= 1) {
            const int64_t a = __shfl_up(it, d, 64);
            const int64_t b = __shfl_up(ib, d, 64);
            if (lane >= d) {
                it += a;
                ib += b;
            }
        }
        if (lane == 63) {
            wave_tok[wave] = it;
            wave_blk[wave] = ib;
        }
        __syncthreads();
        if (wave == 0) {
            const int nw = kScanThreads / 64;
            int64_t wt = lane < nw ? wave_tok[lane] : 0;
            int64_t wb = lane < nw ? wave_blk[lane] : 0;
#pragma unroll
            for (int d = 1; d < nw; d <<= 1) {
                const int64_t a = __shfl_up(wt, d, 64);
                const int64_t b = __shfl_up(wb, d, 64);
                if (lane >= d) {
                    wt += a;
                    wb += b;
                }
            }
            if (lane < nw) {   // exclusive totals of preceding waves
                wave_tok[lane] = wt;
                wave_blk[lane] = wb;
            }
        }
        __syncthreads();
        const int64_t pre_t = carry[0] + (wave ? wave_tok[wave - 1] : 0);
        const int64_t pre_b = carry[1] + (wave ? wave_blk[wave - 1] : 0);
        if (s < S) {
            const int64_t et = pre_t + it - n, eb = pre_b + ib - nb;
            if (et > INT32_MAX || eb > INT32_MAX) bad = true;
            tok_off[s] = static_cast<int32_t>(et < INT32_MAX ? et : INT32_MAX);
            blk_off[s] = static_cast<int32_t>(eb < INT32_MAX ? eb : INT32_MAX);
        }
        __syncthreads();
        if (tid == kScanThreads - 1) {
            carry[0] = pre_t + it;
            carry[1] = pre_b + ib;
        }
        __syncthreads();
    }
    if (tid == 0) {
        tok_off[S] = static_cast<int32_t>(carry[0] < INT32_MAX ? carry[0] : INT32_MAX);
        blk_off[S] = static_cast<int32_t>(carry[1] < INT32_MAX ? carry[1] : INT32_MAX);
    }
    if (bad) *flag = kFlagTables;
}

// One thread per live block: locate its sequence by binary search over the
// block offsets, then read its id from the table row.  Every index is bounded
// by the host-side sizes; an inconsistency yields an empty descriptor and sets
// the flag instead of an out-of-bounds access.
__global__ __launch_bounds__(256) void expand_emit(const int32_t* __restrict__ lens,
                                                   const int32_t* __restrict__ row_off,
                                                   const int32_t* __restrict__ ids, int32_t S, int32_t bs,
                                                   const int32_t* __restrict__ tok_off,
                                                   const int32_t* __restrict__ blk_off, int64_t nnz,
                                                   int64_t num_blocks, int64_t total_tokens, int64_t n_desc,
                                                   BlockDesc* __restrict__ desc, int32_t* __restrict__ flag,
                                                   int32_t* __restrict__ bucket, uint32_t nb,
                                                   uint64_t* __restrict__ stamp_at, uint64_t stamp) {
    const int64_t b = static_cast<int64_t>(blockIdx.x) * blockDim.x + threadIdx.x;
    if (b == 0 && stamp_at) *stamp_at = stamp;   // the descriptors are complete once this kernel is
    if (b >= n_desc) return;
    int32_t lo = 0, hi = S;   // last s in [0, S] with blk_off[s] <= b
    while (lo < hi) {
        const int32_t mid = (lo + hi + 1) >> 1;
        if (blk_off[mid] <= b) lo = mid;
        else hi = mid - 1;
    }
    BlockDesc d{0, 0, 0, 0};
    bool ok = lo < S;
    if (ok) {
        const int32_t s = lo;
        const int64_t j = b - blk_off[s];
        const int64_t n = lens[s];
        const int64_t r = static_cast<int64_t>(row_off[s]) + j;
        ok = r >= 0 && r < nnz;
        if (ok) {
            const int64_t id = ids[r];
            const int64_t tok = static_cast<int64_t>(tok_off[s]) + j * bs;
            const int64_t rest = n - j * bs;
            const int64_t cnt = rest < bs ? rest : bs;
            ok = id >= 0 && id < num_blocks && cnt > 0 && tok >= 0 && tok + cnt <= total_tokens;
            if (ok) d = BlockDesc{static_cast<int32_t>(id), static_cast<int32_t>(tok), static_cast<int32_t>(cnt), s};
        }
    }
    if (!ok) *flag = kFlagTables;
    desc[b] = d;
    if (bucket) atomicAdd(&bucket[block_bucket(d.block, num_blocks > 0 ? num_blocks : 1, nb)], 1);
}

// ---------------------------------------------------------------------------
// ordering of the new descriptors by physical block
// ---------------------------------------------------------------------------

// The new tables come from a serving engine's free list, so consecutive live
// blocks sit at scattered physical addresses, and an unpack in descriptor
// order writes the pool in random 4-64 KiB pieces.  On MI355X random writes
// cost more than random reads (measured, 4 KiB pieces: 5.6 TB/s scattered
// writes against 6.1 TB/s scattered reads), so the new descriptors are
// bucket-sorted by block id first: the expansion clears and counts the
// buckets, then an exclusive scan and a scatter.  Order inside a bucket is
// whatever the atomics give; every order yields the same bytes.

// Exclusive scan of cnt[0, nb) in place (one workgroup, 4 consecutive counters
// per thread, carried over chunks of 4096).
constexpr int kSortScanPerThread = 4;

__global__ __launch_bounds__(kScanThreads) void sort_scan(int32_t* __restrict__ cnt, uint32_t nb) {
    __shared__ int32_t wave_sum[kScanThreads / 64];
    __shared__ int32_t carry;
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    if (tid == 0) carry = 0;
    __syncthreads();
    for (uint32_t base = 0; base < nb; base += kScanThreads * kSortScanPerThread) {
        const uint32_t i0 = base + tid * kSortScanPerThread;
        int32_t c[kSortScanPerThread];
        int32_t v = 0;
#pragma unroll
        for (int k = 0; k < kSortScanPerThread; ++k) {
            c[k] = i0 + k < nb ? cnt[i0 + k] : 0;
            v += c[k];
        }
        int32_t x = v;
#pragma unroll
        for (int d = 1; d < 64; d <<= 1) {
            const int32_t a = __shfl_up(x, d, 64);
            if (lane >= d) x += a;
        }
        if (lane == 63) wave_sum[wave] = x;
        __syncthreads();
        if (wave == 0) {
            const int nw = kScanThreads / 64;
            int32_t w = lane < nw ? wave_sum[lane] : 0;
#pragma unroll
            for (int d = 1; d < nw; d <<= 1) {
                const int32_t a = __shfl_up(w, d, 64);
                if (lane >= d) w += a;
            }
            if (lane < nw) wave_sum[lane] = w;
        }
        __syncthreads();
        int32_t run = carry + (wave ? wave_sum[wave - 1] : 0) + x - v;   // exclusive prefix of counter i0
#pragma unroll
        for (int k = 0; k < kSortScanPerThread; ++k) {
            if (i0 + k < nb) cnt[i0 + k] = run;
            run += c[k];
        }
        const int32_t pre = carry + (wave ? wave_sum[wave - 1] : 0);
        __syncthreads();
        if (tid == kScanThreads - 1) carry = pre + x;
        __syncthreads();
    }
}

__global__ __launch_bounds__(256) void sort_scatter(const BlockDesc* __restrict__ desc, int32_t n, int64_t num_blocks,
                                                    uint32_t nb, int32_t* __restrict__ next,
                                                    BlockDesc* __restrict__ out, uint64_t* __restrict__ stamp_at,
                                                    uint64_t stamp) {
    const int32_t i = static_cast<int32_t>(blockIdx.x * 256 + threadIdx.x);
    if (i == 0 && stamp_at) *stamp_at = stamp;   // the sorted descriptors are complete once this kernel is
    if (i < n) {
        const BlockDesc d = desc[i];
        const int32_t pos = atomicAdd(&next[block_bucket(d.block, num_blocks, nb)], 1);
        if (pos >= 0 && pos < n) out[pos] = d;
    }
}

}  // namespace remp
