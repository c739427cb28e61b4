// GPU side of the weight-shard rebuild (Section 3.3): copy each rank's slices
// of the page-locked host store into its shard buffers in HBM.
//
// The copy is bound by the host link (PCIe), not by HBM: a handful of
// workgroups with enough loads in flight saturate it, so the gather kernel
// runs on a capped grid and leaves the other compute units to a KV migration
// running beside it on another stream (Section 3.2).  Each workgroup takes
// 32 KiB chunks of the flattened (segment, row, vector) space in turn; a
// lane's source address is row * pitch + column, its destination is
// contiguous, so every chunk is one coalesced HBM write.  Row-parallel slices
// (a column range of every row) are as cheap as contiguous ones.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cstring>
#include <string>
#include <vector>

#include "device_util.hpp"
#include "plan.hpp"
#include "weights_plan.hpp"

namespace remp {

constexpr int kGatherThreads = 256;
constexpr int kGatherUnroll = 8;
constexpr uint32_t kGatherChunk = kGatherThreads * kGatherUnroll;   // vectors per workgroup step
constexpr int kMaxGatherSegs = 64;                                  // segments per launch
constexpr int kDefaultGatherWgs = 32;                               // default grid cap (saturates PCIe)

struct GatherSeg {
    const char* src;       // device-visible address of the segment's first source byte
    char* dst;             // first destination byte
    int64_t pitch;         // source row pitch, bytes
    uint32_t vpr;          // vectors per row
    uint32_t vpr_magic, vpr_shift;
    uint32_t nvec;         // rows * vpr
    uint32_t chunk_begin;  // first chunk of this segment in the launch
};

struct GatherArgs {
    GatherSeg seg[kMaxGatherSegs];
    int32_t nseg;
    uint32_t total_chunks;
};
static_assert(sizeof(GatherArgs) < 4096, "gather kernel arguments must stay below 4 KiB");

template <int VEC>
__global__ __launch_bounds__(kGatherThreads) void gather_h2d(const GatherArgs a) {
    typedef typename VecT<VEC>::type V;
    for (uint32_t c = blockIdx.x; c < a.total_chunks; c += gridDim.x) {
        // segment holding chunk c (uniform across the workgroup)
        int lo = 0, hi = a.nseg - 1;
        while (lo < hi) {
            const int mid = (lo + hi + 1) >> 1;
            if (a.seg[mid].chunk_begin <= c) lo = mid;
            else hi = mid - 1;
        }
        const GatherSeg& g = a.seg[lo];
        const uint32_t base = (c - g.chunk_begin) * kGatherChunk + threadIdx.x;
        V v[kGatherUnroll];
#pragma unroll
        for (int j = 0; j < kGatherUnroll; ++j) {
            const uint32_t i = base + j * kGatherThreads;
            if (i < g.nvec) {
                const uint32_t row = fast_div(i, g.vpr_magic, g.vpr_shift);
                const uint32_t col = i - row * g.vpr;
                v[j] = *reinterpret_cast<const V*>(g.src + static_cast<int64_t>(row) * g.pitch +
                                                   static_cast<int64_t>(col) * VEC);
            }
        }
#pragma unroll
        for (int j = 0; j < kGatherUnroll; ++j) {
            const uint32_t i = base + j * kGatherThreads;
            if (i < g.nvec) __builtin_nontemporal_store(v[j], reinterpret_cast<V*>(g.dst + static_cast<int64_t>(i) * VEC));
        }
    }
}

// Device-visible address of a page-locked host range, or an error when any
// part of [host, host + bytes) is not page-locked host memory.
static remp_status device_view(const char* host, int64_t bytes, const std::string& what, const char** out) {
    hipPointerAttribute_t a0, a1;
    const hipError_t e0 = hipPointerGetAttributes(&a0, host);
    const hipError_t e1 = hipPointerGetAttributes(&a1, host + bytes - 1);
    if (e0 != hipSuccess || e1 != hipSuccess) (void)hipGetLastError();   // not a sticky error for the caller
    if (e0 != hipSuccess || e1 != hipSuccess || a0.type != hipMemoryTypeHost || a1.type != hipMemoryTypeHost ||
        !a0.devicePointer || !a1.devicePointer)
        return fail(REMP_E_INVALID, what + ": source is not page-locked host memory (allocate it with hipHostMalloc "
                                           "or torch pin_memory=True)");
    if (static_cast<const char*>(a1.devicePointer) - static_cast<const char*>(a0.devicePointer) != bytes - 1)
        return fail(REMP_E_INVALID, what + ": source range is not one page-locked allocation");
    *out = static_cast<const char*>(a0.devicePointer);
    return REMP_OK;
}

// Whether [dst, dst + bytes) lies in one device allocation.
static remp_status check_device_dst(const void* dst, int64_t bytes, const std::string& what) {
    hipPointerAttribute_t a;
    hipError_t e = hipPointerGetAttributes(&a, dst);
    if (e != hipSuccess || a.type != hipMemoryTypeDevice) {
        if (e != hipSuccess) (void)hipGetLastError();
        return fail(REMP_E_INVALID, what + ": destination is not device memory");
    }
    hipDeviceptr_t base = nullptr;
    size_t size = 0;
    e = hipMemGetAddressRange(&base, &size, const_cast<void*>(dst));
    if (e != hipSuccess) {
        (void)hipGetLastError();
        return fail(REMP_E_INVALID, what + ": destination allocation not found");
    }
    if (static_cast<const char*>(dst) + bytes > static_cast<const char*>(base) + size)
        return fail(REMP_E_SIZE, what + ": destination allocation is smaller than the shard");
    return REMP_OK;
}

struct ReadySeg {
    const char* src_host;   // for the DMA engines
    const char* src_dev;    // for the gather kernel
    char* dst;
    int64_t pitch, width, rows;
};

template <int VEC>
static remp_status launch_gather(const std::vector<ReadySeg>& segs, int32_t max_wgs, hipStream_t stream) {
    for (size_t first = 0; first < segs.size(); first += kMaxGatherSegs) {
        const size_t cnt = std::min<size_t>(kMaxGatherSegs, segs.size() - first);
        GatherArgs a;
        std::memset(&a, 0, sizeof(a));
        uint64_t chunks = 0;
        for (size_t k = 0; k < cnt; ++k) {
            const ReadySeg& r = segs[first + k];
            GatherSeg& g = a.seg[k];
            g.src = r.src_dev;
            g.dst = r.dst;
            g.pitch = r.pitch;
            g.vpr = static_cast<uint32_t>(r.width / VEC);
            const FastDiv f = make_fastdiv(g.vpr);
            g.vpr_magic = f.magic;
            g.vpr_shift = f.shift;
            g.nvec = static_cast<uint32_t>(r.rows * (r.width / VEC));
            g.chunk_begin = static_cast<uint32_t>(chunks);
            chunks += (g.nvec + kGatherChunk - 1) / kGatherChunk;
        }
        a.nseg = static_cast<int32_t>(cnt);
        a.total_chunks = static_cast<uint32_t>(chunks);
        const uint32_t grid = static_cast<uint32_t>(std::min<uint64_t>(chunks, static_cast<uint64_t>(max_wgs)));
        hipLaunchKernelGGL(gather_h2d<VEC>, dim3(grid), dim3(kGatherThreads), 0, stream, a);
        if (remp_status st = hip_check(hipGetLastError(), "gather launch")) return st;
    }
    return REMP_OK;
}

}  // namespace remp

using namespace remp;

extern "C" {

remp_status remp_w_load(const remp_w_plan_t* plan, int32_t rank, int32_t tensor_begin, int32_t tensor_end,
                        void* const* dst, uint32_t flags, int32_t max_workgroups, hipStream_t stream) {
    clear_error();
    if (!plan) return fail(REMP_E_INVALID, "plan is NULL");
    const remp_w_plan_t& p = *plan;
    if (rank < 0 || rank >= p.tp * p.pp) return fail(REMP_E_RANGE, "rank out of range");
    if (tensor_begin < 0 || tensor_end < tensor_begin || tensor_end > static_cast<int32_t>(p.tensors.size()))
        return fail(REMP_E_RANGE, "tensor window out of range");
    if (flags & ~REMP_W_COPY_ENGINE) return fail(REMP_E_INVALID, "unknown flags");
    if (max_workgroups < 0) return fail(REMP_E_INVALID, "max_workgroups < 0");

    std::vector<WSeg> segs;
    std::vector<int32_t> seg_tensor;
    for (int32_t i = tensor_begin; i < tensor_end; ++i) {
        w_segments(p, rank, i, segs);
        seg_tensor.resize(segs.size(), i);
    }
    if (segs.empty()) return REMP_OK;
    if (!dst) return fail(REMP_E_INVALID, "dst is NULL");

    // Validate every destination and source before enqueueing anything.
    std::vector<const char*> src_dev(p.parts.size(), nullptr);
    int32_t last_tensor = -1;
    for (size_t k = 0; k < segs.size(); ++k) {
        const WSeg& s = segs[k];
        const int32_t i = seg_tensor[k];
        const std::string what = "tensor " + std::to_string(i);
        if (i != last_tensor) {
            last_tensor = i;
            if (!dst[i]) return fail(REMP_E_INVALID, what + ": destination is NULL");
            if (reinterpret_cast<uintptr_t>(dst[i]) % p.elem_bytes != 0)
                return fail(REMP_E_ALIGN, what + ": destination is not aligned to the element size");
            int64_t r, c;
            remp_w_shard_shape(plan, rank, i, &r, &c);
            if (remp_status st = check_device_dst(dst[i], r * c * p.elem_bytes, what)) return st;
        }
        const WPart& a = p.parts[s.part];
        if (!src_dev[s.part]) {
            if (remp_status st = device_view(a.host, a.rows * a.cols * p.elem_bytes, what, &src_dev[s.part]))
                return st;
        }
    }

    // Ready segments, grouped by the widest vector each one's addresses and sizes allow (a short
    // row-vector part, e.g. a bias, must not narrow the copy of everything else in the call).
    std::vector<ReadySeg> ready[5];   // vector widths 16, 8, 4, 2, 1
    for (size_t k = 0; k < segs.size(); ++k) {
        const WSeg& s = segs[k];
        ReadySeg r;
        r.src_host = p.parts[s.part].host + s.src_off;
        r.src_dev = src_dev[s.part] + s.src_off;
        r.dst = static_cast<char*>(dst[seg_tensor[k]]) + s.dst_off;
        r.pitch = s.pitch;
        r.width = s.width;
        r.rows = s.rows;
        // contiguous rows are one long row: fewer, larger DMA transfers and no row arithmetic
        if (r.pitch == r.width && r.rows > 1) {
            r.width *= r.rows;
            r.pitch = r.width;
            r.rows = 1;
        }
        if (flags & REMP_W_COPY_ENGINE) {
            ready[0].push_back(r);
            continue;
        }
        const uint64_t bits = reinterpret_cast<uintptr_t>(r.src_dev) | reinterpret_cast<uintptr_t>(r.dst) |
                              static_cast<uint64_t>(r.pitch) | static_cast<uint64_t>(r.width) | 16u;
        const int vec = static_cast<int>(bits & (~bits + 1));
        std::vector<ReadySeg>& out = ready[vec == 16 ? 0 : vec == 8 ? 1 : vec == 4 ? 2 : vec == 2 ? 3 : 4];
        // the gather kernel indexes vectors of one segment with 32 bits: split long ones
        const int64_t max_vec = (int64_t(1) << 31);
        if (r.width / vec > max_vec) {
            if (r.rows != 1) return fail(REMP_E_UNSUPPORTED, "a strided shard row exceeds 2^31 vectors");
            const int64_t piece = max_vec * vec;
            for (int64_t off = 0; off < r.width; off += piece) {
                ReadySeg q = r;
                q.src_host += off;
                q.src_dev += off;
                q.dst += off;
                q.width = std::min(piece, r.width - off);
                q.pitch = q.width;
                out.push_back(q);
            }
            continue;
        }
        // rows per segment so that rows * vectors-per-row stays below 2^31
        const int64_t vpr = r.width / vec;
        const int64_t max_rows = std::max<int64_t>(1, max_vec / vpr);
        for (int64_t r0 = 0; r0 < r.rows; r0 += max_rows) {
            ReadySeg q = r;
            q.src_host += r0 * r.pitch;
            q.src_dev += r0 * r.pitch;
            q.dst += r0 * r.width;
            q.rows = std::min(max_rows, r.rows - r0);
            out.push_back(q);
        }
    }

    if (flags & REMP_W_COPY_ENGINE) {
        for (const ReadySeg& r : ready[0]) {
            const hipError_t e = r.rows == 1 ? hipMemcpyAsync(r.dst, r.src_host, r.width, hipMemcpyHostToDevice, stream)
                                             : hipMemcpy2DAsync(r.dst, r.width, r.src_host, r.pitch, r.width, r.rows,
                                                                hipMemcpyHostToDevice, stream);
            if (remp_status st = hip_check(e, "DMA copy")) return st;
        }
        return REMP_OK;
    }
    const int32_t wgs = max_workgroups > 0 ? max_workgroups : kDefaultGatherWgs;
    if (remp_status st = launch_gather<16>(ready[0], wgs, stream)) return st;
    if (remp_status st = launch_gather<8>(ready[1], wgs, stream)) return st;
    if (remp_status st = launch_gather<4>(ready[2], wgs, stream)) return st;
    if (remp_status st = launch_gather<2>(ready[3], wgs, stream)) return st;
    return launch_gather<1>(ready[4], wgs, stream);
}

}  // extern "C"
