// The last stride's change list of a layer, sorted row-major, built on the
// device into a caller's device buffer: the allocation-free, asynchronous
// counterpart of sscater_changed (which synchronises and sorts on the host).
//
// A layer's change list is the set of its grid's cells stamped with the
// stride's epoch (Alg. 1's change map), restricted for a sparse layer to the
// sites active now or in the previous stride.  Enumerating the stamp map in
// cell order yields that set already sorted, so the list is a stream
// compaction: count the matches of each block of cells, scan the counts,
// then write each block's matches at its offset.
//
// The per-block counts live in `scratch`, a fixed device array of this
// library (one per GPU, kept until the process ends), so the call allocates
// nothing and can be captured into a HIP graph.  Calls that overlap on one
// GPU share that array and race; every call overwrites every count it uses.
#include <hip/hip_runtime.h>

#include <mutex>

#include "../../include/sscater.h"
#include "device_common.h"

namespace ssc {

constexpr int CPB = 1024;                    // cells per block: 256 threads x 4 consecutive cells
constexpr int MAX_BLOCKS = 65536;            // 256 KB of counts
constexpr long long MAX_CELLS = (long long)CPB * MAX_BLOCKS;   // 64 Mi cells

static __device__ __align__(256) int32_t scratch[MAX_BLOCKS];

namespace {

// the scratch array's device address on each GPU (hipGetSymbolAddress once
// per device, with that device current)
constexpr int MAX_DEVICES = 64;
std::mutex g_mu;
int32_t* g_scratch[MAX_DEVICES] = {};

__device__ __forceinline__ bool listed(const uint32_t* stamp, const uint64_t* memb, uint32_t epoch, long long q) {
    if (stamp[q] != epoch) return false;
    if (!memb) return true;
    const uint64_t w = memb[q];
    return memb_now(w) || memb_prev(w, epoch);
}

// Exclusive scan of one value per thread over a 256-thread workgroup; returns
// the thread's offset and leaves the total in *total.
__device__ __forceinline__ int block_scan(int v, int* total) {
    __shared__ int part[256];
    const int t = (int)threadIdx.x;
    part[t] = v;
    __syncthreads();
    for (int d = 1; d < 256; d <<= 1) {
        const int x = t >= d ? part[t - d] : 0;
        __syncthreads();
        part[t] += x;
        __syncthreads();
    }
    const int incl = part[t];
    *total = part[255];
    __syncthreads();
    return incl - v;
}

__global__ __launch_bounds__(256) void changed_count_kernel(const uint32_t* __restrict__ stamp,
                                                             const uint64_t* __restrict__ memb, uint32_t epoch,
                                                             long long cells, int32_t* __restrict__ blk) {
    const long long c0 = (long long)blockIdx.x * CPB + 4 * threadIdx.x;
    int n = 0;
#pragma unroll
    for (int j = 0; j < 4; ++j) n += (c0 + j < cells && listed(stamp, memb, epoch, c0 + j)) ? 1 : 0;
    int total;
    block_scan(n, &total);
    if (threadIdx.x == 0) blk[blockIdx.x] = total;
}

// One workgroup: exclusive scan of the block counts in place, the total to
// *count.
__global__ __launch_bounds__(256) void changed_scan_kernel(int32_t* __restrict__ blk, int nblk,
                                                            int32_t* __restrict__ count) {
    int carry = 0;
    for (int b0 = 0; b0 < nblk; b0 += 256) {
        const int b = b0 + (int)threadIdx.x;
        const int v = b < nblk ? blk[b] : 0;
        int total;
        const int off = block_scan(v, &total);
        if (b < nblk) blk[b] = carry + off;
        carry += total;
    }
    if (threadIdx.x == 0) *count = carry;
}

__global__ __launch_bounds__(256) void changed_write_kernel(const uint32_t* __restrict__ stamp,
                                                             const uint64_t* __restrict__ memb, uint32_t epoch,
                                                             long long cells, const int32_t* __restrict__ blk,
                                                             int32_t* __restrict__ dst, int cap) {
    const long long c0 = (long long)blockIdx.x * CPB + 4 * threadIdx.x;
    bool m[4];
    int n = 0;
#pragma unroll
    for (int j = 0; j < 4; ++j) {
        m[j] = c0 + j < cells && listed(stamp, memb, epoch, c0 + j);
        n += m[j] ? 1 : 0;
    }
    int total;
    int at = blk[blockIdx.x] + block_scan(n, &total);
#pragma unroll
    for (int j = 0; j < 4; ++j)
        if (m[j]) {
            if (at < cap) dst[at] = (int32_t)(c0 + j);
            ++at;
        }
}

// The current device's address of `scratch` (the current device is
// `device`); nullptr with *err set on failure.
int32_t* scratch_ptr(int device, hipError_t* err) {
    *err = hipErrorInvalidDevice;
    if (device < 0 || device >= MAX_DEVICES) return nullptr;
    std::lock_guard<std::mutex> lk(g_mu);
    if (!g_scratch[device]) {
        void* p = nullptr;
        *err = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
        if (*err != hipSuccess) return nullptr;
        g_scratch[device] = static_cast<int32_t*>(p);
    }
    *err = hipSuccess;
    return g_scratch[device];
}

}  // namespace
}  // namespace ssc

using namespace ssc;

extern "C" int sscater_changed_noalloc(sscater_t h, int32_t layer, int32_t* dst, int32_t cap, int32_t* count,
                                       void* stream) {
    if (!h || !count || cap < 0 || (cap > 0 && !dst)) return SSCATER_E_INVALID_ARG;
    ChangedSource src;
    if (int rc = changed_source(h, layer, &src)) return rc;
    if (src.cells > MAX_CELLS) return SSCATER_E_SCRATCH;
    int prev = -1;
    hipError_t e = hipGetDevice(&prev);
    if (e != hipSuccess) return report_hip_error(e);
    if (prev != src.device && (e = hipSetDevice(src.device)) != hipSuccess) return report_hip_error(e);
    int rc = SSCATER_OK;
    hipStream_t s = static_cast<hipStream_t>(stream);
    int32_t* blk = scratch_ptr(src.device, &e);
    if (!blk) {
        rc = report_hip_error(e);
    } else {
        // no stride since create / reset: an empty list (the scan of zero
        // blocks writes the count)
        const int nblk = src.have ? (int)((src.cells + CPB - 1) / CPB) : 0;
        if (nblk > 0)
            hipLaunchKernelGGL(changed_count_kernel, dim3(nblk), dim3(256), 0, s, src.stamp, src.memb, src.epoch,
                               src.cells, blk);
        hipLaunchKernelGGL(changed_scan_kernel, dim3(1), dim3(256), 0, s, blk, nblk, count);
        if (nblk > 0)
            hipLaunchKernelGGL(changed_write_kernel, dim3(nblk), dim3(256), 0, s, src.stamp, src.memb, src.epoch,
                               src.cells, blk, dst, cap);
        if ((e = hipGetLastError()) != hipSuccess) rc = report_hip_error(e);
    }
    if (prev != src.device) (void)hipSetDevice(prev);
    return rc;
}
