// Map readout (Y_l = phi(Z_l), not stored between strides) and zero fill.
#include "device_common.h"

namespace ssc {

template <bool BF16>
__global__ __launch_bounds__(256) void read_kernel(const float* __restrict__ Z, void* __restrict__ dst, long long n4,
                                                   int relu) {
    for (long long i = blockIdx.x * (long long)blockDim.x + threadIdx.x; i < n4;
         i += (long long)gridDim.x * blockDim.x) {
        f4v z = reinterpret_cast<const f4v*>(Z)[i];
        if (relu) {
            z.x = fmaxf(z.x, 0.f); z.y = fmaxf(z.y, 0.f); z.z = fmaxf(z.z, 0.f); z.w = fmaxf(z.w, 0.f);
        }
        if constexpr (BF16) {
            uint2 p;
            p.x = f32_to_bf16_bits(z.x) | (f32_to_bf16_bits(z.y) << 16);
            p.y = f32_to_bf16_bits(z.z) | (f32_to_bf16_bits(z.w) << 16);
            reinterpret_cast<uint2*>(dst)[i] = p;
        } else {
            reinterpret_cast<f4v*>(dst)[i] = z;
        }
    }
}

template <bool BF16>
__global__ __launch_bounds__(256) void read_slice_kernel(const float* __restrict__ Z, void* __restrict__ dst,
                                                         long long cells, int ctot, int coff, int cout4, int relu) {
    const long long n4 = cells * cout4;
    for (long long i = blockIdx.x * (long long)blockDim.x + threadIdx.x; i < n4;
         i += (long long)gridDim.x * blockDim.x) {
        const long long cell = i / cout4;
        const long long at = cell * ctot + coff + (i - cell * cout4) * 4;   // element index, a multiple of 4
        f4v z = *reinterpret_cast<const f4v*>(Z + at);
        if (relu) {
            z.x = fmaxf(z.x, 0.f); z.y = fmaxf(z.y, 0.f); z.z = fmaxf(z.z, 0.f); z.w = fmaxf(z.w, 0.f);
        }
        if constexpr (BF16) {
            uint2 p;
            p.x = f32_to_bf16_bits(z.x) | (f32_to_bf16_bits(z.y) << 16);
            p.y = f32_to_bf16_bits(z.z) | (f32_to_bf16_bits(z.w) << 16);
            reinterpret_cast<uint2*>(dst)[at / 4] = p;
        } else {
            reinterpret_cast<f4v*>(dst)[at / 4] = z;
        }
    }
}

// phi(Z) at the active sites of a sparse layer, zero elsewhere.
template <bool BF16>
__global__ __launch_bounds__(256) void read_masked_kernel(const float* __restrict__ Z, void* __restrict__ dst,
                                                          long long cells, int cout4, const uint64_t* __restrict__ memb,
                                                          int relu) {
    const long long n4 = cells * cout4;
    for (long long i = blockIdx.x * (long long)blockDim.x + threadIdx.x; i < n4;
         i += (long long)gridDim.x * blockDim.x) {
        f4v z = reinterpret_cast<const f4v*>(Z)[i];
        if (relu) {
            z.x = fmaxf(z.x, 0.f); z.y = fmaxf(z.y, 0.f); z.z = fmaxf(z.z, 0.f); z.w = fmaxf(z.w, 0.f);
        }
        if (!memb_now(memb[i / cout4])) z = f4v{0.f, 0.f, 0.f, 0.f};
        if constexpr (BF16) {
            uint2 p;
            p.x = f32_to_bf16_bits(z.x) | (f32_to_bf16_bits(z.y) << 16);
            p.y = f32_to_bf16_bits(z.z) | (f32_to_bf16_bits(z.w) << 16);
            reinterpret_cast<uint2*>(dst)[i] = p;
        } else {
            reinterpret_cast<f4v*>(dst)[i] = z;
        }
    }
}

__global__ __launch_bounds__(256) void fill_zero_kernel(uint4* __restrict__ p, long long n16) {
    for (long long i = blockIdx.x * (long long)blockDim.x + threadIdx.x; i < n16;
         i += (long long)gridDim.x * blockDim.x)
        p[i] = make_uint4(0u, 0u, 0u, 0u);
}

static unsigned grid_for(long long n) {
    long long b = (n + 255) / 256;
    if (b < 1) b = 1;
    if (b > 8192) b = 8192;
    return (unsigned)b;
}

// n = element count, a multiple of 4 (channel counts are multiples of 8).
hipError_t launch_read(const float* Z, void* dst, long long n, int relu, bool bf16, hipStream_t s) {
    const long long n4 = n / 4;
    if (bf16) hipLaunchKernelGGL(read_kernel<true>, dim3(grid_for(n4)), dim3(256), 0, s, Z, dst, n4, relu);
    else hipLaunchKernelGGL(read_kernel<false>, dim3(grid_for(n4)), dim3(256), 0, s, Z, dst, n4, relu);
    return hipGetLastError();
}

hipError_t launch_read_masked(const float* Z, void* dst, long long cells, int cout, const uint64_t* memb, int relu,
                              bool bf16, hipStream_t s) {
    const long long n4 = cells * (cout / 4);
    if (bf16)
        hipLaunchKernelGGL(read_masked_kernel<true>, dim3(grid_for(n4)), dim3(256), 0, s, Z, dst, cells, cout / 4, memb,
                           relu);
    else
        hipLaunchKernelGGL(read_masked_kernel<false>, dim3(grid_for(n4)), dim3(256), 0, s, Z, dst, cells, cout / 4,
                           memb, relu);
    return hipGetLastError();
}

// ctot, coff and cout are multiples of 4 (channel counts are multiples of 8).
hipError_t launch_read_slice(const float* Z, void* dst, long long cells, int ctot, int coff, int cout, int relu,
                             bool bf16, hipStream_t s) {
    const long long n4 = cells * (cout / 4);
    if (bf16)
        hipLaunchKernelGGL(read_slice_kernel<true>, dim3(grid_for(n4)), dim3(256), 0, s, Z, dst, cells, ctot, coff,
                           cout / 4, relu);
    else
        hipLaunchKernelGGL(read_slice_kernel<false>, dim3(grid_for(n4)), dim3(256), 0, s, Z, dst, cells, ctot, coff,
                           cout / 4, relu);
    return hipGetLastError();
}

// bytes must be a multiple of 16 (all library buffers are padded to 256 B).
hipError_t launch_fill_zero(void* p, size_t bytes, hipStream_t s) {
    const long long n16 = (long long)(bytes / 16);
    if (n16 == 0) return hipSuccess;
    hipLaunchKernelGGL(fill_zero_kernel, dim3(grid_for(n16)), dim3(256), 0, s, static_cast<uint4*>(p), n16);
    return hipGetLastError();
}

}  // namespace ssc
