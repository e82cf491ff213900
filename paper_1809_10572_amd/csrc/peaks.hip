// Microbenchmarks of the MI355X ceilings used as roofline denominators: the issue rate
// of the SAMD multiply step (v_mad_i64_i32), of full-rate 32-bit integer VALU work, of
// the int8 matrix cores, and achievable HBM bandwidth (copy and read).
#include <hip/hip_runtime.h>

#include "hip_util.hpp"
#include "samd_peaks.h"

namespace samd {

namespace {

constexpr int kPeakBlock = 256;
constexpr int kChains = 8;    // independent accumulators per lane (as the conv kernel's 8 channels)
constexpr int kMfmaAcc = 4;   // independent MFMA accumulators per wave

typedef int v4i __attribute__((ext_vector_type(4)));

// Opaque to the compiler: the value is taken as rewritten here, so loop-invariant work
// cannot be hoisted or summed up across trips.
template <typename T>
__device__ __forceinline__ void opaque(T &v) {
    asm volatile("" : "+v"(v));
}

// kChains exact signed 32x32 -> 64-bit multiply-adds per trip, the multiplier uniform
// (a kernel argument in SGPRs, as the conv kernel's kernel words), the operand per lane.
__global__ __launch_bounds__(kPeakBlock) void peak_mad_kernel(int iters, int32_t k0, int32_t k1, int32_t *out) {
    const int tid = blockIdx.x * kPeakBlock + threadIdx.x;
    int32_t a = tid * 2654435761u;
    int64_t acc[kChains];
#pragma unroll
    for (int j = 0; j < kChains; ++j) acc[j] = j;
    for (int it = 0; it < iters; ++it) {
        opaque(a);
#pragma unroll
        for (int j = 0; j < kChains; ++j) acc[j] += (int64_t)a * (int64_t)(j & 1 ? k1 : k0 + j);
#pragma unroll
        for (int j = 0; j < kChains; ++j) opaque(acc[j]);
    }
    int64_t s = 0;
#pragma unroll
    for (int j = 0; j < kChains; ++j) s ^= acc[j];
    out[tid] = (int32_t)(s ^ (s >> 32));
}

// kChains independent 32-bit adds per trip.
__global__ __launch_bounds__(kPeakBlock) void peak_valu_kernel(int iters, int32_t k0, int32_t k1, int32_t *out) {
    const int tid = blockIdx.x * kPeakBlock + threadIdx.x;
    uint32_t x[kChains];
#pragma unroll
    for (int j = 0; j < kChains; ++j) x[j] = tid + j;
    for (int it = 0; it < iters; ++it) {
#pragma unroll
        for (int j = 0; j < kChains; ++j) x[j] += (uint32_t)(j & 1 ? k1 : k0);
#pragma unroll
        for (int j = 0; j < kChains; ++j) opaque(x[j]);
    }
    uint32_t s = 0;
#pragma unroll
    for (int j = 0; j < kChains; ++j) s ^= x[j];
    out[tid] = (int32_t)s;
}

// kMfmaAcc independent 16x16x64 int8 products per trip and wave (16 x 16 x 64 = 16384
// multiply-adds each).
__global__ __launch_bounds__(kPeakBlock) void peak_mfma_kernel(int iters, int32_t k0, int32_t k1, int32_t *out) {
    const int tid = blockIdx.x * kPeakBlock + threadIdx.x;
    const v4i a = {tid, k0, k1, tid ^ k0}, b = {k1, tid, k0, tid + k1};
    v4i c0 = {tid, 0, 0, 0}, c1 = {0, tid, 0, 0}, c2 = {0, 0, tid, 0}, c3 = {0, 0, 0, tid};
    for (int it = 0; it < iters; ++it) {
        c0 = __builtin_amdgcn_mfma_i32_16x16x64_i8(a, b, c0, 0, 0, 0);
        c1 = __builtin_amdgcn_mfma_i32_16x16x64_i8(a, b, c1, 0, 0, 0);
        c2 = __builtin_amdgcn_mfma_i32_16x16x64_i8(a, b, c2, 0, 0, 0);
        c3 = __builtin_amdgcn_mfma_i32_16x16x64_i8(a, b, c3, 0, 0, 0);
    }
    const v4i s = c0 ^ c1 ^ c2 ^ c3;
    out[tid] = s[0] ^ s[1] ^ s[2] ^ s[3];
}

// 16-byte LDS reads (ds_read_b128), kLdsReads per trip, each lane reading its own 16 bytes
// of a 16 KiB block (consecutive lanes consecutive 16-byte slots: no bank conflicts); the
// data is xor-combined so the reads cannot be dropped.
constexpr int kLdsReads = 8;
__global__ __launch_bounds__(kPeakBlock) void peak_lds_kernel(int iters, int32_t k0, int32_t k1, int32_t *out) {
    __shared__ __attribute__((aligned(16))) int4 buf[kPeakBlock * 4];
    const int tid = blockIdx.x * kPeakBlock + threadIdx.x;
    for (int i = threadIdx.x; i < kPeakBlock * 4; i += kPeakBlock) buf[i] = int4{i, i ^ k0, i + k1, tid};
    __syncthreads();
    int4 x = {0, 0, 0, 0};
    int base = threadIdx.x;
    for (int it = 0; it < iters; ++it) {
        opaque(base);
#pragma unroll
        for (int r = 0; r < kLdsReads; ++r) {
            v4i v = __builtin_bit_cast(v4i, buf[(base + r * 64) & (kPeakBlock * 4 - 1)]);
            opaque(v);   // all 16 bytes stay live: the read stays 16 bytes wide
            x.x ^= v[0];
        }
    }
    out[tid] = x.x ^ x.y ^ x.z ^ x.w;
}

// Grid-stride streaming copy of n16 16-byte chunks.
__global__ __launch_bounds__(kPeakBlock) void peak_copy_kernel(const int4 *__restrict__ src, int4 *__restrict__ dst,
                                                               int64_t n16) {
    const int64_t stride = (int64_t)gridDim.x * kPeakBlock;
    for (int64_t i = (int64_t)blockIdx.x * kPeakBlock + threadIdx.x; i < n16; i += stride) dst[i] = src[i];
}

// Grid-stride streaming write of n16 16-byte chunks.
__global__ __launch_bounds__(kPeakBlock) void peak_write_kernel(int4 *__restrict__ dst, int64_t n16, int32_t v) {
    const int64_t stride = (int64_t)gridDim.x * kPeakBlock;
    for (int64_t i = (int64_t)blockIdx.x * kPeakBlock + threadIdx.x; i < n16; i += stride) dst[i] = int4{v, v, v, v};
}

// Grid-stride streaming read of n16 16-byte chunks; one sum per workgroup.
__global__ __launch_bounds__(kPeakBlock) void peak_read_kernel(const int4 *__restrict__ src, int64_t n16,
                                                               int32_t *__restrict__ out) {
    const int64_t stride = (int64_t)gridDim.x * kPeakBlock;
    int32_t s = 0;
    for (int64_t i = (int64_t)blockIdx.x * kPeakBlock + threadIdx.x; i < n16; i += stride) {
        const int4 v = src[i];
        s += v.x ^ v.y ^ v.z ^ v.w;
    }
    __shared__ int32_t part[kPeakBlock / 64];
    for (int o = 32; o > 0; o >>= 1) s += __shfl_xor(s, o);
    if ((threadIdx.x & 63) == 0) part[threadIdx.x >> 6] = s;
    __syncthreads();
    if (threadIdx.x == 0) out[blockIdx.x] = part[0] + part[1] + part[2] + part[3];
}

bool valid(int kind, int64_t iters, int32_t blocks, int64_t bytes) {
    if (blocks < 1 || blocks > (1 << 20)) return false;
    switch (kind) {
        case SAMD_PEAK_MAD_I64_I32:
        case SAMD_PEAK_VALU_I32:
        case SAMD_PEAK_MFMA_I8:
        case SAMD_PEAK_LDS: return iters >= 1 && iters <= (1 << 24);
        case SAMD_PEAK_COPY:
        case SAMD_PEAK_READ:
        case SAMD_PEAK_WRITE: return bytes >= 16 && bytes % 16 == 0;
        default: return false;
    }
}

}  // namespace

}  // namespace samd

using namespace samd;

extern "C" {

double samd_peak_work(int kind, int64_t iters, int32_t blocks, int64_t bytes) {
    if (!valid(kind, iters, blocks, bytes)) return -1.0;
    const double threads = (double)blocks * kPeakBlock;
    switch (kind) {
        case SAMD_PEAK_MAD_I64_I32:
        case SAMD_PEAK_VALU_I32: return threads * (double)iters * kChains;
        case SAMD_PEAK_MFMA_I8: return threads / 64.0 * (double)iters * kMfmaAcc * 16.0 * 16.0 * 64.0;
        case SAMD_PEAK_COPY: return 2.0 * (double)bytes;
        case SAMD_PEAK_LDS: return threads * (double)iters * kLdsReads * 16.0;
        default: return (double)bytes;
    }
}

int samd_peak_launch(int kind, int64_t iters, int32_t blocks, const void *src, void *dst, int64_t bytes,
                     hipStream_t stream) {
    set_error("");
    if (!valid(kind, iters, blocks, bytes)) {
        set_error("samd_peak_launch: bad kind, iters, blocks or bytes");
        return SAMD_EINVAL;
    }
    if (!dst || ((kind == SAMD_PEAK_COPY || kind == SAMD_PEAK_READ) && !src)) {
        set_error("samd_peak_launch: NULL buffer");
        return SAMD_EINVAL;
    }
    if ((kind == SAMD_PEAK_COPY || kind == SAMD_PEAK_READ || kind == SAMD_PEAK_WRITE) &&
        (((uintptr_t)src | (uintptr_t)dst) & 15)) {
        set_error("samd_peak_launch: src and dst must be 16-byte aligned");
        return SAMD_EALIGN;
    }
    const dim3 grid((unsigned)blocks), block(kPeakBlock);
    int32_t *out = (int32_t *)dst;
    switch (kind) {
        case SAMD_PEAK_MAD_I64_I32:
            hipLaunchKernelGGL(peak_mad_kernel, grid, block, 0, stream, (int)iters, 3, -5, out);
            break;
        case SAMD_PEAK_VALU_I32:
            hipLaunchKernelGGL(peak_valu_kernel, grid, block, 0, stream, (int)iters, 3, -5, out);
            break;
        case SAMD_PEAK_MFMA_I8:
            hipLaunchKernelGGL(peak_mfma_kernel, grid, block, 0, stream, (int)iters, 3, -5, out);
            break;
        case SAMD_PEAK_WRITE:
            hipLaunchKernelGGL(peak_write_kernel, grid, block, 0, stream, (int4 *)dst, bytes / 16, (int32_t)iters);
            break;
        case SAMD_PEAK_LDS:
            hipLaunchKernelGGL(peak_lds_kernel, grid, block, 0, stream, (int)iters, 3, -5, out);
            break;
        case SAMD_PEAK_COPY:
            hipLaunchKernelGGL(peak_copy_kernel, grid, block, 0, stream, (const int4 *)src, (int4 *)dst, bytes / 16);
            break;
        default:
            hipLaunchKernelGGL(peak_read_kernel, grid, block, 0, stream, (const int4 *)src, bytes / 16, out);
            break;
    }
    return check_launch("samd_peak_launch");
}

}  // extern "C"
