// Packing b-bit values into the dense storage format and back (HBM-bound).
//
// Format: a row of `len` values occupies ceil(len / P) uint32 words, P = 32 / b; value j
// sits in bits [(j % P) * b, (j % P) * b + b) of word j / P; unused bits are zero.
#include <hip/hip_runtime.h>

#include "hip_util.hpp"

namespace samd {

namespace {

constexpr int kBlock = 256;

// One thread builds one packed word from its P source bytes.
template <int B, bool SIGNED>
__global__ __launch_bounds__(kBlock) void pack_kernel(const uint8_t *__restrict__ src, int64_t rows, int64_t len,
                                                      int64_t words_per_row, uint32_t *__restrict__ dst,
                                                      int32_t *__restrict__ oor) {
    constexpr int P = 32 / B;
    constexpr uint32_t kMask = (1u << B) - 1;
    const int64_t total = rows * words_per_row;
    int bad = 0;
    for (int64_t w = (int64_t)blockIdx.x * kBlock + threadIdx.x; w < total; w += (int64_t)gridDim.x * kBlock) {
        const int64_t r = w / words_per_row, q = w - r * words_per_row;
        const int64_t j0 = q * P;
        const int cnt = (int)min((int64_t)P, len - j0);
        const uint8_t *s = src + r * len + j0;
        uint32_t word = 0;
#pragma unroll
        for (int i = 0; i < P; ++i) {
            if (i < cnt) {
                const uint32_t byte = s[i];
                if (SIGNED) {
                    const int v = (int)(int8_t)byte;
                    bad += (v < -(1 << (B - 1)) || v > (1 << (B - 1)) - 1) ? 1 : 0;
                } else {
                    bad += (byte > kMask) ? 1 : 0;
                }
                word |= (byte & kMask) << (i * B);
            }
        }
        dst[w] = word;
    }
    if (oor) {
        // wave-wide sum, one atomic per wave
        for (int off = 32; off > 0; off >>= 1) bad += __shfl_xor(bad, off, 64);
        if ((threadIdx.x & 63) == 0 && bad) atomicAdd(oor, bad);
    }
}

// The same for a 4-byte aligned source and 32-bit indices: the P bytes of a word come
// from at most P/4 + 1 dword loads, realigned with byte funnel shifts.
template <int B, bool SIGNED>
__global__ __launch_bounds__(kBlock) void pack_dword_kernel(const uint32_t *__restrict__ src32, uint32_t total_bytes,
                                                            uint32_t len, uint32_t words_per_row, uint32_t total_words,
                                                            uint32_t *__restrict__ dst, int32_t *__restrict__ oor) {
    constexpr int P = 32 / B;
    constexpr int ND = (P + 3) / 4 + 1;
    constexpr uint32_t kMask = (1u << B) - 1;
    int bad = 0;
    for (uint32_t w = blockIdx.x * kBlock + threadIdx.x; w < total_words; w += gridDim.x * kBlock) {
        const uint32_t r = w / words_per_row, q = w - r * words_per_row;
        const uint32_t j0 = q * P;
        const uint32_t cnt = min((uint32_t)P, len - j0);
        const uint32_t o = r * len + j0;          // byte offset of the word's first value
        const uint32_t d0 = o >> 2, dend = (o + cnt + 3) >> 2;
        uint32_t raw[ND];
#pragma unroll
        for (int k = 0; k < ND; ++k) {
            const uint32_t di = d0 + k;
            uint32_t v = 0;
            if (di < dend) {
                if (di * 4 + 4 <= total_bytes) {
                    v = src32[di];
                } else {   // the buffer's last, partial dword: byte by byte
                    const uint8_t *s8 = (const uint8_t *)src32;
                    for (uint32_t e = di * 4; e < total_bytes; ++e) v |= (uint32_t)s8[e] << ((e - di * 4) * 8);
                }
            }
            raw[k] = v;
        }
        uint32_t word = 0;
#pragma unroll
        for (int k = 0; k < ND - 1; ++k) {
            const uint32_t a = __builtin_amdgcn_alignbyte(raw[k + 1], raw[k], o & 3);   // bytes 4k .. 4k+3
#pragma unroll
            for (int e = 0; e < 4; ++e) {
                const int i = 4 * k + e;
                if (i < P && (uint32_t)i < cnt) {
                    const uint32_t byte = (a >> (8 * e)) & 0xffu;
                    if (SIGNED) {
                        const int v = (int)(int8_t)byte;
                        bad += (v < -(1 << (B - 1)) || v > (1 << (B - 1)) - 1) ? 1 : 0;
                    } else {
                        bad += (byte > kMask) ? 1 : 0;
                    }
                    word |= (byte & kMask) << (i * B);
                }
            }
        }
        dst[w] = word;
    }
    if (oor) {
        for (int off = 32; off > 0; off >>= 1) bad += __shfl_xor(bad, off, 64);
        if ((threadIdx.x & 63) == 0 && bad) atomicAdd(oor, bad);
    }
}

// One thread unpacks one word into its P values.
template <int B, bool SIGNED>
__global__ __launch_bounds__(kBlock) void unpack_kernel(const uint32_t *__restrict__ src, int64_t rows, int64_t len,
                                                        int64_t words_per_row, uint8_t *__restrict__ dst) {
    constexpr int P = 32 / B;
    const int64_t total = rows * words_per_row;
    for (int64_t w = (int64_t)blockIdx.x * kBlock + threadIdx.x; w < total; w += (int64_t)gridDim.x * kBlock) {
        const int64_t r = w / words_per_row, q = w - r * words_per_row;
        const int64_t j0 = q * P;
        const int cnt = (int)min((int64_t)P, len - j0);
        const uint32_t word = src[w];
        uint8_t *d = dst + r * len + j0;
#pragma unroll
        for (int i = 0; i < P; ++i) {
            if (i < cnt) {
                int v = (int)((word >> (i * B)) & ((1u << B) - 1));
                if (SIGNED) v = (v << (32 - B)) >> (32 - B);
                d[i] = (uint8_t)v;
            }
        }
    }
}

}  // namespace

int launch_pack(const void *src, int64_t rows, int64_t len, int bits, int is_signed, uint32_t *dst, int32_t *oor,
                hipStream_t s) {
    const int64_t wpr = row_words(len, bits);
    const int grid = grid_for(rows * wpr, kBlock);
    // dword loads need a 4-byte aligned source; both paths need every index in 32 bits
    const bool dword = ((uintptr_t)src & 3) == 0 && rows * len < (int64_t)1 << 31 && rows * wpr < (int64_t)1 << 31;
#define SAMD_PACK_CASE(B, S)                                                                                   \
    if (bits == B && (bool)is_signed == S) {                                                                   \
        if (dword)                                                                                             \
            hipLaunchKernelGGL((pack_dword_kernel<B, S>), dim3(grid), dim3(kBlock), 0, s, (const uint32_t *)src, \
                               (uint32_t)(rows * len), (uint32_t)len, (uint32_t)wpr, (uint32_t)(rows * wpr), dst, oor); \
        else                                                                                                   \
            hipLaunchKernelGGL((pack_kernel<B, S>), dim3(grid), dim3(kBlock), 0, s, (const uint8_t *)src, rows, \
                               len, wpr, dst, oor);                                                            \
        return check_launch("pack");                                                                           \
    }
    SAMD_FOR_EACH_FMT(SAMD_PACK_CASE)
#undef SAMD_PACK_CASE
    set_error("pack: unsupported format");
    return SAMD_EINVAL;
}

int launch_unpack(const uint32_t *src, int64_t rows, int64_t len, int bits, int is_signed, void *dst, hipStream_t s) {
    const int64_t wpr = row_words(len, bits);
    const int grid = grid_for(rows * wpr, kBlock);
#define SAMD_UNPACK_CASE(B, S)                                                                                  \
    if (bits == B && (bool)is_signed == S) {                                                                    \
        hipLaunchKernelGGL((unpack_kernel<B, S>), dim3(grid), dim3(kBlock), 0, s, src, rows, len, wpr,         \
                           (uint8_t *)dst);                                                                     \
        return check_launch("unpack");                                                                          \
    }
    SAMD_FOR_EACH_FMT(SAMD_UNPACK_CASE)
#undef SAMD_UNPACK_CASE
    set_error("unpack: unsupported format");
    return SAMD_EINVAL;
}

}  // namespace samd
