// Between-layer epilogue of the AlexNet-shaped stack: the layer maximum, then ReLU and
// requantisation to unsigned b bits, written in the packed storage format, straight into
// the next layer's operand words (the SAMD chain), or as NHWC uint8 (the 8-bit baseline
// chain).  The paper fixes no rule;
// the library's rule: mx = max(max(acc), 0), s = the smallest s >= 0 with
// mx >> s <= 2^b - 1, q = min((max(v, 0) + (s ? 2^(s-1) : 0)) >> s, 2^b - 1).
#include <hip/hip_runtime.h>

#include <climits>

#include "hip_util.hpp"

namespace samd {

namespace {

constexpr int kBlock = 256;

__global__ void max_init_kernel(int32_t *dev_max) {
    if (threadIdx.x == 0 && blockIdx.x == 0) *dev_max = INT_MIN;
}

// The maximum of n values: each workgroup reduces its grid-stride share (16-byte loads
// when src is 16-byte aligned, four in flight per thread; shuffles, then LDS across its
// waves) and only then touches *dev_max, with one atomic, and only when its maximum
// exceeds what *dev_max already holds.  Atomics on one address serialise (about 12 ns
// each), and the workgroups of one launch finish at nearly the same time, so the grid is
// kept to a few hundred workgroups that each read many values.
constexpr int kMaxGrid = 512;
__global__ __launch_bounds__(kBlock) void max_kernel(const int32_t *__restrict__ src, int64_t n, int32_t *dev_max) {
    __shared__ int32_t part[kBlock / 64];
    int32_t m = INT_MIN;
    const int64_t stride = (int64_t)gridDim.x * kBlock;
    const int64_t tid = (int64_t)blockIdx.x * kBlock + threadIdx.x;
    int64_t head = 0;   // values before the first 16-byte vector
    if (((uintptr_t)src & 15) == 0) {
        const int4 *v = (const int4 *)src;
        const int64_t n4 = n >> 2;
#pragma unroll 4
        for (int64_t i = tid; i < n4; i += stride) {
            const int4 q = v[i];
            m = max(m, max(max(q.x, q.y), max(q.z, q.w)));
        }
        head = n4 << 2;
    }
    for (int64_t i = head + tid; i < n; i += stride) m = max(m, src[i]);
    for (int off = 32; off > 0; off >>= 1) m = max(m, __shfl_xor(m, off, 64));
    if ((threadIdx.x & 63) == 0) part[threadIdx.x >> 6] = m;
    __syncthreads();
    if (threadIdx.x == 0) {
#pragma unroll
        for (int w = 1; w < kBlock / 64; ++w) m = max(m, part[w]);
        if (m > __hip_atomic_load(dev_max, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT)) atomicMax(dev_max, m);
    }
}

__global__ void zero_count_kernel(int32_t *count) {
    if (threadIdx.x == 0 && blockIdx.x == 0) *count = 0;
}

// Number of positions where two int32 arrays differ, added to *count.
__global__ __launch_bounds__(kBlock) void mismatch_kernel(const int32_t *__restrict__ a,
                                                          const int32_t *__restrict__ b, int64_t n,
                                                          int32_t *count) {
    int32_t c = 0;
    for (int64_t i = (int64_t)blockIdx.x * kBlock + threadIdx.x; i < n; i += (int64_t)gridDim.x * kBlock)
        c += a[i] != b[i] ? 1 : 0;
    for (int off = 32; off > 0; off >>= 1) c += __shfl_xor(c, off, 64);
    if ((threadIdx.x & 63) == 0 && c != 0) atomicAdd(count, c);
}

// Requantisation shift for a layer maximum.
__device__ inline int requant_shift(int32_t layer_max, int bits) {
    const uint32_t mx = layer_max > 0 ? (uint32_t)layer_max : 0u;
    const int len = 32 - __clz(mx);   // bit length, 0 for 0
    return len > bits ? len - bits : 0;
}

__device__ inline uint32_t requant(int32_t v, int shift, int bits) {
    const int64_t r = v > 0 ? v : 0;
    const int64_t half = shift ? (int64_t)1 << (shift - 1) : 0;
    const int64_t q = (r + half) >> shift;
    const int64_t top = ((int64_t)1 << bits) - 1;
    return (uint32_t)(q < top ? q : top);
}

// Rows of at most kPackVals values: a workgroup takes whole consecutive rows (their
// values are one contiguous run of acc), reads them coalesced into LDS as requantised
// bytes, then builds and stores one packed word per thread.  Longer rows: one thread
// per packed word, reading its values directly.
constexpr int kPackVals = 4096;

template <int B>
__global__ __launch_bounds__(kBlock) void relu_requant_pack_kernel(const int32_t *__restrict__ acc, int64_t rows,
                                                                   int32_t len, int32_t words_per_row, int32_t rpb,
                                                                   const int32_t *__restrict__ dev_max,
                                                                   uint32_t *__restrict__ dst,
                                                                   int32_t *__restrict__ dev_shift) {
    constexpr int P = 32 / B;
    __shared__ uint8_t q8[kPackVals];
    const int shift = requant_shift(*dev_max, B);
    if (dev_shift && blockIdx.x == 0 && threadIdx.x == 0) *dev_shift = shift;
    const int64_t r0 = (int64_t)blockIdx.x * rpb;
    const int R = (int)min((int64_t)rpb, rows - r0);
    const int nv = R * len;   // <= kPackVals
    const int32_t *a = acc + r0 * len;
#pragma unroll 4
    for (int i = threadIdx.x; i < nv; i += kBlock) q8[i] = (uint8_t)requant(a[i], shift, B);
    __syncthreads();
    const int nw = R * words_per_row;
    for (int k = threadIdx.x; k < nw; k += kBlock) {
        const int r = k / words_per_row, qw = k - r * words_per_row;
        const int j0 = qw * P, cnt = min(P, len - j0);
        const uint8_t *src = q8 + r * len + j0;
        uint32_t word = 0;
#pragma unroll
        for (int i = 0; i < P; ++i)
            if (i < cnt) word |= (uint32_t)src[i] << (i * B);
        dst[(r0 + r) * words_per_row + qw] = word;
    }
}

template <int B>
__global__ __launch_bounds__(kBlock) void relu_requant_pack_long_kernel(const int32_t *__restrict__ acc, int64_t rows,
                                                                        int64_t len, int64_t words_per_row,
                                                                        const int32_t *__restrict__ dev_max,
                                                                        uint32_t *__restrict__ dst,
                                                                        int32_t *__restrict__ dev_shift) {
    constexpr int P = 32 / B;
    const int shift = requant_shift(*dev_max, B);
    if (dev_shift && blockIdx.x == 0 && threadIdx.x == 0) *dev_shift = shift;
    const int64_t total = rows * words_per_row;
    for (int64_t w = (int64_t)blockIdx.x * kBlock + threadIdx.x; w < total; w += (int64_t)gridDim.x * kBlock) {
        const int64_t r = w / words_per_row, q = w - r * words_per_row;
        const int64_t j0 = q * P;
        const int cnt = (int)min((int64_t)P, len - j0);
        const int32_t *a = acc + r * len + j0;
        uint32_t word = 0;
#pragma unroll
        for (int i = 0; i < P; ++i)
            if (i < cnt) word |= requant(a[i], shift, B) << (i * B);
        dst[w] = word;
    }
}

// ReLU + requantisation written straight into the next layer's operand words: the
// activations never take the dense packed form between layers, they go from the int32
// accumulators into lanes with spacer bits (the layout the next layer multiplies).
// Word q of kernel-word variant t of padded row hp of channel c of image n holds, lane
// ii, the requantised activation of column sw (q I + delta_t + ii) + phase_t - pw of row
// hp - ph, minus the next layer's recentring offset; columns and rows outside the image
// are 0.  The same words the next layer's operand spread builds from packed rows.
// A block of 256 threads covers 256 / QP padded rows, as that spread does.
__global__ __launch_bounds__(kBlock) void relu_requant_stage_kernel(const int32_t *__restrict__ acc,
                                                                    const int32_t *__restrict__ dev_max,
                                                                    const Conv2dGeom g, int qshift,
                                                                    int32_t *__restrict__ xs,
                                                                    int32_t *__restrict__ dev_shift) {
    const int shift = requant_shift(*dev_max, g.xbits);
    if (dev_shift && blockIdx.x == 0 && threadIdx.x == 0) *dev_shift = shift;
    const int64_t row = (int64_t)blockIdx.x * (kBlock >> qshift) + (threadIdx.x >> qshift);   // (n*C + c)*Hp + hp
    if (row >= (int64_t)g.N * g.C * g.Hp) return;
    const int hp = (int)(row % g.Hp);
    const int64_t nc = row / g.Hp;
    const int h = hp - g.ph;
    const bool inside = h >= 0 && h < g.H;
    const int32_t *src = acc + (nc * g.H + (inside ? h : 0)) * g.W;
    for (int q = threadIdx.x & ((1 << qshift) - 1); q < g.nq; q += 1 << qshift) {
        int32_t *dst = xs + row * g.ntw * g.nq + q;
        for (int t = 0; t < g.ntw; ++t) {
            const int delta = g.tw_tap0[t] + g.tw_ntaps[t] - g.Kmax;
            const int col0 = g.sw * (q * g.I + delta) + g.tw_phase[t] - g.pw;
            uint32_t word = 0;
            if (inside)
                for (int ii = 0; ii < g.I; ++ii) {
                    const int col = col0 + g.sw * ii;
                    if (col >= 0 && col < g.W)
                        word += (uint32_t)((int32_t)requant(src[col], shift, g.xbits) - g.xoff) << (ii * g.L);
                }
            dst[t * g.nq] = (int32_t)word;
        }
    }
}

// NCHW accumulators to NHWC bytes through an LDS tile: a workgroup takes kNhwcCols
// columns of one image row and kNhwcChans channels (grid: image rows x column tiles x
// channel chunks); it reads each channel's columns as one contiguous run (coalesced,
// several channels' loads in flight per wave), requantises them into the tile, then
// writes the tile's pixels, whose chunk of channel bytes is contiguous in NHWC, with
// consecutive threads on consecutive bytes (whole 32-bit words when aligned).
constexpr int kNhwcCols = 64;
constexpr int kNhwcChans = 64;
__global__ __launch_bounds__(kBlock) void relu_requant_nhwc_kernel(const int32_t *__restrict__ acc, int N, int C,
                                                                   int H, int W, const int32_t *__restrict__ dev_max,
                                                                   int bits, uint8_t *__restrict__ dst) {
    constexpr int kPitch = kNhwcCols + 4;   // bytes per tile row (channel), padded
    __shared__ uint8_t tile[kNhwcChans * kPitch];
    const int shift = requant_shift(*dev_max, bits);
    const int tiles_w = (W + kNhwcCols - 1) / kNhwcCols;
    const int chunks = (C + kNhwcChans - 1) / kNhwcChans;
    int b = blockIdx.x;
    const int ch = b % chunks;
    b /= chunks;
    const int tw = b % tiles_w;
    const int nh = b / tiles_w;   // n H + h
    const int n = nh / H, h = nh - n * H;
    const int w0 = tw * kNhwcCols, c0 = ch * kNhwcChans;
    const int cols = min(kNhwcCols, W - w0), cc = min(kNhwcChans, C - c0);
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    const int32_t *a = acc + (((int64_t)n * C + c0) * H + h) * W + w0 + lane;
    const int64_t cstride = (int64_t)H * W;
#pragma unroll 4
    for (int c = wave; c < cc; c += kBlock / 64)
        if (lane < cols) tile[c * kPitch + lane] = (uint8_t)requant(a[c * cstride], shift, bits);
    __syncthreads();
    // pixel j's channels c0 .. c0 + cc - 1 sit at dst[pix0 + j C + c0 ...]
    const int64_t pix0 = ((int64_t)nh * W + w0) * C + c0;
    const bool words = (cc & 3) == 0 && (C & 3) == 0 && (((uintptr_t)dst + pix0) & 3) == 0;
    if (words) {
        const int per = cc >> 2;   // 32-bit words per pixel
        for (int k = threadIdx.x; k < cols * per; k += kBlock) {
            const int j = k / per, c = (k - j * per) << 2;
            const uint32_t v = (uint32_t)tile[c * kPitch + j] | ((uint32_t)tile[(c + 1) * kPitch + j] << 8) |
                               ((uint32_t)tile[(c + 2) * kPitch + j] << 16) |
                               ((uint32_t)tile[(c + 3) * kPitch + j] << 24);
            *(uint32_t *)(dst + pix0 + (int64_t)j * C + c) = v;
        }
    } else {
        for (int k = threadIdx.x; k < cols * cc; k += kBlock) {
            const int j = k / cc, c = k - j * cc;
            dst[pix0 + (int64_t)j * C + c] = tile[c * kPitch + j];
        }
    }
}

}  // namespace

int launch_max_i32(const int32_t *src, int64_t n, int32_t *dev_max, hipStream_t s) {
    hipLaunchKernelGGL(max_init_kernel, dim3(1), dim3(64), 0, s, dev_max);
    int st = check_launch("max init");
    if (st) return st;
    const int grid = std::min(grid_for((n + 15) / 16, kBlock), kMaxGrid);   // ~16 values per thread or more
    hipLaunchKernelGGL(max_kernel, dim3(grid), dim3(kBlock), 0, s, src, n, dev_max);
    return check_launch("max");
}

int launch_count_mismatch(const int32_t *a, const int32_t *b, int64_t n, int32_t *count, hipStream_t s) {
    hipLaunchKernelGGL(zero_count_kernel, dim3(1), dim3(64), 0, s, count);
    int st = check_launch("mismatch count init");
    if (st) return st;
    const int grid = std::max(1, std::min(grid_for(n, kBlock), 2048));
    hipLaunchKernelGGL(mismatch_kernel, dim3(grid), dim3(kBlock), 0, s, a, b, n, count);
    return check_launch("mismatch count");
}

int launch_relu_requant_pack(const int32_t *acc, int64_t rows, int64_t len, const int32_t *dev_max, int bits,
                             uint32_t *dst, int32_t *dev_shift, hipStream_t s) {
    const int64_t wpr = row_words(len, bits);
    if (len <= kPackVals) {
        const int rpb = (int)(kPackVals / len);
        const int64_t grid = (rows + rpb - 1) / rpb;
        if (grid > INT32_MAX) {
            set_error("relu_requant_pack: too many rows");
            return SAMD_EUNSUPPORTED;
        }
#define SAMD_REQ_CASE(B)                                                                                          \
        if (bits == B) {                                                                                          \
            hipLaunchKernelGGL((relu_requant_pack_kernel<B>), dim3((unsigned)grid), dim3(kBlock), 0, s, acc, rows, \
                               (int32_t)len, (int32_t)wpr, rpb, dev_max, dst, dev_shift);                         \
            return check_launch("relu_requant_pack");                                                             \
        }
        SAMD_REQ_CASE(1) SAMD_REQ_CASE(2) SAMD_REQ_CASE(3) SAMD_REQ_CASE(4)
        SAMD_REQ_CASE(5) SAMD_REQ_CASE(6) SAMD_REQ_CASE(7) SAMD_REQ_CASE(8)
#undef SAMD_REQ_CASE
    } else {
        const int grid = grid_for(rows * wpr, kBlock);
#define SAMD_REQ_CASE(B)                                                                                          \
        if (bits == B) {                                                                                          \
            hipLaunchKernelGGL((relu_requant_pack_long_kernel<B>), dim3(grid), dim3(kBlock), 0, s, acc, rows, len, \
                               wpr, dev_max, dst, dev_shift);                                                     \
            return check_launch("relu_requant_pack");                                                             \
        }
        SAMD_REQ_CASE(1) SAMD_REQ_CASE(2) SAMD_REQ_CASE(3) SAMD_REQ_CASE(4)
        SAMD_REQ_CASE(5) SAMD_REQ_CASE(6) SAMD_REQ_CASE(7) SAMD_REQ_CASE(8)
#undef SAMD_REQ_CASE
    }
    set_error("relu_requant_pack: unsupported bits");
    return SAMD_EINVAL;
}

int launch_relu_requant_stage(const int32_t *acc, const int32_t *dev_max, const Conv2dGeom &g, void *ws,
                              int32_t *dev_shift, hipStream_t s, int32_t *dst) {
    int32_t *xs = dst ? dst : (int32_t *)((char *)ws + conv2d_xs_offset(g));
    const int qshift = spread_qshift(g.nq);   // ~2.5 words per thread, as the spread
    const int64_t nrows = (int64_t)g.N * g.C * g.Hp;
    const int rpb = kBlock >> qshift;
    const int64_t blocks = (nrows + rpb - 1) / rpb;   // one thread group per row, no grid-stride loop
    // the planner refuses layers that would need 2^32 threads or more (addressable())
    if (blocks * kBlock > (int64_t)0xffffffff) {
        set_error("relu_requant_stage: more than 2^32 threads in one launch");
        return SAMD_EUNSUPPORTED;
    }
    hipLaunchKernelGGL(relu_requant_stage_kernel, dim3((unsigned)blocks), dim3(kBlock), 0, s, acc, dev_max, g, qshift,
                       xs, dev_shift);
    return check_launch("relu_requant_stage");
}

int launch_relu_requant_nhwc_u8(const int32_t *acc, int N, int C, int H, int W, const int32_t *dev_max, int bits,
                                uint8_t *dst, hipStream_t s) {
    const int64_t grid = (int64_t)N * H * ((W + kNhwcCols - 1) / kNhwcCols) * ((C + kNhwcChans - 1) / kNhwcChans);
    if (grid > INT32_MAX) {
        set_error("relu_requant_nhwc_u8: too many image rows");
        return SAMD_EUNSUPPORTED;
    }
    hipLaunchKernelGGL(relu_requant_nhwc_kernel, dim3((unsigned)grid), dim3(kBlock), 0, s, acc, N, C, H, W, dev_max,
                       bits, dst);
    return check_launch("relu_requant_nhwc_u8");
}

}  // namespace samd
