// Standalone SAMD 1-D convolution (Sec. 5): unsigned b-bit input, unsigned kernel.
//
// Operand word for output word q and kernel group g: A = sum_i x[q*I + delta_g + i] 2^(i L)
// (I values with L - b temporary spacer bits above each).  Kernel word B_g holds the
// group's taps in natural order, one per lane.  One 32x32 -> 64-bit multiply per group
// gives lanes j = 0 .. I+K-2, lane j holding the partial full-convolution sum for output
// q*I + j - (K - 1) (the "parallelogram" of Sec. 5.1).  An output's complete value is its
// lane in word q plus the low lanes of the following words (overlap-add).
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cstdint>

#include "hip_util.hpp"

namespace samd {

namespace {

constexpr int kBlock = 256;

// The computation is staged through LDS, with the overlap-add done there.  A block of W = 256 threads owns output words q0 .. q0 + W - 1,
// i.e. outputs
// q0 I .. q0 I + W I - 1; word q's lanes reach outputs q I - (K - 1) .. q I + I - 1, so
// those outputs take lanes of words q0 .. q0 + W - 1 + extra.  The block
//   1. unpacks every value those words read into LDS (one value per thread and pass,
//      coalesced reads of the packed row, 32-bit indices, P a compile-time constant);
//   2. builds each word's operand words from LDS, multiplies them by the kernel words
//      (one 32x32 -> 64-bit product per tap group), and adds every lane into its output
//      in an LDS row (atomic adds: lanes of up to 1 + extra words meet in one output);
//   3. stores its W I outputs, coalesced.
// The extra words past the block's own are computed by its first threads (and again,
// as their own, by the next block).  LDS indices are skewed by one word per 16 (sk), so
// that the lanes of neighbouring words, I apart, fall in different banks.
__device__ __forceinline__ int sk(int i) { return i + (i >> 4); }

template <int B>
__global__ __launch_bounds__(kBlock) void conv1d_lds_kernel(const uint32_t *__restrict__ x, int32_t *__restrict__ y,
                                                            Conv1dGeom g, int dmin, int nvals, int nouts) {
    extern __shared__ uint32_t sh[];
    uint32_t *vals = sh;                              // nvals values
    uint32_t *outs = sh + sk(nvals);                  // nouts outputs; outs[sk(K - 1)] is output q0 I
    constexpr int P = 32 / B;
    const int I = g.I, L = g.L, K = g.K, nl = g.nl;
    const int W = blockDim.x;
    const int64_t q0 = (int64_t)blockIdx.x * W;
    const int64_t u0 = q0 * I + dmin;   // 64-bit: rows may hold more than 2^31 values
    for (int t = threadIdx.x; t < nvals; t += W) {
        const int64_t u = u0 + t;
        uint32_t f = 0;
        if (u >= 0 && u < g.n) f = (x[(uint64_t)u / P] >> (((uint64_t)u % P) * B)) & ((1u << B) - 1);
        vals[sk(t)] = f;
    }
    for (int t = threadIdx.x; t < sk(nouts); t += W) outs[t] = 0;
    __syncthreads();
    const uint64_t lmask = (1ull << L) - 1;   // L <= 32
    for (int w = threadIdx.x; w < W + g.extra; w += W) {
        if (q0 + w >= g.nwords + g.extra) break;   // words past the row only reach discarded outputs
        uint64_t p = 0;
        for (int gi = 0; gi < g.ngroups; ++gi) {
            const int v0 = w * I + g.g_delta[gi] - dmin;
            uint32_t A = 0;
            for (int i = 0; i < I; ++i) A |= vals[sk(v0 + i)] << (i * L);
            p += (uint64_t)A * g.g_word[gi];
        }
        // lane j of word w is output w I + j - (K - 1), at outs[sk(w I + j)]
        const int o = w * I;
        for (int j = 0; j < nl - 1; ++j) {
            atomicAdd(outs + sk(o + j), (uint32_t)(p & lmask));
            p >>= L;
        }
        atomicAdd(outs + sk(o + nl - 1), (uint32_t)p);
    }
    __syncthreads();
    const int64_t o0 = q0 * I;
    for (int t = threadIdx.x; t < W * I; t += W) {
        const int64_t o = o0 + t;
        if (o < g.nout) y[o] = (int32_t)outs[sk(t + K - 1)];
    }
}

}  // namespace

int launch_conv1d(const uint32_t *x, const Conv1dGeom &g, int32_t *y, hipStream_t s) {
    const int64_t grid = (g.nwords + kBlock - 1) / kBlock;
    if (grid > INT32_MAX) {
        set_error("conv1d: row too long");
        return SAMD_EUNSUPPORTED;
    }
    // the values a block reads: words q0 .. q0 + kBlock - 1 + extra, each from offset
    // delta_g of its window, I values per operand word
    int dmin = 0, dmax = 0;
    for (int gi = 0; gi < g.ngroups; ++gi) {
        dmin = std::min(dmin, g.g_delta[gi]);
        dmax = std::max(dmax, g.g_delta[gi]);
    }
    const int nvals = (kBlock + g.extra) * g.I + dmax - dmin;
    // lanes of words 0 .. kBlock + extra - 1 land at outs[w I + j], j < nl
    const int nouts = std::max((kBlock + g.extra - 1) * g.I + g.nl, kBlock * g.I + g.K - 1);
    const size_t shm = ((size_t)(nvals + (nvals >> 4) + 1) + (size_t)(nouts + (nouts >> 4) + 1)) * 4;
#define SAMD_C1_CASE(B)                                                                                   \
    if (g.bits == B) {                                                                                    \
        hipLaunchKernelGGL((conv1d_lds_kernel<B>), dim3((unsigned)grid), dim3(kBlock), shm, s, x, y, g, dmin, \
                           nvals, nouts);                                                                 \
        return check_launch("conv1d");                                                                    \
    }
    SAMD_C1_CASE(1) SAMD_C1_CASE(2) SAMD_C1_CASE(3) SAMD_C1_CASE(4)
    SAMD_C1_CASE(5) SAMD_C1_CASE(6) SAMD_C1_CASE(7) SAMD_C1_CASE(8)
#undef SAMD_C1_CASE
    set_error("conv1d: unsupported bits");
    return SAMD_EINVAL;
}

}  // namespace samd
