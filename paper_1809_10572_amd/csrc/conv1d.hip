// Standalone SAMD 1-D convolution (Sec. 5): unsigned b-bit input, unsigned kernel.
//
// Operand word for output word q and kernel group g: A = sum_i x[q*I + delta_g + i] 2^(i L)
// (I values with L - b temporary spacer bits above each).  Kernel word B_g holds the
// group's taps in natural order, one per lane.  One 32x32 -> 64-bit multiply per group
// gives lanes j = 0 .. I+K-2, lane j holding the partial full-convolution sum for output
// q*I + j - (K - 1) (the "parallelogram" of Sec. 5.1).  An output's complete value is its
// lane in word q plus the low lanes of the following words (overlap-add); each thread
// recomputes those few following products instead of exchanging them.
#include <hip/hip_runtime.h>

#include "hip_util.hpp"

namespace samd {

namespace {

constexpr int kBlock = 256;
constexpr int kMaxExtra = kMaxConv1dExtra;

template <int B>
__device__ inline uint32_t field(const uint32_t *__restrict__ x, int64_t n, int64_t u) {
    constexpr int P = 32 / B;
    if (u < 0 || u >= n) return 0u;
    return (x[u / P] >> ((u % P) * B)) & ((1u << B) - 1);
}

template <int B>
__global__ __launch_bounds__(kBlock) void conv1d_kernel(const uint32_t *__restrict__ x, int32_t *__restrict__ y,
                                                        Conv1dGeom g) {
    const int64_t q = (int64_t)blockIdx.x * kBlock + threadIdx.x;
    if (q >= g.nwords) return;
    const int I = g.I, L = g.L, K = g.K;
    const int nl = g.nl;
    uint64_t acc[kMaxExtra + 1];
#pragma unroll
    for (int e = 0; e <= kMaxExtra; ++e) {
        acc[e] = 0;
        if (e <= g.extra) {
            const int64_t base = (q + e) * I;
            for (int gi = 0; gi < g.ngroups; ++gi) {
                uint32_t A = 0;
                for (int i = 0; i < I; ++i) A |= field<B>(x, g.n, base + g.g_delta[gi] + i) << (i * L);
                acc[e] += (uint64_t)A * g.g_word[gi];
            }
        }
    }
    const uint64_t lmask = (L >= 64) ? ~0ull : ((1ull << L) - 1);
    const int64_t o0 = q * I;
    for (int r = 0; r < I; ++r) {
        const int64_t o = o0 + r;
        if (o >= g.nout) break;
        uint64_t sum = 0;
#pragma unroll
        for (int e = 0; e <= kMaxExtra; ++e) {
            const int j = r + K - 1 - e * I;
            if (e <= g.extra && j >= 0 && j < nl) {
                const uint64_t v = acc[e] >> (j * L);
                sum += (j == nl - 1) ? v : (v & lmask);
            }
        }
        y[o] = (int32_t)sum;
    }
}

}  // namespace

int launch_conv1d(const uint32_t *x, const Conv1dGeom &g, int32_t *y, hipStream_t s) {
    const int grid = (int)((g.nwords + kBlock - 1) / kBlock);
#define SAMD_C1_CASE(B)                                                                                  \
    if (g.bits == B) {                                                                                   \
        hipLaunchKernelGGL((conv1d_kernel<B>), dim3(grid), dim3(kBlock), 0, s, x, y, g);                \
        return check_launch("conv1d");                                                                   \
    }
    SAMD_C1_CASE(1) SAMD_C1_CASE(2) SAMD_C1_CASE(3) SAMD_C1_CASE(4)
    SAMD_C1_CASE(5) SAMD_C1_CASE(6) SAMD_C1_CASE(7) SAMD_C1_CASE(8)
#undef SAMD_C1_CASE
    set_error("conv1d: unsupported bits");
    return SAMD_EINVAL;
}

}  // namespace samd
