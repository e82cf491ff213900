// Standalone SAMD 1-D convolution (Sec. 5): unsigned b-bit input, unsigned kernel.
//
// Operand word for output word q and kernel group g: A = sum_i x[q*I + delta_g + i] 2^(i L)
// (I values with L - b temporary spacer bits above each).  Kernel word B_g holds the
// group's taps in natural order, one per lane.  One 32x32 -> 64-bit multiply per group
// gives lanes j = 0 .. I+K-2, lane j holding the partial full-convolution sum for output
// q*I + j - (K - 1) (the "parallelogram" of Sec. 5.1); the groups' lanes line up, so
// their products add into one 64-bit word P_q.  An output's complete value is its lane in
// P_q plus the low lanes of the following words' products (overlap-add).
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cstdint>

#include "hip_util.hpp"

namespace samd {

namespace {

constexpr int kBlock = 256;

// Lane j of the 64-bit product (lo, hi), j L < 64; the highest non-zero lane (nl - 1)
// takes all the remaining bits, every other lane L of them.  Arguments other than the
// product are uniform: the selection compiles to scalar code.
__device__ __forceinline__ uint32_t lane_of(uint32_t lo, uint32_t hi, int j, int L, int nl, uint32_t lmask) {
    const int sh = j * L;
    const uint32_t v = sh < 32 ? __builtin_amdgcn_alignbit(hi, lo, sh) : hi >> (sh - 32);
    return j < nl - 1 ? v & lmask : v;
}

// One thread per output word and row (I <= 4 values per word, IM >= I a compile-time
// bound the per-output registers are unrolled over).  Each (row, wave) stores the
// outputs of own = 64 - extra consecutive words; the last `extra` lanes of each compute
// the products of the following words only, which the storing lanes read with
// whole-wave lane shifts for the overlap-add.  A lane works on kRows rows, which share
// every scalar decision (which lane of which product an output takes).
//   1. The workgroup copies the packed words its lanes read into LDS, with words outside
//      the row and fields past its end cleared (coalesced loads, the only wait on
//      memory).
//   2. Each lane builds its words' operand words per group from the (at most two)
//      packed words its I values occupy, multiplies and sums the groups' products.
//   3. Overlap-add through whole-wave lane shifts; a lane's I outputs are stored next to
//      those of its neighbours.
// Per-lane index arithmetic is 32-bit; 64-bit positions are per workgroup (scalar).
constexpr int kRows = 2;

template <int B, int IM>
__global__ __launch_bounds__(kBlock) void conv1d_kernel(const uint32_t *__restrict__ x, int32_t *__restrict__ y,
                                                        const Conv1dGeom g, int dmin, int nwin, bool aligned) {
    constexpr int P = 32 / B;   // fields per packed word
    constexpr uint32_t vmask = (1u << B) - 1;
    constexpr uint32_t wmask = P * B == 32 ? 0xffffffffu : (1u << (P * B)) - 1;   // the P fields
    constexpr int kWaves = kBlock / 64, R = kRows;
    extern __shared__ uint32_t pk[];   // nwin + 1 packed words
    const int I = g.I, L = g.L, K = g.K, nl = g.nl, extra = g.extra;
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6, own = 64 - extra;
    const int64_t qb = (int64_t)blockIdx.x * (R * kWaves) * own;   // the workgroup's first word
    // field 0 of pk[0] holds value ub - fb (fb < P): the workgroup's first value ub
    const int64_t ub = qb * I + dmin;
    const int64_t kb = ub >= 0 ? ub / P : -((P - 1 - ub) / P);
    const int fb = (int)(ub - kb * P);
    {
        const int64_t wlast = (g.n - 1) / P;   // packed word of the row's last value
        const int keep = (int)((g.n - 1) - wlast * P + 1);
        for (int k = tid; k <= nwin; k += kBlock) {
            const int64_t wi = kb + k;
            uint32_t v = 0;
            if (wi >= 0 && wi <= wlast) {
                v = x[wi] & wmask;
                if (wi == wlast && keep < P) v &= (1u << (keep * B)) - 1;
            }
            pk[k] = v;
        }
    }
    __syncthreads();
    const uint32_t fmask = I * B >= 32 ? 0xffffffffu : (1u << (I * B)) - 1;   // I fields
    int r0[R];   // field of value q I relative to pk[0]'s field 0, per row
#pragma unroll
    for (int r = 0; r < R; ++r) r0[r] = fb + ((r * kWaves + wave) * own + lane) * I - dmin;
    uint64_t prod[R] = {};
    for (int gi = 0; gi < g.ngroups; ++gi) {
        const uint32_t word = g.g_word[gi];
        const int delta = g.g_delta[gi];
#pragma unroll
        for (int r = 0; r < R; ++r) {
            const int f = r0[r] + delta;
            const int k = f / P, fk = f - k * P;
            const uint32_t w0 = pk[k], w1 = pk[k + 1];
            // the two words' fields back to back (w0 has no bits above its P fields)
            uint32_t clo = w0, chi = w1;
            if constexpr (P * B < 32) {
                clo = w0 | (w1 << (P * B));
                chi = w1 >> (32 - P * B);
            }
            const uint32_t bits = __builtin_amdgcn_alignbit(chi, clo, fk * B) & fmask;
            // spread: field i to bit i L (fields past the I-th are zero, whatever their shift)
            uint32_t A = bits & vmask;
#pragma unroll
            for (int i = 1; i < IM; ++i) A |= ((bits >> (i * B)) & vmask) << ((i * L) & 31);
            prod[r] += (uint64_t)A * word;
        }
    }
    const uint32_t lmask = L >= 32 ? 0xffffffffu : (1u << L) - 1;
    uint32_t lo[R], hi[R], out[R][IM];
#pragma unroll
    for (int r = 0; r < R; ++r) {
        lo[r] = (uint32_t)prod[r];
        hi[r] = (uint32_t)(prod[r] >> 32);
    }
#pragma unroll
    for (int t = 0; t < IM; ++t) {
        const int j = t + K - 1;
        const bool take = t < I && j < nl;
#pragma unroll
        for (int r = 0; r < R; ++r) out[r][t] = take ? lane_of(lo[r], hi[r], j, L, nl, lmask) : 0u;
    }
    // the product of the word e lanes up: e whole-wave shifts by one lane (DPP wave_shl,
    // a register move; the top lanes receive zeros and store nothing)
    uint32_t elo[R], ehi[R];
#pragma unroll
    for (int r = 0; r < R; ++r) {
        elo[r] = lo[r];
        ehi[r] = hi[r];
    }
    for (int e = 1; e <= extra; ++e) {
#pragma unroll
        for (int r = 0; r < R; ++r) {
            elo[r] = (uint32_t)__builtin_amdgcn_update_dpp(0, (int)elo[r], 0x130, 0xf, 0xf, false);
            ehi[r] = (uint32_t)__builtin_amdgcn_update_dpp(0, (int)ehi[r], 0x130, 0xf, 0xf, false);
        }
#pragma unroll
        for (int t = 0; t < IM; ++t) {
            const int j = t + K - 1 - e * I;
            if (t < I && j >= 0 && j < nl) {
#pragma unroll
                for (int r = 0; r < R; ++r) out[r][t] += lane_of(elo[r], ehi[r], j, L, nl, lmask);
            }
        }
    }
    if (lane < own) {
#pragma unroll
        for (int r = 0; r < R; ++r) {
            const int64_t o = (qb + (r * kWaves + wave) * own + lane) * I;
            // I = 2, 3 or 4 with y 16-byte aligned: the lane's outputs in one 8-, 12- or 16-byte
            // store (o is a multiple of I, so the store is aligned to its element count's
            // power of two, or to 4 bytes for 3); otherwise, and at the row's end, one by one
            if constexpr (IM == 2 || IM == 4) {
                if (I >= IM - 1 && I > 1 && aligned && o + I <= g.nout) {
                    if constexpr (IM == 2) {
                        *(uint2 *)(y + o) = uint2{out[r][0], out[r][1]};
                    } else if (I == 4) {
                        *(uint4 *)(y + o) = uint4{out[r][0], out[r][1], out[r][2], out[r][3]};
                    } else {
                        *(uint3 *)(y + o) = uint3{out[r][0], out[r][1], out[r][2]};
                    }
                    continue;
                }
            }
#pragma unroll
            for (int t = 0; t < IM; ++t)
                if (t < I && o + t < g.nout) y[o + t] = (int32_t)out[r][t];
        }
    }
}

}  // namespace

int launch_conv1d(const uint32_t *x, const Conv1dGeom &g, int32_t *y, hipStream_t s) {
    const int own = 64 - g.extra;
    const int64_t per_block = (int64_t)kRows * (kBlock / 64) * own;
    const int64_t grid = (g.nwords + per_block - 1) / per_block;
    if (g.extra >= 64 || g.I > kConv1dMaxLanes || grid > INT32_MAX) {
        set_error("conv1d: row too long");
        return SAMD_EUNSUPPORTED;
    }
    int dmin = 0, dmax = 0;
    for (int gi = 0; gi < g.ngroups; ++gi) {
        dmin = std::min(dmin, g.g_delta[gi]);
        dmax = std::max(dmax, g.g_delta[gi]);
    }
    // fields the workgroup reads from pk[0]'s field 0: below fb + kRows 256 I + dmax - dmin
    const int P = 32 / g.bits;
    const int fields = (P - 1) + kRows * kBlock * g.I + dmax - dmin;
    const int nwin = (fields + P - 1) / P;
    const size_t shm = (size_t)(nwin + 1) * 4;
    const int im = g.I <= 1 ? 1 : g.I <= 2 ? 2 : 4;
    const bool aligned = ((uintptr_t)y & 15) == 0;
#define SAMD_C1_CASE(B)                                                                                        \
    if (g.bits == B) {                                                                                         \
        if (im == 1)                                                                                           \
            hipLaunchKernelGGL((conv1d_kernel<B, 1>), dim3((unsigned)grid), dim3(kBlock), shm, s, x, y, g, dmin, nwin, aligned); \
        else if (im == 2)                                                                                      \
            hipLaunchKernelGGL((conv1d_kernel<B, 2>), dim3((unsigned)grid), dim3(kBlock), shm, s, x, y, g, dmin, nwin, aligned); \
        else                                                                                                   \
            hipLaunchKernelGGL((conv1d_kernel<B, 4>), dim3((unsigned)grid), dim3(kBlock), shm, s, x, y, g, dmin, nwin, aligned); \
        return check_launch("conv1d");                                                                         \
    }
    SAMD_C1_CASE(1) SAMD_C1_CASE(2) SAMD_C1_CASE(3) SAMD_C1_CASE(4)
    SAMD_C1_CASE(5) SAMD_C1_CASE(6) SAMD_C1_CASE(7) SAMD_C1_CASE(8)
#undef SAMD_C1_CASE
    set_error("conv1d: unsupported bits");
    return SAMD_EINVAL;
}

}  // namespace samd
