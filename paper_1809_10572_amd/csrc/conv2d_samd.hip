// SAMD 2-D convolution for gfx950: convolution by long multiplication (Sec. 5) with
// signed sign-extension and the underflow fix-up (Sec. 6).
//
// Workgroup = one image n, rows_blk output rows, mblk output channels; each of its wm
// waves owns kWaveM output channels, each lane one operand-word column q of one output
// row.  Per channel chunk the workgroup
//   1. copies the packed input rows it needs into LDS (coalesced),
//   2. spreads them into operand words: I values of one stride phase, L bits apart
//      (temporary spacer bits), negative values sign-extended - every operand word is
//      then the int32 sum_i v_i 2^(i L),
//   3. multiplies every operand word by the kernel words of its kernel rows and adds the
//      exact signed 32x32 -> 64-bit products into one accumulator per output channel
//      (v_mad_i64_i32; the kernel words are wave-uniform and come in through SGPRs).
// After every G channels each accumulator is decoded: the fix-up (add every lane's sign
// bit to itself, then xor it back) makes every lane its own two's-complement value, the
// lanes are extracted and added into an LDS tile of int32 outputs - which also performs
// the overlap-add of neighbouring words' partial lanes.  The tile is finally written to
// HBM row by row.
#include <hip/hip_runtime.h>

#include "hip_util.hpp"

namespace samd {

namespace {

constexpr int RM = kWaveM;

template <int B, bool S>
__device__ inline int32_t packed_field(const uint32_t *row, int col) {
    constexpr int P = 32 / B;
    const uint32_t f = (row[col / P] >> ((col % P) * B)) & ((1u << B) - 1);
    if (S) return (int32_t)(f << (32 - B)) >> (32 - B);
    return (int32_t)f;
}

// Kernel words, laid out [channel block][channel][kernel row x tap word][mblk] so that
// each wave reads its kWaveM words of one (channel, row-tap) as one contiguous run.
template <int B, bool S>
__global__ __launch_bounds__(256) void prep_weights_kernel(const uint32_t *__restrict__ w, const Conv2dGeom g,
                                                           int32_t *__restrict__ kw) {
    const int64_t total = (int64_t)g.nmb * g.C * g.nrt * g.mblk;
    for (int64_t idx = (int64_t)blockIdx.x * 256 + threadIdx.x; idx < total; idx += (int64_t)gridDim.x * 256) {
        const int mm = (int)(idx % g.mblk);
        int64_t t = idx / g.mblk;
        const int rt = (int)(t % g.nrt);
        t /= g.nrt;
        const int c = (int)(t % g.C);
        const int mb = (int)(t / g.C);
        const int m = mb * g.mblk + mm;
        uint32_t word = 0;
        if (m < g.M) {
            const int ky = rt / g.ntw, tw = rt % g.ntw;
            const uint32_t *row = w + ((int64_t)(m * g.C + c) * g.KH + ky) * g.wrw;
            const int k = g.tw_ntaps[tw], a0 = g.tw_tap0[tw], r = g.tw_phase[tw];
            for (int s = 0; s < k; ++s) {
                const int tap = g.sw * (a0 + k - 1 - s) + r;   // reversed: lane s holds tap a0+k-1-s
                word += (uint32_t)packed_field<B, S>(row, tap) << (s * g.L);
            }
        }
        kw[idx] = (int32_t)word;
    }
}

template <int B, bool S>
__global__ __launch_bounds__(256) void conv2d_samd_kernel(const uint32_t *__restrict__ x,
                                                          const int32_t *__restrict__ kw, int32_t *__restrict__ y,
                                                          const Conv2dGeom g) {
    extern __shared__ int32_t lds[];
    int32_t *tile = lds;
    int32_t *spread = lds + g.lds_tile;
    uint32_t *raw = (uint32_t *)(lds + g.lds_tile + g.lds_spread);

    const int tid = threadIdx.x;
    const int nthr = g.wm * 64;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int lane = tid & 63;
    const int ho0 = blockIdx.x * g.rows_blk;
    const int mb = blockIdx.y;
    const int n = blockIdx.z;
    const int rloc_raw = lane / g.nq;
    const bool active = rloc_raw < g.rows_blk && ho0 + rloc_raw < g.Ho;
    const int rloc = active ? rloc_raw : 0;
    const int q = active ? lane - rloc_raw * g.nq : 0;
    const int hin0 = ho0 * g.sh - g.ph;

    for (int i = tid; i < g.lds_tile; i += nthr) tile[i] = 0;

    int64_t acc[RM];
#pragma unroll
    for (int m = 0; m < RM; ++m) acc[m] = 0;
    int pending = 0;

    const int32_t *kwave = kw + (int64_t)mb * g.C * g.nrt * g.mblk + wave * RM;
    int32_t *tile_row = tile + ((wave * RM) * g.rows_blk + rloc) * g.Wo;
    const int tile_mstride = g.rows_blk * g.Wo;
    const int obase = q * g.I - g.Kmax + 1;

    auto decode = [&]() {
#pragma unroll
        for (int m = 0; m < RM; ++m) {
            uint64_t v = (uint64_t)acc[m];
            acc[m] = 0;
            if (g.result_signed) {
                const uint64_t s = v & g.msb_mask;
                v = (v + s) ^ s;
            }
            int32_t *trow = tile_row + m * tile_mstride;
            for (int j = 0; j < g.nl; ++j) {
                int32_t d;
                if (j < g.nl - 1) {
                    const uint32_t w32 = (uint32_t)(v >> (j * g.L));
                    d = g.result_signed ? ((int32_t)(w32 << (32 - g.L)) >> (32 - g.L))
                                        : (int32_t)(w32 & ((1u << g.L) - 1));
                } else {
                    d = g.result_signed ? (int32_t)((int64_t)v >> (j * g.L)) : (int32_t)(v >> (j * g.L));
                }
                const int o = obase + j;
                if (active && o >= 0 && o < g.Wo) atomicAdd(&trow[o], d);
            }
        }
    };

    for (int c0 = 0; c0 < g.C; c0 += g.cc) {
        const int ncc = min(g.cc, g.C - c0);
        __syncthreads();
        // 1. packed input rows of this channel chunk (zero rows above / below the image)
        const int nraw = ncc * g.trows * g.xrw;
        for (int i = tid; i < nraw; i += nthr) {
            const int wd = i % g.xrw;
            const int t = i / g.xrw;
            const int tr = t % g.trows, cc = t / g.trows;
            const int h = hin0 + tr;
            uint32_t v = 0;
            if (h >= 0 && h < g.H) v = x[(((int64_t)n * g.C + c0 + cc) * g.H + h) * g.xrw + wd];
            raw[i] = v;
        }
        __syncthreads();
        // 2. operand words: I values of stride phase r starting at phase index q*I + delta
        const int nsp = ncc * g.trows * g.nvar * g.nq;
        for (int i = tid; i < nsp; i += nthr) {
            const int qq = i % g.nq;
            int t = i / g.nq;
            const int v = t % g.nvar;
            t /= g.nvar;
            const uint32_t *row = raw + t * g.xrw;
            const int col0 = g.sw * (qq * g.I + g.var_delta[v]) + g.var_phase[v] - g.pw;
            uint32_t word = 0;
            for (int ii = 0; ii < g.I; ++ii) {
                const int col = col0 + g.sw * ii;
                if (col >= 0 && col < g.W) word += (uint32_t)packed_field<B, S>(row, col) << (ii * g.L);
            }
            spread[i] = (int32_t)word;
        }
        __syncthreads();
        // 3. multiply-accumulate: one v_mad_i64_i32 per (row-tap, output channel)
        for (int cc = 0; cc < ncc; ++cc) {
            const int32_t *kc = kwave + (int64_t)(c0 + cc) * g.nrt * g.mblk;
            const int32_t *sp = spread + (cc * g.trows + rloc * g.sh) * g.nvar * g.nq + q;
            int rt = 0;
            for (int ky = 0; ky < g.KH; ++ky) {
                for (int tw = 0; tw < g.ntw; ++tw, ++rt) {
                    const int32_t a = active ? sp[(ky * g.nvar + g.tw_var[tw]) * g.nq] : 0;
                    const int32_t *kr = kc + rt * g.mblk;
#pragma unroll
                    for (int m = 0; m < RM; ++m) acc[m] += (int64_t)a * (int64_t)kr[m];
                }
            }
            if (++pending == g.G) {
                decode();
                pending = 0;
            }
        }
    }
    if (pending) decode();
    __syncthreads();
    // 4. write the output tile, whole rows at a time
    const int tile_n = g.mblk * g.rows_blk * g.Wo;
    for (int i = tid; i < tile_n; i += nthr) {
        const int o = i % g.Wo;
        const int t = i / g.Wo;
        const int r = t % g.rows_blk, mm = t / g.rows_blk;
        const int m = mb * g.mblk + mm, ho = ho0 + r;
        if (m < g.M && ho < g.Ho) y[(((int64_t)n * g.M + m) * g.Ho + ho) * g.Wo + o] = tile[i];
    }
}

}  // namespace

int launch_conv2d_prepare(const uint32_t *w, const Conv2dGeom &g, void *ws, hipStream_t s) {
    int32_t *kw = (int32_t *)ws;
    const int64_t nkw = (int64_t)g.nmb * g.C * g.nrt * g.mblk;
    const int pgrid = grid_for(nkw, 256);
    bool launched = false;
#define SAMD_PREP_CASE(B, SG)                                                                            \
    if (!launched && g.wbits == B && (bool)g.wsigned == SG) {                                            \
        hipLaunchKernelGGL((prep_weights_kernel<B, SG>), dim3(pgrid), dim3(256), 0, s, w, g, kw);        \
        launched = true;                                                                                 \
    }
    SAMD_FOR_EACH_FMT(SAMD_PREP_CASE)
#undef SAMD_PREP_CASE
    return check_launch("conv2d weight preparation");
}

int launch_conv2d_samd(const uint32_t *x, const Conv2dGeom &g, int32_t *y, const void *ws, hipStream_t s) {
    const int32_t *kw = (const int32_t *)ws;
    const dim3 grid((g.Ho + g.rows_blk - 1) / g.rows_blk, g.nmb, g.N);
    const size_t shm = (size_t)(g.lds_tile + g.lds_spread + g.lds_raw) * 4;
    bool launched = false;
#define SAMD_CONV_CASE(B, SG)                                                                               \
    if (!launched && g.xbits == B && (bool)g.xsigned == SG) {                                               \
        hipLaunchKernelGGL((conv2d_samd_kernel<B, SG>), grid, dim3(g.wm * 64), shm, s, x, kw, y, g);        \
        launched = true;                                                                                    \
    }
    SAMD_FOR_EACH_FMT(SAMD_CONV_CASE)
#undef SAMD_CONV_CASE
    return check_launch("conv2d");
}

}  // namespace samd
