// Native 8-bit baseline (Sec. 7): the same convolution on values unpacked to 8 bits,
// as an implicit GEMM on the gfx950 int8 matrix cores (v_mfma_i32_16x16x64_i8).
//
// GEMM view: D[m][p] = sum_k Wr[m][k] * X[k][p] with p an output position (n, ho, wo)
// and k = (ky, kx, c); weights are reordered once per call to [M][KH][KW][Cp] (Cp = C
// rounded up to 64) and activations are read in NHWC, so every lane fetches 16
// consecutive channels with one 128-bit load.  Unsigned 8-bit activations do not fit
// int8; they enter as v - 128 and the product gains 128 * (sum of the weights whose
// input lies inside the image) back in the epilogue.
#include <hip/hip_runtime.h>

#include "hip_util.hpp"

namespace samd {

namespace {

typedef int v4i __attribute__((ext_vector_type(4)));

struct I8Geom {
    int N, C, H, W, M, KH, KW, sh, sw, ph, pw, Ho, Wo;
    int Cp;          // channels padded to 64
    int Mp;          // output channels padded to 64
    int zero_point;  // 1: unsigned 8-bit activations, shifted by -128
    int64_t P;       // output positions N * Ho * Wo
};

// Reorder weights to [Mp][KH][KW][Cp] int8 (zero padded) and, for the zero-point path,
// per-(m, ky, kx) channel sums plus per-m totals.
__global__ __launch_bounds__(256) void i8_prep_kernel(const int8_t *__restrict__ w, const I8Geom g,
                                                      int8_t *__restrict__ wr, int32_t *__restrict__ wsum,
                                                      int32_t *__restrict__ wtot) {
    const int64_t total = (int64_t)g.Mp * g.KH * g.KW * g.Cp;
    for (int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x; i < total; i += (int64_t)gridDim.x * 256) {
        const int c = (int)(i % g.Cp);
        int64_t t = i / g.Cp;
        const int kx = (int)(t % g.KW);
        t /= g.KW;
        const int ky = (int)(t % g.KH);
        const int m = (int)(t / g.KH);
        int8_t v = 0;
        if (m < g.M && c < g.C) v = w[(((int64_t)m * g.C + c) * g.KH + ky) * g.KW + kx];
        wr[i] = v;
    }
    if (!g.zero_point) return;
    const int64_t nsum = (int64_t)g.M * g.KH * g.KW;
    for (int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x; i < nsum; i += (int64_t)gridDim.x * 256) {
        const int kx = (int)(i % g.KW);
        const int64_t t = i / g.KW;
        const int ky = (int)(t % g.KH);
        const int m = (int)(t / g.KH);
        int32_t s = 0;
        for (int c = 0; c < g.C; ++c) s += w[(((int64_t)m * g.C + c) * g.KH + ky) * g.KW + kx];
        wsum[i] = s;
    }
    for (int64_t m = (int64_t)blockIdx.x * 256 + threadIdx.x; m < g.M; m += (int64_t)gridDim.x * 256) {
        int32_t s = 0;
        for (int c = 0; c < g.C; ++c)
            for (int k = 0; k < g.KH * g.KW; ++k) s += w[((int64_t)m * g.C + c) * g.KH * g.KW + k];
        wtot[m] = s;
    }
}

// 16 channels [c, c + 16) of one input pixel, as int8 (zero outside the image / channels).
template <bool VEC>
__device__ inline v4i load_pixel16(const uint8_t *__restrict__ x, const I8Geom &g, int n, int hi, int wi, int c,
                                   bool inside, uint32_t flip) {
    v4i r = {0, 0, 0, 0};
    if (!inside || c >= g.C) return r;
    const uint8_t *p = x + (((int64_t)n * g.H + hi) * g.W + wi) * g.C + c;
    if (VEC) {
        r = *(const v4i *)p;
        r ^= (int)flip;
    } else {
        uint32_t b[4] = {0, 0, 0, 0};
        for (int e = 0; e < 16; ++e)
            if (c + e < g.C) b[e >> 2] |= ((uint32_t)p[e] ^ (flip & 0xff)) << ((e & 3) * 8);
        r = v4i{(int)b[0], (int)b[1], (int)b[2], (int)b[3]};
    }
    return r;
}

// Workgroup: 4 waves, 64 output channels x 64 positions; wave w owns channels
// [32*(w/2), +32) and positions [32*(w%2), +32) as 2 x 2 MFMA tiles of 16 x 16.
template <bool VEC>
__global__ __launch_bounds__(256) void conv2d_i8_kernel(const uint8_t *__restrict__ x, const int8_t *__restrict__ wr,
                                                        const int32_t *__restrict__ wsum,
                                                        const int32_t *__restrict__ wtot, int32_t *__restrict__ y,
                                                        const I8Geom g) {
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    const int li = lane & 15, lg = lane >> 4;
    const int m_base = blockIdx.y * 64 + (wave >> 1) * 32;
    const int64_t p_base = (int64_t)blockIdx.x * 64 + (wave & 1) * 32;
    const uint32_t flip = g.zero_point ? 0x80808080u : 0u;

    // the two positions this lane feeds into B (columns li of the two position tiles)
    int pn[2], pho[2], pwo[2];
    bool pvalid[2];
    for (int t = 0; t < 2; ++t) {
        const int64_t p = p_base + t * 16 + li;
        pvalid[t] = p < g.P;
        const int64_t pp = pvalid[t] ? p : 0;
        pwo[t] = (int)(pp % g.Wo);
        const int64_t r = pp / g.Wo;
        pho[t] = (int)(r % g.Ho);
        pn[t] = (int)(r / g.Ho);
    }
    v4i acc[2][2];
    for (int a = 0; a < 2; ++a)
        for (int b = 0; b < 2; ++b) acc[a][b] = v4i{0, 0, 0, 0};

    const int cstep = 64;
    for (int ky = 0; ky < g.KH; ++ky) {
        for (int kx = 0; kx < g.KW; ++kx) {
            int hi[2], wi[2];
            bool inside[2];
            for (int t = 0; t < 2; ++t) {
                hi[t] = pho[t] * g.sh + ky - g.ph;
                wi[t] = pwo[t] * g.sw + kx - g.pw;
                inside[t] = pvalid[t] && hi[t] >= 0 && hi[t] < g.H && wi[t] >= 0 && wi[t] < g.W;
            }
            const int8_t *wk = wr + ((int64_t)ky * g.KW + kx) * g.Cp;
            for (int c0 = 0; c0 < g.Cp; c0 += cstep) {
                const int c = c0 + lg * 16;
                v4i A[2], B[2];
                for (int t = 0; t < 2; ++t) {
                    const int m = m_base + t * 16 + li;
                    A[t] = *(const v4i *)(wk + (int64_t)m * g.KH * g.KW * g.Cp + c);
                    B[t] = load_pixel16<VEC>(x, g, pn[t], hi[t], wi[t], c, inside[t], flip);
                }
                for (int a = 0; a < 2; ++a)
                    for (int b = 0; b < 2; ++b)
                        acc[a][b] = __builtin_amdgcn_mfma_i32_16x16x64_i8(A[a], B[b], acc[a][b], 0, 0, 0);
            }
        }
    }
    // D[row][col]: lane holds rows 4*lg + v (output channels), column li (position)
    for (int b = 0; b < 2; ++b) {
        if (!pvalid[b]) continue;
        const int n = pn[b], ho = pho[b], wo = pwo[b];
        const bool interior = ho * g.sh - g.ph >= 0 && ho * g.sh - g.ph + g.KH <= g.H && wo * g.sw - g.pw >= 0 &&
                              wo * g.sw - g.pw + g.KW <= g.W;
        for (int a = 0; a < 2; ++a) {
            for (int v = 0; v < 4; ++v) {
                const int m = m_base + a * 16 + lg * 4 + v;
                if (m >= g.M) continue;
                int32_t val = acc[a][b][v];
                if (g.zero_point) {
                    int32_t s = 0;
                    if (interior) {
                        s = wtot[m];
                    } else {
                        for (int ky = 0; ky < g.KH; ++ky) {
                            const int hi = ho * g.sh + ky - g.ph;
                            if (hi < 0 || hi >= g.H) continue;
                            for (int kx = 0; kx < g.KW; ++kx) {
                                const int wi = wo * g.sw + kx - g.pw;
                                if (wi >= 0 && wi < g.W) s += wsum[((int64_t)m * g.KH + ky) * g.KW + kx];
                            }
                        }
                    }
                    val += 128 * s;
                }
                y[(((int64_t)n * g.M + m) * g.Ho + ho) * g.Wo + wo] = val;
            }
        }
    }
}

I8Geom make_geom(const samd_conv2d_desc &d, samd_fmt xf) {
    I8Geom g;
    g.N = d.N; g.C = d.C; g.H = d.H; g.W = d.W; g.M = d.M; g.KH = d.KH; g.KW = d.KW;
    g.sh = d.stride_h; g.sw = d.stride_w; g.ph = d.pad_h; g.pw = d.pad_w;
    g.Ho = (d.H + 2 * d.pad_h - d.KH) / d.stride_h + 1;
    g.Wo = (d.W + 2 * d.pad_w - d.KW) / d.stride_w + 1;
    g.Cp = (d.C + 63) / 64 * 64;
    g.Mp = (d.M + 63) / 64 * 64;
    g.zero_point = (!xf.is_signed && xf.bits == 8) ? 1 : 0;
    g.P = (int64_t)d.N * g.Ho * g.Wo;
    return g;
}

size_t align256(size_t v) { return (v + 255) / 256 * 256; }

}  // namespace

size_t conv2d_i8_workspace_bytes(const samd_conv2d_desc &d, samd_fmt xf) {
    I8Geom g = make_geom(d, xf);
    size_t wr = align256((size_t)g.Mp * g.KH * g.KW * g.Cp);
    size_t sums = align256((size_t)g.M * g.KH * g.KW * 4);
    size_t tot = align256((size_t)g.M * 4);
    return wr + sums + tot;
}

namespace {

struct I8Workspace {
    int8_t *wr;
    int32_t *wsum, *wtot;
};

I8Workspace carve(const I8Geom &g, void *ws) {
    I8Workspace w;
    w.wr = (int8_t *)ws;
    w.wsum = (int32_t *)((char *)ws + align256((size_t)g.Mp * g.KH * g.KW * g.Cp));
    w.wtot = (int32_t *)((char *)w.wsum + align256((size_t)g.M * g.KH * g.KW * 4));
    return w;
}

}  // namespace

int launch_conv2d_i8_prepare(const int8_t *w, samd_fmt xf, const samd_conv2d_desc &d, void *ws, hipStream_t s) {
    const I8Geom g = make_geom(d, xf);
    const I8Workspace p = carve(g, ws);
    const int pgrid = grid_for((int64_t)g.Mp * g.KH * g.KW * g.Cp, 256);
    hipLaunchKernelGGL(i8_prep_kernel, dim3(pgrid), dim3(256), 0, s, w, g, p.wr, p.wsum, p.wtot);
    return check_launch("conv2d_int8 weight reorder");
}

int launch_conv2d_i8(const void *x, samd_fmt xf, const samd_conv2d_desc &d, int32_t *y, const void *ws,
                     hipStream_t s) {
    const I8Geom g = make_geom(d, xf);
    const I8Workspace p = carve(g, const_cast<void *>(ws));
    const dim3 grid((unsigned)((g.P + 63) / 64), g.Mp / 64);
    const bool vec = (g.C % 16) == 0 && ((uintptr_t)x % 16) == 0;
    if (vec)
        hipLaunchKernelGGL((conv2d_i8_kernel<true>), grid, dim3(256), 0, s, (const uint8_t *)x, p.wr, p.wsum,
                           p.wtot, y, g);
    else
        hipLaunchKernelGGL((conv2d_i8_kernel<false>), grid, dim3(256), 0, s, (const uint8_t *)x, p.wr, p.wsum,
                           p.wtot, y, g);
    return check_launch("conv2d_int8");
}

}  // namespace samd
