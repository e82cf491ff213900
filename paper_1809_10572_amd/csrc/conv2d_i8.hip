// Native 8-bit baseline (Sec. 7): the same convolution on values unpacked to 8 bits,
// as an implicit GEMM on the gfx950 int8 matrix cores (v_mfma_i32_16x16x64_i8), tiled
// through LDS.
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
    int Mp;          // output channels padded to 128
    int zero_point;  // 1: unsigned 8-bit activations, shifted by -128
    int64_t P;       // output positions N * Ho * Wo
};

// Reorder weights to [Mp][KH][KW][Cp] int8 (zero padded) and, for the zero-point path,
// per-m 2-D prefix sums of the channel-summed kernel (the correction of an output is the
// sum over its in-image taps: a rectangle, four lookups).
__global__ __launch_bounds__(256) void i8_prep_kernel(const int8_t *__restrict__ w, const I8Geom g,
                                                      int8_t *__restrict__ wr, int32_t *__restrict__ pre) {
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
    // pre[m][i][j] = sum of w[m][c][ky][kx] over all c, ky < i, kx < j (i <= KH, j <= KW)
    const int pw = (g.KH + 1) * (g.KW + 1);
    const int64_t npre = (int64_t)g.M * pw;
    for (int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x; i < npre; i += (int64_t)gridDim.x * 256) {
        const int m = (int)(i / pw), e = (int)(i - (int64_t)m * pw);
        const int ii = e / (g.KW + 1), jj = e - ii * (g.KW + 1);
        int32_t sum = 0;
        for (int c = 0; c < g.C; ++c)
            for (int ky = 0; ky < ii; ++ky)
                for (int kx = 0; kx < jj; ++kx) sum += w[(((int64_t)m * g.C + c) * g.KH + ky) * g.KW + kx];
        pre[i] = sum;
    }
}

// Workgroup tile: 128 output channels x 64 output positions, 4 waves of 64 x 32 (4 x 2
// MFMA tiles of 16 x 16).  Per K step (one kernel tap (ky, kx), 64 channels) the A tile
// (weights, 128 x 64 int8) and the B tile (activations of 64 positions, 64 x 64 int8)
// are staged in LDS, double-buffered; the 16-byte chunks of step k + 2 are loaded into
// registers while step k's MFMAs run and stored after step k + 1's (one barrier per
// step).  LDS rows are 64 bytes of data plus 16 of padding (fewer bank conflicts on the
// 16-byte reads).
constexpr int kTM = 128, kTP = 64, kKS = 64, kRowB = 80;
constexpr int kTileA = kTM * kRowB, kTileB = kTP * kRowB;   // bytes of the A and B tiles

// 16 bytes: channels [c, c + 16) of one input pixel as int8 (zero outside the image or
// past the channels); unsigned 8-bit activations are shifted by -128 (flip the top bit).
template <bool VEC>
__device__ inline v4i pixel16(const uint8_t *__restrict__ x, const I8Geom &g, int n, int hi, int wi, int c,
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

template <bool VEC>
__global__ __launch_bounds__(256) void conv2d_i8_kernel(const uint8_t *__restrict__ x, const int8_t *__restrict__ wr,
                                                        const int32_t *__restrict__ pre, int32_t *__restrict__ y,
                                                        const I8Geom g) {
    __shared__ __attribute__((aligned(16))) char sm[2 * (kTileA + kTileB)];   // A0, B0, A1, B1
    const int tid = threadIdx.x;
    const int lane = tid & 63, wave = tid >> 6;
    const int li = lane & 15, lg = lane >> 4;
    const int wy = wave >> 1, wx = wave & 1;   // wave tile: rows wy*64 .., positions wx*32 ..
    const int m0 = blockIdx.y * kTM;
    const int64_t p0 = (int64_t)blockIdx.x * kTP;
    const uint32_t flip = g.zero_point ? 0x80808080u : 0u;

    // staging: thread t moves 16-byte chunk (t & 3) of A rows t >> 2 and (t >> 2) + 64 and
    // of B row t >> 2
    const int qq = tid & 3, srow = tid >> 2;
    int sn, sho, swo;
    bool sval;
    {
        const int64_t p = p0 + srow;
        sval = p < g.P;
        const int64_t pp = sval ? p : 0;
        swo = (int)(pp % g.Wo);
        const int64_t r = pp / g.Wo;
        sho = (int)(r % g.Ho);
        sn = (int)(r / g.Ho);
    }
    const int csteps = g.Cp / kKS;
    const int nk = g.KH * g.KW * csteps;
    struct Chunk {
        v4i a[2], b;
    };
    auto load_step = [&](int k, Chunk &ch) {
        const int tap = k / csteps, c0 = (k - tap * csteps) * kKS + qq * 16;
        const int ky = tap / g.KW, kx = tap - ky * g.KW;
#pragma unroll
        for (int u = 0; u < 2; ++u)
            ch.a[u] = *(const v4i *)(wr + (((int64_t)(m0 + srow + u * 64) * g.KH + ky) * g.KW + kx) * g.Cp + c0);
        const int hi = sho * g.sh + ky - g.ph, wi = swo * g.sw + kx - g.pw;
        const bool inside = sval && hi >= 0 && hi < g.H && wi >= 0 && wi < g.W;
        ch.b = pixel16<VEC>(x, g, sn, hi, wi, c0, inside, flip);
    };
    auto store_step = [&](int buf, const Chunk &ch) {
        char *A = sm + buf * (kTileA + kTileB), *B = A + kTileA;
#pragma unroll
        for (int u = 0; u < 2; ++u) *(v4i *)(A + (srow + u * 64) * kRowB + qq * 16) = ch.a[u];
        *(v4i *)(B + srow * kRowB + qq * 16) = ch.b;
    };

    v4i acc[4][2];
#pragma unroll
    for (int a = 0; a < 4; ++a)
#pragma unroll
        for (int b = 0; b < 2; ++b) acc[a][b] = v4i{0, 0, 0, 0};

    Chunk c0, c1;
    load_step(0, c0);
    if (nk > 1) load_step(1, c1);
    store_step(0, c0);
    __syncthreads();
    for (int k = 0; k < nk; ++k) {
        // c1 holds step k + 1; load step k + 2 into c0 (free once step k was stored)
        if (k + 2 < nk) load_step(k + 2, c0);
        const char *A = sm + (k & 1) * (kTileA + kTileB), *B = A + kTileA;
        v4i fa[4], fb[2];
#pragma unroll
        for (int t = 0; t < 4; ++t) fa[t] = *(const v4i *)(A + (wy * 64 + t * 16 + li) * kRowB + lg * 16);
#pragma unroll
        for (int t = 0; t < 2; ++t) fb[t] = *(const v4i *)(B + (wx * 32 + t * 16 + li) * kRowB + lg * 16);
#pragma unroll
        for (int a = 0; a < 4; ++a)
#pragma unroll
            for (int b = 0; b < 2; ++b) acc[a][b] = __builtin_amdgcn_mfma_i32_16x16x64_i8(fa[a], fb[b], acc[a][b], 0, 0, 0);
        if (k + 1 < nk) store_step((k + 1) & 1, c1);
        c1 = c0;
        __syncthreads();
    }

    // D[row][col]: lane holds rows 4*lg + v (output channels) of column li (position).
    // Zero point: + 128 * (sum of the weights whose input lies inside the image), the
    // rectangle [ky0, ky1) x [kx0, kx1) of in-image taps of the position.
    const int pw = (g.KH + 1) * (g.KW + 1);
#pragma unroll
    for (int b = 0; b < 2; ++b) {
        const int64_t p = p0 + wx * 32 + b * 16 + li;
        if (p >= g.P) continue;
        const int wo = (int)(p % g.Wo);
        const int64_t r = p / g.Wo;
        const int ho = (int)(r % g.Ho), n = (int)(r / g.Ho);
        const int hb = ho * g.sh - g.ph, wb = wo * g.sw - g.pw;
        const int ky0 = max(0, -hb), ky1 = min(g.KH, g.H - hb);
        const int kx0 = max(0, -wb), kx1 = min(g.KW, g.W - wb);
        const int e11 = ky1 * (g.KW + 1) + kx1, e01 = ky0 * (g.KW + 1) + kx1;
        const int e10 = ky1 * (g.KW + 1) + kx0, e00 = ky0 * (g.KW + 1) + kx0;
        int32_t *yo = y + ((int64_t)n * g.M * g.Ho + ho) * g.Wo + wo;
#pragma unroll
        for (int a = 0; a < 4; ++a) {
#pragma unroll
            for (int v = 0; v < 4; ++v) {
                const int m = m0 + wy * 64 + a * 16 + lg * 4 + v;
                if (m >= g.M) continue;
                int32_t val = acc[a][b][v];
                if (g.zero_point) {
                    const int32_t *pm = pre + (int64_t)m * pw;
                    val += 128 * (pm[e11] - pm[e01] - pm[e10] + pm[e00]);
                }
                yo[(int64_t)m * g.Ho * g.Wo] = val;
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
    g.Mp = (d.M + 127) / 128 * 128;
    g.zero_point = (!xf.is_signed && xf.bits == 8) ? 1 : 0;
    g.P = (int64_t)d.N * g.Ho * g.Wo;
    return g;
}

size_t align256(size_t v) { return (v + 255) / 256 * 256; }

}  // namespace

size_t conv2d_i8_workspace_bytes(const samd_conv2d_desc &d, samd_fmt xf) {
    I8Geom g = make_geom(d, xf);
    size_t wr = align256((size_t)g.Mp * g.KH * g.KW * g.Cp);
    size_t pre = align256((size_t)g.M * (g.KH + 1) * (g.KW + 1) * 4);
    return wr + pre;
}

namespace {

struct I8Workspace {
    int8_t *wr;
    int32_t *pre;
};

I8Workspace carve(const I8Geom &g, void *ws) {
    I8Workspace w;
    w.wr = (int8_t *)ws;
    w.pre = (int32_t *)((char *)ws + align256((size_t)g.Mp * g.KH * g.KW * g.Cp));
    return w;
}

}  // namespace

int launch_conv2d_i8_prepare(const int8_t *w, samd_fmt xf, const samd_conv2d_desc &d, void *ws, hipStream_t s) {
    const I8Geom g = make_geom(d, xf);
    const I8Workspace p = carve(g, ws);
    const int pgrid = grid_for((int64_t)g.Mp * g.KH * g.KW * g.Cp, 256);
    hipLaunchKernelGGL(i8_prep_kernel, dim3(pgrid), dim3(256), 0, s, w, g, p.wr, p.pre);
    return check_launch("conv2d_int8 weight reorder");
}

int launch_conv2d_i8(const void *x, samd_fmt xf, const samd_conv2d_desc &d, int32_t *y, const void *ws,
                     hipStream_t s) {
    const I8Geom g = make_geom(d, xf);
    const I8Workspace p = carve(g, const_cast<void *>(ws));
    const dim3 grid((unsigned)((g.P + kTP - 1) / kTP), g.Mp / kTM);
    const bool vec = (g.C % 16) == 0 && ((uintptr_t)x % 16) == 0;
    if (vec)
        hipLaunchKernelGGL((conv2d_i8_kernel<true>), grid, dim3(256), 0, s, (const uint8_t *)x, p.wr, p.pre, y, g);
    else
        hipLaunchKernelGGL((conv2d_i8_kernel<false>), grid, dim3(256), 0, s, (const uint8_t *)x, p.wr, p.pre, y, g);
    return check_launch("conv2d_int8");
}

}  // namespace samd
