// Native 8-bit baseline (Sec. 7): the same convolution on values unpacked to 8 bits,
// as an implicit GEMM on the gfx950 int8 matrix cores (v_mfma_i32_16x16x64_i8), tiled
// through LDS.
//
// GEMM view: D[m][p] = sum_k Wr[m][k] * X[k][p] with p an output position (n, ho, wo)
// and k = (ky, kx, c); weights are reordered once per call to [M][KH][KW][Cp] (Cp = C
// rounded up to the K step, 64 or 128 channels) and activations are read in NHWC, so every lane fetches 16
// consecutive channels with one 128-bit load.  Unsigned 8-bit activations do not fit
// int8; they enter as v - 128 and the product gains 128 * (sum of the weights whose
// input lies inside the image) back in the epilogue.
#include <hip/hip_runtime.h>

#include <type_traits>

#include "hip_util.hpp"

namespace samd {

namespace {

typedef int v4i __attribute__((ext_vector_type(4)));

struct I8Geom {
    int N, C, H, W, M, KH, KW, sh, sw, ph, pw, Ho, Wo;
    int ks;          // channels per K step: 64, or 128 when C > 64
    int Cp;          // channels padded to a multiple of ks
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

// Workgroup tile: 128 output channels x TP output positions (TP = 32 or 64), 4 waves,
// wave w owning output channels w*32 .. +31 of all TP positions (2 x TP/16 MFMA tiles of
// 16 x 16).  Per K step (one kernel tap (ky, kx), KS = 64 or 128 channels) the A tile
// (weights, 128 x KS int8) and the B tile (activations of TP positions, TP x KS int8) are
// staged in LDS, double-buffered, through a register ring: the 16-byte chunks of step
// k + kRing - 1 are loaded while step k's MFMAs run, and step k + 1's are stored after
// them (one barrier per step).  LDS rows are KS bytes of data plus 16 of padding (fewer
// bank conflicts on the 16-byte reads).  The wider step amortises each barrier's fixed
// chain (wait for loads, store, barrier, read) over twice the MFMAs.
//
// The step's tap and channel chunk are uniform and advance by counters (no division in
// the loop); each thread's weight rows and input pixels are fixed 32-bit byte offsets set
// up once, so a step's loads are one add each, through buffer resources.
constexpr int kTM = 128;

__device__ __forceinline__ v4i load16(__amdgpu_buffer_rsrc_t r, int off) {
    return __builtin_bit_cast(v4i, __builtin_amdgcn_raw_buffer_load_b128(r, off, 0, 0));
}

template <int TP, int KS, bool VEC>
__global__ __launch_bounds__(256) void conv2d_i8_kernel(const uint8_t *__restrict__ x, const int8_t *__restrict__ wr,
                                                        const int32_t *__restrict__ pre, int32_t *__restrict__ y,
                                                        const I8Geom g) {
    constexpr int kRowB = KS + 16;
    constexpr int kTileA = kTM * kRowB, kTileB = TP * kRowB;
    constexpr int CPR = KS / 16;                        // 16-byte chunks per row
    constexpr int NA = kTM * CPR / 256;                 // A chunks per thread
    constexpr int NBC = (TP * CPR + 255) / 256;         // B chunks per thread
    constexpr int kNB = TP / 16;                        // MFMA tiles along the positions
    constexpr int KB = KS / 64;                         // MFMA k-blocks per step
    __shared__ __attribute__((aligned(16))) char sm[2 * (kTileA + kTileB)];   // A0, B0, A1, B1
    const int tid = threadIdx.x;
    const int lane = tid & 63, wave = tid >> 6;
    const int li = lane & 15, lg = lane >> 4;
    const int m0 = blockIdx.y * kTM;
    const int64_t p0 = (int64_t)blockIdx.x * TP;
    const int flip = g.zero_point ? (int)0x80808080u : 0;
    const int khw = g.KH * g.KW;

    // A chunk u of this thread: row (t + 256u) / CPR, 16-byte column (t + 256u) % CPR
    int aoff[NA];
#pragma unroll
    for (int u = 0; u < NA; ++u) {
        const int j = tid + 256 * u;
        aoff[u] = (j / CPR) * khw * g.Cp + (j % CPR) * 16;
    }
    const __amdgpu_buffer_rsrc_t wrs = __builtin_amdgcn_make_buffer_rsrc(
        (void *)(wr + (int64_t)m0 * khw * g.Cp), (short)0, kTM * khw * g.Cp, 0x00020000);
    // B chunk u: position p0 + (t + 256u) / CPR, channels ((t + 256u) % CPR) * 16 ..; its
    // input pixel at tap (0, 0) is (n, hb, wb), possibly outside the image
    bool bst[NBC];
    int bhb[NBC], bwb[NBC], bbase[NBC], bcol[NBC];
#pragma unroll
    for (int u = 0; u < NBC; ++u) {
        const int j = tid + 256 * u;
        bst[u] = j < TP * CPR;
        const int64_t p = p0 + j / CPR;
        const bool ok = bst[u] && p < g.P;
        const int64_t pp = ok ? p : 0;
        const int wo = (int)(pp % g.Wo);
        const int64_t r = pp / g.Wo;
        const int ho = (int)(r % g.Ho), n = (int)(r / g.Ho);
        bhb[u] = ok ? ho * g.sh - g.ph : -(1 << 20);   // positions past P are never inside
        bwb[u] = wo * g.sw - g.pw;
        bbase[u] = n * g.H * g.W * g.C;
        bcol[u] = (j % CPR) * 16;
    }
    const __amdgpu_buffer_rsrc_t xrs =
        __builtin_amdgcn_make_buffer_rsrc((void *)x, (short)0, g.N * g.H * g.W * g.C, 0x00020000);

    // raw 16-byte loads and, per B chunk, whether its pixel lies inside the image: the
    // zeroing of outside pixels and the zero-point flip happen at the LDS store, when the
    // data is due anyway (applied at the load, they would make every step wait for all
    // its own loads to arrive)
    struct Chunk {
        v4i a[NA], b[NBC];
        bool in[NBC];
    };
    auto load_step = [&](int ky, int kx, int c0, Chunk &ch) {
        const int ak = (ky * g.KW + kx) * g.Cp + c0;
#pragma unroll
        for (int u = 0; u < NA; ++u) ch.a[u] = load16(wrs, aoff[u] + ak);
#pragma unroll
        for (int u = 0; u < NBC; ++u) {
            const int hi = bhb[u] + ky, wi = bwb[u] + kx, c = c0 + bcol[u];
            const bool inside = hi >= 0 && hi < g.H && wi >= 0 && wi < g.W && c < g.C;
            ch.in[u] = inside;
            if (VEC) {
                ch.b[u] = load16(xrs, inside ? bbase[u] + (hi * g.W + wi) * g.C + c : 0);
            } else {
                // channels past C read as 0 before the flip, like padding
                uint32_t bb[4] = {0, 0, 0, 0};
                if (inside) {
                    const uint8_t *px = x + bbase[u] + (hi * g.W + wi) * g.C + c;
                    for (int e = 0; e < 16; ++e)
                        if (c + e < g.C) bb[e >> 2] |= (uint32_t)px[e] << ((e & 3) * 8);
                        else bb[e >> 2] |= ((uint32_t)flip & 0xff) << ((e & 3) * 8);
                }
                ch.b[u] = v4i{(int)bb[0], (int)bb[1], (int)bb[2], (int)bb[3]};
            }
        }
    };
    auto store_step = [&](int buf, const Chunk &ch) {
        char *A = sm + buf * (kTileA + kTileB), *B = A + kTileA;
#pragma unroll
        for (int u = 0; u < NA; ++u) {
            const int j = tid + 256 * u;
            *(v4i *)(A + (j / CPR) * kRowB + (j % CPR) * 16) = ch.a[u];
        }
#pragma unroll
        for (int u = 0; u < NBC; ++u) {
            const int j = tid + 256 * u;
            const v4i zero = {0, 0, 0, 0};
            if (bst[u]) *(v4i *)(B + (j / CPR) * kRowB + (j % CPR) * 16) = ch.in[u] ? (ch.b[u] ^ flip) : zero;
        }
    };
    // steps in order: channel chunks innermost, then kx, then ky
    int lky = 0, lkx = 0, lc = 0;   // the next step to load
    auto advance = [&]() {
        lc += KS;
        if (lc >= g.Cp) {
            lc = 0;
            if (++lkx == g.KW) {
                lkx = 0;
                ++lky;
            }
        }
    };

    v4i acc[2][kNB];
#pragma unroll
    for (int a = 0; a < 2; ++a)
#pragma unroll
        for (int b = 0; b < kNB; ++b) acc[a][b] = v4i{0, 0, 0, 0};

    const int nk = khw * (g.Cp / KS);
    // Register ring of kRing chunks: at step k the chunk of step k + kRing - 1 is loaded
    // (into the slot step k - 1 used) and the chunk of step k + 1 is stored to LDS buffer
    // (k + 1) & 1, so every load has kRing - 2 steps of MFMA work to arrive.  The loop is
    // unrolled by kRing, so every slot's role is fixed at compile time (no register copy
    // waits for loads still in flight).
    constexpr int kRing = 3;
    // FULL: every load and store of the step exists (no branch around them, so the
    // compiler's load counters stay exact and each store waits only for its own chunk)
    auto body = [&](auto full, int k, Chunk &load_into, const Chunk &store_from) {
        if (full.value || k + kRing - 1 < nk) {
            load_step(lky, lkx, lc, load_into);
            advance();
        }
        const char *A = sm + (k & 1) * (kTileA + kTileB), *B = A + kTileA;
#pragma unroll
        for (int kb = 0; kb < KB; ++kb) {
            v4i fa[2], fb[kNB];
#pragma unroll
            for (int t = 0; t < 2; ++t)
                fa[t] = *(const v4i *)(A + (wave * 32 + t * 16 + li) * kRowB + kb * 64 + lg * 16);
#pragma unroll
            for (int t = 0; t < kNB; ++t) fb[t] = *(const v4i *)(B + (t * 16 + li) * kRowB + kb * 64 + lg * 16);
#pragma unroll
            for (int a = 0; a < 2; ++a)
#pragma unroll
                for (int b = 0; b < kNB; ++b)
                    acc[a][b] = __builtin_amdgcn_mfma_i32_16x16x64_i8(fa[a], fb[b], acc[a][b], 0, 0, 0);
        }
        if (full.value || k + 1 < nk) store_step((k + 1) & 1, store_from);
        __syncthreads();
    };
    Chunk ring[kRing];
#pragma unroll
    for (int i = 0; i < kRing - 1; ++i)
        if (i < nk) {
            load_step(lky, lkx, lc, ring[i]);
            advance();
        }
    store_step(0, ring[0]);
    __syncthreads();
    int k = 0;
    // groups of kRing steps whose loads (up to step k + 2 kRing - 2) all exist
    for (; k + 2 * kRing - 1 <= nk; k += kRing) {
#pragma unroll
        for (int u = 0; u < kRing; ++u)
            body(std::true_type{}, k + u, ring[(u + kRing - 1) % kRing], ring[(u + 1) % kRing]);
    }
    for (; k < nk; k += kRing) {
#pragma unroll
        for (int u = 0; u < kRing; ++u)
            if (k + u < nk) body(std::false_type{}, k + u, ring[(u + kRing - 1) % kRing], ring[(u + 1) % kRing]);
    }

    // D[row][col]: lane holds rows 4*lg + v (output channels) of column li (position).
    // Zero point: + 128 * (sum of the weights whose input lies inside the image), the
    // rectangle [ky0, ky1) x [kx0, kx1) of in-image taps of the position.
    const int pw = (g.KH + 1) * (g.KW + 1);
#pragma unroll
    for (int b = 0; b < kNB; ++b) {
        const int64_t p = p0 + b * 16 + li;
        if (p >= g.P) continue;
        const int wo = (int)(p % g.Wo);
        const int64_t r = p / g.Wo;
        const int ho = (int)(r % g.Ho), n = (int)(r / g.Ho);
        const int hh = ho * g.sh - g.ph, ww = wo * g.sw - g.pw;
        const int ky0 = max(0, -hh), ky1 = min(g.KH, g.H - hh);
        const int kx0 = max(0, -ww), kx1 = min(g.KW, g.W - ww);
        const int e11 = ky1 * (g.KW + 1) + kx1, e01 = ky0 * (g.KW + 1) + kx1;
        const int e10 = ky1 * (g.KW + 1) + kx0, e00 = ky0 * (g.KW + 1) + kx0;
        int32_t *yo = y + ((int64_t)n * g.M * g.Ho + ho) * g.Wo + wo;
#pragma unroll
        for (int a = 0; a < 2; ++a) {
#pragma unroll
            for (int v = 0; v < 4; ++v) {
                const int m = m0 + wave * 32 + a * 16 + lg * 4 + v;
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
    g.ks = d.C > 64 ? 128 : 64;               // channels per K step
    g.Cp = (d.C + g.ks - 1) / g.ks * g.ks;
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
    // 64 positions per workgroup (half the weight re-reads of 32) when that still gives
    // every compute unit a workgroup, else 32
    const int64_t wgs64 = (g.P + 63) / 64 * (g.Mp / kTM);
    const bool vec = (g.C % 16) == 0 && ((uintptr_t)x % 16) == 0;
    const unsigned gy = (unsigned)(g.Mp / kTM);
#define SAMD_I8_LAUNCH(TP_, KS_, VEC_)                                                                          \
    hipLaunchKernelGGL((conv2d_i8_kernel<TP_, KS_, VEC_>), dim3((unsigned)((g.P + TP_ - 1) / TP_), gy), dim3(256), 0, \
                       s, (const uint8_t *)x, p.wr, p.pre, y, g)
#define SAMD_I8_KS(TP_)                                                                                         \
    if (g.ks == 128) {                                                                                          \
        if (vec) SAMD_I8_LAUNCH(TP_, 128, true); else SAMD_I8_LAUNCH(TP_, 128, false);                          \
    } else {                                                                                                    \
        if (vec) SAMD_I8_LAUNCH(TP_, 64, true); else SAMD_I8_LAUNCH(TP_, 64, false);                            \
    }
    if (wgs64 >= 256) {
        SAMD_I8_KS(64)
    } else {
        SAMD_I8_KS(32)
    }
#undef SAMD_I8_KS
#undef SAMD_I8_LAUNCH
    return check_launch("conv2d_int8");
}

}  // namespace samd
