// Native 8-bit baseline (Sec. 7): the same convolution on values unpacked to 8 bits,
// as an implicit GEMM on the gfx950 int8 matrix cores (v_mfma_i32_16x16x64_i8), tiled
// through LDS.
//
// GEMM view: D[m][p] = sum_k Wr[m][k] * X[k][p] with p an output position (n, ho, wo)
// and k = (ky, kx, c); weights are reordered once per call to [M][KH][KW][Cp] (Cp = C
// rounded up to the K step, 64 or 128 channels) and activations are read in NHWC, so
// every lane fetches 16 consecutive channels with one 128-bit load.  Layers with few
// input channels also get the weights in a packed-row K order (k = (ky, kx*C + c), each
// kernel row padded to 16-byte slots), which the packed-row kernel reads instead of
// padding C to 64.  Unsigned 8-bit activations do not fit int8; they enter as v - 128
// and the product gains 128 * (sum of the weights whose input lies inside the image)
// back in the epilogue.
//
// Kernels: im2col tiles (any layer), halo tiles (stride-1 layers with C a multiple of
// 16), weight-resident runs (stride-1 3x3 and 1x1 layers, whole K or K in chunks), and
// packed rows (few input channels, any stride); the host lists the launches that fit a
// layer and a model or a measurement picks one.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <climits>
#include <array>
#include <map>
#include <mutex>
#include <string>
#include <type_traits>
#include <vector>

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
    int rk;          // packed-row K: bytes of one kernel row's window in NHWC, KW * C
    int rs;          // ... 16-byte slots per kernel row, ceil(rk / 16)
    int pkb;         // ... 64-byte k-blocks, ceil(KH * rs / 4); 0 where that layout is not offered
};

// Reorder weights to [Mp][KH][KW][Cp] int8 (zero padded) and, for the zero-point path,
// per-m 2-D prefix sums of the channel-summed kernel (the correction of an output is the
// sum over its in-image taps: a rectangle, four lookups).
//
// Where the packed-row K applies, the weights are also written in that K order, as MFMA B
// fragments: fragment (cb, kb) (filters cb*16 .. +15, k-block kb) is 1 KB at
// (cb * pkb + kb) * 1024, lane l's 16 bytes at l * 16 holding filter cb*16 + (l & 15),
// slot s = kb*4 + (l >> 4): kernel row s / rs, window bytes j = (s % rs)*16 .. +15, byte j
// being tap column j / C, channel j % C (zero past the row's rk bytes, past the last slot
// and past the last filter).
__global__ __launch_bounds__(256) void i8_prep_kernel(const int8_t *__restrict__ w, const I8Geom g,
                                                      int8_t *__restrict__ wr, int32_t *__restrict__ pre,
                                                      int8_t *__restrict__ wk) {
    if (g.pkb) {
        const int64_t ptotal = (int64_t)((g.M + 15) / 16) * g.pkb * 1024;
        for (int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x; i < ptotal; i += (int64_t)gridDim.x * 256) {
            const int f = (int)(i >> 10), l = (int)((i >> 4) & 63), b = (int)(i & 15);
            const int cb = f / g.pkb, kb = f - cb * g.pkb;
            const int m = cb * 16 + (l & 15), sl = kb * 4 + (l >> 4);
            const int ky = sl / g.rs, j = (sl - ky * g.rs) * 16 + b;
            int8_t v = 0;
            if (m < g.M && ky < g.KH && j < g.rk)
                v = w[(((int64_t)m * g.C + j % g.C) * g.KH + ky) * g.KW + j / g.C];
            wk[i] = v;
        }
    }
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

// Halo-tiled implicit GEMM for stride-1 layers whose channel count is a multiple of 16.
// A workgroup computes TM = 4 WM output channels x TP output positions of one image:
// wave w owns channels w*WM .. +WM-1 of all TP positions (WM/16 x TP/16 MFMA tiles of
// 16 x 16).  The K loop walks chunks of KC channels (the weight layout's K step, 64 or
// 128) and, inside each chunk, the KH*KW taps; one step is one tap of one chunk.  The
// input pixels a chunk needs (the tile's output rows plus KH-1 halo rows, every column
// any of its positions reaches, KC channels each) are staged in LDS once and read by
// every tap at a shifted address - the KH*KW-fold re-read of an im2col tile becomes one
// load per chunk - while the next chunk's halo is requested at the first step of a chunk
// and stored into the second LDS buffer after its last step (one barrier per chunk).
// Each wave streams its own weight rows straight from L2 into registers, kRing - 1 steps
// ahead: no two waves share a weight row, so LDS would buy no reuse.  A step reads the
// whole KC-byte segment of each of its weight rows, so every cache line of the weights
// is fetched once per workgroup.
//
// Tiles are either flat runs of TP positions of one image (narrow images: a tile spans
// several output rows and the halo holds whole padded rows) or segments of TP columns of
// one output row (wide images: the halo holds KH rows of TP + KW - 1 columns).
//
// Unsigned 8-bit activations enter as v - 128 (the int8 range), and so do the zero
// padding pixels (0 - 128): every tap then carries the same offset, and the result is
// the accumulator plus 128 times the sum of all of the filter's weights, one constant per
// output channel.
constexpr int kHaloPer = 12;     // halo pieces (16 bytes) per thread and chunk at most
constexpr int kHaloPieces = kHaloPer * 256;
constexpr int kHaloMaxLds = 160 * 1024;   // LDS of one workgroup on gfx950

struct HaloTiles {
    int rowseg;      // 0: flat tiles of TP positions; 1: row segments of TP columns
    int tiles_img;   // tiles per image
    int segs;        // row segments per output row (rowseg)
    int halo_bytes;  // LDS bytes of one halo buffer (the largest tile's)
    int nch;         // chunks of KC channels: Cp / KC
    int items;       // work items: N * tiles_img * channel tiles
    int kc;          // channels per chunk: the K step, or 64 where a 128-channel chunk does not fit
};

// n / d for 0 <= n < 2^22 and 1 <= d < 2^12 by a float reciprocal estimate and one exact
// correction each way (the estimate is within one of the quotient): a few independent VALU
// operations instead of the dependent chain of an integer division, which with one wave
// per SIMD would sit exposed in the kernel's prologue.
struct FastDiv {
    int d;
    float r;
    __device__ explicit FastDiv(int d_) : d(d_), r(1.0f / (float)d_) {}
    __device__ int div(int n) const {
        int q = (int)((float)n * r);
        q += (q + 1) * d <= n ? 1 : 0;
        q -= q * d > n ? 1 : 0;
        return q;
    }
};

template <int WM, int TP, int KC>
__global__ __launch_bounds__(256) void conv2d_i8_halo_kernel(const uint8_t *__restrict__ x, const int8_t *__restrict__ wr,
                                                             const int32_t *__restrict__ pre, int32_t *__restrict__ y,
                                                             const I8Geom g, const HaloTiles ht) {
    constexpr int NI = WM / 16, NJ = TP / 16, TM = 4 * WM;
    constexpr int KB = KC / 64;           // MFMA k-blocks per step
    constexpr int PIX = KC + 16;          // LDS bytes per halo pixel: KC channels + 16 against bank conflicts
    constexpr int PPP = KC / 16;          // 16-byte pieces per pixel
    constexpr int kRing = KC == 128 ? 4 : 6;   // weight register sets: requests kRing - 1 steps ahead
    extern __shared__ __attribute__((aligned(16))) char halo[];
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int li = lane & 15, lg = lane >> 4;
    // Workgroup p runs on XCD p % 8; XCD x takes the contiguous range of work items
    // [x * items / 8, (x + 1) * items / 8), items ordered (image, tile, channel tile), so
    // neighbouring tiles - which share halo rows - and the channel tiles of one position
    // tile meet in one L2.
    const int xcd = blockIdx.x % kNumXcd, k = blockIdx.x / kNumXcd;
    const int ib = (int)((int64_t)xcd * ht.items / kNumXcd), ie = (int)((int64_t)(xcd + 1) * ht.items / kNumXcd);
    if (ib + k >= ie) return;
    const int item = ib + k;
    const int mtiles = (g.M + TM - 1) / TM;
    const int tile = item / mtiles;
    const int m0 = (item - tile * mtiles) * TM;
    const int n = tile / ht.tiles_img, tt = tile - n * ht.tiles_img;
    const int HWo = g.Ho * g.Wo;
    const int khw = g.KH * g.KW;
    const int flip = g.zero_point ? (int)0x80808080u : 0;

    // the tile: positions p0 .. p0 + np - 1 of image n (row-major within the image), output
    // rows ho_a .. ho_b, halo columns col_lo .. col_lo + hw - 1 of input rows ho_a - ph ..
    int p0, np, ho_a, ho_b, col_lo, hw;
    if (!ht.rowseg) {
        p0 = tt * TP;
        np = min(TP, HWo - p0);
        ho_a = p0 / g.Wo;
        ho_b = (p0 + np - 1) / g.Wo;
        col_lo = -g.pw;
        hw = g.Wo + g.KW - 1;
    } else {
        const int ho = tt / ht.segs, wo0 = (tt - ho * ht.segs) * TP;
        np = min(TP, g.Wo - wo0);
        p0 = ho * g.Wo + wo0;
        ho_a = ho_b = ho;
        col_lo = wo0 - g.pw;
        hw = np + g.KW - 1;
    }
    const int npc = (ho_b - ho_a + g.KH) * hw * PPP;   // 16-byte halo pieces of one chunk
    const int ih0 = ho_a - g.ph;

    // halo pieces of this thread: k = tid + 256 u -> pixel (r, jc) = divmod(k / PPP, hw),
    // channels (k % PPP) * 16 .. +15 of the chunk; global byte offset without the chunk's
    // first channel, LDS offset, and whether the pixel lies inside the image
    int gofs[kHaloPer], lofs[kHaloPer];
    uint32_t inside = 0;
    const FastDiv by_hw(hw);
#pragma unroll
    for (int u = 0; u < kHaloPer; ++u) {
        const int k = tid + 256 * u;
        const int q = k & (PPP - 1), rc = k / PPP;
        const int r = by_hw.div(rc), jc = rc - r * hw;
        const int ih = ih0 + r, iw = col_lo + jc;
        const bool in = k < npc && ih >= 0 && ih < g.H && iw >= 0 && iw < g.W;
        inside |= in ? 1u << u : 0u;
        gofs[u] = in ? ((n * g.H + ih) * g.W + iw) * g.C + q * 16 : 0;
        lofs[u] = rc * PIX + q * 16;
    }
    const __amdgpu_buffer_rsrc_t xrs =
        __builtin_amdgcn_make_buffer_rsrc((void *)x, (short)0, g.N * g.H * g.W * g.C, 0x00020000);
    v4i hv[kHaloPer];
    auto halo_load = [&](int c0) {
#pragma unroll
        for (int u = 0; u < kHaloPer; ++u) hv[u] = load16(xrs, gofs[u] + c0);
    };
    auto halo_store = [&](int buf, int c0) {
        char *hb = halo + buf * ht.halo_bytes;
        const v4i pad = {flip, flip, flip, flip};
#pragma unroll
        for (int u = 0; u < kHaloPer; ++u) {
            const int k = tid + 256 * u;
            // padding pixels and channels past C (whose weights are 0) hold the zero point
            const bool in = ((inside >> u) & 1) && c0 + (k & (PPP - 1)) * 16 < g.C;
            if (k < npc) *(v4i *)(hb + lofs[u]) = in ? (hv[u] ^ flip) : pad;
        }
    };

    // weight rows of this wave: A tile i is rows wave*WM + i*16 + li, bytes kb*64 + lg*16
    // .. +15 of each step's KC-byte segment
    int alane[NI];
#pragma unroll
    for (int i = 0; i < NI; ++i) alane[i] = (wave * WM + i * 16 + li) * khw * g.Cp + lg * 16;
    const __amdgpu_buffer_rsrc_t wrs = __builtin_amdgcn_make_buffer_rsrc(
        (void *)(wr + (int64_t)m0 * khw * g.Cp), (short)0, TM * khw * g.Cp, 0x00020000);

    // halo address of each position tile's lane (position p0 + j*16 + li; lanes past the
    // tile read its last position, their sums are not stored), before the tap's shift
    int blane[NJ];
    const FastDiv by_wo(g.Wo);
#pragma unroll
    for (int j = 0; j < NJ; ++j) {
        const int p = p0 + min(j * 16 + li, np - 1);
        const int ho = by_wo.div(p), wo = p - ho * g.Wo;
        blane[j] = ((ho - ho_a) * hw + (wo - g.pw - col_lo)) * PIX + lg * 16;
    }

    v4i acc[NI][NJ];
#pragma unroll
    for (int i = 0; i < NI; ++i)
#pragma unroll
        for (int j = 0; j < NJ; ++j) acc[i][j] = v4i{0, 0, 0, 0};

    const int S = ht.nch * khw;   // steps: chunks x taps
    // The next step whose weights are requested.  Every step requests one step's weights,
    // also past the last step (the last step's rows again, in bounds, never used): loads
    // issued on every path keep the compiler's wait counts exact, so a step waits only for
    // its own weights, requested kRing - 1 steps earlier.
    int ltap = 0, lc = 0;
    const int last_so = (khw - 1) * g.Cp + g.Cp - KC;
    v4i aR[kRing][NI][KB];
    auto a_load = [&](v4i (&a)[NI][KB]) {
        const int so = lc < g.Cp ? ltap * g.Cp + lc : last_so;
#pragma unroll
        for (int i = 0; i < NI; ++i)
#pragma unroll
            for (int kb = 0; kb < KB; ++kb)
                a[i][kb] = __builtin_bit_cast(
                    v4i, __builtin_amdgcn_raw_buffer_load_b128(wrs, alane[i] + kb * 64, so, 0));
        if (++ltap == khw) {
            ltap = 0;
            lc += KC;
        }
    };

    halo_load(0);
#pragma unroll
    for (int r = 0; r < kRing - 1; ++r) a_load(aR[r]);
    halo_store(0, 0);
    __syncthreads();

    // Halo fragments of a step, one k-block (64 channels) at a time: while a k-block's
    // MFMAs run, the fragments of the next k-block (of this step or the next) are read,
    // so LDS reads overlap the matrix work instead of preceding it.  After the last step
    // they read the first tap again (in bounds, never used).
    v4i b[KB][NJ];
    auto b_read = [&](int kb, int buf, int ky, int kx) {
        const char *hb = halo + buf * ht.halo_bytes + (ky * hw + kx) * PIX + kb * 64;
#pragma unroll
        for (int j = 0; j < NJ; ++j) b[kb][j] = *(const v4i *)(hb + blane[j]);
    };
#pragma unroll
    for (int kb = 0; kb < KB; ++kb) b_read(kb, 0, 0, 0);

    int tap = 0, cc = 0, tky = 0, tkx = 0;   // the step being computed
    auto step = [&](auto slot) {
        constexpr int SL = decltype(slot)::value;
        a_load(aR[(SL + kRing - 1) % kRing]);
        if (tap == 0 && cc + 1 < ht.nch) halo_load((cc + 1) * KC);
        // the following step's tap (within this chunk)
        int nky = tky, nkx = tkx + 1;
        if (nkx == g.KW) {
            nkx = 0;
            ++nky;
        }
        const bool last_tap = tap + 1 == khw;
        if (last_tap) nky = nkx = 0;
#pragma unroll
        for (int kb = 0; kb < KB; ++kb) {
#pragma unroll
            for (int i = 0; i < NI; ++i)
#pragma unroll
                for (int j = 0; j < NJ; ++j)
                    acc[i][j] = __builtin_amdgcn_mfma_i32_16x16x64_i8(aR[SL][i][kb], b[kb][j], acc[i][j], 0, 0, 0);
            // this k-block's fragments are consumed: read the next step's (same chunk)
            if (!last_tap) b_read(kb, cc & 1, nky, nkx);
        }
        if (last_tap) {
            if (cc + 1 < ht.nch) {
                halo_store((cc + 1) & 1, (cc + 1) * KC);
                __syncthreads();
            }
            tap = tky = tkx = 0;
            ++cc;
#pragma unroll
            for (int kb = 0; kb < KB; ++kb) b_read(kb, cc & 1, 0, 0);
        } else {
            ++tap;
            tky = nky;
            tkx = nkx;
        }
    };
    int s = 0;
    if constexpr (kRing == 4) {
        for (; s + 4 <= S; s += 4) {
            step(std::integral_constant<int, 0>{});
            step(std::integral_constant<int, 1>{});
            step(std::integral_constant<int, 2>{});
            step(std::integral_constant<int, 3>{});
        }
    } else {
        for (; s + 6 <= S; s += 6) {
            step(std::integral_constant<int, 0>{});
            step(std::integral_constant<int, 1>{});
            step(std::integral_constant<int, 2>{});
            step(std::integral_constant<int, 3>{});
            step(std::integral_constant<int, 4>{});
            step(std::integral_constant<int, 5>{});
        }
    }
    if (s < S) step(std::integral_constant<int, 0>{});
    if (s + 1 < S) step(std::integral_constant<int, 1>{});
    if (s + 2 < S) step(std::integral_constant<int, 2>{});
    if constexpr (kRing == 6) {
        if (s + 3 < S) step(std::integral_constant<int, 3>{});
        if (s + 4 < S) step(std::integral_constant<int, 4>{});
    }

    // D[row][col]: lane holds rows 4*lg + v (output channels) of column li (position);
    // zero point: + 128 * (the sum of all of the filter's weights)
    const int full = g.KH * (g.KW + 1) + g.KW;   // prefix-table entry of the whole filter
#pragma unroll
    for (int i = 0; i < NI; ++i) {
#pragma unroll
        for (int v = 0; v < 4; ++v) {
            const int m = m0 + wave * WM + i * 16 + lg * 4 + v;
            if (m >= g.M) continue;
            const int32_t corr = g.zero_point ? 128 * pre[(int64_t)m * (g.KH + 1) * (g.KW + 1) + full] : 0;
            int32_t *ym = y + ((int64_t)n * g.M + m) * HWo + p0;
#pragma unroll
            for (int j = 0; j < NJ; ++j) {
                const int pp = j * 16 + li;
                if (pp < np) ym[pp] = acc[i][j][v] + corr;
            }
        }
    }
}

// Weight-resident implicit GEMM for stride-1 3x3 and 1x1 layers of 64 or 128 (padded)
// channels.  A workgroup owns one group of 32 filters and one contiguous run of output
// positions of one image (the layer is cut into about one workgroup per compute unit).
// It stages the group's weights (32 x K bytes, K = Cp*KH*KW) and the halo of the whole
// run - every input pixel the run's positions read, all channels - in LDS once; then each
// of its 8 waves (two per SIMD) copies the weights into its registers (2 x K/64 fragments
// of 16 bytes per lane, 144 registers at K = 1152) and walks its share of the run's
// 16-position tiles with no further global reads and no barrier.  A tile's outputs are
// stored as soon as its MFMAs end, so the int32 output writes overlap the matrix work of
// the later tiles.  Owning 32 filters rather than all of them keeps the bytes a compute
// unit pulls from L2 before its first tile small (the group's weights and the halo of a
// longer run): that prologue bounds such a kernel, since every compute unit starts at
// once and they share the L2 bandwidth.
//
// The activations are the MFMA's A operand (rows = output positions, read from the halo
// at the tap's shift) and the weights its B operand (columns = filters), so a lane's four
// accumulator values are four consecutive positions of one filter: one 16-byte store.
//
// Unsigned 8-bit activations and the zero padding enter as v - 128, as in the halo
// kernel: one correction constant per output channel.
// One k-block of a 16 x 16 output tile from the activation fragment a (lane li: position
// li) and the weight fragment w (lane li: filter li).  TR = false: the result's rows are
// positions, so a lane holds 4 consecutive positions of filter li (one 16-byte store
// where the output is 16-byte aligned and an image's positions a multiple of 4); TR =
// true: the rows are filters, so a lane holds position li of filters 4 lg .. 4 lg + 3 and
// 16 lanes store 16 consecutive positions of a filter, 64 contiguous bytes at any
// alignment (the element stores of the other layout would be scattered 4-byte writes).
template <bool TR>
__device__ __forceinline__ v4i mfma_tile(v4i a, v4i w, v4i acc) {
    return TR ? __builtin_amdgcn_mfma_i32_16x16x64_i8(w, a, acc, 0, 0, 0)
              : __builtin_amdgcn_mfma_i32_16x16x64_i8(a, w, acc, 0, 0, 0);
}

constexpr int kResThreads = 512;
constexpr int kResWaves = kResThreads / 64;
constexpr int kResPieces = 5120;   // 16-byte halo pieces of one workgroup at most
constexpr int kResTile = 16;       // output positions per tile
constexpr int kResGroup = 32;      // filters per workgroup

constexpr int kResChunk = 64;      // chunked kernel: input channels per K chunk (or twice that)
constexpr int kResTPW = 4;         // ... tiles per wave at most: runs of at most 512 positions
constexpr int kResHalo = 6;        // ... halo pieces (16 bytes) per thread and chunk at most
constexpr int kResMaxChunks = 8;   // ... padded channels up to 512

struct ResTiles {
    int R;      // position runs per image
    int U;      // tiles of 16 positions per image
    int items;  // work items: N * R * (Mp / 32)
    int nch;    // K chunks of 64 or 128 channels (chunked kernel)
    int halo;   // LDS bytes of the halo (of one chunk's halo, chunked kernel); the weights follow it
    int buf;    // LDS bytes of one chunk buffer: halo and weights (chunked kernel)
    int vec;    // 1: 16-byte output stores (Ho * Wo a multiple of 4, y 16-byte aligned)
};

// Store a 16-position tile (positions p0 .., of which those below pe exist) of NC
// 16-filter tiles from filter m0, adding 128 x the filter sums where the activations carry
// the zero point (corr per lane: filter li, or filters 4 lg + v with TR); lanes follow
// mfma_tile's layouts.  Non-temporal: the outputs are not read again by this kernel.
template <int NC, bool TR>
__device__ __forceinline__ void store_res_tile(const v4i (&acc)[NC], const int32_t (&corr)[NC][TR ? 4 : 1],
                                               int32_t *__restrict__ y, const I8Geom &g, int n, int m0, int p0,
                                               int pe, int HWo, int vec, int li, int lg) {
    if constexpr (TR) {
        // through a buffer over the NC*16 filters' outputs of image n: one per-lane offset
        // and a scalar one per (c, v), so no per-store 64-bit addresses stay live
        const int pos = p0 + li;
        if (pos >= pe) return;
        const __amdgpu_buffer_rsrc_t yrs = __builtin_amdgcn_make_buffer_rsrc(
            (void *)(y + ((int64_t)n * g.M + m0) * HWo), (short)0, min(NC * 16, g.M - m0) * HWo * 4, 0x00020000);
        const int voff = (lg * 4 * HWo + pos) * 4;
#pragma unroll
        for (int c = 0; c < NC; ++c)
#pragma unroll
            for (int v = 0; v < 4; ++v)
                if (m0 + c * 16 + lg * 4 + v < g.M)   // aux 2: non-temporal
                    __builtin_amdgcn_raw_buffer_store_b32(acc[c][v] + (g.zero_point ? 128 * corr[c][v] : 0), yrs,
                                                          voff, (c * 16 + v) * HWo * 4, 2);
    } else {
        const int q0 = p0 + lg * 4;
#pragma unroll
        for (int c = 0; c < NC; ++c) {
            const int m = m0 + c * 16 + li;
            if (m >= g.M) continue;
            int32_t *ym = y + ((int64_t)n * g.M + m) * HWo;
            const v4i o = acc[c] + (g.zero_point ? 128 * corr[c][0] : 0);
            if (vec) {
                if (q0 < pe) __builtin_nontemporal_store(o, (v4i *)(ym + q0));
            } else {
#pragma unroll
                for (int v = 0; v < 4; ++v)
                    if (q0 + v < pe) ym[q0 + v] = o[v];
            }
        }
    }
}

template <int KH, int KW, int CB, bool TR>
__global__ __launch_bounds__(kResThreads) void conv2d_i8_resident_kernel(const uint8_t *__restrict__ x,
                                                                        const int8_t *__restrict__ wr,
                                                                        const int32_t *__restrict__ pre,
                                                                        int32_t *__restrict__ y, const I8Geom g,
                                                                        const ResTiles rt) {
    constexpr int NT = kResThreads, NW = kResWaves;
    constexpr int NC = 2;                 // 16-filter MFMA tiles per wave
    constexpr int KHW = KH * KW;
    constexpr int NKB = KHW * CB;         // k-blocks of 64: taps x channel blocks
    constexpr int KC = 64 * CB;           // padded channels (the weight layout's Cp)
    constexpr int PIX = KC + 16;          // LDS bytes per halo pixel (16 against bank conflicts)
    constexpr int PPP = KC / 16;          // 16-byte pieces per pixel
    constexpr int HPER = kResPieces / NT; // halo pieces per thread at most
    constexpr int WPIECES = NC * NKB * 64;          // the group's weights in 16-byte pieces
    constexpr int WPER = (WPIECES + NT - 1) / NT;
    constexpr int D = NKB % 3 == 0 ? 3 : NKB;       // k-blocks of A fragments read ahead
    extern __shared__ __attribute__((aligned(16))) char smem[];
    char *halo = smem;
    char *wlds = smem + rt.halo;   // fragment (c, kb): 1 KB at (c*NKB + kb)*1024, lane l at l*16

    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int li = lane & 15, lg = lane >> 4;
    // items ordered (image, run, filter group); XCD x takes a contiguous share, so the
    // filter groups of one run and neighbouring runs (which share halo rows) meet in one L2
    const int xcd = blockIdx.x % kNumXcd, kk = blockIdx.x / kNumXcd;
    const int ib = (int)((int64_t)xcd * rt.items / kNumXcd), ie = (int)((int64_t)(xcd + 1) * rt.items / kNumXcd);
    if (ib + kk >= ie) return;
    const int item = ib + kk;
    const int ngrp = g.Mp / kResGroup;
    const int run = item / ngrp;
    const int m0 = (item - run * ngrp) * kResGroup;
    const int n = run / rt.R, r = run - n * rt.R;
    const int HWo = g.Ho * g.Wo;
    const int ua = (int)((int64_t)r * rt.U / rt.R), ub = (int)((int64_t)(r + 1) * rt.U / rt.R);
    const int ps = ua * kResTile, pe = min(ub * kResTile, HWo), nt = ub - ua;
    const int ho_a = ps / g.Wo, ho_b = (pe - 1) / g.Wo;
    const int hw = g.Wo + KW - 1;                  // halo columns: the padded row
    const int npc = (ho_b - ho_a + KH) * hw * PPP;
    const int ih0 = ho_a - g.ph;
    const int flip = g.zero_point ? (int)0x80808080u : 0;

    // halo pieces of this thread: k = tid + NT u -> pixel rc = k / PPP = (row, column) of
    // the halo, channels (k % PPP) * 16 .. +15
    const __amdgpu_buffer_rsrc_t xrs =
        __builtin_amdgcn_make_buffer_rsrc((void *)x, (short)0, g.N * g.H * g.W * g.C, 0x00020000);
    const FastDiv by_hw(hw);
    v4i hv[HPER];
    uint32_t inside = 0;
#pragma unroll
    for (int u = 0; u < HPER; ++u) {
        const int k = tid + NT * u;
        const int q = k % PPP, rc = k / PPP;
        const int rr = by_hw.div(rc), jc = rc - rr * hw;
        const int ih = ih0 + rr, iw = jc - g.pw;
        const bool in = k < npc && ih >= 0 && ih < g.H && iw >= 0 && iw < g.W && q * 16 < g.C;
        inside |= in ? 1u << u : 0u;
        hv[u] = load16(xrs, in ? ((n * g.H + ih) * g.W + iw) * g.C + q * 16 : 0);
    }
    // the group's weights, 16 bytes per piece e = tid + NT u: fragment e / 64, lane e % 64
    // -> filter m0 + c*16 + (lane & 15), bytes kb*64 + (lane >> 4)*16 .. +15 of its K
    const __amdgpu_buffer_rsrc_t wrs = __builtin_amdgcn_make_buffer_rsrc(
        (void *)(wr + (int64_t)m0 * KHW * KC), (short)0, kResGroup * KHW * KC, 0x00020000);
    v4i wv[WPER];
#pragma unroll
    for (int u = 0; u < WPER; ++u) {
        const int e = min(tid + NT * u, WPIECES - 1);
        const int f = e >> 6, l = e & 63;
        const int c = f / NKB, kb = f - c * NKB;
        wv[u] = load16(wrs, (c * 16 + (l & 15)) * KHW * KC + kb * 64 + (l >> 4) * 16);
    }
    // the zero-point correction of this lane's filters
    constexpr int full = KH * (KW + 1) + KW;   // prefix-table entry of the whole filter
    const __amdgpu_buffer_rsrc_t prs = __builtin_amdgcn_make_buffer_rsrc(
        (void *)pre, (short)0, g.M * (KH + 1) * (KW + 1) * 4, 0x00020000);
    constexpr int NV = TR ? 4 : 1;   // filters per lane and 16-filter tile
    int32_t corr[NC][NV];
#pragma unroll
    for (int c = 0; c < NC; ++c)
#pragma unroll
        for (int v = 0; v < NV; ++v) {
            const int m = min(m0 + c * 16 + (TR ? lg * 4 + v : li), g.M - 1);
            corr[c][v] = __builtin_amdgcn_raw_buffer_load_b32(prs, (m * (KH + 1) * (KW + 1) + full) * 4, 0, 0);
        }

    {
        const v4i pad = {flip, flip, flip, flip};
#pragma unroll
        for (int u = 0; u < HPER; ++u) {
            const int k = tid + NT * u;
            if (k < npc) *(v4i *)(halo + (k / PPP) * PIX + (k % PPP) * 16) = ((inside >> u) & 1) ? (hv[u] ^ flip) : pad;
        }
#pragma unroll
        for (int u = 0; u < WPER; ++u) {
            const int e = tid + NT * u;
            if (e < WPIECES) *(v4i *)(wlds + e * 16) = wv[u];
        }
    }
    __syncthreads();

    // this wave's copy of the group's weights: B fragment (c, kb) is column li (filter
    // m0 + c*16 + li), bytes kb*64 + lg*16 .. +15 of the filter's K
    v4i wb[NC][NKB];
#pragma unroll
    for (int c = 0; c < NC; ++c)
#pragma unroll
        for (int kb = 0; kb < NKB; ++kb) wb[c][kb] = *(const v4i *)(wlds + (c * NKB + kb) * 1024 + lane * 16);

    // halo address of this lane's A row (position) in tile t, at tap (0, 0) and channel
    // block 0; lanes past the run read its last position (their sums are not stored)
    const FastDiv by_wo(g.Wo);
    auto lane_addr = [&](int t) {
        const int pos = min(ps + t * kResTile + li, pe - 1);
        const int ho = by_wo.div(pos), wo = pos - ho * g.Wo;
        return ((ho - ho_a) * hw + wo) * PIX + lg * 16;
    };
    const int rowsh = hw * PIX;
    auto shift = [&](int kb) {   // kb is a compile-time constant after unrolling
        const int tap = kb / CB;
        return (tap / KW) * rowsh + (tap % KW) * PIX + (kb % CB) * 64;
    };

    // tile pairs: the wave's i-th tile is 2 (wave + NW (i / 2)) + i % 2, so both 64-byte
    // halves of an output line come from one wave, one right after the other
    auto tile_of = [&](int i) { return 2 * (wave + NW * (i >> 1)) + (i & 1); };
    int cad = lane_addr(min(tile_of(0), nt - 1)), nad;
    v4i a[D];
#pragma unroll
    for (int s = 0; s < D; ++s) a[s] = *(const v4i *)(halo + cad + shift(s));
    for (int i = 0, t = tile_of(0); t < nt; t = tile_of(++i)) {
        nad = lane_addr(min(tile_of(i + 1), nt - 1));
        v4i acc[NC];
#pragma unroll
        for (int c = 0; c < NC; ++c) acc[c] = v4i{0, 0, 0, 0};
#pragma unroll
        for (int kb = 0; kb < NKB; ++kb) {
            const int sl = kb % D;
#pragma unroll
            for (int c = 0; c < NC; ++c) acc[c] = mfma_tile<TR>(a[sl], wb[c][kb], acc[c]);
            // the slot is consumed: read k-block kb + D (of this tile, or of the next)
            const int kn = kb + D;
            a[sl] = *(const v4i *)(halo + (kn < NKB ? cad : nad) + shift(kn % NKB));
        }
        cad = nad;
        store_res_tile<NC, TR>(acc, corr, y, g, n, m0, ps + t * kResTile, pe, HWo, rt.vec, li, lg);
    }
}

// The same for layers of 256 to 512 (padded) channels, whose weights do not fit a wave's
// registers whole.  A workgroup owns one group of 32 filters and one contiguous run of output
// positions of one image (the layer is cut into about one workgroup per compute unit).
// It walks K in chunks of CH = 64 CB input channels (128 where a chunk's halo fits the
// staging registers and two chunks fit the LDS, else 64): for each chunk it stages the
// group's weights of the chunk (32 x KH*KW x CH bytes) and the run's halo of the chunk
// (every input pixel the run's positions read, CH channels) in LDS; for each 64-channel
// block of the chunk, each of its 8 waves (two per SIMD) copies the block's weights into
// registers (2 x KH*KW fragments of 16 bytes per lane, 72 registers at 3x3) and adds the
// block's products of its share of the run's 16-position tiles into accumulators it keeps
// for all its tiles.  128-channel chunks halve the chunk round trips (load, LDS write,
// barrier) that the 256-512-channel layers serialise on.  The next chunk is
// requested before the current one's MFMAs and written to the other LDS buffer after
// them (one barrier per chunk); the outputs are stored during the last chunk, each tile's
// as soon as its MFMAs end, so the int32 output writes overlap the last chunk's MFMAs,
// and no wait for a chunk's loads ever has an output store ahead of it (loads and stores
// complete in order on one counter).  Owning 32 filters rather than all of them keeps the
// bytes a compute unit pulls from L2 small (the group's weights and a halo of a longer
// run); that traffic, with every compute unit starting at once, bounds such a kernel, and
// the chunks let the first MFMAs start after one chunk of it.  Operands, output stores
// and the zero point as in the kernel above.
template <int KH, int KW, int CB, bool TR>
__global__ __launch_bounds__(kResThreads) void conv2d_i8_resident_chunked_kernel(const uint8_t *__restrict__ x,
                                                                        const int8_t *__restrict__ wr,
                                                                        const int32_t *__restrict__ pre,
                                                                        int32_t *__restrict__ y, const I8Geom g,
                                                                        const ResTiles rt) {
    constexpr int NT = kResThreads, NW = kResWaves;
    constexpr int NC = 2;                 // 16-filter MFMA tiles per wave
    constexpr int KHW = KH * KW;
    constexpr int CH = 64 * CB;           // input channels per chunk
    constexpr int NKB = KHW * CB;         // k-blocks of a chunk: taps x 64-channel blocks
    constexpr int PIX = CH + 16;          // LDS bytes per halo pixel (16 against bank conflicts)
    constexpr int PPP = CH / 16;          // 16-byte pieces per pixel
    constexpr int HPER = kResHalo;        // halo pieces per thread and chunk
    constexpr int WPIECES = NC * NKB * 64;          // a chunk's weights in 16-byte pieces
    constexpr int WPER = (WPIECES + NT - 1) / NT;
    constexpr int D = KHW % 3 == 0 ? 3 : KHW;       // taps of A fragments read ahead
    extern __shared__ __attribute__((aligned(16))) char smem[];

    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int li = lane & 15, lg = lane >> 4;
    // items ordered (image, run, filter group); XCD x takes a contiguous share, so the
    // filter groups of one run and neighbouring runs (which share halo rows) meet in one L2
    const int xcd = blockIdx.x % kNumXcd, kk = blockIdx.x / kNumXcd;
    const int ib = (int)((int64_t)xcd * rt.items / kNumXcd), ie = (int)((int64_t)(xcd + 1) * rt.items / kNumXcd);
    if (ib + kk >= ie) return;
    const int item = ib + kk;
    const int ngrp = g.Mp / kResGroup;
    const int run = item / ngrp;
    const int m0 = (item - run * ngrp) * kResGroup;
    const int n = run / rt.R, r = run - n * rt.R;
    const int HWo = g.Ho * g.Wo;
    const int ua = (int)((int64_t)r * rt.U / rt.R), ub = (int)((int64_t)(r + 1) * rt.U / rt.R);
    const int ps = ua * kResTile, pe = min(ub * kResTile, HWo), nt = ub - ua;
    const int ho_a = ps / g.Wo, ho_b = (pe - 1) / g.Wo;
    const int hw = g.Wo + KW - 1;                  // halo columns: the padded row
    const int npc = (ho_b - ho_a + KH) * hw * PPP; // 16-byte pieces of a chunk's halo
    const int ih0 = ho_a - g.ph;
    const int flip = g.zero_point ? (int)0x80808080u : 0;
    const int Kw = KHW * g.Cp;                     // bytes of one filter's weights

    const __amdgpu_buffer_rsrc_t xrs =
        __builtin_amdgcn_make_buffer_rsrc((void *)x, (short)0, g.N * g.H * g.W * g.C, 0x00020000);
    const __amdgpu_buffer_rsrc_t wrs = __builtin_amdgcn_make_buffer_rsrc(
        (void *)(wr + (int64_t)m0 * Kw), (short)0, kResGroup * Kw, 0x00020000);
    const FastDiv by_hw(hw);
    // chunk ch into registers: halo piece k = tid + NT u is pixel k / PPP of the halo (row,
    // column), channels ch*CH + (k % PPP)*16 .. +15; weight piece e = tid + NT u is
    // fragment e / 64 = (c, kb), lane e % 64 -> filter m0 + c*16 + (lane & 15), tap kb / CB,
    // channels ch*CH + (kb % CB)*64 + (lane >> 4)*16 .. +15
    auto chunk_load = [&](int ch, v4i (&hv)[HPER], uint32_t &inside, v4i (&wv)[WPER]) {
        const int c0 = ch * CH;
        inside = 0;
#pragma unroll
        for (int u = 0; u < HPER; ++u) {
            const int k = tid + NT * u;
            const int q = k % PPP, rc = k / PPP;
            const int rr = by_hw.div(rc), jc = rc - rr * hw;
            const int ih = ih0 + rr, iw = jc - g.pw;
            const bool in = k < npc && ih >= 0 && ih < g.H && iw >= 0 && iw < g.W && c0 + q * 16 < g.C;
            inside |= in ? 1u << u : 0u;
            hv[u] = load16(xrs, in ? ((n * g.H + ih) * g.W + iw) * g.C + c0 + q * 16 : 0);
        }
#pragma unroll
        for (int u = 0; u < WPER; ++u) {
            const int e = min(tid + NT * u, WPIECES - 1);
            const int f = e >> 6, l = e & 63;
            const int c = f / NKB, kb = f - c * NKB;
            wv[u] = load16(wrs, (c * 16 + (l & 15)) * Kw + (kb / CB) * g.Cp + c0 + (kb % CB) * 64 + (l >> 4) * 16);
        }
    };
    // ... and from registers into LDS buffer buf: the halo at 0, the weights after it, as
    // fragment (c, kb): 1 KB at (c*NKB + kb)*1024, lane l at l*16
    auto chunk_store = [&](int buf, const v4i (&hv)[HPER], uint32_t inside, const v4i (&wv)[WPER]) {
        char *hb = smem + buf * rt.buf;
        char *wl = hb + rt.halo;
        const v4i pad = {flip, flip, flip, flip};
#pragma unroll
        for (int u = 0; u < HPER; ++u) {
            const int k = tid + NT * u;
            if (k < npc) *(v4i *)(hb + (k / PPP) * PIX + (k % PPP) * 16) = ((inside >> u) & 1) ? (hv[u] ^ flip) : pad;
        }
#pragma unroll
        for (int u = 0; u < WPER; ++u) {
            const int e = tid + NT * u;
            if (e < WPIECES) *(v4i *)(wl + e * 16) = wv[u];
        }
    };

    v4i hv[HPER], wv[WPER];
    uint32_t inside;
    chunk_load(0, hv, inside, wv);
    // the zero-point correction of this lane's filters
    constexpr int full = KH * (KW + 1) + KW;   // prefix-table entry of the whole filter
    const __amdgpu_buffer_rsrc_t prs = __builtin_amdgcn_make_buffer_rsrc(
        (void *)pre, (short)0, g.M * (KH + 1) * (KW + 1) * 4, 0x00020000);
    // (in registers for lane li's filters; with TR, where a lane stores four filters, in
    // LDS after the two chunk buffers and read back only for the stores)
    int32_t corr[NC][1];
    int32_t *corr_lds = (int32_t *)(smem + 2 * rt.buf);
    if constexpr (TR) {
        if (tid < kResGroup) {
            const int m = min(m0 + tid, g.M - 1);
            corr_lds[tid] = __builtin_amdgcn_raw_buffer_load_b32(prs, (m * (KH + 1) * (KW + 1) + full) * 4, 0, 0);
        }
    } else {
#pragma unroll
        for (int c = 0; c < NC; ++c) {
            const int m = min(m0 + c * 16 + li, g.M - 1);
            corr[c][0] = __builtin_amdgcn_raw_buffer_load_b32(prs, (m * (KH + 1) * (KW + 1) + full) * 4, 0, 0);
        }
    }
    chunk_store(0, hv, inside, wv);
    __syncthreads();

    // halo offset of this lane's A row (position) in tile t, at tap (0, 0); lanes past the
    // run read its last position (their sums are not stored)
    const FastDiv by_wo(g.Wo);
    auto lane_addr = [&](int t) {
        const int pos = min(ps + t * kResTile + li, pe - 1);
        const int ho = by_wo.div(pos), wo = pos - ho * g.Wo;
        return ((ho - ho_a) * hw + wo) * PIX + lg * 16;
    };
    const int rowsh = hw * PIX;
    auto shift = [&](int tap) {   // tap is a compile-time constant after unrolling
        return (tap / KW) * rowsh + (tap % KW) * PIX;
    };
    auto store_tile = [&](const v4i (&acc)[NC], int t) {
        if constexpr (TR) {
            int32_t cr[NC][4];
#pragma unroll
            for (int c = 0; c < NC; ++c) {
                const v4i cv = *(const v4i *)(corr_lds + c * 16 + lg * 4);
#pragma unroll
                for (int v = 0; v < 4; ++v) cr[c][v] = cv[v];
            }
            store_res_tile<NC, TR>(acc, cr, y, g, n, m0, ps + t * kResTile, pe, HWo, rt.vec, li, lg);
        } else {
            store_res_tile<NC, TR>(acc, corr, y, g, n, m0, ps + t * kResTile, pe, HWo, rt.vec, li, lg);
        }
    };

    v4i acc[kResTPW][NC];
#pragma unroll
    for (int tt = 0; tt < kResTPW; ++tt)
#pragma unroll
        for (int c = 0; c < NC; ++c) acc[tt][c] = v4i{0, 0, 0, 0};
    for (int ch = 0; ch < rt.nch; ++ch) {
        const bool more = ch + 1 < rt.nch;
        if (more) chunk_load(ch + 1, hv, inside, wv);
        const char *hb = smem + (ch & 1) * rt.buf;
        const char *wl = hb + rt.halo;
#pragma unroll
        for (int h = 0; h < CB; ++h) {
            // this wave's copy of the weights of the chunk's 64-channel block h: B fragment
            // (c, tap) is column li (filter m0 + c*16 + li), channels ch*CH + h*64 + lg*16 .. +15
            v4i wb[NC][KHW];
#pragma unroll
            for (int c = 0; c < NC; ++c)
#pragma unroll
                for (int kb = 0; kb < KHW; ++kb)
                    wb[c][kb] = *(const v4i *)(wl + (c * NKB + kb * CB + h) * 1024 + lane * 16);
            // tiles wave, wave + NW, ... of the run; the first D taps of the next tile are
            // read while a tile's last MFMAs run
            const char *hh = hb + h * 64;
            int cad = lane_addr(min(wave, nt - 1));
            v4i a[D];
#pragma unroll
            for (int s = 0; s < D; ++s) a[s] = *(const v4i *)(hh + cad + shift(s));
#pragma unroll
            for (int tt = 0; tt < kResTPW; ++tt) {
                const int t = wave + tt * NW;
                if (t < nt) {
                    const int nad = lane_addr(min(t + NW, nt - 1));
#pragma unroll
                    for (int kb = 0; kb < KHW; ++kb) {
                        const int sl = kb % D;
#pragma unroll
                        for (int c = 0; c < NC; ++c)
                            acc[tt][c] = mfma_tile<TR>(a[sl], wb[c][kb], acc[tt][c]);
                        const int kn = kb + D;
                        a[sl] = *(const v4i *)(hh + (kn < KHW ? cad : nad) + shift(kn % KHW));
                    }
                    cad = nad;
                    if (!more && h == CB - 1) store_tile(acc[tt], t);
                }
            }
        }
        if (more) {
            chunk_store((ch + 1) & 1, hv, inside, wv);
            __syncthreads();
        }
    }
}

// Packed-row implicit GEMM for layers with few input channels (an image network's first
// layer: 3 channels), where padding C to a 64-channel K step would spend most of the
// matrix-core work and most of the activation reads on zeros (at 3 channels and 3x3,
// 27 useful bytes of K = 576).  In NHWC the KW pixels one kernel row covers at an output
// position are KW*C consecutive bytes, whatever the stride, so K is laid out by kernel
// row: row kh owns rs = ceil(KW*C / 16) slots of 16 bytes, four slots per 64-byte k-block
// (3x3 on 3 channels: one k-block; 11x11 on 3 channels: nine, against 121).  The weight
// fragments of up to 128 filters (the prepared packed layout) are staged in LDS once per
// workgroup; each lane builds its A fragment (16 bytes of one position's slot) from five
// aligned 4-byte loads, a byte shift, and a mask that puts the padding value on bytes of
// pixels outside the image (skipped where the whole window lies inside).  The next step's
// loads (the next k-block, or the next tile's first) are issued before a step's MFMAs,
// and a tile's outputs are stored after the next tile's first loads, so no wait for
// operands has that tile's stores ahead of it.  Output layouts (TR) and the zero point as
// in the weight-resident kernels; the corrections sit in LDS after the fragments.
constexpr int kPkThreads = 256;
constexpr int kPkWaves = kPkThreads / 64;
constexpr int kPkBlocks = 8;    // 16-filter MFMA column blocks per workgroup at most
constexpr int kPkMaxKb = 16;    // k-blocks at most (LDS: 8 blocks x 16 k-blocks x 1 KB)

struct PkTiles {
    int tiles_img;   // 16-position tiles per image
    int tiles;       // N * tiles_img
    int tpw;         // tiles per wave
    int items;       // workgroups along the positions: ceil(tiles / (4 tpw))
    int vec;         // 1: 16-byte output stores
};

template <bool TR>
__global__ __launch_bounds__(kPkThreads) void conv2d_i8_packed_kernel(const uint8_t *__restrict__ x,
                                                                      const int8_t *__restrict__ wk,
                                                                      const int32_t *__restrict__ pre,
                                                                      int32_t *__restrict__ y, const I8Geom g,
                                                                      const PkTiles pt) {
    extern __shared__ __attribute__((aligned(16))) char smem[];
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int li = lane & 15, lg = lane >> 4;
    // items dealt per XCD in contiguous shares: neighbouring tiles read the same input rows
    const int xcd = blockIdx.x % kNumXcd, kk = blockIdx.x / kNumXcd;
    const int ib = (int)((int64_t)xcd * pt.items / kNumXcd), ie = (int)((int64_t)(xcd + 1) * pt.items / kNumXcd);
    if (ib + kk >= ie) return;
    const int item = ib + kk;
    const int nkb = g.pkb;
    const int cb0 = blockIdx.y * kPkBlocks;
    const int ncb = min(kPkBlocks, (g.M + 15) / 16 - cb0);

    // the group's fragments (cb0 + c, kb) to LDS at (c * nkb + kb) * 1024, and after them
    // the zero-point correction (128 x the filter's sum) of each of the group's filters
    {
        const v4i *src = (const v4i *)(wk + (int64_t)cb0 * nkb * 1024);
        const int pieces = ncb * nkb * 64;
        for (int e = tid; e < pieces; e += kPkThreads) *(v4i *)(smem + e * 16) = src[e];
    }
    int32_t *corr = (int32_t *)(smem + ncb * nkb * 1024);
    if (tid < ncb * 16) {
        const int pstride = (g.KH + 1) * (g.KW + 1);
        const int m = min(cb0 * 16 + tid, g.M - 1);
        corr[tid] = g.zero_point ? 128 * pre[m * pstride + pstride - 1] : 0;
    }
    const int flip = g.zero_point ? (int)0x80808080u : 0;
    __syncthreads();

    const int HWo = g.Ho * g.Wo;
    const FastDiv by_wo(g.Wo), by_rs(g.rs);
    const int slots = g.KH * g.rs;
    const int nrec = g.N * g.H * g.W * g.C;   // a whole number of 4-byte words, at least one
    const __amdgpu_buffer_rsrc_t xrs = __builtin_amdgcn_make_buffer_rsrc((void *)x, (short)0, nrec, 0x00020000);

    // a lane's position in tile i of the wave (tiles item*4*tpw + 4 i + wave)
    struct Geo {
        int n, p0;    // image, first position of the tile
        int row0;     // (n*H + ho*sh - ph)*W + wo*sw - pw: the window's first pixel at kernel row 0
        int ih0;      // ho*sh - ph
        int jl, jh;   // window bytes inside the image: [jl, jh)
    };
    auto geo = [&](int i, Geo &o) {
        const int t = item * kPkWaves * pt.tpw + kPkWaves * i + wave;
        if (i >= pt.tpw || t >= pt.tiles) return false;
        o.n = t / pt.tiles_img;
        o.p0 = (t - o.n * pt.tiles_img) * 16;
        const int pos = min(o.p0 + li, HWo - 1);
        const int ho = by_wo.div(pos), wo = pos - ho * g.Wo;
        o.ih0 = ho * g.sh - g.ph;
        const int iw0 = wo * g.sw - g.pw;
        o.row0 = (o.n * g.H + o.ih0) * g.W + iw0;
        // a window inside the image leaves its bytes past KW*C unmasked (their weights are
        // zero), so every slot of an inside window takes the unmasked path below
        o.jl = max(0, -iw0) * g.C;
        o.jh = iw0 + g.KW <= g.W ? 1 << 20 : (g.W - iw0) * g.C;
        return true;
    };
    // step (tile geometry, k-block kb): the lane's five dwords, byte shift and valid range
    struct Ld {
        uint32_t r[5];
        int sb, lo, hi;
    };
    auto issue = [&](const Geo &o, int kb, Ld &ld) {
        const int sl = kb * 4 + lg;
        const int ky = by_rs.div(sl), part = sl - ky * g.rs;
        const int ih = o.ih0 + ky;
        const bool ok = sl < slots && ih >= 0 && ih < g.H;
        const int off = (o.row0 + ky * g.W) * g.C + part * 16;
        ld.lo = ok ? o.jl - part * 16 : 16;
        ld.hi = ok ? o.jh - part * 16 : 0;
        ld.sb = off & 3;
        // each word's offset clamped into the activations: a word before the first byte or
        // past the last holds only bytes of pixels outside the image (or past the window),
        // which the mask replaces, so every load stays in range (and the clamps keep the
        // five loads from being merged into one wider load)
        const int a = ok ? off - ld.sb : 0;
#pragma unroll
        for (int d = 0; d < 5; ++d)
            ld.r[d] = __builtin_amdgcn_raw_buffer_load_b32(xrs, min(max(a + 4 * d, 0), nrec - 4), 0, 0);
    };
    auto build = [&](const Ld &ld) {
        v4i a;
        if (ld.lo <= 0 && ld.hi >= 16) {   // every byte inside the image (or past the window)
#pragma unroll
            for (int d = 0; d < 4; ++d)
                a[d] = (int)(__builtin_amdgcn_alignbyte(ld.r[d + 1], ld.r[d], (uint32_t)ld.sb) ^ (uint32_t)flip);
        } else {
#pragma unroll
            for (int d = 0; d < 4; ++d) {
                const uint32_t v = __builtin_amdgcn_alignbyte(ld.r[d + 1], ld.r[d], (uint32_t)ld.sb);
                const int lo = min(max(ld.lo - 4 * d, 0), 4), hi = min(max(ld.hi - 4 * d, 0), 4);
                const uint32_t m = hi > lo ? (uint32_t)((0xFFFFFFFFull << (8 * lo)) & ((1ull << (8 * hi)) - 1)) : 0u;
                a[d] = (int)(((v ^ (uint32_t)flip) & m) | ((uint32_t)flip & ~m));
            }
        }
        return a;
    };
    // the tile's outputs in mfma_tile's layouts (TR: position o.p0 + li of filters
    // 4 lg .. 4 lg + 3 of each 16-filter block; else positions o.p0 + 4 lg .. of filter li)
    auto store = [&](const v4i (&acc)[kPkBlocks], const Geo &o) {
        if constexpr (TR) {
            const int pos = o.p0 + li;
            if (pos >= HWo) return;
            int32_t *yb = y + ((int64_t)o.n * g.M + cb0 * 16 + lg * 4) * HWo + pos;   // filter cb0*16 + 4 lg
#pragma unroll
            for (int c = 0; c < kPkBlocks; ++c) {
                if (c >= ncb) continue;
                const v4i cv = *(const v4i *)(corr + c * 16 + lg * 4);
#pragma unroll
                for (int v = 0; v < 4; ++v)
                    if ((cb0 + c) * 16 + lg * 4 + v < g.M)
                        __builtin_nontemporal_store(acc[c][v] + cv[v], yb + (int64_t)(c * 16 + v) * HWo);
            }
        } else {
            const int q0 = o.p0 + lg * 4;
#pragma unroll
            for (int c = 0; c < kPkBlocks; ++c) {
                const int m = (cb0 + c) * 16 + li;
                if (c >= ncb || m >= g.M) continue;
                int32_t *ym = y + ((int64_t)o.n * g.M + m) * HWo;
                const v4i v = acc[c] + corr[c * 16 + li];
                if (pt.vec) {
                    if (q0 < HWo) __builtin_nontemporal_store(v, (v4i *)(ym + q0));
                } else {
#pragma unroll
                    for (int e = 0; e < 4; ++e)
                        if (q0 + e < HWo) ym[q0 + e] = v[e];
                }
            }
        }
    };

    Geo cur;
    if (!geo(0, cur)) return;
    Ld ld;
    issue(cur, 0, ld);
    v4i acc[kPkBlocks];
#pragma unroll
    for (int c = 0; c < kPkBlocks; ++c) acc[c] = v4i{0, 0, 0, 0};
    int i = 0, kb = 0;
    while (true) {
        const v4i a = build(ld);
        // the next step: the next k-block of this tile, or the first of the next tile
        Geo nxt = cur;
        int i2 = i, kb2 = kb + 1;
        bool more = true;
        if (kb2 == nkb) {
            kb2 = 0;
            i2 = i + 1;
            more = geo(i2, nxt);
        }
        if (more) issue(nxt, kb2, ld);
        const char *bf = smem + kb * 1024 + lane * 16;
#pragma unroll
        for (int c = 0; c < kPkBlocks; ++c)
            if (c < ncb)
                acc[c] = mfma_tile<TR>(a, *(const v4i *)(bf + c * nkb * 1024), acc[c]);
        if (kb == nkb - 1) {
            store(acc, cur);
#pragma unroll
            for (int c = 0; c < kPkBlocks; ++c) acc[c] = v4i{0, 0, 0, 0};
        }
        if (!more) break;
        cur = nxt;
        i = i2;
        kb = kb2;
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
    // the packed-row K where it at most halves the padded layout's k-blocks, with 32-bit
    // byte offsets into the activations, activations a whole number of 4-byte words (no
    // word straddles the end, which a range-checked load would read as zero), positions
    // below 2^22, output rows below 2^12 (fast divisions) and the group's fragments in LDS
    g.rk = d.KW * d.C;
    g.rs = (g.rk + 15) / 16;
    g.pkb = (d.KH * g.rs + 3) / 4;
    const bool pk = 2 * g.pkb <= d.KH * d.KW * g.Cp / 64 && g.pkb <= kPkMaxKb &&
                    (int64_t)d.N * d.H * d.W * d.C + 64 < INT32_MAX && (int64_t)d.N * d.H * d.W * d.C % 4 == 0 &&
                    (int64_t)g.Ho * g.Wo < (1 << 22) &&
                    g.Wo < 4096 && (int64_t)d.N * ((int64_t)g.Ho * g.Wo + 15) / 16 < INT32_MAX / 2;
    if (!pk) g.pkb = 0;
    return g;
}

size_t align256(size_t v) { return (v + 255) / 256 * 256; }

size_t packed_bytes(const I8Geom &g) { return g.pkb ? align256((size_t)((g.M + 15) / 16) * g.pkb * 1024) : 0; }

}  // namespace

size_t conv2d_i8_workspace_bytes(const samd_conv2d_desc &d, samd_fmt xf) {
    I8Geom g = make_geom(d, xf);
    size_t wr = align256((size_t)g.Mp * g.KH * g.KW * g.Cp);
    size_t pre = align256((size_t)g.M * (g.KH + 1) * (g.KW + 1) * 4);
    return wr + pre + packed_bytes(g);
}

namespace {

struct I8Workspace {
    int8_t *wr;
    int32_t *pre;
    int8_t *wk;   // packed-row weight fragments (null where that layout is not offered)
};

I8Workspace carve(const I8Geom &g, void *ws) {
    I8Workspace w;
    w.wr = (int8_t *)ws;
    const size_t wr = align256((size_t)g.Mp * g.KH * g.KW * g.Cp);
    w.pre = (int32_t *)((char *)ws + wr);
    w.wk = g.pkb ? (int8_t *)ws + wr + align256((size_t)g.M * (g.KH + 1) * (g.KW + 1) * 4) : nullptr;
    return w;
}

}  // namespace

int launch_conv2d_i8_prepare(const int8_t *w, samd_fmt xf, const samd_conv2d_desc &d, void *ws, hipStream_t s) {
    const I8Geom g = make_geom(d, xf);
    const I8Workspace p = carve(g, ws);
    const int pgrid = grid_for((int64_t)g.Mp * g.KH * g.KW * g.Cp, 256);
    hipLaunchKernelGGL(i8_prep_kernel, dim3(pgrid), dim3(256), 0, s, w, g, p.wr, p.pre, p.wk);
    return check_launch("conv2d_int8 weight reorder");
}

namespace {

constexpr int kHaloShapes[4][2] = {{32, 128}, {32, 64}, {16, 128}, {16, 64}};   // (WM, TP)

// Tiling of the halo kernel for (WM, TP); false when the halo does not fit the LDS (one
// buffer, or two when there are several chunks) or the register-held halo pieces.
bool halo_tiles(const I8Geom &g, int wm, int tp, HaloTiles &ht, int64_t &wgs, int &lds) {
    int rmax, hwmax;
    if (g.Wo < tp) {   // flat tiles: whole padded rows
        ht.rowseg = 0;
        ht.tiles_img = (g.Ho * g.Wo + tp - 1) / tp;
        ht.segs = 1;
        rmax = std::min(g.Ho, (tp - 1) / g.Wo + 2) + g.KH - 1;
        hwmax = g.Wo + g.KW - 1;
    } else {           // row segments
        ht.rowseg = 1;
        ht.segs = (g.Wo + tp - 1) / tp;
        ht.tiles_img = g.Ho * ht.segs;
        rmax = g.KH;
        hwmax = tp + g.KW - 1;
    }
    // the kernel's fast divisions need positions per image below 2^22, divisors below 2^12
    if ((int64_t)g.Ho * g.Wo >= (1 << 22) || g.Wo >= 4096 || hwmax >= 4096) return false;
    const int64_t pixels = (int64_t)rmax * hwmax;
    wgs = (int64_t)g.N * ht.tiles_img * ((g.M + 4 * wm - 1) / (4 * wm));
    ht.items = (int)std::min<int64_t>(wgs, INT32_MAX);
    if (wgs >= ((int64_t)1 << 31) - 8) return false;
    // chunks of the weight layout's K step, or of 64 channels where a 128-channel chunk's
    // halo does not fit (the weights of a chunk are the same bytes either way)
    const int opts[2] = {g.ks, 64};
    for (int o = 0; o < (g.ks == 64 ? 1 : 2); ++o) {
        const int kc = opts[o];
        ht.kc = kc;
        ht.halo_bytes = (int)std::min<int64_t>(pixels * (kc + 16), 1 << 30);
        ht.nch = g.Cp / kc;
        lds = (ht.nch > 1 ? 2 : 1) * ht.halo_bytes;
        if (pixels * (kc / 16) <= kHaloPieces && lds <= kHaloMaxLds) return true;
    }
    return false;
}

template <int WM, int TP, int KC>
int launch_halo(const void *x, const I8Geom &g, const HaloTiles &ht, int lds, const I8Workspace &p, int32_t *y,
                hipStream_t s) {
    const void *fn = (const void *)conv2d_i8_halo_kernel<WM, TP, KC>;
    // more than the default 64 KiB of dynamic LDS is opted into once per kernel
    static std::once_flag once;
    static hipError_t attr = hipSuccess;
    std::call_once(once, [&] { attr = hipFuncSetAttribute(fn, hipFuncAttributeMaxDynamicSharedMemorySize, kHaloMaxLds); });
    if (attr != hipSuccess) {
        set_error(std::string("conv2d_int8: LDS attribute: ") + hipGetErrorString(attr));
        return SAMD_EHIP;
    }
    // every XCD gets the same number of workgroups, enough for its share of the items
    const int64_t per_xcd = ((int64_t)ht.items + kNumXcd - 1) / kNumXcd;
    const dim3 grid((unsigned)(per_xcd * kNumXcd));
    hipLaunchKernelGGL((conv2d_i8_halo_kernel<WM, TP, KC>), grid, dim3(256), (size_t)lds, s, (const uint8_t *)x,
                       p.wr, p.pre, y, g, ht);
    return check_launch("conv2d_int8 (halo tiles)");
}

// Position runs of the weight-resident kernels: R runs per image, so that the layer
// gives about `target` workgroups; false when the layer is not one they serve or a run's
// halo exceeds the LDS or the register-held pieces.  Padded channels up to 128: the
// kernel that holds a filter's whole K in registers; 256 to 512: the chunked kernel (no
// run of more than kResTPW tiles per wave).
bool res_tiles(const I8Geom &g, int target, ResTiles &rt, int &lds, int64_t &wgs, int &positions) {
    if (g.sh != 1 || g.sw != 1 || g.C % 16 != 0) return false;
    if (!((g.KH == 3 && g.KW == 3) || (g.KH == 1 && g.KW == 1))) return false;
    const bool chunked = g.Cp > 128;
    if (g.Cp % kResChunk != 0 || g.Cp / kResChunk > kResMaxChunks) return false;
    const int64_t HWo = (int64_t)g.Ho * g.Wo;
    const int hw = g.Wo + g.KW - 1;
    // fast divisions (positions below 2^22, divisors below 2^12) and 32-bit byte offsets
    if (HWo >= (1 << 22) || hw >= 4096 || (int64_t)g.N * g.H * g.W * g.C >= INT32_MAX) return false;
    if ((int64_t)g.Mp * g.KH * g.KW * g.Cp >= INT32_MAX) return false;
    const int ngrp = g.Mp / kResGroup;
    rt.U = (int)((HWo + kResTile - 1) / kResTile);
    const int64_t per_img = (int64_t)g.N * ngrp;
    int64_t R = std::max<int64_t>(1, (target + per_img - 1) / per_img);
    if (chunked) R = std::max<int64_t>(R, (rt.U + kResTPW * kResWaves - 1) / (kResTPW * kResWaves));
    rt.R = (int)std::min<int64_t>(rt.U, R);
    const int maxu = (rt.U + rt.R - 1) / rt.R;
    positions = (int)std::min<int64_t>(HWo, (int64_t)maxu * kResTile);
    // rows a run of that many positions spans (starting anywhere in a row), and its halo
    const int64_t rows = std::min<int64_t>(g.Ho, (positions - 1) / g.Wo + 2) + g.KH - 1;
    const int64_t pixels = rows * hw;
    // channels in LDS at a time: the whole K up to 128 padded channels; above, chunks of
    // 128 channels where a chunk's halo fits the registers that stage it and two chunks
    // fit the LDS, else of 64
    auto bytes = [&](int kc, int64_t &halo) {
        halo = (pixels * (kc + 16) + 15) / 16 * 16;
        return halo + (int64_t)kResGroup * g.KH * g.KW * kc;
    };
    int64_t halo;
    int kc = g.Cp;
    if (chunked) {
        kc = g.Cp % 128 == 0 && pixels * 8 <= (int64_t)kResHalo * kResThreads &&
                     2 * bytes(128, halo) + kResGroup * 4 <= kHaloMaxLds
                 ? 128 : kResChunk;
    }
    const int64_t buf = bytes(kc, halo);
    rt.nch = g.Cp / kc;
    rt.halo = (int)std::min<int64_t>(halo, INT32_MAX);
    rt.buf = (int)std::min<int64_t>(buf, INT32_MAX);
    // chunked: two chunk buffers, then the group's zero-point corrections (transposed stores)
    const int64_t total = chunked ? 2 * buf + kResGroup * 4 : buf;
    lds = (int)std::min<int64_t>(total, INT32_MAX);
    wgs = (int64_t)g.N * rt.R * ngrp;
    rt.items = (int)std::min<int64_t>(wgs, INT32_MAX);
    const bool pieces = chunked ? (maxu <= kResTPW * kResWaves && pixels * (kc / 16) <= (int64_t)kResHalo * kResThreads)
                                : pixels * (kc / 16) <= kResPieces;
    return pieces && total <= kHaloMaxLds && wgs < ((int64_t)1 << 31) - 8;
}

// 16-byte output stores where every image's positions are a multiple of 4 and the output
// 16-byte aligned; else the transposed tile layout (64-byte runs of one filter's positions)
bool vec_out(const I8Geom &g, const int32_t *y) {
    return ((int64_t)g.Ho * g.Wo) % 4 == 0 && ((uintptr_t)y % 16) == 0;
}

template <typename F>
int launch_res_kernel(F kernel, const void *x, const I8Geom &g, ResTiles rt, int lds, const I8Workspace &p,
                      int32_t *y, hipStream_t s, std::once_flag &once, hipError_t &attr) {
    std::call_once(once, [&] {
        attr = hipFuncSetAttribute((const void *)kernel, hipFuncAttributeMaxDynamicSharedMemorySize, kHaloMaxLds);
    });
    if (attr != hipSuccess) {
        set_error(std::string("conv2d_int8: LDS attribute: ") + hipGetErrorString(attr));
        return SAMD_EHIP;
    }
    rt.vec = vec_out(g, y);
    const int64_t per_xcd = ((int64_t)rt.items + kNumXcd - 1) / kNumXcd;
    hipLaunchKernelGGL(kernel, dim3((unsigned)(per_xcd * kNumXcd)), dim3(kResThreads), (size_t)lds, s,
                       (const uint8_t *)x, (const int8_t *)p.wr, (const int32_t *)p.pre, y, g, rt);
    return check_launch("conv2d_int8 (weight-resident)");
}

template <int KH, int KW, int CB, bool TR>
int launch_res_tr(const void *x, const I8Geom &g, const ResTiles &rt, int lds, const I8Workspace &p, int32_t *y,
                  hipStream_t s) {
    static std::once_flag once;
    static hipError_t attr = hipSuccess;
    return launch_res_kernel(conv2d_i8_resident_kernel<KH, KW, CB, TR>, x, g, rt, lds, p, y, s, once, attr);
}

template <int KH, int KW, int CB>
int launch_res(const void *x, const I8Geom &g, const ResTiles &rt, int lds, const I8Workspace &p, int32_t *y,
               hipStream_t s) {
    return vec_out(g, y) ? launch_res_tr<KH, KW, CB, false>(x, g, rt, lds, p, y, s)
                         : launch_res_tr<KH, KW, CB, true>(x, g, rt, lds, p, y, s);
}

template <int KH, int KW, int CB, bool TR>
int launch_res_chunked_tr(const void *x, const I8Geom &g, const ResTiles &rt, int lds, const I8Workspace &p,
                          int32_t *y, hipStream_t s) {
    static std::once_flag once;
    static hipError_t attr = hipSuccess;
    return launch_res_kernel(conv2d_i8_resident_chunked_kernel<KH, KW, CB, TR>, x, g, rt, lds, p, y, s, once, attr);
}

template <int KH, int KW, int CB>
int launch_res_chunked_cb(const void *x, const I8Geom &g, const ResTiles &rt, int lds, const I8Workspace &p,
                          int32_t *y, hipStream_t s) {
    return vec_out(g, y) ? launch_res_chunked_tr<KH, KW, CB, false>(x, g, rt, lds, p, y, s)
                         : launch_res_chunked_tr<KH, KW, CB, true>(x, g, rt, lds, p, y, s);
}

template <int KH, int KW>
int launch_res_chunked(const void *x, const I8Geom &g, const ResTiles &rt, int lds, const I8Workspace &p, int32_t *y,
                       hipStream_t s) {
    return g.Cp / rt.nch == 128 ? launch_res_chunked_cb<KH, KW, 2>(x, g, rt, lds, p, y, s)
                                : launch_res_chunked_cb<KH, KW, 1>(x, g, rt, lds, p, y, s);
}

int launch_res_any(const void *x, const I8Geom &g, const ResTiles &rt, int lds, const I8Workspace &p, int32_t *y,
                   hipStream_t s) {
    const bool k3 = g.KH == 3 && g.KW == 3, k1 = g.KH == 1 && g.KW == 1;
    if (g.Cp > 128) {
        if (k3) return launch_res_chunked<3, 3>(x, g, rt, lds, p, y, s);
        if (k1) return launch_res_chunked<1, 1>(x, g, rt, lds, p, y, s);
    } else if (g.Cp == 128) {
        if (k3) return launch_res<3, 3, 2>(x, g, rt, lds, p, y, s);
        if (k1) return launch_res<1, 1, 2>(x, g, rt, lds, p, y, s);
    } else {
        if (k3) return launch_res<3, 3, 1>(x, g, rt, lds, p, y, s);
        if (k1) return launch_res<1, 1, 1>(x, g, rt, lds, p, y, s);
    }
    set_error("conv2d_int8: no weight-resident kernel for this layer");
    return SAMD_EUNSUPPORTED;
}

constexpr int kResTargets[2] = {256, 512};   // workgroups: one per compute unit, or two

// Tiling of the packed-row kernel with tpw 16-position tiles per wave; false where the
// layer does not take the packed-row K.
bool pk_tiles(const I8Geom &g, int tpw, PkTiles &pt, int &lds, int64_t &wgs) {
    if (!g.pkb) return false;
    const int64_t HWo = (int64_t)g.Ho * g.Wo;
    pt.tiles_img = (int)((HWo + 15) / 16);
    pt.tiles = g.N * pt.tiles_img;
    pt.tpw = tpw;
    pt.items = (int)(((int64_t)pt.tiles + kPkWaves * tpw - 1) / (kPkWaves * tpw));
    pt.vec = 0;
    const int nblk = (g.M + 15) / 16;
    lds = std::min(kPkBlocks, nblk) * g.pkb * 1024 + kPkBlocks * 16 * 4;
    wgs = (int64_t)pt.items * ((nblk + kPkBlocks - 1) / kPkBlocks);
    return lds <= kHaloMaxLds && wgs < ((int64_t)1 << 31) - 8;
}

constexpr int kPkTpw[3] = {4, 2, 1};   // tiles per wave of the packed-row candidates

template <bool TR>
int launch_packed_tr(const void *x, const I8Geom &g, PkTiles pt, int lds, const I8Workspace &p, int32_t *y,
                     hipStream_t s) {
    static std::once_flag once;
    static hipError_t attr = hipSuccess;
    std::call_once(once, [&] {
        attr = hipFuncSetAttribute((const void *)conv2d_i8_packed_kernel<TR>,
                                   hipFuncAttributeMaxDynamicSharedMemorySize, kHaloMaxLds);
    });
    if (attr != hipSuccess) {
        set_error(std::string("conv2d_int8: LDS attribute: ") + hipGetErrorString(attr));
        return SAMD_EHIP;
    }
    pt.vec = vec_out(g, y);
    const int64_t per_xcd = ((int64_t)pt.items + kNumXcd - 1) / kNumXcd;
    const unsigned gy = (unsigned)(((g.M + 15) / 16 + kPkBlocks - 1) / kPkBlocks);
    hipLaunchKernelGGL(conv2d_i8_packed_kernel<TR>, dim3((unsigned)(per_xcd * kNumXcd), gy), dim3(kPkThreads),
                       (size_t)lds, s, (const uint8_t *)x, (const int8_t *)p.wk, (const int32_t *)p.pre, y, g, pt);
    return check_launch("conv2d_int8 (packed rows)");
}

int launch_packed(const void *x, const I8Geom &g, const PkTiles &pt, int lds, const I8Workspace &p, int32_t *y,
                  hipStream_t s) {
    return vec_out(g, y) ? launch_packed_tr<false>(x, g, pt, lds, p, y, s)
                         : launch_packed_tr<true>(x, g, pt, lds, p, y, s);
}

// Every launch the int8 baseline can make for a layer: the halo tiles that fit (stride-1
// layers, C a multiple of 16), then the im2col kernel with 64 and 32 positions per
// workgroup.
void int8_candidates(const I8Geom &g, std::vector<samd_conv2d_int8_plan> &out) {
    out.clear();
    for (int tpw : kPkTpw) {
        PkTiles pt{};
        int lds = 0;
        int64_t wgs = 0;
        if (!pk_tiles(g, tpw, pt, lds, wgs)) continue;
        samd_conv2d_int8_plan c{};
        c.halo = 3;
        c.mtile = std::min(kPkBlocks, (g.M + 15) / 16) * 16;
        c.positions = kPkWaves * kResTile * tpw;
        c.row_segments = 0;
        c.lds_bytes = lds;
        c.waves = kPkWaves;
        c.workgroups = wgs;
        out.push_back(c);
    }
    if (g.sh == 1 && g.sw == 1 && g.C % 16 == 0) {
        for (const auto &sh : kHaloShapes) {
            HaloTiles ht{};
            int64_t wgs = 0;
            int lds = 0;
            if (!halo_tiles(g, sh[0], sh[1], ht, wgs, lds)) continue;
            samd_conv2d_int8_plan c{};
            c.halo = 1;
            c.mtile = 4 * sh[0];
            c.positions = sh[1];
            c.row_segments = ht.rowseg;
            c.lds_bytes = lds;
            c.waves = 4;
            c.workgroups = wgs;
            out.push_back(c);
        }
        for (int target : kResTargets) {
            ResTiles rt{};
            int64_t wgs = 0;
            int lds = 0, positions = 0;
            if (!res_tiles(g, target, rt, lds, wgs, positions)) continue;
            samd_conv2d_int8_plan c{};
            c.halo = 2;
            c.mtile = kResGroup;
            c.positions = positions;
            c.row_segments = 0;
            c.lds_bytes = lds;
            c.waves = kResWaves;
            c.workgroups = wgs;
            bool dup = false;
            for (const auto &o : out) dup = dup || (o.halo == 2 && o.positions == positions);
            if (!dup) out.push_back(c);
        }
    }
    for (int tp : {64, 32}) {
        samd_conv2d_int8_plan c{};
        c.halo = 0;
        c.mtile = kTM;
        c.positions = tp;
        c.lds_bytes = 0;
        c.waves = 4;
        c.workgroups = (g.P + tp - 1) / tp * (g.Mp / kTM);
        out.push_back(c);
    }
}

// The model's choice among the candidates: the weight-resident launch of one workgroup
// per compute unit (at most 256 workgroups, at least 160); else in the order 64 x 128, 128 x 128, 64 x 64,
// 128 x 64 (output channels x positions; the order of their times on the mid-size layer),
// the first halo tile that still gives at least 160 workgroups (about two thirds of the
// compute units), else the halo tile with the most workgroups, else the im2col kernel
// with 64 positions when that gives every compute unit a workgroup, else 32.
samd_conv2d_int8_plan model_choice(const std::vector<samd_conv2d_int8_plan> &cands) {
    // the packed-row kernel where the layer takes it (few input channels), with the most
    // tiles per wave that still gives every compute unit a workgroup
    const samd_conv2d_int8_plan *pk = nullptr;
    for (const auto &c : cands) {
        if (c.halo != 3) continue;
        if (c.workgroups >= 256) return c;
        pk = &c;   // from 4 tiles per wave down to 1: the last has the most workgroups
    }
    if (pk) return *pk;
    // the weight-resident kernel with about one workgroup per compute unit, when the layer
    // fills at least two thirds of them
    for (const auto &c : cands)
        if (c.halo == 2 && c.workgroups >= 160 && c.workgroups <= 256) return c;
    static const int order[4][2] = {{64, 128}, {128, 128}, {64, 64}, {128, 64}};
    for (const auto &o : order)
        for (const auto &c : cands)
            if (c.halo == 1 && c.mtile == o[0] && c.positions == o[1] && c.workgroups >= 160) return c;
    int most = -1;
    for (size_t i = 0; i < cands.size(); ++i) {
        if (cands[i].halo != 1) continue;
        if (most < 0 || cands[i].workgroups > cands[most].workgroups) most = (int)i;
    }
    if (most >= 0) return cands[most];
    for (const auto &c : cands)
        if (!c.halo && c.positions == 64 && c.workgroups >= 256) return c;
    return cands.back();
}

// Plans installed by samd_conv2d_int8_use_plan, per (shape, activation format).
using Int8Key = std::array<int32_t, 13>;
std::mutex int8_mu;
std::map<Int8Key, samd_conv2d_int8_plan> int8_plans;

Int8Key int8_key(const samd_conv2d_desc &d, samd_fmt xf) {
    return {d.N, d.C, d.H, d.W, d.M, d.KH, d.KW, d.stride_h, d.stride_w, d.pad_h, d.pad_w, xf.bits, xf.is_signed};
}

bool same_launch(const samd_conv2d_int8_plan &a, const samd_conv2d_int8_plan &b) {
    return a.halo == b.halo && a.mtile == b.mtile && a.positions == b.positions && a.waves == b.waves;
}

}  // namespace

int conv2d_i8_candidates(const samd_conv2d_desc &d, samd_fmt xf, std::vector<samd_conv2d_int8_plan> &out) {
    int8_candidates(make_geom(d, xf), out);
    return SAMD_OK;
}

int conv2d_i8_tiles(const samd_conv2d_desc &d, samd_fmt xf, samd_conv2d_int8_plan &out) {
    std::vector<samd_conv2d_int8_plan> cands;
    int8_candidates(make_geom(d, xf), cands);
    {
        std::lock_guard<std::mutex> lock(int8_mu);
        auto it = int8_plans.find(int8_key(d, xf));
        if (it != int8_plans.end()) {
            out = it->second;
            return SAMD_OK;
        }
    }
    out = model_choice(cands);
    return SAMD_OK;
}

int conv2d_i8_use_plan(const samd_conv2d_desc &d, samd_fmt xf, const samd_conv2d_int8_plan *plan) {
    std::lock_guard<std::mutex> lock(int8_mu);
    if (!plan) {
        int8_plans.erase(int8_key(d, xf));
        return SAMD_OK;
    }
    std::vector<samd_conv2d_int8_plan> cands;
    int8_candidates(make_geom(d, xf), cands);
    for (const auto &c : cands)
        if (same_launch(c, *plan)) {
            int8_plans[int8_key(d, xf)] = c;
            return SAMD_OK;
        }
    set_error("conv2d_int8: no candidate launch of this layer matches the plan");
    return SAMD_EINVAL;
}

int launch_conv2d_i8(const void *x, samd_fmt xf, const samd_conv2d_desc &d, int32_t *y, const void *ws,
                     hipStream_t s) {
    const I8Geom g = make_geom(d, xf);
    const I8Workspace p = carve(g, const_cast<void *>(ws));
    const bool vec = (g.C % 16) == 0 && ((uintptr_t)x % 16) == 0;
    samd_conv2d_int8_plan plan{};
    conv2d_i8_tiles(d, xf, plan);
    if (plan.halo == 3 && ((uintptr_t)x % 4) == 0) {
        PkTiles pt{};
        int lds = 0;
        int64_t wgs = 0;
        if (pk_tiles(g, plan.positions / (4 * kResTile), pt, lds, wgs)) return launch_packed(x, g, pt, lds, p, y, s);
    }
    if (plan.halo == 2 && vec) {
        // the plan's runs again: the plan records the workgroup count its target gave
        for (int target : kResTargets) {
            ResTiles rt{};
            int64_t wgs = 0;
            int lds = 0, positions = 0;
            if (res_tiles(g, target, rt, lds, wgs, positions) && positions == plan.positions)
                return launch_res_any(x, g, rt, lds, p, y, s);
        }
    }
    if (plan.halo == 1 && vec) {
        const int wm = plan.mtile / 4, tp = plan.positions;
        HaloTiles ht{};
        int64_t wgs = 0;
        int lds = 0;
        if (halo_tiles(g, wm, tp, ht, wgs, lds)) {
#define SAMD_HALO(WM_, TP_)                                                                                  \
    if (wm == WM_ && tp == TP_)                                                                              \
        return ht.kc == 128 ? launch_halo<WM_, TP_, 128>(x, g, ht, lds, p, y, s)                             \
                            : launch_halo<WM_, TP_, 64>(x, g, ht, lds, p, y, s);
            SAMD_HALO(32, 128) SAMD_HALO(32, 64) SAMD_HALO(16, 128) SAMD_HALO(16, 64)
#undef SAMD_HALO
        }
    }
    // the im2col kernel: the chosen plan's positions per workgroup, or (misaligned
    // activations under a halo plan) 64 when that gives every compute unit a workgroup
    int tp = plan.halo ? ((g.P + 63) / 64 * (g.Mp / kTM) >= 256 ? 64 : 32) : plan.positions;
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
    if (tp == 64) {
        SAMD_I8_KS(64)
    } else {
        SAMD_I8_KS(32)
    }
#undef SAMD_I8_KS
#undef SAMD_I8_LAUNCH
    return check_launch("conv2d_int8");
}

}  // namespace samd
