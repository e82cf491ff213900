// SAMD 2-D convolution for gfx950: convolution by long multiplication (Sec. 5) with
// signed sign-extension and the underflow fix-up (Sec. 6).
//
// Three kernels:
//  * prep_weights_kernel: every kernel row -> its kernel words (taps reversed, sign-
//    extended, L bits apart), laid out as one contiguous stream per group of kWaveM
//    output channels, so a wave walks its kernel words with scalar loads;
//  * spread_kernel: every packed input row -> operand words, I values of one stride
//    phase L bits apart (temporary spacer bits), negative values sign-extended, so that
//    each word is the int32 sum_i v_i 2^(i L); rows of the zero padding are written too;
//  * conv2d_samd_kernel: a workgroup owns a tile of output rows of one image and wm*8
//    output channels.  Per chunk of input channels it copies the tile's operand words
//    into LDS (double-buffered, one barrier per chunk); every wave multiplies them by its
//    8 SGPR-resident kernel words and adds the exact signed 32x32 -> 64-bit products
//    into 64-bit accumulators (v_mad_i64_i32).  Every G channels the accumulators are
//    decoded - fix-up, lane extraction - and added into an LDS tile of int32 outputs,
//    which also performs the overlap-add of neighbouring words' partial lanes.
#include <hip/hip_runtime.h>

#include <climits>

#include "hip_util.hpp"

namespace samd {

namespace {

constexpr int RM = kWaveM;
constexpr int kPrefetch = kStagePerThread;   // operand words each thread carries into the next chunk

template <int B, bool S>
__device__ inline int32_t packed_field(const uint32_t *row, int col) {
    constexpr int P = 32 / B;
    const uint32_t f = (row[col / P] >> ((col % P) * B)) & ((1u << B) - 1);
    if (S) return (int32_t)(f << (32 - B)) >> (32 - B);
    return (int32_t)f;
}

// Kernel-word stream of output-channel group wb: step s = c*nrt + ky*ntw + t holds the
// kWaveM words of kernel word t of row ky of channel c; kStreamPad zero steps pad the end.
template <int B, bool S>
__global__ __launch_bounds__(256) void prep_weights_kernel(const uint32_t *__restrict__ w, const Conv2dGeom g,
                                                           int32_t *__restrict__ kw) {
    const int64_t steps = (int64_t)g.C * g.nrt + kStreamPad;
    for (int64_t idx = (int64_t)blockIdx.x * 256 + threadIdx.x; idx < g.kw_words; idx += (int64_t)gridDim.x * 256) {
        const int mm = (int)(idx % RM);
        const int64_t s = (idx / RM) % steps;
        const int64_t wb = idx / (RM * steps);
        const int m = (int)(wb * RM + mm);
        uint32_t word = 0;
        if (m < g.M && s < (int64_t)g.C * g.nrt) {
            const int c = (int)(s / g.nrt), rt = (int)(s % g.nrt);
            const int ky = rt / g.ntw, t = rt % g.ntw;
            const uint32_t *row = w + ((int64_t)(m * g.C + c) * g.KH + ky) * g.wrw;
            const int k = g.tw_ntaps[t], a0 = g.tw_tap0[t], r = g.tw_phase[t];
            for (int si = 0; si < k; ++si) {
                const int tap = g.sw * (a0 + k - 1 - si) + r;   // reversed: lane si holds tap a0+k-1-si
                word += (uint32_t)packed_field<B, S>(row, tap) << (si * g.L);
            }
        }
        kw[idx] = (int32_t)word;
    }
}

// Operand words xs[n][c][hp][t][q] for padded rows hp in [0, H + 2 ph).
template <int B, bool S>
__global__ __launch_bounds__(256) void spread_kernel(const uint32_t *__restrict__ x, const Conv2dGeom g,
                                                     int32_t *__restrict__ xs) {
    for (int64_t idx = (int64_t)blockIdx.x * 256 + threadIdx.x; idx < g.spread_words;
         idx += (int64_t)gridDim.x * 256) {
        const int q = (int)(idx % g.nq);
        int64_t t1 = idx / g.nq;
        const int t = (int)(t1 % g.ntw);
        t1 /= g.ntw;
        const int hp = (int)(t1 % g.Hp);
        const int64_t nc = t1 / g.Hp;
        const int h = hp - g.ph;
        uint32_t word = 0;
        if (h >= 0 && h < g.H) {
            const uint32_t *row = x + (nc * g.H + h) * g.xrw;
            const int delta = g.tw_tap0[t] + g.tw_ntaps[t] - g.Kmax;
            const int col0 = g.sw * (q * g.I + delta) + g.tw_phase[t] - g.pw;
            for (int ii = 0; ii < g.I; ++ii) {
                const int col = col0 + g.sw * ii;
                if (col >= 0 && col < g.W) word += (uint32_t)packed_field<B, S>(row, col) << (ii * g.L);
            }
        }
        xs[idx] = (int32_t)word;
    }
}

// Empty register barrier: the accumulator is treated as rewritten here, so the products
// of successive steps cannot be summed first and added afterwards (integer addition is
// associative, and that rewrite costs one extra 64-bit add per batch); every product
// stays one v_mad_i64_i32 into its accumulator.
__device__ __forceinline__ void keep(int64_t &acc) { asm volatile("" : "+v"(acc)); }

// Sign- or zero-extended field of the low L bits (v_bfe with a uniform width).
template <bool SG>
__device__ __forceinline__ int32_t low_field(uint32_t w, int L) {
    int32_t d;
    if (SG)
        asm("v_bfe_i32 %0, %1, 0, %2" : "=v"(d) : "v"(w), "s"(L));
    else
        asm("v_bfe_u32 %0, %1, 0, %2" : "=v"(d) : "v"(w), "s"(L));
    return d;
}

// Decode of one accumulator (Sec. 6): the fix-up of the signed-convolution figure for
// signed results, then lanes from the bottom - take the low L bits, shift them out -
// each added into its output column (p + j); lane NL-1 takes all remaining bits.
template <bool SG, int NL>
__device__ __forceinline__ void decode_word(uint64_t v, uint64_t msb_mask, int L, int32_t *p) {
    if (SG) {
        const uint64_t s = v & msb_mask;
        v = (v + s) ^ s;
    }
#pragma unroll
    for (int j = 0; j < NL - 1; ++j) {
        atomicAdd(p + j, low_field<SG>((uint32_t)v, L));
        v = SG ? (uint64_t)((int64_t)v >> L) : v >> L;
    }
    atomicAdd(p + NL - 1, (int32_t)v);
}

// The same for a lane count known only at run time.
template <bool SG>
__device__ __forceinline__ void decode_word_n(uint64_t v, uint64_t msb_mask, int L, int nl, int32_t *p) {
    if (SG) {
        const uint64_t s = v & msb_mask;
        v = (v + s) ^ s;
    }
#pragma unroll 1
    for (int j = 0; j < nl - 1; ++j) {
        atomicAdd(p + j, low_field<SG>((uint32_t)v, L));
        v = SG ? (uint64_t)((int64_t)v >> L) : v >> L;
    }
    atomicAdd(p + nl - 1, (int32_t)v);
}

// A workgroup has wm x ks waves.  Wave (kq, mw) owns output channels mw*8 .. +7 of the
// block and multiplies slice kq (cpw channels) of every chunk; the ks waves of one
// output-channel group add their decoded partial sums into the same LDS tile, whose
// atomic adds are also the overlap-add of neighbouring words' partial lanes.
//
// NRT: steps (kernel row x kernel word) per input channel when it is 3 or 6 (every 3x3
// layer), so batches never straddle channels and all LDS offsets are immediates; 0 for
// any other count.  SG: the result is signed (either operand signed), so lanes need
// the fix-up and are sign-extended.
template <int RH, int NRT, bool SG>
__global__ __launch_bounds__(1024) void conv2d_samd_kernel(const int32_t *__restrict__ xs,
                                                           const int32_t *__restrict__ kw, int32_t *__restrict__ y,
                                                           const Conv2dGeom g) {
    extern __shared__ int32_t lds[];
    int32_t *tile = lds;
    int32_t *abuf0 = lds + g.lds_tile;
    int32_t *abuf1 = abuf0 + g.lds_abuf;

    // Consecutive workgroups on one XCD (hardware assigns workgroup p to XCD p % 8) take
    // all channel blocks of one spatial tile, so its operand words are reused from L2.
    const int p = blockIdx.x;
    const int slot = p >> 3;
    const int mb = slot % g.nmb;
    const int tile_id = (slot / g.nmb) * 8 + (p & 7);
    if (tile_id >= g.N * g.row_tiles) return;   // padding workgroup: exits as a whole
    const int n = tile_id / g.row_tiles;
    const int ho0 = (tile_id % g.row_tiles) * g.rows_blk;

    const int tid = threadIdx.x;
    const int nthr = g.wm * g.ks * 64;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int kq = wave / g.wm;
    const int mw = wave - kq * g.wm;
    const int lane = tid & 63;
    const int grp_raw = lane / g.nq;
    const bool lane_ok = grp_raw < g.groups;
    const int grp = lane_ok ? grp_raw : 0;
    const int q = lane_ok ? lane - grp_raw * g.nq : 0;
    const int wb = mb * g.wm + mw;

    for (int i = tid; i < g.lds_tile; i += nthr) tile[i] = 0;

    // LDS chunk layout [cc][q][tr * ntw + t] with an odd stride per q (conflict-free):
    // a thread's steps (ky, t) of one channel and row are consecutive words.
    const int T = g.trows * g.ntw;                 // words per (channel, q)
    const int qs = g.lds_qstride;                  // T rounded up to odd
    const int cs = g.nq * qs;                      // words per channel
    const int gblk = T * g.nq;                     // global words per channel of the tile
    const int64_t ch_stride = (int64_t)g.Hp * g.ntw * g.nq;
    const int in_words = min(g.trows, g.Hp - ho0 * g.sh) * g.ntw * g.nq;   // rows that exist
    const int32_t *xs_tile = xs + ((int64_t)n * g.C * g.Hp + ho0 * g.sh) * g.ntw * g.nq;
    // Thread element j of a chunk: global word i of channel cc (global order [tr][t][q]);
    // the same (cc, i) in every chunk, so offsets are computed once.
    // e_off < 0: the row lies past the padded image and stages as 0; e_lds = INT_MAX: no
    // element (past the chunk).  Channel cc < n of a chunk  <=>  e_lds < n * cs.
    int e_lds[kPrefetch], e_off[kPrefetch];
    const int chunk_words = g.chk * gblk;
#pragma unroll
    for (int j = 0; j < kPrefetch; ++j) {
        const int e = tid + j * nthr;
        const int cc = e / gblk, i = e - cc * gblk;
        const int qq = i % g.nq, rt = i / g.nq;
        e_lds[j] = e < chunk_words ? cc * cs + qq * qs + rt : INT_MAX;
        e_off[j] = i < in_words ? (int)(cc * ch_stride) + i : -1;
    }
    // words past the kPrefetch carried per thread (large staged tiles only): loaded and
    // stored directly
    auto stage_rest = [&](int32_t *dst, const int32_t *src, int ncc) {
        for (int e = tid + kPrefetch * nthr; e < ncc * gblk; e += nthr) {
            const int cc = e / gblk, i = e - cc * gblk;
            const int qq = i % g.nq, rt = i / g.nq;
            dst[cc * cs + qq * qs + rt] = i < in_words ? src[cc * ch_stride + i] : 0;
        }
    };
    const int nchunks = (g.C + g.chk - 1) / g.chk;
    {
        const int ncc = min(g.chk, g.C);
        const int lim = ncc * cs;
#pragma unroll
        for (int j = 0; j < kPrefetch; ++j)
            if (e_lds[j] < lim) abuf0[e_lds[j]] = e_off[j] >= 0 ? xs_tile[e_off[j]] : 0;
        stage_rest(abuf0, xs_tile, ncc);
    }
    __syncthreads();

    int64_t acc[RH][RM];
#pragma unroll
    for (int r = 0; r < RH; ++r)
#pragma unroll
        for (int m = 0; m < RM; ++m) acc[r][m] = 0;

    const int64_t stream_len = ((int64_t)g.C * g.nrt + kStreamPad) * RM;
    const int32_t *kstream = kw + wb * stream_len;
    // LDS word offset of each of the thread's rows within a channel (rows past the tile
    // reuse the last one; their results are never stored)
    int rowoff[RH];
#pragma unroll
    for (int r = 0; r < RH; ++r) rowoff[r] = q * qs + min(grp * RH + r, g.rows_blk - 1) * g.sh * g.ntw;
    const int cw0 = kq * g.cpw;   // first channel of this wave's slice of a chunk

    // Decode: fix-up (signed results), then lane j of word q goes to output column
    // q*I + j - (Kmax-1), stored at tile column q*I + j; the top lane takes the bits left.
    // Tile rows cover every row a wave computes, so no lane needs a bounds check.
    int32_t *const tbase = tile + ((mw * RM) * g.tile_rows + grp * RH) * g.tile_row + q * g.I;
    const int mstride = g.tile_rows * g.tile_row;
    auto decode = [&]() {
        if (lane_ok) {
            const uint64_t msb = g.msb_mask;
            const int L = g.L;
#define SAMD_DECODE_NL(NL_)                                                                           \
    case NL_:                                                                                         \
        _Pragma("unroll") for (int r = 0; r < RH; ++r)                                               \
            _Pragma("unroll") for (int m = 0; m < RM; ++m)                                           \
                decode_word<SG, NL_>((uint64_t)acc[r][m], msb, L, tbase + r * g.tile_row + m * mstride); \
        break;
            switch (g.nl) {
                SAMD_DECODE_NL(2) SAMD_DECODE_NL(3) SAMD_DECODE_NL(4) SAMD_DECODE_NL(5)
                SAMD_DECODE_NL(6) SAMD_DECODE_NL(7) SAMD_DECODE_NL(8)
            default:
#pragma unroll
                for (int r = 0; r < RH; ++r)
#pragma unroll
                    for (int m = 0; m < RM; ++m)
                        decode_word_n<SG>((uint64_t)acc[r][m], msb, L, g.nl, tbase + r * g.tile_row + m * mstride);
            }
#undef SAMD_DECODE_NL
        }
#pragma unroll
        for (int r = 0; r < RH; ++r)
#pragma unroll
            for (int m = 0; m < RM; ++m) acc[r][m] = 0;
    };

    for (int k = 0; k < nchunks; ++k) {
        const int32_t *cur = (k & 1) ? abuf1 : abuf0;
        int32_t *nxt = (k & 1) ? abuf0 : abuf1;
        const int c0 = k * g.chk;
        const int ncc = min(g.chk, g.C - c0);
        const int c1 = c0 + g.chk;
        const int ncc1 = k + 1 < nchunks ? min(g.chk, g.C - c1) : 0;

        // operand words of the next chunk: global loads now, LDS stores after the compute
        int32_t pre[kPrefetch];
        const int32_t *src1 = xs_tile + c1 * ch_stride;
        const int lim1 = ncc1 * cs;
#pragma unroll
        for (int j = 0; j < kPrefetch; ++j) pre[j] = (e_lds[j] < lim1 && e_off[j] >= 0) ? src1[e_off[j]] : 0;

        // This wave's slice: channels cw0 .. cw0 + nch - 1 of the chunk, in batches of
        // kStepBatch steps: kernel words in SGPRs, operand words from LDS.  With 3 or 6
        // steps per channel a slice is a whole number of batches.
        const int nch = min(max(ncc - cw0, 0), g.cpw);
        const int nsteps = nch * g.nrt;
        const int nbat = (nsteps + kStepBatch - 1) / kStepBatch;
        const int32_t *ks = kstream + (int64_t)(c0 + cw0) * g.nrt * RM;
        const int32_t *wcur = cur + cw0 * cs;
        int32_t kA[kStepBatch * RM], aA[kStepBatch][RH], kB[kStepBatch * RM], aB[kStepBatch][RH];
        int gs = 0;   // generic layout: step index of the next batch to load
        auto load_batch = [&](int b, int32_t (&kb)[kStepBatch * RM], int32_t (&ab)[kStepBatch][RH]) {
#pragma unroll
            for (int j = 0; j < kStepBatch * RM; ++j) kb[j] = ks[b * kStepBatch * RM + j];
            if constexpr (NRT != 0) {
                // batch b: channel b / (NRT/3), steps (b % (NRT/3))*3 .. +2 of it
                constexpr int BPC = NRT / kStepBatch;
                const int base = (b / BPC) * cs + (b % BPC) * kStepBatch;
#pragma unroll
                for (int r = 0; r < RH; ++r) {
                    const int32_t *src = wcur + base + rowoff[r];
#pragma unroll
                    for (int j = 0; j < kStepBatch; ++j) ab[j][r] = src[j];
                }
            } else {
#pragma unroll
                for (int j = 0; j < kStepBatch; ++j) {
                    // steps past the slice (its step count need not be a multiple of the
                    // batch) multiply the following channel's kernel words: their operand is 0
                    const bool live = gs + j < nsteps;
                    const int st = min(gs + j, nsteps - 1);
                    const int cc = st / g.nrt, rt = st - cc * g.nrt;
#pragma unroll
                    for (int r = 0; r < RH; ++r) {
                        const int32_t v = wcur[cc * cs + rt + rowoff[r]];
                        ab[j][r] = live ? v : 0;
                    }
                }
                gs += kStepBatch;
            }
        };
        auto mac_batch = [&](const int32_t (&kb)[kStepBatch * RM], const int32_t (&ab)[kStepBatch][RH]) {
#pragma unroll
            for (int j = 0; j < kStepBatch; ++j) {
#pragma unroll
                for (int r = 0; r < RH; ++r)
#pragma unroll
                    for (int m = 0; m < RM; ++m) acc[r][m] += (int64_t)ab[j][r] * (int64_t)kb[j * RM + m];
#pragma unroll
                for (int r = 0; r < RH; ++r)
#pragma unroll
                    for (int m = 0; m < RM; ++m) keep(acc[r][m]);
            }
        };
        // Ping-pong over two register sets.  Before a batch's kernel words are used, all
        // outstanding scalar and LDS loads are waited for, and only then is the next batch
        // requested: scalar loads return out of order, so a wait placed after requesting
        // the next batch would wait for it too.
        // The batch after the slice's last one is fetched too (its results are never
        // used): it reads the next slice's channel, or for the last slice the spare
        // channel block after the LDS buffers and the kStreamPad padding steps of the
        // kernel-word stream.
        if (nbat > 0) {
            load_batch(0, kA, aA);
            int b = 0;
            for (; b + 1 < nbat; b += 2) {
                __builtin_amdgcn_s_waitcnt(0xc07f);   // lgkmcnt(0)
                load_batch(b + 1, kB, aB);
                __builtin_amdgcn_sched_barrier(0);
                mac_batch(kA, aA);
                __builtin_amdgcn_sched_barrier(0);
                __builtin_amdgcn_s_waitcnt(0xc07f);
                load_batch(b + 2, kA, aA);
                __builtin_amdgcn_sched_barrier(0);
                mac_batch(kB, aB);
                __builtin_amdgcn_sched_barrier(0);
            }
            if (b < nbat) {   // odd batch count: the last batch
                __builtin_amdgcn_s_waitcnt(0xc07f);
                mac_batch(kA, aA);
            }
        }

        // the next chunk's operand words into the other buffer (last read a chunk ago,
        // before the previous barrier)
#pragma unroll
        for (int j = 0; j < kPrefetch; ++j)
            if (e_lds[j] < lim1) nxt[e_lds[j]] = pre[j];
        stage_rest(nxt, src1, ncc1);

        if ((k + 1) % g.flush_chunks == 0 || k + 1 == nchunks) decode();
        __syncthreads();
    }

    // output tile -> y, one row per wave at a time
    const int nwaves = g.wm * g.ks;
    for (int rr = wave; rr < g.mblk * g.rows_blk; rr += nwaves) {
        const int mm = rr / g.rows_blk, r = rr - mm * g.rows_blk;
        const int m = mb * g.mblk + mm, ho = ho0 + r;
        if (m >= g.M || ho >= g.Ho) continue;
        const int32_t *src = tile + (mm * g.tile_rows + r) * g.tile_row + (g.Kmax - 1);
        int32_t *dst = y + (((int64_t)n * g.M + m) * g.Ho + ho) * g.Wo;
        for (int o = lane; o < g.Wo; o += 64) dst[o] = src[o];
    }
}

}  // namespace

int launch_conv2d_prepare(const uint32_t *w, const Conv2dGeom &g, void *ws, hipStream_t s) {
    int32_t *kw = (int32_t *)ws;
    const int pgrid = grid_for(g.kw_words, 256);
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

int launch_conv2d_spread(const uint32_t *x, const Conv2dGeom &g, void *ws, hipStream_t s) {
    int32_t *xs = (int32_t *)((char *)ws + conv2d_kw_bytes(g));
    const int sgrid = grid_for(g.spread_words, 256);
    bool launched = false;
#define SAMD_SPREAD_CASE(B, SG)                                                                            \
    if (!launched && g.xbits == B && (bool)g.xsigned == SG) {                                              \
        hipLaunchKernelGGL((spread_kernel<B, SG>), dim3(sgrid), dim3(256), 0, s, x, g, xs);                \
        launched = true;                                                                                   \
    }
    SAMD_FOR_EACH_FMT(SAMD_SPREAD_CASE)
#undef SAMD_SPREAD_CASE
    return check_launch("conv2d operand spread");
}

int launch_conv2d_multiply(const Conv2dGeom &g, int32_t *y, const void *ws, hipStream_t s) {
    const int32_t *kw = (const int32_t *)ws;
    const int32_t *xs = (const int32_t *)((const char *)ws + conv2d_kw_bytes(g));
    const dim3 grid((unsigned)g.tiles * g.nmb), block(g.wm * g.ks * 64);
    const size_t shm = (size_t)g.lds_words * 4;
#define SAMD_CONV_CASE(RH_, NRT_, SG_)                                                                \
    if (g.rh == RH_ && (NRT_ == 0 ? (g.nrt != 3 && g.nrt != 6) : g.nrt == NRT_) &&                     \
        (bool)g.result_signed == SG_) {                                                               \
        hipLaunchKernelGGL((conv2d_samd_kernel<RH_, NRT_, SG_>), grid, block, shm, s, xs, kw, y, g);   \
        return check_launch("conv2d");                                                                \
    }
    SAMD_CONV_CASE(1, 3, false) SAMD_CONV_CASE(1, 6, false) SAMD_CONV_CASE(1, 0, false)
    SAMD_CONV_CASE(2, 3, false) SAMD_CONV_CASE(2, 6, false) SAMD_CONV_CASE(2, 0, false)
    SAMD_CONV_CASE(1, 3, true) SAMD_CONV_CASE(1, 6, true) SAMD_CONV_CASE(1, 0, true)
    SAMD_CONV_CASE(2, 3, true) SAMD_CONV_CASE(2, 6, true) SAMD_CONV_CASE(2, 0, true)
#undef SAMD_CONV_CASE
    set_error("conv2d: no kernel for this geometry");
    return SAMD_EUNSUPPORTED;
}

int launch_conv2d_samd(const uint32_t *x, const Conv2dGeom &g, int32_t *y, const void *ws, hipStream_t s) {
    const int st = launch_conv2d_spread(x, g, const_cast<void *>(ws), s);
    if (st) return st;
    return launch_conv2d_multiply(g, y, ws, s);
}

}  // namespace samd
