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
//    output channels.  Every lane reads its operand words straight from the spread buffer
//    with raw buffer loads (L1/L2-resident: each word is reused by the workgroup's channel
//    waves and kernel rows), every wave holds its 8 kernel words of a step in SGPRs
//    (scalar loads from its kernel-word stream) and adds the exact signed 32x32 -> 64-bit
//    products into 64-bit accumulators (v_mad_i64_i32).  Every G channels the
//    accumulators are decoded - fix-up, lane extraction - and added into an LDS tile of
//    int32 outputs (the tile is the only LDS use), which also performs the overlap-add of
//    neighbouring words' partial lanes and sums the channel-split waves; finished rows
//    are stored from the tile.
#include <hip/hip_runtime.h>

#include <climits>
#include <map>
#include <mutex>
#include <tuple>

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

// Kernel-word stream of output-channel group wb: step s = c*nrt + ky*ntw + t (or
// c*nrt + t*KH + ky on the shared-row path) holds the kWaveM words of kernel word t of
// row ky of channel c; kStreamPad zero steps pad the end.
// Also zeroes the multiply kernel's ticket counters.
template <int B, bool S>
__global__ __launch_bounds__(256) void prep_weights_kernel(const uint32_t *__restrict__ w, const Conv2dGeom g,
                                                           int32_t *__restrict__ kw, int32_t *__restrict__ queue) {
    if (blockIdx.x == 0)
        for (int i = threadIdx.x; i < kQueueBytes / 4; i += 256) queue[i] = 0;
    const int64_t steps = (int64_t)g.C * g.nrt + kStreamPad;
    for (int64_t idx = (int64_t)blockIdx.x * 256 + threadIdx.x; idx < g.kw_words; idx += (int64_t)gridDim.x * 256) {
        const int mm = (int)(idx % RM);
        const int64_t s = (idx / RM) % steps;
        const int64_t wb = idx / (RM * steps);
        const int m = (int)(wb * RM + mm);
        uint32_t word = 0;
        if (m < g.M && s < (int64_t)g.C * g.nrt) {
            const int c = (int)(s / g.nrt), rt = (int)(s % g.nrt);
            // steps of a channel: kernel-row-major, or kernel-word-major for the
            // shared-row path
            const int ky = g.rows_path ? rt % g.KH : rt / g.ntw, t = g.rows_path ? rt / g.KH : rt % g.ntw;
            const uint32_t *row = w + (((int64_t)m * g.C + c) * g.KH + ky) * g.wrw;
            const int k = g.tw_ntaps[t], a0 = g.tw_tap0[t], r = g.tw_phase[t];
            for (int si = 0; si < k; ++si) {
                const int tap = g.sw * (a0 + k - 1 - si) + r;   // reversed: lane si holds tap a0+k-1-si
                word += (uint32_t)packed_field<B, S>(row, tap) << (si * g.L);
            }
        }
        kw[idx] = (int32_t)word;
    }
}

// Correction table of recentred activations: pre[m][i][j] = sum of w[m][c][ky][kx] over
// all c, ky < i, kx < j (i <= KH, j <= KW), so an output's in-image taps [ky0, ky1) x
// [kx0, kx1) sum to a rectangle of four entries.
template <int B, bool S>
__global__ __launch_bounds__(256) void prefix_kernel(const uint32_t *__restrict__ w, const Conv2dGeom g,
                                                     int32_t *__restrict__ pre) {
    const int pwid = (g.KH + 1) * (g.KW + 1);
    const int64_t total = (int64_t)g.M * pwid;
    for (int64_t e = (int64_t)blockIdx.x * 256 + threadIdx.x; e < total; e += (int64_t)gridDim.x * 256) {
        const int m = (int)(e / pwid), ij = (int)(e - (int64_t)m * pwid);
        const int i = ij / (g.KW + 1), j = ij - i * (g.KW + 1);
        int32_t sum = 0;
        for (int c = 0; c < g.C; ++c)
            for (int ky = 0; ky < i; ++ky) {
                const uint32_t *row = w + (((int64_t)m * g.C + c) * g.KH + ky) * g.wrw;
                for (int kx = 0; kx < j; ++kx) sum += packed_field<B, S>(row, kx);
            }
        pre[e] = sum;
    }
}

// Operand words xs[n][c][hp][t][q] for padded rows hp in [0, H + 2 ph), of the
// activations minus xoff (recentred unsigned activations).  A block of 256
// threads covers 256 / QP padded rows (QP, a power of two of at most 256, about nq / 2.5
// threads per row): thread (row, q) builds words q, q + QP, ... of every kernel-word
// variant t of its row from the packed input row (L1-resident; rows of the zero padding
// give zeros).
template <int B, bool S>
__global__ __launch_bounds__(256) void spread_kernel(const uint32_t *__restrict__ x, const Conv2dGeom g, int qshift,
                                                     int32_t *__restrict__ xs) {
    constexpr int P = 32 / B;
    // 32-bit row indices: the planner keeps N * C * Hp below 2^31
    const uint32_t row = blockIdx.x * (256u >> qshift) + (threadIdx.x >> qshift);   // (n*C + c)*Hp + hp
    if (row >= (uint32_t)(g.N * g.C * g.Hp)) return;
    const uint32_t nc = row / (uint32_t)g.Hp;
    const int hp = (int)(row - nc * (uint32_t)g.Hp);
    const int h = hp - g.ph;
    const bool inside = h >= 0 && h < g.H;
    const uint32_t *src = x + ((int64_t)nc * g.H + (inside ? h : 0)) * g.xrw;
    // words q, q + 2^qshift, ... of the row (one pass unless the row has more than 256)
    for (int q = threadIdx.x & ((1 << qshift) - 1); q < g.nq; q += 1 << qshift) {
        int32_t *dst = xs + (int64_t)row * g.ntw * g.nq + q;
        for (int t = 0; t < g.ntw; ++t) {
            const int delta = g.tw_tap0[t] + g.tw_ntaps[t] - g.Kmax;
            const int col0 = g.sw * (q * g.I + delta) + g.tw_phase[t] - g.pw;
            uint32_t word = 0;
            if (inside) {
                for (int ii = 0; ii < g.I; ++ii) {
                    const int col = col0 + g.sw * ii;
                    if (col >= 0 && col < g.W) {
                        const uint32_t f = (src[col / P] >> ((col % P) * B)) & ((1u << B) - 1);
                        const int32_t v = (S ? ((int32_t)(f << (32 - B)) >> (32 - B)) : (int32_t)f) - g.xoff;
                        word += (uint32_t)v << (ii * g.L);
                    }
                }
            }
            dst[t * g.nq] = (int32_t)word;
        }
    }
}

// The same operand words built from unpacked 8-bit values (int8 when S, else uint8; N C H W
// row-major) instead of packed rows: the permanent-spacer layout written straight from
// the values a caller holds.  Each value enters as its low b bits (sign-extended when S).
template <int B, bool S>
__global__ __launch_bounds__(256) void spread_bytes_kernel(const uint8_t *__restrict__ x, const Conv2dGeom g,
                                                           int qshift, int32_t *__restrict__ xs) {
    const uint32_t row = blockIdx.x * (256u >> qshift) + (threadIdx.x >> qshift);   // (n*C + c)*Hp + hp
    if (row >= (uint32_t)(g.N * g.C * g.Hp)) return;
    const uint32_t nc = row / (uint32_t)g.Hp;
    const int hp = (int)(row - nc * (uint32_t)g.Hp);
    const int h = hp - g.ph;
    const bool inside = h >= 0 && h < g.H;
    const uint8_t *src = x + ((int64_t)nc * g.H + (inside ? h : 0)) * g.W;
    for (int q = threadIdx.x & ((1 << qshift) - 1); q < g.nq; q += 1 << qshift) {
        int32_t *dst = xs + (int64_t)row * g.ntw * g.nq + q;
        for (int t = 0; t < g.ntw; ++t) {
            const int delta = g.tw_tap0[t] + g.tw_ntaps[t] - g.Kmax;
            const int col0 = g.sw * (q * g.I + delta) + g.tw_phase[t] - g.pw;
            uint32_t word = 0;
            if (inside) {
                for (int ii = 0; ii < g.I; ++ii) {
                    const int col = col0 + g.sw * ii;
                    if (col >= 0 && col < g.W) {
                        const uint32_t f = src[col] & ((1u << B) - 1);
                        const int32_t v = (S ? ((int32_t)(f << (32 - B)) >> (32 - B)) : (int32_t)f) - g.xoff;
                        word += (uint32_t)v << (ii * g.L);
                    }
                }
            }
            dst[t * g.nq] = (int32_t)word;
        }
    }
}

// Operand words are read through a buffer resource over one image's operand words: the
// per-lane byte offset is a VGPR, the per-step offset an SGPR (no address arithmetic in
// the vector unit).  Word 3 is the gfx9 raw-buffer format (32-bit data, no swizzle).
constexpr int kBufferWord3 = 0x00020000;

__device__ __forceinline__ int32_t buffer_word(__amdgpu_buffer_rsrc_t r, int lane_bytes, int step_bytes) {
    return __builtin_amdgcn_raw_buffer_load_b32(r, lane_bytes, step_bytes, 0);
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
// signed results, after which lane j is the (sign-extended) field at bit j L, each
// added into its output column (p + j); lane NL-1 takes all remaining bits.  Every lane
// is cut from the fixed-up word directly (no chain of shifts), so the lanes' extractions
// are independent instructions.
// PS (permanent spacer bits, Sec. 6.1): every lane's MSB is a spacer bit (the planner
// keeps its values within L - 1 bits), so the fix-up's final xor, which only restores the
// MSB, is left out and each lane is read from its low L - 1 bits.
template <bool SG, int NL, bool PS>
__device__ __forceinline__ void decode_word(uint64_t v, uint64_t msb_mask, int L, int fw, int32_t *p) {
    if (SG) {
        const uint64_t s = v & msb_mask;
        v += s;
        if (!PS) v ^= s;
    }
#pragma unroll
    for (int j = 0; j < NL - 1; ++j) atomicAdd(p + j, low_field<SG>((uint32_t)(v >> (j * L)), PS ? fw : L));
    const int top = (NL - 1) * L;
    atomicAdd(p + NL - 1, (int32_t)(SG ? (uint64_t)((int64_t)v >> top) : v >> top));
}

// The same for a lane count known only at run time.
template <bool SG, bool PS>
__device__ __forceinline__ void decode_word_n(uint64_t v, uint64_t msb_mask, int L, int fw, int nl, int32_t *p) {
    if (SG) {
        const uint64_t s = v & msb_mask;
        v += s;
        if (!PS) v ^= s;
    }
#pragma unroll 1
    for (int j = 0; j < nl - 1; ++j) atomicAdd(p + j, low_field<SG>((uint32_t)(v >> (j * L)), PS ? fw : L));
    const int top = (nl - 1) * L;
    atomicAdd(p + nl - 1, (int32_t)(SG ? (uint64_t)((int64_t)v >> top) : v >> top));
}

// Work item: rows_blk output rows x all Wo columns x mblk output channels of one image,
// computed by one workgroup of wm x ks waves.  Wave (kq, mw) computes output channels
// mw*8 .. +7 of the block over its slice kq of the input channels; lane (grp, q) holds
// output word q of rows grp*RH .. +RH-1.  Operand words come straight from the spread
// buffer (global memory, L1/L2-resident: every word is reused by the block's wm waves and
// its KH kernel rows), kernel words from the wave's stream through scalar loads.  After at
// most G channels the accumulators are decoded into an LDS tile of int32 outputs whose
// atomic adds also sum the ks channel slices and overlap-add neighbouring words' partial
// lanes.
//
// The grid holds at most as many workgroups as the chip keeps resident.  XCD x (hardware
// assigns workgroup p to XCD p % 8) owns one contiguous eighth of the spatial tiles, each
// with all its channel blocks in consecutive items, so a tile's operand words - and the
// halo rows it shares with the next row tile - are fetched into that XCD's L2 once and
// reused there.  Workgroup p first computes item p / 8 of its XCD; the items
// beyond the XCD's workgroups go to whichever workgroup frees up first, through a ticket
// counter per XCD: waves of equal work finish far apart (the SIMD issues the oldest wave
// first), and a fixed assignment would leave the chip draining for much of the launch.
// A launch takes exactly T = extra items + workgroups tickets from each counter (every
// workgroup ends on one ticket past the items), so ticket t stands for local index
// t mod T: the counters never need resetting between launches.  Each workgroup asks for
// its next ticket when it starts an item, so the atomic's latency hides behind the item.
//
// NRT: steps (kernel row x kernel word) per input channel when it is 3 or 6 (every 3x3
// layer), so batches never straddle channels; 0 for any other count.  SG: the result is
// signed (either operand signed), so lanes need the fix-up and are sign-extended.  RNTW:
// 0, or the kernel words per kernel row (1 or 2) of a 3-row, stride-1 kernel whose rows
// share operand loads: output row r with kernel row ky reads input row r + ky, so the
// lane's RH rows need RH + 2 operand words per (channel, kernel word) instead of 3 RH.
// Every operand load costs the compute unit's texture path far more cycles than a
// multiply-add costs a SIMD, and the four SIMDs share that path, so loads, not
// multiply-adds, bound the loop unless each load feeds enough of them.
template <int RH, int NRT, bool SG, int RNTW, bool SEG>
__global__ __launch_bounds__(1024) void conv2d_samd_kernel(const int32_t *__restrict__ xs,
                                                           const int32_t *__restrict__ kw,
                                                           const int32_t *__restrict__ pre, int32_t *__restrict__ y,
                                                           unsigned long long *__restrict__ tickets,
                                                           const Conv2dGeom g) {
    extern __shared__ int32_t lds[];
    int32_t *tile = lds;
    __shared__ int32_t next_item;

    const int xcd = blockIdx.x % kNumXcd;
    const int ntiles = g.tiles;                                          // N x row tiles x column segments
    // XCD x owns the tiles [t0, t1): a contiguous range, so neighbouring row tiles (which
    // share their halo input rows) meet in one L2
    const int t0 = (int)((int64_t)xcd * ntiles / kNumXcd), t1 = (int)((int64_t)(xcd + 1) * ntiles / kNumXcd);
    const int nitems = (t1 - t0) * g.nmb;                                // items of this XCD
    const int nwg = gridDim.x / kNumXcd;                                 // workgroups of this XCD
    const int nextra = max(0, nitems - nwg);                             // items handed out by ticket
    unsigned long long *const counter = tickets + xcd * (kTicketStride / 8);

    const int tid = threadIdx.x;
    const int nthr = g.wm * g.ks * 64;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int kq = wave / g.wm;
    const int mw = wave - kq * g.wm;
    const int lane = tid & 63;
    const int grp_raw = lane / g.nqs;
    const bool lane_ok = grp_raw < g.groups;
    const int grp = lane_ok ? grp_raw : 0;
    const int q = lane_ok ? lane - grp_raw * g.nqs : 0;   // word within the column segment

    {
        int4 *t4 = (int4 *)tile;   // lds_tile is a multiple of 4 words
        for (int i = tid; i < g.lds_tile / 4; i += nthr) t4[i] = int4{0, 0, 0, 0};
    }

    int64_t acc[RH][RM];
#pragma unroll
    for (int r = 0; r < RH; ++r)
#pragma unroll
        for (int m = 0; m < RM; ++m) acc[r][m] = 0;

    // Decode: lane j of word q goes to output column q*I + j - (Kmax-1), stored at tile
    // column q*I + j.  Tile rows cover every row a wave computes, so no lane needs a
    // bounds check.  The tile index of each (row, channel) accumulator is one add away from
    // the previous one; the running index is opaque to the compiler, which would otherwise
    // keep all RH*8 indices (times every lane-count case) live across the main loop and
    // cut the waves a SIMD can hold.
    const int tidx0 = ((mw * RM) * g.tile_rows + grp * RH) * g.tile_row + q * g.I;
    const int mstride = g.tile_rows * g.tile_row;
    auto decode = [&]() {
        if (lane_ok) {
            const uint64_t msb = g.msb_mask;
            const int L = g.L, fw = g.L - 1;
            int ti = tidx0;
#define SAMD_DECODE_LOOP(CALL)                                                                        \
    _Pragma("unroll") for (int m = 0; m < RM; ++m) {                                                 \
        asm volatile("" : "+v"(ti));                                                                  \
        int tr = ti;                                                                                  \
        _Pragma("unroll") for (int r = 0; r < RH; ++r) {                                             \
            CALL;                                                                                     \
            tr += g.tile_row;                                                                         \
        }                                                                                             \
        ti += mstride;                                                                                \
    }
#define SAMD_DECODE_NL(NL_, PS_)                                                                      \
    case NL_:                                                                                         \
        SAMD_DECODE_LOOP((decode_word<SG, NL_, PS_>((uint64_t)acc[r][m], msb, L, fw, tile + tr)))     \
        break;
#define SAMD_DECODE_ALL(PS_)                                                                          \
    switch (g.nl) {                                                                                   \
        SAMD_DECODE_NL(2, PS_) SAMD_DECODE_NL(3, PS_) SAMD_DECODE_NL(4, PS_) SAMD_DECODE_NL(5, PS_)   \
        SAMD_DECODE_NL(6, PS_) SAMD_DECODE_NL(7, PS_) SAMD_DECODE_NL(8, PS_)                          \
    default:                                                                                          \
        SAMD_DECODE_LOOP((decode_word_n<SG, PS_>((uint64_t)acc[r][m], msb, L, fw, g.nl, tile + tr)))  \
    }
            if constexpr (SG) {
                if (g.spacer) {
                    SAMD_DECODE_ALL(true)
                } else {
                    SAMD_DECODE_ALL(false)
                }
            } else {
                SAMD_DECODE_ALL(false)
            }
#undef SAMD_DECODE_ALL
#undef SAMD_DECODE_NL
#undef SAMD_DECODE_LOOP
        }
#pragma unroll
        for (int r = 0; r < RH; ++r)
#pragma unroll
            for (int m = 0; m < RM; ++m) acc[r][m] = 0;
    };

    // orders the tile's zeroing before the first item's decodes
    __syncthreads();
    for (int item = blockIdx.x / kNumXcd; item < nitems;) {
        unsigned long long ticket = 0;
        if (nextra > 0 && tid == 0) ticket = atomicAdd(counter, 1ull);
        const int mb = item % g.nmb;
        const int tile_id = t0 + item / g.nmb;   // (n, row tile, column segment)
        // SEG: rows are split into column segments; without, the segment terms fold away
        // (their run-time divisions and bounds cost measurable time per item)
        const int cs = SEG ? tile_id % g.ncs : 0, rt_id = SEG ? tile_id / g.ncs : tile_id;
        const int n = rt_id / g.row_tiles;
        const int ho0 = (rt_id - n * g.row_tiles) * g.rows_blk;
        const int wb = mb * g.wm + mw;
        // the lane's word in the row; words past the row (last segment) read its last
        // word and only reach columns that are never stored
        const int qg = SEG ? min(cs * g.qseg + q, g.nq - 1) : q;

        // Operand word of step s (s = ky*ntw + t) of channel c for this lane's row r:
        // xs[n][c][hp][t][q] with hp = (ho0 + row)*sh + ky, i.e. word
        // (c*Hp*ntw + (ho0 + row)*sh*ntw + s)*nq + q of image n.  Rows past the image (the last
        // row tile, idle lanes) read the last output row's inputs; their sums are not stored.
        const int ch_stride = g.Hp * g.ntw * g.nq;
        int lb[RH];   // byte offset of the lane's word in channel 0, step 0
#pragma unroll
        for (int r = 0; r < RH; ++r) {
            const int row = min(ho0 + min(grp * RH + r, g.rows_blk - 1), g.Ho - 1);
            lb[r] = (row * g.sh * g.ntw * g.nq + qg) * 4;
        }
        // the image's channels and one spare channel after them
        const __amdgpu_buffer_rsrc_t xrs = __builtin_amdgcn_make_buffer_rsrc(
            (void *)(xs + (int64_t)n * g.C * ch_stride), (short)0, (g.C + 1) * ch_stride * 4, kBufferWord3);

        const int64_t stream_len = ((int64_t)g.C * g.nrt + kStreamPad) * RM;
        const int32_t *kstream = kw + wb * stream_len;

        // This wave's channel slice: channels cbeg .. cend-1, decoded after every G channels.
        const int cbeg = min(kq * g.cpw, g.C), cend = min(cbeg + g.cpw, g.C);
        const int32_t *ks_slice = kstream + (int64_t)cbeg * g.nrt * RM;
        int32_t kA[kStepBatch * RM], aA[kStepBatch][RH], kB[kStepBatch * RM], aB[kStepBatch][RH];
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
        // Batches of kStepBatch steps: kernel words in SGPRs (scalar loads), the lane's operand
        // words from global memory.  Ping-pong over two register sets.  Before a batch's kernel
        // words are used, all outstanding scalar loads are waited for, and only then is the
        // next batch requested: scalar loads return out of order, so a wait placed after
        // requesting the next batch would wait for it too.  Operand loads are vector loads,
        // which complete in order, so the compiler waits for exactly the batch in use.  The
        // batch after the last one is fetched as well (its results are never used): it reads
        // the next channel, which exists (the spread buffer has one spare channel after the
        // last image), and the kStreamPad padding steps of the kernel-word stream.
        if constexpr (RNTW != 0) {
            // batch b: kernel word t = b % RNTW of channel cbeg + b / RNTW, its three kernel
            // rows (the stream is kernel-word-major within a channel, so they are steps
            // 3b .. 3b+2 of the slice); operand words of input rows hp0 + i, i < RH + 2
            // (rows past the padded image are clamped to its last row: they only reach
            // output rows that are never stored)
            constexpr int NA = RH + 2;
            int lbi[NA];
#pragma unroll
            for (int i = 0; i < NA; ++i)
                lbi[i] = (min(ho0 + grp * RH + i, g.Hp - 1) * RNTW * g.nq + qg) * 4;
            const int nbat = (cend - cbeg) * RNTW;
            const int seg = g.G * RNTW;
            int32_t kRA[kStepBatch * RM], aRA[NA], kRB[kStepBatch * RM], aRB[NA];
            auto load_rows = [&](int b, int32_t (&kb)[kStepBatch * RM], int32_t (&ab)[NA]) {
#pragma unroll
                for (int j = 0; j < kStepBatch * RM; ++j) kb[j] = ks_slice[b * kStepBatch * RM + j];
                const int sb = ((cbeg + b / RNTW) * ch_stride + (b % RNTW) * g.nq) * 4;
#pragma unroll
                for (int i = 0; i < NA; ++i) ab[i] = buffer_word(xrs, lbi[i], sb);
            };
            auto mac_rows = [&](const int32_t (&kb)[kStepBatch * RM], const int32_t (&ab)[NA]) {
#pragma unroll
                for (int ky = 0; ky < kStepBatch; ++ky) {
#pragma unroll
                    for (int r = 0; r < RH; ++r)
#pragma unroll
                        for (int m = 0; m < RM; ++m)
                            acc[r][m] += (int64_t)ab[r + ky] * (int64_t)kb[ky * RM + m];
#pragma unroll
                    for (int r = 0; r < RH; ++r)
#pragma unroll
                        for (int m = 0; m < RM; ++m) keep(acc[r][m]);
                }
            };
            if (nbat > 0) {
                int left = seg;   // batches until the next decode
                load_rows(0, kRA, aRA);
                int b = 0;
                for (; b + 1 < nbat; b += 2) {
                    __builtin_amdgcn_s_waitcnt(0xc07f);   // lgkmcnt(0)
                    load_rows(b + 1, kRB, aRB);
                    __builtin_amdgcn_sched_barrier(0);
                    mac_rows(kRA, aRA);
                    __builtin_amdgcn_sched_barrier(0);
                    if (--left == 0) {
                        decode();
                        left = seg;
                    }
                    __builtin_amdgcn_s_waitcnt(0xc07f);
                    load_rows(b + 2, kRA, aRA);
                    __builtin_amdgcn_sched_barrier(0);
                    mac_rows(kRB, aRB);
                    __builtin_amdgcn_sched_barrier(0);
                    if (--left == 0) {
                        decode();
                        left = seg;
                    }
                }
                if (b < nbat) {   // odd batch count: the last batch
                    __builtin_amdgcn_s_waitcnt(0xc07f);
                    mac_rows(kRA, aRA);
                    --left;
                }
                if (left != seg) decode();
            }
        } else if constexpr (NRT != 0) {
            // 3 or 6 steps per channel: batch b is steps (b % BPC)*3 .. +2 of channel
            // cbeg + b / BPC, and the slice is one pipeline; the decode after every G channels
            // runs while the next batch's loads are in flight.
            constexpr int BPC = NRT / kStepBatch;
            const int nbat = (cend - cbeg) * BPC;
            const int seg = g.G * BPC;   // batches between decodes
            auto load_batch = [&](int b, int32_t (&kb)[kStepBatch * RM], int32_t (&ab)[kStepBatch][RH]) {
#pragma unroll
                for (int j = 0; j < kStepBatch * RM; ++j) kb[j] = ks_slice[b * kStepBatch * RM + j];
                const int sb = ((cbeg + b / BPC) * ch_stride + (b % BPC) * kStepBatch * g.nq) * 4;
#pragma unroll
                for (int j = 0; j < kStepBatch; ++j)
#pragma unroll
                    for (int r = 0; r < RH; ++r) ab[j][r] = buffer_word(xrs, lb[r], sb + j * g.nq * 4);
            };
            if (nbat > 0) {
                int left = seg;   // batches until the next decode
                load_batch(0, kA, aA);
                int b = 0;
                for (; b + 1 < nbat; b += 2) {
                    __builtin_amdgcn_s_waitcnt(0xc07f);   // lgkmcnt(0)
                    load_batch(b + 1, kB, aB);
                    __builtin_amdgcn_sched_barrier(0);
                    mac_batch(kA, aA);
                    __builtin_amdgcn_sched_barrier(0);
                    if (--left == 0) {
                        decode();
                        left = seg;
                    }
                    __builtin_amdgcn_s_waitcnt(0xc07f);
                    load_batch(b + 2, kA, aA);
                    __builtin_amdgcn_sched_barrier(0);
                    mac_batch(kB, aB);
                    __builtin_amdgcn_sched_barrier(0);
                    if (--left == 0) {
                        decode();
                        left = seg;
                    }
                }
                if (b < nbat) {   // odd batch count: the last batch
                    __builtin_amdgcn_s_waitcnt(0xc07f);
                    mac_batch(kA, aA);
                    --left;
                }
                if (left != seg) decode();
            }
        } else {
            // any other step count: segments of at most G channels, each its own pipeline;
            // batches straddle channels, and steps past a segment multiply by a zero operand
            for (int c0 = cbeg; c0 < cend; c0 += g.G) {
                const int nsteps = min(g.G, cend - c0) * g.nrt;
                const int nbat = (nsteps + kStepBatch - 1) / kStepBatch;
                const int32_t *ks = ks_slice + (int64_t)(c0 - cbeg) * g.nrt * RM;
                auto load_batch = [&](int b, int32_t (&kb)[kStepBatch * RM], int32_t (&ab)[kStepBatch][RH]) {
#pragma unroll
                    for (int j = 0; j < kStepBatch * RM; ++j) kb[j] = ks[b * kStepBatch * RM + j];
#pragma unroll
                    for (int j = 0; j < kStepBatch; ++j) {
                        const int st0 = b * kStepBatch + j;
                        const bool live = st0 < nsteps;
                        const int st = min(st0, nsteps - 1);
                        const int cc = st / g.nrt, rt = st - cc * g.nrt;
                        const int sb = ((c0 + cc) * ch_stride + rt * g.nq) * 4;
#pragma unroll
                        for (int r = 0; r < RH; ++r) {
                            const int32_t v = buffer_word(xrs, lb[r], sb);
                            ab[j][r] = live ? v : 0;
                        }
                    }
                };
                load_batch(0, kA, aA);
                int b = 0;
                for (; b + 1 < nbat; b += 2) {
                    __builtin_amdgcn_s_waitcnt(0xc07f);
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
                if (b < nbat) {
                    __builtin_amdgcn_s_waitcnt(0xc07f);
                    mac_batch(kA, aA);
                }
                decode();
            }
        }
        if (tid == 0)
            next_item = nextra > 0 ? nwg + (int)(ticket % (unsigned long long)(nextra + nwg)) : nitems;
        __syncthreads();
        const int following = __builtin_amdgcn_readfirstlane(next_item);

        // output tile -> y: wave w copies rows rr = w, w + nwaves, ... (rr = mm * rows_blk + r)
        // of the tile, lanes along the row
        const int nwaves = g.wm * g.ks;
        const int dmm = nwaves / g.rows_blk, dr = nwaves - dmm * g.rows_blk;
        int mm = wave / g.rows_blk, r = wave - mm * g.rows_blk;
        const int c0 = SEG ? cs * g.cw : 0, ncols = SEG ? min(g.cw, g.Wo - c0) : g.Wo;   // the segment's output columns
        const int segw = SEG ? g.cw : g.Wo;
        while (mm < g.mblk) {
            const int m = mb * g.mblk + mm, ho = ho0 + r;
            // every tile word of a segment column (cw of them) is zeroed for the next item
            // once read, also in rows past the image, channels past M and columns past Wo,
            // which another item stores
            int32_t *src = tile + (mm * g.tile_rows + r) * g.tile_row + (g.Kmax - 1);
            if (m < g.M && ho < g.Ho) {
                int32_t *dst = y + (((int64_t)n * g.M + m) * g.Ho + ho) * g.Wo + c0;
                if (g.xoff == 0) {
                    for (int o = lane; o < ncols; o += 64) {
                        dst[o] = src[o];
                        src[o] = 0;
                    }
                } else {
                    // recentred activations: + xoff * (weights over the output's in-image taps)
                    const int hb = ho * g.sh - g.ph, kwid = g.KW + 1;
                    const int ky0 = max(0, -hb) * kwid, ky1 = min(g.KH, g.H - hb) * kwid;
                    const int32_t *pm = pre + (int64_t)m * (g.KH + 1) * kwid;
                    for (int o = lane; o < ncols; o += 64) {
                        const int wbeg = (c0 + o) * g.sw - g.pw;
                        const int kx0 = max(0, -wbeg), kx1 = min(g.KW, g.W - wbeg);
                        const int32_t rect = pm[ky1 + kx1] - pm[ky0 + kx1] - pm[ky1 + kx0] + pm[ky0 + kx0];
                        dst[o] = src[o] + g.xoff * rect;
                        src[o] = 0;
                    }
                }
                // the columns past Wo of the last segment
                if (SEG)
                    for (int o = ncols + lane; o < segw; o += 64) src[o] = 0;
            } else {
                for (int o = lane; o < segw; o += 64) src[o] = 0;
            }
            mm += dmm;
            r += dr;
            if (r >= g.rows_blk) {
                r -= g.rows_blk;
                ++mm;
            }
        }
        item = following;
        // the write-out (and the tile's re-zeroing) ends before the next item's decodes
        if (item < nitems) __syncthreads();
    }
}

}  // namespace

int launch_conv2d_prepare(const uint32_t *w, const Conv2dGeom &g, void *ws, hipStream_t s) {
    int32_t *kw = (int32_t *)ws;
    int32_t *queue = (int32_t *)((char *)ws + conv2d_queue_offset(g));
    const int pgrid = grid_for(g.kw_words, 256);
    bool launched = false;
#define SAMD_PREP_CASE(B, SG)                                                                            \
    if (!launched && g.wbits == B && (bool)g.wsigned == SG) {                                            \
        hipLaunchKernelGGL((prep_weights_kernel<B, SG>), dim3(pgrid), dim3(256), 0, s, w, g, kw, queue);        \
        launched = true;                                                                                 \
    }
    SAMD_FOR_EACH_FMT(SAMD_PREP_CASE)
#undef SAMD_PREP_CASE
    int st = check_launch("conv2d weight preparation");
    if (st || !g.xoff) return st;
    int32_t *pre = (int32_t *)((char *)ws + conv2d_kw_bytes(g));
    const int fgrid = grid_for((int64_t)g.M * (g.KH + 1) * (g.KW + 1), 256);
    launched = false;
#define SAMD_PREFIX_CASE(B, SG)                                                                          \
    if (!launched && g.wbits == B && (bool)g.wsigned == SG) {                                            \
        hipLaunchKernelGGL((prefix_kernel<B, SG>), dim3(fgrid), dim3(256), 0, s, w, g, pre);             \
        launched = true;                                                                                 \
    }
    SAMD_FOR_EACH_FMT(SAMD_PREFIX_CASE)
#undef SAMD_PREFIX_CASE
    return check_launch("conv2d correction table");
}

int launch_conv2d_spread(const uint32_t *x, const Conv2dGeom &g, void *ws, hipStream_t s, int32_t *dst) {
    int32_t *xs = dst ? dst : (int32_t *)((char *)ws + conv2d_xs_offset(g));
    // 2^qshift threads per row, each building about 2.5 of its words (words q, q + 2^qshift,
    // ...): one word per thread was 5-23 % slower at the mid-size layer
    const int qshift = spread_qshift(g.nq);
    const int64_t nrows = (int64_t)g.N * g.C * g.Hp;
    const int rpb = 256 >> qshift;
    const int64_t blocks = (nrows + rpb - 1) / rpb;   // one thread group per row, no grid-stride loop
    // the planner refuses layers that would need 2^32 threads or more (addressable())
    if (blocks * 256 > (int64_t)0xffffffff) {
        set_error("conv2d operand spread: more than 2^32 threads in one launch");
        return SAMD_EUNSUPPORTED;
    }
    const unsigned sgrid = (unsigned)blocks;
    bool launched = false;
#define SAMD_SPREAD_CASE(B, SG)                                                                            \
    if (!launched && g.xbits == B && (bool)g.xsigned == SG) {                                              \
        hipLaunchKernelGGL((spread_kernel<B, SG>), dim3(sgrid), dim3(256), 0, s, x, g, qshift, xs);        \
        launched = true;                                                                                   \
    }
    SAMD_FOR_EACH_FMT(SAMD_SPREAD_CASE)
#undef SAMD_SPREAD_CASE
    return check_launch("conv2d operand spread");
}

int launch_conv2d_spread_bytes(const void *x, const Conv2dGeom &g, int32_t *dst, hipStream_t s) {
    const int qshift = spread_qshift(g.nq);
    const int64_t nrows = (int64_t)g.N * g.C * g.Hp;
    const int rpb = 256 >> qshift;
    const int64_t blocks = (nrows + rpb - 1) / rpb;
    // the planner refuses layers that would need 2^32 threads or more (addressable())
    if (blocks * 256 > (int64_t)0xffffffff) {
        set_error("conv2d spaced pack: more than 2^32 threads in one launch");
        return SAMD_EUNSUPPORTED;
    }
    // the stored values' format: signed when the activations are (recentred unsigned
    // activations are stored unsigned and shifted by xoff inside the kernel)
    const bool sgn = g.xsigned != 0;
    bool launched = false;
#define SAMD_SPREAD_BYTES_CASE(B, SG)                                                                    \
    if (!launched && g.xbits == B && sgn == SG) {                                                        \
        hipLaunchKernelGGL((spread_bytes_kernel<B, SG>), dim3((unsigned)blocks), dim3(256), 0, s,       \
                           (const uint8_t *)x, g, qshift, dst);                                          \
        launched = true;                                                                                 \
    }
    SAMD_FOR_EACH_FMT(SAMD_SPREAD_BYTES_CASE)
#undef SAMD_SPREAD_BYTES_CASE
    return check_launch("conv2d spaced pack");
}

namespace {

// Workgroups of `kernel` the current device keeps resident at once (all compute units),
// looked up once per (device, kernel, block, LDS bytes).
int resident_workgroups(const void *kernel, int block, size_t shm, int &out) {
    static std::mutex mu;
    static std::map<std::tuple<int, const void *, int, size_t>, int> cache;
    int dev = 0;
    if (hipGetDevice(&dev) != hipSuccess) {
        set_error("conv2d: hipGetDevice failed");
        return SAMD_EHIP;
    }
    const auto key = std::make_tuple(dev, kernel, block, shm);
    {
        std::lock_guard<std::mutex> lock(mu);
        auto it = cache.find(key);
        if (it != cache.end()) {
            out = it->second;
            return SAMD_OK;
        }
    }
    int per_cu = 0, cus = 0;
    hipError_t e = hipOccupancyMaxActiveBlocksPerMultiprocessor(&per_cu, kernel, block, shm);
    if (e == hipSuccess) e = hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev);
    if (e != hipSuccess) {
        set_error(std::string("conv2d: occupancy query: ") + hipGetErrorString(e));
        return SAMD_EHIP;
    }
    out = std::max(1, per_cu) * std::max(1, cus);
    std::lock_guard<std::mutex> lock(mu);
    cache[key] = out;
    return SAMD_OK;
}

template <int RH, int NRT, bool SG, int RNTW, bool SEG>
int launch_multiply_seg(const Conv2dGeom &g, int32_t *y, const void *ws, hipStream_t s, const int32_t *src) {
    const int32_t *kw = (const int32_t *)ws;
    const int32_t *pre = (const int32_t *)((const char *)ws + conv2d_kw_bytes(g));
    unsigned long long *tickets =
        (unsigned long long *)((char *)const_cast<void *>(ws) + conv2d_queue_offset(g));
    const int32_t *xs = src ? src : (const int32_t *)((const char *)ws + conv2d_xs_offset(g));
    const int block = g.wm * g.ks * 64;
    const size_t shm = (size_t)g.lds_words * 4;
    const void *fn = (const void *)conv2d_samd_kernel<RH, NRT, SG, RNTW, SEG>;
    int resident = 0;
    const int st = resident_workgroups(fn, block, shm, resident);
    if (st) return st;
    // every XCD gets the same number of workgroups; none gets more than its items
    const int64_t xitems = (int64_t)(g.tiles + kNumXcd - 1) / kNumXcd * g.nmb;
    const int64_t per_xcd = std::max<int64_t>(1, std::min<int64_t>(xitems, resident / kNumXcd));
    hipLaunchKernelGGL((conv2d_samd_kernel<RH, NRT, SG, RNTW, SEG>), dim3((unsigned)(per_xcd * kNumXcd)), dim3(block), shm, s,
                       xs, kw, pre, y, tickets, g);
    return check_launch("conv2d");
}

template <int RH, int NRT, bool SG, int RNTW>
int launch_multiply(const Conv2dGeom &g, int32_t *y, const void *ws, hipStream_t s, const int32_t *src) {
    return g.ncs > 1 ? launch_multiply_seg<RH, NRT, SG, RNTW, true>(g, y, ws, s, src)
                     : launch_multiply_seg<RH, NRT, SG, RNTW, false>(g, y, ws, s, src);
}

}  // namespace

int launch_conv2d_multiply(const Conv2dGeom &g, int32_t *y, const void *ws, hipStream_t s, const int32_t *src) {
    if (g.rows_path) {
#define SAMD_ROWS_CASE(RH_, NTW_, SG_)                                                                \
    if (g.rh == RH_ && g.ntw == NTW_ && (bool)g.result_signed == SG_)                                 \
        return launch_multiply<RH_, 0, SG_, NTW_>(g, y, ws, s, src);
        SAMD_ROWS_CASE(1, 1, false) SAMD_ROWS_CASE(2, 1, false) SAMD_ROWS_CASE(3, 1, false) SAMD_ROWS_CASE(4, 1, false)
        SAMD_ROWS_CASE(1, 2, false) SAMD_ROWS_CASE(2, 2, false) SAMD_ROWS_CASE(3, 2, false) SAMD_ROWS_CASE(4, 2, false)
        SAMD_ROWS_CASE(1, 1, true) SAMD_ROWS_CASE(2, 1, true) SAMD_ROWS_CASE(3, 1, true) SAMD_ROWS_CASE(4, 1, true)
        SAMD_ROWS_CASE(1, 2, true) SAMD_ROWS_CASE(2, 2, true) SAMD_ROWS_CASE(3, 2, true) SAMD_ROWS_CASE(4, 2, true)
#undef SAMD_ROWS_CASE
    } else {
#define SAMD_CONV_CASE(RH_, NRT_, SG_)                                                                \
    if (g.rh == RH_ && (NRT_ == 0 ? (g.nrt != 3 && g.nrt != 6) : g.nrt == NRT_) &&                     \
        (bool)g.result_signed == SG_)                                                                 \
        return launch_multiply<RH_, NRT_, SG_, 0>(g, y, ws, s, src);
        SAMD_CONV_CASE(1, 3, false) SAMD_CONV_CASE(1, 6, false) SAMD_CONV_CASE(1, 0, false)
        SAMD_CONV_CASE(2, 3, false) SAMD_CONV_CASE(2, 6, false) SAMD_CONV_CASE(2, 0, false)
        SAMD_CONV_CASE(1, 3, true) SAMD_CONV_CASE(1, 6, true) SAMD_CONV_CASE(1, 0, true)
        SAMD_CONV_CASE(2, 3, true) SAMD_CONV_CASE(2, 6, true) SAMD_CONV_CASE(2, 0, true)
#undef SAMD_CONV_CASE
    }
    set_error("conv2d: no kernel for this geometry");
    return SAMD_EUNSUPPORTED;
}

int launch_conv2d_samd(const uint32_t *x, const Conv2dGeom &g, int32_t *y, const void *ws, hipStream_t s) {
    const int st = launch_conv2d_spread(x, g, const_cast<void *>(ws), s, nullptr);
    if (st) return st;
    return launch_conv2d_multiply(g, y, ws, s, nullptr);
}

}  // namespace samd
