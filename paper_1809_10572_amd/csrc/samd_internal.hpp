// Internal declarations of the SAMD library: the lane-geometry plans computed on the
// host, the kernel launchers, and small helpers shared by host and device code.
#pragma once

#include <stddef.h>
#include <stdint.h>

#include <functional>
#include <string>
#include <vector>

#include "samd.h"

namespace samd {

constexpr int kMaxTapWords = 16;   // kernel words per (input channel, kernel row)
constexpr int kMaxLanes = 16;      // I: values per operand word
constexpr int kMaxOutLanes = 20;   // I + Kmax - 1: lanes of an accumulator that are decoded
constexpr int kWaveM = 8;          // output channels per wave (kernel words per step, in SGPRs)
constexpr int kMaxConv1dExtra = 15; // following words whose low lanes reach a 1-D output word
// Values per 1-D operand word: the conv1d kernel keeps a lane's outputs in registers and
// stores them directly; more, shorter words per row also give the GPU more lanes to run.
constexpr int kConv1dMaxLanes = 4;
constexpr int kStepBatch = 3;      // kernel-word steps fetched per scalar-load batch
constexpr int kStreamPad = 2 * kStepBatch;  // zero steps after each kernel-word stream
constexpr int kMaxBlockWaves = 16; // waves per conv2d workgroup
constexpr int kMaxLdsBytes = 65536; // LDS per conv2d workgroup
constexpr int kNumXcd = 8;          // accelerator complexes (each with its own L2); workgroup p runs on p % 8
constexpr int kTicketStride = 256;  // bytes between the conv2d ticket counters (one per XCD)
constexpr int kQueueBytes = kNumXcd * kTicketStride;
constexpr int kResidentWavesPerSimd = 6;  // conv2d multiply kernel, as measured (register-limited)

// Geometry of one SAMD 2-D convolution.  Every operand word is a signed 32-bit
// integer A = sum_i v_i 2^(i L) holding I input values of one stride phase of one
// input row (temporary spacer bits between them, negative values sign-extended);
// every kernel word B = sum_s w_s 2^(s L) holds up to Kmax taps of one phase of one
// kernel row, reversed.  A*B accumulates into a 64-bit integer whose L-bit lane j
// holds a partial sum for output column q*I + j - (Kmax - 1).
//
// Kernel word t of a kernel row multiplies operand words whose window starts at phase
// index q*I + delta_t, delta_t = tap0_t + ntaps_t - Kmax; each kernel word has its own
// operand-word variant, stored at index t.
struct Conv2dGeom {
    int32_t N, C, H, W, M, KH, KW, sh, sw, ph, pw, Ho, Wo, Hp;
    int32_t xbits, xsigned, wbits, wsigned;   // xsigned: how stored activations are read
    int32_t xoff;                   // subtracted from every activation (recentred unsigned
                                    // activations: 2^(xbits-1)); 0 otherwise
    int32_t L, I, Kmax, nq, G;      // lane bits, values/word, widest phase, words/row, flush channels
    int32_t nl;                     // decoded lanes per accumulator; lane nl-1 takes the remaining bits
    int32_t result_signed;          // any operand signed: lanes need the fix-up
    int32_t layout_spaced;          // planned for the permanent-spacer layout (caller-held operand words)
    int32_t spacer;                 // layout_spaced and result_signed: every decoded lane keeps its MSB
                                    // as a spacer bit (values fit L - 1 bits), so the decode leaves out
                                    // the fix-up's final xor and reads L - 1-bit fields (Sec. 6.1)
    uint64_t msb_mask;              // sign bit of lanes 0 .. nl-2
    int32_t ntw;                    // kernel words (and operand-word variants) per (channel, kernel row)
    int32_t tw_phase[kMaxTapWords], tw_tap0[kMaxTapWords], tw_ntaps[kMaxTapWords];
    int32_t nrt;                    // steps per channel: KH * ntw
    // launch shape
    int32_t rows_path;              // 1: 3-row stride-1 kernel whose output rows share operand loads
                                    // (kernel-word streams kernel-word-major within a channel)
    int32_t rh;                     // output rows per thread
    int32_t groups;                 // row groups per wave: 64 / nqs
    int32_t rows_blk;               // output rows per workgroup: rh * groups
    int32_t wm;                     // output-channel waves per workgroup, each kWaveM channels
    int32_t ks;                     // channel-split waves: wave (kq, mw) multiplies channel slice kq
    int32_t mblk;                   // output channels per workgroup, wm * kWaveM
    int32_t nmb;                    // output-channel blocks
    int32_t row_tiles;              // ceil(Ho / rows_blk)
    int32_t tiles;                  // spatial tiles: N * row_tiles * ncs
    int32_t chk;                    // ks * cpw (reported)
    int32_t cpw;                    // input channels of one wave's slice: ceil(C / ks)
    int32_t trows;                  // input rows a tile reads, (rows_blk-1)*sh + KH
    int32_t xrw;                    // packed words per input row
    int32_t wrw;                    // packed words per kernel row
    int32_t tile_rows;              // output-tile rows per channel: groups * rh
    int32_t tile_row;               // output-tile words per row: nqs * I + Kmax - 1 (segment column o at o + Kmax - 1)
    int32_t lds_tile;               // LDS words of the output tile (a multiple of 4)
    int32_t lds_words;              // LDS words in all
    int64_t kw_words, spread_words; // workspace: kernel-word streams, operand words (after the
                                    // correction table when xoff != 0)
    double macs_per_mad, cost;
    // column segments (rows of more than 64 operand words)
    int32_t nqs;                    // words of one column segment (<= 64: a lane group's words)
    int32_t cw;                     // output columns per column segment (Wo when ncs == 1)
    int32_t ncs;                    // column segments per output row
    int32_t qseg;                   // words between column segments: cw / I
};

// 1-D convolution geometry (unsigned operands, 32x32 -> 64-bit products).
struct Conv1dGeom {
    int64_t n, nout, nwords;        // inputs, outputs, output words
    int32_t bits, K, L, I, extra;   // extra: following words whose low lanes reach a word's outputs
    int32_t nl;                     // lanes that can be non-zero; lane nl-1 takes all remaining bits
    int32_t ngroups;
    int32_t g_tap0[kMaxTapWords], g_ntaps[kMaxTapWords];
    int32_t g_delta[kMaxTapWords];  // window offset of each kernel word
    uint32_t g_word[kMaxTapWords];  // the kernel words themselves (taps packed, unsigned)
    int32_t xrw;
};

// Host planning (pure C++, no HIP calls).  Return SAMD_OK or an error with `err` set.
// spacer: plan for the permanent-spacer layout (samd_conv2d_spaced*) instead of the
// packed one; the two are planned, cached and tuned separately.
int plan_conv2d(const samd_conv2d_desc &d, samd_fmt xf, samd_fmt wf, Conv2dGeom &g, std::string &err,
                int spacer = 0);
int plan_conv1d(int64_t n, samd_fmt xf, const int32_t *taps, int32_t K, samd_fmt kf, Conv1dGeom &g,
                std::string &err);
// Candidate plans of a shape, ranked by the model's cost, the model's choice first, at
// most max_count of them (distinct lane geometries and launch shapes).
int conv2d_candidates(const samd_conv2d_desc &d, samd_fmt xf, samd_fmt wf, int max_count,
                      std::vector<Conv2dGeom> &out, std::string &err, int spacer = 0);
// The first of all candidate plans (no count limit) that `match` accepts.
int find_conv2d_candidate(const samd_conv2d_desc &d, samd_fmt xf, samd_fmt wf,
                          const std::function<bool(const Conv2dGeom &)> &match, Conv2dGeom &out,
                          std::string &err, int spacer = 0);
// Plans chosen by measurement take precedence in plan_conv2d until cleared (d == NULL:
// every shape; otherwise both layouts of the shape).  A plan is kept under its own
// layout (g.layout_spaced).
void set_tuned_conv2d(const samd_conv2d_desc &d, samd_fmt xf, samd_fmt wf, const Conv2dGeom &g);
void clear_tuned_conv2d(const samd_conv2d_desc *d, samd_fmt xf, samd_fmt wf);
size_t conv2d_workspace_bytes(const Conv2dGeom &g);
size_t conv2d_kw_bytes(const Conv2dGeom &g);
size_t conv2d_pre_bytes(const Conv2dGeom &g);   // the recentring correction table
size_t conv2d_queue_offset(const Conv2dGeom &g); // work queues of the multiply kernel
size_t conv2d_xs_offset(const Conv2dGeom &g);    // operand words

// Kernel launchers (enqueue only; report launch errors through the return value).
int launch_pack(const void *src, int64_t rows, int64_t len, int bits, int is_signed, uint32_t *dst,
                int32_t *oor, hipStream_t s);
int launch_unpack(const uint32_t *src, int64_t rows, int64_t len, int bits, int is_signed, void *dst,
                  hipStream_t s);
int launch_conv1d(const uint32_t *x, const Conv1dGeom &g, int32_t *y, hipStream_t s);
int launch_conv2d_prepare(const uint32_t *w, const Conv2dGeom &g, void *ws, hipStream_t s);
int launch_conv2d_samd(const uint32_t *x, const Conv2dGeom &g, int32_t *y, const void *ws, hipStream_t s);
// The operand spread writes the workspace's operand words, or dst when given (the
// permanent-spacer layout held by the caller); the multiply reads the workspace's, or src.
int launch_conv2d_spread(const uint32_t *x, const Conv2dGeom &g, void *ws, hipStream_t s, int32_t *dst = nullptr);
int launch_conv2d_spread_bytes(const void *x, const Conv2dGeom &g, int32_t *dst, hipStream_t s);
int launch_conv2d_multiply(const Conv2dGeom &g, int32_t *y, const void *ws, hipStream_t s,
                           const int32_t *src = nullptr);
// samd_conv2d with the library's scratch array as the workspace (SAMD_ENOSPC when the
// layer's workspace does not fit it).
int launch_conv2d_noalloc(const uint32_t *x, const uint32_t *w, const Conv2dGeom &g, int32_t *y, hipStream_t s);
size_t conv2d_i8_workspace_bytes(const samd_conv2d_desc &d, samd_fmt xf);
int launch_conv2d_i8_prepare(const int8_t *w, samd_fmt xf, const samd_conv2d_desc &d, void *ws, hipStream_t s);
int launch_conv2d_i8(const void *x, samd_fmt xf, const samd_conv2d_desc &d, int32_t *y, const void *ws,
                     hipStream_t s);
// The int8 kernel and tile samd_conv2d_int8 uses for a layer with 16-byte aligned
// activations (host only).
int conv2d_i8_tiles(const samd_conv2d_desc &d, samd_fmt xf, samd_conv2d_int8_plan &out);
// Every launch the int8 baseline can make for a layer, and the override of its choice
// (plan NULL: back to the model's choice).
int conv2d_i8_candidates(const samd_conv2d_desc &d, samd_fmt xf, std::vector<samd_conv2d_int8_plan> &out);
int conv2d_i8_use_plan(const samd_conv2d_desc &d, samd_fmt xf, const samd_conv2d_int8_plan *plan);
int launch_max_i32(const int32_t *src, int64_t n, int32_t *dev_max, hipStream_t s);
int launch_count_mismatch(const int32_t *a, const int32_t *b, int64_t n, int32_t *count, hipStream_t s);
int launch_lanewise(int op, const uint32_t *a, const uint32_t *b, int64_t nwords, int bits, uint32_t scalar,
                    uint32_t *dst, hipStream_t s);
int launch_relu_requant_pack(const int32_t *acc, int64_t rows, int64_t len, const int32_t *dev_max, int bits,
                             uint32_t *dst, int32_t *dev_shift, hipStream_t s);
int launch_relu_requant_stage(const int32_t *acc, const int32_t *dev_max, const Conv2dGeom &g, void *ws,
                              int32_t *dev_shift, hipStream_t s, int32_t *dst = nullptr);
int launch_relu_requant_nhwc_u8(const int32_t *acc, int N, int C, int H, int W, const int32_t *dev_max,
                                int bits, uint8_t *dst, hipStream_t s);

// Error detail for the calling thread.
void set_error(const std::string &msg);

// Threads per padded row of the operand spread and the fused epilogue, as a power of two
// 2^q: about 2.5 operand words per thread (measured on MI355X, 2-3 words per thread
// amortise the per-thread row and address set-up best), at most 256.
inline int spread_qshift(int nq) {
    int q = 0;
    while ((1 << q) * 5 < 2 * nq && q < 8) ++q;
    return q;
}

inline int64_t row_words(int64_t len, int bits) {
    const int64_t per = 32 / bits;
    return (len + per - 1) / per;
}

}  // namespace samd
