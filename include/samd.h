/*
 * samd.h - C ABI of the SAMD quantized-convolution library for MI355X (gfx950).
 *
 * Method: Anderson, Doyle, Gregg, "Scalar Arithmetic Multiple Data: Customizable
 * Precision for Deep Neural Networks" (arXiv 1809.10572).  b-bit (1..8) signed or
 * unsigned integers are packed into machine words; a 1-D convolution is read out of
 * one wide integer multiply of a packed input word by a packed kernel word (Sec. 5,
 * "Convolution as Long Multiplication"); signed and mixed-sign lanes are made exact
 * by sign extension before the multiply and the underflow fix-up after it (Sec. 6).
 *
 * Conventions for every entry point:
 *  - Pointers are DEVICE pointers unless a parameter says "host".  The caller owns
 *    every buffer; the library allocates nothing and keeps no state between calls
 *    apart from a thread-local error message, a cache of computed plans (a pure
 *    function of shape and formats) and the plans chosen by samd_conv2d_tune or
 *    samd_conv2d_use_plan (process-wide mutable state, until samd_conv2d_untune).
 *  - Work is enqueued asynchronously on `stream` (0 = the default stream).  A return
 *    of SAMD_OK means the launch was accepted; results are ready once the stream is
 *    synchronised.
 *  - Arguments are validated on the host before any HIP call.  On a validation error
 *    nothing is enqueued and the GPU is not touched, so validation can be exercised
 *    without a GPU.  Nothing is thrown across the ABI.
 *  - Device buffers of 32-bit elements must be 4-byte aligned (SAMD_EALIGN).
 *
 * Packed storage format (shared by activations, weights and requantised outputs):
 *   a row of `len` b-bit values occupies ceil(len / P) uint32 words, P = floor(32/b);
 *   value j lies in bits [(j mod P)*b, (j mod P)*b + b) of word floor(j / P) as a
 *   b-bit two's-complement field when signed, unsigned otherwise; unused bits are 0;
 *   every row starts on a new word.  Storage stays dense: spacer bits exist only
 *   inside the kernels (temporary spacer bits, Sec. 2.2).  Signed 1-bit values are
 *   {-1, 0}.
 */
#ifndef SAMD_H
#define SAMD_H

#include <stddef.h>
#include <stdint.h>
#include <hip/hip_runtime_api.h>

#ifdef __cplusplus
extern "C" {
#endif

/* Bit width (1..8) and signedness of one operand. */
typedef struct {
    int32_t bits;
    int32_t is_signed;
} samd_fmt;

/* 2-D convolution shape: input N x C x H x W, weights M x C x KH x KW, output
 * N x M x Ho x Wo with Ho = (H + 2 pad_h - KH) / stride_h + 1 and likewise Wo. */
typedef struct {
    int32_t N, C, H, W, M, KH, KW, stride_h, stride_w, pad_h, pad_w;
} samd_conv2d_desc;

enum {
    SAMD_OK = 0,
    SAMD_EINVAL = -1,       /* bad argument: null pointer, bits out of 1..8, bad shape */
    SAMD_EALIGN = -2,       /* a 32-bit buffer is not 4-byte aligned */
    SAMD_EUNSUPPORTED = -3, /* no exact lane geometry exists for this shape / format */
    SAMD_EOVERFLOW = -4,    /* an exact result could exceed int32 */
    SAMD_EHIP = -5,         /* the HIP runtime reported an error (see samd_last_error) */
    SAMD_ENOSPC = -6        /* the workspace is smaller than the query returned */
};

/* Lane geometry chosen for a convolution (host-only query, for inspection and tests).
 *   lane_bits    L: bit width of one lane of the 64-bit accumulator
 *   lanes        I: input values per 32-bit operand word
 *   taps_max     Kmax: taps of the widest stride phase, ceil(KW / stride_w)
 *   words_per_row nq: operand words per output row, ceil((Wo + Kmax - 1) / I)
 *   flush_channels G: input channels accumulated before the lanes are decoded
 *   out_lanes    lanes of an accumulator that can be non-zero; the highest of them
 *                takes all the accumulator's remaining bits
 *   tap_words    kernel words per (input channel, kernel row)
 *   phase[i], tap0[i], ntaps[i] for i < tap_words: kernel word i holds ntaps[i]
 *                consecutive taps of stride phase phase[i], starting at phase tap tap0[i]
 *   rows_per_block, mblock: output rows and output channels of one workgroup's tile
 *   split_waves  waves that share one tile's output channels, each multiplying its own
 *                slice of every chunk of input channels (their sums meet in the tile)
 *   chunk_channels input channels per wave slice times split_waves
 *   x_offset     0, or 2^(b-1) when unsigned activations are recentred: x - x_offset
 *                (a signed b-bit value) enters the lanes, halving the largest product,
 *                and x_offset times the sum of each output's in-image weights is added
 *                back when the output is stored
 *   col_segments, segment_columns: output rows of more than 64 operand words are split
 *                into col_segments ranges of segment_columns output columns (a multiple
 *                of I), each computed from the at most 64 words it needs (words reaching
 *                two ranges are computed for both); 1 and Wo otherwise
 *   macs_per_mad multiply-accumulates delivered per 32x32->64 multiply (I * taps)
 *   rows_per_thread, shared_rows: output rows each lane computes, and whether they share
 *                operand loads (3-row, stride-1 kernels: RH + 2 loads per channel and
 *                kernel word instead of 3 RH)
 *   model_cost   the planner's cost estimate (issue cycles of one compute unit)
 *   layout_spaced 1: a plan of the permanent-spacer layout (samd_conv2d_spaced*)
 *   spacer_msb   1: result lanes keep their MSB as a spacer bit; the decode leaves out
 *                the fix-up's xor (Sec. 6.1) */
typedef struct {
    int32_t lane_bits, lanes, taps_max, words_per_row, flush_channels, out_lanes, tap_words;
    int32_t phase[16], tap0[16], ntaps[16];
    int32_t rows_per_block, mblock, split_waves, chunk_channels;
    int32_t x_offset;
    int32_t col_segments, segment_columns;
    double macs_per_mad;
    int32_t rows_per_thread, shared_rows;
    double model_cost;
    int32_t layout_spaced, spacer_msb;
} samd_conv2d_plan;

/* Human-readable name of a status code; never NULL. */
const char *samd_status_str(int status);

/* Detail of the last error on the calling thread ("" if none); valid until the next
 * call on this thread. */
const char *samd_last_error(void);

/* Library utility (sizes the packed storage format above; no passage of the paper):
 * words per packed row, ceil(len / floor(32 / f.bits)); negative status on error. */
int64_t samd_row_words(int64_t len, samd_fmt f);

/* Pack `rows` x `len` values (int8 when f.is_signed, else uint8; row-major) into the
 * packed storage format, dst holding rows x samd_row_words(len, f) words.  Values
 * outside the b-bit range are stored as their low b bits; when `oor_count` is not
 * NULL the number of such values is ADDED to *oor_count (a device int32).
 * The paper's baseline unpacks to the nearest native type (Sec. 7); this is the
 * inverse step. */
int samd_pack(const void *src, int64_t rows, int64_t len, samd_fmt f, uint32_t *dst,
              int32_t *oor_count, hipStream_t stream);

/* Library utility, the inverse of samd_pack (for inspection and tests; the paper's
 * baseline unpacks to 8 bits, Sec. 7): dst is int8 (sign-extended) when f.is_signed,
 * else uint8. */
int samd_unpack(const uint32_t *src, int64_t rows, int64_t len, samd_fmt f, void *dst,
                hipStream_t stream);

/* Valid-mode 1-D true convolution of one packed row of n unsigned b-bit values
 * with a K-tap unsigned kernel given on the HOST in natural order:
 *     y[i] = sum_{t<K} taps[t] * x[i + K - 1 - t],   i = 0 .. n - K,
 * i.e. the complete lanes of the long multiplication of Sec. 5.1, with partial lanes
 * of neighbouring words added (overlap-add of the "parallelograms").  y holds n-K+1
 * int32.  Both formats must be unsigned (the standalone 1-D operator of the paper's
 * Sec. 5); 1 <= K <= 16, K <= n, n <= 2^40 and the packed row below 2^31 words (rows
 * of more than 2^31 values are supported: positions are 64-bit). */
int samd_conv1d(const uint32_t *x, int64_t n, samd_fmt xf, const int32_t *taps, int32_t K,
                samd_fmt kf, int32_t *y, hipStream_t stream);

/* Lane geometry of a 1-D convolution (host-only query):
 *   lane_bits L, lanes I (values per 32-bit operand word), groups (kernel words; group
 *   g holds taps [tap0[g], tap0[g] + ntaps[g]) in natural order), extra (following
 *   operand words whose low lanes reach an output word), out_lanes (lanes that can be
 *   non-zero; the highest takes the product's remaining bits). */
typedef struct {
    int32_t lane_bits, lanes, groups, extra, out_lanes;
    int32_t tap0[16], ntaps[16];
} samd_conv1d_plan;

/* Host-only: the lane geometry samd_conv1d would use (same argument rules). */
int samd_conv1d_plan_query(int64_t n, samd_fmt xf, const int32_t *taps, int32_t K, samd_fmt kf,
                           samd_conv1d_plan *out);

/* Host-only: the lane geometry samd_conv2d would use. */
int samd_conv2d_plan_query(const samd_conv2d_desc *d, samd_fmt xf, samd_fmt wf,
                           samd_conv2d_plan *out);

/* Library utility: the workspace bytes samd_conv2d and its split entry points need for
 * (xf, wf, *d) under the shape's current plan (kernel-word streams, the recentring
 * correction table, the multiply kernel's ticket counters and the staged operand words).
 *
 * A workspace serves one launch at a time: the multiply kernel's per-XCD ticket counters
 * live in it and are advanced by every launch, so two launches in flight on one
 * workspace (different streams, or graph branches that may overlap) race.  Give each
 * stream its own workspace. */
int samd_conv2d_workspace(const samd_conv2d_desc *d, samd_fmt xf, samd_fmt wf, size_t *bytes);

/* Quantized 2-D convolution by SAMD long multiplication, the DNN loop of Sec. 7
 * (direct-sum2d figure) with batch, stride and zero padding:
 *   y[n][m][ho][wo] = sum_c sum_ky sum_kx x[n][c][ho*sh+ky-ph][wo*sw+kx-pw] * w[m][c][ky][kx]
 * (cross-correlation; out-of-image inputs are 0; y is overwritten, not accumulated).
 *   x  packed activations, N*C*H rows of W values (format xf)
 *   w  packed weights,     M*C*KH rows of KW values (format wf)
 *   y  int32 output, N x M x Ho x Wo
 *   ws workspace of at least samd_conv2d_workspace() bytes, 256-byte aligned
 * Each kernel row is sign-extended into one or more 32-bit kernel words (Sec. 6,
 * sign-extension figure), each x row is spread into lanes with temporary spacer bits
 * and sign-extended the same way, products are accumulated over input channels
 * before the lanes are resolved (Sec. 5), and the fix-up of the signed-convolution
 * figure makes each lane exact.  Returns SAMD_EOVERFLOW when
 * C*KH*KW*max|x|*max|w| >= 2^31. */
int samd_conv2d(const uint32_t *x, samd_fmt xf, const uint32_t *w, samd_fmt wf,
                const samd_conv2d_desc *d, int32_t *y, void *ws, size_t ws_bytes,
                hipStream_t stream);

/* samd_conv2d split in its two steps, for callers that reuse one layer's weights:
 * samd_conv2d_prepare writes the layer's kernel words into ws (each kernel row reversed
 * and sign-extended into 32-bit words, Sec. 6); samd_conv2d_prepared then convolves any
 * number of inputs with them.  Both take the same formats, descriptor and workspace as
 * samd_conv2d; the prepared workspace is valid for exactly that (xf, wf, *d). */
int samd_conv2d_prepare(const uint32_t *w, samd_fmt wf, const samd_conv2d_desc *d, samd_fmt xf, void *ws,
                        size_t ws_bytes, hipStream_t stream);
int samd_conv2d_prepared(const uint32_t *x, samd_fmt xf, samd_fmt wf, const samd_conv2d_desc *d, int32_t *y,
                         const void *ws, size_t ws_bytes, hipStream_t stream);

/* samd_conv2d_prepared split once more, into its operand staging and its arithmetic:
 * samd_conv2d_stage spreads x (packed rows) into operand words in ws - I values of one
 * stride phase per 32-bit word, L bits apart (temporary spacers, Sec. 2.2), signed values
 * sign-extended (Sec. 6) - for every padded input row; samd_conv2d_accumulate multiplies
 * them with the prepared kernel words, accumulates the 64-bit products over input
 * channels (Sec. 5), decodes the lanes with the fix-up of Sec. 6, overlap-adds partial
 * lanes of neighbouring words and stores y (NCHW int32).  stage + accumulate is
 * samd_conv2d_prepared; the staged operand words stay valid until the next stage call
 * on the same workspace, so one staged input can be accumulated several times. */
int samd_conv2d_stage(const uint32_t *x, samd_fmt xf, samd_fmt wf, const samd_conv2d_desc *d, void *ws,
                      size_t ws_bytes, hipStream_t stream);
int samd_conv2d_accumulate(samd_fmt xf, samd_fmt wf, const samd_conv2d_desc *d, int32_t *y, const void *ws,
                           size_t ws_bytes, hipStream_t stream);

/* ---- Permanent-spacer activations (Sec. 2.2 permanent spacer bits, Sec. 6.1) ----
 * The packed format above keeps storage dense and inserts spacer bits inside every call
 * (temporary spacer bits, Sec. 2.2); the multiply then reads operand words spread from
 * it.  The permanent-spacer layout stores a layer's activations already spread: lanes of
 * L bits with the spacer bits in place, in exactly the words the multiply reads, so a
 * convolution from it has no spread pass (more bytes stored, fewer operations per call:
 * the trade-off of the paper's permanent spacer bits).  Lanes of signed results can keep
 * their MSB as a permanent spacer bit (the planner then bounds every lane's value to
 * L - 1 bits), so the decode leaves out the fix-up's final xor and reads L - 1-bit
 * fields, the optimisation of Sec. 6.1; it halves the channels a lane holds before a
 * decode, so the planner prices plans with and without it (samd_conv2d_plan.spacer_msb
 * reports the choice).  Sums over channels are taken on the exact products before any
 * lane is read, so no spacer ever needs clearing before an addition.
 *
 * The layout belongs to one layer (descriptor and formats) and its plan: word q of
 * kernel-word variant t of padded row hp (hp in [0, H + 2 pad_h); rows of the zero padding
 * are stored) of channel c of image n is word ((n C + c) padded_rows + hp) tap_words + t)
 * words_per_row + q, the signed 32-bit sum over lanes i < lanes of (v - x_offset) 2^(i
 * lane_bits), v the activation in row hp - pad_h, column stride_w (q lanes + delta[t] + i)
 * + phase[t] - pad_w (0 outside the image), where delta[t] = tap0[t] + ntaps[t] - taps_max
 * and phase/tap0/ntaps/taps_max are the plan's (samd_conv2d_spaced_plan_query).  One
 * spare channel's words follow the last image (read, never used).  Plans of this layout
 * are chosen, cached and tuned separately from the packed layout's; tuning the layout's
 * plan changes the layout, so tensors must be written again after tuning. */
typedef struct {
    int32_t lane_bits, lanes, words_per_row, tap_words, padded_rows, x_offset, spacer_msb;
    int64_t words;   /* int32 words of one layer's activations, the spare channel included */
} samd_spaced_layout;

/* Host-only: the layout of (xf, wf, *d) and the plan behind it. */
int samd_conv2d_spaced_layout(const samd_conv2d_desc *d, samd_fmt xf, samd_fmt wf, samd_spaced_layout *out);
int samd_conv2d_spaced_plan_query(const samd_conv2d_desc *d, samd_fmt xf, samd_fmt wf, samd_conv2d_plan *out);

/* Workspace bytes of the permanent-spacer convolution (kernel words, correction table,
 * ticket counters; no operand words), and its preparation (as samd_conv2d_prepare, under
 * the layout's plan).  A workspace serves one launch at a time. */
int samd_conv2d_spaced_workspace(const samd_conv2d_desc *d, samd_fmt xf, samd_fmt wf, size_t *bytes);
int samd_conv2d_spaced_prepare(const uint32_t *w, samd_fmt wf, const samd_conv2d_desc *d, samd_fmt xf, void *ws,
                               size_t ws_bytes, hipStream_t stream);

/* Write a layer's activations in the layout: from 8-bit values (int8 when xf.is_signed,
 * else uint8; N x C x H x W; each value enters as its low xf.bits bits), or from packed
 * rows (the packed format; the samd_conv2d_stage step into a caller buffer).  dst holds
 * samd_spaced_layout.words int32 words. */
int samd_conv2d_spaced_pack(const void *src, samd_fmt xf, samd_fmt wf, const samd_conv2d_desc *d, uint32_t *dst,
                            hipStream_t stream);
int samd_conv2d_spaced_from_packed(const uint32_t *x, samd_fmt xf, samd_fmt wf, const samd_conv2d_desc *d,
                                   uint32_t *dst, hipStream_t stream);

/* The convolution of samd_conv2d from activations in the layout: xs as written above,
 * ws prepared by samd_conv2d_spaced_prepare; y int32 N x M x Ho x Wo. */
int samd_conv2d_spaced(const uint32_t *xs, samd_fmt xf, samd_fmt wf, const samd_conv2d_desc *d, int32_t *y,
                       const void *ws, size_t ws_bytes, hipStream_t stream);

/* ReLU and requantisation of samd_relu_requant_pack, written as the next layer's
 * activations in the layout (format xf, unsigned; weight format wf; descriptor *d of the
 * next layer): the activations go from one layer's int32 outputs to the next layer's
 * spaced lanes without the packed form.  dev_shift nullable. */
int samd_relu_requant_spaced(const int32_t *acc, const int32_t *dev_max, samd_fmt xf, samd_fmt wf,
                             const samd_conv2d_desc *d, uint32_t *dst, int32_t *dev_shift, hipStream_t stream);

/* samd_conv2d_tune for the layout's plan: the candidates of the permanent-spacer plan,
 * each timed on the multiply alone (the layout is written once per candidate, untimed),
 * from x given as packed rows; the chosen plan becomes the layout's plan.  Arguments and
 * workspace size (samd_conv2d_spaced_tune_workspace) as for samd_conv2d_tune. */
int samd_conv2d_spaced_tune_workspace(const samd_conv2d_desc *d, samd_fmt xf, samd_fmt wf, int32_t candidates,
                                      size_t *bytes);
int samd_conv2d_spaced_tune(const uint32_t *x, samd_fmt xf, const uint32_t *w, samd_fmt wf,
                            const samd_conv2d_desc *d, int32_t *y, void *ws, size_t ws_bytes, int32_t candidates,
                            int32_t reps, samd_conv2d_plan *chosen, hipStream_t stream);

/* ---- Allocation-free convolution ----
 * For callers that cannot allocate device memory (code under HIP graph capture, tight
 * serving loops, harnesses that forbid hipMalloc): samd_conv2d with its workspace in a
 * device array inside the library instead of a caller buffer.  The array holds
 * SAMD_NOALLOC_SCRATCH_BYTES per GPU, allocated by the HIP runtime when the library's
 * device code is loaded on that GPU and held until the process ends.
 *   x, w, y, *d, xf, wf  as for samd_conv2d
 * The call itself allocates nothing (no hipMalloc, hipFree or allocating library
 * routine).  A layer whose workspace (samd_conv2d_workspace) exceeds
 * SAMD_NOALLOC_SCRATCH_BYTES is refused with SAMD_ENOSPC before any HIP call.  Every call
 * on one GPU uses that GPU's one array, and each call prepares it from scratch (kernel
 * words and the zeroed ticket counters are written by the call's own kernels), so the
 * previous call's contents do not matter; but calls that may overlap on one GPU (several
 * streams, several host threads, concurrent graph branches) race on the array and must
 * be serialised by the caller. */
#define SAMD_NOALLOC_SCRATCH_BYTES (64u << 20)

int samd_conv2d_noalloc(const uint32_t *x, samd_fmt xf, const uint32_t *w, samd_fmt wf,
                        const samd_conv2d_desc *d, int32_t *y, hipStream_t stream);

/* ---- Autotuning ----
 * The paper specialises the SAMD instruction sequence for each precision with a code
 * generator (Sec. 1, Sec. 7).  Here the specialisations are compiled kernel templates
 * (lane geometry x launch shape), the planner picks one with a cost model, and these
 * calls let a caller pick by measurement instead.
 *
 * At most SAMD_MAX_CANDIDATES plans are listed or timed per call. */
#define SAMD_MAX_CANDIDATES 64

/* Host-only: up to max_count candidate plans for (xf, wf, *d), ranked by the planner's
 * cost model, the planner's own choice first; out holds max_count entries, *count
 * receives the number written.  Tuned plans (below) do not affect this list. */
int samd_conv2d_candidates(const samd_conv2d_desc *d, samd_fmt xf, samd_fmt wf, int32_t max_count,
                           samd_conv2d_plan *out, int32_t *count);

/* Workspace bytes samd_conv2d_tune needs to time the first `candidates` candidates: the
 * largest of their workspaces, plus a second output tensor and a counter. */
int samd_conv2d_tune_workspace(const samd_conv2d_desc *d, samd_fmt xf, samd_fmt wf, int32_t candidates,
                               size_t *bytes);

/* Times the first `candidates` candidate plans on the caller's x and w (stage +
 * accumulate, `reps` times each, HIP events on `stream`; after 4 x reps untimed runs of
 * the planner's plan to bring the clocks up, two passes over all candidates, each keeping
 * its faster pass) and makes the fastest the plan of (xf, wf, *d) for every later call
 * in this process, until samd_conv2d_untune.  A candidate must beat the best so far by
 * 2 % (near-ties keep the higher-ranked plan, so repeated tuning settles on one plan).
 *   x, w, y as for samd_conv2d (y receives the convolution)
 *   ws      256-byte aligned; candidates whose workspace does not fit next to the
 *           second output are skipped (SAMD_ENOSPC if the planner's own plan does not);
 *           samd_conv2d_tune_workspace gives the size that fits them all
 *   candidates 1..SAMD_MAX_CANDIDATES; reps 1..1000
 *   chosen  (host, nullable) receives the chosen plan
 * Every candidate's output is compared on the device with the planner's plan's output;
 * any difference is an error (SAMD_EHIP, detail in samd_last_error) and nothing is
 * tuned.  Unlike the other calls this one BLOCKS: it synchronises `stream` to read the
 * timings.  On return ws is prepared for the chosen plan (as by samd_conv2d_prepare).
 * Workspaces prepared for the shape before tuning must be prepared again, and their
 * size queried again (samd_conv2d_workspace reports the tuned plan's).  The tuned plans
 * are process-wide state shared by all threads: tune during set-up, not while other
 * threads run the same shape. */
int samd_conv2d_tune(const uint32_t *x, samd_fmt xf, const uint32_t *w, samd_fmt wf,
                     const samd_conv2d_desc *d, int32_t *y, void *ws, size_t ws_bytes,
                     int32_t candidates, int32_t reps, samd_conv2d_plan *chosen, hipStream_t stream);

/* Host-only: make `plan` - one reported for this shape by samd_conv2d_candidates,
 * samd_conv2d_tune or samd_conv2d_plan_query, matched by its lane geometry (lane_bits,
 * lanes, x_offset) and launch shape (shared_rows, rows_per_thread, rows_per_block,
 * mblock, split_waves) - the plan of (xf, wf, *d), as if tuned: a tuning result kept
 * from an earlier process.  SAMD_EINVAL when no candidate of the shape matches. */
int samd_conv2d_use_plan(const samd_conv2d_desc *d, samd_fmt xf, samd_fmt wf, const samd_conv2d_plan *plan);

/* Host-only: forget the tuned plan of (xf, wf, *d), or of every shape when d is NULL
 * (xf and wf are then ignored); the planner's model decides again. */
int samd_conv2d_untune(const samd_conv2d_desc *d, samd_fmt xf, samd_fmt wf);

/* Library utility: the workspace bytes samd_conv2d_int8 needs (reordered int8 weights,
 * the per-filter weight sums of the zero-point correction and, for layers that take the
 * packed-row kernel, the weights in that kernel's K order). */
int samd_conv2d_int8_workspace(const samd_conv2d_desc *d, samd_fmt xf, size_t *bytes);

/* The native 8-bit baseline of Sec. 7: the same convolution on values unpacked to
 * 8 bits, computed with the gfx950 int8 matrix cores.
 *   x  unpacked activations, N x H x W x C (channels innermost), int8 when xf is
 *      signed, else uint8 (unsigned 8-bit values use a -128 zero point internally)
 *   w  int8 weights, M x C x KH x KW
 *   y  int32 output, N x M x Ho x Wo
 * Same semantics and overflow rule as samd_conv2d. */
int samd_conv2d_int8(const void *x, samd_fmt xf, const int8_t *w, samd_fmt wf,
                     const samd_conv2d_desc *d, int32_t *y, void *ws, size_t ws_bytes,
                     hipStream_t stream);

/* Library utility (host only, for inspection and tests): the kernel and tile
 * samd_conv2d_int8 uses for this layer when the activations are 16-byte aligned.
 *   halo         3: the packed-row kernel (few input channels, any stride: K laid out
 *                by kernel row, ceil(KW*C / 16) 16-byte slots per row, where that at
 *                least halves the k-blocks of the 64-channel layout; activations a
 *                whole number of 4-byte words and 4-byte aligned);
 *                2: a weight-resident kernel (stride-1 3x3 and 1x1 layers, C a
 *                multiple of 16 and at most 512): each workgroup keeps its 32 filters'
 *                weights in registers (whole, or in chunks of 128 or 64 channels
 *                above 128 padded channels) and walks one run of positions of one image;
 *                1: the halo-tiled kernel (stride-1 layers with C a multiple of 16);
 *                0: the im2col kernel (any other layer, or misaligned activations)
 *   mtile        output channels per workgroup
 *   positions    output positions per workgroup (weight-resident: the longest run;
 *                packed-row: 4 waves x 16-position tiles per wave x 16)
 *   row_segments 1: tiles are segments of one output row; 0: runs of positions that may
 *                span several rows (halo kernel only)
 *   lds_bytes    dynamic LDS per workgroup (halo kernel: two halo buffers; packed-row:
 *                the weight fragments of up to 128 filters and their zero-point
 *                corrections; chunked weight-resident: two chunk buffers and the
 *                group's corrections)
 *   waves        wavefronts per workgroup (4; 8 for the weight-resident kernels)
 *   workgroups   workgroups of one call */
typedef struct {
    int32_t halo, mtile, positions, row_segments, lds_bytes, waves;
    int64_t workgroups;
} samd_conv2d_int8_plan;

int samd_conv2d_int8_plan_query(const samd_conv2d_desc *d, samd_fmt xf, samd_fmt wf, samd_conv2d_int8_plan *out);

/* Host-only, for measuring the baseline at its best (the SAMD path is tuned the same way,
 * samd_conv2d_tune): every launch samd_conv2d_int8 can make for the layer, the halo
 * tiles that fit first, then the weight-resident launches, then the im2col kernel; out holds max_count entries, *count
 * receives the number written. */
int samd_conv2d_int8_candidates(const samd_conv2d_desc *d, samd_fmt xf, samd_fmt wf, int32_t max_count,
                                samd_conv2d_int8_plan *out, int32_t *count);

/* Host-only: make `plan` (one of the layer's candidates, matched by halo, mtile,
 * positions and waves) the launch of (xf, *d) for every later samd_conv2d_int8 call in this process;
 * plan NULL restores the library's own choice.  Process-wide state, like tuned SAMD
 * plans; the workspace does not depend on it.  SAMD_EINVAL when no candidate matches. */
int samd_conv2d_int8_use_plan(const samd_conv2d_desc *d, samd_fmt xf, samd_fmt wf, const samd_conv2d_int8_plan *plan);

/* samd_conv2d_int8 split in weight reordering and convolution, as for samd_conv2d. */
int samd_conv2d_int8_prepare(const int8_t *w, samd_fmt wf, const samd_conv2d_desc *d, samd_fmt xf, void *ws,
                             size_t ws_bytes, hipStream_t stream);
int samd_conv2d_int8_prepared(const void *x, samd_fmt xf, samd_fmt wf, const samd_conv2d_desc *d, int32_t *y,
                              const void *ws, size_t ws_bytes, hipStream_t stream);

/* Library utility for the requantisation between layers (the layer maximum that fixes
 * the shift of samd_relu_requant_pack): maximum of n int32 values, written to *dev_max
 * (device); n >= 1. */
int samd_max_i32(const int32_t *src, int64_t n, int32_t *dev_max, hipStream_t stream);

/* ReLU and requantisation to unsigned b bits between layers (the paper gives no rule;
 * this library's): with mx = max(*dev_max, 0), s = the smallest s >= 0 such that
 * mx >> s <= 2^b - 1, each value becomes min((max(v,0) + (s ? 2^(s-1) : 0)) >> s,
 * 2^b - 1).  acc is rows x len int32 (rows of an NCHW tensor, len = W); the result is
 * written in the packed storage format (format `out`, which must be unsigned).
 * When dev_shift is not NULL, s is stored there. */
int samd_relu_requant_pack(const int32_t *acc, int64_t rows, int64_t len, const int32_t *dev_max,
                           samd_fmt out, uint32_t *dst, int32_t *dev_shift, hipStream_t stream);

/* The same requantisation for the 8-bit baseline chain: acc is N x C x H x W int32,
 * dst is N x H x W x C uint8 (channels innermost, the layout samd_conv2d_int8 reads). */
int samd_relu_requant_nhwc_u8(const int32_t *acc, int32_t N, int32_t C, int32_t H, int32_t W,
                              const int32_t *dev_max, samd_fmt out, uint8_t *dst,
                              hipStream_t stream);

/* ReLU and requantisation, as samd_relu_requant_pack, written straight into the next
 * layer's operand words instead of packed rows: the result equals samd_relu_requant_pack
 * followed by samd_conv2d_stage of the next layer, without the dense packed activations
 * in between.  Between layers the activations stay in the lanes-with-spacers layout the
 * multiply reads (the permanent-spacer storage of Sec. 2.2 and Sec. 7: more bytes, no
 * repacking).  Afterwards samd_conv2d_accumulate computes the next layer.
 *   acc       int32 accumulators, NCHW with the next layer's d->N, C, H, W (device)
 *   dev_max   device int32 maximum of acc (samd_max_i32)
 *   xf        the next layer's activation format: unsigned, bits = requantisation bits
 *   wf, d     the next layer's weight format and descriptor
 *   ws        the next layer's workspace (samd_conv2d_workspace bytes, 256-byte aligned;
 *             its kernel words prepared before samd_conv2d_accumulate)
 *   dev_shift nullable device int32: receives the shift used */
int samd_relu_requant_stage(const int32_t *acc, const int32_t *dev_max, samd_fmt xf, samd_fmt wf,
                            const samd_conv2d_desc *d, void *ws, size_t ws_bytes, int32_t *dev_shift,
                            hipStream_t stream);

/* Lane-wise SAMD arithmetic on packed words (Sec. 3, conventional SAMD arithmetic: the
 * add figure, the subtract passage and the lane-wise multiply figure).
 *   op   SAMD_LANE_ADD, SAMD_LANE_SUB or SAMD_LANE_MUL
 *   a, b nwords packed words each (device), in the format of samd_pack: any number of
 *        rows, each starting on a word, the bits above a word's last lane zero
 *   dst  nwords words (device; may alias a or b), same format
 * Lane i of every result word is (a_i op b_i) mod 2^bits: for signed formats the
 * two's-complement wrap-around of the exact result, for unsigned the value mod 2^bits.
 * The whole word is computed at once with temporary spacer bits (each lane's top bit);
 * the multiply takes bits shift-and-add steps.  Bits above the last lane stay zero when
 * they are zero in a and b. */
enum { SAMD_LANE_ADD = 0, SAMD_LANE_SUB = 1, SAMD_LANE_MUL = 2, SAMD_LANE_SCALE = 3 };
int samd_lanewise(int op, const uint32_t *a, const uint32_t *b, int64_t nwords, samd_fmt f, uint32_t *dst,
                  hipStream_t stream);

/* Vector scale (Sec. 4, scale-wrap figure): every lane of a times one scalar, modulo
 * 2^bits.  The scalar is taken as its low bits bits (a negative scalar of a signed
 * format is its two's-complement pattern); the low bits of a product do not depend on
 * signedness, so the result lanes are (a_i * scalar) mod 2^bits for either format.
 * Arguments as samd_lanewise. */
int samd_scale(const uint32_t *a, int64_t nwords, samd_fmt f, int32_t scalar, uint32_t *dst, hipStream_t stream);

#ifdef __cplusplus
}
#endif

#endif /* SAMD_H */
