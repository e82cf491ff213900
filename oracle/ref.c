/*
 * CPU oracle for the SAMD quantized-convolution path.
 *
 * TEST INFRASTRUCTURE ONLY.  This file is the plain, slow, obviously correct
 * definition of every result the GPU library computes.  Only tests/, the smoke
 * check and the benchmark's CPU-baseline leg may load it; the GPU library shares no
 * code with it.  Everything is exact integer arithmetic in int64.
 *
 * Paper: Anderson, Doyle, Gregg, "Scalar Arithmetic Multiple Data: Customizable
 * Precision for Deep Neural Networks" (arXiv 1809.10572).
 */
#include <stdint.h>
#include <stddef.h>
#ifdef _OPENMP
#include <omp.h>
#endif

/* ---------------------------------------------------------------------------
 * Packed storage format.
 *
 * The paper keeps storage dense and creates spacer bits only inside a routine
 * (temporary spacer bits, Sec. 2.2).  The storage layout itself is not fixed by
 * the paper; this is the library's definition:
 *   a row of `len` b-bit values (1 <= b <= 8) occupies ceil(len / P) uint32 words,
 *   P = floor(32 / b); value j lies in bits [(j mod P)*b, (j mod P)*b + b) of word
 *   floor(j / P), as a b-bit two's-complement field if signed, unsigned otherwise;
 *   bits above P*b in a word, and fields past the row end, are zero.  Every row
 *   starts on a new word.
 * ------------------------------------------------------------------------- */

int64_t orc_row_words(int64_t len, int bits)
{
    int64_t per = 32 / bits;
    return (len + per - 1) / per;
}

/* Returns the number of values outside the b-bit range; such values are stored
 * as their low b bits. */
int64_t orc_pack(const int32_t *vals, int64_t rows, int64_t len, int bits, int is_signed,
                 uint32_t *dst)
{
    int64_t per = 32 / bits, words = orc_row_words(len, bits), bad = 0;
    int64_t lo = is_signed ? -((int64_t)1 << (bits - 1)) : 0;
    int64_t hi = is_signed ? ((int64_t)1 << (bits - 1)) - 1 : ((int64_t)1 << bits) - 1;
    uint32_t field_mask = (uint32_t)(((uint64_t)1 << bits) - 1);
    for (int64_t r = 0; r < rows; ++r) {
        for (int64_t q = 0; q < words; ++q)
            dst[r * words + q] = 0;
        for (int64_t j = 0; j < len; ++j) {
            int64_t v = vals[r * len + j];
            if (v < lo || v > hi)
                ++bad;
            uint32_t f = (uint32_t)v & field_mask;
            dst[r * words + j / per] |= f << ((j % per) * bits);
        }
    }
    return bad;
}

void orc_unpack(const uint32_t *src, int64_t rows, int64_t len, int bits, int is_signed,
                int32_t *vals)
{
    int64_t per = 32 / bits, words = orc_row_words(len, bits);
    uint32_t field_mask = (uint32_t)(((uint64_t)1 << bits) - 1);
    for (int64_t r = 0; r < rows; ++r)
        for (int64_t j = 0; j < len; ++j) {
            uint32_t f = (src[r * words + j / per] >> ((j % per) * bits)) & field_mask;
            int64_t v = f;
            if (is_signed && (f >> (bits - 1)))
                v -= (int64_t)1 << bits;
            vals[r * len + j] = (int32_t)v;
        }
}

/* ---------------------------------------------------------------------------
 * 1-D convolution, valid part only (Sec. 5: the polynomial product computed by
 * convolution; the complete lanes of the long multiplication are the outputs in
 * which every kernel tap meets an input).  True convolution, kernel in natural
 * order:  y[i] = sum_t k[t] * x[i + K - 1 - t],  i = 0 .. n - K.
 * ------------------------------------------------------------------------- */
void orc_conv1d(const int64_t *x, int64_t n, const int64_t *k, int K, int64_t *y)
{
    for (int64_t i = 0; i + K <= n; ++i) {
        int64_t s = 0;
        for (int t = 0; t < K; ++t)
            s += k[t] * x[i + K - 1 - t];
        y[i] = s;
    }
}

/* ---------------------------------------------------------------------------
 * 2-D convolution as the DNN loop computes it (Sec. 7, direct-sum2d figure):
 * a cross-correlation summed over input channels,
 *   y[n][m][ho][wo] = sum_c sum_ky sum_kx x[n][c][ho*sh + ky - ph][wo*sw + kx - pw]
 *                                          * w[m][c][ky][kx],
 * extended with a batch dimension, stride and zero padding (an input position
 * outside the image contributes 0).  The output starts at zero.
 * desc = {N, C, H, W, M, KH, KW, stride_h, stride_w, pad_h, pad_w};
 * Ho = (H + 2 ph - KH) / sh + 1,  Wo = (W + 2 pw - KW) / sw + 1.
 * ------------------------------------------------------------------------- */
static void out_size(const int32_t *d, int64_t *Ho, int64_t *Wo)
{
    *Ho = ((int64_t)d[2] + 2 * d[9] - d[5]) / d[7] + 1;
    *Wo = ((int64_t)d[3] + 2 * d[10] - d[6]) / d[8] + 1;
}

void orc_conv2d(const int32_t *x, const int32_t *w, const int32_t *d, int64_t *y)
{
    int64_t N = d[0], C = d[1], H = d[2], W = d[3], M = d[4], KH = d[5], KW = d[6];
    int64_t sh = d[7], sw = d[8], ph = d[9], pw = d[10], Ho, Wo;
    out_size(d, &Ho, &Wo);
#pragma omp parallel for collapse(2) schedule(dynamic)
    for (int64_t n = 0; n < N; ++n)
        for (int64_t m = 0; m < M; ++m) {
            int64_t *out = y + (n * M + m) * Ho * Wo;
            for (int64_t p = 0; p < Ho * Wo; ++p)
                out[p] = 0;
            /* The sum is reordered only as integer addition allows: for each weight,
             * add its products into every output position. */
            for (int64_t c = 0; c < C; ++c)
                for (int64_t ky = 0; ky < KH; ++ky)
                    for (int64_t kx = 0; kx < KW; ++kx) {
                        int64_t wv = w[((m * C + c) * KH + ky) * KW + kx];
                        for (int64_t ho = 0; ho < Ho; ++ho) {
                            int64_t hi = ho * sh + ky - ph;
                            if (hi < 0 || hi >= H)
                                continue;
                            const int32_t *row = x + ((n * C + c) * H + hi) * W;
                            for (int64_t wo = 0; wo < Wo; ++wo) {
                                int64_t wi = wo * sw + kx - pw;
                                if (wi >= 0 && wi < W)
                                    out[ho * Wo + wo] += (int64_t)row[wi] * wv;
                            }
                        }
                    }
        }
}

/* One output of the same definition, for sampled checks at full size. */
int64_t orc_conv2d_point(const int32_t *x, const int32_t *w, const int32_t *d,
                         int64_t n, int64_t m, int64_t ho, int64_t wo)
{
    int64_t C = d[1], H = d[2], W = d[3], KH = d[5], KW = d[6];
    int64_t s = 0;
    for (int64_t c = 0; c < C; ++c)
        for (int64_t ky = 0; ky < KH; ++ky)
            for (int64_t kx = 0; kx < KW; ++kx) {
                int64_t hi = ho * d[7] + ky - d[9], wi = wo * d[8] + kx - d[10];
                if (hi < 0 || hi >= H || wi < 0 || wi >= W)
                    continue;
                s += (int64_t)x[((n * C + c) * H + hi) * W + wi] *
                     w[((m * C + c) * KH + ky) * KW + kx];
            }
    return s;
}

/* ---------------------------------------------------------------------------
 * ReLU + requantisation to unsigned b bits between the layers of the
 * AlexNet-shaped stack.  The paper gives no requantisation rule; this is the
 * library's definition, integer-only:
 *   r = max(acc, 0);  s = the smallest s >= 0 with (max over the layer of r) >> s
 *   <= 2^b - 1;  q = min((r + (s > 0 ? 2^(s-1) : 0)) >> s, 2^b - 1)
 * (round half up, then clamp).
 * ------------------------------------------------------------------------- */
int orc_requant_shift(const int64_t *acc, int64_t count, int bits)
{
    int64_t mx = 0;
    for (int64_t i = 0; i < count; ++i)
        if (acc[i] > mx)
            mx = acc[i];
    int s = 0;
    while ((mx >> s) > ((int64_t)1 << bits) - 1)
        ++s;
    return s;
}

void orc_relu_requant(const int64_t *acc, int64_t count, int shift, int bits, int32_t *q)
{
    int64_t top = ((int64_t)1 << bits) - 1;
    int64_t half = shift > 0 ? (int64_t)1 << (shift - 1) : 0;
#pragma omp parallel for schedule(static)
    for (int64_t i = 0; i < count; ++i) {
        int64_t r = acc[i] > 0 ? acc[i] : 0;
        int64_t v = (r + half) >> shift;
        q[i] = (int32_t)(v < top ? v : top);
    }
}

int orc_threads(void)
{
#ifdef _OPENMP
    return omp_get_max_threads();
#else
    return 1;
#endif
}
