// Host-side lane-geometry planning for the SAMD convolutions.  Pure C++: no HIP calls,
// so it runs (and is tested) without a GPU.
//
// The paper sizes lanes so that no lane can overflow into its neighbour (Sec. 5.1:
// a K-term sum of b x b-bit products needs 2b + log2 K bits) and keeps one bit of
// margin in signed lanes for the borrow a negative lane hands to the lane above it
// (Sec. 6).  Here the bound is computed exactly, per lane, for the products actually
// accumulated into it before the lanes are decoded, and the planner picks among the
// exact geometries the one with the lowest modelled cost.
#include <algorithm>
#include <cmath>
#include <cstdio>
#include <array>
#include <limits>
#include <functional>
#include <map>
#include <mutex>
#include <vector>

#include "samd_internal.hpp"

namespace samd {

namespace {

typedef __int128 i128;

i128 pow2(int e) { return (i128)1 << e; }

// Range of a b-bit value.
void value_range(int bits, bool is_signed, i128 &lo, i128 &hi) {
    lo = is_signed ? -pow2(bits - 1) : 0;
    hi = is_signed ? pow2(bits - 1) - 1 : pow2(bits) - 1;
}

i128 max_abs(int bits, bool is_signed) { return is_signed ? pow2(bits - 1) : pow2(bits) - 1; }

// Does sum_{i<n} v_i 2^(i L) stay inside [lo_lim, hi_lim] for every b-bit v_i?
bool word_fits(int bits, bool is_signed, int L, int n, i128 lo_lim, i128 hi_lim) {
    if ((n - 1) * L + bits > 64) return false;
    i128 lo, hi, place = 0;
    value_range(bits, is_signed, lo, hi);
    for (int i = 0; i < n; ++i) place += pow2(i * L);
    return lo * place >= lo_lim && hi * place <= hi_lim;
}

const i128 kI32Min = -pow2(31), kI32Max = pow2(31) - 1;
const i128 kI64Max = pow2(63) - 1;

// Products of an I-value word and a k-tap word that land in lane j.
int pairs_in_lane(int j, int I, int k) {
    if (j < 0 || j > I + k - 2) return 0;
    return std::min(std::min(j + 1, k), std::min(I, I + k - 1 - j));
}

// Split `count` consecutive taps into ceil(count / kmax) near-equal groups; false (and
// nothing written) when that is more than kMaxTapWords groups.
bool split_taps(int count, int kmax, int *t0, int *nt, int &ngroups) {
    ngroups = (count + kmax - 1) / kmax;
    if (ngroups > kMaxTapWords) return false;
    int base = count / ngroups, extra = count % ngroups, at = 0;
    for (int g = 0; g < ngroups; ++g) {
        nt[g] = base + (g < extra ? 1 : 0);
        t0[g] = at;
        at += nt[g];
    }
    return true;
}

// Index ranges the kernels assume, checked for every plan before it is used or listed:
//  - one image's operand words (and one spare channel) are addressed with 32-bit byte
//    offsets, and padded rows with 32-bit indices;
//  - a wave's slice of the kernel-word stream (cpw channels, plus the padding steps) is
//    indexed with 32-bit word offsets;
//  - the operand spread and the fused epilogue give every padded row 2^q threads in one
//    launch of fewer than 2^32 threads.
bool addressable(const samd_conv2d_desc &d, const Conv2dGeom &g) {
    const int64_t two31 = (int64_t)1 << 31;
    const int64_t rows = (int64_t)d.N * d.C * g.Hp;
    const int rpb = 256 >> spread_qshift(g.nq);
    return (int64_t)(d.C + 1) * g.Hp * g.ntw * g.nq * 4 < two31 && rows < two31 &&
           ((int64_t)g.cpw * g.nrt + kStreamPad) * kWaveM < two31 &&
           (rows + rpb - 1) / rpb * 256 <= (int64_t)0xffffffff;
}

// Launch shape of one lane geometry: output rows per thread (rh), row groups per wave,
// output-channel waves (wm) and channel-slice waves (ks) per workgroup, and whether the
// lane's rows share operand loads (3-row, stride-1 kernels).  Every candidate is priced
// in issue cycles of one compute unit (units of 4 clocks): its SIMDs' multiply-adds and
// decodes, and its texture path's operand loads (about 12 clocks per wave-wide load on
// MI355X, shared by the 4 SIMDs), whichever binds, divided by an issue efficiency that
// grows with the waves resident per SIMD (latency hiding), plus the last item's drain and
// the operand-spread pass.  Returns false when no tile fits the LDS.  With `all`, every
// launch shape that fits is also appended to it, priced.
bool place_launch(const samd_conv2d_desc &d, Conv2dGeom &c, std::vector<Conv2dGeom> *all, bool &range_limited) {
    const int grp_max = 64 / c.nqs;
    const bool rows_ok = d.KH == 3 && d.stride_h == 1 && (c.ntw == 1 || c.ntw == 2);
    bool found = false;
    Conv2dGeom best = c;
    best.cost = 1e300;
    for (int rows = 0; rows <= (rows_ok ? 1 : 0); ++rows) {
    for (int rh = 1; rh <= (rows ? 4 : 2); ++rh) {
        if (rh > 1 && c.Ho < rh) continue;
        // waves per SIMD the kernel's registers allow (as compiled for gfx950), and at
        // most kResidentWavesPerSimd
        const int reg_waves = std::min(kResidentWavesPerSimd, rh <= 2 ? 7 : (rh == 3 ? 5 : 4));
        for (int gr = grp_max; gr >= 1; --gr) {
            for (int wm : {1, 2, 4}) {
                // at most 8 channel slices: 16-wave workgroups measured 1.0-1.8x slower than
                // 8-wave ones on 512-channel layers (all 16 waves decode into one tile)
                for (int ks : {1, 2, 4, 8}) {
                    if (wm * ks > kMaxBlockWaves) continue;
                    if (ks > 1 && (d.C + ks - 1) / ks < 1) continue;
                    Conv2dGeom t = c;
                    t.rows_path = rows;
                    t.rh = rh;
                    t.groups = gr;
                    t.rows_blk = std::min(rh * gr, c.Ho);
                    t.trows = (t.rows_blk - 1) * d.stride_h + d.KH;
                    t.wm = wm;
                    t.ks = ks;
                    t.mblk = wm * kWaveM;
                    t.nmb = (d.M + t.mblk - 1) / t.mblk;
                    t.tile_rows = gr * rh;
                    // tile row stride: the columns a row needs, padded so that the rows of
                    // neighbouring lane groups start on different LDS banks (row groups are
                    // rh rows apart; their offset mod 32 banks should not be a multiple of
                    // the lane stride I)
                    t.tile_row = c.nqs * c.I + c.Kmax - 1;
                    for (int pad = 0; pad < c.I && c.I > 1; ++pad)
                        if ((rh * (t.tile_row + pad)) % 32 % c.I != 0) {
                            t.tile_row += pad;
                            break;
                        }
                    t.lds_tile = (t.mblk * t.tile_rows * t.tile_row + 3) / 4 * 4;
                    t.lds_words = t.lds_tile;
                    if ((long)t.lds_words * 4 > kMaxLdsBytes) continue;
                    t.cpw = (d.C + ks - 1) / ks;           // channels per slice
                    if (ks > 1 && (long)(ks - 1) * t.cpw >= d.C) continue;   // an empty slice
                    t.chk = t.cpw * ks;
                    t.row_tiles = (c.Ho + t.rows_blk - 1) / t.rows_blk;
                    t.tiles = d.N * t.row_tiles * c.ncs;
                    t.kw_words = (int64_t)t.nmb * wm * ((int64_t)d.C * c.nrt + kStreamPad) * kWaveM;
                    t.spread_words = (int64_t)d.N * d.C * c.Hp * c.ntw * c.nq;
                    if (!addressable(d, t)) {
                        range_limited = true;
                        continue;
                    }

                    // wave-instructions and operand loads of one workgroup's item
                    const double waves = (double)wm * ks;
                    const double nflush = std::ceil((double)t.cpw / c.G);
                    const double mads = waves * kWaveM * rh * t.cpw * c.nrt * 1.08;
                    // fix-up: and, add, xor on 64 bits (6 operations), the xor left out with
                    // a spacer MSB
                    const double decode = waves * nflush * kWaveM * rh *
                                          ((c.result_signed ? (c.spacer ? 3.0 : 5.0) : 0.0) + 1.0 + 2.0 * c.nl);
                    const double fixed = waves * 150.0 + (double)t.lds_tile / 64.0 * 3.0;
                    const double wg = mads + decode + fixed;
                    const double loads = waves * t.cpw * (rows ? c.ntw * (rh + 2.0) : (double)c.nrt * rh);
                    // one compute unit's share of the items (taken as workgroups free up)
                    const double items = std::max(1.0, (double)t.tiles * t.nmb / 256.0);
                    const double valu = items * wg / 4.0;
                    const double tex = items * loads * 3.0;
                    const double busy = std::max(valu, tex) + 0.25 * std::min(valu, tex);
                    // residency: LDS and registers
                    const double res = std::max(1.0, std::min(std::floor(163840.0 / (t.lds_words * 4.0)),
                                                              std::floor(4.0 * reg_waves / waves)));
                    const double occ = std::min(items, res) * waves / 4.0;
                    const double eff = occ / (occ + 0.7);
                    const double drain = 0.5 * wg / waves;
                    const double spread = (double)t.spread_words * (6.0 * c.I + 4.0) / 64.0 / 1024.0;
                    // measured on MI355X: slices of about 32 channels balance the per-wave
                    // fixed costs against scalar-load latency hiding
                    const double slice = 1.0 + 0.15 * std::fabs(std::log2(t.cpw / 32.0));
                    t.cost = (busy / eff + drain) * slice + spread;
                    if (all) all->push_back(t);
                    if (t.cost < best.cost) {
                        best = t;
                        found = true;
                    }
                }
            }
        }
    }
    }
    if (found) {
        const double keep = c.macs_per_mad;
        c = best;
        c.macs_per_mad = keep;
    }
    return found;
}

}  // namespace

namespace {

// xf: the activations as the lanes see them; xoff: the value subtracted from every
// stored activation before it enters a lane (0, or 2^(b-1) for recentred unsigned
// activations, which then behave as signed b-bit values).
// layout: 1 for the permanent-spacer layout (operand words held by the caller).
// msb: lanes of signed results keep their MSB as a spacer bit - their values fit L - 1
// bits - so the decode can leave out the fix-up's final xor (Sec. 6.1); it halves the
// channels a lane holds, so the planner prices both.
int search_lanes(const samd_conv2d_desc &d, samd_fmt xf, samd_fmt wf, int xoff, int layout, int msb,
                 Conv2dGeom &best, std::string &err, std::vector<Conv2dGeom> *all = nullptr) {
    Conv2dGeom g = {};
    g.N = d.N; g.C = d.C; g.H = d.H; g.W = d.W; g.M = d.M; g.KH = d.KH; g.KW = d.KW;
    g.sh = d.stride_h; g.sw = d.stride_w; g.ph = d.pad_h; g.pw = d.pad_w;
    g.Ho = (d.H + 2 * d.pad_h - d.KH) / d.stride_h + 1;
    g.Wo = (d.W + 2 * d.pad_w - d.KW) / d.stride_w + 1;
    g.xbits = xf.bits; g.xsigned = xoff ? 0 : xf.is_signed; g.wbits = wf.bits; g.wsigned = wf.is_signed;
    g.xoff = xoff;
    g.result_signed = (xf.is_signed || wf.is_signed) ? 1 : 0;
    g.layout_spaced = layout ? 1 : 0;
    g.spacer = layout && msb && g.result_signed ? 1 : 0;
    g.xrw = (int32_t)row_words(d.W, xf.bits);
    g.wrw = (int32_t)row_words(d.KW, wf.bits);

    const int S = d.stride_w;
    g.Kmax = (d.KW + S - 1) / S;
    const i128 prod = max_abs(xf.bits, xf.is_signed) * max_abs(wf.bits, wf.is_signed);
    bool found = false, range_limited = false;
    best.cost = 1e300;

    for (int L = 2; L <= 31; ++L) {
        // widest kernel word and input word that stay int32 at this lane width
        int kmax = 0;
        for (int k = 1; k <= g.Kmax; ++k)
            if (word_fits(wf.bits, wf.is_signed, L, k, kI32Min, kI32Max)) kmax = k;
        if (kmax == 0) continue;
        int imax = 0;
        for (int i = 1; i <= kMaxLanes; ++i)
            if (word_fits(xf.bits, xf.is_signed, L, i, kI32Min, kI32Max)) imax = i;
        for (int I = 1; I <= imax; ++I) {
            Conv2dGeom c = g;
            c.L = L;
            c.I = I;
            // kernel words: every stride phase's taps in groups of at most kmax
            c.ntw = 0;
            bool ok = true;
            for (int r = 0; r < S && ok; ++r) {
                int Kr = r < d.KW ? (d.KW - r + S - 1) / S : 0;
                if (Kr == 0) continue;
                int t0[kMaxTapWords], nt[kMaxTapWords], ng;
                if (!split_taps(Kr, kmax, t0, nt, ng)) {
                    ok = false;
                    break;
                }
                for (int q = 0; q < ng; ++q) {
                    if (c.ntw >= kMaxTapWords) { ok = false; break; }
                    c.tw_phase[c.ntw] = r;
                    c.tw_tap0[c.ntw] = t0[q];
                    c.tw_ntaps[c.ntw] = nt[q];
                    ++c.ntw;
                }
            }
            if (!ok) continue;
            // products per lane for one (channel, kernel row)
            if (I + c.Kmax - 1 > kMaxOutLanes) continue;
            int nj[kMaxOutLanes] = {0};
            int top = -1;
            for (int j = 0; j < I + c.Kmax - 1; ++j) {
                for (int t = 0; t < c.ntw; ++t) nj[j] += pairs_in_lane(j, I, c.tw_ntaps[t]);
                if (nj[j] > 0) top = j;
            }
            c.nl = top + 1;
            if (c.nl > kMaxOutLanes) continue;
            // largest number of channels whose sums every lane (and the whole word) holds
            const i128 cap = c.result_signed ? (c.spacer ? pow2(L - 2) - 1 : pow2(L - 1) - 1) : pow2(L) - 1;
            i128 gmax = d.C;
            i128 place = 0;
            for (int j = 0; j < c.nl; ++j) {
                if (nj[j] == 0) continue;
                i128 per = (i128)d.KH * nj[j] * prod;
                if (j < c.nl - 1) gmax = std::min(gmax, cap / per);
                if (j * L > 62) { gmax = 0; break; }
                place += (i128)nj[j] * pow2(j * L);
            }
            if (gmax >= 1) gmax = std::min(gmax, kI64Max / ((i128)d.KH * prod * place));
            if (gmax < 1) continue;
            c.G = (int32_t)gmax;
            c.msb_mask = 0;
            for (int j = 0; j < c.nl - 1; ++j) c.msb_mask |= (uint64_t)1 << (j * L + L - 1);
            c.nq = (c.Wo + c.Kmax - 1 + I - 1) / I;
            if (c.nq <= 64) {
                c.nqs = c.nq;
                c.cw = c.Wo;
                c.ncs = 1;
            } else {
                // a row too wide for one wave's lanes: column segments of cw output
                // columns (a multiple of I), each needing at most 64 words, words
                // [c0/I, (c0 + cw + Kmax - 2)/I]; the words reaching two segments are
                // computed by both
                c.nqs = 64;
                c.cw = ((c.nqs - 1) * I - (c.Kmax - 2)) / I * I;
                if (c.cw < I) continue;
                c.ncs = (c.Wo + c.cw - 1) / c.cw;
            }
            c.qseg = c.cw / I;
            c.nrt = d.KH * c.ntw;
            c.Hp = d.H + 2 * d.pad_h;
            c.macs_per_mad = (double)I * d.KW / (double)c.ntw;
            // the multiply-adds alone, spread perfectly over every SIMD, bound the cost below
            const double floor_cost = (double)d.N * c.Ho * c.ncs * c.nqs * d.M * d.C * c.nrt / 64.0 / 1024.0;
            if (!all && found && floor_cost >= best.cost) continue;
            if (!place_launch(d, c, all, range_limited)) continue;
            if (c.cost < best.cost) {
                best = c;
                found = true;
            }
        }
    }
    if (!found) {
        char buf[256];
        if (range_limited)
            snprintf(buf, sizeof buf, "the layer exceeds the kernels' index ranges (operand words of one image "
                     "above 2 GiB, a kernel-word slice above 2^31 words, or an operand spread of 2^32 threads or more)");
        else
            snprintf(buf, sizeof buf, "no exact SAMD lane geometry for %d-bit x %d-bit, KW=%d stride %d, Wo=%d",
                     xf.bits, wf.bits, d.KW, d.stride_w, g.Wo);
        err = buf;
        return SAMD_EUNSUPPORTED;
    }
    return SAMD_OK;
}

// Unsigned activations with signed weights may also be recentred: x - 2^(b-1) is a
// signed b-bit value, so products are half as large and a lane holds twice as many;
// the offset comes back exactly as 2^(b-1) times the sum of the weights over each
// output's in-image taps.  Both are planned and the cheaper kept.
int search_layout(const samd_conv2d_desc &d, samd_fmt xf, samd_fmt wf, int xoff, int layout, Conv2dGeom &best,
                  std::string &err, std::vector<Conv2dGeom> *all) {
    int st = search_lanes(d, xf, wf, xoff, layout, 1, best, err, all);
    if (!layout || !(xf.is_signed || wf.is_signed || xoff)) return st;
    // the permanent-spacer layout of a signed result: also without the spacer MSB
    Conv2dGeom alt;
    std::string err2;
    if (search_lanes(d, xf, wf, xoff, layout, 0, alt, err2, all) == SAMD_OK && (st != SAMD_OK || alt.cost < best.cost)) {
        best = alt;
        st = SAMD_OK;
    }
    return st;
}

int search_conv2d(const samd_conv2d_desc &d, samd_fmt xf, samd_fmt wf, int spacer, Conv2dGeom &best,
                  std::string &err, std::vector<Conv2dGeom> *all = nullptr) {
    int st = search_layout(d, xf, wf, 0, spacer, best, err, all);
    if (!xf.is_signed && wf.is_signed && xf.bits >= 2) {
        Conv2dGeom alt;
        std::string err2;
        const samd_fmt xs = {xf.bits, 1};
        const size_t first = all ? all->size() : 0;
        if (search_layout(d, xs, wf, 1 << (xf.bits - 1), spacer, alt, err2, all) == SAMD_OK) {
            // the correction: four table lookups and a multiply-add per output, issued after
            // the last barrier where nothing hides their latency (about 40 issue cycles per
            // output in measurements on MI355X)
            const double correction = (double)d.N * d.M * alt.Ho * alt.Wo * 40.0 / 64.0 / 1024.0;
            alt.cost += correction;
            if (all)
                for (size_t i = first; i < all->size(); ++i) (*all)[i].cost += correction;
            if (st != SAMD_OK || alt.cost < best.cost) {
                best = alt;
                st = SAMD_OK;
            }
        }
    }
    return st;
}

// Plans are a pure function of (shape, formats); the search prices thousands of launch
// shapes, so found plans are kept (under a lock) and later calls look them up.
using PlanKey = std::array<int32_t, 16>;
std::mutex plan_mu;
std::map<PlanKey, Conv2dGeom> plan_cache;
constexpr size_t kPlanCacheMax = 4096;
// Plans chosen by measurement (samd_conv2d_tune): they take precedence over the model's
// and are kept until cleared, since workspaces prepared under them depend on them.
std::map<PlanKey, Conv2dGeom> tuned_plans;

PlanKey plan_key(const samd_conv2d_desc &d, samd_fmt xf, samd_fmt wf, int spacer) {
    return {d.N, d.C, d.H, d.W, d.M, d.KH, d.KW, d.stride_h, d.stride_w, d.pad_h, d.pad_w,
            xf.bits, xf.is_signed, wf.bits, wf.is_signed, spacer};
}

}  // namespace

int plan_conv2d(const samd_conv2d_desc &d, samd_fmt xf, samd_fmt wf, Conv2dGeom &g, std::string &err,
                int spacer) {
    const PlanKey key = plan_key(d, xf, wf, spacer);
    {
        std::lock_guard<std::mutex> lock(plan_mu);
        auto tu = tuned_plans.find(key);
        if (tu != tuned_plans.end()) {
            g = tu->second;
            return SAMD_OK;
        }
        auto it = plan_cache.find(key);
        if (it != plan_cache.end()) {
            g = it->second;
            return SAMD_OK;
        }
    }
    int st = search_conv2d(d, xf, wf, spacer, g, err);
    if (st == SAMD_OK && !addressable(d, g)) {
        err = "the layer exceeds the kernels' index ranges (operand words of one image above 2 GiB, a kernel-word "
              "slice above 2^31 words, or an operand spread of 2^32 threads or more)";
        st = SAMD_EUNSUPPORTED;
    }
    if (st == SAMD_OK) {
        std::lock_guard<std::mutex> lock(plan_mu);
        if (plan_cache.size() >= kPlanCacheMax) plan_cache.clear();
        plan_cache.emplace(key, g);
    }
    return st;
}

int conv2d_candidates(const samd_conv2d_desc &d, samd_fmt xf, samd_fmt wf, int max_count,
                      std::vector<Conv2dGeom> &out, std::string &err, int spacer) {
    out.clear();
    // the model alone (no cache, no tuned plan): its choice, then every priced candidate
    Conv2dGeom model;
    std::vector<Conv2dGeom> all;
    int st = search_conv2d(d, xf, wf, spacer, model, err, &all);
    if (st) return st;
    if (!addressable(d, model)) {
        err = "the layer exceeds the kernels' index ranges (operand words of one image above 2 GiB, a kernel-word "
              "slice above 2^31 words, or an operand spread of 2^32 threads or more)";
        return SAMD_EUNSUPPORTED;
    }
    std::vector<Conv2dGeom> keep;
    for (const Conv2dGeom &c : all)
        if (addressable(d, c)) keep.push_back(c);
    std::stable_sort(keep.begin(), keep.end(),
                     [](const Conv2dGeom &a, const Conv2dGeom &b) { return a.cost < b.cost; });
    auto same = [](const Conv2dGeom &a, const Conv2dGeom &b) {
        return a.L == b.L && a.I == b.I && a.xoff == b.xoff && a.rows_path == b.rows_path && a.rh == b.rh &&
               a.groups == b.groups && a.wm == b.wm && a.ks == b.ks && a.spacer == b.spacer;
    };
    out.push_back(model);
    for (const Conv2dGeom &c : keep) {
        if ((int)out.size() >= max_count) break;
        bool dup = false;
        for (const Conv2dGeom &o : out) dup = dup || same(o, c);
        if (!dup) out.push_back(c);
    }
    return SAMD_OK;
}

int find_conv2d_candidate(const samd_conv2d_desc &d, samd_fmt xf, samd_fmt wf,
                          const std::function<bool(const Conv2dGeom &)> &match, Conv2dGeom &out,
                          std::string &err, int spacer) {
    // every priced candidate, unsorted (matching needs no ranking)
    Conv2dGeom model;
    std::vector<Conv2dGeom> all;
    int st = search_conv2d(d, xf, wf, spacer, model, err, &all);
    if (st) return st;
    for (const Conv2dGeom &c : all)
        if (addressable(d, c) && match(c)) {
            out = c;
            return SAMD_OK;
        }
    err = "no candidate plan of this shape matches";
    return SAMD_EINVAL;
}

void set_tuned_conv2d(const samd_conv2d_desc &d, samd_fmt xf, samd_fmt wf, const Conv2dGeom &g) {
    std::lock_guard<std::mutex> lock(plan_mu);
    tuned_plans[plan_key(d, xf, wf, g.layout_spaced)] = g;
}

void clear_tuned_conv2d(const samd_conv2d_desc *d, samd_fmt xf, samd_fmt wf) {
    std::lock_guard<std::mutex> lock(plan_mu);
    if (!d)
        tuned_plans.clear();
    else
        for (int spacer : {0, 1}) tuned_plans.erase(plan_key(*d, xf, wf, spacer));
}

// Workspace: kernel-word streams, the recentring correction table, the work queues of
// the multiply kernel, then the operand words of one call (each 256-byte aligned).
size_t conv2d_kw_bytes(const Conv2dGeom &g) { return ((size_t)g.kw_words * 4 + 255) / 256 * 256; }

size_t conv2d_pre_bytes(const Conv2dGeom &g) {
    return g.xoff ? ((size_t)g.M * (g.KH + 1) * (g.KW + 1) * 4 + 255) / 256 * 256 : 0;
}

size_t conv2d_queue_offset(const Conv2dGeom &g) { return conv2d_kw_bytes(g) + conv2d_pre_bytes(g); }

size_t conv2d_xs_offset(const Conv2dGeom &g) { return conv2d_queue_offset(g) + kQueueBytes; }

size_t conv2d_workspace_bytes(const Conv2dGeom &g) {
    // one spare channel after the last image: the batch fetched after a slice's last one
    // may read it (its products are never used)
    const size_t spare = (size_t)g.Hp * g.ntw * g.nq;
    return conv2d_xs_offset(g) + ((size_t)(g.spread_words + spare) * 4 + 255) / 256 * 256;
}

int plan_conv1d(int64_t n, samd_fmt xf, const int32_t *taps, int32_t K, samd_fmt kf, Conv1dGeom &best,
                std::string &err) {
    Conv1dGeom g = {};
    g.n = n;
    g.nout = n - K + 1;
    g.bits = xf.bits;
    g.K = K;
    g.xrw = (int32_t)row_words(n, xf.bits);
    const i128 xmax = pow2(xf.bits) - 1, kmax_v = pow2(kf.bits) - 1;
    const i128 u32max = pow2(32) - 1, u64max = pow2(64) - 1;
    double best_cost = 1e300;
    bool found = false;
    for (int L = 1; L <= 32; ++L) {
        int kmax = 0;
        for (int k = 1; k <= K; ++k)
            if (word_fits(kf.bits, false, L, k, 0, u32max)) kmax = k;
        if (kmax == 0) continue;
        int imax = 0;
        for (int i = 1; i <= 32; ++i)
            if (word_fits(xf.bits, false, L, i, 0, u32max)) imax = i;
        for (int I = 1; I <= std::min(imax, kConv1dMaxLanes); ++I) {
            Conv1dGeom c = g;
            c.L = L;
            c.I = I;
            int t0[kMaxTapWords], nt[kMaxTapWords];
            if (!split_taps(K, kmax, t0, nt, c.ngroups)) continue;
            // lanes: j <-> output q*I + j - (K - 1); group g's window starts at q*I - t0[g]
            int nl = I + K - 1, top = -1;
            if (nl > 64) continue;
            int nj[64] = {0};
            for (int j = 0; j < nl; ++j) {
                for (int q = 0; q < c.ngroups; ++q) nj[j] += pairs_in_lane(j, I, nt[q]);
                if (nj[j]) top = j;
            }
            bool ok = true;
            i128 total = 0;
            for (int j = 0; j <= top && ok; ++j) {
                i128 dmax = (i128)nj[j] * xmax * kmax_v;
                if (j < top && dmax > pow2(L) - 1) ok = false;
                if (j * L > 63 && dmax > 0) ok = false;
                if (ok) total += dmax * pow2(j * L);
            }
            if (!ok || total > u64max) continue;
            c.nl = top + 1;
            for (int q = 0; q < c.ngroups; ++q) {
                c.g_tap0[q] = t0[q];
                c.g_ntaps[q] = nt[q];
                c.g_delta[q] = -t0[q];
                uint64_t word = 0;
                for (int s = 0; s < nt[q]; ++s) word |= (uint64_t)(uint32_t)taps[t0[q] + s] << (s * L);
                c.g_word[q] = (uint32_t)word;
            }
            c.extra = (K - 1 + I - 1) / I;
            if (c.extra > kMaxConv1dExtra) continue;
            c.nwords = (c.nout + I - 1) / I;
            double cost = (double)c.ngroups * (1 + c.extra) * (2.0 + 3.0 * I) / I + 3.0 * (I + K) * (1 + c.extra) / I;
            if (cost < best_cost) {
                best_cost = cost;
                best = c;
                found = true;
            }
        }
    }
    if (!found) {
        err = "no exact SAMD lane geometry for this 1-D convolution";
        return SAMD_EUNSUPPORTED;
    }
    return SAMD_OK;
}

}  // namespace samd
