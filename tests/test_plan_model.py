"""The lane geometries the library plans, checked on the CPU with Python integers.

For every workload shape and bit width the planner's geometry (lane width L, values per
operand word I, kernel-word tap groups, channels per decode G) is replayed here in plain
Python, independently of the HIP code: operand and kernel words must be int32, the
64-bit accumulator must hold every partial sum, and decoding the lanes with the fix-up
of the signed-convolution figure must give the direct sums - for extreme inputs at the
bound, and for a complete small convolution compared with the oracle."""
import itertools
import random

import numpy as np
import pytest

import paper_1809_10572_amd as samd
import samd_workloads as wl
from oracle import reference as ref
from oracle import samd_model as sm

I32 = (-(1 << 31), (1 << 31) - 1)


def tap_words(plan):
    return [(plan.phase[t], plan.tap0[t], plan.ntaps[t]) for t in range(plan.tap_words)]


def decode_lanes(V, L, nl, signed):
    """Lanes 0..nl-1 of an exact accumulator; the top lane takes all remaining bits."""
    if signed:
        word = V & ((1 << 64) - 1)
        mask = sum(1 << (j * L + L - 1) for j in range(nl - 1))
        s = word & mask
        fixed = ((word + s) & ((1 << 64) - 1)) ^ s
        lanes = sm.word_to_lanes(fixed, L, nl - 1, signed=True)
        top = sm.to_signed(fixed, 64) >> ((nl - 1) * L)
        return lanes + [top]
    lanes = sm.word_to_lanes(V, L, nl - 1, signed=False)
    return lanes + [V >> ((nl - 1) * L)]


def planned_conv2d(x, w, shape, xf, wf, plan):
    """The planned SAMD convolution on Python integers: operand words of I phase values,
    kernel words of reversed taps, exact products summed over G channels, then the
    lanes decoded and added into the outputs they belong to."""
    N, C, H, W, M, KH, KW, sh, sw, ph, pw = shape
    Ho, Wo = ref.out_hw(shape)
    L, I, Kmax, G = plan.lane_bits, plan.lanes, plan.taps_max, plan.flush_channels
    nq = plan.words_per_row
    tws = tap_words(plan)
    off = plan.x_offset
    signed = bool(xf.is_signed or wf.is_signed or off)
    y = np.zeros((N, M, Ho, Wo), dtype=np.int64)

    def xval(n, c, h, col):
        # recentred activations enter the lanes as x - off; the zero padding stays 0
        return int(x[n, c, h, col]) - off if 0 <= h < H and 0 <= col < W else 0

    nl_max = plan.out_lanes
    for n, m, ho in itertools.product(range(N), range(M), range(Ho)):
        for q in range(nq):
            acc = 0
            for c in range(C):
                for ky in range(KH):
                    h = ho * sh + ky - ph
                    for (r, a0, k) in tws:
                        delta = a0 + k - Kmax
                        A = sum(xval(n, c, h, sw * (q * I + delta + i) + r - pw) << (i * L) for i in range(I))
                        B = sum(int(w[m, c, ky, sw * (a0 + k - 1 - s) + r]) << (s * L) for s in range(k))
                        assert I32[0] <= A <= I32[1] and I32[0] <= B <= I32[1]
                        acc += A * B
                        assert -(1 << 63) <= acc < (1 << 63)
                if (c + 1) % G == 0 or c == C - 1:
                    for j, d in enumerate(decode_lanes(acc, L, nl_max, signed)):
                        o = q * I + j - (Kmax - 1)
                        if 0 <= o < Wo:
                            y[n, m, ho, o] += d
                    acc = 0
    if off:
        # add back off * (the weights of every output's in-image taps)
        ones = np.ones((N, C, H, W), dtype=np.int64)
        y += off * ref.conv2d(ones, w, shape)
    return y


SMALL = [
    (wl.Conv2dShape(1, 5, 4, 11, 2, 3, 3, 1, 1, 1, 1), [(1, 0, 4, 1), (4, 0, 4, 1), (8, 0, 8, 1), (3, 1, 3, 1),
                                                       (6, 1, 6, 1), (2, 1, 5, 0)]),
    (wl.Conv2dShape(1, 2, 9, 13, 2, 11, 11, 4, 4, 2, 2), [(4, 0, 4, 1), (8, 0, 8, 1), (2, 1, 2, 1)]),
    (wl.Conv2dShape(1, 3, 6, 9, 2, 5, 5, 1, 1, 2, 2), [(2, 0, 2, 1), (8, 0, 8, 1), (5, 1, 5, 1)]),
]


@pytest.mark.parametrize("shape,fmts", SMALL, ids=["3x3", "11x11s4", "5x5"])
def test_planned_convolution_matches_oracle(shape, fmts):
    rng = np.random.default_rng(sum(shape.as_tuple()))
    for bx, sx, bw, sw_ in fmts:
        xf, wf = samd.Fmt(bx, sx), samd.Fmt(bw, sw_)
        plan = samd.conv2d_plan(shape, xf, wf)
        gen = wl.half_extremes
        x = gen(rng, (shape.N, shape.C, shape.H, shape.W), bx, bool(sx))
        w = gen(rng, (shape.M, shape.C, shape.KH, shape.KW), bw, bool(sw_))
        got = planned_conv2d(x, w, shape.as_tuple(), xf, wf, plan)
        np.testing.assert_array_equal(got, ref.conv2d(x, w, shape.as_tuple()), err_msg=str((bx, sx, bw, sw_)))


def full_shapes():
    out = []
    for cfg, shape in ((1, wl.SINGLE), (3, wl.MID), (4, wl.STRESS)):
        for b in range(1, 9):
            xs, ws = (True, True) if cfg == 4 else (False, True)
            if cfg == 4 and b == 1:
                continue
            out.append((f"cfg{cfg}-b{b}", shape, samd.Fmt(b, xs), samd.Fmt(b, ws)))
    for li, shape in enumerate(wl.ALEXNET_LAYERS):
        for b in (2, 4, 8):
            out.append((f"alex{li + 1}-b{b}", shape, samd.Fmt(b, False), samd.Fmt(b, True)))
    return out


@pytest.mark.parametrize("name,shape,xf,wf", full_shapes(), ids=[f[0] for f in full_shapes()])
def test_planned_geometry_is_exact_at_the_bound(name, shape, xf, wf):
    """Every lane of a word accumulated over G channels of extreme products decodes
    exactly; operand and kernel words are int32 for every value in range."""
    plan = samd.conv2d_plan(shape, xf, wf)
    L, I, Kmax, G = plan.lane_bits, plan.lanes, plan.taps_max, plan.flush_channels
    assert 1 <= G <= shape.C and plan.macs_per_mad > 0
    tws = tap_words(plan)
    assert sum(k for (_, _, k) in tws) == shape.KW
    # recentred unsigned activations reach the lanes as signed b-bit values
    xlo, xhi = wl.value_range(xf.bits, bool(xf.is_signed) or plan.x_offset != 0)
    wlo, whi = wl.value_range(wf.bits, bool(wf.is_signed))
    for lo, hi, n in [(xlo, xhi, I)] + [(wlo, whi, k) for (_, _, k) in tws]:
        place = sum(1 << (i * L) for i in range(n))
        assert lo * place >= I32[0] and hi * place <= I32[1]
    signed = bool(xf.is_signed or wf.is_signed or plan.x_offset)
    rnd = random.Random(hash(name) & 0xFFFF)
    rows = G * shape.KH
    # adversarial operands: every product at its most positive / most negative value,
    # then random mixtures of the extremes
    cases = []
    for mode in ("max", "min", "mix", "mix"):
        xs, wsv = [], []
        for _ in range(rows):
            for (r, a0, k) in tws:
                if mode == "max":
                    xv, wv = (xhi, whi) if xhi * whi >= xlo * wlo else (xlo, wlo)
                    xw = [xv] * I, [wv] * k
                elif mode == "min":
                    xv, wv = (xhi, wlo) if xhi * wlo <= xlo * whi else (xlo, whi)
                    xw = [xv] * I, [wv] * k
                else:
                    xw = [rnd.choice((xlo, xhi)) for _ in range(I)], [rnd.choice((wlo, whi)) for _ in range(k)]
                xs.append(xw[0])
                wsv.append(xw[1])
        cases.append((xs, wsv))
    nl = plan.out_lanes
    assert nl <= I + Kmax - 1
    for xs, wsv in cases:
        acc = 0
        want = [0] * (I + Kmax - 1)
        for idx, (xv, wv) in enumerate(zip(xs, wsv)):
            r, a0, k = tws[idx % len(tws)]
            A = sum(v << (i * L) for i, v in enumerate(xv))
            B = sum(v << (s * L) for s, v in enumerate(wv))
            acc += A * B
            assert -(1 << 63) <= acc < (1 << 63)
            for j, d in enumerate(np.convolve(xv, wv)):
                want[j] += int(d)
        assert all(v == 0 for v in want[nl:])
        assert decode_lanes(acc, L, nl, signed) == want[:nl], name


def test_plan_prefers_more_lanes_for_fewer_bits():
    shape = wl.MID
    mpm = [samd.conv2d_plan(shape, samd.Fmt(b, False), samd.Fmt(b, True)).macs_per_mad for b in (1, 2, 4, 8)]
    assert mpm[0] >= mpm[1] >= mpm[2] >= mpm[3] and mpm[0] > mpm[3]


def test_plan_rejects_what_cannot_be_exact():
    # a 16-tap-wide kernel row of 8-bit values leaves no exact geometry within 32-bit words
    with pytest.raises(samd.SamdError) as e:
        samd.conv2d_plan(wl.Conv2dShape(1, 1, 4, 200, 1, 1, 100, 1, 1, 0, 0), samd.Fmt(8, False), samd.Fmt(8, True))
    assert e.value.status in (samd.SAMD_EUNSUPPORTED,)


def planned_conv1d(x, k, plan):
    """The planned 1-D convolution on Python integers: unsigned operand words of I values
    L bits apart, one kernel word per tap group (natural order), 32x32 -> 64-bit
    products, lanes read out and added into the outputs they belong to."""
    n, K = len(x), len(k)
    L, I, nl = plan.lane_bits, plan.lanes, plan.out_lanes
    nout = n - K + 1
    y = [0] * nout
    nwords = -(-nout // I)
    for q in range(nwords + plan.extra):
        acc = 0
        for g in range(plan.groups):
            t0, kk = plan.tap0[g], plan.ntaps[g]
            A = sum(int(x[q * I - t0 + i]) << (i * L) for i in range(I) if 0 <= q * I - t0 + i < n)
            B = sum(int(k[t0 + s]) << (s * L) for s in range(kk))
            assert A < (1 << 32) and B < (1 << 32)
            acc += A * B
        assert acc < (1 << 64)
        lanes = [(acc >> (j * L)) & ((1 << L) - 1) for j in range(nl - 1)] + [acc >> ((nl - 1) * L)]
        for j, d in enumerate(lanes):
            o = q * I + j - (K - 1)
            if 0 <= o < nout:
                y[o] += d
    return y


@pytest.mark.parametrize("bits", range(1, 9))
def test_planned_conv1d_matches_oracle(bits):
    rng = np.random.default_rng(bits)
    top = (1 << bits) - 1
    for K in (1, 2, 3, 5, 7, 16):
        for n in (K, K + 1, 41, 200):
            for x, k in ((np.full(n, top), np.full(K, top)), (wl.uniform(rng, (n,), bits, False),
                                                             wl.uniform(rng, (K,), bits, False))):
                plan = samd.conv1d_plan(n, bits, k.tolist(), bits)
                assert sum(plan.ntaps[g] for g in range(plan.groups)) == K
                assert planned_conv1d(x, k, plan) == list(ref.conv1d(x, k)), (bits, K, n)
