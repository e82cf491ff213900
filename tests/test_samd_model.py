"""Pins for the model of the paper's SAMD routines (oracle/samd_model.py).

Each routine is checked against an independent element-wise computation, a library
routine (numpy.convolve), the paper's worked examples and claims, or exhaustive
enumeration on tiny widths.  Tests also show where the routines as printed fail,
which is what justifies each reading."""
import itertools
import os
import random

import numpy as np
import pytest

from oracle import samd_model as sm
from oracle import reference as ref

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")
M64 = (1 << 64) - 1


def lanes(word, bits, width=64):
    """Split a word into b-bit lanes (the top one may be partial)."""
    out, pos = [], 0
    while pos < width:
        span = min(bits, width - pos)
        out.append(((word >> pos) & ((1 << span) - 1), span))
        pos += bits
    return out


def lanewise_ref(a, b, bits, op, width=64):
    """Element-wise reference: apply op to each lane pair modulo the lane size."""
    res, pos = 0, 0
    for (x, span), (y, _) in zip(lanes(a, bits, width), lanes(b, bits, width)):
        res |= (op(x, y) % (1 << span)) << pos
        pos += bits
    return res


# --- masks --------------------------------------------------------------------------

def test_masks_hand_written():
    with open(os.path.join(GOLDEN, "lane_masks.txt")) as f:
        rows = [l.split() for l in f if l.strip() and not l.startswith("#")]
    fns = {"MSB": sm.msb_lane_mask, "LSB": sm.lsb_lane_mask, "ODD": sm.odd_lane_mask, "EVEN": sm.even_lane_mask}
    assert len(rows) == 13
    for name, w, hexval in rows:
        assert fns[name](int(w)) == int(hexval, 16), (name, w)


def test_mask_runs_of_31_bits_and_wider():
    # the printed int shift would overflow here; the reading builds the run at full width
    assert sm.build_mask(0, 31, 64) == (1 << 31) - 1
    assert sm.build_mask(0, 40, 64) == (1 << 40) - 1
    assert sm.even_lane_mask(32) == 0xFFFFFFFF
    assert sm.msb_lane_mask(10, 128) == sum(1 << p for p in range(9, 128, 10))


# --- lane-wise arithmetic (Sec. 3) ----------------------------------------------------

@pytest.mark.parametrize("bits", range(1, 9))
def test_lanewise_add_sub_mul_match_elementwise(bits):
    rnd = random.Random(bits)
    for _ in range(300):
        a, b = rnd.getrandbits(64), rnd.getrandbits(64)
        assert sm.lanewise_add(a, b, bits) == lanewise_ref(a, b, bits, lambda x, y: x + y)
        assert sm.lanewise_sub(a, b, bits) == lanewise_ref(a, b, bits, lambda x, y: x - y)
        assert sm.lanewise_mul(a, b, bits) == lanewise_ref(a, b, bits, lambda x, y: x * y)


@pytest.mark.parametrize("bits", [1, 2, 3])
def test_lanewise_ops_exhaustive_16bit_word(bits):
    for a, b in itertools.product(range(1 << 12), range(0, 1 << 12, 37)):
        for fn, op in ((sm.lanewise_add, lambda x, y: x + y), (sm.lanewise_sub, lambda x, y: x - y),
                       (sm.lanewise_mul, lambda x, y: x * y)):
            assert fn(a, b, bits, 12) == lanewise_ref(a, b, bits, op, 12)


def test_printed_multiply_mask_spills_for_wide_lanes():
    rnd = random.Random(5)
    for bits in range(1, 9):
        wrong = 0
        for _ in range(200):
            a, b = rnd.getrandbits(64), rnd.getrandbits(64)
            wrong += sm.lanewise_mul_printed_mask(a, b, bits) != lanewise_ref(a, b, bits, lambda x, y: x * y)
        # b = 1 has a one-bit span either way; every wider lane sees the spill
        assert (wrong == 0) if bits == 1 else (wrong > 150), (bits, wrong)


def test_add_with_permanent_spacers():
    rnd = random.Random(9)
    for bits in (3, 7, 8):
        lane = bits + 1
        n = 64 // lane
        for _ in range(200):
            xs = [rnd.getrandbits(bits) for _ in range(n)]
            ys = [rnd.getrandbits(bits) for _ in range(n)]
            got = sm.word_to_lanes(sm.add_with_spacers(sm.lanes_to_word(xs, lane), sm.lanes_to_word(ys, lane), bits),
                                   lane, n)
            assert got == [x + y for x, y in zip(xs, ys)]  # the carry lands in the spacer


# --- vector scale (Sec. 4) --------------------------------------------------------------

@pytest.mark.parametrize("bits", range(1, 9))
def test_scale_wrap_zero_extended_scalar(bits):
    rnd = random.Random(100 + bits)
    lo = -(1 << (bits - 1))
    for _ in range(300):
        vec = rnd.getrandbits(64)
        s = rnd.randint(lo, (1 << bits) - 1)  # any b-bit pattern, signed or unsigned
        bcast = ((s % (1 << bits)) * sm.lsb_lane_mask(bits)) & M64   # the scalar in every lane
        want = lanewise_ref(vec, bcast, bits, lambda x, y: x * y)
        assert sm.scale_wrap(vec, s % (1 << bits), bits) == want


def test_scale_wrap_sign_extended_scalar_breaks_negative_scalars():
    rnd = random.Random(3)
    bits, wrong = 4, 0
    for _ in range(200):
        vec, s = rnd.getrandbits(64), rnd.randint(-8, -1)
        want = sm.scale_wrap(vec, s % 16, bits)
        ev, od = sm.even_lane_mask(bits), sm.odd_lane_mask(bits)
        sext = s & M64
        got = ((((vec & ev) * sext) & ev) | (((vec & od) * sext) & od)) & M64
        wrong += got != want
    assert wrong > 150


def test_sign_agnostic_low_half_exhaustive():
    # the low b bits of a b x b product agree for unsigned and two's-complement operands
    for bits in range(1, 9):
        m = (1 << bits) - 1
        for x, y in itertools.product(range(1 << bits), repeat=2):
            sx = x - (1 << bits) if x >> (bits - 1) else x
            sy = y - (1 << bits) if y >> (bits - 1) else y
            assert (x * y) & m == (sx * sy) & m


def test_scale_with_spacers_full_products():
    rnd = random.Random(4)
    for bits in (2, 5, 8):
        n = 64 // (2 * bits)
        for _ in range(100):
            xs = [rnd.getrandbits(bits) for _ in range(n)]
            s = rnd.getrandbits(bits)
            vec = sum(x << ((2 * i + 1) * bits) for i, x in enumerate(xs)) | rnd.getrandbits(64) & sm.even_lane_mask(bits)
            p = sm.scale_with_spacers(vec, s, bits)
            # each value's full 2b-bit product sits in its lane and the spacer above it
            for i, x in enumerate(xs):
                lo = (2 * i + 1) * bits
                if lo + 2 * bits <= 64:
                    assert (p >> lo) & ((1 << (2 * bits)) - 1) == x * s


# --- convolution by long multiplication (Sec. 5) -------------------------------------

def test_polynomial_example_through_one_multiply():
    rows = {}
    with open(os.path.join(GOLDEN, "polynomial_product.txt")) as f:
        for l in f:
            if l.strip() and not l.startswith("#"):
                rows[l.split()[0]] = [int(t) for t in l.split()[1:]]
    # coefficients lowest degree first in lanes; 10-bit lanes hold every product sum
    a, b = rows["a"][::-1], rows["b"][::-1]
    got = sm.conv_by_multiply(a, b, 4, True, 4, True, lane=10)
    assert got[::-1] == rows["product"]
    assert sm.kronecker_conv(a, b, 10)[::-1] == rows["product"]


def test_lane_contents_of_the_four_by_three_example():
    # inputs i0..i3 and taps k1..k3; the two complete lanes are k3 i0 + k2 i1 + k1 i2
    # and k3 i1 + k2 i2 + k1 i3 (Sec. 5.1), the other four are partial sums
    rnd = random.Random(1)
    for _ in range(50):
        i = [rnd.randint(0, 15) for _ in range(4)]
        k = [rnd.randint(0, 15) for _ in range(3)]  # k[0] = k1
        got = sm.conv_by_multiply(i, k, 4, False, 4, False, lane=10)
        assert got[2] == k[2] * i[0] + k[1] * i[1] + k[0] * i[2]
        assert got[3] == k[2] * i[1] + k[1] * i[2] + k[0] * i[3]
        assert got[0] == k[0] * i[0] and got[5] == k[2] * i[3]
        assert got[1] == k[1] * i[0] + k[0] * i[1] and got[4] == k[2] * i[2] + k[1] * i[3]


@pytest.mark.parametrize("bits", [1, 3, 5, 8])
@pytest.mark.parametrize("K", [3, 5])
def test_overlap_add_long_unsigned_conv(bits, K):
    rnd = random.Random(bits * 7 + K)
    x = [rnd.getrandbits(bits) for _ in range(257)]
    k = [rnd.getrandbits(bits) for _ in range(K)]
    lane = (K * ((1 << bits) - 1) ** 2).bit_length()
    # the kernel must fit one word (Sec. 5.1); b = 8 with 5 taps needs a 128-bit word
    word = 64 if (K - 1) * lane + bits <= 64 else 128
    per_word = (word - bits) // lane + 1
    full = sm.long_conv_overlap_add(x, k, bits, False, bits, False, lane, per_word, word)
    assert full == list(np.convolve(x, k))
    assert full[K - 1:len(x)] == list(ref.conv1d(np.array(x), np.array(k)))


# --- signed values (Sec. 6) --------------------------------------------------------------

@pytest.mark.parametrize("bits", range(1, 9))
def test_sign_extend4mul_gives_the_integer_value(bits):
    rnd = random.Random(bits)
    lane = 2 * bits + 2
    n = 64 // lane
    for _ in range(200):
        vals = [rnd.randint(-(1 << (bits - 1)), (1 << (bits - 1)) - 1) for _ in range(n)]
        w = sm.sign_extend4mul(sm.lanes_to_word([v & ((1 << bits) - 1) for v in vals], lane), bits, lane)
        assert sm.to_signed(w, 64) == sum(v << (i * lane) for i, v in enumerate(vals))


def random_signed_conv_case(rnd, bits, I, K, sx, sk):
    xs = [rnd.randint(-(1 << (bits - 1)), (1 << (bits - 1)) - 1) if sx else rnd.getrandbits(bits) for _ in range(I)]
    ks = [rnd.randint(-(1 << (bits - 1)), (1 << (bits - 1)) - 1) if sk else rnd.getrandbits(bits) for _ in range(K)]
    return xs, ks


@pytest.mark.parametrize("bits", range(1, 9))
@pytest.mark.parametrize("sx,sk", [(True, True), (False, True), (True, False)])
def test_signed_and_mixed_conv_by_multiply(bits, sx, sk):
    rnd = random.Random(bits * 3 + sx * 2 + sk)
    for K in (1, 3, 5):
        lane = (K * (1 << bits) ** 2).bit_length() + 1   # |sum| <= K 2^(2b), plus a sign bit
        # each packed word is a signed integer: its top lane keeps one bit of headroom
        # for the borrow a negative lane below it hands up
        word = 64 if (K - 1) * lane + bits <= 63 else 128
        I = (word - 1 - bits) // lane + 1
        for _ in range(100):
            xs, ks = random_signed_conv_case(rnd, bits, I, K, sx, sk)
            got = sm.conv_by_multiply(xs, ks, bits, sx, bits, sk, lane, word)
            assert got == list(np.convolve(xs, ks)), (bits, K, xs, ks)


def test_top_lane_without_headroom_overflows_the_word():
    # b = 4, 10-bit lanes, seven lanes: the top field ends at bit 63; with -8 on top and
    # a negative lane below, the word's value is below -2**63
    xs = [0, 0, 0, 0, 0, -1, -8]
    X = sm.pack_lanes_signed(xs, 4, 10, True, 64)
    assert sm.to_signed(X, 64) != sum(v << (10 * i) for i, v in enumerate(xs))
    X6 = sm.pack_lanes_signed(xs[:6], 4, 10, True, 64)
    assert sm.to_signed(X6, 64) == sum(v << (10 * i) for i, v in enumerate(xs[:6]))


def test_printed_zero_extended_product_fails_when_top_lanes_are_high():
    rnd = random.Random(8)
    bits = 4
    lane = 2 * bits + 2
    for K, expect_fail in ((1, False), (3, True), (5, True)):
        I = 64 // lane
        wrong = 0
        for _ in range(300):
            xs, ks = random_signed_conv_case(rnd, bits, I, K, True, True)
            X = sm.pack_lanes_signed(xs, bits, lane, True)
            Kw = sm.pack_lanes_signed(ks, bits, lane, True)
            n = I + K - 1
            good = sm.word_to_lanes(sm.signed_convolution(X, Kw, lane), lane, n, signed=True)
            assert good == list(np.convolve(xs, ks))
            bad = sm.word_to_lanes(sm.signed_convolution_printed(X, Kw, lane), lane, n, signed=True)
            wrong += bad != good
        # with one tap every needed lane is in the low 64 bits, so zero-extension is harmless
        assert (wrong > 150) if expect_fail else (wrong == 0), (K, wrong)


def test_fixup_exhaustive_small_and_obvious_fixup_fails():
    # every b <= 3 input vector of up to 4 lanes and kernel of up to 3 taps, summed over
    # up to 3 channels before one fix-up; lanes sized for the accumulated range
    obvious_failures = 0
    for bits in (1, 2, 3):
        vals = range(-(1 << (bits - 1)), 1 << (bits - 1))
        for I, K, G in ((1, 1, 1), (2, 2, 1), (3, 2, 2), (4, 3, 1), (2, 3, 3)):
            lane = (G * min(I, K) * (1 << (bits - 1)) ** 2).bit_length() + 1
            cases = list(itertools.product(vals, repeat=I))
            kernels = list(itertools.product(vals, repeat=K))
            rnd = random.Random(bits * 100 + I * 10 + K)
            pairs = [(c, k) for c in cases for k in kernels] if len(cases) * len(kernels) <= 4096 else \
                [(rnd.choice(cases), rnd.choice(kernels)) for _ in range(4096)]
            for xs, ks in pairs:
                acc = 0
                want = np.zeros(I + K - 1, dtype=np.int64)
                for g in range(G):
                    xg = [((v + g) % (1 << bits)) - (1 << (bits - 1)) if g else v for v in xs]
                    X = sm.pack_lanes_signed(xg, bits, lane, True)
                    Kw = sm.pack_lanes_signed(ks, bits, lane, True)
                    acc += sm.to_signed(X, 64) * sm.to_signed(Kw, 64)
                    want += np.convolve(xg, ks)
                acc &= (1 << 128) - 1
                n = I + K - 1
                got = sm.word_to_lanes(sm.fixup(acc, lane, 128), lane, n, signed=True)
                assert got == list(want)
                # the lowest lane needs no correction at all
                raw0 = sm.word_to_lanes(acc, lane, 1, signed=True)[0]
                assert raw0 == want[0]
                obvious = sm.word_to_lanes(sm.fixup_obvious(acc, lane, 128), lane, n, signed=True)
                obvious_failures += obvious != got
    assert obvious_failures > 0


def test_obvious_fixup_double_increments_a_zero_lane_next_to_a_negative_one():
    # true lanes [-1, 0, 5]: lane 1 reads as -1 after the borrow, and adding the sign
    # bits one place up both fixes lane 1 and carries into lane 2 a second time
    lane = 8
    value = (-1) + (0 << lane) + (5 << (2 * lane))
    word = value & ((1 << 64) - 1)
    assert sm.word_to_lanes(sm.fixup(word, lane, 64), lane, 3, signed=True) == [-1, 0, 5]
    assert sm.word_to_lanes(sm.fixup_obvious(word, lane, 64), lane, 3, signed=True) == [-1, 0, 6]


def test_msb_states_after_the_fixup_add():
    # Sec. 6.1: after product + sign bits (before the xor) a lane's top bit is set only
    # where the lane read all ones and the lane below it read negative - its true value
    # is then 0 and every other bit of the lane is 0; the lowest lane's top bit is clear
    rnd = random.Random(12)
    lane, n = 9, 7
    mask, seen = (1 << lane) - 1, 0
    for _ in range(3000):
        digits = [rnd.randint(-(1 << (lane - 1)) + 1, (1 << (lane - 1)) - 1) for _ in range(n)]
        digits[rnd.randrange(1, n)] = 0
        value = sum(d << (i * lane) for i, d in enumerate(digits)) & M64
        added = (value + (value & sm.msb_lane_mask(lane, 64))) & M64
        assert (added >> (lane - 1)) & 1 == 0
        for j in range(1, n):
            raw = (value >> (j * lane)) & mask
            below_negative = (value >> (j * lane - 1)) & 1
            top = (added >> (j * lane + lane - 1)) & 1
            assert top == int(raw == mask and below_negative == 1)
            if top:
                seen += 1
                assert digits[j] == 0 and (added >> (j * lane)) & (mask >> 1) == 0
    assert seen > 100


def test_channel_sum_before_resolve():
    rnd = random.Random(21)
    for bits in (1, 2, 4):
        for _ in range(50):
            C, I, K = 12, 4, 3
            xs = [[rnd.getrandbits(bits) for _ in range(I)] for _ in range(C)]
            ks = [[rnd.randint(-(1 << (bits - 1)), (1 << (bits - 1)) - 1) for _ in range(K)] for _ in range(C)]
            lane = (C * K * ((1 << bits) - 1) * (1 << (bits - 1))).bit_length() + 1
            got = sm.channel_sum_then_resolve(xs, ks, bits, False, bits, True, lane)
            want = sum(np.convolve(x, k) for x, k in zip(xs, ks))
            assert got == list(want)


def test_word_digits_per_lane_fixup_matches_kronecker():
    rnd = random.Random(2)
    for _ in range(500):
        lane = rnd.randint(3, 16)
        n = rnd.randint(1, 64 // lane)
        digits = [rnd.randint(-(1 << (lane - 1)) + 1, (1 << (lane - 1)) - 1) for _ in range(n)]
        value = sum(d << (i * lane) for i, d in enumerate(digits))
        got, rest = sm.word_digits(value, lane, n)
        assert got == digits and rest == 0


def test_samd2_holds_the_ternary_set():
    # Sec. 2: the signed 2-bit format holds {-2, -1, 0, 1}, so {-1, 0, +1} fits
    vals = [-1, 0, 1, -1, 1, 0, 0, 1]
    words, bad = ref.pack(np.array(vals), 2, True)
    assert bad == 0 and list(ref.unpack(words, len(vals), 2, True)) == vals


# --- Sec. 6.1: optimisations for permanent spacer bits ------------------------------

def test_spacer_fixup_exhaustive_small():
    # every b <= 3 input vector of up to 4 lanes and kernel of up to 3 taps, summed over up
    # to 3 channels, in lanes one bit wider than the accumulated range needs (the MSB is a
    # permanent spacer): the fix-up without its xor, read from the low lane - 1 bits, gives
    # every lane exactly, as the full fix-up does
    for bits in (1, 2, 3):
        vals = range(-(1 << (bits - 1)), 1 << (bits - 1))
        for I, K, G in ((1, 1, 1), (2, 2, 1), (3, 2, 2), (4, 3, 1), (2, 3, 3)):
            lane = (G * min(I, K) * (1 << (bits - 1)) ** 2).bit_length() + 2
            cases = list(itertools.product(vals, repeat=I))
            kernels = list(itertools.product(vals, repeat=K))
            rnd = random.Random(7 + bits * 100 + I * 10 + K)
            pairs = [(c, k) for c in cases for k in kernels] if len(cases) * len(kernels) <= 4096 else \
                [(rnd.choice(cases), rnd.choice(kernels)) for _ in range(4096)]
            for xs, ks in pairs:
                acc = 0
                want = np.zeros(I + K - 1, dtype=np.int64)
                for g in range(G):
                    xg = [((v + g) % (1 << bits)) - (1 << (bits - 1)) if g else v for v in xs]
                    acc += sm.to_signed(sm.pack_lanes_signed(xg, bits, lane, True), 64) * \
                        sm.to_signed(sm.pack_lanes_signed(ks, bits, lane, True), 64)
                    want += np.convolve(xg, ks)
                acc &= (1 << 128) - 1
                n = I + K - 1
                assert sm.decode_spacer(acc, lane, n, 128) == list(want)
                assert sm.word_to_lanes(sm.fixup(acc, lane, 128), lane, n, signed=True) == list(want)


def test_spacer_fixup_needs_the_spare_msb():
    # a lane value that needs the MSB (outside lane - 1 signed bits) is misread without the
    # xor: -2**(lane-2) - 1 in a 9-bit lane reads as a positive number
    lane = 9
    vals = [3, -(1 << (lane - 2)) - 1, 7]
    word = sum(v << (i * lane) for i, v in enumerate(vals)) & ((1 << 64) - 1)
    assert sm.word_to_lanes(sm.fixup(word, lane, 64), lane, 3, signed=True) == vals
    assert sm.decode_spacer(word, lane, 3, 64)[1] != vals[1]
    # random words whose lanes all fit lane - 1 bits: both decodes agree
    rnd = random.Random(61)
    for _ in range(4000):
        n = rnd.randint(2, 7)
        digits = [rnd.randint(-(1 << (lane - 2)), (1 << (lane - 2)) - 1) for _ in range(n - 1)]
        digits.append(rnd.randint(-(1 << 20), 1 << 20))
        word = sum(d << (i * lane) for i, d in enumerate(digits)) & ((1 << 128) - 1)
        assert sm.decode_spacer(word, lane, n, 128) == digits


def test_spacer_accumulation_needs_no_msb_clearing():
    # Sec. 6.1's second point: results that feed further additions need no clearing of
    # their MSBs.  Here every addition happens on the exact products before any lane is
    # read, so sums over channels decode exactly with the spacer fix-up
    rnd = random.Random(5)
    bits, lane, G = 4, 13, 9
    for _ in range(500):
        xs = [[rnd.randint(-8, 7) for _ in range(4)] for _ in range(G)]
        ks = [[rnd.randint(-8, 7) for _ in range(3)] for _ in range(G)]
        acc = sum(sm.to_signed(sm.pack_lanes_signed(x, bits, lane, True), 64) *
                  sm.to_signed(sm.pack_lanes_signed(k, bits, lane, True), 64) for x, k in zip(xs, ks))
        want = sum(np.convolve(x, k) for x, k in zip(xs, ks))
        assert sm.decode_spacer(acc & ((1 << 128) - 1), lane, 6, 128) == list(want)
