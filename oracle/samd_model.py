"""The paper's SAMD routines on Python integers, with its ambiguous passages read.

TEST INFRASTRUCTURE ONLY (see the package docstring).  A word of ``width`` bits is
a Python int in [0, 2**width); every operation reduces modulo 2**width, as the
scalar machine instruction would.  The functions follow the paper's steps in its
order; names follow its notation (b = value bits, lanes, spacer bits).

Readings of the paper (each one is pinned by a test in tests/test_samd_model.py):

* build-mask figure: the run of ones is built at the full word width, so runs of
  31 bits or more and lanes that straddle the top of the word are well defined
  (the printed ``1 << len`` is an int shift).
* lane-wise multiply figure: the partial product is accumulated with the
  lane-wise add, the write mask covers the lane's bits from the current bit to
  the lane top (``(bit << i) - bit`` with i the bits left), and the sum is
  returned.  The printed mask ``(bit << bits) - bit`` spills into the next lane;
  ``lanewise_mul_printed_mask`` keeps it to show where it fails.
* scale-with-spacers figure: the spacer-cleared vector is the one multiplied.
* scale-wrap figure: the scalar is the zero-extended b-bit pattern.
* signed convolution figure: the product is the exact signed product of the two
  sign-extended words (the printed code zero-extends both to 128 bits, which is
  only right while every needed lane lies in the low word), the kernel is the
  second operand, and the fix-up mask is MSB_LANE_MASK of the result lane width
  over the full result width.
* signed-values section: a negative lane n lowers lane n+1 (the more significant
  neighbour) by one; the fix-up adds lane n's sign bit into lane n+1.
* 1-bit signed values are {-1, 0} (two's complement).
* optimisations for permanent spacer bits (Sec. 6.1): where every result lane keeps its
  MSB as a spacer (its value fits lane - 1 bits), the fix-up's final xor is left out and
  each lane is read from its low lane - 1 bits (``fixup_spacer``, ``decode_spacer``).
"""
from __future__ import annotations

from typing import List, Sequence, Tuple


def wmask(width: int) -> int:
    return (1 << width) - 1


# --- Masks (build-mask figure) --------------------------------------------------

def build_mask(start: int, run: int, stride: int, width: int = 64) -> int:
    """``run`` ones every ``stride`` bits starting at bit ``start``; cut at ``width``."""
    ones = (1 << run) - 1
    m, pos = 0, start
    while pos < width:
        m |= ones << pos
        pos += stride
    return m & wmask(width)


def msb_lane_mask(w: int, width: int = 64) -> int:
    return build_mask(w - 1, 1, w, width)


def lsb_lane_mask(w: int, width: int = 64) -> int:
    return build_mask(0, 1, w, width)


def odd_lane_mask(w: int, width: int = 64) -> int:
    return build_mask(w, w, 2 * w, width)


def even_lane_mask(w: int, width: int = 64) -> int:
    return build_mask(0, w, 2 * w, width)


# --- Lanes <-> words ------------------------------------------------------------

def lanes_to_word(vals: Sequence[int], lane: int, width: int = 64) -> int:
    """Place value i's low ``lane`` bits at lane i (lane 0 least significant)."""
    word = 0
    for i, v in enumerate(vals):
        word |= (v & wmask(lane)) << (i * lane)
    return word & wmask(width)


def word_to_lanes(word: int, lane: int, count: int, signed: bool = False) -> List[int]:
    out = []
    for i in range(count):
        f = (word >> (i * lane)) & wmask(lane)
        if signed and f >> (lane - 1):
            f -= 1 << lane
        out.append(f)
    return out


# --- Conventional SAMD arithmetic (Sec. 3) ----------------------------------------

def add_with_spacers(a: int, b: int, bits: int, width: int = 64) -> int:
    """Unsigned add with one permanent spacer bit on top of every b-bit value
    (lanes of b+1 bits): clear the spacers, then one scalar add."""
    keep = ~msb_lane_mask(bits + 1, width) & wmask(width)
    return ((a & keep) + (b & keep)) & wmask(width)


def lanewise_add(a: int, b: int, bits: int, width: int = 64) -> int:
    """Add modulo 2**bits per lane with a temporary spacer in each lane's top bit:
    add the low bits, then rebuild the top bit as the xor of both top bits and the
    carry caught in it."""
    top = msb_lane_mask(bits, width)
    low = ~top & wmask(width)
    top_xor = (a ^ b) & top
    return (((a & low) + (b & low)) ^ top_xor) & wmask(width)


def lanewise_sub(a: int, b: int, bits: int, width: int = 64) -> int:
    """Subtract modulo 2**bits per lane: force each minuend top bit to 1 so no
    borrow leaves the lane, then correct the top bit."""
    top = msb_lane_mask(bits, width)
    low = ~top & wmask(width)
    top_xor = (a ^ b) & top
    diff = ((a | top) - (b & low)) & wmask(width)
    return (diff ^ top_xor ^ top) & wmask(width)


def _lanewise_mul(a: int, b: int, bits: int, width: int, spill: bool) -> int:
    probe = lsb_lane_mask(bits, width)
    acc = 0
    for left in range(bits, 0, -1):
        sel = b & probe
        span = bits if spill else left
        fill = ((sel << span) - sel) & wmask(width)
        acc = lanewise_add(acc, a & fill, bits, width)
        a = (a << 1) & wmask(width)
        probe = (probe << 1) & wmask(width)
    return acc


def lanewise_mul(a: int, b: int, bits: int, width: int = 64) -> int:
    """Lane-wise product modulo 2**bits by shift-and-add, O(bits) steps: for each
    bit position of b's lanes, add the suitably shifted a into the lanes where
    that bit is set, masked to the lane's remaining bits."""
    return _lanewise_mul(a, b, bits, width, spill=False)


def lanewise_mul_printed_mask(a: int, b: int, bits: int, width: int = 64) -> int:
    """The same loop with the write mask as printed (``(bit << bits) - bit``)."""
    return _lanewise_mul(a, b, bits, width, spill=True)


# --- Vector scale (Sec. 4) ------------------------------------------------------

def scale_with_spacers(vec: int, scalar: int, bits: int, width: int = 64) -> int:
    """b-bit unsigned values in the odd b-bit lanes, b zero spacer bits below each
    in the even lanes: one scalar multiply puts each 2b-bit product in the value's
    lane and the spacer lane above it."""
    cleared = vec & odd_lane_mask(bits, width)
    return (cleared * scalar) & wmask(width)


def scale_wrap(vec: int, scalar: int, bits: int, width: int = 64) -> int:
    """Lane-wise product modulo 2**bits with dense b-bit lanes: split even and odd
    lanes so each has b zero bits above it, multiply both by the zero-extended
    scalar, keep each lane's low half and merge."""
    ev, od = even_lane_mask(bits, width), odd_lane_mask(bits, width)
    s = scalar & wmask(bits)
    return ((((vec & ev) * s) & ev) | (((vec & od) * s) & od)) & wmask(width)


# --- Signed values (Sec. 6) -------------------------------------------------------

def sign_extend4mul(vec: int, bits: int, lane: int, width: int = 64) -> int:
    """b-bit two's-complement values in the low bits of ``lane``-bit lanes (zero
    spacers above): subtract each value's sign bit, moved one place up, so every
    negative value's spacers fill with ones and the lane above loses one.  The word
    then equals sum_i v_i 2**(i*lane) modulo 2**width."""
    sign = vec & build_mask(bits - 1, 1, lane, width)
    return (vec - (sign << 1)) & wmask(width)


def to_signed(word: int, width: int) -> int:
    return word - (1 << width) if word >> (width - 1) else word


def fixup(product: int, lane: int, width: int) -> int:
    """Underflow fix-up: add each lane's sign bit to itself, which carries one into
    the lane above exactly where a negative lane had lowered it (a lane holding -1
    does not pass the carry on), then xor restores the sign bits.  Afterwards every
    lane is its own two's-complement value."""
    s = product & msb_lane_mask(lane, width)
    return ((product + s) & wmask(width)) ^ s


def fixup_spacer(product: int, lane: int, count: int, width: int) -> int:
    """The fix-up with a permanent spacer bit in every lane's MSB (Sec. 6.1): the sign
    bits of the result lanes below the top one are added to themselves as in ``fixup``,
    and the final xor, which only restores the MSBs, is left out.  Lane values must then
    fit lane - 1 bits (the MSB carries no value bit)."""
    s = product & msb_lane_mask(lane, width) & wmask((count - 1) * lane)
    return (product + s) & wmask(width)


def decode_spacer(product: int, lane: int, count: int, width: int) -> List[int]:
    """Signed result lanes with a permanent spacer MSB: ``fixup_spacer``, then every lane
    below the top one from its low lane - 1 bits, sign-extended, and the top lane from
    all remaining bits of the word as a two's-complement number."""
    w = fixup_spacer(product, lane, count, width)
    out = []
    for i in range(count - 1):
        f = (w >> (i * lane)) & wmask(lane - 1)
        out.append(f - (1 << (lane - 1)) if f >> (lane - 2) else f)
    top_bits = width - (count - 1) * lane
    t = w >> ((count - 1) * lane)
    out.append(t - (1 << top_bits) if t >> (top_bits - 1) else t)
    return out


def fixup_obvious(product: int, lane: int, width: int) -> int:
    """The rejected correction: add each sign bit one place up."""
    s = product & msb_lane_mask(lane, width)
    return (product + (s << 1)) & wmask(width)


def signed_convolution(vec: int, kernel: int, lane: int, word: int = 64) -> int:
    """Signed convolution by one multiply (signed convolution figure): the exact
    signed 2*word-bit product of the two sign-extended words, then the fix-up."""
    p = (to_signed(vec, word) * to_signed(kernel, word)) & wmask(2 * word)
    return fixup(p, lane, 2 * word)


def signed_convolution_printed(vec: int, kernel: int, lane: int, word: int = 64) -> int:
    """As printed: both words zero-extended to 2*word bits before the multiply."""
    p = (vec * kernel) & wmask(2 * word)
    return fixup(p, lane, 2 * word)


# --- Convolution by long multiplication (Sec. 5) ---------------------------------

def pack_lanes_signed(vals: Sequence[int], bits: int, lane: int, signed: bool, width: int = 64) -> int:
    """Pack b-bit values into ``lane``-bit lanes with zero spacers, then, for signed
    values, sign-extend them for the multiply."""
    w = lanes_to_word([v & wmask(bits) for v in vals], lane, width)
    return sign_extend4mul(w, bits, lane, width) if signed else w


def decode(product: int, lane: int, count: int, signed: bool, width: int) -> List[int]:
    """Read ``count`` result lanes: unsigned lanes directly, signed lanes after the
    fix-up."""
    if signed:
        return word_to_lanes(fixup(product, lane, width), lane, count, signed=True)
    return word_to_lanes(product, lane, count, signed=False)


def conv_by_multiply(x: Sequence[int], k: Sequence[int], bx: int, sx: bool, bk: int, sk: bool,
                     lane: int, word: int = 64) -> List[int]:
    """Full convolution of a short input and kernel that each fit one word: one
    multiply of the packed words, lane j of the product = sum_t k[t] x[j - t]."""
    X = pack_lanes_signed(x, bx, lane, sx, word)
    K = pack_lanes_signed(k, bk, lane, sk, word)
    signed = sx or sk
    if signed:
        p = (to_signed(X, word) * to_signed(K, word)) & wmask(2 * word)
    else:
        p = X * K
    return decode(p, lane, len(x) + len(k) - 1, signed, 2 * word)


def long_conv_overlap_add(x: Sequence[int], k: Sequence[int], bx: int, sx: bool, bk: int, sk: bool,
                          lane: int, per_word: int, word: int = 64) -> List[int]:
    """Full convolution of an input longer than a word: convolve each word-sized
    chunk of ``per_word`` inputs with the kernel by one multiply, then align the
    chunk results (parallelograms) by their offset and add the overlapping lanes."""
    n, K = len(x), len(k)
    full = [0] * (n + K - 1)
    for q in range(0, n, per_word):
        chunk = list(x[q:q + per_word])
        lanes = conv_by_multiply(chunk, k, bx, sx, bk, sk, lane, word)
        for j, v in enumerate(lanes):
            full[q + j] += v
    return full


def channel_sum_then_resolve(xs: Sequence[Sequence[int]], ks: Sequence[Sequence[int]], bx: int, sx: bool,
                             bk: int, sk: bool, lane: int, word: int = 64) -> List[int]:
    """Sum the packed products of several channels first and resolve the lanes
    once (the accumulate-before-resolve idea of Sec. 5)."""
    signed = sx or sk
    acc = 0
    for x, k in zip(xs, ks):
        X = pack_lanes_signed(x, bx, lane, sx, word)
        Kw = pack_lanes_signed(k, bk, lane, sk, word)
        if signed:
            acc += to_signed(X, word) * to_signed(Kw, word)
        else:
            acc += X * Kw
    acc &= wmask(2 * word)
    return decode(acc, lane, len(xs[0]) + len(ks[0]) - 1, signed, 2 * word)


def kronecker_conv(x: Sequence[int], k: Sequence[int], lane: int) -> List[int]:
    """Textbook Kronecker substitution with unbounded integers: evaluate both
    polynomials at 2**lane, multiply, read the signed base-2**lane digits."""
    X = sum(v << (i * lane) for i, v in enumerate(x))
    K = sum(v << (i * lane) for i, v in enumerate(k))
    P = X * K
    out, base, half = [], 1 << lane, 1 << (lane - 1)
    for _ in range(len(x) + len(k) - 1):
        d = P % base
        if d >= half:
            d -= base
        out.append(d)
        P = (P - d) >> lane
    assert P == 0
    return out


def word_digits(value: int, lane: int, count: int) -> Tuple[List[int], int]:
    """Signed base-2**lane digits of an exact integer, least significant first, by
    the per-lane form of the fix-up: digit j = the sign-extended lane field plus
    the sign bit of lane j-1.  Returns (digits, remaining high part)."""
    digits = []
    for j in range(count):
        f = (value >> (j * lane)) & wmask(lane)
        if f >> (lane - 1):
            f -= 1 << lane
        borrow = (value >> (j * lane - 1)) & 1 if j else 0
        digits.append(f + borrow)
    rest = (value >> (count * lane)) + ((value >> (count * lane - 1)) & 1)
    return digits, rest
