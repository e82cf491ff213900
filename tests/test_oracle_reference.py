"""Pins for the plain oracle (oracle/ref.c): each result is checked against something
other than the oracle itself - hand-worked values, the paper's worked example, a
library routine, closed forms, brute force on tiny inputs."""
import itertools
import os

import numpy as np
import pytest
import torch

from oracle import reference as ref
import samd_workloads as wl

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def _golden_lines(name):
    with open(os.path.join(GOLDEN, name)) as f:
        return [l.strip() for l in f if l.strip() and not l.startswith("#")]


# --- packed storage format -------------------------------------------------------

def test_pack_hand_worked_words():
    rows = _golden_lines("pack_words.txt")
    assert len(rows) == 5
    for line in rows:
        head, vals, words = (s.split() for s in line.split("|"))
        bits, signed = int(head[0]), bool(int(head[1]))
        v = np.array([int(t) for t in vals], dtype=np.int32)
        want = np.array([int(t, 16) for t in words], dtype=np.uint32)
        got, bad = ref.pack(v, bits, signed)
        assert bad == 0
        np.testing.assert_array_equal(got, want)
        np.testing.assert_array_equal(ref.unpack(got, v.size, bits, signed), v)


@pytest.mark.parametrize("bits", range(1, 9))
@pytest.mark.parametrize("signed", [False, True])
def test_pack_roundtrip_every_value_every_position(bits, signed):
    lo, hi = wl.value_range(bits, signed)
    per = 32 // bits
    vals = np.arange(lo, hi + 1, dtype=np.int32)
    # every value at every field position, rows of a ragged length (3 words + 1 field)
    length = 3 * per + 1
    rows = []
    for shift in range(length):
        rows.append(np.resize(np.roll(vals, shift), length))
    x = np.stack(rows)
    words, bad = ref.pack(x, bits, signed)
    assert bad == 0
    assert words.shape == (length, ref.row_words(length, bits)) and words.shape[1] == 4
    np.testing.assert_array_equal(ref.unpack(words, length, bits, signed), x)
    # fields one by one, read with plain integer arithmetic
    for r, j in itertools.product(range(0, length, 7), range(length)):
        f = (int(words[r, j // per]) >> ((j % per) * bits)) & ((1 << bits) - 1)
        assert f == int(x[r, j]) % (1 << bits)
    # unused bits above P*b and fields past the row end are zero
    used = (1 << (per * bits)) - 1
    assert np.all((words.astype(np.uint64) & ~np.uint64(used) & np.uint64(0xFFFFFFFF)) == 0)
    # the last word holds one field; everything above it is zero
    assert np.all(words[:, 3] >> np.uint32(bits) == 0)


@pytest.mark.parametrize("bits", [1, 3, 8])
def test_pack_counts_and_masks_out_of_range(bits):
    lo, hi = wl.value_range(bits, True)
    v = np.array([lo - 1, hi + 1, lo, hi, 0], dtype=np.int32)
    words, bad = ref.pack(v, bits, True)
    assert bad == 2
    back = ref.unpack(words, v.size, bits, True)
    # stored as the low b bits, read back modulo 2^b into the signed range
    assert back[0] == hi and back[1] == lo and list(back[2:]) == [lo, hi, 0]


def test_row_words():
    assert ref.row_words(56, 1) == 2 and ref.row_words(56, 4) == 7 and ref.row_words(56, 8) == 14
    assert ref.row_words(1 << 20, 3) == 104858 and ref.row_words(0, 5) == 0


# --- 1-D convolution ----------------------------------------------------------------

def test_conv1d_polynomial_product_from_paper():
    rows = dict((l.split()[0], [int(t) for t in l.split()[1:]]) for l in _golden_lines("polynomial_product.txt"))
    a, b, want = rows["a"], rows["b"], rows["product"]
    # the full product is the valid convolution of the zero-padded input
    padded = [0] * (len(b) - 1) + a + [0] * (len(b) - 1)
    assert list(ref.conv1d(np.array(padded), np.array(b))) == want


@pytest.mark.parametrize("bits", [1, 4, 8])
@pytest.mark.parametrize("K", [1, 3, 5])
def test_conv1d_matches_numpy_convolve(bits, K):
    rng = np.random.default_rng(bits * 10 + K)
    x = rng.integers(-(1 << 8), 1 << 8, 1000)
    k = rng.integers(-(1 << 8), 1 << 8, K)
    np.testing.assert_array_equal(ref.conv1d(x, k), np.convolve(x, k, mode="valid"))


def test_conv1d_brute_force_and_closed_forms():
    rng = np.random.default_rng(7)
    for n in range(1, 9):
        for K in range(1, n + 1):
            x, k = rng.integers(-9, 10, n), rng.integers(-9, 10, K)
            want = [sum(int(k[t]) * int(x[i + K - 1 - t]) for t in range(K)) for i in range(n - K + 1)]
            assert list(ref.conv1d(x, k)) == want
    x = rng.integers(0, 256, 50)
    assert np.all(ref.conv1d(np.ones(50, int), np.ones(5, int)) == 5)
    # a delta at tap t shifts: y[i] = x[i + K - 1 - t]
    k = np.zeros(5, int)
    k[1] = 1
    np.testing.assert_array_equal(ref.conv1d(x, k), x[3:3 + 46])
    assert ref.conv1d(x[:2], k).size == 0


# --- 2-D convolution ----------------------------------------------------------------

SMALL_SHAPES = [
    wl.Conv2dShape(1, 1, 1, 1, 1, 1, 1),
    wl.Conv2dShape(2, 3, 7, 9, 4, 3, 3, 1, 1, 1, 1),
    wl.Conv2dShape(1, 2, 5, 13, 3, 3, 3, 1, 1, 0, 0),
    wl.Conv2dShape(2, 3, 19, 17, 5, 11, 11, 4, 4, 2, 2),
    wl.Conv2dShape(1, 4, 9, 9, 2, 5, 5, 1, 1, 2, 2),
    wl.Conv2dShape(1, 2, 6, 10, 3, 3, 5, 2, 1, 1, 2),
    wl.Conv2dShape(1, 1, 1, 40, 1, 1, 3, 1, 1, 0, 1),
]


@pytest.mark.parametrize("shape", SMALL_SHAPES, ids=lambda s: "x".join(map(str, s.as_tuple())))
def test_conv2d_matches_torch_float64(shape):
    rng = np.random.default_rng(sum(shape.as_tuple()))
    x = rng.integers(-128, 128, (shape.N, shape.C, shape.H, shape.W)).astype(np.int32)
    w = rng.integers(-128, 128, (shape.M, shape.C, shape.KH, shape.KW)).astype(np.int32)
    got = ref.conv2d(x, w, shape.as_tuple())
    # float64 is exact here: every partial sum is far below 2**53
    want = torch.nn.functional.conv2d(torch.from_numpy(x).double(), torch.from_numpy(w).double(),
                                      stride=(shape.stride_h, shape.stride_w),
                                      padding=(shape.pad_h, shape.pad_w)).numpy()
    assert got.shape == want.shape
    np.testing.assert_array_equal(got, want.astype(np.int64))


def test_conv2d_brute_force_tiny():
    shp = wl.Conv2dShape(1, 2, 4, 5, 2, 3, 2, 2, 1, 1, 1)
    rng = np.random.default_rng(3)
    x = rng.integers(-8, 8, (1, 2, 4, 5)).astype(np.int32)
    w = rng.integers(-8, 8, (2, 2, 3, 2)).astype(np.int32)
    Ho, Wo = (4 + 2 - 3) // 2 + 1, (5 + 2 - 2) // 1 + 1
    want = np.zeros((1, 2, Ho, Wo), np.int64)
    for m, ho, wo, c, ky, kx in itertools.product(range(2), range(Ho), range(Wo), range(2), range(3), range(2)):
        hi, wi = ho * 2 + ky - 1, wo + kx - 1
        if 0 <= hi < 4 and 0 <= wi < 5:
            want[0, m, ho, wo] += int(x[0, c, hi, wi]) * int(w[m, c, ky, kx])
    np.testing.assert_array_equal(ref.conv2d(x, w, shp.as_tuple()), want)


def test_conv2d_special_cases():
    rng = np.random.default_rng(11)
    # 1x1 kernel: a matrix product over channels
    x = rng.integers(0, 16, (2, 5, 6, 7)).astype(np.int32)
    w = rng.integers(-8, 8, (3, 5, 1, 1)).astype(np.int32)
    want = np.einsum("nchw,mc->nmhw", x.astype(np.int64), w[:, :, 0, 0].astype(np.int64))
    np.testing.assert_array_equal(ref.conv2d(x, w, (2, 5, 6, 7, 3, 1, 1, 1, 1, 0, 0)), want)
    # centred delta 3x3 kernel with pad 1 copies channel c into output c
    C = 4
    x = rng.integers(-8, 8, (1, C, 9, 8)).astype(np.int32)
    w = np.zeros((C, C, 3, 3), np.int32)
    for c in range(C):
        w[c, c, 1, 1] = 1
    np.testing.assert_array_equal(ref.conv2d(x, w, (1, C, 9, 8, C, 3, 3, 1, 1, 1, 1)), x)
    # constant input and weights: interior outputs are C*KH*KW*a*b, a corner sees 4 of 9 taps
    x = np.full((1, 3, 6, 6), 5, np.int32)
    w = np.full((2, 3, 3, 3), -7, np.int32)
    y = ref.conv2d(x, w, (1, 3, 6, 6, 2, 3, 3, 1, 1, 1, 1))
    assert np.all(y[:, :, 1:-1, 1:-1] == 3 * 9 * 5 * -7)
    assert np.all(y[:, :, 0, 0] == 3 * 4 * 5 * -7) and np.all(y[:, :, 0, 2] == 3 * 6 * 5 * -7)


def test_conv2d_points_agree_with_full():
    case = wl.conv2d_case(1, 4)
    y = ref.conv2d(case.x, case.w, case.shape.as_tuple())
    rng = np.random.default_rng(0)
    idx = np.stack([rng.integers(0, s, 40) for s in y.shape], axis=1)
    np.testing.assert_array_equal(ref.conv2d_points(case.x, case.w, case.shape.as_tuple(), idx),
                                  y[tuple(idx.T)])


# --- ReLU + requantisation ----------------------------------------------------------

def test_requant_hand_cases():
    acc = np.array([-5, 0, 3, 15], np.int64)
    assert ref.requant_shift(acc, 4) == 0
    assert list(ref.relu_requant(acc, 0, 4)) == [0, 0, 3, 15]
    acc = np.array([16, 7, 8, 9, -1], np.int64)
    # max 16 > 15 -> shift 1; round half up: 7 -> 4, 8 -> 4, 9 -> 5, 16 -> 8
    assert ref.requant_shift(acc, 4) == 1
    assert list(ref.relu_requant(acc, 1, 4)) == [8, 4, 4, 5, 0]
    # b = 2, max 100: 100 >> 5 = 3 <= 3 but 100 >> 4 = 6 > 3 -> shift 5;
    # (100 + 16) >> 5 = 3; 47 -> (47+16) >> 5 = 1; 48 -> 2
    acc = np.array([100, 47, 48, 95, 96], np.int64)
    assert ref.requant_shift(acc, 2) == 5
    assert list(ref.relu_requant(acc, 5, 2)) == [3, 1, 2, 3, 3]
    assert ref.requant_shift(np.array([-9, -1], np.int64), 3) == 0


def test_stack_tiny_chains_layers():
    layers = [wl.Conv2dShape(2, 3, 23, 23, 4, 11, 11, 4, 4, 2, 2), wl.Conv2dShape(2, 4, 5, 5, 3, 3, 3, 1, 1, 1, 1)]
    case = wl.stack_case(4, layers=layers)
    accs, acts, shifts = ref.stack(case.x, case.ws, [l.as_tuple() for l in layers], 4)
    assert len(accs) == 2 and len(acts) == 2 and len(shifts) == 1
    np.testing.assert_array_equal(accs[0], ref.conv2d(case.x, case.ws[0], layers[0].as_tuple()))
    assert acts[1].min() >= 0 and acts[1].max() <= 15 and acts[1].max() > 0
    np.testing.assert_array_equal(accs[1], ref.conv2d(acts[1], case.ws[1], layers[1].as_tuple()))
