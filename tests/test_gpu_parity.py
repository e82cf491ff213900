"""GPU parity: every result of the HIP library, called through its C ABI, compared
element by element with the CPU oracle on the same seeded inputs.  All results are
integers, so the bar is bit-exact equality."""
import numpy as np
import pytest
import torch

import paper_1809_10572_amd as samd
import samd_workloads as wl
from oracle import reference as ref

pytestmark = pytest.mark.gpu
DEV = "cuda:0"


def gpu_vals(a: np.ndarray, signed: bool) -> torch.Tensor:
    return torch.from_numpy(np.ascontiguousarray(a).astype(np.int8 if signed else np.uint8)).to(DEV)


def gpu_words(words: np.ndarray) -> torch.Tensor:
    return torch.from_numpy(np.ascontiguousarray(words).view(np.int32)).to(DEV)


def host_words(t: torch.Tensor) -> np.ndarray:
    return t.cpu().numpy().view(np.uint32)


def run_conv2d(x, w, shape, xf, wf):
    """Pack on the GPU, convolve with SAMD, return int32 numpy."""
    xs = gpu_vals(x, xf.is_signed)
    ws = gpu_vals(w, wf.is_signed)
    xp = samd.pack(xs, xf.bits, xf.is_signed)
    wp = samd.pack(ws, wf.bits, wf.is_signed)
    y = samd.conv2d(xp, xf, wp, wf, shape)
    torch.cuda.synchronize()
    return y.cpu().numpy()


@pytest.mark.parametrize("bits,xs,ws", [(2, 0, 1), (4, 1, 1), (8, 0, 1), (3, 1, 0)])
def test_fully_connected_as_1x1(bits, xs, ws):
    """A fully connected layer (batch 37, 300 -> 70) through conv2d as a 1x1 layer whose
    row is the batch (N = 1, C = inputs, H = 1, W = batch): the vector-scale form of the
    method, one tap per kernel word and I batch elements per operand word, against the
    plain matrix product."""
    rng = np.random.default_rng(bits * 7 + xs)
    batch, nin, nout = 37, 300, 70
    a = wl.uniform(rng, (batch, nin), bits, bool(xs))
    wt = wl.uniform(rng, (nout, nin), bits, bool(ws))
    shape = wl.Conv2dShape(1, nin, 1, batch, nout, 1, 1, 1, 1, 0, 0)
    x = np.ascontiguousarray(a.T).reshape(1, nin, 1, batch)
    w = wt.reshape(nout, nin, 1, 1)
    got = run_conv2d(x, w, shape, samd.Fmt(bits, xs), samd.Fmt(bits, ws)).reshape(nout, batch)
    want = (wt.astype(np.int64) @ a.astype(np.int64).T)
    np.testing.assert_array_equal(got, want)
    np.testing.assert_array_equal(got.reshape(1, nout, 1, batch), ref.conv2d(x, w, shape.as_tuple()))


def run_conv2d_int8(x, w, shape, xf, wf):
    xs = gpu_vals(np.transpose(x, (0, 2, 3, 1)), xf.is_signed)   # NHWC
    ws = gpu_vals(w, True)
    y = samd.conv2d_int8(xs, xf, ws, wf, shape)
    torch.cuda.synchronize()
    return y.cpu().numpy()


# --- packing ---------------------------------------------------------------------------

@pytest.mark.parametrize("bits", range(1, 9))
@pytest.mark.parametrize("signed", [False, True])
def test_pack_unpack_match_oracle(bits, signed):
    rng = np.random.default_rng(bits * 2 + signed)
    for rows, length in ((37, 101), (1, 1), (3, 32 // bits), (5, 32 // bits + 1), (64, 56)):
        v = wl.uniform(rng, (rows, length), bits, signed)
        want, bad = ref.pack(v, bits, signed)
        got = samd.pack(gpu_vals(v, signed), bits, signed)
        np.testing.assert_array_equal(host_words(got), want)
        back = samd.unpack(got, length, bits, signed).cpu().numpy().astype(np.int32)
        np.testing.assert_array_equal(back, v)


@pytest.mark.parametrize("bits", [1, 3, 7])
def test_pack_counts_out_of_range(bits):
    v = np.array([[0, (1 << bits), 255, 1, (1 << bits) - 1]], dtype=np.int32)
    want, bad = ref.pack(v, bits, False)
    oor = torch.zeros(1, dtype=torch.int32, device=DEV)
    got = samd.pack(gpu_vals(v, False), bits, False, oor)
    torch.cuda.synchronize()
    np.testing.assert_array_equal(host_words(got), want)
    assert int(oor.item()) == bad == 2


# --- 1-D convolution (workload 2) ------------------------------------------------------

@pytest.mark.parametrize("bits", range(1, 9))
@pytest.mark.parametrize("K", [3, 5])
def test_conv1d_full_size(bits, K):
    case = wl.conv1d_case(bits, K)
    want = ref.conv1d(case.x, case.k)
    words, _ = ref.pack(case.x, bits, False)
    y = samd.conv1d(gpu_words(words), case.x.size, bits, case.k.tolist(), bits)
    torch.cuda.synchronize()
    np.testing.assert_array_equal(y.cpu().numpy(), want)


@pytest.mark.parametrize("bits,K", [(2, 3), (8, 5)])
def test_conv1d_row_past_2_31_values(bits, K):
    """A row of 2^31 + 1000 values (64-bit value, word and output indices): pack and conv1d
    on the GPU (8.6 GB of outputs), sampled outputs - both ends, around index 2^31, and
    random ones - against the oracle on the windows that define them."""
    n = (1 << 31) + 1000
    gen = torch.Generator(device=DEV).manual_seed(1809 + bits)
    vals = torch.randint(0, 1 << bits, (n,), dtype=torch.uint8, device=DEV, generator=gen)
    taps = [int(t) for t in np.random.default_rng(bits).integers(0, 1 << bits, K)]
    xp = samd.pack(vals.view(1, n), bits, False).view(-1)
    y = samd.conv1d(xp, n, bits, taps, bits)
    torch.cuda.synchronize()
    del xp
    nout = n - K + 1
    rng = np.random.default_rng(bits * 31)
    idx = np.unique(np.concatenate([np.arange(0, 4), np.arange((1 << 31) - 8, (1 << 31) + 8),
                                    np.arange(nout - 4, nout), rng.integers(0, nout, 64)]))
    got = y[torch.from_numpy(idx).to(DEV)].cpu().numpy()
    for o, g in zip(idx, got):
        window = vals[int(o):int(o) + K].cpu().numpy().astype(np.int64)
        assert g == ref.conv1d(window, np.asarray(taps))[0], (bits, K, int(o))
    del y, vals
    torch.cuda.empty_cache()


@pytest.mark.parametrize("bits", range(1, 9))
def test_conv1d_ragged_and_degenerate(bits):
    rng = np.random.default_rng(bits)
    # tiny and degenerate rows, then rows of several blocks of output words with ragged ends
    # and wide kernels (several following words per output word)
    for n, K in ((1, 1), (3, 3), (4, 3), (5, 5), (33, 3), (97, 5), (1000, 7), (257, 16), (65, 1),
                 (100003, 3), (70001, 9), (8197, 16), (4096 * 3 + 1, 2)):
        x = wl.uniform(rng, (n,), bits, False)
        k = wl.uniform(rng, (K,), bits, False)
        words, _ = ref.pack(x, bits, False)
        y = samd.conv1d(gpu_words(words), n, bits, k.tolist(), bits)
        torch.cuda.synchronize()
        np.testing.assert_array_equal(y.cpu().numpy(), ref.conv1d(x, k), err_msg=f"n={n} K={K}")
    # outputs written from an address that is not 16-byte aligned (the one-by-one stores)
    for n, K in ((5000, 3), (4099, 5)):
        x = wl.uniform(rng, (n,), bits, False)
        k = wl.uniform(rng, (K,), bits, False)
        words, _ = ref.pack(x, bits, False)
        buf = torch.full((n - K + 2,), -7, dtype=torch.int32, device=DEV)
        y = samd.conv1d(gpu_words(words), n, bits, k.tolist(), bits, out=buf[1:])
        torch.cuda.synchronize()
        assert buf[1:].data_ptr() % 16 == 4
        np.testing.assert_array_equal(buf[1:].cpu().numpy(), ref.conv1d(x, k), err_msg=f"unaligned n={n} K={K}")
        assert int(buf[0].item()) == -7
    # every value at the top of the range
    x = np.full(999, (1 << bits) - 1, np.int32)
    k = np.full(5, (1 << bits) - 1, np.int32)
    words, _ = ref.pack(x, bits, False)
    y = samd.conv1d(gpu_words(words), 999, bits, k.tolist(), bits)
    torch.cuda.synchronize()
    np.testing.assert_array_equal(y.cpu().numpy(), ref.conv1d(x, k))


# --- lane-wise SAMD arithmetic on packed words ---------------------------------------

def wrap(v: np.ndarray, bits: int, signed: bool) -> np.ndarray:
    """v modulo 2**bits, read as a b-bit two's-complement (signed) or unsigned value."""
    m = np.asarray(v, np.int64) & ((1 << bits) - 1)
    return np.where(m >= (1 << (bits - 1)), m - (1 << bits), m) if signed else m


LANE_CASES = [(3, 61), (5, 256), (2, 7)]   # (rows, values per row): ragged rows, odd word counts


@pytest.mark.parametrize("bits", range(1, 9))
@pytest.mark.parametrize("signed", [False, True])
def test_lanewise_ops_match_elementwise(bits, signed):
    rng = np.random.default_rng(300 + 2 * bits + signed)
    for rows, n in LANE_CASES:
        for gen in (wl.uniform, wl.half_extremes):
            x = gen(rng, (rows, n), bits, signed)
            y = gen(rng, (rows, n), bits, signed)
            xw, _ = ref.pack(x, bits, signed)
            yw, _ = ref.pack(y, bits, signed)
            xg, yg = gpu_words(xw), gpu_words(yw)
            for op, fn in ((samd.LANE_ADD, np.add), (samd.LANE_SUB, np.subtract), (samd.LANE_MUL, np.multiply)):
                got = samd.lanewise(op, xg, yg, bits, signed)
                torch.cuda.synchronize()
                want, _ = ref.pack(wrap(fn(x.astype(np.int64), y), bits, signed), bits, signed)
                np.testing.assert_array_equal(host_words(got), want, err_msg=f"op {op} rows {rows} len {n}")
                np.testing.assert_array_equal(ref.unpack(host_words(got), n, bits, signed),
                                              wrap(fn(x.astype(np.int64), y), bits, signed))
            # in place: dst is a
            samd.lanewise(samd.LANE_ADD, xg, yg, bits, signed, out=xg)
            torch.cuda.synchronize()
            np.testing.assert_array_equal(ref.unpack(host_words(xg), n, bits, signed), wrap(x + y, bits, signed))


@pytest.mark.parametrize("bits", range(1, 9))
@pytest.mark.parametrize("signed", [False, True])
def test_vector_scale_matches_elementwise(bits, signed):
    rng = np.random.default_rng(400 + 2 * bits + signed)
    lo, hi = wl.value_range(bits, signed)
    for rows, n in LANE_CASES:
        x = wl.half_extremes(rng, (rows, n), bits, signed)
        xw, _ = ref.pack(x, bits, signed)
        xg = gpu_words(xw)
        for s in sorted({lo, hi, 0, 1, -1, lo + 1, int(rng.integers(lo, hi + 1))}):
            got = samd.scale(xg, s, bits, signed)
            torch.cuda.synchronize()
            want = wrap(x.astype(np.int64) * s, bits, signed)
            np.testing.assert_array_equal(ref.unpack(host_words(got), n, bits, signed), want, err_msg=f"scalar {s}")
            np.testing.assert_array_equal(host_words(got), ref.pack(want, bits, signed)[0])


# --- 2-D convolution: workloads 1, 3, 4 at full size -----------------------------------

def conv2d_full(cfg, bits):
    case = wl.conv2d_case(cfg, bits)
    xf, wf = samd.Fmt(bits, case.x_signed), samd.Fmt(bits, case.w_signed)
    want = ref.conv2d(case.x, case.w, case.shape.as_tuple())
    return case, xf, wf, want


@pytest.mark.parametrize("bits", range(1, 9))
def test_conv2d_single_layer(bits):
    case, xf, wf, want = conv2d_full(1, bits)
    np.testing.assert_array_equal(run_conv2d(case.x, case.w, case.shape, xf, wf), want)


@pytest.mark.parametrize("bits", range(1, 9))
def test_conv2d_mid_layer_full(bits):
    case, xf, wf, want = conv2d_full(3, bits)
    np.testing.assert_array_equal(run_conv2d(case.x, case.w, case.shape, xf, wf), want)


@pytest.mark.parametrize("bits", range(2, 9))
def test_conv2d_mixed_sign_stress_full(bits):
    case, xf, wf, want = conv2d_full(4, bits)
    np.testing.assert_array_equal(run_conv2d(case.x, case.w, case.shape, xf, wf), want)


EDGE = [
    wl.Conv2dShape(1, 1, 1, 1, 1, 1, 1),                      # a single MAC
    wl.Conv2dShape(1, 1, 1, 7, 1, 1, 3, 1, 1, 0, 1),          # H = 1
    wl.Conv2dShape(2, 3, 5, 61, 17, 3, 3, 1, 1, 1, 1),        # W not a multiple of any lane count, M = 17
    wl.Conv2dShape(1, 9, 13, 13, 33, 3, 3, 1, 1, 0, 0),       # no padding
    wl.Conv2dShape(1, 4, 12, 12, 16, 5, 5, 1, 1, 2, 2),       # 5x5, pad 2
    wl.Conv2dShape(2, 3, 45, 47, 20, 11, 11, 4, 4, 2, 2),     # 11x11 stride 4
    wl.Conv2dShape(1, 5, 17, 19, 8, 3, 3, 2, 2, 1, 1),        # stride 2
    wl.Conv2dShape(1, 2, 9, 30, 4, 3, 5, 1, 2, 1, 2),         # asymmetric kernel and stride
    wl.Conv2dShape(1, 300, 6, 6, 70, 3, 3, 1, 1, 1, 1),       # many channels, several decodes
    wl.Conv2dShape(3, 16, 8, 120, 48, 1, 1, 1, 1, 0, 0),      # 1x1, the vector-scale case
    wl.Conv2dShape(1, 8, 130, 9, 16, 3, 3, 1, 1, 1, 1),       # tall image, many row blocks
    wl.Conv2dShape(2, 5, 6, 300, 12, 3, 3, 1, 1, 1, 1),       # wide rows: several column segments
    wl.Conv2dShape(1, 3, 7, 700, 9, 3, 5, 2, 2, 1, 2),        # wide, strided, 5 taps
    wl.Conv2dShape(1, 2, 3, 1100, 8, 3, 3, 1, 1, 1, 1),       # rows of more than 256 operand words
]


@pytest.mark.parametrize("shape", EDGE, ids=lambda s: "x".join(map(str, s.as_tuple())))
@pytest.mark.parametrize("bx,sx,bw,sw", [(1, 0, 1, 1), (2, 1, 2, 1), (3, 0, 5, 1), (4, 0, 4, 1), (6, 1, 2, 0),
                                         (8, 0, 8, 1), (7, 1, 7, 1), (1, 1, 8, 1), (5, 0, 3, 0)])
def test_conv2d_edge_shapes(shape, bx, sx, bw, sw):
    xf, wf = samd.Fmt(bx, sx), samd.Fmt(bw, sw)
    try:
        samd.conv2d_plan(shape, xf, wf)
    except samd.SamdError as e:
        assert e.status in (samd.SAMD_EOVERFLOW, samd.SAMD_EUNSUPPORTED)
        pytest.skip(f"rejected on the host: {e}")
    rng = np.random.default_rng(sum(shape.as_tuple()) + bx * 100 + bw)
    for gen in (wl.uniform, wl.half_extremes):
        x = gen(rng, (shape.N, shape.C, shape.H, shape.W), bx, bool(sx))
        w = gen(rng, (shape.M, shape.C, shape.KH, shape.KW), bw, bool(sw))
        np.testing.assert_array_equal(run_conv2d(x, w, shape, xf, wf), ref.conv2d(x, w, shape.as_tuple()))
    # every product at the negative extreme: the largest borrow chains
    lo_x, hi_x = wl.value_range(bx, bool(sx))
    lo_w, hi_w = wl.value_range(bw, bool(sw))
    x = np.full((shape.N, shape.C, shape.H, shape.W), hi_x if lo_x == 0 else lo_x, np.int32)
    w = np.full((shape.M, shape.C, shape.KH, shape.KW), lo_w if lo_x == 0 else hi_w, np.int32)
    np.testing.assert_array_equal(run_conv2d(x, w, shape, xf, wf), ref.conv2d(x, w, shape.as_tuple()))


@pytest.mark.parametrize("sx", [0, 1])
def test_conv2d_largest_stack_accumulator(sx):
    """The largest accumulator the AlexNet-shaped stack can reach: 384 channels of 3x3 at
    8 bits with every product at its extreme (u8 x s8: 255 x -128; s8 x s8: -128 x -128),
    through the SAMD path and the int8 baseline; an interior output is the closed form
    384 * 9 * x * w (-112,803,840 and 56,623,104), the borders the oracle's."""
    shape = wl.Conv2dShape(1, 384, 6, 6, 16, 3, 3, 1, 1, 1, 1)
    xv = -128 if sx else 255
    x = np.full((shape.N, shape.C, shape.H, shape.W), xv, np.int32)
    w = np.full((shape.M, shape.C, shape.KH, shape.KW), -128, np.int32)
    want = ref.conv2d(x, w, shape.as_tuple())
    assert int(want[0, 0, 2, 2]) == 384 * 9 * xv * -128
    xf, wf = samd.Fmt(8, sx), samd.Fmt(8, 1)
    np.testing.assert_array_equal(run_conv2d(x, w, shape, xf, wf), want)
    np.testing.assert_array_equal(run_conv2d_int8(x, w, shape, xf, wf), want)


def test_conv2d_rejects_and_leaves_output_untouched():
    shape = wl.Conv2dShape(1, 512, 16, 16, 1, 16, 16, 1, 1, 0, 0)
    x = torch.zeros(512 * 16 * 4, dtype=torch.int32, device=DEV)
    w = torch.zeros(512 * 16 * 4, dtype=torch.int32, device=DEV)
    out = torch.full((1, 1, 1, 1), 7, dtype=torch.int32, device=DEV)
    with pytest.raises(samd.SamdError) as e:
        samd.conv2d(x, samd.Fmt(8, 0), w, samd.Fmt(8, 1), shape, ws=torch.zeros(1 << 20, dtype=torch.uint8,
                                                                                   device=DEV), out=out)
    assert e.value.status == samd.SAMD_EOVERFLOW
    assert int(out.item()) == 7


def test_conv2d_weights_past_2g_rows():
    """A 1x1 layer whose M*C weight rows pass 2^31 (C = 32768, M = 66000, u8 x s8: 8.6 GB
    of packed weights and as much kernel words): rows past the 2^31st are found with
    64-bit indices, and every output matches the oracle."""
    C, M = 32768, 66000
    shape = (1, C, 1, 1, M, 1, 1, 1, 1, 0, 0)
    assert M * C > 1 << 31
    rng = np.random.default_rng(2 ** 31)
    x = rng.integers(0, 256, size=(1, C, 1, 1), dtype=np.uint8)
    w = rng.integers(-128, 128, size=(M, C, 1, 1), dtype=np.int8)
    xf, wf = samd.Fmt(8, False), samd.Fmt(8, True)
    xp = samd.pack(gpu_vals(x, False), 8, False)
    wv = gpu_vals(w, True)
    wp = samd.pack(wv, 8, True)
    del wv
    y = samd.conv2d(xp, xf, wp, wf, shape)
    torch.cuda.synchronize()
    got = y.cpu().numpy()
    del wp, y
    torch.cuda.empty_cache()
    want = ref.conv2d(x, w, shape)
    np.testing.assert_array_equal(got, want)


# --- the native 8-bit baseline -----------------------------------------------------------

@pytest.mark.parametrize("cfg,bits", [(1, 4), (3, 1), (3, 4), (3, 8), (4, 2), (4, 8)])
def test_conv2d_int8_baseline_full(cfg, bits):
    case, xf, wf, want = conv2d_full(cfg, bits)
    np.testing.assert_array_equal(run_conv2d_int8(case.x, case.w, case.shape, xf, wf), want)


@pytest.mark.parametrize("shape", [EDGE[2], EDGE[4], EDGE[5], EDGE[8], wl.Conv2dShape(1, 3, 224, 224, 96, 11, 11, 4, 4, 2, 2)],
                         ids=["W61", "5x5", "11x11s4", "C300", "alex1"])
@pytest.mark.parametrize("bx,sx", [(8, 0), (8, 1), (4, 0)])
def test_conv2d_int8_baseline_edges(shape, bx, sx):
    rng = np.random.default_rng(bx + sx)
    x = wl.half_extremes(rng, (shape.N, shape.C, shape.H, shape.W), bx, bool(sx))
    w = wl.half_extremes(rng, (shape.M, shape.C, shape.KH, shape.KW), 8, True)
    got = run_conv2d_int8(x, w, shape, samd.Fmt(bx, sx), samd.Fmt(8, 1))
    np.testing.assert_array_equal(got, ref.conv2d(x, w, shape.as_tuple()))


# Layers of the halo-tiled int8 kernel (stride 1, C a multiple of 16): flat and
# row-segment tiles, 64- and 128-channel steps, channel counts that leave part of a chunk
# (or a whole chunk) empty, output channels that are not a multiple of the tile, ragged
# last tiles, 1x1 to 7x7 and asymmetric kernels; the last one has no halo that fits and
# takes the im2col kernel.  The stride-1 3x3 and 1x1 layers of at most 128 channels also
# have weight-resident launches (position counts that are and are not multiples of 4 and
# of the 32-position tile, filter counts that leave a wave's filters partly empty).  Every candidate launch of each layer is tested;
# tests/test_abi.py checks on the CPU that they include every tile shape.
HALO = [
    wl.Conv2dShape(2, 16, 9, 20, 24, 3, 3, 1, 1, 1, 1),        # small: 16 x 64 tiles
    wl.Conv2dShape(1, 48, 30, 61, 70, 3, 3, 1, 1, 1, 1),       # C = 48: a partly empty chunk
    wl.Conv2dShape(1, 80, 7, 150, 33, 3, 3, 1, 1, 1, 1),       # wide rows: row segments
    wl.Conv2dShape(2, 32, 12, 12, 130, 5, 5, 1, 1, 2, 2),      # 5x5, M = 130
    wl.Conv2dShape(1, 64, 1, 40, 16, 1, 3, 1, 1, 0, 1),        # H = 1, 1x3
    wl.Conv2dShape(3, 16, 20, 21, 8, 1, 1, 1, 1, 0, 0),        # 1x1
    wl.Conv2dShape(1, 144, 14, 14, 200, 3, 3, 1, 1, 1, 1),     # C = 144: an all-empty fourth chunk
    wl.Conv2dShape(2, 96, 28, 28, 100, 3, 3, 1, 1, 1, 1),      # 128-channel steps, C = 96
    wl.Conv2dShape(1, 256, 10, 10, 64, 3, 3, 1, 1, 1, 1),      # two 128-channel chunks
    wl.Conv2dShape(2, 16, 56, 56, 128, 3, 3, 1, 1, 1, 1),      # the mid-size layer's image size
    wl.Conv2dShape(1, 16, 5, 7, 16, 3, 7, 1, 1, 1, 3),         # 3x7, pad (1, 3)
    wl.Conv2dShape(1, 32, 6, 6, 16, 7, 7, 1, 1, 3, 3),         # 7x7 on a 6x6 image
    wl.Conv2dShape(1, 64, 14, 14, 200, 3, 3, 1, 1, 1, 1),     # two 128-filter tiles, the second partial
    wl.Conv2dShape(2, 128, 7, 9, 96, 1, 1, 1, 1, 0, 0),        # 1x1 with 128-channel steps, 63 positions
    wl.Conv2dShape(1, 256, 9, 11, 40, 3, 3, 1, 1, 1, 1),       # 2 chunks of 128 channels, 99 positions, M = 40
    wl.Conv2dShape(2, 384, 5, 7, 48, 1, 1, 1, 1, 0, 0),        # 1x1 in 3 chunks, 35 positions
    wl.Conv2dShape(1, 256, 4, 150, 40, 3, 3, 1, 1, 1, 1),      # wide rows: 4 chunks of 64 channels
    wl.Conv2dShape(1, 256, 2, 300, 16, 1, 1, 1, 1, 0, 0),      # 1x1, wide rows: 4 chunks of 64 channels
    wl.Conv2dShape(1, 16, 20, 80, 16, 11, 11, 1, 1, 5, 5),     # no halo fits: im2col kernel
    wl.Conv2dShape(1, 96, 12, 40, 40, 5, 5, 1, 1, 2, 2),       # 5x5, 96 channels: 64-channel halo chunks at 128 positions
    # packed-row K (few channels): 3 channels at 3x3 (one k-block), 11x11 stride 4 on 3
    # channels (nine), 1 channel with 130 filters (two workgroup rows), 5x5 with strides
    # (1, 2), 24 channels, and 42 positions per image (per-element output stores)
    wl.Conv2dShape(1, 3, 10, 8, 20, 3, 3, 1, 1, 1, 1),
    wl.Conv2dShape(2, 3, 30, 30, 24, 11, 11, 4, 4, 2, 2),
    wl.Conv2dShape(1, 1, 5, 8, 130, 3, 3, 1, 1, 1, 1),
    wl.Conv2dShape(2, 5, 6, 7, 17, 5, 5, 1, 2, 2, 1),
    wl.Conv2dShape(1, 24, 9, 9, 8, 3, 3, 1, 1, 1, 1),
    wl.Conv2dShape(2, 3, 6, 7, 70, 3, 3, 1, 1, 1, 1),
]


@pytest.mark.parametrize("bits", [8, 5])
def test_conv2d_int8_every_launch_mid(bits):
    """Every launch the int8 baseline can make for the mid-size layer (halo tiles,
    weight-resident runs of 400 and 208 positions, im2col), installed in turn, against the
    oracle at full size."""
    case, xf, wf, want = conv2d_full(3, bits)
    cands = samd.conv2d_int8_candidates(case.shape, xf, wf)
    assert sorted(p.positions for p in cands if p.halo == 2) == [208, 400]
    try:
        for plan in cands:
            samd.conv2d_int8_use_plan(case.shape, xf, wf, plan)
            np.testing.assert_array_equal(run_conv2d_int8(case.x, case.w, case.shape, xf, wf), want,
                                          err_msg=f"halo={plan.halo} {plan.mtile}x{plan.positions} w{plan.waves}")
    finally:
        samd.conv2d_int8_use_plan(case.shape, xf, wf, None)


@pytest.mark.parametrize("shape", [wl.Conv2dShape(2, 16, 56, 56, 128, 3, 3, 1, 1, 1, 1),
                                   wl.Conv2dShape(3, 16, 20, 21, 8, 1, 1, 1, 1, 0, 0),
                                   wl.Conv2dShape(1, 256, 9, 12, 40, 3, 3, 1, 1, 1, 1),
                                   wl.Conv2dShape(2, 384, 4, 8, 48, 1, 1, 1, 1, 0, 0),
                                   wl.Conv2dShape(1, 3, 10, 8, 20, 3, 3, 1, 1, 1, 1)],
                         ids=lambda s: "x".join(map(str, s.as_tuple())))
def test_conv2d_int8_resident_unaligned_output(shape):
    """The weight-resident (whole-K and chunked) and packed-row launches writing into an
    output 4 bytes past a 16-byte boundary (the transposed-tile store path) and into an
    aligned one (16-byte stores), against the oracle; nothing around the output is
    written."""
    rng = np.random.default_rng(5)
    x = wl.uniform(rng, (shape.N, shape.C, shape.H, shape.W), 8, False)
    w = wl.uniform(rng, (shape.M, shape.C, shape.KH, shape.KW), 8, True)
    xf, wf = samd.Fmt(8, 0), samd.Fmt(8, 1)
    want = ref.conv2d(x, w, shape.as_tuple())
    xs = gpu_vals(np.transpose(x, (0, 2, 3, 1)), False)
    ws = gpu_vals(w, True)
    cands = [p for p in samd.conv2d_int8_candidates(shape, xf, wf) if p.halo in (2, 3)]
    assert cands
    buf = torch.full((want.size + 8,), -7, dtype=torch.int32, device=DEV)
    try:
        for plan in cands:
            samd.conv2d_int8_use_plan(shape, xf, wf, plan)
            for off in (1, 4):
                buf.fill_(-7)
                samd.conv2d_int8(xs, xf, ws, wf, shape, out=buf[off:off + want.size])
                torch.cuda.synchronize()
                got = buf.cpu().numpy()
                np.testing.assert_array_equal(got[off:off + want.size].reshape(want.shape), want,
                                              err_msg=f"offset {off} positions {plan.positions}")
                assert (got[:off] == -7).all() and (got[off + want.size:] == -7).all()
    finally:
        samd.conv2d_int8_use_plan(shape, xf, wf, None)


@pytest.mark.parametrize("shape", [wl.Conv2dShape(1, 3, 10, 8, 20, 3, 3, 1, 1, 1, 1),
                                   wl.Conv2dShape(2, 16, 12, 12, 40, 3, 3, 1, 1, 1, 1),
                                   wl.Conv2dShape(1, 256, 9, 12, 40, 3, 3, 1, 1, 1, 1)],
                         ids=lambda s: "x".join(map(str, s.as_tuple())))
def test_conv2d_int8_misaligned_activations(shape):
    """Every int8 launch of the layer with the activations 1 and 4 bytes past a 16-byte
    boundary: the kernels that need 16-byte (weight-resident, halo) or 4-byte (packed-row)
    aligned activations give way to the im2col kernel, or run where their alignment holds;
    every result against the oracle."""
    rng = np.random.default_rng(11)
    x = wl.half_extremes(rng, (shape.N, shape.C, shape.H, shape.W), 8, False)
    w = wl.half_extremes(rng, (shape.M, shape.C, shape.KH, shape.KW), 8, True)
    xf, wf = samd.Fmt(8, 0), samd.Fmt(8, 1)
    want = ref.conv2d(x, w, shape.as_tuple())
    xh = np.ascontiguousarray(np.transpose(x, (0, 2, 3, 1))).astype(np.uint8).reshape(-1)
    ws = gpu_vals(w, True)
    buf = torch.zeros(xh.size + 32, dtype=torch.uint8, device=DEV)
    try:
        for plan in samd.conv2d_int8_candidates(shape, xf, wf):
            samd.conv2d_int8_use_plan(shape, xf, wf, plan)
            for off in (1, 4):
                xs = buf[off:off + xh.size]
                xs.copy_(torch.from_numpy(xh).to(DEV))
                assert xs.data_ptr() % 16 == off % 16
                got = samd.conv2d_int8(xs, xf, ws, wf, shape).cpu().numpy()
                np.testing.assert_array_equal(got, want, err_msg=f"offset {off} halo={plan.halo} "
                                              f"{plan.mtile}x{plan.positions}")
    finally:
        samd.conv2d_int8_use_plan(shape, xf, wf, None)


@pytest.mark.parametrize("shape", HALO, ids=lambda s: "x".join(map(str, s.as_tuple())))
@pytest.mark.parametrize("bx,sx", [(8, 0), (8, 1), (4, 0)])
def test_conv2d_int8_every_launch(shape, bx, sx):
    """Every launch the int8 baseline can make for the layer (the packed-row launches,
    each halo tile and weight-resident run that fits, and the im2col kernel), installed in
    turn, against the oracle; then the library's own choice again."""
    rng = np.random.default_rng(1000 + bx + sx)
    x = wl.half_extremes(rng, (shape.N, shape.C, shape.H, shape.W), bx, bool(sx))
    w = wl.half_extremes(rng, (shape.M, shape.C, shape.KH, shape.KW), 8, True)
    xf, wf = samd.Fmt(bx, sx), samd.Fmt(8, 1)
    want = ref.conv2d(x, w, shape.as_tuple())
    try:
        for plan in samd.conv2d_int8_candidates(shape, xf, wf):
            samd.conv2d_int8_use_plan(shape, xf, wf, plan)
            got = run_conv2d_int8(x, w, shape, xf, wf)
            np.testing.assert_array_equal(got, want, err_msg=f"halo={plan.halo} {plan.mtile}x{plan.positions} w{plan.waves}")
    finally:
        samd.conv2d_int8_use_plan(shape, xf, wf, None)
    np.testing.assert_array_equal(run_conv2d_int8(x, w, shape, xf, wf), want)


# --- requantisation and the AlexNet-shaped stack (workload 5) ---------------------------

@pytest.mark.parametrize("bits", [1, 2, 4, 8])
def test_max_and_relu_requant(bits):
    rng = np.random.default_rng(bits)
    for scale in (0, 3, 1000, 1 << 26):
        acc = rng.integers(-scale - 1, scale + 1, (3, 5, 7, 29)).astype(np.int32)
        a = torch.from_numpy(acc).to(DEV)
        mx = samd.max_i32(a)
        shift = torch.zeros(1, dtype=torch.int32, device=DEV)
        packed = samd.relu_requant_pack(a, mx, bits, shift_out=shift)
        nhwc = samd.relu_requant_nhwc_u8(a, mx, bits)
        torch.cuda.synchronize()
        assert int(mx.item()) == int(acc.max())
        s = ref.requant_shift(acc.astype(np.int64), bits)
        assert int(shift.item()) == s
        q = ref.relu_requant(acc.astype(np.int64), s, bits)
        want, _ = ref.pack(q.reshape(-1, 29), bits, False)
        np.testing.assert_array_equal(host_words(packed).reshape(-1, want.shape[-1]), want)
        np.testing.assert_array_equal(nhwc.cpu().numpy(), np.transpose(q, (0, 2, 3, 1)))


@pytest.mark.parametrize("shape", [(2, 3, 3, 1), (1, 96, 2, 64), (2, 301, 2, 65), (1, 260, 1, 130),
                                   (1, 8, 4, 200)], ids=lambda s: "x".join(map(str, s)))
def test_relu_requant_nhwc_tiles(shape):
    """The NHWC requantisation's tiling: rows wider than one column tile, channel counts
    above one channel chunk and not a multiple of 4 (the byte path), one column."""
    rng = np.random.default_rng(sum(shape))
    acc = rng.integers(-5000, 60000, shape).astype(np.int32)
    a = torch.from_numpy(acc).to(DEV)
    for bits in (2, 8):
        nhwc = samd.relu_requant_nhwc_u8(a, samd.max_i32(a), bits)
        torch.cuda.synchronize()
        s = ref.requant_shift(acc.astype(np.int64), bits)
        q = ref.relu_requant(acc.astype(np.int64), s, bits)
        np.testing.assert_array_equal(nhwc.cpu().numpy(), np.transpose(q, (0, 2, 3, 1)))


@pytest.mark.parametrize("shape", [(40, 11, 55), (7, 3, 5000), (2, 1, 4096), (3, 700, 1), (1, 1, 4097)],
                         ids=lambda s: "x".join(map(str, s)))
def test_relu_requant_pack_row_tiles(shape):
    """The packed requantisation's tiling: many workgroups of whole rows, rows of exactly
    one tile, rows of one value, and rows longer than a tile (one thread per word)."""
    rng = np.random.default_rng(sum(shape))
    acc = rng.integers(-70000, 70000, shape).astype(np.int32)
    a = torch.from_numpy(acc).to(DEV)
    for bits in (1, 3, 8):
        shift = torch.zeros(1, dtype=torch.int32, device=DEV)
        packed = samd.relu_requant_pack(a, samd.max_i32(a), bits, shift_out=shift)
        torch.cuda.synchronize()
        s = ref.requant_shift(acc.astype(np.int64), bits)
        assert int(shift.item()) == s
        q = ref.relu_requant(acc.astype(np.int64), s, bits)
        want, _ = ref.pack(q.reshape(-1, shape[-1]), bits, False)
        np.testing.assert_array_equal(host_words(packed).reshape(-1, want.shape[-1]), want)


@pytest.mark.parametrize("n", [1, 255, 1 << 20, 5_000_003])
def test_max_i32_many_workgroups(n):
    rng = np.random.default_rng(n)
    for where in (0, n // 2, n - 1):
        v = rng.integers(-(1 << 31), (1 << 30), n).astype(np.int32)
        v[where] = (1 << 31) - 1 - where % 7
        got = samd.max_i32(torch.from_numpy(v).to(DEV))
        torch.cuda.synchronize()
        assert int(got.item()) == int(v.max())
    neg = np.full(n, -(1 << 31), dtype=np.int32)
    assert int(samd.max_i32(torch.from_numpy(neg).to(DEV)).item()) == -(1 << 31)
    # a source that starts 4 bytes past a 16-byte boundary (the scalar path)
    v = rng.integers(-1000, 1000, n + 1).astype(np.int32)
    v[-1] = 5000
    t = torch.from_numpy(v).to(DEV)[1:]
    assert t.data_ptr() % 16 == 4
    assert int(samd.max_i32(t).item()) == 5000


def run_stack_samd(case):
    bits = case.bits
    x = samd.pack(gpu_vals(case.x, False), bits, False)
    accs, acts = [], []
    for li, (w, shp) in enumerate(zip(case.ws, case.layers)):
        wp = samd.pack(gpu_vals(w, True), bits, True)
        y = samd.conv2d(x, samd.Fmt(bits, False), wp, samd.Fmt(bits, True), shp)
        accs.append(y)
        if li + 1 < len(case.ws):
            x = samd.relu_requant_pack(y, samd.max_i32(y), bits)
            acts.append(x)
    torch.cuda.synchronize()
    return [a.cpu().numpy() for a in accs], acts


def run_stack_int8(case):
    bits = case.bits
    x = gpu_vals(np.transpose(case.x, (0, 2, 3, 1)), False)
    accs = []
    for li, (w, shp) in enumerate(zip(case.ws, case.layers)):
        y = samd.conv2d_int8(x, samd.Fmt(bits, False), gpu_vals(w, True), samd.Fmt(bits, True), shp)
        accs.append(y)
        if li + 1 < len(case.ws):
            x = samd.relu_requant_nhwc_u8(y, samd.max_i32(y), bits)
    torch.cuda.synchronize()
    return [a.cpu().numpy() for a in accs]


@pytest.mark.parametrize("bits", [2, 4, 8])
def test_alexnet_stack_batch2(bits):
    case = wl.stack_case(bits, batch=2)
    want_accs, want_acts, _ = ref.stack(case.x, case.ws, [l.as_tuple() for l in case.layers], bits)
    got_accs, got_acts = run_stack_samd(case)
    for li, (g, w) in enumerate(zip(got_accs, want_accs)):
        np.testing.assert_array_equal(g, w, err_msg=f"SAMD layer {li + 1}")
    for li, (g, w) in enumerate(zip(got_acts, want_acts[1:])):
        packed, _ = ref.pack(w, bits, False)
        np.testing.assert_array_equal(host_words(g), packed, err_msg=f"activation after layer {li + 1}")
    for li, (g, w) in enumerate(zip(run_stack_int8(case), want_accs)):
        np.testing.assert_array_equal(g, w, err_msg=f"int8 layer {li + 1}")


def run_stack_samd_fused(case):
    """The SAMD chain with the epilogue writing the next layer's operand words directly
    (relu_requant_stage), no packed activations between layers."""
    bits = case.bits
    xf, wf = samd.Fmt(bits, False), samd.Fmt(bits, True)
    wss = [samd.conv2d_prepare(samd.pack(gpu_vals(w, True), bits, True), wf, shp, xf)
           for w, shp in zip(case.ws, case.layers)]
    samd.conv2d_stage(samd.pack(gpu_vals(case.x, False), bits, False), xf, wf, case.layers[0], wss[0])
    accs, shifts = [], []
    for li, shp in enumerate(case.layers):
        y = samd.conv2d_accumulate(xf, wf, shp, wss[li])
        accs.append(y)
        if li + 1 < len(case.layers):
            sh = torch.zeros(1, dtype=torch.int32, device=DEV)
            samd.relu_requant_stage(y, samd.max_i32(y), bits, wf, case.layers[li + 1], wss[li + 1], dev_shift=sh)
            shifts.append(sh)
    torch.cuda.synchronize()
    return [a.cpu().numpy() for a in accs], [int(s.item()) for s in shifts]


@pytest.mark.parametrize("bits", [1, 2, 3, 4, 5, 8])
def test_alexnet_stack_fused_epilogue(bits):
    """ReLU + requantisation straight into the next layer's operand words gives every
    layer's accumulators and shifts of the oracle (batch 2)."""
    case = wl.stack_case(bits, batch=2)
    want_accs, _, want_shifts = ref.stack(case.x, case.ws, [l.as_tuple() for l in case.layers], bits)
    got_accs, got_shifts = run_stack_samd_fused(case)
    assert got_shifts == list(want_shifts)
    for li, (g, w) in enumerate(zip(got_accs, want_accs)):
        np.testing.assert_array_equal(g, w, err_msg=f"SAMD layer {li + 1}")


@pytest.mark.parametrize("bits", [2, 4, 8])
def test_alexnet_stack_full_batch(bits):
    case = wl.stack_case(bits)
    want_accs, _, _ = ref.stack(case.x, case.ws, [l.as_tuple() for l in case.layers], bits)
    got_accs, _ = run_stack_samd(case)
    for li, (g, w) in enumerate(zip(got_accs, want_accs)):
        np.testing.assert_array_equal(g, w, err_msg=f"SAMD layer {li + 1}")


@pytest.mark.parametrize("bits", [2, 8])
def test_alexnet_stack_full_batch_fused_tuned(bits):
    """The chain the stack benchmark times: batch 16, each layer's plan tuned on that
    layer's own input, ReLU + requantisation written straight into the next layer's
    operand words; every layer's accumulators and shifts against the oracle."""
    case = wl.stack_case(bits)
    shapes = [l.as_tuple() for l in case.layers]
    want_accs, want_acts, want_shifts = ref.stack(case.x, case.ws, shapes, bits)
    xf, wf = samd.Fmt(bits, False), samd.Fmt(bits, True)
    try:
        for li, (w, shp) in enumerate(zip(case.ws, case.layers)):
            xp = samd.pack(gpu_vals(want_acts[li], False), bits, False)
            samd.conv2d_tune(xp, xf, samd.pack(gpu_vals(w, True), bits, True), wf, shp, candidates=6, reps=2)
        got_accs, got_shifts = run_stack_samd_fused(case)
        assert got_shifts == list(want_shifts)
        for li, (g, w) in enumerate(zip(got_accs, want_accs)):
            np.testing.assert_array_equal(g, w, err_msg=f"SAMD layer {li + 1}")
    finally:
        for shp in case.layers:
            samd.conv2d_untune(shp, xf, wf)


@pytest.mark.parametrize("bits", [1, 4, 8])
def test_prepared_weights_are_reusable(bits):
    shape = EDGE[2]
    xf, wf = samd.Fmt(bits, False), samd.Fmt(bits, True)
    rng = np.random.default_rng(40 + bits)
    w = wl.uniform(rng, (shape.M, shape.C, shape.KH, shape.KW), bits, True)
    wp = samd.pack(gpu_vals(w, True), bits, True)
    ws = samd.conv2d_prepare(wp, wf, shape, xf)
    ws8 = samd.conv2d_int8_prepare(gpu_vals(w, True), wf, shape, xf)
    for _ in range(2):
        x = wl.uniform(rng, (shape.N, shape.C, shape.H, shape.W), bits, False)
        want = ref.conv2d(x, w, shape.as_tuple())
        y = samd.conv2d_prepared(samd.pack(gpu_vals(x, False), bits, False), xf, wf, shape, ws)
        y8 = samd.conv2d_int8_prepared(gpu_vals(np.transpose(x, (0, 2, 3, 1)), False), xf, wf, shape, ws8)
        torch.cuda.synchronize()
        np.testing.assert_array_equal(y.cpu().numpy(), want)
        np.testing.assert_array_equal(y8.cpu().numpy(), want)


def run_conv2d_spaced(x, w, shape, xf, wf):
    """The permanent-spacer layout: activations written in the layer's spaced words,
    convolved without a spread pass."""
    spaced = samd.conv2d_spaced_pack(gpu_vals(x, xf.is_signed), xf, wf, shape)
    wp = samd.pack(gpu_vals(w, wf.is_signed), wf.bits, wf.is_signed)
    y = samd.conv2d_spaced(spaced, xf, wf, shape, samd.conv2d_spaced_prepare(wp, wf, shape, xf))
    torch.cuda.synchronize()
    return y.cpu().numpy()


@pytest.mark.parametrize("bits", range(2, 9))
def test_vggb_layers(bits):
    """The paper's experiment shapes (Sec. 7): all ten VGG-B convolution layers at batch
    1 with signed N-bit activations and weights, N = 2..8, SAMD with temporary spacer bits
    (packed activations), SAMD with permanent spacer bits (the spaced layout) and the int8
    baseline, every output against the oracle."""
    f = samd.Fmt(bits, True)
    for li in range(len(wl.VGGB_LAYERS)):
        case = wl.vggb_case(li, bits)
        want = ref.conv2d(case.x, case.w, case.shape.as_tuple())
        np.testing.assert_array_equal(run_conv2d(case.x, case.w, case.shape, f, f), want,
                                      err_msg=f"SAMD layer {li + 1}")
        np.testing.assert_array_equal(run_conv2d_spaced(case.x, case.w, case.shape, f, f), want,
                                      err_msg=f"SAMD permanent-spacer layer {li + 1}")
        np.testing.assert_array_equal(run_conv2d_int8(case.x, case.w, case.shape, f, f), want,
                                      err_msg=f"int8 layer {li + 1}")


@pytest.mark.parametrize("bx,sx,bw,sw", [(1, 0, 1, 1), (4, 0, 4, 1), (5, 1, 6, 1), (8, 0, 8, 1)])
def test_conv2d_many_items_per_workgroup(bx, sx, bw, sw):
    """More work items than resident workgroups, a partial last row tile and M not a
    multiple of the channel block: workgroups take several items each, so every tile
    word must be re-zeroed between items.  Three inputs in a row on one workspace also
    check that the work queues are re-armed after every launch."""
    shape = wl.Conv2dShape(32, 16, 61, 23, 44, 3, 3, 1, 1, 1, 1)
    xf, wf = samd.Fmt(bx, sx), samd.Fmt(bw, sw)
    rng = np.random.default_rng(7 * bx + bw)
    w = wl.uniform(rng, (shape.M, shape.C, shape.KH, shape.KW), bw, bool(sw))
    ws = samd.conv2d_prepare(samd.pack(gpu_vals(w, bool(sw)), bw, bool(sw)), wf, shape, xf)
    for gen in (wl.uniform, wl.half_extremes, wl.uniform):
        x = gen(rng, (shape.N, shape.C, shape.H, shape.W), bx, bool(sx))
        y = samd.conv2d_prepared(samd.pack(gpu_vals(x, bool(sx)), bx, bool(sx)), xf, wf, shape, ws)
        torch.cuda.synchronize()
        np.testing.assert_array_equal(y.cpu().numpy(), ref.conv2d(x, w, shape.as_tuple()))


@pytest.mark.parametrize("bits", [2, 5])
def test_staged_input_accumulates_against_several_weight_sets(bits):
    """stage once, then prepare + accumulate two weight sets on the same staged words."""
    shape = EDGE[2]
    xf, wf = samd.Fmt(bits, False), samd.Fmt(bits, True)
    rng = np.random.default_rng(70 + bits)
    x = wl.uniform(rng, (shape.N, shape.C, shape.H, shape.W), bits, False)
    ws = torch.empty(samd.conv2d_workspace(shape, xf, wf), dtype=torch.uint8, device=DEV)
    samd.conv2d_stage(samd.pack(gpu_vals(x, False), bits, False), xf, wf, shape, ws)
    for _ in range(2):
        w = wl.uniform(rng, (shape.M, shape.C, shape.KH, shape.KW), bits, True)
        samd.conv2d_prepare(samd.pack(gpu_vals(w, True), bits, True), wf, shape, xf, ws=ws)
        y = samd.conv2d_accumulate(xf, wf, shape, ws)
        torch.cuda.synchronize()
        np.testing.assert_array_equal(y.cpu().numpy(), ref.conv2d(x, w, shape.as_tuple()))


@pytest.mark.parametrize("bits", [1, 4, 8])
def test_graph_replays_match_eager(bits):
    """pack + stage + accumulate captured in a HIP graph: every replay (with eager work
    and synchronisations in between) equals the eager result and the oracle."""
    shape = EDGE[2]
    xf, wf = samd.Fmt(bits, False), samd.Fmt(bits, True)
    rng = np.random.default_rng(90 + bits)
    x = wl.uniform(rng, (shape.N, shape.C, shape.H, shape.W), bits, False)
    w = wl.uniform(rng, (shape.M, shape.C, shape.KH, shape.KW), bits, True)
    want = ref.conv2d(x, w, shape.as_tuple())
    xg = gpu_vals(x, False)
    ws = samd.conv2d_prepare(samd.pack(gpu_vals(w, True), bits, True), wf, shape, xf)
    xp = torch.empty((shape.N, shape.C, shape.H, samd.row_words(shape.W, bits)), dtype=torch.int32, device=DEV)
    Ho, Wo = samd.out_hw(shape)
    y = torch.empty((shape.N, shape.M, Ho, Wo), dtype=torch.int32, device=DEV)

    def step():
        samd.pack(xg, bits, False, out=xp)
        samd.conv2d_prepared(xp, xf, wf, shape, ws, out=y)

    step()
    torch.cuda.synchronize()
    eager = y.cpu().numpy()
    np.testing.assert_array_equal(eager, want)
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):
        step()
    torch.cuda.current_stream().wait_stream(side)
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph):
        step()
    for i in range(4):
        y.fill_(-1)
        torch.cuda.synchronize()
        graph.replay()
        torch.cuda.synchronize()
        np.testing.assert_array_equal(y.cpu().numpy(), eager, err_msg=f"replay {i}")
        step()   # eager work between replays
        torch.cuda.synchronize()


# --- autotuning ------------------------------------------------------------------------

def plan_key(p):
    return (p.lane_bits, p.lanes, p.x_offset, p.shared_rows, p.rows_per_thread, p.rows_per_block, p.mblock,
            p.split_waves)


TUNE_CASES = [
    # (shape, x bits, x signed, w bits): shared-row candidates, strided and 5-wide kernels,
    # recentred unsigned activations, and a row of more than 64 operand words
    ((2, 24, 17, 45, 20, 3, 3, 1, 1, 1, 1), 2, False, 2),
    ((2, 24, 17, 45, 20, 3, 3, 1, 1, 1, 1), 8, False, 8),
    ((1, 9, 23, 61, 10, 3, 5, 2, 2, 1, 2), 5, True, 4),
    ((1, 6, 5, 300, 9, 3, 3, 1, 1, 1, 1), 6, True, 6),
]


@pytest.mark.parametrize("case", range(len(TUNE_CASES)))
def test_conv2d_tune_keeps_results_exact(case):
    shape, xb, xs, wb = TUNE_CASES[case]
    N, C, H, W, M, KH, KW = shape[:7]
    rng = np.random.default_rng(1000 + case)
    x = wl.uniform(rng, (N, C, H, W), xb, xs)
    w = wl.uniform(rng, (M, C, KH, KW), wb, True)
    xf, wf = samd.Fmt(xb, xs), samd.Fmt(wb, True)
    want = ref.conv2d(x, w, shape)
    xp = samd.pack(gpu_vals(x, xs), xb, xs)
    wp = samd.pack(gpu_vals(w, True), wb, True)
    cands = samd.conv2d_candidates(shape, xf, wf, 12)
    model = samd.conv2d_plan(shape, xf, wf)
    assert plan_key(cands[0]) == plan_key(model)
    try:
        # every candidate's output is checked against the model plan's inside the call
        chosen = samd.conv2d_tune(xp, xf, wp, wf, shape, candidates=12, reps=2)
        assert plan_key(chosen) in [plan_key(c) for c in cands]
        assert plan_key(samd.conv2d_plan(shape, xf, wf)) == plan_key(chosen)
        # later calls use the tuned plan (workspace sized and prepared under it)
        y = samd.conv2d(xp, xf, wp, wf, shape)
        torch.cuda.synchronize()
        np.testing.assert_array_equal(y.cpu().numpy(), want)
    finally:
        samd.conv2d_untune(shape, xf, wf)
    assert plan_key(samd.conv2d_plan(shape, xf, wf)) == plan_key(model)


def test_conv2d_tune_output_and_prepared_workspace():
    # the tuner leaves y holding the result and ws prepared for the chosen plan; with room
    # for the model plan only, the candidates that need more workspace are skipped
    shape = (2, 16, 12, 30, 12, 3, 3, 1, 1, 1, 1)
    rng = np.random.default_rng(77)
    x = wl.uniform(rng, (2, 16, 12, 30), 3, False)
    w = wl.uniform(rng, (12, 16, 3, 3), 3, True)
    xf, wf = samd.Fmt(3, False), samd.Fmt(3, True)
    want = ref.conv2d(x, w, shape)
    xp = samd.pack(gpu_vals(x, False), 3, False)
    wp = samd.pack(gpu_vals(w, True), 3, True)
    full = samd.conv2d_tune_workspace(shape, xf, wf, 8)
    extra = (2 * 12 * 12 * 30 * 4 + 255) // 256 * 256 + 256     # the second output and its counter
    tight = samd.conv2d_workspace(shape, xf, wf) + extra
    # an odd size: the second output still starts 256-byte aligned below the end
    for nbytes in (full, tight, tight + 77):
        ws = torch.empty(nbytes, dtype=torch.uint8, device=DEV)
        y = torch.full((2, 12, 12, 30), -7, dtype=torch.int32, device=DEV)
        try:
            samd.conv2d_tune(xp, xf, wp, wf, shape, candidates=8, reps=1, ws=ws, out=y)
            torch.cuda.synchronize()
            np.testing.assert_array_equal(y.cpu().numpy(), want)
            y2 = samd.conv2d_prepared(xp, xf, wf, shape, ws)
            torch.cuda.synchronize()
            np.testing.assert_array_equal(y2.cpu().numpy(), want)
        finally:
            samd.conv2d_untune(None)


# --- seeded random shapes --------------------------------------------------------------

def random_cases(n, seed, wmax=300, cmax=70, hmax=40):
    """Seeded conv2d shapes and format pairs within the library's limits: kernels 1..7
    (stride 1..3, padding up to the kernel), rows up to wmax values, channels up to cmax."""
    rng = np.random.default_rng(seed)
    out = []
    while len(out) < n:
        KH, KW = int(rng.integers(1, 8)), int(rng.integers(1, 8))
        sh, sw = int(rng.integers(1, 4)), int(rng.integers(1, 4))
        ph, pw = int(rng.integers(0, KH)), int(rng.integers(0, KW))
        H, W = int(rng.integers(max(1, KH - 2 * ph), hmax)), int(rng.integers(max(1, KW - 2 * pw), wmax + 1))
        N, C, M = int(rng.integers(1, 4)), int(rng.integers(1, cmax + 1)), int(rng.integers(1, 41))
        xb, wb = int(rng.integers(1, 9)), int(rng.integers(1, 9))
        xs, ws = bool(rng.integers(0, 2)), bool(rng.integers(0, 2))
        if C * KH * KW * (1 << xb) * (1 << wb) >= (1 << 31):
            continue
        out.append(((N, C, H, W, M, KH, KW, sh, sw, ph, pw), xb, xs, wb, ws))
    return out


# the second set: wide rows (many column segments), fewer channels and rows
RANDOM_CASES = random_cases(40, 1809) + random_cases(24, 2024, wmax=1200, cmax=24, hmax=12)


@pytest.mark.parametrize("case", range(24))
def test_conv1d_random(case):
    rng = np.random.default_rng(4000 + case)
    bits = int(rng.integers(1, 9))
    K = int(rng.integers(1, 17))
    n = int(rng.integers(K, 300001))
    x = wl.uniform(rng, (n,), bits, False)
    k = wl.uniform(rng, (K,), bits, False)
    words, _ = ref.pack(x, bits, False)
    try:
        y = samd.conv1d(gpu_words(words), n, bits, k.tolist(), bits)
    except samd.SamdError as e:
        assert e.status == -3, str(e)      # refused, never computed wrongly
        return
    torch.cuda.synchronize()
    np.testing.assert_array_equal(y.cpu().numpy(), ref.conv1d(x, k), err_msg=f"n={n} K={K} b={bits}")


@pytest.mark.parametrize("case", range(len(RANDOM_CASES)))
def test_conv2d_random_shapes(case):
    shape, xb, xs, wb, ws = RANDOM_CASES[case]
    N, C, H, W, M, KH, KW = shape[:7]
    rng = np.random.default_rng(3000 + case)
    x = wl.uniform(rng, (N, C, H, W), xb, xs)
    w = wl.uniform(rng, (M, C, KH, KW), wb, ws)
    xf, wf = samd.Fmt(xb, xs), samd.Fmt(wb, ws)
    want = ref.conv2d(x, w, shape)
    try:
        got = run_conv2d(x, w, shape, xf, wf)
    except samd.SamdError as e:
        # shapes without an exact lane geometry are refused, never computed wrongly
        assert e.status == -3, str(e)
        return
    np.testing.assert_array_equal(got, want, err_msg=f"{shape} x{xb}{'s' if xs else 'u'} w{wb}{'s' if ws else 'u'}")
    if case % 4 == 0:
        xp = samd.pack(gpu_vals(x, xs), xb, xs)
        wp = samd.pack(gpu_vals(w, ws), wb, ws)
        try:
            samd.conv2d_tune(xp, xf, wp, wf, shape, candidates=6, reps=1)
            y = samd.conv2d(xp, xf, wp, wf, shape)
            torch.cuda.synchronize()
            np.testing.assert_array_equal(y.cpu().numpy(), want)
        finally:
            samd.conv2d_untune(shape, xf, wf)


def random_epilogue_cases(n, seed):
    """Seeded (accumulator shape, next layer) pairs: the next layer's input is the
    accumulator (C = its channels, H x W = its size), any kernel 1..5, stride 1..2."""
    rng = np.random.default_rng(seed)
    out = []
    while len(out) < n:
        N, C = int(rng.integers(1, 3)), int(rng.integers(1, 40))
        H, W = int(rng.integers(3, 20)), int(rng.integers(3, 400))
        KH, KW = int(rng.integers(1, 6)), int(rng.integers(1, 6))
        sh, sw = int(rng.integers(1, 3)), int(rng.integers(1, 3))
        ph, pw = int(rng.integers(0, KH)), int(rng.integers(0, KW))
        if H + 2 * ph < KH or W + 2 * pw < KW:
            continue
        bits = int(rng.integers(1, 9))
        out.append(((N, C, H, W, int(rng.integers(1, 24)), KH, KW, sh, sw, ph, pw), bits))
    return out


EPILOGUE_CASES = random_epilogue_cases(16, 77)


@pytest.mark.parametrize("case", range(len(EPILOGUE_CASES)))
def test_fused_epilogue_random(case):
    """ReLU + requantisation written into the next layer's operand words, under the
    model's plan and under a tuned one, gives that layer's oracle result."""
    shape, bits = EPILOGUE_CASES[case]
    N, C, H, W, M, KH, KW = shape[:7]
    rng = np.random.default_rng(5000 + case)
    acc = rng.integers(-(1 << 20), 1 << 20, size=(N, C, H, W), dtype=np.int64).astype(np.int32)
    w = wl.uniform(rng, (M, C, KH, KW), bits, True)
    xf, wf = samd.Fmt(bits, False), samd.Fmt(bits, True)
    shift = ref.requant_shift(acc, bits)
    want = ref.conv2d(ref.relu_requant(acc, shift, bits), w, shape)
    acc_d = torch.from_numpy(acc).to(DEV)
    wp = samd.pack(gpu_vals(w, True), bits, True)
    try:
        for plan in (["model", "tuned"] if case % 2 == 0 else ["model"]):
            if plan == "tuned":
                xp = samd.pack(gpu_vals(ref.relu_requant(acc, shift, bits), False), bits, False)
                samd.conv2d_tune(xp, xf, wp, wf, shape, candidates=6, reps=1)
            ws = samd.conv2d_prepare(wp, wf, shape, xf)
            sh = torch.zeros(1, dtype=torch.int32, device=DEV)
            samd.relu_requant_stage(acc_d, samd.max_i32(acc_d), bits, wf, shape, ws, dev_shift=sh)
            y = samd.conv2d_accumulate(xf, wf, shape, ws)
            torch.cuda.synchronize()
            assert int(sh.item()) == shift
            np.testing.assert_array_equal(y.cpu().numpy(), want, err_msg=f"{shape} b={bits} {plan} plan")
    finally:
        samd.conv2d_untune(shape, xf, wf)
