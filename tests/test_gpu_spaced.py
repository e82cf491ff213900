"""GPU parity of the permanent-spacer layout (include/samd.h, "Permanent-spacer
activations"; the paper's permanent spacer bits, Sec. 2.2, and their optimisations,
Sec. 6.1): the layout's words against their definition, and every convolution from the
layout against the oracle, bit-exact."""
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


def spaced_words_by_definition(x, shape, xf, wf):
    """The layout's words from its definition: word q of kernel-word variant t of padded
    row hp of channel c of image n is sum_i (v - x_offset) 2^(i L) as a signed 32-bit
    integer, v the activation in row hp - pad_h, column sw (q I + delta_t + i) + phase_t -
    pw, 0 outside the image (rows and columns of the zero padding)."""
    lay = samd.conv2d_spaced_layout(shape, xf, wf)
    plan = samd.conv2d_spaced_plan(shape, xf, wf)
    N, C, H, W = x.shape
    L, I, nq, ntw, Hp, xoff = lay.lane_bits, lay.lanes, lay.words_per_row, lay.tap_words, lay.padded_rows, lay.x_offset
    padded = np.zeros((N, C, Hp, W), dtype=np.int64)
    padded[:, :, shape.pad_h:shape.pad_h + H, :] = x.astype(np.int64) - xoff
    inside_rows = np.zeros(Hp, dtype=bool)
    inside_rows[shape.pad_h:shape.pad_h + H] = True
    words = np.zeros((N, C, Hp, ntw, nq), dtype=np.int64)
    for t in range(ntw):
        delta = plan.tap0[t] + plan.ntaps[t] - plan.taps_max
        for q in range(nq):
            acc = np.zeros((N, C, Hp), dtype=np.int64)
            for i in range(I):
                col = shape.stride_w * (q * I + delta + i) + plan.phase[t] - shape.pad_w
                if 0 <= col < W:
                    acc += padded[:, :, :, col] << (i * L)
            words[:, :, :, t, q] = np.where(inside_rows[None, None, :], acc, 0)
    flat = words.reshape(-1)
    assert np.all(flat >= -(1 << 31)) and np.all(flat < (1 << 31))
    return flat.astype(np.int32), lay


LAYOUT_SHAPES = [
    wl.Conv2dShape(2, 3, 5, 61, 4, 3, 3, 1, 1, 1, 1),
    wl.Conv2dShape(1, 5, 17, 19, 8, 3, 3, 2, 2, 1, 1),      # stride 2: two phases
    wl.Conv2dShape(1, 4, 12, 12, 16, 5, 5, 1, 1, 2, 2),     # 5x5
    wl.Conv2dShape(1, 2, 9, 30, 4, 3, 5, 1, 2, 1, 2),       # asymmetric
    wl.Conv2dShape(1, 3, 7, 150, 5, 3, 3, 1, 1, 1, 1),      # rows of more than 64 operand words
]
FORMATS = [(1, 0, 1, 1), (2, 1, 2, 1), (4, 0, 4, 1), (5, 0, 3, 0), (8, 0, 8, 1), (7, 1, 7, 1), (3, 0, 3, 0)]


@pytest.mark.parametrize("shape", LAYOUT_SHAPES, ids=lambda s: "x".join(map(str, s.as_tuple())))
@pytest.mark.parametrize("bx,sx,bw,sw", FORMATS)
def test_spaced_layout_matches_its_definition(shape, bx, sx, bw, sw):
    xf, wf = samd.Fmt(bx, sx), samd.Fmt(bw, sw)
    rng = np.random.default_rng(31 * bx + sw)
    x = wl.uniform(rng, (shape.N, shape.C, shape.H, shape.W), bx, bool(sx))
    want, lay = spaced_words_by_definition(x, shape, xf, wf)
    got = samd.conv2d_spaced_pack(gpu_vals(x, sx), xf, wf, shape)
    got2 = samd.conv2d_spaced_from_packed(samd.pack(gpu_vals(x, sx), bx, bool(sx)), xf, wf, shape)
    torch.cuda.synchronize()
    n = want.size   # the spare channel after the last image is not part of the definition
    assert lay.words == n + lay.padded_rows * lay.tap_words * lay.words_per_row
    np.testing.assert_array_equal(got.cpu().numpy()[:n], want)
    np.testing.assert_array_equal(got2.cpu().numpy()[:n], want)


def run_spaced(x, w, shape, xf, wf, from_packed=False):
    xs = gpu_vals(x, xf.is_signed)
    wp = samd.pack(gpu_vals(w, wf.is_signed), wf.bits, wf.is_signed)
    if from_packed:
        spaced = samd.conv2d_spaced_from_packed(samd.pack(xs, xf.bits, xf.is_signed), xf, wf, shape)
    else:
        spaced = samd.conv2d_spaced_pack(xs, xf, wf, shape)
    ws = samd.conv2d_spaced_prepare(wp, wf, shape, xf)
    y = samd.conv2d_spaced(spaced, xf, wf, shape, ws)
    torch.cuda.synchronize()
    return y.cpu().numpy()


def spaced_full(cfg, bits):
    case = wl.conv2d_case(cfg, bits)
    xf, wf = samd.Fmt(bits, case.x_signed), samd.Fmt(bits, case.w_signed)
    return case, xf, wf, ref.conv2d(case.x, case.w, case.shape.as_tuple())


@pytest.mark.parametrize("bits", range(1, 9))
def test_spaced_single_layer(bits):
    case, xf, wf, want = spaced_full(1, bits)
    np.testing.assert_array_equal(run_spaced(case.x, case.w, case.shape, xf, wf), want)


@pytest.mark.parametrize("bits", range(1, 9))
def test_spaced_mid_layer_full(bits):
    case, xf, wf, want = spaced_full(3, bits)
    plan = samd.conv2d_spaced_plan(case.shape, xf, wf)
    assert plan.layout_spaced == 1
    np.testing.assert_array_equal(run_spaced(case.x, case.w, case.shape, xf, wf, from_packed=bits % 2 == 0), want)


@pytest.mark.parametrize("bits", wl.BITS_SWEEP[4])
def test_spaced_stress_layer_full(bits):
    case, xf, wf, want = spaced_full(4, bits)
    np.testing.assert_array_equal(run_spaced(case.x, case.w, case.shape, xf, wf), want)


EDGE = [
    wl.Conv2dShape(1, 1, 1, 1, 1, 1, 1),
    wl.Conv2dShape(1, 1, 1, 7, 1, 1, 3, 1, 1, 0, 1),
    wl.Conv2dShape(1, 9, 13, 13, 33, 3, 3, 1, 1, 0, 0),
    wl.Conv2dShape(2, 3, 45, 47, 20, 11, 11, 4, 4, 2, 2),
    wl.Conv2dShape(1, 300, 6, 6, 70, 3, 3, 1, 1, 1, 1),
    wl.Conv2dShape(3, 16, 8, 120, 48, 1, 1, 1, 1, 0, 0),
    wl.Conv2dShape(1, 8, 130, 9, 16, 3, 3, 1, 1, 1, 1),
    wl.Conv2dShape(2, 5, 6, 300, 12, 3, 3, 1, 1, 1, 1),
    wl.Conv2dShape(1, 3, 7, 700, 9, 3, 5, 2, 2, 1, 2),
]


@pytest.mark.parametrize("shape", EDGE, ids=lambda s: "x".join(map(str, s.as_tuple())))
@pytest.mark.parametrize("bx,sx,bw,sw", FORMATS)
def test_spaced_edges(shape, bx, sx, bw, sw):
    rng = np.random.default_rng(bx * 10 + bw)
    x = wl.half_extremes(rng, (shape.N, shape.C, shape.H, shape.W), bx, bool(sx))
    w = wl.half_extremes(rng, (shape.M, shape.C, shape.KH, shape.KW), bw, bool(sw))
    xf, wf = samd.Fmt(bx, sx), samd.Fmt(bw, sw)
    np.testing.assert_array_equal(run_spaced(x, w, shape, xf, wf), ref.conv2d(x, w, shape.as_tuple()))


@pytest.mark.parametrize("bits", [2, 4, 8])
def test_spaced_stack_chain(bits):
    """The AlexNet-shaped stack at batch 2 with the activations in the permanent-spacer
    layout from the input to the last layer: ReLU + requantisation write each next
    layer's spaced words directly; every layer's output against the oracle."""
    case = wl.stack_case(bits, batch=2)
    xf, wf = samd.Fmt(bits, False), samd.Fmt(bits, True)
    accs, _, shifts = ref.stack(case.x, case.ws, [l.as_tuple() for l in case.layers], bits)
    spaced = samd.conv2d_spaced_pack(gpu_vals(case.x, False), xf, wf, case.layers[0])
    mx = torch.empty(1, dtype=torch.int32, device=DEV)
    sh = torch.empty(1, dtype=torch.int32, device=DEV)
    for li, (l, w) in enumerate(zip(case.layers, case.ws)):
        wp = samd.pack(gpu_vals(w, True), bits, True)
        ws = samd.conv2d_spaced_prepare(wp, wf, l, xf)
        y = samd.conv2d_spaced(spaced, xf, wf, l, ws)
        torch.cuda.synchronize()
        np.testing.assert_array_equal(y.cpu().numpy(), accs[li], err_msg=f"layer {li + 1}")
        if li + 1 < len(case.layers):
            samd.max_i32(y, out=mx)
            spaced = samd.relu_requant_spaced(y, mx, bits, wf, case.layers[li + 1], dev_shift=sh)
            torch.cuda.synchronize()
            assert int(sh.item()) == shifts[li]


@pytest.mark.parametrize("cfg,bits", [(3, 4), (4, 6), (1, 3)])
def test_spaced_tune_keeps_results_exact(cfg, bits):
    case, xf, wf, want = spaced_full(cfg, bits)
    xp = samd.pack(gpu_vals(case.x, case.x_signed), bits, case.x_signed)
    wp = samd.pack(gpu_vals(case.w, case.w_signed), bits, case.w_signed)
    try:
        chosen = samd.conv2d_spaced_tune(xp, xf, wp, wf, case.shape, candidates=8, reps=2)
        plan = samd.conv2d_spaced_plan(case.shape, xf, wf)
        assert samd.plan_key(plan) == samd.plan_key(chosen) and plan.layout_spaced == 1
        np.testing.assert_array_equal(run_spaced(case.x, case.w, case.shape, xf, wf), want)
    finally:
        samd.conv2d_untune(case.shape, xf, wf)
    # untuning returns the layout to the model's plan, still exact
    np.testing.assert_array_equal(run_spaced(case.x, case.w, case.shape, xf, wf), want)
