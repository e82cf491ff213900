"""The allocation-free entry point samd_conv2d_noalloc, through the C ABI: bit-exact
against samd_conv2d (the same convolution with a caller workspace) on two calls in a
row, the second on a smaller layer, so the second call runs on whatever the first left
in the library's scratch array."""
import numpy as np
import pytest
import torch

import paper_1809_10572_amd as samd
import samd_workloads as wl
from oracle import reference as ref

pytestmark = pytest.mark.gpu
DEV = torch.device("cuda:0")


def packed(vals, bits, signed):
    t = torch.from_numpy(np.ascontiguousarray(vals).astype(np.int8 if signed else np.uint8)).to(DEV)
    return samd.pack(t, bits, signed)


@pytest.mark.parametrize("first,second", [((3, 8), (1, 4)), ((4, 5), (1, 2))])
def test_noalloc_matches_conv2d_twice(first, second):
    for cfg, bits in (first, second):
        case = wl.conv2d_case(cfg, bits)
        xf, wf = samd.Fmt(bits, case.x_signed), samd.Fmt(bits, case.w_signed)
        xp, wp = packed(case.x, bits, case.x_signed), packed(case.w, bits, case.w_signed)
        Ho, Wo = samd.out_hw(case.shape)
        y_ref = samd.conv2d(xp, xf, wp, wf, case.shape)
        y = torch.full((case.shape.N, case.shape.M, Ho, Wo), -7, dtype=torch.int32, device=DEV)
        samd.conv2d_noalloc(xp, xf, wp, wf, case.shape, out=y)
        torch.cuda.synchronize()
        got, want = y.cpu().numpy(), y_ref.cpu().numpy()
        np.testing.assert_array_equal(got, want, err_msg=f"config {cfg}, b={bits}")
        if cfg == 1:   # the small layer also against the oracle
            np.testing.assert_array_equal(got, ref.conv2d(case.x, case.w, case.shape.as_tuple()))


def test_noalloc_refuses_a_layer_beyond_the_scratch_array():
    # 16 x 512 x 55 x 55 -> 384 at 8 bits needs more than 64 MiB of operand words
    shape = wl.Conv2dShape(16, 512, 55, 55, 384, 3, 3, 1, 1, 1, 1)
    xf, wf = samd.Fmt(8, False), samd.Fmt(8, True)
    assert samd.conv2d_workspace(shape, xf, wf) > samd.NOALLOC_SCRATCH_BYTES
    xp = torch.zeros(16 * 512 * 55 * samd.row_words(55, 8), dtype=torch.int32, device=DEV)
    wp = torch.zeros(384 * 512 * 3 * samd.row_words(3, 8), dtype=torch.int32, device=DEV)
    y = torch.empty(16 * 384 * 55 * 55, dtype=torch.int32, device=DEV)
    with pytest.raises(samd.SamdError) as e:
        samd.conv2d_noalloc(xp, xf, wp, wf, shape, out=y)
    assert e.value.status == -6 and "scratch array" in str(e.value)
