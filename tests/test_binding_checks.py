"""The Python binding checks every tensor before the library sees it: the library takes
plain device pointers and cannot tell how large a buffer is or where it lives, so a
short or host-side tensor must raise here, before any kernel could read or write past
it.  These tests run on the CPU: chosen tensors are treated as device tensors and the
library is replaced by a recorder, so a call that got through would show up as a
recorded entry point."""
import pytest
import torch

import paper_1809_10572_amd as samd
from paper_1809_10572_amd import Fmt

SHAPE = (2, 3, 9, 20, 5, 3, 3, 1, 1, 1, 1)       # N C H W M KH KW sh sw ph pw
N, C, H, W, M, KH, KW = SHAPE[:7]
HO, WO = samd.out_hw(SHAPE)
XF, WF = Fmt(4, False), Fmt(4, True)


class Recorder:
    """Stands in for the library: row-word counts and status strings come from the
    real one, every other entry point only records that it was called."""

    def __init__(self, real):
        self.real, self.calls = real, []

    def __getattr__(self, name):
        if name in ("samd_row_words", "samd_status_str", "samd_last_error"):
            return getattr(self.real, name)

        def call(*args):
            self.calls.append((name, args))
            return samd.SAMD_OK
        return call


@pytest.fixture
def fake(monkeypatch):
    """Returns (t, rec): t(numel, dtype) makes a tensor that the binding takes for a
    device tensor (views of it too); tensors made any other way count as host memory."""
    rec = Recorder(samd.lib())
    gpu = set()

    def t(numel, dtype=torch.int32):
        x = torch.zeros(numel, dtype=dtype)
        gpu.add(x.untyped_storage().data_ptr())
        keep.append(x)
        return x
    keep = []
    monkeypatch.setattr(samd, "lib", lambda: rec)
    monkeypatch.setattr(samd, "_on_gpu", lambda x: x.untyped_storage().data_ptr() in gpu)
    monkeypatch.setattr(samd, "_stream", lambda x: 0)
    return t, rec


def xw(bits=XF.bits):
    return N * C * H * samd.row_words(W, bits)


def ww(bits=WF.bits):
    return M * C * KH * samd.row_words(KW, bits)


def outs():
    return N * M * HO * WO


def expect_refused(rec, fn, *args, **kw):
    before = len(rec.calls)
    with pytest.raises(ValueError):
        fn(*args, **kw)
    assert len(rec.calls) == before, f"{rec.calls[before][0]} was called"


def expect_passed(rec, fn, entry, *args, **kw):
    fn(*args, **kw)
    assert rec.calls and rec.calls[-1][0] == entry


def test_conv2d_entries_check_operand_sizes(fake):
    t, rec = fake
    ws, y = t(1 << 16, torch.uint8), t(outs())
    cases = [
        (samd.conv2d, "samd_conv2d", lambda x, w: ((x, XF, w, WF, SHAPE), dict(ws=ws, out=y))),
        (samd.conv2d_tune, "samd_conv2d_tune", lambda x, w: ((x, XF, w, WF, SHAPE), dict(ws=ws, out=y))),
    ]
    for fn, entry, make in cases:
        args, kw = make(t(xw()), t(ww()))
        expect_passed(rec, fn, entry, *args, **kw)
        args, kw = make(t(xw() - 1), t(ww()))
        expect_refused(rec, fn, *args, **kw)
        args, kw = make(t(xw()), t(ww() - 1))
        expect_refused(rec, fn, *args, **kw)
        args, kw = make(torch.zeros(xw(), dtype=torch.int32), t(ww()))      # host memory
        expect_refused(rec, fn, *args, **kw)
    expect_passed(rec, samd.conv2d_prepare, "samd_conv2d_prepare", t(ww()), WF, SHAPE, XF, ws=ws)
    expect_refused(rec, samd.conv2d_prepare, t(ww() - 1), WF, SHAPE, XF, ws=ws)
    for fn, entry in ((samd.conv2d_prepared, "samd_conv2d_prepared"), (samd.conv2d_stage, "samd_conv2d_stage")):
        kw = dict(out=y) if fn is samd.conv2d_prepared else {}
        expect_passed(rec, fn, entry, t(xw()), XF, WF, SHAPE, ws, **kw)
        expect_refused(rec, fn, t(xw() - 1), XF, WF, SHAPE, ws, **kw)


def test_workspaces_must_be_device_memory_and_count_bytes(fake):
    t, rec = fake
    y = t(outs())
    host_ws = torch.zeros(1 << 16, dtype=torch.uint8)
    expect_refused(rec, samd.conv2d, t(xw()), XF, t(ww()), WF, SHAPE, ws=host_ws, out=y)
    expect_refused(rec, samd.conv2d_accumulate, XF, WF, SHAPE, host_ws, out=y)
    expect_refused(rec, samd.conv2d_prepare, t(ww()), WF, SHAPE, XF, ws=host_ws)
    expect_refused(rec, samd.conv2d_int8_prepare, t(M * C * KH * KW, torch.int8), WF, SHAPE, XF, ws=host_ws)
    # a workspace of another dtype reports its size in bytes
    expect_passed(rec, samd.conv2d_accumulate, "samd_conv2d_accumulate", XF, WF, SHAPE, t(1000, torch.int32), out=y)
    assert rec.calls[-1][1][5] == 4000


def test_pointer_arguments_must_be_device_tensors(fake):
    t, rec = fake
    vals = t(64, torch.uint8).view(4, 16)
    expect_passed(rec, samd.pack, "samd_pack", vals, 4, False, oor=t(1))
    expect_refused(rec, samd.pack, vals, 4, False, oor=torch.zeros(1, dtype=torch.int32))
    expect_refused(rec, samd.pack, vals, 4, False, out=torch.zeros((4, 2), dtype=torch.int32))
    expect_refused(rec, samd.max_i32, t(100), out=torch.zeros(1, dtype=torch.int32))
    acc = t(N * C * H * W).view(N, C, H, W)
    packed = t(N * C * H * samd.row_words(W, 4)).view(N, C, H, -1)
    expect_passed(rec, samd.relu_requant_pack, "samd_relu_requant_pack", acc, t(1), 4, shift_out=t(1), out=packed)
    expect_refused(rec, samd.relu_requant_pack, acc, torch.zeros(1, dtype=torch.int32), 4, out=packed)
    expect_refused(rec, samd.relu_requant_pack, acc, t(1), 4, shift_out=torch.zeros(1, dtype=torch.int32), out=packed)
    expect_refused(rec, samd.relu_requant_pack, acc, t(1), 4, out=t(N * C * H * samd.row_words(W, 4) - 1))
    expect_passed(rec, samd.relu_requant_nhwc_u8, "samd_relu_requant_nhwc_u8", acc, t(1), 4,
                  out=t(N * C * H * W, torch.uint8))
    expect_refused(rec, samd.relu_requant_nhwc_u8, acc, t(1), 4, out=t(N * C * H * W - 1, torch.uint8))
    ws = t(1 << 16, torch.uint8)
    expect_passed(rec, samd.relu_requant_stage, "samd_relu_requant_stage", acc, t(1), 4, WF, SHAPE, ws, dev_shift=t(1))
    expect_refused(rec, samd.relu_requant_stage, t(N * C * H * W - 1), t(1), 4, WF, SHAPE, ws)
    expect_refused(rec, samd.relu_requant_stage, acc, t(1), 4, WF, SHAPE, ws,
                   dev_shift=torch.zeros(1, dtype=torch.int32))


def test_conv1d_unpack_and_int8_check_sizes(fake):
    t, rec = fake
    n, bits = 1000, 3
    y1 = t(n - 2)
    expect_passed(rec, samd.conv1d, "samd_conv1d", t(samd.row_words(n, bits)), n, bits, [1, 2, 3], bits, out=y1)
    expect_refused(rec, samd.conv1d, t(samd.row_words(n, bits) - 1), n, bits, [1, 2, 3], bits, out=y1)
    rw = samd.row_words(50, bits)
    expect_passed(rec, samd.unpack, "samd_unpack", t(4 * rw).view(4, rw), 50, bits, False)
    expect_refused(rec, samd.unpack, t(4 * (rw - 1)).view(4, rw - 1), 50, bits, False)
    xn, wn = N * H * W * C, M * C * KH * KW
    ws, y = t(1 << 16, torch.uint8), t(outs())
    expect_passed(rec, samd.conv2d_int8, "samd_conv2d_int8", t(xn, torch.uint8), XF, t(wn, torch.int8), WF, SHAPE,
                  ws=ws, out=y)
    expect_refused(rec, samd.conv2d_int8, t(xn - 1, torch.uint8), XF, t(wn, torch.int8), WF, SHAPE, ws=ws, out=y)
    expect_refused(rec, samd.conv2d_int8, t(xn, torch.uint8), XF, t(wn - 1, torch.int8), WF, SHAPE, ws=ws, out=y)
    expect_refused(rec, samd.conv2d_int8_prepared, t(xn - 1, torch.uint8), XF, WF, SHAPE, ws, out=y)
