"""The C ABI without a GPU: the library loads, exports every function include/*.h
declares, and rejects bad arguments on the host before any HIP call."""
import ctypes
import glob
import os
import re

import pytest

import paper_1809_10572_amd as samd
from paper_1809_10572_amd import Conv2dDesc, Fmt

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADERS = sorted(glob.glob(os.path.join(ROOT, "include", "*.h")))

OK, EINVAL, EALIGN, EUNSUP, EOVERFLOW, EHIP, ENOSPC = 0, -1, -2, -3, -4, -5, -6
MID = Conv2dDesc(8, 128, 56, 56, 128, 3, 3, 1, 1, 1, 1)
# fake device addresses: validation must reject before anything is dereferenced
P4, P1 = 0x10000, 0x10001


def declared_functions():
    names = set()
    for h in HEADERS:
        text = re.sub(r"/\*.*?\*/", "", open(h).read(), flags=re.S)
        names |= set(re.findall(r"\b(samd_[a-z0-9_]+)\s*\(", text))
    return sorted(names)


def test_library_exports_every_declared_function():
    assert any(h.endswith("samd.h") for h in HEADERS) and any(h.endswith("samd_peaks.h") for h in HEADERS)
    names = declared_functions()
    assert len(names) >= 16 and "samd_peak_launch" in names
    L = ctypes.CDLL(samd.LIB_PATH)
    for n in names:
        assert hasattr(L, n), n


def test_status_strings():
    L = samd.lib()
    for code in (OK, EINVAL, EALIGN, EUNSUP, EOVERFLOW, EHIP, ENOSPC):
        assert L.samd_status_str(code).startswith(b"SAMD_")
    assert L.samd_status_str(12345) == b"unknown SAMD status"


def test_row_words_and_format_checks():
    L = samd.lib()
    assert L.samd_row_words(56, Fmt(4, 0)) == 7 and L.samd_row_words(1 << 20, Fmt(3, 0)) == 104858
    assert L.samd_row_words(10, Fmt(0, 0)) == EINVAL and L.samd_row_words(10, Fmt(9, 1)) == EINVAL
    assert L.samd_row_words(-1, Fmt(4, 0)) == EINVAL
    raw = Fmt(4, 0)
    raw.is_signed = 2          # the ABI accepts only 0 or 1
    assert L.samd_row_words(10, raw) == EINVAL
    assert b"outside 1..8" in L.samd_last_error() or b"must be 0 or 1" in L.samd_last_error()


def test_pack_unpack_validation():
    L = samd.lib()
    assert L.samd_pack(P4, 2, 8, Fmt(9, 0), P4, None, None) == EINVAL
    assert L.samd_pack(None, 2, 8, Fmt(4, 0), P4, None, None) == EINVAL
    assert L.samd_pack(P4, 2, 8, Fmt(4, 0), P1, None, None) == EALIGN
    assert L.samd_pack(P4, 2, 8, Fmt(4, 0), P4, P1, None) == EALIGN
    assert L.samd_pack(P4, -1, 8, Fmt(4, 0), P4, None, None) == EINVAL
    assert L.samd_pack(None, 0, 8, Fmt(4, 0), None, None, None) == OK   # empty: nothing to do
    assert L.samd_unpack(P1, 2, 8, Fmt(4, 0), P4, None) == EALIGN
    assert L.samd_unpack(P4, 2, 8, Fmt(4, 0), None, None) == EINVAL


def test_conv1d_validation():
    L = samd.lib()
    taps = (ctypes.c_int32 * 3)(1, 2, 3)
    assert L.samd_conv1d(P4, 100, Fmt(4, 1), taps, 3, Fmt(4, 0), P4, None) == EINVAL     # signed input
    assert L.samd_conv1d(P4, 100, Fmt(4, 0), None, 3, Fmt(4, 0), P4, None) == EINVAL
    assert L.samd_conv1d(P4, 2, Fmt(4, 0), taps, 3, Fmt(4, 0), P4, None) == EINVAL        # n < K
    assert L.samd_conv1d(P4, 100, Fmt(4, 0), taps, 0, Fmt(4, 0), P4, None) == EINVAL
    bad = (ctypes.c_int32 * 3)(1, 16, 3)
    assert L.samd_conv1d(P4, 100, Fmt(4, 0), bad, 3, Fmt(4, 0), P4, None) == EINVAL       # tap too wide
    assert L.samd_conv1d(P1, 100, Fmt(4, 0), taps, 3, Fmt(4, 0), P4, None) == EALIGN
    # rows past 2^31 values are accepted (64-bit positions) up to 2^31 packed words
    plan = samd.conv1d_plan((1 << 31) + 1000, 8, [1, 2, 3], 8)
    assert plan.lanes >= 1
    with pytest.raises(samd.SamdError):
        samd.conv1d_plan(1 << 36, 1, [1], 1)          # 2^31 words of 1-bit values


def test_conv2d_validation():
    L = samd.lib()
    n = ctypes.c_size_t(0)
    assert L.samd_conv2d_workspace(ctypes.byref(MID), Fmt(4, 0), Fmt(4, 1), ctypes.byref(n)) == OK
    assert n.value > 0
    need = n.value
    args = lambda **kw: dict(dict(x=P4, xf=Fmt(4, 0), w=P4, wf=Fmt(4, 1), d=MID, y=P4, ws=P4 * 16, nb=need), **kw)

    def call(**kw):
        a = args(**kw)
        return L.samd_conv2d(a["x"], a["xf"], a["w"], a["wf"], ctypes.byref(a["d"]) if a["d"] else None, a["y"],
                             a["ws"], a["nb"], None)

    assert call(xf=Fmt(0, 0)) == EINVAL
    raw = Fmt(4, 0)
    raw.is_signed = 3
    assert call(wf=raw) == EINVAL
    assert call(d=None) == EINVAL
    assert call(d=Conv2dDesc(8, 0, 56, 56, 128, 3, 3, 1, 1, 1, 1)) == EINVAL
    assert call(d=Conv2dDesc(8, 128, 56, 56, 128, 3, 3, 0, 1, 1, 1)) == EINVAL
    assert call(d=Conv2dDesc(8, 128, 56, 56, 128, 3, 3, 1, 1, 3, 1)) == EINVAL      # pad >= kernel
    assert call(d=Conv2dDesc(1, 1, 2, 2, 1, 5, 5, 1, 1, 1, 1)) == EINVAL            # kernel > padded input
    assert call(x=None) == EINVAL
    assert call(y=P1) == EALIGN
    assert call(ws=P4 * 16 + 4) == EALIGN
    assert call(nb=need - 1) == ENOSPC
    # 8-bit x 8-bit over 256 channels of 3x3: 256*9*255*128 < 2^31, but 16x16 taps do not fit
    big = Conv2dDesc(1, 512, 16, 16, 1, 16, 16, 1, 1, 0, 0)
    assert call(d=big, xf=Fmt(8, 0), wf=Fmt(8, 1)) == EOVERFLOW
    assert b"does not fit int32" in L.samd_last_error()


def test_conv2d_stage_and_accumulate_validation():
    L = samd.lib()
    n = ctypes.c_size_t(0)
    assert L.samd_conv2d_workspace(ctypes.byref(MID), Fmt(2, 0), Fmt(2, 1), ctypes.byref(n)) == OK
    need = n.value
    assert L.samd_conv2d_stage(None, Fmt(2, 0), Fmt(2, 1), ctypes.byref(MID), P4 * 16, need, None) == EINVAL
    assert L.samd_conv2d_stage(P1, Fmt(2, 0), Fmt(2, 1), ctypes.byref(MID), P4 * 16, need, None) == EALIGN
    assert L.samd_conv2d_stage(P4, Fmt(2, 0), Fmt(2, 1), ctypes.byref(MID), P4 * 16, need - 1, None) == ENOSPC
    assert L.samd_conv2d_stage(P4, Fmt(9, 0), Fmt(2, 1), ctypes.byref(MID), P4 * 16, need, None) == EINVAL
    assert L.samd_conv2d_accumulate(Fmt(2, 0), Fmt(2, 1), ctypes.byref(MID), None, P4 * 16, need, None) == EINVAL
    assert L.samd_conv2d_accumulate(Fmt(2, 0), Fmt(2, 1), ctypes.byref(MID), P1, P4 * 16, need, None) == EALIGN
    assert L.samd_conv2d_accumulate(Fmt(2, 0), Fmt(2, 1), ctypes.byref(MID), P4, None, need, None) == EINVAL
    assert L.samd_conv2d_accumulate(Fmt(2, 0), Fmt(2, 1), None, P4, P4 * 16, need, None) == EINVAL


def test_conv2d_int8_validation():
    L = samd.lib()
    n = ctypes.c_size_t(0)
    assert L.samd_conv2d_int8_workspace(ctypes.byref(MID), Fmt(8, 0), ctypes.byref(n)) == OK and n.value > 0
    call = lambda xf=Fmt(8, 0), wf=Fmt(8, 1), y=P4, ws=P4 * 16, nb=n.value: L.samd_conv2d_int8(
        P4, xf, P4, wf, ctypes.byref(MID), y, ws, nb, None)
    assert call(wf=Fmt(8, 0)) == EINVAL          # unsigned 8-bit weights do not fit int8
    assert call(y=P1) == EALIGN
    assert call(nb=n.value - 1) == ENOSPC
    assert call(ws=P4 + 64) == EALIGN


def test_epilogue_validation():
    L = samd.lib()
    assert L.samd_max_i32(P4, 0, P4, None) == EINVAL
    assert L.samd_max_i32(P1, 10, P4, None) == EALIGN
    assert L.samd_relu_requant_pack(P4, 4, 4, P4, Fmt(4, 1), P4, None, None) == EINVAL   # signed output
    assert L.samd_relu_requant_pack(P4, 4, 4, None, Fmt(4, 0), P4, None, None) == EINVAL
    assert L.samd_relu_requant_nhwc_u8(P4, 1, 0, 1, 1, P4, Fmt(4, 0), P4, None) == EINVAL


def test_calls_fail_loudly_without_a_gpu_tensor():
    import torch
    with pytest.raises(ValueError):
        samd.pack(torch.zeros(4, dtype=torch.uint8), 4, False)


def test_lanewise_and_scale_validation():
    L = samd.lib()
    A16, A4 = 0x10000, 0x10004
    assert L.samd_lanewise(0, A16, A16, 8, Fmt(9, 0), A16, None) == EINVAL      # format
    assert L.samd_lanewise(3, A16, A16, 8, Fmt(4, 0), A16, None) == EINVAL      # scale is samd_scale
    assert L.samd_lanewise(-1, A16, A16, 8, Fmt(4, 0), A16, None) == EINVAL
    assert L.samd_lanewise(0, A16, A16, -1, Fmt(4, 0), A16, None) == EINVAL
    assert L.samd_lanewise(0, None, A16, 8, Fmt(4, 0), A16, None) == EINVAL
    assert L.samd_lanewise(0, A16, A4, 8, Fmt(4, 0), A16, None) == EALIGN
    assert L.samd_lanewise(1, None, None, 0, Fmt(4, 1), None, None) == OK       # empty: nothing to do
    assert L.samd_scale(A16, 8, Fmt(0, 0), 3, A16, None) == EINVAL
    assert L.samd_scale(A16, -2, Fmt(4, 0), 3, A16, None) == EINVAL
    assert L.samd_scale(A16, 8, Fmt(4, 0), 3, A4, None) == EALIGN
    assert L.samd_scale(None, 0, Fmt(4, 0), 3, None, None) == OK


def test_candidates_and_tune_validation():
    L = samd.lib()
    xf, wf = Fmt(4, 0), Fmt(4, 1)
    arr = (samd.Conv2dPlan * 8)()
    cnt = ctypes.c_int32(0)
    assert L.samd_conv2d_candidates(ctypes.byref(MID), xf, wf, 0, arr, ctypes.byref(cnt)) == EINVAL
    assert L.samd_conv2d_candidates(ctypes.byref(MID), xf, wf, samd.MAX_CANDIDATES + 1, arr,
                                    ctypes.byref(cnt)) == EINVAL
    assert L.samd_conv2d_candidates(ctypes.byref(MID), xf, wf, 8, None, ctypes.byref(cnt)) == EINVAL
    assert L.samd_conv2d_candidates(ctypes.byref(MID), Fmt(9, 0), wf, 8, arr, ctypes.byref(cnt)) == EINVAL
    assert L.samd_conv2d_candidates(ctypes.byref(MID), xf, wf, 8, arr, ctypes.byref(cnt)) == OK
    assert 1 <= cnt.value <= 8
    need = ctypes.c_size_t(0)
    assert L.samd_conv2d_tune_workspace(ctypes.byref(MID), xf, wf, 8, ctypes.byref(need)) == OK
    one = ctypes.c_size_t(0)
    assert L.samd_conv2d_workspace(ctypes.byref(MID), xf, wf, ctypes.byref(one)) == OK
    assert need.value >= one.value + 8 * 128 * 56 * 56 * 4      # the second output fits beside it

    def tune(**kw):
        a = dict(dict(x=P4, w=P4, y=P4, ws=P4 * 16, nb=need.value, cands=8, reps=3, d=MID, xf=xf, wf=wf), **kw)
        return L.samd_conv2d_tune(a["x"], a["xf"], a["w"], a["wf"], ctypes.byref(a["d"]), a["y"], a["ws"], a["nb"],
                                  a["cands"], a["reps"], None, None)

    # every rejection happens on the host, before anything is dereferenced or launched
    assert tune(x=None) == EINVAL
    assert tune(ws=None) == EINVAL
    assert tune(cands=0) == EINVAL
    assert tune(reps=0) == EINVAL
    assert tune(reps=1001) == EINVAL
    assert tune(y=P1) == EALIGN
    assert tune(ws=P4 * 16 + 64) == EALIGN
    assert tune(nb=one.value) == ENOSPC
    assert tune(d=Conv2dDesc(1, 512, 16, 16, 1, 16, 16, 1, 1, 0, 0), xf=Fmt(8, 0), wf=Fmt(8, 1)) == EOVERFLOW
    assert L.samd_conv2d_untune(None, Fmt(0, 0), Fmt(0, 0)) == OK       # all shapes: formats ignored
    assert L.samd_conv2d_untune(ctypes.byref(MID), Fmt(0, 0), wf) == EINVAL
    assert L.samd_conv2d_untune(ctypes.byref(MID), xf, wf) == OK


@pytest.mark.parametrize("bits", [1, 4, 8])
def test_candidates_rank_the_planner_choice_first(bits):
    # the planner's own plan leads the list; the rest are distinct shapes priced no lower
    shape = (8, 128, 56, 56, 128, 3, 3, 1, 1, 1, 1)
    xf, wf = Fmt(bits, 0), Fmt(bits, 1)
    plan = samd.conv2d_plan(shape, xf, wf)
    cands = samd.conv2d_candidates(shape, xf, wf, 16)
    key = lambda p: (p.lane_bits, p.lanes, p.x_offset, p.shared_rows, p.rows_per_thread, p.rows_per_block,
                     p.mblock, p.split_waves)
    assert key(cands[0]) == key(plan)
    assert len(set(map(key, cands))) == len(cands)
    assert all(c.model_cost >= cands[0].model_cost for c in cands[1:])
    assert [c.model_cost for c in cands[1:]] == sorted(c.model_cost for c in cands[1:])


def test_use_plan_installs_a_candidate():
    shape = (2, 24, 17, 45, 20, 3, 3, 1, 1, 1, 1)
    xf, wf = Fmt(5, 0), Fmt(5, 1)
    model = samd.conv2d_plan(shape, xf, wf)
    cands = samd.conv2d_candidates(shape, xf, wf, 8)
    try:
        for c in cands[1:4]:
            samd.conv2d_use_plan(shape, xf, wf, samd.plan_key(c))
            assert samd.plan_key(samd.conv2d_plan(shape, xf, wf)) == samd.plan_key(c)
            assert samd.conv2d_workspace(shape, xf, wf) > 0
        bogus = dict(samd.plan_key(model), split_waves=3)
        with pytest.raises(samd.SamdError):
            samd.conv2d_use_plan(shape, xf, wf, bogus)
    finally:
        samd.conv2d_untune(shape, xf, wf)
    assert samd.plan_key(samd.conv2d_plan(shape, xf, wf)) == samd.plan_key(model)
    L = samd.lib()
    assert L.samd_conv2d_use_plan(ctypes.byref(MID), xf, wf, None) == EINVAL


def test_peak_validation():
    L = samd.lib()
    f = L.samd_peak_launch
    f.restype, f.argtypes = ctypes.c_int, [ctypes.c_int, ctypes.c_int64, ctypes.c_int32, ctypes.c_void_p,
                                           ctypes.c_void_p, ctypes.c_int64, ctypes.c_void_p]
    assert f(9, 1, 1, None, P4, 0, None) == EINVAL            # unknown kind
    assert f(0, 0, 1, None, P4, 0, None) == EINVAL            # no trips
    assert f(0, 1, 0, None, P4, 0, None) == EINVAL            # no workgroups
    assert f(0, 1, 1, None, None, 0, None) == EINVAL          # no output
    assert f(3, 1, 1, None, P4, 1024, None) == EINVAL         # copy without a source
    assert f(3, 1, 1, P4, P4, 1000, None) == EINVAL           # not a multiple of 16 bytes
    assert f(3, 1, 1, P4 + 4, P4, 1024, None) == EALIGN       # misaligned source
    assert samd.peak_work(0, 10, 2) == 2 * 256 * 10 * 8
    assert samd.peak_work(2, 10, 2) == 2 * 4 * 10 * 4 * 16 * 16 * 64
    assert samd.peak_work(3, 1, 1, 1 << 20) == 2 * (1 << 20)


def test_planner_keeps_kernel_word_slices_within_32_bit_offsets():
    # 3x3 layer with 10^8 one-bit channels: a single wave slice of every channel would
    # index 2.4e9 kernel words; every listed candidate must split the channels enough
    d = Conv2dDesc(1, 100_000_000, 1, 1, 8, 3, 3, 1, 1, 1, 1)
    for p in samd.conv2d_candidates(d, Fmt(1, False), Fmt(1, False), 64):
        cpw = -(-d.C // p.split_waves)
        assert (cpw * d.KH * p.tap_words + 6) * 8 < 2 ** 31, (p.split_waves, p.tap_words)


def test_planner_refuses_a_spread_of_2_to_the_32_threads():
    # 2^24 padded rows of 651 operand words (8-bit lanes, two values per word) would need
    # 2^32 spread threads: refused by the planner, before any HIP call
    d = Conv2dDesc(65536, 8, 30, 1300, 8, 3, 3, 1, 1, 1, 1)
    L = samd.lib()
    plan = samd.Conv2dPlan()
    st = L.samd_conv2d_plan_query(ctypes.byref(d), Fmt(8, False), Fmt(8, True), ctypes.byref(plan))
    assert st == EUNSUP, st
    assert b"index ranges" in L.samd_last_error()
    n = ctypes.c_size_t(0)
    assert L.samd_conv2d_workspace(ctypes.byref(d), Fmt(8, False), Fmt(8, True), ctypes.byref(n)) == EUNSUP


def test_int8_halo_tiles_cover_every_kernel():
    """The int8 layers of the GPU tests, with all their candidate launches, reach both
    kernels, every halo tile shape, both tile modes and both channel steps (host-only
    queries of the launches the library makes)."""
    import sys
    sys.path.insert(0, os.path.join(ROOT, "tests"))
    import samd_workloads as wl
    from test_gpu_parity import HALO
    seen = set()
    for shape in HALO:
        cands = samd.conv2d_int8_candidates(shape, Fmt(8, False), Fmt(8, True))
        assert cands and cands[-1].halo == 0
        for p in cands:
            kc = 64 if shape.C <= 64 else 128
            seen.add((p.halo, p.mtile, p.positions, p.row_segments, kc if p.halo else 0))
            if p.halo:
                assert p.lds_bytes <= 160 * 1024 and p.workgroups >= 1
        # the library's own choice is one of the candidates
        own = samd.conv2d_int8_plan(shape, Fmt(8, False), Fmt(8, True))
        assert any((own.halo, own.mtile, own.positions) == (c.halo, c.mtile, c.positions) for c in cands)
    assert {(1, 128, 128), (1, 128, 64), (1, 64, 128), (1, 64, 64)} <= {k[:3] for k in seen}, seen
    # weight-resident launches (32 filters per workgroup) for 3x3 and 1x1 layers of 1 to 4
    # blocks of 64 input channels (whole K in registers up to 128 padded channels, K in
    # chunks of 64 channels above)
    res = {(sh.KH, -(-sh.C // 64)) for sh in HALO
           for p in samd.conv2d_int8_candidates(sh, Fmt(8, False), Fmt(8, True)) if p.halo == 2}
    assert {(3, 1), (3, 2), (3, 3), (3, 4), (1, 1), (1, 2)} <= res, res
    # above 128 padded channels both chunk widths (128 and 64 channels), for 3x3 and 1x1
    widths = set()
    for sh in HALO:
        cp = -(-sh.C // 128) * 128
        if cp <= 128:
            continue
        for p in samd.conv2d_int8_candidates(sh, Fmt(8, False), Fmt(8, True)):
            if p.halo != 2:
                continue
            rows = min(sh.H, (p.positions - 1) // sh.W + 2) + sh.KH - 1
            pixels = rows * (sh.W + sh.KW - 1)
            kc = [k for k in (64, 128)
                  if p.lds_bytes == 2 * ((pixels * (k + 16) + 15) // 16 * 16 + 32 * sh.KH * sh.KW * k) + 32 * 4]
            assert len(kc) == 1, (sh, p)
            widths.add((sh.KH, kc[0]))
    assert widths == {(3, 64), (3, 128), (1, 64), (1, 128)}, widths
    mid = samd.conv2d_int8_candidates(wl.MID, Fmt(8, False), Fmt(8, True))
    assert [(p.mtile, p.positions, p.waves, p.workgroups) for p in mid if p.halo == 2] == [(32, 400, 8, 256),
                                                                                          (32, 208, 8, 512)]
    assert {(0, 128, 64), (0, 128, 32)} <= {k[:3] for k in seen}
    assert {0, 1} <= {k[3] for k in seen if k[0] == 1}
    assert {64, 128} <= {k[4] for k in seen if k[0] == 1}
    im2col_only = wl.Conv2dShape(1, 16, 20, 80, 16, 11, 11, 1, 1, 5, 5)
    assert im2col_only in HALO
    assert not any(c.halo for c in samd.conv2d_int8_candidates(im2col_only, Fmt(8, False), Fmt(8, True)))
    # the mid-size layer, the extremes-heavy layer (256 channels) and VGG-B's 3x3 layers of
    # 64 to 512 channels take the weight-resident kernel
    for shape in [wl.MID, wl.STRESS] + list(wl.VGGB_LAYERS[2:]):
        assert samd.conv2d_int8_plan(shape, Fmt(8, False), Fmt(8, True)).halo == 2, shape
    # strided layers and channel counts that are not a multiple of 16 take the packed-row
    # kernel where it at least halves the k-blocks (16 or 24 channels at 3x3), else im2col
    assert samd.conv2d_int8_plan(wl.Conv2dShape(1, 16, 9, 9, 8, 3, 3, 2, 2, 1, 1), Fmt(8, 1), Fmt(8, 1)).halo == 3
    assert samd.conv2d_int8_plan(wl.Conv2dShape(1, 24, 9, 9, 8, 3, 3, 1, 1, 1, 1), Fmt(8, 1), Fmt(8, 1)).halo == 3
    assert samd.conv2d_int8_plan(wl.Conv2dShape(1, 40, 9, 9, 8, 3, 3, 2, 2, 1, 1), Fmt(8, 1), Fmt(8, 1)).halo == 0


def test_int8_packed_rows():
    """The packed-row launches: K laid out by kernel row (ceil(KW*C / 16) slots of 16
    bytes per row, four slots per k-block), offered where that at least halves the
    k-blocks of the 64-channel layout and the activations are whole 4-byte words; the
    group's fragments (up to 8 blocks of 16 filters x k-blocks x 1 KB) in LDS; the
    workspace grows by the packed fragments.  LDS: the fragments, then 8 x 16 zero-point
    corrections of 4 bytes."""
    import samd_workloads as wl
    xf, wf = Fmt(8, False), Fmt(8, True)

    def packed(shape):
        return [(p.mtile, p.positions, p.lds_bytes, p.workgroups)
                for p in samd.conv2d_int8_candidates(shape, xf, wf) if p.halo == 3]
    # VGG-B layer 1: 3x3 on 3 channels = 9 bytes per row, one slot each, one k-block;
    # 224 x 224 positions = 3136 tiles of 16, 4, 2 or 1 per wave and 4 waves
    assert packed(wl.VGGB_LAYERS[0]) == [(64, 256, 4 * 1024 + 512, 196), (64, 128, 4 * 1024 + 512, 392),
                                         (64, 64, 4 * 1024 + 512, 784)]
    # AlexNet layer 1: 11x11 stride 4 on 3 channels = 33 bytes per row, 3 slots, 33 slots =
    # 9 k-blocks (against 121); 96 filters = 6 blocks; 16 images of 55 x 55 = 16 x 190 tiles
    assert packed(wl.ALEXNET_LAYERS[0]) == [(96, 256, 6 * 9 * 1024 + 512, 190), (96, 128, 6 * 9 * 1024 + 512, 380),
                                            (96, 64, 6 * 9 * 1024 + 512, 760)]
    for shape in (wl.VGGB_LAYERS[0], wl.ALEXNET_LAYERS[0]):
        assert samd.conv2d_int8_plan(shape, xf, wf).halo == 3
    # 200 filters: two workgroup rows (8 + 5 blocks), LDS for 8
    assert packed(Conv2dDesc(1, 3, 8, 8, 200, 3, 3, 1, 1, 1, 1))[0][2:] == (8 * 1024 + 512, 2)
    # 64 channels, 1x1 layers and 32 channels at 3x3 keep the 64-channel layout
    assert not packed(wl.MID) and not packed(Conv2dDesc(1, 16, 8, 8, 8, 1, 1, 1, 1, 0, 0))
    assert not packed(Conv2dDesc(1, 32, 8, 8, 8, 3, 3, 1, 1, 1, 1))
    # activations not a whole number of words (3 x 9 x 9 bytes)
    assert not packed(Conv2dDesc(1, 3, 9, 9, 8, 3, 3, 1, 1, 1, 1))
    n = ctypes.c_size_t(0)
    d = Conv2dDesc(*wl.VGGB_LAYERS[0].as_tuple())
    assert samd.lib().samd_conv2d_int8_workspace(ctypes.byref(d), xf, ctypes.byref(n)) == OK
    a256 = lambda v: -(-v // 256) * 256
    assert n.value == a256(128 * 9 * 64) + a256(64 * 16 * 4) + a256(4 * 1 * 1024)


def test_int8_resident_bounds():
    """The weight-resident launches are offered only where their 32-bit offsets and
    register-held chunks hold: not for activations of 2^31 bytes or more, not past 512
    channels, not for strided or 5x5 layers."""
    def resident(shape):
        return [p for p in samd.conv2d_int8_candidates(shape, Fmt(8, False), Fmt(8, True)) if p.halo == 2]
    assert resident(Conv2dDesc(1, 512, 14, 14, 64, 3, 3, 1, 1, 1, 1))
    assert not resident(Conv2dDesc(1, 576, 14, 14, 64, 3, 3, 1, 1, 1, 1))       # 640 padded channels
    assert not resident(Conv2dDesc(1, 64, 14, 14, 64, 3, 3, 2, 2, 1, 1))        # stride 2
    assert not resident(Conv2dDesc(1, 64, 14, 14, 64, 5, 5, 1, 1, 2, 2))        # 5x5
    assert resident(Conv2dDesc(2, 64, 128, 128, 64, 3, 3, 1, 1, 1, 1))
    assert not resident(Conv2dDesc(2048, 64, 128, 128, 64, 3, 3, 1, 1, 1, 1))   # 2^31 bytes of activations


def test_int8_resident_chunk_width():
    """Layers of 256-512 padded channels walk K in 128-channel chunks where a chunk's halo
    fits six 16-byte pieces per thread and two chunks fit 160 KB of LDS, else in 64-channel
    chunks: each chunk buffer holds the halo (pixels x (chunk + 16) bytes) and 32 filters'
    weights of the chunk (32 x 9 x chunk bytes), two buffers alternate, and the 32
    filters' zero-point corrections (4 bytes each) follow them."""
    import samd_workloads as wl

    def lds(pixels, kc):
        return 2 * ((pixels * (kc + 16) + 15) // 16 * 16 + 32 * 9 * kc) + 32 * 4

    def resident(shape):
        return {p.positions: p.lds_bytes
                for p in samd.conv2d_int8_candidates(shape, Fmt(8, False), Fmt(8, True)) if p.halo == 2}
    # 28-wide rows: 112 positions read 5 + 2 halo rows of 30 columns, 64 read 4 + 2
    assert resident(wl.STRESS) == {112: lds(7 * 30, 128), 64: lds(6 * 30, 128)}
    # 56-wide rows: 112 or 64 positions read 3 + 2 rows of 58 columns (290 pixels, 157 KB)
    assert resident(wl.VGGB_LAYERS[5]) == {112: lds(5 * 58, 128), 64: lds(5 * 58, 128)}
    # 112-wide rows: 208 positions read 3 + 2 rows of 114 columns, 570 pixels: too many
    # for 128-channel chunks (8 pieces each), 64-channel ones fit; 400 positions fit neither
    assert resident(Conv2dDesc(1, 256, 112, 112, 256, 3, 3, 1, 1, 1, 1)) == {208: lds(5 * 114, 64)}


def test_int8_use_plan_installs_and_reverts():
    import samd_workloads as wl
    xf, wf = Fmt(8, False), Fmt(8, True)
    own = samd.conv2d_int8_plan(wl.MID, xf, wf)
    cands = samd.conv2d_int8_candidates(wl.MID, xf, wf)
    other = [c for c in cands if (c.halo, c.mtile, c.positions) != (own.halo, own.mtile, own.positions)][0]
    try:
        samd.conv2d_int8_use_plan(wl.MID, xf, wf, other)
        p = samd.conv2d_int8_plan(wl.MID, xf, wf)
        assert (p.halo, p.mtile, p.positions) == (other.halo, other.mtile, other.positions)
        bad = samd.Conv2dInt8Plan(1, 48, 64, 0, 0, 0)
        with pytest.raises(samd.SamdError):
            samd.conv2d_int8_use_plan(wl.MID, xf, wf, bad)
    finally:
        samd.conv2d_int8_use_plan(wl.MID, xf, wf, None)
    p = samd.conv2d_int8_plan(wl.MID, xf, wf)
    assert (p.halo, p.mtile, p.positions) == (own.halo, own.mtile, own.positions)


def test_noalloc_validation_before_any_hip_call():
    L = samd.lib()
    f = L.samd_conv2d_noalloc
    x8, w8 = Fmt(8, False), Fmt(8, True)
    assert f(P4, x8, P4, w8, None, P4, None) == EINVAL
    assert f(None, x8, P4, w8, ctypes.byref(MID), P4, None) == EINVAL
    assert f(P1, x8, P4, w8, ctypes.byref(MID), P4, None) == EALIGN
    assert f(P4, Fmt(9, 0), P4, w8, ctypes.byref(MID), P4, None) == EINVAL
    big = Conv2dDesc(16, 512, 55, 55, 384, 3, 3, 1, 1, 1, 1)   # workspace beyond the 64 MiB array
    assert f(P4, x8, P4, w8, ctypes.byref(big), P4, None) == ENOSPC
    assert b"scratch array" in L.samd_last_error()


def test_spaced_validation_before_any_hip_call():
    L = samd.lib()
    x8, w8 = Fmt(8, False), Fmt(8, True)
    d = ctypes.byref(MID)
    assert L.samd_conv2d_spaced(P4, x8, w8, None, P4, P4, 1 << 30, None) == EINVAL
    assert L.samd_conv2d_spaced(None, x8, w8, d, P4, P4, 1 << 30, None) == EINVAL
    assert L.samd_conv2d_spaced(P1, x8, w8, d, P4, P4, 1 << 30, None) == EALIGN
    assert L.samd_conv2d_spaced(P4, x8, w8, d, P4, 0x10010, 1 << 30, None) == EALIGN   # workspace alignment
    assert L.samd_conv2d_spaced(P4, x8, w8, d, P4, P4, 256, None) == ENOSPC
    assert L.samd_conv2d_spaced_pack(None, x8, w8, d, P4, None) == EINVAL
    assert L.samd_conv2d_spaced_pack(P4, x8, w8, d, P1, None) == EALIGN
    assert L.samd_conv2d_spaced_from_packed(P1, x8, w8, d, P4, None) == EALIGN
    assert L.samd_conv2d_spaced_prepare(None, w8, d, x8, P4, 1 << 30, None) == EINVAL
    assert L.samd_relu_requant_spaced(P4, P4, Fmt(8, 1), w8, d, P4, None, None) == EINVAL   # signed activations
    assert L.samd_relu_requant_spaced(P4, P4, x8, w8, d, P1, None, None) == EALIGN
    assert L.samd_conv2d_spaced_pack(P4, Fmt(0, 0), w8, d, P4, None) == EINVAL
    big = Conv2dDesc(1, 512, 16, 16, 1, 16, 16, 1, 1, 0, 0)
    assert L.samd_conv2d_spaced_pack(P4, x8, w8, ctypes.byref(big), P4, None) == EOVERFLOW


@pytest.mark.parametrize("bits", range(1, 9))
def test_spaced_layout_and_workspace(bits):
    import samd_workloads as wl
    xf, wf = Fmt(bits, False), Fmt(bits, True)
    lay = samd.conv2d_spaced_layout(wl.MID, xf, wf)
    plan = samd.conv2d_spaced_plan(wl.MID, xf, wf)
    assert (lay.lane_bits, lay.lanes, lay.words_per_row, lay.tap_words) == \
        (plan.lane_bits, plan.lanes, plan.words_per_row, plan.tap_words)
    d = wl.MID
    assert lay.padded_rows == d.H + 2 * d.pad_h
    assert lay.words == (d.N * d.C + 1) * lay.padded_rows * lay.tap_words * lay.words_per_row
    assert plan.layout_spaced == 1
    assert samd.conv2d_spaced_workspace(d, xf, wf) < samd.conv2d_workspace(d, xf, wf)
    # unsigned results need no fix-up, so no spacer bit
    assert samd.conv2d_spaced_plan(d, xf, Fmt(bits, False)).spacer_msb == 0
    # signed results: the candidates include plans with and without the spacer MSB, and a
    # spacer MSB never holds more channels per decode than the same lanes without it
    cands = samd.conv2d_candidates(d, xf, wf, 64)
    assert all(c.layout_spaced == 0 and c.spacer_msb == 0 for c in cands)
