"""The C-ABI library without a GPU: it loads, exports every symbol that
include/dqt.h declares, its host helpers match the oracle, and argument checks
reject bad calls before anything is launched (no compute call is made)."""
import ctypes
import os
import re

import numpy as np
import pytest

from oracle import dqt_oracle as O
from paper_2412_04787_amd import dqt

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def declared_functions():
    src = open(os.path.join(ROOT, "include", "dqt.h")).read()
    src = re.sub(r"/\*.*?\*/", "", src, flags=re.S)
    return sorted(set(re.findall(r"\b(dqt_[a-z0-9_]+)\s*\(", src)))


def test_library_exports_every_declared_symbol():
    lib = dqt.load()
    names = declared_functions()
    assert len(names) >= 11
    for n in names:
        assert hasattr(lib, n), n
    assert set(names) == set(dqt.EXPORTS)


def test_version_and_status_strings():
    assert dqt.version() == 10000
    for st in range(9):
        s = dqt.status_string(st)
        assert s.startswith("DQT_")
    assert "unknown" in dqt.status_string(99)


def test_struct_layout_matches_header():
    assert ctypes.sizeof(dqt.DqtWeight) == 32
    assert dqt.DqtWeight.alpha.offset == 20 and dqt.DqtWeight.tensor_id.offset == 24


def test_pack_unpack_match_oracle():
    rng = np.random.default_rng(0)
    q = rng.integers(-1, 2, (33, 64)).astype(np.int8)
    packed = dqt.dqt_pack_ternary(q)
    assert np.array_equal(packed, O.pack_ternary(q))
    assert np.array_equal(dqt.dqt_unpack_ternary(packed, 64), q)
    bad = q.copy()
    bad[3, 5] = 2
    with pytest.raises(dqt.DqtError) as e:
        dqt.dqt_pack_ternary(bad)
    assert e.value.status == dqt.DQT_ERR_RANGE


@pytest.mark.parametrize("qmin,qmax", [(-1, 1), (-127, 127), (-128, 127), (-4, 3)])
def test_absmean_init_matches_oracle(qmin, qmax):
    rng = np.random.default_rng(qmax)
    W0 = (rng.standard_normal((300, 256)) * 0.02).astype(np.float32)
    q_lib, a_lib = dqt.dqt_absmean_init(W0, qmin, qmax)
    q_or, a_or = O.absmean_init(W0, qmin, qmax)
    # the two sum |W0| in different orders; alpha may differ by one fp32 ulp
    assert abs(float(a_lib) - float(a_or)) <= abs(float(np.spacing(a_or)))
    diff = np.count_nonzero(q_lib != q_or)
    assert diff <= 2, diff


def test_absmean_init_rejects_zero_tensor():
    with pytest.raises(dqt.DqtError) as e:
        dqt.dqt_absmean_init(np.zeros((4, 4), np.float32), -1, 1)
    assert e.value.status == dqt.DQT_ERR_RANGE


def _w(**kw):
    base = dict(d_out=64, d_in=64, wfmt=dqt.DQT_TERNARY2, qmin=-1, qmax=1, alpha=0.01, tensor_id=0)
    base.update(kw)
    return dqt.weight(**base)


FAKE = ctypes.c_void_p(1 << 20)          # never dereferenced: calls fail validation first
UNALIGNED = ctypes.c_void_p((1 << 20) + 4)


@pytest.mark.parametrize("kw,status", [
    (dict(d_in=8), dqt.DQT_ERR_SHAPE),
    (dict(d_out=40), dqt.DQT_ERR_SHAPE),
    (dict(d_in=65536 + 16), dqt.DQT_ERR_SHAPE),
    (dict(qmin=-2), dqt.DQT_ERR_RANGE),
    (dict(wfmt=dqt.DQT_I8, qmin=-129, qmax=127), dqt.DQT_ERR_RANGE),
    (dict(wfmt=dqt.DQT_I8, qmin=5, qmax=5), dqt.DQT_ERR_RANGE),
    (dict(alpha=0.0), dqt.DQT_ERR_RANGE),
    (dict(alpha=float("inf")), dqt.DQT_ERR_RANGE),
    (dict(wfmt=dqt.DQT_BF16), dqt.DQT_ERR_DTYPE),
])
def test_bad_weight_descriptor_rejected(kw, status):
    lib = dqt.load()
    w = _w(**kw)
    st = lib.dqt_sr_update(ctypes.byref(w), FAKE, FAKE, 1e-3, 0, 1, None, None)
    assert st == status
    st = lib.dqt_linear_fwd(ctypes.byref(w), FAKE, FAKE, dqt.DQT_F32, 16, dqt.DQT_I8, FAKE, FAKE,
                            FAKE, dqt.DQT_F32, FAKE, 1 << 30, None)
    assert st == status


def test_call_level_checks():
    lib = dqt.load()
    w = _w()
    bw = ctypes.byref(w)
    # fwd
    BIG = 1 << 30
    assert lib.dqt_linear_fwd(bw, FAKE, FAKE, dqt.DQT_F32, -1, dqt.DQT_I8, FAKE, FAKE, FAKE,
                              dqt.DQT_F32, FAKE, BIG, None) == dqt.DQT_ERR_SHAPE
    assert lib.dqt_linear_fwd(bw, None, FAKE, dqt.DQT_F32, 16, dqt.DQT_I8, FAKE, FAKE, FAKE,
                              dqt.DQT_F32, FAKE, BIG, None) == dqt.DQT_ERR_NULL
    assert lib.dqt_linear_fwd(bw, FAKE, FAKE, dqt.DQT_F32, 16, dqt.DQT_I8, FAKE, UNALIGNED, FAKE,
                              dqt.DQT_F32, FAKE, BIG, None) == dqt.DQT_ERR_ALIGN
    assert lib.dqt_linear_fwd(bw, FAKE, FAKE, dqt.DQT_I8, 16, dqt.DQT_I8, FAKE, FAKE, FAKE,
                              dqt.DQT_F32, FAKE, BIG, None) == dqt.DQT_ERR_DTYPE
    assert lib.dqt_linear_fwd(bw, FAKE, FAKE, dqt.DQT_F32, 16, dqt.DQT_F32, FAKE, FAKE, FAKE,
                              dqt.DQT_F32, FAKE, BIG, None) == dqt.DQT_ERR_DTYPE
    # the fastest form expands the codes into the workspace (256 counter
    # bytes + one byte per weight); with d_in a multiple of 64 the counters
    # alone also do (the packed codes go straight to the GEMM), fewer do not
    assert lib.dqt_linear_fwd_workspace(bw) == 256 + w.d_out * w.d_in
    assert lib.dqt_linear_fwd(bw, FAKE, FAKE, dqt.DQT_F32, 16, dqt.DQT_I8, FAKE, FAKE, FAKE,
                              dqt.DQT_F32, FAKE, 255, None) == dqt.DQT_ERR_WORKSPACE
    w48 = _w(d_in=48)
    need_f = lib.dqt_linear_fwd_workspace(ctypes.byref(w48))
    assert need_f == 256 + 64 * 48
    assert lib.dqt_linear_fwd(ctypes.byref(w48), FAKE, FAKE, dqt.DQT_F32, 16, dqt.DQT_I8, FAKE, FAKE,
                              FAKE, dqt.DQT_F32, FAKE, need_f - 1, None) == dqt.DQT_ERR_WORKSPACE
    assert lib.dqt_linear_fwd(ctypes.byref(w48), FAKE, FAKE, dqt.DQT_F32, 16, dqt.DQT_I8, FAKE, FAKE,
                              FAKE, dqt.DQT_F32, None, 0, None) == dqt.DQT_ERR_WORKSPACE
    w8 = _w(wfmt=dqt.DQT_I8, qmin=-127, qmax=127)
    assert lib.dqt_linear_fwd_workspace(ctypes.byref(w8)) == 256
    assert lib.dqt_linear_fwd(ctypes.byref(w8), FAKE, FAKE, dqt.DQT_F32, 16, dqt.DQT_FP8E4M3,
                              FAKE, FAKE, FAKE, dqt.DQT_F32, None, 0, None) == dqt.DQT_ERR_UNSUPPORTED
    # M = 0 is a no-op that launches nothing
    assert lib.dqt_linear_fwd(bw, None, None, dqt.DQT_F32, 0, dqt.DQT_I8, None, None, None,
                              dqt.DQT_F32, None, 0, None) == dqt.DQT_OK
    # bwd
    big = _w(d_out=768, d_in=768)
    need = lib.dqt_linear_bwd_workspace(ctypes.byref(big), 8192)
    # bf16 weights + bf16 X~ + split partials
    assert need >= 768 * 768 * 2 + 8192 * 768 * 2
    assert lib.dqt_linear_bwd(ctypes.byref(big), FAKE, FAKE, dqt.DQT_I8, FAKE, FAKE, dqt.DQT_BF16,
                              8192, dqt.DQT_BF16, None, dqt.DQT_F32, FAKE, None, 0,
                              None) == dqt.DQT_ERR_WORKSPACE
    assert lib.dqt_linear_bwd(ctypes.byref(big), FAKE, FAKE, dqt.DQT_I8, FAKE, FAKE, dqt.DQT_BF16,
                              8192, dqt.DQT_BF16, None, dqt.DQT_F32, FAKE, FAKE, need - 4,
                              None) == dqt.DQT_ERR_WORKSPACE
    assert lib.dqt_linear_bwd(bw, FAKE, FAKE, dqt.DQT_I8, FAKE, FAKE, dqt.DQT_F32, 16,
                              dqt.DQT_BF16, None, dqt.DQT_F32, FAKE, None, 0,
                              None) == dqt.DQT_ERR_UNSUPPORTED
    assert lib.dqt_linear_bwd(bw, FAKE, FAKE, dqt.DQT_I8, FAKE, FAKE, dqt.DQT_F32, 16,
                              dqt.DQT_F32, None, dqt.DQT_F32, None, None, 0, None) == dqt.DQT_OK
    assert lib.dqt_linear_bwd_workspace(ctypes.byref(_w()), 512) >= 64 * 64 * 2 + 512 * 64 * 2
    # sr
    assert lib.dqt_sr_update(bw, FAKE, None, 1e-3, 0, 1, None, None) == dqt.DQT_ERR_NULL
    assert lib.dqt_sr_update(bw, FAKE, FAKE, -1.0, 0, 1, None, None) == dqt.DQT_ERR_RANGE
    assert lib.dqt_sr_update(bw, FAKE, FAKE, float("nan"), 0, 1, None, None) == dqt.DQT_ERR_RANGE
    tiny = _w(alpha=1e-38)
    assert lib.dqt_sr_update(ctypes.byref(tiny), FAKE, FAKE, 1e3, 0, 1, None,
                             None) == dqt.DQT_ERR_RANGE
    assert lib.dqt_sr_update(bw, UNALIGNED, FAKE, 1e-3, 0, 1, None, None) == dqt.DQT_ERR_ALIGN
    # act quant / rng
    assert lib.dqt_act_quant(FAKE, dqt.DQT_F32, 4, 20, dqt.DQT_I8, FAKE, FAKE,
                             None) == dqt.DQT_ERR_SHAPE
    assert lib.dqt_act_quant(FAKE, dqt.DQT_F32, 0, 32, dqt.DQT_I8, None, None, None) == dqt.DQT_OK
    ents = (dqt.DqtActIO * 9)()
    for e in ents:
        e.X, e.Xq, e.xdq, e.K, e.reserved = 1 << 20, 1 << 20, 1 << 20, 64, 0
    assert lib.dqt_act_quant_batch(9, ents, dqt.DQT_BF16, 16, dqt.DQT_I8, None) == dqt.DQT_ERR_SHAPE
    assert lib.dqt_act_quant_batch(2, None, dqt.DQT_BF16, 16, dqt.DQT_I8, None) == dqt.DQT_ERR_NULL
    assert lib.dqt_act_quant_batch(2, ents, dqt.DQT_I8, 16, dqt.DQT_I8, None) == dqt.DQT_ERR_DTYPE
    ents[1].K = 20
    assert lib.dqt_act_quant_batch(2, ents, dqt.DQT_BF16, 16, dqt.DQT_I8, None) == dqt.DQT_ERR_SHAPE
    ents[1].K = 64
    ents[1].Xq = None
    assert lib.dqt_act_quant_batch(2, ents, dqt.DQT_BF16, 16, dqt.DQT_I8, None) == dqt.DQT_ERR_NULL
    ents[1].Xq = (1 << 20) + 8
    assert lib.dqt_act_quant_batch(2, ents, dqt.DQT_BF16, 16, dqt.DQT_I8, None) == dqt.DQT_ERR_ALIGN
    assert lib.dqt_act_quant_batch(2, ents, dqt.DQT_BF16, 0, dqt.DQT_I8, None) == dqt.DQT_ERR_ALIGN
    ents[1].Xq = 1 << 20
    assert lib.dqt_act_quant_batch(2, ents, dqt.DQT_BF16, 0, dqt.DQT_I8, None) == dqt.DQT_OK
    assert lib.dqt_act_quant_batch(2, ents, dqt.DQT_BF16, (1 << 28) + 1, dqt.DQT_I8,
                                   None) == dqt.DQT_ERR_SHAPE
    assert lib.dqt_debug_rng(0, 1, 0, 0, -1, FAKE, None) == dqt.DQT_ERR_SHAPE
    assert lib.dqt_debug_rng(0, 1, 0, 0, 5, None, None) == dqt.DQT_ERR_NULL


def test_workspace_depends_on_shape_only():
    lib = dqt.load()
    a = _w(d_out=2048, d_in=768, tensor_id=3)
    b = _w(d_out=2048, d_in=768, alpha=0.5)
    assert lib.dqt_linear_bwd_workspace(ctypes.byref(a), 8192) == \
        lib.dqt_linear_bwd_workspace(ctypes.byref(b), 8192)


def test_adamw_sr_argument_checks():
    """AdamW with SR: hyper-parameters, step and pointers are checked before
    anything is launched."""
    lib = dqt.load()
    bw = ctypes.byref(_w())

    def call(hp, step=1, m=FAKE, v=FAKE, wq=FAKE, dw=FAKE):
        return lib.dqt_adamw_sr_update(bw, wq, dw, m, v, None if hp is None else ctypes.byref(hp),
                                       0, step, None, None)

    ok = dqt.adamw(1e-3)
    assert call(None) == dqt.DQT_ERR_NULL
    assert call(ok, step=0) == dqt.DQT_ERR_RANGE
    assert call(dqt.adamw(1e-3, eps=0.0)) == dqt.DQT_ERR_RANGE
    assert call(dqt.adamw(1e-3, beta1=1.0)) == dqt.DQT_ERR_RANGE
    assert call(dqt.adamw(1e-3, beta2=-0.1)) == dqt.DQT_ERR_RANGE
    assert call(dqt.adamw(-1e-3)) == dqt.DQT_ERR_RANGE
    assert call(dqt.adamw(float("nan"))) == dqt.DQT_ERR_RANGE
    assert call(dqt.adamw(1e-3, weight_decay=-1.0)) == dqt.DQT_ERR_RANGE
    assert call(ok, m=None) == dqt.DQT_ERR_NULL
    assert call(ok, v=UNALIGNED) == dqt.DQT_ERR_ALIGN
    assert call(ok, wq=None) == dqt.DQT_ERR_NULL
    # a step that overflows fp32 in grid units
    tiny = ctypes.byref(_w(alpha=1e-38))
    assert lib.dqt_adamw_sr_update(tiny, FAKE, FAKE, FAKE, FAKE, ctypes.byref(dqt.adamw(1e3)), 0, 1,
                                   None, None) == dqt.DQT_ERR_RANGE


def test_fused_bwd_sr_argument_checks_host():
    """The fused backward + SR call rejects a dW pointer, the fp32
    environment and a bad learning rate before launching anything."""
    lib = dqt.load()
    io = dqt.linear_io([dict(w=_w())])
    io[0].Wq = io[0].Xq = io[0].xdq = io[0].dY = FAKE.value
    io[0].dW = FAKE.value
    bf, f32 = dqt.DQT_BF16, dqt.DQT_F32
    args = lambda dy, lr: (1, io, 64, dqt.DQT_I8, dy, dy, bf, lr, 0, 1, None, FAKE, 1 << 30, None)
    assert lib.dqt_linear_bwd_sr_batch(*args(bf, 1e-3)) == dqt.DQT_ERR_UNSUPPORTED
    io[0].dW = None
    assert lib.dqt_linear_bwd_sr_batch(*args(f32, 1e-3)) == dqt.DQT_ERR_UNSUPPORTED
    assert lib.dqt_linear_bwd_sr_batch(*args(bf, -1.0)) == dqt.DQT_ERR_RANGE


def test_int4_pack_matches_oracle_and_roundtrips():
    rng = np.random.default_rng(3)
    q = rng.integers(-8, 8, size=(5, 32)).astype(np.int8)
    packed = dqt.dqt_pack_int4(q)
    assert np.array_equal(packed, O.pack_int4(q))
    assert np.array_equal(dqt.dqt_unpack_int4(packed, 32), q)
    # layout: weight k in the low nibble of byte k // 2 when k is even
    two = np.array([[-8, 7, 1, -1]], np.int8)
    assert dqt.dqt_pack_int4(two).tolist() == [[0x78, 0xF1]]
    with pytest.raises(dqt.DqtError):
        dqt.dqt_pack_int4(np.array([[8, 0]], np.int8))
    # descriptor checks: the 4-bit grid must lie in [-8, 7]
    lib = dqt.load()
    ok = _w(wfmt=dqt.DQT_INT4, qmin=-8, qmax=7)
    assert lib.dqt_sr_update(ctypes.byref(ok), FAKE, None, 1e-3, 0, 1, None, None) == dqt.DQT_ERR_NULL
    bad = _w(wfmt=dqt.DQT_INT4, qmin=-9, qmax=7)
    assert lib.dqt_sr_update(ctypes.byref(bad), FAKE, FAKE, 1e-3, 0, 1, None, None) == dqt.DQT_ERR_RANGE
    # e4m3 activations take ternary or 4-bit weights (exact in e4m3), not int8 codes
    i8w = _w(wfmt=dqt.DQT_I8, qmin=-127, qmax=127)
    assert lib.dqt_linear_fwd(ctypes.byref(i8w), FAKE, FAKE, dqt.DQT_F32, 16, dqt.DQT_FP8E4M3, FAKE,
                              FAKE, FAKE, dqt.DQT_F32, FAKE, 1 << 30, None) == dqt.DQT_ERR_UNSUPPORTED


def test_new_batch_entry_points_take_one_to_eight_linears():
    """Like the other linear batches, n outside 1..8 is rejected before
    anything is enqueued, as is an unknown variant mode."""
    lib = dqt.load()
    bf = dqt.DQT_BF16
    hp = ctypes.byref(dqt.adamw(1e-3))
    empty = (dqt.DqtLinearIO * 1)()
    assert lib.dqt_linear_bwd_sr_batch(0, empty, 64, dqt.DQT_I8, bf, bf, bf, 1e-3, 0, 1, None, FAKE,
                                       1 << 30, None) == dqt.DQT_ERR_SHAPE
    assert lib.dqt_adamw_sr_update_batch(0, empty, None, None, hp, 0, 1, None, None) == dqt.DQT_ERR_SHAPE
    assert lib.dqt_update_variant_batch(0, empty, 1e-3, 0, 1, dqt.DQT_UPD_NEAREST, 0.2, None, None, 0,
                                        None) == dqt.DQT_ERR_SHAPE
    nine = dqt.linear_io([dict(w=_w())] * 9)
    assert lib.dqt_linear_bwd_sr_batch(9, nine, 64, dqt.DQT_I8, bf, bf, bf, 1e-3, 0, 1, None, FAKE,
                                       1 << 30, None) == dqt.DQT_ERR_SHAPE
    assert lib.dqt_adamw_sr_update_batch(9, nine, None, None, hp, 0, 1, None, None) == dqt.DQT_ERR_SHAPE
    assert lib.dqt_update_variant_batch(9, nine, 1e-3, 0, 1, 0, 0.2, None, None, 0,
                                        None) == dqt.DQT_ERR_SHAPE
    assert lib.dqt_update_variant_batch(1, dqt.linear_io([dict(w=_w())]), 1e-3, 0, 1, 7, 0.2, None,
                                        None, 0, None) == dqt.DQT_ERR_RANGE


def test_sr_table_build_layout_and_checks():
    """The update table of n tensors: 64-byte entries holding the code and
    gradient addresses, the tensor's chunks of 8 weights, its first tile of
    256 chunks in the launch (a running sum), alpha, the grid and the tensor
    id; the host checks reject bad entries before anything is written to the
    device."""
    lib = dqt.load()
    shapes = [(16, 16), (256, 272), (48, 80), (4096, 4096)]
    ents = []
    for s, (d_out, d_in) in enumerate(shapes):
        w = _w(d_out=d_out, d_in=d_in, wfmt=dqt.DQT_I8, qmin=-127, qmax=127, alpha=0.5 + s,
               tensor_id=9 + s)
        ents.append(w)
    io = dqt.linear_io([dict(w=w) for w in ents])
    for s in range(len(ents)):
        io[s].Wq = 0x10000 * (s + 1)
        io[s].dW = 0x100000 * (s + 1)
    assert dqt.dqt_sr_table_bytes(4) == 256 and dqt.dqt_sr_table_bytes(0) == 0
    tab = dqt.dqt_sr_table_build(io)
    rec = np.frombuffer(tab.tobytes(), dtype=np.dtype([
        ("wq", "<u8"), ("grad", "<u8"), ("nchunks", "<i8"), ("tile0", "<i8"), ("alpha", "<f4"),
        ("qmin", "<i4"), ("qmax", "<i4"), ("tid", "<u4"), ("pad", "<u4", 4)]))
    tile = 0
    for s, (d_out, d_in) in enumerate(shapes):
        r = rec[s]
        assert r["wq"] == 0x10000 * (s + 1) and r["grad"] == 0x100000 * (s + 1)
        assert r["nchunks"] == d_out * d_in // 8 and r["tile0"] == tile
        assert r["alpha"] == np.float32(0.5 + s) and (r["qmin"], r["qmax"]) == (-127, 127)
        assert r["tid"] == 9 + s and not r["pad"].any()
        tile += (d_out * d_in // 8 + 255) // 256
    buf = np.zeros(256, np.uint8)
    assert lib.dqt_sr_table_build(4, io, buf.ctypes.data, 255) == dqt.DQT_ERR_WORKSPACE
    assert lib.dqt_sr_table_build(0, io, buf.ctypes.data, 256) == dqt.DQT_ERR_SHAPE
    assert lib.dqt_sr_table_build(4, io, None, 256) == dqt.DQT_ERR_NULL
    io[2].dW = 0x100008                                       # not 16-byte aligned
    assert lib.dqt_sr_table_build(4, io, buf.ctypes.data, 256) == dqt.DQT_ERR_ALIGN
    io[2].dW = None
    assert lib.dqt_sr_table_build(4, io, buf.ctypes.data, 256) == dqt.DQT_ERR_NULL
    io[2].dW = 0x300000
    mixed = dqt.linear_io([dict(w=ents[0]), dict(w=_w(wfmt=dqt.DQT_TERNARY2))])
    mixed[0].Wq = mixed[1].Wq = mixed[0].dW = mixed[1].dW = 0x10000
    assert lib.dqt_sr_table_build(2, mixed, buf.ctypes.data, 256) == dqt.DQT_ERR_UNSUPPORTED
    # the update call repeats the checks, and refuses a bad lr or table
    assert lib.dqt_sr_update_table(4, io, 0x200000, -1.0, 0, 1, None, None, None) == \
        dqt.DQT_ERR_RANGE
    assert lib.dqt_sr_update_table(4, io, None, 1e-3, 0, 1, None, None, None) == dqt.DQT_ERR_NULL
    assert lib.dqt_sr_update_table(4, io, 0x200008, 1e-3, 0, 1, None, None, None) == \
        dqt.DQT_ERR_ALIGN
    assert lib.dqt_sr_update_table(4, io, 0x200000, 1e-3, 0, 1, None, 0x300004, None) == \
        dqt.DQT_ERR_ALIGN


def test_int3_pack_matches_oracle_and_checks():
    rng = np.random.default_rng(5)
    q = rng.integers(-4, 4, size=(7, 48)).astype(np.int8)
    packed = dqt.dqt_pack_int3(q)
    assert np.array_equal(packed, O.pack_int3(q))
    assert np.array_equal(dqt.dqt_unpack_int3(packed, 48), q)
    with pytest.raises(dqt.DqtError) as e:
        dqt.dqt_pack_int3(np.array([[4] + [0] * 7], np.int8))
    assert e.value.status == dqt.DQT_ERR_RANGE
    lib = dqt.load()
    ok = _w(wfmt=dqt.DQT_INT3, qmin=-4, qmax=3)
    assert lib.dqt_sr_update(ctypes.byref(ok), FAKE, None, 1e-3, 0, 1, None, None) == dqt.DQT_ERR_NULL
    for qmin, qmax in ((-5, 3), (-4, 4), (2, 1)):
        bad = _w(wfmt=dqt.DQT_INT3, qmin=qmin, qmax=qmax)
        assert lib.dqt_sr_update(ctypes.byref(bad), FAKE, FAKE, 1e-3, 0, 1, None, None) == \
            dqt.DQT_ERR_RANGE


def test_launch_timer_argument_checks():
    """The launch timer refuses bad capacities and a stop without a start
    (neither touches a device)."""
    lib = dqt.load()
    assert lib.dqt_launch_timer_start(0) == 2                 # DQT_ERR_SHAPE
    assert lib.dqt_launch_timer_start(65537) == 2
    count = ctypes.c_int32(-1)
    ms = (ctypes.c_float * 4)()
    assert lib.dqt_launch_timer_stop(ms, 4, ctypes.byref(count)) == 7   # DQT_ERR_UNSUPPORTED
    assert count.value == -1


def test_read_stream_argument_checks():
    """The streaming read refuses bad sizes and pointers before launching."""
    lib = dqt.load()
    assert lib.dqt_read_stream(None, 0, None, None) == 0          # nothing to read
    assert lib.dqt_read_stream(None, 16, FAKE, None) == 1         # DQT_ERR_NULL
    assert lib.dqt_read_stream(FAKE, 15, FAKE, None) == 2         # DQT_ERR_SHAPE
    assert lib.dqt_read_stream(UNALIGNED, 16, FAKE, None) == 3    # DQT_ERR_ALIGN
