"""dqt_linear_fwd_batch_noalloc -- the forward batch for callers that cannot
allocate -- gives the bits of dqt_linear_fwd_batch with a workspace, call
after call on the library's static per-GPU scratch (two calls in a row, the
second with a smaller input), runs ternary codes whose expansion does not fit
from the packed codes, and refuses a batch whose smallest workspace exceeds
the array before launching anything."""
import numpy as np
import pytest
import torch

from paper_2412_04787_amd import dqt, workloads as W

from gpu_util import DEV, log, make_weight, to_dev, weight_codes_dev

pytestmark = pytest.mark.gpu


def _batch(M, shapes, wfmt, qmin, qmax, act, seed):
    """Quantised inputs and codes for a batch of linears sharing one input
    per distinct d_in; outputs for the two entry points."""
    a_code = dqt.DQT_I8 if act == "i8" else dqt.DQT_FP8E4M3
    Xq, xdq = {}, {}
    ents_ws, ents_na = [], []
    for li, (d_in, d_out) in enumerate(shapes):
        if d_in not in Xq:
            X, _ = to_dev(W.draw_normal((M, d_in), 1.0, seed, 91, 1, d_in), "bf16")
            Xq[d_in] = torch.empty((M, d_in), dtype=torch.int8 if act == "i8" else torch.uint8,
                                   device=DEV)
            xdq[d_in] = torch.empty((max(M, 1),), dtype=torch.float32, device=DEV)
            dqt.dqt_act_quant(X, a_code, Xq[d_in], xdq[d_in])
        if wfmt == "ternary":
            q = W.draw_ternary((d_out, d_in), seed, 91, 2, li)
        else:
            q = W.draw_int((d_out, d_in), qmin, qmax, seed, 91, 2, li)
        w = make_weight(d_out, d_in, wfmt, qmin, qmax, 0.01 + 0.001 * li, li)
        codes = weight_codes_dev(q, wfmt)
        common = dict(w=w, Wq=codes, Xq=Xq[d_in], xdq=xdq[d_in])
        ents_ws.append(dict(common, Y=torch.full((M, d_out), 7.0, dtype=torch.bfloat16, device=DEV)))
        ents_na.append(dict(common, Y=torch.full((M, d_out), -7.0, dtype=torch.bfloat16, device=DEV)))
    return a_code, ents_ws, ents_na


CALLS = [
    # (M, shapes, wfmt, qmin, qmax, act): each pair runs back to back, the
    # second smaller than the first
    [(2048, [(768, 768), (768, 2048), (2048, 768)], "ternary", -1, 1, "i8"),
     (300, [(256, 512), (512, 256)], "ternary", -1, 1, "i8")],
    # 4-bit codes and a ternary row length that is not a multiple of 64 use
    # the array beyond the counters (the expanded operand bytes)
    [(1000, [(512, 1024), (1024, 512)], "i4", -8, 7, "e4m3"),
     (200, [(96, 208), (208, 96)], "ternary", -1, 1, "i8")],
]


@pytest.mark.parametrize("ci", range(len(CALLS)))
def test_noalloc_forward_matches_workspace_forward(lib, ci):
    for k, (M, shapes, wfmt, qmin, qmax, act) in enumerate(CALLS[ci]):
        log(f"no-alloc forward case {ci}.{k}: M={M} {shapes} {wfmt} {act}")
        a_code, ents_ws, ents_na = _batch(M, shapes, wfmt, qmin, qmax, act, 10 * ci + k)
        io_ws, io_na = dqt.linear_io(ents_ws), dqt.linear_io(ents_na)
        need = dqt.dqt_linear_fwd_batch_workspace(io_ws)
        assert need <= dqt.NOALLOC_SCRATCH_BYTES
        ws = dqt.workspace(need)
        dqt.dqt_linear_fwd_batch(io_ws, M, a_code, dqt.DQT_BF16, ws)
        dqt.dqt_linear_fwd_batch_noalloc(io_na, M, a_code, dqt.DQT_BF16)
        torch.cuda.synchronize()
        for li, (a, b) in enumerate(zip(ents_ws, ents_na)):
            assert torch.equal(a["Y"], b["Y"]), (ci, k, li)


def test_noalloc_forward_large_ternary_runs_packed(lib):
    """Ternary codes whose expansion exceeds the array (2 x 4096 x 4096 bytes
    plus the counters) run from the packed codes, expanded in registers:
    int8 activations give the bits of the workspace call, which expands them."""
    for k, M in enumerate((256, 96)):
        log(f"no-alloc forward, packed ternary: M={M}")
        a_code, ents_ws, ents_na = _batch(M, [(4096, 4096), (4096, 4096)], "ternary", -1, 1, "i8", 70 + k)
        io_ws, io_na = dqt.linear_io(ents_ws), dqt.linear_io(ents_na)
        need = dqt.dqt_linear_fwd_batch_workspace(io_ws)
        assert need > dqt.NOALLOC_SCRATCH_BYTES
        dqt.dqt_linear_fwd_batch(io_ws, M, a_code, dqt.DQT_BF16, dqt.workspace(need))
        dqt.dqt_linear_fwd_batch_noalloc(io_na, M, a_code, dqt.DQT_BF16)
        torch.cuda.synchronize()
        for li, (a, b) in enumerate(zip(ents_ws, ents_na)):
            assert torch.equal(a["Y"], b["Y"]), (k, li)


def test_noalloc_forward_refuses_oversized_scratch(lib):
    # 4-bit codes expand to one byte per weight: 2 x 4096 x 4096 bytes plus
    # the counters exceed the array; nothing is launched
    w = make_weight(4096, 4096, "i4", -8, 7, 0.01)
    t = torch.zeros((16,), dtype=torch.int8, device=DEV)
    io = dqt.linear_io([dict(w=w, Wq=t, Xq=t, xdq=t, Y=t)] * 2)
    assert dqt.dqt_linear_fwd_batch_workspace(io) > dqt.NOALLOC_SCRATCH_BYTES
    with pytest.raises(dqt.DqtError) as e:
        dqt.dqt_linear_fwd_batch_noalloc(io, 64, dqt.DQT_I8, dqt.DQT_BF16)
    assert e.value.status == dqt.DQT_ERR_WORKSPACE
    # invalid arguments are refused as dqt_linear_fwd_batch refuses them
    io_bad = dqt.linear_io([dict(w=make_weight(64, 64, "ternary", -1, 1, 0.01), Wq=None, Xq=t,
                                 xdq=t, Y=t)])
    with pytest.raises(dqt.DqtError) as e:
        dqt.dqt_linear_fwd_batch_noalloc(io_bad, 64, dqt.DQT_I8, dqt.DQT_BF16)
    assert e.value.status == dqt.DQT_ERR_NULL
