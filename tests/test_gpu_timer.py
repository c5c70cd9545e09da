"""The launch timer: one pair of events per GEMM kernel launch, in issue
order, up to its capacity; its durations fit inside the calls they belong to;
calls after the stop run untimed."""
import os
import sys

import numpy as np
import pytest
import torch

from paper_2412_04787_amd import dqt, workloads as W

from gpu_util import DEV, log

sys.path.insert(0, os.path.dirname(os.path.dirname(os.path.abspath(__file__))))
import bench  # noqa: E402

pytestmark = pytest.mark.gpu


def _calls(blk, kind, n, step0):
    def only(k, fn):
        if k == kind:
            fn()
    for r in range(n):
        bench.run_step(blk, dqt, step0 + r, None, only, split_bwd=kind in ("bwd_dx", "bwd_dw"),
                       sr="fused" if kind == "bwd_sr" else "separate")


@pytest.fixture(scope="module")
def h768(lib):
    blk = bench.Block(W.WORKLOADS["llama_h768"], torch, dqt, W)
    _calls(blk, "act_quant", 1, 1)      # quantised inputs in place
    torch.cuda.synchronize()
    return blk


@pytest.mark.parametrize("kind,per_call", [("fwd", 1), ("bwd_sr", 1), ("bwd", 1), ("bwd_dx", 1),
                                           ("bwd_dw", 1)])
def test_timer_counts_gemm_launches(h768, kind, per_call):
    log(f"launch timer: llama_h768 {kind}")
    blk = h768
    n = 3
    ev = [torch.cuda.Event(enable_timing=True) for _ in range(2)]
    dqt.dqt_launch_timer_start(16)
    ev[0].record()
    _calls(blk, kind, n, 10)
    ev[1].record()
    torch.cuda.synchronize()
    ms, count = dqt.dqt_launch_timer_stop(16)
    assert count == n * per_call, count
    assert all(t > 0 for t in ms), ms
    # the GEMM kernels are part of the calls: their sum cannot exceed the
    # calls' own span
    assert sum(ms) <= ev[0].elapsed_time(ev[1]) * 1.001 + 0.01, (ms, ev[0].elapsed_time(ev[1]))
    # stopped: later calls run untimed, and a second stop is refused
    _calls(blk, kind, 1, 20)
    torch.cuda.synchronize()
    with pytest.raises(dqt.DqtError) as e:
        dqt.dqt_launch_timer_stop(16)
    assert e.value.status == dqt.DQT_ERR_UNSUPPORTED


def test_timer_capacity_and_restart(lib):
    log("launch timer: capacity 2 over 3 forward calls, then a second timer")
    wl = W.WORKLOADS["single_256"]
    blk = bench.Block(wl, torch, dqt, W)
    dqt.dqt_launch_timer_start(2)
    with pytest.raises(dqt.DqtError) as e:
        dqt.dqt_launch_timer_start(2)           # one timer at a time
    assert e.value.status == dqt.DQT_ERR_UNSUPPORTED
    _calls(blk, "fwd", 3, 1)
    torch.cuda.synchronize()
    ms, count = dqt.dqt_launch_timer_stop(2)
    assert count == 2 and len(ms) == 2 and all(t > 0 for t in ms)
    dqt.dqt_launch_timer_start(4)
    _calls(blk, "fwd", 1, 5)
    torch.cuda.synchronize()
    ms, count = dqt.dqt_launch_timer_stop(1)
    assert count == 1 and len(ms) == 1


@pytest.mark.parametrize("nbytes", [16, 16 * 1000003, 64 << 20])
def test_read_stream_reads_every_word_once(lib, nbytes):
    """The xor of the sink is the xor of every 32-bit word of the buffer (each
    word read exactly once), ragged sizes included."""
    log(f"read stream: {nbytes} bytes")
    g = torch.Generator(device=DEV)
    g.manual_seed(nbytes)
    src = torch.randint(-2**31, 2**31 - 1, (nbytes // 4,), dtype=torch.int32, device=DEV, generator=g)
    sink = torch.full((dqt.READ_STREAM_SINK_WORDS,), 12345, dtype=torch.int32, device=DEV)
    dqt.dqt_read_stream(src, sink)
    torch.cuda.synchronize()
    want = np.bitwise_xor.reduce(src.cpu().numpy().view(np.uint32))
    got = np.bitwise_xor.reduce(sink.cpu().numpy().view(np.uint32))
    assert got == want
