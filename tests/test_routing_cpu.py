"""Kernel routing by shape, on the host (no GPU needed).

albireo_sample_route runs the same decision every sampling entry point takes before it enqueues
anything.  Each shape class below is routed once: rows too short for a 16-byte slot, rows that fit one
workgroup's registers (16 to 38 x 512 x 16 bytes), wider rows up to the streaming kernels' 64 chunks of
4864 slots, rows beyond that, rows with a prompt history or a penalty state (streaming kernels only),
batches whose chunk count reaches 2^31 (the cooperative kernel) and invalid arguments.  A routing
step that called itself without end would overflow the host stack here and kill the test process.
"""
import pytest
import torch

from paper_2606_01927_amd import (ROUTE_COOPERATIVE, ROUTE_NONE, ROUTE_ONE_WORKGROUP, ROUTE_STREAM,
                                  PenaltyState, SamplingParams, _lib, sample_route)

F32, BF16 = torch.float32, torch.bfloat16
REG_SLOTS = 38 * 512     # 16-byte slots one workgroup holds in registers
STREAM_SLOTS = 64 * 4864  # 16-byte slots of the streaming kernels' widest row
VEC = {F32: 4, BF16: 8}  # logits per 16-byte slot


def _limits(dt):
    v = VEC[dt]
    return v, (REG_SLOTS + 1) * v - 1, (STREAM_SLOTS + 1) * v - 1


@pytest.mark.parametrize("dt", [F32, BF16])
def test_route_by_width(dt):
    v, reg_max, stream_max = _limits(dt)
    cases = [(1, ROUTE_STREAM), (v - 1, ROUTE_STREAM), (v, ROUTE_ONE_WORKGROUP),
             (32000, ROUTE_ONE_WORKGROUP), (reg_max, ROUTE_ONE_WORKGROUP), (reg_max + 1, ROUTE_STREAM),
             (256000, ROUTE_STREAM), (stream_max, ROUTE_STREAM), (stream_max + 1, ROUTE_NONE)]
    for V, want in cases:
        for B in (0, 1, 64, 4096):
            for sharded in (False, True):
                assert sample_route(B, V, dt, sharded=sharded) == want, (dt, V, B, sharded)


@pytest.mark.parametrize("dt", [F32, BF16])
def test_prompt_or_state_takes_the_streaming_kernels(dt):
    v, reg_max, stream_max = _limits(dt)
    with_prompt = SamplingParams(prompt_offsets=torch.zeros(2, dtype=torch.int64),
                                 prompt_ids=torch.zeros(0, dtype=torch.int32))
    st = PenaltyState.__new__(PenaltyState)  # only whether a state is given is read
    with_state = SamplingParams(state=st)
    for p in (with_prompt, with_state):
        for V in (v, 32000, reg_max, reg_max + 1, stream_max):
            assert sample_route(8, V, dt, p) == ROUTE_STREAM, (dt, V)
        assert sample_route(8, stream_max + 1, dt, p) == ROUTE_NONE
    # output history and per-row scalars alone keep the width rule
    only_hist = SamplingParams(hist_offsets=torch.zeros(2, dtype=torch.int64),
                               hist_ids=torch.zeros(0, dtype=torch.int32))
    assert sample_route(8, 32000, dt, only_hist) == ROUTE_ONE_WORKGROUP


def test_cooperative_route_when_the_chunk_grid_overflows():
    # fp32 V = 100000: 25000 slots, 6 streaming chunks, 2 cooperative chunks
    chunks = -(-25000 // 4864)
    b_max = ((1 << 31) - 1) // chunks
    assert sample_route(b_max, 100000, F32) == ROUTE_STREAM
    assert sample_route(b_max + 1, 100000, F32) == ROUTE_COOPERATIVE
    # rows that fit one workgroup stay there whatever the batch
    assert sample_route(1 << 40, 32000, F32) == ROUTE_ONE_WORKGROUP


def test_invalid_arguments_route_nowhere():
    assert sample_route(8, 0, F32) == ROUTE_NONE
    assert sample_route(-1, 32000, F32) == ROUTE_NONE
    assert sample_route(8, (1 << 31) - 16, BF16) == ROUTE_NONE
    assert _lib.albireo_sample_route(8, 32000, 7, None, 0) == ROUTE_NONE


def test_refused_launch_refills_the_workspace(monkeypatch):
    """After ALBIREO_E_LAUNCH the binding zero-fills its Workspace before raising; other errors leave it."""
    import paper_2606_01927_amd as alb

    ws = alb.Workspace("cpu")
    calls = []
    monkeypatch.setattr(ws, "refill", lambda stream=None: calls.append(stream))
    with pytest.raises(alb.AlbireoError):
        alb._fail(alb.E_INVALID, "albireo_sample", ws)
    assert calls == []
    with pytest.raises(alb.AlbireoError):
        alb._fail(alb.E_LAUNCH, "albireo_sample", ws, "s")
    assert calls == ["s"]
    with pytest.raises(alb.AlbireoError):
        alb._fail(alb.E_LAUNCH, "albireo_sample", None)  # a caller's raw pointer: nothing to refill
