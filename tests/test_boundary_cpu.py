"""Host-side checks of the C-ABI library that need no GPU: it loads, it exports every entry point the
header declares, and argument errors come back as status codes before anything is launched."""
from __future__ import annotations

import ctypes
import os
import re

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "albireo.h")


def _declared():
    text = open(HEADER).read()
    return sorted(set(re.findall(r"^\s*(?:albireo_status_t|albireo_route_t|size_t|const char\*)\s+(albireo_\w+)\s*\(", text, re.M)))


@pytest.fixture(scope="module")
def alb():
    lib = os.path.join(ROOT, "paper_2606_01927_amd", "libalbireo.so")
    if not os.path.exists(lib):
        pytest.skip("library not built")
    import paper_2606_01927_amd

    return paper_2606_01927_amd


def test_header_declares_the_entry_points():
    assert _declared() == sorted(["albireo_apply_penalties", "albireo_backfill", "albireo_philox_uniforms",
                                  "albireo_penalty_state_append", "albireo_penalty_state_init",
                                  "albireo_sample", "albireo_sample_noalloc", "albireo_sample_route",
                                  "albireo_sample_sharded",
                                  "albireo_sample_step",
                                  "albireo_status_string",
                                  "albireo_topk_topp", "albireo_workspace_size"])


def test_library_exports_every_declared_symbol(alb):
    lib = ctypes.CDLL(alb.LIB_PATH)
    for name in _declared():
        assert hasattr(lib, name), name
    assert set(_declared()) == set(alb.EXPORTED)


def test_status_strings(alb):
    for st in range(6):
        assert alb.status_string(st)
    assert alb.status_string(99) == "unknown status"


def _sample(alb, **kw):
    args = dict(logits=0x1000, dtype=alb.BF16, B=4, V=1000, ld=1000, params=None, uniforms=0x2000,
                ids=0x3000, lps=0x4000, n_top=0, tids=None, tlps=None, flags=None, ws=None, wsb=0, stream=None)
    args.update(kw)
    f = alb.raw_call("albireo_sample")
    return f(args["logits"], args["dtype"], args["B"], args["V"], args["ld"], args["params"], args["uniforms"],
             args["ids"], args["lps"], args["n_top"], args["tids"], args["tlps"], args["flags"], args["ws"],
             args["wsb"], args["stream"])


def test_argument_errors_return_before_any_launch(alb):
    E = alb.E_INVALID
    assert _sample(alb, dtype=7) == E
    assert _sample(alb, B=-1) == E
    assert _sample(alb, V=0) == E
    assert _sample(alb, ld=999) == E
    assert _sample(alb, n_top=33) == E
    assert _sample(alb, n_top=-1) == E
    assert _sample(alb, logits=None) == E
    assert _sample(alb, logits=0x1001) == E           # misaligned for bf16
    assert _sample(alb, uniforms=None) == E
    assert _sample(alb, ids=None) == E
    assert _sample(alb, n_top=5) == E                  # top-n outputs missing
    assert _sample(alb, V=1 << 31, ld=1 << 31) == alb.E_UNSUPPORTED
    assert _sample(alb, B=0) == alb.OK                 # nothing to do, nothing launched


def test_penalty_and_filter_entry_points_validate(alb):
    pen = alb.raw_call("albireo_apply_penalties")
    assert pen(0x1000, alb.BF16, 2, 100, 50, None, 0x2000, None, 0, None) == alb.E_INVALID     # ld < V
    assert pen(0x1000, alb.BF16, 2, 100, 100, None, None, None, 0, None) == alb.E_INVALID     # no output
    assert pen(0x1000, alb.BF16, 2, 100, 100, None, 0x1000, None, 0, None) == alb.E_INVALID   # bf16 alias
    assert pen(0x1000, alb.F32, 0, 100, 100, None, 0x2000, None, 0, None) == alb.OK
    tt = alb.raw_call("albireo_topk_topp")
    assert tt(0x1002, 2, 100, 100, None, None, None, None, None, None, None, 0, None) == alb.E_INVALID
    assert tt(0x1000, 0, 100, 100, None, None, None, None, None, None, None, 0, None) == alb.OK
    # history length must be non-negative and come with ids
    p = alb.Params()
    p.hist_offsets = 0x5000
    p.hist_ids = None
    p.hist_len = 10
    assert _sample(alb, params=ctypes.pointer(p)) == alb.E_INVALID
    p.hist_len = -1
    assert _sample(alb, params=ctypes.pointer(p)) == alb.E_INVALID


def test_workspace_size_without_rows(alb):
    assert alb.workspace_size(0, 1000, __import__("torch").bfloat16) == 256


def test_step_rng_and_backfill_entry_points_validate(alb):
    step_fn = alb.raw_call("albireo_sample_step")

    def call(st, **kw):
        a = dict(logits=0x1000, dtype=alb.BF16, B=4, V=1000, ld=1000, ids=0x3000, lps=0x4000, n_top=0)
        a.update(kw)
        return step_fn(a["logits"], a["dtype"], a["B"], a["V"], a["ld"], None, st, a["ids"], a["lps"], a["n_top"],
                       None, None, None, None, 0, None)

    assert call(None) == alb.E_INVALID                           # no step struct
    st = alb._Step(seed=1, step=2, seq_ids=None, next_tokens=0x6000, backfill_dest=None, next_len=8)
    assert call(ctypes.pointer(st)) == alb.E_INVALID             # backfill without destinations
    st.backfill_dest = 0x7000
    st.next_len = -1
    assert call(ctypes.pointer(st)) == alb.E_INVALID             # negative slot count
    st.next_len = 8
    assert call(ctypes.pointer(st), B=0) == alb.OK               # nothing to do, nothing launched
    assert call(ctypes.pointer(st), ids=None) == alb.E_INVALID
    rng = alb.raw_call("albireo_philox_uniforms")
    assert rng(1, 2, None, -1, 0x1000, None) == alb.E_INVALID
    assert rng(1, 2, None, 5, None, None) == alb.E_INVALID
    assert rng(1, 2, None, 0, None, None) == alb.OK
    bf = alb.raw_call("albireo_backfill")
    assert bf(0x1000, 0x2000, -1, 0x3000, 4, None) == alb.E_INVALID
    assert bf(0x1000, None, 3, 0x3000, 4, None) == alb.E_INVALID
    assert bf(0x1000, 0x2000, 3, 0x3000, -1, None) == alb.E_INVALID
    assert bf(None, None, 0, None, 0, None) == alb.OK


def test_sharded_entry_point_validates(alb):
    fn = alb.raw_call("albireo_sample_sharded")
    st = alb._Step(seed=1, step=2, seq_ids=None, next_tokens=None, backfill_dest=None, next_len=0)

    def call(shards, uniforms=0x5000, step=None, **kw):
        a = dict(logits=0x10000, dtype=alb.BF16, B=4, V=1000, ld=256, ids=0x3000, lps=0x4000)
        a.update(kw)
        sh = None if shards is None else ctypes.pointer(alb._Shards(*shards))
        return fn(a["logits"], a["dtype"], a["B"], a["V"], a["ld"], sh, None, uniforms, step, a["ids"], a["lps"],
                  0, None, None, None, None, 0, None)

    assert call(None) == alb.E_INVALID                                   # no layout
    assert call((256, 1024), uniforms=None) == alb.E_INVALID             # neither uniforms nor step
    assert call((256, 1024), step=ctypes.pointer(st)) == alb.E_INVALID   # both
    assert call((0, 1024)) == alb.E_INVALID                              # empty blocks
    assert call((256, 128)) == alb.E_INVALID                             # blocks of a row overlap
    assert call((256, 1024), ld=100) == alb.E_INVALID                    # rows overlap inside a block
    assert call((252, 1024)) == alb.E_UNSUPPORTED                        # a 16-byte slot crosses blocks
    assert call((256, 1028)) == alb.E_UNSUPPORTED                        # misaligned block stride
    assert call((256, 1024), logits=0x10008) == alb.E_UNSUPPORTED        # misaligned base
    assert call((256, 1024), ld=260) == alb.E_UNSUPPORTED                # misaligned row stride
    assert call((256, 1024), B=0) == alb.OK                              # nothing to do, nothing launched
    assert call((256, 1024), ids=None) == alb.E_INVALID


def test_batch_padding_and_shard_length(alb):
    import torch

    assert [alb.padded_batch(s, 8) for s in (0, 1, 8, 9, 250, 256)] == [0, 8, 8, 16, 256, 256]
    assert alb.shard_len_for(152064, 8, torch.bfloat16) == 19008
    assert alb.shard_len_for(32000, 8, torch.bfloat16) == 4000
    assert alb.shard_len_for(32001, 8, torch.bfloat16) == 4008    # ceil(V / t), whole 16-byte slots
    assert alb.shard_len_for(32001, 8, torch.float32) == 4004
    assert alb.shard_len_for(10, 3, torch.float32) == 4
