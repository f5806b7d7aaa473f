"""GPU parity of the decoding-step extras: device uniforms (Philox-4x32-10, sec. 6.2) and the
early-feedback backfill (sec. 5), through the C ABI against the CPU oracle."""
from __future__ import annotations

import sys

import numpy as np
import pytest

import workloads
from tests.parity import compare_sample, np_

pytestmark = pytest.mark.gpu


def _say(*a):
    print(*a, flush=True)
    sys.stdout.flush()


@pytest.fixture(scope="module")
def lib():
    import torch

    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    import paper_2606_01927_amd as alb

    return alb


SEEDS = [(0, 0), (2026, 7), (0xFFFFFFFFFFFFFFFF, 2**32 + 5), (0x0123456789ABCDEF, 2**63 + 11)]


@pytest.mark.parametrize("B", [1, 255, 256, 1000, 100003])
def test_philox_uniforms_bit_exact(B, lib, oracle_mod):
    import torch

    rng = np.random.default_rng(B)
    for seed, step in SEEDS:
        _say("philox", B, hex(seed), step)
        seq = rng.integers(-(2**62), 2**62, size=B, dtype=np.int64)
        got = np_(lib.philox_uniforms(seed, step, torch.from_numpy(seq).cuda()))
        ref = oracle_mod.philox_uniforms(seed, step, seq)
        assert np.array_equal(got.view(np.uint32), ref.view(np.uint32))
        got0 = np_(lib.philox_uniforms(seed, step, B=B, device="cuda"))  # no ids: the row index
        assert np.array_equal(got0.view(np.uint32), oracle_mod.philox_uniforms(seed, step, B=B).view(np.uint32))


def _seq_ids(B, salt):
    return np.random.default_rng(1000 + salt).integers(0, 2**40, size=B, dtype=np.int64)


CASES = [(1, 4, 32000), (2, 64, 30011), (3, 32, 152064), (4, 8, 152064), (5, 16, 60013), (5, 16, 256000)]


@pytest.mark.parametrize("cfg,B,V", CASES, ids=["c%d_B%d_V%d" % c for c in CASES])
def test_sample_step_matches_sample_and_oracle(cfg, B, V, lib, oracle_mod):
    """Same results as albireo_sample on the uniforms the generator returns (bit-exact), and parity
    with the oracle fed the oracle's own generator."""
    import torch
    from workloads.device import to_device

    w = workloads.generate(cfg, B=B, V=V, H=min(2048, V // 4) if cfg in (3, 5) else None, variant=2)
    seed, step = 0xC0FFEE + cfg, 41 + cfg
    seq = _seq_ids(B, cfg)
    _say("sample_step", cfg, B, V)
    logits, _, p = to_device(w)
    seq_d = torch.from_numpy(seq).cuda()
    out = lib.sample_step(logits, seed, step, seq_d, p, n_top=w.n_top, V=w.V)
    u = lib.philox_uniforms(seed, step, seq_d)
    ref_gpu = lib.sample(logits, u, p, n_top=w.n_top, V=w.V)
    torch.cuda.synchronize()
    for a, b in zip(out, ref_gpu):
        assert np.array_equal(np_(a), np_(b))
    w.uniforms = oracle_mod.philox_uniforms(seed, step, seq)
    rep = compare_sample(oracle_mod.sample(w), out, n_top=w.n_top)
    _say("  ", rep)
    assert rep["band"] <= max(2, B // 8)


def test_rank_slices_sample_what_one_worker_samples(lib):
    """sec. 6.2: a worker that samples a slice of the rows, generating the uniforms of its rows from
    their sequence ids, gets exactly the single-worker ids and logprobs for those rows."""
    import torch
    from workloads.device import to_device

    w = workloads.generate(3, B=96, V=152064, H=2048, variant=3)
    seq = torch.from_numpy(_seq_ids(w.B, 77)).cuda()
    logits, _, p = to_device(w)
    full = lib.sample_step(logits, 99, 3, seq, p, V=w.V)
    torch.cuda.synchronize()
    for t in (2, 4, 8):
        for lo, hi in zip(range(0, w.B, w.B // t), range(w.B // t, w.B + 1, w.B // t)):
            part_w = w.row_slice(lo, hi)
            lg, _, pp = to_device(part_w)
            part = lib.sample_step(lg, 99, 3, seq[lo:hi].contiguous(), pp, V=w.V)
            torch.cuda.synchronize()
            assert np.array_equal(np_(part[0]), np_(full[0])[lo:hi])
            assert np.array_equal(np_(part[1]), np_(full[1])[lo:hi])


@pytest.mark.parametrize("B,n_next", [(1, 1), (7, 3), (256, 300), (1000, 1000), (4099, 5000)])
def test_backfill_bit_exact(B, n_next, lib, oracle_mod):
    import torch

    rng = np.random.default_rng(B + n_next)
    ids = rng.integers(0, 150000, size=B, dtype=np.int32)
    # distinct slots for the scheduled rows; the rest padding (-1) or out of range
    dest = np.full(B, -1, np.int32)
    k = min(B, n_next)
    rows = rng.permutation(B)[:k]
    dest[rows] = rng.permutation(n_next)[:k].astype(np.int32)
    extra = rng.permutation(B)[: B // 10]
    dest[extra] = np.where(rng.random(extra.size) < 0.5, -7, n_next + 3).astype(np.int32)
    nxt = rng.integers(-5, 5, size=n_next, dtype=np.int32)
    _say("backfill", B, n_next)
    got = lib.backfill(torch.from_numpy(ids).cuda(), torch.from_numpy(dest).cuda(), torch.from_numpy(nxt).cuda())
    torch.cuda.synchronize()
    assert np.array_equal(np_(got), oracle_mod.backfill(ids, dest, nxt))


@pytest.mark.parametrize("V", [30011, 200003], ids=["one_workgroup", "streamed"])
def test_sample_step_backfill(V, lib, oracle_mod):
    """The fused backfill writes what the standalone scatter of the same call's ids writes; an empty
    row sends -1; unnamed slots keep their contents.  The streamed width also sends the ids of the
    rows the chunk-parallel general path resolves (the mix's top-p rows without top-k)."""
    import torch
    from workloads.device import to_device

    w = workloads.generate(2, B=64, V=V, variant=4)
    w.logits = np.array(w.logits, copy=True)
    w.logits[5, :] = 0xFF80  # bf16 -inf: an empty row
    logits, _, p = to_device(w)
    rng = np.random.default_rng(5)
    dest = np.full(w.B, -1, np.int32)
    dest[: w.B - 8] = rng.permutation(80)[: w.B - 8].astype(np.int32)
    dest[5] = 3 if 3 not in dest else dest[5]
    nxt0 = np.full(80, 12345, np.int32)
    nxt = torch.from_numpy(nxt0).cuda()
    out = lib.sample_step(logits, 5, 6, None, p, V=w.V, next_tokens=nxt, backfill_dest=torch.from_numpy(dest).cuda())
    torch.cuda.synchronize()
    ids = np_(out[0])
    assert ids[5] == -1 and (np_(out[4])[5] & lib.FLAG_EMPTY)
    assert np.array_equal(np_(nxt), oracle_mod.backfill(ids, dest, nxt0))
