"""Pins for the oracle's device-random-number and backfill definitions (O-11, O-12).

* Philox-4x32-10 against the generator's published known-answer vectors (tests/golden/philox_kat.json);
* the uniform mapping: 24-bit multiples in [0, 1), the first output word's top 24 bits, a loose
  uniformity check, and the counter layout (step in words 0-1, sequence id in words 2-3);
* the paper's determinism claim for sequence-parallel sampling (sec. 6.2): a worker that generates the
  numbers of its own rows from their sequence ids gets what a single worker gets for those rows;
* backfill (sec. 5): a hand-worked scatter, and skipped rows leave slots untouched.
"""
from __future__ import annotations

import json
import os

import numpy as np

HERE = os.path.dirname(os.path.abspath(__file__))
KAT = json.load(open(os.path.join(HERE, "golden", "philox_kat.json")))["cases"]


def _words(hexes):
    return np.array([int(h, 16) for h in hexes], dtype=np.uint32)


def test_philox_known_answers(oracle_mod):
    for case in KAT:
        got = oracle_mod.philox4x32_10(_words(case["counter"]), _words(case["key"]))
        assert list(got) == list(_words(case["out"])), case


def test_uniform_is_top_24_bits_of_word0(oracle_mod):
    seed, step = 0x0123456789ABCDEF, 77
    seq = np.array([0, 1, 5, -1, 2**40 + 3], dtype=np.int64)
    u = oracle_mod.philox_uniforms(seed, step, seq)
    for i, s in enumerate(seq.astype(np.uint64)):
        ctr = np.array([step & 0xFFFFFFFF, step >> 32, int(s) & 0xFFFFFFFF, int(s) >> 32], np.uint32)
        key = np.array([seed & 0xFFFFFFFF, seed >> 32], np.uint32)
        w0 = int(oracle_mod.philox4x32_10(ctr, key)[0])
        assert u[i] == np.float32((w0 >> 8) / 2.0**24)


def test_uniform_range_and_grid(oracle_mod):
    u = oracle_mod.philox_uniforms(1234, 5, B=200000)
    assert u.dtype == np.float32
    assert np.all(u >= 0.0) and np.all(u < 1.0)
    k = u.astype(np.float64) * 2.0**24
    assert np.all(k == np.floor(k))


def test_uniformity_loose(oracle_mod):
    u = oracle_mod.philox_uniforms(99, 3, B=1 << 16).astype(np.float64)
    assert abs(u.mean() - 0.5) < 0.01
    h, _ = np.histogram(u, bins=16, range=(0.0, 1.0))
    exp = u.size / 16
    chi2 = float(((h - exp) ** 2 / exp).sum())
    assert chi2 < 60.0  # 15 degrees of freedom; a broken mapping is far above this


def test_counter_layout_and_defaults(oracle_mod):
    a = oracle_mod.philox_uniforms(7, 11, B=64)
    b = oracle_mod.philox_uniforms(7, 11, np.arange(64))
    assert np.array_equal(a, b)  # no sequence ids: the row index
    c = oracle_mod.philox_uniforms(7, 12, np.arange(64))
    d = oracle_mod.philox_uniforms(8, 11, np.arange(64))
    assert not np.array_equal(a, c) and not np.array_equal(a, d)
    # step 2^32 differs from step 0 (the high word of the step is in the counter)
    e = oracle_mod.philox_uniforms(7, 0, np.arange(64))
    f = oracle_mod.philox_uniforms(7, 2**32, np.arange(64))
    assert not np.array_equal(e, f)


def test_rank_slices_draw_what_one_worker_draws(oracle_mod):
    seq = np.random.default_rng(0).integers(0, 2**50, size=96, dtype=np.int64)
    full = oracle_mod.philox_uniforms(2026, 9, seq)
    for t in (2, 3, 4, 8):
        parts = [oracle_mod.philox_uniforms(2026, 9, part) for part in np.array_split(seq, t)]
        assert np.array_equal(np.concatenate(parts), full)


def test_backfill_hand_worked(oracle_mod):
    nxt = np.array([10, 11, 12, 13], np.int32)
    out = oracle_mod.backfill([5, 7, 9], [2, -1, 0], nxt)
    assert list(out) == [9, 11, 5, 13]
    assert list(nxt) == [10, 11, 12, 13]  # the input is not modified


def test_backfill_skips_out_of_range_rows(oracle_mod):
    out = oracle_mod.backfill([1, 2, 3, 4], [4, -5, 100, 1], np.zeros(4, np.int32))
    assert list(out) == [0, 4, 0, 0]
