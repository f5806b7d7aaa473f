"""Pins for the oracle's all-to-all receive layout (O-13).

The all-to-all that replaces the gather (sec. 6.1, Eq. opt_sample; sec. 6.2, "Efficient logit
exchange") sends each worker the vocabulary-shard columns of its own rows.  The pins build such
buffers from first principles (numpy block copies of one worker's shard for another worker's rows),
never from the element formula, and check that the oracle reads the original rows back:

* an emulated exchange over t workers, including a vocabulary that does not divide by t (the last
  shard partly used, its padding NaN and never read);
* blocks placed with row and block strides larger than the packed ones (gaps full of NaN);
* one block (t = 1) is the row-major matrix;
* sampling the received rows is sampling the original rows (sec. 6: the per-row computation does not
  change when the rows are split across workers).
"""
from __future__ import annotations

import numpy as np
import pytest

import workloads


def _exchange(X, t, L, pad_value):
    """Emulate the exchange: worker w owns columns [w L, (w + 1) L) of every row (past V: padding);
    worker j's receive buffer is, for w = 0 .. t-1, the block of w's shard for j's rows.  Returns
    the t receive buffers (flat) and the rows per worker."""
    s, V = X.shape
    assert s % t == 0
    b = s // t
    shards = []
    for w in range(t):
        sh = np.full((s, L), pad_value, dtype=X.dtype)
        cols = X[:, w * L:min((w + 1) * L, V)]
        sh[:, :cols.shape[1]] = cols
        shards.append(sh)
    recv = []
    for j in range(t):
        blocks = [shards[w][j * b:(j + 1) * b] for w in range(t)]  # what worker w sends to worker j
        recv.append(np.stack(blocks).reshape(-1))
    return recv, b


@pytest.mark.parametrize("t,s,V,L", [(2, 6, 40, 20), (4, 8, 30, 8), (8, 16, 100, 16), (3, 3, 7, 3)])
def test_exchange_round_trip_f32(t, s, V, L, oracle_mod):
    X = np.arange(s * V, dtype=np.float32).reshape(s, V) + 0.5
    recv, b = _exchange(X, t, L, np.float32(np.nan))
    for j in range(t):
        got = oracle_mod.receive_rows(recv[j], b, V, L, L, b * L)
        assert np.array_equal(got, X[j * b:(j + 1) * b]), j


def test_exchange_round_trip_bf16_bits(oracle_mod):
    t, s, V, L = 4, 12, 150, 40  # last shard holds 30 of its 40 columns
    rng = np.random.default_rng(3)
    X = rng.integers(0, 0x7F00, size=(s, V)).astype(np.uint16)
    recv, b = _exchange(X, t, L, np.uint16(0x7FC0))  # bf16 NaN in the padding columns
    for j in range(t):
        got = oracle_mod.receive_rows(recv[j], b, V, L, L, b * L)
        assert np.array_equal(got, X[j * b:(j + 1) * b])
        assert not np.any(got == 0x7FC0)


def test_strided_blocks(oracle_mod):
    B, V, L, ld, S = 5, 37, 10, 13, 80  # row stride > L, block stride > B * ld
    t = -(-V // L)
    rng = np.random.default_rng(11)
    X = rng.standard_normal((B, V)).astype(np.float32)
    buf = np.full((t, S), np.nan, dtype=np.float32)
    for w in range(t):
        blk = buf[w, :B * ld].reshape(B, ld)
        cols = X[:, w * L:min((w + 1) * L, V)]
        blk[:, :cols.shape[1]] = cols
    got = oracle_mod.receive_rows(buf, B, V, ld, L, S)
    assert np.array_equal(got, X)


def test_one_block_is_row_major(oracle_mod):
    rng = np.random.default_rng(5)
    B, V, ld = 4, 33, 40
    M = rng.standard_normal((B, ld)).astype(np.float32)
    got = oracle_mod.receive_rows(M, B, V, ld, V, 10**6)  # the block stride is never used
    assert np.array_equal(got, M[:, :V])


def test_sampling_the_received_rows(oracle_mod):
    t = 4
    w = workloads.generate(3, B=8, V=2048, H=300)
    L = w.V // t
    recv, b = _exchange(w.logits, t, L, np.uint16(0))
    for j in range(t):
        part = w.row_slice(j * b, (j + 1) * b)
        ref = oracle_mod.sample(part)
        part.logits = oracle_mod.receive_rows(recv[j], b, w.V, L, L, b * L)
        part.ld = w.V
        got = oracle_mod.sample(part)
        assert np.array_equal(got["ids"], ref["ids"])
        assert np.array_equal(got["logprobs"], ref["logprobs"])
