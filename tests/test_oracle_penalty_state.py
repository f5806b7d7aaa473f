"""Pins for the oracle's split penalties and penalty state (O-14, O-15).

* hand-worked rows with a prompt history and an output history (tests/golden/prompt_split.json):
  repetition over prompt and output ids, frequency and presence over output counts only;
* the state of a sequence (distinct ids of prompt and output, output counts, prompt flags) on a
  hand-worked example, and its invariants on random histories;
* the incremental property the on-device state relies on: folding one more sampled id into the state
  gives the state of the longer output.
"""
from __future__ import annotations

import json
import os

import numpy as np
import pytest

from tests.test_oracle_pins import row_workload

HERE = os.path.dirname(os.path.abspath(__file__))
CASES = json.load(open(os.path.join(HERE, "golden", "prompt_split.json")))["cases"]


def _split_workload(c):
    w = row_workload(c["x"], T=c.get("T", 1.0), rep=c["rep"], freq=c["freq"], pres=c["pres"], hist=c["out"])
    w.prompt_offsets = np.array([0, len(c["prompt"])], np.int64)
    w.prompt_ids = np.array(c["prompt"], np.int32)
    return w


@pytest.mark.parametrize("case", CASES, ids=[c["name"] for c in CASES])
def test_split_worked_example(case, oracle_mod):
    r = oracle_mod.sample(_split_workload(case), penalised=True)
    got = r["penalised"][0]
    assert np.array_equal(got, np.array(case["expect_penalised"], np.float32))
    if case.get("expect_signbit0"):
        assert np.signbit(got[0])
    if "expect_id" in case:
        assert r["ids"][0] == case["expect_id"]
    if "expect_flags" in case:
        assert r["flags"][0] == case["expect_flags"]
    if "expect_flag_bits" in case:
        assert r["flags"][0] & case["expect_flag_bits"]


def test_state_worked_example(oracle_mod):
    st = oracle_mod.penalty_state([5, 3, 5], [3, 9, 9, 9, -1, 12], V=10)
    assert st == {5: (0, True), 3: (1, True), 9: (3, False)}


def test_state_invariants(oracle_mod):
    rng = np.random.default_rng(7)
    V = 500
    for _ in range(20):
        prompt = rng.integers(-5, V + 5, size=rng.integers(0, 80))
        out = rng.integers(-5, V + 5, size=rng.integers(0, 80))
        st = oracle_mod.penalty_state(prompt, out, V)
        valid_out = out[(out >= 0) & (out < V)]
        valid_prompt = prompt[(prompt >= 0) & (prompt < V)]
        assert sum(c for c, _ in st.values()) == valid_out.size
        assert {t for t, (_, f) in st.items() if f} == set(valid_prompt.tolist())
        assert set(st) == set(valid_out.tolist()) | set(valid_prompt.tolist())
        for t, (c, _) in st.items():
            assert c == int(np.sum(valid_out == t))


def test_state_folds_one_sampled_id(oracle_mod):
    rng = np.random.default_rng(8)
    V = 64
    prompt = rng.integers(0, V, size=30)
    out = list(rng.integers(0, V, size=10))
    st = oracle_mod.penalty_state(prompt, out, V)
    for t in rng.integers(0, V, size=25):
        c, f = st.get(int(t), (0, False))
        st[int(t)] = (c + 1, f)
        out.append(int(t))
        assert st == oracle_mod.penalty_state(prompt, out, V)


def test_split_matches_single_history_without_prompt(oracle_mod):
    """With an empty prompt for every row the split rule is the single-history rule: the same rows
    sampled both ways agree exactly (a prompt history of length 0 adds nothing)."""
    import workloads

    w = workloads.generate(3, B=6, V=3000, H=400)
    ref = oracle_mod.sample(w, penalised=True)
    w.prompt_offsets = np.zeros(w.B + 1, np.int64)
    w.prompt_ids = np.zeros(0, np.int32)
    got = oracle_mod.sample(w, penalised=True)
    assert np.array_equal(ref["penalised"], got["penalised"])
    assert np.array_equal(ref["ids"], got["ids"])
