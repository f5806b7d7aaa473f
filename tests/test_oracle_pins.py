"""Pins for the CPU oracle: values it must reproduce that come from somewhere other than itself.

* hand-worked examples with closed-form answers (tests/golden/worked_examples.json);
* special cases that reduce to numpy routines (float64 log-softmax, cumsum + searchsorted for the
  inverse CDF, argmax, partition for the k-th largest);
* brute-force enumeration on tiny vocabularies (nucleus as a minimal subset, interval measure of the
  inverse CDF);
* invariants that hold at any size (mass sums, nesting of kept sets, logprob identities);
* the paper's two correctness claims for sequence-parallel sampling (sec. 6.2): splitting the rows
  across workers with each worker consuming its slice of the pre-generated randoms does not change
  any row's result, and padded rows do not affect real rows.
"""
from __future__ import annotations

import json
import math
import os

import numpy as np
import pytest

import workloads
from tests import brute

HERE = os.path.dirname(os.path.abspath(__file__))
CASES = json.load(open(os.path.join(HERE, "golden", "worked_examples.json")))["cases"]


def _f(v):
    return -np.inf if v == "-inf" else (np.inf if v == "inf" else float(v))


def row_workload(x, T=1.0, k=0, p=1.0, min_p=0.0, rep=None, freq=None, pres=None, hist=None, u=0.5,
                 n_top=0, dtype="f32"):
    x = np.array([[_f(v) for v in x]], dtype=np.float32)
    V = x.shape[1]
    w = workloads.Workload(name="row", B=1, V=V, dtype=dtype, ld=V,
                           logits=workloads.to_bf16_bits(x) if dtype == "bf16" else x,
                           uniforms=np.array([u], np.float32),
                           temperature=np.array([T], np.float32), top_k=np.array([k], np.int32),
                           top_p=np.array([p], np.float32), min_p=np.array([min_p], np.float32),
                           n_top=n_top)
    if hist is not None:
        w.repetition_penalty = np.array([1.0 if rep is None else rep], np.float32)
        w.frequency_penalty = np.array([0.0 if freq is None else freq], np.float32)
        w.presence_penalty = np.array([0.0 if pres is None else pres], np.float32)
        w.hist_offsets = np.array([0, len(hist)], np.int64)
        w.hist_ids = np.array(hist, np.int32)
    return w


def _case_workload(c):
    return row_workload(c["x"], T=c.get("T", 1.0), k=c.get("k", 0), p=c.get("p", 1.0),
                        min_p=c.get("min_p", 0.0), rep=c.get("rep"), freq=c.get("freq"),
                        pres=c.get("pres"), hist=c.get("hist"), u=c.get("u", 0.5),
                        n_top=c.get("n_top", 0))


@pytest.mark.parametrize("case", CASES, ids=[c["name"] for c in CASES])
def test_worked_example(case, oracle_mod):
    w = _case_workload(case)
    r = oracle_mod.sample(w, probs=True, penalised=True)
    tol = case.get("tol", 0.0)
    if "expect_penalised" in case:
        np.testing.assert_allclose(r["penalised"][0], np.array(case["expect_penalised"], np.float32),
                                   rtol=0, atol=tol)
    if "expect_S" in case:
        S = set(np.nonzero(r["probs"][0] > 0)[0].tolist())
        assert S == set(case["expect_S"])
        assert r["kept"][0] == len(case["expect_S"])
    if "expect_threshold" in case:
        assert r["threshold"][0] == case["expect_threshold"]
    if "expect_probs" in case:
        np.testing.assert_allclose(r["probs"][0], case["expect_probs"], rtol=0, atol=max(tol, 1e-12))
    if "expect_id" in case:
        assert r["ids"][0] == case["expect_id"]
    if "expect_cdf_margin" in case:
        assert abs(r["cdf_margin"][0] - case["expect_cdf_margin"]) <= max(tol, 1e-12)
    if "expect_topp_margin" in case:
        assert abs(r["topp_margin"][0] - case["expect_topp_margin"]) <= max(tol, 1e-12)
    if "expect_log_norm" in case:
        assert abs(r["log_norm"][0] - case["expect_log_norm"]) <= max(tol, 1e-12)
    if "expect_flags" in case:
        assert r["flags"][0] == case["expect_flags"]
    if "expect_logprob" in case:
        assert abs(r["logprobs"][0] - case["expect_logprob"]) <= tol
    if "expect_top_ids" in case:
        assert r["top_ids"][0].tolist() == case["expect_top_ids"]
    if "expect_top_logprobs" in case:
        want = np.array([_f(v) for v in case["expect_top_logprobs"]])
        got = r["top_logprobs"][0]
        assert (np.isinf(got) == np.isinf(want)).all()
        fin = np.isfinite(want)
        np.testing.assert_allclose(got[fin], want[fin], rtol=0, atol=max(tol, 1e-12))


# ---------------------------------------------------------------- numpy special cases

def _rand_rows(seed, B, V, scale=2.0):
    rng = np.random.default_rng(seed)
    return rng.normal(0, scale, size=(B, V)).astype(np.float32), rng.random(B).astype(np.float32)


def _plain(x, u, **kw):
    B, V = x.shape
    w = workloads.Workload(name="plain", B=B, V=V, dtype="f32", ld=V, logits=x, uniforms=u, **kw)
    return w


def test_no_filters_is_softmax_and_searchsorted(oracle_mod):
    """T=1, no penalties, no filters: logprobs are float64 log-softmax of the fp32 logits and the draw
    is numpy's searchsorted over the cumulative distribution (first index with cumsum > u)."""
    x, u = _rand_rows(1, 16, 777)
    r = oracle_mod.sample(_plain(x, u), probs=True)
    xd = x.astype(np.float64)
    lsm = xd - xd.max(1, keepdims=True)
    lsm = lsm - np.log(np.exp(lsm).sum(1, keepdims=True))
    for i in range(16):
        pi = np.exp(lsm[i])
        np.testing.assert_allclose(r["probs"][i], pi, rtol=1e-12, atol=1e-15)
        want = int(np.searchsorted(np.cumsum(pi), float(u[i]), side="right"))
        if r["cdf_margin"][i] > 1e-9:
            assert r["ids"][i] == want
        assert abs(r["logprobs"][i] - lsm[i, r["ids"][i]]) < 1e-12
        assert r["kept"][i] == 777


def test_greedy_is_argmax_with_ties(oracle_mod):
    x, u = _rand_rows(2, 8, 501)
    x[3, [17, 400]] = x[3].max() + 1.0  # tie at the maximum: the lower id wins
    r = oracle_mod.sample(_plain(x, u, temperature=np.zeros(8, np.float32)))
    assert (r["ids"] == np.argmax(x, axis=1)).all()
    assert r["ids"][3] == 17
    assert (r["flags"] & oracle_mod.GREEDY).all()


def test_topk_threshold_is_partition(oracle_mod):
    x, u = _rand_rows(3, 12, 1000)
    x[5, :300] = np.float32(0.25)  # heavy ties
    ks = np.array([1, 2, 5, 40, 999, 300, 7, 8, 64, 100, 500, 10], np.int32)
    r = oracle_mod.sample(_plain(x, u, top_k=ks), probs=True)
    for i in range(12):
        kth = np.partition(x[i], 1000 - ks[i])[1000 - ks[i]]
        assert r["threshold"][i] == kth
        assert r["kept"][i] == int((x[i] >= kth).sum())
        assert set(np.nonzero(r["probs"][i])[0]) == set(np.nonzero(x[i] >= kth)[0])


def test_minp_matches_probability_ratio(oracle_mod):
    """min-p keeps p_v >= min_p * p_max; away from the boundary this equals the canonical fp32 rule."""
    x, u = _rand_rows(4, 10, 3000, scale=1.5)
    mp = np.linspace(0.01, 0.5, 10).astype(np.float32)
    r = oracle_mod.sample(_plain(x, u, min_p=mp), probs=True)
    for i in range(10):
        ratio = np.exp(x[i].astype(np.float64) - x[i].max())
        away = np.abs(ratio - mp[i]) > 1e-5
        kept = r["probs"][i] > 0
        assert (kept[away] == (ratio[away] >= mp[i])).all()


# ---------------------------------------------------------------- brute force on tiny vocabularies

@pytest.mark.parametrize("seed", range(40))
def test_nucleus_and_topk_by_enumeration(seed, oracle_mod):
    rng = np.random.default_rng(100 + seed)
    V = int(rng.integers(2, 9))
    x = rng.normal(0, 1.5, size=V).astype(np.float32)
    while len(set(x.tolist())) < V:
        x = rng.normal(0, 1.5, size=V).astype(np.float32)
    p = float(rng.uniform(0.05, 0.99))
    k = int(rng.integers(0, V + 1))
    T = float(rng.uniform(0.5, 1.5))
    w = row_workload(x, T=T, k=k, p=p)
    r = oracle_mod.sample(w, probs=True)
    # reconstruct the canonical z and masses exactly as defined, then enumerate
    rr = np.float32(1.0 / np.float64(np.float32(T)))
    z = (x * rr).astype(np.float32)
    S2 = brute.topk_by_definition(z.tolist(), k)
    ids = sorted(S2)
    m = float(z.max())
    mass = [math.exp(float(z[i]) - m) for i in ids]
    if r["topp_margin"][0] > 1e-9:
        nuc = brute.nucleus_by_enumeration(mass, np.float32(p))
        want = set(ids[j] for j in nuc)
        assert set(np.nonzero(r["probs"][0])[0]) == want


@pytest.mark.parametrize("seed", range(10))
def test_draw_interval_measure(seed, oracle_mod):
    """For tiny V the set of u drawing id v has measure pi_v (checked on a grid of u)."""
    rng = np.random.default_rng(200 + seed)
    V = int(rng.integers(2, 7))
    x = rng.normal(0, 1.0, size=V).astype(np.float32)
    x[rng.integers(0, V)] = -np.inf if V > 2 else x[0]
    grid = 4000
    us = ((np.arange(grid) + 0.5) / grid).astype(np.float32)
    B = grid
    X = np.repeat(x[None, :], B, axis=0)
    w = workloads.Workload(name="g", B=B, V=V, dtype="f32", ld=V, logits=X, uniforms=us,
                           top_p=np.full(B, 0.9, np.float32))
    r = oracle_mod.sample(w, probs=True)
    pi = r["probs"][0]
    frac = np.bincount(r["ids"], minlength=V) / grid
    np.testing.assert_allclose(frac, pi, atol=2.0 / grid)


# ---------------------------------------------------------------- invariants on the real recipes

@pytest.mark.parametrize("cfg,B,V", [(1, 4, 32000), (2, 32, 4099), (3, 16, 5003), (4, 16, 6007), (5, 32, 7001)])
def test_invariants(cfg, B, V, oracle_mod):
    w = workloads.generate(cfg, B=B, V=V, H=64)
    r = oracle_mod.sample(w, probs=True, penalised=True)
    for i in range(B):
        if r["flags"][i] & (oracle_mod.EMPTY | oracle_mod.BAD_INPUT):
            continue
        pr = r["probs"][i]
        assert abs(pr.sum() - 1.0) < 1e-9
        S = pr > 0
        assert S[r["ids"][i]]
        # S is an upper set of z
        T = w.temperature[i]
        rr = np.float32(1.0) if T < 1e-5 else np.float32(1.0 / np.float64(T))
        z = r["penalised"][i] * rr
        assert z[S].min() >= z[~S & np.isfinite(z)].max(initial=-np.inf) or S.all()
        assert r["logprobs"][i] <= 1e-12
        assert abs(r["logprobs"][i] - (float(z[r["ids"][i]]) - r["lse"][i])) < 1e-9
        if T >= 1e-5 and w.top_p is not None and w.top_p[i] < 1:
            # filtered mass >= top_p: S carries at least p of the mass renormalised over S2
            tau2 = -np.inf
            if w.top_k is not None and 0 < w.top_k[i] < V:
                tau2 = np.sort(z)[::-1][w.top_k[i] - 1]
            if w.min_p is not None and w.min_p[i] > 0:
                tau2 = max(tau2, np.float32(z.max() + np.float32(np.log(np.float64(min(w.min_p[i], 1.0))))))
            S2 = np.isfinite(z) & (z >= tau2)
            mass = np.exp(z.astype(np.float64) - z.max())
            assert mass[S].sum() / mass[S2].sum() >= w.top_p[i] - 1e-9
        if T >= 1e-5 and w.top_k is not None and w.top_k[i] == 1:
            assert z[r["ids"][i]] == z.max()


def test_topk1_and_p_to_zero_pick_the_argmax_group(oracle_mod):
    x, u = _rand_rows(5, 20, 900)
    x[:, 3] = x.max() + 2
    x[:, 11] = x[:, 3]
    for kw in (dict(top_k=np.ones(20, np.int32)), dict(top_p=np.full(20, 1e-7, np.float32))):
        r = oracle_mod.sample(_plain(x.copy(), u, **kw))
        assert set(r["ids"].tolist()) <= {3, 11}


# ---------------------------------------------------------------- the paper's parallel-sampling claims

def test_row_split_invariance(oracle_mod):
    """sec. 6.2: each worker samples its slice of rows with its slice of the pre-generated uniforms;
    the outcome must equal single-worker sampling."""
    w = workloads.generate(5, B=24, V=3001, H=50)
    full = oracle_mod.sample(w)
    for t in (2, 3, 4, 8):
        step = -(-24 // t)
        parts = [oracle_mod.sample(w.row_slice(a, min(a + step, 24))) for a in range(0, 24, step)]
        for k in ("ids", "logprobs", "top_ids", "top_logprobs", "flags"):
            assert np.array_equal(np.concatenate([p[k] for p in parts]), full[k])


def test_padding_rows_do_not_change_real_rows(oracle_mod):
    """sec. 6.2 batch padding: synthetic rows appended to reach a multiple of t are dropped and must not
    affect real rows."""
    w = workloads.generate(2, B=10, V=2003)
    base = oracle_mod.sample(w)
    pad = workloads.generate(1, B=6, V=2003)
    ww = w.row_slice(0, 10)
    ww.B = 16
    ww.logits = np.concatenate([w.logits, workloads.to_bf16_bits(pad.logits)])
    ww.uniforms = np.concatenate([w.uniforms, pad.uniforms])
    for f in ("temperature", "top_k", "top_p"):
        ww.__dict__[f] = np.concatenate([getattr(w, f), getattr(pad, f)])
    got = oracle_mod.sample(ww)
    for k in ("ids", "logprobs", "flags"):
        assert np.array_equal(got[k][:10], base[k])


# ---------------------------------------------------------------- data faults and parameters

def test_bad_inputs_and_params_are_flagged(oracle_mod):
    w = row_workload([1.0, float("nan"), 0.5], u=0.2)
    assert oracle_mod.sample(w)["flags"][0] & oracle_mod.BAD_INPUT
    w = row_workload([1.0, 2.0, 0.5], hist=[0, 7], rep=1.1, u=0.2)
    assert oracle_mod.sample(w)["flags"][0] & oracle_mod.BAD_INPUT
    w = row_workload([1.0, 2.0, 0.5], hist=[0], rep=-1.0, u=0.2)
    r = oracle_mod.sample(w, penalised=True)
    assert r["flags"][0] & oracle_mod.BAD_PARAM
    assert r["penalised"][0].tolist() == [1.0, 2.0, 0.5]  # treated as rep = 1
    w = row_workload([1.0, 2.0, 0.5], p=float("nan"), u=0.2)
    assert oracle_mod.sample(w)["flags"][0] & oracle_mod.BAD_PARAM


def test_bf16_widening_is_exact(oracle_mod):
    x = np.array([[1.0, -2.5, 3.140625, 1e-3]], np.float32)
    bits = workloads.to_bf16_bits(x)
    w = row_workload(x[0], dtype="bf16")
    r = oracle_mod.sample(w, penalised=True)
    want = (bits.astype(np.uint32) << 16).view(np.float32)
    assert np.array_equal(r["penalised"], want)
