"""GPU parity of the prompt/output penalty split and the per-sequence penalty state, through the C ABI.

* sampling with a prompt history (repetition over prompt and output ids, frequency and presence over the
  output counts) against the oracle (O-14), on single-chunk and multi-chunk rows;
* the state built from the two histories, and the state after several steps of sampled ids, against the
  oracle's state (O-15): the same distinct ids in ascending order, the same output counts and prompt
  marks, bad ids skipped and flagged, rows over capacity flagged;
* sampling from the state against sampling from the histories it stands for (bit-identical outputs) and
  the oracle, before and after the state has followed the sampled tokens.
"""
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


def _with_penalties(w, seed=0):
    rng = np.random.default_rng(seed)
    if w.repetition_penalty is None:
        w.repetition_penalty = rng.uniform(1.05, 1.5, size=w.B).astype(np.float32)
        w.frequency_penalty = rng.uniform(0.0, 0.5, size=w.B).astype(np.float32)
        w.presence_penalty = rng.uniform(-0.2, 0.4, size=w.B).astype(np.float32)
    return w


def _rows(offs, ids, b):
    return np.asarray(ids[offs[b]:offs[b + 1]])


def _csr(lists):
    offs = np.cumsum([0] + [len(x) for x in lists]).astype(np.int64)
    ids = np.concatenate([np.asarray(x, np.int32) for x in lists]) if offs[-1] else np.zeros(0, np.int32)
    return offs, ids


def _state_rows(st):
    ids, cnt, ln, fl = np_(st.ids), np_(st.counts).view(np.uint32), np_(st.len), np_(st.flags)
    rows = []
    for b in range(st.B):
        n = int(ln[b])
        e_ids, e_cnt = ids[b, :n], cnt[b, :n]
        assert np.all(np.diff(e_ids) > 0), "entries of row %d not in ascending id order" % b
        rows.append(({int(i): (int(c & 0x7FFFFFFF), bool(c >> 31)) for i, c in zip(e_ids, e_cnt)}, int(fl[b])))
    return rows


def _dev(a, dt):
    import torch

    return torch.from_numpy(np.ascontiguousarray(a)).to(device="cuda", dtype=dt)


# (config, rows, V, prompt length): single-chunk and multi-chunk rows, bf16 and fp32, top-n
CASES = [(3, 24, 152064, 1024), (5, 16, 60013, 512), (1, 4, 32000, 300), (4, 4, 152064, 256),
         (2, 8, 30011, 2000)]


@pytest.mark.parametrize("cfg,B,V,P", CASES, ids=["c%d_B%d_V%d_P%d" % c for c in CASES])
def test_prompt_split_parity(cfg, B, V, P, lib, oracle_mod):
    import torch

    from workloads.device import to_device

    w = workloads.generate(cfg, B=B, V=V, H=min(2048, V // 4) if cfg in (3, 5) else None, variant=7)
    workloads.add_prompt(w, P, seed=cfg)
    _with_penalties(w, seed=cfg)
    _say("prompt split", cfg, B, V, P)
    logits, u, p = to_device(w)
    out = lib.sample(logits, u, p, n_top=w.n_top, V=V)
    torch.cuda.synchronize()
    rep = compare_sample(oracle_mod.sample(w), out, n_top=w.n_top)
    _say("  ", rep)
    assert rep["band"] <= max(2, B // 8)


def _histories(B, V, seed, P=600, H=400):
    rng = np.random.default_rng(seed)
    prompts = [rng.integers(0, V, size=rng.integers(0, P)) for _ in range(B)]
    outs = [rng.integers(0, V // 8, size=rng.integers(0, H)) for _ in range(B)]  # repeats
    return prompts, outs


def test_state_init_matches_oracle(lib, oracle_mod):
    import torch

    B, V = 37, 5000
    prompts, outs = _histories(B, V, 1)
    prompts[3] = np.concatenate([prompts[3], [-1, V + 3]])  # skipped and flagged
    prompts[4] = np.zeros(0, np.int64)                       # output only
    outs[5] = np.zeros(0, np.int64)                          # prompt only
    prompts[6], outs[6] = np.zeros(0, np.int64), np.zeros(0, np.int64)
    po, pi = _csr(prompts)
    oo, oi = _csr(outs)
    st = lib.PenaltyState(B, cap=2048).init(V, _dev(po, torch.int64), _dev(pi, torch.int32), _dev(oo, torch.int64),
                                           _dev(oi, torch.int32))
    torch.cuda.synchronize()
    got = _state_rows(st)
    for b in range(B):
        ref = oracle_mod.penalty_state(prompts[b], outs[b], V)
        assert got[b][0] == ref, b
        assert got[b][1] == (lib.FLAG_BAD_INPUT if b == 3 else 0), b


def test_state_append_matches_oracle(lib, oracle_mod):
    import torch

    B, V = 21, 3000
    prompts, outs = _histories(B, V, 2)
    po, pi = _csr(prompts)
    oo, oi = _csr(outs)
    st = lib.PenaltyState(B, cap=4096).init(V, _dev(po, torch.int64), _dev(pi, torch.int32), _dev(oo, torch.int64),
                                           _dev(oi, torch.int32))
    rng = np.random.default_rng(3)
    hist = [list(o) for o in outs]
    for step in range(12):
        ids = rng.integers(0, V, size=B).astype(np.int32)
        ids[rng.random(B) < 0.4] = rng.integers(0, V // 8, size=1)[0]   # a repeat of an output id
        ids[step % B] = -1                                               # an EMPTY row
        ids[(step + 5) % B] = V + 7                                      # out of range: no change
        st.append(_dev(ids, torch.int32), V)
        for b in range(B):
            if 0 <= ids[b] < V:
                hist[b].append(int(ids[b]))
    torch.cuda.synchronize()
    got = _state_rows(st)
    for b in range(B):
        assert got[b][0] == oracle_mod.penalty_state(prompts[b], hist[b], V), b
        assert got[b][1] == 0


def test_state_capacity_limit(lib, oracle_mod):
    import torch

    B, V, cap = 3, 1000, 8
    prompts = [np.arange(5), np.arange(20), np.arange(3)]
    outs = [np.array([7, 7]), np.array([]), np.array([100, 200, 300, 400, 500])]
    po, pi = _csr(prompts)
    oo, oi = _csr(outs)
    st = lib.PenaltyState(B, cap=cap).init(V, _dev(po, torch.int64), _dev(pi, torch.int32), _dev(oo, torch.int64),
                                          _dev(oi, torch.int32))
    st.append(_dev(np.array([900, 901, 902], np.int32), torch.int32), V)
    torch.cuda.synchronize()
    got = _state_rows(st)
    assert got[0][0] == oracle_mod.penalty_state(prompts[0], [7, 7, 900], V) and got[0][1] == 0
    assert len(got[1][0]) == cap and got[1][1] == lib.FLAG_LIMIT          # 20 prompt ids, 8 kept
    assert got[1][0] == {i: (0, True) for i in range(cap)}                # the smallest ids
    assert len(got[2][0]) == cap and got[2][1] == lib.FLAG_LIMIT          # full: 902 finds no room
    assert got[2][0] == oracle_mod.penalty_state(prompts[2], outs[2], V)


@pytest.mark.parametrize("cfg,B,V", [(3, 16, 152064), (5, 8, 60013)], ids=["c3_B16_V152064", "c5_B8_V60013"])
def test_sample_with_state_equals_histories(cfg, B, V, lib, oracle_mod):
    import torch

    from workloads.device import to_device

    w = workloads.generate(cfg, B=B, V=V, H=1024, variant=8)
    workloads.add_prompt(w, 700, seed=10 + cfg)
    logits, u, p = to_device(w)
    st = lib.PenaltyState(B, cap=4096).init(V, p.prompt_offsets, p.prompt_ids, p.hist_offsets, p.hist_ids)
    ps = lib.SamplingParams(temperature=p.temperature, top_k=p.top_k, top_p=p.top_p, min_p=p.min_p,
                            repetition_penalty=p.repetition_penalty, frequency_penalty=p.frequency_penalty,
                            presence_penalty=p.presence_penalty, state=st)
    outs = [np_(o.reshape(-1)) for o in [lib.sample(logits, u, p, n_top=w.n_top, V=V)[0]]]
    for step in range(3):
        _say("state step", cfg, step)
        a = lib.sample(logits, u, p, n_top=w.n_top, V=V)
        b = lib.sample(logits, u, ps, n_top=w.n_top, V=V)
        torch.cuda.synchronize()
        for x, y in zip(a, b):
            assert np.array_equal(np_(x), np_(y))
        rep = compare_sample(oracle_mod.sample(w), b, n_top=w.n_top)
        assert rep["band"] <= 2
        # the sampled tokens join the output history and the state
        ids = np_(b[0]).astype(np.int32)
        st.append(b[0], V)
        rows = [list(_rows(w.hist_offsets, w.hist_ids, r)) + ([int(ids[r])] if ids[r] >= 0 else [])
                for r in range(B)]
        w.hist_offsets, w.hist_ids = _csr(rows)
        p.hist_offsets, p.hist_ids = _dev(w.hist_offsets, torch.int64), _dev(w.hist_ids, torch.int32)
        outs.append(ids)
    assert len(outs) == 4


@pytest.mark.parametrize("cfg,B,V,H,P", [(3, 8, 20011, 1000, 600), (5, 4, 170011, 1024, 6000),
                                         (4, 6, 60013, 0, 300)],
                         ids=["c3_B8_V20011", "c5_B4_V170011_long_prompt", "c4_B6_V60013_prompt_only"])
def test_apply_penalties_prompt_and_state_bit_exact(cfg, B, V, H, P, lib, oracle_mod):
    """albireo_apply_penalties with a prompt history, then with the penalty state built from the same
    two histories: both bit-identical to the oracle's penalised logits (the long prompt gives each row
    thousands of distinct ids, within the state's 8192 entries)."""
    import torch

    from workloads.device import to_device

    w = _with_penalties(workloads.generate(cfg, B=B, V=V, H=H if H else None, variant=8), seed=cfg)
    if not H:
        w.hist_offsets, w.hist_ids = _csr([[] for _ in range(B)])
    workloads.add_prompt(w, P, seed=20 + cfg, s=0.6)
    ref = oracle_mod.sample(w, penalised=True)["penalised"]
    logits, u, p = to_device(w)
    _say("apply_penalties prompt", cfg, B, V, H, P)
    got = lib.apply_penalties(logits, p, V=V)
    torch.cuda.synchronize()
    assert np.array_equal(np_(got).view(np.uint32), ref.view(np.uint32))
    st = lib.PenaltyState(B, cap=8192).init(V, p.prompt_offsets, p.prompt_ids, p.hist_offsets, p.hist_ids)
    assert not (np_(st.flags) & lib.FLAG_LIMIT).any()
    ps = lib.SamplingParams(repetition_penalty=p.repetition_penalty, frequency_penalty=p.frequency_penalty,
                            presence_penalty=p.presence_penalty, state=st)
    _say("apply_penalties state", cfg, B, V, H, P)
    got_s = lib.apply_penalties(logits, ps, V=V)
    torch.cuda.synchronize()
    assert np.array_equal(np_(got_s).view(np.uint32), ref.view(np.uint32))
