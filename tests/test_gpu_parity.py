"""GPU parity: the HIP sampling path through the C ABI against the CPU oracle on seeded inputs."""
from __future__ import annotations

import sys

import numpy as np
import pytest

import workloads
from tests.parity import BAND, TOL, compare_sample, np_

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


def _run(alb, w, n_top=None, offset_bytes=0):
    import torch
    from workloads.device import to_device

    logits, u, p = to_device(w, row_offset_bytes=offset_bytes)
    out = alb.sample(logits, u, p, n_top=w.n_top if n_top is None else n_top, V=w.V)
    torch.cuda.synchronize()
    return out


# reduced sizes that still span several register slots, ragged tails and (for the wide fp32 case)
# two chunks per row
SMALL = [
    (1, 4, 32000), (1, 16, 4099), (2, 64, 30011), (2, 32, 128256), (3, 32, 20011),
    (3, 16, 152064), (4, 16, 60013), (4, 8, 100003), (5, 24, 40009), (5, 8, 170011),
]


@pytest.mark.parametrize("cfg,B,V", SMALL, ids=["c%d_B%d_V%d" % c for c in SMALL])
def test_sample_reduced(cfg, B, V, lib, oracle_mod):
    w = workloads.generate(cfg, B=B, V=V, H=min(2048, V // 4) if cfg in (3, 5) else None, variant=1)
    _say("sample", cfg, B, V)
    out = _run(lib, w)
    ref = oracle_mod.sample(w)
    rep = compare_sample(ref, out, n_top=w.n_top)
    _say("  ", rep)
    assert rep["band"] <= max(2, B // 8)


FULL = [1, 2, 3, 4, 5]


@pytest.mark.parametrize("cfg", FULL)
def test_sample_full_size(cfg, lib, oracle_mod):
    """The configuration at its full size in the launch the benchmark times, every row against the
    oracle; rows whose draw or nucleus boundary lies within the flag band of a decision are counted,
    and must stay few (at most one in 32)."""
    w = workloads.generate(cfg)
    _say("full config", cfg, w.B, w.V)
    out = _run(lib, w)
    ref = oracle_mod.sample(w)
    rep = compare_sample(ref, out, n_top=w.n_top)
    _say("   config %d: %d rows, %d compared, %d in the flag band, max |dlogprob| %.3g" % (
        cfg, rep["rows"], rep["compared"], rep["band"], rep["max_dlogprob"]))
    assert rep["rows"] == w.B
    assert rep["band"] * 32 <= w.B, "%d of %d rows in the flag band" % (rep["band"], w.B)


def test_determinism_and_shard_invariance(lib):
    """sec. 6.2: splitting the rows across workers, each consuming its slice of the pre-generated
    uniforms, gives the single-worker result -- here bit-exact, logprobs included."""
    import torch

    w = workloads.generate(5, B=32, V=50021, H=512, ld=50024)  # rows 16-byte aligned in every slice
    full = [np_(x) for x in _run(lib, w)]
    again = [np_(x) for x in _run(lib, w)]
    for a, b in zip(full, again):
        assert np.array_equal(a, b)
    for t in (2, 4, 8):
        step = 32 // t
        parts = [[np_(x) for x in _run(lib, w.row_slice(a, a + step))] for a in range(0, 32, step)]
        for k in range(5):
            assert np.array_equal(np.concatenate([p[k] for p in parts]), full[k]), (t, k)
    torch.cuda.synchronize()


def test_padding_rows_do_not_change_real_rows(lib):
    w = workloads.generate(2, B=10, V=20011)
    base = [np_(x) for x in _run(lib, w)]
    pad = workloads.generate(2, B=6, V=20011, variant=7)
    ww = w.row_slice(0, 10)
    ww.B = 16
    ww.logits = np.concatenate([w.logits, pad.logits])
    ww.uniforms = np.concatenate([w.uniforms, pad.uniforms])
    for f in ("temperature", "top_k", "top_p"):
        setattr(ww, f, np.concatenate([getattr(w, f), getattr(pad, f)]))
    got = [np_(x) for x in _run(lib, ww)]
    for k in range(5):
        assert np.array_equal(got[k][:10], base[k])


@pytest.mark.parametrize("offset", [0, 2, 6, 12])
@pytest.mark.parametrize("cfg,ld_pad", [(3, 13), (4, 7)])
def test_strided_and_misaligned_rows(cfg, ld_pad, offset, lib, oracle_mod):
    es = 2 if cfg in (2, 3, 5) else 4
    V = 9001
    if offset % es:
        # rows that do not start on an element boundary: refused before anything is enqueued
        import ctypes

        import torch

        buf = torch.zeros(8 * (V + ld_pad) * es + 64, dtype=torch.uint8, device="cuda")
        u = torch.zeros(8, dtype=torch.float32, device="cuda")
        outs = [torch.zeros(8, dtype=torch.int32, device="cuda") for _ in range(2)]
        st = lib.raw_call("albireo_sample")(buf.data_ptr() + offset, lib.F32, 8, V, V + ld_pad, None, u.data_ptr(),
                                              outs[0].data_ptr(), outs[1].data_ptr(), 0, None, None, None, None, 0,
                                              None)
        assert st == lib.E_INVALID
        return
    w = workloads.generate(cfg, B=8, V=V, ld=V + ld_pad, H=300 if cfg in (3, 5) else None)
    _say("strided", cfg, ld_pad, offset)
    out = _run(lib, w, offset_bytes=offset)
    compare_sample(oracle_mod.sample(w), out, n_top=w.n_top)


def _rowset(rows, dtype="f32", **params):
    """Workload built from explicit rows (list of lists), same V for all."""
    B = len(rows)
    V = len(rows[0])
    x = np.array([[(-np.inf if v == "-inf" else (np.inf if v == "inf" else (np.nan if v == "nan" else v)))
                   for v in r] for r in rows], dtype=np.float32)
    w = workloads.Workload(name="edge", B=B, V=V, dtype=dtype, ld=V,
                           logits=workloads.to_bf16_bits(x) if dtype == "bf16" else x,
                           uniforms=np.asarray(params.pop("u", np.linspace(0.05, 0.95, B)), np.float32))
    for k, v in params.items():
        setattr(w, k, v)
    return w


def test_edge_cases(lib, oracle_mod):
    rng = np.random.default_rng(5)
    V = 1000
    base = rng.normal(0, 1, size=V).astype(np.float32)
    rows, T, K, Pp, MP = [], [], [], [], []

    def add(x, t=1.0, k=0, p=1.0, mp=0.0):
        rows.append(list(x)); T.append(t); K.append(k); Pp.append(p); MP.append(mp)

    allneg = np.full(V, -np.inf, np.float32)
    add(allneg)                                   # empty row
    ties = np.zeros(V, np.float32)
    add(ties, t=0.0)                              # greedy, every entry tied: lowest id
    add(ties, k=5)                                # top-k ties keep all
    add(ties, p=0.3)                              # nucleus of all-equal mass
    x = base.copy(); x[[10, 700]] = 9.0
    add(x, t=0.0)                                 # greedy tie between two ids
    add(x, k=1)                                   # top_k = 1 with a tied maximum
    add(x, p=1e-7)                                # p -> 0 keeps the top group
    add(base, mp=2.0)                             # min_p > 1 behaves as 1
    add(base, t=1e6)                              # huge temperature
    add(base, t=1e-4, k=3, p=0.5, mp=0.05)        # tiny temperature, all filters
    y = base.copy(); y[::3] = -np.inf
    add(y, p=0.9, k=50)                           # masked entries
    add(y, k=V - 1)                               # top-k nearly off
    add(base, k=V + 5)                            # top-k beyond V is off
    add(base, p=-1.0)                             # p <= 0
    z = base.copy(); z[17] = np.nan
    add(z)                                        # NaN -> BAD_INPUT
    w = _rowset(rows, temperature=np.array(T, np.float32), top_k=np.array(K, np.int32),
                top_p=np.array(Pp, np.float32), min_p=np.array(MP, np.float32))
    w.n_top = 7
    out = _run(lib, w)
    ref = oracle_mod.sample(w)
    compare_sample(ref, out, n_top=7)


@pytest.mark.parametrize("n_top", [0, 4])
def test_topk_ties_on_streamed_rows(n_top, lib, oracle_mod):
    """Rows of the streaming route (many chunks per row) whose top-k boundary value is tied, inside one
    chunk's list beyond its first k entries and across chunks: every tied value is kept (ties kept at
    the k-th value), with and without top-n."""
    rng = np.random.default_rng(21)
    V = 200003  # fp32: 11 chunks per row
    base = rng.normal(0, 1, size=V).astype(np.float32)
    rows, K, Pp = [], [], []

    def add(pos, vals, k, p=1.0):
        x = base.copy()
        x[pos] = vals
        rows.append(x); K.append(k); Pp.append(p)

    add([10, 20], 9.0, 1)                          # tied maximum, one chunk
    add([10, 150000], 9.0, 1)                      # tied maximum, two chunks
    add([10, 20, 30], 9.0, 2)                      # three-way tie at the top, k = 2
    add([5, 6, 7, 8], [9.0, 8.5, 8.0, 8.0], 3)     # tie at the k-th value, one chunk
    add([5, 6, 90000, 190000], [9.0, 8.5, 8.0, 8.0], 3)  # tie at the k-th value, across chunks
    add([10, 20, 30, 40], 9.0, 1, p=0.5)           # tied maximum with a nucleus
    add(list(range(100, 140)), 9.0, 7)             # 40 tied values above k = 7
    w = _rowset(rows, temperature=np.full(len(rows), 0.9, np.float32), top_k=np.array(K, np.int32),
                top_p=np.array(Pp, np.float32))
    w.n_top = n_top
    import torch

    assert lib.sample_route(w.B, V, torch.float32) == lib.ROUTE_STREAM
    out = _run(lib, w)
    ref = oracle_mod.sample(w)
    compare_sample(ref, out, n_top=n_top)


def test_overflowing_kept_set_lists_keep_top_n(lib, oracle_mod):
    """Streamed rows whose min-p or top-k bound lets far more candidates into a chunk than its list
    holds: the kept set goes to the general path, while the chunk lists fall back to the top-n bound
    and still give the top-n logprobs (ties at the n-th value included)."""
    import torch

    rng = np.random.default_rng(31)
    V = 200003  # fp32: 11 chunks per row
    base = rng.normal(0, 0.5, size=V).astype(np.float32)  # flat: thousands within ln(1/min_p) of the max
    rows, K, MP, Pp = [], [], [], []

    def add(x, k=0, mp=0.0, p=1.0):
        rows.append(x); K.append(k); MP.append(mp); Pp.append(p)

    add(base.copy(), mp=0.001)                     # min-p keeps most of every chunk
    add(base.copy(), mp=0.01, p=0.9)               # min-p and a nucleus
    add(base.copy(), k=5000)                       # top-k beyond the list capacity
    t = base.copy(); t[[3, 40000, 90000, 150000, 199999]] = 4.0; t[[7, 8]] = 3.5
    add(t, mp=0.001)                               # distinct top values, then a tie inside one chunk
    w = _rowset(rows, temperature=np.full(len(rows), 1.0, np.float32), top_k=np.array(K, np.int32),
                min_p=np.array(MP, np.float32), top_p=np.array(Pp, np.float32))
    w.n_top = 6
    assert lib.sample_route(w.B, V, torch.float32) == lib.ROUTE_STREAM
    out = _run(lib, w)
    ref = oracle_mod.sample(w)
    compare_sample(ref, out, n_top=6)


@pytest.mark.parametrize("dtype,extras", [("f32", False), ("bf16", False), ("bf16", True)],
                         ids=["f32", "bf16", "bf16_topn_penalties"])
def test_general_path_wide_rows(dtype, extras, lib, oracle_mod):
    """Wide rows whose kept sets are too large for candidate lists: the selections over the whole row
    (top-k above the list capacity, top-p without top-k), including rows whose boundary values are so
    often tied that they do not fit in the on-chip staging and take the whole-row selection."""
    rng = np.random.default_rng(11)
    V = 100003
    rows, K, Pp, MP = [], [], [], []

    def add(x, k=0, p=1.0, mp=0.0):
        rows.append(np.asarray(x, np.float32)); K.append(k); Pp.append(p); MP.append(mp)

    base = rng.normal(0, 2, size=V).astype(np.float32)
    add(base, k=2000, p=0.9)                      # count selection, then the nucleus
    add(base, p=0.6)                              # nucleus alone
    add(base, k=600)                              # top-k just above the list capacity
    tied = base.copy(); tied[rng.random(V) < 0.5] = 1.5
    add(tied, p=0.95)                             # ~50000 equal values around the boundary
    add(tied, k=30000, p=0.99)                    # the K-th value among them
    q = np.round(base * 16) / 16
    add(q, p=0.8)                                 # coarse values: many ties in every bucket
    add(rng.standard_t(3, size=V) * 2, p=0.98, mp=0.02)  # heavy tail with min-p
    half = base.copy(); half[rng.random(V) < 0.5] = -np.inf
    add(half, p=0.7, k=5000)                      # masked entries
    x = np.stack(rows)
    w = workloads.Workload(name="wide", B=len(rows), V=V, dtype=dtype, ld=V,
                           logits=workloads.to_bf16_bits(x) if dtype == "bf16" else x,
                           uniforms=np.linspace(0.07, 0.93, len(rows)).astype(np.float32),
                           temperature=np.full(len(rows), 0.9, np.float32), top_k=np.array(K, np.int32),
                           top_p=np.array(Pp, np.float32), min_p=np.array(MP, np.float32))
    if extras:  # top-5 logprobs and penalties from 1500-id histories over the same rows
        hr = np.random.default_rng(12)
        B = len(rows)
        lens = hr.integers(200, 1500, size=B)
        w.hist_offsets = np.concatenate([[0], np.cumsum(lens)]).astype(np.int64)
        w.hist_ids = hr.integers(0, V, size=int(lens.sum())).astype(np.int32)
        w.repetition_penalty = hr.uniform(1.05, 1.4, size=B).astype(np.float32)
        w.frequency_penalty = hr.uniform(0.0, 0.4, size=B).astype(np.float32)
        w.presence_penalty = hr.uniform(-0.1, 0.3, size=B).astype(np.float32)
        w.n_top = 5
    _say("wide rows", dtype, extras)
    out = _run(lib, w)
    rep = compare_sample(oracle_mod.sample(w), out, n_top=w.n_top)
    _say("  ", rep)
    assert rep["band"] <= 1


def test_penalty_edge_cases(lib, oracle_mod):
    rng = np.random.default_rng(6)
    V = 3001
    B = 6
    x = rng.normal(0, 2, size=(B, V)).astype(np.float32)
    hist = [
        [0, 0, 0, 5, 5, V - 1],            # repeats and the last id
        [V + 3, -1, 7],                     # out of range ids are skipped and flagged
        list(range(0, V, 2)),               # half the vocabulary penalised
        [],                                 # empty history
        [42] * 500,                         # one id many times
        list(rng.integers(0, V, size=2500)),
    ]
    offs = np.cumsum([0] + [len(h) for h in hist]).astype(np.int64)
    w = workloads.Workload(name="pen", B=B, V=V, dtype="f32", ld=V, logits=x,
                           uniforms=rng.random(B).astype(np.float32),
                           repetition_penalty=np.array([1.3, 1.1, 0.0, 1.2, 2.0, 1.05], np.float32),
                           frequency_penalty=np.array([0.5, 0.2, 0.1, 0.3, 0.01, np.inf], np.float32),
                           presence_penalty=np.array([0.25, 0.1, -0.5, 0.1, 1.0, 0.2], np.float32),
                           hist_offsets=offs, hist_ids=np.concatenate([np.array(h, np.int32) for h in hist]),
                           temperature=np.array([0.9, 1.0, 0.0, 1.1, 0.7, 1.0], np.float32),
                           top_k=np.array([0, 10, 0, 0, 50, 0], np.int32),
                           top_p=np.array([0.9, 1.0, 1.0, 0.8, 0.95, 0.99], np.float32))
    w.n_top = 5
    out = _run(lib, w)
    compare_sample(oracle_mod.sample(w), out, n_top=5)


def test_topk_topp_dense(lib, oracle_mod):
    import torch
    from workloads.device import to_device

    for cfg, B, V in [(1, 4, 32000), (4, 8, 100003), (2, 16, 20011)]:
        w = workloads.generate(cfg, B=B, V=V)
        if w.dtype == "bf16":
            w.logits = (w.logits.astype(np.uint32) << 16).view(np.float32)
            w.dtype = "f32"
        _say("topk_topp", cfg, B, V)
        logits, u, p = to_device(w)
        pr, thr, kept, lnorm, flags = lib.topk_topp(logits, p, V=V)
        torch.cuda.synchronize()
        ref = oracle_mod.sample(w, probs=True, draw=False)
        ok = ref["topp_margin"] >= BAND
        assert np.array_equal(np_(kept)[ok], ref["kept"][ok])
        assert np.array_equal(np_(thr)[ok].astype(np.float64), ref["threshold"][ok])
        assert (np.abs(np_(lnorm)[ok] - ref["log_norm"][ok]) <= TOL).all()
        d = np.abs(np_(pr)[ok].astype(np.float64) - ref["probs"][ok])
        assert d.max() <= TOL, d.max()


def test_apply_penalties_bit_exact(lib, oracle_mod):
    import torch
    from workloads.device import to_device

    for cfg, B, V in [(3, 8, 20011), (5, 4, 170011)]:
        w = workloads.generate(cfg, B=B, V=V, H=1000)
        logits, u, p = to_device(w)
        out = lib.apply_penalties(logits, p, V=V)
        torch.cuda.synchronize()
        ref = oracle_mod.sample(w, penalised=True)["penalised"]
        assert np.array_equal(np_(out).view(np.uint32), ref.view(np.uint32))


def test_workspace_left_zero_after_deferred_rows(lib, oracle_mod):
    """The workspace contract on the streaming route with rows that the chunk-parallel general path
    resolves: after calls whose rows are deferred (nucleus rows whose crossing bucket fits the
    staging, rows where it does not, plain rows, rows with penalties and top-n), every byte of the
    caller's workspace is zero again, and a second call through the same workspace gives the same
    outputs."""
    import torch

    from workloads.device import to_device

    rng = np.random.default_rng(41)
    V = 200003  # bf16: 6 chunks per row
    base = rng.normal(0, 2, size=V).astype(np.float32)
    tied = base.copy(); tied[rng.random(V) < 0.4] = 1.25
    rows = [base, base * 0.5, tied, np.round(base * 8) / 8, base]
    P_ = np.array([0.9, 0.6, 0.95, 0.8, 1.0], np.float32)  # the last row: no filter at all
    w = _rowset(rows, dtype="bf16", temperature=np.array([1.0, 1.3, 0.9, 1.0, 0.8], np.float32),
                top_k=np.zeros(len(rows), np.int32), top_p=P_)
    hr = np.random.default_rng(42)
    lens = hr.integers(100, 900, size=w.B)
    w.hist_offsets = np.concatenate([[0], np.cumsum(lens)]).astype(np.int64)
    w.hist_ids = hr.integers(0, V, size=int(lens.sum())).astype(np.int32)
    w.repetition_penalty = np.full(w.B, 1.2, np.float32)
    w.n_top = 3
    assert lib.sample_route(w.B, V, torch.bfloat16) == lib.ROUTE_STREAM
    logits, u, p = to_device(w)
    ws = lib.Workspace("cuda")
    out = lib.sample(logits, u, p, n_top=3, V=V, workspace=ws)
    torch.cuda.synchronize()
    first = [np_(x) for x in out]
    assert int(torch.count_nonzero(ws.buf)) == 0
    second = [np_(x) for x in lib.sample(logits, u, p, n_top=3, V=V, workspace=ws)]
    torch.cuda.synchronize()
    assert int(torch.count_nonzero(ws.buf)) == 0
    for x, y in zip(first, second):
        assert np.array_equal(x, y)
    compare_sample(oracle_mod.sample(w), out, n_top=3)


def test_deferred_rows_edge_cases(lib, oracle_mod):
    """Edge cases of the chunk-parallel general path on streamed rows (no top-k): p <= 0 and p -> 0
    (the top group only), a nucleus cut inside a group of equal values spread over chunks, min-p
    together with a nucleus, masked entries, a row whose finite values are all in one chunk, no filter
    at all, and a greedy row beside them."""
    import torch

    rng = np.random.default_rng(51)
    V = 200003  # fp32: 11 chunks per row
    base = rng.normal(0, 1.5, size=V).astype(np.float32)
    rows, T, Pp, MP = [], [], [], []

    def add(x, t=1.0, p=1.0, mp=0.0):
        rows.append(np.asarray(x, np.float32)); T.append(t); Pp.append(p); MP.append(mp)

    x = base.copy(); x[[10, 90000, 180000]] = 7.0
    add(x, p=-1.0)                                  # p <= 0: the tied top group only
    add(x, p=1e-7)                                  # p -> 0: the same
    g = base.copy(); g[rng.choice(V, 3000, replace=False)] = 4.0
    add(g, p=0.5)                                   # the cut falls inside 3000 equal values
    add(base, p=0.9, mp=0.05)                       # min-p and a nucleus
    h = base.copy(); h[rng.random(V) < 0.7] = -np.inf
    add(h, p=0.8)                                   # masked entries
    one = np.full(V, -np.inf, np.float32); one[100:5000] = base[100:5000]
    add(one, p=0.7)                                 # every finite value in the first chunk
    add(base, t=1.3)                                # no filter
    add(base, t=0.0)                                # greedy
    w = _rowset(rows, temperature=np.array(T, np.float32), top_k=np.zeros(len(rows), np.int32),
                top_p=np.array(Pp, np.float32), min_p=np.array(MP, np.float32))
    assert lib.sample_route(w.B, V, torch.float32) == lib.ROUTE_STREAM
    out = _run(lib, w)
    compare_sample(oracle_mod.sample(w), out)


def test_deferred_rows_beyond_one_grid(lib, oracle_mod):
    """More deferred rows than the general-path launches have workgroups: about 780 nucleus rows
    without top-k (more than the 512 row workgroups) of 6 chunks each (more than the 1024 chunk
    workgroups), interleaved with top-k rows the resolution kernel finishes itself, so that each
    workgroup walks several items of the deferred-row list.  Parity with the oracle, and the workspace
    (list included) is zero again after the call."""
    import torch

    from workloads.device import to_device

    rng = np.random.default_rng(61)
    B, V = 1040, 100003  # fp32: 6 chunks per row
    # N(0, 4) at T in [0.5, 1]: peaked enough that few rows fall in the flag band (about 40 of 1040
    # against the oracle; flatter rows put most of them within 1e-5 of a boundary)
    x = (rng.normal(0, 1, size=(B, V)) * 4).astype(np.float32)
    K = np.where(np.arange(B) % 4 == 3, 50, 0).astype(np.int32)
    w = workloads.Workload(name="deferred_many", B=B, V=V, dtype="f32", ld=V, logits=x,
                           uniforms=rng.random(B).astype(np.float32))
    w.temperature = rng.uniform(0.5, 1.0, size=B).astype(np.float32)
    w.top_k = K
    w.top_p = rng.uniform(0.5, 1.0, size=B).astype(np.float32)
    assert lib.sample_route(B, V, torch.float32) == lib.ROUTE_STREAM
    _say("deferred rows beyond one grid", B, V)
    logits, u, p = to_device(w)
    ws = lib.Workspace("cuda")
    out = lib.sample(logits, u, p, V=V, workspace=ws)
    torch.cuda.synchronize()
    assert int(torch.count_nonzero(ws.buf)) == 0
    rep = compare_sample(oracle_mod.sample(w), out)
    _say("  ", rep)
    assert rep["band"] <= max(2, B // 8)
