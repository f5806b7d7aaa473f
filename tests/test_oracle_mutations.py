"""Mutation check of the oracle's pins: plausible mistakes planted in copies of the oracle source (on
the CPU, in a temporary directory) must each make at least one pin fail.

Every mutant below is a one-token slip of the kind the pins are meant to catch: a dropped term, a
wrong sign, a transposed operand, an off-by-one index, a non-strict comparison, a missing
renormalisation, a wrong tie order.
"""
from __future__ import annotations

import inspect
import os
import tempfile

import pytest

import oracle
from tests import test_oracle_pins as pins
from tests import test_oracle_penalty_state as state_pins
from tests import test_oracle_receive_layout as layout_pins
from tests import test_oracle_rng_backfill as rng_pins

SRC = os.path.join(os.path.dirname(oracle.__file__), "albireo_oracle.c")

MUTANTS = [
    ("presence penalty dropped", "xv = xv - pres;", "xv = xv;"),
    ("frequency penalty sign", "xv = xv - fc;", "xv = xv + fc;"),
    ("repetition operand transposed", "if (xv > 0.0f) xv = xv / rep;", "if (xv > 0.0f) xv = xv * rep;"),
    ("frequency ignores the count", "float fc = freq * (float)c;", "float fc = freq;"),
    ("presence applied to prompt-only ids", "      if (c > 0) {\n        float fc", "      if (1) {\n        float fc"),
    ("prompt ids not penalised", "if (c == 0 && !(have_p && inS[v])) continue;", "if (c == 0) continue;"),
    ("non-strict inverse CDF", "if (C > u) {", "if (C >= u) {"),
    ("top-p not renormalised over S2", "c = c + gm / Z2;", "c = c + gm / sum;"),
    ("top-k off by one", "tau_k = ord[k - 1].z;", "tau_k = ord[k].z;"),
    ("ties ordered by descending id", "return (p->id > q->id) - (p->id < q->id);",
     "return (p->id < q->id) - (p->id > q->id);"),
    ("min-p threshold sign", "tau_m = m + lm;", "tau_m = m - lm;"),
    ("temperature multiplies", "const float r = greedy ? 1.0f : (float)(1.0 / (double)T);",
     "const float r = greedy ? 1.0f : T;"),
    ("logprob drops the max", "out->logprobs[i] = id >= 0 ? (double)z[id] - (double)m - L : -INFINITY;",
     "out->logprobs[i] = id >= 0 ? (double)z[id] - L : -INFINITY;"),
    ("top-p splits tie groups", "while (g_end < n2 && ord[g_end].z == ord[t].z) {",
     "while (g_end < n2 && g_end == t) {"),
    ("draw ignores the kept set", "if (!inS[v]) continue;", "if (0) continue;"),
    ("greedy takes the highest id", "const int32_t id = ord[0].id;",
     "int32_t id = ord[0].id; for (int64_t q = 1; q < V && ord[q].z == ord[0].z; ++q) id = ord[q].id;"),
    ("Philox multipliers swapped", "const uint64_t p0 = (uint64_t)0xD2511F53u * (uint64_t)c[0];",
     "const uint64_t p0 = (uint64_t)0xCD9E8D57u * (uint64_t)c[0];"),
    ("Philox key not advanced", "k[1] += 0xBB67AE85u;", "k[1] += 0u;"),
    ("Philox halves crossed", "const uint32_t n0 = hi1 ^ c[1] ^ k[0];", "const uint32_t n0 = hi0 ^ c[1] ^ k[0];"),
    ("uniform from 23 bits", "out[i] = (float)((double)(w[0] >> 8) * (1.0 / 16777216.0));",
     "out[i] = (float)((double)(w[0] >> 9) * (1.0 / 16777216.0));"),
    ("step low word only", "const uint32_t ctr[4] = {(uint32_t)step, (uint32_t)(step >> 32),",
     "const uint32_t ctr[4] = {(uint32_t)step, 0u,"),
    ("backfill skips slot 0", "if (d >= 0 && d < n_next) next_tokens[d] = ids[i];",
     "if (d > 0 && d < n_next) next_tokens[d] = ids[i];"),
    ("nucleus margin forced to zero", "double a = c - (double)p, b = (double)p - c_prev;\n      out->topp_margin[i] = a < b ? a : b;",
     "double a = c - (double)p, b = (double)p - c_prev;\n      out->topp_margin[i] = 0.0 * (a < b ? a : b);"),
    ("CDF margin forced to zero", "double a = u - Cb, b = C - u;\n        out->cdf_margin[i] = a < b ? a : b;",
     "double a = u - Cb, b = C - u;\n        out->cdf_margin[i] = 0.0 * (a < b ? a : b);"),
    ("log-normaliser drops the max", "out->log_norm[i] = (double)m + log(ZS);", "out->log_norm[i] = log(ZS);"),
    ("top-n logprobs drop the max", "out->top_logprobs[i * nt + t] = (double)ord[t].z - (double)m - L;",
     "out->top_logprobs[i * nt + t] = (double)ord[t].z - L;"),
    ("block stride taken as the row stride", "const int64_t at = (v / L) * S + i * ld + v % L;",
     "const int64_t at = (v / L) * ld + i * ld + v % L;"),
    ("row stride taken as the block length", "const int64_t at = (v / L) * S + i * ld + v % L;",
     "const int64_t at = (v / L) * S + i * L + v % L;"),
    ("column taken modulo the row stride", "const int64_t at = (v / L) * S + i * ld + v % L;",
     "const int64_t at = (v / L) * S + i * ld + v % ld;"),
]


def _pin_calls():
    """(name, callable) for every pin test, with its parametrisations expanded."""
    calls = []
    members = (inspect.getmembers(pins, inspect.isfunction) + inspect.getmembers(rng_pins, inspect.isfunction)
               + inspect.getmembers(layout_pins, inspect.isfunction)
               + inspect.getmembers(state_pins, inspect.isfunction))
    for name, fn in members:
        if not name.startswith("test_"):
            continue
        params = getattr(fn, "pytestmark", [])
        sets = [{}]
        for mark in params:
            if mark.name != "parametrize":
                continue
            argnames, values = mark.args[0], mark.args[1]
            names = [a.strip() for a in argnames.split(",")] if isinstance(argnames, str) else list(argnames)
            new = []
            for s in sets:
                for v in values:
                    vv = v if len(names) > 1 else (v,)
                    d = dict(s)
                    d.update(zip(names, vv))
                    new.append(d)
            sets = new
        for kw in sets:
            calls.append((name, fn, kw))
    return calls


@pytest.mark.parametrize("desc,old,new", MUTANTS, ids=[m[0] for m in MUTANTS])
def test_mutant_is_killed(desc, old, new):
    src = open(SRC).read()
    assert src.count(old) == 1, "mutation anchor not unique: %r" % old
    with tempfile.TemporaryDirectory() as d:
        path = os.path.join(d, "mutant.c")
        with open(path, "w") as f:
            f.write(src.replace(old, new))
        lib = oracle.build(force=True, src=path, out=os.path.join(d, "libmutant.so"))
        variant = oracle.Variant(lib)
        killed_by = None
        for name, fn, kw in _pin_calls():
            try:
                fn(oracle_mod=variant, **kw)
            except Exception:  # noqa: BLE001 - any failure of a pin kills the mutant
                killed_by = name
                break
        assert killed_by is not None, "mutant survived every pin: " + desc
