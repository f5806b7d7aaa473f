"""CPU oracle for the per-sequence sampling step -- TEST INFRASTRUCTURE ONLY.

Only ``tests/``, ``__graft_entry__.smoke()`` and the CPU-baseline leg of ``bench.py`` may import this
package.  The product path (``paper_2606_01927_amd``) never imports it and shares no code with it.

``albireo_oracle.c`` holds the definition (plain C, double-precision mass arithmetic, a full sort per
row); this module compiles it with gcc and calls it through ctypes.  ``brute.py`` holds pure-Python
brute-force checks for tiny vocabularies.

Oracle flag bits: 1 GREEDY, 2 EMPTY, 4 BAD_INPUT, 8 BAD_PARAM.  Two margins come back per row:
``cdf_margin`` (distance of the uniform to the ends of the drawn token's CDF interval) and
``topp_margin`` (distance of top_p to the cumulative masses on both sides of the nucleus cut); the
parity tests exclude rows whose margin is below 1e-5 from the exact token-id comparison.
"""
from __future__ import annotations

import ctypes
import os
import subprocess

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "albireo_oracle.c")
_LIB = os.path.join(_HERE, "liboracle.so")

GREEDY, EMPTY, BAD_INPUT, BAD_PARAM = 1, 2, 4, 8


def build(force: bool = True, src: str = _SRC, out: str = _LIB) -> str:
    """Compile the oracle with gcc into ``oracle/liboracle.so`` (or ``out``)."""
    if force or not os.path.exists(out) or os.path.getmtime(out) < os.path.getmtime(src):
        tmp = out + ".tmp%d" % os.getpid()
        cmd = ["gcc", "-O2", "-std=c99", "-ffp-contract=off", "-fno-fast-math", "-fopenmp", "-fPIC",
               "-shared", src, "-o", tmp, "-lm"]
        subprocess.check_call(cmd)
        os.replace(tmp, out)
    return out


class _In(ctypes.Structure):
    _fields_ = [
        ("logits", ctypes.c_void_p), ("is_bf16", ctypes.c_int32),
        ("B", ctypes.c_int64), ("V", ctypes.c_int64), ("ld", ctypes.c_int64),
        ("temperature", ctypes.c_void_p), ("top_k", ctypes.c_void_p), ("top_p", ctypes.c_void_p),
        ("min_p", ctypes.c_void_p), ("rep", ctypes.c_void_p), ("freq", ctypes.c_void_p),
        ("pres", ctypes.c_void_p), ("hist_offsets", ctypes.c_void_p), ("hist_ids", ctypes.c_void_p),
        ("hist_len", ctypes.c_int64), ("uniforms", ctypes.c_void_p), ("n_top", ctypes.c_int32),
        ("prompt_offsets", ctypes.c_void_p), ("prompt_ids", ctypes.c_void_p), ("prompt_len", ctypes.c_int64),
    ]


class _Out(ctypes.Structure):
    _fields_ = [(n, ctypes.c_void_p) for n in (
        "ids", "logprobs", "top_ids", "top_logprobs", "flags", "cdf_margin", "topp_margin",
        "threshold", "kept", "log_norm", "lse", "probs", "penalised")]


_libs = {}


def _load(path: str = _LIB):
    if path not in _libs:
        if path == _LIB and not os.path.exists(_LIB):
            build(force=True)
        lib = ctypes.CDLL(path)
        lib.oracle_sample.argtypes = [ctypes.POINTER(_In), ctypes.POINTER(_Out), ctypes.c_int]
        lib.oracle_sample.restype = ctypes.c_int
        lib.oracle_max_threads.restype = ctypes.c_int
        lib.oracle_philox4x32_10.argtypes = [ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p]
        lib.oracle_philox4x32_10.restype = None
        lib.oracle_philox_uniforms.argtypes = [ctypes.c_uint64, ctypes.c_uint64, ctypes.c_void_p,
                                               ctypes.c_int64, ctypes.c_void_p]
        lib.oracle_philox_uniforms.restype = None
        lib.oracle_backfill.argtypes = [ctypes.c_void_p, ctypes.c_void_p, ctypes.c_int64, ctypes.c_void_p,
                                        ctypes.c_int64]
        lib.oracle_backfill.restype = None
        lib.oracle_receive_rows.argtypes = [ctypes.c_void_p, ctypes.c_int32, ctypes.c_int64, ctypes.c_int64,
                                            ctypes.c_int64, ctypes.c_int64, ctypes.c_int64, ctypes.c_void_p]
        lib.oracle_receive_rows.restype = None
        _libs[path] = lib
    return _libs[path]


def max_threads() -> int:
    return _load().oracle_max_threads()


def _ptr(a):
    return None if a is None else a.ctypes.data


def sample(w, nthreads: int = 0, probs: bool = False, penalised: bool = False, draw: bool = True,
           rows=None, lib_path: str = _LIB) -> dict:
    """Run the oracle on workload ``w`` (a ``workloads.Workload``; only ``rows`` if given).

    Returns numpy arrays: ids, logprobs, top_ids, top_logprobs, flags, cdf_margin, topp_margin,
    threshold, kept, log_norm, lse, and optionally probs [B, V] (float64) and penalised [B, V] (float32).
    """
    if rows is not None:
        rows = np.asarray(rows, dtype=np.int64)
        res = [sample(w.row_slice(int(r), int(r) + 1), nthreads, probs, penalised, draw, lib_path=lib_path)
               for r in rows]
        return {k: np.concatenate([r[k] for r in res]) for k in res[0]}
    lib = _load(lib_path)
    B, V = w.B, w.V
    keep = []

    def c(a, dt):
        if a is None:
            return None
        a = np.ascontiguousarray(a, dtype=dt)
        keep.append(a)
        return a

    logits = c(w.logits, np.uint16 if w.dtype == "bf16" else np.float32)
    n_top = int(w.n_top)
    ho = c(w.hist_offsets, np.int64)
    hi = None
    hist_len = 0
    if ho is not None:
        hist_len = 0 if w.hist_ids is None else int(np.asarray(w.hist_ids).size)
        hi = c(w.hist_ids if hist_len else np.zeros(1, np.int32), np.int32)
    po = c(getattr(w, "prompt_offsets", None), np.int64)
    pi = None
    prompt_len = 0
    if po is not None:
        prompt_len = 0 if w.prompt_ids is None else int(np.asarray(w.prompt_ids).size)
        pi = c(w.prompt_ids if prompt_len else np.zeros(1, np.int32), np.int32)
    inp = _In(
        logits=_ptr(logits), is_bf16=1 if w.dtype == "bf16" else 0, B=B, V=V, ld=w.ld,
        temperature=_ptr(c(w.temperature, np.float32)), top_k=_ptr(c(w.top_k, np.int32)),
        top_p=_ptr(c(w.top_p, np.float32)), min_p=_ptr(c(w.min_p, np.float32)),
        rep=_ptr(c(w.repetition_penalty, np.float32)), freq=_ptr(c(w.frequency_penalty, np.float32)),
        pres=_ptr(c(w.presence_penalty, np.float32)), hist_offsets=_ptr(ho),
        hist_ids=_ptr(hi), hist_len=hist_len,
        uniforms=_ptr(c(w.uniforms, np.float32)) if draw else None, n_top=n_top,
        prompt_offsets=_ptr(po), prompt_ids=_ptr(pi), prompt_len=prompt_len)
    o = dict(
        ids=np.zeros(B, np.int32), logprobs=np.zeros(B, np.float64),
        top_ids=np.zeros((B, n_top), np.int32), top_logprobs=np.zeros((B, n_top), np.float64),
        flags=np.zeros(B, np.uint32), cdf_margin=np.zeros(B, np.float64),
        topp_margin=np.zeros(B, np.float64), threshold=np.zeros(B, np.float64),
        kept=np.zeros(B, np.int64), log_norm=np.zeros(B, np.float64), lse=np.zeros(B, np.float64))
    if probs:
        o["probs"] = np.zeros((B, V), np.float64)
    if penalised:
        o["penalised"] = np.zeros((B, V), np.float32)
    out = _Out(**{k: (v.ctypes.data if (v.size or k in ("top_ids", "top_logprobs")) else None)
                  for k, v in o.items()})
    if n_top == 0:
        out.top_ids = None
        out.top_logprobs = None
    rc = lib.oracle_sample(ctypes.byref(inp), ctypes.byref(out), int(nthreads))
    if rc != 0:
        raise RuntimeError("oracle_sample failed with code %d" % rc)
    return o


def philox4x32_10(counter, key, lib_path: str = _LIB) -> np.ndarray:
    """Philox-4x32-10 of a 4-word counter under a 2-word key (O-11): four uint32 words."""
    c = np.ascontiguousarray(counter, dtype=np.uint32)
    k = np.ascontiguousarray(key, dtype=np.uint32)
    assert c.shape == (4,) and k.shape == (2,)
    out = np.zeros(4, np.uint32)
    _load(lib_path).oracle_philox4x32_10(c.ctypes.data, k.ctypes.data, out.ctypes.data)
    return out


def philox_uniforms(seed: int, step: int, seq_ids=None, B: int = None, lib_path: str = _LIB) -> np.ndarray:
    """The per-row uniforms of O-11: row i uses sequence id seq_ids[i] (the row index when None)."""
    if seq_ids is not None:
        seq = np.ascontiguousarray(seq_ids, dtype=np.int64)
        B = seq.size
    out = np.zeros(B, np.float32)
    _load(lib_path).oracle_philox_uniforms(ctypes.c_uint64(seed & (2**64 - 1)), ctypes.c_uint64(step & (2**64 - 1)),
                                           None if seq_ids is None else seq.ctypes.data, B, out.ctypes.data)
    return out


def backfill(ids, dest, next_tokens, lib_path: str = _LIB) -> np.ndarray:
    """O-12: a copy of next_tokens with row i's id written to slot dest[i] where that slot exists."""
    ids = np.ascontiguousarray(ids, dtype=np.int32)
    dest = np.ascontiguousarray(dest, dtype=np.int32)
    out = np.array(next_tokens, dtype=np.int32, copy=True)
    _load(lib_path).oracle_backfill(ids.ctypes.data, dest.ctypes.data, ids.size, out.ctypes.data, out.size)
    return out


def penalty_state(prompt_ids, output_ids, V: int) -> dict:
    """O-15: a sequence's penalty state after its prompt and outputs: {id: (output count, in prompt)}
    over the distinct ids of both that lie in [0, V)."""
    st = {}
    for t in np.asarray(prompt_ids, dtype=np.int64).ravel():
        if 0 <= t < V:
            c, _ = st.get(int(t), (0, False))
            st[int(t)] = (c, True)
    for t in np.asarray(output_ids, dtype=np.int64).ravel():
        if 0 <= t < V:
            c, f = st.get(int(t), (0, False))
            st[int(t)] = (c + 1, f)
    return st


def receive_rows(buf, B: int, V: int, ld: int, L: int, S: int, lib_path: str = _LIB) -> np.ndarray:
    """O-13: the [B, V] rows held in an all-to-all receive buffer (flat array of bf16 bit patterns or
    fp32) with blocks of L columns, S elements apart, row stride ld inside a block."""
    buf = np.ascontiguousarray(buf).reshape(-1)
    assert buf.dtype in (np.uint16, np.float32)
    out = np.zeros((B, V), buf.dtype)
    if B and V:
        assert (V - 1) // L * S + (B - 1) * ld + min(L, V) - 1 < buf.size
    _load(lib_path).oracle_receive_rows(buf.ctypes.data, buf.itemsize, B, V, ld, L, S, out.ctypes.data)
    return out


class Variant:
    """The oracle's interface bound to another build of the same source (used by the mutation test,
    which compiles deliberately broken copies and checks that the pins reject them)."""

    GREEDY, EMPTY, BAD_INPUT, BAD_PARAM = GREEDY, EMPTY, BAD_INPUT, BAD_PARAM

    def __init__(self, lib_path: str):
        self.lib_path = lib_path

    def sample(self, w, **kw):
        return sample(w, lib_path=self.lib_path, **kw)

    def philox4x32_10(self, counter, key):
        return philox4x32_10(counter, key, lib_path=self.lib_path)

    def philox_uniforms(self, seed, step, seq_ids=None, B=None):
        return philox_uniforms(seed, step, seq_ids, B, lib_path=self.lib_path)

    def backfill(self, ids, dest, next_tokens):
        return backfill(ids, dest, next_tokens, lib_path=self.lib_path)

    def penalty_state(self, prompt_ids, output_ids, V):
        return penalty_state(prompt_ids, output_ids, V)

    def receive_rows(self, buf, B, V, ld, L, S):
        return receive_rows(buf, B, V, ld, L, S, lib_path=self.lib_path)
