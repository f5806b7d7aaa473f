"""Python binding of the gfx950 per-sequence sampling library (``include/albireo.h``).

Argument marshalling only: every step of the sampling path runs in the HIP kernels of
``libalbireo.so``.  PyTorch supplies device memory and the current HIP stream.  Importing this package
fails loudly when the built library is missing; there is no CPU fallback.
"""
from __future__ import annotations

import ctypes
import dataclasses
import os
from typing import Optional

import torch

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libalbireo.so")

if not os.path.exists(LIB_PATH):
    raise ImportError(
        "libalbireo.so is not built (expected at %s); run `python paper_2606_01927_amd/build.py` "
        "or __graft_entry__.build()" % LIB_PATH)

_lib = ctypes.CDLL(LIB_PATH)

F32, BF16 = 0, 1
OK, E_INVALID, E_UNSUPPORTED, E_WORKSPACE, E_LAUNCH, E_SCRATCH = 0, 1, 2, 3, 4, 5
ROUTE_NONE, ROUTE_ONE_WORKGROUP, ROUTE_STREAM, ROUTE_COOPERATIVE = 0, 1, 2, 3
FLAG_GREEDY, FLAG_EMPTY, FLAG_BAD_INPUT, FLAG_BAD_PARAM, FLAG_LIMIT = 1, 2, 4, 8, 16
MAX_TOP_N = 32


class _State(ctypes.Structure):
    _fields_ = [("cap", ctypes.c_int32), ("ids", ctypes.c_void_p), ("counts", ctypes.c_void_p),
                ("len", ctypes.c_void_p), ("flags", ctypes.c_void_p)]


class _Params(ctypes.Structure):
    _fields_ = [
        ("temperature", ctypes.c_void_p), ("top_k", ctypes.c_void_p), ("top_p", ctypes.c_void_p),
        ("min_p", ctypes.c_void_p), ("repetition_penalty", ctypes.c_void_p),
        ("frequency_penalty", ctypes.c_void_p), ("presence_penalty", ctypes.c_void_p),
        ("hist_offsets", ctypes.c_void_p), ("hist_ids", ctypes.c_void_p), ("hist_len", ctypes.c_int64),
        ("prompt_offsets", ctypes.c_void_p), ("prompt_ids", ctypes.c_void_p), ("prompt_len", ctypes.c_int64),
        ("state", ctypes.POINTER(_State)),
    ]


class _Step(ctypes.Structure):
    _fields_ = [
        ("seed", ctypes.c_uint64), ("step", ctypes.c_uint64), ("seq_ids", ctypes.c_void_p),
        ("next_tokens", ctypes.c_void_p), ("backfill_dest", ctypes.c_void_p), ("next_len", ctypes.c_int64),
    ]


class _Shards(ctypes.Structure):
    _fields_ = [("shard_len", ctypes.c_int64), ("shard_stride", ctypes.c_int64)]


_vp, _i64, _i32, _sz = ctypes.c_void_p, ctypes.c_int64, ctypes.c_int32, ctypes.c_size_t
_lib.albireo_workspace_size.argtypes = [_i64, _i64, ctypes.c_int, _i32]
_lib.albireo_workspace_size.restype = _sz
_lib.albireo_sample_route.argtypes = [_i64, _i64, ctypes.c_int, ctypes.POINTER(_Params), _i32]
_lib.albireo_sample_route.restype = ctypes.c_int
_lib.albireo_sample.argtypes = [_vp, ctypes.c_int, _i64, _i64, _i64, ctypes.POINTER(_Params), _vp, _vp, _vp,
                                _i32, _vp, _vp, _vp, _vp, _sz, _vp]
_lib.albireo_sample.restype = ctypes.c_int
_lib.albireo_sample_noalloc.argtypes = [_vp, ctypes.c_int, _i64, _i64, _i64, ctypes.POINTER(_Params), _vp, _vp,
                                        _vp, _i32, _vp, _vp, _vp, _vp]
_lib.albireo_sample_noalloc.restype = ctypes.c_int
_lib.albireo_apply_penalties.argtypes = [_vp, ctypes.c_int, _i64, _i64, _i64, ctypes.POINTER(_Params), _vp,
                                         _vp, _sz, _vp]
_lib.albireo_apply_penalties.restype = ctypes.c_int
_lib.albireo_topk_topp.argtypes = [_vp, _i64, _i64, _i64, ctypes.POINTER(_Params), _vp, _vp, _vp, _vp, _vp,
                                   _vp, _sz, _vp]
_lib.albireo_topk_topp.restype = ctypes.c_int
_lib.albireo_sample_step.argtypes = [_vp, ctypes.c_int, _i64, _i64, _i64, ctypes.POINTER(_Params),
                                     ctypes.POINTER(_Step), _vp, _vp, _i32, _vp, _vp, _vp, _vp, _sz, _vp]
_lib.albireo_sample_step.restype = ctypes.c_int
_lib.albireo_sample_sharded.argtypes = [_vp, ctypes.c_int, _i64, _i64, _i64, ctypes.POINTER(_Shards),
                                        ctypes.POINTER(_Params), _vp, ctypes.POINTER(_Step), _vp, _vp, _i32, _vp,
                                        _vp, _vp, _vp, _sz, _vp]
_lib.albireo_sample_sharded.restype = ctypes.c_int
_lib.albireo_philox_uniforms.argtypes = [ctypes.c_uint64, ctypes.c_uint64, _vp, _i64, _vp, _vp]
_lib.albireo_philox_uniforms.restype = ctypes.c_int
_lib.albireo_backfill.argtypes = [_vp, _vp, _i64, _vp, _i64, _vp]
_lib.albireo_backfill.restype = ctypes.c_int
_lib.albireo_penalty_state_init.argtypes = [ctypes.POINTER(_State), _i64, _i64, _vp, _vp, _i64, _vp, _vp, _i64, _vp]
_lib.albireo_penalty_state_init.restype = ctypes.c_int
_lib.albireo_penalty_state_append.argtypes = [ctypes.POINTER(_State), _i64, _i64, _vp, _vp]
_lib.albireo_penalty_state_append.restype = ctypes.c_int
_lib.albireo_status_string.argtypes = [ctypes.c_int]
_lib.albireo_status_string.restype = ctypes.c_char_p

EXPORTED = ("albireo_workspace_size", "albireo_sample", "albireo_sample_step", "albireo_sample_sharded",
            "albireo_philox_uniforms",
            "albireo_backfill", "albireo_apply_penalties", "albireo_topk_topp", "albireo_status_string",
            "albireo_penalty_state_init", "albireo_penalty_state_append", "albireo_sample_noalloc",
            "albireo_sample_route")


class AlbireoError(RuntimeError):
    def __init__(self, status: int, where: str):
        super().__init__("%s: %s (status %d)" % (where, status_string(status), status))
        self.status = status


def status_string(status: int) -> str:
    return _lib.albireo_status_string(int(status)).decode()


@dataclasses.dataclass
class SamplingParams:
    """Per-row sampling metadata as device tensors ([B] each; None turns a feature off)."""
    temperature: Optional[torch.Tensor] = None         # float32
    top_k: Optional[torch.Tensor] = None               # int32
    top_p: Optional[torch.Tensor] = None               # float32
    min_p: Optional[torch.Tensor] = None               # float32
    repetition_penalty: Optional[torch.Tensor] = None  # float32
    frequency_penalty: Optional[torch.Tensor] = None   # float32
    presence_penalty: Optional[torch.Tensor] = None    # float32
    hist_offsets: Optional[torch.Tensor] = None        # int64 [B + 1]
    hist_ids: Optional[torch.Tensor] = None            # int32
    prompt_offsets: Optional[torch.Tensor] = None      # int64 [B + 1]: with it, hist_* is the output only
    prompt_ids: Optional[torch.Tensor] = None          # int32
    state: Optional["PenaltyState"] = None             # in place of hist_* and prompt_*


_DT = {"temperature": torch.float32, "top_k": torch.int32, "top_p": torch.float32, "min_p": torch.float32,
       "repetition_penalty": torch.float32, "frequency_penalty": torch.float32,
       "presence_penalty": torch.float32, "hist_offsets": torch.int64, "hist_ids": torch.int32,
       "prompt_offsets": torch.int64, "prompt_ids": torch.int32}


def _ptr(t: Optional[torch.Tensor], name: str, device) -> Optional[int]:
    if t is None:
        return None
    if t.device != device or t.dtype != _DT[name] or not t.is_contiguous():
        raise ValueError("%s must be a contiguous %s tensor on %s" % (name, _DT[name], device))
    return t.data_ptr()


def _params(p: Optional[SamplingParams], device) -> Optional[_Params]:
    if p is None:
        return None
    s = _Params()
    for f in ("temperature", "top_k", "top_p", "min_p", "repetition_penalty", "frequency_penalty",
              "presence_penalty", "hist_offsets", "hist_ids", "prompt_offsets", "prompt_ids"):
        setattr(s, f, _ptr(getattr(p, f), f, device))
    s.hist_len = 0 if p.hist_ids is None else int(p.hist_ids.numel())
    s.prompt_len = 0 if p.prompt_ids is None else int(p.prompt_ids.numel())
    if p.state is not None:
        s._state = p.state._struct(device)  # kept alive with the struct
        s.state = ctypes.pointer(s._state)
    return s


class PenaltyState:
    """Per-sequence penalty state of B rows on the device (the distinct ids of each row's prompt and
    output with their output counts and prompt marks), built from histories by init() and advanced by
    one sampled token per row with append()."""

    def __init__(self, B: int, cap: int, device=None):
        self.device = torch.device("cuda") if device is None else torch.device(device)
        self.B, self.cap = B, cap
        self.ids = torch.zeros((B, cap), dtype=torch.int32, device=self.device)
        self.counts = torch.zeros((B, cap), dtype=torch.int32, device=self.device)  # uint32 bit patterns
        self.len = torch.zeros(B, dtype=torch.int32, device=self.device)
        self.flags = torch.zeros(B, dtype=torch.int32, device=self.device)
        self.device = self.ids.device  # with its index

    def _struct(self, device) -> _State:
        if self.ids.device != device:
            raise ValueError("penalty state lives on %s, not %s" % (self.ids.device, device))
        return _State(cap=self.cap, ids=self.ids.data_ptr(), counts=self.counts.data_ptr(),
                      len=self.len.data_ptr(), flags=self.flags.data_ptr())

    def init(self, V: int, prompt_offsets=None, prompt_ids=None, out_offsets=None, out_ids=None, stream=None):
        st = self._struct(self.device)
        po = _ptr(prompt_offsets, "prompt_offsets", self.device)
        pi = _ptr(prompt_ids, "prompt_ids", self.device)
        oo = _ptr(out_offsets, "hist_offsets", self.device)
        oi = _ptr(out_ids, "hist_ids", self.device)
        rc = _lib.albireo_penalty_state_init(ctypes.byref(st), self.B, V, po, pi,
                                             0 if prompt_ids is None else int(prompt_ids.numel()), oo, oi,
                                             0 if out_ids is None else int(out_ids.numel()), _stream(stream))
        if rc != OK:
            raise AlbireoError(rc, "albireo_penalty_state_init")
        return self

    def append(self, ids: torch.Tensor, V: int, stream=None):
        if ids.device != self.device or ids.dtype != torch.int32 or not ids.is_contiguous():
            raise ValueError("ids must be a contiguous int32 tensor on %s" % self.device)
        st = self._struct(self.device)
        rc = _lib.albireo_penalty_state_append(ctypes.byref(st), self.B, V, ids.data_ptr(), _stream(stream))
        if rc != OK:
            raise AlbireoError(rc, "albireo_penalty_state_append")
        return self


def _dtype_code(t: torch.Tensor) -> int:
    if t.dtype == torch.bfloat16:
        return BF16
    if t.dtype == torch.float32:
        return F32
    raise ValueError("logits must be bfloat16 or float32")


def _stream(stream) -> int:
    s = torch.cuda.current_stream() if stream is None else stream
    return s.cuda_stream


def workspace_size(B: int, V: int, dtype: torch.dtype, n_top: int = 0) -> int:
    return int(_lib.albireo_workspace_size(B, V, BF16 if dtype == torch.bfloat16 else F32, n_top))


def sample_route(B: int, V: int, dtype: torch.dtype, params: Optional[SamplingParams] = None,
                 sharded: bool = False) -> int:
    """albireo_sample_route: which kernels a sampling call of this shape takes (ROUTE_*); host only."""
    cp = None
    if params is not None and (params.prompt_offsets is not None or params.state is not None):
        cp = _Params()  # only whether a prompt history or a penalty state is given is read
        if params.prompt_offsets is not None:
            cp.prompt_offsets = params.prompt_offsets.data_ptr()
        if params.state is not None:
            cp._route_state = _State()
            cp.state = ctypes.pointer(cp._route_state)
    return int(_lib.albireo_sample_route(B, V, BF16 if dtype == torch.bfloat16 else F32,
                                         ctypes.byref(cp) if cp is not None else None, 1 if sharded else 0))


class Workspace:
    """A zero-filled device workspace for the calls of one stream, grown on demand (the library leaves
    it zeroed).  A new buffer is allocated and zero-filled on the stream that asks for it, so the fill
    is ordered before that stream's launches."""

    def __init__(self, device=None):
        self.device = torch.device("cuda") if device is None else torch.device(device)
        self.buf = None

    def get(self, nbytes: int, stream=None):
        if nbytes == 0:
            return None, 0
        if self.buf is None or self.buf.numel() < nbytes + 256:
            s = torch.cuda.current_stream(self.device) if stream is None else stream
            with torch.cuda.stream(s):
                self.buf = torch.zeros(max(nbytes, 256) + 256, dtype=torch.uint8, device=self.device)
        base = self.buf.data_ptr()
        off = (-base) % 256
        return base + off, self.buf.numel() - off

    def refill(self, stream=None) -> None:
        """Zero the buffer again on the stream: a call that returned ALBIREO_E_LAUNCH may have run part
        of its launches and left it non-zero."""
        if self.buf is not None:
            s = torch.cuda.current_stream(self.device) if stream is None else stream
            with torch.cuda.stream(s):
                self.buf.zero_()


def _fail(st, name, ws=None, stream=None):
    """Raise the error of a sampling call, zeroing its Workspace first after a refused launch."""
    if st == E_LAUNCH and isinstance(ws, Workspace):
        try:
            ws.refill(stream)
        except RuntimeError:
            pass  # the device refused the fill as well; the launch error is the one to report
    raise AlbireoError(st, name)


_default_ws = {}


def _ws_for(device, workspace, stream=None):
    """The caller's workspace, else the default one of (device, stream): calls on different streams
    never share a workspace."""
    if workspace is not None:
        return workspace
    s = torch.cuda.current_stream(device) if stream is None else stream
    key = (device.type, device.index, s.cuda_stream)
    if key not in _default_ws:
        _default_ws[key] = Workspace(device)
    return _default_ws[key]


def _rows(logits: torch.Tensor, V: Optional[int]):
    if logits.dim() != 2 or logits.stride(1) != 1:
        raise ValueError("logits must be a 2-D tensor with unit stride along the vocabulary")
    B = logits.shape[0]
    V = logits.shape[1] if V is None else V
    ld = logits.stride(0) if B > 1 else max(V, logits.shape[1])
    return B, V, ld


def sample(logits: torch.Tensor, uniforms: torch.Tensor, params: Optional[SamplingParams] = None,
           n_top: int = 0, V: Optional[int] = None, workspace: Optional[Workspace] = None, stream=None,
           out=None):
    """Sample one token per row.  Returns (ids int32 [B], logprobs float32 [B], top_ids [B, n_top],
    top_logprobs [B, n_top], flags int32 [B])."""
    dev = logits.device
    B, V, ld = _rows(logits, V)
    if uniforms.dtype != torch.float32 or uniforms.device != dev or uniforms.numel() < B:
        raise ValueError("uniforms must be a float32 [B] tensor on the logits' device")
    if out is None:
        ids = torch.empty(B, dtype=torch.int32, device=dev)
        lps = torch.empty(B, dtype=torch.float32, device=dev)
        tids = torch.empty((B, n_top), dtype=torch.int32, device=dev)
        tlps = torch.empty((B, n_top), dtype=torch.float32, device=dev)
        flags = torch.empty(B, dtype=torch.int32, device=dev)
    else:
        ids, lps, tids, tlps, flags = out
    dt = _dtype_code(logits)
    ws = _ws_for(dev, workspace, stream)
    wptr, wbytes = ws.get(int(_lib.albireo_workspace_size(B, V, dt, n_top)), stream)
    prm = _params(params, dev)
    st = _lib.albireo_sample(logits.data_ptr(), dt, B, V, ld, ctypes.byref(prm) if prm else None,
                             uniforms.data_ptr(), ids.data_ptr(), lps.data_ptr(), n_top,
                             tids.data_ptr() if n_top else None, tlps.data_ptr() if n_top else None,
                             flags.data_ptr(), wptr, wbytes, _stream(stream))
    if st != OK:
        _fail(st, "albireo_sample", ws, stream)
    return ids, lps, tids, tlps, flags


def sample_noalloc(logits: torch.Tensor, uniforms: torch.Tensor, params: Optional[SamplingParams] = None,
                   n_top: int = 0, V: Optional[int] = None, stream=None, out=None):
    """albireo_sample_noalloc: sample() with the library's fixed device scratch in place of a workspace
    (nothing is allocated when `out` is given).  Same return value as sample()."""
    dev = logits.device
    B, V, ld = _rows(logits, V)
    if uniforms.dtype != torch.float32 or uniforms.device != dev or uniforms.numel() < B:
        raise ValueError("uniforms must be a float32 [B] tensor on the logits' device")
    ids, lps, tids, tlps, flags = _outs(B, n_top, dev, out)
    prm = _params(params, dev)
    st = _lib.albireo_sample_noalloc(logits.data_ptr(), _dtype_code(logits), B, V, ld,
                                     ctypes.byref(prm) if prm else None, uniforms.data_ptr(), ids.data_ptr(),
                                     lps.data_ptr(), n_top, tids.data_ptr() if n_top else None,
                                     tlps.data_ptr() if n_top else None, flags.data_ptr(), _stream(stream))
    if st != OK:
        raise AlbireoError(st, "albireo_sample_noalloc")
    return ids, lps, tids, tlps, flags


class PreparedSample:
    """albireo_sample with its arguments marshalled once; calling it enqueues one launch with the
    given logits pointer (same shape, dtype and stride as at preparation)."""

    def __init__(self, logits: torch.Tensor, uniforms: torch.Tensor, params: Optional[SamplingParams],
                 n_top: int, V: Optional[int], out, workspace: Optional[Workspace] = None, stream=None):
        dev = logits.device
        self.B, self.V, self.ld = _rows(logits, V)
        self.dt = _dtype_code(logits)
        ws = _ws_for(dev, workspace, stream)
        self.wptr, self.wbytes = ws.get(int(_lib.albireo_workspace_size(self.B, self.V, self.dt, n_top)), stream)
        self.prm = _params(params, dev)
        self.prm_ref = ctypes.byref(self.prm) if self.prm else None
        ids, lps, tids, tlps, flags = out
        # the workspace buffer too: a later, larger call may give the Workspace a new one
        self.keep = (uniforms, params, out, ws.buf)
        self.tail = (self.prm_ref, uniforms.data_ptr(), ids.data_ptr(), lps.data_ptr(), n_top,
                     tids.data_ptr() if n_top else None, tlps.data_ptr() if n_top else None, flags.data_ptr(),
                     self.wptr, self.wbytes, _stream(stream))
        self.fn = _lib.albireo_sample
        self.stream = stream

    def __call__(self, logits_ptr: int) -> None:
        st = self.fn(logits_ptr, self.dt, self.B, self.V, self.ld, *self.tail)
        if st != OK:
            if st == E_LAUNCH and self.keep[3] is not None:  # zero this call's buffer again (the Workspace may hold a newer one)
                buf, dev = self.keep[3], self.keep[3].device
                with torch.cuda.stream(torch.cuda.current_stream(dev) if self.stream is None else self.stream):
                    buf.zero_()
            raise AlbireoError(st, "albireo_sample")


def _step_arg(dev, B, seed, step, seq_ids, next_tokens, backfill_dest):
    if seq_ids is not None and (seq_ids.dtype != torch.int64 or seq_ids.device != dev or seq_ids.numel() < B):
        raise ValueError("seq_ids must be an int64 [B] tensor on the logits' device")
    if next_tokens is not None:
        if next_tokens.dtype != torch.int32 or next_tokens.device != dev or not next_tokens.is_contiguous():
            raise ValueError("next_tokens must be a contiguous int32 tensor on the logits' device")
        if backfill_dest is None or backfill_dest.dtype != torch.int32 or backfill_dest.device != dev \
                or backfill_dest.numel() < B:
            raise ValueError("backfill_dest must be an int32 [B] tensor on the logits' device")
    return _Step(seed=seed & (2**64 - 1), step=step & (2**64 - 1),
                 seq_ids=seq_ids.data_ptr() if seq_ids is not None else None,
                 next_tokens=next_tokens.data_ptr() if next_tokens is not None else None,
                 backfill_dest=backfill_dest.data_ptr() if next_tokens is not None else None,
                 next_len=next_tokens.numel() if next_tokens is not None else 0)


def _outs(B, n_top, dev, out):
    if out is not None:
        return out
    return (torch.empty(B, dtype=torch.int32, device=dev), torch.empty(B, dtype=torch.float32, device=dev),
            torch.empty((B, n_top), dtype=torch.int32, device=dev),
            torch.empty((B, n_top), dtype=torch.float32, device=dev), torch.empty(B, dtype=torch.int32, device=dev))


def sample_step(logits: torch.Tensor, seed: int, step: int, seq_ids: Optional[torch.Tensor] = None,
                params: Optional[SamplingParams] = None, n_top: int = 0, V: Optional[int] = None,
                next_tokens: Optional[torch.Tensor] = None, backfill_dest: Optional[torch.Tensor] = None,
                workspace: Optional[Workspace] = None, stream=None, out=None):
    """albireo_sample_step: uniforms generated on the device from (seed, step, seq_ids), and the sampled
    ids optionally backfilled into next_tokens at backfill_dest.  Returns what sample() returns."""
    dev = logits.device
    B, V, ld = _rows(logits, V)
    stp = _step_arg(dev, B, seed, step, seq_ids, next_tokens, backfill_dest)
    ids, lps, tids, tlps, flags = _outs(B, n_top, dev, out)
    dt = _dtype_code(logits)
    ws = _ws_for(dev, workspace, stream)
    wptr, wbytes = ws.get(int(_lib.albireo_workspace_size(B, V, dt, n_top)), stream)
    prm = _params(params, dev)
    st = _lib.albireo_sample_step(logits.data_ptr(), dt, B, V, ld, ctypes.byref(prm) if prm else None,
                                  ctypes.byref(stp), ids.data_ptr(), lps.data_ptr(), n_top,
                                  tids.data_ptr() if n_top else None, tlps.data_ptr() if n_top else None,
                                  flags.data_ptr(), wptr, wbytes, _stream(stream))
    if st != OK:
        _fail(st, "albireo_sample_step", ws, stream)
    return ids, lps, tids, tlps, flags


def shard_len_for(V: int, t: int, dtype: torch.dtype) -> int:
    """Columns per vocabulary shard when V is split over t workers: ceil(V / t) rounded up to whole
    16-byte slots, the block length albireo_sample_sharded accepts (the last shard is partly used)."""
    vec = 16 // torch.empty((), dtype=dtype).element_size()
    per = (V + t - 1) // t
    return (per + vec - 1) // vec * vec


def padded_batch(s: int, t: int) -> int:
    """Batch size after batch padding: the smallest multiple of t that holds s rows (sec. 6.2,
    "Batch padding")."""
    if s < 0 or t <= 0:
        raise ValueError("need s >= 0 and t > 0")
    return -(-s // t) * t


def sample_sharded(recv: torch.Tensor, V: Optional[int] = None, uniforms: Optional[torch.Tensor] = None,
                   seed: Optional[int] = None, step: int = 0, seq_ids: Optional[torch.Tensor] = None,
                   params: Optional[SamplingParams] = None, n_top: int = 0,
                   next_tokens: Optional[torch.Tensor] = None, backfill_dest: Optional[torch.Tensor] = None,
                   workspace: Optional[Workspace] = None, stream=None, out=None):
    """albireo_sample_sharded on an all-to-all receive buffer recv [t, B, shard_len] (unit stride along
    the last axis; recv.stride(0) is the block stride and recv.stride(1) the row stride): row i is the
    concatenation of recv[0, i], recv[1, i], ... cut at V (default t * shard_len).  Give uniforms
    (as sample()) or seed (as sample_step(), with step, seq_ids and the optional backfill)."""
    if recv.dim() != 3 or recv.stride(2) != 1:
        raise ValueError("recv must be a 3-D tensor [t, B, shard_len] with unit stride along the last axis")
    if (uniforms is None) == (seed is None):
        raise ValueError("give exactly one of uniforms and seed")
    dev = recv.device
    t, B, L = recv.shape
    V = t * L if V is None else V
    if not (t - 1) * L < V <= t * L:
        raise ValueError("V must lie in ((t - 1) * shard_len, t * shard_len]")
    stp = None
    if seed is not None:
        stp = _step_arg(dev, B, seed, step, seq_ids, next_tokens, backfill_dest)
    elif uniforms.dtype != torch.float32 or uniforms.device != dev or uniforms.numel() < B:
        raise ValueError("uniforms must be a float32 [B] tensor on the logits' device")
    ids, lps, tids, tlps, flags = _outs(B, n_top, dev, out)
    dt = _dtype_code(recv)
    ws = _ws_for(dev, workspace, stream)
    wptr, wbytes = ws.get(int(_lib.albireo_workspace_size(B, V, dt, n_top)), stream)
    prm = _params(params, dev)
    shards = _Shards(shard_len=L, shard_stride=recv.stride(0))
    st = _lib.albireo_sample_sharded(recv.data_ptr(), dt, B, V, recv.stride(1), ctypes.byref(shards),
                                     ctypes.byref(prm) if prm else None,
                                     uniforms.data_ptr() if uniforms is not None else None,
                                     ctypes.byref(stp) if stp is not None else None, ids.data_ptr(),
                                     lps.data_ptr(), n_top, tids.data_ptr() if n_top else None,
                                     tlps.data_ptr() if n_top else None, flags.data_ptr(), wptr, wbytes,
                                     _stream(stream))
    if st != OK:
        _fail(st, "albireo_sample_sharded", ws, stream)
    return ids, lps, tids, tlps, flags


def philox_uniforms(seed: int, step: int, seq_ids: Optional[torch.Tensor] = None, B: Optional[int] = None,
                    device=None, stream=None) -> torch.Tensor:
    """albireo_philox_uniforms: float32 [B] uniforms for (seed, step, seq_ids) (seq_ids None: row index)."""
    if seq_ids is not None:
        if seq_ids.dtype != torch.int64 or not seq_ids.is_contiguous():
            raise ValueError("seq_ids must be a contiguous int64 tensor")
        B = seq_ids.numel()
        device = seq_ids.device
    out = torch.empty(B, dtype=torch.float32, device=device)
    st = _lib.albireo_philox_uniforms(seed & (2**64 - 1), step & (2**64 - 1),
                                      seq_ids.data_ptr() if seq_ids is not None else None, B,
                                      out.data_ptr() if B else None, _stream(stream))
    if st != OK:
        raise AlbireoError(st, "albireo_philox_uniforms")
    return out


def backfill(ids: torch.Tensor, dest: torch.Tensor, next_tokens: torch.Tensor, stream=None) -> torch.Tensor:
    """albireo_backfill: next_tokens[dest[i]] = ids[i] where the slot exists (in place; returned)."""
    for t, name in ((ids, "ids"), (dest, "dest"), (next_tokens, "next_tokens")):
        if t.dtype != torch.int32 or not t.is_contiguous():
            raise ValueError("%s must be a contiguous int32 tensor" % name)
    B = ids.numel()
    if dest.numel() < B:
        raise ValueError("dest must have one slot per id")
    st = _lib.albireo_backfill(ids.data_ptr(), dest.data_ptr(), B, next_tokens.data_ptr(), next_tokens.numel(),
                               _stream(stream))
    if st != OK:
        raise AlbireoError(st, "albireo_backfill")
    return next_tokens


def apply_penalties(logits: torch.Tensor, params: SamplingParams, V: Optional[int] = None, out=None,
                    stream=None) -> torch.Tensor:
    """Penalised logits as fp32 [B, V]."""
    dev = logits.device
    B, V, ld = _rows(logits, V)
    if out is None:
        out = torch.empty((B, V), dtype=torch.float32, device=dev)
    prm = _params(params, dev)
    st = _lib.albireo_apply_penalties(logits.data_ptr(), _dtype_code(logits), B, V, ld,
                                      ctypes.byref(prm) if prm else None, out.data_ptr(), None, 0,
                                      _stream(stream))
    if st != OK:
        raise AlbireoError(st, "albireo_apply_penalties")
    return out


def topk_topp(logits: torch.Tensor, params: Optional[SamplingParams] = None, V: Optional[int] = None,
              probs: bool = True, workspace: Optional[Workspace] = None, stream=None):
    """Filtered distribution of fp32 logits.  Returns (probs [B, V] or None, threshold [B], kept [B],
    log_norm [B], flags [B])."""
    if logits.dtype != torch.float32:
        raise ValueError("topk_topp takes float32 logits")
    dev = logits.device
    B, V, ld = _rows(logits, V)
    pr = torch.empty((B, V), dtype=torch.float32, device=dev) if probs else None
    thr = torch.empty(B, dtype=torch.float32, device=dev)
    kept = torch.empty(B, dtype=torch.int32, device=dev)
    lnorm = torch.empty(B, dtype=torch.float32, device=dev)
    flags = torch.empty(B, dtype=torch.int32, device=dev)
    ws = _ws_for(dev, workspace, stream)
    wptr, wbytes = ws.get(int(_lib.albireo_workspace_size(B, V, F32, 0)), stream)
    prm = _params(params, dev)
    st = _lib.albireo_topk_topp(logits.data_ptr(), B, V, ld, ctypes.byref(prm) if prm else None,
                                pr.data_ptr() if pr is not None else None, thr.data_ptr(), kept.data_ptr(),
                                lnorm.data_ptr(), flags.data_ptr(), wptr, wbytes, _stream(stream))
    if st != OK:
        _fail(st, "albireo_topk_topp", ws, stream)
    return pr, thr, kept, lnorm, flags


def raw_call(name: str):
    """The C entry point itself (for tests that exercise the boundary's argument checks)."""
    return getattr(_lib, name)


Params = _Params
