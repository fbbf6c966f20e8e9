"""Thin ctypes binding of liblocks (include/locks.h).

Argument marshalling only: every step of the decode path runs in the HIP
kernels of liblocks.so.  Tensors are torch device tensors (PyTorch provides the
device memory and the stream); the binding passes their data pointers and the
current HIP stream.  If the library is not built, every call raises.
"""
from __future__ import annotations

import ctypes
import math
import os
from dataclasses import dataclass
from typing import Optional

import torch

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "liblocks.so")

LOCKS_BF16 = 0
LOCKS_FP32 = 1
LOCKS_BASIS_INT4 = 0
LOCKS_BASIS_INT8 = 1
LOCKS_BASIS_BF16 = 2
BASIS_NAMES = {LOCKS_BASIS_INT4: "int4", LOCKS_BASIS_INT8: "int8", LOCKS_BASIS_BF16: "bf16"}
PAGE = 16
HEAD_DIM = 128


class LocksError(RuntimeError):
    pass


class _Cfg(ctypes.Structure):
    _fields_ = [(n, ctypes.c_int32) for n in (
        "num_seqs", "num_q_heads", "num_kv_heads", "head_dim", "page_size", "rank",
        "budget_tokens", "max_pages_per_seq", "num_blocks", "kv_dtype", "q_dtype", "basis")]


@dataclass
class Config:
    num_seqs: int
    num_q_heads: int
    num_kv_heads: int
    rank: int
    budget_tokens: int
    max_pages_per_seq: int
    num_blocks: int
    kv_dtype: int = LOCKS_BF16
    q_dtype: int = LOCKS_BF16
    head_dim: int = HEAD_DIM
    page_size: int = PAGE
    basis: int = LOCKS_BASIS_INT4

    @property
    def group(self) -> int:
        return self.num_q_heads // self.num_kv_heads

    @property
    def k(self) -> int:
        return (self.budget_tokens + self.page_size - 1) // self.page_size

    def c(self) -> _Cfg:
        return _Cfg(self.num_seqs, self.num_q_heads, self.num_kv_heads, self.head_dim,
                    self.page_size, self.rank, self.budget_tokens, self.max_pages_per_seq,
                    self.num_blocks, self.kv_dtype, self.q_dtype, self.basis)


LOCKS_KIVI_POST = 0
LOCKS_KIVI_PRE = 1


class Kivi(ctypes.Structure):
    """KIVI fake quantisation of finalised pages: bits, value channel group, stage."""
    _fields_ = [("bits", ctypes.c_int32), ("v_group", ctypes.c_int32), ("stage", ctypes.c_int32)]


class StepOpts(ctypes.Structure):
    """Options of locks_decode_step_ex: KIVI, and the step's new KV rows."""
    _fields_ = [("kivi", ctypes.POINTER(Kivi)), ("k_new", ctypes.c_void_p),
                ("v_new", ctypes.c_void_p)]


_lib = None
_P = ctypes.c_void_p
_SZ = ctypes.c_size_t
_I = ctypes.c_int32

_SIGS = {
    "locks_summary_payload_bytes": (_SZ, [_I]),
    "locks_summary_stride": (_SZ, [_I]),
    "locks_summary_payload_bytes_ex": (_SZ, [_I, _I]),
    "locks_summary_stride_ex": (_SZ, [_I, _I]),
    "locks_summary_payload_bytes_page": (_SZ, [_I, _I, _I]),
    "locks_summary_stride_page": (_SZ, [_I, _I, _I]),
    "locks_workspace_bytes": (_SZ, [ctypes.POINTER(_Cfg)]),
    "locks_build_summaries": (ctypes.c_int, [ctypes.POINTER(_Cfg), _P, _P, _P, _P, _I, _P, _P]),
    "locks_build_factors": (ctypes.c_int, [ctypes.POINTER(_Cfg), _P, _P, _P, _P, _I, _P, _P, _P,
                                           _P, _P]),
    "locks_select": (ctypes.c_int, [ctypes.POINTER(_Cfg), _P, _P, _P, _P, _P, _P, _P, _P, _SZ,
                                    _P]),
    "locks_score_pages": (ctypes.c_int, [ctypes.POINTER(_Cfg), _P, _P, _P, _P, _P, _P, _SZ, _P]),
    "locks_sparse_attend": (ctypes.c_int, [ctypes.POINTER(_Cfg), _P, _P, _P, _P, _P, _P, _P, _P,
                                           _P, _SZ, _P]),
    "locks_dense_attend": (ctypes.c_int, [ctypes.POINTER(_Cfg), _P, _P, _P, _P, _P, _P, _P, _P,
                                          _SZ, _P]),
    "locks_decode_step": (ctypes.c_int, [ctypes.POINTER(_Cfg), _P, _P, _P, _P, _P, _P, _P, _I,
                                         _P, _P, _P, _P, _P, _SZ, _P]),
    "locks_kivi_quantize": (ctypes.c_int, [ctypes.POINTER(_Cfg), ctypes.POINTER(Kivi), _P, _P, _P,
                                           _P, _P, _I, _P]),
    "locks_decode_step_ex": (ctypes.c_int, [ctypes.POINTER(_Cfg), ctypes.POINTER(StepOpts), _P,
                                            _P, _P, _P, _P, _P, _P, _I, _P, _P, _P, _P, _P, _SZ,
                                            _P]),
    "locks_append_kv": (ctypes.c_int, [ctypes.POINTER(_Cfg), _P, _P, _P, _P, _P, _P, _P]),
    "locks_init": (ctypes.c_int, []),
    "locks_decode_step_static": (ctypes.c_int, [ctypes.POINTER(_Cfg), _P, _P, _P, _P, _P, _P, _P,
                                                _I, _P, _P, _P, _P, _P]),
    "locks_set_table_checks": (ctypes.c_int, [_I]),
    "locks_table_error_offset": (_SZ, [ctypes.POINTER(_Cfg)]),
    "locks_strerror": (ctypes.c_char_p, [ctypes.c_int]),
    "locks_last_hip_error": (ctypes.c_int, []),
}


def lib():
    """Load liblocks.so (raises LocksError when it has not been built)."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise LocksError(f"{LIB_PATH} is missing: build it with "
                             "`python -m paper_2607_24555_amd.build_lib`")
        L = ctypes.CDLL(LIB_PATH)
        for name, (res, args) in _SIGS.items():
            f = getattr(L, name)
            f.restype = res
            f.argtypes = args
        _lib = L
    return _lib


def _ptr(t: Optional[torch.Tensor]):
    if t is None:
        return None
    if not t.is_cuda:
        raise LocksError("liblocks takes device tensors")
    if not t.is_contiguous():
        raise LocksError("liblocks takes contiguous tensors")
    return ctypes.c_void_p(t.data_ptr())


_TORCH_OF = {LOCKS_BF16: torch.bfloat16, LOCKS_FP32: torch.float32}


def _need(name: str, t: Optional[torch.Tensor], shape, dtype, optional: bool = False):
    """Checks a tensor argument against the layout include/locks.h documents for
    cfg before anything reaches the library: the kernels trust shapes and dtypes,
    so a mismatch would read or write outside the allocation."""
    if t is None:
        if optional:
            return
        raise LocksError(f"{name} is required")
    if t.dtype != dtype:
        raise LocksError(f"{name}: dtype {t.dtype}, expected {dtype}")
    if tuple(t.shape) != tuple(shape):
        raise LocksError(f"{name}: shape {tuple(t.shape)}, expected {tuple(shape)}")


def _same_device(*ts):
    devs = {t.device for t in ts if t is not None}
    if len(devs) > 1:
        raise LocksError(f"tensors on several devices: {sorted(map(str, devs))}")


def _check_q(cfg: "Config", q):
    _need("q", q, (cfg.num_seqs, cfg.num_q_heads, cfg.head_dim), _TORCH_OF[cfg.q_dtype])


def _check_tables(cfg: "Config", page_table, seq_lens):
    _need("page_table", page_table, (cfg.num_seqs, cfg.max_pages_per_seq), torch.int32)
    _need("seq_lens", seq_lens, (cfg.num_seqs,), torch.int32)


def _check_cache(cfg: "Config", name: str, cache):
    _need(name, cache, (cfg.num_blocks, cfg.num_kv_heads, cfg.page_size, cfg.head_dim),
          _TORCH_OF[cfg.kv_dtype])


def _check_summaries(cfg: "Config", summaries):
    _need("summaries", summaries,
          (cfg.num_blocks, cfg.num_kv_heads, summary_stride(cfg.rank, cfg.basis, cfg.page_size)),
          torch.uint8)


def _check_list(name: str, lst):
    if lst is not None and (lst.dtype != torch.int32 or lst.dim() != 2 or lst.shape[1] != 2):
        raise LocksError(f"{name}: expected int32 [n][2] (sequence, page) pairs, got "
                         f"{lst.dtype} {tuple(lst.shape)}")


def _check_ws(ws):
    if ws is None or ws.dtype != torch.uint8 or ws.dim() != 1:
        raise LocksError("ws: expected a 1-D uint8 workspace (alloc_workspace)")


def _check_select_out(cfg: "Config", out_ids, out_sel_lse, out_all_lse=None):
    _need("out_ids", out_ids, (cfg.num_seqs, cfg.num_kv_heads, cfg.k), torch.int32)
    _need("out_sel_lse", out_sel_lse, (cfg.num_seqs, cfg.num_q_heads, cfg.k), torch.float32)
    _need("out_all_lse", out_all_lse, (cfg.num_seqs, cfg.num_q_heads, cfg.max_pages_per_seq),
          torch.float32, optional=True)


def _check_attend_out(cfg: "Config", out, out_lse):
    _need("out", out, (cfg.num_seqs, cfg.num_q_heads, cfg.head_dim), torch.float32)
    _need("out_lse", out_lse, (cfg.num_seqs, cfg.num_q_heads), torch.float32, optional=True)


def _stream(stream) -> Optional[ctypes.c_void_p]:
    s = torch.cuda.current_stream() if stream is None else stream
    return ctypes.c_void_p(s.cuda_stream)


def _check(rc: int):
    if rc != 0:
        L = lib()
        msg = L.locks_strerror(rc).decode()
        raise LocksError(f"liblocks status {rc}: {msg} (hip error {L.locks_last_hip_error()})")


def init():
    """locks_init: create the current device's side stream before any capture."""
    _check(lib().locks_init())


LOCKS_TABLE_E_LENGTH = 1
LOCKS_TABLE_E_BLOCK = 2


def set_table_checks(enable: bool) -> bool:
    """locks_set_table_checks: device-side checks of page_table / seq_lens in every
    call that takes a workspace (clamped copies, error word in the workspace).
    Returns the previous setting."""
    return bool(lib().locks_set_table_checks(1 if enable else 0))


def table_errors(cfg: Config, ws: torch.Tensor):
    """The last checked call's error word (LOCKS_TABLE_E_* bits) and the per-sequence
    words, read from the workspace (waits for the work queued on it)."""
    c = cfg.c()
    off = int(lib().locks_table_error_offset(ctypes.byref(c)))
    if off == ctypes.c_size_t(-1).value:
        raise LocksError("invalid configuration")
    words = ws[off:off + 4 * (1 + cfg.num_seqs)].view(torch.int32).cpu()
    return int(words[0]), [int(x) for x in words[1:]]


def summary_payload_bytes(rank: int) -> int:
    return int(lib().locks_summary_payload_bytes(rank))


def summary_stride(rank: int, basis: int = LOCKS_BASIS_INT4, page_size: int = PAGE) -> int:
    return int(lib().locks_summary_stride_page(rank, basis, page_size))


def summary_payload_bytes_ex(rank: int, basis: int, page_size: int = PAGE) -> int:
    return int(lib().locks_summary_payload_bytes_page(rank, basis, page_size))


def workspace_bytes(cfg: Config) -> int:
    c = cfg.c()
    return int(lib().locks_workspace_bytes(ctypes.byref(c)))


def alloc_workspace(cfg: Config, device="cuda") -> torch.Tensor:
    n = workspace_bytes(cfg)
    if n == 0:
        raise LocksError("invalid configuration")
    return torch.empty(n, dtype=torch.uint8, device=device)


def alloc_summaries(cfg: Config, device="cuda") -> torch.Tensor:
    return torch.zeros(cfg.num_blocks, cfg.num_kv_heads,
                       summary_stride(cfg.rank, cfg.basis, cfg.page_size), dtype=torch.uint8,
                       device=device)


def build_summaries(cfg: Config, k_cache, page_table, seq_lens, summaries,
                    build_list: Optional[torch.Tensor] = None, stream=None):
    _check_cache(cfg, "k_cache", k_cache)
    _check_tables(cfg, page_table, seq_lens)
    _check_summaries(cfg, summaries)
    _check_list("build_list", build_list)
    _same_device(k_cache, page_table, seq_lens, summaries, build_list)
    c = cfg.c()
    n = 0 if build_list is None else int(build_list.shape[0])
    _check(lib().locks_build_summaries(ctypes.byref(c), _ptr(k_cache), _ptr(page_table),
                                       _ptr(seq_lens), _ptr(build_list), n, _ptr(summaries),
                                       _stream(stream)))


def build_factors(cfg: Config, k_cache, page_table, seq_lens, build_list: torch.Tensor,
                  stream=None):
    _check_cache(cfg, "k_cache", k_cache)
    _check_tables(cfg, page_table, seq_lens)
    _check_list("build_list", build_list)
    if build_list is None:
        raise LocksError("build_factors needs a build list")
    _same_device(k_cache, page_table, seq_lens, build_list)
    n = int(build_list.shape[0])
    dev = k_cache.device
    mu = torch.zeros(n, cfg.num_kv_heads, HEAD_DIM, device=dev)
    basis = torch.zeros(n, cfg.num_kv_heads, HEAD_DIM, cfg.rank, device=dev)
    coef = torch.zeros(n, cfg.num_kv_heads, cfg.page_size, cfg.rank, device=dev)
    sigma2 = torch.zeros(n, cfg.num_kv_heads, cfg.page_size, device=dev)
    c = cfg.c()
    _check(lib().locks_build_factors(ctypes.byref(c), _ptr(k_cache), _ptr(page_table),
                                     _ptr(seq_lens), _ptr(build_list), n, _ptr(mu), _ptr(basis),
                                     _ptr(coef), _ptr(sigma2), _stream(stream)))
    return mu, basis, coef, sigma2


def alloc_select_outputs(cfg: Config, device="cuda"):
    ids = torch.empty(cfg.num_seqs, cfg.num_kv_heads, cfg.k, dtype=torch.int32, device=device)
    sel = torch.empty(cfg.num_seqs, cfg.num_q_heads, cfg.k, dtype=torch.float32, device=device)
    return ids, sel


def select(cfg: Config, q, summaries, page_table, seq_lens, ws, out_ids=None, out_sel_lse=None,
           out_all_lse=None, stream=None):
    if out_ids is None:
        out_ids, out_sel_lse = alloc_select_outputs(cfg, q.device)
    _check_q(cfg, q)
    _check_summaries(cfg, summaries)
    _check_tables(cfg, page_table, seq_lens)
    _check_ws(ws)
    _check_select_out(cfg, out_ids, out_sel_lse, out_all_lse)
    _same_device(q, summaries, page_table, seq_lens, ws, out_ids, out_sel_lse, out_all_lse)
    c = cfg.c()
    _check(lib().locks_select(ctypes.byref(c), _ptr(q), _ptr(summaries), _ptr(page_table),
                              _ptr(seq_lens), _ptr(out_ids), _ptr(out_sel_lse), _ptr(out_all_lse),
                              _ptr(ws), ws.numel(), _stream(stream)))
    return out_ids, out_sel_lse


def score_pages(cfg: Config, q, summaries, page_table, seq_lens, ws, out_all_lse=None,
                stream=None):
    call = prepare_score_pages(cfg, q, summaries, page_table, seq_lens, ws, out_all_lse)
    call(stream)
    return call.outputs


def prepare_score_pages(cfg: Config, q, summaries, page_table, seq_lens, ws,
                        out_all_lse=None) -> "PreparedCall":
    """score_pages' checks and marshalling, done once (see PreparedCall)."""
    if out_all_lse is None:
        out_all_lse = torch.empty(cfg.num_seqs, cfg.num_q_heads, cfg.max_pages_per_seq,
                                  dtype=torch.float32, device=q.device)
    _check_q(cfg, q)
    _check_summaries(cfg, summaries)
    _check_tables(cfg, page_table, seq_lens)
    _check_ws(ws)
    _need("out_all_lse", out_all_lse, (cfg.num_seqs, cfg.num_q_heads, cfg.max_pages_per_seq),
          torch.float32)
    _same_device(q, summaries, page_table, seq_lens, ws, out_all_lse)
    return PreparedCall(lib().locks_score_pages, cfg.c(),
                        (_ptr(q), _ptr(summaries), _ptr(page_table), _ptr(seq_lens),
                         _ptr(out_all_lse), _ptr(ws), ws.numel()), None, out_all_lse)


def alloc_attend_outputs(cfg: Config, device="cuda"):
    out = torch.empty(cfg.num_seqs, cfg.num_q_heads, HEAD_DIM, dtype=torch.float32, device=device)
    lse = torch.empty(cfg.num_seqs, cfg.num_q_heads, dtype=torch.float32, device=device)
    return out, lse


def sparse_attend(cfg: Config, q, k_cache, v_cache, page_table, seq_lens, page_ids, ws,
                  out=None, out_lse=None, stream=None):
    if out is None:
        out, out_lse = alloc_attend_outputs(cfg, q.device)
    _check_q(cfg, q)
    _check_cache(cfg, "k_cache", k_cache)
    _check_cache(cfg, "v_cache", v_cache)
    _check_tables(cfg, page_table, seq_lens)
    _need("page_ids", page_ids, (cfg.num_seqs, cfg.num_kv_heads, cfg.k), torch.int32)
    _check_ws(ws)
    _check_attend_out(cfg, out, out_lse)
    _same_device(q, k_cache, v_cache, page_table, seq_lens, page_ids, ws, out, out_lse)
    c = cfg.c()
    _check(lib().locks_sparse_attend(ctypes.byref(c), _ptr(q), _ptr(k_cache), _ptr(v_cache),
                                     _ptr(page_table), _ptr(seq_lens), _ptr(page_ids), _ptr(out),
                                     _ptr(out_lse), _ptr(ws), ws.numel(), _stream(stream)))
    return out, out_lse


def dense_attend(cfg: Config, q, k_cache, v_cache, page_table, seq_lens, ws, out=None,
                 out_lse=None, stream=None):
    call = prepare_dense_attend(cfg, q, k_cache, v_cache, page_table, seq_lens, ws, out, out_lse)
    call(stream)
    return call.outputs


def prepare_dense_attend(cfg: Config, q, k_cache, v_cache, page_table, seq_lens, ws, out=None,
                         out_lse=None) -> "PreparedCall":
    """dense_attend's checks and marshalling, done once (see PreparedCall)."""
    if out is None:
        out, out_lse = alloc_attend_outputs(cfg, q.device)
    _check_q(cfg, q)
    _check_cache(cfg, "k_cache", k_cache)
    _check_cache(cfg, "v_cache", v_cache)
    _check_tables(cfg, page_table, seq_lens)
    _check_ws(ws)
    _check_attend_out(cfg, out, out_lse)
    _same_device(q, k_cache, v_cache, page_table, seq_lens, ws, out, out_lse)
    return PreparedCall(lib().locks_dense_attend, cfg.c(),
                        (_ptr(q), _ptr(k_cache), _ptr(v_cache), _ptr(page_table), _ptr(seq_lens),
                         _ptr(out), _ptr(out_lse), _ptr(ws), ws.numel()), None, (out, out_lse))


def decode_step(cfg: Config, q, k_cache, v_cache, page_table, seq_lens, summaries, ws,
                build_list: Optional[torch.Tensor] = None, out_ids=None, out_sel_lse=None,
                out=None, out_lse=None, stream=None, kivi: Optional[Kivi] = None,
                k_new=None, v_new=None):
    """The fused step.  With `kivi` the listed pages are KIVI fake-quantised in place
    (before or after their build, per kivi.stage); with k_new / v_new [S][H_kv][128]
    the step first writes each sequence's newest token (seq_lens counting it) --
    locks_decode_step_ex."""
    step = prepare_decode_step(cfg, q, k_cache, v_cache, page_table, seq_lens, summaries, ws,
                               build_list, out_ids, out_sel_lse, out, out_lse, kivi, k_new, v_new)
    step(stream)
    return step.outputs


class PreparedCall:
    """One library call with its arguments checked and marshalled once: every call
    of the object enqueues the same call on the given or current stream.  For
    fixed-shape loops over fixed buffers (the deployment pattern of Sec. 4
    "Implementation"), where per-call argument checks would cost host time."""

    def __init__(self, fn, cfg_struct, args, opts, outputs):
        self._fn, self._c, self._args, self._opts = fn, cfg_struct, args, opts
        self.outputs = outputs

    def __call__(self, stream=None):
        if self._opts is None:
            _check(self._fn(ctypes.byref(self._c), *self._args, _stream(stream)))
        else:
            _check(self._fn(ctypes.byref(self._c), ctypes.byref(self._opts), *self._args,
                            _stream(stream)))


def prepare_decode_step(cfg: Config, q, k_cache, v_cache, page_table, seq_lens, summaries, ws,
                        build_list: Optional[torch.Tensor] = None, out_ids=None,
                        out_sel_lse=None, out=None, out_lse=None, kivi: Optional[Kivi] = None,
                        k_new=None, v_new=None) -> PreparedCall:
    """decode_step's checks and marshalling, done once; returns the PreparedCall.
    The tensors must stay alive (and keep their storage) while it is used."""
    if out_ids is None:
        out_ids, out_sel_lse = alloc_select_outputs(cfg, q.device)
    if out is None:
        out, out_lse = alloc_attend_outputs(cfg, q.device)
    _check_q(cfg, q)
    _check_cache(cfg, "k_cache", k_cache)
    _check_cache(cfg, "v_cache", v_cache)
    _check_tables(cfg, page_table, seq_lens)
    _check_summaries(cfg, summaries)
    _check_list("build_list", build_list)
    _check_ws(ws)
    _check_select_out(cfg, out_ids, out_sel_lse)
    _check_attend_out(cfg, out, out_lse)
    for name, t in (("k_new", k_new), ("v_new", v_new)):
        _need(name, t, (cfg.num_seqs, cfg.num_kv_heads, cfg.head_dim), _TORCH_OF[cfg.kv_dtype],
              optional=True)
    _same_device(q, k_cache, v_cache, page_table, seq_lens, summaries, build_list, ws, out_ids,
                 out_sel_lse, out, out_lse, k_new, v_new)
    n = 0 if build_list is None else int(build_list.shape[0])
    c = cfg.c()
    args = (_ptr(q), _ptr(k_cache), _ptr(v_cache), _ptr(page_table), _ptr(seq_lens),
            _ptr(summaries), _ptr(build_list), n, _ptr(out_ids), _ptr(out_sel_lse), _ptr(out),
            _ptr(out_lse), _ptr(ws), ws.numel())
    outputs = (out_ids, out_sel_lse, out, out_lse)
    if kivi is None and k_new is None and v_new is None:
        return PreparedCall(lib().locks_decode_step, c, args, None, outputs)
    opts = StepOpts(ctypes.pointer(kivi) if kivi is not None else None, _ptr(k_new), _ptr(v_new))
    return PreparedCall(lib().locks_decode_step_ex, c, args, opts, outputs)


STATIC_SCRATCH_BYTES = 64 << 20


def decode_step_static(cfg: Config, q, k_cache, v_cache, page_table, seq_lens, summaries,
                       build_list: Optional[torch.Tensor] = None, out_ids=None, out_sel_lse=None,
                       out=None, out_lse=None, stream=None):
    """locks_decode_step_static: the fused step on the library's static device scratch
    (no workspace argument; the call allocates nothing)."""
    if out_ids is None:
        out_ids, out_sel_lse = alloc_select_outputs(cfg, q.device)
    if out is None:
        out, out_lse = alloc_attend_outputs(cfg, q.device)
    _check_q(cfg, q)
    _check_cache(cfg, "k_cache", k_cache)
    _check_cache(cfg, "v_cache", v_cache)
    _check_tables(cfg, page_table, seq_lens)
    _check_summaries(cfg, summaries)
    _check_list("build_list", build_list)
    _check_select_out(cfg, out_ids, out_sel_lse)
    _check_attend_out(cfg, out, out_lse)
    _same_device(q, k_cache, v_cache, page_table, seq_lens, summaries, build_list, out_ids,
                 out_sel_lse, out, out_lse)
    n = 0 if build_list is None else int(build_list.shape[0])
    c = cfg.c()
    _check(lib().locks_decode_step_static(
        ctypes.byref(c), _ptr(q), _ptr(k_cache), _ptr(v_cache), _ptr(page_table), _ptr(seq_lens),
        _ptr(summaries), _ptr(build_list), n, _ptr(out_ids), _ptr(out_sel_lse), _ptr(out),
        _ptr(out_lse), _stream(stream)))
    return out_ids, out_sel_lse, out, out_lse


def append_kv(cfg: Config, k_new, v_new, k_cache, v_cache, page_table, seq_lens, stream=None):
    """Write each sequence's newest token (token seq_lens[s] - 1) from k_new / v_new
    [S][H_kv][128] into the paged caches -- locks_append_kv."""
    for name, t in (("k_new", k_new), ("v_new", v_new)):
        _need(name, t, (cfg.num_seqs, cfg.num_kv_heads, cfg.head_dim), _TORCH_OF[cfg.kv_dtype])
    _check_cache(cfg, "k_cache", k_cache)
    _check_cache(cfg, "v_cache", v_cache)
    _check_tables(cfg, page_table, seq_lens)
    _same_device(k_new, v_new, k_cache, v_cache, page_table, seq_lens)
    c = cfg.c()
    _check(lib().locks_append_kv(ctypes.byref(c), _ptr(k_new), _ptr(v_new), _ptr(k_cache),
                                 _ptr(v_cache), _ptr(page_table), _ptr(seq_lens), _stream(stream)))


def kivi_quantize(cfg: Config, kivi: Kivi, k_cache, v_cache, page_table, seq_lens,
                  page_list: Optional[torch.Tensor] = None, stream=None):
    """KIVI fake quantisation, in place, of every complete page (page_list None) or of
    the listed (seq, page) pairs [n][2] int32 -- locks_kivi_quantize."""
    n = 0 if page_list is None else int(page_list.shape[0])
    if page_list is not None and n == 0:
        return                      # an empty list names no page (NULL would mean all)
    _check_cache(cfg, "k_cache", k_cache)
    _check_cache(cfg, "v_cache", v_cache)
    _check_tables(cfg, page_table, seq_lens)
    _check_list("page_list", page_list)
    _same_device(k_cache, v_cache, page_table, seq_lens, page_list)
    c = cfg.c()
    _check(lib().locks_kivi_quantize(ctypes.byref(c), ctypes.byref(kivi), _ptr(k_cache),
                                     _ptr(v_cache), _ptr(page_table), _ptr(seq_lens),
                                     _ptr(page_list), n, _stream(stream)))


def config_for(spec, num_blocks: int, max_pages: int) -> Config:
    """Config of a workloads.WorkloadSpec laid out with num_blocks / max_pages."""
    dt = {"bf16": LOCKS_BF16, "fp32": LOCKS_FP32}
    return Config(spec.num_seqs, spec.num_q_heads, spec.num_kv_heads, spec.rank,
                  spec.budget_tokens, max_pages, num_blocks, dt[spec.kv_dtype], dt[spec.q_dtype],
                  page_size=getattr(spec, "page_size", PAGE))


def page_count(seq_len: int, page_size: int = PAGE) -> int:
    return math.ceil(seq_len / page_size)
