"""TokenTiming verification hot path on AMD Instinct MI355X (gfx950).

Thin ctypes binding over the C-ABI in include/tt.h (libtt.so, built from csrc/).
Each function marshals torch device tensors into pointers and calls the library on
the current HIP stream; all arithmetic happens in the HIP kernels.  Nothing here
falls back to the CPU: if libtt.so is missing or a call fails, an exception is
raised.

    align     tt_align     Dynamic Token Warping + backtrack + mapping (Sec. 4.1, Alg. 1, App. A.2)
    transfer  tt_transfer  draft probability of the aligned draft token (Alg. 2, App. A.2)
    verify    tt_verify    acceptance, residual / bonus sampling (Sec. 3, 4.2.2-4.2.3, App. D Alg. 4)
    verify_dense  tt_verify_dense  the same with dense proposals over one vocabulary (App. D Alg. 4)
    delta_histogram  tt_delta_histogram  |i - j| over the optimal paths' cells (Fig. CDF, App. K)
    delta_quantile / w_at_quantile  tt_delta_quantile  where that distribution reaches 0.9 (App. K)
    token_index / retokenize  tt_token_index_build / tt_retokenize  draft tokens -> proxy target
              tokens by greedy longest match (Sec. 4.2.1, Alg. 2, App. A.1)
    vocab_intersection / tli_proposal / verify_tli  the Token-Level Intersection proposal
              (App. D Alg. 3): the intersection maps, q' rows, and the verification with q'
              formed on the fly
    verify_logits  tt_verify_logits  verification from bf16 logits and a temperature (App. F)
"""
from __future__ import annotations

import ctypes
import os

__all__ = ["Vocab", "align", "align_workspace", "transfer", "verify", "verify_noalloc", "verify_dense", "verify_workspace", "lib",
           "delta_histogram", "delta_quantile", "w_at_quantile", "token_index", "retokenize", "LIB_PATH",
           "vocab_intersection", "tli_proposal", "verify_tli", "verify_logits",
           "TTError", "path_capacity"]

LIB_PATH = os.path.join(os.path.dirname(os.path.abspath(__file__)), "libtt.so")

TT_OK, TT_EINVAL, TT_EUNSUPPORTED, TT_ELAUNCH, TT_EWORKSPACE = 0, -1, -2, -3, -4


class TTError(RuntimeError):
    def __init__(self, status: int, where: str):
        self.status = status
        super().__init__(f"{where}: {lib().tt_status_string(status).decode()} (status {status})")


class c_tt_vocab(ctypes.Structure):
    _fields_ = [("bytes", ctypes.c_void_p), ("offsets", ctypes.c_void_p),
                ("n_tokens", ctypes.c_int32), ("max_token_bytes", ctypes.c_int32)]


_lib = None


def lib():
    """The loaded libtt.so with argument types declared (raises if it is not built)."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise RuntimeError(f"{LIB_PATH} is not built; run paper_2510_15545_amd/build.py "
                               "(or __graft_entry__.build())")
        L = ctypes.CDLL(LIB_PATH)
        P, i32, i64, sz = ctypes.c_void_p, ctypes.c_int32, ctypes.c_int64, ctypes.c_size_t
        VP = ctypes.POINTER(c_tt_vocab)
        L.tt_status_string.argtypes = [ctypes.c_int]
        L.tt_status_string.restype = ctypes.c_char_p
        L.tt_version.argtypes = []
        L.tt_version.restype = ctypes.c_int
        L.tt_align_workspace_size.argtypes = [i32, i32, i32, i32, i32, ctypes.POINTER(sz)]
        L.tt_align_workspace_size.restype = ctypes.c_int
        L.tt_align.argtypes = [VP, VP, i32, P, P, P, P, i32, i32, i32, P, P, P, P, P, sz, P]
        L.tt_align.restype = ctypes.c_int
        L.tt_transfer.argtypes = [i32, i32, P, P, P, P, P, i64, P, P]
        L.tt_transfer.restype = ctypes.c_int
        L.tt_verify_workspace_size.argtypes = [i32, i32, ctypes.POINTER(sz)]
        L.tt_verify_workspace_size.restype = ctypes.c_int
        L.tt_verify.argtypes = [i32, i32, P, P, P, P, i64, P, P, i32, P, P, P, P, sz, P]
        L.tt_verify.restype = ctypes.c_int
        L.tt_verify_noalloc.argtypes = [i32, i32, P, P, P, P, i64, P, P, i32, P, P, P, P]
        L.tt_verify_noalloc.restype = ctypes.c_int
        L.tt_verify_dense.argtypes = [i32, i32, P, P, P, i64, P, i64, P, P, i32, P, P, P, P, sz, P]
        L.tt_verify_dense.restype = ctypes.c_int
        L.tt_verify_logits.argtypes = [i32, i32, P, P, P, P, i64, P, P, P, P, i32, P, P, P]
        L.tt_verify_logits.restype = ctypes.c_int
        L.tt_delta_histogram.argtypes = [i32, P, P, P, P, i32, P, P]
        L.tt_delta_histogram.restype = ctypes.c_int
        L.tt_delta_quantile.argtypes = [P, i32, i32, i32, P, P]
        L.tt_delta_quantile.restype = ctypes.c_int
        L.tt_token_index_size.argtypes = [i32, ctypes.POINTER(sz)]
        L.tt_token_index_size.restype = ctypes.c_int
        L.tt_token_index_build.argtypes = [VP, P, sz, P]
        L.tt_token_index_build.restype = ctypes.c_int
        L.tt_retokenize_workspace_size.argtypes = [i32, i32, ctypes.POINTER(sz)]
        L.tt_retokenize_workspace_size.restype = ctypes.c_int
        L.tt_retokenize.argtypes = [VP, VP, P, sz, i32, P, P, i32, i32, P, P, P, sz, P]
        L.tt_retokenize.restype = ctypes.c_int
        L.tt_vocab_intersection.argtypes = [VP, P, sz, VP, P, sz, P, P, P]
        L.tt_vocab_intersection.restype = ctypes.c_int
        L.tt_tli_proposal.argtypes = [i32, i32, i32, P, P, P, i64, P, i64, P]
        L.tt_tli_proposal.restype = ctypes.c_int
        L.tt_verify_tli.argtypes = [i32, i32, i32, P, P, P, P, P, i64, P, P, i64, P, P, i32, P, P, P]
        L.tt_verify_tli.restype = ctypes.c_int
        L.tt_step_workspace_size.argtypes = [i32, i32, i32, i32, i32, i32, ctypes.POINTER(sz)]
        L.tt_step_workspace_size.restype = ctypes.c_int
        L.tt_step.argtypes = [VP, VP, i32, i32, i32, P, P, P, P, i32, i32, i32, P, i64, P, i64, P, P,
                              P, P, P, P, P, P, P, P, P, sz, P]
        L.tt_step.restype = ctypes.c_int
        _lib = L
    return _lib


def _torch():
    import torch

    return torch


def _stream_handle(stream):
    torch = _torch()
    s = torch.cuda.current_stream() if stream is None else stream
    return ctypes.c_void_p(s.cuda_stream)


def _ptr(t, dtype, name, allow_none=False):
    if t is None:
        if allow_none:
            return None
        raise ValueError(f"{name} is required")
    if not t.is_cuda:
        raise ValueError(f"{name} must be a device tensor")
    if t.dtype != dtype:
        raise ValueError(f"{name} must be {dtype}, got {t.dtype}")
    if not t.is_contiguous():
        raise ValueError(f"{name} must be contiguous")
    return ctypes.c_void_p(t.data_ptr())


def _check(status: int, where: str):
    if status != TT_OK:
        raise TTError(status, where)


class Vocab:
    """Token byte table on the device: token t is data[offsets[t]:offsets[t+1]]."""

    def __init__(self, data, offsets, max_token_bytes: int):
        torch = _torch()
        self.data = data if data.numel() else torch.zeros(1, dtype=torch.uint8, device=offsets.device)
        self.offsets = offsets
        self.n_tokens = int(offsets.numel()) - 1
        self.max_token_bytes = int(max_token_bytes)
        self._c = c_tt_vocab(_ptr(self.data, torch.uint8, "vocab bytes").value,
                             _ptr(self.offsets, torch.int32, "vocab offsets").value,
                             self.n_tokens, self.max_token_bytes)

    @classmethod
    def from_host(cls, data, offsets, max_token_bytes: int, device="cuda"):
        torch = _torch()
        return cls(torch.as_tensor(data, dtype=torch.uint8).to(device),
                   torch.as_tensor(offsets, dtype=torch.int32).to(device), max_token_bytes)


def path_capacity(draft_off_last: int, target_off_last: int) -> int:
    """int32 entries the path output needs: 2 * (sum K + sum M)."""
    return 2 * (int(draft_off_last) + int(target_off_last))


def align_workspace(n_pairs: int, max_k: int, max_m: int, w: int, max_token_bytes: int, device="cuda"):
    """A workspace for tt_align with these bounds (None when none is needed)."""
    torch = _torch()
    n = ctypes.c_size_t(0)
    _check(lib().tt_align_workspace_size(int(n_pairs), int(max_k), int(max_m), int(w), int(max_token_bytes),
                                         ctypes.byref(n)), "tt_align_workspace_size")
    return torch.empty(n.value, dtype=torch.uint8, device=device) if n.value else None


def align(vd: Vocab, vt: Vocab, draft_ids, draft_off, target_ids, target_off, w: int,
          max_k: int, max_m: int, n_path: int | None = None, out=None, workspace=None, stream=None):
    """tt_align.  Returns (cost, path_len, path, map) device tensors (int32).

    n_path: length of the path buffer (2 * (sum K + sum M)); read from the CSR
    offsets on the host if not given (one small device->host copy).
    workspace: from align_workspace(); allocated here when needed and not given.
    """
    torch = _torch()
    i32 = torch.int32
    n = int(draft_off.numel()) - 1
    dev = draft_off.device
    if workspace is None:
        workspace = align_workspace(n, max_k, max_m, w, max(vd.max_token_bytes, vt.max_token_bytes), dev)
    if out is None:
        if n_path is None:
            n_path = path_capacity(draft_off[-1].item(), target_off[-1].item())
        m_total = int(target_ids.numel())
        out = (torch.empty(n, dtype=i32, device=dev), torch.empty(n, dtype=i32, device=dev),
               torch.empty(max(1, n_path), dtype=i32, device=dev),
               torch.empty(max(1, m_total), dtype=i32, device=dev))
    cost, plen, path, mp = out
    di = draft_ids if draft_ids.numel() else torch.zeros(1, dtype=i32, device=dev)
    ti = target_ids if target_ids.numel() else torch.zeros(1, dtype=i32, device=dev)
    st = lib().tt_align(ctypes.byref(vd._c), ctypes.byref(vt._c), n,
                        _ptr(di, i32, "draft_ids"), _ptr(draft_off, i32, "draft_off"),
                        _ptr(ti, i32, "target_ids"), _ptr(target_off, i32, "target_off"),
                        int(max_k), int(max_m), int(w),
                        _ptr(cost, i32, "cost"), _ptr(plen, i32, "path_len"),
                        _ptr(path, i32, "path"), _ptr(mp, i32, "map"),
                        None if workspace is None else ctypes.c_void_p(workspace.data_ptr()),
                        0 if workspace is None else int(workspace.numel()), _stream_handle(stream))
    _check(st, "tt_align")
    return out


def transfer(v_d: int, draft_ids, draft_off, target_off, mp, draft_probs, out=None, stream=None):
    """tt_transfer.  Returns q (float32, one per target position)."""
    torch = _torch()
    i32 = torch.int32
    n = int(draft_off.numel()) - 1
    if draft_probs.dim() != 2 or draft_probs.stride(1) != 1:
        raise ValueError("draft_probs must be a 2-D row-major tensor")
    if draft_probs.dtype != torch.float32 or not draft_probs.is_cuda:
        raise ValueError("draft_probs must be a float32 device tensor")
    if out is None:
        out = torch.empty(max(1, int(mp.numel())), dtype=torch.float32, device=mp.device)
    st = lib().tt_transfer(n, int(v_d), _ptr(draft_ids, i32, "draft_ids"), _ptr(draft_off, i32, "draft_off"),
                           _ptr(target_off, i32, "target_off"), _ptr(mp, i32, "map"),
                           ctypes.c_void_p(draft_probs.data_ptr()),
                           int(draft_probs.stride(0)), _ptr(out, torch.float32, "q"), _stream_handle(stream))
    _check(st, "tt_transfer")
    return out


def verify_workspace(n_streams: int, v_t: int, device="cuda"):
    """A workspace for tt_verify (reusable by calls that do not overlap in time)."""
    torch = _torch()
    n = ctypes.c_size_t(0)
    _check(lib().tt_verify_workspace_size(int(n_streams), int(v_t), ctypes.byref(n)),
           "tt_verify_workspace_size")
    return torch.zeros(max(1, n.value), dtype=torch.uint8, device=device)


def verify(v_t: int, target_ids, target_off, q, target_probs, u_accept, u_sample, max_m: int,
           workspace=None, residual: bool = False, out=None, stream=None):
    """tt_verify.  Returns (n_accepted, out_token, residual or None)."""
    torch = _torch()
    i32, f32 = torch.int32, torch.float32
    n = int(target_off.numel()) - 1
    dev = target_off.device
    if target_probs.dim() != 2 or target_probs.stride(1) != 1:
        raise ValueError("target_probs must be a 2-D row-major tensor")
    if workspace is None:
        workspace = verify_workspace(n, v_t, dev)
    if out is None:
        out = (torch.empty(n, dtype=i32, device=dev), torch.empty(n, dtype=i32, device=dev),
               torch.zeros((n, target_probs.stride(0)), dtype=f32, device=dev) if residual else None)
    nacc, tok, res = out
    ti = target_ids if target_ids.numel() else torch.zeros(1, dtype=i32, device=dev)
    qq = q if q.numel() else torch.zeros(1, dtype=f32, device=dev)
    ua = u_accept if u_accept.numel() else torch.zeros(1, dtype=f32, device=dev)
    if target_probs.dtype != f32 or not target_probs.is_cuda:
        raise ValueError("target_probs must be a float32 device tensor")
    st = lib().tt_verify(n, int(v_t), _ptr(ti, i32, "target_ids"), _ptr(target_off, i32, "target_off"),
                         _ptr(qq, f32, "q"), ctypes.c_void_p(target_probs.data_ptr()),
                         int(target_probs.stride(0)), _ptr(ua, f32, "u_accept"),
                         _ptr(u_sample, f32, "u_sample"), int(max_m), _ptr(nacc, i32, "n_accepted"),
                         _ptr(tok, i32, "out_token"), _ptr(res, f32, "residual", allow_none=True),
                         ctypes.c_void_p(workspace.data_ptr()), int(workspace.numel()), _stream_handle(stream))
    _check(st, "tt_verify")
    return out


def verify_noalloc(v_t: int, target_ids, target_off, q, target_probs, u_accept, u_sample, max_m: int,
                   residual: bool = False, out=None, stream=None):
    """tt_verify_noalloc: tt_verify with the library's own scratch (no workspace).  Returns
    (n_accepted, out_token, residual or None); pass `out` to allocate nothing here either."""
    torch = _torch()
    i32, f32 = torch.int32, torch.float32
    n = int(target_off.numel()) - 1
    dev = target_off.device
    if target_probs.dim() != 2 or target_probs.stride(1) != 1 or target_probs.dtype != f32 or not target_probs.is_cuda:
        raise ValueError("target_probs must be a 2-D row-major float32 device tensor")
    if out is None:
        out = (torch.empty(n, dtype=i32, device=dev), torch.empty(n, dtype=i32, device=dev),
               torch.zeros((n, target_probs.stride(0)), dtype=f32, device=dev) if residual else None)
    nacc, tok, res = out
    st = lib().tt_verify_noalloc(n, int(v_t), _ptr(target_ids, i32, "target_ids"), _ptr(target_off, i32, "target_off"),
                                 _ptr(q, f32, "q"), ctypes.c_void_p(target_probs.data_ptr()),
                                 int(target_probs.stride(0)), _ptr(u_accept, f32, "u_accept"),
                                 _ptr(u_sample, f32, "u_sample"), int(max_m), _ptr(nacc, i32, "n_accepted"),
                                 _ptr(tok, i32, "out_token"), _ptr(res, f32, "residual", allow_none=True),
                                 _stream_handle(stream))
    _check(st, "tt_verify_noalloc")
    return out


def verify_dense(v: int, draft_ids, off, draft_probs, target_probs, u_accept, u_sample, max_m: int,
                 workspace=None, residual: bool = False, out=None, stream=None):
    """tt_verify_dense.  Returns (n_accepted, out_token, residual or None)."""
    torch = _torch()
    i32, f32 = torch.int32, torch.float32
    n = int(off.numel()) - 1
    dev = off.device
    for name, t in (("draft_probs", draft_probs), ("target_probs", target_probs)):
        if t.dim() != 2 or t.stride(1) != 1 or t.dtype != f32 or not t.is_cuda:
            raise ValueError(f"{name} must be a 2-D row-major float32 device tensor")
    if workspace is None:
        workspace = verify_workspace(n, v, dev)
    if out is None:
        out = (torch.empty(n, dtype=i32, device=dev), torch.empty(n, dtype=i32, device=dev),
               torch.zeros((n, target_probs.stride(0)), dtype=f32, device=dev) if residual else None)
    nacc, tok, res = out
    ids = draft_ids if draft_ids.numel() else torch.zeros(1, dtype=i32, device=dev)
    ua = u_accept if u_accept.numel() else torch.zeros(1, dtype=f32, device=dev)
    st = lib().tt_verify_dense(n, int(v), _ptr(ids, i32, "draft_ids"), _ptr(off, i32, "off"),
                               ctypes.c_void_p(draft_probs.data_ptr()), int(draft_probs.stride(0)),
                               ctypes.c_void_p(target_probs.data_ptr()), int(target_probs.stride(0)),
                               _ptr(ua, f32, "u_accept"), _ptr(u_sample, f32, "u_sample"), int(max_m),
                               _ptr(nacc, i32, "n_accepted"), _ptr(tok, i32, "out_token"),
                               _ptr(res, f32, "residual", allow_none=True),
                               ctypes.c_void_p(workspace.data_ptr()), int(workspace.numel()), _stream_handle(stream))
    _check(st, "tt_verify_dense")
    return out


def verify_logits(v_t: int, target_ids, target_off, q, target_logits, inv_temperature, u_accept, u_sample,
                  max_m: int, lse=None, out=None, stream=None):
    """tt_verify_logits: target_logits is a 2-D row-major device tensor of bf16 (or its int16 / uint16
    bit patterns); inv_temperature float32 [n_streams]; lse optional float32 [rows], the rows'
    log-sum-exp of logit * inv_temperature.  Returns (n_accepted, out_token)."""
    torch = _torch()
    i32, f32 = torch.int32, torch.float32
    n = int(target_off.numel()) - 1
    dev = target_off.device
    if target_logits.dim() != 2 or target_logits.stride(1) != 1 or not target_logits.is_cuda or \
            target_logits.element_size() != 2:
        raise ValueError("target_logits must be a 2-D row-major 16-bit device tensor")
    if out is None:
        out = (torch.empty(n, dtype=i32, device=dev), torch.empty(n, dtype=i32, device=dev))
    nacc, tok = out
    ids = target_ids if target_ids.numel() else torch.zeros(1, dtype=i32, device=dev)
    qq = q if q.numel() else torch.zeros(1, dtype=f32, device=dev)
    ua = u_accept if u_accept.numel() else torch.zeros(1, dtype=f32, device=dev)
    st = lib().tt_verify_logits(n, int(v_t), _ptr(ids, i32, "target_ids"), _ptr(target_off, i32, "target_off"),
                                _ptr(qq, f32, "q"), ctypes.c_void_p(target_logits.data_ptr()),
                                int(target_logits.stride(0)), _ptr(inv_temperature, f32, "inv_temperature"),
                                _ptr(lse, f32, "lse", allow_none=True), _ptr(ua, f32, "u_accept"), _ptr(u_sample, f32, "u_sample"), int(max_m),
                                _ptr(nacc, i32, "n_accepted"), _ptr(tok, i32, "out_token"), _stream_handle(stream))
    _check(st, "tt_verify_logits")
    return out


def delta_histogram(draft_off, target_off, path_len, path, n_bins: int, out=None, stream=None):
    """tt_delta_histogram: int32 counts of |i - j| over every aligned pair's path cells (last bin
    collects |i - j| >= n_bins - 1)."""
    torch = _torch()
    i32 = torch.int32
    n = int(draft_off.numel()) - 1
    hist = torch.empty(int(n_bins), dtype=i32, device=draft_off.device) if out is None else out
    st = lib().tt_delta_histogram(n, _ptr(draft_off, i32, "draft_off"), _ptr(target_off, i32, "target_off"),
                                  _ptr(path_len, i32, "path_len"), _ptr(path, i32, "path"), int(n_bins),
                                  _ptr(hist, i32, "hist"), _stream_handle(stream))
    _check(st, "tt_delta_histogram")
    return hist


def delta_quantile(hist, num: int = 9, den: int = 10, out=None, stream=None):
    """tt_delta_quantile: (int32 device tensor of one element) the smallest deviation d at which
    the cumulative counts of `hist` reach num/den of their total (App. K)."""
    torch = _torch()
    i32 = torch.int32
    d = torch.empty(1, dtype=i32, device=hist.device) if out is None else out
    st = lib().tt_delta_quantile(_ptr(hist, i32, "hist"), int(hist.numel()), int(num), int(den), _ptr(d, i32, "d_out"),
                                 _stream_handle(stream))
    _check(st, "tt_delta_quantile")
    return d


def w_at_quantile(hist, num: int = 9, den: int = 10) -> int:
    """App. K's bound on w from a device histogram: tt_delta_quantile's result as a host int."""
    return int(delta_quantile(hist, num, den).item())


def token_index(v: Vocab, stream=None):
    """tt_token_index_build: the longest-match index of a token table (a uint8 device tensor)."""
    torch = _torch()
    n = ctypes.c_size_t(0)
    _check(lib().tt_token_index_size(v.n_tokens, ctypes.byref(n)), "tt_token_index_size")
    idx = torch.empty(n.value, dtype=torch.uint8, device=v.offsets.device)
    _check(lib().tt_token_index_build(ctypes.byref(v._c), ctypes.c_void_p(idx.data_ptr()), n.value,
                                      _stream_handle(stream)), "tt_token_index_build")
    return idx


def retokenize(vd: Vocab, vt: Vocab, vt_index, draft_ids, draft_off, max_bytes: int, max_m: int,
               out=None, workspace=None, stream=None):
    """tt_retokenize.  Returns (target_ids, target_off) device tensors; target_ids has room for
    n_streams * max_m ids (the first target_off[-1] are valid)."""
    torch = _torch()
    i32 = torch.int32
    n = int(draft_off.numel()) - 1
    dev = draft_off.device
    if workspace is None:
        nb = ctypes.c_size_t(0)
        _check(lib().tt_retokenize_workspace_size(n, int(max_m), ctypes.byref(nb)), "tt_retokenize_workspace_size")
        workspace = torch.empty(max(1, nb.value), dtype=torch.uint8, device=dev)
    if out is None:
        out = (torch.empty(max(1, n * int(max_m)), dtype=i32, device=dev), torch.empty(n + 1, dtype=i32, device=dev))
    tids, toff = out
    ids = draft_ids if draft_ids.numel() else torch.zeros(1, dtype=i32, device=dev)
    st = lib().tt_retokenize(ctypes.byref(vd._c), ctypes.byref(vt._c), ctypes.c_void_p(vt_index.data_ptr()),
                             int(vt_index.numel()), n, _ptr(ids, i32, "draft_ids"), _ptr(draft_off, i32, "draft_off"),
                             int(max_bytes), int(max_m), _ptr(tids, i32, "target_ids"),
                             _ptr(toff, i32, "target_off"), ctypes.c_void_p(workspace.data_ptr()),
                             int(workspace.numel()), _stream_handle(stream))
    _check(st, "tt_retokenize")
    return out


def vocab_intersection(vd: Vocab, vd_index, vt: Vocab, vt_index, out=None, stream=None):
    """tt_vocab_intersection (App. D Alg. 3's T ∩ D by byte strings).  Returns (d2t, t2d) int32
    device tensors of vd.n_tokens and vt.n_tokens entries (-1 outside the intersection)."""
    torch = _torch()
    i32 = torch.int32
    dev = vd.offsets.device
    if out is None:
        out = (torch.empty(vd.n_tokens, dtype=i32, device=dev), torch.empty(vt.n_tokens, dtype=i32, device=dev))
    d2t, t2d = out
    st = lib().tt_vocab_intersection(ctypes.byref(vd._c), ctypes.c_void_p(vd_index.data_ptr()), int(vd_index.numel()),
                                     ctypes.byref(vt._c), ctypes.c_void_p(vt_index.data_ptr()), int(vt_index.numel()),
                                     _ptr(d2t, i32, "d2t"), _ptr(t2d, i32, "t2d"), _stream_handle(stream))
    _check(st, "tt_vocab_intersection")
    return out


def tli_proposal(d2t, t2d, draft_probs, v_d: int | None = None, out=None, stream=None):
    """tt_tli_proposal: q' rows over the target vocabulary (App. D Alg. 3) from draft rows
    [n, >= V_d] float32.  Returns out [n, V_t] (or the given tensor, any row stride >= V_t)."""
    torch = _torch()
    i32, f32 = torch.int32, torch.float32
    v_d = int(d2t.numel()) if v_d is None else int(v_d)
    v_t = int(t2d.numel())
    if draft_probs.dim() != 2 or draft_probs.stride(1) != 1 or draft_probs.dtype != f32 or not draft_probs.is_cuda:
        raise ValueError("draft_probs must be a 2-D row-major float32 device tensor")
    n = int(draft_probs.shape[0])
    if out is None:
        out = torch.empty((n, v_t), dtype=f32, device=draft_probs.device)
    if out.dim() != 2 or out.stride(1) != 1 or out.dtype != f32 or not out.is_cuda:
        raise ValueError("out must be a 2-D row-major float32 device tensor")
    st = lib().tt_tli_proposal(n, v_d, v_t, _ptr(d2t, i32, "d2t"), _ptr(t2d, i32, "t2d"),
                               ctypes.c_void_p(draft_probs.data_ptr()), int(draft_probs.stride(0)),
                               ctypes.c_void_p(out.data_ptr()), int(out.stride(0)), _stream_handle(stream))
    _check(st, "tt_tli_proposal")
    return out


def verify_tli(d2t, t2d, target_ids, target_off, draft_probs, target_probs, u_accept, u_sample, max_m: int,
               draft_mass=None, v_d: int | None = None, out=None, stream=None):
    """tt_verify_tli: standard speculative sampling with the TLI proposal formed on the fly from
    draft rows [sum M, >= V_d] float32 (row target_off[b] + j for position j) against target rows
    [rows, >= V_t]; draft_mass optional float32 [sum M], the drafter's S_j.  Returns
    (n_accepted, out_token)."""
    torch = _torch()
    i32, f32 = torch.int32, torch.float32
    v_d = int(d2t.numel()) if v_d is None else int(v_d)
    v_t = int(t2d.numel())
    n = int(target_off.numel()) - 1
    dev = target_off.device
    for name, t in (("draft_probs", draft_probs), ("target_probs", target_probs)):
        if t.dim() != 2 or t.stride(1) != 1 or t.dtype != f32 or not t.is_cuda:
            raise ValueError(f"{name} must be a 2-D row-major float32 device tensor")
    if out is None:
        out = (torch.empty(n, dtype=i32, device=dev), torch.empty(n, dtype=i32, device=dev))
    nacc, tok = out
    ids = target_ids if target_ids.numel() else torch.zeros(1, dtype=i32, device=dev)
    ua = u_accept if u_accept.numel() else torch.zeros(1, dtype=f32, device=dev)
    st = lib().tt_verify_tli(n, v_d, v_t, _ptr(d2t, i32, "d2t"), _ptr(t2d, i32, "t2d"), _ptr(ids, i32, "target_ids"),
                             _ptr(target_off, i32, "target_off"), ctypes.c_void_p(draft_probs.data_ptr()),
                             int(draft_probs.stride(0)), _ptr(draft_mass, f32, "draft_mass", allow_none=True),
                             ctypes.c_void_p(target_probs.data_ptr()), int(target_probs.stride(0)),
                             _ptr(ua, f32, "u_accept"), _ptr(u_sample, f32, "u_sample"), int(max_m),
                             _ptr(nacc, i32, "n_accepted"), _ptr(tok, i32, "out_token"), _stream_handle(stream))
    _check(st, "tt_verify_tli")
    return out


def step_workspace(n_streams: int, v_t: int, max_k: int, max_m: int, w: int, max_token_bytes: int,
                   device="cuda"):
    """A workspace for tt_step (reusable by calls that do not overlap in time)."""
    torch = _torch()
    n = ctypes.c_size_t(0)
    _check(lib().tt_step_workspace_size(int(n_streams), int(v_t), int(max_k), int(max_m), int(w),
                                        int(max_token_bytes), ctypes.byref(n)), "tt_step_workspace_size")
    return torch.empty(max(1, n.value), dtype=torch.uint8, device=device)


def step(vd: Vocab, vt: Vocab, v_d: int, v_t: int, draft_ids, draft_off, target_ids, target_off, w: int,
         max_k: int, max_m: int, draft_probs, target_probs, u_accept, u_sample, n_path: int | None = None,
         workspace=None, residual: bool = False, out=None, stream=None):
    """tt_step (align + transfer + verify).  Returns
    (cost, path_len, path, map, q, n_accepted, out_token, residual or None)."""
    torch = _torch()
    i32, f32 = torch.int32, torch.float32
    n = int(draft_off.numel()) - 1
    dev = draft_off.device
    for name, t in (("draft_probs", draft_probs), ("target_probs", target_probs)):
        if t.dim() != 2 or t.stride(1) != 1 or t.dtype != f32 or not t.is_cuda:
            raise ValueError(name + " must be a 2-D row-major float32 device tensor")
    if workspace is None:
        workspace = step_workspace(n, v_t, max_k, max_m, w, max(vd.max_token_bytes, vt.max_token_bytes), dev)
    if out is None:
        if n_path is None:
            n_path = path_capacity(draft_off[-1].item(), target_off[-1].item())
        m_total = max(1, int(target_ids.numel()))
        out = (torch.empty(n, dtype=i32, device=dev), torch.empty(n, dtype=i32, device=dev),
               torch.empty(max(1, n_path), dtype=i32, device=dev), torch.empty(m_total, dtype=i32, device=dev),
               torch.empty(m_total, dtype=f32, device=dev), torch.empty(n, dtype=i32, device=dev),
               torch.empty(n, dtype=i32, device=dev),
               torch.zeros((n, target_probs.stride(0)), dtype=f32, device=dev) if residual else None)
    cost, plen, path, mp, q, nacc, tok, res = out
    di = draft_ids if draft_ids.numel() else torch.zeros(1, dtype=i32, device=dev)
    ti = target_ids if target_ids.numel() else torch.zeros(1, dtype=i32, device=dev)
    ua = u_accept if u_accept.numel() else torch.zeros(1, dtype=f32, device=dev)
    st = lib().tt_step(ctypes.byref(vd._c), ctypes.byref(vt._c), n, int(v_d), int(v_t),
                       _ptr(di, i32, "draft_ids"), _ptr(draft_off, i32, "draft_off"),
                       _ptr(ti, i32, "target_ids"), _ptr(target_off, i32, "target_off"),
                       int(max_k), int(max_m), int(w),
                       ctypes.c_void_p(draft_probs.data_ptr()), int(draft_probs.stride(0)),
                       ctypes.c_void_p(target_probs.data_ptr()), int(target_probs.stride(0)),
                       _ptr(ua, f32, "u_accept"), _ptr(u_sample, f32, "u_sample"),
                       _ptr(cost, i32, "cost"), _ptr(plen, i32, "path_len"), _ptr(path, i32, "path"),
                       _ptr(mp, i32, "map"), _ptr(q, f32, "q"), _ptr(nacc, i32, "n_accepted"),
                       _ptr(tok, i32, "out_token"), _ptr(res, f32, "residual", allow_none=True),
                       ctypes.c_void_p(workspace.data_ptr()), int(workspace.numel()), _stream_handle(stream))
    _check(st, "tt_step")
    return out
