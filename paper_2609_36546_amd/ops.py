"""Thin ctypes binding of libipdv.so (argument marshalling only).

Every function takes device tensors, checks dtype / device / contiguity /
shape, passes raw pointers and the current HIP stream to the C ABI of the
same name, and raises RuntimeError with the library's message on a non-OK
status.  All arithmetic runs in the library's gfx950 kernels; there is no
other path.  Outputs and workspaces can be passed in (to keep a call free of
allocations) or are allocated here with torch.
"""
from __future__ import annotations

import ctypes
import math
import os
from typing import Optional

import torch

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libipdv.so")

IPDV_F32 = 0
IPDV_BF16 = 1
MAX_K = 32

_lib = None


class IpdvError(RuntimeError):
    def __init__(self, func: str, status: int, msg: str):
        super().__init__(f"{func} failed with status {status}: {msg}")
        self.status = status


def lib() -> ctypes.CDLL:
    """The loaded library (raises if it has not been built)."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise RuntimeError(f"{LIB_PATH} is missing: build it with "
                               "`python -m paper_2609_36546_amd.build`")
        L = ctypes.CDLL(LIB_PATH)
        vp, i32p, u8p, f32p = ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p
        ci, cf, cs = ctypes.c_int, ctypes.c_float, ctypes.c_size_t
        L.ipdv_attn_workspace_size.argtypes = [ci] * 7
        L.ipdv_attn_workspace_size.restype = cs
        L.verify_attn_paged.argtypes = [vp, vp, vp, vp, vp, i32p, ci, i32p, i32p, i32p, ci, ci, vp,
                                        ci, ci, ci, ci, ci, cf, ci, vp, cs, vp]
        L.verify_attn_paged.restype = ci
        L.ipdv_lmhead_workspace_size.argtypes = [ci] * 4
        L.ipdv_lmhead_workspace_size.restype = cs
        L.ipdv_workspace_size.argtypes = [ci, ctypes.POINTER(ctypes.c_int32), ci]
        L.ipdv_workspace_size.restype = cs
        L.ipdv_check_page_table.argtypes = [vp, ci, ci, vp, vp, vp, ci, ci, ci, ci,
                                            ctypes.POINTER(ctypes.c_int32)]
        L.ipdv_check_page_table.restype = ci
        L.verify_attn_paged_noalloc.argtypes = [vp, vp, vp, vp, vp, i32p, ci, i32p, i32p, i32p, ci,
                                                ci, vp, ci, ci, ci, ci, ci, cf, ci, vp]
        L.verify_attn_paged_noalloc.restype = ci
        L.lmhead_logsoftmax_verify.argtypes = [vp, vp, i32p, i32p, ci, ci, ci, ci, f32p, f32p, i32p,
                                               i32p, f32p, f32p, ci, vp, cs, vp]
        L.lmhead_logsoftmax_verify.restype = ci
        L.accept_scan.argtypes = [i32p, i32p, i32p, ci, u8p, i32p, i32p, ctypes.c_int32,
                                  ctypes.c_int32, ci, i32p, i32p, u8p, u8p, i32p, u8p, vp]
        L.accept_scan.restype = ci
        L.accept_scan_rule.argtypes = [i32p, i32p, i32p, ci, u8p, i32p, i32p, ctypes.c_int32,
                                       ctypes.c_int32, ci, ci, ci, f32p, ctypes.c_float,
                                       ctypes.c_float, i32p, i32p, u8p, u8p, i32p, u8p, vp]
        L.accept_scan_rule.restype = ci
        L.lmhead_sample.argtypes = [vp, vp, ci, ci, ci, ci, vp, cs, f32p, i32p, ci, vp]
        L.lmhead_sample.restype = ci
        L.ipdv_lmhead_packed_w_size.argtypes = [ci, ci]
        L.ipdv_lmhead_packed_w_size.restype = cs
        L.lmhead_pack_w.argtypes = [vp, ci, ci, vp, ci, vp]
        L.lmhead_pack_w.restype = ci
        L.lmhead_logp_gather.argtypes = [vp, vp, ci, ci, ci, f32p, i32p, ci, f32p, ci, vp]
        L.lmhead_logp_gather.restype = ci
        L.source_split_kl.argtypes = [ci, ci, i32p, f32p, f32p, i32p, f32p, f32p, u8p, ci, ci,
                                      f32p, f32p, f32p, f32p, i32p, ci, f32p, f32p, vp]
        L.source_split_kl.restype = ci
        L.sample_takeover.argtypes = [vp, vp, ci, ci, ci, ci, vp, cs, i32p, ci, i32p, u8p, i32p,
                                      i32p, f32p, ctypes.c_int32, i32p, u8p, ci, vp]
        L.sample_takeover.restype = ci
        L.ipdv_trace_events.argtypes = [ctypes.c_void_p, ci]
        L.ipdv_trace_events.restype = ci
        L.ipdv_trace_count.restype = ci
        L.ipdv_last_error.restype = ctypes.c_char_p
        L.ipdv_version.restype = ctypes.c_char_p
        _lib = L
    return _lib


def _check(func: str, status: int):
    if status != 0:
        raise IpdvError(func, status, lib().ipdv_last_error().decode())


def _ptr(t: Optional[torch.Tensor]):
    return None if t is None else ctypes.c_void_p(t.data_ptr())


def _stream(device: torch.device):
    return ctypes.c_void_p(torch.cuda.current_stream(device).cuda_stream)


def _need(t: torch.Tensor, name: str, dtype=None, device=None, ndim=None):
    if not isinstance(t, torch.Tensor):
        raise TypeError(f"{name} must be a torch.Tensor")
    if device is not None and t.device != device:
        raise ValueError(f"{name} must be on {device} (is on {t.device})")
    if t.device.type != "cuda":
        raise ValueError(f"{name} must be a GPU tensor")
    if dtype is not None and t.dtype != dtype:
        raise ValueError(f"{name} must be {dtype} (is {t.dtype})")
    if ndim is not None and t.dim() != ndim:
        raise ValueError(f"{name} must have {ndim} dims (has {t.dim()})")
    if not t.is_contiguous():
        raise ValueError(f"{name} must be contiguous")


def _dtype_code(dt: torch.dtype) -> int:
    if dt == torch.bfloat16:
        return IPDV_BF16
    if dt == torch.float32:
        return IPDV_F32
    raise ValueError(f"unsupported dtype {dt}")


def trace_events(events) -> None:
    """Bracket every kernel the library launches with these torch.cuda.Event
    objects (in order; see ipdv_trace_events).  None turns tracing off."""
    global _trace_keep
    if not events:
        lib().ipdv_trace_events(None, 0)
        _trace_keep = None
        return
    for e in events:            # torch creates the HIP event on first record
        if e.cuda_event == 0:
            e.record()
    arr = (ctypes.c_void_p * len(events))(*[e.cuda_event for e in events])
    _trace_keep = arr
    lib().ipdv_trace_events(ctypes.cast(arr, ctypes.c_void_p), len(events))


def trace_count() -> int:
    return int(lib().ipdv_trace_count())


_trace_keep = None


def version() -> str:
    return lib().ipdv_version().decode()


# ---------------------------------------------------------------------------

def attn_workspace_size(n_seq, Hq, Hkv, D, max_q, max_pages, page_size) -> int:
    return int(lib().ipdv_attn_workspace_size(n_seq, Hq, Hkv, D, max_q, max_pages, page_size))


def check_page_table(page_table, ctx_lens, cu_q, max_q: int, page_size: int, num_pages: int,
                     seq_ids=None, n_seq: Optional[int] = None):
    """ipdv_check_page_table on host copies of the arrays (tensors on any
    device, or numpy arrays).  Raises IpdvError naming the first contract
    violation; returns None when the table is valid."""
    import numpy as np

    def host(x):
        if isinstance(x, torch.Tensor):
            x = x.detach().cpu().numpy()
        return np.ascontiguousarray(np.asarray(x, np.int32))

    pt, ctx, cu = host(page_table), host(ctx_lens), host(cu_q)
    sid = None if seq_ids is None else host(seq_ids)
    B = ctx.shape[0]
    if pt.ndim != 2 or pt.shape[0] != B or cu.shape[0] != B + 1:
        raise ValueError("page_table must be [B, maxp] and cu_q [B+1]")
    if n_seq is None:
        n_seq = B if sid is None else sid.shape[0]
    p = lambda a: None if a is None else a.ctypes.data_as(ctypes.c_void_p)
    bad = ctypes.c_int32(-1)
    st = lib().ipdv_check_page_table(p(pt), B, pt.shape[1], p(ctx), p(cu), p(sid), n_seq, max_q,
                                     page_size, num_pages, ctypes.byref(bad))
    _check("ipdv_check_page_table", st)


def verify_attn_paged(q, k_new, v_new, k_cache, v_cache, page_table, ctx_lens, cu_q,
                      max_q: int, seq_ids=None, n_seq: Optional[int] = None,
                      scale: Optional[float] = None, out=None, workspace=None,
                      validate: bool = False):
    """Append the window to the paged cache and attend (see include/ipdv.h).

    q [T,Hq,D], k_new/v_new [T,Hkv,D], k_cache [P,Hkv,D/32,ps,32], v_cache [P,Hkv,D,ps]
    (bf16 or fp32), page_table [B,maxp] int32, ctx_lens [B] int32, cu_q [B+1]
    int32, seq_ids [n] int32 or None.  Returns out [T,Hq,D].  validate=True
    first runs check_page_table on host copies (a device-to-host copy and a
    synchronisation; for debugging).
    """
    dev = q.device
    dt = q.dtype
    _need(q, "q", dt, dev, 3)
    T, Hq, D = q.shape
    _need(k_new, "k_new", dt, dev, 3)
    _need(v_new, "v_new", dt, dev, 3)
    Hkv = k_new.shape[1]
    _need(k_cache, "k_cache", dt, dev, 5)
    _need(v_cache, "v_cache", dt, dev, 4)
    P, ps = k_cache.shape[0], k_cache.shape[3]
    if tuple(k_cache.shape) != (P, Hkv, D // 32, ps, 32) or tuple(v_cache.shape) != (P, Hkv, D, ps):
        raise ValueError("k_cache must be [P,Hkv,D/32,ps,32] and v_cache [P,Hkv,D,ps]")
    if tuple(k_new.shape) != (T, Hkv, D) or tuple(v_new.shape) != (T, Hkv, D):
        raise ValueError("k_new / v_new must be [T,Hkv,D]")
    _need(page_table, "page_table", torch.int32, dev, 2)
    _need(ctx_lens, "ctx_lens", torch.int32, dev, 1)
    _need(cu_q, "cu_q", torch.int32, dev, 1)
    B = ctx_lens.shape[0]
    if cu_q.shape[0] != B + 1 or page_table.shape[0] != B:
        raise ValueError("cu_q must be [B+1] and page_table [B, maxp]")
    if seq_ids is not None:
        _need(seq_ids, "seq_ids", torch.int32, dev, 1)
        n_seq = seq_ids.shape[0] if n_seq is None else n_seq
    elif n_seq is None:
        n_seq = B
    if scale is None:
        scale = 1.0 / math.sqrt(D)
    if out is None:
        out = torch.empty_like(q)
    else:
        _need(out, "out", dt, dev, 3)
    maxp = page_table.shape[1]
    if validate:
        check_page_table(page_table, ctx_lens, cu_q, max_q, ps, P, seq_ids=seq_ids, n_seq=n_seq)
    need = attn_workspace_size(n_seq, Hq, Hkv, D, max_q, maxp, ps)
    if workspace is None:
        workspace = torch.empty(max(need, 1), dtype=torch.uint8, device=dev)
    st = lib().verify_attn_paged(
        _ptr(q), _ptr(k_new), _ptr(v_new), _ptr(k_cache), _ptr(v_cache), _ptr(page_table),
        maxp, _ptr(ctx_lens), _ptr(cu_q), _ptr(seq_ids), n_seq, max_q, _ptr(out),
        Hq, Hkv, D, ps, P, float(scale), _dtype_code(dt), _ptr(workspace),
        workspace.numel() * workspace.element_size(), _stream(dev))
    _check("verify_attn_paged", st)
    return out


NOALLOC_SCRATCH_BYTES = 128 << 20


def verify_attn_paged_noalloc(q, k_new, v_new, k_cache, v_cache, page_table, ctx_lens, cu_q,
                              max_q: int, seq_ids=None, n_seq: Optional[int] = None,
                              scale: Optional[float] = None, out=None):
    """verify_attn_paged_noalloc (see include/ipdv.h): verify_attn_paged with
    its split-KV partials in the library's per-device scratch.  Allocates
    nothing when `out` is given."""
    dev = q.device
    dt = q.dtype
    _need(q, "q", dt, dev, 3)
    T, Hq, D = q.shape
    _need(k_new, "k_new", dt, dev, 3)
    _need(v_new, "v_new", dt, dev, 3)
    Hkv = k_new.shape[1]
    _need(k_cache, "k_cache", dt, dev, 5)
    _need(v_cache, "v_cache", dt, dev, 4)
    P, ps = k_cache.shape[0], k_cache.shape[3]
    if tuple(k_cache.shape) != (P, Hkv, D // 32, ps, 32) or tuple(v_cache.shape) != (P, Hkv, D, ps):
        raise ValueError("k_cache must be [P,Hkv,D/32,ps,32] and v_cache [P,Hkv,D,ps]")
    if tuple(k_new.shape) != (T, Hkv, D) or tuple(v_new.shape) != (T, Hkv, D):
        raise ValueError("k_new / v_new must be [T,Hkv,D]")
    _need(page_table, "page_table", torch.int32, dev, 2)
    _need(ctx_lens, "ctx_lens", torch.int32, dev, 1)
    _need(cu_q, "cu_q", torch.int32, dev, 1)
    B = ctx_lens.shape[0]
    if cu_q.shape[0] != B + 1 or page_table.shape[0] != B:
        raise ValueError("cu_q must be [B+1] and page_table [B, maxp]")
    if seq_ids is not None:
        _need(seq_ids, "seq_ids", torch.int32, dev, 1)
        n_seq = seq_ids.shape[0] if n_seq is None else n_seq
    elif n_seq is None:
        n_seq = B
    if scale is None:
        scale = 1.0 / math.sqrt(D)
    if out is None:
        out = torch.empty_like(q)
    else:
        _need(out, "out", dt, dev, 3)
    st = lib().verify_attn_paged_noalloc(
        _ptr(q), _ptr(k_new), _ptr(v_new), _ptr(k_cache), _ptr(v_cache), _ptr(page_table),
        page_table.shape[1], _ptr(ctx_lens), _ptr(cu_q), _ptr(seq_ids), n_seq, max_q, _ptr(out),
        Hq, Hkv, D, ps, P, float(scale), _dtype_code(dt), _stream(dev))
    _check("verify_attn_paged_noalloc", st)
    return out


def lmhead_workspace_size(M, Hd, V, K) -> int:
    return int(lib().ipdv_lmhead_workspace_size(M, Hd, V, K))


W_TILED = 0x10


class PackedW:
    """The LM-head weight in the tiled layout written by lmhead_pack_w (see
    include/ipdv.h): ``data`` is the flat bf16 buffer; ``V`` and ``Hd`` the
    logical shape.  Accepted wherever a row-major W is."""

    def __init__(self, data, V: int, Hd: int):
        self.data, self.V, self.Hd = data, int(V), int(Hd)

    @property
    def device(self):
        return self.data.device

    @property
    def dtype(self):
        return self.data.dtype


def lmhead_pack_w(W) -> PackedW:
    """Repack a row-major bf16 W [V, Hd] into the tiled layout (one launch)."""
    dev = W.device
    _need(W, "W", torch.bfloat16, dev, 2)
    V, Hd = W.shape
    n = int(lib().ipdv_lmhead_packed_w_size(V, Hd))
    if n == 0:
        raise ValueError(f"unsupported LM-head shape V={V} Hd={Hd}")
    data = torch.empty(n // 2, dtype=torch.bfloat16, device=dev)
    st = lib().lmhead_pack_w(_ptr(W), V, Hd, _ptr(data), _dtype_code(torch.bfloat16), _stream(dev))
    _check("lmhead_pack_w", st)
    return PackedW(data, V, Hd)


def _w_arg(W, dt, dev, Hd):
    """(pointer, V, dtype code) for a row-major W [V, Hd] or a PackedW."""
    if isinstance(W, PackedW):
        if W.dtype != torch.bfloat16 or dt != torch.bfloat16:
            raise ValueError("a packed W needs bf16 hidden rows and weights")
        if W.device != dev:
            raise ValueError(f"W must be on {dev}")
        if W.Hd != Hd:
            raise ValueError("packed W has another hidden size")
        return _ptr(W.data), W.V, _dtype_code(dt) | W_TILED
    _need(W, "W", dt, dev, 2)
    if W.shape[1] != Hd:
        raise ValueError("W must be [V, Hd]")
    return _ptr(W), W.shape[0], _dtype_code(dt)


def lmhead_logsoftmax_verify(hidden, W, prop_tok, K: int, out_rows=None, n_out_rows=None,
                             with_entropy: bool = True, outs=None, workspace=None):
    """Verifier log-softmax outputs for each row (see include/ipdv.h).

    hidden [M,Hd], W [V,Hd] (bf16 or fp32), prop_tok [M] int32, out_rows [M]
    int32 or None.  Returns dict lse, logp_prop, argmax, topk_idx, topk_logp,
    entropy (rows = n_out_rows if out_rows is given, else M).
    """
    dev = hidden.device
    dt = hidden.dtype
    _need(hidden, "hidden", dt, dev, 2)
    M, Hd = hidden.shape
    w_ptr, V, code = _w_arg(W, dt, dev, Hd)
    _need(prop_tok, "prop_tok", torch.int32, dev, 1)
    if prop_tok.shape[0] != M:
        raise ValueError("prop_tok must be [M]")
    if out_rows is not None:
        _need(out_rows, "out_rows", torch.int32, dev, 1)
        R = int(n_out_rows)
    else:
        R = M
    if outs is None:
        outs = {
            "lse": torch.empty(R, dtype=torch.float32, device=dev),
            "logp_prop": torch.empty(R, dtype=torch.float32, device=dev),
            "argmax": torch.empty(R, dtype=torch.int32, device=dev),
            "topk_idx": torch.empty(R, K, dtype=torch.int32, device=dev),
            "topk_logp": torch.empty(R, K, dtype=torch.float32, device=dev),
            "entropy": torch.empty(R, dtype=torch.float32, device=dev) if with_entropy else None,
        }
    need = lmhead_workspace_size(M, Hd, V, K)
    if workspace is None:
        workspace = torch.empty(max(need, 1), dtype=torch.uint8, device=dev)
    st = lib().lmhead_logsoftmax_verify(
        _ptr(hidden), w_ptr, _ptr(prop_tok), _ptr(out_rows), M, Hd, V, K,
        _ptr(outs["lse"]), _ptr(outs["logp_prop"]), _ptr(outs["argmax"]), _ptr(outs["topk_idx"]),
        _ptr(outs["topk_logp"]), _ptr(outs["entropy"]), code, _ptr(workspace),
        workspace.numel() * workspace.element_size(), _stream(dev))
    _check("lmhead_logsoftmax_verify", st)
    return outs


TAKE_COVERAGE, TAKE_ENTROPY = 0, 1
HAND_COVERAGE, HAND_FIXED_ONE, HAND_ENTROPY = 0, 1, 2


def _scan_args(cu_q, prop_tok, topk_idx, K, driver, ctx_lens, seq_lens, ent, uses_ent, outs):
    """Checks the verdict inputs and allocates the outputs when none are given."""
    dev = cu_q.device
    _need(cu_q, "cu_q", torch.int32, dev, 1)
    B = cu_q.shape[0] - 1
    _need(prop_tok, "prop_tok", torch.int32, dev, 1)
    T = prop_tok.shape[0]
    if uses_ent:
        _need(ent, "ent", torch.float32, dev, 1)
        if ent.shape[0] != T:
            raise ValueError("ent must be [T]")
    if K > 0 and topk_idx is not None:
        _need(topk_idx, "topk_idx", torch.int32, dev, 2)
        if topk_idx.shape[0] != T or topk_idx.shape[1] != K:
            raise ValueError("topk_idx must be [T, K]")
    _need(driver, "driver", torch.uint8, dev, 1)
    _need(ctx_lens, "ctx_lens", torch.int32, dev, 1)
    _need(seq_lens, "seq_lens", torch.int32, dev, 1)
    if outs is None:
        outs = {
            "n_acc": torch.empty(B, dtype=torch.int32, device=dev),
            "event_row": torch.empty(B, dtype=torch.int32, device=dev),
            "next_driver": torch.empty(B, dtype=torch.uint8, device=dev),
            "finished": torch.empty(B, dtype=torch.uint8, device=dev),
            "new_cache_len": torch.empty(B, dtype=torch.int32, device=dev),
            "src": torch.empty(T, dtype=torch.uint8, device=dev),
        }
    tk = _ptr(topk_idx) if (K > 0 and topk_idx is not None) else None
    return dev, B, tk, outs


def _scan_outs(outs):
    return (_ptr(outs["n_acc"]), _ptr(outs["event_row"]), _ptr(outs["next_driver"]),
            _ptr(outs["finished"]), _ptr(outs["new_cache_len"]), _ptr(outs["src"]))


def accept_scan(cu_q, prop_tok, topk_idx, K: int, driver, ctx_lens, seq_lens, eos_id: int,
                max_len: int, outs=None):
    """Verdict for each sequence's window (see include/ipdv.h).  Returns dict
    n_acc, event_row, next_driver, finished, new_cache_len, src."""
    dev, B, tk, outs = _scan_args(cu_q, prop_tok, topk_idx, K, driver, ctx_lens, seq_lens, None,
                                  False, outs)
    st = lib().accept_scan(_ptr(cu_q), _ptr(prop_tok), tk, K, _ptr(driver), _ptr(ctx_lens),
                           _ptr(seq_lens), int(eos_id), int(max_len), B, *_scan_outs(outs),
                           _stream(dev))
    _check("accept_scan", st)
    return outs


def accept_scan_rule(cu_q, prop_tok, topk_idx, K: int, driver, ctx_lens, seq_lens, eos_id: int,
                     max_len: int, take_rule: int = TAKE_COVERAGE, hand_rule: int = HAND_COVERAGE,
                     ent=None, tau_take: float = 0.0, tau_hand: float = 0.0, outs=None):
    """Verdict with the takeover / handback rule variants (see
    include/ipdv.h, accept_scan_rule).  ``ent`` is a [T] float32 entropy per
    row, needed by the entropy rules."""
    uses_ent = take_rule == TAKE_ENTROPY or hand_rule == HAND_ENTROPY
    dev, B, tk, outs = _scan_args(cu_q, prop_tok, topk_idx, K, driver, ctx_lens, seq_lens, ent,
                                  uses_ent, outs)
    st = lib().accept_scan_rule(
        _ptr(cu_q), _ptr(prop_tok), tk, K, _ptr(driver), _ptr(ctx_lens), _ptr(seq_lens),
        int(eos_id), int(max_len), B, int(take_rule), int(hand_rule),
        _ptr(ent) if uses_ent else None, float(tau_take), float(tau_hand), *_scan_outs(outs),
        _stream(dev))
    _check("accept_scan_rule", st)
    return outs


def sample_takeover(hidden, W, K: int, workspace, cu_q, driver, event_row, u, eos_id: int,
                    finished, row_local=None, seq_ids=None, token=None):
    """Teacher replacement tokens at the takeovers (see include/ipdv.h).

    hidden, W, K and workspace as passed to the preceding
    lmhead_logsoftmax_verify call (its records are read); cu_q [B+1] int32,
    driver [B] uint8, event_row [B] int32 (accept_scan's), u [B] float32
    uniforms in [0, 1), row_local [T] int32 or None, seq_ids [n] int32 or None
    (the sequences handled; None: all B), finished [B] uint8 (updated in
    place).  Returns token [B] int32 (-1: no draw; entries of sequences not
    handled are left as they were in `token`)."""
    dev = hidden.device
    dt = hidden.dtype
    _need(hidden, "hidden", dt, dev, 2)
    M, Hd = hidden.shape
    w_ptr, V, code = _w_arg(W, dt, dev, Hd)
    _need(cu_q, "cu_q", torch.int32, dev, 1)
    B = cu_q.shape[0] - 1
    _need(driver, "driver", torch.uint8, dev, 1)
    _need(event_row, "event_row", torch.int32, dev, 1)
    _need(u, "u", torch.float32, dev, 1)
    _need(finished, "finished", torch.uint8, dev, 1)
    if row_local is not None:
        _need(row_local, "row_local", torch.int32, dev, 1)
    n_seq = B
    if seq_ids is not None:
        _need(seq_ids, "seq_ids", torch.int32, dev, 1)
        n_seq = seq_ids.shape[0]
    if token is None:
        token = torch.full((B,), -1, dtype=torch.int32, device=dev)
    st = lib().sample_takeover(
        _ptr(hidden), w_ptr, M, Hd, V, K, _ptr(workspace),
        workspace.numel() * workspace.element_size(), _ptr(seq_ids), n_seq, _ptr(cu_q),
        _ptr(driver), _ptr(event_row), _ptr(row_local), _ptr(u), int(eos_id), _ptr(token),
        _ptr(finished), code, _stream(dev))
    _check("sample_takeover", st)
    return token


def lmhead_logp_gather(hidden, W, lse, idx, out=None):
    """log-softmax of hidden . W^T at idx [M, n] (see include/ipdv.h);
    lse [M] float32 from the same model's lmhead_logsoftmax_verify.  Returns
    logp [M, n] float32 (-inf for indices outside [0, V))."""
    dev = hidden.device
    dt = hidden.dtype
    _need(hidden, "hidden", dt, dev, 2)
    M, Hd = hidden.shape
    w_ptr, V, code = _w_arg(W, dt, dev, Hd)
    _need(lse, "lse", torch.float32, dev, 1)
    _need(idx, "idx", torch.int32, dev, 2)
    if lse.shape[0] != M or idx.shape[0] != M:
        raise ValueError("lse and idx must have M rows")
    n = idx.shape[1]
    if out is None:
        out = torch.empty(M, n, dtype=torch.float32, device=dev)
    st = lib().lmhead_logp_gather(_ptr(hidden), w_ptr, M, Hd, V, _ptr(lse), _ptr(idx), n,
                                  _ptr(out), code, _stream(dev))
    _check("lmhead_logp_gather", st)
    return out


SUPPORT_UNION, SUPPORT_STUDENT, SUPPORT_TEACHER, SUPPORT_INTERSECTION = 0, 1, 2, 3
LOSS_IPD_SPLIT, LOSS_PURE_REVERSE, LOSS_PURE_FORWARD, LOSS_INVERSE_SPLIT = 0, 1, 2, 3


def source_split_kl(s_idx, s_logp, s_at_t, t_idx, t_logp, t_at_s, src, support=SUPPORT_UNION,
                    loss_mode=LOSS_IPD_SPLIT, cu=None):
    """Per-position source-split KL values (see include/ipdv.h).  Inputs
    [M, K] (int32 indices, float32 log-probs) and src [M] uint8; cu [B+1]
    int32 segment offsets or None.  Returns dict kl_rev, kl_fwd, loss,
    overlap [M] and, with cu, seq_loss, t_ratio [B] (float32)."""
    dev = s_idx.device
    for t, name, dt in ((s_idx, "s_idx", torch.int32), (t_idx, "t_idx", torch.int32),
                        (s_logp, "s_logp", torch.float32), (s_at_t, "s_at_t", torch.float32),
                        (t_logp, "t_logp", torch.float32), (t_at_s, "t_at_s", torch.float32)):
        _need(t, name, dt, dev, 2)
    M, K = s_idx.shape
    for t in (s_logp, s_at_t, t_idx, t_logp, t_at_s):
        if tuple(t.shape) != (M, K):
            raise ValueError("every list input must be [M, K]")
    _need(src, "src", torch.uint8, dev, 1)
    if src.shape[0] != M:
        raise ValueError("src must be [M]")
    out = {k: torch.empty(M, dtype=torch.float32, device=dev)
           for k in ("kl_rev", "kl_fwd", "loss", "overlap")}
    B = 0
    if cu is not None:
        _need(cu, "cu", torch.int32, dev, 1)
        B = cu.shape[0] - 1
        out["seq_loss"] = torch.empty(B, dtype=torch.float32, device=dev)
        out["t_ratio"] = torch.empty(B, dtype=torch.float32, device=dev)
    st = lib().source_split_kl(
        M, K, _ptr(s_idx), _ptr(s_logp), _ptr(s_at_t), _ptr(t_idx), _ptr(t_logp), _ptr(t_at_s),
        _ptr(src), int(support), int(loss_mode), _ptr(out["kl_rev"]), _ptr(out["kl_fwd"]),
        _ptr(out["loss"]), _ptr(out["overlap"]), _ptr(cu), B, _ptr(out.get("seq_loss")),
        _ptr(out.get("t_ratio")), _stream(dev))
    _check("source_split_kl", st)
    return out


def lmhead_sample(hidden, W, K: int, workspace, u, token=None):
    """One temperature-1 draw per row (see include/ipdv.h): hidden, W, K and
    workspace as passed to the preceding lmhead_logsoftmax_verify call; u [M]
    float32 uniforms in [0, 1).  Returns token [M] int32."""
    dev = hidden.device
    dt = hidden.dtype
    _need(hidden, "hidden", dt, dev, 2)
    M, Hd = hidden.shape
    w_ptr, V, code = _w_arg(W, dt, dev, Hd)
    _need(u, "u", torch.float32, dev, 1)
    if u.shape[0] != M:
        raise ValueError("u must be [M]")
    if token is None:
        token = torch.empty(M, dtype=torch.int32, device=dev)
    st = lib().lmhead_sample(_ptr(hidden), w_ptr, M, Hd, V, K, _ptr(workspace),
                             workspace.numel() * workspace.element_size(), _ptr(u), _ptr(token),
                             code, _stream(dev))
    _check("lmhead_sample", st)
    return token
