"""torch-facing wrappers of the C ABI (include/rcllm.h).

Argument marshalling only: shapes, dtypes and pointers are checked and passed
to librcllm, which enqueues its HIP kernels on torch's current stream. torch
provides device memory and streams; no step of the path runs in torch, and
there is no fallback: without the built library every call raises.
"""
from __future__ import annotations

import ctypes
import math
import os
from dataclasses import dataclass

import numpy as np
import torch

from . import _lib
from ._lib import RcPool, RcShape, check
from .inputs import LayerWeights


# Debug mode (RCLLM_DEBUG=1): row lists are checked after the selection and
# before attention, at the cost of a synchronisation per call. The library
# marks a request whose segment table disagrees with n_fresh (or whose budget
# exceeds its class) with -1 entries in its row list instead of failing, since
# it cannot read device tables without a synchronisation.
DEBUG = os.environ.get("RCLLM_DEBUG", "") not in ("", "0")


def check_rows(rows: torch.Tensor, N: int, what: str) -> None:
    """Raise if any listed row lies outside [0, N); names the requests."""
    if rows.numel() == 0:
        return
    r = rows.detach().cpu()
    bad = ((r < 0) | (r >= N)).any(dim=1).nonzero().flatten().tolist()
    if bad:
        raise RuntimeError(f"{what}: requests {bad} have row-list entries outside [0, {N}) "
                           f"(segment table disagreeing with n_fresh, or a budget above its class)")


def _dtype_code(t: torch.Tensor) -> int:
    if t.dtype == torch.bfloat16:
        return _lib.RC_BF16
    if t.dtype == torch.float32:
        return _lib.RC_F32
    raise TypeError(f"storage dtype must be bfloat16 or float32, got {t.dtype}")


def _dev(t: torch.Tensor, name: str) -> int:
    if not isinstance(t, torch.Tensor):
        raise TypeError(f"{name} must be a torch.Tensor")
    if not t.is_cuda:
        raise ValueError(f"{name} must be a device tensor")
    if not t.is_contiguous():
        raise ValueError(f"{name} must be contiguous")
    return t.data_ptr()


def _pool_ptr(t: torch.Tensor, name: str) -> int:
    """Device tensors, or pinned host tensors (read by the kernels over PCIe)."""
    if isinstance(t, torch.Tensor) and not t.is_cuda and t.is_pinned():
        if not t.is_contiguous():
            raise ValueError(f"{name} must be contiguous")
        return t.data_ptr()
    return _dev(t, name)


def _stream(stream=None) -> ctypes.c_void_p:
    s = torch.cuda.current_stream() if stream is None else stream
    return ctypes.c_void_p(s.cuda_stream)


def _shape(B, N, Hq, Hkv, D, dtype_code) -> RcShape:
    return RcShape(int(B), int(N), int(Hq), int(Hkv), int(D), int(dtype_code))


# ---------------------------------------------------------------- segments

@dataclass
class Segments:
    """A validated, uploaded segment table."""
    dev: torch.Tensor       # [B, S, 4] int32 on the device
    host: np.ndarray        # [B, S, 4] int32
    n_fresh: int            # fresh positions per request (same for every request)
    N: int

    @property
    def S(self) -> int:
        return int(self.host.shape[1])

    @property
    def n_reused(self) -> int:
        return self.N - self.n_fresh


def prepare_segments(segs, N: int, pools, device, check_blocks: bool = True) -> Segments:
    """Check on the host that every request's segments tile [0, N) in order,
    name existing pools and blocks and share one fresh count, then upload.
    check_blocks=False: a status table (fresh / cached-from-pool runs) that
    only the selection reads, e.g. for a token-granular gather."""
    h = np.ascontiguousarray(np.asarray(segs.cpu() if isinstance(segs, torch.Tensor) else segs,
                                        dtype=np.int32))
    if h.ndim != 3 or h.shape[2] != 4 or h.shape[1] < 1:
        raise ValueError("segments must have shape [B, S, 4]")
    n_fresh = None
    for b, req in enumerate(h):
        pos, fresh = 0, 0
        for dst, ln, p, blk in req.tolist():
            if dst != pos or ln < 1:
                raise ValueError(f"request {b}: segments must tile [0, N) in order")
            if p >= 0:
                if p >= len(pools):
                    raise ValueError(f"request {b}: pool {p} does not exist")
                pk = pools[p][0]
                if check_blocks and (not (0 <= blk < pk.shape[0]) or ln > pk.shape[1]):
                    raise ValueError(f"request {b}: block {blk}/len {ln} outside pool {p}")
            else:
                fresh += ln
            pos += ln
        if pos != N:
            raise ValueError(f"request {b}: segments cover {pos} positions, N = {N}")
        if n_fresh is None:
            n_fresh = fresh
        elif fresh != n_fresh:
            raise ValueError("every request must have the same number of fresh positions")
    dev = torch.from_numpy(h).to(device)
    return Segments(dev=dev, host=h, n_fresh=int(n_fresh), N=int(N))


# ----------------------------------------------------------------- calls

def rope_table(max_pos: int, D: int, base: float, device=None):
    """cos/sin tables [max_pos, D/2] fp32 built by the library (host) and
    uploaded to `device` when given."""
    cos = torch.empty((max_pos, D // 2), dtype=torch.float32)
    sin = torch.empty((max_pos, D // 2), dtype=torch.float32)
    check(_lib.load().rc_rope_table(int(max_pos), int(D), float(base),
                                    ctypes.c_void_p(cos.data_ptr()), ctypes.c_void_p(sin.data_ptr())))
    if device is not None:
        cos, sin = cos.to(device), sin.to(device)
    return cos, sin


def _pool_array(pools, dtype, Hkv, D):
    arr = (RcPool * len(pools))()
    for i, (pk, pv) in enumerate(pools):
        if pk.dtype != dtype or pv.dtype != dtype:
            raise TypeError("pool dtype differs from the fresh tensors")
        if pk.shape != pv.shape or pk.dim() != 4 or pk.shape[2] != Hkv or pk.shape[3] != D:
            raise ValueError("pool K/V must be [num_blocks, block_len, Hkv, D]")
        arr[i] = RcPool(_pool_ptr(pk, "pool k"), _pool_ptr(pv, "pool v"), pk.shape[0], pk.shape[1])
    return arr


def kv_assemble(pools, segs: Segments, k_fresh, v_fresh, cos=None, sin=None, k_out=None,
                v_out=None, scores_out=None, stream=None, score_only=False):
    """rc_kv_assemble: gather + fused re-alignment (+ deviation scores into
    `scores_out` [B, N] fp32 when given). Returns (k_asm, v_asm); with
    score_only the rows are only scored (nothing stored) and (None, None) is
    returned."""
    B, N, Hkv, D = k_fresh.shape
    if v_fresh.shape != k_fresh.shape or v_fresh.dtype != k_fresh.dtype:
        raise ValueError("k_fresh and v_fresh must match")
    if score_only:
        if scores_out is None:
            raise ValueError("score_only needs scores_out")
    else:
        k_out = torch.empty_like(k_fresh) if k_out is None else k_out
        v_out = torch.empty_like(v_fresh) if v_out is None else v_out
    code = _dtype_code(k_fresh)
    parr = _pool_array(pools, k_fresh.dtype, Hkv, D)
    max_pos = 0 if cos is None else int(cos.shape[0])
    check(_lib.load().rc_kv_assemble(
        ctypes.byref(_shape(B, N, 1, Hkv, D, code)), parr, len(pools), _dev(segs.dev, "segs"),
        segs.S, _dev(k_fresh, "k_fresh"), _dev(v_fresh, "v_fresh"),
        None if cos is None else _dev(cos, "cos"), None if sin is None else _dev(sin, "sin"),
        max_pos, None if score_only else _dev(k_out, "k_out"),
        None if score_only else _dev(v_out, "v_out"),
        None if scores_out is None else _dev(scores_out, "scores_out"), _stream(stream)))
    return (None, None) if score_only else (k_out, v_out)


def kv_assemble_vref(pools, segs: Segments, k_fresh, v_fresh, cos=None, sin=None, k_out=None,
                     v_ref=None, scores_out=None, stream=None):
    """rc_kv_assemble_vref: gather + fused re-alignment of K (+ deviation
    scores), and a table v_ref [B, N] int64 of value-row byte addresses (pool
    or fresh row) instead of a copy of V. The table refers to the pool tensors
    and to v_fresh: they must outlive its use. Returns (k_asm, v_ref)."""
    B, N, Hkv, D = k_fresh.shape
    if v_fresh.shape != k_fresh.shape or v_fresh.dtype != k_fresh.dtype:
        raise ValueError("k_fresh and v_fresh must match")
    k_out = torch.empty_like(k_fresh) if k_out is None else k_out
    if v_ref is None:
        v_ref = torch.empty((B, N), dtype=torch.int64, device=k_fresh.device)
    elif v_ref.dtype != torch.int64 or tuple(v_ref.shape) != (B, N):
        raise ValueError("v_ref must be int64 [B, N]")
    parr = _pool_array(pools, k_fresh.dtype, Hkv, D)
    max_pos = 0 if cos is None else int(cos.shape[0])
    check(_lib.load().rc_kv_assemble_vref(
        ctypes.byref(_shape(B, N, 1, Hkv, D, _dtype_code(k_fresh))), parr, len(pools),
        _dev(segs.dev, "segs"), segs.S, _dev(k_fresh, "k_fresh"), _dev(v_fresh, "v_fresh"),
        None if cos is None else _dev(cos, "cos"), None if sin is None else _dev(sin, "sin"),
        max_pos, _dev(k_out, "k_out"), _dev(v_ref, "v_ref"),
        None if scores_out is None else _dev(scores_out, "scores_out"), _stream(stream)))
    return k_out, v_ref


def kv_gather_tokens(pools, token_map, k_fresh, v_fresh, cos=None, sin=None, k_out=None,
                     v_out=None, scores_out=None, stream=None, max_workgroups=0):
    """rc_kv_gather_tokens: per-position map gather + alignment (+ deviation
    scores). token_map: device int32 [B, N, 4]. Pools may be pinned host
    tensors. Returns (k_asm, v_asm)."""
    B, N, Hkv, D = k_fresh.shape
    if tuple(token_map.shape) != (B, N, 4) or token_map.dtype != torch.int32:
        raise ValueError("token_map must be int32 [B, N, 4]")
    k_out = torch.empty_like(k_fresh) if k_out is None else k_out
    v_out = torch.empty_like(v_fresh) if v_out is None else v_out
    parr = _pool_array(pools, k_fresh.dtype, Hkv, D)
    max_pos = 0 if cos is None else int(cos.shape[0])
    check(_lib.load().rc_kv_gather_tokens(
        ctypes.byref(_shape(B, N, 1, Hkv, D, _dtype_code(k_fresh))), parr, len(pools),
        _dev(token_map, "token_map"), _dev(k_fresh, "k_fresh"), _dev(v_fresh, "v_fresh"),
        None if cos is None else _dev(cos, "cos"), None if sin is None else _dev(sin, "sin"),
        max_pos, _dev(k_out, "k_out"), _dev(v_out, "v_out"),
        None if scores_out is None else _dev(scores_out, "scores_out"), int(max_workgroups),
        _stream(stream)))
    return k_out, v_out


def pin_pool(pool):
    """Pinned host copy of a (pool_k, pool_v) pair: the pool then stays in host
    memory and the gather reads it over PCIe."""
    return tuple(t.detach().cpu().contiguous().pin_memory() for t in pool)


def rerope(k, delta, cos, sin, stream=None):
    """rc_rerope: rotate K[b,i] by delta[b,i] in place. Returns k."""
    B, N, Hkv, D = k.shape
    if delta.dtype != torch.int32 or tuple(delta.shape) != (B, N):
        raise ValueError("delta must be int32 [B, N]")
    check(_lib.load().rc_rerope(ctypes.byref(_shape(B, N, 1, Hkv, D, _dtype_code(k))),
                                _dev(k, "k"), _dev(delta, "delta"), _dev(cos, "cos"),
                                _dev(sin, "sin"), int(cos.shape[0]), _stream(stream)))
    return k


def select_tokens(segs: Segments, k: int, k_fresh, v_fresh, k_asm, v_asm, scores_in=None,
                  scores_out=None, rows_out=None, patch=True, stream=None):
    """rc_select_tokens: score, top-k, patch. Returns (rows, scores)."""
    B, N, Hkv, D = k_fresh.shape
    R = segs.n_fresh + int(k)
    rows = torch.empty((B, R), dtype=torch.int32, device=k_fresh.device) if rows_out is None else rows_out
    if scores_in is None and scores_out is None:
        scores_out = torch.empty((B, N), dtype=torch.float32, device=k_fresh.device)
    check(_lib.load().rc_select_tokens(
        ctypes.byref(_shape(B, N, 1, Hkv, D, _dtype_code(k_fresh))), _dev(segs.dev, "segs"),
        segs.S, segs.n_fresh, int(k), _dev(k_fresh, "k_fresh"), _dev(v_fresh, "v_fresh"),
        None if k_asm is None else _dev(k_asm, "k_asm"),
        None if v_asm is None else _dev(v_asm, "v_asm"),
        None if scores_in is None else _dev(scores_in, "scores_in"),
        None if scores_out is None else _dev(scores_out, "scores_out"),
        _dev(rows, "rows"), 1 if patch else 0, _stream(stream)))
    if DEBUG:
        check_rows(rows, N, "rc_select_tokens")
    return rows, (scores_out if scores_out is not None else scores_in)


def select_tokens_vref(segs: Segments, k: int, k_fresh, v_fresh, k_asm, v_ref, scores_in=None,
                       scores_out=None, rows_out=None, stream=None):
    """rc_select_tokens_vref: score, top-k, and the correction over a value
    reference table (fresh K rows copied, value entries of the selected
    positions pointed at their fresh rows). Returns (rows, scores)."""
    B, N, Hkv, D = k_fresh.shape
    R = segs.n_fresh + int(k)
    if v_ref.dtype != torch.int64 or tuple(v_ref.shape) != (B, N):
        raise ValueError("v_ref must be int64 [B, N]")
    rows = torch.empty((B, R), dtype=torch.int32, device=k_fresh.device) if rows_out is None else rows_out
    if scores_in is None and scores_out is None:
        scores_out = torch.empty((B, N), dtype=torch.float32, device=k_fresh.device)
    check(_lib.load().rc_select_tokens_vref(
        ctypes.byref(_shape(B, N, 1, Hkv, D, _dtype_code(k_fresh))), _dev(segs.dev, "segs"),
        segs.S, segs.n_fresh, int(k), _dev(k_fresh, "k_fresh"), _dev(v_fresh, "v_fresh"),
        _dev(k_asm, "k_asm"), _dev(v_ref, "v_ref"),
        None if scores_in is None else _dev(scores_in, "scores_in"),
        None if scores_out is None else _dev(scores_out, "scores_out"),
        _dev(rows, "rows"), _stream(stream)))
    if DEBUG:
        check_rows(rows, N, "rc_select_tokens_vref")
    return rows, (scores_out if scores_out is not None else scores_in)


def selective_attention_vref(q, k, v_ref, rows=None, scale=None, out=None, stream=None):
    """rc_selective_attention_vref: rc_selective_attention with V read
    through v_ref [B, N] int64 (value-row byte addresses); bf16, D = 128."""
    B, N, Hq, D = q.shape
    Hkv = k.shape[2]
    if k.shape[:2] != q.shape[:2] or k.shape[3] != D:
        raise ValueError("q [B,N,Hq,D] and k [B,N,Hkv,D] do not match")
    if v_ref.dtype != torch.int64 or tuple(v_ref.shape) != (B, N):
        raise ValueError("v_ref must be int64 [B, N]")
    R = N if rows is None else int(rows.shape[1])
    if rows is not None and (rows.dtype != torch.int32 or rows.shape[0] != B):
        raise ValueError("rows must be int32 [B, R]")
    scale = 1.0 / math.sqrt(D) if scale is None else float(scale)
    out = torch.empty((B, R, Hq, D), dtype=q.dtype, device=q.device) if out is None else out
    if DEBUG and rows is not None:
        check_rows(rows, N, "rc_selective_attention_vref")
    check(_lib.load().rc_selective_attention_vref(
        ctypes.byref(_shape(B, N, Hq, Hkv, D, _dtype_code(q))), _dev(q, "q"),
        None if rows is None else _dev(rows, "rows"), R, _dev(k, "k"), _dev(v_ref, "v_ref"),
        ctypes.c_float(scale), _dev(out, "out"), _stream(stream)))
    return out


def selective_attention(q, k, v, rows=None, scale=None, out=None, stream=None):
    """rc_selective_attention: causal GQA attention of `rows` (all rows if None)."""
    B, N, Hq, D = q.shape
    Hkv = k.shape[2]
    if k.shape != v.shape or k.shape[:2] != q.shape[:2] or k.shape[3] != D:
        raise ValueError("q [B,N,Hq,D] and k, v [B,N,Hkv,D] do not match")
    R = N if rows is None else int(rows.shape[1])
    if rows is not None and (rows.dtype != torch.int32 or rows.shape[0] != B):
        raise ValueError("rows must be int32 [B, R]")
    scale = 1.0 / math.sqrt(D) if scale is None else float(scale)
    out = torch.empty((B, R, Hq, D), dtype=q.dtype, device=q.device) if out is None else out
    if DEBUG and rows is not None:
        check_rows(rows, N, "rc_selective_attention")
    check(_lib.load().rc_selective_attention(
        ctypes.byref(_shape(B, N, Hq, Hkv, D, _dtype_code(q))), _dev(q, "q"),
        None if rows is None else _dev(rows, "rows"), R, _dev(k, "k"), _dev(v, "v"),
        ctypes.c_float(scale), _dev(out, "out"), _stream(stream)))
    return out


def selective_attention_lse(q, k, v, rows=None, scale=None, out=None, lse=None, stream=None):
    """rc_selective_attention_lse: attention plus each row's natural
    log-sum-exp [B, R, Hq] fp32. Returns (out, lse)."""
    B, N, Hq, D = q.shape
    Hkv = k.shape[2]
    if k.shape != v.shape or k.shape[:2] != q.shape[:2] or k.shape[3] != D:
        raise ValueError("q [B,N,Hq,D] and k, v [B,N,Hkv,D] do not match")
    R = N if rows is None else int(rows.shape[1])
    if rows is not None and (rows.dtype != torch.int32 or rows.shape[0] != B):
        raise ValueError("rows must be int32 [B, R]")
    scale = 1.0 / math.sqrt(D) if scale is None else float(scale)
    out = torch.empty((B, R, Hq, D), dtype=q.dtype, device=q.device) if out is None else out
    lse = torch.empty((B, R, Hq), dtype=torch.float32, device=q.device) if lse is None else lse
    check(_lib.load().rc_selective_attention_lse(
        ctypes.byref(_shape(B, N, Hq, Hkv, D, _dtype_code(q))), _dev(q, "q"),
        None if rows is None else _dev(rows, "rows"), R, _dev(k, "k"), _dev(v, "v"),
        ctypes.c_float(scale), _dev(out, "out"), _dev(lse, "lse"), _stream(stream)))
    return out, lse


def attention_mass(q, k, lse, scale=None, mass=None, stream=None):
    """rc_attention_mass: attention weight each key receives from every row
    of its KV group's heads, [B, Hkv, N] fp32."""
    B, N, Hq, D = q.shape
    Hkv = k.shape[2]
    if k.shape[:2] != q.shape[:2] or k.shape[3] != D:
        raise ValueError("q [B,N,Hq,D] and k [B,N,Hkv,D] do not match")
    if tuple(lse.shape) != (B, N, Hq) or lse.dtype != torch.float32:
        raise ValueError("lse must be fp32 [B, N, Hq] (every row of the full pass)")
    scale = 1.0 / math.sqrt(D) if scale is None else float(scale)
    mass = torch.empty((B, Hkv, N), dtype=torch.float32, device=q.device) if mass is None else mass
    check(_lib.load().rc_attention_mass(
        ctypes.byref(_shape(B, N, Hq, Hkv, D, _dtype_code(q))), _dev(q, "q"), _dev(k, "k"),
        _dev(lse, "lse"), ctypes.c_float(scale), _dev(mass, "mass"), _stream(stream)))
    return mass


def component_counts(segs: Segments, item_mask: int):
    """Cached positions per request in the history and item classes."""
    h = segs.host
    cached = h[..., 2] >= 0
    item = cached & (((item_mask >> np.clip(h[..., 2], 0, 31)) & 1) == 1)
    lens = h[..., 1]
    return (np.where(cached & ~item, lens, 0).sum(1), np.where(item, lens, 0).sum(1))


def select_tokens_eq3(segs: Segments, item_mask: int, lam: float, k_hist: int, k_item: int,
                      k_fresh, v_fresh, k_asm, v_asm, mass=None, scores_in=None,
                      scores_out=None, rows_out=None, patch=True, stream=None):
    """rc_select_tokens_eq3: Eq. (3) score, separate history/item top-k,
    patch. Returns (rows, scores)."""
    B, N, Hkv, D = k_fresh.shape
    nh, ni = component_counts(segs, item_mask)
    if k_hist > nh.min() or k_item > ni.min():
        raise ValueError(f"budgets ({k_hist}, {k_item}) exceed a request's history/item "
                         f"counts ({nh.min()}, {ni.min()})")
    R = segs.n_fresh + int(k_hist) + int(k_item)
    rows = torch.empty((B, R), dtype=torch.int32, device=k_fresh.device) if rows_out is None else rows_out
    if scores_in is None and scores_out is None:
        scores_out = torch.empty((B, N), dtype=torch.float32, device=k_fresh.device)
    check(_lib.load().rc_select_tokens_eq3(
        ctypes.byref(_shape(B, N, 1, Hkv, D, _dtype_code(k_fresh))), _dev(segs.dev, "segs"),
        segs.S, segs.n_fresh, int(item_mask), ctypes.c_float(lam), int(k_hist), int(k_item),
        None if mass is None else _dev(mass, "mass"), _dev(k_fresh, "k_fresh"),
        _dev(v_fresh, "v_fresh"), None if k_asm is None else _dev(k_asm, "k_asm"),
        None if v_asm is None else _dev(v_asm, "v_asm"),
        None if scores_in is None else _dev(scores_in, "scores_in"),
        None if scores_out is None else _dev(scores_out, "scores_out"),
        _dev(rows, "rows"), 1 if patch else 0, _stream(stream)))
    if DEBUG:
        check_rows(rows, N, "rc_select_tokens_eq3")
    return rows, (scores_out if scores_out is not None else scores_in)


def paged_attention(q, k_fresh, v_fresh, pools, segs: Segments, rows, cos=None, sin=None,
                    scale=None, out=None, stream=None):
    """rc_paged_attention: selective attention straight from the pools and
    fresh tensors through the segment table (no assembled copy)."""
    B, N, Hq, D = q.shape
    Hkv = k_fresh.shape[2]
    if rows.dtype != torch.int32 or rows.dim() != 2 or rows.shape[0] != B:
        raise ValueError("rows must be int32 [B, R]")
    R = int(rows.shape[1])
    scale = 1.0 / math.sqrt(D) if scale is None else float(scale)
    out = torch.empty((B, R, Hq, D), dtype=q.dtype, device=q.device) if out is None else out
    parr = _pool_array(pools, k_fresh.dtype, Hkv, D)
    max_pos = 0 if cos is None else int(cos.shape[0])
    check(_lib.load().rc_paged_attention(
        ctypes.byref(_shape(B, N, Hq, Hkv, D, _dtype_code(q))), _dev(q, "q"), _dev(rows, "rows"), R,
        parr, len(pools), _dev(segs.dev, "segs"), segs.S, _dev(k_fresh, "k_fresh"),
        _dev(v_fresh, "v_fresh"), None if cos is None else _dev(cos, "cos"),
        None if sin is None else _dev(sin, "sin"), max_pos, ctypes.c_float(scale),
        _dev(out, "out"), _stream(stream)))
    return out


def segments_with_window(segs, N: int, W: int) -> np.ndarray:
    """rc_segments_with_window (host): the last W positions of every request
    become fresh segments. Returns the new [B, S', 4] int32 table."""
    h = np.ascontiguousarray(np.asarray(segs.cpu() if isinstance(segs, torch.Tensor) else segs,
                                        dtype=np.int32))
    B, S = h.shape[:2]
    cap = S + 1
    out = np.zeros((B * cap, 4), np.int32)
    s_out = ctypes.c_int32(0)
    check(_lib.load().rc_segments_with_window(h.ctypes.data_as(ctypes.c_void_p), B, S, int(N), int(W),
                                              out.ctypes.data_as(ctypes.c_void_p), cap,
                                              ctypes.byref(s_out)))
    return out[:B * s_out.value].reshape(B, s_out.value, 4).copy()


# ------------------------------------------------------------- the pipeline

@dataclass
class PrefillBuffers:
    k_asm: torch.Tensor
    v_asm: torch.Tensor | None      # assembled V (None: value rows by reference)
    scores: torch.Tensor
    rows: torch.Tensor
    out: torch.Tensor
    v_ref: torch.Tensor | None = None   # [B, N] int64 value-row addresses

    @staticmethod
    def alloc(B, N, Hq, Hkv, D, R, dtype, device, v_copy=True, v_ref=False):
        return PrefillBuffers(
            k_asm=torch.empty((B, N, Hkv, D), dtype=dtype, device=device),
            v_asm=torch.empty((B, N, Hkv, D), dtype=dtype, device=device) if v_copy else None,
            scores=torch.empty((B, N), dtype=torch.float32, device=device),
            rows=torch.empty((B, R), dtype=torch.int32, device=device),
            out=torch.empty((B, R, Hq, D), dtype=dtype, device=device),
            v_ref=torch.empty((B, N), dtype=torch.int64, device=device) if v_ref else None)


def selective_prefill(q, k_fresh, v_fresh, pools, segs: Segments, k: int, cos, sin,
                      scale=None, bufs: PrefillBuffers | None = None, stream=None):
    """One layer of selective prefill on one stream: assemble (fused
    re-alignment and deviation score) -> top-k, patch -> attention of the fresh
    and selected rows. Returns the buffers (k_asm, v_asm patched, scores, rows,
    out)."""
    B, N, Hq, D = q.shape
    Hkv = k_fresh.shape[2]
    R = segs.n_fresh + int(k)
    if bufs is None:
        bufs = PrefillBuffers.alloc(B, N, Hq, Hkv, D, R, q.dtype, q.device)
    kv_assemble(pools, segs, k_fresh, v_fresh, cos, sin, bufs.k_asm, bufs.v_asm,
                scores_out=bufs.scores, stream=stream)
    select_tokens(segs, k, k_fresh, v_fresh, bufs.k_asm, bufs.v_asm, scores_in=bufs.scores,
                  rows_out=bufs.rows, patch=True, stream=stream)
    if R > 0:
        selective_attention(q, bufs.k_asm, bufs.v_asm, bufs.rows, scale, bufs.out, stream)
    return bufs


def selective_prefill_vref(q, k_fresh, v_fresh, pools, segs: Segments, k: int, cos, sin,
                           scale=None, bufs: PrefillBuffers | None = None, stream=None):
    """selective_prefill with the value rows taken by reference: the gather
    copies and aligns K and writes a table of value-row addresses, the patch
    copies fresh K rows and redirects their value entries, and the attention
    reads V through the table (bf16, D = 128). The pools and v_fresh must
    outlive the use of bufs.v_ref. Returns the buffers (k_asm patched,
    v_ref, scores, rows, out)."""
    B, N, Hq, D = q.shape
    Hkv = k_fresh.shape[2]
    R = segs.n_fresh + int(k)
    if bufs is None:
        bufs = PrefillBuffers.alloc(B, N, Hq, Hkv, D, R, q.dtype, q.device, v_copy=False,
                                    v_ref=True)
    kv_assemble_vref(pools, segs, k_fresh, v_fresh, cos, sin, bufs.k_asm, bufs.v_ref,
                     scores_out=bufs.scores, stream=stream)
    select_tokens_vref(segs, k, k_fresh, v_fresh, bufs.k_asm, bufs.v_ref, scores_in=bufs.scores,
                       rows_out=bufs.rows, stream=stream)
    if R > 0:
        selective_attention_vref(q, bufs.k_asm, bufs.v_ref, bufs.rows, scale, bufs.out, stream)
    return bufs


@dataclass
class Eq3Buffers:
    k_asm: torch.Tensor
    v_asm: torch.Tensor
    out_full: torch.Tensor   # the first layer's attention output, every row
    lse: torch.Tensor
    mass: torch.Tensor
    scores: torch.Tensor
    rows: torch.Tensor

    @staticmethod
    def alloc(B, N, Hq, Hkv, D, R, dtype, device):
        return Eq3Buffers(
            k_asm=torch.empty((B, N, Hkv, D), dtype=dtype, device=device),
            v_asm=torch.empty((B, N, Hkv, D), dtype=dtype, device=device),
            out_full=torch.empty((B, N, Hq, D), dtype=dtype, device=device),
            lse=torch.empty((B, N, Hq), dtype=torch.float32, device=device),
            mass=torch.empty((B, Hkv, N), dtype=torch.float32, device=device),
            scores=torch.empty((B, N), dtype=torch.float32, device=device),
            rows=torch.empty((B, R), dtype=torch.int32, device=device))


def eq3_select(q, k_fresh, v_fresh, pools, segs: Segments, item_mask: int, lam: float,
               k_hist: int, k_item: int, cos, sin, scale=None, bufs: Eq3Buffers | None = None,
               stream=None):
    """Selection by the full Eq. (3) score on one stream: the first layer in
    full (attention of every row over the fresh K/V, with log-sum-exp) ->
    attention mass -> assemble (gather + alignment) -> score, separate
    history/item top-k, patch. Returns the buffers."""
    B, N, Hq, D = q.shape
    Hkv = k_fresh.shape[2]
    R = segs.n_fresh + int(k_hist) + int(k_item)
    if bufs is None:
        bufs = Eq3Buffers.alloc(B, N, Hq, Hkv, D, R, q.dtype, q.device)
    selective_attention_lse(q, k_fresh, v_fresh, None, scale, bufs.out_full, bufs.lse, stream)
    attention_mass(q, k_fresh, bufs.lse, scale, bufs.mass, stream)
    kv_assemble(pools, segs, k_fresh, v_fresh, cos, sin, bufs.k_asm, bufs.v_asm, stream=stream)
    select_tokens_eq3(segs, item_mask, lam, k_hist, k_item, k_fresh, v_fresh, bufs.k_asm,
                      bufs.v_asm, mass=bufs.mass, scores_out=bufs.scores, rows_out=bufs.rows,
                      patch=True, stream=stream)
    return bufs


def paged_prefill(q, k_fresh, v_fresh, pools, segs: Segments, k: int, cos, sin, scale=None,
                  bufs: PrefillBuffers | None = None, stream=None):
    """Zero-copy selective prefill of one layer: deviation scores of the
    aligned pool keys without assembling -> top-k (no patch) -> attention
    that reads K/V through the segment table. Same rows and output as
    selective_prefill; bufs.k_asm / v_asm are not used."""
    B, N, Hq, D = q.shape
    Hkv = k_fresh.shape[2]
    R = segs.n_fresh + int(k)
    if bufs is None:
        bufs = PrefillBuffers.alloc(B, N, Hq, Hkv, D, R, q.dtype, q.device)
    kv_assemble(pools, segs, k_fresh, v_fresh, cos, sin, scores_out=bufs.scores, stream=stream,
                score_only=True)
    select_tokens(segs, k, k_fresh, v_fresh, None, None, scores_in=bufs.scores, rows_out=bufs.rows,
                  patch=False, stream=stream)
    if R > 0:
        paged_attention(q, k_fresh, v_fresh, pools, segs, bufs.rows, cos, sin, scale, bufs.out,
                        stream)
    return bufs


# Workgroups of a gather that overlaps the first layer: few enough to leave the
# compute units to the first layer while the gather waits on PCIe (measured
# best of 24..128 on the 3,008- and 2,080-position workloads).
OVERLAP_GATHER_WORKGROUPS = 64


def eq3_select_tokens_path(q, k_fresh, v_fresh, pools, token_map, status: Segments, item_mask: int,
                           lam: float, k_hist: int, k_item: int, cos, sin, scale=None,
                           bufs: Eq3Buffers | None = None, gather_stream=None,
                           gather_workgroups: int = OVERLAP_GATHER_WORKGROUPS):
    """Eq. (3) selection with token-granular sources (pool rows possibly in
    pinned host memory). With gather_stream, the gather runs there, overlapping
    the first layer in full (attention with log-sum-exp, attention mass) on the
    current stream, which needs no pool row (Sec. III-C.3 hides the transfer of
    cached KV under the first layer); the score then waits for the gather.
    Without it everything runs in order on the current stream. The
    overlapped gather runs on about gather_workgroups workgroups, so that it
    leaves the compute units to the first layer while it waits on PCIe."""
    B, N, Hq, D = q.shape
    Hkv = k_fresh.shape[2]
    R = status.n_fresh + int(k_hist) + int(k_item)
    if bufs is None:
        bufs = Eq3Buffers.alloc(B, N, Hq, Hkv, D, R, q.dtype, q.device)
    main = torch.cuda.current_stream()
    if gather_stream is None:
        kv_gather_tokens(pools, token_map, k_fresh, v_fresh, cos, sin, bufs.k_asm, bufs.v_asm)
    else:
        gather_stream.wait_stream(main)   # inputs written on the current stream
        kv_gather_tokens(pools, token_map, k_fresh, v_fresh, cos, sin, bufs.k_asm, bufs.v_asm,
                         stream=gather_stream, max_workgroups=gather_workgroups)
        done = torch.cuda.Event()
        done.record(gather_stream)
    selective_attention_lse(q, k_fresh, v_fresh, None, scale, bufs.out_full, bufs.lse)
    attention_mass(q, k_fresh, bufs.lse, scale, bufs.mass)
    if gather_stream is not None:
        main.wait_event(done)
    select_tokens_eq3(status, item_mask, lam, k_hist, k_item, k_fresh, v_fresh, bufs.k_asm,
                      bufs.v_asm, mass=bufs.mass, scores_out=bufs.scores, rows_out=bufs.rows,
                      patch=True)
    return bufs


def full_prefill(q, k_fresh, v_fresh, scale=None, out=None, stream=None):
    """Full-Recompute baseline: causal attention of every row over fresh K/V."""
    return selective_attention(q, k_fresh, v_fresh, None, scale, out, stream)


# ------------------------------------------------------- several layers

def gemm(x, w, residual=None, out=None, stream=None):
    """rc_gemm_bf16: out[M, n] = x[M, k] @ w[n, k]^T (+ residual)."""
    M, k = x.shape
    n = w.shape[0]
    if w.shape[1] != k:
        raise ValueError(f"x [M, {k}] and w [{n}, {w.shape[1]}] do not match")
    out = torch.empty((M, n), dtype=x.dtype, device=x.device) if out is None else out
    check(_lib.load().rc_gemm_bf16(
        int(M), int(n), int(k), _dev(x, "x"), _dev(w, "w"),
        None if residual is None else _dev(residual, "residual"), _dev(out, "out"), _stream(stream)))
    return out


def rmsnorm(x, gamma, eps=1e-5, out=None, stream=None):
    M, Hd = x.shape
    out = torch.empty_like(x) if out is None else out
    check(_lib.load().rc_rmsnorm(int(M), int(Hd), _dev(x, "x"), _dev(gamma, "gamma"),
                                 ctypes.c_float(eps), _dev(out, "out"), _stream(stream)))
    return out


def qkv_rope(qkv, B, N, Hq, Hkv, D, rows, cos, sin, q_out, k_out, v_out, stream=None):
    R = N if rows is None else int(rows.shape[1])
    check(_lib.load().rc_qkv_rope(
        ctypes.byref(_shape(B, N, Hq, Hkv, D, _lib.RC_BF16)), _dev(qkv, "qkv"),
        None if rows is None else _dev(rows, "rows"), R,
        None if cos is None else _dev(cos, "cos"), None if sin is None else _dev(sin, "sin"),
        0 if cos is None else int(cos.shape[0]), _dev(q_out, "q_out"), _dev(k_out, "k_out"),
        _dev(v_out, "v_out"), _stream(stream)))


def silu_mul(gate_up, out=None, stream=None):
    M, I2 = gate_up.shape
    out = torch.empty((M, I2 // 2), dtype=gate_up.dtype, device=gate_up.device) if out is None else out
    check(_lib.load().rc_silu_mul(int(M), int(I2 // 2), _dev(gate_up, "gate_up"), _dev(out, "out"),
                                  _stream(stream)))
    return out


def gather_rows(src, rows, out=None, stream=None):
    """dst[b, r] = src[b, rows[b, r]] for src [B, Nsrc, ...]."""
    B, Nsrc = src.shape[:2]
    R = int(rows.shape[1])
    row_bytes = src[0, 0].numel() * src.element_size()
    out = torch.empty((B, R) + tuple(src.shape[2:]), dtype=src.dtype, device=src.device) if out is None else out
    check(_lib.load().rc_gather_rows(int(B), int(Nsrc), R, int(row_bytes), _dev(src, "src"),
                                     _dev(rows, "rows"), _dev(out, "out"), _stream(stream)))
    return out


def _mlp_and_residual(h, L: "LayerWeights", eps):
    n2 = rmsnorm(h, L.g_mlp, eps)
    act = silu_mul(gemm(n2, L.w_gu))
    return gemm(act, L.w_down, residual=h)


def stack_prefill(x, layers, pools_by_layer, segs: Segments, k: int, cos, sin, eps=1e-5):
    """Selective prefill through a stack of decoder layers (Sec. III-C.2b).
    Layer 1 is computed for every row: its fresh K are scored against the
    layer's aligned cache (score-only pass), the top-k picks the rows, and the
    rows' attention runs over the layer's fresh K/V. Layers 2..L recompute only
    those rows: each layer's cache is assembled (gather + alignment), the rows'
    projected K/V overwrite their positions in it, and the rows attend over
    it. x: [B, N, H] bf16 input states. Returns (hidden [B, R, H] of the
    rows after the last layer, rows, layer-1 scores)."""
    B, N, Hd = x.shape
    L0 = layers[0]
    Hkv = pools_by_layer[0][0][0].shape[2]
    D = pools_by_layer[0][0][0].shape[3]
    Hq = L0.w_o.shape[1] // D
    R = segs.n_fresh + int(k)
    dev, dt = x.device, x.dtype
    # ---- layer 1, every row
    n = rmsnorm(x.view(B * N, Hd), L0.g_attn, eps)
    qkv = gemm(n, L0.w_qkv)
    q = torch.empty((B, N, Hq, D), dtype=dt, device=dev)
    k1 = torch.empty((B, N, Hkv, D), dtype=dt, device=dev)
    v1 = torch.empty_like(k1)
    qkv_rope(qkv, B, N, Hq, Hkv, D, None, cos, sin, q, k1, v1)
    del qkv, n
    scores = torch.empty((B, N), dtype=torch.float32, device=dev)
    kv_assemble(pools_by_layer[0], segs, k1, v1, cos, sin, scores_out=scores, score_only=True)
    rows, _ = select_tokens(segs, k, k1, v1, None, None, scores_in=scores, patch=False)
    attn = selective_attention(q, k1, v1, rows)
    x_rows = gather_rows(x, rows).view(B * R, Hd)
    h = gemm(attn.view(B * R, Hq * D), L0.w_o, residual=x_rows)
    xs = _mlp_and_residual(h, L0, eps)
    # ---- layers 2..L, the selected rows only
    zeros = torch.zeros((B, N, Hkv, D), dtype=dt, device=dev)  # fresh positions are all rows
    for L, pools in zip(layers[1:], pools_by_layer[1:]):
        k_asm, v_asm = kv_assemble(pools, segs, zeros, zeros, cos, sin)
        n = rmsnorm(xs, L.g_attn, eps)
        qkv = gemm(n, L.w_qkv)
        qkv_rope(qkv, B, N, Hq, Hkv, D, rows, cos, sin, q, k_asm, v_asm)
        attn = selective_attention(q, k_asm, v_asm, rows)
        h = gemm(attn.view(B * R, Hq * D), L.w_o, residual=xs)
        xs = _mlp_and_residual(h, L, eps)
    return xs.view(B, R, Hd), rows, scores


def stack_full(x, layers, Hq, Hkv, D, cos, sin, eps=1e-5):
    """Full recompute through the stack: every row of every layer over fresh
    K/V. Returns hidden [B, N, H] after the last layer."""
    B, N, Hd = x.shape
    dev, dt = x.device, x.dtype
    q = torch.empty((B, N, Hq, D), dtype=dt, device=dev)
    kk = torch.empty((B, N, Hkv, D), dtype=dt, device=dev)
    vv = torch.empty_like(kk)
    xs = x.reshape(B * N, Hd)
    for L in layers:
        n = rmsnorm(xs, L.g_attn, eps)
        qkv_rope(gemm(n, L.w_qkv), B, N, Hq, Hkv, D, None, cos, sin, q, kk, vv)
        attn = selective_attention(q, kk, vv)
        h = gemm(attn.view(B * N, Hq * D), L.w_o, residual=xs)
        xs = _mlp_and_residual(h, L, eps)
    return xs.view(B, N, Hd)
