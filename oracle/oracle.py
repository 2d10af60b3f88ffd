"""Python bindings of the CPU oracle (``rcref.c``) for RcLLM's selective prefill.

TEST INFRASTRUCTURE ONLY: the test suite, the smoke check and the benchmark's
CPU-baseline leg are its only users. The GPU path never imports it.

Every function takes and returns host numpy arrays. Storage dtypes: ``float32``
arrays are fp32 tensors; ``uint16`` arrays hold bf16 bit patterns. Layouts are
the token-major layouts documented in ``rcref.c``.

Paper passages followed (arXiv 2605.07443):
  * Sec. III-C.3, end-to-end prefill pipeline: (i) assembly, (ii) alignment by
    RoPE rotation, (iii) heavy-hitter update;
  * Sec. III-C.2b and Eq. (3): importance score (deviation term, K only,
    lambda = 1) and the heavy-hitter top-k; the full score (attention mass of
    the first layer computed in full, K and V divergence, lambda, no divergence
    for item blocks) with separate history and item budgets (Sec. IV-A);
  * Eq. (1): scaled dot-product attention, causal, grouped-query;
  * Sec. IV-A: Full-Recompute baseline (every row recomputed);
  * Sec. III-C.2b, several layers: the first computed in full, later layers
    recomputing only the selected rows over their aligned caches.
"""
from __future__ import annotations

import ctypes
import os
import subprocess

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
SRC_PATH = os.path.join(_HERE, "rcref.c")
# RCREF_LIB names another build of rcref.c (the sanitizer test loads an
# ASan/UBSan build this way)
LIB_PATH = os.environ.get("RCREF_LIB") or os.path.join(_HERE, "librcref.so")

_lib = None


def build(force: bool = True) -> str:
    """Compile ``rcref.c`` with gcc: no FMA contraction, no fast-math, OpenMP."""
    if not force and os.path.exists(LIB_PATH):
        return LIB_PATH
    tmp = LIB_PATH + ".tmp"
    cmd = ["gcc", "-O2", "-std=c11", "-fPIC", "-shared", "-fopenmp", "-ffp-contract=off",
           "-fno-fast-math", "-Wall", "-Wextra", "-o", tmp, SRC_PATH, "-lm"]
    subprocess.run(cmd, check=True)
    os.replace(tmp, LIB_PATH)
    return LIB_PATH


def lib():
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            build()
        L = ctypes.CDLL(LIB_PATH)
        vp, i32, f64 = ctypes.c_void_p, ctypes.c_int, ctypes.c_double
        L.rcref_rope_table.argtypes = [i32, i32, f64, vp, vp]
        L.rcref_assemble.argtypes = [i32, i32, i32, i32, i32, vp, vp, vp, vp, i32, vp, i32,
                                     vp, vp, vp, vp, vp, vp]
        L.rcref_rerope.argtypes = [i32, i32, i32, i32, i32, vp, vp, vp, vp]
        L.rcref_deviation.argtypes = [i32, i32, i32, i32, i32, vp, vp, vp]
        L.rcref_topk.argtypes = [i32, i32, vp, i32, i32, vp, vp]
        L.rcref_topk.restype = i32
        L.rcref_patch.argtypes = [i32, i32, i32, i32, i32, vp, i32, vp, i32, vp, vp, vp, vp]
        L.rcref_attention.argtypes = [i32, i32, i32, i32, i32, i32, vp, vp, i32, vp, vp, f64, vp]
        L.rcref_selective_prefill.argtypes = [i32, i32, i32, i32, i32, i32, vp, vp, vp, vp, i32,
                                              vp, i32, i32, vp, vp, vp, vp, vp, f64,
                                              vp, vp, vp, vp, vp]
        L.rcref_selective_prefill.restype = i32
        L.rcref_attention_lse.argtypes = [i32, i32, i32, i32, i32, i32, vp, vp, f64, vp]
        L.rcref_attention_mass.argtypes = [i32, i32, i32, i32, i32, i32, vp, vp, f64, vp]
        u32 = ctypes.c_uint32
        L.rcref_score_eq3.argtypes = [i32, i32, i32, i32, i32, vp, i32, u32, f64, vp, vp, vp, vp,
                                      vp, vp]
        L.rcref_topk_split.argtypes = [i32, i32, vp, i32, u32, i32, i32, vp, vp]
        L.rcref_topk_split.restype = i32
        L.rcref_eq3_select.argtypes = [i32, i32, i32, i32, i32, i32, vp, vp, vp, vp, i32, vp, i32,
                                       u32, f64, i32, i32, vp, vp, vp, vp, vp, f64, vp, vp, vp,
                                       vp, vp]
        L.rcref_eq3_select.restype = i32
        L.rcref_gather_tokens.argtypes = [i32, i32, i32, i32, i32, vp, vp, vp, vp, vp, vp, vp, vp,
                                          vp]
        L.rcref_num_threads.argtypes = []
        L.rcref_num_threads.restype = i32
        _lib = L
    return _lib


def num_threads() -> int:
    """OpenMP threads the oracle's parallel loops use."""
    return int(lib().rcref_num_threads())


def _dt(a: np.ndarray) -> int:
    if a.dtype == np.float32:
        return 0
    if a.dtype == np.uint16:
        return 1
    raise TypeError(f"storage dtype must be float32 or uint16 (bf16 bits), got {a.dtype}")


def _p(a):
    return None if a is None else a.ctypes.data_as(ctypes.c_void_p)


def _c(a, dtype=None):
    return np.ascontiguousarray(a if dtype is None else a.astype(dtype, copy=False))


def fresh_count(segs: np.ndarray) -> np.ndarray:
    """Per-request number of fresh positions (segments with pool < 0)."""
    segs = np.asarray(segs)
    return np.where(segs[..., 2] < 0, segs[..., 1], 0).sum(axis=1)


def rope_table(max_pos: int, D: int, base: float):
    cos = np.empty((max_pos, D // 2), np.float32)
    sin = np.empty((max_pos, D // 2), np.float32)
    lib().rcref_rope_table(max_pos, D, float(base), _p(cos), _p(sin))
    return cos, sin


def assemble(k_fresh, v_fresh, pools, segs, cos=None, sin=None):
    """Gather (and, given tables, re-align) K/V rows. ``pools`` is a list of
    (pool_k, pool_v) arrays of shape [num_blocks, block_len, Hkv, D]."""
    k_fresh, v_fresh = _c(k_fresh), _c(v_fresh)
    B, N, Hkv, D = k_fresh.shape
    dt = _dt(k_fresh)
    segs = _c(segs, np.int32)
    S = segs.shape[1]
    pools = [(_c(pk), _c(pv)) for pk, pv in pools]
    n = len(pools)
    pk_arr = (ctypes.c_void_p * max(n, 1))(*[pk.ctypes.data for pk, _ in pools])
    pv_arr = (ctypes.c_void_p * max(n, 1))(*[pv.ctypes.data for _, pv in pools])
    nb = np.array([pk.shape[0] for pk, _ in pools] or [0], np.int32)
    bl = np.array([pk.shape[1] for pk, _ in pools] or [0], np.int32)
    k_asm = np.empty_like(k_fresh)
    v_asm = np.empty_like(v_fresh)
    cos = None if cos is None else _c(cos, np.float32)
    sin = None if sin is None else _c(sin, np.float32)
    lib().rcref_assemble(B, N, Hkv, D, dt, pk_arr, pv_arr, _p(nb), _p(bl), n, _p(segs), S,
                         _p(k_fresh), _p(v_fresh), _p(cos), _p(sin), _p(k_asm), _p(v_asm))
    return k_asm, v_asm


def gather_tokens(k_fresh, v_fresh, pools, token_map, cos=None, sin=None):
    """Token-granular gather: token_map [B, N, 4] int32 = {pool, row, delta, -};
    pools as for ``assemble`` (rows counted across blocks)."""
    k_fresh, v_fresh = _c(k_fresh), _c(v_fresh)
    B, N, Hkv, D = k_fresh.shape
    token_map = _c(token_map, np.int32)
    pools = [(_c(pk), _c(pv)) for pk, pv in pools]
    n = len(pools)
    pk_arr = (ctypes.c_void_p * max(n, 1))(*[pk.ctypes.data for pk, _ in pools])
    pv_arr = (ctypes.c_void_p * max(n, 1))(*[pv.ctypes.data for _, pv in pools])
    k_asm = np.empty_like(k_fresh)
    v_asm = np.empty_like(v_fresh)
    cos = None if cos is None else _c(cos, np.float32)
    sin = None if sin is None else _c(sin, np.float32)
    lib().rcref_gather_tokens(B, N, Hkv, D, _dt(k_fresh), pk_arr, pv_arr, _p(token_map),
                              _p(k_fresh), _p(v_fresh), _p(cos), _p(sin), _p(k_asm), _p(v_asm))
    return k_asm, v_asm


def rerope(k, delta, cos, sin):
    """Return a copy of K [B,N,Hkv,D] with row (b,i) rotated by delta[b,i]."""
    out = np.array(k, copy=True)
    B, N, Hkv, D = out.shape
    delta = _c(delta, np.int32)
    lib().rcref_rerope(B, N, Hkv, D, _dt(out), _p(out), _p(delta), _p(_c(cos, np.float32)),
                       _p(_c(sin, np.float32)))
    return out


def deviation(k_fresh, k_asm):
    k_fresh, k_asm = _c(k_fresh), _c(k_asm)
    B, N, Hkv, D = k_fresh.shape
    scores = np.empty((B, N), np.float32)
    lib().rcref_deviation(B, N, Hkv, D, _dt(k_fresh), _p(k_fresh), _p(k_asm), _p(scores))
    return scores


def topk(segs, N: int, k: int, scores):
    segs = _c(segs, np.int32)
    B, S = segs.shape[:2]
    F = int(fresh_count(segs)[0])
    scores = _c(scores, np.float32)
    rows = np.empty((B, F + k), np.int32)
    st = lib().rcref_topk(B, N, _p(segs), S, int(k), _p(scores), _p(rows))
    if st != 0:
        raise ValueError("k exceeds the cached positions of a request, or fresh counts differ")
    return rows


def patch(segs, rows, k_fresh, v_fresh, k_asm, v_asm):
    segs = _c(segs, np.int32)
    rows = _c(rows, np.int32)
    k_fresh, v_fresh = _c(k_fresh), _c(v_fresh)
    k_out = np.array(k_asm, copy=True)
    v_out = np.array(v_asm, copy=True)
    B, N, Hkv, D = k_fresh.shape
    lib().rcref_patch(B, N, Hkv, D, _dt(k_fresh), _p(segs), segs.shape[1], _p(rows),
                      rows.shape[1], _p(k_fresh), _p(v_fresh), _p(k_out), _p(v_out))
    return k_out, v_out


def attention(q, k, v, rows=None, scale=None):
    """Causal GQA attention of the listed rows (all rows if ``rows`` is None)."""
    q, k, v = _c(q), _c(k), _c(v)
    B, N, Hq, D = q.shape
    Hkv = k.shape[2]
    if scale is None:
        scale = 1.0 / np.sqrt(D)
    if rows is not None:
        rows = _c(rows, np.int32)
        R = rows.shape[1]
    else:
        R = N
    out = np.empty((B, R, Hq, D), q.dtype)
    lib().rcref_attention(B, N, Hq, Hkv, D, _dt(q), _p(q), _p(rows), R, _p(k), _p(v),
                          float(scale), _p(out))
    return out


def selective_prefill(q, k_fresh, v_fresh, pools, segs, k: int, cos, sin, scale=None):
    """The whole pipeline; returns a dict with every intermediate."""
    q, k_fresh, v_fresh = _c(q), _c(k_fresh), _c(v_fresh)
    B, N, Hq, D = q.shape
    Hkv = k_fresh.shape[2]
    dt = _dt(q)
    segs = _c(segs, np.int32)
    S = segs.shape[1]
    F = int(fresh_count(segs)[0])
    R = F + int(k)
    pools = [(_c(pk), _c(pv)) for pk, pv in pools]
    n = len(pools)
    pk_arr = (ctypes.c_void_p * max(n, 1))(*[pk.ctypes.data for pk, _ in pools])
    pv_arr = (ctypes.c_void_p * max(n, 1))(*[pv.ctypes.data for _, pv in pools])
    nb = np.array([pk.shape[0] for pk, _ in pools] or [0], np.int32)
    bl = np.array([pk.shape[1] for pk, _ in pools] or [0], np.int32)
    if scale is None:
        scale = 1.0 / np.sqrt(D)
    k_asm = np.empty_like(k_fresh)
    v_asm = np.empty_like(v_fresh)
    scores = np.empty((B, N), np.float32)
    rows = np.empty((B, R), np.int32)
    out = np.empty((B, R, Hq, D), q.dtype)
    st = lib().rcref_selective_prefill(
        B, N, Hq, Hkv, D, dt, pk_arr, pv_arr, _p(nb), _p(bl), n, _p(segs), S, int(k), _p(q),
        _p(k_fresh), _p(v_fresh), _p(_c(cos, np.float32)), _p(_c(sin, np.float32)),
        float(scale), _p(k_asm), _p(v_asm), _p(scores), _p(rows), _p(out))
    if st != 0:
        raise ValueError("k exceeds the cached positions of a request, or fresh counts differ")
    return dict(k_asm=k_asm, v_asm=v_asm, scores=scores, rows=rows, out=out)


def pool_mask(item_pools) -> int:
    """Bit mask of the pools whose blocks are items (no divergence term)."""
    m = 0
    for p in item_pools:
        m |= 1 << int(p)
    return m


def attention_lse(q, k, scale=None):
    """Natural log-sum-exp [B, N, Hq] (fp64) of every row's scaled causal scores."""
    q, k = _c(q), _c(k)
    B, N, Hq, D = q.shape
    Hkv = k.shape[2]
    scale = 1.0 / np.sqrt(D) if scale is None else scale
    lse = np.empty((B, N, Hq), np.float64)
    lib().rcref_attention_lse(B, N, Hq, Hkv, D, _dt(q), _p(q), _p(k), float(scale), _p(lse))
    return lse


def attention_mass(q, k, scale=None):
    """Attention mass [B, Hkv, N] (fp64) each key receives per KV group."""
    q, k = _c(q), _c(k)
    B, N, Hq, D = q.shape
    Hkv = k.shape[2]
    scale = 1.0 / np.sqrt(D) if scale is None else scale
    mass = np.empty((B, Hkv, N), np.float64)
    lib().rcref_attention_mass(B, N, Hq, Hkv, D, _dt(q), _p(q), _p(k), float(scale), _p(mass))
    return mass


def score_eq3(segs, item_mask: int, lam: float, mass, k_fresh, v_fresh, k_asm, v_asm):
    """Eq. (3) scores [B, N] fp32 from fp32 mass [B, Hkv, N]."""
    segs = _c(segs, np.int32)
    k_fresh, v_fresh, k_asm, v_asm = _c(k_fresh), _c(v_fresh), _c(k_asm), _c(v_asm)
    B, N, Hkv, D = k_fresh.shape
    mass = _c(mass, np.float32)
    scores = np.empty((B, N), np.float32)
    lib().rcref_score_eq3(B, N, Hkv, D, _dt(k_fresh), _p(segs), segs.shape[1], int(item_mask),
                          float(lam), _p(mass), _p(k_fresh), _p(v_fresh), _p(k_asm), _p(v_asm),
                          _p(scores))
    return scores


def topk_split(segs, N: int, item_mask: int, k_hist: int, k_item: int, scores):
    """Separate history / item top-k; rows [B, F + k_hist + k_item] ascending."""
    segs = _c(segs, np.int32)
    B, S = segs.shape[:2]
    F = int(fresh_count(segs)[0])
    scores = _c(scores, np.float32)
    rows = np.empty((B, F + k_hist + k_item), np.int32)
    st = lib().rcref_topk_split(B, N, _p(segs), S, int(item_mask), int(k_hist), int(k_item),
                                _p(scores), _p(rows))
    if st != 0:
        raise ValueError("a budget exceeds its component's cached positions, or fresh counts differ")
    return rows


def eq3_select(q, k_fresh, v_fresh, pools, segs, item_mask: int, lam: float, k_hist: int,
               k_item: int, cos, sin, scale=None):
    """Selection by the full Eq. (3) score; returns every intermediate."""
    q, k_fresh, v_fresh = _c(q), _c(k_fresh), _c(v_fresh)
    B, N, Hq, D = q.shape
    Hkv = k_fresh.shape[2]
    segs = _c(segs, np.int32)
    S = segs.shape[1]
    F = int(fresh_count(segs)[0])
    R = F + int(k_hist) + int(k_item)
    pools = [(_c(pk), _c(pv)) for pk, pv in pools]
    n = len(pools)
    pk_arr = (ctypes.c_void_p * max(n, 1))(*[pk.ctypes.data for pk, _ in pools])
    pv_arr = (ctypes.c_void_p * max(n, 1))(*[pv.ctypes.data for _, pv in pools])
    nb = np.array([pk.shape[0] for pk, _ in pools] or [0], np.int32)
    bl = np.array([pk.shape[1] for pk, _ in pools] or [0], np.int32)
    scale = 1.0 / np.sqrt(D) if scale is None else scale
    k_asm = np.empty_like(k_fresh)
    v_asm = np.empty_like(v_fresh)
    mass = np.empty((B, Hkv, N), np.float32)
    scores = np.empty((B, N), np.float32)
    rows = np.empty((B, R), np.int32)
    st = lib().rcref_eq3_select(
        B, N, Hq, Hkv, D, _dt(q), pk_arr, pv_arr, _p(nb), _p(bl), n, _p(segs), S, int(item_mask),
        float(lam), int(k_hist), int(k_item), _p(q), _p(k_fresh), _p(v_fresh),
        _p(_c(cos, np.float32)), _p(_c(sin, np.float32)), float(scale), _p(k_asm), _p(v_asm),
        _p(mass), _p(scores), _p(rows))
    if st != 0:
        raise ValueError("a budget exceeds its component's cached positions, or fresh counts differ")
    return dict(k_asm=k_asm, v_asm=v_asm, mass=mass, scores=scores, rows=rows)


def position_map(segs_b, N: int) -> list:
    """Per position of one request: None (fresh) or (pool, block row, rotation
    delta) -- the row the position reads and the angle it is aligned by."""
    m = [None] * N
    for dst, ln, p, blk in np.asarray(segs_b).tolist():
        for t in range(ln):
            m[dst + t] = None if p < 0 else (p, blk, t, dst)
    return m


def segments_with_window(segs, N: int, W: int) -> np.ndarray:
    """The local sliding window (Sec. III-C.2b: heavy hitters and the local
    sliding window are recomputed): positions [N - W, N) of every request
    become fresh. Segments are clipped at N - W and one fresh segment covers
    the window; requests with fewer segments split their window segment so
    that the table stays [B, S] (a cached segment is never split: its
    dst_start fixes both the block offset and the rotation)."""
    segs = np.asarray(segs, np.int32)
    cut = N - W
    tables = []
    for req in segs.tolist():
        runs = []
        for dst, ln, p, blk in req:
            end = min(dst + ln, cut)
            if dst < end:
                runs.append([dst, end - dst, p, blk])
        if W > 0:
            runs.append([cut, W, -1, 0])
        tables.append(runs)
    S = max(len(t) for t in tables)
    out = np.zeros((len(tables), S, 4), np.int32)
    for b, runs in enumerate(tables):
        while len(runs) < S:
            dst, ln, p, blk = runs[-1]
            if p >= 0 or ln < 2:
                raise ValueError("the window is too short to pad the segment table")
            runs[-1:] = [[dst, ln - 1, -1, 0], [dst + ln - 1, 1, -1, 0]]
        out[b] = np.array(runs, np.int32)
    return out


# ---------------------------------------------------------------------------
# Several layers: the first computed in full, later ones only for the
# selected rows (Sec. III-C.2b), with pre-norm decoder layers
# ---------------------------------------------------------------------------

def f64(a):
    """Storage array (fp32, or bf16 bits) as fp64 values."""
    a = np.asarray(a)
    return as_f32(a).astype(np.float64) if a.dtype in (np.uint16, np.float32) else a.astype(np.float64)


def rmsnorm64(x, gamma, eps):
    x = np.asarray(x, np.float64)
    return x / np.sqrt(np.mean(x * x, axis=-1, keepdims=True) + eps) * np.asarray(gamma, np.float64)


def silu_mul64(gu):
    gu = np.asarray(gu, np.float64)
    I = gu.shape[-1] // 2
    g, u = gu[..., :I], gu[..., I:]
    return g / (1.0 + np.exp(-g)) * u


def rope_at(x, pos, base):
    """Rotate-half rotary encoding of x [..., T, H, D] at absolute positions
    pos [..., T], angles pos * base^(-2j/D), in fp64."""
    x = np.asarray(x, np.float64)
    D = x.shape[-1]
    half = D // 2
    inv = base ** (-2.0 * np.arange(half) / D)
    ang = np.asarray(pos, np.float64)[..., None, None] * inv
    c, sn = np.cos(ang), np.sin(ang)
    a, b = x[..., :half], x[..., half:]
    return np.concatenate([a * c - b * sn, a * sn + b * c], axis=-1)


def _attend(q, k, v, rows):
    """Causal GQA attention (the pinned oracle, fp32 storage of fp64 values)."""
    return f64(attention(q.astype(np.float32), k.astype(np.float32), v.astype(np.float32),
                         rows=None if rows is None else np.ascontiguousarray(rows, np.int32)))


def _layer_w(L):
    return {k: f64(v) for k, v in L.items()}


def decoder_stack_full(x, layers, Hq, Hkv, D, rope_base, eps, return_kv=False):
    """Every row through every layer: h = x + O(attn(norm(x))), x' = h +
    down(silu(gate) * up)(norm(h)). layers: dicts of storage arrays w_qkv,
    w_o, w_gu, w_down, g_attn, g_mlp. Returns [B, N, H] fp64 (and each
    layer's pre-rotation keys and values)."""
    X = f64(x)
    B, N, _ = X.shape
    pos = np.broadcast_to(np.arange(N), (B, N))
    kv = []
    for L in layers:
        W = _layer_w(L)
        qkv = rmsnorm64(X, W["g_attn"], eps) @ W["w_qkv"].T
        q = qkv[..., :Hq * D].reshape(B, N, Hq, D)
        kr = qkv[..., Hq * D:(Hq + Hkv) * D].reshape(B, N, Hkv, D)
        v = qkv[..., (Hq + Hkv) * D:].reshape(B, N, Hkv, D)
        kv.append((kr, v))
        att = _attend(rope_at(q, pos, rope_base), rope_at(kr, pos, rope_base), v, None)
        h = X + att.reshape(B, N, Hq * D) @ W["w_o"].T
        X = h + silu_mul64(rmsnorm64(h, W["g_mlp"], eps) @ W["w_gu"].T) @ W["w_down"].T
    return (X, kv) if return_kv else X


def decoder_stack_selective(x, layers, pools_by_layer, segs, rows, cos, sin, Hq, rope_base, eps,
                            dt=1):
    """The stack for the listed rows [B, R] (the selection is made by the
    caller): layer 1 runs every row's projections and attends the listed rows
    over its fresh K/V; layers 2..L project only the listed rows, put their
    rotated keys and values into the layer's aligned cache (pinned assembly of
    its pools, storage dtype dt) and attend over it. Returns the listed rows'
    states [B, R, H] fp64 and layer 1's rotated keys [B, N, Hkv, D] fp64."""
    X = f64(x)
    B, N, Hd = X.shape
    rows = np.asarray(rows)
    R = rows.shape[1]
    pool0 = pools_by_layer[0][0][0]
    Hkv, D = pool0.shape[2], pool0.shape[3]
    pos = np.broadcast_to(np.arange(N), (B, N))
    bidx = np.arange(B)[:, None]
    W = _layer_w(layers[0])
    qkv = rmsnorm64(X, W["g_attn"], eps) @ W["w_qkv"].T
    q = rope_at(qkv[..., :Hq * D].reshape(B, N, Hq, D), pos, rope_base)
    k1 = rope_at(qkv[..., Hq * D:(Hq + Hkv) * D].reshape(B, N, Hkv, D), pos, rope_base)
    v1 = qkv[..., (Hq + Hkv) * D:].reshape(B, N, Hkv, D)
    att = _attend(q, k1, v1, rows)
    h = X[bidx, rows] + att.reshape(B, R, Hq * D) @ W["w_o"].T
    xs = h + silu_mul64(rmsnorm64(h, W["g_mlp"], eps) @ W["w_gu"].T) @ W["w_down"].T
    store = (lambda a: f32_to_bf16(a.astype(np.float32))) if dt == 1 else (lambda a: a.astype(np.float32))
    zeros = store(np.zeros((B, N, Hkv, D)))
    for L, pools in zip(layers[1:], pools_by_layer[1:]):
        W = _layer_w(L)
        ka, va = assemble(zeros, zeros, pools, segs, cos, sin)
        ka, va = f64(ka), f64(va)
        qkv = rmsnorm64(xs, W["g_attn"], eps) @ W["w_qkv"].T
        qf = np.zeros((B, N, Hq, D))
        qf[bidx, rows] = rope_at(qkv[..., :Hq * D].reshape(B, R, Hq, D), rows, rope_base)
        ka[bidx, rows] = rope_at(qkv[..., Hq * D:(Hq + Hkv) * D].reshape(B, R, Hkv, D), rows, rope_base)
        va[bidx, rows] = qkv[..., (Hq + Hkv) * D:].reshape(B, R, Hkv, D)
        att = _attend(qf, ka, va, rows)
        h = xs + att.reshape(B, R, Hq * D) @ W["w_o"].T
        xs = h + silu_mul64(rmsnorm64(h, W["g_mlp"], eps) @ W["w_gu"].T) @ W["w_down"].T
    return xs, k1


# ---------------------------------------------------------------------------
# bf16 conversions for host-side comparisons (exact widening; RNE narrowing)
# ---------------------------------------------------------------------------

def bf16_to_f32(a: np.ndarray) -> np.ndarray:
    return (np.asarray(a, np.uint16).astype(np.uint32) << 16).view(np.float32)


def f32_to_bf16(a: np.ndarray) -> np.ndarray:
    u = np.ascontiguousarray(a, np.float32).view(np.uint32).astype(np.uint64)
    nan = (u & 0x7FFFFFFF) > 0x7F800000
    r = ((u + 0x7FFF + ((u >> 16) & 1)) >> 16).astype(np.uint16)
    return np.where(nan, ((u >> 16) | 0x40).astype(np.uint16), r)


def as_f32(a: np.ndarray) -> np.ndarray:
    return bf16_to_f32(a) if a.dtype == np.uint16 else np.asarray(a, np.float32)
