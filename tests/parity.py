"""Shared helpers for the GPU parity tests: run the HIP path step by step
through the C ABI and compare every intermediate with the CPU oracle on the
same seeded inputs."""
from __future__ import annotations

import sys

import numpy as np
import torch

from oracle import oracle as O
from paper_2605_07443_amd import inputs, ops

H = inputs.to_host_bits

# tolerances for attention outputs (fp32 accumulation)
BF16_MAX, BF16_MEAN = 2e-2, 2e-3
F32_MAX = 1e-4


def say(msg: str) -> None:
    print(msg, flush=True)
    sys.stdout.flush()


def assert_attn_close(gpu: np.ndarray, ref: np.ndarray, dtype: str, what: str = "") -> dict:
    g, r = O.as_f32(gpu).astype(np.float64), O.as_f32(ref).astype(np.float64)
    assert g.shape == r.shape, (g.shape, r.shape)
    assert np.all(np.isfinite(g)), f"{what}: non-finite GPU output"
    err = np.abs(g - r)
    mx, mean = float(err.max()) if err.size else 0.0, float(err.mean()) if err.size else 0.0
    if dtype == "bf16":
        assert mx <= BF16_MAX and mean <= BF16_MEAN, f"{what}: max {mx:.3e} mean {mean:.3e}"
    else:
        assert mx <= F32_MAX, f"{what}: max {mx:.3e}"
    return dict(max=mx, mean=mean)


def sample_rows(B: int, R: int, stride: int):
    """All rows of the first and last request, every `stride`-th row elsewhere."""
    out = []
    for b in range(B):
        idx = np.arange(R) if b in (0, B - 1) or stride <= 1 else np.arange(0, R, stride)
        out.append(idx)
    return out


def oracle_attention_rows(q, k, v, rows, sel):
    """Oracle attention for rows[b][sel[b]] of each request b (one request at a time)."""
    res = []
    for b, idx in enumerate(sel):
        r = np.ascontiguousarray(rows[b:b + 1, idx])
        res.append(O.attention(q[b:b + 1], k[b:b + 1], v[b:b + 1], rows=r)[0])
    return res


def run_stepwise(cfg, w, k: int, device, stride: int = 1, check_attention: bool = True):
    """Run assemble -> select (score, top-k, patch) -> attention on the GPU and
    check each step against the oracle. Returns a dict of error statistics."""
    stats = {}
    segs = ops.prepare_segments(w.segs, cfg.N, w.pools, device)
    cos, sin = ops.rope_table(cfg.N, cfg.D, cfg.rope_base, device)
    fused = torch.empty((cfg.B, cfg.N), dtype=torch.float32, device=device)
    k_asm, v_asm = ops.kv_assemble(w.pools, segs, w.k_fresh, w.v_fresh, cos, sin,
                                   scores_out=fused)
    k_pre, v_pre = k_asm.clone(), v_asm.clone()
    # scores computed by rc_select_tokens' own deviation kernel drive this run
    rows, scores = ops.select_tokens(segs, k, w.k_fresh, w.v_fresh, k_asm, v_asm, patch=True)
    out = ops.selective_attention(w.q, k_asm, v_asm, rows) if rows.shape[1] > 0 else None
    torch.cuda.synchronize()

    # ---- (i)+(ii) assembly with fused re-alignment: bit-exact
    ocos, osin = O.rope_table(cfg.N, cfg.D, cfg.rope_base)
    subpools, segs_sub = inputs.referenced_subpools(w)
    kf, vf = H(w.k_fresh), H(w.v_fresh)
    ka_o, va_o = O.assemble(kf, vf, subpools, segs_sub, ocos, osin)
    np.testing.assert_array_equal(H(k_pre), ka_o, err_msg="assembled K differs")
    np.testing.assert_array_equal(H(v_pre), va_o, err_msg="assembled V differs")

    # ---- deviation scores: fp32 accumulation vs fp64
    sc_g = scores.cpu().numpy()
    sc_o = O.deviation(kf, ka_o)
    np.testing.assert_allclose(sc_g, sc_o, rtol=1e-5, atol=1e-5, err_msg="deviation scores")
    sc_f = fused.cpu().numpy()
    np.testing.assert_allclose(sc_f, sc_o, rtol=1e-5, atol=1e-5,
                               err_msg="deviation scores fused into the gather")
    stats["score_rel"] = float(np.max(np.abs(sc_g - sc_o) / np.maximum(np.abs(sc_o), 1e-30)))
    stats["fused_score_rel"] = float(np.max(np.abs(sc_f - sc_o) / np.maximum(np.abs(sc_o), 1e-30)))

    # ---- top-k: bit-exact on identical scores, both ways
    segs_h = w.segs.numpy()
    rows_g = rows.cpu().numpy()
    np.testing.assert_array_equal(rows_g, O.topk(segs_h, cfg.N, k, sc_g),
                                  err_msg="GPU rows differ from oracle top-k of the GPU scores")
    sc_in = torch.from_numpy(sc_o).to(device)
    rows_g2, _ = ops.select_tokens(segs, k, w.k_fresh, w.v_fresh, k_asm, v_asm, scores_in=sc_in,
                                   patch=False)
    np.testing.assert_array_equal(rows_g2.cpu().numpy(), O.topk(segs_h, cfg.N, k, sc_o),
                                  err_msg="GPU top-k of the oracle scores differs")
    rows_g3, _ = ops.select_tokens(segs, k, w.k_fresh, w.v_fresh, k_asm, v_asm, scores_in=fused,
                                   patch=False)
    np.testing.assert_array_equal(rows_g3.cpu().numpy(), O.topk(segs_h, cfg.N, k, sc_f),
                                  err_msg="GPU top-k of the fused scores differs")
    stats["rows_agree_own_scores"] = float(np.mean(rows_g == O.topk(segs_h, cfg.N, k, sc_o)))

    # ---- (iii) patch: bit-exact
    kp_o, vp_o = O.patch(segs_h, rows_g, kf, vf, ka_o, va_o)
    np.testing.assert_array_equal(H(k_asm), kp_o, err_msg="patched K differs")
    np.testing.assert_array_equal(H(v_asm), vp_o, err_msg="patched V differs")

    # ---- attention of the selected rows
    if check_attention and out is not None:
        qh = H(w.q)
        sel = sample_rows(cfg.B, rows_g.shape[1], stride)
        ref = oracle_attention_rows(qh, kp_o, vp_o, rows_g, sel)
        outh = H(out)
        g = np.concatenate([outh[b, idx] for b, idx in enumerate(sel)])
        r = np.concatenate(ref)
        stats.update(assert_attn_close(g, r, cfg.dtype, "selective attention"))
    return stats, dict(segs=segs, cos=cos, sin=sin, k_asm=k_asm, v_asm=v_asm, rows=rows,
                       scores=scores, out=out)


# ------------------------------------------------------------ Eq. (3) selection

# log-sum-exp: scores of bf16/fp32 inputs accumulated in fp32 (bf16 products
# are exact in fp32), exponentials and their sums in fp32, so the error is a
# few fp32 ulps of the score scale (|lse| < 30): measured <= 1.7e-6 on every
# workload. Mass: each weight exp(s - lse) carries the lse and exp2 errors
# (relative, a few 1e-7 .. 1e-6) and is summed in fp32: measured <= 1.3e-6
# relative. The bounds below leave a margin of about 10x.
LSE_ATOL = 2e-5
MASS_RTOL, MASS_ATOL = 2e-5, 1e-6


def group_slice(q, k, g, G):
    """Q heads and the K head of KV group g (oracle cost of one group)."""
    return (np.ascontiguousarray(q[:, :, g * G:(g + 1) * G]), np.ascontiguousarray(k[:, :, g:g + 1]))


def run_eq3_stepwise(cfg, w, lam, k_hist, k_item, device, check_requests=None, check_groups=None):
    """First layer in full with lse -> mass -> assemble -> Eq. (3) score ->
    split top-k -> patch on the GPU; each step checked against the oracle.
    check_requests / check_groups bound the oracle's quadratic work (None:
    all)."""
    stats = {}
    G = cfg.Hq // cfg.Hkv
    mask = inputs.ITEM_POOL_MASK
    lam = float(np.float32(lam))
    segs = ops.prepare_segments(w.segs, cfg.N, w.pools, device)
    cos, sin = ops.rope_table(cfg.N, cfg.D, cfg.rope_base, device)
    bufs = ops.eq3_select(w.q, w.k_fresh, w.v_fresh, w.pools, segs, mask, lam, k_hist, k_item,
                          cos, sin)
    torch.cuda.synchronize()
    qh, kf, vf = H(w.q), H(w.k_fresh), H(w.v_fresh)
    lse_g = bufs.lse.cpu().numpy()
    mass_g = bufs.mass.cpu().numpy()
    reqs = range(cfg.B) if check_requests is None else check_requests
    groups = range(cfg.Hkv) if check_groups is None else check_groups

    # ---- the first layer's log-sum-exp and attention mass
    lse_err, mass_rel = 0.0, 0.0
    for b in reqs:
        for g in groups:
            qg, kg = group_slice(qh[b:b + 1], kf[b:b + 1], g, G)
            lse_o = O.attention_lse(qg, kg)[0]                       # N, G
            d = np.abs(lse_g[b, :, g * G:(g + 1) * G] - lse_o)
            assert d.max() <= LSE_ATOL, f"lse b={b} g={g}: max err {d.max():.3e}"
            lse_err = max(lse_err, float(d.max()))
            m_o = O.attention_mass(qg, kg)[0, 0]                      # N
            np.testing.assert_allclose(mass_g[b, g], m_o, rtol=MASS_RTOL, atol=MASS_ATOL,
                                       err_msg=f"mass b={b} g={g}")
            mass_rel = max(mass_rel, float(np.max(np.abs(mass_g[b, g] - m_o) / np.maximum(m_o, 1e-6))))
    # every row's weights sum to 1: each group's mass sums to G * N
    np.testing.assert_allclose(mass_g.astype(np.float64).sum(-1), G * cfg.N, rtol=1e-5)
    stats.update(lse_max_err=lse_err, mass_max_rel=mass_rel)

    # ---- assembly: bit-exact (the Eq. (3) path assembles without scoring)
    ocos, osin = O.rope_table(cfg.N, cfg.D, cfg.rope_base)
    subpools, segs_sub = inputs.referenced_subpools(w)
    ka_o, va_o = O.assemble(kf, vf, subpools, segs_sub, ocos, osin)

    # ---- score from the GPU's mass: fp32 vs fp64
    segs_h = w.segs.numpy()
    sc_g = bufs.scores.cpu().numpy()
    sc_o = O.score_eq3(segs_h, mask, lam, mass_g, kf, vf, ka_o, va_o)
    np.testing.assert_allclose(sc_g, sc_o, rtol=1e-5, atol=1e-5, err_msg="Eq. (3) scores")
    stats["score_rel"] = float(np.max(np.abs(sc_g - sc_o) / np.maximum(np.abs(sc_o), 1e-30)))

    # ---- split top-k: bit-exact on identical scores, both ways
    rows_g = bufs.rows.cpu().numpy()
    np.testing.assert_array_equal(rows_g, O.topk_split(segs_h, cfg.N, mask, k_hist, k_item, sc_g),
                                  err_msg="GPU rows differ from the oracle split top-k of the GPU scores")
    k_asm2, v_asm2 = ops.kv_assemble(w.pools, segs, w.k_fresh, w.v_fresh, cos, sin)
    rows2, _ = ops.select_tokens_eq3(segs, mask, lam, k_hist, k_item, w.k_fresh, w.v_fresh, k_asm2,
                                     v_asm2, scores_in=torch.from_numpy(sc_o).to(device), patch=False)
    np.testing.assert_array_equal(rows2.cpu().numpy(),
                                  O.topk_split(segs_h, cfg.N, mask, k_hist, k_item, sc_o),
                                  err_msg="GPU split top-k of the oracle scores differs")
    np.testing.assert_array_equal(H(k_asm2), ka_o, err_msg="assembled K differs")
    np.testing.assert_array_equal(H(v_asm2), va_o, err_msg="assembled V differs")

    # ---- patch: bit-exact
    kp_o, vp_o = O.patch(segs_h, rows_g, kf, vf, ka_o, va_o)
    np.testing.assert_array_equal(H(bufs.k_asm), kp_o, err_msg="patched K differs")
    np.testing.assert_array_equal(H(bufs.v_asm), vp_o, err_msg="patched V differs")
    return stats, bufs
