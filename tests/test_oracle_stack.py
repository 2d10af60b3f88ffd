"""Pins for the oracle's decoder stack (arXiv 2605.07443, Sec. III-C.2b: the
first layer computed in full, later layers recomputing only the selected
rows over cached K/V): closed forms, agreement with separately pinned oracle
functions, and the invariants the method must satisfy (every row selected ==
full recompute; a cache holding exactly the full computation's K/V makes the
selected rows exact)."""
import math

import numpy as np
import pytest

from oracle import oracle as O
from paper_2605_07443_amd import inputs

EPS = 1e-5


def _weights(n_layers, H, Hq, Hkv, D, I, seed, zero_out=False, dt="f32"):
    rng = np.random.default_rng(seed)
    layers = []
    for _ in range(n_layers):
        def w(r, c):
            a = (rng.standard_normal((r, c)) / math.sqrt(c)).astype(np.float32)
            return O.f32_to_bf16(a) if dt == "bf16" else a
        L = dict(w_qkv=w((Hq + 2 * Hkv) * D, H), w_o=w(H, Hq * D), w_gu=w(2 * I, H),
                 w_down=w(H, I), g_attn=(1 + 0.1 * rng.standard_normal(H)).astype(np.float32),
                 g_mlp=(1 + 0.1 * rng.standard_normal(H)).astype(np.float32))
        if zero_out:
            L["w_o"] = np.zeros_like(L["w_o"])
            L["w_down"] = np.zeros_like(L["w_down"])
        layers.append(L)
    return layers


def test_rmsnorm_and_silu_closed_forms():
    rng = np.random.default_rng(1)
    x = rng.standard_normal((5, 64)) * 3.0
    y = O.rmsnorm64(x, np.ones(64), 0.0)
    np.testing.assert_allclose(np.sqrt(np.mean(y * y, -1)), 1.0, rtol=1e-12)
    np.testing.assert_allclose(O.rmsnorm64(7.5 * x, np.ones(64), 0.0), y, rtol=1e-12)
    g = np.array([[0.0, 1.0, -1.0, 40.0, -40.0, 2.0, 2.0, 2.0, 2.0, 2.0]])
    gu = np.concatenate([g, np.ones_like(g)], -1)
    want = np.array([0.0, 1 / (1 + math.exp(-1)), -1 / (1 + math.e), 40.0, 0.0, 2 / (1 + math.exp(-2)),
                     2 / (1 + math.exp(-2)), 2 / (1 + math.exp(-2)), 2 / (1 + math.exp(-2)),
                     2 / (1 + math.exp(-2))])
    np.testing.assert_allclose(O.silu_mul64(gu)[0], want, rtol=1e-12, atol=1e-15)


def test_rope_at_matches_the_pinned_rotation():
    """fp64 rotation at absolute positions vs the pinned table-driven
    rotation (fp32 tables, fp32 arithmetic): equal to fp32 rounding."""
    B, N, H, D = 2, 33, 3, 64
    x = np.random.default_rng(2).standard_normal((B, N, H, D)).astype(np.float32)
    cos, sin = O.rope_table(N, D, 10000.0)
    delta = np.broadcast_to(np.arange(N, dtype=np.int32), (B, N)).copy()
    want = O.rerope(x, delta, cos, sin)
    got = O.rope_at(x, np.broadcast_to(np.arange(N), (B, N)), 10000.0)
    np.testing.assert_allclose(got, want, rtol=0, atol=2e-6)


def _small_case(seed=3, n_layers=3):
    cfg = inputs.TEST_WORKLOADS["tiny-f32-gqa"]
    w = inputs.make(cfg, seed)
    H, I = 96, 128
    x = np.random.default_rng(seed).standard_normal((cfg.B, cfg.N, H)).astype(np.float32)
    return cfg, w, x, H, I


def test_zero_output_projections_make_the_stack_the_identity():
    cfg, w, x, H, I = _small_case()
    layers = _weights(3, H, cfg.Hq, cfg.Hkv, cfg.D, I, 4, zero_out=True)
    full = O.decoder_stack_full(x, layers, cfg.Hq, cfg.Hkv, cfg.D, cfg.rope_base, EPS)
    np.testing.assert_array_equal(full, x.astype(np.float64))
    cos, sin = O.rope_table(cfg.N, cfg.D, cfg.rope_base)
    pools = [[(a.numpy(), b.numpy()) for a, b in w.pools]] * 3
    rows = O.topk(w.segs.numpy(), cfg.N, cfg.k, np.random.default_rng(5).random((cfg.B, cfg.N)).astype(np.float32))
    sel, _ = O.decoder_stack_selective(x, layers, pools, w.segs.numpy(), rows, cos, sin, cfg.Hq,
                                       cfg.rope_base, EPS, dt=0)
    np.testing.assert_array_equal(sel, np.stack([x[b, rows[b]] for b in range(cfg.B)]).astype(np.float64))


def test_every_row_selected_equals_full_recompute():
    cfg, w, x, H, I = _small_case()
    layers = _weights(3, H, cfg.Hq, cfg.Hkv, cfg.D, I, 6)
    full = O.decoder_stack_full(x, layers, cfg.Hq, cfg.Hkv, cfg.D, cfg.rope_base, EPS)
    cos, sin = O.rope_table(cfg.N, cfg.D, cfg.rope_base)
    pools = [[(a.numpy(), b.numpy()) for a, b in w.pools]] * 3
    rows = np.broadcast_to(np.arange(cfg.N, dtype=np.int32), (cfg.B, cfg.N)).copy()
    sel, _ = O.decoder_stack_selective(x, layers, pools, w.segs.numpy(), rows, cos, sin, cfg.Hq,
                                       cfg.rope_base, EPS, dt=0)
    np.testing.assert_allclose(sel, full, rtol=0, atol=2e-5)


def test_exact_cache_makes_the_selected_rows_exact():
    """Pools holding each layer's keys (rotated to block-local positions) and
    values from the full computation: after alignment the cache equals the
    full computation's K/V, so every selected row equals its full-recompute
    row, whichever rows are selected."""
    cfg, w, x, H, I = _small_case(seed=7)
    layers = _weights(3, H, cfg.Hq, cfg.Hkv, cfg.D, I, 8)
    full, kv = O.decoder_stack_full(x, layers, cfg.Hq, cfg.Hkv, cfg.D, cfg.rope_base, EPS,
                                    return_kv=True)
    segs = w.segs.numpy().copy()
    B, S = segs.shape[:2]
    Lmax = int(segs[..., 1].max())
    cos, sin = O.rope_table(cfg.N, cfg.D, cfg.rope_base)
    pools_by_layer = []
    new = segs.copy()
    for kr, v in kv:
        pk = np.zeros((B * S, Lmax, cfg.Hkv, cfg.D), np.float32)
        pv = np.zeros_like(pk)
        for b in range(B):
            for s in range(S):
                dst, ln, p, _ = segs[b, s]
                if p < 0:
                    continue
                pk[b * S + s, :ln] = O.rope_at(kr[b, dst:dst + ln], np.arange(ln), cfg.rope_base)
                pv[b * S + s, :ln] = v[b, dst:dst + ln]
                new[b, s, 2], new[b, s, 3] = 0, b * S + s
        pools_by_layer.append([(pk, pv)])
    rng = np.random.default_rng(9)
    for _ in range(2):
        rows = O.topk(new, cfg.N, cfg.k, rng.random((B, cfg.N)).astype(np.float32))
        sel, _ = O.decoder_stack_selective(x, layers, pools_by_layer, new, rows, cos, sin, cfg.Hq,
                                           cfg.rope_base, EPS, dt=0)
        want = np.stack([full[b, rows[b]] for b in range(B)])
        np.testing.assert_allclose(sel, want, rtol=0, atol=2e-4)
    # a noisy cache (the workload's own pools) does move the selected rows
    pools = [[(a.numpy(), b.numpy()) for a, b in w.pools]] * 3
    sel_n, _ = O.decoder_stack_selective(x, layers, pools, segs, rows, cos, sin, cfg.Hq,
                                         cfg.rope_base, EPS, dt=0)
    assert np.abs(sel_n - want).max() > 1e-2


# ---------------------------------------------------------------------------
# Closed form of the whole block (no oracle code on the expected side).
# With the query projection zero every score is 0, so each row's causal
# softmax is uniform and the attention output of row p is the mean of the
# value rows 0..p of its KV group. With gate rows [A; -A], up rows [B; B] and
# down columns [C, -C] the MLP is C((A n) * (B n)), because
# silu(t) - silu(-t) = t. One layer is then
#     n  = x / sqrt(mean(x^2) + eps) * g_attn
#     h  = x + concat_h(prefix-mean of V n over j <= p, group h // G) W_o^T
#     n2 = h / sqrt(mean(h^2) + eps) * g_mlp
#     x' = h + ((A n2) * (B n2)) C^T
# which fixes the q/k/v split order, the GQA head-to-group map, the causal
# mask (j <= p), the orientation of W_o, both residuals, both norm gains and
# their places, the gate/up order and pairing, and the orientation of W_down.
# ---------------------------------------------------------------------------

def _closed_form_layers(n_layers, H, Hq, Hkv, D, m, seed):
    rng = np.random.default_rng(seed)
    layers = []
    for _ in range(n_layers):
        w_qkv = rng.standard_normal(((Hq + 2 * Hkv) * D, H)) / math.sqrt(H)
        w_qkv[:Hq * D] = 0.0                                   # q = 0: uniform softmax
        A = rng.standard_normal((m, H)) / math.sqrt(H)
        Bm = rng.standard_normal((m, H)) / math.sqrt(H)
        C = rng.standard_normal((H, m)) / math.sqrt(m)
        layers.append(dict(
            w_qkv=w_qkv.astype(np.float32),
            w_o=(rng.standard_normal((H, Hq * D)) / math.sqrt(Hq * D)).astype(np.float32),
            w_gu=np.concatenate([A, -A, Bm, Bm]).astype(np.float32),    # gate [A; -A], up [B; B]
            w_down=np.concatenate([C, -C], axis=1).astype(np.float32),  # [C, -C]
            g_attn=(1 + 0.2 * rng.standard_normal(H)).astype(np.float32),
            g_mlp=(1 + 0.2 * rng.standard_normal(H)).astype(np.float32)))
    return layers


def _cf_norm(x, g):
    return x / np.sqrt(np.mean(x * x, axis=-1, keepdims=True) + EPS) * g


def _cf_prefix_mean(v, upto):
    """mean of v[0..p] for every p in upto: v [N, Hkv, D] -> [len(upto), Hkv, D]."""
    csum = np.cumsum(v, axis=0)
    return np.stack([csum[p] / (p + 1) for p in upto])


def _cf_mlp(h, L, m):
    n2 = _cf_norm(h, L["g_mlp"].astype(np.float64))
    A = L["w_gu"][:m].astype(np.float64)
    Bm = L["w_gu"][2 * m:3 * m].astype(np.float64)
    C = L["w_down"][:, :m].astype(np.float64)
    return h + ((n2 @ A.T) * (n2 @ Bm.T)) @ C.T


def _cf_attend_rows(vals, rows, Hq, Hkv, Wo):
    """Uniform causal attention of `rows` over value rows `vals` [N, Hkv, D],
    heads mapped to groups h // (Hq / Hkv), through W_o."""
    G = Hq // Hkv
    pm = _cf_prefix_mean(vals, rows)                       # [R, Hkv, D]
    heads = pm[:, np.arange(Hq) // G]                      # [R, Hq, D]
    return heads.reshape(len(rows), -1) @ Wo.T


@pytest.mark.parametrize("Hq,Hkv", [(4, 2), (6, 3), (4, 4)])
def test_full_stack_matches_closed_form(Hq, Hkv):
    B, N, H, D, m = 2, 11, 20, 8, 6
    layers = _closed_form_layers(2, H, Hq, Hkv, D, m, seed=Hq * 10 + Hkv)
    x = np.random.default_rng(3).standard_normal((B, N, H)).astype(np.float32)
    got = O.decoder_stack_full(x, layers, Hq, Hkv, D, 500000.0, EPS)
    X = x.astype(np.float64)
    for L in layers:
        Wv = L["w_qkv"][(Hq + Hkv) * D:].astype(np.float64)
        Wo = L["w_o"].astype(np.float64)
        nxt = np.empty_like(X)
        for b in range(B):
            n = _cf_norm(X[b], L["g_attn"].astype(np.float64))
            v = (n @ Wv.T).reshape(N, Hkv, D)
            h = X[b] + _cf_attend_rows(v, np.arange(N), Hq, Hkv, Wo)
            nxt[b] = _cf_mlp(h, L, m)
        X = nxt
    # the oracle's attention stores its inputs and outputs in fp32
    np.testing.assert_allclose(got, X, rtol=2e-6, atol=2e-6)


def test_selective_stack_matches_closed_form():
    """Later layers attend over their cache: pool value rows at cached
    positions that are not listed, the listed rows' own projected values
    elsewhere. Checks the gather's block and offset, the overwrite of listed
    positions, and that later layers continue from the listed rows' states."""
    Hq, Hkv, D, H, m, N = 4, 2, 8, 20, 6, 12
    rng = np.random.default_rng(5)
    # fresh [0, 3), pool 0 block 1 at [3, 8), pool 1 block 0 at [8, 12)
    segs = np.array([[[0, 3, -1, 0], [3, 5, 0, 1], [8, 4, 1, 0]]], np.int32)
    pools_by_layer = []
    for _ in range(3):
        p0 = [rng.standard_normal((2, 5, Hkv, D)).astype(np.float32) for _ in range(2)]
        p1 = [rng.standard_normal((1, 4, Hkv, D)).astype(np.float32) for _ in range(2)]
        pools_by_layer.append([tuple(p0), tuple(p1)])
    rows = np.array([[0, 1, 2, 5, 9, 11]], np.int32)
    layers = _closed_form_layers(3, H, Hq, Hkv, D, m, seed=17)
    x = rng.standard_normal((1, N, H)).astype(np.float32)
    cos, sin = O.rope_table(N, D, 500000.0)
    got, _ = O.decoder_stack_selective(x, layers, pools_by_layer, segs, rows, cos, sin, Hq,
                                       500000.0, EPS, dt=0)
    r = rows[0]
    X = x[0].astype(np.float64)
    # layer 1: every row projected, the listed rows attend over the fresh values
    L = layers[0]
    Wv = L["w_qkv"][(Hq + Hkv) * D:].astype(np.float64)
    v = (_cf_norm(X, L["g_attn"].astype(np.float64)) @ Wv.T).reshape(N, Hkv, D)
    h = X[r] + _cf_attend_rows(v, r, Hq, Hkv, L["w_o"].astype(np.float64))
    xs = _cf_mlp(h, L, m)
    for L, pools in zip(layers[1:], pools_by_layer[1:]):
        Wv = L["w_qkv"][(Hq + Hkv) * D:].astype(np.float64)
        cache = np.zeros((N, Hkv, D))
        cache[3:8] = pools[0][1][1, :5]          # pool 0 block 1, offsets 0..4
        cache[8:12] = pools[1][1][0, :4]         # pool 1 block 0
        cache[r] = (_cf_norm(xs, L["g_attn"].astype(np.float64)) @ Wv.T).reshape(len(r), Hkv, D)
        h = xs + _cf_attend_rows(cache, r, Hq, Hkv, L["w_o"].astype(np.float64))
        xs = _cf_mlp(h, L, m)
    np.testing.assert_allclose(got[0], xs, rtol=2e-6, atol=2e-6)
