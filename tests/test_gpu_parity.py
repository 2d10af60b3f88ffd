"""GPU parity: the HIP path, called through the C ABI, against the CPU oracle
on the same seeded inputs.

Bar: assembled K/V, selected rows and patched K/V bit-exact (rows compared on
identical scores); deviation scores within 1e-5 relative; attention outputs
within max-abs 2e-2 / mean-abs 2e-3 (bf16) or 1e-4 (fp32)."""
import numpy as np
import pytest
import torch

from oracle import oracle as O
from paper_2605_07443_amd import inputs, ops

from parity import (H, assert_attn_close, oracle_attention_rows, run_stepwise, sample_rows,
                    say)

pytestmark = pytest.mark.gpu

DEV = torch.device("cuda:0")


@pytest.fixture(scope="module", autouse=True)
def _lib_loaded():
    from paper_2605_07443_amd import _lib
    _lib.load()
    yield
    torch.cuda.synchronize()


# ---------------------------------------------------------------- small shapes

SMALL = ["tiny-bf16", "ragged-bf16", "mha-d64-bf16", "miss-bf16", "tiny-f32-gqa", "allfresh-bf16"]


@pytest.mark.parametrize("name", SMALL)
@pytest.mark.parametrize("pct", [0, 15, 40, 100])
def test_stepwise_small(name, pct):
    cfg = inputs.TEST_WORKLOADS[name]
    say(f"[stepwise] {name} pct={pct} N={cfg.N} B={cfg.B}")
    w = inputs.make(cfg, 100 + pct, device=DEV)
    stats, _ = run_stepwise(cfg, w, cfg.k_for(pct), DEV)
    say(f"  {stats}")


def test_stepwise_config1_tiny_fp32():
    cfg = inputs.WORKLOADS[1]
    say(f"[stepwise] config 1 N={cfg.N}")
    w = inputs.make(cfg, 1000, device=DEV)
    stats, _ = run_stepwise(cfg, w, cfg.k, DEV)
    say(f"  {stats}")


def test_planted_heavy_hitters_selected_on_gpu():
    cfg = inputs.TEST_WORKLOADS["tiny-bf16"]
    w = inputs.make(cfg, 5, device=DEV, planted=6)
    _, r = run_stepwise(cfg, w, cfg.k, DEV)
    rows = r["rows"].cpu().numpy()
    for b in range(cfg.B):
        assert set(w.planted[b].tolist()) <= set(rows[b].tolist())


# ----------------------------------------------------- standalone re-alignment

@pytest.mark.parametrize("dtype,D,Hkv", [("bf16", 128, 8), ("bf16", 64, 2), ("f32", 64, 8),
                                         ("f32", 128, 1)])
def test_rerope_standalone_bitexact(dtype, D, Hkv):
    B, N, max_pos = 3, 301, 5000
    g = torch.Generator(device="cpu").manual_seed(7)
    tdt = torch.bfloat16 if dtype == "bf16" else torch.float32
    k = torch.randn((B, N, Hkv, D), generator=g).to(tdt)
    delta = torch.randint(-(max_pos - 1), max_pos, (B, N), generator=g, dtype=torch.int32)
    delta[:, ::7] = 0
    delta[0, 5] = max_pos          # out of range: skipped
    delta[1, 9] = -max_pos
    cos, sin = ops.rope_table(max_pos, D, 500000.0, DEV)
    kd = k.to(DEV)
    ops.rerope(kd, delta.to(DEV), cos, sin)
    torch.cuda.synchronize()
    ocos, osin = O.rope_table(max_pos, D, 500000.0)
    d_np = delta.numpy().copy()
    d_np[0, 5] = 0
    d_np[1, 9] = 0
    want = O.rerope(H(k), d_np, ocos, osin)
    np.testing.assert_array_equal(H(kd), want)


# ------------------------------------------------------------ attention shapes

@pytest.mark.parametrize("Hq,Hkv", [(8, 8), (8, 4), (16, 4), (16, 2), (32, 2)])
@pytest.mark.parametrize("D", [64, 128])
def test_attention_unsorted_rows_and_groups(Hq, Hkv, D):
    B, N, R = 2, 333, 150
    g = torch.Generator(device="cpu").manual_seed(Hq * 100 + Hkv + D)
    q = torch.randn((B, N, Hq, D), generator=g).to(torch.bfloat16)
    k = torch.randn((B, N, Hkv, D), generator=g).to(torch.bfloat16)
    v = torch.randn((B, N, Hkv, D), generator=g).to(torch.bfloat16)
    rows = torch.randint(0, N, (B, R), generator=g, dtype=torch.int32)
    rows[0, :3] = torch.tensor([N - 1, 0, N - 1], dtype=torch.int32)   # duplicates, extremes
    out = ops.selective_attention(q.to(DEV), k.to(DEV), v.to(DEV), rows.to(DEV))
    full = ops.full_prefill(q.to(DEV), k.to(DEV), v.to(DEV))
    torch.cuda.synchronize()
    ref = O.attention(H(q), H(k), H(v), rows=rows.numpy())
    assert_attn_close(H(out), ref, "bf16", "selective")
    reff = O.attention(H(q), H(k), H(v))
    assert_attn_close(H(full), reff, "bf16", "full prefill")


@pytest.mark.parametrize("Hq,Hkv", [(32, 1), (64, 1), (128, 1), (128, 2)])
def test_attention_large_groups(Hq, Hkv):
    """Group sizes 32, 64 and 128 (the largest that divides a workgroup's 128
    query vectors): a workgroup then holds 4, 2 or 1 rows of all G heads;
    selective rows (unsorted, duplicated) and full prefill against the
    oracle, bf16 and D = 64."""
    B, N, R, D = 2, 200, 37, 64
    g = torch.Generator(device="cpu").manual_seed(Hq * 10 + Hkv)
    q = torch.randn((B, N, Hq, D), generator=g).to(torch.bfloat16)
    k = torch.randn((B, N, Hkv, D), generator=g).to(torch.bfloat16)
    v = torch.randn((B, N, Hkv, D), generator=g).to(torch.bfloat16)
    rows = torch.randint(0, N, (B, R), generator=g, dtype=torch.int32)
    rows[1, :2] = torch.tensor([N - 1, N - 1], dtype=torch.int32)
    say(f"[attention groups] Hq={Hq} Hkv={Hkv}")
    out = ops.selective_attention(q.to(DEV), k.to(DEV), v.to(DEV), rows.to(DEV))
    full = ops.full_prefill(q.to(DEV), k.to(DEV), v.to(DEV))
    torch.cuda.synchronize()
    assert_attn_close(H(out), O.attention(H(q), H(k), H(v), rows=rows.numpy()), "bf16", "selective")
    assert_attn_close(H(full), O.attention(H(q), H(k), H(v)), "bf16", "full prefill")


@pytest.mark.parametrize("N", [1, 17, 63, 64, 65, 127, 128, 129])
@pytest.mark.parametrize("D", [64, 128])
def test_attention_tile_boundary_lengths(N, D):
    """Prompts shorter than, equal to and just past one 64-key tile and two:
    the partial last tile, a single tile and a single key."""
    B, Hq, Hkv = 2, 8, 2
    g = torch.Generator(device="cpu").manual_seed(N * 10 + D)
    q = torch.randn((B, N, Hq, D), generator=g).to(torch.bfloat16)
    k = torch.randn((B, N, Hkv, D), generator=g).to(torch.bfloat16)
    v = torch.randn((B, N, Hkv, D), generator=g).to(torch.bfloat16)
    R = min(N, 5)
    rows = torch.sort(torch.randint(0, N, (B, R), generator=g, dtype=torch.int32), dim=1).values
    rows[:, -1] = N - 1
    say(f"[attention boundary] N={N} D={D}")
    out = ops.selective_attention(q.to(DEV), k.to(DEV), v.to(DEV), rows.to(DEV))
    full = ops.full_prefill(q.to(DEV), k.to(DEV), v.to(DEV))
    torch.cuda.synchronize()
    assert_attn_close(H(out), O.attention(H(q), H(k), H(v), rows=rows.numpy()), "bf16", "selective")
    assert_attn_close(H(full), O.attention(H(q), H(k), H(v)), "bf16", "full prefill")


def test_attention_fp32_full_and_selected():
    B, N, Hq, Hkv, D = 2, 190, 8, 2, 128
    g = torch.Generator(device="cpu").manual_seed(3)
    q, k, v = (torch.randn((B, N, h, D), generator=g) for h in (Hq, Hkv, Hkv))
    rows = torch.sort(torch.randperm(N, generator=g)[:70]).values.to(torch.int32).repeat(B, 1)
    out = ops.selective_attention(q.to(DEV), k.to(DEV), v.to(DEV), rows.to(DEV).contiguous())
    full = ops.full_prefill(q.to(DEV), k.to(DEV), v.to(DEV))
    torch.cuda.synchronize()
    assert_attn_close(H(out), O.attention(H(q), H(k), H(v), rows=rows.numpy()), "f32", "sel")
    assert_attn_close(H(full), O.attention(H(q), H(k), H(v)), "f32", "full")


# ------------------------------------------------------------------ invariants

@pytest.mark.parametrize("name", ["tiny-bf16", "tiny-f32-gqa", "miss-bf16"])
def test_full_ratio_equals_full_prefill_on_gpu(name):
    """Selecting every cached token = Full-Recompute, bit for bit on the GPU."""
    cfg = inputs.TEST_WORKLOADS[name]
    w = inputs.make(cfg, 31, device=DEV)
    segs = ops.prepare_segments(w.segs, cfg.N, w.pools, DEV)
    cos, sin = ops.rope_table(cfg.N, cfg.D, cfg.rope_base, DEV)
    bufs = ops.selective_prefill(w.q, w.k_fresh, w.v_fresh, w.pools, segs, cfg.n_reused, cos, sin)
    full = ops.full_prefill(w.q, w.k_fresh, w.v_fresh)
    torch.cuda.synchronize()
    assert torch.equal(bufs.rows.cpu(), torch.arange(cfg.N, dtype=torch.int32).repeat(cfg.B, 1))
    assert torch.equal(bufs.k_asm, w.k_fresh) and torch.equal(bufs.v_asm, w.v_fresh)
    assert torch.equal(bufs.out, full)


@pytest.mark.parametrize("pct", [0, 10, 50])
def test_zero_perturbation_equals_full_prefill_on_gpu(pct):
    cfg = inputs.TEST_WORKLOADS["ragged-bf16"]
    w = inputs.make(cfg, 32, device=DEV, sigma=0.0)
    segs = ops.prepare_segments(w.segs, cfg.N, w.pools, DEV)
    cos, sin = ops.rope_table(cfg.N, cfg.D, cfg.rope_base, DEV)
    bufs = ops.selective_prefill(w.q, w.k_fresh, w.v_fresh, w.pools, segs, cfg.k_for(pct), cos, sin)
    full = ops.full_prefill(w.q, w.k_fresh, w.v_fresh)
    torch.cuda.synchronize()
    rows = bufs.rows.long()
    sel_full = torch.stack([full[b, rows[b]] for b in range(cfg.B)])
    assert_attn_close(H(bufs.out), H(sel_full), "bf16", "zero noise")


def test_instruction_rows_equal_full_prefill_at_any_noise():
    cfg = inputs.TEST_WORKLOADS["tiny-bf16"]
    w = inputs.make(cfg, 33, device=DEV, sigma=0.3)
    segs = ops.prepare_segments(w.segs, cfg.N, w.pools, DEV)
    cos, sin = ops.rope_table(cfg.N, cfg.D, cfg.rope_base, DEV)
    bufs = ops.selective_prefill(w.q, w.k_fresh, w.v_fresh, w.pools, segs, cfg.k, cos, sin)
    full = ops.full_prefill(w.q, w.k_fresh, w.v_fresh)
    torch.cuda.synchronize()
    rows = bufs.rows.cpu().numpy()
    for b in range(cfg.B):
        first = np.nonzero(rows[b] < cfg.F)[0]
        ref = H(full[b])[rows[b][first]]
        assert_attn_close(H(bufs.out[b])[first], ref, "bf16", "instruction rows")


def test_pipeline_is_deterministic():
    cfg = inputs.TEST_WORKLOADS["ragged-bf16"]
    w = inputs.make(cfg, 34, device=DEV)
    segs = ops.prepare_segments(w.segs, cfg.N, w.pools, DEV)
    cos, sin = ops.rope_table(cfg.N, cfg.D, cfg.rope_base, DEV)
    a = ops.selective_prefill(w.q, w.k_fresh, w.v_fresh, w.pools, segs, cfg.k, cos, sin)
    b = ops.selective_prefill(w.q, w.k_fresh, w.v_fresh, w.pools, segs, cfg.k, cos, sin)
    torch.cuda.synchronize()
    for name in ("k_asm", "v_asm", "scores", "rows", "out"):
        assert torch.equal(getattr(a, name), getattr(b, name)), name


# ---------------------------------------------------------------- edge cases

def test_single_token_segments_and_all_cached_prompt():
    """Segments of length 1 and 2, no fresh positions at all (n_fresh = 0),
    k = 0 (nothing recomputed, empty row list) and k = n_r."""
    B, Hkv, Hq, D = 2, 2, 8, 128
    pk = torch.randn((5, 3, Hkv, D)).to(torch.bfloat16).to(DEV)
    pv = torch.randn((5, 3, Hkv, D)).to(torch.bfloat16).to(DEV)
    spans = [(0, 1, 0, 4), (1, 2, 0, 0), (3, 1, 0, 2), (4, 3, 0, 1), (7, 1, 0, 3)]
    segs_h = np.array([spans, spans[::-1]], np.int32)
    # second request: same blocks in reverse order, re-tiled
    pos = 0
    for s in range(len(spans)):
        segs_h[1, s, 0] = pos
        pos += segs_h[1, s, 1]
    N = 8
    kf = torch.randn((B, N, Hkv, D)).to(torch.bfloat16).to(DEV)
    vf = torch.randn((B, N, Hkv, D)).to(torch.bfloat16).to(DEV)
    q = torch.randn((B, N, Hq, D)).to(torch.bfloat16).to(DEV)
    segs = ops.prepare_segments(segs_h, N, [(pk, pv)], DEV)
    assert segs.n_fresh == 0
    cos, sin = ops.rope_table(N, D, 10000.0, DEV)
    ka, va = ops.kv_assemble([(pk, pv)], segs, kf, vf, cos, sin)
    torch.cuda.synchronize()
    ocos, osin = O.rope_table(N, D, 10000.0)
    ka_o, va_o = O.assemble(H(kf), H(vf), [(H(pk), H(pv))], segs_h, ocos, osin)
    np.testing.assert_array_equal(H(ka), ka_o)
    np.testing.assert_array_equal(H(va), va_o)
    rows0, _ = ops.select_tokens(segs, 0, kf, vf, ka.clone(), va.clone())
    assert rows0.shape == (B, 0)
    rows8, sc = ops.select_tokens(segs, N, kf, vf, ka, va)
    out = ops.selective_attention(q, ka, va, rows8)
    torch.cuda.synchronize()
    assert torch.equal(rows8.cpu(), torch.arange(N, dtype=torch.int32).repeat(B, 1))
    assert_attn_close(H(out), O.attention(H(q), H(kf), H(vf)), "bf16", "all selected")


def test_scores_in_special_values_match_oracle():
    cfg = inputs.TEST_WORKLOADS["ragged-bf16"]
    w = inputs.make(cfg, 35, device=DEV)
    segs = ops.prepare_segments(w.segs, cfg.N, w.pools, DEV)
    rng = np.random.default_rng(0)
    sc = rng.integers(0, 4, (cfg.B, cfg.N)).astype(np.float32)     # many ties
    sc[0, 20] = np.nan
    sc[0, 30] = np.inf
    sc[1, 40] = -np.inf
    sc[2, 50:60] = -1.5
    sc[2, 61] = -0.0
    for k in (0, 1, 7, cfg.n_reused // 2, cfg.n_reused):
        rows, _ = ops.select_tokens(segs, k, w.k_fresh, w.v_fresh, torch.empty_like(w.k_fresh),
                                    torch.empty_like(w.v_fresh), scores_in=torch.from_numpy(sc).to(DEV),
                                    patch=False)
        torch.cuda.synchronize()
        np.testing.assert_array_equal(rows.cpu().numpy(), O.topk(w.segs.numpy(), cfg.N, k, sc))


# ------------------------------------------------------------- full workloads

@pytest.mark.parametrize("cid,pct,stride", [(2, 15, 16), (3, 10, 32), (5, 15, 64),
                                            (4, 0, 16), (4, 5, 16), (4, 10, 16), (4, 15, 16),
                                            (4, 25, 32), (4, 50, 64), (4, 100, 128)])
def test_stepwise_full_workloads(cid, pct, stride):
    cfg = inputs.WORKLOADS[cid]
    say(f"[full workload] config {cid} pct={pct} B={cfg.B} N={cfg.N} pools="
        f"{cfg.hist_pool}x{cfg.hist_len},{cfg.item_pool}x{cfg.item_len}")
    w = inputs.make(cfg, 1000 * cid, device=DEV)
    stats, _ = run_stepwise(cfg, w, cfg.k_for(pct), DEV, stride=stride)
    say(f"  {stats}")
    del w
    torch.cuda.empty_cache()


@pytest.mark.parametrize("cid,stride", [(2, 64), (3, 256), (4, 128), (5, 256)])
def test_full_prefill_full_workloads(cid, stride):
    cfg = inputs.WORKLOADS[cid]
    say(f"[full prefill] config {cid}")
    g = torch.Generator(device=DEV).manual_seed(cid)
    q = torch.randn((cfg.B, cfg.N, cfg.Hq, cfg.D), generator=g, device=DEV).to(torch.bfloat16)
    k = torch.randn((cfg.B, cfg.N, cfg.Hkv, cfg.D), generator=g, device=DEV).to(torch.bfloat16)
    v = torch.randn((cfg.B, cfg.N, cfg.Hkv, cfg.D), generator=g, device=DEV).to(torch.bfloat16)
    out = ops.full_prefill(q, k, v)
    torch.cuda.synchronize()
    all_rows = np.arange(cfg.N, dtype=np.int32)[None].repeat(cfg.B, 0)
    sel = [np.concatenate([np.arange(0, cfg.N, stride), [cfg.N - 1]]) for _ in range(cfg.B)]
    ref = oracle_attention_rows(H(q), H(k), H(v), all_rows, sel)
    outh = H(out)
    g_ = np.concatenate([outh[b, idx] for b, idx in enumerate(sel)])
    assert_attn_close(g_, np.concatenate(ref), "bf16", "full prefill")


@pytest.mark.parametrize("D", [64, 128])
def test_attention_max_jumps_inside_tiles(D):
    """Scores that jump by more than the lazy-rescale margin in the second
    half of every 64-key tile (keys j with j % 64 >= 32 align with the
    queries more than all earlier keys): the running max is raised inside a
    tile, after the first half's probabilities were formed, on every tile.
    Output and log-sum-exp against the oracle."""
    B, N, Hq, Hkv = 1, 320, 8, 2
    g = torch.Generator(device="cpu").manual_seed(77 + D)
    u = torch.ones(D) / D ** 0.25   # scale * (u . 8u) * log2(e) = 11.5 log2 units per amplitude step
    amp = torch.tensor([(j // 64) + (1.0 if j % 64 >= 32 else 0.0) for j in range(N)])
    q = (u + 0.05 * torch.randn((B, N, Hq, D), generator=g)).to(torch.bfloat16)
    k = (amp[None, :, None, None] * u * 8.0 + 0.05 * torch.randn((B, N, Hkv, D), generator=g)).to(torch.bfloat16)
    v = torch.randn((B, N, Hkv, D), generator=g).to(torch.bfloat16)
    rows = torch.tensor([[5, 40, 63, 64, 95, 96, 127, 150, 191, 200, 255, 256, 300, 319]], dtype=torch.int32)
    say(f"[attention max jumps] D={D}")
    out = ops.selective_attention(q.to(DEV), k.to(DEV), v.to(DEV), rows.to(DEV))
    full = ops.full_prefill(q.to(DEV), k.to(DEV), v.to(DEV))
    _, lse = ops.selective_attention_lse(q.to(DEV), k.to(DEV), v.to(DEV))
    torch.cuda.synchronize()
    assert_attn_close(H(out), O.attention(H(q), H(k), H(v), rows=rows.numpy()), "bf16", "selective")
    assert_attn_close(H(full), O.attention(H(q), H(k), H(v)), "bf16", "full prefill")
    lse_o = O.attention_lse(H(q), H(k))
    # lse reaches about 45 here: the absolute bound of the eq3 tests plus fp32 rounding of it
    err = np.abs(lse.cpu().numpy().astype(np.float64) - lse_o)
    assert np.all(err <= 2e-5 + 1e-6 * np.abs(lse_o)), f"lse max err {err.max():.3e}"


def test_patch_with_more_than_64_segments():
    """Requests of 150 segments, more than the 64 that the wave-level gather
    keeps in lane registers (the workgroup gather runs instead) and a long
    class search in the selection: assembly, selection and patched K/V
    bit-exact with the oracle."""
    B, Hkv, D, BL = 2, 2, 64, 16
    rng = np.random.default_rng(11)
    lens = rng.integers(1, BL + 1, 150)
    kinds = np.where(np.arange(150) % 3 == 0, -1, np.arange(150) % 2)  # fresh, pool 0, pool 1
    starts = np.concatenate([[0], np.cumsum(lens)[:-1]])
    N = int(lens.sum())
    blocks = rng.integers(0, 40, 150)
    seg = np.stack([starts, lens, kinds, np.where(kinds < 0, 0, blocks)], 1).astype(np.int32)
    segs_h = np.ascontiguousarray(np.broadcast_to(seg, (B, 150, 4)))
    g = torch.Generator(device="cpu").manual_seed(11)
    pools = [(torch.randn((40, BL, Hkv, D), generator=g).to(torch.bfloat16).to(DEV),
              torch.randn((40, BL, Hkv, D), generator=g).to(torch.bfloat16).to(DEV)) for _ in range(2)]
    kf = torch.randn((B, N, Hkv, D), generator=g).to(torch.bfloat16).to(DEV)
    vf = torch.randn((B, N, Hkv, D), generator=g).to(torch.bfloat16).to(DEV)
    segs = ops.prepare_segments(segs_h, N, pools, DEV)
    k = (N - segs.n_fresh) // 4
    say(f"[patch, 150 segments] N={N} k={k}")
    ka, va = ops.kv_assemble(pools, segs, kf, vf)
    torch.cuda.synchronize()
    hp = [(H(pk), H(pv)) for pk, pv in pools]
    ka0, va0 = O.assemble(H(kf), H(vf), hp, segs_h)
    np.testing.assert_array_equal(H(ka), ka0)
    rows, sc = ops.select_tokens(segs, k, kf, vf, ka, va)
    torch.cuda.synchronize()
    rows_h = rows.cpu().numpy()
    np.testing.assert_array_equal(rows_h, O.topk(segs_h, N, k, sc.cpu().numpy()))
    kp, vp = O.patch(segs_h, rows_h, H(kf), H(vf), ka0, va0)
    np.testing.assert_array_equal(H(ka), kp)
    np.testing.assert_array_equal(H(va), vp)


# ------------------------------------------------------- the most pools a call takes

@pytest.mark.parametrize("dtype,D,Hq", [("bf16", 128, 8), ("f32", 64, 8), ("bf16", 64, 64)])
def test_eight_pools_in_one_request(dtype, D, Hq):
    """Eight pools (the most a call takes), each with its own block length and
    block count, all referenced by every request, with a fresh segment between
    them and blocks used whole and in part: fused gather + rotation bit-exact
    with the oracle, scores within 1e-5, rows and patched K/V bit-exact,
    attention within tolerance of the oracle; for bf16 the paged path equals
    the assembled one bit for bit (also with 32 query heads per KV head)."""
    B, Hkv, F = 2, 2, 8
    tdt = torch.bfloat16 if dtype == "bf16" else torch.float32
    rng = np.random.default_rng(800 + D + Hq)
    bls = [8, 12, 16, 20, 24, 32, 40, 48]
    nbs = [5, 6, 7, 8, 9, 10, 11, 12]
    order = list(range(8)) + list(range(7, -1, -1))
    lens = [bls[p] if j < 8 else int(rng.integers(1, bls[p] + 1)) for j, p in enumerate(order)]
    segs_h = []
    for b in range(B):
        seg, pos = [(0, F, -1, 0)], F
        for j, p in enumerate(order):
            seg.append((pos, lens[j], p, int(rng.integers(0, nbs[p]))))
            pos += lens[j]
            if j == 3:
                seg.append((pos, 5, -1, 0))
                pos += 5
        segs_h.append(seg)
    segs_h = np.ascontiguousarray(np.array(segs_h, np.int32))
    N = int(segs_h[0, -1, 0] + segs_h[0, -1, 1])
    g = torch.Generator().manual_seed(80 + D + Hq)
    pools = [(torch.randn((nb, bl, Hkv, D), generator=g).to(tdt).to(DEV),
              torch.randn((nb, bl, Hkv, D), generator=g).to(tdt).to(DEV)) for nb, bl in zip(nbs, bls)]
    kf = torch.randn((B, N, Hkv, D), generator=g).to(tdt).to(DEV)
    vf = torch.randn((B, N, Hkv, D), generator=g).to(tdt).to(DEV)
    q = torch.randn((B, N, Hq, D), generator=g).to(tdt).to(DEV)
    segs = ops.prepare_segments(segs_h, N, pools, DEV)
    assert segs.n_fresh == F + 5
    k = (segs.n_reused * 30 + 99) // 100
    cos, sin = ops.rope_table(N, D, 10000.0, DEV)
    say(f"[8 pools] {dtype} D={D} Hq={Hq} N={N} S={segs.S} k={k}")
    scores = torch.empty((B, N), dtype=torch.float32, device=DEV)
    ka, va = ops.kv_assemble(pools, segs, kf, vf, cos, sin, scores_out=scores)
    a = ops.selective_prefill(q, kf, vf, pools, segs, k, cos, sin)
    torch.cuda.synchronize()
    hp = [(H(pk), H(pv)) for pk, pv in pools]
    ocos, osin = O.rope_table(N, D, 10000.0)
    ka0, va0 = O.assemble(H(kf), H(vf), hp, segs_h, ocos, osin)
    np.testing.assert_array_equal(H(ka), ka0)
    np.testing.assert_array_equal(H(va), va0)
    np.testing.assert_allclose(scores.cpu().numpy(), O.deviation(H(kf), ka0), rtol=1e-5, atol=1e-5)
    sc = a.scores.cpu().numpy()
    rows = a.rows.cpu().numpy()
    np.testing.assert_array_equal(rows, O.topk(segs_h, N, k, sc))
    kp, vp = O.patch(segs_h, rows, H(kf), H(vf), ka0, va0)
    np.testing.assert_array_equal(H(a.k_asm), kp)
    np.testing.assert_array_equal(H(a.v_asm), vp)
    sel = sample_rows(B, rows.shape[1], 1)
    ref = np.concatenate(oracle_attention_rows(H(q), kp, vp, rows, sel))
    got = np.concatenate([H(a.out)[b, idx] for b, idx in enumerate(sel)])
    assert_attn_close(got, ref, dtype, "attention over eight pools")
    if dtype == "bf16":
        p = ops.paged_prefill(q, kf, vf, pools, segs, k, cos, sin)
        torch.cuda.synchronize()
        assert torch.equal(a.scores, p.scores)
        assert torch.equal(a.rows, p.rows)
        assert torch.equal(a.out, p.out), "paged attention differs from the assembled path"
    if dtype == "bf16" and D == 128:
        # V by reference over the same eight pools: identical outputs, and
        # every table entry the address of the row the copy would have taken
        r = ops.selective_prefill_vref(q, kf, vf, pools, segs, k, cos, sin)
        torch.cuda.synchronize()
        assert torch.equal(r.scores, a.scores) and torch.equal(r.rows, a.rows)
        assert torch.equal(r.k_asm, a.k_asm)
        assert torch.equal(r.out, a.out), "attention through V references differs"
        row_bytes = Hkv * D * 2
        fresh = vf.data_ptr() + row_bytes * np.arange(B * N, dtype=np.int64).reshape(B, N)
        want = fresh.copy()
        for b in range(B):
            for dst, ln, pool, blk in segs_h[b].tolist():
                if pool >= 0:
                    pv = pools[pool][1]
                    want[b, dst:dst + ln] = (pv.data_ptr() + (blk * pv.shape[1]) * row_bytes
                                             + row_bytes * np.arange(ln, dtype=np.int64))
            want[b, rows[b]] = fresh[b, rows[b]]
        np.testing.assert_array_equal(r.v_ref.cpu().numpy(), want)


# ------------------------------------------------- cache misses, bad row lists

def test_all_fresh_prompt_equals_full_prefill():
    """Every segment a cache miss (computed on the fly, Sec. III-C.2a): nothing
    is reused, the assembled K/V are the fresh rows, no position is selected
    (k = 0 at any ratio), every position is a row, and the output is the
    Full-Recompute output bit for bit."""
    cfg = inputs.TEST_WORKLOADS["allfresh-bf16"]
    assert cfg.n_reused == 0
    w = inputs.make(cfg, 41, device=DEV)
    segs = ops.prepare_segments(w.segs, cfg.N, w.pools, DEV)
    cos, sin = ops.rope_table(cfg.N, cfg.D, cfg.rope_base, DEV)
    bufs = ops.selective_prefill(w.q, w.k_fresh, w.v_fresh, w.pools, segs, cfg.k_for(15), cos, sin)
    full = ops.full_prefill(w.q, w.k_fresh, w.v_fresh)
    torch.cuda.synchronize()
    assert torch.equal(bufs.rows.cpu(), torch.arange(cfg.N, dtype=torch.int32).repeat(cfg.B, 1))
    assert torch.equal(bufs.k_asm, w.k_fresh) and torch.equal(bufs.v_asm, w.v_fresh)
    assert bool((bufs.scores == 0).all())
    assert torch.equal(bufs.out, full)


def test_row_list_marks_inconsistent_fresh_count():
    """A segment table whose fresh count differs from the n_fresh passed in
    (possible only when the caller builds the table itself): the library
    cannot read the device table on the host, so it marks the request's row
    list with -1 (short list: unfilled tail; long list: last entry), the
    attention writes NaN for those rows and leaves the others exact, and the
    wrapper's debug check names the request."""
    cfg = inputs.TEST_WORKLOADS["tiny-bf16"]
    w = inputs.make(cfg, 42, device=DEV)
    good = ops.prepare_segments(w.segs, cfg.N, w.pools, DEV)
    cos, sin = ops.rope_table(cfg.N, cfg.D, cfg.rope_base, DEV)
    k = cfg.k
    k_asm, v_asm = ops.kv_assemble(w.pools, good, w.k_fresh, w.v_fresh, cos, sin)
    rows_ok, sc = ops.select_tokens(good, k, w.k_fresh, w.v_fresh, k_asm.clone(), v_asm.clone(),
                                    patch=False)
    for delta in (3, -3):
        bad = ops.Segments(dev=good.dev, host=good.host, n_fresh=good.n_fresh + delta, N=good.N)
        rows, _ = ops.select_tokens(bad, k, w.k_fresh, w.v_fresh, k_asm.clone(), v_asm.clone(),
                                    scores_in=sc, patch=False)
        torch.cuda.synchronize()
        r, ok = rows.cpu().numpy(), rows_ok.cpu().numpy()
        R = r.shape[1]
        if delta > 0:     # short list: the taken rows, then -1
            np.testing.assert_array_equal(r[:, :ok.shape[1]], ok)
            assert (r[:, ok.shape[1]:] == -1).all()
        else:             # long list: truncated, last entry -1
            np.testing.assert_array_equal(r[:, :R - 1], ok[:, :R - 1])
            assert (r[:, R - 1] == -1).all()
        with pytest.raises(RuntimeError, match="requests \\[0, 1\\]"):
            ops.check_rows(rows, cfg.N, "test")
        out = ops.selective_attention(w.q, k_asm, v_asm, rows)
        torch.cuda.synchronize()
        o = H(out)
        neg = r < 0
        assert np.isnan(O.as_f32(o[neg])).all()
        good_rows = np.where(neg, 0, r).astype(np.int32)
        ref = O.attention(H(w.q), H(k_asm), H(v_asm), rows=good_rows)
        assert_attn_close(o[~neg], ref[~neg], "bf16", "rows next to marked rows")


@pytest.mark.parametrize("dtype", ["bf16", "f32"])
def test_attention_rows_outside_range_give_nan(dtype):
    """Listed rows outside [0, N) yield NaN outputs (and lse), nothing else
    changes: the kernels read only in-range rows."""
    B, N, Hq, Hkv, D = 2, 200, 8, 2, 128
    g = torch.Generator(device="cpu").manual_seed(9)
    tdt = torch.bfloat16 if dtype == "bf16" else torch.float32
    q, k, v = (torch.randn((B, N, h, D), generator=g).to(tdt) for h in (Hq, Hkv, Hkv))
    rows = torch.tensor([[-1, 3, 50, 199], [0, N, 120, 1 << 30]], dtype=torch.int32)
    out, lse = ops.selective_attention_lse(q.to(DEV), k.to(DEV), v.to(DEV), rows.to(DEV))
    torch.cuda.synchronize()
    bad = np.array([[1, 0, 0, 0], [0, 1, 0, 1]], bool)
    o, l = O.as_f32(H(out)), lse.cpu().numpy()
    assert np.isnan(o[bad]).all() and np.isnan(l[bad]).all()
    assert np.isfinite(o[~bad]).all() and np.isfinite(l[~bad]).all()
    ref = O.attention(H(q), H(k), H(v), rows=np.where(bad, 0, rows.numpy()).astype(np.int32))
    assert_attn_close(H(out)[~bad], ref[~bad], dtype, "in-range rows")
