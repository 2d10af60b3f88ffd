"""GPU parity of the value-reference chain (rc_kv_assemble_vref ->
rc_select_tokens_vref -> rc_selective_attention_vref), called through the C
ABI, against the CPU oracle and against the assembled chain on the same
seeded inputs.

Bar: assembled and patched K bit-exact against the oracle; deviation scores
and selected rows bit-identical to the assembled chain's; every value-row
address equal to the one computed on the host from the segment table, the
pool tensors and the selected rows; attention outputs bit-identical to
rc_selective_attention over the assembled copy, and within max-abs 2e-2 /
mean-abs 2e-3 of the oracle on the rows checked."""
import numpy as np
import pytest
import torch

from oracle import oracle as O
from paper_2605_07443_amd import _lib, inputs, ops

from parity import H, assert_attn_close, oracle_attention_rows, sample_rows, say

pytestmark = pytest.mark.gpu

DEV = torch.device("cuda:0")


@pytest.fixture(scope="module", autouse=True)
def _lib_loaded():
    _lib.load()
    yield
    torch.cuda.synchronize()


def expected_vref(w, rows: np.ndarray) -> np.ndarray:
    """Byte address of the value row each position reads: the pool row of a
    cached position, the fresh row of a fresh or selected one."""
    B, N, Hkv, D = w.v_fresh.shape
    row_bytes = Hkv * D * w.v_fresh.element_size()
    fresh = w.v_fresh.data_ptr() + row_bytes * np.arange(B * N, dtype=np.int64).reshape(B, N)
    exp = fresh.copy()
    for b, req in enumerate(w.segs.numpy()):
        for dst, ln, p, blk in req.tolist():
            if p < 0:
                continue
            pv = w.pools[p][1]
            base = pv.data_ptr() + (blk * pv.shape[1]) * row_bytes
            exp[b, dst:dst + ln] = base + row_bytes * np.arange(ln, dtype=np.int64)
        r = rows[b][rows[b] >= 0]
        exp[b, r] = fresh[b, r]
    return exp


def run_both(cfg, w, k):
    """The assembled chain and the value-reference chain on the same inputs."""
    segs = ops.prepare_segments(w.segs, cfg.N, w.pools, DEV)
    cos, sin = ops.rope_table(cfg.N, cfg.D, cfg.rope_base, DEV)
    sc_a = torch.empty((cfg.B, cfg.N), dtype=torch.float32, device=DEV)
    k_asm, v_asm = ops.kv_assemble(w.pools, segs, w.k_fresh, w.v_fresh, cos, sin, scores_out=sc_a)
    rows_a, _ = ops.select_tokens(segs, k, w.k_fresh, w.v_fresh, k_asm, v_asm, scores_in=sc_a,
                                  patch=True)
    R = rows_a.shape[1]
    out_a = ops.selective_attention(w.q, k_asm, v_asm, rows_a) if R > 0 else None

    sc_r = torch.empty((cfg.B, cfg.N), dtype=torch.float32, device=DEV)
    k_ref, v_ref = ops.kv_assemble_vref(w.pools, segs, w.k_fresh, w.v_fresh, cos, sin,
                                        scores_out=sc_r)
    table_pre = v_ref.clone()
    k_pre = k_ref.clone()
    rows_r, _ = ops.select_tokens_vref(segs, k, w.k_fresh, w.v_fresh, k_ref, v_ref, scores_in=sc_r)
    out_r = ops.selective_attention_vref(w.q, k_ref, v_ref, rows_r) if R > 0 else None
    torch.cuda.synchronize()
    return dict(segs=segs, sc_a=sc_a, rows_a=rows_a, k_asm=k_asm, v_asm=v_asm, out_a=out_a,
                sc_r=sc_r, rows_r=rows_r, k_ref=k_ref, v_ref=v_ref, out_r=out_r,
                table_pre=table_pre, k_pre=k_pre)


def check_against_assembled(w, r):
    np.testing.assert_array_equal(r["sc_r"].cpu().numpy(), r["sc_a"].cpu().numpy(),
                                  err_msg="scores of the value-reference gather differ")
    rows = r["rows_r"].cpu().numpy()
    np.testing.assert_array_equal(rows, r["rows_a"].cpu().numpy(), err_msg="rows differ")
    np.testing.assert_array_equal(H(r["k_ref"]), H(r["k_asm"]), err_msg="patched K differs")
    # the table before the patch: every position's gather source
    no_sel = np.full((rows.shape[0], 0), -1, np.int32)
    np.testing.assert_array_equal(r["table_pre"].cpu().numpy(), expected_vref(w, no_sel),
                                  err_msg="value-row addresses of the gather differ")
    np.testing.assert_array_equal(r["v_ref"].cpu().numpy(), expected_vref(w, rows),
                                  err_msg="value-row addresses after the patch differ")
    if r["out_a"] is not None:
        np.testing.assert_array_equal(H(r["out_r"]), H(r["out_a"]),
                                      err_msg="attention through references differs")
    return rows


SMALL = ["tiny-bf16", "ragged-bf16", "miss-bf16", "allfresh-bf16"]


@pytest.mark.parametrize("name", SMALL)
@pytest.mark.parametrize("pct", [0, 15, 100])
def test_vref_chain_small(name, pct):
    cfg = inputs.TEST_WORKLOADS[name]
    say(f"[vref] {name} pct={pct} N={cfg.N} B={cfg.B}")
    w = inputs.make(cfg, 300 + pct, device=DEV)
    k = cfg.k_for(pct)
    r = run_both(cfg, w, k)
    rows = check_against_assembled(w, r)

    # against the oracle: assembled K before the patch, patched K, attention
    ocos, osin = O.rope_table(cfg.N, cfg.D, cfg.rope_base)
    subpools, segs_sub = inputs.referenced_subpools(w)
    kf, vf = H(w.k_fresh), H(w.v_fresh)
    ka_o, va_o = O.assemble(kf, vf, subpools, segs_sub, ocos, osin)
    np.testing.assert_array_equal(H(r["k_pre"]), ka_o, err_msg="assembled K differs from the oracle")
    sc_o = O.deviation(kf, ka_o)
    np.testing.assert_allclose(r["sc_r"].cpu().numpy(), sc_o, rtol=1e-5, atol=1e-5)
    kp_o, vp_o = O.patch(w.segs.numpy(), rows, kf, vf, ka_o, va_o)
    np.testing.assert_array_equal(H(r["k_ref"]), kp_o, err_msg="patched K differs from the oracle")
    if r["out_r"] is not None:
        sel = sample_rows(cfg.B, rows.shape[1], 1)
        ref = oracle_attention_rows(H(w.q), kp_o, vp_o, rows, sel)
        g = np.concatenate([H(r["out_r"])[b, idx] for b, idx in enumerate(sel)])
        say(f"  {assert_attn_close(g, np.concatenate(ref), cfg.dtype, 'vref attention')}")


@pytest.mark.parametrize("Hq,Hkv", [(8, 1), (16, 1)])
def test_vref_chain_one_kv_head(Hq, Hkv):
    """One KV head (a key row of 256 bytes): the wave gather then owns 8
    positions per wave and writes 8 table entries per wave."""
    cfg = inputs.Config(f"mqa{Hq}-bf16", "bf16", B=2, Hq=Hq, Hkv=Hkv, D=128, rope_base=500000.0,
                        F=9, hist_len=70, hist_pool=3, n_items=4, item_len=33, item_pool=6, pct=25)
    w = inputs.make(cfg, 55 + Hq, device=DEV)
    r = run_both(cfg, w, cfg.k)
    rows = check_against_assembled(w, r)
    ocos, osin = O.rope_table(cfg.N, cfg.D, cfg.rope_base)
    subpools, segs_sub = inputs.referenced_subpools(w)
    kf, vf = H(w.k_fresh), H(w.v_fresh)
    ka_o, va_o = O.assemble(kf, vf, subpools, segs_sub, ocos, osin)
    kp_o, vp_o = O.patch(w.segs.numpy(), rows, kf, vf, ka_o, va_o)
    np.testing.assert_array_equal(H(r["k_ref"]), kp_o)
    sel = sample_rows(cfg.B, rows.shape[1], 1)
    ref = oracle_attention_rows(H(w.q), kp_o, vp_o, rows, sel)
    g = np.concatenate([H(r["out_r"])[b, idx] for b, idx in enumerate(sel)])
    assert_attn_close(g, np.concatenate(ref), cfg.dtype, f"vref attention, Hq={Hq}, one KV head")


def test_vref_chain_single_partial_tile():
    """A prompt shorter than one key tile (N = 40): the attention's only tile
    is partial and takes its V rows through the table too."""
    cfg = inputs.Config("short-bf16", "bf16", B=3, Hq=8, Hkv=2, D=128, rope_base=500000.0, F=8,
                        hist_len=16, hist_pool=3, n_items=1, item_len=16, item_pool=4, pct=40)
    assert cfg.N < 64
    w = inputs.make(cfg, 77, device=DEV)
    r = run_both(cfg, w, cfg.k)
    rows = check_against_assembled(w, r)
    ocos, osin = O.rope_table(cfg.N, cfg.D, cfg.rope_base)
    subpools, segs_sub = inputs.referenced_subpools(w)
    kf, vf = H(w.k_fresh), H(w.v_fresh)
    ka_o, va_o = O.assemble(kf, vf, subpools, segs_sub, ocos, osin)
    kp_o, vp_o = O.patch(w.segs.numpy(), rows, kf, vf, ka_o, va_o)
    np.testing.assert_array_equal(H(r["k_ref"]), kp_o)
    sel = sample_rows(cfg.B, rows.shape[1], 1)
    ref = oracle_attention_rows(H(w.q), kp_o, vp_o, rows, sel)
    g = np.concatenate([H(r["out_r"])[b, idx] for b, idx in enumerate(sel)])
    assert_attn_close(g, np.concatenate(ref), cfg.dtype, "vref attention, one partial tile")


@pytest.mark.parametrize("cid,stride", [(2, 16), (3, 32), (4, 16), (5, 64)])
def test_vref_chain_full_workloads(cid, stride):
    """Full sizes at 15% recompute, in the launch configuration the benchmark
    times: the chain is bit-identical to the assembled one, K against the
    oracle, and sampled rows of the attention against the oracle."""
    cfg = inputs.WORKLOADS[cid]
    k = cfg.k_for(15)
    say(f"[vref] workload {cid} B={cfg.B} N={cfg.N} k={k}")
    w = inputs.make(cfg, 4200 + cid, device=DEV)
    r = run_both(cfg, w, k)
    rows = check_against_assembled(w, r)
    ocos, osin = O.rope_table(cfg.N, cfg.D, cfg.rope_base)
    subpools, segs_sub = inputs.referenced_subpools(w)
    kf, vf = H(w.k_fresh), H(w.v_fresh)
    ka_o, va_o = O.assemble(kf, vf, subpools, segs_sub, ocos, osin)
    np.testing.assert_array_equal(H(r["k_pre"]), ka_o, err_msg="assembled K differs from the oracle")
    kp_o, vp_o = O.patch(w.segs.numpy(), rows, kf, vf, ka_o, va_o)
    np.testing.assert_array_equal(H(r["k_ref"]), kp_o, err_msg="patched K differs from the oracle")
    sel = sample_rows(cfg.B, rows.shape[1], stride)
    ref = oracle_attention_rows(H(w.q), kp_o, vp_o, rows, sel)
    outh = H(r["out_r"])
    g = np.concatenate([outh[b, idx] for b, idx in enumerate(sel)])
    say(f"  {assert_attn_close(g, np.concatenate(ref), cfg.dtype, 'vref attention')}")
    del w, r
    torch.cuda.empty_cache()


def test_vref_full_prefill_mode_equals_plain():
    """rows = NULL (every row, the Full-Recompute baseline) through a table
    that points at the rows of V itself: bit-identical to the plain call."""
    cfg = inputs.TEST_WORKLOADS["ragged-bf16"]
    w = inputs.make(cfg, 11, device=DEV)
    B, N, Hkv, D = w.v_fresh.shape
    row_bytes = Hkv * D * w.v_fresh.element_size()
    table = (w.v_fresh.data_ptr() + row_bytes * torch.arange(B * N, device=DEV, dtype=torch.int64)).view(B, N)
    ref = ops.selective_attention(w.q, w.k_fresh, w.v_fresh)
    got = ops.selective_attention_vref(w.q, w.k_fresh, table)
    torch.cuda.synchronize()
    np.testing.assert_array_equal(H(got), H(ref))


def test_vref_unresolved_positions_point_at_fresh_rows():
    """A segment naming a block outside its pool leaves its positions
    unresolved: the gather writes no key row there (as rc_kv_assemble) and
    their table entries address the fresh V rows, so that the table never
    holds an unreadable address."""
    cfg = inputs.TEST_WORKLOADS["tiny-bf16"]
    w = inputs.make(cfg, 21, device=DEV)
    segs_h = w.segs.clone()
    bad = [s for s in range(segs_h.shape[1]) if int(segs_h[0, s, 2]) >= 0][0]
    pool = int(segs_h[0, bad, 2])
    segs_h[0, bad, 3] = w.pools[pool][0].shape[0] + 5          # block past the pool's end
    segs = ops.prepare_segments(segs_h, cfg.N, w.pools, DEV, check_blocks=False)
    cos, sin = ops.rope_table(cfg.N, cfg.D, cfg.rope_base, DEV)
    k_ref = torch.zeros_like(w.k_fresh)
    k_ref, v_ref = ops.kv_assemble_vref(w.pools, segs, w.k_fresh, w.v_fresh, cos, sin, k_out=k_ref)
    torch.cuda.synchronize()
    dst, ln = int(segs_h[0, bad, 0]), int(segs_h[0, bad, 1])
    row_bytes = cfg.Hkv * cfg.D * w.v_fresh.element_size()
    want = w.v_fresh.data_ptr() + row_bytes * (np.arange(dst, dst + ln, dtype=np.int64))
    np.testing.assert_array_equal(v_ref.cpu().numpy()[0, dst:dst + ln], want)
    assert not k_ref[0, dst:dst + ln].any(), "unresolved key rows must not be written"
    # the other entries are those of the well-formed table
    good = expected_vref(w, np.full((cfg.B, 0), -1, np.int32))
    got = v_ref.cpu().numpy()
    mask = np.ones_like(got, dtype=bool)
    mask[0, dst:dst + ln] = False
    np.testing.assert_array_equal(got[mask], good[mask])


def test_vref_fp32_gather_and_patch_exact_attention_rejected():
    """The tiny fp32 workload (workload 1): the gather and the patch through
    references work for any dtype and match the assembled chain; the
    attention through references is bf16-only and says so."""
    cfg = inputs.WORKLOADS[1]
    w = inputs.make(cfg, 1001, device=DEV)
    segs = ops.prepare_segments(w.segs, cfg.N, w.pools, DEV)
    cos, sin = ops.rope_table(cfg.N, cfg.D, cfg.rope_base, DEV)
    sc_a = torch.empty((cfg.B, cfg.N), dtype=torch.float32, device=DEV)
    k_asm, v_asm = ops.kv_assemble(w.pools, segs, w.k_fresh, w.v_fresh, cos, sin, scores_out=sc_a)
    rows_a, _ = ops.select_tokens(segs, cfg.k, w.k_fresh, w.v_fresh, k_asm, v_asm, scores_in=sc_a)
    sc_r = torch.empty_like(sc_a)
    k_ref, v_ref = ops.kv_assemble_vref(w.pools, segs, w.k_fresh, w.v_fresh, cos, sin, scores_out=sc_r)
    rows_r, _ = ops.select_tokens_vref(segs, cfg.k, w.k_fresh, w.v_fresh, k_ref, v_ref, scores_in=sc_r)
    torch.cuda.synchronize()
    np.testing.assert_array_equal(sc_r.cpu().numpy(), sc_a.cpu().numpy())
    rows = rows_r.cpu().numpy()
    np.testing.assert_array_equal(rows, rows_a.cpu().numpy())
    np.testing.assert_array_equal(H(k_ref), H(k_asm))
    np.testing.assert_array_equal(v_ref.cpu().numpy(), expected_vref(w, rows))
    with pytest.raises(_lib.RcError) as e:
        ops.selective_attention_vref(w.q, k_ref, v_ref, rows_r)
    assert e.value.status == _lib.RC_ERR_UNSUPPORTED


def test_vref_rejects_unsupported_shapes():
    cfg = inputs.TEST_WORKLOADS["mha-d64-bf16"]
    w = inputs.make(cfg, 7, device=DEV)
    segs = ops.prepare_segments(w.segs, cfg.N, w.pools, DEV)
    cos, sin = ops.rope_table(cfg.N, cfg.D, cfg.rope_base, DEV)
    k_ref, v_ref = ops.kv_assemble_vref(w.pools, segs, w.k_fresh, w.v_fresh, cos, sin)
    rows, _ = ops.select_tokens_vref(segs, cfg.k, w.k_fresh, w.v_fresh, k_ref, v_ref)
    with pytest.raises(_lib.RcError) as e:
        ops.selective_attention_vref(w.q, k_ref, v_ref, rows)
    assert e.value.status == _lib.RC_ERR_UNSUPPORTED
    torch.cuda.synchronize()
