"""GPU parity of the zero-copy path (paged attention through the segment
table, score-only alignment pass) and of the local sliding window (arXiv
2605.07443, Sec. III-A block mapping, Sec. III-C.2b, III-C.3), called
through the C ABI.

Bar: the paged path computes the assembled path's tiles bit for bit, so its
rows and outputs equal the assembled path's exactly; its outputs are within
the attention tolerance of the oracle (assemble -> patch -> attention); the
score-only pass equals the fused gather scores exactly."""
import numpy as np
import pytest
import torch

from oracle import oracle as O
from paper_2605_07443_amd import inputs, ops

from parity import H, assert_attn_close, oracle_attention_rows, sample_rows, say

pytestmark = pytest.mark.gpu

DEV = torch.device("cuda:0")


@pytest.fixture(scope="module", autouse=True)
def _lib_loaded():
    from paper_2605_07443_amd import _lib
    _lib.load()
    yield
    torch.cuda.synchronize()


def _both(cfg, w, segs_np, k, check_oracle=True, stride=1):
    segs = ops.prepare_segments(segs_np, cfg.N, w.pools, DEV)
    cos, sin = ops.rope_table(cfg.N, cfg.D, cfg.rope_base, DEV)
    a = ops.selective_prefill(w.q, w.k_fresh, w.v_fresh, w.pools, segs, k, cos, sin)
    p = ops.paged_prefill(w.q, w.k_fresh, w.v_fresh, w.pools, segs, k, cos, sin)
    torch.cuda.synchronize()
    assert torch.equal(a.scores, p.scores), "score-only pass differs from the fused gather scores"
    assert torch.equal(a.rows, p.rows), "rows differ"
    assert torch.equal(a.out, p.out), "paged attention differs from the assembled path"
    if check_oracle and a.rows.shape[1] > 0:
        ocos, osin = O.rope_table(cfg.N, cfg.D, cfg.rope_base)
        sub = inputs.Workload(cfg=cfg, seed=w.seed, q=w.q, k_fresh=w.k_fresh, v_fresh=w.v_fresh,
                              pools=w.pools, segs=torch.from_numpy(np.asarray(segs_np)),
                              item_ids=w.item_ids, hist_ids=w.hist_ids)
        subpools, segs_sub = inputs.referenced_subpools(sub)
        kf, vf = H(w.k_fresh), H(w.v_fresh)
        ka, va = O.assemble(kf, vf, subpools, segs_sub, ocos, osin)
        rows = p.rows.cpu().numpy()
        kp, vp = O.patch(np.asarray(segs_np), rows, kf, vf, ka, va)
        sel = sample_rows(cfg.B, rows.shape[1], stride)
        ref = np.concatenate(oracle_attention_rows(H(w.q), kp, vp, rows, sel))
        got = np.concatenate([H(p.out)[b, idx] for b, idx in enumerate(sel)])
        return assert_attn_close(got, ref, cfg.dtype, "paged attention")
    return {}


SMALL = ["tiny-bf16", "ragged-bf16", "mha-d64-bf16", "miss-bf16"]


@pytest.mark.parametrize("name", SMALL)
@pytest.mark.parametrize("pct", [0, 15, 100])
def test_paged_equals_assembled_small(name, pct):
    cfg = inputs.TEST_WORKLOADS[name]
    say(f"[paged] {name} pct={pct}")
    w = inputs.make(cfg, 500 + pct, device=DEV)
    say(f"  {_both(cfg, w, w.segs.numpy(), cfg.k_for(pct))}")


@pytest.mark.parametrize("name", ["tiny-bf16", "miss-bf16", "ragged-bf16"])
@pytest.mark.parametrize("W", [1, 16, 50])
def test_sliding_window_both_paths(name, W):
    """The last W positions become fresh segments: they are always rows, carry
    fresh K/V, and both paths agree with each other and the oracle."""
    cfg = inputs.TEST_WORKLOADS[name]
    say(f"[window] {name} W={W}")
    w = inputs.make(cfg, 600 + W, device=DEV)
    segs_w = ops.segments_with_window(w.segs.numpy(), cfg.N, W)
    F = int(O.fresh_count(segs_w)[0])
    n_r = cfg.N - F
    k = (n_r * 15 + 99) // 100
    _both(cfg, w, segs_w, k)
    segs = ops.prepare_segments(segs_w, cfg.N, w.pools, DEV)
    cos, sin = ops.rope_table(cfg.N, cfg.D, cfg.rope_base, DEV)
    bufs = ops.selective_prefill(w.q, w.k_fresh, w.v_fresh, w.pools, segs, k, cos, sin)
    torch.cuda.synchronize()
    rows = bufs.rows.cpu().numpy()
    for b in range(cfg.B):
        assert set(range(cfg.N - W, cfg.N)) <= set(rows[b].tolist())
    assert torch.equal(bufs.k_asm[:, cfg.N - W:], w.k_fresh[:, cfg.N - W:])
    assert torch.equal(bufs.v_asm[:, cfg.N - W:], w.v_fresh[:, cfg.N - W:])


def test_paged_unsorted_rows_and_duplicates():
    """Rows in any order, with repeats, still read fresh K/V for every listed
    position and match the assembled path patched at the same rows."""
    cfg = inputs.TEST_WORKLOADS["ragged-bf16"]
    w = inputs.make(cfg, 77, device=DEV)
    segs = ops.prepare_segments(w.segs, cfg.N, w.pools, DEV)
    cos, sin = ops.rope_table(cfg.N, cfg.D, cfg.rope_base, DEV)
    g = torch.Generator().manual_seed(3)
    rows = torch.randint(0, cfg.N, (cfg.B, 37), generator=g, dtype=torch.int32)
    rows[:, 5] = rows[:, 9]
    rows = rows.to(DEV)
    out_p = ops.paged_attention(w.q, w.k_fresh, w.v_fresh, w.pools, segs, rows, cos, sin)
    k_asm, v_asm = ops.kv_assemble(w.pools, segs, w.k_fresh, w.v_fresh, cos, sin)
    for b in range(cfg.B):
        idx = rows[b].long()
        k_asm[b, idx] = w.k_fresh[b, idx]
        v_asm[b, idx] = w.v_fresh[b, idx]
    out_a = ops.selective_attention(w.q, k_asm, v_asm, rows)
    torch.cuda.synchronize()
    assert torch.equal(out_p, out_a)


@pytest.mark.parametrize("cid,stride", [(2, 16), (5, 64), (3, 64)])
def test_paged_full_workloads(cid, stride):
    """Workload sizes in the benchmark's launch configuration: exact equality
    with the assembled path everywhere, oracle check on sampled rows."""
    cfg = inputs.WORKLOADS[cid]
    say(f"[paged] config {cid} B={cfg.B} N={cfg.N} S={cfg.n_items + 2}")
    w = inputs.make(cfg, 1000 * cid, device=DEV)
    say(f"  {_both(cfg, w, w.segs.numpy(), cfg.k, stride=stride)}")
    del w
    torch.cuda.empty_cache()
