"""GPU parity of the heavy-hitter top-k (Sec. III-C.2b) on requests longer than
one workgroup's 1024 threads: every thread then holds several positions, and
equal scores straddle the per-thread chunks. Rows are compared bit for bit
with the oracle on identical scores, for the single budget and for the
separate history / item budgets."""
import numpy as np
import pytest
import torch

from oracle import oracle as O
from paper_2605_07443_amd import ops

from parity import H

pytestmark = pytest.mark.gpu

DEV = torch.device("cuda:0")


def _segments(N, S, B, rng):
    """S runs tiling [0, N), each fresh (pool -1) or cached from pool 0 or 1;
    the same runs for every request (one fresh count)."""
    cuts = np.sort(rng.choice(np.arange(1, N), S - 1, replace=False))
    starts = np.concatenate([[0], cuts])
    lens = np.diff(np.concatenate([starts, [N]]))
    kinds = rng.integers(-1, 2, S)
    kinds[0] = 0  # at least one cached run
    seg = np.stack([starts, lens, kinds, np.zeros(S, np.int64)], 1).astype(np.int32)
    return np.ascontiguousarray(np.broadcast_to(seg, (B, S, 4)))


def _scores(kind, B, N, rng):
    if kind == "ties":
        sc = rng.integers(0, 6, (B, N)).astype(np.float32)
    else:  # keys spread over many binades: several radix passes
        sc = (np.exp(rng.normal(0.0, 6.0, (B, N))) * rng.choice([-1.0, 1.0], (B, N))).astype(np.float32)
        sc[:, ::7] = sc[:, 3:4]  # a repeated value in every chunk
    sc[0, N // 2] = np.nan
    sc[0, N - 1] = np.inf
    sc[1 % B, 1] = -np.inf
    sc[1 % B, N // 3] = -0.0
    return sc


def _dummy_kv(B, N):
    return torch.empty((B, N, 1, 64), dtype=torch.bfloat16, device=DEV)


@pytest.mark.parametrize("N,S", [(1025, 9), (3008, 40), (5000, 1024), (16384, 300)])
@pytest.mark.parametrize("kind", ["ties", "spread"])
def test_topk_several_chunks_per_thread(N, S, kind):
    B = 3
    rng = np.random.default_rng(N + S)
    segs_h = _segments(N, S, B, rng)
    segs = ops.prepare_segments(segs_h, N, [(None, None)] * 2, DEV, check_blocks=False)
    n_reused = N - segs.n_fresh
    sc = _scores(kind, B, N, rng)
    kf = _dummy_kv(B, N)
    sc_d = torch.from_numpy(sc).to(DEV)
    for k in sorted({0, 1, n_reused // 3, n_reused - 1, n_reused}):
        print(f"topk N={N} S={S} {kind} k={k}", flush=True)
        rows, _ = ops.select_tokens(segs, k, kf, kf, None, None, scores_in=sc_d, patch=False)
        torch.cuda.synchronize()
        np.testing.assert_array_equal(rows.cpu().numpy(), O.topk(segs_h, N, k, sc), err_msg=f"k={k}")


@pytest.mark.parametrize("N,S", [(2048, 33), (9000, 700)])
def test_split_topk_several_chunks_per_thread(N, S):
    B = 2
    rng = np.random.default_rng(7 * N + S)
    segs_h = _segments(N, S, B, rng)
    segs = ops.prepare_segments(segs_h, N, [(None, None)] * 2, DEV, check_blocks=False)
    mask = 0b10  # pool 1 holds items
    nh, ni = ops.component_counts(segs, mask)
    nh, ni = int(nh.min()), int(ni.min())
    kf = _dummy_kv(B, N)
    for kind in ("ties", "spread"):
        sc = _scores(kind, B, N, rng)
        sc_d = torch.from_numpy(sc).to(DEV)
        for kh, ki in [(0, 1), (1, 0), (nh // 2, ni // 3), (nh, ni), (nh - 1, 0), (3, ni)]:
            print(f"split topk N={N} S={S} {kind} kh={kh} ki={ki}", flush=True)
            rows, _ = ops.select_tokens_eq3(segs, mask, 0.5, kh, ki, kf, kf, None, None,
                                            scores_in=sc_d, patch=False)
            torch.cuda.synchronize()
            np.testing.assert_array_equal(rows.cpu().numpy(),
                                          O.topk_split(segs_h, N, mask, kh, ki, sc),
                                          err_msg=f"kh={kh} ki={ki}")


def _random_scores(kind, B, N, rng):
    if kind == "zero":        # every key equal: selection by position alone
        return np.zeros((B, N), np.float32)
    if kind == "signed-zero":
        return np.where(rng.random((B, N)) < 0.5, np.float32(-0.0), np.float32(0.0)).astype(np.float32)
    if kind == "nan-heavy":
        sc = rng.random((B, N)).astype(np.float32)
        sc[rng.random((B, N)) < 0.3] = np.nan
        sc[rng.random((B, N)) < 0.1] = np.inf
        return sc
    if kind == "few-values":
        return rng.choice(np.array([0.25, 0.5, 1.0, 3.0], np.float32), (B, N))
    return np.abs(rng.standard_normal((B, N))).astype(np.float32)


SWEEP_N = [1, 2, 3, 64, 1023, 1024, 1025, 2047, 2048, 2049, 3008, 16383, 16384]


@pytest.mark.parametrize("case", range(len(SWEEP_N)))
def test_topk_and_patch_random_sweep(case):
    """Seeded random requests at the chunk boundaries of the 1024-thread
    selection (and N = 1..3, 16384), random segment tables (fresh and cached
    runs), budgets from 0 to every cached position, and degenerate score sets
    (all zero, signed zeros, many NaN/inf, four values): rows bit-exact with
    the oracle; with the patch, the assembled K/V rows bit-exact with the
    oracle's patch."""
    N = SWEEP_N[case]
    rng = np.random.default_rng(9000 + case)
    B = 2
    S = int(rng.integers(1, min(N, 1024) + 1))
    if S == 1:
        segs_h = np.ascontiguousarray(np.broadcast_to(np.array([[0, N, 0, 0]], np.int32), (B, 1, 4)))
    else:
        segs_h = _segments(N, S, B, rng)
    segs = ops.prepare_segments(segs_h, N, [(None, None)] * 2, DEV, check_blocks=False)
    n_reused = N - segs.n_fresh
    g = torch.Generator().manual_seed(case)
    kf = torch.randn((B, N, 1, 64), generator=g).to(torch.bfloat16).to(DEV)
    vf = torch.randn((B, N, 1, 64), generator=g).to(torch.bfloat16).to(DEV)
    ka0 = torch.randn((B, N, 1, 64), generator=g).to(torch.bfloat16)
    va0 = torch.randn((B, N, 1, 64), generator=g).to(torch.bfloat16)
    kinds = ["zero", "signed-zero", "nan-heavy", "few-values", "spread"]
    for kind in kinds:
        sc = _random_scores(kind, B, N, rng)
        sc_d = torch.from_numpy(sc).to(DEV)
        ks = sorted({0, n_reused, int(rng.integers(0, n_reused + 1)), min(1, n_reused)})
        for k in ks:
            print(f"sweep N={N} S={S} {kind} k={k}", flush=True)
            ka, va = ka0.to(DEV), va0.to(DEV)
            rows, _ = ops.select_tokens(segs, k, kf, vf, ka, va, scores_in=sc_d, patch=True)
            torch.cuda.synchronize()
            rows_h = rows.cpu().numpy()
            np.testing.assert_array_equal(rows_h, O.topk(segs_h, N, k, sc), err_msg=f"{kind} k={k}")
            kp, vp = O.patch(segs_h, rows_h, H(kf), H(vf), H(ka0), H(va0))
            np.testing.assert_array_equal(H(ka), kp, err_msg=f"patched K, {kind} k={k}")
            np.testing.assert_array_equal(H(va), vp, err_msg=f"patched V, {kind} k={k}")
