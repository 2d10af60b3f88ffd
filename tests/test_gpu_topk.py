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
