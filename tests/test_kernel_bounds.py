"""Host models of the launch geometry and index arithmetic of the row kernels
that run in the decoder-stack path, at the Llama-3-8B-layer shapes of the
stack test (B = 8, N = 3008, hidden 4096, MLP 14336, 32/8 heads of 128,
R = 520 rows per request after a 16-position window): every global read and
write of every thread must fall inside its buffer. Each model restates the
kernel's own index expressions (csrc/layer.hip, csrc/assemble.hip) for the
whole grid, vectorised over blocks and threads; the kernels' compile-time
constants are read from the sources so that a change there is seen here.
CPU only."""
import os
import re

import numpy as np
import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
CSRC = os.path.join(ROOT, "paper_2605_07443_amd", "csrc")

B, N, HID, INTER, R, HQ, HKV, D = 8, 3008, 4096, 14336, 520, 32, 8, 128


def _const(src, name):
    text = open(os.path.join(CSRC, src)).read()
    m = re.search(rf"constexpr int [^;]*\b{name} = ([^,;]+)[,;]", text)
    assert m, f"{name} not found in {src}"
    return m.group(1).strip()


def _check(what, lo, hi_excl, size):
    """Every access [lo, hi_excl) (element offsets) lies inside [0, size)."""
    lo, hi_excl = np.asarray(lo), np.asarray(hi_excl)
    assert lo.size == 0 or (lo.min() >= 0 and hi_excl.max() <= size), (
        f"{what}: accesses [{lo.min()}, {hi_excl.max()}) outside [0, {size})")


def _rows_with_window(seed=0):
    """Row lists like the stack's: fresh positions, the last 16 positions and
    sorted random others, R per request."""
    rng = np.random.default_rng(seed)
    rows = np.empty((B, R), np.int64)
    fixed = np.r_[np.arange(64), np.arange(N - 16, N)]
    for b in range(B):
        rest = rng.choice(np.arange(64, N - 16), R - fixed.size, replace=False)
        rows[b] = np.sort(np.r_[fixed, rest])
    return rows


THREADS = int(_const("layer.hip", "kRowThreads"))
NORM_UNITS = int(_const("layer.hip", "kNormMaxUnits"))


@pytest.mark.parametrize("M", [B * N, B * R])
def test_rmsnorm_bounds(M):
    """rmsnorm_kernel: block = row, thread t handles 16-byte units
    t + j * threads (j < kNormMaxUnits) that are below H / 8."""
    H = HID
    units = H // 8
    assert units <= NORM_UNITS * THREADS          # the host's H <= 8192 check
    t = np.arange(THREADS)[:, None]
    j = np.arange(NORM_UNITS)[None, :]
    u = (t + j * THREADS).ravel()
    u = u[u < units]
    row = np.array([0, M - 1])[:, None]           # offsets are affine in the row
    x_lo = row * H + u * 8
    _check("rmsnorm x / y", x_lo, x_lo + 8, M * H)
    _check("rmsnorm gamma", u * 8, u * 8 + 8, H)


@pytest.mark.parametrize("layer1", [True, False])
def test_qkv_rope_bounds(layer1):
    """qkv_rope_kernel: block m = b * R + r, position rows[m] (r when rows is
    NULL); threads loop over q pairs, k pairs and v units."""
    Rr = N if layer1 else R
    M = B * Rr
    rows = np.broadcast_to(np.arange(N), (B, N)) if layer1 else _rows_with_window()
    pos = rows.reshape(-1)
    assert pos.min() >= 0 and pos.max() < N
    m = np.arange(M)
    b = m // Rr
    half_units = D // 16
    q_pairs, k_pairs, v_units = HQ * half_units, HKV * half_units, HKV * 2 * half_units
    row_w = (HQ + 2 * HKV) * D                    # elements of one qkv row
    its = np.arange(q_pairs + k_pairs + v_units)
    # every thread visits it = tid, tid + 256, ...: together all of `its`
    assert set(np.concatenate([np.arange(t, its.size, THREADS) for t in range(THREADS)])) == set(its)
    pq = its[its < q_pairs + k_pairs]
    isq = pq < q_pairs
    p = np.where(isq, pq, pq - q_pairs)
    head = p // half_units
    u = p - head * half_units
    base = np.where(isq, 0, HQ * 2 * half_units) + head * 2 * half_units
    src_units = np.r_[base + u, base + u + half_units]
    for mm in (m[:1], m[-1:]):                    # affine in m: the extremes bound it
        lo = mm[:, None] * row_w + src_units[None, :] * 8
        _check("qkv source (q, k pairs)", lo, lo + 8, M * row_w)
    vu = its[its >= q_pairs + k_pairs] - q_pairs - k_pairs
    lo = m[-1] * row_w + ((HQ + HKV) * 2 * half_units + vu) * 8
    _check("qkv source (v units)", lo, lo + 8, M * row_w)
    # destinations at the row's position
    row_q = (b * N + pos) * HQ * D
    row_kv = (b * N + pos) * HKV * D
    hq, uq = head[isq], u[isq]
    hk, uk = head[~isq], u[~isq]
    for r0 in (row_q.min(), row_q.max()):
        lo = r0 + np.r_[hq * D + uq * 8, hq * D + (uq + half_units) * 8]
        _check("q_out", lo, lo + 8, B * N * HQ * D)
    for r0 in (row_kv.min(), row_kv.max()):
        lo = r0 + np.r_[hk * D + uk * 8, hk * D + (uk + half_units) * 8]
        _check("k_out", lo, lo + 8, B * N * HKV * D)
        lo = r0 + vu * 8
        _check("v_out", lo, lo + 8, B * N * HKV * D)
    # cos/sin at the row's position (tables of N positions)
    lo = pos.max() * (D // 2) + u * 8
    _check("rope tables", lo, lo + 8, N * (D // 2))


@pytest.mark.parametrize("M", [B * R, B * N])
def test_silu_mul_bounds(M):
    """silu_mul_kernel: flat index over M * I / 8 units, blocks of 256; the
    grid's last block is cut by idx < M * upr."""
    I = INTER
    upr = I // 8
    items = M * upr
    blocks = (items + THREADS - 1) // THREADS
    idx = np.array([0, items - 1, blocks * THREADS - 1])
    idx = idx[idx < items]
    mrow = idx // upr
    u = idx - mrow * upr
    g_lo = mrow * 2 * I + u * 8
    _check("silu gate", g_lo, g_lo + 8, M * 2 * I)
    _check("silu up", g_lo + I, g_lo + I + 8, M * 2 * I)
    o_lo = mrow * I + u * 8
    _check("silu out", o_lo, o_lo + 8, M * I)
    assert blocks < 2 ** 31


def test_gather_rows_bounds():
    """gather_rows_kernel: block m = b * R + r copies source row rows[m] of
    request b (skipped when outside [0, Nsrc)) to destination row m."""
    rows = _rows_with_window()
    row_bytes = HID * 2
    units = row_bytes // 16
    m = np.arange(B * R)
    b = m // R
    p = rows.reshape(-1)
    ok = (p >= 0) & (p < N)
    u = np.arange(units)
    src = (b[ok] * N + p[ok]) * units
    _check("gather_rows src", src.min() * 16, (src.max() + units) * 16, B * N * row_bytes)
    _check("gather_rows dst", m.min() * units * 16, (m.max() + 1) * units * 16, B * R * row_bytes)
    assert u.max() < units


ASM_THREADS = int(_const("assemble.hip", "kThreads"))
ASM_KPER = int(_const("assemble.hip", "kKPer"))
ASM_VPER = int(_const("assemble.hip", "kVPer"))
ASM_MAXTOK = int(_const("assemble.hip", "kMaxTok"))


def _window_segments():
    """The stack's table: 64 fresh, a 1024-token history block, 20 items of 96,
    the last 16 positions cut off into fresh single-token pieces and one
    remainder (the library's window rewrite)."""
    segs = [[0, 64, -1, 0], [64, 1024, 0, 3]]
    pos = 1088
    for i in range(20):
        segs.append([pos, 96, 1, 17 * i + 5])
        pos += 96
    # window of 16: the last item is cut at N - 16, the window is fresh
    last = segs[-1]
    last[1] -= 16
    segs.append([N - 16, 16, -1, 0])
    return np.array(segs, np.int64)


@pytest.mark.parametrize("score_only", [False, True])
def test_kv_rows_kernel_bounds(score_only):
    """kv_rows_kernel (assembly with the fused rotation and score, and the
    score-only pass): one block per TOK positions of a request; positions
    resolve to pool rows through the table; key pairs, fresh key pairs, value
    units, table entries and scores indexed as in the kernel."""
    es = 2
    row_bytes = HKV * D * es
    row_units = row_bytes // 16
    head_units = D * es // 16
    half_units = head_units // 2
    E = 16 // es
    half = D // 2
    k_items_cap = ASM_KPER * ASM_THREADS
    tok = max(1, min(ASM_MAXTOK, k_items_cap * 32 // row_bytes))
    segs = _window_segments()
    pools = {0: (256, 1024), 1: (400, 96)}                 # num_blocks, block_len
    ppr = row_units // 2
    assert tok * ppr <= k_items_cap                        # the host's scoring check
    pos = np.arange(N)
    seg_of = np.searchsorted(segs[:, 0], pos, side="right") - 1
    g = segs[seg_of]
    assert np.all(pos < g[:, 0] + g[:, 1])
    cached = g[:, 2] >= 0
    for p, (nb, bl) in pools.items():
        m = g[:, 2] == p
        src_row = g[m, 3] * bl + (pos[m] - g[m, 0])
        assert g[m, 3].max() < nb and (pos[m] - g[m, 0]).max() < bl
        _check(f"pool {p} rows", src_row * row_bytes, (src_row + 1) * row_bytes, nb * bl * row_bytes)
    delta = np.where(cached, g[:, 0], 0)
    assert delta.max() < N                                  # max_pos = N
    n_blk = (N + tok - 1) // tok
    for blk in (0, n_blk - 1):
        i0 = blk * tok
        tok_cnt = min(tok, N - i0)
        k_items = tok_cnt * ppr
        v_items = 0 if score_only else tok_cnt * row_units
        it = 0
        while it * k_items_cap < k_items or it * ASM_VPER * ASM_THREADS < v_items:
            idx = it * k_items_cap + np.arange(ASM_KPER)[:, None] * ASM_THREADS + np.arange(ASM_THREADS)
            idx = idx[idx < k_items]
            ktok = idx // ppr
            pr = idx - ktok * ppr
            head = pr // half_units
            kunit = head * head_units + (pr - head * half_units)
            assert (kunit + half_units).max() < row_units
            j0 = (kunit % head_units) * E
            assert (kunit % head_units).max() < half_units and (j0 + E).max() <= half
            for b in (0, B - 1):
                rows = b * N + i0 + ktok
                _check("fresh key pairs", rows * row_bytes + kunit * 16,
                       rows * row_bytes + (kunit + half_units) * 16 + 16, B * N * row_bytes)
                if not score_only:
                    _check("assembled key pairs", rows * row_bytes + kunit * 16,
                           rows * row_bytes + (kunit + half_units) * 16 + 16, B * N * row_bytes)
            vidx = it * ASM_VPER * ASM_THREADS + np.arange(ASM_VPER * ASM_THREADS)
            vidx = vidx[vidx < v_items]
            vtok, vunit = vidx // row_units, vidx % row_units
            assert vunit.max(initial=0) < row_units and vtok.max(initial=0) < tok_cnt
            d = delta[i0 + ktok]
            _check("rope tables", d * half + j0, d * half + j0 + E, N * half)
            it += 1
        assert k_items <= k_items_cap                        # one scoring pass (s_part size)
    _check("scores", np.array([0]), np.array([B * N]), B * N)


WAVE_KP = int(_const("assemble.hip", "kWaveGatherKP"))


@pytest.mark.parametrize("score_only", [False, True])
def test_kv_gather_kernel_bounds(score_only):
    """kv_gather_kernel (the wave-level assembly used when a request has at
    most 64 segments and a key row has a power-of-two pair count): wave w of
    block x owns positions (4x + w) T .. + T; lane l carries key pairs
    k * 64 + l and value units k * 64 + l of them."""
    es = 2
    row_bytes = HKV * D * es
    row_units = row_bytes // 16
    head_units = D * es // 16
    half_units = head_units // 2
    E = 16 // es
    half = D // 2
    ppr = row_units // 2
    assert ppr & (ppr - 1) == 0 and ppr <= 64 * WAVE_KP
    log2_ppr = ppr.bit_length() - 1
    T = (64 * WAVE_KP) >> log2_ppr
    waves = ASM_THREADS // 64
    grid_x = (N + waves * T - 1) // (waves * T)
    segs = _window_segments()
    assert segs.shape[0] <= 64
    lane = np.arange(64)
    for x in (0, grid_x - 1):
        for w in range(waves):
            i0 = (x * waves + w) * T
            if i0 >= N:
                continue
            k = np.arange(WAVE_KP)[:, None]
            q = k * 64 + lane                              # [KP, 64]
            kt = q >> log2_ppr
            pr = q & (ppr - 1)
            head = pr // half_units
            kunit = head * head_units + (pr - head * half_units)
            assert (kunit + half_units).max() < row_units
            live = i0 + kt < N
            for b in (0, B - 1):
                rows = (b * N + i0 + kt)[live]
                ku = kunit[live]
                _check("fresh / assembled key pairs", rows * row_bytes + ku * 16,
                       rows * row_bytes + (ku + half_units) * 16 + 16, B * N * row_bytes)
                _check("scores", b * N + i0 + kt[live], b * N + i0 + kt[live] + 1, B * N)
            if not score_only:
                kv = np.arange(2 * WAVE_KP)[:, None] * 64 + lane
                vt, vu = kv // row_units, kv % row_units
                vl = i0 + vt < N
                rows = ((B - 1) * N + i0 + vt)[vl]
                _check("value units", rows * row_bytes + vu[vl] * 16, rows * row_bytes + vu[vl] * 16 + 16,
                       B * N * row_bytes)
            j0 = (kunit % head_units) * E
            assert (j0 + E).max() <= half


def _gemm_split_plan(M, n, k):
    """rc_gemm_bf16's choice for a row tail, restated: (M_main, M_tail, splits)
    with splits >= 2 when the tail goes to split-K, else splits = 0."""
    kBM, kGM, kGN, kGK = (int(_const("gemm.hip", c)) for c in ("kBM", "kGM", "kGN", "kGK"))
    kSM, kSN = int(_const("gemm.hip", "kSM")), int(_const("gemm.hip", "kSN"))
    M_main = (M // kBM) * kBM
    M_tail = M - M_main
    KT = k // kGK
    small_tiles = -(-M_tail // kGM) * -(-n // kGN)
    split_tiles = -(-M_tail // kSM) * -(-n // kSN)
    s = 512 // max(split_tiles, 1)
    s = min(s, KT // 2)
    if M_tail > 0:
        s = min(s, M_main // (2 * M_tail))
    use = M_tail > 0 and small_tiles < 128 and s >= 2
    return M_main, M_tail, (s if use else 0)


@pytest.mark.parametrize("M,n,k", [(B * R, 3 * HQ * D // 2, HID), (B * R, HID, HID),
                                   (B * R, 2 * INTER, HID), (B * R, HID, INTER),
                                   (300, 650, 512), (1279, 512, 1024), (300, 640, 256)])
def test_gemm_split_tail_bounds(M, n, k):
    """The split-K row tail of rc_gemm_bf16 (gemm_bf16_splitk_kernel, then
    gemm_tail_reduce_kernel) at the stack's 4,160-row projection shapes and
    the GEMM test shapes: every X, W and partial access of every lane is in
    its buffer, every split covers at least two k tiles, the partials fit
    in the first M_main rows of y (whose bf16 bytes they borrow) and stay
    clear of the tail rows the reduction writes."""
    kSM, kSN, kGK = int(_const("gemm.hip", "kSM")), int(_const("gemm.hip", "kSN")), int(_const("gemm.hip", "kGK"))
    threads = int(_const("gemm.hip", "kSThreads"))
    M_main, M_tail, S = _gemm_split_plan(M, n, k)
    if S == 0:
        pytest.skip("tail not on split-K for this shape")
    KT = k // kGK
    assert S * M_tail * n * 4 <= M_main * n * 2          # partials inside y's body
    for s in range(S):
        kt0, kt1 = s * KT // S, (s + 1) * KT // S
        assert kt1 - kt0 >= 2 and 0 <= kt0 and kt1 <= KT
    # X staging: unit u = tid + i * threads, row u // 8 (guarded by M_tail),
    # 16-byte unit at k offset kt * 64 + (u % 8) * 8 of row M_main + row
    u = np.arange(threads)[:, None] + np.arange(kSM * 8 // threads)[None, :] * threads
    rows = (np.arange(-(-M_tail // kSM))[:, None, None] * kSM + (u // 8)[None]).ravel()
    rows = rows[rows < M_tail]
    kk_max = (KT - 1) * kGK + 7 * 8
    _check("split-K X", (M_main + rows) * k, (M_main + rows) * k + kk_max + 8, M * k)
    # W fragments: row min(n0 + 16 * wave + c16, n - 1), k offset kt * 64 + ks * 32 + q4 * 8
    n0 = np.arange(-(-n // kSN))[:, None] * kSN
    wrow = np.minimum(n0 + np.arange(kSN)[None, :], n - 1).ravel()
    _check("split-K W", wrow * k, wrow * k + (KT - 1) * kGK + 32 + 3 * 8 + 8, n * k)
    # partial stores: part[s][row][col], row < M_tail, col < n (floats)
    _check("split-K partials", 0, S * M_tail * n, S * M_tail * n)
    # the reduction reads part[s * count + e] and writes y[M_main * n + e], e < count
    count = M_tail * n
    _check("reduce partials", 0, (S - 1) * count + count, S * count)
    _check("reduce output", M_main * n, M_main * n + count, M * n)
    # partial bytes end before the tail rows of y begin
    assert S * count * 4 <= M_main * n * 2


@pytest.mark.parametrize("Hkv,D,es", [(1, 128, 2), (2, 128, 2), (4, 128, 2), (8, 128, 2),
                                      (2, 64, 2), (8, 64, 4)])
@pytest.mark.parametrize("n", [1, 40, 64, 65, 1000, 3008])
def test_value_reference_table_coverage(Hkv, D, es, n):
    """The gather with V by reference: lane t < T of wave (4x + w) writes the
    entry of position (4x + w) T + t. Every entry of [B, N] is written
    exactly once (so that the attention never reads an unwritten address),
    and the attention's table loads (lane l of wave w reads, for the pair of
    tiles starting at t, the entry of key (t + (l / 16) % 2) * 64 + 16 w +
    l % 16, clamped to N - 1) stay inside the request's N entries."""
    row_units = Hkv * D * es // 16
    ppr = row_units // 2
    assert ppr & (ppr - 1) == 0 and 1 <= ppr <= 64 * WAVE_KP
    T = (64 * WAVE_KP) // ppr
    assert T <= 64
    waves = ASM_THREADS // 64
    grid_x = (n + waves * T - 1) // (waves * T)
    hits = np.zeros(n, np.int64)
    lane = np.arange(64)
    for x in range(grid_x):
        for w in range(waves):
            i0 = (x * waves + w) * T
            if i0 >= n:
                continue
            live = (lane < T) & (i0 + lane < n)
            np.add.at(hits, (i0 + lane)[live], 1)
    assert (hits == 1).all(), "table entries written other than once"
    kkt = 64
    n_kv = (n - 1) // kkt + 1
    for t in range(0, n_kv + 1, 2):          # the prologue's pair and every even tile's
        for w in range(4):
            key = np.minimum((t + ((lane >> 4) & 1)) * kkt + w * 16 + (lane & 15), n - 1)
            assert key.min() >= 0 and key.max() < n
