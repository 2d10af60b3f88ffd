"""CPU-side checks of the C ABI: the library loads, exports every symbol the
header declares, builds the same RoPE tables as the oracle, and rejects bad
arguments on the host before anything is enqueued (no GPU needed)."""
import ctypes
import os
import re

import numpy as np
import pytest

from oracle import oracle as O
from paper_2605_07443_amd import _lib

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "rcllm.h")


@pytest.fixture(scope="module")
def lib():
    if not os.path.exists(_lib.LIB_PATH):
        from paper_2605_07443_amd import build
        build.build()
    return _lib.load()


def test_header_declarations_are_exported(lib):
    text = open(HEADER).read()
    declared = set(re.findall(r"^\s*(?:const\s+)?\w+\*?\s+\*?(rc_\w+)\s*\(", text, re.M))
    assert declared == set(_lib.EXPORTS)
    for name in declared:
        assert hasattr(lib, name), name


def test_binding_argument_counts_match_header(lib):
    """Every ctypes binding passes as many arguments as its header
    declaration has parameters."""
    text = re.sub(r"/\*.*?\*/", "", open(HEADER).read(), flags=re.S)
    decls = re.findall(r"^\s*(?:const\s+)?\w+\*?\s+\*?(rc_\w+)\s*\(([^)]*)\)\s*;", text, re.M)
    assert {name for name, _ in decls} == set(_lib.EXPORTS)
    for name, params in decls:
        p = params.strip()
        n = 0 if p in ("", "void") else p.count(",") + 1
        assert len(getattr(lib, name).argtypes) == n, name


def test_status_strings(lib):
    assert _lib.status_string(0) == "RC_OK"
    assert _lib.status_string(-1) == "RC_ERR_INVALID_ARG"
    assert _lib.status_string(-2) == "RC_ERR_UNSUPPORTED"
    assert _lib.status_string(-3) == "RC_ERR_HIP"


@pytest.mark.parametrize("max_pos,D,base", [(416, 64, 10000.0), (8160, 128, 500000.0)])
def test_rope_table_bitwise_equals_oracle_table(lib, max_pos, D, base):
    """Two independent fp64 -> fp32 table builders agree bit for bit, so the
    fused re-alignment can be compared bit-exactly."""
    cos = np.empty((max_pos, D // 2), np.float32)
    sin = np.empty((max_pos, D // 2), np.float32)
    assert lib.rc_rope_table(max_pos, D, base, cos.ctypes.data, sin.ctypes.data) == 0
    ocos, osin = O.rope_table(max_pos, D, base)
    np.testing.assert_array_equal(cos, ocos)
    np.testing.assert_array_equal(sin, osin)


FAKE = 0x1000  # never dereferenced: every case below fails host validation

# Belt and braces: on a machine with a GPU a validation bug would launch a
# kernel on these fake pointers, so the fake-pointer cases only run without
# one (device_count() does not initialise the GPU).
import torch  # noqa: E402

no_gpu = pytest.mark.skipif(torch.cuda.device_count() > 0,
                            reason="fake-pointer validation cases run only on GPU-less hosts")


def _shape(B=2, N=64, Hq=8, Hkv=2, D=128, dtype=1):
    return ctypes.byref(_lib.RcShape(B, N, Hq, Hkv, D, dtype))


def _pools(n=1, nb=4, bl=16):
    arr = (_lib.RcPool * max(n, 1))()
    for i in range(n):
        arr[i] = _lib.RcPool(FAKE, FAKE + 64, nb, bl)
    return arr


def _err(status, lib):
    return status, lib.rc_last_error().decode()


def test_rope_table_rejects_bad_args(lib):
    buf = np.empty(8, np.float32)
    assert lib.rc_rope_table(4, 4, 10000.0, None, buf.ctypes.data) == -1
    assert lib.rc_rope_table(0, 4, 10000.0, buf.ctypes.data, buf.ctypes.data) == -1
    assert lib.rc_rope_table(2, 3, 10000.0, buf.ctypes.data, buf.ctypes.data) == -1
    assert lib.rc_rope_table(2, 4, -1.0, buf.ctypes.data, buf.ctypes.data) == -1


@no_gpu
def test_assemble_validation(lib):
    ok = dict(pools=_pools(), n=1, segs=FAKE, S=3, kf=FAKE, vf=FAKE + 8, cos=FAKE, sin=FAKE,
              max_pos=64, ka=FAKE + 16, va=FAKE + 24)

    def call(shape=None, **kw):
        a = dict(ok, **kw)
        return lib.rc_kv_assemble(_shape() if shape is None else shape, a["pools"], a["n"], a["segs"],
                                  a["S"], a["kf"], a["vf"], a["cos"], a["sin"], a["max_pos"], a["ka"],
                                  a["va"], None, None)

    assert call(shape=ctypes.cast(0, ctypes.POINTER(_lib.RcShape))) == -1
    assert call(segs=None) == -1
    assert call(kf=None) == -1
    assert call(ka=None) == -1
    assert call(S=0) == -1
    assert call(S=1025) == -2
    assert call(n=0) == -1
    assert call(n=9, pools=_pools(9)) == -2
    assert call(pools=_pools(1, nb=0)) == -1
    assert call(cos=None) == -1                       # one table without the other
    st, msg = _err(call(max_pos=63), lib)             # tables shorter than the prompt
    assert st == -1 and "max_pos" in msg
    assert call(shape=_shape(D=96)) == -2
    assert call(shape=_shape(dtype=7)) == -2
    assert call(shape=_shape(N=0)) == -1
    assert call(ka=FAKE) == -1                        # output aliases an input


@no_gpu
def test_value_reference_validation(lib):
    """The value-reference chain checks what rc_kv_assemble, rc_select_tokens
    and rc_selective_attention check, plus its own limits: the wave-level
    gather's shapes (S <= 64, a key row of 32 bytes times a power of two up to
    64) and bf16 with D = 128 for the attention."""
    ok = dict(pools=_pools(), n=1, segs=FAKE, S=3, kf=FAKE, vf=FAKE + 8, cos=FAKE, sin=FAKE,
              max_pos=64, ka=FAKE + 16, vr=FAKE + 24, sc=None)

    def asm(shape=None, **kw):
        a = dict(ok, **kw)
        return lib.rc_kv_assemble_vref(_shape() if shape is None else shape, a["pools"], a["n"],
                                       a["segs"], a["S"], a["kf"], a["vf"], a["cos"], a["sin"],
                                       a["max_pos"], a["ka"], a["vr"], a["sc"], None)

    assert asm(segs=None) == -1
    assert asm(vr=None) == -1
    assert asm(ka=None, vr=None, sc=FAKE + 32) == -1      # no score-only form
    assert asm(vr=FAKE + 8) == -1                          # table aliases v_fresh
    assert asm(max_pos=63) == -1
    st, msg = _err(asm(S=65), lib)
    assert st == -2 and "S=65" in msg
    assert asm(shape=_shape(Hkv=3)) == -2                  # 24 pairs: not a power of two
    assert asm(shape=_shape(Hkv=16)) == -2                 # 128 pairs
    assert asm(shape=_shape(D=96)) == -2

    def sel(shape=None, k=10, rows=FAKE, vr=FAKE + 24, ka=FAKE + 16, scores_in=FAKE + 32):
        return lib.rc_select_tokens_vref(_shape() if shape is None else shape, FAKE, 3, 8, k, FAKE,
                                         FAKE + 8, ka, vr, scores_in, None, rows, None)

    assert sel(vr=None) == -1
    assert sel(ka=None) == -1
    assert sel(k=57) == -1
    assert sel(rows=None) == -1
    assert sel(shape=_shape(N=16385)) == -2

    def att(shape=None, q=FAKE, vr=FAKE + 8, R=10):
        return lib.rc_selective_attention_vref(_shape() if shape is None else shape, q, FAKE, R,
                                               FAKE + 16, vr, ctypes.c_float(0.088), FAKE + 24,
                                               None)

    assert att(q=None) == -1
    assert att(vr=None) == -1
    assert att(shape=_shape(dtype=0)) == -2                # fp32
    assert att(shape=_shape(D=64)) == -2
    assert att(R=0) == 0


@no_gpu
def test_rerope_validation(lib):
    assert lib.rc_rerope(_shape(), None, FAKE, FAKE, FAKE, 8, None) == -1
    assert lib.rc_rerope(_shape(), FAKE, FAKE, FAKE, FAKE, 0, None) == -1
    assert lib.rc_rerope(_shape(D=32), FAKE, FAKE, FAKE, FAKE, 8, None) == -2


@no_gpu
def test_select_validation(lib):
    def call(shape=None, S=3, n_fresh=8, k=10, scores_in=None, scores_out=FAKE, rows=FAKE, patch=1,
             kf=FAKE, vf=FAKE, ka=FAKE, va=FAKE):
        return lib.rc_select_tokens(_shape() if shape is None else shape, FAKE, S, n_fresh, k, kf, vf, ka, va, scores_in,
                                    scores_out, rows, patch, None)

    assert call(k=-1) == -1
    assert call(k=57) == -1                           # k > N - n_fresh
    assert call(n_fresh=65) == -1
    assert call(rows=None) == -1
    assert call(scores_out=None) == -1                # must score without scores_in
    assert call(patch=1, va=None) == -1
    assert call(shape=_shape(N=16385)) == -2
    assert call(S=0) == -1
    st, msg = _err(call(k=100), lib)
    assert "k=100" in msg


@no_gpu
def test_attention_validation(lib):
    def call(shape=None, rows=FAKE, R=10, scale=0.088, q=FAKE, out=FAKE):
        return lib.rc_selective_attention(_shape() if shape is None else shape, q, rows, R, FAKE, FAKE,
                                          ctypes.c_float(scale), out, None)

    assert call(q=None) == -1
    assert call(R=-1) == -1
    assert call(rows=None, R=10) == -1                # full mode needs R == N
    assert call(scale=0.0) == -1
    assert call(scale=float("nan")) == -1
    assert call(shape=_shape(Hq=6, Hkv=4)) == -1      # Hq % Hkv
    assert call(shape=_shape(Hq=12, Hkv=4)) == -2     # bf16 group of 3 does not divide 128
    assert call(shape=_shape(D=256)) == -2
    assert call(R=0) == 0                             # nothing to do, nothing enqueued


@no_gpu
def test_attention_lse_and_mass_validation(lib):
    def att(shape=None, rows=None, R=64, lse=FAKE):
        return lib.rc_selective_attention_lse(_shape() if shape is None else shape, FAKE, rows, R, FAKE,
                                              FAKE, ctypes.c_float(0.088), FAKE, lse, None)

    assert att(lse=None) == -1
    assert att(R=10) == -1                            # full mode needs R == N
    assert att(shape=_shape(Hq=12, Hkv=4)) == -2
    assert att(R=0, rows=FAKE, lse=None) == 0         # nothing to do

    def mass(shape=None, q=FAKE, lse=FAKE, out=FAKE, scale=0.088):
        return lib.rc_attention_mass(_shape() if shape is None else shape, q, FAKE, lse,
                                     ctypes.c_float(scale), out, None)

    assert mass(q=None) == -1
    assert mass(lse=None) == -1
    assert mass(out=None) == -1
    assert mass(scale=-1.0) == -1
    assert mass(shape=_shape(D=96)) == -2
    assert mass(shape=_shape(Hq=12, Hkv=4)) == -2     # bf16 group of 3 does not divide 128
    assert mass(shape=_shape(Hq=6, Hkv=4)) == -1


@no_gpu
def test_select_eq3_validation(lib):
    def call(shape=None, n_fresh=8, mask=2, lam=0.5, kh=5, ki=5, mass=FAKE, scores_in=None,
             scores_out=FAKE, rows=FAKE, patch=1, vf=FAKE, va=FAKE):
        return lib.rc_select_tokens_eq3(_shape() if shape is None else shape, FAKE, 3, n_fresh, mask,
                                        ctypes.c_float(lam), kh, ki, mass, FAKE, vf, FAKE, va,
                                        scores_in, scores_out, rows, patch, None)

    assert call(kh=-1) == -1
    assert call(kh=30, ki=27) == -1                   # budgets exceed N - n_fresh
    assert call(mass=None) == -1                      # scoring needs the mass
    assert call(vf=None, patch=0) == -1               # scoring needs V
    assert call(lam=1.5) == -1
    assert call(lam=float("nan")) == -1
    assert call(mask=1 << 8) == -1                    # pools beyond 8
    assert call(rows=None) == -1
    assert call(scores_out=None) == -1
    assert call(shape=_shape(N=16385)) == -2
    # lambda = 1 scores every item token 0: an item budget is rejected, a
    # history-only budget is not
    st, msg = _err(call(lam=1.0, kh=5, ki=1), lib)
    assert st == -1 and "lambda = 1" in msg


def test_window_transform_matches_oracle(lib):
    """The library's host-side window transform and the oracle's describe the
    same per-position rows and rotations (their tables may split differently)."""
    from paper_2605_07443_amd import inputs, ops
    for name in ("miss-bf16", "ragged-bf16", "tiny-bf16"):
        cfg = inputs.TEST_WORKLOADS[name]
        w = inputs.make(cfg, 9)
        segs = w.segs.numpy()
        for W in (0, 1, 3, 37, 64, cfg.N - 1, cfg.N):
            got = ops.segments_with_window(segs, cfg.N, W)
            want = O.segments_with_window(segs, cfg.N, W)
            assert got.shape[1] <= segs.shape[1] + 1
            for b in range(cfg.B):
                assert O.position_map(got[b], cfg.N) == O.position_map(want[b], cfg.N), (name, W, b)
    segs = np.array([[[0, 4, -1, 0], [4, 4, 0, 1]]], np.int32)
    with pytest.raises(_lib.RcError):
        ops.segments_with_window(segs, 8, 9)                 # W > N
    with pytest.raises(_lib.RcError):
        ops.segments_with_window(np.array([[[0, 4, -1, 0], [5, 3, 0, 1]]], np.int32), 8, 2)  # gap


@no_gpu
def test_paged_attention_validation(lib):
    def call(shape=None, rows=FAKE, n=1, pools=None, S=3, cos=FAKE, sin=FAKE, max_pos=64):
        return lib.rc_paged_attention(_shape() if shape is None else shape, FAKE, rows, 10,
                                      _pools() if pools is None else pools, n, FAKE, S, FAKE, FAKE,
                                      cos, sin, max_pos, ctypes.c_float(0.088), FAKE, None)

    assert call(rows=None) == -1
    assert call(n=0) == -1
    assert call(S=0) == -1
    assert call(S=65) == -2                           # paged tables live in LDS
    assert call(cos=None) == -1
    assert call(max_pos=10) == -1
    assert call(shape=_shape(dtype=0)) == -2          # bf16 only
    assert call(shape=_shape(N=16385)) == -2
    assert call(pools=_pools(1, nb=0)) == -1


@no_gpu
def test_layer_calls_validation(lib):
    """Host checks of the decoder-layer calls: bad sizes, NULL pointers and
    aliasing fail with a status and a message before anything is enqueued;
    zero rows succeed without a launch."""
    def gemm(M=300, n=64, k=64, x=FAKE, w=FAKE + 8, res=None, y=FAKE + 16):
        return lib.rc_gemm_bf16(M, n, k, x, w, res, y, None)

    assert gemm(x=None) == -1 and gemm(w=None) == -1 and gemm(y=None) == -1
    assert gemm(M=-1) == -1 and gemm(n=0) == -1
    for k in (0, 4, 12, 100):
        st, msg = _err(gemm(k=k), lib)
        assert st == -1 and "k" in msg
    st, msg = _err(gemm(res=FAKE + 16), lib)          # residual aliases the output
    assert st == -1 and "alias" in msg
    far = 1 << 30                                     # x, w and y apart; each overlap alone
    st, msg = _err(gemm(x=FAKE, w=FAKE + far, y=FAKE + 300 * 64 * 2 - 2), lib)    # y's first element in x
    assert st == -1 and "overlap" in msg
    st, msg = _err(gemm(x=FAKE, w=FAKE + far, y=FAKE + 2 * far, res=FAKE + 2 * far + 2), lib)
    assert st == -1 and "overlap" in msg
    st, msg = _err(gemm(x=FAKE, w=FAKE + 2 * far - 2, y=FAKE + 2 * far - 64 * 64 * 2 + 2), lib)
    assert st == -1 and "overlap" in msg
    assert gemm(M=0) == 0

    def norm(M=4, H=64, eps=1e-5, x=FAKE, g=FAKE + 8, y=FAKE + 16):
        return lib.rc_rmsnorm(M, H, x, g, ctypes.c_float(eps), y, None)

    assert norm(x=None) == -1 and norm(g=None) == -1
    assert norm(H=12) == -1 and norm(H=0) == -1 and norm(M=-1) == -1
    assert norm(H=8192 + 8) == -2
    assert norm(eps=-1.0) == -1 and norm(eps=float("inf")) == -1 and norm(eps=float("nan")) == -1
    assert norm(M=0) == 0

    assert lib.rc_silu_mul(4, 12, FAKE, FAKE + 8, None) == -1
    assert lib.rc_silu_mul(-1, 16, FAKE, FAKE + 8, None) == -1
    assert lib.rc_silu_mul(4, 16, None, FAKE + 8, None) == -1
    assert lib.rc_silu_mul(0, 16, FAKE, FAKE + 8, None) == 0

    rows = ctypes.cast(FAKE + 32, ctypes.POINTER(ctypes.c_int32))
    assert lib.rc_gather_rows(2, 8, 4, 24, FAKE, rows, FAKE + 8, None) == -1   # row_bytes % 16
    assert lib.rc_gather_rows(0, 8, 4, 32, FAKE, rows, FAKE + 8, None) == -1
    assert lib.rc_gather_rows(2, 8, 4, 32, None, rows, FAKE + 8, None) == -1
    assert lib.rc_gather_rows(2, 8, 0, 32, FAKE, rows, FAKE + 8, None) == 0
