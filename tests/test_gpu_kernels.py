"""GPU parity: each entry point of libfp8train against the CPU oracle on
seeded inputs, element by element, at sizes that span several tiles and a
ragged tail.  Exact-mode GEMMs, quantization and the update must be
bit-identical; fast-mode GEMMs must lie within the tolerance derived in
`fast_tolerance` (see below)."""
import os

import numpy as np
import pytest
import torch

import oracle
import paper_1812_08011_amd as fp8t
from tests.gpu_util import DEV, dev, gemm, host, q8, q16, say
from tests.helpers import within_fast_bounds

pytestmark = pytest.mark.gpu

U = 2.0 ** -10


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    fp8t.lib()
    yield


def fast_tolerance(absum, K, CL):
    """A loose tolerance in units of sum_k |a_k b_k|: both the fast mode and
    the fast oracle are within nch*u*(1+u)^2*sum|p| of the exact dot product
    (u = 2^-10, nch = ceil(K/CL); recursive summation applied to the chunk
    roundings and the inter-chunk chain), plus the error of the fast mode's
    chunk sums: on the matrix cores each product is truncated to 2^-13 of its
    group's largest exponent and the group sums are combined within
    2^-17 sum|p| (measured; 2^-16 taken), in FP32 on the vector ALUs within
    CL 2^-22 sum|p|."""
    nch = -(-K // CL) if K else 0
    cl = min(CL, K) if K else 0
    chunk_err = cl * 2.0 ** -13 + 2.0 ** -16 + cl * 2.0 ** -22
    return (2 * nch * U * (1 + U) ** 2 + chunk_err * (1 + U)) * absum


def abs_dot(A_vals, B_vals):
    """sum_k |a(i,k) b(k,j)| for every output."""
    return np.abs(A_vals) @ np.abs(B_vals)


def check_fast(Cg, A, B, CL, ta, tb, what, *, rows=None, cols=None, Co=None, absum=None,
               K=None):
    """Fast-mode results against the oracle's bounds: every output must lie
    between the two monotone FP16 chains built from each chunk's sum minus
    and plus its error bound -- for chunks of a multiple of 16 products, the
    FP8 matrix cores' sum (groups of 8 products truncated to 2^-13 of the
    group's largest exponent, the measured arithmetic), otherwise an FP32 sum
    in any order.  Where the bounds coincide the output is forced.  The
    looser tolerance in units of sum|p| (`fast_tolerance`) is checked as
    well, and the fraction bit-identical to the fast oracle (exact chunk
    sums) is reported."""
    Kf = A.shape[0] if ta else A.shape[1]
    matrix_core = Kf > 0 and min(CL, Kf) % 16 == 0
    lo, hi = oracle.chunk_gemm_fast_bounds(A, B, CL, ta, tb, rows, cols,
                                           matrix_core=matrix_core)
    ok = within_fast_bounds(Cg, lo, hi)
    bad = np.flatnonzero(~ok.ravel())
    assert bad.size == 0, (what, bad[:5], Cg.ravel()[bad[:5]], lo.ravel()[bad[:5]],
                           hi.ravel()[bad[:5]])
    single = float(np.mean(lo == hi))
    msg = (f"{what}: inside the fast-mode bounds ({'matrix-core' if matrix_core else 'FP32'} "
           f"chunk sums); single-valued bounds {single:.4f}")
    if Co is not None:
        msg += f", bit-identical to the fast oracle {float(np.mean(Cg == Co)):.4f}"
    say(msg)
    if absum is not None:
        vg, vo = oracle.p16_value(Cg), oracle.p16_value(Co)
        tol = fast_tolerance(absum, K, CL)
        both_nan = np.isnan(vg) & np.isnan(vo)
        same_inf = np.isinf(vg) & (vg == vo)
        fin = ~(both_nan | same_inf)
        assert np.all(np.isfinite(vg[fin])), what
        diff = np.abs(vg[fin] - vo[fin])
        assert not (diff > tol[fin] + 1e-300).any(), what
    return single


# ---- quantization -------------------------------------------------------------

def test_fp8_quantize_f32_bit_patterns():
    rng = np.random.default_rng(500)
    bits = rng.integers(0, 2 ** 32, size=2_000_003, dtype=np.uint64).astype(np.uint32)
    x = np.concatenate([bits.view(np.float32),
                        rng.standard_normal(1_000_000).astype(np.float32),
                        (rng.standard_normal(1_000_000) * 1e-5).astype(np.float32)])
    vals = np.unique(oracle.p8_value(np.arange(0x7C, dtype=np.uint8)))
    mids = ((vals[1:] + vals[:-1]) / 2).astype(np.float32)
    x = np.concatenate([x, mids, -mids, np.nextafter(mids, np.float32(np.inf)),
                        np.nextafter(mids, np.float32(0)),
                        np.float32([0.0, -0.0, np.inf, -np.inf, np.nan, 61440, 61439.996,
                                    57344, 1e30, -1e30])])
    for scale in (1.0, 1000.0, 0.25):
        say(f"fp8_quantize f32 n={x.size} scale={scale}")
        got = host(q8(dev(x), scale))
        ref = oracle.fp8_quantize(x, scale)
        assert np.array_equal(got, ref), np.flatnonzero(got != ref)[:10]


def test_fp8_quantize_every_f32_prefix():
    """Every sign, exponent and top-7-bit mantissa prefix of a float, with the
    low 16 bits at the rounding-relevant patterns (ties have them all zero)
    and at random values: the conversion is correct in every binade."""
    rng = np.random.default_rng(503)
    hi = np.arange(65536, dtype=np.uint32) << 16
    lows = np.concatenate([np.uint32([0, 1, 0x7FFF, 0x8000, 0x8001, 0xFFFF]),
                           rng.integers(0, 65536, size=6, dtype=np.uint32)])
    x = (hi[:, None] | lows[None, :]).ravel().view(np.float32)
    for scale in (1.0, 3.0):
        say(f"fp8_quantize f32 every prefix n={x.size} scale={scale}")
        got = host(q8(dev(x), scale))
        ref = oracle.fp8_quantize(x, scale)
        assert np.array_equal(got, ref), np.flatnonzero(got != ref)[:10]


def test_fp8_quantize_all_fp16_codes_and_odd_offsets():
    codes = np.arange(65536, dtype=np.uint16)
    for scale in (1.0, 1000.0, 2.0 ** -3):
        say(f"fp8_quantize fp16 all codes scale={scale}")
        got = host(q8(dev(codes), scale))
        assert np.array_equal(got, oracle.fp8_quantize(codes, scale))
    # misaligned pointers and ragged lengths take the scalar path
    rng = np.random.default_rng(501)
    x = rng.standard_normal(10_007).astype(np.float32)
    xd = dev(x)
    out = torch.empty(10_007, dtype=torch.uint8, device=DEV)
    for off in (1, 2, 3):
        say(f"fp8_quantize misaligned offset {off}")
        n = x.size - off
        fp8t.lib().fp8_quantize(xd.data_ptr() + 4 * off, 0, 1.0, out.data_ptr() + off, n,
                                torch.cuda.current_stream().cuda_stream)
        got = host(out)[off:off + n]
        assert np.array_equal(got, oracle.fp8_quantize(x[off:]))


def test_fp16_quantize_bit_patterns():
    rng = np.random.default_rng(502)
    bits = rng.integers(0, 2 ** 32, size=2_000_001, dtype=np.uint64).astype(np.uint32)
    vals = oracle.p16_value(np.arange(0x7E00, dtype=np.uint16))
    mids = ((vals[1:] + vals[:-1]) / 2).astype(np.float32)
    x = np.concatenate([bits.view(np.float32), mids, -mids,
                        rng.standard_normal(100_000).astype(np.float32) * np.float32(1e-10),
                        np.float32([0.0, -0.0, np.inf, -np.inf, np.nan, 4290772992.0,
                                    4292870144.0, 1e38])])
    say(f"fp16_quantize n={x.size}")
    got = host(q16(dev(x)))
    ref = oracle.fp16_quantize(x)
    assert np.array_equal(got, ref), np.flatnonzero(got != ref)[:10]


# ---- chunk_gemm -----------------------------------------------------------------

SHAPES = [
    # M, N, K, CL
    (1, 1, 1, 1),
    (3, 5, 7, 2),
    (37, 29, 100, 16),
    (130, 67, 333, 64),       # ragged in all three dimensions, last chunk 13
    (64, 128, 256, 64),
    (257, 131, 129, 1),       # CL = 1: sequential sum
    (100, 90, 500, 500),      # CL = K: one chunk
    (45, 61, 300, 1000),      # CL > K
    (33, 47, 400, 48),        # fast mode: multiple of 16 but not of 64
    (19, 23, 1030, 256),
]


def _operands(rng, M, N, K, ta, tb, scale=1.0):
    a = (rng.standard_normal((M, K)) * scale).astype(np.float32)
    b = rng.standard_normal((K, N)).astype(np.float32)
    # sprinkle exact zeros, large values and ties
    a[rng.random(a.shape) < 0.05] = 0.0
    b[rng.random(b.shape) < 0.02] *= 64.0
    A = oracle.fp8_quantize(np.ascontiguousarray(a.T if ta else a))
    B = oracle.fp8_quantize(np.ascontiguousarray(b.T if tb else b))
    return A, B


# 0-8: register tiles of the main exact kernel; 9: the chain kernel (whole
# 32 x 32 tiles, 4-k groups; CL = 2 falls back to the others)
VALU_TILES = ["auto", "0", "1", "2", "3", "4", "5", "6", "7", "8", "9"]


@pytest.mark.parametrize("guard", ["1", "0"])
@pytest.mark.parametrize("tile", VALU_TILES)
@pytest.mark.parametrize("ta,tb", [(0, 0), (0, 1), (1, 0), (1, 1)])
def test_chunk_gemm_exact_matches_oracle(tile, ta, tb, guard, monkeypatch):
    """Both paths of the exact kernel (guarded: plain values with Veltkamp
    rounding; safe: scaled by 2^96 with integer rounding) on every tile."""
    if tile != "auto":
        monkeypatch.setenv("FP8T_VALU_TILE", tile)
    monkeypatch.setenv("FP8T_GEMM_GUARD", guard)
    rng = np.random.default_rng(510 + 2 * ta + tb)
    for (M, N, K, CL) in SHAPES:
        A, B = _operands(rng, M, N, K, ta, tb)
        say(f"chunk_gemm exact tile={tile} guard={guard} ta={ta} tb={tb} M={M} N={N} K={K} "
            f"CL={CL}")
        Cg = host(gemm(dev(A), dev(B), M, N, K, CL, ta, tb))
        Co = oracle.chunk_gemm(A, B, CL, ta, tb)
        assert np.array_equal(Cg, Co), (M, N, K, CL, np.argwhere(Cg != Co)[:5])


# Shapes whose tiles get shared out over few workgroups: tiles split at chunk
# boundaries, pieces of one chunk, ragged last chunks, shared and whole tiles
# in one launch.
SPLIT_SHAPES = [
    # M, N, K, CL
    (130, 67, 333, 64),
    (200, 150, 1000, 16),
    (64, 64, 4096, 64),
    (33, 47, 700, 48),
    (17, 300, 64, 8),
]


@pytest.mark.parametrize("tile", ["1", "2", "4", "5", "6", "7", "8"])
@pytest.mark.parametrize("wgs", ["1", "3", "7", "50"])
@pytest.mark.parametrize("ta,tb", [(0, 0), (1, 0), (0, 1)])
def test_chunk_gemm_exact_shared_tiles(tile, wgs, ta, tb, monkeypatch):
    """Every plan (whole tiles, shared tiles continued by the fold pass) gives
    the oracle's bits: the chunk sums and their order do not depend on it."""
    monkeypatch.setenv("FP8T_VALU_TILE", tile)
    monkeypatch.setenv("FP8T_GEMM_WGS", wgs)
    monkeypatch.setenv("FP8T_GEMM_SPLIT", "1")
    rng = np.random.default_rng(550 + 2 * ta + tb)
    for (M, N, K, CL) in SPLIT_SHAPES:
        A, B = _operands(rng, M, N, K, ta, tb)
        ws = fp8t.chunk_gemm_workspace_size(ta, tb, M, N, K, CL, fp8t.EXACT)
        say(f"chunk_gemm exact shared tile={tile} wgs={wgs} ta={ta} tb={tb} M={M} N={N} "
            f"K={K} CL={CL} ws={ws}")
        Cg = host(gemm(dev(A), dev(B), M, N, K, CL, ta, tb))
        Co = oracle.chunk_gemm(A, B, CL, ta, tb)
        assert np.array_equal(Cg, Co), (M, N, K, CL, np.argwhere(Cg != Co)[:5])


@pytest.mark.parametrize("guard", ["1", "0"])
@pytest.mark.parametrize("wgs", ["3", "7"])
def test_chunk_gemm_fold_decodes_every_kind_of_chunk_sum(wgs, guard, monkeypatch):
    """Shared tiles only, so the fold pass continues every output over chunk
    sums of each kind: zeros (rows of -0 / +0 codes), FP16 subnormals of both
    signs (one 2^-16 x 2^-16 product per chunk: 2^-32), normal values, an Inf
    chunk and a NaN chunk part-way along K.  The fold decodes each chunk
    sum's FP16 code and must give the oracle's bits."""
    monkeypatch.setenv("FP8T_GEMM_SPLIT", "1")
    monkeypatch.setenv("FP8T_GEMM_WGS", wgs)
    monkeypatch.setenv("FP8T_GEMM_GUARD", guard)
    rng = np.random.default_rng(591)
    M, N, CL, nch = 10, 64, 64, 40
    K = CL * nch
    A = np.zeros((M, K), np.uint8)
    A[0, :] = 0x80                                   # -0
    A[1, :] = 0x00                                   # +0
    A[2, ::CL] = 0x01                                # 2^-16, one per chunk
    A[3, ::CL] = 0x81                                # -2^-16
    A[4, ::CL] = np.where(rng.random(nch) < 0.5, 0x01, 0x81)
    A[4, 5::CL] = np.where(rng.random(nch) < 0.5, 0x02, 0x82)
    A[5, :] = rng.integers(0x30, 0x48, K) | (rng.integers(0, 2, K) << 7)
    A[6, :] = A[5, :]
    A[6, CL * 20 + 3] = 0x7C                         # +Inf in chunk 20
    A[7, :] = A[5, :]
    A[7, CL * 11 + 9] = 0x7D                         # NaN in chunk 11
    A[8, :] = 0x80
    A[8, CL * 30] = 0x01                             # -0 until chunk 30
    A[9, ::CL] = 0x81
    A[9, CL * 35:] = 0x00                            # negative subnormal sums, then +0
    B = np.empty((K, N), np.uint8)
    B[:, :32] = 0x01                                 # 2^-16: subnormal products
    B[:, 32:] = rng.integers(0x30, 0x48, (K, 32)) | (rng.integers(0, 2, (K, 32)) << 7)
    B[:, 40] = 0x3C                                  # 1.0
    ws = fp8t.chunk_gemm_workspace_size(0, 0, M, N, K, CL, fp8t.EXACT)
    assert ws > 0
    say(f"fold decodes every kind of chunk sum wgs={wgs} guard={guard}")
    Cg = host(gemm(dev(A), dev(B), M, N, K, CL))
    Co = oracle.chunk_gemm(A, B, CL)
    assert np.array_equal(Cg, Co), np.argwhere(Cg != Co)[:5]
    assert np.all(Cg[:2] == 0)
    assert np.all((Cg[6] & 0x7FFF) == 0x7E00) and np.all(Cg[7] == 0x7F00)


def test_chunk_gemm_workspace_contract():
    """No workspace: a plan that needs none, same bits.  Too small a
    workspace is rejected before anything is enqueued."""
    rng = np.random.default_rng(560)
    M, N, K, CL = 96, 200, 2048, 64
    A, B = _operands(rng, M, N, K, 0, 0)
    Ad, Bd = dev(A), dev(B)
    Co = oracle.chunk_gemm(A, B, CL)
    ws = fp8t.chunk_gemm_workspace_size(0, 0, M, N, K, CL, fp8t.EXACT)
    say(f"workspace contract ws={ws}")
    C = torch.empty((M, N), dtype=torch.uint16, device=DEV)
    fp8t.chunk_gemm(0, 0, M, N, K, CL, Ad, K, Bd, N, C, N, fp8t.EXACT)
    assert np.array_equal(host(C), Co)
    if ws > 0:
        small = torch.empty(ws - 1, dtype=torch.uint8, device=DEV)
        with pytest.raises(fp8t.Fp8tError) as e:
            fp8t.chunk_gemm(0, 0, M, N, K, CL, Ad, K, Bd, N, C, N, fp8t.EXACT, small, ws - 1)
        assert e.value.status == fp8t.EWORKSPACE
        big = torch.full((ws,), 0xA5, dtype=torch.uint8, device=DEV)
        C.fill_(0)
        fp8t.chunk_gemm(0, 0, M, N, K, CL, Ad, K, Bd, N, C, N, fp8t.EXACT, big, ws)
        assert np.array_equal(host(C), Co)


@pytest.mark.parametrize("mtile", ["auto", "0", "1", "2", "3", "4", "5"])
@pytest.mark.parametrize("ta,tb", [(0, 0), (0, 1), (1, 0), (1, 1)])
def test_chunk_gemm_fast_within_tolerance(ta, tb, mtile, monkeypatch):
    """Fast mode against the fast oracle within the derived tolerance, for
    every matrix-core tile; the guarded and safe epilogues give the same
    bits."""
    if mtile != "auto":
        monkeypatch.setenv("FP8T_MFMA_TILE", mtile)
    rng = np.random.default_rng(520 + 2 * ta + tb)
    for (M, N, K, CL) in SHAPES:
        A, B = _operands(rng, M, N, K, ta, tb)
        say(f"chunk_gemm fast mtile={mtile} ta={ta} tb={tb} M={M} N={N} K={K} CL={CL}")
        Ad, Bd = dev(A), dev(B)
        monkeypatch.setenv("FP8T_GEMM_GUARD", "1")
        Cg = host(gemm(Ad, Bd, M, N, K, CL, ta, tb, mode=fp8t.FAST))
        monkeypatch.setenv("FP8T_GEMM_GUARD", "0")
        Cs = host(gemm(Ad, Bd, M, N, K, CL, ta, tb, mode=fp8t.FAST))
        assert np.array_equal(Cg, Cs), (M, N, K, CL, np.argwhere(Cg != Cs)[:5])
        Co = oracle.chunk_gemm(A, B, CL, ta, tb, mode=oracle.FAST)
        va = oracle.p8_value(A.T if ta else A)
        vb = oracle.p8_value(B.T if tb else B)
        check_fast(Cg, A, B, CL, ta, tb, f"fast {M}x{N}x{K} CL={CL}", Co=Co,
                   absum=abs_dot(va, vb), K=K)
        if CL == 1:
            assert np.array_equal(Cg, oracle.chunk_gemm(A, B, CL, ta, tb))


@pytest.mark.parametrize("ta,tb", [(0, 0), (0, 1), (1, 0), (1, 1)])
def test_chunk_gemm_fast_vector_alu_tiles_same_bits(ta, tb, monkeypatch):
    """The fast mode for chunk lengths the matrix cores cannot split (CL not
    a multiple of 16): every vector-ALU kernel that has it -- the register
    tiles 4, 5, 6 of the main kernel and the chain kernel's 2 x 2, 1 x 2 and
    1 x 1 (9, 10, 11) -- sums a chunk's products in FP32 in ascending k and
    rounds once, so all give the same bits: ragged M, N and K (a last 4-k
    group with zero-filled products), CL 4 to 36, Inf/NaN operands; within
    the fast oracle's bounds."""
    rng = np.random.default_rng(700 + 2 * ta + tb)
    shapes = [(130, 67, 333, 8), (64, 96, 1000, 12), (33, 47, 700, 4), (70, 150, 602, 20),
              (5, 3, 17, 4), (128, 64, 2048, 36)]
    for si, (M, N, K, CL) in enumerate(shapes):
        A, B = _operands(rng, M, N, K, ta, tb)
        if si == 1:
            (A.T if ta else A)[5, 900] = 0x7C          # +Inf
            (A.T if ta else A)[60, 500] = 0x7F         # NaN
        Ad, Bd = dev(A), dev(B)
        got = {}
        for tile in ("6", "4", "5", "9", "10", "11"):
            monkeypatch.setenv("FP8T_VALU_TILE", tile)
            say(f"fast vector-ALU tile={tile} ta={ta} tb={tb} {M}x{N}x{K} CL={CL}")
            got[tile] = host(gemm(Ad, Bd, M, N, K, CL, ta, tb, mode=fp8t.FAST))
        monkeypatch.delenv("FP8T_VALU_TILE")
        for tile, C in got.items():
            assert np.array_equal(C, got["6"]), (tile, M, N, K, CL,
                                                 np.argwhere(C != got["6"])[:5])
        Co = oracle.chunk_gemm(A, B, CL, ta, tb, mode=oracle.FAST)
        check_fast(got["6"], A, B, CL, ta, tb, f"fast valu {M}x{N}x{K} CL={CL}", Co=Co)


@pytest.mark.parametrize("mtile", ["0", "1", "2"])
@pytest.mark.parametrize("wgs", ["2", "9"])
@pytest.mark.parametrize("ta,tb", [(0, 0), (1, 0), (0, 1)])
def test_chunk_gemm_fast_shared_tiles(mtile, wgs, ta, tb, monkeypatch):
    """Fast mode with tiles shared out over few workgroups (chunk sums through
    the workspace and the fold pass) gives the bits of the whole-tile plan."""
    monkeypatch.setenv("FP8T_MFMA_TILE", mtile)
    rng = np.random.default_rng(580 + 2 * ta + tb)
    for (M, N, K, CL) in [(130, 67, 1000, 64), (64, 96, 4096, 32), (33, 47, 700, 32)]:
        A, B = _operands(rng, M, N, K, ta, tb)
        Ad, Bd = dev(A), dev(B)
        monkeypatch.setenv("FP8T_GEMM_SPLIT", "0")
        monkeypatch.delenv("FP8T_GEMM_WGS", raising=False)
        say(f"fast shared mtile={mtile} wgs={wgs} ta={ta} tb={tb} {M}x{N}x{K} CL={CL}")
        Cw = host(gemm(Ad, Bd, M, N, K, CL, ta, tb, mode=fp8t.FAST))
        monkeypatch.setenv("FP8T_GEMM_SPLIT", "1")
        monkeypatch.setenv("FP8T_GEMM_WGS", wgs)
        Cs = host(gemm(Ad, Bd, M, N, K, CL, ta, tb, mode=fp8t.FAST))
        assert np.array_equal(Cw, Cs), (M, N, K, CL, np.argwhere(Cw != Cs)[:5])


@pytest.mark.parametrize("mtile,split", [("0", "0"), ("1", "0"), ("2", "0"), ("3", "0"),
                                         ("4", "0"), ("5", "0"), ("0", "1"), ("1", "1")])
def test_chunk_gemm_fast_specials(mtile, split, monkeypatch):
    """Inf and NaN operands through every matrix-core kernel, in whole tiles
    and in the later pieces of shared tiles (chunk sums through the
    workspace): the guarded epilogue's rounding turns an Inf chunk sum into
    NaN, so its guard must catch it and the safe epilogue give Inf -- the
    same bits as an all-safe run, inside the oracle's bounds."""
    monkeypatch.setenv("FP8T_MFMA_TILE", mtile)
    rng = np.random.default_rng(585)
    M, N, K, CL = 130, 67, 1000, 64
    A, B = _operands(rng, M, N, K, 0, 0)
    A[5, 900] = 0x7C            # +Inf in chunk 14
    A[60, 500] = 0x7F           # NaN in chunk 7
    B[950, 3] = 0xFC            # -Inf in chunk 14
    A[77, 640] = 0x7C           # +Inf meeting zero and finite partners
    Ad, Bd = dev(A), dev(B)
    got = {}
    for guard in ("1", "0"):
        monkeypatch.setenv("FP8T_GEMM_GUARD", guard)
        monkeypatch.setenv("FP8T_GEMM_SPLIT", split)
        monkeypatch.setenv("FP8T_GEMM_WGS", "7" if split == "1" else "0")
        say(f"fast specials mtile={mtile} split={split} guard={guard}")
        got[guard] = host(gemm(Ad, Bd, M, N, K, CL, mode=fp8t.FAST))
    assert np.array_equal(got["1"], got["0"]), np.argwhere(got["1"] != got["0"])[:5]
    Co = oracle.chunk_gemm(A, B, CL, mode=oracle.FAST)
    assert np.any((Co & 0x7FFF) == 0x7E00) and np.any(Co == 0x7F00)
    check_fast(got["1"], A, B, CL, 0, 0, f"fast specials mtile={mtile} split={split}", Co=Co)


@pytest.mark.parametrize("ta,tb", [(0, 0), (0, 1), (1, 0), (1, 1)])
def test_chunk_gemm_fast_chunks_over_waves_same_bits(ta, tb, monkeypatch):
    """The kernel that spreads a step's four chunks over the waves of a
    64 x 64 tile (CL = 64) feeds the matrix cores the same bytes per chunk as
    the streamed 64 x 64 kernel and adds the chunk sums in the same order, so
    the two give the same bits: ragged M, N and K (steps with 1-3 chunks and
    a short last chunk), padded leading dimensions and misaligned bases
    (4-byte and byte-wise loads), both epilogues; and the fast oracle's
    tolerance holds."""
    rng = np.random.default_rng(590 + 2 * ta + tb)
    # the last three are whole 64 x 64 tiles with K a multiple of 256 and
    # 16-byte rows (the kernel's single-load-path variant); the last one has
    # tiles that fail the overflow guard
    cases = [(32, 32, 64, 0, 0), (33, 31, 65, 0, 0), (100, 70, 64 * 9 + 17, 0, 0),
             (64, 96, 64 * 14, 0, 0), (70, 45, 64 * 23 + 40, 5, 1), (40, 72, 64 * 6, 3, 3),
             (128, 64, 1024, 0, 0), (64, 128, 768, 0, 0), (128, 192, 512, 0, 0)]
    for ci, (M, N, K, pad, off) in enumerate(cases):
        A, B = _operands(rng, M, N, K, ta, tb)
        if ci == len(cases) - 1:
            (A.T if ta else A)[37, :] = 0x7B                     # 57344
            (B if tb else B.T)[70, :] = np.where(rng.random(K) < 0.5, 0x7A, 0xFA)
        # rows of lda (ldb) bytes starting off bytes into the allocation
        lda, ldb = A.shape[1] + pad, B.shape[1] + pad
        Ap = np.zeros((A.shape[0], lda), np.uint8)
        Bp = np.zeros((B.shape[0], ldb), np.uint8)
        Ap[:, :A.shape[1]] = A
        Bp[:, :B.shape[1]] = B
        Ad = dev(np.concatenate([np.zeros(off, np.uint8), Ap.ravel()]))[off:]
        Bd = dev(np.concatenate([np.zeros(off, np.uint8), Bp.ravel()]))[off:]
        got = {}
        for mtile, wgs in (("2", "0"), ("3", "0"), ("3", "3")):
            monkeypatch.setenv("FP8T_MFMA_TILE", mtile)
            monkeypatch.setenv("FP8T_GEMM_WGS", wgs)     # 3: several tiles per workgroup
            for guard in ("1", "0"):
                monkeypatch.setenv("FP8T_GEMM_GUARD", guard)
                say(f"fast chunks over waves mtile={mtile} wgs={wgs} guard={guard} ta={ta} "
                    f"tb={tb} {M}x{N}x{K} pad={pad} off={off}")
                got[mtile + wgs, guard] = host(gemm(Ad, Bd, M, N, K, 64, ta, tb,
                                                    mode=fp8t.FAST, lda=lda, ldb=ldb))
        monkeypatch.delenv("FP8T_GEMM_WGS")
        ref = got["20", "1"]
        for key, C in got.items():
            assert np.array_equal(C, ref), (key, M, N, K, np.argwhere(C != ref)[:5])
        # the FP8 result in the same pass (with and without the FP16 one)
        monkeypatch.setenv("FP8T_GEMM_GUARD", "1")
        q8s = {}
        for mtile in ("2", "3"):
            monkeypatch.setenv("FP8T_MFMA_TILE", mtile)
            for with_c in (True, False):
                C8 = torch.full((M, N + 3), 0xEE, dtype=torch.uint8, device=DEV)
                C = torch.empty((M, N), dtype=torch.uint16, device=DEV) if with_c else None
                ws_b = fp8t.chunk_gemm_fp8_workspace_size(ta, tb, M, N, K, 64, fp8t.FAST)
                ws = torch.empty(max(ws_b, 1), dtype=torch.uint8, device=DEV)
                fp8t.chunk_gemm_fp8(ta, tb, M, N, K, 64, Ad, lda, Bd, ldb, C, N, C8, N + 3,
                                    0.5, fp8t.FAST, ws, ws_b)
                q8s[mtile, with_c] = host(C8)
                if with_c:
                    assert np.array_equal(host(C), ref)
        for key, Q in q8s.items():
            assert np.array_equal(Q, q8s["2", True]), key
        assert np.all(q8s["3", True][:, N:] == 0xEE)
        assert np.array_equal(q8s["3", True][:, :N], oracle.fp8_quantize(ref, 0.5))
        Co = oracle.chunk_gemm(A, B, 64, ta, tb, mode=oracle.FAST)
        va = oracle.p8_value(A.T if ta else A)
        vb = oracle.p8_value(B.T if tb else B)
        check_fast(got["30", "1"], A, B, 64, ta, tb, f"fast kx {M}x{N}x{K}", Co=Co,
                   absum=abs_dot(va, vb), K=K)


@pytest.mark.parametrize("ta,tb", [(0, 0), (0, 1), (1, 0), (1, 1)])
def test_chunk_gemm_fast_block_per_wave_same_bits(ta, tb, monkeypatch):
    """The 64 x 64-tile kernel whose 16 waves each own a 16 x 16 block over
    the whole K (CL = 64) forms every chunk sum with the instruction sequence
    of the 16 x 16 block kernel (two 16x16x32 steps from zero) and adds them
    in the same order, so the two give the same bits: ragged M, N and K,
    padded leading dimensions and misaligned bases, several tiles per
    workgroup, both epilogues, tiles failing the overflow guard, the FP8
    result in the same pass; and the fast oracle's bounds hold."""
    rng = np.random.default_rng(600 + 2 * ta + tb)
    cases = [(32, 32, 64, 0, 0), (33, 31, 65, 0, 0), (100, 70, 64 * 9 + 17, 0, 0),
             (64, 96, 64 * 14, 0, 0), (70, 45, 64 * 23 + 40, 5, 1), (40, 72, 64 * 6, 3, 3),
             (128, 64, 1024, 0, 0), (64, 128, 768, 0, 0), (128, 192, 512, 0, 0)]
    for ci, (M, N, K, pad, off) in enumerate(cases):
        A, B = _operands(rng, M, N, K, ta, tb)
        if ci == len(cases) - 1:
            (A.T if ta else A)[37, :] = 0x7B                     # 57344
            (B if tb else B.T)[70, :] = np.where(rng.random(K) < 0.5, 0x7A, 0xFA)
        if ci == 4:
            (A.T if ta else A)[3, 70] = 0x7C                     # +Inf
            (B if tb else B.T)[9, 1000] = 0x7D                   # NaN
        lda, ldb = A.shape[1] + pad, B.shape[1] + pad
        Ap = np.zeros((A.shape[0], lda), np.uint8)
        Bp = np.zeros((B.shape[0], ldb), np.uint8)
        Ap[:, :A.shape[1]] = A
        Bp[:, :B.shape[1]] = B
        Ad = dev(np.concatenate([np.zeros(off, np.uint8), Ap.ravel()]))[off:]
        Bd = dev(np.concatenate([np.zeros(off, np.uint8), Bp.ravel()]))[off:]
        got = {}
        for mtile, wgs in (("1", "0"), ("4", "0"), ("4", "3")):
            monkeypatch.setenv("FP8T_MFMA_TILE", mtile)
            monkeypatch.setenv("FP8T_GEMM_WGS", wgs)     # 3: several tiles per workgroup
            for guard in ("1", "0"):
                monkeypatch.setenv("FP8T_GEMM_GUARD", guard)
                say(f"fast block per wave mtile={mtile} wgs={wgs} guard={guard} ta={ta} "
                    f"tb={tb} {M}x{N}x{K} pad={pad} off={off}")
                got[mtile + wgs, guard] = host(gemm(Ad, Bd, M, N, K, 64, ta, tb,
                                                    mode=fp8t.FAST, lda=lda, ldb=ldb))
        monkeypatch.delenv("FP8T_GEMM_WGS")
        ref = got["10", "1"]
        for key, C in got.items():
            assert np.array_equal(C, ref), (key, M, N, K, np.argwhere(C != ref)[:5])
        monkeypatch.setenv("FP8T_GEMM_GUARD", "1")
        monkeypatch.setenv("FP8T_MFMA_TILE", "4")
        for with_c in (True, False):
            C8 = torch.full((M, N + 3), 0xEE, dtype=torch.uint8, device=DEV)
            C = torch.empty((M, N), dtype=torch.uint16, device=DEV) if with_c else None
            ws_b = fp8t.chunk_gemm_fp8_workspace_size(ta, tb, M, N, K, 64, fp8t.FAST)
            ws = torch.empty(max(ws_b, 1), dtype=torch.uint8, device=DEV)
            fp8t.chunk_gemm_fp8(ta, tb, M, N, K, 64, Ad, lda, Bd, ldb, C, N, C8, N + 3,
                                0.5, fp8t.FAST, ws, ws_b)
            q8 = host(C8)
            assert np.all(q8[:, N:] == 0xEE)
            assert np.array_equal(q8[:, :N], oracle.fp8_quantize(ref, 0.5))
            if with_c:
                assert np.array_equal(host(C), ref)
        if ci != 4:
            Co = oracle.chunk_gemm(A, B, 64, ta, tb, mode=oracle.FAST)
            va = oracle.p8_value(A.T if ta else A)
            vb = oracle.p8_value(B.T if tb else B)
            check_fast(got["40", "1"], A, B, 64, ta, tb, f"fast kx16 {M}x{N}x{K}", Co=Co,
                       absum=abs_dot(va, vb), K=K)



@pytest.mark.parametrize("tb", [0, 1])
def test_chunk_gemm_fast_wave_kernel_same_bits(tb, monkeypatch, capfd):
    """The wave-independent 32 x 128-tile kernel (each wave streams its own
    32 x 32 block; loads of whole 128-byte row pieces re-laid out through
    wave-private LDS; B stored with n contiguous copied k-contiguous first)
    issues the streamed kernel's matrix-core instructions with the same lane
    layout and the same epilogue, so the two give the same bits: ragged M, N
    and K (K not a multiple of 16 or 64), padded leading dimensions, CL 64 and
    128, one and several tiles per workgroup, both epilogues, Inf/NaN
    operands and tiles failing the overflow guard, the FP8 result in the same
    pass; within the fast oracle's bounds.  Operands that rule out its
    16-byte loads fall back to another plan with the same bits."""
    rng = np.random.default_rng(640 + tb)
    cases = [(32, 128, 128, 64, 0), (33, 31, 65, 64, 0), (100, 70, 64 * 9 + 17, 64, 0),
             (64, 200, 64 * 14, 128, 0), (70, 45, 64 * 23 + 40, 64, 16),
             (40, 72, 64 * 6 + 5, 128, 32), (128, 256, 1024, 64, 0), (96, 384, 512, 64, 0)]
    for ci, (M, N, K, CL, pad) in enumerate(cases):
        A, B = _operands(rng, M, N, K, 0, tb)
        if ci == len(cases) - 1:
            A[37, :] = 0x7B                                     # 57344
            (B if tb else B.T)[70, :] = np.where(rng.random(K) < 0.5, 0x7A, 0xFA)
        if ci == 4:
            A[3, 70] = 0x7C                                     # +Inf
            (B if tb else B.T)[9, 1000] = 0x7D                  # NaN
        # leading dimensions that keep 16-byte loads (the kernel's condition)
        lda = -(-A.shape[1] // 16) * 16 + pad
        ldb = (-(-B.shape[1] // 16) * 16 if tb else B.shape[1]) + pad
        Ap = np.zeros((A.shape[0], lda), np.uint8)
        Bp = np.zeros((B.shape[0], ldb), np.uint8)
        Ap[:, :A.shape[1]] = A
        Bp[:, :B.shape[1]] = B
        Ad, Bd = dev(Ap), dev(Bp)
        got = {}
        for mtile, wgs in (("2", "0"), ("5", "0"), ("5", "3")):
            monkeypatch.setenv("FP8T_MFMA_TILE", mtile)
            monkeypatch.setenv("FP8T_GEMM_WGS", wgs)     # 3: several tiles per workgroup
            for guard in ("1", "0"):
                monkeypatch.setenv("FP8T_GEMM_GUARD", guard)
                monkeypatch.setenv("FP8T_GEMM_VERBOSE", "1")
                say(f"fast wave kernel mtile={mtile} wgs={wgs} guard={guard} tb={tb} "
                    f"{M}x{N}x{K} CL={CL} pad={pad}")
                capfd.readouterr()
                got[mtile + wgs, guard] = host(gemm(Ad, Bd, M, N, K, CL, 0, tb,
                                                    mode=fp8t.FAST, lda=lda, ldb=ldb))
                monkeypatch.delenv("FP8T_GEMM_VERBOSE")
                # the forced configuration is the one that ran
                assert f"chose kind 2 cfg {mtile} " in capfd.readouterr().err
        monkeypatch.delenv("FP8T_GEMM_WGS")
        ref = got["20", "1"]
        for key, C in got.items():
            assert np.array_equal(C, ref), (key, M, N, K, np.argwhere(C != ref)[:5])
        monkeypatch.setenv("FP8T_GEMM_GUARD", "1")
        monkeypatch.setenv("FP8T_MFMA_TILE", "5")
        for with_c in (True, False):
            C8 = torch.full((M, N + 3), 0xEE, dtype=torch.uint8, device=DEV)
            C = torch.empty((M, N), dtype=torch.uint16, device=DEV) if with_c else None
            ws_b = fp8t.chunk_gemm_fp8_workspace_size(0, tb, M, N, K, CL, fp8t.FAST)
            ws = torch.empty(max(ws_b, 1), dtype=torch.uint8, device=DEV)
            fp8t.chunk_gemm_fp8(0, tb, M, N, K, CL, Ad, lda, Bd, ldb, C, N, C8, N + 3,
                                0.5, fp8t.FAST, ws, ws_b)
            q8 = host(C8)
            assert np.all(q8[:, N:] == 0xEE)
            assert np.array_equal(q8[:, :N], oracle.fp8_quantize(ref, 0.5))
            if with_c:
                assert np.array_equal(host(C), ref)
        # a misaligned A base rules the kernel out: another plan, same bits
        Am = torch.zeros(Ap.size + 1, dtype=torch.uint8, device=DEV)
        Am[1:] = Ad.reshape(-1)
        C = torch.empty((M, N), dtype=torch.uint16, device=DEV)
        ws_b = fp8t.chunk_gemm_workspace_size(0, tb, M, N, K, CL, fp8t.FAST)
        ws = torch.empty(max(ws_b, 1), dtype=torch.uint8, device=DEV)
        say(f"fast wave kernel misaligned A tb={tb} {M}x{N}x{K}")
        fp8t.chunk_gemm(0, tb, M, N, K, CL, Am.data_ptr() + 1, lda, Bd, ldb, C, N, fp8t.FAST,
                        ws, ws_b)
        assert np.array_equal(host(C), ref)
        if ci != 4:
            Co = oracle.chunk_gemm(A, B, CL, 0, tb, mode=oracle.FAST)
            va = oracle.p8_value(A)
            vb = oracle.p8_value(B.T if tb else B)
            check_fast(got["50", "1"], A, B, CL, 0, tb, f"fast wave {M}x{N}x{K}", Co=Co,
                       absum=abs_dot(va, vb), K=K)

def test_chunk_gemm_padded_leading_dims_and_misaligned_bases():
    rng = np.random.default_rng(530)
    M, N, K, CL = 150, 70, 260, 64
    for ta, tb in ((0, 0), (1, 1), (0, 1), (1, 0)):
        for off in (0, 1, 3):
            A, B = _operands(rng, M, N, K, ta, tb)
            lda, ldb, ldc = A.shape[1] + 5, B.shape[1] + 3, N + 7
            Ap = np.zeros((A.shape[0], lda + off), np.uint8)
            Bp = np.zeros((B.shape[0], ldb + off), np.uint8)
            Ap[:, off:off + A.shape[1]] = A
            Bp[:, off:off + B.shape[1]] = B
            Ad, Bd = dev(Ap.ravel()), dev(Bp.ravel())
            for mode in (fp8t.EXACT, fp8t.FAST):
                say(f"chunk_gemm padded ta={ta} tb={tb} off={off} mode={mode}")
                C = dev(np.full((M, ldc), 0xABCD, np.uint16))
                ldap, ldbp = lda + off, ldb + off
                fp8t.chunk_gemm(ta, tb, M, N, K, CL, Ad.data_ptr() + off, ldap,
                                Bd.data_ptr() + off, ldbp, C, ldc, mode)
                Ch = host(C)
                assert np.all(Ch[:, N:] == 0xABCD)          # padding untouched
                Co = oracle.chunk_gemm(A, B, CL, ta, tb, mode=mode)
                if mode == fp8t.EXACT:
                    assert np.array_equal(Ch[:, :N], Co)
                else:
                    check_fast(Ch[:, :N], A, B, CL, ta, tb, "padded fast", Co=Co,
                               absum=abs_dot(oracle.p8_value(A.T if ta else A),
                                             oracle.p8_value(B.T if tb else B)), K=K)


def test_chunk_gemm_degenerate():
    say("chunk_gemm K=0")
    C = gemm(dev(np.zeros((5, 1), np.uint8)), dev(np.zeros((1, 7), np.uint8)), 5, 7, 0, 64,
             lda=1, ldb=7)
    assert np.all(host(C) == 0)
    # -0 products give +0; Inf/NaN propagate
    A = np.array([[0x80, 0x80, 0x80], [0x7C, 0x3C, 0x00], [0x7D, 0x3C, 0x3C],
                  [0x7B, 0x7B, 0x7B]], np.uint8)
    B = np.array([[0x3C, 0x3C], [0xFC, 0x3C], [0x3C, 0x7C]], np.uint8)
    for mode in (fp8t.EXACT, fp8t.FAST):
        for CL in (1, 2, 16):
            say(f"chunk_gemm specials mode={mode} CL={CL}")
            Cg = host(gemm(dev(A), dev(B), 4, 2, 3, CL, mode=mode))
            assert np.array_equal(Cg, oracle.chunk_gemm(A, B, CL, mode=mode))


@pytest.mark.parametrize("guard", ["1", "0"])
@pytest.mark.parametrize("ta,tb", [(0, 0), (0, 1), (1, 0), (1, 1)])
def test_chunk_gemm_decodes_every_code(ta, tb, guard, monkeypatch):
    """All 256 FP8 codes (finite, subnormal, +-0, Inf, NaN) through both
    operands: a selection-like partner (1, 0, -1) makes the outputs the
    codes' own values and simple sums of them."""
    monkeypatch.setenv("FP8T_GEMM_GUARD", guard)
    codes = np.arange(256, dtype=np.uint8)
    X = np.stack([codes, codes[::-1]], axis=1)                 # 256 x 2
    Y = np.array([[0x3C, 0x00, 0xBC], [0x00, 0x3C, 0x3C]], np.uint8)   # 2 x 3
    for A, B, M, N in ((X, Y, 256, 3), (Y.T.copy(), X.T.copy(), 3, 256)):
        As = np.ascontiguousarray(A.T) if ta else A
        Bs = np.ascontiguousarray(B.T) if tb else B
        for CL in (1, 2):
            say(f"decode every code ta={ta} tb={tb} guard={guard} M={M} N={N} CL={CL}")
            Cg = host(gemm(dev(As), dev(Bs), M, N, 2, CL, ta, tb))
            Co = oracle.chunk_gemm(As, Bs, CL, ta, tb)
            assert np.array_equal(Cg, Co), np.argwhere(Cg != Co)[:5]


def test_chunk_gemm_guard_falls_back_per_piece(monkeypatch):
    """Tiles whose operands could overflow (or hold Inf/NaN) fail the guarded
    path's check and are recomputed on the safe path, in the same launch as
    tiles that pass; shared tiles mix both paths across their pieces."""
    rng = np.random.default_rng(570)
    M, N, K, CL = 300, 140, 1536, 64
    A, B = _operands(rng, M, N, K, 0, 0)
    A[5, :] = 0x7B                      # 57344: 9 K max|a| max|b| far above 2^31
    A[200, 700] = 0xFC                  # -Inf
    B[:, 3] = np.where(rng.random(K) < 0.5, 0x7A, 0xFA)   # +-49152
    Co = oracle.chunk_gemm(A, B, CL)
    for tile, split, wgs in (("auto", "0", "0"), ("auto", "0", "7"), ("auto", "1", "0"),
                             ("auto", "1", "7"), ("9", "0", "0"), ("9", "0", "7")):
        if tile == "auto":
            monkeypatch.delenv("FP8T_VALU_TILE", raising=False)
        else:
            monkeypatch.setenv("FP8T_VALU_TILE", tile)
        monkeypatch.setenv("FP8T_GEMM_SPLIT", split)
        monkeypatch.setenv("FP8T_GEMM_WGS", wgs)
        say(f"guard fallback tile={tile} split={split} wgs={wgs}")
        Cg = host(gemm(dev(A), dev(B), M, N, K, CL))
        assert np.array_equal(Cg, Co), np.argwhere(Cg != Co)[:5]


@pytest.mark.parametrize("tile", ["auto", "4", "9", "11"])
@pytest.mark.parametrize("CL", [64, 1024])
@pytest.mark.parametrize("b0", [0x50, 0x52, 0x56])
def test_chunk_gemm_guard_threshold(b0, CL, tile, monkeypatch):
    """All-positive operands whose running sums end near the guard's 2^31:
    A mostly 57344 and B mostly b0 = 32 (results 1.6e9 - 1.7e9: the guarded
    path), 48 (2.3e9 - 2.5e9: the tracked running sum fails the guard, the
    safe path) or 96 (beyond 4.29e9: FP16 overflow to Inf), with 10% smaller
    entries; CL = 64 keeps the chunk bound 3 CL max|a| max|b| below 2^31,
    CL = K = 1024 does not.  Every register tile and plan gives the oracle's
    bits."""
    if tile != "auto":
        monkeypatch.setenv("FP8T_VALU_TILE", tile)
    rng = np.random.default_rng(571 + b0)
    M, N, K = 192, 200, 1024
    A = np.full((M, K), 0x7B, np.uint8)
    B = np.full((K, N), b0, np.uint8)
    ma = rng.random(A.shape) < 0.1
    A[ma] = rng.integers(0x60, 0x7B, int(ma.sum()))
    mb = rng.random(B.shape) < 0.1
    B[mb] = rng.integers(0x40, b0, int(mb.sum()))
    Co = oracle.chunk_gemm(A, B, CL)
    v = oracle.p16_value(Co)
    say(f"guard threshold b0={b0:#x} CL={CL} tile={tile}: largest result {np.max(v):.4g}")
    for split, wgs in (("0", "0"), ("1", "7")):
        for guard in ("1", "0"):
            monkeypatch.setenv("FP8T_GEMM_SPLIT", split)
            monkeypatch.setenv("FP8T_GEMM_WGS", wgs)
            monkeypatch.setenv("FP8T_GEMM_GUARD", guard)
            say(f"guard threshold b0={b0:#x} CL={CL} tile={tile} split={split} wgs={wgs} "
                f"guard={guard}")
            Cg = host(gemm(dev(A), dev(B), M, N, K, CL))
            assert np.array_equal(Cg, Co), np.argwhere(Cg != Co)[:5]


@pytest.mark.parametrize("mtile", ["0", "1", "2", "3", "4"])
@pytest.mark.parametrize("wgs", ["0", "1"])
def test_chunk_gemm_fast_guard_falls_back(mtile, wgs, monkeypatch):
    """Fast mode: pieces whose chunk sums reach 2^32 are recomputed on the
    safe epilogue and give the bits of an all-safe run -- a few failing tiles
    among passing ones, and (one workgroup, every one of its 121 tiles
    failing) more failures than a workgroup remembers."""
    monkeypatch.setenv("FP8T_MFMA_TILE", mtile)
    monkeypatch.setenv("FP8T_GEMM_WGS", wgs)
    rng = np.random.default_rng(575)
    M, N, K, CL = 700, 650, 640, 64
    for case in ("some", "all"):
        A, B = _operands(rng, M, N, K, 0, 0)
        if case == "some":
            A[5, :] = 0x7B                  # 57344
            B[:, 300] = np.where(rng.random(K) < 0.5, 0x7A, 0xFA)   # +-49152
        else:
            A[:, :2] = 0x7B                 # first chunk of every output > 2^32
            B[:2, :] = 0x7B
        Ad, Bd = dev(A), dev(B)
        say(f"fast guard fallback mtile={mtile} wgs={wgs} case={case}")
        monkeypatch.setenv("FP8T_GEMM_GUARD", "1")
        Cg = host(gemm(Ad, Bd, M, N, K, CL, mode=fp8t.FAST))
        monkeypatch.setenv("FP8T_GEMM_GUARD", "0")
        Cs = host(gemm(Ad, Bd, M, N, K, CL, mode=fp8t.FAST))
        assert np.array_equal(Cg, Cs), np.argwhere(Cg != Cs)[:5]
        if case == "all":
            assert np.all(Cg == 0x7E00)
            assert np.array_equal(Cg, oracle.chunk_gemm(A, B, CL, mode=oracle.FAST))


@pytest.mark.parametrize("guard", ["1", "0"])
def test_chunk_gemm_overflow_to_inf(guard, monkeypatch):
    """Sums beyond the largest FP16 value become Inf and stay Inf."""
    monkeypatch.setenv("FP8T_GEMM_GUARD", guard)
    K = 64 * 40
    A = np.full((2, K), 0x7B, np.uint8)          # 57344
    B = np.full((K, 2), 0x7B, np.uint8)
    B[::2, 1] = 0xFB                              # alternate signs in column 1
    for mode in (fp8t.EXACT, fp8t.FAST):
        say(f"chunk_gemm overflow mode={mode} guard={guard}")
        Cg = host(gemm(dev(A), dev(B), 2, 2, K, 64, mode=mode))
        Co = oracle.chunk_gemm(A, B, 64, mode=mode)
        assert np.array_equal(Cg, Co)
        assert Cg[0, 0] == 0x7E00


def test_fig3b_stall_on_gpu():
    """Sec. 2.3, Fig. 3(b): CL = 1 stalls at exactly 4096, chunking does not."""
    import workloads
    x = workloads.accumulation_vector(12000)
    a = oracle.fp8_quantize(x)[None, :]
    ones = np.full((12000, 1), 0x3C, np.uint8)
    for CL in (1, 32, 64, 12000):
        say(f"fig3b CL={CL}")
        Cg = host(gemm(dev(a), dev(ones), 1, 1, 12000, CL))
        assert np.array_equal(Cg, oracle.chunk_gemm(a, ones, CL))
        if CL in (1, 12000):
            assert oracle.p16_value(Cg)[0, 0] == 4096.0


# ---- sr_weight_update --------------------------------------------------------------

def _update_case(rng, n, with_v=True, with_w8=True, lr=0.1, mu=0.9, wd=1e-4, seed=7, offset=0):
    w = oracle.fp16_quantize((rng.standard_normal(n) * 0.02).astype(np.float32))
    g = oracle.fp16_quantize((rng.standard_normal(n) * 1e-4).astype(np.float32))
    v = oracle.fp16_quantize((rng.standard_normal(n) * 1e-4).astype(np.float32)) if with_v else None
    wd_, gd = dev(w), dev(g)
    vd = dev(v) if with_v else None
    w8d = torch.zeros(n, dtype=torch.uint8, device=DEV) if with_w8 else None
    say(f"sr_weight_update n={n} v={with_v} w8={with_w8} lr={lr} mu={mu} wd={wd} seed={seed}"
        f" offset={offset}")
    fp8t.sr_weight_update(wd_, gd, vd, w8d, n, lr, mu if with_v else 0.0, wd, seed, offset)
    ow, ov, ow8 = oracle.sr_weight_update(w, g, v, lr=lr, momentum=mu if with_v else 0.0,
                                          weight_decay=wd, seed=seed, offset=offset,
                                          want_w8=with_w8)
    assert np.array_equal(host(wd_), ow)
    if with_v:
        assert np.array_equal(host(vd), ov)
    if with_w8:
        assert np.array_equal(host(w8d), ow8)


def test_sr_update_variants():
    rng = np.random.default_rng(540)
    for n in (1, 2, 3, 4097, 100_001):
        for with_v in (True, False):
            for with_w8 in (True, False):
                _update_case(rng, n, with_v, with_w8)
    _update_case(rng, 50_000, seed=2 ** 63 + 12345, offset=2 ** 40 + 7)
    _update_case(rng, 50_000, lr=0.0, mu=0.0, wd=0.0)


@pytest.mark.parametrize("n", [200_003, 4_500_001])
def test_sr_update_mixed_ranges(n):
    """Elements outside FP16's normal range (zeros, subnormals, values whose
    update leaves the range or overflows, Inf, NaN) scattered among ordinary
    ones: the groups holding them take the general path, the others the
    normal-range one, and both must agree with the oracle (at the larger size
    every thread of the capped grid loops over several pairs)."""
    rng = np.random.default_rng(544)
    w = oracle.fp16_quantize((rng.standard_normal(n) * 0.02).astype(np.float32))
    g = oracle.fp16_quantize((rng.standard_normal(n) * 1e-4).astype(np.float32))
    v = oracle.fp16_quantize((rng.standard_normal(n) * 1e-4).astype(np.float32))
    specials = np.uint16([0x0000, 0x8000, 0x0001, 0x81FF, 0x0200, 0x7DFF, 0xFDFF, 0x7C00,
                          0x7E00, 0xFE00, 0x7F00, 0x3E00])
    for arr in (w, g, v):
        idx = rng.choice(n, size=n // 500, replace=False)
        arr[idx] = rng.choice(specials, size=idx.size)
    wd_, gd, vd = dev(w), dev(g), dev(v)
    w8d = torch.zeros(n, dtype=torch.uint8, device=DEV)
    for lr, mu, wdk in ((0.1, 0.9, 1e-4), (3e4, 0.9, 0.5), (0.1, 0.0, 0.0)):
        say(f"sr_weight_update mixed ranges n={n} lr={lr} mu={mu} wd={wdk}")
        wd_.copy_(dev(w)); vd.copy_(dev(v))
        fp8t.sr_weight_update(wd_, gd, vd if mu else None, w8d, n, lr, mu, wdk, 11, 5)
        ow, ov, ow8 = oracle.sr_weight_update(w, g, v if mu else None, lr=lr, momentum=mu,
                                              weight_decay=wdk, seed=11, offset=5)
        assert np.array_equal(host(wd_), ow)
        if mu:
            assert np.array_equal(host(vd), ov)
        assert np.array_equal(host(w8d), ow8)


@pytest.mark.parametrize("lr", [float("inf"), float("nan"), -float("inf")])
def test_sr_update_non_finite_rate(lr):
    rng = np.random.default_rng(545)
    n = 4099
    _update_case(rng, n, lr=lr)
    _update_case(rng, n, lr=0.1, mu=float("nan"))


def test_sr_update_misaligned_pointers():
    rng = np.random.default_rng(541)
    n = 10_001
    w = oracle.fp16_quantize((rng.standard_normal(n + 1) * 0.02).astype(np.float32))
    g = oracle.fp16_quantize((rng.standard_normal(n + 1) * 1e-3).astype(np.float32))
    wd_, gd = dev(w), dev(g)
    w8d = torch.zeros(n + 1, dtype=torch.uint8, device=DEV)
    say("sr_weight_update misaligned")
    fp8t.lib().sr_weight_update(wd_.data_ptr() + 2, gd.data_ptr() + 2, None,
                                w8d.data_ptr() + 1, n, 0.1, 0.0, 0.0, 3, 9,
                                torch.cuda.current_stream().cuda_stream)
    ow, _, ow8 = oracle.sr_weight_update(w[1:], g[1:], None, lr=0.1, seed=3, offset=9)
    assert np.array_equal(host(wd_)[1:], ow)
    assert np.array_equal(host(w8d)[1:], ow8)


def test_sr_update_specials():
    w = np.array([0x7E00, 0xFE00, 0x7F00, 0x0000, 0x8000, 0x0001, 0x7DFF, 0x01FF], np.uint16)
    g = np.array([0x3C00, 0x3C00, 0x0000, 0x0001, 0x8001, 0x0000, 0xFDFF, 0x0001], np.uint16)
    v = np.array([0x0000, 0x7E00, 0x0000, 0x0000, 0x0000, 0x0200, 0x0000, 0x0003], np.uint16)
    wd_, gd, vd = dev(w), dev(g), dev(v)
    w8d = torch.zeros(8, dtype=torch.uint8, device=DEV)
    say("sr_weight_update specials")
    fp8t.sr_weight_update(wd_, gd, vd, w8d, 8, 1.5, 0.9, 1e-4, 1, 2)
    ow, ov, ow8 = oracle.sr_weight_update(w, g, v, lr=1.5, momentum=0.9, weight_decay=1e-4,
                                          seed=1, offset=2)
    assert np.array_equal(host(wd_), ow)
    assert np.array_equal(host(vd), ov)
    assert np.array_equal(host(w8d), ow8)
