"""FP8 GEMM parity on the GPU against the oracle's float64 product.

Bar: max |G - O| / max |O| <= 1e-3 per output (FP32 accumulation against an
exact-product float64 sum); bit-exact where every partial sum is an integer
below 2^24 (then FP32 accumulation is exact in any order)."""
import numpy as np
import pytest

from oracle import fp8, gemm
from tests.gpu_util import dev, rel_err, torch
from tests.libqe import need_lib

pytestmark = pytest.mark.gpu
FMTS = {0: "E4M3", 1: "E5M2"}


def rup16(v):
    return (v + 15) // 16 * 16


def random_codes(rng, rows, cols, fmt, ld):
    c = rng.integers(0, 256, size=(rows, ld), dtype=np.uint8)
    if fmt == 0:
        c[(c & 0x7F) == 0x7F] = 0x3C          # no NaN
    else:
        c[(c & 0x7C) == 0x7C] = 0x3C          # no inf / NaN
        c &= 0xBF                             # keep |values| <= 2^0 range-ish (exponent field < 16)
    return c


def run_gemm(qe, d, A, fa, B, fb, m, n, k, sa, sb, out, ldc, mode=0, c_init=None):
    lda, ldb = A.shape[1], B.shape[1]
    a_t = torch.from_numpy(A).to(d)
    b_t = torch.from_numpy(B).to(d)
    s = torch.tensor([sa, sb], dtype=torch.float32, device=d)
    if out == qe.BF16:
        c_t = torch.zeros(max(m * ldc, 1), dtype=torch.int16, device=d)
    else:
        c_t = torch.from_numpy(c_init.copy()).to(d) if c_init is not None else \
            torch.zeros(max(m * ldc, 1), dtype=torch.float32, device=d)
    st = qe.qe_fp8_gemm_tn(a_t, fa, lda, b_t, fb, ldb, m, n, k, s[0:1], s[1:2], c_t, out, ldc, mode)
    assert st == "OK", st
    torch.cuda.synchronize()
    c = c_t.cpu().numpy()
    if out == qe.BF16:
        c = (c.view(np.uint16).astype(np.uint32) << 16).view(np.float32)
    return c


SHAPES = [(1, 1, 1), (16, 16, 128), (37, 53, 100), (256, 256, 128), (300, 520, 384), (513, 257, 1000),
          (128, 256, 256), (64, 96, 16), (255, 511, 129)]


@pytest.mark.parametrize("shape", SHAPES, ids=lambda s: "x".join(map(str, s)))
@pytest.mark.parametrize("fa,fb", [(0, 0), (1, 0), (0, 1), (1, 1)])
def test_random_codes(shape, fa, fb):
    qe = need_lib()
    d = dev()
    m, n, k = shape
    rng = np.random.default_rng(m * 7 + n * 13 + k + fa * 2 + fb)
    A = random_codes(rng, m, k, fa, rup16(k))
    B = random_codes(rng, n, k, fb, rup16(k))
    sa, sb = 2.0 ** -3, 2.0 ** 5
    ref = gemm.gemm_tn(A[:, :k], FMTS[fa], B[:, :k], FMTS[fb], sa, sb)
    got = run_gemm(qe, d, A, fa, B, fb, m, n, k, sa, sb, qe.F32, n)[: m * n].reshape(m, n)
    assert rel_err(got, ref) <= 1e-3


@pytest.mark.parametrize("shape", [(37, 53, 100), (300, 520, 384), (256, 512, 4096)], ids=str)
def test_integer_operands_bit_exact(shape):
    """Codes of small integers: every partial sum is an integer < 2^24, so the
    FP32 result must equal the exact integer product bit for bit."""
    qe = need_lib()
    d = dev()
    m, n, k = shape
    rng = np.random.default_rng(5)
    ai = rng.integers(-6, 7, size=(m, k))
    bi = rng.integers(-6, 7, size=(n, k))
    A = np.zeros((m, rup16(k)), dtype=np.uint8)
    B = np.zeros((n, rup16(k)), dtype=np.uint8)
    A[:, :k] = fp8.encode(ai.astype(np.float64), "E4M3")
    B[:, :k] = fp8.encode(bi.astype(np.float64), "E5M2")
    got = run_gemm(qe, d, A, 0, B, 1, m, n, k, 1.0, 0.5, qe.F32, n)[: m * n].reshape(m, n)
    np.testing.assert_array_equal(got, (ai @ bi.T).astype(np.float32) * np.float32(0.5))


def test_bf16_output():
    qe = need_lib()
    d = dev()
    m, n, k = 200, 300, 512
    rng = np.random.default_rng(9)
    A = random_codes(rng, m, k, 0, k)
    B = random_codes(rng, n, k, 0, k)
    ref = gemm.gemm_tn(A, "E4M3", B, "E4M3", 0.25, 0.125)
    got = run_gemm(qe, d, A, 0, B, 0, m, n, k, 0.25, 0.125, qe.BF16, n)[: m * n].reshape(m, n)
    # a bf16 result is within half a bf16 ulp (2^-9 relative, 2^-8 at worst
    # across a binade edge) of the FP32 accumulation, which is within 1e-3
    assert rel_err(got, ref) <= 2.0 ** -8 + 1e-3


@pytest.mark.parametrize("shape", [(40, 70, 64), (256, 256, 256), (300, 257, 130)], ids=str)
def test_accumulate_strided_view_untouched_elsewhere(shape):
    """ACCUM into a strided view of a flat buffer: the view gets fl32(G + D);
    every other element (before, after, and the row gaps) keeps its sentinel."""
    qe = need_lib()
    d = dev()
    m, n, k = shape
    ldc, off = n + 9, 37
    rng = np.random.default_rng(3)
    A = random_codes(rng, m, k, 1, rup16(k))
    B = random_codes(rng, n, k, 0, rup16(k))
    total = off + (m - 1) * ldc + n + 50
    G = rng.standard_normal(total).astype(np.float32)
    a_t, b_t = torch.from_numpy(A).to(d), torch.from_numpy(B).to(d)
    s = torch.tensor([0.5, 2.0], dtype=torch.float32, device=d)
    g_t = torch.from_numpy(G.copy()).to(d)
    view = g_t[off:]
    assert qe.qe_fp8_gemm_tn(a_t, 1, A.shape[1], b_t, 0, B.shape[1], m, n, k, s[0:1], s[1:2], view, qe.F32, ldc,
                             qe.ACCUM) == "OK"
    torch.cuda.synchronize()
    got = g_t.cpu().numpy()
    ref = G.copy()
    gemm.place(ref, gemm.gemm_tn(A[:, :k], "E5M2", B[:, :k], "E4M3", 0.5, 2.0), off, ldc, accumulate=True)
    idx = gemm.view_index(off, ldc, m, n)
    mask = np.ones(total, dtype=bool)
    mask[idx.ravel()] = False
    np.testing.assert_array_equal(got[mask], G[mask])
    assert rel_err(got[idx], ref[idx]) <= 1e-3


def test_k_zero_and_empty():
    qe = need_lib()
    d = dev()
    A = np.zeros((8, 16), dtype=np.uint8)
    B = np.zeros((4, 16), dtype=np.uint8)
    got = run_gemm(qe, d, A, 0, B, 0, 8, 4, 0, 1.0, 1.0, qe.F32, 4, c_init=np.full(32, 3.0, dtype=np.float32))
    np.testing.assert_array_equal(got, np.zeros(32, dtype=np.float32))
    got = run_gemm(qe, d, A, 0, B, 0, 8, 4, 0, 1.0, 1.0, qe.F32, 4, mode=1,
                   c_init=np.full(32, 3.0, dtype=np.float32))
    np.testing.assert_array_equal(got, np.full(32, 3.0, dtype=np.float32))
    assert qe.qe_fp8_gemm_tn(0, 0, 16, 0, 0, 16, 0, 4, 16, 0, 0, 0, qe.F32, 4) == "OK"


@pytest.mark.parametrize("shape", [(4096, 4096, 1024), (4096, 6144, 1024), (4100, 4100, 1040)], ids=str)
def test_large_grids_bit_exact(shape):
    """Grids large enough to select each macro-tile shape (256 x 256 when the
    grid fills whole rounds of CUs, 256 x 128 otherwise), integer operands so
    the result is exact."""
    qe = need_lib()
    d = dev()
    m, n, k = shape
    g = torch.Generator(device=d)
    g.manual_seed(11)
    ai = torch.randint(-6, 7, (m, k), device=d, generator=g)
    bi = torch.randint(-6, 7, (n, k), device=d, generator=g)
    lut = torch.from_numpy(fp8.encode(np.arange(-6, 7, dtype=np.float64), "E4M3")).to(d)
    a_t = lut[(ai + 6)].contiguous()
    b_t = lut[(bi + 6)].contiguous()
    s = torch.tensor([1.0, 1.0], dtype=torch.float32, device=d)
    c = torch.empty((m, n), dtype=torch.float32, device=d)
    assert qe.qe_fp8_gemm_tn(a_t, 0, k, b_t, 0, k, m, n, k, s[0:1], s[1:2], c, qe.F32, n) == "OK"
    ref = (ai.double() @ bi.double().T).float()
    assert torch.equal(c, ref)


@pytest.fixture
def forced_tile():
    """Sets a forced macro-tile shape for one test and restores the cost model after it."""
    qe = need_lib()
    yield qe
    assert qe.qe_set_gemm_tile(qe.TILE_AUTO) == "OK"


def _int_operands(d, m, n, k, seed):
    """Integer-valued E4M3 operands with rows padded to a multiple of 16 bytes
    (padding codes are arbitrary and must be ignored)."""
    g = torch.Generator(device=d)
    g.manual_seed(seed)
    ld = rup16(k)
    ai = torch.randint(-6, 7, (m, ld), device=d, generator=g)
    bi = torch.randint(-6, 7, (n, ld), device=d, generator=g)
    lut = torch.from_numpy(fp8.encode(np.arange(-6, 7, dtype=np.float64), "E4M3")).to(d)
    return ai[:, :k], bi[:, :k], lut[(ai + 6)].contiguous(), lut[(bi + 6)].contiguous()


# full tiles of every shape, ragged edges in M, N and K, a partial last K tile,
# and grids of several rounds
TILE_SHAPES = [(768, 768, 256), (1000, 700, 320), (576, 4096, 384), (4096, 576, 130), (2304, 2304, 512),
               (193, 191, 129), (4096, 6144, 256), (2048, 7168, 384)]


@pytest.mark.parametrize("tile", [1, 2, 3, 4, 5], ids=["256x256", "256x192", "192x256", "256x128", "256x224"])
@pytest.mark.parametrize("shape", TILE_SHAPES, ids=lambda s: "x".join(map(str, s)))
def test_forced_tile_shapes_exact(forced_tile, tile, shape):
    """Each macro-tile shape on integer operands: FP32 store, BF16 store and
    FP32 accumulate into a strided view are exact (every partial sum is an
    integer below 2^24), on full tiles (the branch-free epilogue) and on ragged
    edges (the checked one)."""
    qe = forced_tile
    d = dev()
    assert qe.qe_set_gemm_tile(tile) == "OK"
    m, n, k = shape
    ai, bi, a_t, b_t = _int_operands(d, m, n, k, 5 + tile)
    lda = a_t.shape[1]
    ref = ai.double() @ bi.double().T
    s = torch.tensor([1.0, 1.0], dtype=torch.float32, device=d)
    c = torch.empty((m, n), dtype=torch.float32, device=d)
    assert qe.qe_fp8_gemm_tn(a_t, 0, lda, b_t, 0, lda, m, n, k, s[0:1], s[1:2], c, qe.F32, n) == "OK"
    assert torch.equal(c, ref.float())
    # bf16: the exact FP32 result rounded to nearest even
    cb = torch.empty((m, n), dtype=torch.int16, device=d)
    assert qe.qe_fp8_gemm_tn(a_t, 0, lda, b_t, 0, lda, m, n, k, s[0:1], s[1:2], cb, qe.BF16, n) == "OK"
    assert torch.equal(cb.view(torch.bfloat16), ref.float().to(torch.bfloat16))
    # accumulate into a view with ld > n; the padding columns stay untouched
    ld = n + 8
    base = torch.randint(-50, 50, (m, ld), device=d, generator=torch.Generator(device=d).manual_seed(3)).float()
    ca = base.clone()
    assert qe.qe_fp8_gemm_tn(a_t, 0, lda, b_t, 0, lda, m, n, k, s[0:1], s[1:2], ca, qe.F32, ld, qe.ACCUM) == "OK"
    torch.cuda.synchronize()
    assert torch.equal(ca[:, :n], (base[:, :n].double() + ref).float())
    assert torch.equal(ca[:, n:], base[:, n:])


@pytest.mark.parametrize("shape", [(768, 768, 1000), (1000, 700, 320), (576, 4096, 384), (1024, 1344, 640)], ids=str)
def test_tile_shapes_same_bits(forced_tile, shape):
    """Every macro-tile shape (256x256, 256x224, 256x192, 192x256 with four
    waves, 256x128 with eight) runs the same MFMA with the same reduction bytes per
    lane in the same K order: on random codes (inexact FP32 sums) their outputs
    are bit-identical."""
    qe = forced_tile
    d = dev()
    m, n, k = shape
    rng = np.random.default_rng(m + n + k)
    A = random_codes(rng, m, k, 0, rup16(k))
    B = random_codes(rng, n, k, 1, rup16(k))
    outs = []
    for tile in (1, 2, 3, 4, 5):
        assert qe.qe_set_gemm_tile(tile) == "OK"
        outs.append(run_gemm(qe, d, A, 0, B, 1, m, n, k, 2.0 ** -2, 2.0 ** 3, qe.F32, n)[: m * n])
    ref = gemm.gemm_tn(A[:, :k], "E4M3", B[:, :k], "E5M2", 2.0 ** -2, 2.0 ** 3)
    assert rel_err(outs[0].reshape(m, n), ref) <= 1e-3
    for o in outs[1:]:
        np.testing.assert_array_equal(o, outs[0])


def _lut_codes(d, seed, rows, cols, lo, hi, fmt):
    """Device operands of small integers lo..hi as FP8 codes (exact in either
    format), drawn on the device; returns (the values as uint8 offsets from lo,
    on the host, for the reference; the codes, on the device)."""
    g = torch.Generator(device=d)
    g.manual_seed(seed)
    vals = torch.randint(0, hi - lo + 1, (rows, cols), dtype=torch.uint8, device=d, generator=g)
    lut = torch.from_numpy(fp8.encode(np.arange(lo, hi + 1, dtype=np.float64), fmt)).to(d)
    codes = lut[vals.int()]
    return vals.cpu().numpy(), codes


def _rows_exact(vals, lo, idx, other_vals, other_lo):
    """Exact integer products of the sampled rows `idx` of one operand with every row of the other."""
    a = vals[idx].astype(np.int64) + lo
    b = other_vals.astype(np.int64) + other_lo
    return a @ b.T


@pytest.mark.parametrize("split", ["rows_of_a", "rows_of_b"])
def test_operands_of_2gib_split_into_row_blocks(split):
    """An operand of 2 GiB or more (the kernel's 32-bit offsets) runs as
    launches over row blocks of whole 256-row tiles: 524,588 rows of 4,096
    bytes split at row 524,032.  Integer operands, so every output is exact:
    sampled rows and columns (either side of the split, the ends, random ones)
    against the integer product, and every column (or row) sum of the output
    against the sum of the integer operand rows times the other operand.  A
    split of A stores FP32, then BF16 (the rounding of that exact FP32); a
    split of B accumulates into an FP32 destination of integers."""
    qe = need_lib()
    d = dev()
    big, small, k = 524_588, 200, 4096
    assert big * k >= 1 << 31
    cut = (((1 << 31) - 1) // k) // 256 * 256
    rng = np.random.default_rng(2031)
    bv, big_t = _lut_codes(d, 2031, big, k, -6, 6, "E4M3")
    sv, small_t = _lut_codes(d, 2032, small, k, -6, 6, "E5M2")
    s = torch.tensor([1.0, 1.0], dtype=torch.float32, device=d)
    picks = np.unique(np.concatenate([[0, 1, cut - 1, cut, cut + 1, big - 2, big - 1],
                                      rng.integers(0, big, size=9)]))
    big_sum = bv.sum(axis=0, dtype=np.int64) - 6 * big        # sum over the big operand's rows
    sum_ref = (big_sum @ (sv.astype(np.int64) - 6).T)         # per row of the small operand
    ref_picks = _rows_exact(bv, -6, picks, sv, -6)            # [picks, small]
    if split == "rows_of_a":
        m, n = big, small
        c = torch.empty((m, n), dtype=torch.float32, device=d)
        assert qe.qe_fp8_gemm_tn(big_t, 0, k, small_t, 1, k, m, n, k, s[0:1], s[1:2], c, qe.F32, n) == "OK"
        cb = torch.empty((m, n), dtype=torch.int16, device=d)
        assert qe.qe_fp8_gemm_tn(big_t, 0, k, small_t, 1, k, m, n, k, s[0:1], s[1:2], cb, qe.BF16, n) == "OK"
        torch.cuda.synchronize()
        np.testing.assert_array_equal(c[torch.from_numpy(picks).to(d)].cpu().numpy(), ref_picks.astype(np.float32))
        np.testing.assert_array_equal(c.double().sum(dim=0).cpu().numpy(), sum_ref.astype(np.float64))
        assert torch.equal(cb.view(torch.bfloat16), c.to(torch.bfloat16))
    else:
        m, n = small, big
        base = rng.integers(-50, 50, size=(m, n)).astype(np.float32)
        c = torch.from_numpy(base).to(d)
        assert qe.qe_fp8_gemm_tn(small_t, 1, k, big_t, 0, k, m, n, k, s[0:1], s[1:2], c, qe.F32, n,
                                 qe.ACCUM) == "OK"
        torch.cuda.synchronize()
        got = c[:, torch.from_numpy(picks).to(d)].cpu().numpy()
        np.testing.assert_array_equal(got, (base[:, picks] + ref_picks.T).astype(np.float32))
        np.testing.assert_array_equal(c.double().sum(dim=1).cpu().numpy(),
                                      base.astype(np.float64).sum(axis=1) + sum_ref.astype(np.float64))


def test_long_reduction_blocks_below_one_tile():
    """A reduction of 2^23 + 100 bytes per row: a 256-row tile of A would pass
    2 GiB, so A runs in blocks of 255 rows (then 5), each a partial tile, with a
    partial last K tile.  Operands in {-1, 0, 1}: every partial sum is an
    integer of magnitude <= 2^23, so the FP32 result is exact in any order."""
    qe = need_lib()
    d = dev()
    m, n, k = 260, 16, (1 << 23) + 100
    ld = rup16(k)
    assert ((1 << 31) - 1) // ld == 255
    av, a_t = _lut_codes(d, 23, m, ld, -1, 1, "E4M3")
    bv, b_t = _lut_codes(d, 24, n, ld, -1, 1, "E4M3")
    a_t[:, k:] = 0x38                             # padding bytes past k (code of 1.0) must be ignored
    b_t[:, k:] = 0x38
    s = torch.tensor([1.0, 0.5], dtype=torch.float32, device=d)
    c = torch.empty((m, n), dtype=torch.float32, device=d)
    assert qe.qe_fp8_gemm_tn(a_t, 0, ld, b_t, 0, ld, m, n, k, s[0:1], s[1:2], c, qe.F32, n) == "OK"
    torch.cuda.synchronize()
    got = c.cpu().numpy()
    # exact: small integers in float32 BLAS (every partial sum an integer below 2^24)
    b = bv[:, :k].astype(np.float32) - 1.0
    for r in range(0, m, 32):
        a = av[r:r + 32, :k].astype(np.float32) - 1.0
        np.testing.assert_array_equal(got[r:r + 32], (a @ b.T) * np.float32(0.5))


# K at and around every count of K tiles the load pipeline treats differently
# (1 to 9 tiles of 128, full or with a partial last tile), with ragged M and N
K_EDGE_SHAPES = [(596, 126, 1), (19, 448, 15), (256, 327, 16), (56, 259, 17), (450, 249, 127), (581, 553, 128),
                 (493, 633, 129), (505, 124, 255), (601, 457, 256), (69, 209, 257), (116, 676, 383),
                 (509, 643, 384), (198, 445, 385), (423, 527, 640), (83, 361, 897), (451, 578, 1152)]


@pytest.mark.parametrize("shape", K_EDGE_SHAPES, ids=lambda s: "x".join(map(str, s)))
def test_k_tile_counts_exact_every_tile_shape(forced_tile, shape):
    """Every macro-tile shape at every small count of K tiles (the prologue,
    the split loads of the K loop, the partial last tile through registers):
    integer operands, FP32 store and FP32 accumulate exact against the integer
    product, and the shapes' outputs identical."""
    qe = forced_tile
    d = dev()
    m, n, k = shape
    ai, bi, a_t, b_t = _int_operands(d, m, n, k, k + 3)
    lda = a_t.shape[1]
    ref = (ai.double() @ bi.double().T).float()
    s = torch.tensor([1.0, 1.0], dtype=torch.float32, device=d)
    base = torch.randint(-50, 50, (m, n), device=d, generator=torch.Generator(device=d).manual_seed(k)).float()
    outs = []
    for tile in (1, 2, 3, 4, 5):
        assert qe.qe_set_gemm_tile(tile) == "OK"
        c = torch.empty((m, n), dtype=torch.float32, device=d)
        assert qe.qe_fp8_gemm_tn(a_t, 0, lda, b_t, 0, lda, m, n, k, s[0:1], s[1:2], c, qe.F32, n) == "OK"
        ca = base.clone()
        assert qe.qe_fp8_gemm_tn(a_t, 0, lda, b_t, 0, lda, m, n, k, s[0:1], s[1:2], ca, qe.F32, n, qe.ACCUM) == "OK"
        torch.cuda.synchronize()
        assert torch.equal(c, ref), tile
        assert torch.equal(ca, base + ref), tile
        outs.append(c)
    for o in outs[1:]:
        assert torch.equal(o, outs[0])


def _sweep_shapes(count, seed):
    rng = np.random.default_rng(seed)
    return [(int(rng.integers(1, 1300)), int(rng.integers(1, 1300)), int(rng.integers(1, 2600)))
            for _ in range(count)]


@pytest.mark.parametrize("shape", _sweep_shapes(40, 77), ids=lambda s: "x".join(map(str, s)))
def test_seeded_shape_sweep_exact(shape):
    """Forty seeded random shapes (M, N up to 1,300, K up to 2,600) under the
    automatic tile choice: FP32 store, BF16 store and FP32 accumulate into a
    padded view, exact on integer operands."""
    qe = need_lib()
    d = dev()
    m, n, k = shape
    ai, bi, a_t, b_t = _int_operands(d, m, n, k, m + n + k)
    lda = a_t.shape[1]
    ref = ai.double() @ bi.double().T
    s = torch.tensor([1.0, 1.0], dtype=torch.float32, device=d)
    c = torch.empty((m, n), dtype=torch.float32, device=d)
    assert qe.qe_fp8_gemm_tn(a_t, 0, lda, b_t, 0, lda, m, n, k, s[0:1], s[1:2], c, qe.F32, n) == "OK"
    cb = torch.empty((m, n), dtype=torch.int16, device=d)
    assert qe.qe_fp8_gemm_tn(a_t, 0, lda, b_t, 0, lda, m, n, k, s[0:1], s[1:2], cb, qe.BF16, n) == "OK"
    ld = n + 5
    base = torch.randint(-50, 50, (m, ld), device=d, generator=torch.Generator(device=d).manual_seed(k)).float()
    ca = base.clone()
    assert qe.qe_fp8_gemm_tn(a_t, 0, lda, b_t, 0, lda, m, n, k, s[0:1], s[1:2], ca, qe.F32, ld, qe.ACCUM) == "OK"
    torch.cuda.synchronize()
    assert torch.equal(c, ref.float())
    assert torch.equal(cb.view(torch.bfloat16), ref.float().to(torch.bfloat16))
    assert torch.equal(ca[:, :n], (base[:, :n].double() + ref).float())
    assert torch.equal(ca[:, n:], base[:, n:])
