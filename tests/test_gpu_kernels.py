"""Parity of the gfx950 kernels with the CPU oracle (through the C ABI).

Integer results (codes, zero points, accumulators, code sums) must be
bit-exact; fp32 results that both sides compute with the same IEEE operations
(recovery factors, recovered products, gate functions) are required bit-exact
as well, which is stronger than the 1e-4 tolerance on float outputs."""
import numpy as np
import pytest
import torch

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def ql():
    assert torch.cuda.is_available(), "GPU tests need an MI355X"
    from paper_1607_04683_amd import qlstm
    qlstm.load()
    return qlstm


def u8(codes_dev, cols):
    """Device-layout int8 codes -> the paper's uint8 V' (numpy)."""
    return (codes_dev[:, :cols].contiguous().cpu().numpy().view(np.uint8) ^ 0x80)


def test_gate_functions_bit_exact(ql, orc):
    x = np.concatenate([np.linspace(-100, 100, 1_000_001, dtype=np.float32),
                        np.float32([0.0, -0.0, 1e-38, -1e-38, 87.0, -87.0, 88.5, -88.5, 1e30])])
    xd = torch.from_numpy(x).cuda()
    for fn, ref in ((0, orc.expf), (1, orc.sigmoidf), (2, orc.tanhf)):
        got = ql.gate_fn(fn, xd).cpu().numpy()
        want = ref(x)
        assert np.array_equal(got.view(np.uint32), want.view(np.uint32)), fn


def test_gate_reciprocal_equals_ieee_division(ql):
    """The reciprocal inside sigmoid (v_rcp_f32 + two Newton steps) against
    IEEE fp32 division 1 / d on the CPU: every mantissa at the bottom, middle
    and top binades of the gate denominators 1 + e^-x (x clamped to 87, so
    d <= 1 + e^87 < 6.1e37), and the whole top range up to 6.1e37."""
    mant = np.arange(1 << 23, dtype=np.uint32)
    top = np.float32(6.1e37).view(np.uint32)
    chunks = [(np.uint32(e + 127) << np.uint32(23)) | mant for e in (0, 1, 2, 23, 24, 60, 100)]
    chunks.append(np.arange(np.uint32(125 + 127) << np.uint32(23), top + 1, dtype=np.uint32))
    for bits in chunks:
        d = bits.view(np.float32)
        got = ql.gate_fn(3, torch.from_numpy(d).cuda()).cpu().numpy()
        want = np.float32(1.0) / d
        bad = np.flatnonzero(got.view(np.uint32) != want.view(np.uint32))
        assert bad.size == 0, (d[bad[:4]], got[bad[:4]], want[bad[:4]])


@pytest.mark.parametrize("rows,cols,nblocks", [(2000, 320, 4), (2000, 500, 4), (256, 128, 1),
                                               (8192, 512, 1), (37, 5, 1), (64, 1, 4),
                                               (12, 130, 3)])
def test_quantize_matches_oracle(ql, orc, rows, cols, nblocks):
    rng = np.random.default_rng(rows * 7 + cols)
    W = rng.uniform(-0.08, 0.08, (rows, cols)).astype(np.float32)
    if nblocks > 1:
        W[: rows // nblocks] *= 3.0
    q = ql.quantize(torch.from_numpy(W).cuda(), nblocks)
    o = orc.quantize(W, nblocks)
    assert np.array_equal(u8(q.codes, cols), o.codes)
    assert np.array_equal(q.zero.cpu().numpy(), o.zero)
    assert np.array_equal(q.inv_q.cpu().numpy().view(np.uint32), o.inv_q.view(np.uint32))
    assert np.array_equal(q.range.cpu().numpy(), o.range)
    assert np.array_equal(q.row_sums.cpu().numpy(), o.row_sums)
    assert (q.codes[:, cols:] == 0).all()   # padding is 0 in the signed layout
    back = ql.dequantize(q).cpu().numpy()
    assert np.array_equal(back.view(np.uint32), orc.dequantize(o).view(np.uint32))


def test_quantize_degenerate_blocks(ql, orc):
    W = np.zeros((8, 9), np.float32)
    W[2:4] = 1.5          # constant positive block
    W[4:6] = -0.25        # constant negative block
    W[6:8] = np.float32([[1000.0] * 9, [1000.0001] * 9])  # ill-conditioned block
    q = ql.quantize(torch.from_numpy(W).cuda(), 4)
    o = orc.quantize(W, 4)
    assert np.array_equal(u8(q.codes, 9), o.codes)
    assert np.array_equal(q.zero.cpu().numpy(), o.zero)
    assert np.array_equal(q.inv_q.cpu().numpy(), o.inv_q)


def _qmm_case(ql, orc, W, X, gran, nblocks=1, bias=None):
    q = ql.quantize(torch.from_numpy(W).cuda(), nblocks)
    b = None if bias is None else torch.from_numpy(bias).cuda()
    Y, acc = ql.quantized_matmul(q, torch.from_numpy(X).cuda(), gran, b, want_acc=True)
    o = orc.quantized_matmul(orc.quantize(W, nblocks), X, act_gran=gran, bias=bias)
    return Y.cpu().numpy(), acc.cpu().numpy(), o


def test_qmatmul_standalone_256x128_per_tensor(ql, orc):
    """The standalone product: W 256x128 ~ N(0, 0.1), X 16x128 ~ U[-1, 1],
    both quantized per tensor -> 16x256 fp32."""
    from paper_1607_04683_amd.workloads import qmatmul_operands
    W, X = qmatmul_operands()
    Y, acc, o = _qmm_case(ql, orc, W, X, gran=0)
    assert np.array_equal(acc, o["acc"])
    assert np.array_equal(Y.view(np.uint32), o["Y"].view(np.uint32))
    assert np.max(np.abs(Y - o["Y"])) <= 1e-4


@pytest.mark.parametrize("m,rows,cols,nblocks", [(1, 1, 1, 1), (5, 33, 7, 1), (130, 257, 129, 1),
                                                 (300, 2000, 320, 4), (77, 100, 500, 4),
                                                 (129, 8192, 512, 1), (3, 16, 2048, 4)])
@pytest.mark.parametrize("gran", [0, 1])
def test_qmatmul_ragged_shapes(ql, orc, m, rows, cols, nblocks, gran):
    rng = np.random.default_rng(m * 1000 + rows + cols)
    W = rng.normal(0, 0.05, (rows, cols)).astype(np.float32)
    X = rng.standard_normal((m, cols)).astype(np.float32)
    bias = rng.normal(0, 0.1, rows).astype(np.float32)
    Y, acc, o = _qmm_case(ql, orc, W, X, gran, nblocks, bias)
    assert np.array_equal(acc, o["acc"])
    assert np.array_equal(Y.view(np.uint32), o["Y"].view(np.uint32))


@pytest.mark.parametrize("m,rows,cols", [(2100, 8200, 333), (4096, 4100, 64)])
def test_qmatmul_large_tiles_sampled_rows(ql, orc, m, rows, cols):
    """Products large enough for the 256x256 tiles (K of 333 and of 64 take
    the two pipeline depths), ragged in rows and columns: sampled rows of the
    recovered output and of the accumulators against the oracle (per-row
    activation quantization keeps rows independent)."""
    rng = np.random.default_rng(m + rows + cols)
    W = rng.normal(0, 0.05, (rows, cols)).astype(np.float32)
    X = rng.standard_normal((m, cols)).astype(np.float32)
    bias = rng.normal(0, 0.1, rows).astype(np.float32)
    q = ql.quantize(torch.from_numpy(W).cuda(), 4)
    Y, acc = ql.quantized_matmul(q, torch.from_numpy(X).cuda(), 1, torch.from_numpy(bias).cuda(),
                                 want_acc=True)
    sel = np.unique(np.concatenate([[0, 1, 255, 256, m - 257, m - 1], rng.choice(m, 24, replace=False)]))
    o = orc.quantized_matmul(orc.quantize(W, 4), X[sel], act_gran=1, bias=bias)
    idx = torch.from_numpy(sel).cuda()
    assert np.array_equal(acc[idx].cpu().numpy(), o["acc"])
    assert np.array_equal(Y[idx].cpu().numpy().view(np.uint32), o["Y"].view(np.uint32))


def test_qmatmul_max_k_accumulator(ql, orc):
    """K = 33025 with nearly all codes 255: sum_k 255*255 is just below 2^31."""
    K = 33025
    W = np.ones((4, K), np.float32)
    W[:, 0] = 0.0
    X = np.ones((2, K), np.float32)
    X[:, 1] = -1.0
    Y, acc, o = _qmm_case(ql, orc, W, X, gran=1)
    assert np.array_equal(acc, o["acc"])
    assert acc.max() > 2 ** 31 - 2 ** 20
    assert np.array_equal(Y, o["Y"])


def test_qmatmul_empty(ql):
    """m = 0 rows: a no-op, with null data pointers accepted."""
    q = ql.quantize(torch.randn(8, 16, device="cuda"), 1)
    Y, acc = ql.quantized_matmul(q, torch.empty(0, 16, device="cuda"), 1, want_acc=True)
    assert Y.shape == (0, 8)


@pytest.mark.parametrize("M,N,K", [(1, 1, 1), (129, 130, 131), (256, 256, 64), (300, 77, 1000),
                                   (64, 2000, 500)])
def test_gemm_u8_matches_oracle(ql, orc, M, N, K):
    rng = np.random.default_rng(M + N + K)
    A = rng.integers(0, 256, (M, K), dtype=np.uint8)
    Bm = rng.integers(0, 256, (N, K), dtype=np.uint8)
    got = ql.gemm_u8(ql.device_codes(A), ql.device_codes(Bm), K).cpu().numpy()
    assert np.array_equal(got, orc.gemm_u8(A, Bm))


@pytest.mark.parametrize("M,N,K", [(4100, 4000, 1000), (4096, 4352, 64), (8192, 2048, 2000)])
def test_gemm_u8_large_tiles_ragged(ql, orc, M, N, K):
    """Shapes large enough for the 256x256 tiles, with ragged M, N and K:
    sampled rows (first and last tile rows included) against the oracle."""
    rng = np.random.default_rng(M ^ N ^ K)
    A = rng.integers(0, 256, (M, K), dtype=np.uint8)
    Bm = rng.integers(0, 256, (N, K), dtype=np.uint8)
    got = ql.gemm_u8(ql.device_codes(A), ql.device_codes(Bm), K)
    rows = np.unique(np.concatenate([[0, 1, 255, 256, M - 257, M - 1],
                                     rng.choice(M, 16, replace=False)]))
    want = orc.gemm_u8(A[rows], Bm)
    assert np.array_equal(got[torch.from_numpy(rows).cuda()].cpu().numpy(), want)


@pytest.mark.parametrize("n", [4096, 8192])
def test_gemm_u8_sweep_sizes_sampled_rows(ql, orc, n):
    """M = N = K = n with U{0..255} operands: sampled rows of C against the
    oracle's integer product of those rows."""
    from paper_1607_04683_amd.workloads import gemm_operands
    A, Bm = gemm_operands(n, n, n, seed=0)
    got = ql.gemm_u8(ql.device_codes(A), ql.device_codes(Bm), n)
    rows = np.sort(np.random.default_rng(n).choice(n, 24, replace=False))
    rows = np.concatenate([[0], rows, [n - 1]])
    want = orc.gemm_u8(A[rows], Bm)
    assert np.array_equal(got[torch.from_numpy(rows).cuda()].cpu().numpy(), want)


@pytest.mark.parametrize("m,cols", [(1, 1), (7, 5), (300, 320), (64, 500), (33, 2048), (0, 16)])
def test_quantize_activations_per_vector(ql, orc, m, cols):
    """Every row quantized as its own vector (eq. 2): the oracle's per-block
    quantizer with one block per row gives the same codes and params."""
    rng = np.random.default_rng(m * 31 + cols)
    X = rng.standard_normal((m, cols)).astype(np.float32)
    if m >= 3:
        X[1] = 0.0        # all-zero vector
        X[2] = 0.75       # constant vector
    q = ql.quantize_activations(torch.from_numpy(X).cuda())
    if m == 0:
        return
    o = orc.quantize(X, m)
    assert np.array_equal(u8(q.codes, cols), o.codes)
    assert np.array_equal(q.zero.cpu().numpy(), o.zero)
    assert np.array_equal(q.inv_q.cpu().numpy().view(np.uint32), o.inv_q.view(np.uint32))
    assert np.array_equal(q.sums.cpu().numpy(), o.codes.astype(np.int64).sum(1))
    assert (q.codes[:, cols:] == 0).all()
