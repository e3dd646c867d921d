"""Parity of the bf16 MFMA GEMM (layup_gemm_bf16) and the float32 GEMM with
float64 products of the same (bf16-valued) inputs: the dX = dY W and
dW = dY^T X products of the linear layers' backward (Algorithm 1, backward
pass at one layer), the forward product and the batched attention products.
Tolerance: rel 2e-2 for bf16-input GEMMs (float32 output is additionally held
to 1e-4 normwise)."""
import numpy as np
import pytest

from paper_2410_05985_amd import synthetic as S
import oracle as O
from tests.parity import compare

pytestmark = pytest.mark.gpu
torch = pytest.importorskip("torch")
from paper_2410_05985_amd import layup as LU  # noqa: E402

DEV = "cuda"


def bf16_tensor(shape, seed, std=1.0):
    x = torch.from_numpy(S.normal(shape, seed, std)).to(torch.bfloat16)
    return x


def as_f64(t):
    return t.float().cpu().numpy().astype(np.float64)


def run(layout, M, N, K, out_f32=True, bias=False, seed=0, ws=False):
    """layout: 'kk' (C = A B^T, forward), 'kn' (C = A B, dX), 'mn' (C = A^T B, dW)."""
    ak, bk = {"kk": (True, True), "kn": (True, False), "mn": (False, False)}[layout]
    A = bf16_tensor((M, K) if ak else (K, M), seed)
    B = bf16_tensor((N, K) if bk else (K, N), seed + 1)
    a64, b64 = as_f64(A), as_f64(B)
    ref = (a64 if ak else a64.T) @ (b64.T if bk else b64)
    bvec = None
    if bias:
        bvec = torch.from_numpy(S.normal((N,), seed + 2)).to(DEV)
        ref = ref + bvec.cpu().numpy().astype(np.float64)
    Ad, Bd = A.to(DEV), B.to(DEV)
    Cd = torch.empty((M, N), dtype=torch.float32 if out_f32 else torch.bfloat16, device=DEV)
    w = torch.empty(64 << 20, dtype=torch.uint8, device=DEV) if ws else None
    d = LU.gemm_desc(Ad, Bd, Cd, M, N, K, K if ak else M, K if bk else N, N, ak, bk, out_f32,
                     bias=bvec, workspace=w, workspace_bytes=(64 << 20) if ws else 0)
    LU.layup_gemm_bf16(d, torch.cuda.current_stream())
    torch.cuda.synchronize()
    return Cd.float().cpu().numpy().astype(np.float64), ref


@pytest.mark.parametrize("layout", ["kk", "kn", "mn"])
@pytest.mark.parametrize("M,N,K", [(64, 64, 64), (128, 128, 128), (256, 384, 192),
                                   (200, 136, 72), (1000, 520, 264), (8, 8, 8), (40, 24, 8),
                                   (128, 64, 1000)])
def test_gemm_layouts_and_ragged_shapes(layout, M, N, K):
    got, ref = run(layout, M, N, K, out_f32=True, seed=M + N + K)
    compare(got, ref, 2e-2, f"{layout} {M}x{N}x{K}")
    assert np.linalg.norm(got - ref) <= 1e-4 * np.linalg.norm(ref)


@pytest.mark.parametrize("layout", ["kk", "kn", "mn"])
def test_gemm_bf16_output_and_bias(layout):
    got, ref = run(layout, 320, 192, 136, out_f32=False, bias=True, seed=5)
    compare(got, ref, 2e-2, "bf16 out")
    # a bf16 result is the float32 result rounded once: within half a bf16 ulp
    assert np.all(np.abs(got - ref) <= 2.0 ** -8 * np.abs(ref) + 1e-3 * np.sqrt(np.mean(ref ** 2)))


@pytest.mark.parametrize("layout", ["mn", "kn"])
def test_gemm_split_k_deterministic(layout):
    """Few output tiles and a long K take the split-K path: float32 partials
    summed in a fixed order -- the result is reproducible bit for bit."""
    a, ref = run(layout, 256, 256, 8192, ws=True, seed=11)
    b, _ = run(layout, 256, 256, 8192, ws=True, seed=11)
    compare(a, ref, 2e-2, "split-K")
    assert np.linalg.norm(a - ref) <= 1e-4 * np.linalg.norm(ref)
    assert np.array_equal(a, b)


@pytest.mark.parametrize("layout", ["kn", "kk"])
def test_gemm_long_k_split(layout):
    """K >= 16384 with a float32 output (the tied head's dX over the
    vocabulary) takes the 256x256 tile with an 8-way split of K; ragged M, N
    and K, reproducible bit for bit."""
    a, ref = run(layout, 520, 264, 16400, ws=True, seed=13)
    b, _ = run(layout, 520, 264, 16400, ws=True, seed=13)
    compare(a, ref, 2e-2, "long-K split")
    assert np.linalg.norm(a - ref) <= 1e-4 * np.linalg.norm(ref)
    assert np.array_equal(a, b)


def test_gemm_split_k_unaligned_columns():
    """Split-K whose output rows are not a multiple of four floats (N = 130,
    k-major B): the partial sums take the per-column path, with the bias;
    reproducible bit for bit."""
    a, ref = run("kk", 200, 130, 16400, bias=True, ws=True, seed=19)
    b, _ = run("kk", 200, 130, 16400, bias=True, ws=True, seed=19)
    compare(a, ref, 2e-2, "split-K N=130")
    assert np.linalg.norm(a - ref) <= 1e-4 * np.linalg.norm(ref)
    assert np.array_equal(a, b)


@pytest.mark.parametrize("layout", ["kk", "kn", "mn"])
def test_gemm_degenerate_sizes(layout):
    """K = 0: C = bias (float32 and bf16 outputs, and the float32 GEMM), the
    row sums of A are 0, and the operands, never read, may be NULL.  M = 0 or
    N = 0: nothing is written."""
    ak, bk = {"kk": (True, True), "kn": (True, False), "mn": (False, False)}[layout]
    M, N = 72, 40
    bvec = torch.from_numpy(S.normal((N,), 3)).to(DEV)
    lda, ldb = (0 if ak else M), (0 if bk else N)
    s = torch.cuda.current_stream()
    for f32 in (True, False):
        C = torch.full((M, N), float("nan"), dtype=torch.float32 if f32 else torch.bfloat16, device=DEV)
        rs = torch.full((M,), float("nan"), dtype=torch.float32, device=DEV) if not ak else None
        d = LU.gemm_desc(None, None, C, M, N, 0, lda, ldb, N, ak, bk, f32, bias=bvec, a_rowsum=rs)
        LU.layup_gemm_bf16(d, s)
        torch.cuda.synchronize()
        want = bvec if f32 else bvec.to(torch.bfloat16)
        assert torch.equal(C, want.expand(M, N)), f32
        if rs is not None:
            assert torch.equal(rs, torch.zeros_like(rs))
    C = torch.full((M, N), float("nan"), dtype=torch.float32, device=DEV)
    LU.layup_gemm_f32(LU.gemm_desc(None, None, C, M, N, 0, lda, ldb, N, ak, bk, True, bias=bvec), s)
    torch.cuda.synchronize()
    assert torch.equal(C, bvec.expand(M, N))
    # M = 0 or N = 0: a sentinel output is left as it is
    A = bf16_tensor((M, 64) if ak else (64, M), 5).to(DEV)
    B = bf16_tensor((N, 64) if bk else (64, N), 6).to(DEV)
    sentinel = torch.full((M, N), 7.0, dtype=torch.float32, device=DEV)
    for m_, n_ in ((0, N), (M, 0)):
        d = LU.gemm_desc(A, B, sentinel, m_, n_, 64, 64 if ak else max(m_, 8), 64 if bk else max(n_, 8),
                         max(n_, 8), ak, bk, True)
        LU.layup_gemm_bf16(d, s)
    torch.cuda.synchronize()
    assert torch.equal(sentinel, torch.full_like(sentinel, 7.0))


def test_gemm_dw_many_tiles():
    """dW = dY^T X with at least 512 output tiles (the head's dW) takes the
    256x128 tile; ragged N and K."""
    got, ref = run("mn", 4096, 2200, 200, seed=17)
    compare(got, ref, 2e-2, "dW many tiles")
    assert np.linalg.norm(got - ref) <= 1e-4 * np.linalg.norm(ref)


@pytest.mark.parametrize("M,N,K,ws", [(256, 384, 192, False), (200, 136, 72, False),
                                      (256, 256, 8192, True), (520, 264, 3000, True),
                                      (2304, 768, 8192, True)])
def test_gemm_dw_bias_row_sums(M, N, K, ws):
    """dW = dY^T X with the bias gradient db = column sums of dY accumulated
    by the same kernel (a_rowsum), with and without split-K (ragged shapes):
    both against the oracle's linear-layer backward of the same bf16 values,
    db at 1e-4 (float32 sums of K terms)."""
    A = bf16_tensor((K, M), 41 + M, 0.5)   # dY, tokens x out
    B = bf16_tensor((K, N), 42 + N, 0.5)   # X, tokens x in
    dy, x = as_f64(A), as_f64(B)
    dw_ref, db_ref, _ = O.linear_bwd(dy, x, None, need_dx=False)
    Cd = torch.empty((M, N), dtype=torch.float32, device=DEV)
    db = torch.full((M,), float("nan"), dtype=torch.float32, device=DEV)
    w = torch.empty(64 << 20, dtype=torch.uint8, device=DEV) if ws else None
    d = LU.gemm_desc(A.to(DEV), B.to(DEV), Cd, M, N, K, M, N, N, False, False, True,
                     workspace=w, workspace_bytes=(64 << 20) if ws else 0, a_rowsum=db)
    LU.layup_gemm_bf16(d, torch.cuda.current_stream())
    torch.cuda.synchronize()
    compare(Cd.cpu().numpy(), dw_ref, 2e-2, f"dW {M}x{N}x{K}")
    compare(db.cpu().numpy(), db_ref, 1e-4, f"db {M}x{N}x{K}")


def test_gemm_row_sums_need_m_major_a():
    A = bf16_tensor((64, 64), 1).to(DEV)
    Cd = torch.empty((64, 64), dtype=torch.float32, device=DEV)
    db = torch.empty(64, dtype=torch.float32, device=DEV)
    d = LU.gemm_desc(A, A, Cd, 64, 64, 64, 64, 64, 64, True, False, True, a_rowsum=db)
    with pytest.raises(RuntimeError):
        LU.layup_gemm_bf16(d, torch.cuda.current_stream())


def test_gemm_batched_attention_strides():
    """Batched products over z = b*H + h with two-level operand offsets, as the
    attention core uses them: S_z = Q_h K_h^T from a packed qkv matrix."""
    B, T, H, dh = 2, 96, 3, 32
    d = H * dh
    qkv = bf16_tensor((B * T, 3 * d), 21)
    q64 = as_f64(qkv).reshape(B, T, 3, H, dh)
    ref = np.einsum("bihk,bjhk->bhij", q64[:, :, 0], q64[:, :, 1])
    dq = qkv.to(DEV)
    Sd = torch.empty((B, H, T, T), dtype=torch.float32, device=DEV)
    ptr = dq.data_ptr()
    d_ = LU.gemm_desc(ptr, ptr + 2 * d, Sd, T, T, dh, 3 * d, 3 * d, T, True, True, True,
                      batch=B * H, inner=H, a_strides=(T * 3 * d, dh), b_strides=(T * 3 * d, dh),
                      c_strides=(H * T * T, T * T))
    LU.layup_gemm_bf16(d_, torch.cuda.current_stream())
    torch.cuda.synchronize()
    compare(Sd.cpu().numpy(), ref, 2e-2, "batched scores")


@pytest.mark.parametrize("M,N,K,layout", [
    (8192, 768, 2304, "kn"),    # qkv dX, GPT-2-small
    (2304, 768, 8192, "mn"),    # qkv dW
    (8192, 3072, 768, "kn"),    # mlp-proj dX
    (768, 3072, 8192, "mn"),    # mlp-proj dW
    (768, 768, 8192, "mn"),     # attn-proj dW
    (8192, 2304, 768, "kk"),    # qkv forward
    (1024, 768, 50304, "kn"),   # head dX over the vocabulary (1024 of the 8192 rows)
    (50304, 768, 1024, "mn"),   # head dW (K = 1024 of the 8192 tokens)
    (8192, 1024, 4096, "kn"),   # GPT-2-medium fc dX
    (4096, 1024, 8192, "mn"),   # GPT-2-medium fc dW (split K)
    (8192, 8192, 2048, "kn"),   # 1.3B mlp-proj dX (256x256 tiles)
    (2048, 8192, 8192, "mn"),   # 1.3B mlp-proj dW (256x256 tiles, long K)
    (8192, 6144, 2048, "kk"),   # 1.3B qkv forward
])
def test_gemm_full_size_sampled(M, N, K, layout):
    """Full backward shapes of the GPT-2-small, GPT-2-medium and 1.3B blocks
    (8192 tokens), checked on 4096 sampled outputs, each an independent
    float64 dot product."""
    ak, bk = {"kk": (True, True), "kn": (True, False), "mn": (False, False)}[layout]
    A = bf16_tensor((M, K) if ak else (K, M), 31, 0.5)
    B = bf16_tensor((N, K) if bk else (K, N), 32, 0.5)
    Cd = torch.empty((M, N), dtype=torch.float32, device=DEV)
    w = torch.empty(64 << 20, dtype=torch.uint8, device=DEV)
    d = LU.gemm_desc(A.to(DEV), B.to(DEV), Cd, M, N, K, K if ak else M, K if bk else N, N, ak, bk,
                     True, workspace=w, workspace_bytes=64 << 20)
    LU.layup_gemm_bf16(d, torch.cuda.current_stream())
    torch.cuda.synchronize()
    rng = np.random.default_rng(M + N)
    mi, ni = rng.integers(0, M, 4096), rng.integers(0, N, 4096)
    a64, b64 = as_f64(A), as_f64(B)
    arows = a64[mi] if ak else a64[:, mi].T
    bcols = b64[ni] if bk else b64[:, ni].T
    ref = np.sum(arows * bcols, axis=1)
    got = Cd.cpu().numpy()[mi, ni].astype(np.float64)
    compare(got, ref, 2e-2, f"{M}x{N}x{K}")
    assert np.linalg.norm(got - ref) <= 1e-4 * np.linalg.norm(ref)


@pytest.mark.parametrize("layout", ["kk", "kn", "mn"])
def test_gemm_f32(layout):
    ak, bk = {"kk": (True, True), "kn": (True, False), "mn": (False, False)}[layout]
    M, N, K = 32, 10, 256
    A = S.normal((M, K) if ak else (K, M), 41)
    B = S.normal((N, K) if bk else (K, N), 42)
    ref = (A.astype(np.float64) if ak else A.T.astype(np.float64)) @ \
        (B.T.astype(np.float64) if bk else B.astype(np.float64))
    Cd = torch.empty((M, N), dtype=torch.float32, device=DEV)
    d = LU.gemm_desc(torch.from_numpy(A).to(DEV), torch.from_numpy(B).to(DEV), Cd, M, N, K,
                     K if ak else M, K if bk else N, N, ak, bk, True)
    LU.layup_gemm_f32(d, torch.cuda.current_stream())
    torch.cuda.synchronize()
    compare(Cd.cpu().numpy(), ref, 1e-5, "f32 gemm")
