"""Single kernels of the HIP path against CPU references (through metro_ops.h).

Weight packing: bit-exact against the operand-order layout written out.
GEMM: every epilogue, in the skinny (M <= 64) and tiled (M > 64) kernels,
with ragged M, K padded to 128 and N covering several tiles plus a tail.
The reference products are exact-value float64 sums of the same bf16
operands; the GPU accumulates in fp32, so the bound is a few fp32 ulps of
the row's absolute sum.
"""

import numpy as np
import pytest

from oracle import bf16_bits_to_f64, bf16_round, greedy_argmax, rms_norm, swiglu
from paper_2411_03519_amd import synth

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")


@pytest.fixture(scope="module")
def metro():
    if not torch.cuda.is_available():
        pytest.skip("no HIP device")
    from paper_2411_03519_amd import metro as m
    return m


def dev_u16(a):
    return torch.from_numpy(np.ascontiguousarray(a.view(np.int16))).cuda()


def rand_bf16(rng, shape, scale=1.0):
    return synth.f32_to_bf16_bits(rng.standard_normal(shape).astype(np.float32) * np.float32(scale))


def packed_layout(W, K, Kp):
    """The operand-order layout of metro_ops.h written out element by element:
    W[n, k] (k < K, else 0) at ((n/16 * Kp/32 + k/32) * 64 + n%16 + 16*((k/8)%4)) * 8 + k%8."""
    N = W.shape[0]
    n, k = np.meshgrid(np.arange(N), np.arange(Kp), indexing="ij")
    idx = ((n // 16 * (Kp // 32) + k // 32) * 64 + n % 16 + 16 * ((k // 8) % 4)) * 8 + k % 8
    out = np.zeros(N * Kp, np.uint16)
    vals = np.zeros((N, Kp), np.uint16)
    vals[:, :K] = W[:, :K]
    out[idx.ravel()] = vals.ravel()
    return out


def pack_dev(metro, W, K, Kp):
    """Device copy of row-major W [N, ld] in the GEMM's packed layout."""
    N, ld = W.shape
    out = torch.zeros(N * Kp, dtype=torch.int16, device="cuda")
    metro.op_pack_weight(dev_u16(W), ld, N, K, Kp, out)
    return out


@pytest.mark.parametrize("N,K,ld,Kp", [(16, 128, 128, 128), (48, 200, 208, 256), (96, 688, 700, 768)])
def test_pack_weight_layout(metro, N, K, ld, Kp):
    rng = np.random.default_rng(N + K)
    W = rng.integers(0, 1 << 16, size=(N, ld), dtype=np.uint16)
    got = pack_dev(metro, W, K, Kp)
    torch.cuda.synchronize()
    np.testing.assert_array_equal(got.cpu().numpy().view(np.uint16), packed_layout(W, K, Kp))


def test_pack_weight_rejects_bad_shapes(metro):
    W = torch.zeros(64 * 256, dtype=torch.int16, device="cuda")
    out = torch.zeros(64 * 256, dtype=torch.int16, device="cuda")
    for N, K, ld, Kp in [(24, 128, 128, 128), (16, 100, 128, 120), (16, 300, 300, 256), (16, 128, 64, 128)]:
        with pytest.raises(metro.MetroError):
            metro.op_pack_weight(W, ld, N, K, Kp, out)


# (M, K, N): decode kernel at M <= 64; above it the tiled kernel with 128 x 128
# blocks (narrow products up to 1000 rows, wide ones up to 192 while they fit
# the CUs), 256 x 128 blocks (wide products otherwise, up to 256 rows) or 256 x
# 256 blocks, with or without a k split (plan_gemm); the 256-row tiles split
# only the tiles of the last round of workgroups (on 256 CUs) when given a
# workspace
GEMM_CASES = [(1, 256, 64), (7, 640, 96), (16, 256, 32), (25, 4096, 512), (33, 768, 160), (64, 384, 1376),
              (65, 256, 160), (200, 1152, 416), (129, 128, 96), (300, 4096, 256), (1100, 384, 160),
              (200, 256, 16384), (70, 128, 65536),
              (129, 1024, 512),      # 128 x 128 tiles; no k split (slice sums would pass half the weights)
              (80, 4096, 4096),      # 32 tiles of 128 x 128, with a workspace 8 k slices (one round of 256)
              (200, 4096, 4096),     # 64 tiles of 128 x 128, with a workspace 4 k slices
              (65, 1024, 160),       # 2 ragged tiles x 2 k slices: fewer workgroups than XCDs
              (150, 2048, 416),      # 8 ragged tiles x 2 k slices
              (200, 4096, 5120),     # narrow, 80 tiles of 128 x 128 x 2 slices -> 40 of 256 x 128 x 4 slices
              (300, 4096, 16384),    # 256 x 256 tiles, 2 k slices with a workspace
              (600, 2048, 288),      # 128 x 128 tiles, ragged in both M and N
              (1300, 2048, 4096),    # 256 x 256 tiles, 96 in one partial round: with a workspace 2 k slices each
              (4300, 1024, 4000),    # 272 ragged 256 x 256 tiles: the 16 past the first round in 8 k slices
              (129, 256, 20480),     # wide: 160 tiles of 256 x 128 over two row blocks
              (100, 256, 69632),     # wide: 272 tiles of 256 x 128, the 16 past the first round in 2 k slices
              (200, 256, 16384),     # wide: 128 tiles of 256 x 128, with a workspace 2 k slices each
              (90, 128, 57344),      # wide: 224 tiles of 256 x 128 (70B gate/up-sized, one round)
              (128, 4096, 6144),     # 48 tiles of 128 x 128 x 4 k slices (8B QKV-sized)
              (256, 4096, 4096),     # 64 tiles of 128 x 128 x 4 k slices
              (129, 2048, 1056),     # ragged N: 18 tiles of 128 x 128, the last 32 rows of W past a 128 block
              (250, 512, 288)]       # ragged in M and N, 128 x 128 tiles


@pytest.mark.parametrize("M,K,N", GEMM_CASES + [(25, 14336, 512), (3, 1024, 4096)])
@pytest.mark.parametrize("epi", [0, 1])
@pytest.mark.parametrize("split", [False, True])
def test_gemm_f32_epilogues(metro, M, K, N, epi, split):
    print(f"gemm M={M} K={K} N={N} epi={epi} split={split}", flush=True)
    rng = np.random.default_rng(M * 7 + K + N + epi)
    Kp = (K + 127) // 128 * 128
    X = np.zeros((M, Kp), np.uint16)
    W = np.zeros((N, Kp), np.uint16)
    X[:, :K] = rand_bf16(rng, (M, K))
    W[:, :K] = rand_bf16(rng, (N, K), 0.05)
    ref = bf16_bits_to_f64(X) @ bf16_bits_to_f64(W).T
    ldo = N + 4
    init = rng.standard_normal((M, ldo)).astype(np.float32)
    out = torch.from_numpy(init.copy()).cuda()
    ws = torch.full((8, M, N), float("nan"), device="cuda") if split else None
    metro.op_gemm(dev_u16(X), pack_dev(metro, W, Kp, Kp), M, N, Kp, epi, out, ldo, workspace=ws)
    torch.cuda.synchronize()
    got = out.cpu().numpy().astype(np.float64)
    want = ref + (init[:, :N] if epi == 1 else 0.0)
    bound = 1e-5 * (np.abs(bf16_bits_to_f64(X)) @ np.abs(bf16_bits_to_f64(W)).T) + 1e-6
    assert np.all(np.abs(got[:, :N] - want) <= bound), np.max(np.abs(got[:, :N] - want) - bound)
    np.testing.assert_array_equal(got[:, N:], init[:, N:])  # padding columns untouched


@pytest.mark.parametrize("M,K,F", [(3, 256, 688), (25, 256, 48), (64, 512, 112), (96, 256, 688), (130, 384, 80),
                                   (150, 128, 8192), (25, 128, 14336), (40, 128, 14336), (300, 128, 14336),
                                   (100, 256, 14336), (180, 128, 16384),
                                   (300, 256, 8192),     # 128 tiles of 256 x 256: with a workspace 2 k slices each
                                   (1300, 256, 2048),    # 96 ragged tiles: with a workspace 2 k slices each
                                   (90, 128, 28672),     # 224 tiles of 256 x 128 (70B gate/up-sized)
                                   (200, 256, 14336)])   # 224 tiles of 256 x 128 over two row blocks
@pytest.mark.parametrize("split", [False, True])
def test_gemm_swiglu_epilogue(metro, M, K, F, split):
    print(f"swiglu M={M} K={K} F={F} split={split}", flush=True)
    rng = np.random.default_rng(M + K + F)
    X = rand_bf16(rng, (M, K))
    Wg = rand_bf16(rng, (F, K), 0.1)
    Wu = rand_bf16(rng, (F, K), 0.1)
    packed = np.zeros((2 * F, K), np.uint16)  # blocks of 8 gate rows, then the 8 matching up rows
    for b in range(F // 8):
        packed[16 * b:16 * b + 8] = Wg[8 * b:8 * b + 8]
        packed[16 * b + 8:16 * b + 16] = Wu[8 * b:8 * b + 8]
    ldo = (F + 127) // 128 * 128
    out = torch.zeros((M, ldo), dtype=torch.int16, device="cuda")
    ws = torch.full((8, M, 2 * F), float("nan"), device="cuda") if split else None
    metro.op_gemm(dev_u16(X), pack_dev(metro, packed, K, K), M, 2 * F, K, 2, out, ldo, workspace=ws)
    torch.cuda.synchronize()
    got = bf16_bits_to_f64(out.cpu().numpy().view(np.uint16))
    xf, wg, wu = bf16_bits_to_f64(X), bf16_bits_to_f64(Wg), bf16_bits_to_f64(Wu)
    g, u = xf @ wg.T, xf @ wu.T
    want = bf16_round(swiglu(g, u))
    # fp32 accumulation error of g and u (bounded by the sums of |products|),
    # carried through silu(g)*u, plus one bf16 ulp of the rounding
    err_g = 1e-5 * (np.abs(xf) @ np.abs(wg).T)
    err_u = 1e-5 * (np.abs(xf) @ np.abs(wu).T)
    prop = 1.1 * np.abs(u) * err_g + np.abs(swiglu(g, np.ones_like(g))) * err_u
    big = np.maximum(np.abs(want), np.abs(got[:, :F]))
    ulp = np.ldexp(1.0, np.frexp(big)[1] - 8)
    assert np.all(np.abs(got[:, :F] - want) <= ulp + 2 * prop + 1e-30)
    assert np.mean(got[:, :F] == want) > 0.98
    assert not np.any(got[:, F:])


def test_rmsnorm(metro):
    rng = np.random.default_rng(5)
    rows, d = 37, 4096
    x = (rng.standard_normal((rows, d)) * 3).astype(np.float32)
    g = rand_bf16(rng, (d,), 1.0)
    h = torch.zeros((rows, d), dtype=torch.int16, device="cuda")
    metro.op_rmsnorm(torch.from_numpy(x).cuda(), dev_u16(g), 1e-5, h, rows, d)
    torch.cuda.synchronize()
    got = bf16_bits_to_f64(h.cpu().numpy().view(np.uint16))
    want = bf16_round(rms_norm(x.astype(np.float64), bf16_bits_to_f64(g), 1e-5))
    ulp = np.ldexp(1.0, np.frexp(np.abs(want))[1] - 8)
    assert np.all(np.abs(got - want) <= ulp)
    assert np.mean(got == want) > 0.99


def test_argmax_lowest_index_and_nan(metro):
    rng = np.random.default_rng(6)
    V = 128256
    L = rng.standard_normal((6, V)).astype(np.float32)
    L[1, [5, 77, 128000]] = 50.0          # tie: lowest index wins
    L[2, :] = -3.0                        # all equal
    L[3, 100] = np.nan
    L[3, 64000] = 40.0
    L[4, :] = np.nan                      # no value left
    L[5, V - 1] = 99.0                    # last element
    out = torch.zeros(6, dtype=torch.int32, device="cuda")
    metro.op_argmax(torch.from_numpy(L).cuda(), 6, V, out)
    torch.cuda.synchronize()
    got = out.cpu().numpy()
    want = greedy_argmax(np.where(np.isnan(L), -np.inf, L))
    want[4] = -1
    np.testing.assert_array_equal(got, want)


@pytest.mark.parametrize("V", [32, 4096, 4 * 8 * 1024 + 36])
def test_argmax_short_and_ragged_rows(metro, V):
    # rows shorter than one batch of loads per thread, and one that ends a few
    # float4 into a second batch; ties planted across threads and batches
    rng = np.random.default_rng(V)
    L = rng.standard_normal((3, V)).astype(np.float32)
    L[0, [V - 1, 3]] = 30.0
    L[1, V // 2:] = np.nan
    L[2, [V - 4, V - 8]] = 7.0
    out = torch.zeros(3, dtype=torch.int32, device="cuda")
    metro.op_argmax(torch.from_numpy(L).cuda(), 3, V, out)
    torch.cuda.synchronize()
    want = greedy_argmax(np.where(np.isnan(L), -np.inf, L))
    np.testing.assert_array_equal(out.cpu().numpy(), want)


# One shape per kernel kind and epilogue: decode kernel with 1, 2 and 4
# activation tiles and 2, 4 and 7 row tiles per wave, 128 x 128, 256 x 128 and
# 256 x 256 tiles, k slices, a split last round, SwiGLU.
REPEAT_CASES = [(7, 4096, 6144, 0, True), (25, 4096, 4096, 1, True), (25, 4096, 28672, 2, False),
                (60, 14336, 4096, 1, True), (128, 4096, 4096, 1, True), (128, 4096, 28672, 2, False),
                (200, 4096, 10240, 0, True), (1300, 2048, 4096, 1, True), (2600, 4096, 6144, 0, False)]


def test_gemm_repeated_launches_are_bitwise_stable(metro):
    """Every kernel kind gives the same bits launch after launch, also when
    other GEMMs run in between (a result that depended on when the matrix
    pipeline drained, or on a race between waves, would differ from launch to
    launch), and its first result is within the fp32 bound of the exact one."""
    rng = np.random.default_rng(77)
    cases = []
    for M, K, N, epi, split in REPEAT_CASES:
        X = rand_bf16(rng, (M, K))
        W = rand_bf16(rng, (N, K), 0.05)
        swig = epi == 2
        ldo = N // 2 if swig else N
        out = (torch.zeros((M, ldo), dtype=torch.int16, device="cuda") if swig
               else torch.zeros((M, ldo), device="cuda"))
        ws = torch.full((8, M, N), float("nan"), device="cuda") if split else None
        cases.append((M, K, N, epi, dev_u16(X), pack_dev(metro, W, K, K), out, ws, X, W))
    first = [None] * len(cases)
    for rep in range(24):
        order = range(len(cases)) if rep % 2 == 0 else reversed(range(len(cases)))
        for i in order:
            M, K, N, epi, Xd, Wd, out, ws, X, W = cases[i]
            if epi == 1:
                out.zero_()
            metro.op_gemm(Xd, Wd, M, N, K, epi, out, out.shape[1], workspace=ws)
        torch.cuda.synchronize()
        for i, c in enumerate(cases):
            got = c[6].cpu().numpy().copy()
            if first[i] is None:
                first[i] = got
                M, K, N, epi, X, W = c[0], c[1], c[2], c[3], c[8], c[9]
                if epi != 2:
                    ref = bf16_bits_to_f64(X) @ bf16_bits_to_f64(W).T
                    bound = 1e-5 * (np.abs(bf16_bits_to_f64(X)) @ np.abs(bf16_bits_to_f64(W)).T) + 1e-6
                    assert np.all(np.abs(got.astype(np.float64) - ref) <= bound), f"case {i}"
            else:
                np.testing.assert_array_equal(got, first[i], err_msg=f"case {c[:5]} launch {rep}")
