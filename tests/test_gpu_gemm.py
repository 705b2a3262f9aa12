"""GPU parity of forge_gemm: every supported layout / epilogue, ragged shapes.

Integer-valued inputs in [-4, 4] are exact in bf16 and every partial sum stays
below 2^24, so fp32 accumulation is exact: fp32 outputs must match the exact
product bit for bit, bf16 outputs must equal its round-to-nearest-even.
Random-normal inputs check the large-tile paths against an fp64 product.
"""
import numpy as np
import pytest

import forge_inputs as fi
from gpu_util import rel_fro, dev_bf16, host_f64, banner

pytestmark = pytest.mark.gpu

KC, MC = 0, 1
STORE_BF16, RESID_BF16, ACC_F32, STORE_F32 = 0, 1, 2, 3
COMBOS = [(KC, KC, STORE_BF16), (KC, KC, RESID_BF16), (KC, KC, ACC_F32), (KC, KC, STORE_F32),
          (KC, MC, STORE_BF16), (KC, MC, RESID_BF16), (MC, MC, ACC_F32), (MC, MC, STORE_F32)]


def _operands(la, lb, M, N, K, rng, integer):
    def draw(shape):
        if integer:
            return rng.integers(-4, 5, size=shape).astype(np.float32)
        return rng.standard_normal(shape, dtype=np.float32)
    A = draw((M, K) if la == KC else (K, M))
    B = draw((N, K) if lb == KC else (K, N))
    return A, B


def run_gemm(la, lb, epi, M, N, K, seed=0, integer=True):
    import torch
    from paper_2609_13645_amd import _lib
    rng = np.random.default_rng(seed)
    A, B = _operands(la, lb, M, N, K, rng, integer)
    Ab, Bb = fi.to_bf16_bits(A), fi.to_bf16_bits(B)
    Al64 = fi.bf16_bits_to_f64(Ab).reshape(A.shape)
    Bl64 = fi.bf16_bits_to_f64(Bb).reshape(B.shape)
    Al64 = Al64 if la == KC else Al64.T
    Bl64 = Bl64.T if lb == KC else Bl64
    prod = Al64 @ Bl64
    dA, dB = dev_bf16(Ab), dev_bf16(Bb)
    R = None
    ref = prod.copy()
    if epi in (STORE_BF16, RESID_BF16):
        C = torch.empty((M, N), dtype=torch.bfloat16, device="cuda")
        if epi == RESID_BF16:
            rb = fi.to_bf16_bits(rng.integers(-8, 9, size=(M, N)).astype(np.float32) if integer
                                 else rng.standard_normal((M, N), dtype=np.float32))
            R = dev_bf16(rb)
            ref = ref + fi.bf16_bits_to_f64(rb)
    else:
        init = (rng.integers(-8, 9, size=(M, N)).astype(np.float32) if epi == ACC_F32
                else np.full((M, N), np.nan, np.float32))
        C = torch.from_numpy(init).cuda()
        if epi == ACC_F32:
            ref = ref + init
    _lib.forge_gemm(la, lb, epi, dA, dB, C, R, M, N, K, A.shape[1], B.shape[1], N,
                    N if R is not None else 0)
    torch.cuda.synchronize()
    return host_f64(C), ref


@pytest.mark.parametrize("la,lb,epi", COMBOS)
@pytest.mark.parametrize("M,N,K", [(64, 64, 64), (136, 200, 688), (264, 392, 40),
                                   (8, 8, 8), (520, 136, 1000)])
def test_gemm_integer_exact(la, lb, epi, M, N, K):
    banner(f"gemm int la={la} lb={lb} epi={epi} M={M} N={N} K={K}")
    got, ref = run_gemm(la, lb, epi, M, N, K, seed=M + N + K)
    if epi in (STORE_BF16, RESID_BF16):
        want = fi.bf16_bits_to_f64(fi.to_bf16_bits(ref.astype(np.float32)))
    else:
        want = ref
    assert np.array_equal(got, want)


@pytest.mark.parametrize("la,lb,epi", [(KC, KC, STORE_BF16), (KC, MC, STORE_BF16),
                                       (MC, MC, ACC_F32)])
@pytest.mark.parametrize("M,N,K", [(4096, 4096, 64), (4096, 2048, 72), (1024, 1536, 256),
                                   (4096, 6144, 64), (4096, 4096, 1000)])
def test_gemm_tile_paths_random(la, lb, epi, M, N, K):
    banner(f"gemm rand la={la} lb={lb} epi={epi} M={M} N={N} K={K}")
    got, ref = run_gemm(la, lb, epi, M, N, K, seed=7, integer=False)
    tol = 1e-2 if epi == STORE_BF16 else 1e-5
    assert rel_fro(got, ref) <= tol


@pytest.mark.parametrize("la,lb,epi", [(KC, MC, STORE_BF16), (MC, MC, ACC_F32), (MC, MC, STORE_F32)])
def test_gemm_large_tiles_long_k_integer_exact(la, lb, epi):
    """256 x 256 tiles over a long ragged reduction (K = 1000: 31 full
    32-deep stages and a partial one), exact in fp32."""
    M, N, K = 4096, 4096, 1000
    banner(f"gemm int big tiles la={la} lb={lb} epi={epi} K={K}")
    got, ref = run_gemm(la, lb, epi, M, N, K, seed=epi + 3)
    want = (fi.bf16_bits_to_f64(fi.to_bf16_bits(ref.astype(np.float32)))
            if epi in (STORE_BF16, RESID_BF16) else ref)
    assert np.array_equal(got, want)


@pytest.mark.parametrize("la,lb,epi", [(KC, KC, STORE_BF16), (KC, KC, RESID_BF16),
                                       (KC, MC, RESID_BF16), (MC, MC, STORE_F32)])
def test_gemm_large_tiles_ragged_n_integer_exact(la, lb, epi):
    """256 x 256 tiles (16 x 16 = 256 of them: one full round) whose last
    column of tiles ends in a half 16-wide block (N % 16 == 8), over a ragged
    reduction (K % 32 == 8): the paired 16-byte bf16 stores fall back to
    element stores at the edge."""
    M, N, K = 4096, 4008, 264
    banner(f"gemm int big tiles ragged N la={la} lb={lb} epi={epi}")
    got, ref = run_gemm(la, lb, epi, M, N, K, seed=epi + 11)
    want = (fi.bf16_bits_to_f64(fi.to_bf16_bits(ref.astype(np.float32)))
            if epi in (STORE_BF16, RESID_BF16) else ref)
    assert np.array_equal(got, want)


@pytest.mark.parametrize("la,lb,epi", [(KC, KC, STORE_BF16), (KC, KC, RESID_BF16),
                                       (KC, KC, STORE_F32), (KC, MC, STORE_BF16)])
def test_gemm_single_round_long_k_integer_exact(la, lb, epi):
    """One round of 256 x 256 tiles over a long reduction (the shape of the
    down projection and the gate/up data gradient): ragged M and N edges
    (M % 256 == 160, N % 16 == 8) and a ragged reduction (K % 32 == 8), exact
    in fp32."""
    M, N, K = 4000, 4008, 8200
    banner(f"gemm int single round long K la={la} lb={lb} epi={epi}")
    got, ref = run_gemm(la, lb, epi, M, N, K, seed=epi + 17)
    want = (fi.bf16_bits_to_f64(fi.to_bf16_bits(ref.astype(np.float32)))
            if epi in (STORE_BF16, RESID_BF16) else ref)
    assert np.array_equal(got, want)


@pytest.mark.parametrize("M,N,K", [(4096, 6144, 264), (4000, 6136, 200), (1280, 13312, 72),
                                   (4864, 6912, 40), (4096, 5896, 40)])
@pytest.mark.parametrize("epi", [STORE_BF16, RESID_BF16, ACC_F32, STORE_F32])
def test_gemm_split_last_round_integer_exact(M, N, K, epi):
    """Forward-layout products whose 256 x 256 tiles leave a last round at
    most half full (384 = 256 + 128, 260 = 256 + 4 and 513 = 2 * 256 + 1
    tiles): the whole rounds run as 256 x 256 tiles and the rest as 256 x 128
    halves in a second launch. Ragged M, N and K on the second shape (the
    last column of halves ends inside a 16-wide block); on the last shape the
    last half of the last column of tiles lies wholly past N (N % 256 = 8)
    and must store nothing. Exact in fp32."""
    banner(f"gemm int split last round M={M} N={N} K={K} epi={epi}")
    got, ref = run_gemm(KC, KC, epi, M, N, K, seed=M + N + K + epi)
    want = (fi.bf16_bits_to_f64(fi.to_bf16_bits(ref.astype(np.float32)))
            if epi in (STORE_BF16, RESID_BF16) else ref)
    assert np.array_equal(got, want)


def test_gemm_zero_k_and_empty():
    banner("gemm K=0 / empty")
    got, ref = run_gemm(KC, KC, ACC_F32, 64, 64, 0)
    assert np.array_equal(got, ref)
    got, ref = run_gemm(MC, MC, STORE_F32, 16, 24, 0)
    assert np.array_equal(got, np.zeros_like(ref))


@pytest.mark.parametrize("epi", [STORE_BF16, RESID_BF16, ACC_F32, STORE_F32])
def test_gemm_256x192_tiles_integer_exact(epi):
    """A K-contiguous product whose 256 x 256 tiles would leave the last wave
    of workgroups half empty runs on 256 x 192 tiles; N = 6136 also leaves a
    ragged last tile column."""
    M, N, K = 4096, 6136, 40
    banner(f"gemm 256x192 tiles epi={epi}")
    got, ref = run_gemm(KC, KC, epi, M, N, K, seed=epi + 11)
    want = (fi.bf16_bits_to_f64(fi.to_bf16_bits(ref.astype(np.float32)))
            if epi in (STORE_BF16, RESID_BF16) else ref)
    assert np.array_equal(got, want)


GROUP_SIZES = [0, 37, 256, 1, 300, 0, 129, 8, 513]


@pytest.mark.parametrize("lb", [KC, MC])
@pytest.mark.parametrize("N,K", [(136, 64), (264, 200)])
def test_grouped_rows_integer_exact(lb, N, K):
    """Per-group products over expert-major rows, ragged and empty groups;
    rows past the last offset are never written."""
    import torch
    from paper_2609_13645_amd import _lib
    banner(f"grouped rows lb={lb} N={N} K={K}")
    rng = np.random.default_rng(N + K + lb)
    off = np.concatenate([[0], np.cumsum(GROUP_SIZES)]).astype(np.int32)
    G, rows = len(GROUP_SIZES), int(off[-1]) + 40          # a slack of unused rows
    A = rng.integers(-4, 5, size=(rows, K)).astype(np.float32)
    B = rng.integers(-4, 5, size=(G, N, K) if lb == KC else (G, K, N)).astype(np.float32)
    C = torch.full((rows, N), float("nan"), dtype=torch.bfloat16, device="cuda")
    _lib.forge_gemm_grouped_rows(lb, dev_bf16(fi.to_bf16_bits(A)), dev_bf16(fi.to_bf16_bits(B)),
                                 C, torch.from_numpy(off).cuda(), G, rows, N, K, K,
                                 K if lb == KC else N, N, N * K)
    torch.cuda.synchronize()
    got = host_f64(C)
    for e in range(G):
        r0, r1 = off[e], off[e + 1]
        Be = B[e].T if lb == KC else B[e]
        want = A[r0:r1].astype(np.float64) @ Be
        assert np.array_equal(got[r0:r1], fi.bf16_bits_to_f64(fi.to_bf16_bits(want.astype(np.float32)))), e
    assert np.all(np.isnan(got[off[-1]:]))


@pytest.mark.parametrize("M,N", [(64, 136), (264, 128)])
def test_grouped_wgrad_integer_exact(M, N):
    """C_e += A_e^T B_e over each group's rows; empty groups leave C_e as is."""
    import torch
    from paper_2609_13645_amd import _lib
    banner(f"grouped wgrad M={M} N={N}")
    rng = np.random.default_rng(M * N)
    off = np.concatenate([[0], np.cumsum(GROUP_SIZES)]).astype(np.int32)
    G, rows = len(GROUP_SIZES), int(off[-1])
    A = rng.integers(-4, 5, size=(rows, M)).astype(np.float32)
    B = rng.integers(-4, 5, size=(rows, N)).astype(np.float32)
    init = rng.integers(-8, 9, size=(G, M, N)).astype(np.float32)
    C = torch.from_numpy(init).cuda()
    _lib.forge_gemm_grouped_wgrad(dev_bf16(fi.to_bf16_bits(A)), dev_bf16(fi.to_bf16_bits(B)), C,
                                  torch.from_numpy(off).cuda(), G, M, N, M, N, N, M * N)
    torch.cuda.synchronize()
    got = host_f64(C)
    for e in range(G):
        r0, r1 = off[e], off[e + 1]
        want = init[e] + A[r0:r1].T.astype(np.float64) @ B[r0:r1]
        assert np.array_equal(got[e], want), e
