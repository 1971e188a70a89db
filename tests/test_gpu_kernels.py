"""Kernel-level parity of the HIP GEMM and shared-prefix attention against CPU references."""
import numpy as np
import pytest
import torch

import oracle
import paper_2606_09937_amd as rk
from gpu_util import log

pytestmark = pytest.mark.gpu
DEV = "cuda"


def _rand(shape, dtype, seed, std=1.0):
    g = torch.Generator(device="cpu").manual_seed(seed)
    return (std * torch.randn(*shape, generator=g)).to(dtype)


@pytest.mark.parametrize("dtype", [torch.bfloat16, torch.float32], ids=["bf16", "f32"])
@pytest.mark.parametrize("M,N,K,splits", [
    (1, 64, 64, 0), (64, 100, 688, 0), (100, 200, 256, 1), (128, 192, 4096, 0),
    (300, 136, 128, 3), (513, 264, 512, 0), (77, 64, 1000, 5),
    # 256 x 256 tiles (512 rows and more): ragged rows, columns and K, forced splits
    (777, 700, 1000, 3), (1024, 512, 2048, 0), (2048, 1536, 4104, 0),
    # one row tile: the 7B projections at 128 rows with the planner's tile width and split count
    (128, 4096, 14336, 0), (128, 4096, 4096, 0), (128, 6144, 4096, 0),
    # the planner's 256- and 192-column weight tiles (ragged N and K, two row tiles)
    (130, 14376, 1000, 0), (70, 6016, 4104, 0),
    # the planner's 256 x 256 tiles over K splits at 512 and 1024 rows (3 and 4 splits)
    (1024, 4608, 3584, 0), (512, 6144, 4096, 0),
    # short K loops of the 128-row kernel's ring (3 slots): splits of 1, 2 and 3 stages, a partial last one
    (128, 4096, 64, 1), (128, 4096, 136, 2), (128, 4096, 192, 1), (128, 4096, 200, 2),
])
def test_gemm_matches_fp64(dtype, M, N, K, splits):
    log(f"gemm {dtype} M={M} N={N} K={K} splits={splits}")
    A = _rand((M, K), torch.float32, 1 + M, 0.5)     # activations are fp32 in every mode
    W = _rand((N, K), dtype, 2 + N, 0.05)
    if dtype == torch.bfloat16:
        # bf16 models feed the projection the hi/lo bf16 planes of the fp32 activation (RNE split).
        a_hi = A.to(torch.bfloat16)
        a_lo = (A - a_hi.float()).to(torch.bfloat16)
        A = a_hi.float() + a_lo.float()                # the value the planes carry
        P = rk.rksc_test_gemm((a_hi.to(DEV), a_lo.to(DEV)), W.to(DEV), splits=splits)
    else:
        P = rk.rksc_test_gemm(A.to(DEV), W.to(DEV), splits=splits)
    torch.cuda.synchronize()
    if splits:
        # a split never gets less than one K tile, so tiny K can use fewer splits than asked
        assert 1 <= P.shape[0] <= splits
    got = P.double().sum(0).cpu().numpy()
    a = A.double().numpy()
    w = W.double().numpy()
    ref = a @ w.T
    # fp32-level accuracy in both modes (bf16 weights meet a hi+lo split of A)
    bound = 1e-5 * (np.abs(a) @ np.abs(w).T) + 1e-7
    err = np.abs(got - ref)
    assert (err <= bound).all(), f"max err {err.max():.3e} at {np.unravel_index(err.argmax(), err.shape)}"


@pytest.mark.parametrize("M,N,K,splits", [
    (1, 16, 32, 0), (100, 200, 256, 0), (300, 700, 1000, 0), (256, 256, 8, 0), (513, 260, 4104, 3),
    (777, 513, 1000, 5), (1024, 1024, 2048, 0), (260, 1030, 3000, 8),
])
def test_gemm_wide_tiles_match_fp64(M, N, K, splits):
    """The 256 x 256-tile kernel (the verify pass's choice for projections with many rows), forced on
    ragged rows, columns and K (K % 32 != 0 included) and on forced K splits."""
    log(f"gemm wide M={M} N={N} K={K} splits={splits}")
    A = _rand((M, K), torch.float32, 11 + M, 0.5)
    W = _rand((N, K), torch.bfloat16, 12 + N, 0.05)
    a_hi = A.to(torch.bfloat16)
    a_lo = (A - a_hi.float()).to(torch.bfloat16)
    A = a_hi.float() + a_lo.float()
    P = rk.rksc_test_gemm((a_hi.to(DEV), a_lo.to(DEV)), W.to(DEV), splits=splits, kind=1)
    torch.cuda.synchronize()
    if splits:
        assert 1 <= P.shape[0] <= splits
    got = P.double().sum(0).cpu().numpy()
    a, w = A.double().numpy(), W.double().numpy()
    bound = 1e-5 * (np.abs(a) @ np.abs(w).T) + 1e-7
    err = np.abs(got - a @ w.T)
    assert (err <= bound).all(), f"max err {err.max():.3e} at {np.unravel_index(err.argmax(), err.shape)}"


@pytest.mark.parametrize("M,N,K,kind", [
    (1, 16, 32, 2), (3, 4, 8, 2), (8, 260, 504, 2), (16, 1000, 2048, 2), (5, 6144, 4096, 2),
    (8, 4096, 14336, 2), (13, 1028, 4104, 2), (16, 200, 20000, 2), (8, 28672, 4096, -1), (7, 4096, 14336, -1),
    # two 16-row activation blocks (17 to 32 rows): ragged rows, N and K, the 7B shapes
    (17, 1000, 2048, 2), (20, 260, 1000, 2), (24, 1028, 4104, 2), (32, 6144, 4096, 2), (32, 28672, 4096, -1),
    (29, 4096, 14336, 2), (17, 16384, 1000, -1),
])
def test_gemm_skinny_matches_fp64(M, N, K, kind):
    """The weight-streaming kernel for at most 32 rows (a decode step's projections), forced and as
    the planner's choice: ragged N (a partial last 16-row weight tile), K not a multiple of 512, one
    to eight K splits of 2048, the 4096-wide splits of a K above 16384 (at most 16 rows), and two
    16-row activation blocks from 17 rows."""
    log(f"gemm skinny M={M} N={N} K={K} kind={kind}")
    A = _rand((M, K), torch.float32, 21 + M, 0.5)
    W = _rand((N, K), torch.bfloat16, 22 + N, 0.05)
    a_hi = A.to(torch.bfloat16)
    a_lo = (A - a_hi.float()).to(torch.bfloat16)
    A = a_hi.float() + a_lo.float()
    P = rk.rksc_test_gemm((a_hi.to(DEV), a_lo.to(DEV)), W.to(DEV), kind=kind)
    torch.cuda.synchronize()
    per_split = 2048 if -(-K // 2048) <= 8 else 4096
    assert P.shape[0] == -(-K // per_split)
    got = P.double().sum(0).cpu().numpy()
    a, w = A.double().numpy(), W.double().numpy()
    bound = 1e-5 * (np.abs(a) @ np.abs(w).T) + 1e-7
    err = np.abs(got - a @ w.T)
    assert (err <= bound).all(), f"max err {err.max():.3e} at {np.unravel_index(err.argmax(), err.shape)}"


@pytest.mark.parametrize("M,N,K,splits,kind,live,s", [
    # 256 x 256 tiles: a live set that ends inside a row tile, inside a wave's 64 rows, on a tile edge
    (1024, 700, 1000, 3, 1, 3, 128), (1024, 4608, 3584, 0, -1, 5, 128), (1024, 512, 2048, 0, 1, 1, 200),
    (8192, 4096, 14336, 0, -1, 7, 256), (8192, 1024, 4096, 2, 1, 31, 256),
    # 128-row tiles: partial waves and tiles
    (1024, 512, 2048, 0, 0, 2, 128), (128, 4096, 4096, 0, -1, 3, 16), (128, 6144, 4096, 0, 0, 1, 5),
    (2048, 1536, 4104, 0, 0, 9, 100),
    # the weight stream of a decode step
    (32, 28672, 4096, 0, -1, 5, 1), (16, 4096, 14336, 0, 2, 11, 1), (32, 1028, 4104, 0, 2, 17, 1),
])
def test_gemm_live_rows_match_fp64(M, N, K, splits, kind, live, s):
    """Projections after branch exits: the plan of an M-row call with only live * s rows live
    (a control block in device memory, as the verify pass keeps it). Live rows match fp64
    (sampled at the largest shapes); rows past the live ones are not written."""
    log(f"gemm live M={M} N={N} K={K} splits={splits} kind={kind} live={live}x{s}")
    A = _rand((M, K), torch.float32, 31 + M, 0.5)
    W = _rand((N, K), torch.bfloat16, 32 + N, 0.05)
    a_hi = A.to(torch.bfloat16)
    a_lo = (A - a_hi.float()).to(torch.bfloat16)
    A = a_hi.float() + a_lo.float()
    P = torch.full((8, M, N), float("nan"), dtype=torch.float32, device=DEV)
    used = rk.rksc_test_gemm_live((a_hi.to(DEV), a_lo.to(DEV)), W.to(DEV), live, s, P, splits=splits, kind=kind)
    torch.cuda.synchronize()
    rows = live * s
    Pc = P[:used].cpu()
    assert torch.isnan(Pc[:, rows:]).all(), "rows past the live set were written"
    assert not torch.isnan(Pc[:, :rows]).any(), "a live row was not written"
    sample = np.arange(rows) if rows * N * K <= 4e9 else np.unique(np.r_[np.arange(0, rows, 37), rows - 1])
    got = Pc[:, sample].double().sum(0).numpy()
    a, w = A[sample].double().numpy(), W.double().numpy()
    bound = 1e-5 * (np.abs(a) @ np.abs(w).T) + 1e-7
    err = np.abs(got - a @ w.T)
    assert (err <= bound).all(), f"max err {err.max():.3e} at {np.unravel_index(err.argmax(), err.shape)}"


@pytest.mark.parametrize("kind", [1, 0])
def test_gemm_row_offsets_past_2_31(kind):
    """Both dense kernels where row * K passes 2^31 elements (150000 rows x 14336, the 7B down
    projection's K; the planner takes the 256 x 256 tiles for such row counts at the full width):
    sampled rows on both sides of the boundary match fp64."""
    M, N, K = 150000, 256, 14336
    assert (M - 1) * K >= 2 ** 31
    assert rk.rksc_test_gemm_plan(153600, 4096, K)["kind"] == 1
    assert rk.rksc_test_gemm_plan(M, N, K, kind=kind)["kind"] == kind
    log(f"gemm offsets kind={kind} M={M} N={N} K={K}")
    g = torch.Generator(device=DEV).manual_seed(5)
    a_hi = torch.randn((M, K), generator=g, device=DEV, dtype=torch.bfloat16)
    a_lo = torch.randn((M, K), generator=g, device=DEV, dtype=torch.bfloat16) * (2.0 ** -9)
    W = (torch.randn((N, K), generator=g, device=DEV, dtype=torch.float32) * 0.05).to(torch.bfloat16)
    P = rk.rksc_test_gemm((a_hi, a_lo), W, kind=kind)
    torch.cuda.synchronize()
    first_past = -(-(2 ** 31) // K)
    rows = np.unique(np.r_[0, 1, 255, 256, first_past - 3, first_past - 1, first_past, first_past + 1,
                           np.arange(first_past + 2, M, 97), M - 2, M - 1])
    idx = torch.from_numpy(rows).to(DEV)
    got = P[:, idx].double().sum(0).cpu().numpy()
    a = (a_hi[idx].double() + a_lo[idx].double()).cpu().numpy()
    w = W.double().cpu().numpy()
    bound = 1e-5 * (np.abs(a) @ np.abs(w).T) + 1e-7
    err = np.abs(got - a @ w.T)
    assert (err <= bound).all(), f"max err {err.max():.3e} at row {rows[np.unravel_index(err.argmax(), err.shape)[0]]}"
    del a_hi, a_lo, P


@pytest.mark.parametrize("M,F,K,fused", [
    (777, 712, 1000, 1), (1024, 2048, 1024, 1), (300, 136, 4104, 1), (4096, 1792, 4096, 1),
    (513, 264, 512, 0), (128, 1024, 4096, 0),
])
def test_gate_up_swiglu_matches_fp64(M, F, K, fused):
    """The gate|up projection with its SwiGLU: the 256 x 256 kernel with the SwiGLU in its epilogue
    (ragged rows, F not a multiple of its 128-column half tiles, ragged K) and the split path."""
    log(f"gate_up swiglu M={M} F={F} K={K} fused={fused}")
    A = _rand((M, K), torch.float32, 41 + M, 0.5)
    W = _rand((2 * F, K), torch.bfloat16, 42 + F, 0.05)
    a_hi = A.to(torch.bfloat16)
    a_lo = (A - a_hi.float()).to(torch.bfloat16)
    A = a_hi.float() + a_lo.float()
    got = rk.rksc_test_gate_up_swiglu((a_hi.to(DEV), a_lo.to(DEV)), W.to(DEV), bool(fused))
    torch.cuda.synchronize()
    got = got.double().cpu().numpy()
    a, w = A.double().numpy(), W.double().numpy()
    gu = a @ w.T
    g, u = gu[:, :F], gu[:, F:]
    sig = 1.0 / (1.0 + np.exp(-g))
    ref = g * sig * u
    eb = 1e-5 * (np.abs(a) @ np.abs(w).T) + 1e-7
    dsilu = np.abs(sig * (1 + g * (1 - sig)))
    bound = dsilu * eb[:, :F] * np.abs(u) + np.abs(g * sig) * eb[:, F:] + 1e-6 * np.abs(ref) + 1e-7
    err = np.abs(got - ref)
    assert (err <= bound).all(), f"max err {err.max():.3e} at {np.unravel_index(err.argmax(), err.shape)}"


def _attention_cases():
    """bf16 at every shape; fp32 (the plain per-thread kernel) only where it finishes quickly."""
    shapes = [
        (1, 0, 1, 4, 4, 64), (2, 37, 16, 8, 2, 64), (3, 130, 70, 28, 4, 128),
        (1, 1024, 128, 32, 8, 128), (2, 64, 200, 4, 4, 128), (4, 64, 16, 4, 4, 64),
        # fewer than 64 query rows per branch and KV head: branches share prefix tiles
        (5, 300, 1, 8, 2, 128), (3, 64, 3, 4, 4, 64), (8, 1000, 2, 32, 8, 128), (4, 0, 5, 8, 2, 64),
        (2, 130, 15, 8, 2, 128), (32, 2100, 1, 32, 8, 128), (64, 64, 1, 4, 1, 64),
        # full-size decode and long-prefix verify tiles: many prefix tiles per chunk
        # stream through the LDS ring (slots reused while others are in flight)
        (32, 16384, 1, 32, 8, 128), (4, 16384, 32, 32, 8, 128), (64, 1024, 32, 8, 2, 128),
    ]
    cases = []
    for shp in shapes:
        B, n, s, H, Hkv, hd = shp
        cases.append(pytest.param(torch.bfloat16, *shp, id=f"bf16-{B}-{n}-{s}-{H}-{Hkv}-{hd}"))
        if n * s * H <= 1024 * 128 * 8:
            cases.append(pytest.param(torch.float32, *shp, id=f"f32-{B}-{n}-{s}-{H}-{Hkv}-{hd}"))
    return cases


@pytest.mark.parametrize("dtype,B,n,s,H,Hkv,hd", _attention_cases())
def test_attention_matches_oracle(dtype, B, n, s, H, Hkv, hd):
    log(f"attention {dtype} B={B} n={n} s={s} H={H} Hkv={Hkv} hd={hd}")
    std = 1.28
    f32 = torch.float32
    q = _rand((B * s, H, hd), f32, 10, std)          # queries and the branch's own K/V are fp32
    pk = _rand((Hkv, n, hd), dtype, 11, std)         # the shared prefix is in the model dtype
    pv = _rand((Hkv, n, hd), dtype, 12, std)
    ko = _rand((B, Hkv, s, hd), f32, 13, std)
    vo = _rand((B, Hkv, s, hd), f32, 14, std)
    o = rk.rksc_test_attention(q.to(DEV), pk.to(DEV) if n else None, pv.to(DEV) if n else None,
                               ko.to(DEV), vo.to(DEV), dtype)
    torch.cuda.synchronize()
    got = o.float().cpu().numpy().reshape(B, s, H, hd)
    tol = 5e-5
    for b in range(B):
        qb = q[b * s:(b + 1) * s].float().numpy()
        kk = np.concatenate([pk.float().numpy(), ko[b].float().numpy()], axis=1)
        vv = np.concatenate([pv.float().numpy(), vo[b].float().numpy()], axis=1)
        ref = oracle.attention(qb, kk, vv, n)
        rel = np.linalg.norm(got[b] - ref) / np.linalg.norm(ref)
        row_rel = np.linalg.norm(got[b] - ref, axis=-1) / np.linalg.norm(ref, axis=-1)
        assert rel < tol / 2 and row_rel.max() < tol, f"branch {b}: rel {rel:.3e}, worst row {row_rel.max():.3e}"
