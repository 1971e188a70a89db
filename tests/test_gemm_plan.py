"""Host-side pins of the projection planner (rksc_test_gemm_plan launches nothing)."""
import pytest

import paper_2606_09937_amd as rk

# The 7B projections: (N, K) of QKV, O, gate|up, down.
P7B = {"qkv": (6144, 4096), "o": (4096, 4096), "gu": (28672, 4096), "down": (4096, 14336)}


@pytest.mark.parametrize("M", [33, 64, 128])
def test_128_row_plans_at_the_headline_shape(M):
    """Up to 128 rows: one row tile, the widest column tile that reaches ~224 workgroups with at most
    8 K splits (the HBM-bound verify pass of one branch)."""
    want = {"qkv": (192, 8), "o": (128, 8), "gu": (256, 2), "down": (128, 8)}
    for name, (N, K) in P7B.items():
        p = rk.rksc_test_gemm_plan(M, N, K)
        assert (p["kind"], p["bm"]) == (0, 128), (name, p)
        assert (p["bn"], p["splits"]) == want[name], (name, p)


@pytest.mark.parametrize("M", [1, 8, 16, 17, 32])
def test_weight_stream_for_decode_rows(M):
    """Up to 16 rows every projection streams the weights; from 17 to 32 rows (two 16-row activation
    blocks) only the wide gate|up does, the others keep the 128-row tiles."""
    for name, (N, K) in P7B.items():
        p = rk.rksc_test_gemm_plan(M, N, K)
        if M <= 16 or name == "gu":
            assert p["kind"] == 2 and p["k_per_split"] == 2048 and p["splits"] == -(-K // 2048), (name, p)
            assert p["bm"] == (16 if M <= 16 else 32), (name, p)
        else:
            assert p["kind"] == 0 and p["bm"] == 128, (name, p)


def test_two_row_blocks_need_one_half_slice():
    """Two row blocks hold one 256-wide half-slice per wave: K above 16384 falls back to 128-row tiles
    from 17 rows, while 16 rows take 4096-wide splits."""
    assert rk.rksc_test_gemm_plan(16, 4096, 20000)["kind"] == 2
    assert rk.rksc_test_gemm_plan(16, 4096, 20000)["k_per_split"] == 4096
    assert rk.rksc_test_gemm_plan(17, 28672, 20000)["kind"] == 0
    assert rk.rksc_test_gemm_plan(17, 28672, 4096)["kind"] == 2
    assert rk.rksc_test_gemm_plan(33, 28672, 4096)["kind"] == 0


@pytest.mark.parametrize("M,N,K,want", [
    # measured on MI355X: 108 -> 71 us with 256 x 256 tiles over 3 K splits (28-layer QKV, 1024 rows)
    (1024, 4608, 3584, (1, 3)),
    # 259 -> 224 us: one round of 224 wide workgroups instead of 448 128-row ones (7B gate|up, 512 rows)
    (512, 28672, 4096, (1, 1)),
    # equal within noise: the 128-row plan stays (7B O, 1024 rows)
    (1024, 4096, 4096, (0, 2)),
    # many rows: whole rounds of wide tiles without splitting K
    (8192, 4096, 14336, (1, 1)), (4096, 37888, 3584, (1, 1)),
])
def test_mfma_bound_plans(M, N, K, want):
    p = rk.rksc_test_gemm_plan(M, N, K)
    assert (p["kind"], p["splits"]) == want, p
    assert p["bm"] == (256 if p["kind"] == 1 else 128)


@pytest.mark.parametrize("M", [129, 256, 511, 512, 777, 1024, 2048, 4096, 8192])
@pytest.mark.parametrize("N,K", list(P7B.values()) + [(4608, 3584), (3584, 18944), (37888, 3584), (260, 1000)])
def test_plan_invariants(M, N, K):
    """Every plan covers K exactly with at most 8 splits (the row kernels sum at most 8 partials), in
    whole pipeline stages (64 K elements for 128-row tiles, 32 for 256 x 256), none of them empty."""
    for bf16 in (True, False):
        p = rk.rksc_test_gemm_plan(M, N, K, bf16=bf16)
        sp, kps = p["splits"], p["k_per_split"]
        assert 1 <= sp <= 8, p
        assert (sp - 1) * kps < K <= sp * kps, p
        if bf16:
            assert kps % (32 if p["kind"] == 1 else 64) == 0 or sp == 1, p
        else:
            assert p["kind"] == 0, p


def test_large_row_counts_take_wide_tiles():
    """Row counts where row * K passes 2^31 (a 150k-token root forward, 64 branches x 2400 tokens at
    the 7B width) reach the 256 x 256-tile kernel through the planner; its row offsets are 64-bit."""
    for M in (153600, 262144):
        assert rk.rksc_test_gemm_plan(M, 4096, 14336)["kind"] == 1


def _attn_chunks(B, n, s, H, Hkv, hd=128):
    """Split-KV chunks of the attention planner, read back from the test hook's scratch size
    (4096 bytes + one (hd + 2)-float partial per chunk, row and head; no partials for one chunk)."""
    lib = rk.load_library()
    size = int(lib.rksc_test_attention_scratch_size(1, B, n, s, H, Hkv, hd))
    parts = (size - 4096) // (B * s * H * (hd + 2) * 4)
    assert 4096 + parts * B * s * H * (hd + 2) * 4 == size
    return max(parts, 1)


@pytest.mark.parametrize("name,B,n,s,H,Hkv,chunks", [
    ("7b_single", 1, 1024, 128, 32, 8, 8),       # 32 query tiles: 8 chunks fill one round of 256
    ("7b_paper_verify", 8, 1024, 128, 28, 4, 1),   # 224 query tiles: a second chunk would need two rounds
    ("7b_large_vocab", 8, 4096, 128, 28, 4, 1),
    ("7b_tot", 16, 2048, 256, 32, 8, 1),
    ("decode_8", 8, 1024, 1, 32, 8, 8),            # packed: 8 tiles, at least 2 prefix tiles per chunk
    ("10b_decode", 32, 16384, 1, 32, 8, 32),       # packed: 8 tiles x 32 chunks = 256
])
def test_attention_split_fits_one_round(name, B, n, s, H, Hkv, chunks):
    """The prefix is split into chunks only while the launch still fits one round of 256 workgroups
    (one per CU), with at least two key tiles per chunk."""
    assert _attn_chunks(B, n, s, H, Hkv) == chunks, name


def test_attention_split_rule_over_a_sweep():
    for B in (1, 2, 3, 8, 16, 32):
        for s in (1, 16, 128, 256):
            for n in (64, 1024, 16384):
                G = 4
                cross = G * s < 64
                base = (-(-B * s * G // 128) if cross else -(-G * s // 128) * B) * 8
                c = _attn_chunks(B, n, s, 32, 8)
                min_tiles = -(-n // 64) + (0 if cross else 1)
                assert 2 * c <= max(min_tiles, 2), (B, s, n, c)
                assert c == 1 or base * c <= 256, (B, s, n, c, base)
                # one more chunk would break a rule
                assert base * (c + 1) > 256 or 2 * (c + 1) > min_tiles, (B, s, n, c, base)
