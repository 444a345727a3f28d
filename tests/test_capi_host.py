"""Host-side tests of libpixelfly.so (no GPU): every declared symbol is
exported, the C++ layout builder matches the oracle's independently built
mask bit for bit, the kernel work lists cover every kept block once, and
every argument error is reported before anything is enqueued."""
import ctypes

import numpy as np
import pytest

import synth
from oracle import mask as om

pf = pytest.importorskip("paper_2112_00029_amd.pixelfly")


def test_every_header_symbol_is_exported():
    names = pf.header_functions()
    assert len(names) >= 18
    lib = ctypes.CDLL(pf.LIB_PATH)
    for n in names:
        assert hasattr(lib, n), n


LAYOUTS = [
    (1024, 1024, 32, 32), (3072, 768, 32, 16), (4096, 1024, 64, 16), (1024, 4096, 64, 16),
    (4096, 4096, 64, 64), (16384, 4096, 128, 32), (16384, 4096, 64, 32), (16384, 4096, 32, 32),
    (64, 64, 32, 1), (64, 64, 32, 4), (128, 64, 32, 2), (96, 160, 32, 8), (384, 128, 64, 1024),
    (768, 768, 32, 1), (256, 256, 128, 2),
]


@pytest.mark.parametrize("n_out,n_in,b,ms", LAYOUTS)
def test_layout_bit_exact_vs_oracle(n_out, n_in, b, ms):
    L = pf.pf_layout_create(n_out, n_in, b, ms)
    info = pf.pf_layout_info_get(L)
    M, ref = om.layout(n_out, n_in, b, ms)
    for name, r in zip(["row_ptr", "col_idx", "col_ptr", "row_idx", "tperm"], ref):
        assert info[name].dtype == np.int32
        assert np.array_equal(info[name], r), name
    assert info["nnzb"] == M.sum()
    assert info["s"] == min(n_out // b, n_in // b)
    pf.pf_layout_check(L)
    st = pf.pf_layout_plan_get(L)
    assert st["tn_kept"] == info["nnzb"]


def test_random_layout_sweep():
    rng = np.random.default_rng(0)
    for _ in range(40):
        b = int(rng.choice([1, 2, 4, 32]))
        nbo, nbi = int(rng.integers(1, 40)), int(rng.integers(1, 40))
        ms = int(2 ** rng.integers(0, 7))
        L = pf.pf_layout_create(nbo * b, nbi * b, b, ms)
        info = pf.pf_layout_info_get(L)
        _, ref = om.layout(nbo * b, nbi * b, b, ms)
        for name, r in zip(["row_ptr", "col_idx", "col_ptr", "row_idx", "tperm"], ref):
            assert np.array_equal(info[name], r), (name, b, nbo, nbi, ms)
        pf.pf_layout_check(L)


def test_tiled_layouts_group_rows():
    # tiled copies along the output dim form 4-row tiles for the forward
    st = pf.pf_layout_plan_get(pf.pf_layout_create(3072, 768, 32, 16))
    assert st["G_fwd"] == 4 and st["fwd_tiles"] == 24
    # tiles are at most 128 columns wide
    st = pf.pf_layout_plan_get(pf.pf_layout_create(16384, 4096, 128, 32))
    assert st["G_fwd"] == 1 and st["fwd_tiles"] == 128
    # wide lists: the four tiled copies pair up (256 columns per tile)
    assert st["G_fwd_wide"] == 2 and st["fwd_tiles_wide"] == 64
    st = pf.pf_layout_plan_get(pf.pf_layout_create(16384, 4096, 64, 32))
    assert st["G_fwd"] == 2 and st["fwd_tiles"] == 128
    assert st["G_fwd_wide"] == 4 and st["fwd_tiles_wide"] == 64
    # tiled copies along the input dim form 2-column tiles for backward-data
    st = pf.pf_layout_plan_get(pf.pf_layout_create(1024, 4096, 64, 16))
    assert st["G_bwd"] == 2 and st["bwd_tiles"] == 32
    assert st["G_bwd_wide"] == 4 and st["bwd_tiles_wide"] == 16


def test_pair_block_plans():
    """b = 32 layers with T x K >= 4M and a rank that is a multiple of 64 run
    backward-data on 64-wide pair tiles and the weight gradient on pair items
    of 256 x 256; smaller products, odd ranks and fp32 keep the 32-wide
    tiles (host planning only, no kernel runs)."""
    L = pf.pf_layout_create(16384, 4096, 32, 32)
    p = pf.pf_linear_plan_get(L, "bf16", 16384, 256)
    assert (p["bwd_tile_n"], p["bwd_direct_lds"]) == (64, 1), p
    assert (p["tn_tile"], p["tn_items"], p["tn_shared"], p["tn_split"]) == (256, 208, 0, 1), p
    # room for the pair blocks (1280 of 64 x 64 bf16) on top of the rest
    assert p["workspace_bytes"] >= 1280 * 64 * 64 * 2
    for T, r, dt in [(512, 256, "bf16"), (16384, 96, "bf16"), (16384, 256, "fp32")]:
        q = pf.pf_linear_plan_get(L, dt, T, r)
        assert q["bwd_tile_n"] == 32 and q["tn_tile"] == 128, (T, r, dt, q)
    # 2048 tokens x 1024: below 4M, the gather would not pay
    q = pf.pf_linear_plan_get(pf.pf_layout_create(1024, 1024, 32, 32), "bf16", 2048, 64)
    assert q["bwd_tile_n"] == 32, q


def test_layout_create_errors():
    for args in [(100, 64, 32, 2), (64, 64, 0, 2), (64, 64, 32, 3), (64, 64, 32, 0), (0, 64, 32, 1)]:
        with pytest.raises(pf.PixelflyError) as e:
            pf.pf_layout_create(*args)
        assert e.value.status == pf.PF_ERR_INVALID_ARG


def test_eff_stride_clamped():
    info = pf.pf_layout_info_get(pf.pf_layout_create(24 * 32, 24 * 32, 32, 1024))
    assert info["max_stride"] == 1024 and info["eff_stride"] == 32


A16 = 0x10000  # a 16-byte aligned fake address: never dereferenced


def _fwd(L, **kw):
    args = dict(dtype=pf.PF_BF16, T=128, r=32, X=A16, Wblk=A16, U=A16, V=A16, Y=A16, T_lr=A16,
                epi=pf.PF_EPI_NONE, Y_pre=None)
    args.update(kw)
    pf.pf_linear_fwd(L, args["dtype"], args["T"], args["r"], args["X"], args["Wblk"], args["U"],
                     args["V"], args["Y"], args["T_lr"], args["epi"], args["Y_pre"], stream=0)


def test_compute_call_errors_before_any_launch():
    L = pf.pf_layout_create(256, 256, 32, 4)
    cases = [
        (dict(T=0), pf.PF_ERR_INVALID_ARG), (dict(r=16), pf.PF_ERR_INVALID_ARG),
        (dict(r=-32), pf.PF_ERR_INVALID_ARG), (dict(X=None), pf.PF_ERR_INVALID_ARG),
        (dict(X=A16 + 2), pf.PF_ERR_INVALID_ARG), (dict(dtype=7), pf.PF_ERR_INVALID_ARG),
        (dict(epi=5), pf.PF_ERR_INVALID_ARG), (dict(epi=pf.PF_EPI_GELU), pf.PF_ERR_INVALID_ARG),
        (dict(Y_pre=A16), pf.PF_ERR_INVALID_ARG), (dict(U=None), pf.PF_ERR_INVALID_ARG),
        (dict(), pf.PF_ERR_STATE),  # valid arguments, layout never uploaded
        (dict(r=0, U=None, V=None, T_lr=None), pf.PF_ERR_STATE),
    ]
    for kw, want in cases:
        with pytest.raises(pf.PixelflyError) as e:
            _fwd(L, **kw)
        assert e.value.status == want, (kw, e.value)
    with pytest.raises(pf.PixelflyError) as e:
        pf.pf_linear_bwd_data(L, pf.PF_BF16, 128, 32, A16, A16, A16, A16, A16, None, stream=0)
    assert e.value.status == pf.PF_ERR_INVALID_ARG
    with pytest.raises(pf.PixelflyError) as e:
        pf.pf_linear_bwd_weight(L, pf.PF_BF16, 128, 32, A16, A16, A16, A16, A16, A16, A16,
                                A16, 1 << 30, stream=0)
    assert e.value.status == pf.PF_ERR_STATE
    # unsupported block size for the kernels
    L16 = pf.pf_layout_create(256, 256, 16, 4)
    with pytest.raises(pf.PixelflyError) as e:
        _fwd(L16)
    assert e.value.status == pf.PF_ERR_UNSUPPORTED
    # attention: wrong head dim / non-square layout
    La = pf.pf_layout_create(512, 512, 64, 8)
    with pytest.raises(pf.PixelflyError) as e:
        pf.pf_attn_fwd(La, 1, 1, 512, 128, 0.1, A16, A16, A16, A16, A16, stream=0)
    assert e.value.status == pf.PF_ERR_UNSUPPORTED
    with pytest.raises(pf.PixelflyError) as e:
        pf.pf_attn_fwd(La, 1, 1, 256, 64, 0.1, A16, A16, A16, A16, A16, stream=0)
    assert e.value.status == pf.PF_ERR_INVALID_ARG
    with pytest.raises(pf.PixelflyError) as e:
        pf.pf_attn_bwd(La, 1, 1, 512, 64, 0.1, A16, A16, A16, A16, A16, A16, A16, A16, A16,
                       A16, 16, stream=0)
    assert e.value.status == pf.PF_ERR_WORKSPACE
    # dense comparator shape checks
    with pytest.raises(pf.PixelflyError) as e:
        pf.pf_dense_gemm(pf.PF_BF16, pf.PF_OP_NT, 100, 64, 64, A16, A16, A16, stream=0)
    assert e.value.status == pf.PF_ERR_UNSUPPORTED
    with pytest.raises(pf.PixelflyError) as e:
        pf.pf_dense_gemm(pf.PF_BF16, 9, 64, 64, 64, A16, A16, A16, stream=0)
    assert e.value.status == pf.PF_ERR_INVALID_ARG
    # GELU backward with n = 0 is a no-op
    pf.pf_gelu_bwd(pf.PF_BF16, 0, None, None, None, stream=0)


def test_workspace_sizes():
    L = pf.pf_layout_create(3072, 768, 32, 16)
    ws = pf.pf_workspace_bytes(L, 4096, 96, pf.PF_BF16)
    assert ws > 0 and ws % 4 == 0
    assert pf.pf_workspace_bytes(L, 4096, 95, pf.PF_BF16) == 0
    # split partials scale with the tokens
    assert pf.pf_workspace_bytes(L, 64, 96, pf.PF_BF16) < ws
    assert pf.pf_workspace_bytes(L, 4096, 0, pf.PF_BF16) <= ws
    assert pf.pf_attn_workspace_bytes(8, 12, 4096) >= 8 * 12 * 4096 * 4
    assert pf.pf_dense_workspace_bytes(pf.PF_BF16, pf.PF_OP_NT, 128, 128, 128) == 0


def test_layout_from_mask():
    rng = np.random.default_rng(5)
    for b in [32, 64, 1]:
        for _ in range(10):
            nbo, nbi = int(rng.integers(1, 20)), int(rng.integers(1, 20))
            M = rng.random((nbo, nbi)) < 0.3
            M[np.arange(nbo), rng.integers(0, nbi, nbo)] = True  # no empty block row
            L = pf.pf_layout_create_from_mask(nbo, nbi, b, M)
            info = pf.pf_layout_info_get(L)
            for name, r in zip(["row_ptr", "col_idx", "col_ptr", "row_idx", "tperm"], om.block_csr(M)):
                assert np.array_equal(info[name], r), name
            assert info["max_stride"] == 0
            pf.pf_layout_check(L)
            assert pf.pf_layout_plan_get(L)["tn_kept"] == M.sum()
    with pytest.raises(pf.PixelflyError):
        pf.pf_layout_create_from_mask(2, 2, 32, np.array([[1, 0], [0, 0]]))


def test_timing_hook_errors_before_any_hip_call():
    with pytest.raises(pf.PixelflyError) as e:
        pf.pf_timing_begin(0)
    assert e.value.status == pf.PF_ERR_INVALID_ARG
    with pytest.raises(pf.PixelflyError) as e:
        pf.pf_timing_end()
    assert e.value.status == pf.PF_ERR_STATE
    assert len(pf.KERNEL_CLASSES) == pf.PF_KERNEL_COUNT == 12


@pytest.mark.parametrize("seq,b,ms,g", [(4096, 64, 64, 1), (4096, 64, 64, 2), (512, 64, 8, 1),
                                        (1536, 64, 16, 3), (256, 32, 4, 0), (640, 64, 1024, 10)])
def test_attention_layout_bit_exact_vs_oracle(seq, b, ms, g):
    """Flat butterfly + global stripes: the C++ builder against the oracle's
    independently built union of supports."""
    L = pf.pf_layout_create_attention(seq, b, ms, g)
    info = pf.pf_layout_info_get(L)
    M, ref = om.attention_layout(seq, b, ms, g)
    for name, r in zip(["row_ptr", "col_idx", "col_ptr", "row_idx", "tperm"], ref):
        assert np.array_equal(info[name], r), name
    assert info["nnzb"] == M.sum()
    pf.pf_layout_check(L)


def test_attention_layout_errors():
    for args in [(4096, 64, 64, -1), (4096, 64, 64, 65), (4000, 64, 64, 1), (4096, 64, 3, 1),
                 (64 * 20000, 64, 64, 1)]:
        with pytest.raises(pf.PixelflyError):
            pf.pf_layout_create_attention(*args)


@pytest.mark.parametrize("n_out,n_in,b", [(3072, 768, 32), (4096, 1024, 64), (16384, 4096, 128),
                                          (1024, 1024, 32), (768, 768, 32), (96, 160, 32)])
def test_select_mask_matches_oracle(n_out, n_in, b):
    from oracle import select as osel
    for k in range(1, 21):
        for share in (0.0, 0.25, 1 / 3):
            got = pf.pf_select_mask(n_out, n_in, b, k / 20, share)
            r, ms, entries = osel.select(n_out, n_in, b, k / 20, share)
            assert (got["r"], got["max_stride"], got["params"]) == (r, ms, entries), (k, share)


def test_select_mask_errors():
    for args in [(1024, 1024, 32, 0.0, 0.25), (1024, 1024, 32, 1.5, 0.25), (1024, 1024, 32, 0.5, -0.1),
                 (1000, 1024, 32, 0.5, 0.25), (1024, 1024, 0, 0.5, 0.25)]:
        with pytest.raises(pf.PixelflyError):
            pf.pf_select_mask(*args)


@pytest.mark.parametrize("n,p,d,b", [(1024, 4, 0.05, 32), (1024, 16, 0.2, 32), (512, 8, 0.1, 64),
                                      (768, 1, 0.002, 32), (256, 32, 0.5, 128)])
def test_cover_layout_bit_exact_vs_oracle(n, p, d, b):
    """pf_layout_create_from_element_mask against the oracle's block cover."""
    E = synth.random_block_mask(n, n, p, d, seed=5)
    C = om.block_cover(E, b, b)
    Mb = C[::b, ::b]
    if not Mb.any(axis=1).all():
        pytest.skip("draw left an empty block row")
    L = pf.pf_layout_create_from_element_mask(n, n, b, E)
    info = pf.pf_layout_info_get(L)
    ref = om.block_csr(Mb)
    for name, r in zip(["row_ptr", "col_idx", "col_ptr", "row_idx", "tperm"], ref):
        assert np.array_equal(info[name], r), name
    pf.pf_layout_check(L)


def test_cover_layout_errors():
    E = np.ones((64, 64), bool)
    for args in [(64, 64, 0, E), (64, 60, 32, E[:, :60]), (64, 64, 48, E)]:
        with pytest.raises(pf.PixelflyError):
            pf.pf_layout_create_from_element_mask(*args)
    E2 = np.zeros((64, 64), bool)
    E2[:32] = True  # second block row empty
    with pytest.raises(pf.PixelflyError):
        pf.pf_layout_create_from_element_mask(64, 64, 32, E2)


@pytest.mark.parametrize("n,b,k", [(1024, 32, 2), (1024, 32, 32), (512, 64, 4), (64, 1, 64)])
def test_factor_layout_vs_oracle(n, b, k):
    """pf_layout_create_factor against the oracle's factor-matrix support
    (built from the butterfly factor definition) plus the identity."""
    L = pf.pf_layout_create_factor(n, b, k)
    info = pf.pf_layout_info_get(L)
    S = om.factor_matrix_support(n // b, k) | np.eye(n // b, dtype=bool)
    ref = om.block_csr(S)
    for name, r in zip(["row_ptr", "col_idx", "col_ptr", "row_idx", "tperm"], ref):
        assert np.array_equal(info[name], r), name
    assert info["nnzb"] == 2 * (n // b)


def test_factor_layout_errors():
    for args in [(1024, 32, 3), (1024, 32, 64), (1000, 32, 2), (1024, 32, 1)]:
        with pytest.raises(pf.PixelflyError):
            pf.pf_layout_create_factor(*args)


def test_mixed_call_errors_before_any_launch():
    """The mixing-weight calls check gamma and every argument before the
    layout state (no HIP work happens for any of these)."""
    L = pf.pf_layout_create(256, 256, 32, 4)
    nan = float("nan")
    with pytest.raises(pf.PixelflyError) as e:
        pf.pf_linear_fwd_mixed(L, pf.PF_BF16, 128, 32, nan, A16, A16, A16, A16, A16, A16, stream=0)
    assert e.value.status == pf.PF_ERR_INVALID_ARG
    with pytest.raises(pf.PixelflyError) as e:
        pf.pf_linear_fwd_mixed(L, pf.PF_BF16, 128, 32, 0.5, A16, A16, A16, A16, A16, A16, stream=0)
    assert e.value.status == pf.PF_ERR_STATE
    with pytest.raises(pf.PixelflyError) as e:
        pf.pf_linear_bwd_data_mixed(L, pf.PF_BF16, 128, 32, float("inf"), A16, A16, A16, A16, A16,
                                    A16, stream=0)
    assert e.value.status == pf.PF_ERR_INVALID_ARG
    with pytest.raises(pf.PixelflyError) as e:
        pf.pf_linear_bwd_data_mixed(L, pf.PF_BF16, 128, 32, 0.5, A16, A16, A16, A16, None, A16,
                                    stream=0)
    assert e.value.status == pf.PF_ERR_INVALID_ARG
    args = [A16] * 8  # dY, X, Wblk, T_lr, S, dW, dU, dV
    for dg, want in [(None, pf.PF_ERR_INVALID_ARG), (A16 + 2, pf.PF_ERR_INVALID_ARG),
                     (A16, pf.PF_ERR_STATE)]:
        with pytest.raises(pf.PixelflyError) as e:
            pf.pf_linear_bwd_weight_mixed(L, pf.PF_BF16, 128, 32, 0.5, *args, dg, A16, 1 << 30,
                                          stream=0)
        assert e.value.status == want, dg
    with pytest.raises(pf.PixelflyError) as e:  # Wblk is required (the dgamma term)
        pf.pf_linear_bwd_weight_mixed(L, pf.PF_BF16, 128, 32, 0.5, A16, A16, None, A16, A16, A16,
                                      A16, A16, A16, A16, 1 << 30, stream=0)
    assert e.value.status == pf.PF_ERR_INVALID_ARG


@pytest.mark.parametrize("n,b,ms", [(1024, 32, 32), (1024, 32, 2), (2048, 32, 16), (512, 64, 8),
                                    (96, 3, 4)])
def test_butterfly_product_layout_bit_exact_vs_oracle(n, b, ms):
    """Stacked factor supports of the product form: the C++ builder against
    the oracle's block-diagonal factor mask, bit for bit."""
    from oracle import butterfly as ob
    L = pf.pf_layout_create_butterfly(n, b, ms)
    info = pf.pf_layout_info_get(L)
    nfac = ms.bit_length() - 1
    M = ob.product_factor_mask(n // b, nfac)
    row_ptr, col_idx, *_r = om.block_csr(M)
    assert info["nb_out"] == info["nb_in"] == nfac * (n // b)
    assert np.array_equal(info["row_ptr"], row_ptr) and np.array_equal(info["col_idx"], col_idx)
    pf.pf_layout_check(L)


def test_butterfly_product_errors():
    for args in [(1024, 32, 3), (1024, 32, 1), (1000, 32, 4), (1024, 32, 64)]:
        with pytest.raises(pf.PixelflyError) as e:
            pf.pf_layout_create_butterfly(*args)
        assert e.value.status == pf.PF_ERR_INVALID_ARG
    fake = 1 << 40
    flat = pf.pf_layout_create(1024, 1024, 32, 8)
    with pytest.raises(pf.PixelflyError) as e:  # not a product layout
        pf.pf_butterfly_fwd(flat, 64, fake, fake, fake)
    assert e.value.status == pf.PF_ERR_INVALID_ARG
    wide = pf.pf_layout_create_butterfly(4096, 32, 64)  # 64 x 32 features per group
    with pytest.raises(pf.PixelflyError) as e:
        pf.pf_butterfly_fwd(wide, 64, fake, fake, fake)
    assert e.value.status == pf.PF_ERR_UNSUPPORTED
    b64 = pf.pf_layout_create_butterfly(1024, 64, 4)
    with pytest.raises(pf.PixelflyError) as e:
        pf.pf_butterfly_bwd_data(b64, 64, fake, fake, fake)
    assert e.value.status == pf.PF_ERR_UNSUPPORTED
    L = pf.pf_layout_create_butterfly(1024, 32, 8)
    with pytest.raises(pf.PixelflyError) as e:
        pf.pf_butterfly_fwd(L, 64, fake + 2, fake, fake)  # misaligned X
    assert e.value.status == pf.PF_ERR_INVALID_ARG
