"""GPU parity of the sparse + low-rank linear layer against the fp64 oracle.

Every case runs forward, backward-data and backward-weight through the C ABI
(libpixelfly.so) and compares each output with the oracle element by element
(relative Frobenius error; bf16 <= 2e-2, fp32 <= 1e-5), plus bit-exact cases
on integer-valued inputs.
"""
import numpy as np
import pytest

import synth
from oracle import linear as ol
from oracle import mask as om
from tests._gpu_util import (TOL, bf16_round, check_close, empty, rel_fro, to_dev, to_host,
                             torch_cuda)

pytestmark = pytest.mark.gpu


def _inputs(n_out, n_in, b, ms, T, r, dtype, seed=0, std=(0.02, 0.02, 0.02, 0.02), ints=None):
    """Seeded inputs; W drawn directly as packed kept blocks (oracle CSR)."""
    M, (row_ptr, col_idx, *_r) = om.layout(n_out, n_in, b, ms)
    nnzb = int(M.sum())
    sx, sw, suv, sdy = std
    if ints is None:
        X, Xr = synth.draw((T, n_in), sx, seed, 1, dtype)
        W, Wr = synth.draw((nnzb, b, b), sw, seed, 2, dtype)
        U, Ur = synth.draw((n_out, r), suv, seed, 3, dtype)
        V, Vr = synth.draw((r, n_in), suv, seed, 4, dtype)
        dY, dYr = synth.draw((T, n_out), sdy, seed, 5, dtype)
    else:
        lo, hi = ints
        X, Xr = synth.draw_int((T, n_in), lo, hi, seed, 1, dtype)
        W, Wr = synth.draw_int((nnzb, b, b), lo, hi, seed, 2, dtype)
        U, Ur = synth.draw_int((n_out, r), lo, hi, seed, 3, dtype)
        V, Vr = synth.draw_int((r, n_in), lo, hi, seed, 4, dtype)
        dY, dYr = synth.draw_int((T, n_out), lo, hi, seed, 5, dtype)
    Wd = ol.unpack(W, row_ptr, col_idx, n_out // b, n_in // b, b)
    return dict(M=M, Mel=om.element_mask(M, b), X=X, W=W, Wd=Wd, U=U, V=V, dY=dY,
                raw=dict(X=Xr, W=Wr, U=Ur, V=Vr, dY=dYr))


def _run_gpu_dev(n_out, n_in, b, ms, T, r, dtype, raw, timing=False):
    """fwd, bwd-data, bwd-weight through the C ABI; returns the device
    outputs, the layout and (timing) the launches per kernel class."""
    torch = torch_cuda()
    from paper_2112_00029_amd import pixelfly as pf
    print(f"[linear] n_out={n_out} n_in={n_in} b={b} ms={ms} T={T} r={r} {dtype}", flush=True)
    L = pf.pf_layout_create(n_out, n_in, b, ms)
    pf.pf_layout_upload(L)
    d = {k: to_dev(v) for k, v in raw.items()}
    Y = empty((T, n_out), dtype)
    dX = empty((T, n_in), dtype)
    dW = empty(tuple(d["W"].shape), dtype)
    Tl = empty((T, max(r, 1)), dtype)
    S = empty((T, max(r, 1)), dtype)
    dU = empty((n_out, max(r, 1)), dtype)
    dV = empty((max(r, 1), n_in), dtype)
    U = d["U"] if r else None
    V = d["V"] if r else None
    ws_bytes = pf.pf_workspace_bytes(L, T, r, dtype)
    ws = torch.empty(max(ws_bytes, 256), dtype=torch.uint8, device="cuda")
    if timing:
        pf.pf_timing_begin(8)
    try:
        pf.pf_linear_fwd(L, dtype, T, r, d["X"], d["W"], U, V, Y, Tl if r else None,
                         workspace=ws, ws_bytes=ws_bytes)
        pf.pf_linear_bwd_data(L, dtype, T, r, d["dY"], d["W"], U, V, S if r else None, dX,
                              workspace=ws, ws_bytes=ws_bytes)
        pf.pf_linear_bwd_weight(L, dtype, T, r, d["dY"], d["X"], Tl if r else None,
                                S if r else None, dW, dU if r else None, dV if r else None,
                                ws, ws_bytes)
        torch.cuda.synchronize()
    finally:
        kt = pf.pf_timing_end() if timing else None
    out = dict(Y=Y, dX=dX, dW=dW)
    if r:
        out.update(T_lr=Tl, S=S, dU=dU, dV=dV)
    return out, L, kt


def _run_gpu(n_out, n_in, b, ms, T, r, dtype, inp):
    """As _run_gpu_dev, outputs read back as float64 arrays."""
    out, L, _kt = _run_gpu_dev(n_out, n_in, b, ms, T, r, dtype, inp["raw"])
    return {k: to_host(v) for k, v in out.items()}, L


def _oracle(inp, r, b):
    U = inp["U"] if r else None
    V = inp["V"] if r else None
    Y, Tlr = ol.forward(inp["X"], inp["Wd"], U, V)
    g = ol.backward(inp["X"], inp["Wd"], inp["Mel"], inp["dY"], U, V)
    ref = dict(Y=Y, dX=g["dX"], dW_dense=g["dW"])
    if r:
        ref.update(T_lr=Tlr, S=g["S"], dU=g["dU"], dV=g["dV"])
    return ref


def _pack_ref(ref, n_out, n_in, b, ms):
    _, (row_ptr, col_idx, *_r) = om.layout(n_out, n_in, b, ms)
    return ol.pack(ref["dW_dense"], row_ptr, col_idx, n_out // b, b)


CASES = [
    # (n_out, n_in, b, max_stride, T, r, dtype)
    pytest.param(1024, 1024, 32, 32, 256, 32, "fp32", id="fp32_1024sq_b32_full"),
    pytest.param(3072, 768, 32, 16, 4096, 96, "bf16", id="mlp_fc1_full"),
    pytest.param(3072, 768, 32, 16, 300, 96, "bf16", id="mlp_fc1_ragged300"),
    pytest.param(4096, 1024, 64, 16, 520, 128, "bf16", id="fc1_1024x4096_b64_T520"),
    pytest.param(1024, 4096, 64, 16, 520, 128, "bf16", id="fc2_4096x1024_b64_T520"),
    # >= 2048 tokens: 256 x 256 tiles where four block rows (columns) share
    # their kept set, 256 x 64 tiles where none do; ragged last token tile
    pytest.param(4096, 1024, 64, 16, 2100, 128, "bf16", id="fc1_1024x4096_b64_T2100_wide"),
    pytest.param(1024, 4096, 64, 16, 2100, 128, "bf16", id="fc2_4096x1024_b64_T2100_wide"),
    pytest.param(2048, 1024, 128, 8, 2100, 128, "bf16", id="b128_T2100_wide"),
    # 512-token tiles (128-column outputs with 512+ workgroups)
    pytest.param(4096, 4096, 128, 32, 8000, 128, "bf16", id="b128_4096sq_T8000_tall"),
    pytest.param(16384, 4096, 128, 32, 200, 256, "bf16", id="large_b128_T200"),
    # S = dY U 8256 deep with r = 512: two 256-wide columns of the split
    # 256 x 256 rank-r tiles, ragged last token tile
    pytest.param(8256, 1024, 64, 16, 2100, 512, "bf16", id="deep_S_r512_T2100"),
    pytest.param(16384, 4096, 64, 32, 200, 256, "bf16", id="large_b64_T200"),
    # b = 32 backward-data on 64-wide pair tiles (T x K >= 4M), ragged
    # last token tile
    pytest.param(2048, 1024, 32, 16, 4100, 64, "bf16", id="b32_pairs_T4100"),
    # forward in bands of output tiles (64+ tiles): 68 tiles of 128 columns
    # in bands of 9 (the last of 5), 5 token tiles (a last group of one)
    pytest.param(8320, 512, 32, 16, 600, 64, "bf16", id="band_ragged_N8320_T600"),
    pytest.param(16384, 4096, 32, 32, 200, 256, "bf16", id="large_b32_T200"),
    # rank-r kernel edges: r = 32 (half of a 64-column tile past r), K and N
    # = 32 mod 64 (the last 64-wide step half outside), 3 steps for 4 waves
    pytest.param(480, 160, 32, 4, 70, 32, "bf16", id="rank32_K160_N480_T70"),
    pytest.param(512, 512, 32, 1, 130, 0, "bf16", id="blockdiag_r0"),
    pytest.param(128, 128, 64, 2, 1, 64, "bf16", id="dense_mask_T1"),
    pytest.param(384, 640, 64, 1024, 77, 64, "bf16", id="clamped_stride_rect"),
    pytest.param(768, 256, 128, 2, 129, 128, "fp32", id="fp32_b128"),
    pytest.param(512, 256, 64, 4, 200, 64, "fp32", id="fp32_b64"),
]


@pytest.mark.parametrize("n_out,n_in,b,ms,T,r,dtype", CASES)
def test_linear_parity(n_out, n_in, b, ms, T, r, dtype):
    std = (1.0, 1.0 / np.sqrt(6 * 32), 1.0 / 32, 1.0) if dtype == "fp32" else (0.02,) * 4
    inp = _inputs(n_out, n_in, b, ms, T, r, dtype, std=std)
    got, _ = _run_gpu(n_out, n_in, b, ms, T, r, dtype, inp)
    ref = _oracle(inp, r, b)
    ref["dW"] = _pack_ref(ref, n_out, n_in, b, ms)
    for k in ["Y", "dX", "dW"] + (["T_lr", "S", "dU", "dV"] if r else []):
        check_close(k, got[k], ref[k], dtype)


def test_fp32_integer_inputs_bit_exact():
    """Integer inputs in [-2, 2], fp32 I/O: every partial sum is an integer
    below 2^24, so the GPU result equals the oracle exactly."""
    n_out, n_in, b, ms, T, r = 1024, 1024, 32, 32, 256, 32
    inp = _inputs(n_out, n_in, b, ms, T, r, "fp32", ints=(-2, 2))
    got, _ = _run_gpu(n_out, n_in, b, ms, T, r, "fp32", inp)
    ref = _oracle(inp, r, b)
    ref["dW"] = _pack_ref(ref, n_out, n_in, b, ms)
    for k in ["Y", "dX", "dW", "T_lr", "S", "dU", "dV"]:
        assert np.array_equal(got[k], ref[k]), k


@pytest.mark.parametrize("b", [32, 64])
def test_bf16_integer_inputs_bit_exact(b):
    """Values in [-1, 1] and small dims keep T_lr and S integers <= 256
    (exact in bf16); outputs must equal the oracle rounded once to bf16."""
    n_out, n_in, ms, T, r = 2 * b, 2 * b, 2, 96, b
    inp = _inputs(n_out, n_in, b, ms, T, r, "bf16", ints=(-1, 1))
    got, _ = _run_gpu(n_out, n_in, b, ms, T, r, "bf16", inp)
    ref = _oracle(inp, r, b)
    ref["dW"] = _pack_ref(ref, n_out, n_in, b, ms)
    assert np.abs(ref["T_lr"]).max() <= 256 and np.abs(ref["S"]).max() <= 256
    for k in ["Y", "dX", "dW", "T_lr", "S", "dU", "dV"]:
        assert np.array_equal(got[k], bf16_round(ref[k])), k


@pytest.mark.parametrize("T", [390, 8192], ids=["T390", "T8192_full"])
def test_mlp_pair_gelu(T):
    """Two layers 1024 -> 4096 -> GELU -> 1024 (b = 64, stride 16, r = 128)
    with the GELU epilogues: forward keeps the pre-activation, backward-data
    of the second layer applies gelu'(pre-activation).  At the workload's
    8192 tokens the GELU epilogues run on 256 x 256 tiles and the rank-r
    products on the split-K tile kernel."""
    torch = torch_cuda()
    from paper_2112_00029_amd import pixelfly as pf
    K, N, b, ms, r = 1024, 4096, 64, 16, 128
    dtype = "bf16"
    l1 = _inputs(N, K, b, ms, T, r, dtype, seed=0)
    l2 = _inputs(K, N, b, ms, T, r, dtype, seed=1)
    print(f"[mlp_pair] T={T}", flush=True)
    L1 = pf.pf_layout_create(N, K, b, ms)
    L2 = pf.pf_layout_create(K, N, b, ms)
    if T == 8192:
        p1, p2 = pf.pf_linear_plan_get(L1, dtype, T, r), pf.pf_linear_plan_get(L2, dtype, T, r)
        assert p1["fwd_tile_n"] == 256, p1  # GELU forward on wide tiles
        assert p2["bwd_tile_n"] == 256, p2  # GELU backward on wide tiles
        assert p1["lowrank_t_kernel"] == 2 and p1["lowrank_s_split"] > 1, p1
        assert p2["lowrank_t_kernel"] == 2 and p2["lowrank_t_split"] > 1, p2
    pf.pf_layout_upload(L1)
    pf.pf_layout_upload(L2)
    X = to_dev(l1["raw"]["X"])
    W1, U1, V1 = (to_dev(l1["raw"][k]) for k in ("W", "U", "V"))
    W2, U2, V2 = (to_dev(l2["raw"][k]) for k in ("W", "U", "V"))
    dY = to_dev(l2["raw"]["dY"])
    ws_b = max(pf.pf_workspace_bytes(L1, T, r, dtype), pf.pf_workspace_bytes(L2, T, r, dtype))
    ws = torch.empty(max(ws_b, 256), dtype=torch.uint8, device="cuda")
    W = dict(workspace=ws, ws_bytes=ws_b)
    Hpre, H, T1 = empty((T, N), dtype), empty((T, N), dtype), empty((T, r), dtype)
    Y, T2 = empty((T, K), dtype), empty((T, r), dtype)
    pf.pf_linear_fwd(L1, dtype, T, r, X, W1, U1, V1, H, T1, pf.PF_EPI_GELU, Hpre, **W)
    pf.pf_linear_fwd(L2, dtype, T, r, H, W2, U2, V2, Y, T2, **W)
    dHpre, S2, dX, S1 = empty((T, N), dtype), empty((T, r), dtype), empty((T, K), dtype), empty((T, r), dtype)
    pf.pf_linear_bwd_data(L2, dtype, T, r, dY, W2, U2, V2, S2, dHpre, pf.PF_EPI_GELU, Hpre, **W)
    pf.pf_linear_bwd_data(L1, dtype, T, r, dHpre, W1, U1, V1, S1, dX, **W)
    dW1, dU1, dV1 = empty(tuple(W1.shape), dtype), empty((N, r), dtype), empty((r, K), dtype)
    dW2, dU2, dV2 = empty(tuple(W2.shape), dtype), empty((K, r), dtype), empty((r, N), dtype)
    pf.pf_linear_bwd_weight(L2, dtype, T, r, dY, H, T2, S2, dW2, dU2, dV2, ws, ws_b)
    pf.pf_linear_bwd_weight(L1, dtype, T, r, dHpre, X, T1, S1, dW1, dU1, dV1, ws, ws_b)
    # standalone GELU backward agrees with the fused epilogue's definition
    dHpre2 = empty((T, N), dtype)
    dH_alone = empty((T, N), dtype)
    pf.pf_linear_bwd_data(L2, dtype, T, r, dY, W2, U2, V2, S2, dH_alone, **W)
    pf.pf_gelu_bwd(dtype, T * N, dH_alone, Hpre, dHpre2)
    torch.cuda.synchronize()

    ref_f = ol.mlp_pair_forward(l1["X"], l1["Wd"], l1["U"], l1["V"], l2["Wd"], l2["U"], l2["V"])
    ref_b = ol.mlp_pair_backward(l1["X"], l1["Wd"], l1["Mel"], l1["U"], l1["V"], l2["Wd"],
                                 l2["Mel"], l2["U"], l2["V"], l2["dY"], fwd=ref_f)
    _, (rp1, ci1, *_a) = om.layout(N, K, b, ms)
    _, (rp2, ci2, *_b) = om.layout(K, N, b, ms)
    checks = {
        "H_pre": (Hpre, ref_f["H_pre"]), "H": (H, ref_f["H"]), "Y": (Y, ref_f["Y"]),
        "dH_pre": (dHpre, ref_b["dH_pre"]), "dH_pre_standalone": (dHpre2, ref_b["dH_pre"]),
        "dX": (dX, ref_b["l1"]["dX"]),
        "dW2": (dW2, ol.pack(ref_b["l2"]["dW"], rp2, ci2, K // b, b)),
        "dU2": (dU2, ref_b["l2"]["dU"]), "dV2": (dV2, ref_b["l2"]["dV"]),
        "dW1": (dW1, ol.pack(ref_b["l1"]["dW"], rp1, ci1, N // b, b)),
        "dU1": (dU1, ref_b["l1"]["dU"]), "dV1": (dV1, ref_b["l1"]["dV"]),
    }
    for k, (g, rf) in checks.items():
        check_close(k, to_host(g), rf, dtype)


@pytest.mark.parametrize("n_out,n_in,b,ms,T,r", [
    (3072, 768, 32, 16, 4096, 96),   # split-token weight gradient
    (2048, 1024, 32, 16, 4100, 64),  # b = 32 backward-data on pair blocks
    (8320, 512, 32, 16, 600, 64),    # forward in bands of output tiles
])
def test_repeat_calls_are_deterministic(n_out, n_in, b, ms, T, r):
    """Split-token weight gradients combine partials in a fixed order, and no
    output is summed by racing workgroups: two runs give identical bits."""
    inp = _inputs(n_out, n_in, b, ms, T, r, "bf16", seed=3)
    a, _ = _run_gpu(n_out, n_in, b, ms, T, r, "bf16", inp)
    c, _ = _run_gpu(n_out, n_in, b, ms, T, r, "bf16", inp)
    for k in a:
        assert np.array_equal(a[k], c[k]), k


def test_kernel_timing_hook_counts_launches():
    """The timing hook sees every launch of a forward + backward step in its
    kernel class (reductions only when a split ran)."""
    from paper_2112_00029_amd import pixelfly as pf
    n_out, n_in, b, ms, T, r = 3072, 768, 32, 16, 512, 96
    inp = _inputs(n_out, n_in, b, ms, T, r, "bf16", seed=5)
    pf.pf_timing_begin(8)
    try:
        _run_gpu(n_out, n_in, b, ms, T, r, "bf16", inp)
    finally:
        kt = pf.pf_timing_end()
    for c in ("spmm_fwd", "spmm_bwd_data", "sddmm"):
        assert kt[c][0] == 1 and kt[c][1] > 0, (c, kt[c])
    for c in ("lowrank_t", "lowrank_s"):
        assert kt[c][0] == 1 and kt[c][1] > 0, (c, kt[c])
    for c in ("gelu_bwd", "attn_fwd", "attn_bwd_dq", "attn_bwd_dkv", "dense"):
        assert kt[c][0] == 0, (c, kt[c])


# ---------------------------------------------------------------------------
# The 16384 x 4096 layer (4096 -> 16384, r = 256, strides < 32 blocks) on the
# paths its full size runs: split-K rank-r products with the bf16 row
# reduction, the weight gradient's many-items token split, wide and tall
# tiles.
# ---------------------------------------------------------------------------
LARGE = dict(n_out=16384, n_in=4096, ms=32, r=256)


def _reductions(kt):
    return kt["reduce"][0]


@pytest.mark.parametrize("b", [128, 64, 32])
def test_large_layer_T4096_all_outputs(b):
    """Every output element against the oracle at 4096 tokens: T_lr and S run
    on the tile kernel with an 8-way K split and the bf16 row reduction, the
    weight gradient on its many-items token split."""
    from paper_2112_00029_amd import pixelfly as pf
    n_out, n_in, ms, r, T = LARGE["n_out"], LARGE["n_in"], LARGE["ms"], LARGE["r"], 4096
    plan = pf.pf_linear_plan_get(pf.pf_layout_create(n_out, n_in, b, ms), "bf16", T, r)
    print(f"[plan b={b} T={T}] {plan}", flush=True)
    assert plan["lowrank_t_kernel"] == 2 and plan["lowrank_t_split"] > 1, plan
    assert plan["lowrank_s_kernel"] == 2 and plan["lowrank_s_split"] > 1, plan
    # S = dY U is 16384 deep: 256 x 256 tiles (T_lr, 4096 deep, 128 x 128).
    assert (plan["lowrank_s_tile_m"], plan["lowrank_s_tile_n"]) == (256, 256), plan
    assert (plan["lowrank_t_tile_m"], plan["lowrank_t_tile_n"]) == (128, 128), plan
    if b == 128:
        # 256 x 256 weight-gradient tiles: whole items, then items shared by
        # several workgroups, summed from their partial slots by a second pass.
        assert plan["tn_tile"] == 256 and plan["tn_split"] == 1 and plan["tn_shared"] > 0, plan
    elif b == 64:
        # 208 items of 256 x 256, fewer than the 256 workgroups: one
        # workgroup per item, nothing shared, no second pass.
        assert plan["tn_tile"] == 256 and plan["tn_items"] == 208 and plan["tn_shared"] == 0, plan
    else:
        # Pair blocks (64 x 64): the weight gradient on 208 items of 256 x 256
        # as at b = 64, then the scatter of the kept quarters; backward-data
        # on 64-wide pair tiles after the pair-block gather.
        assert plan["tn_tile"] == 256 and plan["tn_items"] == 208 and plan["tn_shared"] == 0, plan
        assert (plan["bwd_tile_n"], plan["bwd_direct_lds"]) == (64, 1), plan
    inp = _inputs(n_out, n_in, b, ms, T, r, "bf16")
    out, _L, kt = _run_gpu_dev(n_out, n_in, b, ms, T, r, "bf16", inp["raw"], timing=True)
    # T_lr and S split their K range; the weight gradient splits its tokens
    # (128 x 128) or shares items between workgroups (256 x 256), except
    # with one workgroup per item (b = 64 and b = 32: no second pass); b = 32
    # adds the pair-block gather and scatter.
    assert _reductions(kt) == {128: 3, 64: 2, 32: 4}[b], kt
    got = {k: to_host(v) for k, v in out.items()}
    ref = _oracle(inp, r, b)
    ref["dW"] = _pack_ref(ref, n_out, n_in, b, ms)
    for k in ["Y", "dX", "dW", "T_lr", "S", "dU", "dV"]:
        check_close(k, got[k], ref[k], "bf16")


@pytest.mark.parametrize("T,r,b", [(2509, 256, 128), (2049, 256, 128), (2509, 128, 128),
                                   (2509, 256, 64), (2049, 128, 64), (2509, 256, 32),
                                   (2049, 128, 32)])
def test_large_layer_ragged_T_wide_weight_gradient(T, r, b):
    """The 16384 x 4096 layer at b = 128 with a token count that is not a
    multiple of the 32-token step: the 256 x 256 weight gradient's segments
    end inside a step (rows past T read as zeros) and the shares of the 16
    remaining items start mid-item.  At r = 128 the dU and dV tiles are half
    empty (one 128-column or 128-row block of the 256 x 256 tile), so waves
    whose quarter holds nothing skip their MFMAs and the stores drop the
    empty half.  At b = 64 (208 items, one workgroup per item) every item
    runs whole over the ragged token range; b = 32 runs the same way on its
    pair blocks (64 x 64, dropped quarters computed and not stored) and
    scatters them.  Every output element against the oracle."""
    from paper_2112_00029_amd import pixelfly as pf
    n_out, n_in, ms = LARGE["n_out"], LARGE["n_in"], LARGE["ms"]
    plan = pf.pf_linear_plan_get(pf.pf_layout_create(n_out, n_in, b, ms), "bf16", T, r)
    print(f"[plan b={b} T={T}] {plan}", flush=True)
    assert plan["tn_tile"] == 256 and (plan["tn_shared"] > 0) == (b == 128), plan
    inp = _inputs(n_out, n_in, b, ms, T, r, "bf16")
    out, _L, kt = _run_gpu_dev(n_out, n_in, b, ms, T, r, "bf16", inp["raw"], timing=True)
    assert kt["sddmm"][0] == 1, kt
    got = {k: to_host(v) for k, v in out.items()}
    ref = _oracle(inp, r, b)
    ref["dW"] = _pack_ref(ref, n_out, n_in, b, ms)
    for k in ["Y", "dX", "dW", "T_lr", "S", "dU", "dV"]:
        check_close(k, got[k], ref[k], "bf16")


@pytest.fixture(scope="module")
def large_full_inputs():
    """Seeded inputs of the full 16384-token layer shared by every block size
    (X, U, V, dY do not depend on b)."""
    T, n_out, n_in, r = 16384, LARGE["n_out"], LARGE["n_in"], LARGE["r"]
    X, Xr = synth.draw((T, n_in), 0.02, 0, 1, "bf16")
    U, Ur = synth.draw((n_out, r), 0.02, 0, 3, "bf16")
    V, Vr = synth.draw((r, n_in), 0.02, 0, 4, "bf16")
    dY, dYr = synth.draw((T, n_out), 0.02, 0, 5, "bf16")
    return dict(T=T, X=X, U=U, V=V, dY=dY, raw=dict(X=Xr, U=Ur, V=Vr, dY=dYr))


@pytest.mark.parametrize("b", [128, 64, 32])
def test_large_layer_full_size_sampled(large_full_inputs, b):
    """The 16384-token workload in the launch configuration the benchmark
    times.  The oracle computes sampled outputs one by one: token rows of Y,
    dX, T_lr and S (row t depends on row t of X or dY only), kept blocks of
    dW (block (i, j) is dY[:, i]^T X[:, j] by the gradient lemma), and all
    of S, dU and dV."""
    inp = large_full_inputs
    n_out, n_in, ms, r, T = LARGE["n_out"], LARGE["n_in"], LARGE["ms"], LARGE["r"], inp["T"]
    from paper_2112_00029_amd import pixelfly as pf
    plan = pf.pf_linear_plan_get(pf.pf_layout_create(n_out, n_in, b, ms), "bf16", T, r)
    print(f"[plan b={b} T={T}] {plan}", flush=True)
    assert plan["lowrank_t_kernel"] == 2 and plan["lowrank_s_kernel"] == 2, plan
    assert plan["tn_tile"] == 256, plan
    assert (plan["lowrank_s_tile_n"], plan["lowrank_s_split"]) == (256, 4), plan
    M, (row_ptr, col_idx, *_x) = om.layout(n_out, n_in, b, ms)
    nnzb = int(M.sum())
    W, Wr = synth.draw((nnzb, b, b), 0.02, 0, 2, "bf16")
    raw = dict(inp["raw"], W=Wr)
    out, _L, kt = _run_gpu_dev(n_out, n_in, b, ms, T, r, "bf16", raw, timing=True)
    splits = sum(int(plan[k] > 1) for k in ("lowrank_t_split", "lowrank_s_split", "tn_split"))
    gather = 2 * int(b == 32)  # b = 32: pair-block gather and scatter
    if b == 32:
        assert (plan["bwd_tile_n"], plan["bwd_direct_lds"]) == (64, 1), plan
    assert _reductions(kt) == splits + int(plan["tn_shared"] > 0) + gather, (kt, plan)

    rng = np.random.default_rng([b, 77])
    edges = [0, 1, 127, 128, 255, 256, 511, 512, T // 2 - 1, T // 2, T - 512, T - 1]
    rows = np.unique(np.concatenate([edges, rng.integers(0, T, 20)]))
    Wd = ol.unpack(W, row_ptr, col_idx, n_out // b, n_in // b, b)
    Mel = om.element_mask(M, b)
    X, U, V, dY = inp["X"], inp["U"], inp["V"], inp["dY"]

    Y_ref, Tl_ref = ol.forward(X[rows], Wd, U, V)
    g_rows = ol.backward(X[rows], Wd, Mel, dY[rows], U, V)
    sel = lambda t: to_host(t[torch_cuda().as_tensor(rows, device="cuda")])
    check_close("Y[rows]", sel(out["Y"]), Y_ref, "bf16")
    check_close("T_lr[rows]", sel(out["T_lr"]), Tl_ref, "bf16")
    check_close("dX[rows]", sel(out["dX"]), g_rows["dX"], "bf16")

    # Kept blocks of dW: first and last of the CSR order and random ones.
    blks = np.unique(np.concatenate([[0, nnzb - 1], rng.integers(0, nnzb, 22)]))
    dW_got = to_host(out["dW"][torch_cuda().as_tensor(blks, device="cuda")])
    blk_row = np.searchsorted(row_ptr, blks, side="right") - 1
    dW_ref = np.empty((len(blks), b, b))
    for q, (p, i) in enumerate(zip(blks, blk_row)):
        j = col_idx[p]
        I, J = slice(i * b, (i + 1) * b), slice(j * b, (j + 1) * b)
        dW_ref[q] = ol.backward(X[:, J], Wd[I, J], Mel[I, J], dY[:, I])["dW"]
    check_close("dW[blocks]", dW_got, dW_ref, "bf16")

    # All of S, dU and dV (the low-rank gradients need no dense weight).
    lr = ol.lowrank_grads(X, dY, U, V)
    for k in ("S", "dU", "dV"):
        check_close(k, to_host(out[k]), lr[k], "bf16")
