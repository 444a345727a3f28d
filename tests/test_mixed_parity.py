"""GPU parity of the layer with the learnable mixing weight gamma (Section
3.3, model sparsification: W = gamma B + (1 - gamma) U V^T) against the fp64
oracle: forward, backward-data and backward-weight incl. dgamma, through the
C ABI.  Outputs: relative Frobenius error (bf16 <= 2e-2, fp32 <= 1e-5);
dgamma: absolute error over the size of its two terms, same bounds; repeat
calls give the same dgamma bit for bit (fixed summation order)."""
import numpy as np
import pytest

import synth
from oracle import linear as ol
from oracle import mask as om
from tests._gpu_util import TOL, check_close, empty, rel_fro, to_dev, to_host, torch_cuda
from tests.test_linear_parity import _inputs

pytestmark = pytest.mark.gpu

CASES = [
    # (n_out, n_in, b, max_stride, T, r, dtype, gamma, epi)
    pytest.param(3072, 768, 32, 16, 600, 96, "bf16", 0.3, 0, id="fc1_T600_g0.3"),
    pytest.param(3072, 768, 32, 16, 4096, 96, "bf16", 0.7, 0, id="fc1_T4096_g0.7"),
    pytest.param(3072, 768, 32, 16, 300, 96, "bf16", 1.0, 0, id="fc1_g1"),
    pytest.param(3072, 768, 32, 16, 300, 96, "bf16", 0.0, 0, id="fc1_g0"),
    pytest.param(4096, 1024, 64, 16, 2100, 128, "bf16", 0.6, 1, id="b64_wide_gelu_g0.6"),
    pytest.param(1024, 4096, 64, 16, 520, 128, "bf16", 0.45, 0, id="b64_fc2_g0.45"),
    pytest.param(4096, 4096, 128, 32, 2048, 128, "bf16", 0.8, 0, id="b128_tall_g0.8"),
    pytest.param(1024, 1024, 32, 32, 256, 32, "fp32", 0.25, 0, id="fp32_g0.25"),
    # b = 32 backward-data on 64-wide pair tiles, GELU epilogues
    pytest.param(2048, 1024, 32, 16, 4100, 64, "bf16", 0.4, 1, id="b32_pairs_gelu_g0.4"),
]


@pytest.mark.parametrize("n_out,n_in,b,ms,T,r,dtype,gamma,epi", CASES)
def test_mixed_parity(n_out, n_in, b, ms, T, r, dtype, gamma, epi):
    torch = torch_cuda()
    from paper_2112_00029_amd import pixelfly as pf
    print(f"[mixed] n_out={n_out} n_in={n_in} b={b} T={T} r={r} {dtype} gamma={gamma} epi={epi}",
          flush=True)
    std = (1.0, 1.0 / np.sqrt(6 * 32), 1.0 / 32, 1.0) if dtype == "fp32" else (0.02,) * 4
    inp = _inputs(n_out, n_in, b, ms, T, r, dtype, std=std)
    L = pf.pf_layout_create(n_out, n_in, b, ms)
    pf.pf_layout_upload(L)
    d = {k: to_dev(v) for k, v in inp["raw"].items()}
    Y, Tl, S, dX = empty((T, n_out), dtype), empty((T, r), dtype), empty((T, r), dtype), empty((T, n_in), dtype)
    Ypre = empty((T, n_out), dtype) if epi else None
    dW, dU, dV = empty(tuple(d["W"].shape), dtype), empty((n_out, r), dtype), empty((r, n_in), dtype)
    dg = torch.zeros(4, dtype=torch.float32, device="cuda")
    wsb = pf.pf_workspace_bytes(L, T, r, dtype)
    ws = torch.empty(max(wsb, 256), dtype=torch.uint8, device="cuda")
    pf.pf_linear_fwd_mixed(L, dtype, T, r, gamma, d["X"], d["W"], d["U"], d["V"], Y, Tl,
                           pf.PF_EPI_GELU if epi else pf.PF_EPI_NONE, Ypre, ws, wsb)
    pf.pf_linear_bwd_data_mixed(L, dtype, T, r, gamma, d["dY"], d["W"], d["U"], d["V"], S, dX,
                                workspace=ws, ws_bytes=wsb)
    pf.pf_linear_bwd_weight_mixed(L, dtype, T, r, gamma, d["dY"], d["X"], d["W"], Tl, S, dW, dU,
                                  dV, dg, ws, wsb)
    torch.cuda.synchronize()
    g1 = float(dg[0].item())
    pf.pf_linear_bwd_weight_mixed(L, dtype, T, r, gamma, d["dY"], d["X"], d["W"], Tl, S, dW, dU,
                                  dV, dg[1:], ws, wsb)
    torch.cuda.synchronize()
    assert float(dg[1].item()) == g1, "dgamma not reproducible"

    X, Wd, U, V, dY = inp["X"], inp["Wd"], inp["U"], inp["V"], inp["dY"]
    Yref, Tref = ol.forward_mixed(X, Wd, U, V, gamma)
    g = ol.backward_mixed(X, Wd, inp["Mel"], dY, U, V, gamma)
    _, (row_ptr, col_idx, *_x) = om.layout(n_out, n_in, b, ms)
    ref = {"Y": ol.gelu(Yref) if epi else Yref, "T_lr": Tref, "S": g["S"], "dX": g["dX"],
           "dW": ol.pack(g["dW"], row_ptr, col_idx, n_out // b, b), "dU": g["dU"], "dV": g["dV"]}
    got = {"Y": to_host(Y), "T_lr": to_host(Tl), "S": to_host(S), "dX": to_host(dX),
           "dW": to_host(dW), "dU": to_host(dU), "dV": to_host(dV)}
    if epi:
        ref["Y_pre"], got["Y_pre"] = Yref, to_host(Ypre)
    tol = TOL[dtype]
    for k in ref:
        if np.abs(ref[k]).max() == 0:  # gamma at an endpoint zeroes a gradient
            assert np.abs(got[k]).max() == 0, k
            continue
        check_close(k, got[k], ref[k], dtype)
    terms = abs(np.sum(dY * (X @ Wd.T))) + abs(np.sum(dY * (Tref @ U.T)))
    eg = abs(g1 - g["dgamma"]) / terms
    print(f"  dgamma: got={g1:.6e} ref={g['dgamma']:.6e} rel={eg:.3e}", flush=True)
    assert eg <= tol


@pytest.mark.parametrize("dtype,shape", [
    ("bf16", (768, 3072, 32, 16, 700, 96)),
    ("fp32", (768, 3072, 32, 16, 700, 96)),
    # 64-wide pair tiles of b = 32 (T x K >= 4M), ragged last token tile
    ("bf16", (2048, 1024, 32, 16, 4100, 64)),
], ids=["bf16", "fp32", "bf16_pairs"])
def test_mixed_bwd_data_gelu_epilogue(dtype, shape):
    """Backward-data of the mixed layer with the GELU-derivative epilogue:
    dX = (dY (gamma B) + (1 - gamma) (dY U) V) * gelu'(aux), the form the
    second layer of an MLP hands back through the activation."""
    torch = torch_cuda()
    from paper_2112_00029_amd import pixelfly as pf
    n_out, n_in, b, ms, T, r = shape
    gamma = 0.35
    print(f"[mixed-gelu] {n_out}x{n_in} b={b} T={T} r={r} {dtype} gamma={gamma}", flush=True)
    std = (1.0, 1.0 / np.sqrt(6 * 32), 1.0 / 32, 1.0) if dtype == "fp32" else (0.02,) * 4
    inp = _inputs(n_out, n_in, b, ms, T, r, dtype, std=std)
    aux, aux_raw = synth.draw((T, n_in), 1.0, 0, 9, dtype)  # pre-activation, ~N(0, 1)
    L = pf.pf_layout_create(n_out, n_in, b, ms)
    pf.pf_layout_upload(L)
    d = {k: to_dev(v) for k, v in inp["raw"].items()}
    a_dev = to_dev(aux_raw)
    S, dX = empty((T, r), dtype), empty((T, n_in), dtype)
    wsb = pf.pf_workspace_bytes(L, T, r, dtype)
    ws = torch.empty(max(wsb, 256), dtype=torch.uint8, device="cuda")
    pf.pf_linear_bwd_data_mixed(L, dtype, T, r, gamma, d["dY"], d["W"], d["U"], d["V"], S, dX,
                                pf.PF_EPI_GELU, a_dev, ws, wsb)
    torch.cuda.synchronize()
    g = ol.backward_mixed(inp["X"], inp["Wd"], inp["Mel"], inp["dY"], inp["U"], inp["V"], gamma)
    tol = TOL[dtype]
    for k, got, ref in [("S", to_host(S), g["S"]), ("dX", to_host(dX), g["dX"] * ol.gelu_grad(aux))]:
        check_close(k, got, ref, dtype)
