"""GPU parity of the butterfly product form (Section 3.2: a product of
factors with the support of I + B_k, largest stride leftmost) run as a chain
of block-sparse layers on pf_layout_create_factor layouts, against the dense
product of the same factors: forward, input gradient through the chain, and
the gradient of the last factor on its blocks.  bf16, rel. Frobenius <= 2e-2
(every link stores its activation in bf16)."""
import numpy as np
import pytest

import synth
from oracle import linear as ol
from oracle import mask as om
from tests._gpu_util import TOL, check_close, empty, rel_fro, to_dev, to_host, torch_cuda

pytestmark = pytest.mark.gpu


@pytest.mark.parametrize("n,b,ms,T", [(1024, 32, 8, 300), (1024, 32, 32, 2048), (512, 64, 8, 130)])
def test_product_chain(n, b, ms, T):
    torch = torch_cuda()
    from paper_2112_00029_amd import pixelfly as pf
    print(f"[butterfly] n={n} b={b} max_stride={ms} T={T}", flush=True)
    nb = n // b
    ks = [k for k in (2, 4, 8, 16, 32, 64, 128) if k <= min(ms, nb)]
    X, Xr = synth.draw((T, n), 1.0, 3, 1, "bf16")
    dY, dYr = synth.draw((T, n), 1.0, 3, 5, "bf16")
    F, layouts, Wdev = {}, {}, {}
    for i, k in enumerate(ks):
        S = om.factor_matrix_support(nb, k)
        row_ptr, col_idx, *_r = om.block_csr(S)
        P, Pr = synth.draw((2 * nb, b, b), 1.0 / np.sqrt(2 * b), 3, 20 + i, "bf16")
        F[k] = ol.unpack(P, row_ptr, col_idx, nb, nb, b)
        L = pf.pf_layout_create_factor(n, b, k)
        pf.pf_layout_upload(L)
        layouts[k], Wdev[k] = L, to_dev(Pr)
    wsb = max(pf.pf_workspace_bytes(layouts[k], T, 0, "bf16") for k in ks)
    ws = torch.empty(max(wsb, 256), dtype=torch.uint8, device="cuda")
    acts = [to_dev(Xr)]
    for k in ks:  # x <- x F_k^T, smallest stride first
        y = empty((T, n), "bf16")
        pf.pf_linear_fwd(layouts[k], "bf16", T, 0, acts[-1], Wdev[k], None, None, y, None,
                         workspace=ws, ws_bytes=wsb)
        acts.append(y)
    g = to_dev(dYr)
    dF_last = None
    for i, k in reversed(list(enumerate(ks))):
        if i == len(ks) - 1:
            dF_last = empty((2 * nb, b, b), "bf16")
            pf.pf_linear_bwd_weight(layouts[k], "bf16", T, 0, g, acts[i], None, None, dF_last,
                                    None, None, ws, wsb)
        gx = empty((T, n), "bf16")
        pf.pf_linear_bwd_data(layouts[k], "bf16", T, 0, g, Wdev[k], None, None, None, gx,
                              workspace=ws, ws_bytes=wsb)
        g = gx
    torch.cuda.synchronize()
    M = np.eye(n)
    for k in reversed(ks):
        M = M @ F[k]  # F_kmax ... F_2
    x_prev = X.copy()
    for k in ks[:-1]:
        x_prev = x_prev @ F[k].T
    S_last = om.element_mask(om.factor_matrix_support(nb, ks[-1]), b)
    row_ptr, col_idx, *_r = om.block_csr(om.factor_matrix_support(nb, ks[-1]))
    ref = {"Y": X @ M.T, "dX": dY @ M, "dF_last": ol.pack((dY.T @ x_prev) * S_last, row_ptr, col_idx, nb, b)}
    got = {"Y": to_host(acts[-1]), "dX": to_host(g), "dF_last": to_host(dF_last)}
    for key in ref:
        check_close(key, got[key], ref[key], "bf16")


@pytest.mark.parametrize("n,ms,T", [(1024, 32, 2048), (1024, 8, 300), (1024, 2, 33),
                                    (2048, 16, 520)])
def test_product_kernel(n, ms, T):
    """The one-launch product form (pf_butterfly_fwd / pf_butterfly_bwd_data,
    b = 32) and every factor's gradient in one masked product on the stacked
    layout, against the oracle's product layer: output, input gradient, each
    factor's gradient, and the saved factor inputs and output gradients."""
    from oracle import butterfly as ob
    torch = torch_cuda()
    from paper_2112_00029_amd import pixelfly as pf
    b = 32
    nb, L = n // b, ms.bit_length() - 1
    print(f"[butterfly product] n={n} max_stride={ms} factors={L} T={T}", flush=True)
    X, Xr = synth.draw((T, n), 1.0, 4, 1, "bf16")
    dY, dYr = synth.draw((T, n), 1.0, 4, 5, "bf16")
    P, Pr = synth.draw((L * nb * 2, b, b), 1.0 / np.sqrt(2 * b), 4, 30, "bf16")
    Fd, Sd = [], []
    for f in range(L):
        Sb = om.factor_matrix_support(nb, 2 ** (f + 1))
        row_ptr, col_idx, *_r = om.block_csr(Sb)
        Fd.append(ol.unpack(P[f * 2 * nb:(f + 1) * 2 * nb], row_ptr, col_idx, nb, nb, b))
        Sd.append(om.element_mask(Sb, b))
    Lp = pf.pf_layout_create_butterfly(n, b, ms)
    pf.pf_layout_upload(Lp)
    x, dy, F = to_dev(Xr), to_dev(dYr), to_dev(Pr)
    Y, dX = empty((T, n), "bf16"), empty((T, n), "bf16")
    acts, grads = empty((T, L * n), "bf16"), empty((T, L * n), "bf16")
    dF = empty((L * nb * 2, b, b), "bf16")
    pf.pf_butterfly_fwd(Lp, T, x, F, Y, acts)
    pf.pf_butterfly_bwd_data(Lp, T, dy, F, dX, grads)
    wsb = pf.pf_workspace_bytes(Lp, T, 0, "bf16")
    ws = torch.empty(max(wsb, 256), dtype=torch.uint8, device="cuda")
    pf.pf_linear_bwd_weight(Lp, "bf16", T, 0, grads, acts, None, None, dF, None, None, ws, wsb)
    torch.cuda.synchronize()

    Yr, xs = ob.product_layer_forward(X, Fd)
    dXr, dFr, gs = ob.product_layer_backward(xs, Fd, Sd, dY)
    check_close("Y", to_host(Y), Yr, "bf16")
    check_close("dX", to_host(dX), dXr, "bf16")
    A, G, D = to_host(acts), to_host(grads), to_host(dF)
    for f in range(L):
        check_close(f"x_{f}", A[:, f * n:(f + 1) * n], xs[f], "bf16")
        check_close(f"g_{f + 1}", G[:, f * n:(f + 1) * n], gs[f], "bf16")
        Sb = om.factor_matrix_support(nb, 2 ** (f + 1))
        row_ptr, col_idx, *_r = om.block_csr(Sb)
        check_close(f"dF_{f + 1}", D[f * 2 * nb:(f + 1) * 2 * nb],
                    ol.pack(dFr[f], row_ptr, col_idx, nb, b), "bf16")
