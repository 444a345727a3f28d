"""GPU parity of the block-sparse layer on layouts built from arbitrary
element masks through their 32 x 32 block cover (the random block patterns
of the pattern microbenchmark).  W is zero inside kept cover blocks wherever
the finer element mask is zero, so forward and backward-data reproduce the
dense product with the element mask; the weight gradient is the full
(dY^T X) on every kept cover block.  bf16, rel. Frobenius <= 2e-2."""
import numpy as np
import pytest

import synth
from oracle import linear as ol
from oracle import mask as om
from tests._gpu_util import TOL, check_close, empty, rel_fro, to_dev, to_host, torch_cuda

pytestmark = pytest.mark.gpu


@pytest.mark.parametrize("n,p,d,T", [(1024, 4, 0.1, 512), (1024, 16, 0.1, 300), (2048, 8, 0.05, 600)])
def test_cover_layout_parity(n, p, d, T):
    torch = torch_cuda()
    from paper_2112_00029_amd import pixelfly as pf
    b = 32
    print(f"[pattern] n={n} p={p} density={d} T={T}", flush=True)
    E = synth.random_block_mask(n, n, p, d, seed=1)
    C = om.block_cover(E, b, b)
    Mb = C[::b, ::b]
    row_ptr, col_idx, *_r = om.block_csr(Mb)
    X, Xr = synth.draw((T, n), 0.02, 1, 1, "bf16")
    Wfull, _ = synth.draw((n, n), 0.02, 1, 2, "bf16")
    Wd = Wfull * E
    Wblk = ol.pack(Wd, row_ptr, col_idx, n // b, b)
    Wraw = synth.bf16_bits_from_f32(Wblk.astype(np.float32))
    dY, dYr = synth.draw((T, n), 0.02, 1, 5, "bf16")
    L = pf.pf_layout_create_from_element_mask(n, n, b, E)
    pf.pf_layout_upload(L)
    x, w, dy = to_dev(Xr), to_dev(Wraw), to_dev(dYr)
    Y, dX, dW = empty((T, n), "bf16"), empty((T, n), "bf16"), empty(tuple(Wblk.shape), "bf16")
    wsb = pf.pf_workspace_bytes(L, T, 0, "bf16")
    ws = torch.empty(max(wsb, 256), dtype=torch.uint8, device="cuda")
    pf.pf_linear_fwd(L, "bf16", T, 0, x, w, None, None, Y, None, workspace=ws, ws_bytes=wsb)
    pf.pf_linear_bwd_data(L, "bf16", T, 0, dy, w, None, None, None, dX, workspace=ws, ws_bytes=wsb)
    pf.pf_linear_bwd_weight(L, "bf16", T, 0, dy, x, None, None, dW, None, None, ws, wsb)
    torch.cuda.synchronize()
    ref = {"Y": X @ Wd.T, "dX": dY @ Wd,
           "dW": ol.pack((dY.T @ X) * C, row_ptr, col_idx, n // b, b)}
    got = {"Y": to_host(Y), "dX": to_host(dX), "dW": to_host(dW)}
    for k in ref:
        print(f"  cover density {C.mean():.4f}", flush=True)
        check_close(k, got[k], ref[k], "bf16")


@pytest.mark.parametrize("b,T,r,empty_cols", [
    (32, 300, 32, (0, 9, 23)),
    (64, 520, 64, (0, 9, 23)),
    # b = 32 on pair blocks (T x K >= 4M): pair column 11 = block columns
    # 22, 23 keeps nothing, pair columns 0 and 4 keep one of their two
    (32, 5500, 64, (0, 9, 22, 23)),
])
def test_empty_block_columns_with_lowrank(b, T, r, empty_cols):
    """Block masks whose first, an inner and the last block column keep no
    block: the backward-data tiles of those columns have no kept step and
    carry only the low-rank term (dX columns = (dY U) V there)."""
    torch = torch_cuda()
    from paper_2112_00029_amd import pixelfly as pf
    nb = 24
    n = nb * b
    print(f"[empty-cols] n={n} b={b} T={T} r={r}", flush=True)
    rng = np.random.default_rng([2112, b])
    Mb = rng.random((nb, nb)) < 0.2
    Mb[:, list(empty_cols)] = False
    Mb[np.arange(nb), rng.choice([j for j in range(nb) if j not in empty_cols], nb)] = True
    assert not Mb[:, list(empty_cols)].any() and Mb.any(axis=1).all()
    row_ptr, col_idx, *_r = om.block_csr(Mb)
    nnzb = int(Mb.sum())
    X, Xr = synth.draw((T, n), 0.02, 3, 1, "bf16")
    W, Wr = synth.draw((nnzb, b, b), 0.02, 3, 2, "bf16")
    U, Ur = synth.draw((n, r), 0.02, 3, 3, "bf16")
    V, Vr = synth.draw((r, n), 0.02, 3, 4, "bf16")
    dY, dYr = synth.draw((T, n), 0.02, 3, 5, "bf16")
    Wd = ol.unpack(W, row_ptr, col_idx, nb, nb, b)
    L = pf.pf_layout_create_from_mask(nb, nb, b, Mb.astype(np.uint8))
    pf.pf_layout_upload(L)
    plan = pf.pf_linear_plan_get(L, "bf16", T, r)
    assert (plan["bwd_tile_n"] == 64) == (b == 64 or T * n >= (1 << 22)), plan
    x, w, u, v, dy = (to_dev(a) for a in (Xr, Wr, Ur, Vr, dYr))
    Y, Tl, S, dX = empty((T, n), "bf16"), empty((T, r), "bf16"), empty((T, r), "bf16"), empty((T, n), "bf16")
    dW, dU, dV = empty((nnzb, b, b), "bf16"), empty((n, r), "bf16"), empty((r, n), "bf16")
    wsb = pf.pf_workspace_bytes(L, T, r, "bf16")
    ws = torch.empty(max(wsb, 256), dtype=torch.uint8, device="cuda")
    pf.pf_linear_fwd(L, "bf16", T, r, x, w, u, v, Y, Tl, workspace=ws, ws_bytes=wsb)
    pf.pf_linear_bwd_data(L, "bf16", T, r, dy, w, u, v, S, dX, workspace=ws, ws_bytes=wsb)
    pf.pf_linear_bwd_weight(L, "bf16", T, r, dy, x, Tl, S, dW, dU, dV, ws, wsb)
    torch.cuda.synchronize()
    Yref, Tref = ol.forward(X, Wd, U, V)
    g = ol.backward(X, Wd, om.element_mask(Mb, b), dY, U, V)
    ref = {"Y": Yref, "T_lr": Tref, "S": g["S"], "dX": g["dX"],
           "dW": ol.pack(g["dW"], row_ptr, col_idx, nb, b), "dU": g["dU"], "dV": g["dV"]}
    got = {"Y": to_host(Y), "T_lr": to_host(Tl), "S": to_host(S), "dX": to_host(dX),
           "dW": to_host(dW), "dU": to_host(dU), "dV": to_host(dV)}
    for k in ref:
        check_close(k, got[k], ref[k], "bf16")
    # the empty columns of dX hold only the low-rank term
    cols = np.concatenate([np.arange(j * b, (j + 1) * b) for j in empty_cols])
    check_close("dX empty columns", got["dX"][:, cols], (g["S"] @ V)[:, cols], "bf16")
