"""GPU parity of the in-library dense comparator GEMM (NT, NN, TN) against
numpy float64 matmul on the same bf16 / fp32 inputs."""
import numpy as np
import pytest

import synth
from tests._gpu_util import check_close, empty, to_dev, to_host, torch_cuda

pytestmark = pytest.mark.gpu


@pytest.mark.parametrize("op", ["NT", "NN", "TN"])
@pytest.mark.parametrize("M,N,K,dtype", [(4096, 3072, 768, "bf16"), (2112, 512, 256, "bf16"),
                                         (8192, 4224, 256, "bf16"),
                                         (320, 192, 128, "bf16"),
                                         (256, 128, 200, "bf16"), (192, 256, 128, "fp32")])
def test_dense(op, M, N, K, dtype):
    torch = torch_cuda()
    from paper_2112_00029_amd import pixelfly as pf
    print(f"[dense] {op} M={M} N={N} K={K} {dtype}", flush=True)
    shapes = {"NT": ((M, K), (N, K)), "NN": ((M, K), (K, N)), "TN": ((K, M), (K, N))}[op]
    A, Ar = synth.draw(shapes[0], 1.0, 0, 21, dtype)
    B, Br = synth.draw(shapes[1], 1.0, 0, 22, dtype)
    C = empty((M, N), dtype)
    opc = {"NT": pf.PF_OP_NT, "NN": pf.PF_OP_NN, "TN": pf.PF_OP_TN}[op]
    wsb = pf.pf_dense_workspace_bytes(dtype, opc, M, N, K)
    ws = torch.empty(max(wsb, 256), dtype=torch.uint8, device="cuda")
    if op != "TN" and K % 64:
        # NT / NN step over K in whole 64-wide steps: the call refuses the
        # shape on the host and enqueues nothing.
        with pytest.raises(pf.PixelflyError) as ei:
            pf.pf_dense_gemm(dtype, opc, M, N, K, to_dev(Ar), to_dev(Br), C, ws, wsb)
        assert ei.value.status == pf.PF_ERR_UNSUPPORTED
        return
    pf.pf_dense_gemm(dtype, opc, M, N, K, to_dev(Ar), to_dev(Br), C, ws, wsb)
    torch.cuda.synchronize()
    ref = {"NT": lambda: A @ B.T, "NN": lambda: A @ B, "TN": lambda: A.T @ B}[op]()
    check_close("C", to_host(C), ref, dtype)
