"""GPU parity of block-sparse attention (forward and backward) against the
fp64 oracle, one head at a time.  bf16 inputs, rel. Frobenius <= 2e-2."""
import numpy as np
import pytest

import synth
from oracle import attention as oa
from oracle import mask as om
from tests._gpu_util import check_close, empty, to_dev, to_host, torch_cuda

pytestmark = pytest.mark.gpu


def _run(B, H, S, ms, heads, seed=0, check_bwd=True, g=0):
    torch = torch_cuda()
    from paper_2112_00029_amd import pixelfly as pf
    d, b = 64, 64
    print(f"[attn] B={B} H={H} S={S} ms={ms} global_blocks={g}", flush=True)
    Q, Qr = synth.draw((B, H, S, d), 1.0, seed, 11, "bf16")
    K, Kr = synth.draw((B, H, S, d), 1.0, seed, 12, "bf16")
    V, Vr = synth.draw((B, H, S, d), 1.0, seed, 13, "bf16")
    dO, dOr = synth.draw((B, H, S, d), 1.0, seed, 14, "bf16")
    scale = 1.0 / np.sqrt(d)
    L = pf.pf_layout_create_attention(S, b, ms, g)
    pf.pf_layout_upload(L)
    q, k, v, do = to_dev(Qr), to_dev(Kr), to_dev(Vr), to_dev(dOr)
    O = empty((B, H, S, d), "bf16")
    lse = torch.empty((B, H, S), dtype=torch.float32, device="cuda")
    pf.pf_attn_fwd(L, B, H, S, d, scale, q, k, v, O, lse)
    dQ, dK, dV = (empty((B, H, S, d), "bf16") for _ in range(3))
    wsb = pf.pf_attn_workspace_bytes(B, H, S)
    ws = torch.empty(wsb, dtype=torch.uint8, device="cuda")
    pf.pf_attn_bwd(L, B, H, S, d, scale, q, k, v, O, lse, do, dQ, dK, dV, ws, wsb)
    torch.cuda.synchronize()
    M, _ = om.attention_layout(S, b, ms, g)
    Mel = om.element_mask(M, b)
    Og, lg = to_host(O), lse.cpu().numpy().astype(np.float64)
    dQg, dKg, dVg = to_host(dQ), to_host(dK), to_host(dV)
    for (x, y) in heads:
        print(f"  head {(x, y)}", flush=True)
        o, l, _ = oa.forward_head(Q[x, y], K[x, y], V[x, y], Mel, scale)
        # Each query (key) row against at least the RMS row norm: gradient
        # rows of keys that receive little attention are small next to the
        # rounding of the probabilities that feed them.
        pairs = [("O", Og[x, y], o), ("lse", lg[x, y], l)]
        if check_bwd:
            rq, rk, rv = oa.backward_head(Q[x, y], K[x, y], V[x, y], Mel, scale, dO[x, y])
            pairs += [("dQ", dQg[x, y], rq), ("dK", dKg[x, y], rk), ("dV", dVg[x, y], rv)]
        for kk, gv, rv_ in pairs:
            check_close(kk, gv, rv_, "bf16", row_floor=1.0)


def test_attention_full_sequence_sampled_heads():
    """Sequence 4096, 64x64 blocks, strides < 64 (7 blocks per row); batch 2
    x 3 heads on the GPU, three heads checked against the oracle."""
    _run(2, 3, 4096, 64, heads=[(0, 0), (1, 1), (1, 2)])


def test_attention_workload_shape_sampled_heads():
    """The 8 x 12 x 4096 x 64 workload in the benchmark's launch
    configuration; two heads checked against the oracle."""
    _run(8, 12, 4096, 64, heads=[(0, 0), (7, 11)])


def test_attention_all_kept_is_dense():
    _run(1, 2, 128, 2, heads=[(0, 0), (0, 1)])


def test_attention_block_diagonal():
    _run(1, 1, 512, 1, heads=[(0, 0)])


def test_attention_small_stride():
    _run(2, 2, 1024, 4, heads=[(0, 1), (1, 0)])


def test_attention_global_component_full_sequence():
    """Butterfly + one 64-wide global stripe (appendix on method details,
    low-rank in attention): the first query block attends to all 64 key
    blocks, every query to the first key block; sequence 4096."""
    _run(2, 3, 4096, 64, heads=[(0, 0), (1, 2)], g=1)


def test_attention_global_workload_shape():
    """The attn_global_8x12x4096x64 benchmark configuration, sampled heads."""
    _run(8, 12, 4096, 64, heads=[(3, 5)], g=1)


def test_attention_global_wide_stripes_small_stride():
    _run(1, 2, 1024, 4, heads=[(0, 0), (0, 1)], g=3)


def test_attention_global_every_row():
    """Stripes as wide as the sequence: every block row is long (only the
    grouped kernels run) and the mask is dense."""
    _run(1, 2, 512, 8, heads=[(0, 0), (0, 1)], g=8)


def test_attention_global_rows_shorter_than_groups():
    """Two key blocks per row: two of the four groups of the forward / dQ
    kernels own no block and must contribute nothing."""
    _run(1, 2, 128, 2, heads=[(0, 0), (0, 1)], g=1)


def test_attention_single_block_sequence():
    """Sequence of one 64-row block (every row keeps exactly one block, the
    prefetched next-block index clamps onto it), five heads."""
    _run(1, 5, 64, 1, heads=[(0, 0), (0, 4)])


def test_attention_repeat_calls_bitwise():
    """Forward and backward of the 8 x 12 x 4096 global-stripe workload (the
    grouped and the plain kernels, many workgroups per CU) three times on the
    same inputs: every output identical to the bit.  Each output element is
    summed in a fixed order, so any difference would be a race."""
    torch = torch_cuda()
    from paper_2112_00029_amd import pixelfly as pf
    B, H, S, d, b, ms, g = 8, 12, 4096, 64, 64, 64, 1
    print(f"[attn-repeat] B={B} H={H} S={S} global_blocks={g}", flush=True)
    draw = lambda sid: to_dev(synth.draw((B, H, S, d), 1.0, 5, sid, "bf16")[1])
    q, k, v, do = draw(11), draw(12), draw(13), draw(14)
    L = pf.pf_layout_create_attention(S, b, ms, g)
    pf.pf_layout_upload(L)
    wsb = pf.pf_attn_workspace_bytes(B, H, S)
    ws = torch.empty(wsb, dtype=torch.uint8, device="cuda")
    runs = []
    for _ in range(3):
        O = empty((B, H, S, d), "bf16")
        lse = torch.empty((B, H, S), dtype=torch.float32, device="cuda")
        pf.pf_attn_fwd(L, B, H, S, d, 1.0 / np.sqrt(d), q, k, v, O, lse)
        dQ, dK, dV = (empty((B, H, S, d), "bf16") for _ in range(3))
        pf.pf_attn_bwd(L, B, H, S, d, 1.0 / np.sqrt(d), q, k, v, O, lse, do, dQ, dK, dV, ws, wsb)
        torch.cuda.synchronize()
        runs.append({"O": O, "lse": lse, "dQ": dQ, "dK": dK, "dV": dV})
    for r in runs[1:]:
        for name in runs[0]:
            assert torch.equal(r[name], runs[0][name]), name
