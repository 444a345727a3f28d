"""The allocation-free attention backward (pf_attn_bwd_noalloc) against the
workspace form pf_attn_bwd: same kernels, same inputs, so every output must
be bit-identical; two calls in a row, the second on a smaller input (the
device scratch keeps the first call's contents in between)."""
import numpy as np
import pytest

import synth
from tests._gpu_util import to_dev, torch_cuda


def _case(pf, torch, B, H, S, ms, g, seed):
    d = 64
    print(f"[noalloc] B={B} H={H} S={S} ms={ms} global_blocks={g} seed={seed}", flush=True)
    L = pf.pf_layout_create_attention(S, 64, ms, g)
    pf.pf_layout_upload(L)
    t = {k: to_dev(synth.draw((B, H, S, d), 1.0, seed, sid, "bf16", values=False)[1])
         for k, sid in (("Q", 11), ("K", 12), ("V", 13), ("dO", 14))}
    scale = 1.0 / np.sqrt(d)
    O = torch.empty_like(t["Q"])
    lse = torch.empty((B, H, S), dtype=torch.float32, device="cuda")
    pf.pf_attn_fwd(L, B, H, S, d, scale, t["Q"], t["K"], t["V"], O, lse)
    ref = [torch.empty_like(O) for _ in range(3)]
    wsb = pf.pf_attn_workspace_bytes(B, H, S)
    ws = torch.empty(wsb, dtype=torch.uint8, device="cuda")
    pf.pf_attn_bwd(L, B, H, S, d, scale, t["Q"], t["K"], t["V"], O, lse, t["dO"], *ref, ws, wsb)
    got = [torch.full_like(O, float("nan")) for _ in range(3)]
    pf.pf_attn_bwd_noalloc(L, B, H, S, d, scale, t["Q"], t["K"], t["V"], O, lse, t["dO"], *got)
    torch.cuda.synchronize()
    for name, a, b in zip(("dQ", "dK", "dV"), got, ref):
        same = torch.equal(a.view(torch.int16), b.view(torch.int16))
        print(f"  {name}: bit-identical={same}", flush=True)
        assert same, name


@pytest.mark.gpu
def test_noalloc_matches_workspace_form_twice():
    torch = torch_cuda()
    from paper_2112_00029_amd import pixelfly as pf
    _case(pf, torch, 2, 3, 2048, 64, 1, seed=4)   # global stripes: grouped + plain kernels
    _case(pf, torch, 1, 2, 512, 8, 0, seed=5)     # smaller, second call on the same scratch


def test_noalloc_rejects_rows_beyond_scratch():
    """B * H * Sq above 2^22 rows: refused on the host before any device
    work (the layout need not even be uploaded)."""
    from paper_2112_00029_amd import pixelfly as pf
    L = pf.pf_layout_create_attention(4096, 64, 64, 0)
    fake = 1 << 40  # 16-byte aligned, never dereferenced
    with pytest.raises(pf.PixelflyError) as ei:
        pf.pf_attn_bwd_noalloc(L, 64, 17, 4096, 64, 0.125, *([fake] * 9))
    assert ei.value.status == pf.PF_ERR_UNSUPPORTED
    assert "scratch" in pf.pf_last_error()
