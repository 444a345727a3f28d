"""Benchmark of the Pixelated Butterfly hot path on one MI355X.

    python bench.py [--gpus 1] [--steps K] [--warmup W] [--workload NAME]

A step is one pass of the whole hot path over one batch of synthetic input
that is already resident in HBM:
  linear workloads   forward (T_lr = X V^T, Y = X (M o W)^T + T_lr U^T),
                     backward-data (S = dY U, dX = dY (M o W) + S V) and
                     backward-weight (dW on the mask, dU, dV);
  mlp_pair           both layers with the GELU epilogues, forward + backward;
  attention          block-sparse attention forward + backward.
Prints ONE JSON line.  `value` is nonzero-block TFLOP/s of the step (only the
kept b x b blocks' FLOPs of the three block-sparse products, or of the six
attention block products), the metric of the workload table.  The same line
carries the fraction of the bf16 MFMA peak, the speedup over the dense layer
of the same shape run with the library's own dense MFMA GEMM, and the CPU
oracle timed on a bounded sample of the workload.  The timed region holds
only the steps between two events; a second region repeats the steps with
the library's kernel timing hook armed (every dispatch records its own start
and end events), which gives per_kernel and the roofline entry of the
dominant kernel.
"""
from __future__ import annotations

import argparse
import json
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

import synth  # noqa: E402

METRIC = "nonzero-block TFLOP/s fwd+bwd and % bf16 MFMA peak; speedup vs dense GEMM"
PEAK_BF16_TFLOPS = 2500.0   # MI355X dense bf16 MFMA (no sparsity)
PEAK_FP32_TFLOPS = 157.3
PEAK_HBM_GBS = 8000.0
RIDGE_BF16 = PEAK_BF16_TFLOPS * 1e12 / (PEAK_HBM_GBS * 1e9)


def parse():
    p = argparse.ArgumentParser()
    p.add_argument("--gpus", type=int, default=1)
    p.add_argument("--steps", type=int, default=100)
    p.add_argument("--warmup", type=int, default=10)
    p.add_argument("--workload", default="linear_16384x4096_b128", choices=sorted(synth.WORKLOADS))
    p.add_argument("--no-sweep", action="store_true",
                   help="skip the block-size sweep that follows the 16384 x 4096 layer")
    p.add_argument("--no-cold", action="store_true",
                   help="skip the cold-cache pass (1 GiB written between steps)")
    p.add_argument("--no-cpu-baseline", action="store_true")
    p.add_argument("--no-dense", action="store_true")
    p.add_argument("--no-kernel-timing", action="store_true",
                   help="skip the per-kernel HIP events of the second region (no roofline entry)")
    p.add_argument("--calls-only", default="", help="comma list of calls to loop (profiling aid)")
    p.add_argument("--copy-probe", type=int, default=0, metavar="MIB",
                   help="before the steps, copy MIB MiB device to device three times: a plain "
                        "copy of known size that calibrates HBM byte counters (profiling aid)")
    return p.parse_args()


def library_source_hash():
    """sha256 over the library's sources (csrc/ and the public header): HBM
    traffic taken with counters is only reported while it still matches."""
    import hashlib
    h = hashlib.sha256()
    csrc = os.path.join(ROOT, "paper_2112_00029_amd", "csrc")
    files = sorted(os.path.join(csrc, f) for f in os.listdir(csrc)) + [os.path.join(ROOT, "include", "pixelfly.h")]
    for f in files:
        h.update(os.path.basename(f).encode())
        with open(f, "rb") as fh:
            h.update(fh.read())
    return h.hexdigest()[:16]


def measured_traffic(workload, kernel):
    """HBM bytes per launch of a kernel class from the committed counter
    summaries (lines of profiles/*.md of the form
    `traffic workload=W kernel=C bytes=B fetch=F write=X source=H`), or
    (None, reason) when none matches the current sources."""
    pdir = os.path.join(ROOT, "profiles")
    if not os.path.isdir(pdir):
        return None, "no counter summary"
    cur = library_source_hash()
    stale = False
    for f in sorted(os.listdir(pdir)):
        if not f.endswith(".md"):
            continue
        with open(os.path.join(pdir, f)) as fh:
            for line in fh:
                line = line.strip().strip("`")
                if not line.startswith("traffic "):
                    continue
                kv = dict(x.split("=", 1) for x in line.split()[1:] if "=" in x)
                if kv.get("workload") != workload or kv.get("kernel") != kernel:
                    continue
                if kv.get("source") != cur:
                    stale = True
                    continue
                return {"bytes": float(kv["bytes"]), "fetch": float(kv["fetch"]),
                        "write": float(kv["write"]), "file": f}, None
    return None, ("kernel sources changed since the counters were taken" if stale else "no counter summary")


def dev_bf16(torch, raw):
    return torch.from_numpy(raw.view(np.int16)).cuda().view(torch.bfloat16)


def dev_any(torch, raw):
    if raw.dtype == np.uint16:
        return dev_bf16(torch, raw)
    return torch.from_numpy(raw).cuda()


# Device copies of seeded inputs, shared by the workloads of one run (the
# block-size sweep draws the same X, U, V, dY for every block size).
_DEV_CACHE = {}


def dev_draw(torch, shape, std, seed, stream, dtype):
    key = (tuple(shape), float(std), seed, stream, dtype)
    if key not in _DEV_CACHE:
        _DEV_CACHE[key] = dev_any(torch, synth.draw(shape, std, seed, stream, dtype, values=False)[1])
    return _DEV_CACHE[key]


# ---------------------------------------------------------------------------
# Linear layer workloads
# ---------------------------------------------------------------------------
class Linear:
    calls = ["fwd", "bwd_data", "bwd_weight"]

    def __init__(self, torch, pf, wl, seed=0):
        self.torch, self.pf, self.wl = torch, pf, wl
        T, K, N, b, ms, r, dt = wl.T, wl.K, wl.N, wl.b, wl.max_stride, wl.r, wl.dtype
        self.L = pf.pf_layout_create(N, K, b, ms)
        pf.pf_layout_upload(self.L)
        self.nnzb = pf.pf_layout_info_get(self.L)["nnzb"]
        dr = lambda shape, std, stream: dev_draw(torch, shape, std, seed, stream, dt)
        self.X = dr((T, K), wl.std_x, 1)
        self.W = dr((self.nnzb, b, b), wl.std_w, 2)
        self.U = dr((N, r), wl.std_uv, 3)
        self.V = dr((r, K), wl.std_uv, 4)
        self.dY = dr((T, N), wl.std_dy, 5)
        tdt = torch.bfloat16 if dt == "bf16" else torch.float32
        e = lambda *s: torch.empty(*s, dtype=tdt, device="cuda")
        self.Y, self.Tl, self.S, self.dX = e(T, N), e(T, r), e(T, r), e(T, K)
        self.dW, self.dU, self.dV = torch.empty_like(self.W), e(N, r), e(r, K)
        self.wsb = pf.pf_workspace_bytes(self.L, T, r, dt)
        self.ws = torch.empty(max(self.wsb, 256), dtype=torch.uint8, device="cuda")
        self.dtype = dt

    def call(self, name):
        pf, T, r, dt = self.pf, self.wl.T, self.wl.r, self.dtype
        if name == "fwd":
            pf.pf_linear_fwd(self.L, dt, T, r, self.X, self.W, self.U, self.V, self.Y, self.Tl,
                             workspace=self.ws, ws_bytes=self.wsb)
        elif name == "bwd_data":
            pf.pf_linear_bwd_data(self.L, dt, T, r, self.dY, self.W, self.U, self.V, self.S, self.dX,
                                  workspace=self.ws, ws_bytes=self.wsb)
        else:
            pf.pf_linear_bwd_weight(self.L, dt, T, r, self.dY, self.X, self.Tl, self.S, self.dW,
                                    self.dU, self.dV, self.ws, self.wsb)

    def flops(self):
        wl = self.wl
        sparse = 3 * 2 * wl.T * self.nnzb * wl.b * wl.b
        lowrank = 3 * 2 * wl.T * wl.r * (wl.K + wl.N)
        dense = 3 * 2 * wl.T * wl.N * wl.K
        return sparse, lowrank, dense

    def kernel_work(self):
        """Algorithmic (flops, bytes) per step of each kernel class: every
        operand read once, every output written once."""
        wl, e = self.wl, (2 if self.dtype == "bf16" else 4)
        return _layer_work(wl.T, wl.K, wl.N, wl.r, self.nnzb * wl.b * wl.b, e)

    def dense_setup(self):
        torch, wl = self.torch, self.wl
        tdt = torch.bfloat16 if self.dtype == "bf16" else torch.float32
        self.Wd = torch.randn(wl.N, wl.K, dtype=tdt, device="cuda") * 0.02
        self.Yd = torch.empty(wl.T, wl.N, dtype=tdt, device="cuda")
        self.dXd = torch.empty(wl.T, wl.K, dtype=tdt, device="cuda")
        self.dWd = torch.empty(wl.N, wl.K, dtype=tdt, device="cuda")
        self.dwsb = self.pf.pf_dense_workspace_bytes(self.dtype, self.pf.PF_OP_TN, wl.N, wl.K, wl.T)
        self.dws = torch.empty(max(self.dwsb, 256), dtype=torch.uint8, device="cuda")

    def dense_step(self):
        pf, wl, dt = self.pf, self.wl, self.dtype
        pf.pf_dense_gemm(dt, pf.PF_OP_NT, wl.T, wl.N, wl.K, self.X, self.Wd, self.Yd)
        pf.pf_dense_gemm(dt, pf.PF_OP_NN, wl.T, wl.K, wl.N, self.dY, self.Wd, self.dXd)
        pf.pf_dense_gemm(dt, pf.PF_OP_TN, wl.N, wl.K, wl.T, self.dY, self.X, self.dWd,
                         self.dws, self.dwsb)

    def torch_dense_step(self):
        torch = self.torch
        torch.matmul(self.X, self.Wd.t(), out=self.Yd)
        torch.matmul(self.dY, self.Wd, out=self.dXd)
        torch.matmul(self.dY.t(), self.X, out=self.dWd)

    def cpu_baseline(self, budget_s=12.0):
        """The fp64 oracle (dense masked) on the same workload shape for a
        bounded number of tokens; rate in nonzero-block TFLOP/s."""
        from oracle import linear as ol
        from oracle import mask as om
        wl = self.wl
        M, (row_ptr, col_idx, *_x) = om.layout(wl.N, wl.K, wl.b, wl.max_stride)
        Mel = om.element_mask(M, wl.b)
        Ts = min(wl.T, 1024)
        X = synth.draw((Ts, wl.K), wl.std_x, 0, 1, wl.dtype)[0]
        W = synth.draw((int(M.sum()), wl.b, wl.b), wl.std_w, 0, 2, wl.dtype)[0]
        U = synth.draw((wl.N, wl.r), wl.std_uv, 0, 3, wl.dtype)[0]
        V = synth.draw((wl.r, wl.K), wl.std_uv, 0, 4, wl.dtype)[0]
        dY = synth.draw((Ts, wl.N), wl.std_dy, 0, 5, wl.dtype)[0]
        Wd = ol.unpack(W, row_ptr, col_idx, wl.N // wl.b, wl.K // wl.b, wl.b)
        reps, t0 = 0, time.perf_counter()
        while True:
            ol.forward(X, Wd, U, V)
            ol.backward(X, Wd, Mel, dY, U, V)
            reps += 1
            el = time.perf_counter() - t0
            if el >= budget_s or reps >= 1000:
                break
        fl = 3 * 2 * Ts * int(M.sum()) * wl.b * wl.b * reps
        return fl / el / 1e12, f"oracle fwd+bwd (fp64, dense masked) on {Ts} of {wl.T} tokens x {reps} reps, {el:.1f} s"


class MlpPair(Linear):
    calls = ["fwd1", "fwd2", "bwd_data2", "bwd_weight2", "bwd_data1", "bwd_weight1"]

    def __init__(self, torch, pf, wl, seed=0):
        self.torch, self.pf, self.wl, self.dtype = torch, pf, wl, wl.dtype
        T, K, N, b, ms, r = wl.T, wl.K, wl.N, wl.b, wl.max_stride, wl.r
        self.L1 = pf.pf_layout_create(N, K, b, ms)
        self.L2 = pf.pf_layout_create(K, N, b, ms)
        pf.pf_layout_upload(self.L1)
        pf.pf_layout_upload(self.L2)
        self.nnzb1 = pf.pf_layout_info_get(self.L1)["nnzb"]
        self.nnzb2 = pf.pf_layout_info_get(self.L2)["nnzb"]
        dr = lambda shape, st, s: dev_bf16(torch, synth.draw(shape, st, seed, s, "bf16")[1])
        self.X = dr((T, K), wl.std_x, 1)
        self.W1, self.U1, self.V1 = dr((self.nnzb1, b, b), wl.std_w, 2), dr((N, r), wl.std_uv, 3), dr((r, K), wl.std_uv, 4)
        self.W2, self.U2, self.V2 = dr((self.nnzb2, b, b), wl.std_w, 6), dr((K, r), wl.std_uv, 7), dr((r, N), wl.std_uv, 8)
        self.dY = dr((T, K), wl.std_dy, 5)
        e = lambda *s: torch.empty(*s, dtype=torch.bfloat16, device="cuda")
        self.Hpre, self.H, self.T1, self.Y, self.T2 = e(T, N), e(T, N), e(T, r), e(T, K), e(T, r)
        self.dHpre, self.S2, self.dX, self.S1 = e(T, N), e(T, r), e(T, K), e(T, r)
        self.dW1, self.dU1, self.dV1 = torch.empty_like(self.W1), e(N, r), e(r, K)
        self.dW2, self.dU2, self.dV2 = torch.empty_like(self.W2), e(K, r), e(r, N)
        self.wsb = max(pf.pf_workspace_bytes(self.L1, T, r, "bf16"), pf.pf_workspace_bytes(self.L2, T, r, "bf16"))
        self.ws = torch.empty(max(self.wsb, 256), dtype=torch.uint8, device="cuda")
        self.nnzb = self.nnzb1

    def call(self, name):
        pf, T, r, dt = self.pf, self.wl.T, self.wl.r, "bf16"
        if name == "fwd1":
            pf.pf_linear_fwd(self.L1, dt, T, r, self.X, self.W1, self.U1, self.V1, self.H, self.T1,
                             pf.PF_EPI_GELU, self.Hpre, self.ws, self.wsb)
        elif name == "fwd2":
            pf.pf_linear_fwd(self.L2, dt, T, r, self.H, self.W2, self.U2, self.V2, self.Y, self.T2,
                             workspace=self.ws, ws_bytes=self.wsb)
        elif name == "bwd_data2":
            pf.pf_linear_bwd_data(self.L2, dt, T, r, self.dY, self.W2, self.U2, self.V2, self.S2,
                                  self.dHpre, pf.PF_EPI_GELU, self.Hpre, self.ws, self.wsb)
        elif name == "bwd_weight2":
            pf.pf_linear_bwd_weight(self.L2, dt, T, r, self.dY, self.H, self.T2, self.S2, self.dW2,
                                    self.dU2, self.dV2, self.ws, self.wsb)
        elif name == "bwd_data1":
            pf.pf_linear_bwd_data(self.L1, dt, T, r, self.dHpre, self.W1, self.U1, self.V1, self.S1,
                                  self.dX, workspace=self.ws, ws_bytes=self.wsb)
        else:
            pf.pf_linear_bwd_weight(self.L1, dt, T, r, self.dHpre, self.X, self.T1, self.S1, self.dW1,
                                    self.dU1, self.dV1, self.ws, self.wsb)

    def flops(self):
        wl = self.wl
        sparse = 3 * 2 * wl.T * (self.nnzb1 + self.nnzb2) * wl.b * wl.b
        lowrank = 2 * 3 * 2 * wl.T * wl.r * (wl.K + wl.N)
        dense = 2 * 3 * 2 * wl.T * wl.N * wl.K
        return sparse, lowrank, dense

    def kernel_work(self):
        wl = self.wl
        w1 = _layer_work(wl.T, wl.K, wl.N, wl.r, self.nnzb1 * wl.b * wl.b, 2)
        w2 = _layer_work(wl.T, wl.N, wl.K, wl.r, self.nnzb2 * wl.b * wl.b, 2)
        out = {k: (w1[k][0] + w2[k][0], w1[k][1] + w2[k][1]) for k in w1}
        # GELU: the forward of layer 1 also writes the pre-activation, the
        # backward-data of layer 2 also reads it.
        gelu = 2 * wl.T * wl.N
        out["spmm_fwd"] = (out["spmm_fwd"][0], out["spmm_fwd"][1] + gelu)
        out["spmm_bwd_data"] = (out["spmm_bwd_data"][0], out["spmm_bwd_data"][1] + gelu)
        return out

    def dense_setup(self):
        torch, wl = self.torch, self.wl
        bf = dict(dtype=torch.bfloat16, device="cuda")
        self.Wd1 = torch.randn(wl.N, wl.K, **bf) * 0.02
        self.Wd2 = torch.randn(wl.K, wl.N, **bf) * 0.02
        self.Hd, self.Yd = torch.empty(wl.T, wl.N, **bf), torch.empty(wl.T, wl.K, **bf)
        self.dHd, self.dXd = torch.empty(wl.T, wl.N, **bf), torch.empty(wl.T, wl.K, **bf)
        self.dW1d, self.dW2d = torch.empty(wl.N, wl.K, **bf), torch.empty(wl.K, wl.N, **bf)
        self.dwsb = max(self.pf.pf_dense_workspace_bytes("bf16", self.pf.PF_OP_TN, wl.N, wl.K, wl.T),
                        self.pf.pf_dense_workspace_bytes("bf16", self.pf.PF_OP_TN, wl.K, wl.N, wl.T))
        self.dws = torch.empty(max(self.dwsb, 256), dtype=torch.uint8, device="cuda")

    def dense_step(self):
        pf, wl, d = self.pf, self.wl, "bf16"
        T, K, N = wl.T, wl.K, wl.N
        pf.pf_dense_gemm(d, pf.PF_OP_NT, T, N, K, self.X, self.Wd1, self.Hd)
        pf.pf_dense_gemm(d, pf.PF_OP_NT, T, K, N, self.Hd, self.Wd2, self.Yd)
        pf.pf_dense_gemm(d, pf.PF_OP_NN, T, N, K, self.dY, self.Wd2, self.dHd)
        pf.pf_dense_gemm(d, pf.PF_OP_TN, K, N, T, self.dY, self.Hd, self.dW2d, self.dws, self.dwsb)
        pf.pf_dense_gemm(d, pf.PF_OP_NN, T, K, N, self.dHd, self.Wd1, self.dXd)
        pf.pf_dense_gemm(d, pf.PF_OP_TN, N, K, T, self.dHd, self.X, self.dW1d, self.dws, self.dwsb)

    def torch_dense_step(self):
        torch = self.torch
        torch.matmul(self.X, self.Wd1.t(), out=self.Hd)
        torch.matmul(self.Hd, self.Wd2.t(), out=self.Yd)
        torch.matmul(self.dY, self.Wd2, out=self.dHd)
        torch.matmul(self.dY.t(), self.Hd, out=self.dW2d)
        torch.matmul(self.dHd, self.Wd1, out=self.dXd)
        torch.matmul(self.dHd.t(), self.X, out=self.dW1d)

    def cpu_baseline(self, budget_s=12.0):
        from oracle import linear as ol
        from oracle import mask as om
        wl = self.wl
        M1, (rp1, ci1, *_a) = om.layout(wl.N, wl.K, wl.b, wl.max_stride)
        M2, (rp2, ci2, *_b) = om.layout(wl.K, wl.N, wl.b, wl.max_stride)
        Ts = min(wl.T, 512)
        g = lambda shape, st, s: synth.draw(shape, st, 0, s, "bf16")[0]
        X, dY = g((Ts, wl.K), wl.std_x, 1), g((Ts, wl.K), wl.std_dy, 5)
        W1 = ol.unpack(g((int(M1.sum()), wl.b, wl.b), wl.std_w, 2), rp1, ci1, wl.N // wl.b, wl.K // wl.b, wl.b)
        W2 = ol.unpack(g((int(M2.sum()), wl.b, wl.b), wl.std_w, 6), rp2, ci2, wl.K // wl.b, wl.N // wl.b, wl.b)
        U1, V1 = g((wl.N, wl.r), wl.std_uv, 3), g((wl.r, wl.K), wl.std_uv, 4)
        U2, V2 = g((wl.K, wl.r), wl.std_uv, 7), g((wl.r, wl.N), wl.std_uv, 8)
        E1, E2 = om.element_mask(M1, wl.b), om.element_mask(M2, wl.b)
        reps, t0 = 0, time.perf_counter()
        while True:
            ol.mlp_pair_backward(X, W1, E1, U1, V1, W2, E2, U2, V2, dY)
            reps += 1
            el = time.perf_counter() - t0
            if el >= budget_s or reps >= 1000:
                break
        fl = 3 * 2 * Ts * (int(M1.sum()) + int(M2.sum())) * wl.b * wl.b * reps
        return fl / el / 1e12, f"oracle 2-layer fwd+bwd (fp64, dense masked) on {Ts} of {wl.T} tokens x {reps} reps, {el:.1f} s"


# ---------------------------------------------------------------------------
# Attention workload
# ---------------------------------------------------------------------------
class Attention:
    calls = ["attn_fwd", "attn_bwd"]

    def __init__(self, torch, pf, wl, seed=0):
        self.torch, self.pf, self.wl, self.dtype = torch, pf, wl, "bf16"
        B, H, S, d = wl.B, wl.H, wl.S, wl.d
        self.L = pf.pf_layout_create_attention(S, wl.b, wl.max_stride, wl.global_blocks)
        pf.pf_layout_upload(self.L)
        self.nnzb = pf.pf_layout_info_get(self.L)["nnzb"]
        dr = lambda s: dev_bf16(torch, synth.draw((B, H, S, d), 1.0, seed, s, "bf16")[1])
        self.Q, self.K, self.V, self.dO = dr(11), dr(12), dr(13), dr(14)
        self.O = torch.empty_like(self.Q)
        self.lse = torch.empty(B, H, S, dtype=torch.float32, device="cuda")
        self.dQ, self.dK, self.dV = torch.empty_like(self.Q), torch.empty_like(self.Q), torch.empty_like(self.Q)
        self.wsb = pf.pf_attn_workspace_bytes(B, H, S)
        self.ws = torch.empty(self.wsb, dtype=torch.uint8, device="cuda")
        self.scale = 1.0 / np.sqrt(d)

    def call(self, name):
        pf, wl = self.pf, self.wl
        if name == "attn_fwd":
            pf.pf_attn_fwd(self.L, wl.B, wl.H, wl.S, wl.d, self.scale, self.Q, self.K, self.V, self.O, self.lse)
        else:
            pf.pf_attn_bwd(self.L, wl.B, wl.H, wl.S, wl.d, self.scale, self.Q, self.K, self.V, self.O,
                           self.lse, self.dO, self.dQ, self.dK, self.dV, self.ws, self.wsb)

    def flops(self):
        wl = self.wl
        per = 2 * wl.b * wl.b * wl.d * self.nnzb * wl.B * wl.H
        return 6 * per, 0, 6 * 2 * wl.S * wl.S * wl.d * wl.B * wl.H

    def kernel_work(self):
        """Useful flops: two b x b x d block products per kept block in the
        forward, four in the backward (dP and dQ in the dQ kernel, dV and dK
        in the dK/dV kernel); recomputed scores are not counted."""
        wl = self.wl
        per = 2 * wl.b * wl.b * wl.d * self.nnzb * wl.B * wl.H
        t = wl.B * wl.H * wl.S * wl.d * 2
        rows = wl.B * wl.H * wl.S * 4
        return {"attn_fwd": (2 * per, 4 * t + rows),            # Q, K, V -> O, lse
                "attn_bwd_dq": (2 * per, 6 * t + 2 * rows),     # Q, K, V, O, dO, lse -> dQ, delta
                "attn_bwd_dkv": (2 * per, 6 * t + 2 * rows)}    # Q, K, V, dO, lse, delta -> dK, dV

    def dense_setup(self):
        torch, wl = self.torch, self.wl
        nb = wl.S // wl.b  # every block kept: the dense attention of the same shape
        self.Ld = self.pf.pf_layout_create_from_mask(nb, nb, wl.b, np.ones((nb, nb), bool))
        self.pf.pf_layout_upload(self.Ld)

    def dense_step(self):
        pf, wl = self.pf, self.wl
        pf.pf_attn_fwd(self.Ld, wl.B, wl.H, wl.S, wl.d, self.scale, self.Q, self.K, self.V, self.O, self.lse)
        pf.pf_attn_bwd(self.Ld, wl.B, wl.H, wl.S, wl.d, self.scale, self.Q, self.K, self.V, self.O,
                       self.lse, self.dO, self.dQ, self.dK, self.dV, self.ws, self.wsb)

    def torch_dense_step(self):
        pass

    def cpu_baseline(self, budget_s=12.0):
        from oracle import attention as oa
        from oracle import mask as om
        wl = self.wl
        M, _ = om.attention_layout(wl.S, wl.b, wl.max_stride, wl.global_blocks)
        Mel = om.element_mask(M, wl.b)
        g = lambda s: synth.draw((1, 1, wl.S, wl.d), 1.0, 0, s, "bf16")[0][0, 0]
        Q, K, V, dO = g(11), g(12), g(13), g(14)
        reps, t0 = 0, time.perf_counter()
        while True:
            oa.backward_head(Q, K, V, Mel, 1.0 / np.sqrt(wl.d), dO)
            reps += 1
            el = time.perf_counter() - t0
            if el >= budget_s or reps >= 1000:
                break
        fl = 6 * 2 * wl.b * wl.b * wl.d * int(M.sum()) * reps
        return fl / el / 1e12, f"oracle fwd+bwd (fp64, dense masked) on {reps} heads of {wl.B * wl.H}, {el:.1f} s"


# ---------------------------------------------------------------------------
# Pattern microbenchmark
# ---------------------------------------------------------------------------
class Patterns:
    """Forward block-sparse product of an N x N weight over T tokens for the
    flat block butterfly + low-rank layer selected for a 10% budget (the
    timed step) and, measured beside it, random p x p block patterns of 10%
    expected density run on their 32 x 32 block cover (appendix on
    microbenchmarking): the kernels touch every kept cover block, so a fine
    random pattern costs close to the dense product."""
    calls = ["pixelfly"]
    BLOCKS = (1, 2, 4, 8, 16, 32)
    DENSITY = 0.10

    def __init__(self, torch, pf, wl, seed=0):
        self.torch, self.pf, self.wl, self.dtype = torch, pf, wl, "bf16"
        T, n, b = wl.T, wl.N, wl.b
        sel = pf.pf_select_mask(n, n, b, self.DENSITY, 0.25)
        self.r, self.ms = sel["r"], sel["max_stride"]
        dr = lambda shape, s: dev_bf16(torch, synth.draw(shape, 0.02, seed, s, "bf16")[1])
        e = lambda *sh: torch.empty(*sh, dtype=torch.bfloat16, device="cuda")
        self.X, self.Y = dr((T, n), 1), e(T, n)
        self.cases = []
        L = pf.pf_layout_create(n, n, b, self.ms)
        pf.pf_layout_upload(L)
        nnzb = pf.pf_layout_info_get(L)["nnzb"]
        self.nnzb = nnzb
        self.cases.append(dict(name="pixelfly", block=b, L=L, nnzb=nnzb, r=self.r,
                               W=dr((nnzb, b, b), 2), U=dr((n, self.r), 3), V=dr((self.r, n), 4),
                               Tl=e(T, max(self.r, 1)),
                               expected_density=(nnzb * b * b + 2 * n * self.r) / (n * n)))
        for p in self.BLOCKS:
            E = synth.random_block_mask(n, n, p, self.DENSITY, seed)
            Lr = pf.pf_layout_create_from_element_mask(n, n, b, E)
            pf.pf_layout_upload(Lr)
            nz = pf.pf_layout_info_get(Lr)["nnzb"]
            self.cases.append(dict(name=f"random_{p}x{p}", block=p, L=Lr, nnzb=nz, r=0,
                                   W=dr((nz, b, b), 2), U=None, V=None, Tl=None,
                                   expected_density=float(E.mean())))
        self.wsb = max(pf.pf_workspace_bytes(c["L"], T, c["r"], "bf16") for c in self.cases)
        self.ws = torch.empty(max(self.wsb, 256), dtype=torch.uint8, device="cuda")

    def _fwd(self, c):
        self.pf.pf_linear_fwd(c["L"], "bf16", self.wl.T, c["r"], self.X, c["W"], c["U"], c["V"],
                              self.Y, c["Tl"] if c["r"] else None, workspace=self.ws,
                              ws_bytes=self.wsb)

    def call(self, name):
        self._fwd(next(c for c in self.cases if c["name"] == name))

    def flops(self):
        wl = self.wl
        return (2 * wl.T * self.nnzb * wl.b * wl.b, 2 * wl.T * self.r * 2 * wl.N,
                2 * wl.T * wl.N * wl.K)

    def kernel_work(self):
        wl = self.wl
        w = _layer_work(wl.T, wl.K, wl.N, self.r, self.nnzb * wl.b * wl.b, 2)
        return {k: w[k] for k in ("spmm_fwd", "lowrank_t")}

    def extra(self):
        """Latency of each pattern's forward (events around 20 launches)."""
        wl, rows = self.wl, []
        for c in self.cases:
            ms = timed(self.torch, lambda c=c: self._fwd(c), 20, 3)
            kept = 2 * wl.T * c["nnzb"] * wl.b * wl.b
            rows.append({"pattern": c["name"], "block": c["block"],
                         "expected_density": c["expected_density"],
                         "actual_density": c["nnzb"] * wl.b * wl.b / (wl.N * wl.K),
                         "ms": ms, "tflops_on_cover": kept / (ms * 1e-3) / 1e12})
        return {"patterns": rows, "pass": "forward"}

    def dense_setup(self):
        torch, wl = self.torch, self.wl
        self.Wd = torch.randn(wl.N, wl.K, dtype=torch.bfloat16, device="cuda") * 0.02

    def dense_step(self):
        wl = self.wl
        self.pf.pf_dense_gemm("bf16", self.pf.PF_OP_NT, wl.T, wl.N, wl.K, self.X, self.Wd, self.Y)

    def torch_dense_step(self):
        self.torch.matmul(self.X, self.Wd.t(), out=self.Y)

    def cpu_baseline(self, budget_s=12.0):
        from oracle import linear as ol
        from oracle import mask as om
        wl = self.wl
        M, (row_ptr, col_idx, *_x) = om.layout(wl.N, wl.K, wl.b, self.ms)
        Ts = 512
        X = synth.draw((Ts, wl.K), 0.02, 0, 1, "bf16")[0]
        W = synth.draw((int(M.sum()), wl.b, wl.b), 0.02, 0, 2, "bf16")[0]
        U = synth.draw((wl.N, self.r), 0.02, 0, 3, "bf16")[0]
        V = synth.draw((self.r, wl.K), 0.02, 0, 4, "bf16")[0]
        Wd = ol.unpack(W, row_ptr, col_idx, wl.N // wl.b, wl.K // wl.b, wl.b)
        reps, t0 = 0, time.perf_counter()
        while True:
            ol.forward(X, Wd, U, V)
            reps += 1
            el = time.perf_counter() - t0
            if el >= budget_s or reps >= 1000:
                break
        fl = 2 * Ts * int(M.sum()) * wl.b * wl.b * reps
        return fl / el / 1e12, f"oracle forward (fp64, dense masked) on {Ts} of {wl.T} tokens x {reps} reps, {el:.1f} s"


# ---------------------------------------------------------------------------
# Flat butterfly vs product form
# ---------------------------------------------------------------------------
class Butterfly:
    """Forward + backward of the flat block butterfly (one block-sparse layer
    with every stride up to the maximum; the timed step, at the workload's
    maximum stride) and, measured beside it for each maximum stride, the
    product form: a chain of factor layers I + B_k, forward through every
    factor, then backward-data and backward-weight through each in reverse.
    Appendix on benchmarking the butterfly multiply."""
    calls = ["flat"]

    def __init__(self, torch, pf, wl, seed=0):
        self.torch, self.pf, self.wl, self.dtype = torch, pf, wl, "bf16"
        T, n, b = wl.T, wl.N, wl.b
        dr = lambda shape, st, s: dev_bf16(torch, synth.draw(shape, st, seed, s, "bf16")[1])
        e = lambda *sh: torch.empty(*sh, dtype=torch.bfloat16, device="cuda")
        self.X, self.dY = dr((T, n), 1.0, 1), dr((T, n), 1.0, 5)
        self.Y, self.dX = e(T, n), e(T, n)
        self.strides = [k for k in (2, 4, 8, 16, 32) if k <= min(wl.max_stride, n // b)]
        self.flat = {}
        for ms in self.strides:
            L = pf.pf_layout_create(n, n, b, ms)
            pf.pf_layout_upload(L)
            nz = pf.pf_layout_info_get(L)["nnzb"]
            self.flat[ms] = dict(L=L, nnzb=nz, W=dr((nz, b, b), 1.0 / np.sqrt(nz * b / (n // b)), 2),
                                 dW=e(nz, b, b))
        self.fac = {}
        for k in self.strides:
            L = pf.pf_layout_create_factor(n, b, k)
            pf.pf_layout_upload(L)
            nz = 2 * (n // b)
            self.fac[k] = dict(L=L, W=dr((nz, b, b), 1.0 / np.sqrt(2 * b), 20 + k), dW=e(nz, b, b),
                               act=e(T, n), g=e(T, n))
        # The product form in one launch per pass: factors packed [L][nb][2][b][b]
        # on the stacked layout, factor inputs / output gradients saved [T][L][n].
        self.prod = {}
        for ms in self.strides:
            Lp = pf.pf_layout_create_butterfly(n, b, ms)
            pf.pf_layout_upload(Lp)
            nf = ms.bit_length() - 1
            nz = pf.pf_layout_info_get(Lp)["nnzb"]
            self.prod[ms] = dict(L=Lp, F=dr((nz, b, b), 1.0 / np.sqrt(2 * b), 40 + ms), dF=e(nz, b, b),
                                 acts=e(T, nf * n), grads=e(T, nf * n))
        self.wsb = max(pf.pf_workspace_bytes(c["L"], T, 0, "bf16")
                       for c in list(self.flat.values()) + list(self.fac.values())
                       + list(self.prod.values()))
        self.ws = torch.empty(max(self.wsb, 256), dtype=torch.uint8, device="cuda")
        self.nnzb = self.flat[self.strides[-1]]["nnzb"]

    def _flat(self, ms):
        pf, T, c = self.pf, self.wl.T, self.flat[ms]
        kw = dict(workspace=self.ws, ws_bytes=self.wsb)
        pf.pf_linear_fwd(c["L"], "bf16", T, 0, self.X, c["W"], None, None, self.Y, None, **kw)
        pf.pf_linear_bwd_data(c["L"], "bf16", T, 0, self.dY, c["W"], None, None, None, self.dX, **kw)
        pf.pf_linear_bwd_weight(c["L"], "bf16", T, 0, self.dY, self.X, None, None, c["dW"], None,
                                None, self.ws, self.wsb)

    def _product(self, ms):
        pf, T = self.pf, self.wl.T
        kw = dict(workspace=self.ws, ws_bytes=self.wsb)
        ks = [k for k in self.strides if k <= ms]
        x = self.X
        for k in ks:
            c = self.fac[k]
            pf.pf_linear_fwd(c["L"], "bf16", T, 0, x, c["W"], None, None, c["act"], None, **kw)
            x = c["act"]
        g = self.dY
        for i in reversed(range(len(ks))):
            c = self.fac[ks[i]]
            xin = self.X if i == 0 else self.fac[ks[i - 1]]["act"]
            pf.pf_linear_bwd_weight(c["L"], "bf16", T, 0, g, xin, None, None, c["dW"], None, None,
                                    self.ws, self.wsb)
            pf.pf_linear_bwd_data(c["L"], "bf16", T, 0, g, c["W"], None, None, None, c["g"], **kw)
            g = c["g"]

    def _product_kernel(self, ms):
        pf, T, c = self.pf, self.wl.T, self.prod[ms]
        pf.pf_butterfly_fwd(c["L"], T, self.X, c["F"], self.Y, c["acts"])
        pf.pf_butterfly_bwd_data(c["L"], T, self.dY, c["F"], self.dX, c["grads"])
        pf.pf_linear_bwd_weight(c["L"], "bf16", T, 0, c["grads"], c["acts"], None, None, c["dF"],
                                None, None, self.ws, self.wsb)

    def call(self, name):
        self._flat(self.strides[-1])

    def flops(self):
        wl = self.wl
        return 3 * 2 * wl.T * self.nnzb * wl.b * wl.b, 0, 3 * 2 * wl.T * wl.N * wl.K

    def kernel_work(self):
        wl = self.wl
        w = _layer_work(wl.T, wl.K, wl.N, 0, self.nnzb * wl.b * wl.b, 2)
        return {k: w[k] for k in ("spmm_fwd", "spmm_bwd_data", "sddmm")}

    def extra(self):
        rows = []
        for ms in self.strides:
            tf = timed(self.torch, lambda ms=ms: self._flat(ms), 20, 3)
            tk = timed(self.torch, lambda ms=ms: self._product_kernel(ms), 20, 3)
            tc = timed(self.torch, lambda ms=ms: self._product(ms), 20, 3)
            rows.append({"max_stride": ms, "flat_ms": tf, "product_ms": tk,
                         "product_over_flat": tk / tf, "product_chain_ms": tc,
                         "factors": len([k for k in self.strides if k <= ms])})
        return {"flat_vs_product": rows,
                "product_form": "one launch applies every factor (activation tile in LDS) "
                                "forward and backward-data, plus one launch for all factors' "
                                "gradients; product_chain_ms runs each factor as its own layer"}

    def dense_setup(self):
        torch, wl = self.torch, self.wl
        self.Wd = torch.randn(wl.N, wl.K, dtype=torch.bfloat16, device="cuda") * 0.02
        self.dWd = torch.empty(wl.N, wl.K, dtype=torch.bfloat16, device="cuda")
        self.dwsb = self.pf.pf_dense_workspace_bytes("bf16", self.pf.PF_OP_TN, wl.N, wl.K, wl.T)
        self.dws = torch.empty(max(self.dwsb, 256), dtype=torch.uint8, device="cuda")

    def dense_step(self):
        pf, wl = self.pf, self.wl
        pf.pf_dense_gemm("bf16", pf.PF_OP_NT, wl.T, wl.N, wl.K, self.X, self.Wd, self.Y)
        pf.pf_dense_gemm("bf16", pf.PF_OP_NN, wl.T, wl.K, wl.N, self.dY, self.Wd, self.dX)
        pf.pf_dense_gemm("bf16", pf.PF_OP_TN, wl.N, wl.K, wl.T, self.dY, self.X, self.dWd,
                         self.dws, self.dwsb)

    def torch_dense_step(self):
        torch = self.torch
        torch.matmul(self.X, self.Wd.t(), out=self.Y)
        torch.matmul(self.dY, self.Wd, out=self.dX)
        torch.matmul(self.dY.t(), self.X, out=self.dWd)

    def cpu_baseline(self, budget_s=12.0):
        from oracle import linear as ol
        from oracle import mask as om
        wl = self.wl
        M, (row_ptr, col_idx, *_x) = om.layout(wl.N, wl.K, wl.b, wl.max_stride)
        Mel = om.element_mask(M, wl.b)
        Ts = 1024
        X = synth.draw((Ts, wl.K), 1.0, 0, 1, "bf16")[0]
        dY = synth.draw((Ts, wl.N), 1.0, 0, 5, "bf16")[0]
        W = synth.draw((int(M.sum()), wl.b, wl.b), 0.1, 0, 2, "bf16")[0]
        Wd = ol.unpack(W, row_ptr, col_idx, wl.N // wl.b, wl.K // wl.b, wl.b)
        reps, t0 = 0, time.perf_counter()
        while True:
            ol.forward(X, Wd)
            ol.backward(X, Wd, Mel, dY)
            reps += 1
            el = time.perf_counter() - t0
            if el >= budget_s or reps >= 1000:
                break
        fl = 3 * 2 * Ts * int(M.sum()) * wl.b * wl.b * reps
        return fl / el / 1e12, f"oracle flat fwd+bwd (fp64, dense masked) on {Ts} of {wl.T} tokens x {reps} reps, {el:.1f} s"


def _layer_work(T, K, N, r, w, e):
    """(flops, bytes) per step of the kernel classes of one K -> N layer with
    w kept weight elements, r-rank factors and e-byte elements."""
    return {
        "spmm_fwd": (2 * T * (w + r * N), e * (T * K + w + T * r + N * r + T * N)),
        "spmm_bwd_data": (2 * T * (w + r * K), e * (T * N + w + T * r + r * K + T * K)),
        "sddmm": (2 * T * (w + N * r + r * K), e * (T * N + T * K + 2 * T * r + w + N * r + r * K)),
        "lowrank_t": (2 * T * K * r, e * (T * K + r * K + T * r)),   # T_lr = X V^T
        "lowrank_s": (2 * T * N * r, e * (T * N + N * r + T * r)),   # S = dY U
    }


def cpu_meta():
    """CPU model (from /proc/cpuinfo, as lscpu reports it) and the BLAS
    library numpy runs the oracle on."""
    model = None
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    model = line.split(":", 1)[1].strip()
                    break
    except OSError:
        pass
    blas = None
    try:
        from threadpoolctl import threadpool_info
        for i in threadpool_info():
            if i.get("user_api") == "blas":
                blas = f"{i.get('internal_api')} {i.get('version')} ({i.get('threading_layer', '')})"
                break
    except Exception:
        pass
    return {"cpu_model": model, "blas": blas, "host_cpus": len(os.sched_getaffinity(0))}


def blas_threads():
    try:
        from threadpoolctl import threadpool_info
        n = [i.get("num_threads", 0) for i in threadpool_info() if i.get("user_api") == "blas"]
        if n:
            return int(max(n))
    except Exception:
        pass
    return len(os.sched_getaffinity(0))


def timed(torch, fn, steps, warmup):
    for _ in range(warmup):
        fn()
    torch.cuda.synchronize()
    s, e = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    s.record()
    for _ in range(steps):
        fn()
    e.record()
    torch.cuda.synchronize()
    return s.elapsed_time(e) / steps


def measure(torch, pf, R, args, calls):
    """Warmup, the timed region (K whole steps between two events), the
    kernel-timing region and the cold-cache pass.  Returns (ms_per_step,
    per_kernel, cold_ms_per_step)."""
    for _ in range(args.warmup):
        for c in calls:
            R.call(c)
    torch.cuda.synchronize()
    start, end = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    start.record()
    for _ in range(args.steps):
        for c in calls:
            R.call(c)
    end.record()
    torch.cuda.synchronize()
    ms = start.elapsed_time(end) / args.steps

    # Kernel-timing region: the same K steps again with the library's
    # per-launch events (pf_timing_begin: each dispatch records its start and
    # end), which give per-kernel durations and the roofline entry.
    per_kernel = {}
    if not args.no_kernel_timing:
        pf.pf_timing_begin(args.steps * 8)
        for _ in range(args.steps):
            for c in calls:
                R.call(c)
        torch.cuda.synchronize()
        kt = pf.pf_timing_end()
        per_kernel = {c: {"launches_per_step": n / args.steps, "avg_ms": avg,
                          "ms_per_step": n * avg / args.steps} for c, (n, avg) in kt.items() if n}

    # Cold cache: 1 GiB written between steps (outside each step's event
    # pair) evicts the operands from the L2s and the 256 MB MALL, so every
    # step starts from HBM.
    cold = None
    if not args.no_cold:
        scratch = torch.empty(1 << 30, dtype=torch.uint8, device="cuda")
        n = max(3, min(args.steps, 20))
        evs = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))
               for _ in range(n)]
        for i in range(n):
            scratch.fill_(i & 0xff)
            evs[i][0].record()
            for c in calls:
                R.call(c)
            evs[i][1].record()
        torch.cuda.synchronize()
        cold = sum(a.elapsed_time(b) for a, b in evs) / n
        del scratch
    return ms, per_kernel, cold


def roofline(R, wl, per_kernel):
    """Roofline of the dominant kernel: the kernel class with the most time
    per step, its algorithmic work per launch over its mean launch time (HIP
    events recorded by the library around each launch, in the kernel-timing
    region, on the stream the kernel ran on)."""
    work = R.kernel_work()
    cand = {c: v for c, v in per_kernel.items() if c in work}
    if not cand:
        return None
    dom = max(cand, key=lambda c: cand[c]["ms_per_step"])
    lps, t = cand[dom]["launches_per_step"], cand[dom]["avg_ms"] * 1e-3
    fl, by = work[dom][0] / lps, work[dom][1] / lps
    ai = fl / by
    if R.dtype == "bf16" and ai >= RIDGE_BF16:
        roof = {"bound": "mfma", "achieved": fl / t / 1e12, "peak": PEAK_BF16_TFLOPS, "unit": "TFLOP/s"}
    elif R.dtype == "bf16":
        roof = {"bound": "hbm", "achieved": by / t / 1e9, "peak": PEAK_HBM_GBS, "unit": "GB/s"}
    else:  # fp32: MFMA fp32 peak vs HBM by the same ridge rule
        if ai >= PEAK_FP32_TFLOPS * 1e12 / (PEAK_HBM_GBS * 1e9):
            roof = {"bound": "mfma", "achieved": fl / t / 1e12, "peak": PEAK_FP32_TFLOPS, "unit": "TFLOP/s"}
        else:
            roof = {"bound": "hbm", "achieved": by / t / 1e9, "peak": PEAK_HBM_GBS, "unit": "GB/s"}
    roof["frac"] = roof["achieved"] / roof["peak"]
    tr, why = measured_traffic(wl.name, dom)
    roof["traffic"] = tr["bytes"] if tr else None
    if tr:
        roof["traffic_detail"] = {"fetch_bytes": tr["fetch"], "write_bytes": tr["write"],
                                  "over_algorithmic": tr["bytes"] / by, "source": "profiles/" + tr["file"]}
    else:
        roof["traffic_detail"] = why
    roof.update({"kernel": dom, "avg_launch_ms": cand[dom]["avg_ms"], "launches_per_step": lps,
                 "algorithmic_bytes_per_launch": by, "flops_per_launch": fl,
                 "flop_per_byte": ai,
                 "tflops_per_launch": fl / t / 1e12, "gbs_per_launch": by / t / 1e9})
    # Every kernel class of the step on the same footing (fraction of the
    # peak its arithmetic intensity makes it bound by).
    kinds = {}
    for c, v in cand.items():
        f, b_ = work[c][0] / v["launches_per_step"], work[c][1] / v["launches_per_step"]
        tt = v["avg_ms"] * 1e-3
        mf = R.dtype == "bf16" and f / b_ >= RIDGE_BF16
        kinds[c] = {"bound": "mfma" if mf else "hbm",
                    "frac": (f / tt / 1e12 / PEAK_BF16_TFLOPS) if mf else (b_ / tt / 1e9 / PEAK_HBM_GBS),
                    "tflops": f / tt / 1e12, "gbs": b_ / tt / 1e9}
    roof["per_kernel_frac"] = kinds
    return roof


def config_of(wl, R):
    cfg = {"workload": wl.name}
    if wl.kind == "attention":
        cfg.update(B=wl.B, H=wl.H, S=wl.S, d=wl.d, b=wl.b, max_stride=wl.max_stride,
                   global_blocks=wl.global_blocks)
    elif wl.kind == "butterfly":
        cfg.update(T=wl.T, K=wl.K, N=wl.N, b=wl.b, max_stride=wl.max_stride, r=0)
    elif wl.kind == "patterns":
        cfg.update(T=wl.T, K=wl.K, N=wl.N, b=wl.b, max_stride=R.ms, r=R.r, budget=Patterns.DENSITY)
    else:
        cfg.update(T=wl.T, K=wl.K, N=wl.N, b=wl.b, max_stride=wl.max_stride, r=wl.r)
    return cfg


def run_workload(torch, pf, args, name, dense=None, cpu=True):
    """One workload: its measurement, dense comparator and CPU baseline.
    dense: (in-library, torch) ms per step already measured at this dense
    shape (the block-size sweep shares it), else measured here."""
    wl = synth.WORKLOADS[name]
    R = {"linear": Linear, "mlp_pair": MlpPair, "attention": Attention,
         "patterns": Patterns, "butterfly": Butterfly}[wl.kind](torch, pf, wl)
    calls = [c for c in args.calls_only.split(",") if c] or R.calls
    if "dense" in calls:  # profiling aid: the dense comparator step as one call
        R.dense_setup()
        base_call = R.call
        R.call = lambda c: R.dense_step() if c == "dense" else base_call(c)
    ms, per_kernel, cold = measure(torch, pf, R, args, calls)
    if args.calls_only:
        return {"calls_only": calls, "ms_per_step": ms, "per_kernel": per_kernel}, R

    sparse, lowrank, dense_fl = R.flops()
    value = sparse / (ms * 1e-3) / 1e12
    peak = PEAK_BF16_TFLOPS if R.dtype == "bf16" else PEAK_FP32_TFLOPS
    if dense is None:
        dense_ms = torch_ms = None
        if not args.no_dense:
            R.dense_setup()
            dense_ms = timed(torch, R.dense_step, max(5, args.steps // 4), 3)
            if wl.kind != "attention":
                torch_ms = timed(torch, R.torch_dense_step, max(5, args.steps // 4), 3)
    else:
        dense_ms, torch_ms = dense
    best_dense = min(x for x in (dense_ms, torch_ms) if x) if (dense_ms or torch_ms) else None
    extra = R.extra() if hasattr(R, "extra") else {}

    cpu_b = None
    if cpu and not args.no_cpu_baseline:
        v, sample = R.cpu_baseline()
        cpu_b = {"value": v, "unit": "TFLOP/s", "cores": blas_threads(), "kind": "oracle",
                 "sample": sample, **cpu_meta()}

    out = {
        "metric": METRIC, "value": value, "unit": "TFLOP/s", "n_gpus": 1, "steps": args.steps,
        "warmup": args.warmup, "ms_per_step": ms, "higher_is_better": True, "scaling": "weak",
        "vs_baseline": None, "dtype": R.dtype, "data": "synthetic (seeded, shapes of the workload)",
        "config": config_of(wl, R),
        "pct_peak": 100.0 * value / peak,
        "useful_tflops_incl_lowrank": (sparse + lowrank) / (ms * 1e-3) / 1e12,
        "cold_ms_per_step": cold,
        "cold_value": (sparse / (cold * 1e-3) / 1e12) if cold else None,
        # Speedup over the faster of the two dense steps of the same shape:
        # the library's own MFMA GEMM and torch.matmul (hipBLASLt).
        "speedup_vs_dense": (best_dense / ms) if best_dense else None,
        "speedup_vs_library_dense": (dense_ms / ms) if dense_ms else None,
        "speedup_vs_torch_dense": (torch_ms / ms) if torch_ms else None,
        "dense_ms_per_step": dense_ms,
        "dense_tflops": (dense_fl / (dense_ms * 1e-3) / 1e12) if dense_ms else None,
        "torch_dense_ms_per_step": torch_ms,
        "torch_dense_tflops": (dense_fl / (torch_ms * 1e-3) / 1e12) if torch_ms else None,
        "per_kernel": per_kernel,
        "roofline": roofline(R, wl, per_kernel),
        "cpu_baseline": cpu_b,
    }
    out.update(extra)
    return out, R


def main():
    args = parse()
    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) > 1:
        print("bench.py runs on one GPU only: this build has no multi-GPU path "
              "(see the sharding design notes); use --gpus 1", file=sys.stderr)
        sys.exit(2)
    import torch
    from paper_2112_00029_amd import pixelfly as pf
    assert torch.cuda.is_available(), "bench.py needs a GPU"

    if args.copy_probe:
        n = args.copy_probe << 20
        src = torch.ones(n, dtype=torch.uint8, device="cuda")
        dst = torch.empty_like(src)
        torch.cuda.synchronize()
        for _ in range(3):
            dst.copy_(src)
        torch.cuda.synchronize()
        del src, dst

    out, R = run_workload(torch, pf, args, args.workload)
    if args.calls_only:
        print(json.dumps(out))
        return
    # The 16384 x 4096 layer is quoted as a sweep over the block size (the
    # MFMA-utilisation curve): the other two block sizes run in the same
    # process on the same inputs and the same dense comparator.
    sweep_of = {f"linear_16384x4096_b{b}": b for b in (128, 64, 32)}
    if args.workload in sweep_of and not args.no_sweep:
        dense = (out["dense_ms_per_step"], out["torch_dense_ms_per_step"])
        rows = [{"b": sweep_of[args.workload], "workload": args.workload,
                 "ms_per_step": out["ms_per_step"], "value": out["value"],
                 "pct_peak": out["pct_peak"], "cold_ms_per_step": out["cold_ms_per_step"],
                 "speedup_vs_dense": out["speedup_vs_dense"],
                 "dominant": out["roofline"] and {k: out["roofline"][k] for k in ("kernel", "bound", "frac")}}]
        del R
        for name in sweep_of:
            if name == args.workload:
                continue
            o, R2 = run_workload(torch, pf, args, name, dense=dense, cpu=False)
            rows.append({"b": sweep_of[name], "workload": name, "ms_per_step": o["ms_per_step"],
                         "value": o["value"], "pct_peak": o["pct_peak"],
                         "cold_ms_per_step": o["cold_ms_per_step"],
                         "speedup_vs_dense": o["speedup_vs_dense"],
                         "useful_tflops_incl_lowrank": o["useful_tflops_incl_lowrank"],
                         "per_kernel": o["per_kernel"],
                         "dominant": o["roofline"] and {k: o["roofline"][k] for k in ("kernel", "bound", "frac")}})
            del R2
        out["block_size_sweep"] = sorted(rows, key=lambda r: -r["b"])
    print(json.dumps(out))


if __name__ == "__main__":
    main()
