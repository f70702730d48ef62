#!/usr/bin/env python3
"""Benchmark of the UniSVQ 2-bit affine-lattice product on one MI355X.

Headline workload: the LLaMA-7B decoder linears at M = 1 token (q/k/v/o
4096x4096, gate/up 11008x4096, down 4096x11008), 2-bit codes in d = 4 vectors
along K with one fp16 (A, B) set per (row, 128-column group), fp16
activations.  One step = one pass of the seven linears in the decoder's launch
schedule (q+k+v in one batched launch, o, gate+up in one batched launch,
down).  Weights, activations and outputs are resident in HBM before timing
starts; the steps rotate over enough copies of the layer set (> 512 MB) that
the 256 MB Infinity Cache cannot serve them.  The K timed steps are one HIP
graph of exactly K steps, replayed once between two events.

value = algorithmic bytes per step / time per step (codes N*K/4 + affine
N*(K/128)*40 + activations + outputs; dense fp16 weights are never counted).

The same JSON line carries a sub-record per configured workload ("configs"):
one 4096x4096 layer at M = 1; the 7B set at M = 4, 16, 64 (outlier
channels); the 70B set at M = 1 and 16; prefill at M = 2048 (bf16) through
the decode path and the Eq. 9 fold, with eager and in-graph dense bf16
products of the same shapes; each with its own roofline, graph-timed
per-launch durations and, for the bandwidth-bound ones, a plain read of the
same buffers in the same launch structure ("achievable").

Prints one JSON line.
"""
from __future__ import annotations

import argparse
import ctypes
import json
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

from paper_2606_10520_amd import workloads as wl  # noqa: E402

PEAK_HBM_GBS = 8000.0      # MI355X HBM3E, datasheet
PEAK_BF16_TFLOPS = 2500.0  # MI355X dense bf16/fp16 matrix, datasheet
MALL_BYTES = 256 << 20
METRIC = "2-bit GEMV achieved HBM GB/s (% peak) + µs/layer at 7B shapes, M=1"
SUB_WORKLOADS = ("layer4096_m1", "llama7b_smallbatch_m4", "llama7b_smallbatch_m16", "llama7b_smallbatch_m64",
                 "llama70b_decode_m1", "llama70b_decode_m16", "llama7b_prefill_m2048")
CONFIG_INDEX = {"layer4096_m1": 0, "llama7b_decode_m1": 1, "llama7b_smallbatch_m4": 2, "llama7b_smallbatch_m16": 2,
                "llama7b_smallbatch_m64": 2, "llama70b_decode_m1": 3, "llama70b_decode_m16": 3,
                "llama7b_prefill_m2048": 4}


def affine_groups(K: int, affine: str) -> int:
    """Pairs of a row-shared mode: 1 per matrix, or one per 128-column group."""
    return 1 if affine == "matrix" else K // 128


def algorithmic_bytes(N: int, K: int, M: int, x_bytes: int = 2, y_bytes: int = 2, affine: str = "row_group",
                      bits: int = 2, d: int = 4) -> int:
    """Codes + affine parameters + activations + outputs.  Row-shared pairs
    are read from their packed block of records (one per two groups, a single
    one for a per-matrix pair): 80 bytes for 2-bit d = 4 codes, 160 (d = 4) or
    576 (d = 8) bytes for the format variants."""
    if affine == "row_group":
        par = N * (K // 128) * 40
    else:
        rec = 80 if (bits, d) == (2, 4) else (160 if d == 4 else 576)
        par = rec if affine == "matrix" else rec * ((K // 128 + 1) // 2)
    return N * K * bits // 8 + par + M * K * x_bytes + M * N * y_bytes


def parse():
    p = argparse.ArgumentParser()
    p.add_argument("--gpus", type=int, default=1)
    p.add_argument("--steps", type=int, default=200)
    p.add_argument("--warmup", type=int, default=20)
    p.add_argument("--workload", default=None,
                   choices=["llama7b_decode_m1", *SUB_WORKLOADS, "quantize_llama7b", "ldlq_layer4096"],
                   help="time this workload only (default: the 7B M = 1 headline plus a sub-record per "
                        "configured workload)")
    p.add_argument("--fold", action="store_true",
                   help="with --affine matrix/group and a workload above 3 tokens: the Eq. 9 fold "
                        "(unisvq_gemm_shared_fold) instead of the decode path")
    p.add_argument("--affine", default="row_group", choices=["row_group", "matrix", "group"],
                   help="row_group: one (A, B) pair per (row, 128-column group), stored with the codes (the "
                        "default workload); matrix: one pair per weight matrix shared by all rows (the paper's "
                        "setting), codes-only weights; group: one pair per 128-column group shared by the rows")
    p.add_argument("--format", default="2x4", choices=["2x4", "3x4", "2x8", "3x8"],
                   help="code bits x vector dimension; the variants (3-bit codes, d = 8) keep row-shared pairs "
                        "(--affine matrix unless group is given)")
    p.add_argument("--schedule", default="decoder", choices=["decoder", "per_layer", "single"],
                   help="decoder: q/k/v in one batched launch, o, gate/up in one batched launch, down "
                        "(how a decode step runs them); per_layer: one launch per linear; single: all "
                        "linears in one batched launch")
    p.add_argument("--rht", action="store_true",
                   help="also time the decoder step of a layer quantised in the rotated basis (Eq. 5)")
    p.add_argument("--calibrate-copy", type=int, default=0, metavar="BYTES",
                   help="only run a plain device-to-device copy of BYTES bytes 10 times (counter calibration)")
    p.add_argument("--no-schedules", action="store_true",
                   help="skip the other launch schedules, the per-launch pass and the plain-read line "
                        "(profiling runs)")
    p.add_argument("--no-sub", action="store_true", help="skip the per-config sub-records")
    p.add_argument("--no-cpu-baseline", action="store_true")
    p.add_argument("--cpu-seconds", type=float, default=10.0, help="target CPU work of the oracle sample")
    return p.parse_args()


# Sources that define each kernel (its translation unit and the headers it is built from).
KERNEL_SOURCES = {"gemv": ("gemv.hip", "gemv_kernel.hpp", "common.hpp"),
                  "gemm": ("gemm.hip", "decode.hpp", "common.hpp"),
                  "skinny": ("skinny.hip", "decode.hpp", "common.hpp")}


def kernel_source_hash(kernel: str) -> str:
    import hashlib
    h = hashlib.sha256()
    for f in KERNEL_SOURCES.get(kernel, (f"{kernel}.hip",)):
        h.update(open(os.path.join(ROOT, "paper_2606_10520_amd", "csrc", f), "rb").read())
    return h.hexdigest()[:16]


def measured_traffic(kernel: str, workload: str, schedule: str):
    """HBM bytes per launch from the committed counter summary, if it was taken
    on the current kernel source; else None."""
    path = os.path.join(ROOT, "profiles", f"{kernel}_{workload}_{schedule}_traffic.json")
    if not os.path.exists(path):
        return None
    d = json.load(open(path))
    if d.get("source_sha256_16") != kernel_source_hash(kernel):
        return None
    return d.get("hbm_bytes_per_launch")


def calibrate_copy(nbytes: int):
    import torch
    a = torch.empty(nbytes, dtype=torch.uint8, device="cuda:0")
    b = torch.empty_like(a)
    a.fill_(1)
    torch.cuda.synchronize()
    for _ in range(10):
        b.copy_(a)
    torch.cuda.synchronize()
    print(json.dumps({"calibrate_copy_bytes": nbytes, "launches": 10}), flush=True)


def workload_spec(name: str):
    """(layers, M, activation dtype, outlier channels)"""
    if name == "llama7b_decode_m1":
        return wl.LLAMA7B, 1, "f16", False
    if name == "layer4096_m1":
        return (wl.Layer("layer", 4096, 4096),), 1, "f16", False
    if name == "llama70b_decode_m1":
        return wl.LLAMA70B, 1, "f16", False
    if name == "llama70b_decode_m16":
        return wl.LLAMA70B, 16, "f16", False
    if name.startswith("llama7b_smallbatch_m"):
        return wl.LLAMA7B, int(name.rsplit("m", 1)[1]), "f16", True
    if name == "llama7b_prefill_m2048":
        return wl.PREFILL7B, 2048, "bf16", False
    raise ValueError(name)


def cpu_model() -> str:
    try:
        for line in open("/proc/cpuinfo"):
            if line.startswith("model name"):
                return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return "unknown"


PEAK_FP64_TFLOPS = 78.6   # MI355X fp64 vector, datasheet
QUANT_FLOP_PER_CANDIDATE = 44  # per component: 4 multiplies, 4 adds, 1 subtract, 1 fma (2)


def bench_quantize(args):
    """Nearest-codeword quantiser over the 7B weight shapes: W ~ N(0, 1) fp32,
    one pair per (row, group) from the paper's initial grid (Eq. 6: A = s G with
    G a random orthogonal 4x4 matrix, B = -1.5 s G 1, s = sqrt(12/15), App. A.1),
    fp16.  Reports vectors per second, the fp64 rate, and the weight SNR."""
    import torch
    import paper_2606_10520_amd.unisvq as u

    u.load()
    dev = torch.device("cuda:0")
    layers = wl.LLAMA7B
    rng = np.random.default_rng(0)
    s = np.sqrt(12.0 / 15.0)
    data = []
    for li, L in enumerate(layers):
        G = np.linalg.qr(rng.standard_normal((L.N * (L.K // 128), 4, 4)))[0]  # random orthogonal per set
        A = (s * G).astype(np.float16).reshape(L.N, L.K // 128, 4, 4)
        B = (-1.5 * s * G.sum(axis=2)).astype(np.float16).reshape(L.N, L.K // 128, 4)
        W = torch.randn(L.N, L.K, device=dev, generator=torch.Generator(device=dev).manual_seed(li))
        Ad = torch.from_numpy(A.view(np.int16)).view(torch.float16).to(dev)
        Bd = torch.from_numpy(B.view(np.int16)).view(torch.float16).to(dev)
        data.append((L, W, Ad, Bd, A, B, torch.empty((L.N, L.K), dtype=torch.uint8, device=dev)))
    lib = u.load()
    stream = torch.cuda.current_stream()

    def step():
        for (L, W, Ad, Bd, _, _, q) in data:
            st = lib.unisvq_quantize(L.N, L.K, W.data_ptr(), Ad.data_ptr(), Bd.data_ptr(), 0, q.data_ptr(),
                                     stream.cuda_stream)
            if st != 0:
                raise RuntimeError(f"unisvq_quantize failed with status {st}")

    for _ in range(max(1, args.warmup // 10)):
        step()
    torch.cuda.synchronize()
    steps = max(1, args.steps // 20)
    t0 = torch.cuda.Event(enable_timing=True)
    t1 = torch.cuda.Event(enable_timing=True)
    t0.record(stream)
    for _ in range(steps):
        step()
    t1.record(stream)
    torch.cuda.synchronize()
    ms = t0.elapsed_time(t1) / steps
    vecs = sum(L.N * L.K // 4 for L in layers)
    flops = vecs * 256 * QUANT_FLOP_PER_CANDIDATE
    ach = flops / (ms * 1e-3) / 1e12
    # weight SNR of the result on a slice of rows, decoded by the library
    L, W, Ad, Bd, A, B, q = data[0]
    rows = 64
    Wh = decoded_rows(u, q[:rows], Ad[:rows], Bd[:rows])
    W64 = W[:rows].double().cpu().numpy()
    snr = 10 * np.log10((W64 ** 2).sum() / ((W64 - Wh) ** 2).sum())
    cpu = None
    if not args.no_cpu_baseline:
        import oracle
        Wc = W[:16].cpu().numpy()
        c0 = time.perf_counter()
        n = 0
        while time.perf_counter() - c0 < min(args.cpu_seconds, 5.0) or n == 0:
            oracle.quantize(Wc, A[:16], B[:16])
            n += 1
        dt = time.perf_counter() - c0
        cpu = {"value": round(n * 16 * L.K / 4 / dt / 1e6, 4), "unit": "Mvectors/s", "cores": 1, "kind": "oracle",
               "sample": f"{n} pass(es) over 16 rows of {L.N}x{L.K}, fp64 C oracle, one thread, {dt:.1f} s"}
    out = {
        "metric": "nearest-codeword quantiser throughput (7B weight shapes)",
        "value": round(vecs / (ms * 1e-3) / 1e9, 3), "unit": "Gvectors/s", "n_gpus": 1, "steps": steps,
        "warmup": max(1, args.warmup // 10), "ms_per_step": round(ms, 4), "higher_is_better": True,
        "scaling": "weak", "vs_baseline": None, "dtype": "f64", "data": "synthetic",
        "config": {"workload": "quantize_llama7b", "layers": {L.name: [L.N, L.K] for L in layers},
                   "grid": "Eq. 6 initial grid, one pair per (row, group)", "vectors": vecs},
        "weight_snr_db": round(float(snr), 2),
        "roofline": {"bound": "alu", "achieved": round(ach, 1), "peak": PEAK_FP64_TFLOPS, "unit": "TFLOP/s",
                     "frac": round(ach / PEAK_FP64_TFLOPS, 4), "traffic": None, "kernel": "quantize_kernel",
                     "avg_launch_us": round(ms * 1e3 / len(layers), 3)},
        "cpu_baseline": cpu,
    }
    print(json.dumps(out), flush=True)


def decoded_rows(u, q, Ad, Bd):
    """W_hat of a few rows (per-(row, group) pairs), decoded by the library:
    the prefill product with identity activations returns W_hat^T (each
    decoded weight rounded once to fp16)."""
    import torch
    N, K = q.shape
    pk = u.pack(q.contiguous(), Ad.contiguous(), Bd.contiguous())
    eye = torch.eye(K, dtype=torch.float16, device=q.device)
    y = u.gemm(pk, N, K, eye, out_dtype=torch.float32)  # [K][N]
    return y.t().double().cpu().numpy()


LDLQ_FLOP_PER_FEEDBACK = 2  # one fma per (row, earlier column, column)


def bench_ldlq(args):
    """LDLQ (Eq. 7) on one 4096 x 4096 layer: W ~ N(0, 1) fp32, the paper's
    initial grid (Eq. 6) with one pair per (row, group), and a synthetic
    Hessian with coupled columns (X^T X / S, S = 2K activations sharing a
    common component, + mu I, mu = 0.01, Sec. 4.2) factorised H = U D U^T by
    unisvq_ldl (timed on its own).  Reports vectors per second, the fp64 rate,
    and the Hessian proxy loss tr(E H E^T) against plain nearest-codeword
    rounding on a slice of rows."""
    import torch
    import paper_2606_10520_amd.unisvq as u

    lib = u.load()
    dev = torch.device("cuda:0")
    N = K = 4096
    rng = np.random.default_rng(0)
    s = np.sqrt(12.0 / 15.0)
    G = np.linalg.qr(rng.standard_normal((N * (K // 128), 4, 4)))[0]
    A = (s * G).astype(np.float16).reshape(N, K // 128, 4, 4)
    B = (-1.5 * s * G.sum(axis=2)).astype(np.float16).reshape(N, K // 128, 4)
    S = 2 * K
    X = np.sqrt(0.1) * rng.standard_normal((S, K)) + np.sqrt(0.9) * rng.standard_normal((S, 1)) * rng.standard_normal((1, K))
    H = X.T @ X / S + 0.01 * np.eye(K)
    del X
    # the factorisation on the GPU (timed separately from the quantiser)
    Hd = torch.from_numpy(H).to(dev)
    Ud = torch.empty_like(Hd)
    info = torch.zeros(1, dtype=torch.int32, device=dev)
    ws_ldl = torch.empty(u.ldl_workspace_bytes(K), dtype=torch.uint8, device=dev)
    stream = torch.cuda.current_stream()

    def factor():
        st = lib.unisvq_ldl(K, Hd.data_ptr(), Ud.data_ptr(), None, info.data_ptr(), ws_ldl.data_ptr(),
                            ws_ldl.numel(), stream.cuda_stream)
        if st != 0:
            raise RuntimeError(f"unisvq_ldl failed with status {st}")

    factor()
    torch.cuda.synchronize()
    if int(info.item()) != 0:
        raise RuntimeError(f"the synthetic Hessian is not positive definite (info {int(info.item())})")
    f0 = torch.cuda.Event(enable_timing=True)
    f1 = torch.cuda.Event(enable_timing=True)
    f0.record(stream)
    for _ in range(3):
        factor()
    f1.record(stream)
    torch.cuda.synchronize()
    ldl_ms = f0.elapsed_time(f1) / 3
    U = Ud.cpu().numpy()
    W = torch.randn(N, K, device=dev, generator=torch.Generator(device=dev).manual_seed(1))
    Ad = torch.from_numpy(A.view(np.int16)).view(torch.float16).to(dev)
    Bd = torch.from_numpy(B.view(np.int16)).view(torch.float16).to(dev)
    q = torch.empty((N, K), dtype=torch.uint8, device=dev)
    ws = torch.empty(u.ldlq_workspace_bytes(N, K), dtype=torch.uint8, device=dev)

    def step():
        st = lib.unisvq_ldlq(N, K, W.data_ptr(), Ud.data_ptr(), Ad.data_ptr(), Bd.data_ptr(), 0, q.data_ptr(),
                             ws.data_ptr(), ws.numel(), stream.cuda_stream)
        if st != 0:
            raise RuntimeError(f"unisvq_ldlq failed with status {st}")

    step()
    torch.cuda.synchronize()
    steps = max(1, args.steps // 40)
    t0 = torch.cuda.Event(enable_timing=True)
    t1 = torch.cuda.Event(enable_timing=True)
    t0.record(stream)
    for _ in range(steps):
        step()
    t1.record(stream)
    torch.cuda.synchronize()
    ms = t0.elapsed_time(t1) / steps
    vecs = N * K // 4
    flops = vecs * 256 * QUANT_FLOP_PER_CANDIDATE + N * (K * K // 2) * LDLQ_FLOP_PER_FEEDBACK
    ach = flops / (ms * 1e-3) / 1e12
    # proxy loss on a slice of rows, against plain nearest-codeword rounding
    rows = 64
    q_rtn = torch.empty((rows, K), dtype=torch.uint8, device=dev)
    st = lib.unisvq_quantize(rows, K, W.data_ptr(), Ad.data_ptr(), Bd.data_ptr(), 0, q_rtn.data_ptr(),
                             stream.cuda_stream)
    if st != 0:
        raise RuntimeError(f"unisvq_quantize failed with status {st}")
    W64 = W[:rows].double().cpu().numpy()
    E_l = W64 - decoded_rows(u, q[:rows], Ad[:rows], Bd[:rows])
    E_r = W64 - decoded_rows(u, q_rtn, Ad[:rows], Bd[:rows])
    loss = lambda E: float(np.einsum("rk,kl,rl->", E, H, E))
    mse = lambda E: float((E ** 2).mean())
    cpu = None
    if not args.no_cpu_baseline:
        import oracle
        Wc = W[:2].cpu().numpy()
        c0 = time.perf_counter()
        n = 0
        while time.perf_counter() - c0 < min(args.cpu_seconds, 5.0) or n == 0:
            oracle.ldlq(Wc, U, A[:2], B[:2], threads=2)
            n += 1
        dt = time.perf_counter() - c0
        cpu = {"value": round(n * 2 * K / 4 / dt / 1e6, 5), "unit": "Mvectors/s", "cores": 2, "kind": "oracle",
               "sample": f"{n} pass(es) over 2 rows of {N}x{K}, fp64 C oracle, two threads, {dt:.1f} s"}
    out = {
        "metric": "LDLQ quantiser throughput (one 4096x4096 layer, Hessian feedback)",
        "value": round(vecs / (ms * 1e-3) / 1e6, 2), "unit": "Mvectors/s", "n_gpus": 1, "steps": steps,
        "warmup": 1, "ms_per_step": round(ms, 3), "higher_is_better": True, "scaling": "weak",
        "vs_baseline": None, "dtype": "f64", "data": "synthetic",
        "config": {"workload": "ldlq_layer4096", "N": N, "K": K,
                   "grid": "Eq. 6 initial grid, one pair per (row, group)",
                   "hessian": "X^T X / S, S = 2K, X = sqrt(0.1) Z + sqrt(0.9) common component, + 0.01 I",
                   "launches": 1 + 2 * (K // 128) - 1},
        "factorisation": {"what": "unisvq_ldl, H = U D U^T with 4 x 4 pivot blocks, fp64",
                          "ms": round(ldl_ms, 3), "launches": 1 + 3 * (K // 64) - 2,
                          "fp64_TFLOP_s": round(K ** 3 / 3 / (ldl_ms * 1e-3) / 1e12, 2)},
        "proxy_loss_over_nearest": round(loss(E_l) / loss(E_r), 4),
        "weight_mse": {"ldlq": round(mse(E_l), 5), "nearest": round(mse(E_r), 5)},
        "roofline": {"bound": "alu", "achieved": round(ach, 2), "peak": PEAK_FP64_TFLOPS, "unit": "TFLOP/s",
                     "frac": round(ach / PEAK_FP64_TFLOPS, 4), "traffic": None,
                     "kernel": "ldlq_block_kernel + ldlq_update_kernel", "avg_launch_us": None},
        "cpu_baseline": cpu,
    }
    print(json.dumps(out), flush=True)




# ---------------------------------------------------------------------------
# Product workloads: packed weight sets, launch schedules, graph timing.

class WeightSet:
    """A layer set packed on the GPU in one weight format, with enough copies
    (> 2x the 256 MB Infinity Cache) for every step to stream from HBM."""

    def __init__(self, u, torch, layers, affine="row_group", bits=2, dim=4, keep_host=False):
        self.u, self.torch = u, torch
        self.layers, self.affine, self.bits, self.dim = layers, affine, bits, dim
        self.var = (bits, dim) != (2, 4)
        self.shared = affine != "row_group"
        dev = torch.device("cuda:0")

        def dev_half(a):
            return torch.from_numpy(a.view(np.int16)).view(torch.float16).to(dev)

        self.host = []
        packed0 = []
        for li, L in enumerate(layers):
            if self.var:
                Q, A, B = wl.gen_var_weights(L.N, L.K, bits, dim, affine_groups(L.K, affine), seed=li)
                pk = u.var_pack(torch.from_numpy(Q).to(dev), dev_half(A), dev_half(B), bits, dim)
            elif self.shared:
                Q, A, B = wl.gen_shared_weights(L.N, L.K, affine_groups(L.K, affine), seed=li)
                pk = u.pack_shared(torch.from_numpy(Q).to(dev), dev_half(A), dev_half(B))
            else:
                Q, A, B = wl.gen_weights(L.N, L.K, seed=li)
                pk = u.pack(torch.from_numpy(Q).to(dev), dev_half(A), dev_half(B))
            packed0.append(pk)
            self.host.append((Q, A, B) if keep_host else None)
        self.packed_bytes = sum((u.var_codes_bytes(L.N, L.K, bits, dim) if self.var else
                                 u.codes_bytes(L.N, L.K) if self.shared else u.packed_bytes(L.N, L.K))
                                for L in layers)
        self.copies = max(2, -(-2 * MALL_BYTES // self.packed_bytes) + 1)
        self.packed = [packed0]
        for _ in range(1, self.copies):
            self.packed.append([tuple(t.clone() for t in pk) if isinstance(pk, tuple) else pk.clone()
                                for pk in packed0])
        torch.cuda.synchronize()

    def weight_buffers(self, c, li):
        """Device tensors the product streams for layer li of copy c."""
        pk = self.packed[c][li]
        return [pk[0]] if isinstance(pk, tuple) else [pk]


class Case:
    """One workload (weight set, token count, activation type) with its launch
    schedule; x and y per layer and copy."""

    def __init__(self, ws: WeightSet, M: int, xdt: str, outliers: bool, fold: bool = False):
        u, torch = ws.u, ws.torch
        self.ws, self.u, self.torch = ws, u, torch
        self.M, self.xdt, self.outliers, self.fold = M, xdt, outliers, fold
        self.lib = u.load()
        self.tdt = torch.float16 if xdt == "f16" else torch.bfloat16
        self.xcode = u.F16 if xdt == "f16" else u.BF16
        self.kernel = "gemv" if M <= 3 else "gemm"
        dev = torch.device("cuda:0")
        layers = ws.layers
        # a decoder's query, key and value projections read one activation
        # matrix (the normalised hidden state), and so do gate and up: those
        # layers share the rows of the first of them, in one device buffer
        names = [L.name for L in layers]
        lead = list(range(len(layers)))
        for grp in (("q", "k", "v"), ("gate", "up")):
            if set(grp) <= set(names):
                for n in grp[1:]:
                    lead[names.index(n)] = names.index(grp[0])
        self.x_host = [wl.gen_activations(M, L.K, seed=wl.activation_seed(li, M), dtype=xdt, outliers=outliers)
                       if lead[li] == li else None for li, L in enumerate(layers)]
        self.x_host = [self.x_host[lead[li]] for li in range(len(layers))]
        self.xs, self.ys = [], []
        for c in range(ws.copies):
            xc = [torch.from_numpy(xb.view(np.int16)).view(self.tdt).to(dev) if lead[li] == li else None
                  for li, xb in enumerate(self.x_host)]
            self.xs.append([xc[lead[li]] for li in range(len(layers))])
            self.ys.append([torch.empty((M, L.N), dtype=torch.float16, device=dev) for L in layers])
        self.set_bytes = sum(algorithmic_bytes(L.N, L.K, M, affine=ws.affine, bits=ws.bits, d=ws.dim)
                             for L in layers)
        self.flops = sum(2 * M * L.N * L.K for L in layers)
        ws_bytes = 0
        if self.kernel == "gemm" and not ws.shared and not ws.var and not fold:
            # batched launches (q+k+v, gate+up): the slices of all problems of a batch
            for grp in (layers[:3], layers[4:6], layers):
                arr = (u.GemvProblem * len(grp))(*[u.GemvProblem(L.N, L.K, None, None, None) for L in grp])
                ws_bytes = max(ws_bytes, self.lib.unisvq_gemm_batched_workspace_bytes(arr, len(grp), M, self.xcode))
        if self.kernel == "gemm":
            for L in layers:
                if ws.var:
                    need = u.var_gemm_workspace_bytes(L.N, L.K, M, self.tdt)
                elif fold:
                    need = u.gemm_fold_workspace_bytes(L.N, L.K, M)
                else:
                    need = u.gemm_workspace_bytes(L.N, L.K, M, self.tdt)
                ws_bytes = max(ws_bytes, need)
        # one workspace serves every call: the calls run in order on one stream
        self.ws_bytes = ws_bytes
        self.wsbuf = torch.empty(max(ws_bytes, 256), dtype=torch.uint8, device=dev)
        self.names = [L.name for L in layers]
        # the plain-read reference's sink: one word per wavefront of the largest launch
        self.sink = torch.zeros(2 * (self.set_bytes // 8192 + 16 * len(layers)), dtype=torch.int32, device=dev)
        torch.cuda.synchronize()

    # ---- schedules
    def batched_gemm(self):
        """unisvq_gemm_batched takes batches (q+k+v, gate+up) in one launch."""
        return self.kernel == "gemm" and not self.ws.shared and not self.ws.var and not self.fold

    def groups(self, sched):
        full_set = {"q", "k", "v", "o", "gate", "up", "down"} <= set(self.names)
        if self.kernel != "gemv" and not self.batched_gemm():
            return "per_layer", [[n] for n in self.names]
        if sched == "decoder" and full_set:
            return "decoder", [["q", "k", "v"], ["o"], ["gate", "up"], ["down"]]
        if sched == "single" and len(self.names) <= self.u.MAX_BATCH:
            return "single", [self.names]
        return "per_layer", [[n] for n in self.names]

    def calls(self, groups):
        """Per buffer copy: the step's launches, each (label, [layer indices])."""
        idx = {n: i for i, n in enumerate(self.names)}
        return [[("+".join(g), [idx[n] for n in g]) for g in groups] for _ in range(self.ws.copies)]

    def launch(self, c, lis, sptr):
        u, lib, ws, M = self.u, self.lib, self.ws, self.M
        Ls = [ws.layers[i] for i in lis]
        if len(lis) > 1 and self.kernel == "gemm":
            arr = (u.GemvProblem * len(lis))()
            for j, li in enumerate(lis):
                L = ws.layers[li]
                arr[j] = u.GemvProblem(L.N, L.K, ws.packed[c][li].data_ptr(), self.xs[c][li].data_ptr(),
                                       self.ys[c][li].data_ptr())
            return lib.unisvq_gemm_batched(arr, len(lis), M, self.xcode, u.F16, self.wsbuf.data_ptr(), self.ws_bytes,
                                           sptr)
        if len(lis) > 1:
            if ws.shared or ws.var:
                arr = (u.GemvSharedProblem * len(lis))()
                for j, li in enumerate(lis):
                    L, (pc, pa) = ws.layers[li], ws.packed[c][li]
                    arr[j] = u.GemvSharedProblem(L.N, L.K, affine_groups(L.K, ws.affine), pc.data_ptr(),
                                                 pa.data_ptr(), self.xs[c][li].data_ptr(), self.ys[c][li].data_ptr())
                if ws.var:
                    return lib.unisvq_var_gemv_batched(arr, len(lis), ws.bits, ws.dim, M, self.xcode, u.F16, sptr)
                return lib.unisvq_gemv_shared_batched(arr, len(lis), M, self.xcode, u.F16, sptr)
            arr = (u.GemvProblem * len(lis))()
            for j, li in enumerate(lis):
                L = ws.layers[li]
                arr[j] = u.GemvProblem(L.N, L.K, ws.packed[c][li].data_ptr(), self.xs[c][li].data_ptr(),
                                       self.ys[c][li].data_ptr())
            return lib.unisvq_gemv_batched(arr, len(lis), M, self.xcode, u.F16, sptr)
        li = lis[0]
        L, pk, x, y = Ls[0], ws.packed[c][li], self.xs[c][li].data_ptr(), self.ys[c][li].data_ptr()
        wsp, wsb = self.wsbuf.data_ptr(), self.ws_bytes
        if ws.var:
            pc, pa = pk
            ga = affine_groups(L.K, ws.affine)
            if self.kernel == "gemv":
                return lib.unisvq_var_gemv(L.N, L.K, ws.bits, ws.dim, ga, pc.data_ptr(), pa.data_ptr(), M, x,
                                           self.xcode, y, u.F16, sptr)
            return lib.unisvq_var_gemm(L.N, L.K, ws.bits, ws.dim, ga, pc.data_ptr(), pa.data_ptr(), M, x,
                                       self.xcode, y, u.F16, wsp, wsb, sptr)
        if ws.shared:
            pc, pa = pk
            ga = affine_groups(L.K, ws.affine)
            if self.kernel == "gemv":
                return lib.unisvq_gemv_shared(L.N, L.K, ga, pc.data_ptr(), pa.data_ptr(), M, x, self.xcode, y,
                                              u.F16, sptr)
            fn = lib.unisvq_gemm_shared_fold if self.fold else lib.unisvq_gemm_shared
            return fn(L.N, L.K, ga, pc.data_ptr(), pa.data_ptr(), M, x, self.xcode, y, u.F16, wsp, wsb, sptr)
        if self.kernel == "gemv":
            return lib.unisvq_gemv(L.N, L.K, pk.data_ptr(), M, x, self.xcode, y, u.F16, sptr)
        return lib.unisvq_gemm(L.N, L.K, pk.data_ptr(), M, x, self.xcode, y, u.F16, wsp, wsb, sptr)

    def read_only(self, c, lis, sptr):
        return self.read(c, lis, sptr, 0)

    def read_store(self, c, lis, sptr):
        return self.read(c, lis, sptr, 1)

    def read(self, c, lis, sptr, store):
        """The plain-read reference of one launch: the same weight and
        activation buffers, one launch; with `store` each wavefront also
        stores one word (about 4 bytes per KB read, of the order of the
        product's output)."""
        bufs = []
        for li in lis:
            bufs += self.ws.weight_buffers(c, li) + [self.xs[c][li]]
        arr = (self.u.ByteRange * len(bufs))()
        for j, t in enumerate(bufs):
            arr[j] = self.u.ByteRange(t.data_ptr(), (t.numel() * t.element_size()) // 16 * 16)
        return self.lib.unisvq_read_bytes(arr, len(bufs), store, self.sink.data_ptr(), self.sink.numel(), sptr)

    def run_step(self, calls, i, sptr, fn=None):
        fn = fn or self.launch
        n = len(calls)  # one entry per buffer copy
        for _, lis in calls[i % n]:
            st = fn(i % n, lis, sptr)
            if st != 0:
                raise RuntimeError(f"{self.kernel} launch failed with status {st}")

    def time_steps(self, calls, nsteps, warmup, fn=None, replays=1):
        """Warm up eagerly, capture exactly `nsteps` steps (rotating over the
        copies) in one HIP graph, replay it once untimed and then `replays`
        times, each between two events; returns ms per step (the median over
        the timed replays)."""
        torch = self.torch
        stream = torch.cuda.current_stream()
        for i in range(warmup):
            self.run_step(calls, i, stream.cuda_stream, fn)
        torch.cuda.synchronize()
        graph = torch.cuda.CUDAGraph()
        with torch.cuda.graph(graph):
            cap = torch.cuda.current_stream().cuda_stream
            for i in range(nsteps):
                self.run_step(calls, i, cap, fn)
        torch.cuda.synchronize()
        graph.replay()
        torch.cuda.synchronize()
        times = []
        for _ in range(replays):
            t0 = torch.cuda.Event(enable_timing=True)
            t1 = torch.cuda.Event(enable_timing=True)
            t0.record(stream)
            graph.replay()
            t1.record(stream)
            torch.cuda.synchronize()
            times.append(t0.elapsed_time(t1) / nsteps)
        del graph
        return sorted(times)[len(times) // 2]

    def per_launch_us(self, groups, reps):
        """Graph-timed duration of each launch of the schedule: `reps`
        back-to-back launches of that launch alone, rotating over enough
        copies of its own weights (> 2x the 256 MB Infinity Cache; extra
        copies are cloned for the measurement) that every launch streams them
        from HBM, as in the step."""
        ws, torch = self.ws, self.torch
        idx = {n: i for i, n in enumerate(self.names)}
        out = {}
        for g in groups:
            lis = [idx[n] for n in g]
            gbytes = sum(sum(t.numel() for t in ws.weight_buffers(0, li)) for li in lis)
            need = max(ws.copies, -(-2 * MALL_BYTES // max(gbytes, 1)) + 1)
            base = ws.copies
            for c in range(base, need):
                ws.packed.append([(tuple(t.clone() for t in pk) if isinstance(pk, tuple) else pk.clone())
                                  if li in lis else pk for li, pk in enumerate(ws.packed[0])])
                self.xs.append(self.xs[c % base])
                self.ys.append(self.ys[c % base])
            one = [[("+".join(g), lis)] for _ in range(need)]
            try:
                out["+".join(g)] = round(self.time_steps(one, max(reps, need), 2) * 1e3, 3)
            finally:
                del ws.packed[base:], self.xs[base:], self.ys[base:]
                torch.cuda.synchronize()
        return out


def hbm_roofline(kernel_name, bytes_per_step, launches, ms_per_step, traffic=None):
    avg_us = ms_per_step * 1e3 / launches
    bpl = bytes_per_step / launches
    ach = bpl / (avg_us * 1e-6) / 1e9
    return {"bound": "hbm", "achieved": round(ach, 1), "peak": PEAK_HBM_GBS, "unit": "GB/s",
            "frac": round(ach / PEAK_HBM_GBS, 4), "traffic": None if traffic is None else int(traffic),
            "kernel": kernel_name, "avg_launch_us": round(avg_us, 3), "bytes_per_launch": int(bpl)}


def mfma_roofline(kernel_name, flops_per_step, launches, ms_per_step, traffic=None):
    avg_us = ms_per_step * 1e3 / launches
    ach = flops_per_step / launches / (avg_us * 1e-6) / 1e12
    return {"bound": "mfma", "achieved": round(ach, 1), "peak": PEAK_BF16_TFLOPS, "unit": "TFLOP/s",
            "frac": round(ach / PEAK_BF16_TFLOPS, 4), "traffic": None if traffic is None else int(traffic),
            "kernel": kernel_name, "avg_launch_us": round(avg_us, 3)}


def product_kernel_name(case):
    if case.kernel == "gemv":
        return "gemv_kernel"
    if not case.ws.var and not case.fold and case.M <= SKINNY_MAX_M:
        return "skinny_kernel"
    if not case.ws.var and not case.fold and case.M <= 32:
        return "skinny_kernel or gemm_kernel (by launch width)"
    return "gemm_kernel"


# Largest batch the 2x4 product always sends to the small-batch kernel (from
# 17 to 32 tokens only launches of fewer than 64 tiles of 128 rows go there).
SKINNY_MAX_M = 16


def measure_case(case, sched_name, nsteps, warmup, extras=True, traffic_key=None):
    """Time one workload: the step (graph of nsteps steps), and optionally the
    per-launch durations and the plain read of the same buffers."""
    sched, groups = case.groups(sched_name)
    calls = case.calls(groups)
    ms = case.time_steps(calls, nsteps, warmup)
    rec = {"schedule": sched, "launches_per_step": len(groups), "steps": nsteps, "ms_per_step": round(ms, 5),
           "buffer_copies": case.ws.copies, "set_bytes": case.set_bytes}
    kname = product_kernel_name(case)
    bandwidth_bound = case.M <= 64
    traffic = None
    if traffic_key is not None:
        traffic = measured_traffic(kname.replace("_kernel", ""), traffic_key, sched)
    if bandwidth_bound:
        gbs = case.set_bytes / (ms * 1e-3) / 1e9
        rec.update({"value": round(gbs, 2), "unit": "GB/s", "pct_peak_hbm": round(100 * gbs / PEAK_HBM_GBS, 2)})
        rec["roofline"] = hbm_roofline(kname, case.set_bytes, len(groups), ms, traffic)
    else:
        tf = case.flops / (ms * 1e-3) / 1e12
        rec.update({"value": round(tf, 2), "unit": "TFLOP/s"})
        rec["roofline"] = mfma_roofline(kname, case.flops, len(groups), ms, traffic)
    if extras:
        rec["per_launch_us"] = case.per_launch_us(groups, max(8, min(nsteps, 60)))
        if bandwidth_bound:
            rms = case.time_steps(calls, nsteps, 2, fn=case.read_only, replays=3)
            sms = case.time_steps(calls, nsteps, 2, fn=case.read_store, replays=3)
            rec["achievable"] = {
                "what": "plain read (unisvq_read_bytes) of the same weight and activation buffers, one launch per "
                        "launch of the schedule; read_only writes nothing, read_and_store also stores one word per "
                        "wavefront (a kernel that writes any output pays a fixed end-of-launch cost); the median "
                        "of three timed replays of the graph of the same steps",
                "read_only": {"ms_per_step": round(rms, 5), "GB_per_s": round(case.set_bytes / (rms * 1e-3) / 1e9, 1),
                              "product_over_read_time": round(ms / rms, 4)},
                "read_and_store": {"ms_per_step": round(sms, 5),
                                   "GB_per_s": round(case.set_bytes / (sms * 1e-3) / 1e9, 1),
                                   "product_over_read_time": round(ms / sms, 4)}}
    return rec, calls, groups


def dense_baseline(torch, layers, M, tdt, x_host, reps):
    """Dense products of the same shapes (random bf16/fp16 weights): torch.matmul
    (hipBLASLt) eagerly, each shape timed between events, and the same
    products captured in one graph."""
    dev = torch.device("cuda:0")
    wts = [torch.randn(L.K, L.N, device=dev).to(tdt) for L in layers]  # K x N, contiguous
    xs = [torch.from_numpy(xb.view(np.int16)).view(tdt).to(dev) for xb in x_host]
    stream = torch.cuda.current_stream()
    for _ in range(3):
        for x_, w_ in zip(xs, wts):
            torch.matmul(x_, w_)
    torch.cuda.synchronize()
    eager_ms = 0.0
    per = {}
    for L, x_, w_ in zip(layers, xs, wts):
        e0 = torch.cuda.Event(enable_timing=True)
        e1 = torch.cuda.Event(enable_timing=True)
        e0.record(stream)
        for _ in range(reps):
            torch.matmul(x_, w_)
        e1.record(stream)
        torch.cuda.synchronize()
        t = e0.elapsed_time(e1) / reps
        per[L.name] = round(t * 1e3, 2)
        eager_ms += t
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        outs = [torch.matmul(x_, w_) for x_, w_ in zip(xs, wts)]
    g.replay()
    torch.cuda.synchronize()
    e0 = torch.cuda.Event(enable_timing=True)
    e1 = torch.cuda.Event(enable_timing=True)
    e0.record(stream)
    for _ in range(reps):
        g.replay()
    e1.record(stream)
    torch.cuda.synchronize()
    graph_ms = e0.elapsed_time(e1) / reps
    del outs, g, wts, xs
    flops = sum(2 * M * L.N * L.K for L in layers)
    kind = "bf16" if tdt == torch.bfloat16 else "fp16"
    return {"what": f"torch.matmul (hipBLASLt), dense {kind} weights of the same shapes",
            "eager": {"ms_per_step": round(eager_ms, 5), "TFLOP_per_s": round(flops / (eager_ms * 1e-3) / 1e12, 1),
                      "per_shape_us": per},
            "graph": {"ms_per_step": round(graph_ms, 5), "TFLOP_per_s": round(flops / (graph_ms * 1e-3) / 1e12, 1)}}


def rotated_step(case, nsteps, warmup):
    """Decoder step of a layer quantised in the rotated basis (Eq. 5): per
    launch group one input transform, the batched product, one output
    transform of the group's stacked outputs (12 launches); and the same with
    the input transforms of the q+k+v and o groups inside their products."""
    torch, u, lib, ws, M = case.torch, case.u, case.lib, case.ws, case.M
    dev = torch.device("cuda:0")
    rgroups = [["q", "k", "v"], ["o"], ["gate", "up"], ["down"]]
    idx = {n: i for i, n in enumerate(case.names)}
    rng = np.random.default_rng(123)
    signs = {}
    for grp in rgroups:
        L0 = ws.layers[idx[grp[0]]]
        signs[grp[0]] = (torch.from_numpy(rng.choice(np.array([-1, 1], np.int8), L0.K)).to(dev),
                         torch.from_numpy(rng.choice(np.array([-1, 1], np.int8), L0.N)).to(dev))
    bufs = []
    for c in range(ws.copies):
        cc = []
        for grp in rgroups:
            L0 = ws.layers[idx[grp[0]]]
            xin = case.xs[c][idx[grp[0]]]
            cc.append((grp, L0.N, L0.K, xin, torch.empty_like(xin),
                       torch.empty((len(grp) * M, L0.N), dtype=torch.float16, device=dev),
                       torch.empty((len(grp) * M, L0.N), dtype=torch.float16, device=dev)))
        bufs.append(cc)

    def step(i, sptr, fused):
        c = i % ws.copies
        for (grp, N, K, xin, xrot, ystk, yout) in bufs[c]:
            sV, sU = signs[grp[0]]
            cnt = len(grp)
            arr = (u.GemvProblem * cnt)()
            # fused where the launch has at most 3 row blocks per CU: beyond that
            # the transform each workgroup repeats outweighs the saved launch
            fuse = fused and K in (4096, 8192) and N * cnt // 16 <= 768
            for j, n in enumerate(grp):
                L = ws.layers[idx[n]]
                arr[j] = u.GemvProblem(L.N, L.K, ws.packed[c][idx[n]].data_ptr(),
                                       (xin if fuse else xrot).data_ptr(), ystk[j * M:(j + 1) * M].data_ptr())
            if fuse:
                sg = (ctypes.c_void_p * cnt)(*([sV.data_ptr()] * cnt))
                sts = (lib.unisvq_gemv_rht_batched(arr, cnt, M, case.xcode, u.F16, sg, sptr),)
            else:
                sts = (lib.unisvq_rht(K, M, xin.data_ptr(), case.xcode, sV.data_ptr(), 0, xrot.data_ptr(), u.F16,
                                      sptr),
                       lib.unisvq_gemv_batched(arr, cnt, M, u.F16, u.F16, sptr))
            sts += (lib.unisvq_rht(N, cnt * M, ystk.data_ptr(), u.F16, sU.data_ptr(), 1, yout.data_ptr(), u.F16,
                                   sptr),)
            for st in sts:
                if st != 0:
                    raise RuntimeError(f"rotated step failed with status {st}")

    def timed(fused):
        stream = torch.cuda.current_stream()
        for i in range(warmup):
            step(i, stream.cuda_stream, fused)
        torch.cuda.synchronize()
        g = torch.cuda.CUDAGraph()
        with torch.cuda.graph(g):
            cap = torch.cuda.current_stream().cuda_stream
            for i in range(nsteps):
                step(i, cap, fused)
        g.replay()
        torch.cuda.synchronize()
        e0 = torch.cuda.Event(enable_timing=True)
        e1 = torch.cuda.Event(enable_timing=True)
        e0.record(stream)
        g.replay()
        e1.record(stream)
        torch.cuda.synchronize()
        del g
        return e0.elapsed_time(e1) / nsteps

    rms, fms = timed(False), timed(True)
    return {"what": "decoder step of a layer quantised in the rotated basis: 4 input transforms, 4 batched "
                    "products, 4 output transforms (12 launches)",
            "ms_per_step": round(rms, 5), "GB_per_s": round(case.set_bytes / (rms * 1e-3) / 1e9, 1),
            "fused": {"what": "the same step with the input transforms of the q+k+v and o launch groups inside "
                              "their products (unisvq_gemv_rht_batched; 10 launches)",
                      "ms_per_step": round(fms, 5), "GB_per_s": round(case.set_bytes / (fms * 1e-3) / 1e9, 1)}}


def cpu_baseline(case, workload, seconds):
    """The fp64 oracle (test infrastructure, untuned) on the host cores over
    the same layer set: T threads for about `seconds`, then one thread on a
    slice of the output rows."""
    import oracle
    ws = case.ws
    threads = oracle.default_threads()
    if ws.var:
        packed_h = [oracle.var_pack_codes(Q, ws.bits, ws.dim)[0] for (Q, A, B) in ws.host]
    elif ws.shared:
        packed_h = [oracle.pack_codes(Q)[0] for (Q, A, B) in ws.host]
    else:
        packed_h = [oracle.pack(Q, A, B)[0] for (Q, A, B) in ws.host]
    xs = [oracle.half_to_double(xb) if case.xdt == "f16" else oracle.bf16_to_double(xb) for xb in case.x_host]

    def run(rows_frac, nthreads, budget):
        done, t_cpu, passes = 0.0, 0.0, 0
        while t_cpu < budget or passes == 0:
            for li, L in enumerate(ws.layers):
                Q, A, B = ws.host[li]
                nrows = max(16, int(L.N * rows_frac))
                rows = None if nrows >= L.N else np.arange(nrows)
                s0 = time.perf_counter()
                if ws.var:
                    oracle.var_matmul(packed_h[li], L.N, L.K, ws.bits, A, B, xs[li], rows=rows, threads=nthreads)
                elif ws.shared:
                    oracle.matmul_shared(packed_h[li], L.N, L.K, A, B, xs[li], rows=rows, threads=nthreads)
                else:
                    oracle.matmul(packed_h[li], L.N, L.K, xs[li], rows=rows, threads=nthreads)
                t_cpu += time.perf_counter() - s0
                done += algorithmic_bytes(L.N, L.K, case.M, affine=ws.affine, bits=ws.bits, d=ws.dim) * (nrows / L.N)
            passes += 1
        return done / t_cpu / 1e9, passes, t_cpu

    frac = 1.0 if case.M <= 16 else 1.0 / 64
    v, passes, t = run(frac, threads, seconds)
    v1, p1, t1 = run(frac / 8, 1, seconds / 2)
    return {"value": round(v, 3), "unit": "GB/s", "cores": threads, "kind": "oracle",
            "sample": f"{passes} pass(es) over the {workload} layer set"
                      + ("" if frac == 1.0 else f" (1/{int(1 / frac)} of output rows)")
                      + f", fp64 C oracle, {threads} threads, {t:.1f} s",
            "one_thread": {"value": round(v1, 4), "unit": "GB/s",
                           "sample": f"{p1} pass(es) over 1/{int(8 / frac)} of the output rows of each layer, "
                                     f"one thread, {t1:.1f} s"},
            "cpu_model": cpu_model()}


def sub_records(u, torch, main_ws, args):
    """One record per configured workload besides the headline."""
    out = {}
    ws4096 = WeightSet(u, torch, (wl.Layer("layer", 4096, 4096),))
    c = Case(ws4096, 1, "f16", False)
    out["layer4096_m1"], _, _ = measure_case(c, "decoder", 100, 10)
    del c, ws4096
    for M in (4, 16, 64):
        c = Case(main_ws, M, "f16", True)
        out[f"llama7b_smallbatch_m{M}"], _, _ = measure_case(c, "decoder", 60, 5)
        del c
    ws70 = WeightSet(u, torch, wl.LLAMA70B)
    for M in (1, 16):
        c = Case(ws70, M, "f16", False)
        out[f"llama70b_decode_m{M}"], _, _ = measure_case(c, "decoder", 30, 3)
        del c
    del ws70
    wsp = WeightSet(u, torch, wl.PREFILL7B)
    c = Case(wsp, 2048, "bf16", False)
    rec, _, _ = measure_case(c, "decoder", 10, 2)
    rec["what"] = "decode path, one (A, B) pair per (row, 128-column group)"
    rec["dense_bf16"] = dense_baseline(torch, wsp.layers, 2048, c.tdt, c.x_host, 10)
    rec["over_dense_eager_time"] = round(rec["ms_per_step"] / rec["dense_bf16"]["eager"]["ms_per_step"], 3)
    del c, wsp
    wsm = WeightSet(u, torch, wl.PREFILL7B, affine="matrix")
    c = Case(wsm, 2048, "bf16", False, fold=True)
    fold, _, _ = measure_case(c, "decoder", 10, 2)
    fold["what"] = "Eq. 9 fold (unisvq_gemm_shared_fold), one (A, B) pair per matrix (the paper's setting)"
    fold["over_dense_eager_time"] = round(fold["ms_per_step"] / rec["dense_bf16"]["eager"]["ms_per_step"], 3)
    rec["fold"] = fold
    del c, wsm
    out["llama7b_prefill_m2048"] = rec
    for k, v in out.items():
        v["config_index"] = CONFIG_INDEX[k]
    return out


def main():
    args = parse()
    if args.calibrate_copy:
        calibrate_copy(args.calibrate_copy)
        return
    if args.gpus != 1:
        print(f"bench.py measures one GPU only (asked for --gpus {args.gpus}): the library has no multi-GPU "
              "path (column-parallel layers would split N with no exchange, row-parallel ones K on packet "
              "boundaries followed by one all-reduce of the partial outputs).", file=sys.stderr)
        sys.exit(2)
    if args.workload == "ldlq_layer4096":
        bench_ldlq(args)
        return
    if args.workload == "quantize_llama7b":
        bench_quantize(args)
        return

    import torch
    import paper_2606_10520_amd.unisvq as u

    u.load()  # fails loudly if libunisvq.so is missing
    headline = args.workload or "llama7b_decode_m1"
    layers, M, xdt, outliers = workload_spec(headline)
    bits, dim = (int(v) for v in args.format.split("x"))
    var = (bits, dim) != (2, 4)
    if var and args.affine == "row_group":
        args.affine = "matrix"  # the variants keep their pairs shared by the rows
    shared = args.affine != "row_group"
    if args.fold and (not shared or var or M <= 3):
        print("--fold needs row-shared pairs (--affine matrix or group), the 2x4 format and more than 3 tokens "
              "(the fold is a unisvq_gemm_shared_fold path)", file=sys.stderr)
        sys.exit(2)
    wname = headline if not shared else f"{headline}_{args.affine}_shared" + ("_fold" if args.fold else "")
    if var:
        wname += f"_b{bits}d{dim}"

    ws = WeightSet(u, torch, layers, args.affine, bits, dim, keep_host=not args.no_cpu_baseline)
    case = Case(ws, M, xdt, outliers, fold=args.fold)
    rec, calls, groups = measure_case(case, args.schedule, args.steps, args.warmup, extras=not args.no_schedules,
                                      traffic_key=wname)
    schedules = {}
    if case.kernel == "gemv" and not args.no_schedules:
        for other in ("per_layer", "decoder", "single"):
            oname, ogroups = case.groups(other)
            if oname != other:
                continue
            oms = rec["ms_per_step"] if oname == rec["schedule"] else case.time_steps(case.calls(ogroups), 60, 2)
            schedules[oname] = {"launches_per_step": len(ogroups), "ms_per_step": round(oms, 5),
                                "GB_per_s": round(case.set_bytes / (oms * 1e-3) / 1e9, 1)}
    dense = None
    if M > 64:
        dense = dense_baseline(torch, layers, M, case.tdt, case.x_host, 10)
    rot = None
    full_set = {"q", "k", "v", "o", "gate", "up", "down"} <= set(case.names)
    if (args.rht or args.workload is None) and case.kernel == "gemv" and not shared and full_set \
            and not args.no_schedules:
        rot = rotated_step(case, 60, 5)
    cpu = None
    if not args.no_cpu_baseline:
        cpu = cpu_baseline(case, headline, args.cpu_seconds)
    configs = None
    if args.workload is None and not args.no_sub and not shared and not var:
        configs = sub_records(u, torch, ws, args)

    if case.M <= 64:
        metric = METRIC if (M == 1 and not shared and not var) else f"2-bit decode achieved HBM GB/s at M={M}"
        if var:
            metric = f"{bits}-bit d={dim} decode achieved HBM GB/s at M={M}"
        if shared:
            metric += f" (codes-only, one (A, B) pair per {'matrix' if args.affine == 'matrix' else 'group'})"
    else:
        metric = "unisvq_gemm effective TFLOP/s (2MNK)"
        if var:
            metric = f"unisvq_var_gemm ({bits}-bit codes, d={dim}) effective TFLOP/s (2MNK)"
        if args.fold:
            metric = "unisvq_gemm_shared_fold effective TFLOP/s (2MNK)"
    out = {
        "metric": metric,
        "value": rec["value"],
        "unit": rec["unit"],
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": rec["ms_per_step"],
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        # arithmetic type of the matrix cores: the GEMM multiplies in fp16
        # (bf16 activations are carried exactly as scaled fp16)
        "dtype": "f16" if (xdt == "f16" or case.kernel == "gemm") else "bf16",
        "data": "synthetic",
        "config": {"workload": headline, "layers": {L.name: [L.N, L.K] for L in layers}, "M": M,
                   "activations": xdt, "affine": args.affine, "d": dim, "bits": bits, "group": 128,
                   "kernel": case.kernel, "schedule": rec["schedule"],
                   "launches_per_step": rec["launches_per_step"], "buffer_copies": ws.copies,
                   "set_bytes": case.set_bytes,
                   "timing": "warmup steps eager; the timed steps are one HIP graph of exactly `steps` steps "
                             "(captured, replayed once untimed, then once between two events)"},
        "pct_peak_hbm": rec.get("pct_peak_hbm"),
        "per_launch_us": rec.get("per_launch_us"),
        "achievable": rec.get("achievable"),
        "schedules": schedules or None,
        "dense_matmul": dense,
        "rotated_layer": rot,
        "roofline": rec["roofline"],
        "cpu_baseline": cpu,
        "configs": configs,
    }
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
