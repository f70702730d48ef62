#!/usr/bin/env python3
"""Benchmark of the UniSVQ 2-bit affine-lattice product on one MI355X.

Default workload: the LLaMA-7B decoder linears at M = 1 token (q/k/v/o
4096x4096, gate/up 11008x4096, down 4096x11008), 2-bit codes in d = 4
vectors along K with one fp16 (A, B) set per (row, 128-column group), fp16
activations.  One step = one pass of the seven linears through unisvq_gemv,
launched back to back on one stream.  Weights, activations and outputs are
resident in HBM before timing starts; the step rotates over enough copies of
the layer set (> 512 MB) that the 256 MB Infinity Cache cannot serve them.

Prints one JSON line.  value = algorithmic bytes per step / time per step
(codes N*K/4 + affine N*(K/128)*40 + activations + outputs; dense fp16
weights are never counted).
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
    p.add_argument("--workload", default="llama7b_decode_m1",
                   choices=["llama7b_decode_m1", "layer4096_m1", "llama70b_decode_m1",
                            "llama70b_decode_m16", "llama7b_smallbatch_m4", "llama7b_smallbatch_m16",
                            "llama7b_smallbatch_m64", "llama7b_prefill_m2048", "quantize_llama7b", "ldlq_layer4096"])
    p.add_argument("--fold", action="store_true",
                   help="with --affine matrix/group and a GEMM workload: the Eq. 9 fold "
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
                   help="also time the decoder step of a layer quantised in the rotated basis (Eq. 5): per "
                        "launch group, one input transform of its activations, the batched product and one "
                        "output transform of the group's stacked outputs")
    p.add_argument("--calibrate-copy", type=int, default=0, metavar="BYTES",
                   help="only run a plain device-to-device copy of BYTES bytes 10 times (counter calibration)")
    p.add_argument("--no-schedules", action="store_true",
                   help="time only the --schedule launch sequence (for profiling runs)")
    p.add_argument("--no-cpu-baseline", action="store_true")
    p.add_argument("--cpu-seconds", type=float, default=10.0, help="target CPU work of the oracle sample")
    p.add_argument("--no-launch-events", action="store_true",
                   help="skip the per-launch event pass (roofline fields become null)")
    return p.parse_args()


# Sources that define each kernel (its translation unit and the headers it is built from).
KERNEL_SOURCES = {"gemv": ("gemv.hip", "gemv_kernel.hpp", "common.hpp"),
                  "gemm": ("gemm.hip", "decode.hpp", "common.hpp"),
                  "skinny": ("skinny.hip", "decode.hpp", "common.hpp")}


# Largest batch the 2x4 product sends to the skinny kernel (kSkinnyMaxM).
SKINNY_MAX_M = 32


def kernel_source_hash(kernel: str) -> str:
    import hashlib
    h = hashlib.sha256()
    for f in KERNEL_SOURCES.get(kernel, (f"{kernel}.hip",)):
        h.update(open(os.path.join(ROOT, "paper_2606_10520_amd", "csrc", f), "rb").read())
    return h.hexdigest()[:16]


def measured_traffic(kernel: str, workload: str, schedule: str):
    """HBM bytes per launch from the committed counter summary, if it was taken
    on the current kernel source; else None.  (workload carries a suffix for
    the row-shared modes.)"""
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
    """(layers, M, activation dtype, outliers, kernel)"""
    if name == "llama7b_decode_m1":
        return wl.LLAMA7B, 1, "f16", False, "gemv"
    if name == "layer4096_m1":
        return (wl.Layer("layer", 4096, 4096),), 1, "f16", False, "gemv"
    if name == "llama70b_decode_m1":
        return wl.LLAMA70B, 1, "f16", False, "gemv"
    if name == "llama70b_decode_m16":
        return wl.LLAMA70B, 16, "f16", False, "gemm"
    if name.startswith("llama7b_smallbatch_m"):
        M = int(name.rsplit("m", 1)[1])
        return wl.LLAMA7B, M, "f16", True, ("gemv" if M <= 4 else "gemm")
    if name == "llama7b_prefill_m2048":
        return wl.PREFILL7B, 2048, "bf16", False, "gemm"
    raise ValueError(name)


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


def ldl_factor(H, d=4):
    """H = U D U^T with U unit upper block triangular (the caller's factorisation
    that unisvq_ldlq takes): Cholesky of H with its index order reversed."""
    C = np.linalg.cholesky(H[::-1, ::-1])
    R = np.ascontiguousarray(C[::-1, ::-1])
    U = np.empty_like(R)
    for j in range(H.shape[0] // d):
        sl = slice(d * j, d * (j + 1))
        U[:, sl] = np.linalg.solve(R[sl, sl].T, R[:, sl].T).T
        U[sl, sl] = np.eye(d)
    return U


LDLQ_FLOP_PER_FEEDBACK = 2  # one fma per (row, earlier column, column)


def bench_ldlq(args):
    """LDLQ (Eq. 7) on one 4096 x 4096 layer: W ~ N(0, 1) fp32, the paper's
    initial grid (Eq. 6) with one pair per (row, group), and a synthetic
    Hessian with coupled columns (X^T X / S, S = 2K activations sharing a
    common component, + mu I, mu = 0.01, Sec. 4.2) factorised on the host.
    Reports vectors per second, the fp64 rate, and the Hessian proxy loss
    tr(E H E^T) against plain nearest-codeword rounding on a slice of rows."""
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
    U = ldl_factor(H)
    W = torch.randn(N, K, device=dev, generator=torch.Generator(device=dev).manual_seed(1))
    Ad = torch.from_numpy(A.view(np.int16)).view(torch.float16).to(dev)
    Bd = torch.from_numpy(B.view(np.int16)).view(torch.float16).to(dev)
    Ud = torch.from_numpy(U).to(dev)
    q = torch.empty((N, K), dtype=torch.uint8, device=dev)
    ws = torch.empty(u.ldlq_workspace_bytes(N, K), dtype=torch.uint8, device=dev)
    stream = torch.cuda.current_stream()

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
        "proxy_loss_over_nearest": round(loss(E_l) / loss(E_r), 4),
        "weight_mse": {"ldlq": round(mse(E_l), 5), "nearest": round(mse(E_r), 5)},
        "roofline": {"bound": "alu", "achieved": round(ach, 2), "peak": PEAK_FP64_TFLOPS, "unit": "TFLOP/s",
                     "frac": round(ach / PEAK_FP64_TFLOPS, 4), "traffic": None,
                     "kernel": "ldlq_block_kernel + ldlq_update_kernel", "avg_launch_us": None},
        "cpu_baseline": cpu,
    }
    print(json.dumps(out), flush=True)


def main():
    args = parse()
    if args.calibrate_copy:
        calibrate_copy(args.calibrate_copy)
        return
    if args.workload == "ldlq_layer4096":
        if args.gpus != 1:
            print(f"bench.py measures one GPU only (asked for --gpus {args.gpus})", file=sys.stderr)
            sys.exit(2)
        bench_ldlq(args)
        return
    if args.workload == "quantize_llama7b":
        if args.gpus != 1:
            print("bench.py measures one GPU only", file=sys.stderr)
            sys.exit(2)
        bench_quantize(args)
        return
    if args.gpus != 1:
        print(f"bench.py measures one GPU only (asked for --gpus {args.gpus}); "
              "this build has no multi-GPU path.", file=sys.stderr)
        sys.exit(2)

    import torch
    import paper_2606_10520_amd.unisvq as u

    u.load()  # fails loudly if libunisvq.so is missing
    dev = torch.device("cuda:0")
    layers, M, xdt, outliers, kernel = workload_spec(args.workload)
    tdt = torch.float16 if xdt == "f16" else torch.bfloat16
    bits, dim = (int(v) for v in args.format.split("x"))
    var = (bits, dim) != (2, 4)
    if var and args.affine == "row_group":
        args.affine = "matrix"  # the variants keep their pairs shared by the rows
    shared = args.affine != "row_group"
    wname = args.workload if not shared else f"{args.workload}_{args.affine}_shared" + ("_fold" if args.fold else "")
    if var:
        wname += f"_b{bits}d{dim}"

    # ---- inputs: canonical arrays drawn on the host, packed on the GPU
    canon = []
    for li, L in enumerate(layers):
        if var:
            Q, A, B = wl.gen_var_weights(L.N, L.K, bits, dim, affine_groups(L.K, args.affine), seed=li)
        elif shared:
            Q, A, B = wl.gen_shared_weights(L.N, L.K, affine_groups(L.K, args.affine), seed=li)
        else:
            Q, A, B = wl.gen_weights(L.N, L.K, seed=li)
        xb = wl.gen_activations(M, L.K, seed=wl.activation_seed(li, M), dtype=xdt, outliers=outliers)
        canon.append((Q, A, B, xb))
    set_bytes = sum(algorithmic_bytes(L.N, L.K, M, affine=args.affine, bits=bits, d=dim) for L in layers)
    set_packed = sum((u.var_codes_bytes(L.N, L.K, bits, dim) if var else
                      u.codes_bytes(L.N, L.K) if shared else u.packed_bytes(L.N, L.K)) for L in layers)
    copies = max(2, -(-2 * MALL_BYTES // set_packed) + 1)

    def dev_half(a):
        return torch.from_numpy(a.view(np.int16)).view(torch.float16).to(dev)

    packed0 = []
    for (Q, A, B, _), L in zip(canon, layers):
        if var:
            packed0.append(u.var_pack(torch.from_numpy(Q).to(dev), dev_half(A), dev_half(B), bits, dim))
        elif shared:
            packed0.append(u.pack_shared(torch.from_numpy(Q).to(dev), dev_half(A), dev_half(B)))
        else:
            packed0.append(u.pack(torch.from_numpy(Q).to(dev), dev_half(A), dev_half(B)))
    sets = []
    for c in range(copies):
        s = []
        for li, L in enumerate(layers):
            if shared:
                pk = packed0[li] if c == 0 else tuple(t.clone() for t in packed0[li])
            else:
                pk = packed0[li] if c == 0 else packed0[li].clone()
            x = torch.from_numpy(canon[li][3].view(np.int16)).view(tdt).to(dev)
            y = torch.empty((M, L.N), dtype=torch.float16, device=dev)
            s.append((L, pk, x, y))
        sets.append(s)
    torch.cuda.synchronize()

    lib = u.load()
    xcode = u.F16 if xdt == "f16" else u.BF16
    # GEMM workspace (bf16 activation copy, K-split partials): one buffer
    # serves every call, since the calls run in order on one stream.
    ws_bytes = 0
    if kernel == "gemm":
        wsf = u.var_gemm_workspace_bytes if var else u.gemm_workspace_bytes
        ws_bytes = max(wsf(L.N, L.K, M, tdt) for L in layers)
    if args.fold and shared and kernel == "gemm":
        ws_bytes = max(ws_bytes, max(u.gemm_fold_workspace_bytes(L.N, L.K, M) for L in layers))
    ws = torch.empty(max(ws_bytes, 256), dtype=torch.uint8, device=dev)
    names = [L.name for L in layers]
    full_set = {"q", "k", "v", "o", "gate", "up", "down"} <= set(names)

    def schedule_groups(sched):
        if kernel != "gemv":
            return "per_layer", [[n] for n in names]
        if sched == "decoder" and full_set:
            return "decoder", [["q", "k", "v"], ["o"], ["gate", "up"], ["down"]]
        if sched == "single" and len(names) <= u.MAX_BATCH:
            return "single", [names]
        return "per_layer", [[n] for n in names]

    def build_calls(groups_):
        calls = []  # per buffer copy: list of (label, single-problem tuple or ctypes problem array)
        for s_ in sets:
            by = {L.name: (L, pk, x, y) for (L, pk, x, y) in s_}
            cc = []
            for grp in groups_:
                if len(grp) == 1:
                    cc.append(("+".join(grp), by[grp[0]]))
                elif shared:
                    arr = (u.GemvSharedProblem * len(grp))()
                    for i, n in enumerate(grp):
                        L, (pc, pa), x, y = by[n]
                        arr[i] = u.GemvSharedProblem(L.N, L.K, affine_groups(L.K, args.affine), pc.data_ptr(),
                                                     pa.data_ptr(), x.data_ptr(), y.data_ptr())
                    cc.append(("+".join(grp), arr))
                else:
                    arr = (u.GemvProblem * len(grp))()
                    for i, n in enumerate(grp):
                        L, pk, x, y = by[n]
                        arr[i] = u.GemvProblem(L.N, L.K, pk.data_ptr(), x.data_ptr(), y.data_ptr())
                    cc.append(("+".join(grp), arr))
            calls.append(cc)
        return calls

    def launch(item, sptr):
        if var:
            if not isinstance(item, tuple):
                return lib.unisvq_var_gemv_batched(item, len(item), bits, dim, M, xcode, u.F16, sptr)
            L, (pc, pa), x, y = item
            ga = affine_groups(L.K, args.affine)
            if kernel == "gemv":
                return lib.unisvq_var_gemv(L.N, L.K, bits, dim, ga, pc.data_ptr(), pa.data_ptr(), M, x.data_ptr(),
                                           xcode, y.data_ptr(), u.F16, sptr)
            return lib.unisvq_var_gemm(L.N, L.K, bits, dim, ga, pc.data_ptr(), pa.data_ptr(), M, x.data_ptr(),
                                       xcode, y.data_ptr(), u.F16, ws.data_ptr(), ws_bytes, sptr)
        if isinstance(item, tuple) and shared:
            L, (pc, pa), x, y = item
            ga = affine_groups(L.K, args.affine)
            if kernel == "gemv":
                return lib.unisvq_gemv_shared(L.N, L.K, ga, pc.data_ptr(), pa.data_ptr(), M, x.data_ptr(), xcode,
                                              y.data_ptr(), u.F16, sptr)
            if args.fold:
                return lib.unisvq_gemm_shared_fold(L.N, L.K, ga, pc.data_ptr(), pa.data_ptr(), M, x.data_ptr(),
                                                   xcode, y.data_ptr(), u.F16, ws.data_ptr(), ws_bytes, sptr)
            return lib.unisvq_gemm_shared(L.N, L.K, ga, pc.data_ptr(), pa.data_ptr(), M, x.data_ptr(), xcode,
                                          y.data_ptr(), u.F16, ws.data_ptr(), ws_bytes, sptr)
        if shared:
            return lib.unisvq_gemv_shared_batched(item, len(item), M, xcode, u.F16, sptr)
        if isinstance(item, tuple):
            L, pk, x, y = item
            if kernel == "gemv":
                return lib.unisvq_gemv(L.N, L.K, pk.data_ptr(), M, x.data_ptr(), xcode, y.data_ptr(), u.F16, sptr)
            return lib.unisvq_gemm(L.N, L.K, pk.data_ptr(), M, x.data_ptr(), xcode, y.data_ptr(), u.F16,
                                   ws.data_ptr(), ws_bytes, sptr)
        return lib.unisvq_gemv_batched(item, len(item), M, xcode, u.F16, sptr)

    def run_step(calls, i, sptr):
        for _, item in calls[i % copies]:
            st = launch(item, sptr)
            if st != 0:
                raise RuntimeError(f"{kernel} failed with status {st}")

    stream = torch.cuda.current_stream()

    def time_schedule(calls):
        """Warm up, capture the steps of all buffer copies in one HIP graph, and
        time ceil(steps / copies) replays between two events."""
        for i in range(args.warmup):
            run_step(calls, i, stream.cuda_stream)
        torch.cuda.synchronize()
        graph = torch.cuda.CUDAGraph()
        with torch.cuda.graph(graph):
            cap = torch.cuda.current_stream().cuda_stream
            for c in range(copies):
                run_step(calls, c, cap)
        torch.cuda.synchronize()
        graph.replay()  # one untimed replay
        torch.cuda.synchronize()
        replays = max(1, -(-args.steps // copies))
        t0 = torch.cuda.Event(enable_timing=True)
        t1 = torch.cuda.Event(enable_timing=True)
        t0.record(stream)
        for _ in range(replays):
            graph.replay()
        t1.record(stream)
        torch.cuda.synchronize()
        return t0.elapsed_time(t1) / (replays * copies), replays * copies

    sched, groups_ = schedule_groups(args.schedule)
    calls = build_calls(groups_)
    ms_per_step, steps_done = time_schedule(calls)
    value_gbs = set_bytes / (ms_per_step * 1e-3) / 1e9

    # a dense product of the same shapes (random weights, the activation
    # dtype), timed the same way: the library GEMM the decode would compete with
    dense = None
    if kernel == "gemm":
        wts = [torch.randn(L.K, L.N, device=dev).to(tdt) for L in layers]  # K x N, contiguous
        xs_d = [torch.from_numpy(canon[li][3].view(np.int16)).view(tdt).to(dev) for li in range(len(layers))]
        for i in range(3):
            for x_, w_ in zip(xs_d, wts):
                torch.matmul(x_, w_)
        torch.cuda.synchronize()
        g_d = torch.cuda.CUDAGraph()
        with torch.cuda.graph(g_d):
            outs = [torch.matmul(x_, w_) for x_, w_ in zip(xs_d, wts)]
        g_d.replay()
        torch.cuda.synchronize()
        reps = max(3, args.steps // 4)
        d0 = torch.cuda.Event(enable_timing=True)
        d1 = torch.cuda.Event(enable_timing=True)
        d0.record(stream)
        for _ in range(reps):
            g_d.replay()
        d1.record(stream)
        torch.cuda.synchronize()
        dms = d0.elapsed_time(d1) / reps
        dflops = sum(2 * M * L.N * L.K for L in layers)
        dense = {"what": f"torch.matmul, dense {'fp16' if xdt == 'f16' else 'bf16'} weights of the same shapes",
                 "ms_per_step": round(dms, 5), "TFLOP_per_s": round(dflops / (dms * 1e-3) / 1e12, 1),
                 "unisvq_over_dense_time": round(ms_per_step / dms, 3)}
        del wts, xs_d, outs, g_d

    # the other launch schedules of the same step, for context
    schedules = {}
    if kernel == "gemv" and not args.no_schedules:
        for other in ("per_layer", "decoder", "single"):
            oname, ogroups = schedule_groups(other)
            if oname != other:
                continue
            oms = ms_per_step if oname == sched else time_schedule(build_calls(ogroups))[0]
            schedules[oname] = {"launches_per_step": len(ogroups), "ms_per_step": round(oms, 5),
                                "GB_per_s": round(set_bytes / (oms * 1e-3) / 1e9, 1)}

    # ---- the rotated layer (Eq. 5): transforms around each launch group
    rht = None
    if args.rht and kernel == "gemv" and not shared and full_set:
        rgroups = [["q", "k", "v"], ["o"], ["gate", "up"], ["down"]]
        rng = np.random.default_rng(123)
        rcalls = []
        for s_ in sets:
            by = {L.name: (L, pk, x, y) for (L, pk, x, y) in s_}
            cc = []
            for grp in rgroups:
                Ls = [by[n][0] for n in grp]
                N, K = Ls[0].N, Ls[0].K
                sV = torch.from_numpy(rng.choice(np.array([-1, 1], np.int8), K)).to(dev)
                sU = torch.from_numpy(rng.choice(np.array([-1, 1], np.int8), N)).to(dev)
                xin = by[grp[0]][2]                                   # the group's activations
                xrot = torch.empty_like(xin)
                ystk = torch.empty((len(grp) * M, N), dtype=torch.float16, device=dev)
                yout = torch.empty_like(ystk)
                arr = (u.GemvProblem * len(grp))()
                for i, n in enumerate(grp):
                    L, pk, _, _ = by[n]
                    arr[i] = u.GemvProblem(L.N, L.K, pk.data_ptr(), xrot.data_ptr(), ystk[i * M:(i + 1) * M].data_ptr())
                cc.append((K, M, xin, xcode, sV, xrot, arr, len(grp), N, ystk, sU, yout))
            rcalls.append(cc)

        def rstep(i, sptr, fused):
            for (K, M_, xin, xc, sV, xrot, arr, cnt, N, ystk, sU, yout) in rcalls[i % copies]:
                # fused where the launch has at most 3 row blocks per CU: beyond that
                # the transform each workgroup repeats outweighs the saved launch
                if fused and K in (4096, 8192) and N * cnt // 16 <= 768:
                    # input transform inside the product launch: x enters unrotated
                    farr = (u.GemvProblem * cnt)()
                    for j in range(cnt):
                        farr[j] = u.GemvProblem(arr[j].N, arr[j].K, arr[j].packed, xin.data_ptr(), arr[j].y)
                    sg = (ctypes.c_void_p * cnt)(*([sV.data_ptr()] * cnt))
                    calls_ = (lib.unisvq_gemv_rht_batched(farr, cnt, M_, xc, u.F16, sg, sptr),)
                else:
                    calls_ = (lib.unisvq_rht(K, M_, xin.data_ptr(), xc, sV.data_ptr(), 0, xrot.data_ptr(), u.F16,
                                             sptr),
                              lib.unisvq_gemv_batched(arr, cnt, M_, u.F16, u.F16, sptr))
                calls_ += (lib.unisvq_rht(N, cnt * M_, ystk.data_ptr(), u.F16, sU.data_ptr(), 1, yout.data_ptr(),
                                          u.F16, sptr),)
                for st in calls_:
                    if st != 0:
                        raise RuntimeError(f"rotated step failed with status {st}")

        def time_rotated(fused):
            for i in range(args.warmup):
                rstep(i, stream.cuda_stream, fused)
            torch.cuda.synchronize()
            g_r = torch.cuda.CUDAGraph()
            with torch.cuda.graph(g_r):
                cap = torch.cuda.current_stream().cuda_stream
                for c in range(copies):
                    rstep(c, cap, fused)
            g_r.replay()
            torch.cuda.synchronize()
            reps = max(1, -(-args.steps // copies))
            r0 = torch.cuda.Event(enable_timing=True)
            r1 = torch.cuda.Event(enable_timing=True)
            r0.record(stream)
            for _ in range(reps):
                g_r.replay()
            r1.record(stream)
            torch.cuda.synchronize()
            del g_r
            return r0.elapsed_time(r1) / (reps * copies)

        rms = time_rotated(False)
        fms = time_rotated(True)
        rht = {"what": "decoder step of a layer quantised in the rotated basis: 4 input transforms, 4 batched "
                       "products, 4 output transforms (12 launches)",
               "ms_per_step": round(rms, 5), "over_plain_step": round(rms / ms_per_step, 3),
               "GB_per_s": round(set_bytes / (rms * 1e-3) / 1e9, 1),
               "fused": {"what": "the same step with the input transforms of the q+k+v and o launch groups "
                                 "inside their products (unisvq_gemv_rht_batched; 10 launches)",
                         "ms_per_step": round(fms, 5), "over_plain_step": round(fms / ms_per_step, 3),
                         "GB_per_s": round(set_bytes / (fms * 1e-3) / 1e9, 1)}}

    # ---- per-launch breakdown: HIP events on the launch stream around each
    # launch.  A spin kernel first lets the host queue a chunk of launches ahead
    # of the GPU, so an interval brackets GPU work rather than host latency;
    # each interval still includes one dispatch and two marker packets.
    per_layer_us = {}
    if not args.no_launch_events:
        ev = []
        chunk = 8
        for c0 in range(0, args.steps, chunk):
            torch.cuda.synchronize()
            torch.cuda._sleep(20_000_000)  # ~8 ms of spinning at 2.4 GHz
            for i in range(c0, min(args.steps, c0 + chunk)):
                for label, item in calls[i % copies]:
                    a = torch.cuda.Event(enable_timing=True)
                    b = torch.cuda.Event(enable_timing=True)
                    a.record(stream)
                    launch(item, stream.cuda_stream)
                    b.record(stream)
                    ev.append((label, a, b))
        torch.cuda.synchronize()
        durs = {}
        for name, a, b in ev:
            durs.setdefault(name, []).append(a.elapsed_time(b) * 1e3)
        per_layer_us = {k: float(np.mean(v)) for k, v in durs.items()}

    # The roofline's launch duration comes from the timed region itself: the
    # graph-timed step divided by its launches (events around single launches
    # would add two marker packets and a dispatch to every interval).
    launches_per_step = len(groups_)
    avg_us = ms_per_step * 1e3 / launches_per_step
    bytes_per_launch = set_bytes / launches_per_step
    if kernel == "gemv":
        ach = bytes_per_launch / (avg_us * 1e-6) / 1e9
        traffic = measured_traffic("gemv", wname, sched)
        roofline = {"bound": "hbm", "achieved": round(ach, 1), "peak": PEAK_HBM_GBS, "unit": "GB/s",
                    "frac": round(ach / PEAK_HBM_GBS, 4),
                    "traffic": None if traffic is None else int(traffic),
                    "kernel": "gemv_kernel", "avg_launch_us": round(avg_us, 3),
                    "bytes_per_launch": int(bytes_per_launch)}
    elif M <= 64:
        # small batch: still bound by the weight stream.  The 2x4 format at
        # M <= 32 runs the skinny kernel, everything else the tiled one.
        kname = "skinny" if (not var and M <= SKINNY_MAX_M) else "gemm"
        ach = bytes_per_launch / (avg_us * 1e-6) / 1e9
        traffic = measured_traffic(kname, wname, sched)
        roofline = {"bound": "hbm", "achieved": round(ach, 1), "peak": PEAK_HBM_GBS, "unit": "GB/s",
                    "frac": round(ach / PEAK_HBM_GBS, 4),
                    "traffic": None if traffic is None else int(traffic),
                    "kernel": f"{kname}_kernel", "avg_launch_us": round(avg_us, 3),
                    "bytes_per_launch": int(bytes_per_launch)}
    else:
        flops = sum(2 * M * L.N * L.K for L in layers) / launches_per_step
        ach = flops / (avg_us * 1e-6) / 1e12
        traffic = measured_traffic("gemm", wname, sched)
        roofline = {"bound": "mfma", "achieved": round(ach, 1), "peak": PEAK_BF16_TFLOPS,
                    "unit": "TFLOP/s", "frac": round(ach / PEAK_BF16_TFLOPS, 4),
                    "traffic": None if traffic is None else int(traffic),
                    "kernel": "gemm_kernel", "avg_launch_us": round(avg_us, 3)}

    # ---- CPU baseline: the fp64 oracle on the host cores, bounded sample
    cpu = None
    if not args.no_cpu_baseline:
        import oracle
        threads = oracle.default_threads()
        if var:
            packed_h = [oracle.var_pack_codes(Q, bits, dim)[0] for (Q, A, B, _) in canon]
        elif shared:
            packed_h = [oracle.pack_codes(Q)[0] for (Q, A, B, _) in canon]
        else:
            packed_h = [oracle.pack(Q, A, B)[0] for (Q, A, B, _) in canon]
        xs = [oracle.half_to_double(xb) if xdt == "f16" else oracle.bf16_to_double(xb) for (_, _, _, xb) in canon]
        rows_frac = 1.0
        if M > 16:  # prefill: a bounded slice of output rows per layer
            rows_frac = 1.0 / 64
        done_bytes, t_cpu, passes = 0.0, 0.0, 0
        while t_cpu < args.cpu_seconds or passes == 0:
            for li, L in enumerate(layers):
                nrows = max(16, int(L.N * rows_frac))
                rows = None if nrows >= L.N else np.arange(nrows)
                s0 = time.perf_counter()
                if var:
                    oracle.var_matmul(packed_h[li], L.N, L.K, bits, canon[li][1], canon[li][2], xs[li], rows=rows,
                                      threads=threads)
                elif shared:
                    oracle.matmul_shared(packed_h[li], L.N, L.K, canon[li][1], canon[li][2], xs[li], rows=rows,
                                         threads=threads)
                else:
                    oracle.matmul(packed_h[li], L.N, L.K, xs[li], rows=rows, threads=threads)
                t_cpu += time.perf_counter() - s0
                done_bytes += algorithmic_bytes(L.N, L.K, M, affine=args.affine, bits=bits, d=dim) * (nrows / L.N)
            passes += 1
        cpu = {"value": round(done_bytes / t_cpu / 1e9, 3), "unit": "GB/s", "cores": threads,
               "kind": "oracle",
               "sample": f"{passes} pass(es) over the {args.workload} layer set"
                         + ("" if rows_frac == 1.0 else f" (1/{int(1 / rows_frac)} of output rows)")
                         + f", fp64 C oracle, {threads} threads, {t_cpu:.1f} s"}

    if kernel == "gemv" or M <= 64:
        metric = METRIC if (M == 1 and not shared) else f"2-bit decode achieved HBM GB/s at M={M}"
        if var:
            metric = f"{bits}-bit d={dim} decode achieved HBM GB/s at M={M}"
        if shared:
            metric += f" (codes-only, one (A, B) pair per {'matrix' if args.affine == 'matrix' else 'group'})"
        value, unit = value_gbs, "GB/s"
    else:
        flops = sum(2 * M * L.N * L.K for L in layers)
        metric, value, unit = "unisvq_gemm effective TFLOP/s (2MNK)", flops / (ms_per_step * 1e-3) / 1e12, "TFLOP/s"
        if var:
            metric = f"unisvq_var_gemm ({bits}-bit codes, d={dim}) effective TFLOP/s (2MNK)"
    out = {
        "metric": metric,
        "value": round(value, 2),
        "unit": unit,
        "n_gpus": 1,
        "steps": steps_done,
        "warmup": args.warmup,
        "ms_per_step": round(ms_per_step, 5),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        # arithmetic type of the matrix cores: the GEMM multiplies in fp16
        # (bf16 activations are carried exactly as scaled fp16)
        "dtype": "f16" if (xdt == "f16" or kernel == "gemm") else "bf16",
        "data": "synthetic",
        "config": {"workload": args.workload, "layers": {L.name: [L.N, L.K] for L in layers}, "M": M,
                   "activations": xdt, "affine": args.affine,
                   "d": dim, "bits": bits, "group": 128, "kernel": kernel, "schedule": sched,
                   "launches_per_step": len(groups_), "buffer_copies": copies,
                   "set_bytes": set_bytes},
        "pct_peak_hbm": round(100 * value_gbs / PEAK_HBM_GBS, 2) if (kernel == "gemv" or M <= 64) else None,
        "dense_matmul": dense,
        "event_us_per_launch": {k: round(v, 3) for k, v in per_layer_us.items()},
        "schedules": schedules,
        "rotated_layer": rht,
        "roofline": roofline,
        "cpu_baseline": cpu,
    }
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
