#!/usr/bin/env python3
"""Throughput of quantized LSTM acoustic-model inference on one MI355X.

One step = one full forward pass of the acoustic model (activation
quantization, hoisted input products, the recurrence of every layer and the
quantized softmax output layer) over one batch of synthetic frames already
resident in HBM.  The headline value is frames/s of the 5-layer 500-cell
model with an 8192-way softmax at batch 64 x T=1000.  Also reported: the same
model at batch 1 (streaming latency case), the 4-layer LSTMP(2048, P=512)
model with a 16384-way softmax at batch 256 x T=800, the raw 8-bit GEMM
sweep (M=N=K in {4096, 8192}), the dominant kernel against its roofline, and
the CPU oracle timed on this host's cores on a bounded sample.

    python bench.py [--steps K] [--warmup W] [--gpus 1] [--skip-cpu] [--quick]
"""
from __future__ import annotations

import argparse
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

METRIC = "quantized LSTM AM frames/sec at batch 1 and 64; int8 GEMM TOPS vs MFMA peak"
HBM_PEAK_GBS = 8000.0      # MI355X HBM3E
INT8_PEAK_TOPS = 5000.0    # MI355X dense int8 MFMA
FP32_PEAK_TFLOPS = 157.3   # MI355X dense fp32 (MFMA)

# HBM bytes per launch of the dominant kernel (the wavefront launch over the
# first layers of the 5x500 model at batch 64, T = 1000), from two rocprofv3
# --pmc passes (FETCH_SIZE, WRITE_SIZE) scaled by the same counters on a plain
# 1 GiB copy; valid only for the kernel sources with this digest (any edit
# makes it stale -> null).
TRAFFIC = dict(bytes=3.4146e+08, read=1.6776e+08, written=1.7371e+08,
               sources=("ql_stack.hip", "ql_xstack.hip", "ql_xcd.h", "ql_rec_common.h",
                        "ql_device.h", "ql_exchange.h", "ql_launch.h"),
               sha256="0dec05fd50f7ed0487cf1bb21fa55bb7691a9dbcff5dba8e0caaf48345ffe611",
               summary="profiles/k_xstack_5x500_B64_T1000_counters.md")


def measured_traffic():
    import hashlib
    h = hashlib.sha256()
    for f in TRAFFIC["sources"]:
        with open(os.path.join(ROOT, "paper_1607_04683_amd", "csrc", f), "rb") as fh:
            h.update(fh.read())
    return TRAFFIC["bytes"] if h.hexdigest() == TRAFFIC["sha256"] else None


def log(msg):
    print(f"[bench] {msg}", file=sys.stderr, flush=True)


def parse():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--skip-cpu", action="store_true", help="do not time the CPU oracle")
    ap.add_argument("--quick", action="store_true", help="headline workload only")
    ap.add_argument("--cpu-frames", type=int, default=32000,
                    help="frames of the batch-64 workload the CPU oracle is timed on")
    ap.add_argument("--profile-target", default=None,
                    choices=["stack_b64", "stack_b1", "recurrence_b64", "recurrence_b1",
                             "gemm8192", "lstmp_b256", "lstmp_rec", "pstack_b1", "table1",
                             "qat_b64", "copy"],
                    help="run only one piece (for hardware-counter passes) and exit")
    return ap.parse_args()


class Timer:
    """HIP events on torch's current stream (the stream the library launches on)."""

    def __init__(self, torch):
        self.torch = torch
        self.a = torch.cuda.Event(enable_timing=True)
        self.b = torch.cuda.Event(enable_timing=True)

    def __enter__(self):
        self.a.record()
        return self

    def __exit__(self, *exc):
        self.b.record()
        self.b.synchronize()
        self.ms = self.a.elapsed_time(self.b)


def model_on_device(ql, workload, torch):
    from paper_1607_04683_amd import workloads as wl
    w, _ = wl.model_weights(workload)
    M = ql.quantize_model(w, device="cuda")
    x = torch.from_numpy(wl.features(workload)).cuda()
    return w, M, x


def time_model(ql, torch, M, x, steps, warmup, frames=False):
    """ms per forward pass (events + wall clock), posteriors preallocated.
    frames: x holds base frames [nframes][B][dim]; the frontend's stacking runs
    inside the input quantizer."""
    if frames:
        T, B = ql.stacked_input_count(x.shape[0]), x.shape[1]
        fwd = ql.acoustic_model_forward_frames
    else:
        T, B, _ = x.shape
        fwd = ql.acoustic_model_forward
    ws = ql.Workspace()
    post = torch.empty(T, B, M.Wy.rows, dtype=torch.float32, device="cuda")
    for _ in range(warmup):
        fwd(M, x, workspace=ws, post=post, check=False)
    ql._check(ql.load().ql_workspace_status(ql._ptr(ws.buf), ql._stream()), "warmup")
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    with Timer(torch) as tm:
        for _ in range(steps):
            fwd(M, x, workspace=ws, post=post, check=False)
    torch.cuda.synchronize()
    wall = (time.perf_counter() - t0) * 1e3
    ql._check(ql.load().ql_workspace_status(ql._ptr(ws.buf), ql._stream()), "timed steps")
    return tm.ms / steps, wall / steps


def table1_sweep(ql, torch, wl, steps, warmup):
    """The ten architectures of Table 1 (4-5 layers of 300-500 cells; 5 x 500
    with projections of 100-400 units) with synthetic weights and an 8192-way
    softmax, streaming one utterance of T = 500 presented frames."""
    import numpy as np
    out = []
    T = 500
    x = torch.from_numpy(wl.stacked_features(np.random.Generator(np.random.PCG64(0)), T, 1)).cuda()
    for (layers, hidden, proj) in ((4, 300, 0), (5, 300, 0), (4, 400, 0), (5, 400, 0),
                                   (4, 500, 0), (5, 500, 0), (5, 500, 100), (5, 500, 200),
                                   (5, 500, 300), (5, 500, 400)):
        w = wl.random_model(320, hidden, layers, proj=proj, states=8192, seed=0)
        M = ql.quantize_model(w, device="cuda")
        ms, _ = time_model(ql, torch, M, x, steps, warmup)
        # weight codes a frame streams through the layers (decode-style bytes)
        wbytes = sum(4 * L.hidden * (L.n_in + L.width) + L.proj * L.hidden for L in M.layers)
        us = ms * 1e3 / T
        out.append(dict(arch=f"{layers}x{hidden}" + (f" P{proj}" if proj else ""),
                        ms_per_step=round(ms, 3), frames_per_s=round(T / (ms * 1e-3), 1),
                        us_per_frame=round(us, 2),
                        wavefront_layers=ql.stack_layers_per_launch(M, T, 1),
                        weight_bytes_per_frame=wbytes,
                        weight_frac_of_hbm=round(wbytes / (us * 1e-6) / 1e9 / HBM_PEAK_GBS, 4)))
        del M
    return out


def recurrence_kernel(ql, torch, M, x, reps):
    """Average duration of one persistent-recurrence launch (layer 2 of the
    model, its real input pre-activations), by HIP events around each call."""
    T, B, _ = x.shape
    L1, L2 = M.layers[0], M.layers[1]
    h1 = ql.lstm_layer_forward(L1, x)["h"]
    gx, _ = ql.quantized_matmul(L2.Wx, h1.reshape(T * B, -1), ql.QL_ACT_PER_ROW, L2.bias)
    gx = gx.reshape(T, B, -1)
    ws = ql.Workspace()
    out = {"h": torch.empty(T, B, L2.width, dtype=torch.float32, device="cuda")}
    for _ in range(2):
        ql.lstm_recurrence(L2, gx, workspace=ws, out=out, check=False)
    torch.cuda.synchronize()
    ms = []
    for _ in range(reps):
        with Timer(torch) as tm:
            ql.lstm_recurrence(L2, gx, workspace=ws, out=out, check=False)
        ms.append(tm.ms)
    ql._check(ql.load().ql_workspace_status(ql._ptr(ws.buf), ql._stream()), "recurrence")
    H, R = L2.hidden, L2.width
    wh_bytes = 4 * H * R                       # W_h' codes streamed once per step
    alg = (T * wh_bytes                        # weights, per step (decode-style)
           + T * B * 4 * H * 4                 # read W_x x + b (fp32)
           + T * B * R * 4                     # write h (fp32)
           + T * B * R + T * B * 12)           # write codes of h + per-row params
    avg = sum(ms) / len(ms)
    return dict(avg_ms=avg, min_ms=min(ms), alg_bytes=alg, per_step_us=avg * 1e3 / T,
                wh_bytes_per_step=wh_bytes)


def time_f32_model(ql, torch, workload, steps, warmup):
    """ms per forward pass of the unquantized fp32 model on the same workload."""
    from paper_1607_04683_amd import workloads as wl
    w, _ = wl.model_weights(workload)
    M = ql.f32_model(w, device="cuda")
    x = torch.from_numpy(wl.features(workload)).cuda()
    T, B, _ = x.shape
    ws = ql.Workspace()
    post = torch.empty(T, B, M.Wy.shape[0], dtype=torch.float32, device="cuda")
    for _ in range(warmup):
        ql.f32_acoustic_model_forward(M, x, workspace=ws, post=post, check=False)
    torch.cuda.synchronize()
    with Timer(torch) as tm:
        for _ in range(steps):
            ql.f32_acoustic_model_forward(M, x, workspace=ws, post=post, check=False)
    ql._check(ql.load().ql_workspace_status(ql._ptr(ws.buf), ql._stream()), "fp32 steps")
    return tm.ms / steps


def time_layer(ql, torch, workload, steps, warmup):
    """ms per lstm_layer_forward call of a one-layer workload (no output layer)."""
    from paper_1607_04683_amd import workloads as wl
    w, _ = wl.model_weights(workload)
    L = ql.quantize_layer(w["layers"][0])
    x = torch.from_numpy(wl.features(workload)).cuda()
    ws = ql.Workspace()
    for _ in range(warmup):
        ql.lstm_layer_forward(L, x, workspace=ws, check=False)
    torch.cuda.synchronize()
    with Timer(torch) as tm:
        for _ in range(steps):
            ql.lstm_layer_forward(L, x, workspace=ws, check=False)
    ql._check(ql.load().ql_workspace_status(ql._ptr(ws.buf), ql._stream()), "layer steps")
    return tm.ms / steps


def stack_kernel(ql, torch, M, x, n, reps):
    """Average duration of one wavefront launch over the model's first n
    layers (their real input codes), by HIP events around each call, and its
    algorithmic bytes: every layer-step streams both weight matrices once
    (decode-style), plus the codes (and per-row params) read and written."""
    T, B, n_in = x.shape
    layers = M.layers[:n]
    H = layers[0].hidden
    xq = ql.quantize_activations(x.reshape(T * B, n_in))
    outs = [ql.QAct.empty(T * B, H, x.device) for _ in range(n)]
    ws = ql.Workspace()
    for _ in range(2):
        ql.lstm_stack_forward(layers, xq, T, B, outs=outs, workspace=ws, check=False)
    torch.cuda.synchronize()
    ms = []
    for _ in range(reps):
        with Timer(torch) as tm:
            ql.lstm_stack_forward(layers, xq, T, B, outs=outs, workspace=ws, check=False)
        ms.append(tm.ms)
    ql._check(ql.load().ql_workspace_status(ql._ptr(ws.buf), ql._stream()), "stack")
    w_step = sum(4 * L.hidden * (L.n_in + L.hidden) for L in layers)
    rows = T * B
    alg = (T * w_step                          # W_x' and W_h' of every layer, per step
           + rows * (n_in + 12)                # input codes + params
           + n * rows * (H + 12)               # codes + params written by every layer
           + (n - 1) * rows * (H + 12))        # read again by the next layer
    avg = sum(ms) / len(ms)
    ops = 2 * T * B * w_step                   # every 8-bit multiply-accumulate, both products
    return dict(avg_ms=avg, min_ms=min(ms), alg_bytes=alg, layers=n, int8_ops=ops,
                us_per_frame=avg * 1e3 / T, weight_bytes_per_frame=w_step)


def lstmp_recurrence_kernel(ql, torch, M, x, reps):
    """One persistent-recurrence launch of the LSTMP model's second layer (its
    real pre-activations): per-step time against the bandwidth floor of
    streaming W_h' and W_r' (decode-style) and the int8 MFMA peak."""
    T, B, _ = x.shape
    L1, L2 = M.layers[0], M.layers[1]
    h1 = ql.lstm_layer_forward(L1, x)["h"]
    gx, _ = ql.quantized_matmul(L2.Wx, h1.reshape(T * B, -1), ql.QL_ACT_PER_ROW, L2.bias)
    gx = gx.reshape(T, B, -1)
    del h1
    ws = ql.Workspace()
    out = {"h": torch.empty(T, B, L2.width, dtype=torch.float32, device="cuda")}
    ql.lstm_recurrence(L2, gx, workspace=ws, out=out, check=False)
    torch.cuda.synchronize()
    ms = []
    for _ in range(reps):
        with Timer(torch) as tm:
            ql.lstm_recurrence(L2, gx, workspace=ws, out=out, check=False)
        ms.append(tm.ms)
    ql._check(ql.load().ql_workspace_status(ql._ptr(ws.buf), ql._stream()), "lstmp recurrence")
    H, P = L2.hidden, L2.proj
    w_bytes = 4 * H * P + P * H                # W_h' and W_r' codes per step
    ops = 2 * B * (4 * H * P + P * H)          # per step
    avg = sum(ms) / len(ms)
    us = avg * 1e3 / T
    return dict(kernel="k_xrec (LSTMP 2048/512 layer 2, B=256, T=800; an eighth of the batch per XCD)",
                avg_ms=round(avg, 3), us_per_step=round(us, 2),
                weight_bytes_per_step=w_bytes,
                weight_frac_of_hbm=round(w_bytes / (us * 1e-6) / 1e9 / HBM_PEAK_GBS, 5),
                int8_ops_per_step=ops,
                mfma_frac=round(ops / (us * 1e-6) / 1e12 / INT8_PEAK_TOPS, 5))


def qat_step(ql, torch, W, steps, warmup):
    """The quantization-aware training step (Section 3.2, Algorithm 1) on the
    5 x 500 + 8192 model: a mini-batch of B utterances x T frames with
    synthetic frame targets; parameters updated in place every step."""
    from paper_1607_04683_amd import workloads as wl
    w, _ = wl.model_weights(W)
    P = ql.train_params(w)
    x = torch.from_numpy(wl.features(W)).cuda()
    y = torch.from_numpy(wl.frame_targets(W)).cuda()
    ws = ql.Workspace()
    g = None
    for _ in range(warmup):
        _, g = ql.train_step(P, x, y, 0.1, grads=g, workspace=ws, check=False)
    torch.cuda.synchronize()
    with Timer(torch) as tm:
        for _ in range(steps):
            loss, g = ql.train_step(P, x, y, 0.1, grads=g, workspace=ws, check=False)
    ql._check(ql.load().ql_workspace_status(ql._ptr(ws.buf), ql._stream()), "train steps")
    ms = tm.ms / steps
    T, B = W.T, W.B
    N = T * B
    m = W.model
    # fp32 flops of the gradient products (2 per multiply-add): the output
    # layer's dW_y and dh_L, every layer's dW_x, dW_h and (but the first) dx
    fl = 2 * N * m.states * m.hidden * 2
    for l, (i, h, _) in enumerate(m.layer_dims()):
        fl += 2 * N * 4 * h * i + 2 * N * 4 * h * h + (2 * N * 4 * h * i if l > 0 else 0)
    return dict(workload=W.name + ", quantization-aware SGD step, synthetic frame targets",
                ms_per_step=round(ms, 3), frames_per_s=round(N / (ms * 1e-3), 1),
                loss=round(float(loss.item()), 4),
                grad_product_tflop=round(fl / 1e12, 3),
                grad_product_tflops_over_step=round(fl / (ms * 1e-3) / 1e12, 2),
                note="the step's whole time against the fp32 flops of its gradient products "
                     "(a lower bound on their MFMA rate; fp32 peak 157.3 TF/s)")


def gemm_sweep(ql, torch, n, reps):
    from paper_1607_04683_amd import workloads as wl
    A, Bm = wl.gemm_operands(n, n, n, seed=0)
    Ad, Bd = ql.device_codes(A), ql.device_codes(Bm)
    sa = torch.from_numpy(A.sum(1, dtype="int64").astype("int32")).cuda()
    sb = torch.from_numpy(Bm.sum(1, dtype="int64").astype("int32")).cuda()
    Cm = torch.empty(n, n, dtype=torch.int32, device="cuda")
    for _ in range(2):
        ql.gemm_u8(Ad, Bd, n, sa, sb, out=Cm)
    torch.cuda.synchronize()
    with Timer(torch) as tm:
        for _ in range(reps):
            ql.gemm_u8(Ad, Bd, n, sa, sb, out=Cm)
    ms = tm.ms / reps
    tops = 2.0 * n ** 3 / (ms * 1e-3) / 1e12
    return dict(n=n, ms=ms, tops=tops, frac_of_peak=tops / INT8_PEAK_TOPS)


def _cpu_name():
    try:
        for line in open("/proc/cpuinfo"):
            if line.startswith("model name"):
                return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return "unknown"


def cpu_baselines_all(threads):
    """The oracle on every workload (bounded samples), with `threads` OpenMP
    threads and, for the three smallest, one thread as well."""
    import numpy as np

    from oracle import oracle
    from paper_1607_04683_amd import workloads as wl
    oracle.lib()
    out = []

    def run(name, fn, unit, scale, sample, nthreads):
        oracle.set_threads(nthreads)
        t0 = time.perf_counter()
        fn()
        dt = time.perf_counter() - t0
        out.append(dict(workload=name, value=round(scale / dt, 2), unit=unit, cores=nthreads,
                        kind="oracle", sample=f"{sample}, {dt:.2f} s"))

    W0 = wl.QMATMUL_16x128x256
    Wm, Xm = wl.qmatmul_operands(W0)
    q = oracle.quantize(Wm, 1)
    reps = 2000
    for n in (threads, 1):
        run(W0.name, lambda: [oracle.quantized_matmul(q, Xm, act_gran=0) for _ in range(reps)],
            "qmatmul/s", reps, f"{reps} calls", n)
    for W, Tcap1 in ((wl.LSTM1x500_T300_B1, 300), (wl.LSTM5x500_S8192_T500_B1, 100)):
        w, _ = wl.model_weights(W)
        x = wl.features(W)
        x1 = np.ascontiguousarray(x[:Tcap1])
        if W.model.states:
            Mq = oracle.quantize_model(w)
            f = lambda xx, Mq=Mq: oracle.acoustic_model_forward(Mq, xx)
        else:
            Lq = oracle.quantize_layer(w["layers"][0])
            f = lambda xx, Lq=Lq: oracle.lstm_layer_forward(Lq, xx)
        run(W.name, lambda: f(x), "frames/s", x.shape[0], f"{x.shape[0]} frames", threads)
        run(W.name, lambda: f(x1), "frames/s", x1.shape[0], f"first {x1.shape[0]} frames", 1)
    W5 = wl.LSTMP4x2048P512_S16384_T800_B256
    w5, _ = wl.model_weights(W5)
    Mq5 = oracle.quantize_model(w5)
    nu, T5 = 32, 50
    x5 = np.ascontiguousarray(wl.features(W5, utterances=list(range(nu)))[:T5])
    run(W5.name, lambda: oracle.acoustic_model_forward(Mq5, x5), "frames/s", nu * T5,
        f"{nu} utterances x {T5} frames", threads)
    oracle.set_threads(threads)
    return out


def cpu_baseline(workload, frames):
    """The oracle (untuned) on a bounded sample of the same workload: the first
    `frames` frames of the first utterances (utterances are independent)."""
    import numpy as np

    from oracle import oracle
    from paper_1607_04683_amd import workloads as wl
    w, _ = wl.model_weights(workload)
    threads = max(1, int(os.environ.get("OMP_NUM_THREADS", os.cpu_count() or 1)))
    n_utt = min(workload.B, max(threads, -(-frames // workload.T)))
    T = max(1, min(workload.T, frames // n_utt))
    x = wl.features(workload, utterances=list(range(n_utt)))[:T]
    Mq = oracle.quantize_model(w)
    oracle.lib()
    t0 = time.perf_counter()
    oracle.acoustic_model_forward(Mq, np.ascontiguousarray(x))
    dt = time.perf_counter() - t0
    cores = int(os.environ.get("OMP_NUM_THREADS", 0)) or len(os.sched_getaffinity(0))
    cpu = _cpu_name()
    return dict(value=T * n_utt / dt, unit="frames/s", cores=cores, kind="oracle",
                sample=f"{n_utt} utterances x {T} frames of the batch-64 workload "
                       f"({T * n_utt} frames, {dt:.1f} s, {cpu})")


def profile_target(ql, torch, target, reps):
    """One piece of the benchmark alone, so a counter pass sees only its kernels."""
    from paper_1607_04683_amd import workloads as wl
    if target.startswith("stack"):
        W = wl.LSTM5x500_S8192_T1000_B64 if target.endswith("b64") else wl.LSTM5x500_S8192_T500_B1
        _, M, x = model_on_device(ql, W, torch)
        n = ql.stack_layers_per_launch(M, W.T, W.B)
        out = stack_kernel(ql, torch, M, x, n, reps)
        out["workload"] = W.name
    elif target.startswith("recurrence"):
        W = wl.LSTM5x500_S8192_T1000_B64 if target.endswith("b64") else wl.LSTM5x500_S8192_T500_B1
        _, M, x = model_on_device(ql, W, torch)
        out = recurrence_kernel(ql, torch, M, x, reps)
        out["workload"] = W.name
    elif target == "pstack_b1":
        import numpy as np
        T = 500
        w = wl.random_model(320, 500, 5, proj=200, states=8192, seed=0)
        M = ql.quantize_model(w, device="cuda")
        x = torch.from_numpy(wl.stacked_features(np.random.Generator(np.random.PCG64(0)), T,
                                                 1)).cuda()
        ms, _ = time_model(ql, torch, M, x, 5, 2)
        out = dict(workload="5xLSTM500 P200 + softmax8192, T500 B1", ms_per_step=round(ms, 3),
                   us_per_frame=round(ms * 1e3 / T, 2))
    elif target == "table1":
        out = dict(table1_b1=table1_sweep(ql, torch, wl, 5, 2))
    elif target == "gemm8192":
        out = gemm_sweep(ql, torch, 8192, reps)
    elif target == "lstmp_b256":
        W = wl.LSTMP4x2048P512_S16384_T800_B256
        _, M, x = model_on_device(ql, W, torch)
        ms, _ = time_model(ql, torch, M, x, 2, 1)
        out = dict(workload=W.name, ms_per_step=round(ms, 3))
    elif target == "lstmp_rec":
        W = wl.LSTMP4x2048P512_S16384_T800_B256
        _, M, x = model_on_device(ql, W, torch)
        out = lstmp_recurrence_kernel(ql, torch, M, x, reps)
    elif target == "qat_b64":
        out = qat_step(ql, torch, wl.LSTM5x500_S8192_T1000_B64, 2, 1)
    else:  # a plain device copy of 1 GiB: calibrates the byte counters
        n = 1 << 28
        src = torch.ones(n, dtype=torch.float32, device="cuda")
        dst = torch.empty_like(src)
        for _ in range(reps):
            dst.copy_(src)
        torch.cuda.synchronize()
        out = dict(bytes_read=4 * n, bytes_written=4 * n, copies=reps)
    out["target"] = target
    print(json.dumps(out), flush=True)


def main():
    args = parse()
    if args.gpus != 1:
        print(f"bench.py measures one GPU: this build has no multi-GPU path "
              f"(--gpus {args.gpus} requested). Utterances are independent, so a "
              f"data-parallel run is N copies of this one.", file=sys.stderr)
        sys.exit(2)
    import torch

    from paper_1607_04683_amd import qlstm as ql
    from paper_1607_04683_amd import workloads as wl
    ql.load()
    torch.cuda.set_device(0)
    if args.profile_target:
        profile_target(ql, torch, args.profile_target, reps=3)
        return

    # ---- headline: 5x500 + softmax 8192 at batch 64 x T=1000
    W64 = wl.LSTM5x500_S8192_T1000_B64
    log(f"setup {W64.name}")
    _, M64, x64 = model_on_device(ql, W64, torch)
    ms, wall_ms = time_model(ql, torch, M64, x64, args.steps, args.warmup)
    frames = W64.T * W64.B
    value = frames / (ms * 1e-3)
    log(f"batch 64: {ms:.3f} ms/step (wall {wall_ms:.3f}) -> {value:.0f} frames/s")

    nst = ql.stack_layers_per_launch(M64, W64.T, W64.B)
    rec = stack_kernel(ql, torch, M64, x64, nst, reps=5)
    achieved = rec["alg_bytes"] / (rec["avg_ms"] * 1e-3) / 1e9
    log(f"wavefront kernel ({nst} layers): {rec['avg_ms']:.3f} ms/launch, "
        f"{rec['us_per_frame']:.2f} us/frame, {achieved:.1f} GB/s algorithmic")
    roofline = dict(bound="hbm", kernel=f"k_xstack ({nst} 500-cell layers, B=64, T=1000; one XCD per layer)",
                    achieved=round(achieved, 2), peak=HBM_PEAK_GBS, unit="GB/s",
                    frac=round(achieved / HBM_PEAK_GBS, 5), traffic=measured_traffic(),
                    traffic_unit="bytes per launch", traffic_source=TRAFFIC["summary"],
                    avg_launch_ms=round(rec["avg_ms"], 4), alg_bytes=rec["alg_bytes"],
                    int8_ops=rec["int8_ops"],
                    mfma_frac=round(rec["int8_ops"] / (rec["avg_ms"] * 1e-3) / 1e12 /
                                    INT8_PEAK_TOPS, 5))

    extra = {}
    if not args.quick:
        fr64 = torch.from_numpy(wl.frames(W64)).cuda()
        msf, _ = time_model(ql, torch, M64, fr64, max(3, args.steps // 2), args.warmup,
                            frames=True)
        extra["frontend_fused"] = dict(
            workload=W64.name + ", fed 40-dim base frames (8 stacked, every 3rd presented)",
            ms_per_step=round(msf, 3), frames_per_s=round(frames / (msf * 1e-3), 1))
        log(f"fused frontend: {extra['frontend_fused']}")
        del fr64
        W1 = wl.LSTM5x500_S8192_T500_B1
        log(f"setup {W1.name}")
        _, M1, x1 = model_on_device(ql, W1, torch)
        ms1, _ = time_model(ql, torch, M1, x1, max(3, args.steps // 2), args.warmup)
        n1 = ql.stack_layers_per_launch(M1, W1.T, W1.B)
        rec1 = stack_kernel(ql, torch, M1, x1, n1, reps=5)
        extra["batch1"] = dict(workload=W1.name, ms_per_step=round(ms1, 3),
                               frames_per_s=round(W1.T / (ms1 * 1e-3), 1),
                               wavefront_layers=n1,
                               wavefront_us_per_frame=round(rec1["us_per_frame"], 3),
                               weight_GBs=round(rec1["weight_bytes_per_frame"] /
                                                (rec1["us_per_frame"] * 1e-6) / 1e9, 1),
                               weight_frac_of_hbm=round(rec1["weight_bytes_per_frame"] /
                                                        (rec1["us_per_frame"] * 1e-6) / 1e9 /
                                                        HBM_PEAK_GBS, 5))
        log(f"batch 1: {extra['batch1']}")
        del M1, x1
        W0 = wl.LSTM1x500_T300_B1
        ms0 = time_layer(ql, torch, W0, max(3, args.steps // 2), args.warmup)
        extra["layer_b1"] = dict(workload=W0.name, ms_per_step=round(ms0, 3),
                                 frames_per_s=round(W0.T / (ms0 * 1e-3), 1))
        log(f"one layer, batch 1: {extra['layer_b1']}")
        f64 = time_f32_model(ql, torch, W64, 3, 1)
        f1 = time_f32_model(ql, torch, W1, 3, 1)
        extra["fp32_model"] = dict(
            note="unquantized fp32 model, same API and kernel structure",
            batch64=dict(ms_per_step=round(f64, 3), frames_per_s=round(frames / (f64 * 1e-3), 1),
                         int8_speedup=round(f64 / ms, 3)),
            batch1=dict(ms_per_step=round(f1, 3), frames_per_s=round(W1.T / (f1 * 1e-3), 1),
                        int8_speedup=round(f1 / ms1, 3)))
        log(f"fp32 model: {extra['fp32_model']}")
        extra["table1_b1"] = table1_sweep(ql, torch, wl, max(3, args.steps // 4), args.warmup)
        log(f"Table 1 architectures, batch 1: {extra['table1_b1']}")
        W5 = wl.LSTMP4x2048P512_S16384_T800_B256
        log(f"setup {W5.name}")
        _, M5, x5 = model_on_device(ql, W5, torch)
        ms5, _ = time_model(ql, torch, M5, x5, 3, 1)
        extra["lstmp_b256"] = dict(workload=W5.name, ms_per_step=round(ms5, 3),
                                   frames_per_s=round(W5.T * W5.B / (ms5 * 1e-3), 1),
                                   recurrence=lstmp_recurrence_kernel(ql, torch, M5, x5, 3))
        log(f"LSTMP batch 256: {extra['lstmp_b256']}")
        del M5, x5
        torch.cuda.empty_cache()
        extra["qat_b64"] = qat_step(ql, torch, W64, 3, 1)
        log(f"quantization-aware training step: {extra['qat_b64']}")
        torch.cuda.empty_cache()
        extra["gemm_sweep"] = [gemm_sweep(ql, torch, n, reps=10) for n in wl.GEMM_SWEEP]
        for g in extra["gemm_sweep"]:
            g.update({k: round(v, 4) for k, v in g.items() if isinstance(v, float)})
            g["note"] = ("row sums of the code operands computed on the host before timing "
                         "(an O(n^2) pass outside the timed region)")
        log(f"GEMM sweep: {extra['gemm_sweep']}")

    cpu = None
    if not args.skip_cpu:
        log("timing the CPU oracle")
        cpu = cpu_baseline(W64, args.cpu_frames)
        cpu["value"] = round(cpu["value"], 2)
        log(f"cpu baseline: {cpu}")
        if not args.quick:
            extra["cpu_baselines"] = cpu_baselines_all(cpu["cores"])
            log(f"cpu baselines: {extra['cpu_baselines']}")

    line = {
        "metric": METRIC, "value": round(value, 1), "unit": "frames/s", "n_gpus": 1,
        "steps": args.steps, "warmup": args.warmup, "ms_per_step": round(ms, 4),
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None, "dtype": "u8",
        "data": "synthetic",
        "config": {"workload": W64.name, "layers": 5, "cells": 500, "input": 320,
                   "states": 8192, "batch": W64.B, "T": W64.T,
                   "quantization": "uint8 weights per gate block, uint8 activations per vector"},
        "roofline": roofline, "cpu_baseline": cpu, **extra,
    }
    print(json.dumps(line), flush=True)


if __name__ == "__main__":
    main()
