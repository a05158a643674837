"""Benchmark of the SONIQ mixed-precision quantized GEMM on one MI355X.

One step = the whole per-call hot path on one batch: quantize, permute and
pack the fp32 activations (soniq_quantize_act), then the packed x packed
integer MAC with the bf16 epilogue (soniq_mp_gemm).  Weights are packed
before timing (they are static per layer); their packing time is reported
separately.  Inputs are resident in HBM when timing starts.  Both operands
rotate over distinct copies (fp32 activations up to 512 MB, packed weights
up to 1 GiB), so every step reads them from HBM rather than from the 256 MB
Infinity Cache, as a layer of a real network would.

Prints one JSON line.  The metric has two halves, both measured in the
default run: `value` is the TOPS of the large square GEMM step
(8192 x 8192 x 8192, 4/8-bit operands; 2*M*N*K integer ops per step over
the whole step), with `roofline` on its dominant kernel, timed with HIP
events on the stream it runs on; `gemv` holds the batch-1 decode GEMV
(W[11008, 4096], 2/4-bit weights) as HBM GB/s on the packed weight bytes,
with its own roofline.  The bf16 comparators (torch's GEMM on the same
shapes) are timed with the same protocol: operands rotated the same way,
the timed calls replayed from one captured HIP graph.  `cpu_baseline` is
the CPU oracle on a bounded sample of the headline workload.

`--copy-calibration` instead runs a plain 1 GiB device copy, whose
FETCH_SIZE / WRITE_SIZE counters calibrate the HBM traffic figures.
"""
from __future__ import annotations

import argparse
import hashlib
import json
import math
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

METRIC = "mixed-precision GEMM TOPS & GEMV HBM GB/s (1 MI355X); speedup vs bf16 GEMM"
DEFAULT_WORKLOAD = "square_8192"
DEFAULT_GEMV_WORKLOAD = "decode_11008_m1"
HBM_PEAK_GBS = 8000.0     # MI355X HBM3E
INT8_PEAK_TOPS = 5000.0   # MI355X dense int8 MFMA
ROTATE_A_BYTES = 512 << 20
ROTATE_W_BYTES = 1 << 30
MAX_W_COPIES = 96
TRAFFIC_FILE = os.path.join(ROOT, "profiles", "hbm_traffic.txt")
KERNEL_SOURCE = os.path.join(ROOT, "paper_2311_14114_amd", "csrc", "soniq_kernels.hip")


def container(b: int) -> int:
    return 1 if b <= 1 else 2 if b <= 2 else 4 if b <= 4 else 8


def algorithmic(case, info):
    """Algorithmic bytes and ops of one step: no padding, no debug dumps."""
    M, N, K = case["M"], case["N"], case["K"]
    ab = case["a_bits"]
    act_packed = sum(M * int((ab == b).sum()) * container(int(b)) // 8 for b in np.unique(ab))
    S = len(np.unique(ab))
    return dict(
        ops=2 * M * N * K,
        a_fp32=M * K * 4,
        a_packed=act_packed,
        # the dense copy holds each weight in its own width; the container
        # layout rounds a width up to 1, 2, 4 or 8 bits
        w_packed=(int(case["w_bits"].astype(np.int64).sum()) * K // 8 if case.get("dense")
                  else int(info.packed_w_bytes_algorithmic)),
        # per output channel: scale and one code sum per activation group
        w_side=N * (4 + 4 * S),
        y=M * N * 2,
    )


def sign_nibbles(case) -> bool:
    """1-bit weight channels are packed in 4-bit containers where the MFMA
    GEMM or the block-sum GEMV (which takes containers of 2 bits and up)
    runs the layer; the plain GEMV keeps bits."""
    return bool((case["w_bits"] == 1).any()) and (not uses_gemv(case) or
                                                  bool(case.get("act_group_bits", 0)))


def uses_gemv(case) -> bool:
    # batches of at most 8 rows run a GEMV form (with sub-group scales the
    # block-sum GEMV)
    return case["M"] <= 8


def gemv_kernel(case) -> str:
    if case.get("act_group_bits", 0):
        return "k_gemv_g"
    if case.get("dense"):
        return "k_gemv_dense"
    return "k_gemv" if case["M"] == 1 else "k_gemv_mfma"


def run_gpu(case, steps, warmup, rotate=True, graph=True, conv_input=False, f8f6f4=False,
            implicit=False):
    """Pack, quantize and time one workload; case["dense"] asks for the dense
    weight copy (SONIQ_WPACK_DENSE), which the GEMV forms read."""
    import torch
    import paper_2311_14114_amd as sq

    torch.cuda.set_device(0)
    dev = torch.device("cuda")
    M, N, K = case["M"], case["N"], case["K"]
    stream = torch.cuda.current_stream()
    W = torch.from_numpy(case["W"]).to(dev)
    A0 = torch.from_numpy(case["A"]).to(dev)

    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    e0.record(stream)
    gbits = case.get("act_group_bits", 0)
    nib = sign_nibbles(case)
    if implicit:
        # the filter as [N, C, 3, 3] and one width per input channel
        Cin = case["X"].shape[1]
        Wf = W.view(N, Cin, 3, 3)
        ch_bits = case["a_bits"][::9]

        def pack():
            return sq.soniq_pack_weights_conv3x3(Wf, case["w_bits"], ch_bits, case["a_signed"],
                                                 sign_nibbles=nib)
    else:
        def pack():
            return sq.soniq_pack_weights(W, case["w_bits"], case["a_bits"], case["a_signed"],
                                         act_group_bits=gbits, sign_nibbles=nib, f8f6f4=f8f6f4,
                                         dense=bool(case.get("dense")))
    ws = [pack()]
    e1.record(stream)
    torch.cuda.synchronize()
    pack_ms = e0.elapsed_time(e1)
    info = ws[0].info
    nw = 1
    if rotate:
        nw = max(1, min(MAX_W_COPIES, math.ceil(ROTATE_W_BYTES / int(info.packed_w_bytes))))
    for _ in range(nw - 1):
        ws.append(pack())
    if implicit:
        Bx, _, Hx, Wx = case["X"].shape
        acts = [sq.soniq_act_create_conv3x3(w, Bx, Hx, Wx) for w in ws]
    else:
        acts = [sq.soniq_act_create(w, M) for w in ws]
    # the quantizer's input: the lowered matrix A, or (conv_input) the
    # convolution's NCHW tensor X, whose 3x3 lowering A is
    src0 = torch.from_numpy(case["X"]).to(dev) if conv_input else A0
    na = max(1, min(8, math.ceil(ROTATE_A_BYTES / (src0.numel() * 4)))) if rotate else 1
    As = [src0] + [src0.clone() for _ in range(na - 1)]
    Y = torch.empty((M, N), dtype=torch.bfloat16, device=dev)

    def step(i):
        act = acts[i % nw]
        if conv_input:
            sq.soniq_quantize_act_conv3x3(act, As[i % na])
        else:
            sq.soniq_quantize_act(act, As[i % na])
        return act, ws[i % nw]

    for i in range(warmup):
        act, w = step(i)
        sq.soniq_mp_gemm(act, w, out=Y)
    torch.cuda.synchronize()

    def full(i):
        # one layer: the conv entry point then the GEMM, or the one-call
        # quantize + GEMM (a single launch for a batch of one row)
        if conv_input or implicit:
            act, w = step(i)
            sq.soniq_mp_gemm(act, w, out=Y)
        else:
            sq.soniq_quantize_mp_gemm(acts[i % nw], ws[i % nw], As[i % na], out=Y)

    def gemm_only(i):
        sq.soniq_mp_gemm(acts[i % nw], ws[i % nw], out=Y)

    def timed(fn):
        # ms per call of fn(0..steps-1) run back to back on the stream
        # between two events, launched eagerly or as one captured HIP graph
        # (the launch overhead of small calls otherwise starves the GPU)
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        if graph:
            g = torch.cuda.CUDAGraph()
            side = torch.cuda.Stream()
            side.wait_stream(stream)
            with torch.cuda.graph(g, stream=side):
                for i in range(steps):
                    fn(i)
            torch.cuda.synchronize()
            g.replay()  # first replay uploads the graph
            torch.cuda.synchronize()
            e0.record(stream)
            g.replay()
            e1.record(stream)
        else:
            torch.cuda.synchronize()
            e0.record(stream)
            for i in range(steps):
                fn(i)
            e1.record(stream)
        torch.cuda.synchronize()
        return e0.elapsed_time(e1) / steps

    # The timed region: exactly `steps` steps between two events, nothing
    # else on the stream.  Then the per-call breakdown (and the roofline's
    # launch durations): each entry point alone, back to back.
    t0 = time.perf_counter()
    total_ms = timed(full) * steps
    wall = time.perf_counter() - t0
    q_ms = timed(step)
    g_ms = timed(gemm_only)
    # the same calls on one weight copy, which then stays in the 256 MB
    # Infinity Cache (reported beside the rotated figure, never as it)
    g_hot_ms = timed(lambda i: sq.soniq_mp_gemm(acts[0], ws[0], out=Y))
    # Decode batches are bandwidth-bound: the plain-read time of the same
    # packed weight bytes (one trivial read per call, rotated over 1 GiB
    # like the weights, timed the same way) is the ceiling the GEMV is held
    # against.
    read_ms = None
    if M <= 8:
        nbytes = int(info.dense_w_bytes if case.get("dense") else info.packed_w_bytes) // 16 * 16
        rbuf = torch.empty(ROTATE_W_BYTES, dtype=torch.uint8, device=dev)
        nsl = max(1, ROTATE_W_BYTES // nbytes) if rotate else 1
        sink = torch.empty((nbytes + 8191) // 8192, dtype=torch.int32, device=dev)
        read_ms = timed(lambda i: sq.soniq_debug_stream_read(rbuf, nbytes, sink,
                                                             offset=(i % nsl) * nbytes))
        del rbuf, sink
    del acts, ws

    # bf16 comparator: torch's GEMM (hipBLASLt) on the same shapes, the same
    # protocol, operands rotated the same way.
    # (always on the lowered matrix A: a bf16 GEMM has no other input form)
    del As
    nab = max(1, min(8, math.ceil(ROTATE_A_BYTES / (A0.numel() * 4)))) if rotate else 1
    Ab = [A0.to(torch.bfloat16) for _ in range(nab)]
    nwb = max(1, min(nw, math.ceil(ROTATE_W_BYTES / (N * K * 2))))
    Wb = [W.to(torch.bfloat16) for _ in range(nwb)]
    for i in range(warmup):
        torch.nn.functional.linear(Ab[i % nab], Wb[i % nwb])
    torch.cuda.synchronize()
    bf16_ms = timed(lambda i: torch.nn.functional.linear(Ab[i % nab], Wb[i % nwb]))
    del Ab, Wb
    return dict(total_ms=total_ms, wall_s=wall, q_ms=q_ms, g_ms=g_ms, g_hot_ms=g_hot_ms,
                pack_ms=pack_ms, read_ms=read_ms,
                bf16_ms=bf16_ms, info=info, na=na, nw=nw)


def source_digest() -> str:
    with open(KERNEL_SOURCE, "rb") as f:
        return hashlib.sha256(f.read()).hexdigest()[:16]


def measured_traffic(kernel: str, workload: str):
    """HBM bytes per launch from the committed counter summary, or None when
    it is missing or was taken on a different kernel source."""
    if not os.path.exists(TRAFFIC_FILE):
        return None
    digest = source_digest()
    with open(TRAFFIC_FILE) as f:
        for line in f:
            if line.startswith("#") or not line.strip():
                continue
            kv = dict(t.split("=", 1) for t in line.split() if "=" in t)
            if kv.get("kernel") == kernel and kv.get("workload") == workload:
                if kv.get("source") != digest:
                    return None
                return int(float(kv["traffic_bytes"]))
    return None


def fused_one_row(case) -> bool:
    """Whether soniq_quantize_mp_gemm runs the step as one k_gemv_fused
    launch (its documented conditions: one row, one scale per precision
    group, the narrow group in 4-bit containers and the wide one, if any,
    in bytes, no 1-bit group, K a multiple of 4 up to 4096)."""
    if case["M"] != 1 or case.get("act_group_bits", 0) or case.get("dense"):
        return False
    widths = sorted(set(int(b) for b in case["a_bits"]))
    return (case["K"] % 4 == 0 and case["K"] <= 4096 and 3 <= widths[0] <= 4
            and (len(widths) == 1 or widths[1] >= 5))


def roofline(case, alg, r, steps):
    """Roofline of the dominant kernel of one step."""
    if fused_one_row(case):
        # the step is one launch: the row's quantization and the GEMV
        t = r["total_ms"] / steps * 1e-3
        byt = alg["a_fp32"] + alg["w_packed"] + alg["w_side"] + alg["y"]
        ach = byt / t / 1e9
        return dict(bound="hbm", achieved=ach, peak=HBM_PEAK_GBS, unit="GB/s",
                    frac=ach / HBM_PEAK_GBS, traffic=measured_traffic("k_gemv_fused", case["name"]),
                    kernel="k_gemv_fused", algorithmic_bytes=byt, launch_us=t * 1e6)
    if r["q_ms"] >= r["g_ms"]:
        kernel = "soniq_quantize_act"
        byt = alg["a_fp32"] + alg["a_packed"]
        t = r["q_ms"] * 1e-3
        ach = byt / t / 1e9
        return dict(bound="hbm", achieved=ach, peak=HBM_PEAK_GBS, unit="GB/s",
                    frac=ach / HBM_PEAK_GBS, traffic=measured_traffic(kernel, case["name"]),
                    kernel=kernel, algorithmic_bytes=byt, launch_us=t * 1e6)
    t = r["g_ms"] * 1e-3
    byt = alg["a_packed"] + alg["w_packed"] + alg["w_side"] + alg["y"]
    kernel = (gemv_kernel(case) if uses_gemv(case) else
              "k_gemm_g" if case.get("act_group_bits", 0) else "k_gemm")
    traffic = measured_traffic(kernel, case["name"])
    # the bound is whichever resource needs longer at its peak
    if uses_gemv(case) or byt / (HBM_PEAK_GBS * 1e9) >= alg["ops"] / (INT8_PEAK_TOPS * 1e12):
        ach = byt / t / 1e9
        return dict(bound="hbm", achieved=ach, peak=HBM_PEAK_GBS, unit="GB/s",
                    frac=ach / HBM_PEAK_GBS, traffic=traffic, kernel=kernel,
                    algorithmic_bytes=byt, launch_us=t * 1e6)
    ach = alg["ops"] / t / 1e12
    return dict(bound="mfma", achieved=ach, peak=INT8_PEAK_TOPS, unit="TFLOP/s",
                frac=ach / INT8_PEAK_TOPS, traffic=traffic, kernel=kernel,
                algorithmic_ops=alg["ops"], launch_us=t * 1e6)


def gemv_record(case, r, steps):
    """The batch-1 (or batch-8) decode half of the metric: HBM GB/s on the
    packed weight bytes, the GEMV kernel's roofline (soniq_mp_gemm alone,
    after a separate quantize call) and the one-call step's (for a one-row
    batch soniq_quantize_mp_gemm is one launch that also quantizes the row),
    against torch's bf16 GEMM timed the same way."""
    alg = algorithmic(case, r["info"])
    step_s = r["total_ms"] / steps * 1e-3
    g_s = r["g_ms"] * 1e-3
    kbytes = alg["a_packed"] + alg["w_packed"] + alg["w_side"] + alg["y"]
    kernel = gemv_kernel(case)
    ach = kbytes / g_s / 1e9
    rec = {
        "workload": case["name"], "M": case["M"], "N": case["N"], "K": case["K"],
        "a_bits": sorted(set(case["a_bits"].tolist())),
        "w_bits": sorted(set(case["w_bits"].tolist())),
        "weight_copies": r["nw"], "packed_weight_bytes": alg["w_packed"],
        "dense_weights": bool(case.get("dense")),
        "packed_weight_gbs": alg["w_packed"] / g_s / 1e9,
        "step_packed_weight_gbs": alg["w_packed"] / step_s / 1e9,
        "step_us": step_s * 1e6, "mp_gemm_us": g_s * 1e6, "quantize_act_us": r["q_ms"] * 1e3,
        "mp_gemm_weights_cache_hot_us": r["g_hot_ms"] * 1e3,
        # a plain read of the packed weight bytes, rotated and timed the same
        # way, and the GEMV's time as a fraction of it
        "plain_read_us": r["read_ms"] * 1e3,
        "plain_read_gbs": alg["w_packed"] / (r["read_ms"] * 1e-3) / 1e9,
        "of_plain_read": r["read_ms"] / r["g_ms"],
        "roofline": dict(bound="hbm", achieved=ach, peak=HBM_PEAK_GBS, unit="GB/s",
                         frac=ach / HBM_PEAK_GBS, traffic=measured_traffic(kernel, case["name"]),
                         kernel=kernel, algorithmic_bytes=kbytes, launch_us=g_s * 1e6),
        "bf16_linear_us": r["bf16_ms"] * 1e3,
        "speedup_vs_bf16": {"gemv": r["bf16_ms"] / r["g_ms"], "step": r["bf16_ms"] * 1e-3 / step_s},
    }
    if fused_one_row(case):
        sbytes = alg["a_fp32"] + alg["w_packed"] + alg["w_side"] + alg["y"]
        sa = sbytes / step_s / 1e9
        rec["roofline_step"] = dict(bound="hbm", achieved=sa, peak=HBM_PEAK_GBS, unit="GB/s",
                                    frac=sa / HBM_PEAK_GBS,
                                    traffic=measured_traffic("k_gemv_fused", case["name"]),
                                    kernel="k_gemv_fused", algorithmic_bytes=sbytes,
                                    launch_us=step_s * 1e6)
    return rec


def cpu_baseline(case, budget_s=12.0):
    """The CPU oracle, as it stands, on a bounded sample of the workload: the
    weights are quantized once, untimed (as the GPU packs them once); each
    timed run quantizes the first `rows` activation rows, runs the integer
    MAC and the epilogue.  Rows grow until one run takes about a second."""
    import oracle
    oracle.lib()
    M, N, K = case["M"], case["N"], case["K"]
    q_w, s_w = oracle.quantize_weights(case["W"], case["w_bits"])

    def one(rows):
        A = np.ascontiguousarray(case["A"][:rows])
        t0 = time.perf_counter()
        if case.get("act_group_bits", 0):
            q_a, s_a, seg_bits, seg_of = oracle.quantize_act_grouped(
                A, case["a_bits"], case["a_signed"], case["act_group_bits"])
        else:
            q_a, s_a, seg_bits, seg_of = oracle.quantize_act(A, case["a_bits"], case["a_signed"])
        acc = oracle.mac(q_a, q_w, seg_of, len(seg_bits))
        oracle.epilogue_replay(acc, s_a, s_w)
        return time.perf_counter() - t0

    rows = min(M, 8)
    while True:
        dt = one(rows)
        if rows == M or dt >= 1.0:
            break
        rows = min(M, max(rows + 1, int(rows * min(8.0, 1.2 / max(dt, 1e-3)))))
    reps, el = 1, dt
    while el < budget_s:
        el += one(rows)
        reps += 1
    ops = 2 * rows * N * K * reps
    return dict(value=ops / el / 1e12, unit="TOPS", cores=oracle.threads(), kind="oracle",
                sample=(f"{rows} of {M} activation rows x all {N} outputs, K={K}: "
                        f"quantize_act + MAC + epilogue, {reps} runs in {el:.1f} s"))


def copy_calibration(nbytes=1 << 30, reps=5):
    import torch
    torch.cuda.set_device(0)
    src = torch.ones(nbytes // 4, dtype=torch.float32, device="cuda")
    dst = torch.empty_like(src)
    for _ in range(reps):
        dst.copy_(src)
    torch.cuda.synchronize()
    print(json.dumps({"copy_calibration_bytes": nbytes, "reps": reps}))


def graph_ms(fn, steps, warmup):
    """Milliseconds per call of fn: `steps` calls captured in one HIP graph,
    replayed once untimed and once between two events on the stream."""
    import torch
    stream = torch.cuda.current_stream()
    for _ in range(warmup):
        fn()
    g = torch.cuda.CUDAGraph()
    side = torch.cuda.Stream()
    side.wait_stream(stream)
    with torch.cuda.graph(g, stream=side):
        for _ in range(steps):
            fn()
    torch.cuda.synchronize()
    g.replay()
    torch.cuda.synchronize()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record(stream)
    g.replay()
    e1.record(stream)
    torch.cuda.synchronize()
    return e0.elapsed_time(e1) / steps


def run_conv_chain(steps, warmup):
    """Two 3x3 convolutions in a row (the CNN workload's layer: 32 images of
    256 x 14 x 14 -> 256 channels, then the same again), both as implicit
    GEMMs, timed two ways as `steps` steps in one HIP graph: the second
    convolution's input quantized in the first one's epilogue with static
    scales straight into its haloed code image (soniq_mp_gemm_quantize_next),
    and the unfused form (bf16 Y of layer 1, turned into an fp32 NCHW tensor
    by torch, then soniq_quantize_act_conv3x3 with the batch maximum).  The
    static scales are calibrated once, untimed, from the unfused form.  The
    two-pass form with the batch maximum (soniq_mp_gemm_quantize_next_max:
    Y stored with its tiles' maxima, then the image from Y) is timed too."""
    import torch
    import paper_2311_14114_amd as sq
    import workloads

    torch.cuda.set_device(0)
    l1 = workloads.make("conv3x3_im2col")
    B, C, H, W = l1["X"].shape
    N = l1["N"]
    l2 = workloads.conv3x3(B, N, H, W, N, seed=l1["seed"] + 100, name="conv3x3_second")
    M = B * H * W
    dev = torch.device("cuda")
    X1 = torch.from_numpy(l1["X"]).to(dev)

    def pack(case, cin):
        Wf = torch.from_numpy(np.ascontiguousarray(case["W"].reshape(case["N"], cin, 3, 3))).to(dev)
        return sq.soniq_pack_weights_conv3x3(Wf, case["w_bits"], case["a_bits"][::9], False,
                                             sign_nibbles=True)

    wh1, wh2 = pack(l1, C), pack(l2, N)
    act1 = sq.soniq_act_create_conv3x3(wh1, B, H, W)
    act2 = sq.soniq_act_create_conv3x3(wh2, B, H, W)
    Y1 = torch.empty((M, N), dtype=torch.bfloat16, device=dev)
    X2 = torch.empty((B, N, H, W), dtype=torch.float32, device=dev)
    Y2 = torch.empty((M, N), dtype=torch.bfloat16, device=dev)

    def unfused():
        sq.soniq_quantize_act_conv3x3(act1, X1)
        sq.soniq_mp_gemm(act1, wh1, out=Y1)
        X2.copy_(Y1.view(B, H, W, N).permute(0, 3, 1, 2))
        sq.soniq_quantize_act_conv3x3(act2, X2)
        sq.soniq_mp_gemm(act2, wh2, out=Y2)

    unfused()
    torch.cuda.synchronize()
    s2 = sq.soniq_act_unpack_debug(act2)[1].copy()

    def fused():
        sq.soniq_quantize_act_conv3x3(act1, X1)
        sq.soniq_mp_gemm_quantize_next(act1, wh1, act2, s2)
        sq.soniq_mp_gemm(act2, wh2, out=Y2)

    fused()  # prepares act2 for this producer (allocates outside the graph)

    def fused_max():
        sq.soniq_quantize_act_conv3x3(act1, X1)
        sq.soniq_mp_gemm_quantize_next_max(act1, wh1, act2, out=Y1)
        sq.soniq_mp_gemm(act2, wh2, out=Y2)

    fused_max()
    t_f, t_u = graph_ms(fused, steps, warmup), graph_ms(unfused, steps, warmup)
    t_m = graph_ms(fused_max, steps, warmup)
    ops = 2 * 2 * M * N * 9 * C
    print(json.dumps({
        "chain": "conv3x3 -> conv3x3 (implicit GEMM)", "input": [int(B), int(C), int(H), int(W)],
        "N": int(N), "launch": "graph", "steps": steps, "warmup": warmup,
        "fused_us": t_f * 1e3, "unfused_us": t_u * 1e3, "fused_tops": ops / (t_f * 1e-3) / 1e12,
        "unfused_tops": ops / (t_u * 1e-3) / 1e12, "fused_batch_max_us": t_m * 1e3,
        "static_scales": [float(v) for v in s2], "data": "synthetic"}), flush=True)


def run_chain(steps, warmup, group_bits=0, rows=0):
    """Two transformer linears in a row (FFN up, 4096x3072x768, then FFN
    down, 4096x768x3072), timed two ways, each as `steps` steps captured
    in one HIP graph: the next layer's activations quantized in the first
    GEMM's epilogue with static scales (soniq_mp_gemm_quantize_next), the
    two-pass form with the batch maximum (soniq_mp_gemm_quantize_next_max:
    the epilogue folds the maxima, one pass quantizes the stored bf16 Y),
    and the unfused form (bf16 Y of layer 1, widened to fp32 by torch, then
    soniq_quantize_act with the batch maximum).  The static scales are
    calibrated once, untimed, from the unfused form's batch maxima.  With
    group_bits > 0 both layers are packed with sub-group activation scales
    of that many bits (one static scale per block).  rows > 0 takes only
    the first `rows` rows (a decode batch: the GEMV forms carry the
    epilogue)."""
    import torch
    import paper_2311_14114_amd as sq
    import workloads

    torch.cuda.set_device(0)
    up, down = workloads.xfmr_ffn_up(), workloads.xfmr_ffn_down()
    if rows > 0:
        up["A"] = np.ascontiguousarray(up["A"][:rows])
        up["M"] = down["M"] = rows
    M = up["M"]
    dev = torch.device("cuda")
    A = torch.from_numpy(up["A"]).to(dev)
    wh1 = sq.soniq_pack_weights(torch.from_numpy(up["W"]).to(dev), up["w_bits"], up["a_bits"], True,
                                act_group_bits=group_bits)
    wh2 = sq.soniq_pack_weights(torch.from_numpy(down["W"]).to(dev), down["w_bits"], down["a_bits"],
                                down["a_signed"], act_group_bits=group_bits)
    act1, act2 = sq.soniq_act_create(wh1, M), sq.soniq_act_create(wh2, M)
    Y1 = torch.empty((M, up["N"]), dtype=torch.bfloat16, device=dev)
    Y1f = torch.empty((M, up["N"]), dtype=torch.float32, device=dev)
    Y2 = torch.empty((M, down["N"]), dtype=torch.bfloat16, device=dev)

    def unfused():
        sq.soniq_quantize_act(act1, A)
        sq.soniq_mp_gemm(act1, wh1, out=Y1)
        Y1f.copy_(Y1)
        sq.soniq_quantize_act(act2, Y1f)
        sq.soniq_mp_gemm(act2, wh2, out=Y2)

    unfused()
    torch.cuda.synchronize()
    s2 = sq.soniq_act_unpack_debug(act2)[1].copy()

    def fused():
        sq.soniq_quantize_act(act1, A)
        sq.soniq_mp_gemm_quantize_next(act1, wh1, act2, s2)
        sq.soniq_mp_gemm(act2, wh2, out=Y2)

    def fused_max():
        sq.soniq_quantize_act(act1, A)
        sq.soniq_mp_gemm_quantize_next_max(act1, wh1, act2, out=Y1)
        sq.soniq_mp_gemm(act2, wh2, out=Y2)

    fused()  # prepares act2 for this producer (allocates outside the graph)
    t_f, t_u = graph_ms(fused, steps, warmup), graph_ms(unfused, steps, warmup)
    # the two-pass form (batch maximum, no calibration): layers without blocks
    t_m = graph_ms(fused_max, steps, warmup) if group_bits == 0 else None
    ops = 2 * M * (up["N"] * up["K"] + down["N"] * down["K"])
    print(json.dumps({
        "chain": "xfmr_ffn_up -> xfmr_ffn_down", "M": M, "act_group_bits": group_bits,
        "launch": "graph",
        "steps": steps, "warmup": warmup,
        "fused_us": t_f * 1e3, "unfused_us": t_u * 1e3,
        "fused_batch_max_us": t_m * 1e3 if t_m is not None else None,
        "fused_tops": ops / (t_f * 1e-3) / 1e12,
        "unfused_tops": ops / (t_u * 1e-3) / 1e12, "static_scales": [float(v) for v in s2],
        "data": "synthetic"}), flush=True)


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=100)
    ap.add_argument("--warmup", type=int, default=10)
    ap.add_argument("--workload", default=DEFAULT_WORKLOAD)
    ap.add_argument("--gemv-workload", default=None,
                    help="the decode GEMV measured in the same run (default: "
                         f"{DEFAULT_GEMV_WORKLOAD} when --workload is the default; 'none' skips it)")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-rotate", action="store_true")
    ap.add_argument("--copy-calibration", action="store_true")
    ap.add_argument("--chain", action="store_true",
                    help="time FFN up -> FFN down with the next layer quantized in the first "
                         "GEMM's epilogue, against the unfused form")
    ap.add_argument("--conv-chain", action="store_true",
                    help="time two 3x3 convolutions in a row (the CNN workload's layer twice, "
                         "implicit GEMMs), the second's input quantized in the first's epilogue, "
                         "against the unfused form")
    ap.add_argument("--chain-rows", type=int, default=0,
                    help="--chain: only the first ROWS activation rows (a decode batch)")
    ap.add_argument("--chain-group-bits", type=int, default=0,
                    help="--chain with sub-group activation scales of this many bits "
                         "(512: the transformer setting) in both layers")
    ap.add_argument("--conv-input", action="store_true",
                    help="conv workloads: quantize from the NCHW input tensor "
                         "(soniq_quantize_act_conv3x3) instead of the lowered matrix")
    ap.add_argument("--implicit-conv", action="store_true",
                    help="conv workloads: the implicit-GEMM convolution (weights packed with "
                         "soniq_pack_weights_conv3x3; the input quantized once into a code image "
                         "whose taps the GEMM gathers)")
    ap.add_argument("--f8f6f4", action="store_true",
                    help="pack the weights with SONIQ_WPACK_F8F6F4: narrow x narrow tiles run on the "
                         "fp4/fp6 MFMA")
    ap.add_argument("--dense", action="store_true",
                    help="decode batches: pack the weights with SONIQ_WPACK_DENSE (every code in "
                         "its own width) so the GEMV reads the dense copy")
    ap.add_argument("--launch", choices=["graph", "eager"], default="graph",
                    help="replay the timed steps as one captured HIP graph (default) or "
                         "launch every call from the host")
    args = ap.parse_args()
    if args.gpus != 1:
        print("bench.py measures one GPU only: the quantized GEMM runs on a single MI355X; "
              "how it would shard over several GPUs is a design note, not a measured path.",
              file=sys.stderr)
        sys.exit(2)
    if args.copy_calibration:
        copy_calibration()
        return
    if args.chain:
        run_chain(args.steps, args.warmup, args.chain_group_bits, args.chain_rows)
        return
    if args.conv_chain:
        run_conv_chain(args.steps, args.warmup)
        return

    import workloads
    case = workloads.make(args.workload)
    if args.dense:
        if case["M"] > 8 or args.f8f6f4 or args.implicit_conv or case.get("act_group_bits", 0):
            print("--dense: the dense copy serves decode batches (M <= 8) of plain linear "
                  "layers with one scale per precision group", file=sys.stderr)
            sys.exit(2)
        case["dense"] = True
    if args.implicit_conv:
        args.conv_input = True
    if args.conv_input and "X" not in case:
        print(f"--conv-input needs a convolution workload; {args.workload} has no input tensor",
              file=sys.stderr)
        sys.exit(2)
    r = run_gpu(case, args.steps, args.warmup, rotate=not args.no_rotate,
                graph=args.launch == "graph", conv_input=args.conv_input, f8f6f4=args.f8f6f4,
                implicit=args.implicit_conv)
    alg = algorithmic(case, r["info"])
    if args.conv_input:
        alg["a_fp32"] = int(case["X"].nbytes)  # the quantizer reads X, not its lowering
    ms = r["total_ms"] / args.steps
    tops = alg["ops"] / (ms * 1e-3) / 1e12

    rec = {
        "metric": METRIC, "value": tops, "unit": "TOPS", "n_gpus": 1, "steps": args.steps,
        "warmup": args.warmup, "ms_per_step": ms, "higher_is_better": True, "scaling": "weak",
        "vs_baseline": None, "dtype": "int8", "data": "synthetic",
        "config": {"workload": case["name"], "M": case["M"], "N": case["N"], "K": case["K"],
                   "a_bits": sorted(set(case["a_bits"].tolist())),
                   "w_bits": sorted(set(case["w_bits"].tolist())),
                   "a_signed": bool(case["a_signed"]),
                   "act_group_bits": int(case.get("act_group_bits", 0)),
                   "sign_weights_container": 4 if sign_nibbles(case) else 1,
                   "f8f6f4_copies": bool(args.f8f6f4),
                   "activation_copies": r["na"], "weight_copies": r["nw"],
                   "launch": args.launch, "input": "nchw" if args.conv_input else "lowered",
                   "implicit_conv": bool(args.implicit_conv),
                   "dense_weights": bool(case.get("dense")),
                   "entry": ("soniq_quantize_act_conv3x3 + soniq_mp_gemm" if args.conv_input
                             else "soniq_quantize_mp_gemm")},
        "roofline": roofline(case, alg, r, args.steps),
        "breakdown_ms": {"quantize_act": r["q_ms"], "mp_gemm": r["g_ms"],
                         "pack_weights_once": r["pack_ms"]},
        "gemm_tops": alg["ops"] / (r["g_ms"] * 1e-3) / 1e12,
        "packed_weight_gbs": alg["w_packed"] / (r["g_ms"] * 1e-3) / 1e9,
        "mp_gemm_weights_cache_hot_ms": r["g_hot_ms"],
        "plain_read_weights_ms": r["read_ms"],
        "bf16_linear_ms": r["bf16_ms"],
        "speedup_vs_bf16": {"gemm": r["bf16_ms"] / r["g_ms"], "step": r["bf16_ms"] / ms},
    }
    if args.conv_input and rec["roofline"]["kernel"] == "soniq_quantize_act":
        rec["roofline"]["traffic"] = None  # the counters on file are the lowered path's
    gname = args.gemv_workload
    if gname is None:
        gname = DEFAULT_GEMV_WORKLOAD if args.workload == DEFAULT_WORKLOAD else "none"
    if gname != "none":
        gcase = workloads.make(gname)
        if args.dense and not gcase.get("act_group_bits", 0):
            gcase["dense"] = True
        if gcase["M"] > 8:
            print(f"--gemv-workload {gname} is not a decode batch (M > 8)", file=sys.stderr)
            sys.exit(2)
        gr = run_gpu(gcase, args.steps, args.warmup, rotate=not args.no_rotate,
                     graph=args.launch == "graph")
        rec["gemv"] = gemv_record(gcase, gr, args.steps)
    if not args.no_cpu_baseline:
        rec["cpu_baseline"] = cpu_baseline(case)
    print(json.dumps(rec))


if __name__ == "__main__":
    main()
