#!/usr/bin/env python3
"""Benchmark of the TCL Mamba cost model on one MI355X.

Default workload: one tuning round of B = 4096 candidate programs, L = 25,
F = 164, d_model = 256, 4 blocks, fp32 -- scored by tcl_score with the
features already resident in HBM. A step is one tcl_score call (every
kernel of the scoring pass over the whole batch). Prints one JSON line:
programs scored per second, the roofline position of the dominant kernel
(algorithmic flops or bytes per launch over its event-timed duration on
the launch stream) and the fp64 oracle timed on this host's cores.

    python bench.py [--steps K] [--warmup W] [--workload NAME] [--kernels]
"""
from __future__ import annotations

import argparse
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

HBM_PEAK_GBS = 8000.0          # MI355X HBM3E, GB/s
FP32_MFMA_PEAK_TFS = 157.3     # MI355X dense fp32 matrix, TFLOP/s
BF16_MFMA_PEAK_TFS = 2516.6    # MI355X dense bf16 matrix, TFLOP/s
# fp32 GEMMs on the split path deliver fp32 results from the 16-bit matrix
# cores: in_proj, out_proj and the encoder's Linear layers with two-part fp16
# operands (three part products per fp32 product); split_bf16 runs them with
# three-part bf16 operands (six). They are reported against the fp32 matrix peak (the
# arithmetic they deliver) and, beside it, as the 16-bit matrix-core work they
# issue against the dense fp16 / bf16 peak (the same 2.5 PFLOP/s).
F16_SPLIT_KERNELS = ("gemm_input", "gemm_encoder", "gemm_in_proj", "gemm_out_proj")
BF16_SPLIT_KERNELS = ()


def split_form(name: str, f32_matmul: str):
    """(products per fp32 product, matrix dtype) of a split-path GEMM, or None."""
    if f32_matmul == "split":
        if name in F16_SPLIT_KERNELS:
            return 3, "fp16"
        if name in BF16_SPLIT_KERNELS:
            return 6, "bf16"
    if f32_matmul == "split_bf16" and name in F16_SPLIT_KERNELS + BF16_SPLIT_KERNELS:
        return 6, "bf16"
    return None


# VALU issue: 256 CUs x 4 SIMDs x 2.4 GHz, one wave64 VALU instruction per 4
# cycles per SIMD (16 lanes a cycle: the non-packed half of the 157.3 TFLOP/s
# fp32 vector peak); a transcendental takes two such slots (fitted to the
# scan's VALU busy cycles, profiles/*_counters.md)
VALU_SLOT_PEAK_G = 256 * 4 * 2.4 / 4  # 614.4 G wave64 VALU slots/s
# the paper's end-to-end results (tuning time to reach Tenset-MLP's latency
# after 2000 trials, section 7.3, Fig. 10): context only, not this metric
PAPER_CONTEXT = {
    "tuning_time_speedup_vs_tenset_mlp": {"cpu": {"value": 16.8, "hardware": "Intel i7-12700F"},
                                          "gpu": {"value": 12.48, "hardware": "NVIDIA RTX 3080 Ti"}},
    "note": "end-to-end tuning speedups from the paper (TVM search with measurements on the named hardware); "
            "context, not a target: the paper reports no cost-model throughput",
}


METRIC = "candidate programs scored/sec (B=4096,L=25) + % of HBM / MFMA peak"


def kernel_work(shape, M_v: int, B: int, dtype: str, L: int = 0) -> dict:
    """Algorithmic work per launch of each kernel of the scoring pass.

    Counts use the valid tokens M_v only (padding is never computed) and each
    kernel's minimal inputs and outputs read or written once.
    Returns {name: (kind, amount)} with kind "flop" (MFMA-bound) or "byte"
    (HBM-bound). The selective scan is reported against HBM (its bytes: u,
    z and y at the activation width, [dt_r | B | C] in fp32); its VALU and
    transcendental issue is measured with rocprofv3 counters (profiles/).
    """
    d, E, N, R, F = shape.d_model, shape.d_inner, shape.d_state, shape.dt_rank, shape.F
    XW = R + 2 * N
    a = 4 if dtype == "f32" else 2  # bytes per activation element
    dims = [F, *shape.enc_hidden, d]
    # the hidden encoder layers are timed together: their mean work per launch
    enc = [2 * M_v * dims[i] * dims[i + 1] for i in range(1, len(dims) - 1)]
    ldf = (F + 3) // 4 * 4
    h, h2 = shape.head_hidden, shape.dec_hidden2
    return {
        "gemm_input": ("flop", 2 * M_v * F * dims[1]),
        "gemm_encoder": ("flop", sum(enc) / max(len(enc), 1)),
        # F % 4 != 0: every row of the [B, L, F] input is copied into rows of 4k floats
        "pad_features": ("byte", B * L * (F + ldf) * 4),
        "gemm_in_proj": ("flop", 2 * M_v * d * 2 * E),
        "gemm_x_proj": ("byte", M_v * (E * a + XW * 4)),
        "gemm_out_proj": ("flop", 2 * M_v * E * d),
        "conv_silu": ("byte", M_v * 2 * E * a),
        # the conv fused in front of x_proj: reads x, writes u and [dt_r | B | C]
        "gemm_x_proj_conv": ("byte", M_v * (2 * E * a + XW * 4)),
        "token_pos": ("byte", B * 8 + M_v),
        # reads u and z, writes y (in place of u), reads [dt_r | B | C]
        "scan": ("byte", M_v * (3 * E * a + XW * 4)),
        "scan_chunked": ("byte", M_v * (3 * E * a + XW * 4)),
        "tail": ("byte", M_v * d * 4 + B * 8 + 4 * (d * h + h + h * h2 + 2 * h2)),
        "offsets": ("byte", B * 8),
        "mask_scores": ("byte", B * 8),
    }


def gemm_bytes(shape, M_v: int, dtype: str) -> dict:
    """Minimal HBM bytes per pass of the projections (their operands and
    results read or written once): the byte side of their roofline. The
    residual stream H is fp32 in both dtypes."""
    d, E, F = shape.d_model, shape.d_inner, shape.F
    a = 4 if dtype == "f32" else 2
    return {
        "gemm_input": M_v * 4 * (F + d),               # gathered features in, H out
        "gemm_in_proj": M_v * (4 * d + 2 * E * a),     # H in, xz out
        "gemm_out_proj": M_v * (E * a + 2 * 4 * d),    # y and H in, H out
    }


def expected_launches(name: str, shape) -> int:
    """Launches of a kernel per pass of the model over one batch."""
    if name in ("gemm_in_proj", "gemm_x_proj", "gemm_x_proj_conv", "conv_silu", "scan", "scan_chunked",
                "gemm_out_proj"):
        return shape.n_layers
    if name == "gemm_encoder":
        return max(len(shape.enc_hidden), 1)
    return 1


def roofline_entry(kind, amount, ms_per_launch, dtype, split=None):
    """split: (products, matrix dtype) of a split-path fp32 GEMM, else None."""
    if kind == "flop":
        achieved = amount / (ms_per_launch * 1e-3) / 1e12
        peak = BF16_MFMA_PEAK_TFS if dtype != "f32" else FP32_MFMA_PEAK_TFS
        e = {"bound": "mfma", "achieved": achieved, "peak": peak, "unit": "TFLOP/s", "frac": achieved / peak}
        if dtype == "f32" and split:
            products, mdt = split
            issued = products * achieved
            e["matrix_core"] = {"dtype": mdt, "products": products, "achieved": issued,
                                "peak": BF16_MFMA_PEAK_TFS, "unit": "TFLOP/s", "frac": issued / BF16_MFMA_PEAK_TFS}
            e["peak_note"] = ("fp32 results against the fp32 matrix peak; computed on the 16-bit matrix cores "
                              "with both operands in exact parts (two fp16 parts, three part products, or three "
                              "bf16 parts, six products): matrix_core is that issued work against the dense "
                              "fp16/bf16 peak")
        return e
    achieved = amount / (ms_per_launch * 1e-3) / 1e9
    return {"bound": "hbm", "achieved": achieved, "peak": HBM_PEAK_GBS, "unit": "GB/s",
            "frac": achieved / HBM_PEAK_GBS}


def _roof(name: str, d: dict) -> dict:
    """The bench line's roofline object from a kernel's entry."""
    roof = {"kernel": name, "bound": d["bound"], "achieved": round(d["achieved"], 3), "peak": d["peak"],
            "unit": d["unit"], "frac": round(d["frac"], 4), "traffic": None,
            "ms_per_launch": round(d["ms_per_launch"], 5)}
    if "matrix_core" in d:
        roof["matrix_core"] = {k: (round(v, 4) if isinstance(v, float) else v) for k, v in d["matrix_core"].items()}
    if "hbm" in d:
        roof["hbm"] = {k: (round(v, 4) if isinstance(v, float) else v) for k, v in d["hbm"].items()}
        roof["alu_note"] = d["alu_note"]
    if "peak_note" in d:
        roof["peak_note"] = d["peak_note"]
    if "memory" in d:
        roof["memory"] = {k: (round(v, 4) if isinstance(v, float) else v) for k, v in d["memory"].items()}
    return roof


def measured_traffic(workload: str) -> dict:
    """HBM bytes per launch from the committed rocprofv3 counter summary of
    this workload, for each kernel whose source file still has the hash
    recorded with the measurement (a changed kernel gets no number)."""
    import hashlib
    path = os.path.join(ROOT, "profiles", f"{workload}_hbm_traffic.md")
    out = {}
    if not os.path.exists(path):
        return out
    for line in open(path):
        parts = line.split()
        if len(parts) == 5 and parts[0] == "traffic_bytes_per_launch:":
            cat, nbytes, src, digest = parts[1], float(parts[2]), parts[3], parts[4]
            f = os.path.join(ROOT, "paper_2604_12891_amd", "csrc", src)
            if os.path.exists(f) and hashlib.sha256(open(f, "rb").read()).hexdigest()[:16] == digest:
                out[cat] = nbytes
    return out


def measured_valu_slots(workload: str) -> dict:
    """VALU issue slots per valid token of a kernel (SQ_INSTS_VALU plus one more
    per transcendental), from the committed counter summary of this workload,
    while the kernel's source file still has the hash recorded with them."""
    import hashlib
    path = os.path.join(ROOT, "profiles", f"{workload}_counters.md")
    out = {}
    if not os.path.exists(path):
        return out
    for line in open(path):
        parts = line.split()
        if len(parts) == 5 and parts[0] == "valu_slots_per_token:":
            cat, slots, src, digest = parts[1], float(parts[2]), parts[3], parts[4]
            f = os.path.join(ROOT, "paper_2604_12891_amd", "csrc", src)
            if os.path.exists(f) and hashlib.sha256(open(f, "rb").read()).hexdigest()[:16] == digest:
                out[cat] = slots
    return out


def alu_entry(hbm_entry: dict, slots: float, ms_per_launch: float) -> dict:
    """A VALU-issue-bound kernel: its counted issue slots per launch over its
    duration against the issue peak, with its HBM rate beside it."""
    achieved = slots / (ms_per_launch * 1e-3) / 1e9
    return {"bound": "alu", "achieved": achieved, "peak": VALU_SLOT_PEAK_G, "unit": "G VALU slots/s",
            "frac": achieved / VALU_SLOT_PEAK_G,
            "hbm": {"achieved": hbm_entry["achieved"], "peak": HBM_PEAK_GBS, "unit": "GB/s",
                    "frac": hbm_entry["frac"]},
            "alu_note": "wave64 VALU instructions per launch (rocprofv3 SQ_INSTS_VALU, transcendentals "
                        "counted twice) over the launch's duration, against 256 CUs x 4 SIMDs x 2.4 GHz / 4 "
                        "cycles per instruction"}


def cpu_baseline(w, blob, X, lengths, target_s: float) -> dict:
    """The fp64 oracle, as it stands, on a bounded sample of the same batch."""
    import numpy as np
    from threadpoolctl import threadpool_info

    from oracle import model as om

    cfg = dict(F=w.model.F, d_model=w.model.d_model, d_inner=w.model.d_inner, d_state=w.model.d_state,
               d_conv=w.model.d_conv, dt_rank=w.model.dt_rank, n_layers=w.model.n_layers,
               head_hidden=w.model.head_hidden, final_norm=w.model.final_norm, norm_eps=w.model.norm_eps,
               enc_hidden=tuple(w.model.enc_hidden), dec_hidden2=w.model.dec_hidden2)
    om.score(blob, X[:4], lengths[:4], cfg)  # warm-up (first-call overheads)
    n0 = 32
    t = time.perf_counter()
    om.score(blob, X[:n0], lengths[:n0], cfg)
    dt0 = time.perf_counter() - t
    n = int(min(len(lengths), max(n0, target_s / max(dt0, 1e-6) * n0)))
    idx = np.linspace(0, len(lengths) - 1, n).astype(np.int64)
    t = time.perf_counter()
    om.score(blob, X[idx], lengths[idx], cfg)
    dt = time.perf_counter() - t
    blas = [p for p in threadpool_info() if p.get("user_api") == "blas"]
    threads = max([p.get("num_threads", 1) for p in blas] or [1])
    libs = sorted({f"{p.get('internal_api', '?')} {p.get('version', '')}".strip() for p in blas})
    return {"value": n / dt, "unit": "programs/s", "cores": threads, "kind": "oracle",
            "sample": f"{n} of {len(lengths)} programs (evenly strided) of the same batch, numpy fp64, "
                      f"{dt:.1f} s; host has {os.cpu_count()} CPUs, affinity {len(os.sched_getaffinity(0))}, "
                      f"BLAS {', '.join(libs) or 'none'} with {threads} threads"}


def distill_kernel_work(tshape, sshape, M_v: int, B: int) -> dict:
    """Algorithmic work per step of the distillation step's kernels: the
    teacher's scoring kernels (bf16, as in kernel_work) and the student's
    projection backward GEMMs (flops) and scan backward (bytes)."""
    d, E, N, R, F, h, nl = (sshape.d_model, sshape.d_inner, sshape.d_state, sshape.dt_rank, sshape.F,
                            sshape.head_hidden, sshape.n_layers)
    XW = R + 2 * N
    per_layer = d * E + E * R + XW * E + 2 * E * d  # out_proj, dt_proj, x_proj, in_proj
    tw = kernel_work(tshape, M_v, B, "bf16")
    per_block = ("gemm_in_proj", "gemm_x_proj", "gemm_x_proj_conv", "gemm_out_proj", "conv_silu", "scan")
    out = {}
    for k, (kind, amount) in tw.items():
        reps = tshape.n_layers if k in per_block else 1
        # the scan's work is a (flops, bytes) pair; scale both
        amount = tuple(a * reps for a in amount) if isinstance(amount, tuple) else amount * reps
        out["teacher:" + k] = (kind, amount)
    out.update({
        "gemm_dX": ("flop", 2 * M_v * per_layer * nl),
        "gemm_dW": ("flop", 2 * M_v * per_layer * nl + 2 * B * h * d + 2 * M_v * d * F),
        # reads u, z, y (bf16), dyg, xdbl (fp32); writes dz, du, dv (fp32), dB/dC
        "scan_bwd": ("byte", nl * M_v * (3 * E * 2 + E * 4 + XW * 4 + 3 * E * 4 + 2 * N * 4)),
    })
    return out


def progressive_work(shape, a: int, M_v: int, B: int, L: int) -> dict:
    """Algorithmic work per step of each kernel category of the progressive
    forward ("kb:", "ac:" and "lat:" prefixes): the plain model's per-launch
    counts for each column's own kernels, and the adapters' GEMMs (2 flops
    per multiply-add; token rows for the encoder and blocks, pooled rows for
    the decoder)."""
    from paper_2604_12891_amd import workload as wl

    per = kernel_work(shape, M_v, B, "f32", L)
    widths = wl.layer_widths(shape)
    n_tok = len(shape.enc_hidden) + 1 + shape.n_layers  # layers on token rows
    # the adapters' GEMMs have K = n_in (V) and K = a (U): with a = 8 they move
    # more bytes than they compute, so they are counted as HBM work: V reads
    # the KB's input and writes [rows, a]; U reads [rows, a] and the AC's
    # output and writes it back
    V = U = F = 0
    for i, (n_in, n_out) in enumerate(widths[1:], start=1):
        rows = M_v if i < n_tok else B
        V += rows * (n_in + a) * 4
        U += rows * (a + 2 * n_out) * 4
        F += rows * (n_in + 2 * n_out) * 4  # the fused adapter: input read, output read and written
    dec = [2 * B * n_in * n_out for n_in, n_out in widths[n_tok:]]
    pool = ("byte", M_v * shape.d_model * 4 + B * shape.d_model * 4)
    totals = {"lat:gemm_V": ("byte", V), "lat:gemm_U": ("byte", U), "lat:adapter": ("byte", F),
              # the KB's decoder stops before its output layer (no adapter reads it)
              "ac:gemm_decoder": ("flop", sum(dec)), "kb:gemm_decoder": ("flop", sum(dec[:-1])),
              "ac:pool": pool, "kb:pool": pool}
    return per, totals


def bench_progressive(args, w):
    """The CKD framework's continual-learning forward (Eq. (7)): the KB and
    the AC of the paper's model joined by lateral adapters, one step = one
    tcl_progressive_score call over the whole batch."""
    import numpy as np
    import torch

    from paper_2604_12891_amd import binding as tb

    from paper_2604_12891_amd import workload as wl

    (kb, ac, lat), X, lengths = wl.make_workload(w.name)
    dev = torch.device("cuda:0")
    cfg = tb.config_from_shape(w.model, "f32", args.f32_matmul)
    K, A = tb.CostModel(cfg, kb), tb.CostModel(cfg, ac)
    prog = tb.Progressive(K, A, w.adapter, lat)
    Xd, Ld = torch.from_numpy(X).to(dev), torch.from_numpy(lengths).to(dev)
    ws = prog.workspace(w.B, w.L)
    out = torch.empty(w.B, dtype=torch.float32, device=dev)
    M_v = int(lengths.sum())
    for _ in range(args.warmup):
        prog.score(Xd, Ld, out=out, workspace=ws)
    torch.cuda.synchronize()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    t0 = time.perf_counter()
    e0.record()
    for _ in range(args.steps):
        prog.score(Xd, Ld, out=out, workspace=ws)
    e1.record()
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    ms = e0.elapsed_time(e1) / args.steps
    assert torch.isfinite(out).all().item(), "non-finite scores"
    A.timing(True)
    A.timing_reset()
    for _ in range(args.steps):
        prog.score(Xd, Ld, out=out, workspace=ws)
    torch.cuda.synchronize()
    rep = A.timing_report()
    A.timing(False)

    per, totals = progressive_work(w.model, w.adapter, M_v, w.B, w.L)
    split = args.f32_matmul == "split"
    kernels = {}
    for name, (tot, n) in rep.items():
        base = name.split(":", 1)[-1]
        launches = n // args.steps
        if name in totals:  # per-step totals: the mean per launch
            kind, amount = totals[name]
            amount = amount / launches
        else:  # each column's own kernels: per-launch counts of the plain model
            kind, amount = per[base]
        e = roofline_entry(kind, amount, tot / n, "f32", split_form(base, args.f32_matmul))
        e.update({"ms_per_launch": tot / n, "launches_per_step": launches, "ms_per_step": tot / args.steps,
                  "work_per_launch": amount, "work_unit": kind})
        kernels[name] = e
    dom = max(kernels, key=lambda k: kernels[k]["ms_per_step"])
    d = kernels[dom]
    roof = _roof(dom, d)
    if args.kernels:
        for k, e in sorted(kernels.items(), key=lambda kv: -kv[1]["ms_per_step"]):
            print(f"{k:20s} {e['ms_per_step']:9.4f} ms/step x{e['launches_per_step']:3d} {e['achieved']:10.2f} "
                  f"{e['unit']:8s} {e['frac']:6.3f}", file=sys.stderr)
    cpu = None
    if not args.no_cpu_baseline:
        from threadpoolctl import threadpool_info

        from oracle import progressive as op
        ocfg = dict(F=w.model.F, d_model=w.model.d_model, d_inner=w.model.d_inner, d_state=w.model.d_state,
                    d_conv=w.model.d_conv, dt_rank=w.model.dt_rank, n_layers=w.model.n_layers,
                    head_hidden=w.model.head_hidden, final_norm=w.model.final_norm, norm_eps=w.model.norm_eps,
                    enc_hidden=tuple(w.model.enc_hidden), dec_hidden2=w.model.dec_hidden2)
        n = 64
        t = time.perf_counter()
        op.progressive_scores(kb, ac, lat, w.adapter, X[:n], lengths[:n], ocfg)
        dt0 = time.perf_counter() - t
        n = int(min(w.B, max(n, args.cpu_seconds / max(dt0, 1e-6) * n)))
        idx = np.linspace(0, w.B - 1, n).astype(np.int64)
        t = time.perf_counter()
        op.progressive_scores(kb, ac, lat, w.adapter, X[idx], lengths[idx], ocfg)
        dt = time.perf_counter() - t
        blas = [p for p in threadpool_info() if p.get("user_api") == "blas"]
        cpu = {"value": n / dt, "unit": "programs/s", "cores": max([p.get("num_threads", 1) for p in blas] or [1]),
               "kind": "oracle",
               "sample": f"{n} of {w.B} programs (evenly strided) of the same batch, numpy fp64, {dt:.1f} s"}
    rec = {
        "metric": f"KB+AC progressive forward: programs scored/sec (B={w.B},L={w.L}) + % of HBM / MFMA peak",
        "value": w.B / (ms * 1e-3), "unit": "programs/s", "n_gpus": 1, "steps": args.steps, "warmup": args.warmup,
        "ms_per_step": ms, "higher_is_better": True, "scaling": "weak", "vs_baseline": None, "dtype": "f32",
        "data": "synthetic",
        "config": {"workload": w.name, "B": w.B, "L": w.L, "F": w.model.F, "adapter": w.adapter,
                   "f32_matmul": args.f32_matmul, "encoder": [w.model.F, *w.model.enc_hidden, w.model.d_model],
                   "d_state": w.model.d_state, "n_layers": w.model.n_layers,
                   "lengths": f"uniform {w.len_lo}..{w.len_hi}", "valid_tokens": M_v,
                   # the library picks the sequential scan when the batch alone fills the GPU
                   # (B * d_inner / 64 >= 1024 wavefronts) and the chunked two-level scan below
                   "scan": "chunked two-level" if "scan_chunked" in kernels else "sequential"},
        "wall_ms_per_step": wall * 1e3 / args.steps, "roofline": roof,
        "kernels": {k: {kk: (round(vv, 5) if isinstance(vv, float) else vv) for kk, vv in e.items()}
                    for k, e in kernels.items()},
        "cpu_baseline": cpu,
    }
    print(json.dumps(rec), flush=True)


def bench_distill(args, w):
    import numpy as np
    import torch

    from paper_2604_12891_amd import binding as tb
    from paper_2604_12891_amd import workload as wl

    (tblob, sblob), X, lengths = wl.make_workload(w.name)
    dev = torch.device("cuda:0")
    Xd = torch.from_numpy(X).to(dev)
    Ld = torch.from_numpy(lengths).to(dev)
    teacher = tb.CostModel(tb.config_from_shape(w.model, w.dtype), tblob)
    student = tb.CostModel(tb.config_from_shape(w.student, w.dtype), sblob)
    # labels: the teacher's score plus seeded N(0, 0.05^2) noise (prepared once, untimed)
    t = teacher.score(Xd, Ld)
    Yd = (t + torch.from_numpy(wl.label_noise(w.B)).to(dev)).contiguous()
    tr = tb.Trainer(teacher, student, lr=1e-3, max_B=w.B, max_L=w.L)
    ws = tr.workspace(w.B, w.L)
    kd = args.objective == "kd"
    loss = torch.empty(4 if kd else 3, dtype=torch.float32, device=dev)
    M_v = int(lengths.sum())
    if kd:
        # Eq. (9) with the paper's beta = 0.5 and lambda = 1e4; a fixed gate
        # phi = 0.7 and a seeded Fisher diagonal / previous-task parameters
        krng = np.random.default_rng(12891)
        fisher = torch.from_numpy(krng.random(sblob.size).astype(np.float32)).to(dev)
        theta_prev = torch.from_numpy((sblob + 1e-3 * krng.standard_normal(sblob.size)).astype(np.float32)).to(dev)
        kd_args = dict(beta=0.5, phi=0.7, sigma=1.0, ewc_lambda=1e4, fisher=fisher, theta_prev=theta_prev)

    def one_step():
        if kd:
            tr.step_kd(Xd, Ld, Yd, loss=loss, workspace=ws, **kd_args)
        else:
            tr.step(Xd, Ld, Yd, loss=loss, workspace=ws)

    for _ in range(args.warmup):
        one_step()
    torch.cuda.synchronize()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    t0 = time.perf_counter()
    e0.record()
    for _ in range(args.steps):
        one_step()
    e1.record()
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    ms = e0.elapsed_time(e1) / args.steps
    assert torch.isfinite(loss).all().item(), "non-finite loss"

    # the same step captured once into a HIP graph and replayed K times (each
    # replay is one more step): what launching ~90 kernels one by one costs
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph):
        one_step()
    for _ in range(args.warmup):
        graph.replay()
    torch.cuda.synchronize()
    e0.record()
    for _ in range(args.steps):
        graph.replay()
    e1.record()
    torch.cuda.synchronize()
    ms_graph = e0.elapsed_time(e1) / args.steps
    assert torch.isfinite(loss).all().item(), "non-finite loss after graph replays"
    del graph

    tr.timing(True)
    teacher.timing(True)
    tr.timing_reset()
    teacher.timing_reset()
    for _ in range(args.steps):
        one_step()
    torch.cuda.synchronize()
    rep = {("teacher:" + k): v for k, v in teacher.timing_report().items()}
    rep.update(tr.timing_report())
    tr.timing(False)
    teacher.timing(False)
    work = distill_kernel_work(w.model, w.student, M_v, w.B)
    kernels = {}
    for name, (tot, n) in rep.items():
        per = tot / n
        e = {"ms_per_launch": per, "launches_per_step": n // args.steps, "ms_per_step": tot / args.steps}
        if name in work:
            kind, amount = work[name]  # per step; the launches of a category share it
            dtype = "bf16" if name.startswith("teacher:") else "f32"
            e.update(roofline_entry(kind, amount, tot / args.steps, dtype))
            e["work_per_step"] = amount
        kernels[name] = e
    launches = sum(e["launches_per_step"] for e in kernels.values())
    dom = max((k for k in kernels if "frac" in kernels[k]), key=lambda k: kernels[k]["ms_per_step"])
    d = kernels[dom]
    roof = _roof(dom, d)
    roof["launches_per_step"] = d["launches_per_step"]
    if args.kernels:
        for k, e in sorted(kernels.items(), key=lambda kv: -kv[1]["ms_per_step"]):
            print(f"{k:28s} {e['ms_per_step']:9.4f} ms/step  x{e['launches_per_step']:3d}  "
                  f"{e.get('achieved', float('nan')):10.2f} {e.get('unit', '')}", file=sys.stderr)
    cpu = None
    if not args.no_cpu_baseline:
        from threadpoolctl import threadpool_info

        from oracle import model as om

        def ocfg(m):
            return dict(F=m.F, d_model=m.d_model, d_inner=m.d_inner, d_state=m.d_state, d_conv=m.d_conv,
                        dt_rank=m.dt_rank, n_layers=m.n_layers, head_hidden=m.head_hidden,
                        final_norm=m.final_norm, norm_eps=m.norm_eps)
        n = 64
        labels = Yd.cpu().numpy()
        t0 = time.perf_counter()
        if kd:
            from oracle import kd as okd
            okd.distill_step_kd(tblob, ocfg(w.model), sblob, ocfg(w.student), X[:n], lengths[:n], labels[:n],
                                beta=0.5, phi=0.7, lam=1e4, fisher=fisher.cpu().numpy(),
                                theta_prev=theta_prev.cpu().numpy())
        else:
            om.distill_step(tblob, ocfg(w.model), sblob, ocfg(w.student), X[:n], lengths[:n], labels[:n])
        dt = time.perf_counter() - t0
        blas = [p for p in threadpool_info() if p.get("user_api") == "blas"]
        cpu = {"value": 1.0 / (dt * w.B / n), "unit": "steps/s", "cores": max([p.get("num_threads", 1) for p in blas] or [1]),
               "kind": "oracle",
               "sample": f"one fp64 numpy step on {n} of the {w.B} programs ({dt:.1f} s), scaled linearly "
                         f"to the full batch (programs are independent)"}
    rec = {
        "metric": "distillation steps/sec (B=1024,L=25)" + (", Eq. (9) ranking objective" if kd else ""),
        "value": 1000.0 / ms, "unit": "steps/s",
        "n_gpus": 1, "steps": args.steps, "warmup": args.warmup, "ms_per_step": ms,
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None, "dtype": w.dtype, "data": "synthetic",
        "config": {"workload": w.name, "B": w.B, "L": w.L, "teacher": "d256 E512 N16 x4",
                   "student": "d128 E256 N16 x2", "valid_tokens": M_v, "launches_per_step": launches,
                   "objective": ("beta 0.5 LambdaRank(s; labels) + 0.5 phi LambdaRank(s; teacher) + EWC "
                                 "(lambda 1e4), phi 0.7" if kd else "mse(s, teacher) + mse(s, labels)")},
        "wall_ms_per_step": wall * 1e3 / args.steps, "roofline": roof,
        "graph_replay": {"ms_per_step": ms_graph, "steps_per_s": 1000.0 / ms_graph,
                         "vs_launched": ms / ms_graph,
                         "note": "the same step captured into one HIP graph (stream capture) and replayed"},
        "kernels": {k: {kk: (round(vv, 5) if isinstance(vv, float) else vv) for kk, vv in e.items()}
                    for k, e in kernels.items()},
        "cpu_baseline": cpu,
    }
    print(json.dumps(rec), flush=True)


def bench_consumers(args):
    """What consumes the scores: per-segment top-K over a large round's scores
    and the RDU selection over a dataset-sized pool, each against HBM."""
    import numpy as np
    import torch

    from paper_2604_12891_amd import binding as tb

    dev = torch.device("cuda:0")
    rng = np.random.default_rng(12891)
    res = {}

    def timed(fn, steps):
        for _ in range(max(1, args.warmup)):
            fn()
        torch.cuda.synchronize()
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record()
        for _ in range(steps):
            fn()
        e1.record()
        torch.cuda.synchronize()
        return e0.elapsed_time(e1) / steps

    # top-K: 65,536 scores (the bf16 pool workload's round) as 16 tasks of 4,096, K = 64
    B, n_seg, K = 65536, 16, 64
    s = torch.from_numpy((0.3 * rng.standard_normal(B)).astype(np.float32)).to(dev)
    offs = torch.arange(0, B + 1, B // n_seg, dtype=torch.int32, device=dev)
    ms = timed(lambda: tb.topk(s, offs, K), args.steps)
    nbytes = B * 4 + n_seg * K * 4
    res["topk"] = {"ms_per_call": ms, "candidates_per_s": B / (ms * 1e-3),
                   "config": f"{B} scores, {n_seg} segments of {B // n_seg}, K={K}",
                   "roofline": {"bound": "hbm", "achieved": nbytes / (ms * 1e-3) / 1e9, "peak": HBM_PEAK_GBS,
                                "unit": "GB/s", "frac": nbytes / (ms * 1e-3) / 1e9 / HBM_PEAK_GBS,
                                "traffic": None, "bytes_per_call": nbytes}}
    # RDU: a pool the size of one platform's dataset (8.65 M programs), 20
    # operator types, 1,024 initial labeled programs, 64 selections
    N, n_ops, n_init, n_sel = 8_650_000, 20, 1024, 64
    sc = torch.from_numpy((0.3 * rng.standard_normal(N)).astype(np.float32)).to(dev)
    p = rng.random(n_ops) + 0.1
    op = torch.from_numpy(rng.choice(n_ops, N, p=p / p.sum()).astype(np.int32)).to(dev)
    init = torch.from_numpy(rng.choice(N, n_init, replace=False).astype(np.int32)).to(dev)
    ws = torch.empty(tb.lib().tcl_rdu_workspace_bytes(N, n_ops), dtype=torch.uint8, device=dev)
    steps = max(2, args.steps // 10)
    ms = timed(lambda: tb.rdu_select(sc, op, n_ops, init, n_sel, workspace=ws), steps)
    per_sel = ms / n_sel
    nbytes = N * 16  # per selection: score, operator type and running distance of every program, read once
    res["rdu_select"] = {"ms_per_call": ms, "ms_per_selection": per_sel, "selections_per_s": 1e3 / per_sel,
                         "config": f"pool {N}, {n_ops} operator types, {n_init} initial, {n_sel} selections",
                         "roofline": {"bound": "hbm", "achieved": nbytes / (per_sel * 1e-3) / 1e9,
                                      "peak": HBM_PEAK_GBS, "unit": "GB/s",
                                      "frac": nbytes / (per_sel * 1e-3) / 1e9 / HBM_PEAK_GBS, "traffic": None,
                                      "bytes_per_selection": nbytes,
                                      "note": "includes the setup pass (normalisation, budgets, distances "
                                              "to the initial set) amortised over the selections"}}
    cpu = None
    if not args.no_cpu_baseline:
        from oracle import select as osel
        n_cpu, sel_cpu = 20000, 4
        t0 = time.perf_counter()
        osel.rdu_select(sc[:n_cpu].cpu().numpy().astype(np.float64), op[:n_cpu].cpu().numpy(), n_ops,
                        np.arange(64), sel_cpu)
        dt = time.perf_counter() - t0
        cpu = {"value": sel_cpu / dt * n_cpu / N, "unit": "selections/s (scaled to the 8.65 M pool)", "cores": 1,
               "kind": "oracle", "sample": f"{sel_cpu} selections from a pool of {n_cpu} with 64 initial "
                                           f"({dt:.1f} s), scaled linearly in the pool size"}
    rec = {"metric": "score consumers: top-K candidates/s and RDU selections/s", "value": res["rdu_select"]["selections_per_s"],
           "unit": "selections/s", "n_gpus": 1, "steps": args.steps, "warmup": args.warmup,
           "ms_per_step": res["rdu_select"]["ms_per_selection"], "higher_is_better": True, "scaling": "weak",
           "vs_baseline": None, "dtype": "f64", "data": "synthetic",
           "config": {"workload": "rdu_N8650000_topk_B65536"}, "roofline": res["rdu_select"]["roofline"],
           "consumers": res, "cpu_baseline": cpu}
    print(json.dumps(rec), flush=True)


def scan_sweep(args):
    """Time the sequential scan and the chunked two-level scan on their own
    (kernel-level entry point, HIP events on the launch stream) for programs
    of length 64..256, batch sizes from the long-sequence workload (8192)
    down to 16. Prints one JSON line."""
    import numpy as np
    import torch

    from paper_2604_12891_amd import binding as tb

    E, N, R, L = 512, 16, 16, 256
    rng = np.random.default_rng(7)
    out = []
    for B in (8192, 1024, 256, 64, 16):
        lengths = rng.integers(64, L + 1, size=B).astype(np.int32)
        rows = int(lengths.sum())
        offs = torch.from_numpy(np.concatenate([[0], np.cumsum(lengths)]).astype(np.int32)).cuda()
        u = torch.randn(rows, E, device="cuda")
        z = torch.randn(rows, E, device="cuda")
        xdbl = 0.5 * torch.randn(rows, R + 2 * N, device="cuda")
        W_dt = 0.25 * torch.rand(E, R, device="cuda") - 0.125
        b_dt = torch.full((E,), -4.0, device="cuda")
        A_log = torch.log(torch.arange(1, N + 1, device="cuda", dtype=torch.float32)).repeat(E, 1)
        D = torch.ones(E, device="cuda")
        res = torch.empty_like(u)
        rec = {"B": B, "valid_tokens": rows}
        for chunks in (0, 2, 4, 8):
            for _ in range(3):
                tb.scan_f32(offs, u, xdbl, z, W_dt, b_dt, A_log, D, res, chunks=chunks)
            e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            reps = max(3, min(50, int(2e6 // rows)))
            e0.record()
            for _ in range(reps):
                tb.scan_f32(offs, u, xdbl, z, W_dt, b_dt, A_log, D, res, chunks=chunks)
            e1.record()
            torch.cuda.synchronize()
            ms = e0.elapsed_time(e1) / reps
            key = "sequential" if chunks == 0 else f"chunked{chunks}"
            rec[key + "_ms"] = round(ms, 5)
            rec[key + "_GBps"] = round(rows * (3 * E * 4 + (R + 2 * N) * 4) / (ms * 1e-3) / 1e9, 1)
        out.append(rec)
        del u, z, xdbl, res
        torch.cuda.empty_cache()
    print(json.dumps({"scan_sweep": out, "L": L, "E": E, "N": N, "dtype": "f32",
                      "lengths": "uniform 64..256"}), flush=True)


def other_workloads(args) -> dict:
    """The other configurations, timed the same way on the same GPU in the
    same run (warmup, then events around K steps on the current stream):
    programs/s of the small, the large bf16 and the long-sequence scoring
    workloads, and steps/s of the distillation step on both objectives.
    Parity of each is in the GPU tests; these are their rates."""
    import numpy as np
    import torch

    from paper_2604_12891_amd import binding as tb
    from paper_2604_12891_amd import workload as wl

    dev = torch.device("cuda:0")
    steps, warmup = max(5, args.steps // 4), max(2, args.warmup // 2)

    def timed(fn):
        for _ in range(warmup):
            fn()
        torch.cuda.synchronize()
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record()
        for _ in range(steps):
            fn()
        e1.record()
        torch.cuda.synchronize()
        return e0.elapsed_time(e1) / steps

    out = {}
    for name in ("score_B64_L25_d64_f32", "score_B65536_L25_d256_bf16", "score_B8192_L256_d256_f32"):
        w = wl.WORKLOADS[name]
        blob, X, lengths = wl.make_workload(name)
        model = tb.CostModel(tb.config_from_shape(w.model, w.dtype, args.f32_matmul), blob)
        Xd, Ld = torch.from_numpy(X).to(dev), torch.from_numpy(lengths).to(dev)
        del X
        ws = model.workspace(w.B, w.L)
        o = torch.empty(w.B, dtype=torch.float32, device=dev)
        ms = timed(lambda: model.score(Xd, Ld, out=o, workspace=ws))
        assert torch.isfinite(o).all().item()
        waves = w.B * ((w.model.d_inner + 63) // 64)
        graph = None
        if w.B <= 1024:
            # a small batch is bound by its launches: the same pass replayed from a HIP graph
            g = torch.cuda.CUDAGraph()
            with torch.cuda.graph(g):
                model.score(Xd, Ld, out=o, workspace=ws)
            ms_g = timed(g.replay)
            assert torch.isfinite(o).all().item()
            graph = {"ms_per_step": ms_g, "value": w.B / (ms_g * 1e-3), "vs_launched": ms / ms_g}
            del g
        out[name] = {"value": w.B / (ms * 1e-3), "unit": "programs/s", "ms_per_step": ms, "dtype": w.dtype,
                     "graph_replay": graph,
                     "B": w.B, "L": w.L, "valid_tokens": int(lengths.sum()), "steps": steps,
                     # the library's rule: the chunked two-level scan only for L >= 64 with
                     # fewer than 1024 wavefronts of (program, 64 channels)
                     "scan": ("chunked two-level" if w.L >= 64 and waves < 1024 else "sequential")
                             + f" ({waves} wavefronts)"}
        del model, Xd, Ld, ws, o
        torch.cuda.empty_cache()
    w = wl.WORKLOADS["distill_B1024_L25_t256_s128_bf16"]
    (tblob, sblob), X, lengths = wl.make_workload(w.name)
    Xd, Ld = torch.from_numpy(X).to(dev), torch.from_numpy(lengths).to(dev)
    teacher = tb.CostModel(tb.config_from_shape(w.model, w.dtype), tblob)
    Yd = (teacher.score(Xd, Ld) + torch.from_numpy(wl.label_noise(w.B)).to(dev)).contiguous()
    krng = np.random.default_rng(12891)
    fisher = torch.from_numpy(krng.random(sblob.size).astype(np.float32)).to(dev)
    theta_prev = torch.from_numpy((sblob + 1e-3 * krng.standard_normal(sblob.size)).astype(np.float32)).to(dev)
    for objective in ("mse", "kd"):
        student = tb.CostModel(tb.config_from_shape(w.student, w.dtype), sblob)
        tr = tb.Trainer(teacher, student, lr=1e-3, max_B=w.B, max_L=w.L)
        ws = tr.workspace(w.B, w.L)
        loss = torch.empty(4, dtype=torch.float32, device=dev)
        if objective == "kd":
            fn = lambda: tr.step_kd(Xd, Ld, Yd, beta=0.5, phi=0.7, sigma=1.0, ewc_lambda=1e4, fisher=fisher,
                                    theta_prev=theta_prev, loss=loss, workspace=ws)
        else:
            fn = lambda: tr.step(Xd, Ld, Yd, loss=loss[:3], workspace=ws)
        ms = timed(fn)
        assert torch.isfinite(loss[:3]).all().item()
        out[f"{w.name}:{objective}"] = {"value": 1e3 / ms, "unit": "steps/s", "ms_per_step": ms, "dtype": w.dtype,
                                        "B": w.B, "L": w.L, "steps": steps,
                                        "objective": "mse(s, teacher) + mse(s, labels)" if objective == "mse" else
                                        "Eq. (9): beta 0.5, phi 0.7, LambdaRank terms, EWC lambda 1e4"}
        tr.close()
        del student, tr, ws
    return out


def main():
    ap = argparse.ArgumentParser(description=__doc__, formatter_class=argparse.RawDescriptionHelpFormatter)
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=50)
    ap.add_argument("--warmup", type=int, default=10)
    ap.add_argument("--workload", default="score_B4096_L25_d256_f32")
    ap.add_argument("--cpu-seconds", type=float, default=22.0, help="oracle sample budget")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--kernels", action="store_true", help="print the per-kernel table to stderr")
    ap.add_argument("--scan-sweep", action="store_true",
                    help="time the sequential against the chunked scan over batch sizes and exit")
    ap.add_argument("--consumers", action="store_true",
                    help="time the score consumers (top-K, RDU selection) instead of a model workload")
    ap.add_argument("--objective", choices=["mse", "kd"], default="mse",
                    help="distillation workload: the two-MSE loss, or the paper's ranking objective "
                         "(LambdaRank terms, teacher gate, EWC)")
    ap.add_argument("--no-single-stream", action="store_true",
                    help="skip the second per-kernel timing pass with the batch in one pass (so that a "
                         "profiler's per-dispatch averages cover the timed configuration only)")
    ap.add_argument("--f32-matmul", choices=["split", "split_bf16", "native"], default="split",
                    help="fp32 models: projections on the 16-bit matrix cores with split operands (two-part "
                         "fp16 where the shape allows, else three-part bf16; split_bf16: three-part bf16 "
                         "everywhere), or on the fp32 matrix cores")
    ap.add_argument("--no-others", action="store_true",
                    help="with the headline workload, skip timing the other configurations")
    ap.add_argument("--copy-calibration", action="store_true",
                    help="first run 3 elementwise passes over 256 MiB (known bytes for HBM counters)")
    args = ap.parse_args()

    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) != 1:
        print("bench.py measures one GPU only: the scoring and distillation paths are single-GPU "
              "(batches shard across GPUs by program with no exchange but the scores); run with --gpus 1.",
              file=sys.stderr)
        sys.exit(2)

    if args.scan_sweep:
        scan_sweep(args)
        return
    if args.consumers:
        bench_consumers(args)
        return

    import numpy as np
    import torch

    from paper_2604_12891_amd import binding as tb
    from paper_2604_12891_amd import workload as wl

    w = wl.WORKLOADS[args.workload]
    if w.student is not None:
        bench_distill(args, w)
        return
    if w.adapter:
        bench_progressive(args, w)
        return
    blob, X, lengths = wl.make_workload(w.name)
    dev = torch.device("cuda:0")
    if args.copy_calibration:
        # an elementwise kernel that reads 256 MiB and writes 256 MiB, for
        # scaling FETCH_SIZE / WRITE_SIZE
        src = torch.ones(64 << 20, dtype=torch.float32, device=dev)
        dst = torch.empty_like(src)
        for _ in range(3):
            torch.mul(src, 2.0, out=dst)
        torch.cuda.synchronize()
        del src, dst
    Xd = torch.from_numpy(X).to(dev)
    Ld = torch.from_numpy(lengths).to(dev)
    model = tb.CostModel(tb.config_from_shape(w.model, w.dtype, args.f32_matmul), blob)
    split = w.dtype == "f32" and args.f32_matmul in ("split", "split_bf16")
    ws = model.workspace(w.B, w.L)
    out = torch.empty(w.B, dtype=torch.float32, device=dev)
    M_v = int(lengths.sum())

    for _ in range(args.warmup):
        model.score(Xd, Ld, out=out, workspace=ws)
    torch.cuda.synchronize()

    # timed region: K steps, synchronised on both sides
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    e0.record()
    for _ in range(args.steps):
        model.score(Xd, Ld, out=out, workspace=ws)
    e1.record()
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    ms = e0.elapsed_time(e1) / args.steps
    assert torch.isfinite(out).all().item(), "non-finite scores"

    # context only (never the value): the same steps with the features copied
    # from pinned host memory on the same stream first
    Xh = torch.from_numpy(X).pin_memory()
    Lh = torch.from_numpy(lengths).pin_memory()
    torch.cuda.synchronize()
    e2, e3 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e2.record()
    for _ in range(args.steps):
        Xd.copy_(Xh, non_blocking=True)
        Ld.copy_(Lh, non_blocking=True)
        model.score(Xd, Ld, out=out, workspace=ws)
    e3.record()
    torch.cuda.synchronize()
    ms_h2d = e2.elapsed_time(e3) / args.steps

    work = kernel_work(w.model, M_v, w.B, w.dtype, w.L)
    gbytes = gemm_bytes(w.model, M_v, w.dtype)
    valu_slots = measured_valu_slots(w.name)

    def timed_pass(streams: int):
        """The same K steps with every kernel bracketed by events on its
        stream; per-kernel achieved rates against the roofline."""
        model.set_score_streams(streams)
        model.timing(True)
        model.timing_reset()
        for _ in range(args.steps):
            model.score(Xd, Ld, out=out, workspace=ws)
        torch.cuda.synchronize()
        rep = model.timing_report()
        model.timing(False)
        model.set_score_streams(2)
        kernels = {}
        for name, (tot, n) in rep.items():
            per = tot / n
            kind, amount = work[name]
            # launches of one kernel per step (e.g. one per block) all do the
            # same work; a batch scored as concurrent halves launches each
            # kernel once per half, each with (about) half the work
            parts = max(1, round(n / args.steps / expected_launches(name, w.model)))
            amount = tuple(a / parts for a in amount) if isinstance(amount, tuple) else amount / parts
            e = roofline_entry(kind, amount, per, w.dtype, split_form(name, args.f32_matmul) if split else None)
            if name in valu_slots:
                e = alu_entry(e, valu_slots[name] * M_v / parts, per)
            if name in gbytes:
                # the projections' bytes at their time: how close to HBM they run
                gb = gbytes[name] / parts / (per * 1e-3) / 1e9
                e["memory"] = {"bytes": gbytes[name] / parts, "achieved": gb, "peak": HBM_PEAK_GBS,
                               "unit": "GB/s", "frac": gb / HBM_PEAK_GBS}
            e.update({"ms_per_launch": per, "launches_per_step": n // args.steps,
                      "ms_per_step": tot / args.steps, "work_per_launch": amount, "work_unit": kind})
            kernels[name] = e
        dom = max(kernels, key=lambda k: kernels[k]["ms_per_step"])
        d = kernels[dom]
        roof = _roof(dom, d)
        if args.kernels:
            print(f"-- {streams} stream(s)", file=sys.stderr)
            print(f"{'kernel':16s} {'ms/step':>9s} {'ms/launch':>10s} {'achieved':>10s} {'unit':8s} "
                  f"{'frac':>6s}", file=sys.stderr)
            for k, e in sorted(kernels.items(), key=lambda kv: -kv[1]["ms_per_step"]):
                extra = (f"  ({e['matrix_core']['dtype']} matrix cores {e['matrix_core']['frac']:.3f})"
                         if "matrix_core" in e else
                         f"  (HBM {e['hbm']['achieved']:.0f} GB/s = {e['hbm']['frac']:.3f})" if "hbm" in e else "")
                if "memory" in e:
                    extra += f"  (bytes at {e['memory']['achieved']:.0f} GB/s = {e['memory']['frac']:.3f} of HBM)"
                print(f"{k:16s} {e['ms_per_step']:9.4f} {e['ms_per_launch']:10.5f} {e['achieved']:10.2f} "
                      f"{e['unit']:8s} {e['frac']:6.3f}{extra}", file=sys.stderr)
        return kernels, roof

    # as timed (batches of >= 2048 programs as two concurrent halves), and
    # each kernel on its own (one pass: no other kernel beside it)
    kernels, roof = timed_pass(2)
    kernels1, roof1 = timed_pass(1) if not args.no_single_stream else ({}, None)
    traffic = measured_traffic(w.name).get(roof["kernel"])
    if traffic is not None:
        roof["traffic"] = int(traffic)
        roof["traffic_note"] = ("HBM bytes per launch, rocprofv3 FETCH_SIZE + WRITE_SIZE scaled by an "
                                "elementwise kernel of known size (profiles/)")
    concurrent = any(e["launches_per_step"] > expected_launches(k, w.model) for k, e in kernels.items())
    if concurrent:
        roof["concurrency_note"] = ("the batch runs as two halves on two streams: each launch does half the "
                                    "work while the other half's kernels share the GPU")

    cpu = None
    if not args.no_cpu_baseline:
        cpu = cpu_baseline(w, blob, X, lengths, args.cpu_seconds)
    others = None
    if w.name == "score_B4096_L25_d256_f32" and not args.no_others:
        del Xh, Lh
        others = other_workloads(args)

    rec = {
        "metric": METRIC if w.name == "score_B4096_L25_d256_f32" else
                  f"candidate programs scored/sec (B={w.B},L={w.L}) + % of HBM / MFMA peak",
        "value": w.B / (ms * 1e-3),
        "unit": "programs/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": ms,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": w.dtype,
        "data": "synthetic",
        "config": {"workload": w.name, "B": w.B, "L": w.L, "F": w.model.F, "d_model": w.model.d_model,
                   "f32_matmul": args.f32_matmul if w.dtype == "f32" else None,
                   "d_inner": w.model.d_inner, "d_state": w.model.d_state, "n_layers": w.model.n_layers,
                   "encoder": [w.model.F, *w.model.enc_hidden, w.model.d_model],
                   "decoder": [w.model.d_model, w.model.head_hidden, *([w.model.dec_hidden2] if w.model.dec_hidden2 else []), 1],
                   "lengths": f"uniform {w.len_lo}..{w.len_hi}", "valid_tokens": M_v,
                   # the library picks the sequential scan when the batch alone fills the GPU
                   # (B * d_inner / 64 >= 1024 wavefronts) and the chunked two-level scan below
                   "scan": "chunked two-level" if "scan_chunked" in kernels else "sequential"},
        "wall_ms_per_step": wall * 1e3 / args.steps,
        "roofline": roof,
        "roofline_single_stream": roof1,
        "kernels": {k: {kk: (round(vv, 5) if isinstance(vv, float) else vv) for kk, vv in e.items()}
                    for k, e in kernels.items()},
        "kernels_single_stream": {k: {kk: (round(vv, 5) if isinstance(vv, float) else vv) for kk, vv in e.items()}
                                  for k, e in kernels1.items()},
        "pcie_context": {"ms_per_step_incl_h2d": round(ms_h2d, 5),
                         "programs_per_s_incl_h2d": w.B / (ms_h2d * 1e-3),
                         "h2d_bytes": int(X.nbytes + lengths.nbytes),
                         "note": "features copied from pinned host memory on the scoring stream before every "
                                 "step; context only, value excludes it"},
        "cpu_baseline": cpu,
        "other_workloads": others,
        "paper_context": PAPER_CONTEXT,
    }
    print(json.dumps(rec), flush=True)


if __name__ == "__main__":
    main()
