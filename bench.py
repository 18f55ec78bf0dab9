"""Benchmark: forward + backward branch attention of one context-parallel rank
share on one MI355X, through the C ABI.

One step = branch_attn_fwd + branch_attn_bwd over the whole rank share (every
ring step's main-prefix attention, the branch-local attention and the LSE
merge, then the replayed backward), inputs resident in HBM.

Default workload: one 262144-token sequence, 32 query / 8 KV heads,
head_dim 128, EAGLE-3 chains of depth 3, the zigzag share of rank 0 at CP = 8
(32768 main + 98304 branch queries against 262144 main keys), bf16 inputs
with fp32 accumulation.

Prints ONE JSON line.  `value` is useful TFLOP/s of the whole step (allowed
query-key pairs x heads x 14 d, forward 4d + backward 10d).  `roofline`
describes the dominant kernel (timed live with HIP events recorded by the
library around its ring-kernel launches); `cpu_baseline` is the fp64 CPU
oracle timed on a bounded sample of query rows of the same share.
"""

from __future__ import annotations

import argparse
import ctypes
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

PEAK_BF16_TFLOPS = 256 * 4096 * 2.4e9 / 1e12  # 256 CUs x 4096 dense bf16 FLOP/clk x 2.4 GHz

# HBM bytes per launch measured with rocprofv3 FETCH_SIZE / WRITE_SIZE runs of
# this benchmark (256K headline share; the fused schedule, the plan's choice,
# in profiles/traffic_eagle3-K3-L262144-cp8r0.md, and the per-step schedule
# taken on the same sources), scaled by a plain-copy calibration.  A figure
# only applies while the kernel's source is the one that was measured.
MEASURED_TRAFFIC = {
    ("bwd_kv_kernel", "fused"): {"source": "bwd.hip", "sha256_16": "f3011df620efb2e7", "bytes": 9961742616},
    ("bwd_dq_kernel", "fused"): {"source": "bwd.hip", "sha256_16": "f3011df620efb2e7", "bytes": 38219996059},
    ("fwd_kernel", "fused"): {"source": "fwd.hip", "sha256_16": "0b9b2bab93598c2e", "bytes": 37982780076},
    ("bwd_kv_kernel", "per_step"): {"source": "bwd.hip", "sha256_16": "f3011df620efb2e7", "bytes": 9976401605},
    ("bwd_dq_kernel", "per_step"): {"source": "bwd.hip", "sha256_16": "f3011df620efb2e7", "bytes": 7824389477},
    ("fwd_kernel", "per_step"): {"source": "fwd.hip", "sha256_16": "0b9b2bab93598c2e", "bytes": 7168648699},
}

def measured_traffic(kernel: str, workload: str, mode: str):
    """HBM bytes per launch of `kernel`, or None if not measured for this
    workload and schedule or if the kernel changed since."""
    import hashlib
    m = MEASURED_TRAFFIC.get((kernel, mode))
    if m is None or workload != "eagle3-K3-L262144-cp8r0":
        return None
    path = os.path.join(ROOT, "paper_2609_07108_amd", "csrc", m["source"])
    if hashlib.sha256(open(path, "rb").read()).hexdigest()[:16] != m["sha256_16"]:
        return None  # the kernel changed since the counters were taken
    return m["bytes"]
PEAK_HBM_GBS = 8000.0
METRIC = "branch-attn fwd+bwd ms & TFLOP/s (% bf16 MFMA peak), 256K-token rank share"


class HipEvents:
    """Raw hipEvent_t handles from the HIP runtime torch already loaded."""

    def __init__(self):
        self.h = ctypes.CDLL("libamdhip64.so.7")
        self.h.hipEventCreate.argtypes = [ctypes.POINTER(ctypes.c_void_p)]
        self.h.hipEventElapsedTime.argtypes = [ctypes.POINTER(ctypes.c_float), ctypes.c_void_p, ctypes.c_void_p]
        self.h.hipEventDestroy.argtypes = [ctypes.c_void_p]
        self.h.hipEventRecord.argtypes = [ctypes.c_void_p, ctypes.c_void_p]

    def create(self):
        ev = ctypes.c_void_p()
        rc = self.h.hipEventCreate(ctypes.byref(ev))
        if rc != 0:
            raise RuntimeError(f"hipEventCreate failed ({rc})")
        return ev

    def record(self, ev, stream):
        rc = self.h.hipEventRecord(ev, ctypes.c_void_p(stream))
        if rc != 0:
            raise RuntimeError(f"hipEventRecord failed ({rc})")

    def ms(self, a, b):
        out = ctypes.c_float()
        rc = self.h.hipEventElapsedTime(ctypes.byref(out), a, b)
        if rc != 0:
            raise RuntimeError(f"hipEventElapsedTime failed ({rc})")
        return out.value


def cpu_baseline(prob, rows: int, seed: int = 1234):
    """Time the fp64 oracle on `rows` query rows of the share (fwd + bwd)."""
    import numpy as np
    import oracle

    mq, bq = oracle.select_queries(prob)
    rng = np.random.default_rng(seed)
    n_m = max(1, rows // 4)
    sm = np.sort(rng.choice(mq, size=min(n_m, len(mq)), replace=False)) if len(mq) else mq[:0]
    sb = np.sort(rng.choice(bq, size=min(rows - len(sm), len(bq)), replace=False)) if len(bq) else bq[:0]
    H, Hk, d = prob.hq, prob.hkv, prob.head_dim

    def sparse(name, sel, total, heads):
        a = np.zeros((total, heads, d), np.float32)  # untouched pages stay unallocated
        if len(sel):
            a[sel] = prob.draw(name, sel).float().numpy()
        return a

    # branch keys the sampled rows can reach: every member of their groups
    grp = np.repeat(np.arange(len(prob.g_len)), prob.g_len)
    gsel = np.unique(grp[sb]) if len(sb) else np.zeros(0, np.int64)
    brows = np.concatenate([np.arange(prob.g_row0[g], prob.g_row0[g] + prob.g_len[g]) for g in gsel]) \
        if len(gsel) else np.zeros(0, np.int64)
    t = dict(qm=sparse("qm", sm, prob.n_main, H), qb=sparse("qb", sb, prob.n_branch, H),
             km=prob.draw("km").float().numpy(), vm=prob.draw("vm").float().numpy(),
             kb=sparse("kb", brows, prob.n_branch, Hk), vb=sparse("vb", brows, prob.n_branch, Hk))
    dom = prob.draw("dom", sm).float().numpy() if len(sm) else np.zeros((0, H, d), np.float32)
    dob = prob.draw("dob", sb).float().numpy() if len(sb) else np.zeros((0, H, d), np.float32)
    args = [t[k] for k in ("qm", "km", "vm", "qb", "kb", "vb")]
    t0 = time.perf_counter()
    ref_f = oracle.forward(prob, *args, sm, sb)
    t1 = time.perf_counter()
    ref_b = oracle.backward(prob, *args, dom, dob, sm, sb)
    t2 = time.perf_counter()
    dt, dt_f, dt_b = t2 - t0, t1 - t0, t2 - t1
    pm, pl = oracle.allowed_pair_counts(prob, sm, sb)
    f_fwd, f_bwd = oracle.useful_flops(prob, pm + pl)
    try:
        from threadpoolctl import threadpool_info
        cores = max([i.get("num_threads", 1) for i in threadpool_info()] or [1])
    except Exception:
        cores = os.cpu_count()
    cpu = ""
    try:
        with open("/proc/cpuinfo") as f:
            cpu = next((l.split(":", 1)[1].strip() for l in f if l.startswith("model name")), "")
    except OSError:
        pass
    # the oracle materialises every key of a row's sequence, so its cost per
    # row is about constant within a share: extrapolate by rows
    n_rows = len(mq) + len(bq)
    scale_rows = n_rows / max(1, len(sm) + len(sb))
    res = {"value": (f_fwd + f_bwd) / dt / 1e12, "unit": "TFLOP/s", "cores": int(cores), "kind": "oracle",
           "sample": f"{len(sm)} main + {len(sb)} branch query rows of the share, fp64 fwd+bwd against "
                     f"all their keys, {dt:.1f} s", "seconds": round(dt, 2), "cpu": cpu,
           "cpu_ms_fwd": round(dt_f * 1e3 * scale_rows, 1), "cpu_ms_bwd": round(dt_b * 1e3 * scale_rows, 1),
           "extrapolated": scale_rows > 1.0,
           "extrapolation": f"x{scale_rows:.1f}: the sample's wall time scaled by rows ({n_rows} query rows)"}
    return res, (sm, sb, ref_f, ref_b)


def sample_parity(share, out, sample):
    """Errors of the GPU outputs of the timed run on the CPU sample's rows
    (O and LSE max-abs, dQ relative L2), against the oracle values the CPU
    baseline computed on the same inputs."""
    import numpy as np
    import torch
    sm, sb, ref_f, ref_b = sample
    g2l = {int(g): i for i, g in enumerate(share.l2g)}
    bmap = {int(g): int(l) for g, l in zip(share.br_rows_global, share.br_rows_local)}
    mi = torch.tensor([g2l[int(g)] for g in sm], dtype=torch.long, device=out["o_main"].device)
    bi = torch.tensor([bmap[int(g)] for g in sb], dtype=torch.long, device=out["o_main"].device)
    f = lambda x: x.double().cpu().numpy()
    o_err = lse_err = 0.0
    dq, dq_ref = [], []
    for idx, o, lse, dqg, ro, rl, rdq in ((mi, "o_main", "lse_main", "dq_main", ref_f[0], ref_f[1], ref_b["dq_main"]),
                                          (bi, "o_br", "lse_br", "dq_br", ref_f[2], ref_f[3], ref_b["dq_br"])):
        if len(idx) == 0:
            continue
        o_err = max(o_err, float(np.abs(f(out[o][idx]) - ro).max()))
        lse_err = max(lse_err, float(np.abs(f(out[lse][:, idx]) - rl).max()))
        dq.append(f(out[dqg][idx]).ravel())
        dq_ref.append(rdq.ravel())
    dq, dq_ref = np.concatenate(dq), np.concatenate(dq_ref)
    rel = float(np.linalg.norm(dq - dq_ref) / max(np.linalg.norm(dq_ref), 1e-300))
    return {"rows": int(len(sm) + len(sb)), "o_max_abs": o_err, "lse_max_abs": lse_err, "dq_rel_l2": rel,
            "bars": {"o_max_abs": 2e-2, "lse_max_abs": 1e-3, "dq_rel_l2": 1e-2}}


QKV_METRIC = "qkv projection + rotary fwd+bwd TFLOP/s (% bf16 MFMA peak), rank-share rows"


def bench_qkv(args):
    """Forward + backward of the QKV projection of one rank share: the main rows
    and the branch rows projected in two calls each (the weight gradient
    accumulated over both), positions from the plan, inputs resident in HBM.
    FLOPs: 2 rows hidden (hq + 2 hkv) 128 per product, three products."""
    import numpy as np
    import torch
    from paper_2609_07108_amd import binding as B
    from paper_2609_07108_amd import rankshare as RS
    from paper_2609_07108_amd import workloads as W

    assert torch.cuda.is_available(), "bench.py needs a GPU"
    torch.cuda.set_device(0)
    prob = W.config(args.config)
    theta = args.rope if args.rope else 5.0e5
    hidden, hq, hkv = args.qkv_hidden, prob.hq, prob.hkv
    share = RS.build_share(prob, materialize=False)
    parts = [p for p in share.plan.positions(share.n_local, share.num_branch_rows) if len(p)]
    n = (hq + 2 * hkv) * 128
    g = torch.Generator(device="cuda")
    g.manual_seed(7)

    def randn(shape, scale=1.0, dtype=torch.bfloat16):
        return (torch.randn(shape, generator=g, device="cuda") * scale).to(dtype)

    w = randn((n, hidden), 1.0 / hidden ** 0.5)
    dw = torch.empty((n, hidden), dtype=torch.float32, device="cuda")
    io = []
    for pos in parts:
        r = len(pos)
        io.append(dict(x=randn((r, hidden)), pos=torch.as_tensor(pos, dtype=torch.int32, device="cuda"),
                       q=torch.empty((r, hq, 128), dtype=torch.bfloat16, device="cuda"),
                       k=torch.empty((r, hkv, 128), dtype=torch.bfloat16, device="cuda"),
                       v=torch.empty((r, hkv, 128), dtype=torch.bfloat16, device="cuda"),
                       dq=randn((r, hq, 128)), dk=randn((r, hkv, 128)), dv=randn((r, hkv, 128)),
                       dx=torch.empty((r, hidden), dtype=torch.bfloat16, device="cuda")))
    ws = torch.empty(max(B.branch_attn_qkv_workspace_size(max(len(p) for p in parts), hq, hkv), 256),
                     dtype=torch.uint8, device="cuda")
    rows = sum(len(p) for p in parts)
    flops = 2.0 * rows * hidden * n  # one product
    ev = HipEvents()
    stream = torch.cuda.current_stream().cuda_stream

    def fwd():
        for t in io:
            B.branch_attn_qkv_fwd(t["x"], w, hq, hkv, t["pos"], theta, t["q"], t["k"], t["v"])

    def bwd():
        for i, t in enumerate(io):
            B.branch_attn_qkv_bwd(t["x"], w, hq, hkv, t["pos"], theta, t["dq"], t["dk"], t["dv"], t["dx"], dw,
                                  i > 0, ws)

    for _ in range(args.warmup):
        fwd()
        bwd()
    torch.cuda.synchronize()
    marks = [[ev.create() for _ in range(3)] for _ in range(args.steps)]
    for m in marks:
        ev.record(m[0], stream)
        fwd()
        ev.record(m[1], stream)
        bwd()
        ev.record(m[2], stream)
    torch.cuda.synchronize()
    fwd_ms = sum(ev.ms(m[0], m[1]) for m in marks) / args.steps
    bwd_ms = sum(ev.ms(m[1], m[2]) for m in marks) / args.steps
    step_ms = fwd_ms + bwd_ms
    print(f"[bench] qkv {args.steps} steps: fwd {fwd_ms:.3f} ms ({flops / fwd_ms / 1e9:.0f} TFLOP/s), "
          f"bwd {bwd_ms:.3f} ms ({2 * flops / bwd_ms / 1e9:.0f} TFLOP/s)", file=sys.stderr, flush=True)

    cpu = None
    if args.cpu_rows > 0:
        from oracle import qkv as OQ
        sample = 1024 * args.cpu_rows  # about 10 s of fp64 BLAS on 16 cores at the default
        rng = np.random.default_rng(3)
        x = rng.standard_normal((sample, hidden))
        wn = w.float().cpu().numpy().astype(np.float64)
        pos = rng.integers(0, 262144, sample)
        dq, dk, dv = (rng.standard_normal((sample, h, 128)) for h in (hq, hkv, hkv))
        t0 = time.perf_counter()
        OQ.forward(x, wn, hq, hkv, pos, theta)
        OQ.backward(x, wn, hq, hkv, pos, theta, dq, dk, dv)
        dt = time.perf_counter() - t0
        cpu = {"value": round(3 * 2.0 * sample * hidden * n / dt / 1e12, 4), "unit": "TFLOP/s",
               "cores": os.cpu_count(), "kind": "oracle",
               "sample": f"{sample} rows, fp64 forward + backward, {dt:.1f} s"}

    achieved = flops / (fwd_ms / 1e3) / 1e12
    value = 3 * flops / (step_ms / 1e3) / 1e12
    line = {
        "metric": QKV_METRIC, "value": round(value, 2), "unit": "TFLOP/s", "n_gpus": 1, "steps": args.steps,
        "warmup": args.warmup, "ms_per_step": round(step_ms, 3), "higher_is_better": True, "scaling": "weak",
        "vs_baseline": None, "dtype": "bf16", "data": "synthetic",
        "config": {"workload": f"qkv-{prob.name}", "rows": rows, "calls": [len(p) for p in parts],
                   "hidden": hidden, "hq": hq, "hkv": hkv, "rope_theta": theta},
        "pct_bf16_peak": round(100 * value / PEAK_BF16_TFLOPS, 2),
        "ms": {"fwd": round(fwd_ms, 3), "bwd": round(bwd_ms, 3)},
        "roofline": {"kernel": "proj_gemm_wide_kernel (forward, rotary epilogue)", "bound": "mfma",
                     "achieved": round(achieved, 2), "peak": round(PEAK_BF16_TFLOPS, 1), "unit": "TFLOP/s",
                     "frac": round(achieved / PEAK_BF16_TFLOPS, 4), "traffic": None,
                     "launches_per_step": len(parts), "launch_ms": round(fwd_ms / len(parts), 3)},
        "cpu_baseline": cpu,
    }
    print(json.dumps(line), flush=True)


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=5)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--config", type=int, default=4, help="named workload 1..5 (4 = 256K headline)")
    ap.add_argument("--mode", choices=["auto", "fused", "per_step"], default="auto",
                    help="per_step: one launch per ring step (the ring's schedule); fused: one walk over all "
                         "blocks; auto (default): the plan's choice (fused)")
    ap.add_argument("--cpu-rows", type=int, default=48,
                    help="query rows of the CPU oracle sample (about 12 s on 16 cores; 0 disables)")
    ap.add_argument("--rope", type=float, default=0.0, metavar="THETA",
                    help="rotate queries and keys by their positions (rotary embedding, base THETA) "
                         "in front of the attention; 0 (default) leaves them as they are")
    ap.add_argument("--qkv-hidden", type=int, default=0, metavar="HIDDEN",
                    help="instead of the attention step, time the grouped-query QKV projection with rotary "
                         "embedding (forward + backward) of the workload's main and branch rows from HIDDEN "
                         "features (its own JSON line)")
    ap.add_argument("--calibrate-copy", type=int, default=0, metavar="MIB",
                    help="only run a plain device-to-device copy of MIB mebibytes (HBM counter calibration)")
    args = ap.parse_args()
    if args.calibrate_copy:
        import torch
        n = args.calibrate_copy * 2 ** 20 // 4
        x = torch.ones(n, dtype=torch.float32, device="cuda:0")
        y = torch.empty_like(x)
        torch.cuda.synchronize()
        y.copy_(x)
        torch.cuda.synchronize()
        print(json.dumps({"calibration": "copy", "bytes_read": n * 4, "bytes_written": n * 4}))
        return
    if args.gpus != 1:
        print(json.dumps({"error": "the benchmark evaluates one context-parallel rank share on ONE GPU; "
                                   "--gpus > 1 is not supported (the ring exchange between GPUs is not "
                                   "implemented)"}))
        sys.exit(2)

    if args.qkv_hidden:
        bench_qkv(args)
        return

    import torch
    from paper_2609_07108_amd import binding as B
    from paper_2609_07108_amd import rankshare as RS
    from paper_2609_07108_amd import workloads as W

    assert torch.cuda.is_available(), "bench.py needs a GPU"
    torch.cuda.set_device(0)
    prob = W.config(args.config)
    t0 = time.perf_counter()
    share = RS.build_share(prob, device="cuda:0", with_grad=True, rope_theta=args.rope)
    mode = share.plan.mode({"fused": B.BA_MODE_FUSED, "per_step": B.BA_MODE_PER_STEP,
                            "auto": B.BA_MODE_AUTO}[args.mode])
    mode_name = "fused" if mode == B.BA_MODE_FUSED else "per_step"
    out = RS.alloc_outputs(share, grads=True)
    ws = RS.workspace(share, mode, backward=True)
    torch.cuda.synchronize()
    print(f"[bench] inputs ready in {time.perf_counter() - t0:.1f} s", file=sys.stderr, flush=True)

    f_fwd, f_bwd = share.plan.useful_flops()
    main_pairs, local_pairs = share.plan.pair_counts()
    d, hq = prob.head_dim, prob.hq
    ring_fwd_flops = main_pairs * hq * 4 * d
    ring_bwd_flops = main_pairs * hq * 10 * d

    ev = HipEvents()
    stream = torch.cuda.current_stream().cuda_stream
    fb, fe, bb, be, bk = [], [], [], [], []
    c0, c1, c2 = [], [], []  # whole-call boundaries: before fwd, between fwd and bwd, after bwd

    def step(i=None):
        evf = (fb[i], fe[i]) if i is not None else (None, None)
        evb = (bb[i], be[i], bk[i]) if i is not None else (None, None, None)
        if i is not None:
            ev.record(c0[i], stream)
        RS.run_fwd(share, out, mode, ws, ring_events=evf)
        if i is not None:
            ev.record(c1[i], stream)
        RS.run_bwd(share, out, mode, ws, ring_events=evb)
        if i is not None:
            ev.record(c2[i], stream)

    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()
    print("[bench] warmup done", file=sys.stderr, flush=True)
    for _ in range(args.steps):
        fb.append(ev.create()); fe.append(ev.create()); bb.append(ev.create()); be.append(ev.create())
        bk.append(ev.create())
        c0.append(ev.create()); c1.append(ev.create()); c2.append(ev.create())
    torch.cuda.reset_peak_memory_stats()
    start, stop = ev.create(), ev.create()
    torch.cuda.synchronize()
    ev.record(start, stream)
    for i in range(args.steps):
        step(i)
    ev.record(stop, stream)
    torch.cuda.synchronize()
    total_ms = ev.ms(start, stop)
    ms_step = total_ms / args.steps
    peak_mem = torch.cuda.max_memory_allocated()
    gpu_ms_fwd = sum(ev.ms(a, b) for a, b in zip(c0, c1)) / args.steps
    gpu_ms_bwd = sum(ev.ms(a, b) for a, b in zip(c1, c2)) / args.steps
    fwd_ring_ms = sum(ev.ms(a, b) for a, b in zip(fb, fe)) / args.steps
    bwd_ring_ms = sum(ev.ms(a, b) for a, b in zip(bb, be)) / args.steps
    # the backward ring part is two kernels: dK/dV (S, dP, dV, dK: 8d per
    # pair) then dQ (S, dP, dQ: 6d per pair); a kernel's time and FLOPs are
    # summed over its launches of the call, so their ratio is per launch too
    kv_ms = sum(ev.ms(a, b) for a, b in zip(bb, bk)) / args.steps
    kern = {"fwd_kernel": (fwd_ring_ms, ring_fwd_flops),
            "bwd_kv_kernel": (kv_ms, main_pairs * hq * 8 * d),
            "bwd_dq_kernel": (bwd_ring_ms - kv_ms, main_pairs * hq * 6 * d)}
    print(f"[bench] {args.steps} steps: {ms_step:.2f} ms/step; " +
          ", ".join(f"{k} {v[0]:.2f} ms ({v[1] / v[0] / 1e9:.0f} TFLOP/s)" for k, v in kern.items()),
          file=sys.stderr, flush=True)

    # launches per call: dK/dV once per ring step in both schedules, the
    # forward and dQ once (fused) or once per ring step
    per_call = 1 if mode == B.BA_MODE_FUSED else prob.cp_size
    launches_of = {"fwd_kernel": per_call, "bwd_kv_kernel": prob.cp_size, "bwd_dq_kernel": per_call}
    dom_name = max(kern, key=lambda k: kern[k][0])
    launches = launches_of[dom_name]
    dom_ms, dom_flops = kern[dom_name]
    achieved = dom_flops / (dom_ms / 1e3) / 1e12
    value = (f_fwd + f_bwd) / (ms_step / 1e3) / 1e12

    cpu = parity = None
    if args.cpu_rows > 0:
        print("[bench] timing the CPU oracle sample", file=sys.stderr, flush=True)
        cpu, sample = cpu_baseline(prob, args.cpu_rows)
        parity = sample_parity(share, out, sample) if not args.rope else None

    # minimum HBM traffic of one step: every input read once and every output
    # written once (fwd: Q, K/V of every ring block, branch K/V in; O, LSE out;
    # bwd: Q, K, V, O, dO, LSE in; dQ, dK, dV out, bf16)
    row_q = hq * d * 2
    row_kv = prob.hkv * d * 2
    nq = share.plan.info()[1]  # query rows of the share (main + branch)
    n_kv = prob.cp_size * share.n_local + share.num_branch_rows
    alg_fwd = nq * (row_q * 2 + hq * 4) + n_kv * row_kv * 2
    alg_bwd = nq * (row_q * 4 + hq * 4) + n_kv * row_kv * 4
    alg_bytes = alg_fwd + alg_bwd
    meas = [measured_traffic(k, prob.name, mode_name) for k in kern] if not args.rope else [None]
    meas_bytes = sum(m * launches_of[k] for k, m in zip(kern, meas)) if all(m is not None for m in meas) else None

    n_local, ntok = share.plan.info()
    traffic = measured_traffic(dom_name, prob.name, mode_name) if not args.rope else None
    line = {
        "metric": METRIC, "value": round(value, 2), "unit": "TFLOP/s", "n_gpus": 1, "steps": args.steps,
        "warmup": args.warmup, "ms_per_step": round(ms_step, 3), "higher_is_better": True, "scaling": "weak",
        "vs_baseline": None, "dtype": "bf16", "data": "synthetic",
        "config": {"workload": prob.name, "describe": prob.describe, "mode": mode_name,
                   "mode_requested": args.mode,
                   "query_rows": ntok, "main_keys": prob.n_main, "hq": prob.hq, "hkv": prob.hkv,
                   "head_dim": d, "cp_size": prob.cp_size, "cp_rank": prob.cp_rank,
                   "rope_theta": args.rope},
        "pct_bf16_peak": round(100 * value / PEAK_BF16_TFLOPS, 2),
        "useful_tflop_per_step": {"fwd": round(f_fwd / 1e12, 3), "bwd": round(f_bwd / 1e12, 3)},
        "gpu_ms_fwd": round(gpu_ms_fwd, 3), "gpu_ms_bwd": round(gpu_ms_bwd, 3),
        "ring_ms": {"fwd": round(fwd_ring_ms, 3), "bwd": round(bwd_ring_ms, 3)},
        "hbm_gbps": round(alg_bytes / (ms_step / 1e3) / 1e9, 1),
        "hbm": {"algorithmic_bytes_per_step": int(alg_bytes), "peak_gbps": PEAK_HBM_GBS,
                "measured_bytes_per_step": meas_bytes,
                "measured_gbps": None if meas_bytes is None else round(meas_bytes / (ms_step / 1e3) / 1e9, 1),
                "note": "hbm_gbps: algorithmic bytes (inputs read once, outputs written once) per step time; "
                        "measured: rocprofv3 FETCH_SIZE + WRITE_SIZE of the three ring kernels, when taken on "
                        "the current sources"},
        "peak_mem_gb": round(peak_mem / 1e9, 3),
        "workspace_gb": round(ws.numel() / 1e9, 3),
        "parity": parity,
        "kernels": {k: {"ms": round(v[0], 3), "tflops": round(v[1] / v[0] / 1e9, 1)} for k, v in kern.items()},
        "roofline": {"kernel": dom_name, "bound": "mfma", "achieved": round(achieved, 2),
                     "peak": round(PEAK_BF16_TFLOPS, 1), "unit": "TFLOP/s",
                     "frac": round(achieved / PEAK_BF16_TFLOPS, 4),
                     "traffic": traffic,
                     "launches_per_step": launches,
                     "launch_ms": round(dom_ms / launches, 3)},
        "cpu_baseline": cpu,
    }
    print(json.dumps(line), flush=True)


if __name__ == "__main__":
    main()
