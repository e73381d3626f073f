"""Benchmark of the LaCT fast-weight layer forward on one MI355X.

One step = one full forward of the layer's fast-weight path (every chunk:
apply, key forward/backward, gradient contractions, weight update) over one
batch of seeded synthetic input already resident in HBM. The fast weights
carry over from step to step (a longer sequence of the same shape); the work
per step does not depend on their values.

Prints ONE JSON line (see the keys below). `value` is algorithmic TFLOP/s of
the whole path (App. A FLOP count: 18*d*h per token per head, plus Muon);
tokens/s and the fraction of the bf16 MFMA peak are reported beside it.

Two helper modes serve the HBM-traffic figure of the roofline:
  --copy-calibration        runs a plain device copy of known size (for the
                            rocprofv3 FETCH_SIZE / WRITE_SIZE scale factor)
  --traffic-report F W CF CW  turns four rocprofv3 --pmc CSVs (FETCH_SIZE and
                            WRITE_SIZE of this bench and of the copy) into
                            profiles/lact_<config>_traffic.json, stamped with
                            the hash of the kernel source it was taken on
"""
from __future__ import annotations

import argparse
import csv
import hashlib
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

METRIC = "LaCT layer fwd TFLOP/s + tokens/s at 32K ctx; % of bf16 MFMA peak"
METRIC_BWD = "LaCT fast-weight backward TFLOP/s + tokens/s; % of bf16 MFMA peak"
PEAK_BF16_TFLOPS = 2516.6   # MI355X dense bf16 MFMA: 256 CU x 2.4 GHz x 4096 FLOP/clk
PEAK_FP32_MFMA_TFLOPS = 157.3
PEAK_HBM_GBS = 8000.0
KERNEL_SOURCES = ("paper_2505_23884_amd/csrc/lact_kernels.hip", "paper_2505_23884_amd/csrc/lact_api.hip",
                  "paper_2505_23884_amd/csrc/lact_internal.h")   # the path's kernels (lact_io.hip is outside it)
DOMINANT_KERNEL = {"fwd": "k_fwd", "bwd": "k_bwd", "update": "k_update", "ns": "k_ns"}
COPY_MIB = 1024


def parse():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=10)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--config", default="lm32k")
    ap.add_argument("--chunk", type=int, default=0,
                    help="override the workload's chunk size (a chunk-size sweep of one shape)")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-roofline", action="store_true")
    ap.add_argument("--cpu-seconds", type=float, default=10.0)
    ap.add_argument("--copy-calibration", action="store_true")
    ap.add_argument("--graph", action="store_true",
                    help="time the step replayed from a HIP graph captured once (host launch cost removed)")
    ap.add_argument("--library-gemms", action="store_true",
                    help="time the path's plain contractions as library GEMMs (torch.matmul), for context")
    ap.add_argument("--no-secondary", action="store_true",
                    help="skip the 1M-token NVS workload measured after the default one")
    ap.add_argument("--device-inputs", action="store_true",
                    help="draw the inputs on the device (plain uniform-chunk workloads)")
    ap.add_argument("--backward", action="store_true",
                    help="time the backward (lact_backward; lact_backward_linear on a linear workload, lact_backward_momentum with momentum)")
    ap.add_argument("--traffic-report", nargs=4, metavar=("FETCH_CSV", "WRITE_CSV", "COPY_FETCH_CSV", "COPY_WRITE_CSV"))
    return ap.parse_args()


def _code_only(text):
    """Source text without comments and with whitespace collapsed: what the
    compiler sees (an edit to a comment does not change the kernels). String
    and character literals are kept as they are."""
    out, i, n = [], 0, len(text)
    while i < n:
        c = text[i]
        if c in "\"'":
            j = i + 1
            while j < n and text[j] != c:
                j += 2 if text[j] == "\\" else 1
            out.append(text[i:j + 1])
            i = j + 1
        elif text.startswith("//", i):
            j = text.find("\n", i)
            i = n if j < 0 else j
        elif text.startswith("/*", i):
            j = text.find("*/", i + 2)
            i = n if j < 0 else j + 2
            out.append(" ")
        else:
            out.append(c)
            i += 1
    return " ".join("".join(out).split())


def source_hash():
    """Hash of the path's kernel sources as the compiler sees them."""
    h = hashlib.sha256()
    for rel in KERNEL_SOURCES:
        with open(os.path.join(ROOT, rel), encoding="utf-8") as f:
            h.update(_code_only(f.read()).encode())
    return h.hexdigest()


def copy_calibration():
    """A plain elementwise copy of COPY_MIB MiB (read once, written once), five times."""
    import torch
    n = COPY_MIB << 20
    src = torch.ones(n, dtype=torch.uint8, device="cuda:0")
    dst = torch.empty_like(src)
    for _ in range(5):
        torch.mul(src, 1, out=dst)
    torch.cuda.synchronize()
    print(json.dumps({"copy_bytes": n, "reps": 5}), flush=True)


def library_gemms(cfg, reps):
    """The path's contractions of one step as plain bf16 library GEMMs
    (torch.matmul, hipBLASLt), without any of the fused elementwise work:
    per chunk of C tokens and instance, Z = X [W1; W3]^T for the queries and
    for the keys, D = V W2, O = H W2^T, G13 = [dz1 | dz3]^T K, G2 = V^T H;
    the apply-only tail adds its Z and O. Reported per contraction and summed
    over the step, beside nothing else: a reference point for the kernels,
    which do this work and the elementwise steps in three launches per chunk."""
    import torch
    if cfg.linear or cfg.schedule or cfg.io != "bf16":
        raise SystemExit("--library-gemms covers the uniform-chunk SwiGLU bf16 workloads")
    BH, d, h, C = cfg.BH, cfg.d, cfg.h, cfg.chunk
    tail = cfg.n_q - cfg.n_kv
    gen = torch.Generator(device="cuda:0").manual_seed(0)

    def timed(m, k, n, count):
        a = torch.randn(BH, m, k, generator=gen, device="cuda:0").to(torch.bfloat16)
        b = torch.randn(BH, k, n, generator=gen, device="cuda:0").to(torch.bfloat16)
        if BH == 1:
            a, b = a[0], b[0]
        for _ in range(3):
            torch.matmul(a, b)
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record()
        for _ in range(reps):
            torch.matmul(a, b)
        e1.record()
        torch.cuda.synchronize()
        us = e0.elapsed_time(e1) / reps * 1e3
        fl = 2.0 * BH * m * k * n
        del a, b
        return {"shape": f"[{BH}] {m}x{k} . {k}x{n}", "us": round(us, 2), "tflops": round(fl / us / 1e6, 1),
                "per_step": count, "step_us": round(us * count, 1)}

    nc = cfg.n_chunks
    rows = {
        "Z_queries": timed(C, d, 2 * h, nc),
        "Z_keys": timed(C, d, 2 * h, nc),
        "D": timed(C, d, h, nc),
        "O": timed(C, h, d, nc),
        "G13": timed(2 * h, C, d, nc),
        "G2": timed(d, C, h, nc),
    }
    if tail > 0:
        rows["Z_tail"] = timed(tail, d, 2 * h, 1)
        rows["O_tail"] = timed(tail, h, d, 1)
    total = sum(r["step_us"] for r in rows.values())
    print(json.dumps({"library_gemms": describe(cfg), "contractions": rows,
                      "ms_per_step_gemms_only": round(total / 1e3, 4),
                      "tflops_gemms_only": round(workload_flops(cfg.with_(use_muon=0)) / (total * 1e-6) / 1e12, 1)}),
          flush=True)


def _pmc(path, counter):
    """Per-dispatch values of one counter from a rocprofv3 counter_collection CSV:
    {kernel name: [values]}."""
    out = {}
    with open(path) as f:
        for r in csv.DictReader(f):
            if r["Counter_Name"] != counter:
                continue
            out.setdefault(r["Kernel_Name"], []).append(float(r["Counter_Value"]))
    return out


def kernel_short_name(name):
    """k_fwd, k_bwd, ... from a mangled (…5k_fwdI…) or demangled (…::k_fwd<…) kernel name."""
    for k in ("k_fwd_narrow_keep", "k_fwd_narrow", "k_fwd_keep", "k_fwd", "k_bwd", "k_update", "k_prep", "k_scale_rows", "k_beta_mean", "k_zero_rows",
              "k_ns_fused_pair_out", "k_ns_fused_pair", "k_ns_fused", "k_ns_final", "k_ns_prep", "k_ns_scale", "k_ns",
              "k_prologue", "k_rmsnorm_out", "k_vjp", "k_lin_tokens", "k_copies", "k_accum", "k_swiglu_apply_rows",
              "k_swiglu_rows", "k_mom_bwd", "k_mom_dbeta", "k_mom_adv", "k_slot_dot_part", "k_slot_dot_sum", "k_ns_lin", "k_sym"):
        m = str(len(k)) + k
        if m + "I" in name or m + "E" in name or "::" + k + "<" in name or "::" + k + "(" in name:
            return k
    return None


def traffic_report(cfg_name, fetch_csv, write_csv, cfetch_csv, cwrite_csv):
    """HBM bytes per launch of every lact kernel: the counter's mean per
    dispatch (the same average over launches as the roofline's average launch
    time; a kernel may serve launches of different sizes, such as the key
    forward and the apply of the NVS workloads), scaled by
    copy_bytes / (the same counter for the copy kernel)."""
    import statistics
    cf, cw = _pmc(cfetch_csv, "FETCH_SIZE"), _pmc(cwrite_csv, "WRITE_SIZE")
    copy_fetch = max(max(v) for v in cf.values())
    copy_write = max(max(v) for v in cw.values())
    n = COPY_MIB << 20
    scale = {"fetch": n / copy_fetch, "write": n / copy_write}
    f, w = _pmc(fetch_csv, "FETCH_SIZE"), _pmc(write_csv, "WRITE_SIZE")
    kernels = {}
    for name in f:
        short = kernel_short_name(name)
        if short is None or name not in w:
            continue
        fb = statistics.mean(f[name]) * scale["fetch"]
        wb = statistics.mean(w[name]) * scale["write"]
        kernels[short] = {"fetch_bytes": round(fb), "write_bytes": round(wb), "traffic_bytes": round(fb + wb),
                          "dispatches": len(f[name])}
    rep = {"config": cfg_name, "kernels_source_sha256": source_hash(),
           "calibration": {"copy_bytes": n, "copy_fetch_counter": copy_fetch, "copy_write_counter": copy_write,
                           "fetch_scale": scale["fetch"], "write_scale": scale["write"]},
           "kernels": kernels}
    out = os.path.join(ROOT, "profiles", f"lact_{cfg_name}_traffic.json")
    with open(out, "w") as fh:
        json.dump(rep, fh, indent=1)
    print(json.dumps(rep), flush=True)


def measured_traffic(cfg_name, kernel):
    """Calibrated HBM bytes per launch of `kernel` from the committed counter
    report, or None when there is none or the kernels changed since."""
    path = os.path.join(ROOT, "profiles", f"lact_{cfg_name}_traffic.json")
    try:
        with open(path) as fh:
            rep = json.load(fh)
    except (OSError, ValueError):
        return None
    if rep.get("kernels_source_sha256") != source_hash():
        return None
    k = rep.get("kernels", {}).get(kernel)
    return k["traffic_bytes"] if k else None


def workload_flops(cfg, BH=None):
    """Algorithmic FLOPs of one step (App. A, FLOPs calculation): 12*d*h per
    updated token and 6*d*h per applied token per head, plus per update and
    matrix 3*steps*(4*m^2*n + 2*m^3) with Muon (m <= n the sides)."""
    BH = cfg.BH if BH is None else BH
    if cfg.linear:   # f_W(x) = W x: 2 d^2 per updated and per applied token; Muon on one d x d matrix
        ns = cfg.n_chunks * cfg.ns_steps * 6.0 * float(cfg.d) ** 3 if cfg.use_muon else 0.0
        return BH * (2.0 * cfg.d * cfg.d * (cfg.n_kv + cfg.n_q) + ns)
    dh = float(cfg.d) * cfg.h
    m, n = min(cfg.d, cfg.h), max(cfg.d, cfg.h)
    ns = 3.0 * cfg.ns_steps * (4.0 * m * m * n + 2.0 * m ** 3) if cfg.use_muon else 0.0
    if cfg.schedule:
        from lact_synth import make_schedule
        f = 0.0
        for mode, b, e in make_schedule(cfg):
            if mode != "apply_only":
                f += 12.0 * dh * (e - b) + ns
            if mode != "update_only":
                f += 6.0 * dh * (e - b)
        return BH * f
    return BH * (12.0 * dh * cfg.n_kv + 6.0 * dh * cfg.n_q + cfg.n_chunks * ns)


def backward_flops(cfg, BH=None):
    """Algorithmic FLOPs of the backward (2 per multiply-add of each product).
    Linear fast weight: the replayed chunk gradients (2 d^2 per key token),
    dv = eta dU k and dk = eta dU^T v (4 d^2 per key token), the apply's
    dW += dO^T Q and dq = W^T dO (4 d^2 per query token). SwiGLU: the replayed
    update (key forward and gradient, 12 d h per key token), the update's
    reverse (K U1^T, K U3^T, V U2, dk over 4h, dv over 2h and the three weight
    cotangents: 24 d h per key token) and the apply's (Q W1^T, Q W3^T, dO W2,
    dq over 2h and three weight cotangents: 16 d h per query token). Products
    that the implementation evaluates a second time instead of keeping them
    (K W1^T, K W3^T, V W2 in the reverse) are not counted. With Muon, per
    chunk and matrix: the replayed iteration (App. A: 4 m^2 n + 2 m^3 per
    step, m <= n its sides) and its reverse (dX' X^T, B dX', M X and S A:
    6 m^2 n + 2 m^3 per step). The iteration runs once, in the replay, with
    its iterates kept (where they fit; else it is replayed per chunk in the
    reverse, which is not counted). Momentum adds elementwise passes
    over the state only (no products). A schedule counts its update
    segments' key tokens and its apply segments' query tokens."""
    BH = cfg.BH if BH is None else BH
    nmat = 1 if cfg.linear else 3
    m, n = float(min(cfg.d, cfg.h)), float(max(cfg.d, cfg.h))
    ns1 = nmat * cfg.ns_steps * (10.0 * m * m * n + 4.0 * m ** 3) if cfg.use_muon else 0.0
    ns = cfg.n_chunks * ns1
    if cfg.schedule:
        from lact_synth import make_schedule
        dh = float(cfg.d) * cfg.h
        f = 0.0
        for mode, b, e in make_schedule(cfg):
            if mode != "apply_only":
                f += 36.0 * dh * (e - b) + ns1
            if mode != "update_only":
                f += 16.0 * dh * (e - b)
        return BH * f
    if cfg.linear:
        return BH * (float(cfg.d) * cfg.d * (6.0 * cfg.n_kv + 4.0 * cfg.n_q) + ns)
    return BH * (float(cfg.d) * cfg.h * (36.0 * cfg.n_kv + 16.0 * cfg.n_q) + ns)


def describe(cfg):
    order = "apply-then-update" if cfg.order == 0 else "update-then-apply"
    muon = f", Muon {cfg.ns_steps} NS steps" if cfg.use_muon else ""
    mom = ", momentum (chunk-mean beta)" if cfg.momentum else ""
    lr3 = ", per-matrix rates" if cfg.lr3 else ""
    if cfg.linear:
        lr3 += ", linear fast weight W x"
    if cfg.layer_io:
        lr3 += ", with prologue (SiLU, q/k norm, softplus rates) and per-head RMSNorm"
    if cfg.schedule:
        order = f"schedule {cfg.schedule}"
    return (f"{cfg.name}: B={cfg.B} H={cfg.H} d={cfg.d} h={cfg.h} n_kv={cfg.n_kv} n_q={cfg.n_q} "
            f"chunk={cfg.chunk} {order}{muon}{mom}{lr3}, io {cfg.io}, fp32 state")


def cpu_model():
    """The host CPU's model name and the CPUs this process may run on."""
    name = "unknown"
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    name = line.split(":", 1)[1].strip()
                    break
    except OSError:
        pass
    try:
        ncpu = len(os.sched_getaffinity(0))
    except AttributeError:
        ncpu = os.cpu_count() or 1
    return name, ncpu


def _oracle_sample(cfg, min_seconds, backward=False):
    """The fp64 oracle, as it is, on a bounded sample of the same workload:
    whole (b, h) instances (every chunk), one after another, until at least
    `min_seconds` of host time have passed. When one instance is too large for
    that budget (NVS: 1M tokens in one chunk is ~22 TFLOP), the sample is the
    first tokens of one instance with the same d, h, order and options,
    chunked at the same size up to the sample length.
    With backward, the oracle's reverse of the chunk loop.
    Returns (FLOPs done, seconds, sample description, tokens done)."""
    from lact_synth import make_cotangents, make_inputs
    from oracle import lact_oracle as O

    flops_of = backward_flops if backward else workload_flops
    one = flops_of(cfg, BH=1)
    scfg, note = cfg, ""
    if one > 4e12:   # roughly 30 s or more of fp64 NumPy for one instance
        n = 16384
        scfg = cfg.with_(name=cfg.name + "_sample", B=1, H=1, n_kv=min(cfg.n_kv, n),
                         n_q=min(cfg.n_q, n) + min(cfg.n_q - cfg.n_kv, 4096), chunk=min(cfg.chunk, n))
        note = (f"; token sample of one instance: n_kv={scfg.n_kv}, n_q={scfg.n_q}, chunk={scfg.chunk} "
                f"(same d, h, order, options)")
    done, dt = 0, 0.0
    while done < scfg.BH and dt < min_seconds:
        x = make_inputs(scfg, 0, heads=[done])
        ct = make_cotangents(scfg, 0, heads=[done]) if backward else None
        if backward and scfg.momentum:
            from lact_synth import make_momentum_state
            st = make_momentum_state(scfg, 0, heads=[done])
            W0 = x["W1"][0] if scfg.linear else tuple(x[w][0] for w in ("W1", "W2", "W3"))
            M0 = st["M"][0] if scfg.linear else tuple(st[m][0] for m in ("M1", "M2", "M3"))
        t0 = time.perf_counter()
        if backward and scfg.momentum:
            O.lact_backward_momentum_instance(x["q"][0], x["k"][0], x["v"][0], x["eta"][0], x["beta"][0], W0, M0,
                                              ct["do"][0], scfg.chunk, scfg.order, use_muon=bool(scfg.use_muon),
                                              ns_steps=scfg.ns_steps)
        elif backward and scfg.linear:
            O.lact_backward_linear_instance(x["q"][0], x["k"][0], x["v"][0], x["eta"][0], x["W1"][0], ct["do"][0],
                                            scfg.chunk, scfg.order, use_muon=bool(scfg.use_muon),
                                            ns_steps=scfg.ns_steps)
        elif backward:
            O.lact_backward_instance(x["q"][0], x["k"][0], x["v"][0], x["eta"][0], x["W1"][0], x["W2"][0],
                                     x["W3"][0], ct["do"][0], scfg.chunk, scfg.order, use_muon=bool(scfg.use_muon),
                                     ns_steps=scfg.ns_steps)
        elif scfg.linear:
            O.lact_forward_linear(x["q"], x["k"], x["v"], x["eta"], x["W1"], scfg.chunk, scfg.order,
                                  bool(scfg.use_muon), scfg.ns_steps)
        elif scfg.schedule:
            from lact_synth import make_schedule
            O.lact_forward_schedule(x["q"], x["k"], x["v"], x["eta"], x["W1"], x["W2"], x["W3"],
                                    make_schedule(scfg), use_muon=bool(scfg.use_muon), ns_steps=scfg.ns_steps,
                                    beta=x.get("beta"))
        elif scfg.momentum:
            O.lact_forward_momentum(x["q"], x["k"], x["v"], x["eta"], x["beta"], x["W1"], x["W2"], x["W3"],
                                    chunk=scfg.chunk, order=scfg.order, use_muon=bool(scfg.use_muon),
                                    ns_steps=scfg.ns_steps)
        else:
            O.lact_forward(x["q"], x["k"], x["v"], x["eta"], x["W1"], x["W2"], x["W3"], chunk=scfg.chunk,
                           order=scfg.order, use_muon=bool(scfg.use_muon), ns_steps=scfg.ns_steps)
        dt += time.perf_counter() - t0
        done += 1
    desc = (f"{done} of {scfg.BH} (b,h) instances, all {scfg.n_chunks} chunks each ({done * scfg.n_q} tokens), "
            f"fp64 NumPy, {dt:.1f} s{note}")
    return done * flops_of(scfg, BH=1), dt, desc, done * scfg.n_q


def cpu_baseline(cfg, min_seconds, backward=False):
    """The oracle timed on this host: once with every core the BLAS library
    uses by default, once limited to one thread (a smaller time budget)."""
    from threadpoolctl import threadpool_info, threadpool_limits

    fl, dt, desc, toks = _oracle_sample(cfg, min_seconds, backward)
    threads = max([i.get("num_threads", 1) for i in threadpool_info()] + [1])
    with threadpool_limits(limits=1):
        fl1, dt1, desc1, toks1 = _oracle_sample(cfg, min_seconds / 2, backward)
    model, ncpu = cpu_model()
    return {"value": round(fl / dt / 1e12, 5), "unit": "TFLOP/s", "cores": int(threads), "kind": "oracle",
            "sample": desc, "tokens_per_s": round(toks / dt, 1), "cpu_model": model, "host_cpus": ncpu,
            "one_core": {"value": round(fl1 / dt1 / 1e12, 5), "unit": "TFLOP/s", "cores": 1, "sample": desc1,
                         "tokens_per_s": round(toks1 / dt1, 1)}}


def device_inputs(cfg, dev, seed=0):
    """Inputs of the recipe's distributions drawn on the device (a seeded torch
    generator): q, k, v ~ N(0, 1) with unit rows, eta = 0.01 softplus(N(0, 1)),
    W with N(0, 1/d) entries and unit rows. For workloads whose host draw
    would cost tens of seconds and several GB of host memory (1M tokens)."""
    import torch
    gen = torch.Generator(device=dev).manual_seed(seed)
    io = torch.bfloat16 if cfg.io == "bf16" else torch.float32

    def tok(n):
        x = torch.randn(cfg.B, cfg.H, n, cfg.d, generator=gen, device=dev)
        return (x / x.norm(dim=-1, keepdim=True)).to(io)

    def unit_rows(r, c):
        w = torch.randn(cfg.H, r, c, generator=gen, device=dev) / cfg.d ** 0.5
        w = w / w.norm(dim=-1, keepdim=True)
        return w.unsqueeze(0).expand(cfg.B, -1, -1, -1).contiguous()

    q, k, v = tok(cfg.n_q), tok(cfg.n_kv), tok(cfg.n_kv)
    eta = 0.01 * torch.nn.functional.softplus(torch.randn(cfg.B, cfg.H, cfg.n_kv, generator=gen, device=dev))
    return q, k, v, eta, [unit_rows(cfg.h, cfg.d), unit_rows(cfg.d, cfg.h), unit_rows(cfg.h, cfg.d)]


def kernel_alg_bytes(cfg, kernel, launches_per_step):
    """Algorithmic bytes per launch of the first (k_fwd) or second (k_bwd)
    launch class: the path's inputs each reads and the outputs each writes,
    at their own widths, with the materialised intermediates left out.
    k_fwd reads q, k, v and eta once per step and the 16-bit weight copies
    once per launch (3 d h for an update, 2 d h for an apply-only launch);
    k_bwd reads k and v once and a weight copy once per launch, writes o once,
    and, where it applies the weight update itself (256 < d, h <= 512 without
    Muon), reads and writes the fp32 state and writes its copy per chunk.
    None for other kernels and layouts."""
    if cfg.schedule or cfg.linear or cfg.io != "bf16" or not launches_per_step:
        return None
    esz, dh, C = 2, cfg.d * cfg.h, cfg.chunk
    nch = cfg.n_chunks
    if kernel == "k_fwd":
        upd = nch
        applies = launches_per_step - upd
        b = esz * cfg.d * (2 * cfg.n_kv + cfg.n_q) + 4 * cfg.n_kv + (3 * upd + 2 * applies) * dh * esz
    elif kernel == "k_bwd":
        fused = not cfg.use_muon and 256 < cfg.d <= 512 and 256 < cfg.h <= 512
        b = esz * cfg.d * (2 * cfg.n_kv + cfg.n_q) + launches_per_step * dh * esz
        if fused:
            b += nch * 3 * dh * (4 + 4 + 2)
    else:
        return None
    return cfg.BH * b / launches_per_step


def measure(cfg, args, P, on_device=False):
    """One workload: inputs resident in HBM, warmup, the timed steps, then the
    per-launch timing pass (HIP events on the launch stream) for the roofline."""
    import torch
    from lact_synth import make_inputs

    dev = torch.device("cuda:0")
    io = torch.bfloat16 if cfg.io == "bf16" else torch.float32
    if on_device:
        q, k, v, eta, W = device_inputs(cfg, dev)
        if cfg.momentum or cfg.schedule or cfg.linear or cfg.layer_io or cfg.lr3:
            raise SystemExit("device-drawn inputs cover the plain uniform-chunk workloads")
    else:
        x = make_inputs(cfg, 0)
        sh = lambda a: a.reshape(cfg.B, cfg.H, *a.shape[1:])
        q, k, v = (torch.from_numpy(sh(x[n])).to(dev, io) for n in ("q", "k", "v"))
        eta = torch.from_numpy(sh(x["eta"])).to(dev, torch.float32)
        W = [torch.from_numpy(sh(x[n])).to(dev, torch.float32) for n in ("W1", "W2", "W3")]
        if cfg.momentum:
            beta = torch.from_numpy(sh(x["beta"])).to(dev, torch.float32)
        del x
    if cfg.momentum:
        M = [torch.zeros_like(w) for w in W]
    out = torch.empty_like(q)
    desc = P.binding.make_desc(cfg.B, cfg.H, cfg.d, cfg.h, cfg.n_kv, cfg.n_q, cfg.chunk, cfg.order,
                               cfg.use_muon, cfg.ns_steps, P.IO_BF16 if cfg.io == "bf16" else P.IO_FP32,
                               bool(cfg.lr3), P.FW_LINEAR if cfg.linear else P.FW_SWIGLU)
    ws = torch.empty(P.workspace_bytes(desc), dtype=torch.uint8, device=dev)
    stream = torch.cuda.current_stream(dev)
    launch_on = [stream]   # None while a step is captured into a HIP graph: torch's current stream

    def launch_stream():
        return launch_on[0].cuda_stream if launch_on[0] is not None else None

    io_step = None
    if cfg.layer_io:
        # raw projections and rates, seeded on the device; the prologue makes q, k, v, eta
        gen = torch.Generator(device=dev).manual_seed(0)
        qkv_raw = torch.randn(cfg.B, cfg.n_q, 3, cfg.H, cfg.d, generator=gen, device=dev).to(io)
        lr_raw = torch.randn(cfg.B, cfg.n_q, cfg.H, *((3,) if cfg.lr3 else ()), generator=gen, device=dev)
        rms_w = torch.randn(cfg.H, cfg.d, generator=gen, device=dev)
        y = torch.empty(cfg.B, cfg.n_q, cfg.H, cfg.d, dtype=io, device=dev)
        io_step = {
            "prologue": lambda: P.prologue(qkv_raw, lr_raw, -4.6, n_kv=cfg.n_kv, out=(q, k, v, eta, None),
                                           stream=launch_stream()),
            "rmsnorm": lambda: P.rmsnorm_out(out, rms_w, 1e-6, out=y, stream=launch_stream()),
        }
        esz = 2 if cfg.io == "bf16" else 4
        R = 3 if cfg.lr3 else 1
        io_bytes = {
            "prologue": cfg.B * cfg.n_q * cfg.H * (3 * cfg.d * esz + 4 * R)
                        + cfg.BH * (cfg.n_q * cfg.d * esz + cfg.n_kv * (2 * cfg.d * esz + 4 * R)),
            "rmsnorm": 2 * cfg.BH * cfg.n_q * cfg.d * esz + cfg.H * cfg.d * 4,
        }
        if args.backward:
            # the layer's training step: the norm's reverse (its dO feeds the
            # path's reverse), the path's, then the prologue's; dy and the
            # norm's input o seeded on the device like the projections
            dy_l = torch.randn(cfg.B, cfg.n_q, cfg.H, cfg.d, generator=gen, device=dev).to(io)
            o_l = torch.randn(cfg.B, cfg.H, cfg.n_q, cfg.d, generator=gen, device=dev).to(io)
            dqkv_l, dlr_l, dw_l = torch.empty_like(qkv_raw), torch.empty_like(lr_raw), torch.empty_like(rms_w)
            io_step = {
                "rmsnorm_backward": lambda: P.rmsnorm_out_backward(o_l, dy_l, rms_w, 1e-6, out=(dout, dw_l),
                                                                   stream=launch_stream()),
                "prologue_backward": lambda: P.prologue_backward(qkv_raw, lr_raw, -4.6, None, grads[0], grads[1],
                                                                 grads[2], grads[3], None, out=(dqkv_l, dlr_l, None),
                                                                 stream=launch_stream()),
            }
            # algorithmic bytes: every input read once, every output written once
            io_bytes = {
                "prologue_backward": cfg.B * cfg.n_q * cfg.H * (6 * cfg.d * esz + 8 * R)
                                     + cfg.BH * (cfg.n_q * cfg.d * esz + cfg.n_kv * (2 * cfg.d * esz + 4 * R)),
                "rmsnorm_backward": 3 * cfg.BH * cfg.n_q * cfg.d * esz + 2 * cfg.H * cfg.d * 4,
            }
    sched = None
    if cfg.schedule:
        from lact_synth import make_schedule
        sched = make_schedule(cfg)

    def step():
        if io_step is not None and args.backward:
            io_step["rmsnorm_backward"]()
            path()
            io_step["prologue_backward"]()
            return
        if io_step is not None:
            io_step["prologue"]()
        path()
        if io_step is not None:
            io_step["rmsnorm"]()

    if args.backward:
        from lact_synth import make_cotangents
        if on_device:
            raise SystemExit("--backward runs on host-drawn inputs")
        ct = make_cotangents(cfg, 0)
        dout = torch.from_numpy(ct["do"].reshape(cfg.B, cfg.H, cfg.n_q, cfg.d)).to(dev, io)
        del ct
        Wb = W[:1] if cfg.linear else W
        grads = (torch.empty_like(q), torch.empty_like(k), torch.empty_like(v), torch.empty_like(eta),
                 *(torch.empty_like(w) for w in Wb))
        if sched is not None:   # lact_backward_schedule (no momentum here)
            if cfg.momentum:
                raise SystemExit("--backward of a scheduled workload runs without momentum")
            ws = torch.empty(P.binding.backward_schedule_workspace_bytes(desc, sched), dtype=torch.uint8, device=dev)
        elif cfg.momentum:   # from a seeded nonzero state; the factor's and the state's cotangents too
            from lact_synth import make_momentum_state
            st = make_momentum_state(cfg, 0)
            M = [torch.from_numpy(st[m].reshape(cfg.B, cfg.H, *st[m].shape[1:])).to(dev, torch.float32)
                 for m in (("M",) if cfg.linear else ("M1", "M2", "M3"))]
            del st
            pick = (lambda t: t[0]) if cfg.linear else tuple
            grads = grads[:4] + (torch.empty_like(beta), pick(grads[4:]), pick([torch.empty_like(m) for m in M]))
            ws = torch.empty(P.backward_momentum_workspace_bytes(desc), dtype=torch.uint8, device=dev)
        else:
            ws = torch.empty(P.backward_workspace_bytes(desc), dtype=torch.uint8, device=dev)

    def path():
        if args.backward and sched is not None:
            P.backward_schedule(q, k, v, eta, *W, dout, sched, use_muon=bool(cfg.use_muon), ns_steps=cfg.ns_steps,
                                chunk=cfg.chunk, workspace=ws, stream=launch_stream(),
                                out=grads[:4] + (tuple(grads[4:]),))
        elif args.backward and cfg.momentum:
            P.backward_momentum(q, k, v, eta, beta, Wb[0] if cfg.linear else tuple(Wb), M[0] if cfg.linear else tuple(M),
                                dout, cfg.chunk, order=cfg.order, use_muon=bool(cfg.use_muon), ns_steps=cfg.ns_steps,
                                out=grads, workspace=ws, stream=launch_stream())
        elif args.backward and cfg.linear:
            P.backward_linear(q, k, v, eta, W[0], dout, cfg.chunk, order=cfg.order, use_muon=bool(cfg.use_muon),
                              ns_steps=cfg.ns_steps, out=grads, workspace=ws, stream=launch_stream())
        elif args.backward:
            P.backward(q, k, v, eta, *W, dout, cfg.chunk, order=cfg.order, use_muon=bool(cfg.use_muon),
                       ns_steps=cfg.ns_steps, out=grads, workspace=ws, stream=launch_stream())
        elif cfg.linear:
            P.forward_linear(q, k, v, eta, W[0], cfg.chunk, order=cfg.order, use_muon=bool(cfg.use_muon),
                             ns_steps=cfg.ns_steps, out=out, workspace=ws, stream=launch_stream())
        elif sched is not None:
            P.forward_schedule(q, k, v, eta, *W, sched, use_muon=bool(cfg.use_muon), ns_steps=cfg.ns_steps,
                               chunk=cfg.chunk, out=out, workspace=ws, stream=launch_stream(),
                               **({"beta": beta, "M1": M[0], "M2": M[1], "M3": M[2]} if cfg.momentum else {}))
        elif cfg.momentum:
            P.forward_momentum(q, k, v, eta, beta, *W, *M, chunk=cfg.chunk, order=cfg.order,
                               use_muon=bool(cfg.use_muon), ns_steps=cfg.ns_steps, out=out, workspace=ws,
                               stream=launch_stream())
        else:
            P.forward(q, k, v, eta, *W, chunk=cfg.chunk, order=cfg.order, use_muon=bool(cfg.use_muon),
                      ns_steps=cfg.ns_steps, out=out, workspace=ws, stream=launch_stream())

    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()
    run = step
    if args.graph:
        # the whole step captured once into a HIP graph and replayed: the
        # entry points launch kernels only, so the replay does the same work
        graph = torch.cuda.CUDAGraph()
        launch_on[0] = None
        with torch.cuda.graph(graph):
            step()
        launch_on[0] = stream
        torch.cuda.synchronize()
        run = graph.replay
    t0 = time.perf_counter()
    for _ in range(args.steps):
        run()
    torch.cuda.synchronize()
    dt = (time.perf_counter() - t0) / max(args.steps, 1)

    flops = backward_flops(cfg) if args.backward else workload_flops(cfg)
    tflops = flops / dt / 1e12
    tokens = cfg.B * cfg.n_q
    peak = PEAK_BF16_TFLOPS if cfg.io == "bf16" else PEAK_FP32_MFMA_TFLOPS
    res = {
        "metric": METRIC_BWD if args.backward else METRIC, "value": round(tflops, 3), "unit": "TFLOP/s", "n_gpus": 1,
        "steps": args.steps, "warmup": args.warmup, "ms_per_step": round(dt * 1e3, 4),
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None,
        "dtype": "bf16" if cfg.io == "bf16" else "fp32", "data": "synthetic",
        "config": {"workload": describe(cfg) + ((", backward (lact_rmsnorm_out_backward, lact_backward, "
                                                 "lact_prologue_backward)" if cfg.layer_io else
                                                 ", backward (lact_backward_schedule)" if cfg.schedule else
                                                 ", backward (lact_backward_momentum)" if cfg.momentum else
                                                 ", backward (lact_backward_linear)" if cfg.linear else
                                                 ", backward (lact_backward)") if args.backward else ""),
                   "tokens_per_step": tokens, "flops_per_step": flops},
        "tokens_per_s": round(tokens / dt, 1),
        "launch": "hip_graph" if args.graph else "eager",
        "pct_of_peak": round(100.0 * tflops / peak, 2),
    }
    if on_device:
        res["data"] = "synthetic, drawn on the device (seeded torch generator, the recipe's distributions)"
    if cfg.use_muon:   # the same time over the token FLOPs alone (Newton-Schulz FLOPs left out)
        res["value_without_muon_flops"] = round(workload_flops(cfg.with_(use_muon=0)) / dt / 1e12, 3)

    if not args.no_roofline:
        P.timing_reset()
        P.timing_enable(True)
        for _ in range(args.steps):
            step()
        torch.cuda.synchronize()
        P.timing_enable(False)
        per = {}
        for kc, name in enumerate(P.KCLASS_NAMES):
            n, ms, fl = P.timing_read(kc)
            if n:
                per[name] = {"launches": n, "avg_us": round(1e3 * ms / n, 3), "total_ms": round(ms, 4),
                             "tflops": round(fl / (ms * 1e-3) / 1e12, 2) if ms > 0 and fl > 0 else None}
        P.timing_reset()
        dom = max(per, key=lambda kname: per[kname]["total_ms"])
        d = per[dom]
        achieved = d["tflops"] or 0.0
        kname = DOMINANT_KERNEL.get(dom, dom)
        # the counter reports and the byte counts are the forward's launches;
        # the backward's k_bwd launches are other products (no report: null)
        traffic = None if args.backward else measured_traffic(cfg.name, kname)
        alg = None if args.backward else kernel_alg_bytes(cfg, kname, d["launches"] / max(args.steps, 1))
        res["roofline"] = {"bound": "mfma", "kernel": kname,
                           "achieved": achieved, "peak": peak, "unit": "TFLOP/s",
                           "frac": round(achieved / peak, 4), "traffic": traffic,
                           "traffic_unit": "bytes per launch (HBM, rocprofv3 FETCH_SIZE + WRITE_SIZE, copy-calibrated)",
                           "alg_bytes_per_launch": round(alg) if alg else None,
                           "traffic_over_alg": round(traffic / alg, 3) if (traffic and alg) else None,
                           "avg_launch_us": d["avg_us"],
                           "flops_per_launch": round(achieved * 1e12 * d["avg_us"] * 1e-6),
                           "per_class": per}
        if io_step is not None:
            res["io_kernels"] = {}
            for name, fn in io_step.items():
                P.timing_reset()
                P.timing_enable(True)
                for _ in range(args.steps):
                    fn()
                torch.cuda.synchronize()
                P.timing_enable(False)
                n, ms, _ = P.timing_read(P.KCLASS_NAMES.index("io"))
                P.timing_reset()
                avg = ms / n * 1e-3
                gbs = io_bytes[name] / avg / 1e9
                res["io_kernels"][name] = {"bound": "hbm", "achieved": round(gbs, 1), "peak": PEAK_HBM_GBS,
                                           "unit": "GB/s", "frac": round(gbs / PEAK_HBM_GBS, 4),
                                           "bytes_per_launch": io_bytes[name], "avg_launch_us": round(avg * 1e6, 3)}
    return res


# The second workload that the performance target names, measured in the same
# process after the default one: NVS with a million context tokens; then the
# backward at the LM shape: SwiGLU without and with Muon, the linear fast weight, and SwiGLU with momentum.
SECONDARY = "nvs1m"
SECONDARY_BWD = ("lm32k", "lm32k_muon", "lm32k_linear", "lm32k_mom")


def main():
    args = parse()
    if args.traffic_report:
        traffic_report(args.config, *args.traffic_report)
        return
    if args.gpus != 1:
        print(json.dumps({"error": "this build runs on one GPU only; --gpus must be 1",
                          "n_gpus": args.gpus}))
        sys.exit(2)
    if args.copy_calibration:
        copy_calibration()
        return
    import torch

    import paper_2505_23884_amd as P
    from lact_synth import CONFIGS

    cfg = CONFIGS[args.config]
    if args.chunk:
        if cfg.schedule or cfg.layer_io:
            raise SystemExit("--chunk applies to the uniform-chunk workloads")
        cfg = cfg.with_(name=f"{cfg.name}_c{args.chunk}", chunk=args.chunk)
    if args.backward and not args.no_secondary:
        args.no_secondary = True   # the backward line stands alone
    if args.library_gemms:
        library_gemms(cfg, max(args.steps, 5))
        return
    res = measure(cfg, args, P, on_device=args.device_inputs)
    if not args.no_secondary and args.config == "lm32k" and not args.chunk:
        torch.cuda.empty_cache()
        sec = measure(CONFIGS[SECONDARY], args, P, on_device=True)
        keep = ("value", "unit", "ms_per_step", "tokens_per_s", "pct_of_peak", "data", "config", "roofline")
        res["secondary"] = {SECONDARY: {k: sec[k] for k in keep if k in sec}}
        torch.cuda.empty_cache()
        # the backward at the LM shape, SwiGLU and linear fast weight (its own metric)
        bargs = argparse.Namespace(**{**vars(args), "backward": True})
        for name in SECONDARY_BWD:
            bwd = measure(CONFIGS[name], bargs, P)
            res["secondary"][name + "_backward"] = {"metric": bwd["metric"], **{k: bwd[k] for k in keep if k in bwd}}
            torch.cuda.empty_cache()
    if not args.no_cpu_baseline:
        res["cpu_baseline"] = cpu_baseline(cfg, args.cpu_seconds, args.backward)
    print(json.dumps(res), flush=True)


if __name__ == "__main__":
    main()
