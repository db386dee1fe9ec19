#!/usr/bin/env python3
"""Benchmark: one paper-scale PPO optimizer step on one MI355X.

Workload: the full optimizer step of OpenAI Five's method at the paper's LSTM
size -- GAE over 128 segments of 256 steps, the cut into 2048 samples of 16
steps, the 4096-unit LSTM forward pass (input width 4096), four categorical
heads (30, 8, 32, 4) plus a value head with the PPO loss and its gradient,
truncated BPTT, and Adam with the +-5 sqrt(v) clip over every parameter
(fp32 master weights, bf16 GEMM operands).  Inputs are synthetic and resident
in device memory before the timed region; the behaviour-policy data (actions,
log-probabilities, values) come from an untimed pass of the same library with
perturbed weights.

Prints one JSON line: timesteps/s (B*T per step), the roofline of the
dominant kernel (device time from HIP events recorded by the library on the
launch stream during the timed region), per-site kernel times, and the CPU
oracle timed on a bounded sample of the same workload.
"""
import argparse
import json
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

METRIC = "PPO train timesteps/sec at LSTM H=4096,T=16 (1 GPU); % bf16 MFMA peak"
PEAK_BF16_TFLOPS = 2500.0      # MI355X dense bf16 MFMA
PEAK_HBM_GBS = 8000.0          # MI355X HBM3E


def log(msg):
    print(f"[bench] {msg}", file=sys.stderr, flush=True)


def source_digest():
    """sha256 over the library's kernel sources (csrc/*), in name order."""
    import hashlib
    d = os.path.join(ROOT, "paper_1912_06680_amd", "csrc")
    h = hashlib.sha256()
    for f in sorted(os.listdir(d)):
        h.update(f.encode())
        with open(os.path.join(d, f), "rb") as fh:
            h.update(fh.read())
    return h.hexdigest()


def measured_traffic(kernel, path=None):
    """HBM bytes per launch of `kernel` from the counter runs summarised in
    profiles/traffic.json (or `path`), or None when absent or taken on other
    sources."""
    path = path or os.path.join(ROOT, "profiles", "traffic.json")
    try:
        with open(path) as fh:
            t = json.load(fh)
    except (OSError, ValueError):
        return None
    if t.get("source_digest") != source_digest():
        return None
    k = t.get("kernels", {}).get(kernel)
    if not k:
        return None
    return k["fetch_bytes_per_launch"] + k["write_bytes_per_launch"]


# Kernel (symbol substring) behind each timed site, for the counter summary.
# Where one symbol serves several sites the most frequent (symbol, grid)
# group is taken: the recurrent GEMM runs T times per step.
SITE_SYMBOLS = {
    "lstm_fwd_gemm": "EpiLstmCell",
    "lstm_dh_gemm": "o5::EpiStoreF32, unsigned short>(o5::KRows2",
    "lstm_dw_gemm": "EpiStoreF32Split2",
    "lstm_bwd_cell": "lstm_bwd_cell",
    "adam_step": "adam_kernel",
    "gae": "gae_",
}
COPY_REF_N = 1 << 26   # fp32 elements of the reference conversion (256 MiB read, 128 MiB written)


def summarize_counters(fetch_dir, write_dir, path=None):
    """Turn two `rocprofv3 --pmc FETCH_SIZE` / `--pmc WRITE_SIZE` runs of
    `bench.py --copy-ref` into profiles/traffic.json: bytes per launch of
    each timed site's kernel within the step (dispatches before the
    reference conversion).  Both counters read KiB per dispatch; each is
    scaled by bytes/counter of the reference conversion (COPY_REF_N fp32
    elements read, as many bf16 written)."""
    out = {"source_digest": source_digest(), "kernels": {}}
    for name, d, ref_bytes in (("FETCH_SIZE", fetch_dir, 4.0 * COPY_REF_N), ("WRITE_SIZE", write_dir, 2.0 * COPY_REF_N)):
        g = _pmc_groups(d, {name})
        ref = [v[name] for (ph, k, grid), v in g.items() if ph == "ref"]
        if len(ref) != 1:
            raise SystemExit(f"{name}: reference conversion not found exactly once")
        counted = 1024.0 * sum(ref[0]) / len(ref[0])
        scale = ref_bytes / counted
        out[name] = {"copy_ref_counted_bytes": counted, "copy_ref_bytes": ref_bytes, "scale": scale}
        for site, sym in SITE_SYMBOLS.items():
            cand = [(len(v[name]), k, grid, v[name]) for (ph, k, grid), v in g.items() if ph == "step" and sym in k]
            if not cand:
                continue
            _, kname, grid, v = max(cand, key=lambda c: c[0])
            e = out["kernels"].setdefault(site, {"symbol": kname[:160], "grid_threads": grid})
            key = "fetch_bytes_per_launch" if name == "FETCH_SIZE" else "write_bytes_per_launch"
            e[key] = round(scale * 1024.0 * sum(v) / len(v))
            e["dispatches_" + name.lower()] = len(v)
    out["kernels"] = {k: v for k, v in out["kernels"].items()
                      if "fetch_bytes_per_launch" in v and "write_bytes_per_launch" in v}
    path = path or os.path.join(ROOT, "profiles", "traffic.json")
    with open(path, "w") as fh:
        json.dump(out, fh, indent=1)
        fh.write("\n")
    print(json.dumps(out, indent=1))
    return out


def _copy_ref_dispatch(rows, grid_of):
    """Dispatch id of the reference conversion (the one o5_f32_to_bf16 launch
    with COPY_REF_N / 8 threads), which bench.py --copy-ref runs right after
    the timed steps and before the other workloads."""
    ids = [int(r["Dispatch_Id"]) for r in rows
           if "f32_to_bf16_kernel" in r["Kernel_Name"] and grid_of(r) == COPY_REF_N // 8]
    if len(set(ids)) != 1:
        raise SystemExit("reference conversion not found exactly once")
    return ids[0]


def _phase(dispatch, ref):
    return "step" if dispatch < ref else ("ref" if dispatch == ref else "other")


def _pmc_groups(d, counters):
    """{(phase, kernel, grid threads): {counter: [values per dispatch]}} from
    the counter_collection CSVs of one rocprofv3 --pmc run; phase "step" for
    dispatches before the reference conversion, "ref" for it, "other" after."""
    import csv
    import glob
    rows = []
    for f in glob.glob(os.path.join(d, "**", "*counter_collection.csv"), recursive=True):
        with open(f) as fh:
            rows += [r for r in csv.DictReader(fh) if r["Counter_Name"] in counters]
    ref = _copy_ref_dispatch(rows, lambda r: int(r["Grid_Size"]))
    out = {}
    for r in rows:
        key = (_phase(int(r["Dispatch_Id"]), ref), r["Kernel_Name"], int(r["Grid_Size"]))
        out.setdefault(key, {}).setdefault(r["Counter_Name"], []).append(float(r["Counter_Value"]))
    return out


def _trace_groups(d):
    """{(phase, kernel, grid threads): [durations in us]} from a
    --kernel-trace run (phases as in _pmc_groups)."""
    import csv
    import glob
    rows = []
    for f in glob.glob(os.path.join(d, "**", "*kernel_trace.csv"), recursive=True):
        with open(f) as fh:
            rows += list(csv.DictReader(fh))
    grid = lambda r: int(r["Grid_Size_X"]) * int(r["Grid_Size_Y"]) * int(r["Grid_Size_Z"])  # noqa: E731
    ref = _copy_ref_dispatch(rows, grid)
    out = {}
    for r in rows:
        us = (int(r["End_Timestamp"]) - int(r["Start_Timestamp"])) / 1e3
        out.setdefault((_phase(int(r["Dispatch_Id"]), ref), r["Kernel_Name"], grid(r)), []).append(us)
    return out


def _short(name):
    """Kernel symbol without namespaces and parameter list, template
    arguments kept (shortened)."""
    n = name.replace("void ", "").replace("o5::", "").replace("unsigned short", "bf16")
    depth, cut = 0, len(n)
    for i, ch in enumerate(n):
        if ch == "<":
            depth += 1
        elif ch == ">":
            depth -= 1
        elif ch == "(" and depth == 0:
            cut = i
            break
    return n[:cut][:70]


N_XCD, N_SIMD = 8, 1024   # MI355X: 8 XCDs, 256 CUs x 4 SIMDs


def counter_table(fetch_dir, write_dir, mfma_dir, trace_dir, out_md, command):
    """Per-kernel table from four rocprofv3 runs of bench.py --copy-ref:
    FETCH_SIZE and WRITE_SIZE (scaled by the reference conversion as in
    summarize_counters), SQ_INSTS_MFMA / SQ_VALU_MFMA_BUSY_CYCLES /
    GRBM_GUI_ACTIVE, and the kernel trace.  MFMA busy is the fraction of
    SIMD cycles the matrix pipes were busy: SQ_VALU_MFMA_BUSY_CYCLES /
    (1024 SIMDs x GRBM_GUI_ACTIVE / 8 XCDs) (GRBM_GUI_ACTIVE sums the 8
    XCDs' busy cycles); the clock is those cycles over the traced duration.
    Two sections: the optimizer step at the benchmark shape (dispatches
    before the reference conversion: warmup, instrumented and timed steps)
    and the other workloads (after it).  One row per (kernel, grid) group."""
    tr = _trace_groups(trace_dir)
    fe = _pmc_groups(fetch_dir, {"FETCH_SIZE"})
    wr = _pmc_groups(write_dir, {"WRITE_SIZE"})
    mf = _pmc_groups(mfma_dir, {"SQ_INSTS_MFMA", "SQ_VALU_MFMA_BUSY_CYCLES", "GRBM_GUI_ACTIVE", "SQ_BUSY_CYCLES"})

    def scale(groups, counter, ref_bytes):
        ref = [v[counter] for (ph, k, grid), v in groups.items() if ph == "ref"]
        if len(ref) != 1:
            raise SystemExit(f"{counter}: reference conversion not found exactly once")
        return ref_bytes / (1024.0 * sum(ref[0]) / len(ref[0]))

    sf, sw = scale(fe, "FETCH_SIZE", 4.0 * COPY_REF_N), scale(wr, "WRITE_SIZE", 2.0 * COPY_REF_N)
    mean = lambda v: sum(v) / len(v)  # noqa: E731
    rows = []
    for key, durs in tr.items():
        if key[0] == "ref" or "at::native" in key[1] or "rocclr" in key[1]:
            continue
        r = {"phase": key[0], "kernel": _short(key[1]), "grid": key[2], "n": len(durs), "us": mean(durs)}
        if key in fe:
            r["fetch_mb"] = sf * 1024.0 * mean(fe[key]["FETCH_SIZE"]) / 1e6
        if key in wr:
            r["write_mb"] = sw * 1024.0 * mean(wr[key]["WRITE_SIZE"]) / 1e6
        if "fetch_mb" in r and "write_mb" in r:
            r["gbs"] = (r["fetch_mb"] + r["write_mb"]) * 1e6 / (r["us"] * 1e-6) / 1e9
        m = mf.get(key)
        if m and "SQ_INSTS_MFMA" in m and mean(m["SQ_INSTS_MFMA"]) > 0:
            grbm = mean(m["GRBM_GUI_ACTIVE"]) / N_XCD
            r["mfma_instr"] = mean(m["SQ_INSTS_MFMA"])
            r["mfma_tflops"] = r["mfma_instr"] * 32768.0 / (r["us"] * 1e-6) / 1e12
            r["mfma_busy"] = mean(m["SQ_VALU_MFMA_BUSY_CYCLES"]) / (N_SIMD * grbm)
            r["clock_ghz"] = grbm / (r["us"] * 1e3)
        rows.append(r)
    rows.sort(key=lambda r: (r["phase"] != "step", -r["us"] * r["n"]))
    f = lambda r, k, fmt: (fmt.format(r[k]) if k in r else "")  # noqa: E731
    head = ["| kernel | grid threads | dispatches | avg us | fetch MB | write MB | GB/s (counted) | MFMA instr | "
            "MFMA TFLOP/s | MFMA busy | GHz |",
            "|---|---:|---:|---:|---:|---:|---:|---:|---:|---:|---:|"]
    lines = ["# Per-kernel counters: the PPO optimizer step at H = 4096 (B = 2048 x T = 16), then the other "
             "workloads", "", "Command (four runs on one MI355X; the table by the last line, on the CPU):", "", "```",
             command, "```", "",
             f"Counter scaling from the reference conversion (2^26 fp32 read, 2^26 bf16 written): FETCH_SIZE x "
             f"{sf:.3f}, WRITE_SIZE x {sw:.3f}. WRITE_SIZE misses lines still dirty in the L2 when a kernel "
             f"ends, so it can read below the bytes a kernel writes. MFMA busy = SQ_VALU_MFMA_BUSY_CYCLES / "
             f"(1024 SIMDs x GRBM_GUI_ACTIVE / 8), at the clock the kernel ran at (column `GHz`); MFMA TFLOP/s = "
             f"SQ_INSTS_MFMA x 32768 FLOP (v_mfma_f32_32x32x16_bf16) / traced time.", ""]
    for phase, title in (("step", "## The optimizer step (warmup, instrumented and timed steps)"),
                         ("other", "## The other workloads (tiny and mid steps, LSTM forward + BPTT at B = 1024, "
                                   "rollout inference at B = 4096)")):
        lines += [title, ""] + head
        for r in rows:
            if r["phase"] != phase:
                continue
            lines.append(f"| `{r['kernel']}` | {r['grid']} | {r['n']} | {r['us']:.1f} | {f(r, 'fetch_mb', '{:.1f}')} | "
                         f"{f(r, 'write_mb', '{:.1f}')} | {f(r, 'gbs', '{:.0f}')} | {f(r, 'mfma_instr', '{:.0f}')} | "
                         f"{f(r, 'mfma_tflops', '{:.0f}')} | {f(r, 'mfma_busy', '{:.3f}')} | "
                         f"{f(r, 'clock_ghz', '{:.2f}')} |")
        lines.append("")
    with open(out_md, "w") as fh:
        fh.write("\n".join(lines))
    print("\n".join(lines))
    return rows


def trace_summary(trace_dir, out_md, command, bench_log=None):
    """The rocprofv3 --kernel-trace --stats summary of a bench.py --copy-ref
    run as a table (every symbol's calls and durations), and, for the
    forward GEMM, the average over the launches of the timed steps (the last
    `steps` x T forward launches before the reference conversion) beside the
    per-launch time bench.py printed for the same steps (from its JSON line
    in bench_log)."""
    import csv
    import glob
    stats = []
    for f in glob.glob(os.path.join(trace_dir, "**", "*kernel_stats.csv"), recursive=True):
        with open(f) as fh:
            stats += list(csv.DictReader(fh))
    rows = []
    for f in glob.glob(os.path.join(trace_dir, "**", "*kernel_trace.csv"), recursive=True):
        with open(f) as fh:
            rows += list(csv.DictReader(fh))
    rows.sort(key=lambda r: int(r["Start_Timestamp"]))
    line = None
    if bench_log:
        with open(bench_log) as fh:
            for ln in fh:
                if ln.startswith("{"):
                    line = json.loads(ln)
    lines = ["# Kernel trace: the PPO optimizer step at H = 4096 (B = 2048 x T = 16, bf16), then the other workloads",
             "", "Command (from the repository root, `TMPDIR=/tmp`, on one MI355X; the table by `bench.py "
             "--trace-summary` on the CPU):", "", "```", command, "```", "",
             "The run holds 2 warmup, 5 instrumented (an event pair around every launch site) and 5 timed steps, "
             "then the other workloads (tiny and mid steps, LSTM forward + BPTT at B = 1024, rollout inference at "
             "B = 4096); `--stats` pools every dispatch of a symbol, so a symbol that serves several shapes averages "
             "over them (the counter table splits them by grid and phase)."]
    if line is not None:
        grid = lambda r: int(r["Grid_Size_X"]) * int(r["Grid_Size_Y"]) * int(r["Grid_Size_Z"])  # noqa: E731
        ref = _copy_ref_dispatch(rows, grid)
        fwd = [r for r in rows if int(r["Dispatch_Id"]) < ref and "EpiLstmCell" in r["Kernel_Name"]
               and grid(r) == 262144]
        n = line["steps"] * line["config"]["seq_len"]
        us = [(int(r["End_Timestamp"]) - int(r["Start_Timestamp"])) / 1e3 for r in fwd]
        timed, inst = us[-n:], us[-2 * n:-n]
        lines += ["", f"The timed steps of this run under the profiler: {line['ms_per_step']:.2f} ms per step. The "
                      f"dominant kernel, the fused forward GEMM (`gemm_kk<256, true, EpiLstmCell<bf16>, bf16>`, grid "
                      f"262144): its {n} launches inside the timed steps average {sum(timed) / n:.1f} µs in this "
                      f"trace, and bench.py's HIP events over the same steps gave "
                      f"{1e3 * line['roofline']['ms_per_launch']:.1f} µs per launch (`roofline.ms_per_launch`); "
                      f"the {n} launches of the instrumented pass, with an event pair around each, average "
                      f"{sum(inst) / n:.1f} µs."]
    lines += ["", "| kernel | calls | avg µs | min µs | max µs | total ms | % |", "|---|---:|---:|---:|---:|---:|---:|"]
    for r in sorted(stats, key=lambda r: -float(r["TotalDurationNs"])):
        if float(r["Percentage"]) < 0.05:
            continue
        lines.append(f"| `{_short(r['Name'])}` | {r['Calls']} | {float(r['AverageNs']) / 1e3:.1f} | "
                     f"{float(r['MinNs']) / 1e3:.1f} | {float(r['MaxNs']) / 1e3:.1f} | "
                     f"{float(r['TotalDurationNs']) / 1e6:.2f} | {float(r['Percentage']):.2f} |")
    with open(out_md, "w") as fh:
        fh.write("\n".join(lines) + "\n")
    print("\n".join(lines))


def gpu_behaviour(st, inp):
    """Untimed: actions, log-probabilities and values of a perturbed policy,
    produced by the library itself (forward pass + sampler)."""
    import torch
    from paper_1912_06680_amd import o5
    from paper_1912_06680_amd.step import PARAM_ORDER
    cfg = st.cfg
    T, B, D, H, L, S = cfg.T, cfg.B, cfg.D, cfg.H, cfg.L, cfg.S
    J = L // T
    st.load_params({k: inp[k] + inp["noise_" + k] for k in PARAM_ORDER})
    st.load_x(inp["x"])
    dev = st.p32.device
    f32 = dict(dtype=torch.float32, device=dev)
    st.h0.copy_(torch.from_numpy(inp["h0"]))
    st.c0.copy_(torch.from_numpy(inp["c0"]))
    st.dones.copy_(torch.from_numpy(inp["dones"]))
    zeros = torch.zeros((L, S), **f32)
    o5.o5_segments_to_samples(L, S, T, zeros, zeros, st.dones, st.adv_s, st.ret_s, st.reset)
    o5.o5_lstm_fwd(st.dt, T, B, D, H, st.x, st.W["Wx"], st.W["Wh"], st.P["b"], st.h0, st.c0, st.reset,
                   st.h, st.c, None, st.ws)
    N = T * B
    val = torch.empty(N, **f32)
    sws = torch.empty(max(o5.o5_policy_sample_workspace_bytes(st.dt, N, H, st.heads), 256),
                      dtype=torch.uint8, device=dev)
    o5.o5_policy_sample(st.dt, N, H, st.heads, st.h, st.W["Wp"], st.P["bp"], 1, 0, st.act, st.logp_old, val, sws)
    values = torch.empty((L + 1, S), **f32)
    values[:L] = val.view(T, S, J).permute(2, 0, 1).reshape(L, S)
    last = torch.arange(S, device=dev) * J + (J - 1)
    hT = st.h[T - 1, last].float().contiguous()
    cT = st.c[T - 1, last].contiguous()
    xb32 = torch.from_numpy(inp["x_boot"]).to(dev)
    xb = torch.empty_like(xb32, dtype=st.x.dtype)
    if st.bf16:
        o5.o5_f32_to_bf16(xb32.numel(), xb32, xb)
    else:
        xb.copy_(xb32)
    hb = torch.empty((1, S, H), dtype=st.h.dtype, device=dev)
    cb = torch.empty((1, S, H), **f32)
    bws = torch.empty(max(o5.o5_lstm_fwd_workspace_bytes(st.dt, 1, S, D, H), 256), dtype=torch.uint8, device=dev)
    o5.o5_lstm_fwd(st.dt, 1, S, D, H, xb, st.W["Wx"], st.W["Wh"], st.P["b"], hT, cT, None, hb, cb, None, bws)
    act_b = torch.empty((S, len(st.heads)), dtype=torch.int32, device=dev)
    lp_b = torch.empty(S, **f32)
    vb = torch.empty(S, **f32)
    o5.o5_policy_sample(st.dt, S, H, st.heads, hb, st.W["Wp"], st.P["bp"], 1, 1, act_b, lp_b, vb, sws)
    values[L] = vb
    st.values.copy_(values)
    st.rewards.copy_(torch.from_numpy(inp["rewards"]))
    torch.cuda.synchronize()


def _oracle_step_inputs(sub, seed=1):
    """Seeded inputs of one oracle step at config `sub` (behaviour data drawn
    at random: the timing does not depend on it)."""
    from paper_1912_06680_amd import synth
    inp = synth.make_inputs(sub, seed)
    rng = np.random.default_rng(2)
    N = sub.T * sub.B
    act = np.stack([rng.integers(0, n, N) for n in sub.head_sizes], axis=1)
    logp_old = -np.log(np.prod(sub.head_sizes)) + rng.normal(0, 0.05, N)
    values = rng.standard_normal((sub.L + 1, sub.S))
    return inp, act, logp_old, values


def _time_oracle_step(sub, dtype, reps=1):
    """Median wall time of `reps` full oracle steps (GAE, LSTM forward, heads
    and loss, BPTT, Adam over every parameter) at config `sub`, with arrays
    of `dtype`; bf16 configs round their GEMM inputs as the oracle does."""
    from oracle.precision import working
    from oracle.step import ppo_step
    inp, act, logp_old, values = _oracle_step_inputs(sub)
    params = {k: inp[k] for k in ("Wx", "Wh", "b", "Wp", "bp")}
    ts = []
    with working(dtype):
        for _ in range(reps):
            t0 = time.perf_counter()
            ppo_step(params, inp["x"], inp["h0"], inp["c0"], inp["rewards"], inp["dones"], values, act, logp_old,
                     sub.head_sizes, sub.T, sub.gamma, sub.lam, sub.clip_eps, sub.vf_coef, sub.ent_coef, None, sub.lr,
                     sub.beta1, sub.beta2, sub.adam_eps, sub.clip_k, 1, bf16=sub.dtype == "bf16")
            ts.append(time.perf_counter() - t0)
    return float(np.median(ts))


def _time_oracle_lstm(T, B, D, H, dtype, reps=1, seed=3):
    """Median wall time of the oracle's LSTM forward pass and truncated BPTT
    (no input gradient) over B samples of T steps, arrays of `dtype`."""
    from oracle.lstm import lstm_bptt, lstm_forward
    from oracle.precision import working
    rng = np.random.Generator(np.random.PCG64(seed))
    bound = 1.0 / np.sqrt(H)
    Wx = (rng.random((4 * H, D), dtype=np.float32) * 2 - 1) * bound
    Wh = (rng.random((4 * H, H), dtype=np.float32) * 2 - 1) * bound
    b = (rng.random(4 * H, dtype=np.float32) * 2 - 1) * bound
    x = rng.standard_normal((T, B, D), dtype=np.float32)
    h0 = rng.standard_normal((B, H), dtype=np.float32) * 0.1
    c0 = rng.standard_normal((B, H), dtype=np.float32) * 0.1
    dh = rng.standard_normal((T, B, H), dtype=np.float32)
    ts = []
    with working(dtype):
        for _ in range(reps):
            t0 = time.perf_counter()
            h, c, g = lstm_forward(x, Wx, Wh, b, h0, c0)
            lstm_bptt(x, Wx, Wh, h0, c0, None, h, c, g, dh)
            ts.append(time.perf_counter() - t0)
    return float(np.median(ts))


def cpu_threads():
    """Threads the oracle's BLAS actually uses (the pool size it reports)."""
    try:
        from threadpoolctl import threadpool_info
        return max([i.get("num_threads", 1) for i in threadpool_info()] or [1])
    except Exception:
        return os.cpu_count() or 1


def cpu_baseline(cfg, target_s=12.0):
    """Time the CPU oracle (plain NumPy, as it stands) on the host.

    Headline: the full step at the benchmark shape (T = 16, D = H = 4096,
    four heads) on a bounded sample in fp64 -- the same per-sample shapes
    with fewer samples, each its own GAE segment of T steps, plus Adam over
    every parameter (a fixed cost, found from a 2- and a 6-sample run; the
    third run is sized to about target_s).  Beside it, the other workloads
    in fp64 and with the same code in fp32 (``oracle.precision.working``):
    the tiny step (8 x 16, H = 128) and the mid step (256 x 16, H = 1024)
    whole, median of 3 and 1 repetitions; the LSTM forward + BPTT at
    D = H = 4096 on a sample of 8 of its 1024 sequences; the headline slice
    again in fp32."""
    from paper_1912_06680_amd import synth
    threads = cpu_threads()

    def run5(nb, dtype=np.float64):
        sub = synth.scaled(cfg, S=nb, B=nb, L=cfg.T)
        return _time_oracle_step(sub, dtype), sub

    dt1, _ = run5(2)
    dt2, sub = run5(6)
    dt = dt2
    per = max((dt2 - dt1) / 4, 0.02 * dt2 / 6)   # floor against timing noise
    nb = int(min(cfg.B, max(6, round(6 + (target_s - dt2) / per))))
    if nb > 6:
        dt, sub = run5(nb)
    out = {"value": sub.B * sub.T / dt, "unit": "timesteps/s", "cores": int(threads), "kind": "oracle",
           "sample": f"{sub.B} samples x T={sub.T} (D=H={sub.H}, heads {tuple(sub.head_sizes)}, each sample "
                     f"its own GAE segment), one full step of the fp64 NumPy oracle incl. Adam over all "
                     f"{synth.n_params(sub)} params, {dt:.2f} s",
           "host": {"cpu_model": cpu_model(), "os_cpu_count": os.cpu_count(),
                    "threads_env": {k: os.environ.get(k) for k in ("OMP_NUM_THREADS", "OPENBLAS_NUM_THREADS",
                                                                      "MKL_NUM_THREADS")}}}
    others = []
    # fp32: the same code on the plain fp32 configuration (no bf16 operand rounding)
    sub32 = synth.scaled(sub, dtype="f32")
    dt32 = _time_oracle_step(sub32, np.float32)
    others.append({"config": f"full step, sample of the benchmark shape ({sub.B} samples x T={sub.T}, D=H={sub.H})",
                   "dtype": "f32", "s": round(dt32, 3), "timesteps_per_s": round(sub.B * sub.T / dt32, 1)})
    for name, reps in (("tiny", 3), ("mid", 1)):
        c = synth.CONFIGS[name]
        for dtype, dn in ((np.float64, "f64"), (np.float32, "f32")):
            t = _time_oracle_step(c, dtype, reps)
            others.append({"config": f"full step {name}: B={c.B} x T={c.T}, D={c.D} H={c.H}, heads "
                                     f"{list(c.head_sizes)}", "dtype": dn, "s": round(t, 4),
                           "timesteps_per_s": round(c.B * c.T / t, 1)})
    B3 = 8
    for dtype, dn in ((np.float64, "f64"), (np.float32, "f32")):
        t = _time_oracle_lstm(16, B3, 4096, 4096, dtype)
        others.append({"config": f"LSTM forward + BPTT, sample of {B3} of 1024 sequences x T=16, "
                                 f"D=H=4096", "dtype": dn, "s": round(t, 3), "timesteps_per_s": round(B3 * 16 / t, 1)})
    out["other_configs"] = others
    return out


def other_configs(cfg, reps=5, warm=2):
    """The two other single-GPU workloads of the method at paper scale, each
    timed warm with events on the launch stream (median of `reps` after
    `warm` untimed runs): the LSTM forward pass and truncated BPTT alone at
    B = 1024 samples x T = 16 (D = H = 4096, no input gradient), and one
    rollout inference step for B = 4096 environments (one LSTM step without
    saved gates, then the heads and the Gumbel-max draw).  Inputs are
    synthetic: x ~ N(0, 1), weights U(-1/sqrt(H), 1/sqrt(H)), h0, c0 and
    the upstream gradient ~ N(0, 0.1^2) and N(0, 1)."""
    import torch
    from paper_1912_06680_amd import o5
    dev = "cuda"
    gen = torch.Generator(device=dev)
    gen.manual_seed(1)
    dt = o5.O5_BF16
    et = torch.bfloat16
    D = H = cfg.H
    G = 4 * H
    bound = H ** -0.5

    def uni(shape):
        return ((torch.rand(shape, generator=gen, device=dev) * 2 - 1) * bound).to(et)

    def timed(fn):
        ts = []
        for i in range(warm + reps):
            e0 = torch.cuda.Event(enable_timing=True)
            e1 = torch.cuda.Event(enable_timing=True)
            e0.record()
            fn()
            e1.record()
            torch.cuda.synchronize()
            if i >= warm:
                ts.append(e0.elapsed_time(e1))
        return float(np.median(ts))

    out = []
    # configs 1 and 2: the whole optimizer step at the tiny and mid sizes
    # (latency-bound), as the step runs in the benchmark
    from paper_1912_06680_amd import synth
    from paper_1912_06680_amd.step import PARAM_ORDER, PPOStep
    for name in ("tiny", "mid", "mid_bf16"):
        c = synth.CONFIGS[name]
        inp = synth.make_inputs(c, 0)
        st = PPOStep(c)
        gpu_behaviour(st, inp)
        st.load_params({k: inp[k] for k in PARAM_ORDER})
        st.m.zero_()
        st.v.zero_()
        ms_small = timed(st.run)
        out.append({"workload": f"full PPO step {name}: B={c.B} x T={c.T}, D={c.D} H={c.H}, heads "
                                f"{list(c.head_sizes)} + value, GAE {c.S} x {c.L}, Adam over {st.n_params} params",
                    "dtype": c.dtype, "ms": round(ms_small, 4), "timesteps_per_s": round(c.B * c.T / (ms_small * 1e-3), 1)})
        del st
    torch.cuda.empty_cache()
    Wx, Wh = uni((G, D)), uni((G, H))
    b = (torch.rand(G, generator=gen, device=dev) * 2 - 1) * bound
    T, B = 16, 1024
    x = torch.randn((T, B, D), generator=gen, device=dev).to(et)
    h0 = torch.randn((B, H), generator=gen, device=dev) * 0.1
    c0 = torch.randn((B, H), generator=gen, device=dev) * 0.1
    h = torch.empty((T, B, H), dtype=et, device=dev)
    c = torch.empty((T, B, H), device=dev)
    gates = torch.empty((T, B, G), dtype=et, device=dev)
    dh = torch.randn((T, B, H), generator=gen, device=dev)
    dWx, dWh, db = torch.empty((G, D), device=dev), torch.empty((G, H), device=dev), torch.empty(G, device=dev)
    ws = torch.empty(max(o5.o5_lstm_fwd_workspace_bytes(dt, T, B, D, H), o5.o5_lstm_bptt_workspace_bytes(dt, T, B, D, H)),
                     dtype=torch.uint8, device=dev)

    def lstm_step():
        o5.o5_lstm_fwd(dt, T, B, D, H, x, Wx, Wh, b, h0, c0, None, h, c, gates, ws)
        o5.o5_lstm_bptt(dt, T, B, D, H, x, Wx, Wh, h0, c0, None, h, c, gates, dh, None, None, dWx, dWh, db, None, ws)

    ms = timed(lstm_step)
    flop = 2.0 * T * B * G * (D + H) + 2.0 * G * ((T - 1) * B * H + T * B * H + T * B * D)
    out.append({"workload": f"LSTM forward + truncated BPTT, B={B} x T={T}, D=H={H}, no input gradient",
                "ms": round(ms, 3), "timesteps_per_s": round(B * T / (ms * 1e-3), 1),
                "tflops": round(flop / (ms * 1e-3) / 1e12, 2),
                "frac_mfma_peak": round(flop / (ms * 1e-3) / 1e12 / PEAK_BF16_TFLOPS, 4)})
    del x, h0, c0, h, c, gates, dh, dWx, dWh, db, ws
    B = 4096
    heads = tuple(cfg.head_sizes)
    A1 = sum(heads) + 1
    Wp = uni((A1, H))
    bp = torch.zeros(A1, device=dev)
    x = torch.randn((1, B, D), generator=gen, device=dev).to(et)
    h0 = torch.randn((B, H), generator=gen, device=dev) * 0.1
    c0 = torch.randn((B, H), generator=gen, device=dev) * 0.1
    h = torch.empty((1, B, H), dtype=et, device=dev)
    c = torch.empty((1, B, H), device=dev)
    ws = torch.empty(max(o5.o5_lstm_fwd_workspace_bytes(dt, 1, B, D, H), 256), dtype=torch.uint8, device=dev)
    act = torch.empty((B, len(heads)), dtype=torch.int32, device=dev)
    logp = torch.empty(B, device=dev)
    val = torch.empty(B, device=dev)
    sws = torch.empty(max(o5.o5_policy_sample_workspace_bytes(dt, B, H, heads), 256), dtype=torch.uint8, device=dev)
    counter = [0]

    def rollout():
        o5.o5_lstm_fwd(dt, 1, B, D, H, x, Wx, Wh, b, h0, c0, None, h, c, None, ws)
        o5.o5_policy_sample(dt, B, H, heads, h[0], Wp, bp, 0, counter[0], act, logp, val, sws)
        counter[0] += 1

    ms = timed(rollout)
    flop = 2.0 * B * G * (D + H) + 2.0 * B * A1 * H
    out.append({"workload": f"rollout inference: one LSTM step for B={B} environments (D=H={H}), heads "
                            f"{list(heads)} + value, Gumbel-max sampling",
                "ms": round(ms, 3), "env_steps_per_s": round(B / (ms * 1e-3), 1),
                "tflops": round(flop / (ms * 1e-3) / 1e12, 2),
                "frac_mfma_peak": round(flop / (ms * 1e-3) / 1e12 / PEAK_BF16_TFLOPS, 4)})
    return out


def hbm_kernels(cfg, reps=20, warm=3):
    """The HBM-bound kernels on their own, at the sizes their bandwidth is
    quoted at: GAE over L=256-step segments at S = 128 (the step's size,
    latency-bound), 11,520 (the paper's 2.9M-timestep batch) and 131,072
    (33.5M timesteps, beyond the 256 MB infinity cache); the reward
    post-processing ahead of GAE at 1,152 and 13,107 games of ten heroes;
    the PPO loss with a unit-selection head scoring 189 units against
    128-wide embeddings at the step's shape (bytes: the embeddings read once
    each way, h read twice, dh written); the LSTM's input side
    (observation normalisation, pre-LSTM layer with
    the cross-hero pool, and its backward) at the step's shape with teams of
    five (B = 2040); the surgery that widens the LSTM from 2048 to 4096
    units; Adam at the step's parameter count and at 158,502,815.
    The input-side layer entries also give the warm TFLOP/s of their GEMM
    work (2 N D Do each way) over the whole call.  Each is timed with events on the
    launch stream, median of `reps` after `warm` untimed calls, cold (a
    512 MB buffer read before every call) and warm."""
    import torch
    from paper_1912_06680_amd import o5, synth
    dev = "cuda"
    gen = torch.Generator(device=dev)
    gen.manual_seed(0)
    flush = torch.ones(128 << 20, dtype=torch.float32, device=dev)
    flush_sum = torch.zeros((), dtype=torch.float32, device=dev)

    def timed(fn, cold):
        ts = []
        for i in range(warm + reps):
            if cold:
                # read 512 MB: evicts the inputs from the L2s and the infinity
                # cache without leaving dirty lines to be written back during
                # the timed call
                flush_sum.copy_(flush.sum())
            e0 = torch.cuda.Event(enable_timing=True)
            e1 = torch.cuda.Event(enable_timing=True)
            e0.record()
            fn()
            e1.record()
            torch.cuda.synchronize()
            if i >= warm:
                ts.append(e0.elapsed_time(e1) * 1e3)
        return float(np.median(ts))

    def entry(kernel, size, nbytes, fn, moved=None):
        """`nbytes`: what the operation must move once; `moved`: what the
        method moves when it is more (a second pass over inputs that exceed
        the caches)."""
        cold, hot = timed(fn, True), timed(fn, False)
        e = {"kernel": kernel, "size": size, "bytes": int(nbytes), "cold_us": round(cold, 2),
             "warm_us": round(hot, 2), "cold_gbs": round(nbytes / cold * 1e-3, 1),
             "frac_hbm_peak_cold": round(nbytes / cold * 1e-3 / PEAK_HBM_GBS, 4)}
        if moved is not None:
            e.update({"moved_bytes": int(moved), "cold_gbs_moved": round(moved / cold * 1e-3, 1),
                      "frac_hbm_peak_cold_moved": round(moved / cold * 1e-3 / PEAK_HBM_GBS, 4)})
        return e

    out = []
    L = 256
    for S in (cfg.S, 11520, 131072):
        r = torch.randn((L, S), generator=gen, device=dev)
        v = torch.randn((L + 1, S), generator=gen, device=dev)
        done = (torch.rand((L, S), generator=gen, device=dev) < 0.002).to(torch.uint8)
        adv = torch.empty((L, S), device=dev)
        ret = torch.empty((L, S), device=dev)
        out.append(entry("gae", f"L={L} S={S}", 17 * L * S + 4 * S,
                         lambda: o5.o5_gae(L, S, r, v, done, cfg.gamma, cfg.lam, adv, ret)))
        del r, v, done, adv, ret
    for G in (1152, 13107):   # 11,520 and 131,070 segments: 5v5 games
        ri = synth.reward_inputs(L, G, seed=G)
        sh, oc, gt = (torch.from_numpy(ri[k]).to(dev) for k in ("shaped", "outcome", "game_time"))
        stats = torch.zeros(3, dtype=torch.float64, device=dev)
        rr = torch.empty((L, 10 * G), device=dev)
        rws = torch.empty(max(o5.o5_reward_process_workspace_bytes(L, G), 256), dtype=torch.uint8, device=dev)
        # two passes (the normalisation needs this call's statistics first):
        # shaped, outcome and game time read twice, r written once
        out.append(entry("reward_process", f"L={L} G={G} (S={10 * G})", 12 * L * 10 * G + 4 * L * G,
                         lambda: o5.o5_reward_process(L, G, sh, oc, gt, 0.3, 0.6, 10.0, 1e-8, stats, rr, rws),
                         moved=20 * L * 10 * G + 8 * L * G))
        del sh, oc, gt, stats, rr, rws
    # the LSTM's input side at the step's shape: 408 teams x 5 replicas x 16
    # steps of a 4096-wide observation into the 4096-wide LSTM input
    Tq, Bq, Do, D = cfg.T, 2040, cfg.D, cfg.D
    Nq = Tq * Bq
    dtq = o5.O5_BF16 if cfg.dtype == "bf16" else o5.O5_F32
    et = torch.bfloat16 if dtq == o5.O5_BF16 else torch.float32
    obs = torch.randn((Nq, Do), generator=gen, device=dev) * 2.0 + 1.0
    ostats = torch.zeros((3, Do), dtype=torch.float64, device=dev)
    oq = torch.empty((Nq, Do), dtype=et, device=dev)
    ows = torch.empty(o5.o5_obs_normalize_workspace_bytes(Nq, Do), dtype=torch.uint8, device=dev)
    # two passes (statistics first, this call's rows included): obs read twice
    out.append(entry("obs_normalize", f"N={Nq} Do={Do}", Nq * Do * (4 + oq.element_size()),
                     lambda: o5.o5_obs_normalize(dtq, Nq, Do, obs, ostats, 5.0, 1e-8, oq, ows),
                     moved=Nq * Do * (8 + oq.element_size())))
    del obs
    Wq = (torch.randn((D, Do), generator=gen, device=dev) / Do ** 0.5).to(et)
    bq = torch.zeros(D, device=dev)
    yq = torch.empty((Nq, D), device=dev)
    xq = torch.empty((Nq, D), dtype=et, device=dev)
    fl = 2.0 * Nq * D * Do
    e = entry("prelstm_fwd", f"T={Tq} B={Bq} Do={Do} D={D}", Nq * Do * 2 + D * Do * 2 + Nq * D * (4 + 4 + 2),
              lambda: o5.o5_prelstm_fwd(dtq, Tq, Bq, Do, D, oq, Wq, bq, yq, xq))
    e["tflops_warm"] = round(fl / e["warm_us"] * 1e-6, 1)
    out.append(e)
    dxq = torch.randn((Nq, D), generator=gen, device=dev).to(et)
    dWq = torch.empty((D, Do), device=dev)
    dbq = torch.empty(D, device=dev)
    pws = torch.empty(o5.o5_prelstm_bwd_workspace_bytes(dtq, Tq, Bq, Do, D), dtype=torch.uint8, device=dev)
    e = entry("prelstm_bwd", f"T={Tq} B={Bq} Do={Do} D={D}", Nq * D * (4 + 2 + 2 + 2) + Nq * Do * 2 + D * Do * 4,
              lambda: o5.o5_prelstm_bwd(dtq, Tq, Bq, Do, D, oq, yq, dxq, dWq, dbq, pws))
    e["tflops_warm"] = round(fl / e["warm_us"] * 1e-6, 1)
    out.append(e)
    del oq, Wq, bq, yq, xq, dxq, dWq, dbq, pws, ows, ostats
    # the PPO loss at the step's shape with a unit-selection head: head 1
    # scores 189 units (the paper's count) against 128-wide embeddings
    uheads = (cfg.head_sizes[0], 189) + tuple(cfg.head_sizes[2:])
    Nu, Hu, du = cfg.T * cfg.B, cfg.H, 128
    A1u = sum(uheads) + 1
    dtu = o5.O5_BF16 if cfg.dtype == "bf16" else o5.O5_F32
    etu = torch.bfloat16 if dtu == o5.O5_BF16 else torch.float32
    hu = torch.tanh(torch.randn((Nu, Hu), generator=gen, device=dev)).to(etu)
    Wpu = (torch.randn((A1u, Hu), generator=gen, device=dev) / Hu ** 0.5).to(etu)
    bpu = torch.zeros(A1u, device=dev)
    Wqu = (torch.randn((du, Hu), generator=gen, device=dev) / Hu ** 0.5).to(etu)
    bqu = torch.zeros(du, device=dev)
    Eu = (torch.randn((Nu, 189, du), generator=gen, device=dev) / du ** 0.5).to(etu)
    actu = torch.stack([torch.randint(0, n, (Nu,), generator=gen, device=dev) for n in uheads], 1).to(torch.int32)
    lpu = torch.full((Nu,), -10.0, device=dev)
    advu, retu = torch.randn(Nu, generator=gen, device=dev), torch.randn(Nu, generator=gen, device=dev)
    stu, dhu = torch.empty(8, device=dev), torch.empty((Nu, Hu), device=dev)
    dWpu, dbpu = torch.empty((A1u, Hu), device=dev), torch.empty(A1u, device=dev)
    dWqu, dbqu = torch.empty((du, Hu), device=dev), torch.empty(du, device=dev)
    uh = o5.unit_head(1, du, Wqu, bqu, Eu, dWqu, dbqu)
    uws = torch.empty(o5.o5_ppo_loss_grad_workspace_bytes(dtu, Nu, Hu, uheads, unit=uh), dtype=torch.uint8,
                      device=dev)
    ebytes = Nu * 189 * du * Eu.element_size()
    out.append(entry("ppo_loss_grad_unit_head", f"N={Nu} H={Hu} heads={list(uheads)} unit head 1 d={du}",
                     2 * ebytes + Nu * Hu * (2 * hu.element_size() + 4),
                     lambda: o5.o5_ppo_loss_grad(dtu, Nu, Hu, uheads, hu, Wpu, bpu, actu, lpu, advu, retu, None, 0.2,
                                                 1.0, 0.01, stu, dhu, dWpu, dbpu, uws, unit=uh)))
    del hu, Wpu, Wqu, Eu, dhu, uws
    # surgery: the paper's LSTM widening 2048 -> 4096 units (input 4096,
    # heads 75), parameters and both moments
    A1q = sum(cfg.head_sizes) + 1
    n_old, n_new = o5.o5_param_count(D, 2048, A1q), o5.o5_param_count(D, 4096, A1q)
    olds = [torch.randn(n_old, generator=gen, device=dev) * 0.02 for _ in range(3)]
    news = [torch.empty(n_new, device=dev) for _ in range(3)]
    out.append(entry("surgery_widen", f"D={D} H=2048->4096 A1={A1q}", 12 * (n_old + n_new),
                     lambda: o5.o5_surgery_widen(D, 2048, A1q, D, 4096, *olds, *news, 1e-3, 7)))
    del olds, news
    for n in (synth.n_params(cfg), 158502815):
        p = torch.randn(n, generator=gen, device=dev) * 0.02
        g = torch.randn(n, generator=gen, device=dev) * 1e-3
        m = g * 0.1
        v = g * g
        pb = torch.empty(n, dtype=torch.bfloat16, device=dev)
        out.append(entry("adam_step", f"n={n}", 30 * n,
                         lambda: o5.o5_adam_step(n, p, m, v, g, pb, cfg.lr, cfg.beta1, cfg.beta2, cfg.adam_eps,
                                                 cfg.clip_k, 10)))
        del p, g, m, v, pb
    del flush
    torch.cuda.empty_cache()
    return out


def stream_copy_gbs(reps=10, warm=3):
    """Device-to-device copy of 1 GiB of fp32 (torch's copy kernel): bytes
    read plus written per second, median of `reps` -- the bandwidth a plain
    streaming kernel reaches on this GPU, a second reference beside the
    published 8 TB/s."""
    import torch
    n = 1 << 28
    src = torch.ones(n, dtype=torch.float32, device="cuda")
    dst = torch.empty_like(src)
    ts = []
    for i in range(warm + reps):
        e0 = torch.cuda.Event(enable_timing=True)
        e1 = torch.cuda.Event(enable_timing=True)
        e0.record()
        dst.copy_(src)
        e1.record()
        torch.cuda.synchronize()
        if i >= warm:
            ts.append(e0.elapsed_time(e1) * 1e-3)
    del src, dst
    torch.cuda.empty_cache()
    return 2.0 * 4 * n / float(np.median(ts)) / 1e9


def cpu_model():
    try:
        with open("/proc/cpuinfo") as fh:
            for line in fh:
                if line.startswith("model name"):
                    return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return "unknown CPU"


def main():
    ap = argparse.ArgumentParser(description=__doc__.split("\n")[0])
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=10)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--config", default="full4096")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-kernel-timers", action="store_true",
                    help="time the steps without the per-launch events (no roofline or per-kernel figures)")
    ap.add_argument("--no-other-configs", action="store_true",
                    help="skip the paper-scale LSTM-only and rollout-inference timings")
    ap.add_argument("--no-hbm-kernels", action="store_true",
                    help="skip the standalone GAE / Adam bandwidth measurements")
    ap.add_argument("--copy-ref", action="store_true",
                    help="after timing, run one conversion of 2^26 fp32 elements (counter scale reference)")
    ap.add_argument("--summarize-counters", nargs=2, metavar=("FETCH_DIR", "WRITE_DIR"),
                    help="write profiles/traffic.json from two rocprofv3 --pmc runs and exit (no GPU)")
    ap.add_argument("--counter-table", nargs=5, metavar=("FETCH_DIR", "WRITE_DIR", "MFMA_DIR", "TRACE_DIR", "OUT_MD"),
                    help="write the per-kernel counter table from four rocprofv3 runs and exit (no GPU)")
    ap.add_argument("--trace-summary", nargs=2, metavar=("TRACE_DIR", "OUT_MD"),
                    help="write the kernel-trace summary of a rocprofv3 --kernel-trace --stats run and exit (no GPU)")
    ap.add_argument("--bench-log", default=None, help="the traced run's output (its JSON line), for --trace-summary")
    ap.add_argument("--command", default="", help="the command recorded in the counter table or trace summary")
    args = ap.parse_args()
    if args.summarize_counters:
        summarize_counters(*args.summarize_counters)
        return
    if args.counter_table:
        counter_table(*args.counter_table, command=args.command)
        return
    if args.trace_summary:
        trace_summary(*args.trace_summary, command=args.command, bench_log=args.bench_log)
        return
    if args.gpus != 1:
        print(f"bench.py runs on one GPU only (got --gpus {args.gpus}); the multi-GPU path "
              "(gradient all-reduce before Adam) is not built", file=sys.stderr)
        sys.exit(2)

    import torch
    from paper_1912_06680_amd import o5, synth
    from paper_1912_06680_amd.step import PARAM_ORDER, PPOStep

    assert torch.cuda.is_available(), "bench.py needs a GPU"
    o5.lib()  # fail loudly if the library is missing
    cfg = synth.CONFIGS[args.config]
    T, B, D, H = cfg.T, cfg.B, cfg.D, cfg.H
    log(f"config {cfg.name}: B={B} T={T} D={D} H={H} heads={cfg.head_sizes} L={cfg.L} S={cfg.S} {cfg.dtype}")
    inp = synth.make_inputs(cfg, 0)
    st = PPOStep(cfg)
    gpu_behaviour(st, inp)
    st.load_params({k: inp[k] for k in PARAM_ORDER})
    st.m.zero_()
    st.v.zero_()
    torch.cuda.synchronize()
    log("inputs resident; warmup")
    for _ in range(args.warmup):
        st.run()
    torch.cuda.synchronize()
    # per-site device time and algorithmic work: one pass of K steps with an
    # event pair around every launch site (the events add ~2 % to a step),
    # then the K timed steps with events around the dominant kernel only
    A1 = sum(cfg.head_sizes) + 1
    n = st.n_params
    # the bf16 step passes the heads' gradient in factored form: the
    # recurrent product of each step t < T-1 also takes the heads' K = ld
    # columns, the last step has those alone (T launches), the loss call
    # writes P (ld bf16 per row) instead of dh, and the cell reads no dh
    ld = st.ld if st.bf16 else 0
    flops = {
        "lstm_fwd_gemm": 2.0 * B * 4 * H * (D + H),
        "lstm_dh_gemm": (2.0 * B * H * ((T - 1) * (4 * H + ld) + ld) / T) if st.bf16 else 2.0 * B * H * 4 * H,
        "lstm_dw_gemm": 2.0 * 4 * H * (D + H) * T * B,
    }
    bytes_ = {
        "lstm_fwd_cell": 34.0 * B * H,
        "lstm_bwd_cell": (36.0 if st.bf16 else 40.0) * B * H,
        "adam_step": 30.0 * n,
        "gae": 17.0 * cfg.L * cfg.S + 4.0 * cfg.S,
        "ppo_loss_grad": (2 * 2.0 * H + (2.0 * ld if st.bf16 else 4.0 * H) + 4.0 * A1 + 16.0) * T * B,
    }
    copy_gbs = stream_copy_gbs()
    log(f"streaming copy: {copy_gbs:.0f} GB/s")
    kernels = {}
    dom = None
    if not args.no_kernel_timers:
        log(f"per-kernel times over {args.steps} instrumented steps")
        o5.o5_ktimer_enable(True)
        for _ in range(args.steps):
            st.run()
        torch.cuda.synchronize()
        o5.o5_ktimer_enable(False)
        for site, name in enumerate(o5.KTIMER_SITES):
            tot, cnt = o5.o5_ktimer_read(site)
            if cnt == 0:
                continue
            per = tot / cnt
            k = {"ms_per_launch": round(per, 5), "launches_per_step": cnt / args.steps,
                 "ms_per_step": round(tot / args.steps, 4)}
            if name in flops:
                k["tflops"] = round(flops[name] / (per * 1e-3) / 1e12, 2)
                k["frac_mfma_peak"] = round(k["tflops"] / PEAK_BF16_TFLOPS, 4)
            if name in bytes_:
                k["gbs"] = round(bytes_[name] / (per * 1e-3) / 1e9, 1)
                k["frac_hbm_peak"] = round(k["gbs"] / PEAK_HBM_GBS, 4)
                k["frac_stream_copy"] = round(k["gbs"] / copy_gbs, 4)
            kernels[name] = k
        if any(s_ in kernels for s_ in flops):
            dom = max(flops, key=lambda s_: kernels.get(s_, {}).get("ms_per_step", 0.0))

    log(f"timing {args.steps} steps")
    # the forward GEMM's T launches per step are timed as one span (a pair of
    # events around the whole o5_lstm_fwd call): an event pair around each
    # launch would add ~10 us of stream time per launch to the timed steps
    span = "lstm_fwd_call" if dom == "lstm_fwd_gemm" else dom
    if dom is not None:
        o5.o5_ktimer_enable_sites([span])
    t0 = time.perf_counter()
    for _ in range(args.steps):
        st.run()
    torch.cuda.synchronize()
    elapsed = time.perf_counter() - t0
    o5.o5_ktimer_enable(False)
    ms_step = elapsed * 1e3 / args.steps
    value = B * T * args.steps / elapsed
    stats = st.stats.cpu().numpy().tolist()
    if args.copy_ref:
        src = torch.ones(COPY_REF_N, dtype=torch.float32, device="cuda")
        dst = torch.empty(COPY_REF_N, dtype=torch.bfloat16, device="cuda")
        o5.o5_f32_to_bf16(COPY_REF_N, src, dst)
        torch.cuda.synchronize()
        del src, dst
    log(f"{ms_step:.3f} ms/step, {value:.0f} timesteps/s, loss {stats[0]:.5f}")
    gemm_ms = sum(kernels[s_]["ms_per_step"] for s_ in flops if s_ in kernels)
    gemm_flop = sum(flops[s_] * kernels[s_]["launches_per_step"] for s_ in flops if s_ in kernels)
    lstm_gemm_tflops = gemm_flop / (gemm_ms * 1e-3) / 1e12 if gemm_ms > 0 else 0.0
    roofline = None
    if dom is not None:
        # the dominant kernel's launches inside the timed steps (for the
        # forward GEMM: the forward calls' span over their T launches each,
        # which also holds the h0 conversion ahead of them, so `achieved`
        # errs low)
        tot, cnt = o5.o5_ktimer_read(o5.KTIMER_SITES.index(span))
        launches = cnt * (T if span == "lstm_fwd_call" else 1)
        per = tot / launches
        tf = flops[dom] / (per * 1e-3) / 1e12
        roofline = {"bound": "mfma", "achieved": round(tf, 2), "peak": PEAK_BF16_TFLOPS, "unit": "TFLOP/s",
                    "frac": round(tf / PEAK_BF16_TFLOPS, 4), "traffic": measured_traffic(dom),
                    "kernel": dom, "flop_per_launch": flops[dom], "ms_per_launch": round(per, 5),
                    "timed_as": f"{span}: {launches} launches in {cnt} spans"}
    step_flop = 2.0 * T * B * 4 * H * (D + H) + 2.0 * 4 * H * ((T - 1) * B * H + T * B * H + T * B * D) + \
        3 * 2.0 * T * B * A1 * H

    others = None
    if not args.no_other_configs:
        log("paper-scale LSTM fwd + BPTT and rollout inference")
        others = other_configs(cfg)

    hbm = None
    if not args.no_hbm_kernels:
        log("standalone HBM-bound kernels (GAE, Adam), cold and warm")
        hbm = hbm_kernels(cfg)
        for e in hbm:
            e["frac_stream_copy_cold"] = round(e["cold_gbs"] / copy_gbs, 4)

    cpu = None
    if not args.no_cpu_baseline:
        log("timing the CPU oracle on a bounded sample")
        cpu = cpu_baseline(cfg)
        log(f"cpu oracle: {cpu['value']:.1f} timesteps/s ({cpu['sample']})")

    out = {
        "metric": METRIC, "value": round(value, 1), "unit": "timesteps/s", "n_gpus": 1,
        "steps": args.steps, "warmup": args.warmup, "ms_per_step": round(ms_step, 4),
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None, "dtype": cfg.dtype,
        "data": "synthetic",
        "config": {"workload": f"full PPO optimizer step: B={B} samples x T={T}, LSTM D={D} H={H}, heads "
                               f"{list(cfg.head_sizes)} + value, GAE {cfg.S} segments x {cfg.L} steps, Adam over "
                               f"{n} params", "global_batch": B * T, "seq_len": T, "parallelism": "none (1 GPU)"},
        "roofline": roofline,
        "cpu_baseline": cpu,
        "stream_copy_gbs": round(copy_gbs, 1),
        "lstm_gemm_mfma_frac": round(lstm_gemm_tflops / PEAK_BF16_TFLOPS, 4),
        "lstm_gemm_tflops": round(lstm_gemm_tflops, 2),
        "step_tflops": round(step_flop / (ms_step * 1e-3) / 1e12, 2),
        "kernels": kernels,
        "other_configs": others,
        "hbm_kernels": hbm,
        "loss_stats": [round(s, 6) for s in stats],
    }
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
