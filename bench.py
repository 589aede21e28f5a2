"""Benchmark of the LiteVLM select + prefill path on one MI355X.

One step = the whole path on one batch: litevlm_select_score_topk (view
selection inside the scoring kernels, scores, top-k, gather) ->
litevlm_prefill_attn, all on one stream with no host synchronisation in
between; the same steps with litevlm_patch_select as its own call before
litevlm_token_score_topk are reported beside them. The workload is the
6-view x 1024-visual-token + 128-text-token multi-camera prompt (GQA 32/8
heads, head dim 128, bf16, batch 1) at keep ratio 0.5; the keep-ratio sweep
{1.0, 0.5, 0.25} is reported alongside.

Prints ONE JSON line. Inputs are seeded synthetic tensors already resident in
HBM; the timed steps rotate over several input sets whose total exceeds the
256 MB last-level cache. The headline steps are timed with events only around
the whole timed region; per-call durations come from a second pass of the same
steps with HIP events recorded on the launch stream around each call.
"""
from __future__ import annotations

import argparse
import hashlib
import json
import math
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

METRIC = "select+prefill latency (ms) and prefill attn TFLOP/s, 6 views×1024 tok, 1 GPU"
PEAK_BF16_TFLOPS = 2500.0     # MI355X dense bf16 MFMA, published
PEAK_FP8_TFLOPS = 5000.0
PEAK_HBM_GBS = 8000.0
HEADLINE_R = 0.5
SWEEP = (1.0, 0.5, 0.25)
TRAFFIC_FILE = os.path.join(ROOT, "profiles", "traffic_cfg3_keep050.json")
CSRC = os.path.join(ROOT, "paper_2506_07416_amd", "csrc")
# source file of each kernel family, for keying counter figures to the code they measured
KERNEL_SOURCES = (("attn_", "attn.hip"), ("score_", "score.hip"), ("topk_", "score.hip"),
                  ("gather_rows", "score.hip"), ("patch_select", "patch_select.hip"))


def parse():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=50)
    ap.add_argument("--warmup", type=int, default=10)
    ap.add_argument("--sets", type=int, default=4, help="rotating input sets (cold-cache)")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--settle-s", type=float, default=0.3,
                    help="seconds of untimed back-to-back steps before the timed region (clock settle)")
    ap.add_argument("--no-sweep", action="store_true")
    ap.add_argument("--keep-ratio", type=float, default=None,
                    help="keep ratio of the timed workload (default 0.5 for the 6x1024 workload, "
                         "the workload's own ratio otherwise)")
    ap.add_argument("--workload", type=int, default=3, choices=(3, 4, 5),
                    help="3: 6x1024+128 batch 1 bf16 (the reported line); 4/5: batch-8 ragged bf16/fp8, "
                         "for profiling")
    ap.add_argument("--traffic-calibrate", type=float, metavar="MB", default=None,
                    help="run only a plain fp32 copy of MB megabytes (read, and the same written) 5 times: "
                         "profiled with --pmc FETCH_SIZE and then WRITE_SIZE it calibrates the counters")
    ap.add_argument("--traffic-reduce", nargs=4, metavar=("FETCH_CSV", "WRITE_CSV", "COPY_FETCH_CSV",
                                                          "COPY_WRITE_CSV"), default=None,
                    help="reduce four rocprofv3 counter_collection.csv files (the step's FETCH_SIZE and "
                         "WRITE_SIZE runs, the calibration copy's) into per-kernel HBM bytes per launch, "
                         "written to --traffic-out")
    ap.add_argument("--copy-mb", type=float, default=256.0, help="size of the calibration copy (MB)")
    ap.add_argument("--traffic-out", default=TRAFFIC_FILE)
    return ap.parse_args()


def attn_flops(seqlens, Hq, D):
    """Algorithmic causal attention FLOPs: QK^T and PV over j <= i, 2*D*Hq*S'(S'+1) per sample."""
    return sum(2.0 * D * Hq * s * (s + 1) for s in seqlens)


def score_flops(V_b, T, Hq, D):
    """Each text-row logit once: 2*D*Hq*sum_t(V_b + t + 1)."""
    return sum(2.0 * D * Hq * (T * (v + 1) + T * (T - 1) / 2) for v in V_b)


def gather_bytes(seqlens, Hq, Hkv, D, e):
    return sum(2.0 * s * (Hq + 2 * Hkv) * D * e for s in seqlens)


def source_hash(path):
    """Hash of a kernel source together with the device headers it includes
    (every .hpp beside it), so that a change to either voids old counters."""
    h = hashlib.sha256()
    d = os.path.dirname(path)
    for p in [path] + sorted(os.path.join(d, f) for f in os.listdir(d) if f.endswith(".hpp")):
        with open(p, "rb") as f:
            h.update(f.read())
    return h.hexdigest()[:16]


def kernel_base(name):
    """'void litevlm::attn_bf16_kernel<128, true, 1>(...)' -> 'attn_bf16_kernel<128, true, 1>'."""
    n = name.split("(", 1)[0]
    if n.startswith("void "):
        n = n[5:]
    return n.split("litevlm::", 1)[1] if "litevlm::" in n else n


def kernel_source(name):
    base = kernel_base(name)
    for prefix, src in KERNEL_SOURCES:
        if base.startswith(prefix):
            return src
    return None


def max_len_bound(r, V_full, T):
    """Host bound on every compacted length at keep ratio r, known without a
    device sync: at most floor(r*V_full + 1e-6) visual tokens survive (V_b <=
    V_full) and every text token does. It sizes the attention grid."""
    return min(V_full, int(math.floor(r * V_full + 1e-6))) + T


def traffic_calibrate(mb):
    import torch
    n = int(mb * 1e6) // 4
    x = torch.ones(n, dtype=torch.float32, device="cuda")
    y = torch.empty_like(x)
    for _ in range(5):
        torch.add(x, 0.0, out=y)
    torch.cuda.synchronize()
    print(f"copy: {n * 4} bytes read and {n * 4} written per launch, 5 launches", flush=True)


def _per_dispatch(path, counter):
    """{kernel name: median over dispatches of counter (KiB)} from a rocprofv3
    counter_collection.csv (values of one dispatch summed over its rows)."""
    import csv
    from statistics import median
    vals = {}
    for r in csv.DictReader(open(path)):
        if r["Counter_Name"] != counter:
            continue
        key = (r["Kernel_Name"], r.get("Dispatch_Id") or r.get("Correlation_Id"))
        vals[key] = vals.get(key, 0.0) + float(r["Counter_Value"])
    per = {}
    for (name, _), v in vals.items():
        per.setdefault(name, []).append(v)
    return {k: (median(v), len(v)) for k, v in per.items()}


def traffic_reduce(fa, wa, fc, wc, mb, out):
    """HBM bytes per launch of every kernel in the step's counter runs: each
    counter scaled by (known bytes / measured) of the calibration copy."""
    known = int(mb * 1e6) // 4 * 4
    fetch, write = _per_dispatch(fa, "FETCH_SIZE"), _per_dispatch(wa, "WRITE_SIZE")
    cf = [v for k, v in _per_dispatch(fc, "FETCH_SIZE").items() if "_add<" in k]
    cw = [v for k, v in _per_dispatch(wc, "WRITE_SIZE").items() if "_add<" in k]
    if not cf or not cw:
        raise SystemExit("no elementwise copy dispatches in the calibration files")
    kf = known / (cf[0][0] * 1024.0)
    kw = known / (cw[0][0] * 1024.0)
    rec = {"copy_known_bytes": known, "copy_fetch_kib": cf[0][0], "copy_write_kib": cw[0][0],
           "fetch_scale": kf, "write_scale": kw, "kernels": {}}
    for name in sorted(set(fetch) & set(write)):
        src = kernel_source(name)
        if src is None:
            continue
        f_kib, n_f = fetch[name]
        w_kib, n_w = write[name]
        rec["kernels"][kernel_base(name)] = {
            "fetch_kib_per_dispatch": f_kib, "write_kib_per_dispatch": w_kib, "dispatches": [n_f, n_w],
            "hbm_bytes_per_launch": round(f_kib * 1024.0 * kf + w_kib * 1024.0 * kw),
            "source": src, "source_sha256_16": source_hash(os.path.join(CSRC, src))}
    with open(out, "w") as f:
        json.dump(rec, f, indent=1)
    print(json.dumps(rec, indent=1))


def measured_traffic(prefix):
    """HBM bytes per launch of the first kernel whose name starts with prefix,
    from the counter file, or None when absent or when its source file has
    changed since the counters were taken."""
    if not os.path.exists(TRAFFIC_FILE):
        return None
    with open(TRAFFIC_FILE) as f:
        tr = json.load(f)
    for name, k in tr.get("kernels", {}).items():
        if name.startswith(prefix):
            if k.get("source_sha256_16") == source_hash(os.path.join(CSRC, k["source"])):
                return k["hbm_bytes_per_launch"]
            return None
    return None


def host_description():
    """CPU model and NumPy's BLAS build, for the CPU baseline."""
    import numpy as np
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
        cfg = np.show_config(mode="dicts")
        b = cfg["Build Dependencies"]["blas"]
        blas = f"{b.get('name')} {b.get('version')}"
    except Exception:  # pragma: no cover
        pass
    return {"cpu_model": model, "logical_cpus": os.cpu_count(), "numpy": np.__version__, "blas": blas}


def cpu_baseline(case, r, budget_s=10.0):
    """The CPU oracle timed on the same workload: the whole step (patch
    select, scores, top-k, gather, then prefill attention over every query
    row), run back to back until about budget_s seconds of CPU work have
    accrued (at least two runs); the median run is reported."""
    import numpy as np
    import oracle
    from oracle import litevlm as O
    try:
        from threadpoolctl import threadpool_info
        cores = max([x.get("num_threads", 1) for x in threadpool_info()] or [1])
    except Exception:  # pragma: no cover
        cores = os.cpu_count() or 1
    q, k, v = oracle.decode_inputs(case)
    runs, t_begin = [], time.perf_counter()
    while len(runs) < 2 or (time.perf_counter() - t_begin < budget_s and len(runs) < 50):
        t0 = time.perf_counter()
        res = oracle.run_path(case, keep_ratio=r, attention=False)
        t_sel = time.perf_counter() - t0
        cu = res["cu_seqlens"]
        t0 = time.perf_counter()
        qc = O.gather_rows(q, res["kept_index"], cu)
        kc = O.gather_rows(k, res["kept_index"], cu)
        vc = O.gather_rows(v, res["kept_index"], cu)
        oracle.prefill_attention(qc, kc, vc, cu, case.Hq, case.Hkv, 1 / math.sqrt(case.D))
        runs.append((t_sel, time.perf_counter() - t0))
    from statistics import median
    tot = [a + b for a, b in runs]
    med = median(tot)
    t_sel = median(a for a, _ in runs)
    t_att = median(b for _, b in runs)
    return {"value": round(med * 1e3, 1), "unit": "ms", "cores": int(cores), "kind": "oracle",
            "host": host_description(),
            "sample": f"the whole step on the same inputs, {len(runs)} runs in {sum(tot):.1f} s "
                      f"(median run: selection stage {t_sel:.2f} s, gather + attention over all "
                      f"{int(res['cu_seqlens'][-1])} query rows {t_att:.2f} s)"}


def clocks_under_load(run_steps, seconds=1.0):
    """GPU clocks and socket power sampled with amd-smi (a child process) while
    `run_steps(n)` keeps the GPU busy for about `seconds`; None if amd-smi is
    unavailable or its output cannot be read."""
    import shutil
    import subprocess
    import threading
    exe = shutil.which("amd-smi") or "/opt/rocm/bin/amd-smi"
    if not os.path.exists(exe):
        return None
    box = {}

    def sample():
        time.sleep(0.25 * seconds)
        try:
            r = subprocess.run([exe, "metric", "--clock", "--power", "--json"], capture_output=True,
                               text=True, timeout=20)
            box["out"] = r.stdout
        except Exception as e:  # pragma: no cover
            box["err"] = repr(e)

    th = threading.Thread(target=sample)
    th.start()
    t0 = time.perf_counter()
    while th.is_alive() or time.perf_counter() - t0 < seconds:
        run_steps(50)
        if time.perf_counter() - t0 > 30:
            break
    th.join(timeout=30)
    try:
        txt = box["out"]
        data = json.loads(txt[txt.index("{"):])
        g = data["gpu_data"][0] if isinstance(data, dict) else data[0]
        clk = g.get("clock", {})
        gfx = [v["clk"]["value"] for k, v in sorted(clk.items()) if k.startswith("gfx") and isinstance(v, dict)
               and isinstance(v.get("clk"), dict)]
        mem = clk.get("mem_0", {}).get("clk", {}).get("value") if isinstance(clk.get("mem_0"), dict) else None
        pw = g.get("power", {}).get("socket_power", {})
        return {"gfx_mhz": gfx, "mem_mhz": mem, "socket_power_w": pw.get("value") if isinstance(pw, dict) else None,
                "note": "amd-smi metric --clock --power, sampled while the headline step runs back to back"}
    except Exception:
        return None


def main():
    args = parse()
    if args.traffic_reduce is not None:
        traffic_reduce(*args.traffic_reduce, args.copy_mb, args.traffic_out)
        return
    if args.traffic_calibrate is not None:
        traffic_calibrate(args.traffic_calibrate)
        return
    if args.gpus != 1:
        print(f"bench.py runs on exactly one GPU; --gpus {args.gpus} is not supported "
              "(the path has no multi-GPU mode in this build).", file=sys.stderr)
        sys.exit(2)
    import numpy as np
    import torch
    import paper_2506_07416_amd as lv
    import synth

    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    stream = torch.cuda.current_stream(dev)

    def up(x, dtype):
        if dtype == "bf16":
            return torch.from_numpy(np.ascontiguousarray(x).view(np.int16)).view(torch.bfloat16).to(dev)
        if dtype == "fp8":
            return torch.from_numpy(np.ascontiguousarray(x)).to(dev)
        return torch.from_numpy(np.ascontiguousarray(x, dtype=np.float32)).to(dev)

    class Runner:
        """Preallocated buffers and the calls of one select + prefill step:
        litevlm_select_score_topk (the patch selection inside the scoring call)
        then litevlm_prefill_attn, or, unfused (always with query_rows),
        litevlm_patch_select, the scoring call, then the attention."""

        def __init__(self, cases, query_rows=None, fused=None):
            self.query_rows = query_rows
            self.fused = (query_rows is None) if fused is None else fused
            self.sets = [dict(case=c, q=up(c.q, c.dtype), k=up(c.k, c.dtype), v=up(c.v, c.dtype),
                              logit=torch.from_numpy(c.view_logit).to(dev)) for c in cases]
            c = cases[0]
            self.case = c
            B, S, Hq, Hkv, D, V = c.B, c.S, c.Hq, c.Hkv, c.D, c.V_full
            t = self.sets[0]["q"].dtype
            self.outs = dict(scores=torch.empty((B, V), dtype=torch.float32, device=dev),
                             kept_index=torch.empty((B * S,), dtype=torch.int32, device=dev),
                             cu_seqlens=torch.empty((B + 1,), dtype=torch.int32, device=dev),
                             qc=torch.empty((B * S, Hq, D), dtype=t, device=dev),
                             kc=torch.empty((B * S, Hkv, D), dtype=t, device=dev),
                             vc=torch.empty((B * S, Hkv, D), dtype=t, device=dev),
                             view_keep=torch.empty((B, c.N), dtype=torch.uint8, device=dev),
                             n_visual_kept=torch.empty((B,), dtype=torch.int32, device=dev),
                             workspace=torch.empty((lv.workspace_bytes(B, S, V, Hq, Hkv, D, query_rows),),
                                                   dtype=torch.uint8, device=dev))
            self.o = torch.empty((B * S, Hq, D), dtype=torch.bfloat16, device=dev)

        def step(self, st, r, ev=None):
            c = self.case
            if ev is not None:
                ev[0].record(stream)
            if self.fused:
                lv.select_score_topk(st["logit"], c.view_offsets, st["q"], st["k"], st["v"], r, c.V_full,
                                     w_lexical=c.w_lexical, threshold=c.threshold, q_scale=c.q_scale,
                                     k_scale=c.k_scale, v_scale=c.v_scale, token_keep=False, out=self.outs)
                if ev is not None:
                    ev[1].record(stream)
            else:
                _, tk, _ = lv.patch_select(st["logit"], c.view_offsets, c.S, c.w_lexical, c.threshold)
                if ev is not None:
                    ev[1].record(stream)
                lv.token_score_topk(st["q"], st["k"], st["v"], tk, r, c.V_full, q_scale=c.q_scale,
                                    k_scale=c.k_scale, v_scale=c.v_scale, out=self.outs,
                                    query_rows=self.query_rows)
            if ev is not None:
                ev[2].record(stream)
            lv.prefill_attn(self.outs["qc"], self.outs["kc"], self.outs["vc"], self.outs["cu_seqlens"],
                            max_len_bound(r, c.V_full, c.S - c.V_full), B=c.B, q_scale=c.q_scale,
                            k_scale=c.k_scale, v_scale=c.v_scale, out=self.o)
            if ev is not None:
                ev[3].record(stream)

        def measure(self, r, steps, warmup):
            """ms per step over `steps` timed steps with no event between the
            calls (an event record between two kernels adds a gap of a few us to
            the stream), then the per-call durations from a second pass of the
            same steps with events around each call."""
            for i in range(warmup):
                self.step(self.sets[i % len(self.sets)], r)
            torch.cuda.synchronize()
            t_start = torch.cuda.Event(enable_timing=True)
            t_end = torch.cuda.Event(enable_timing=True)
            torch.cuda.synchronize()
            t_start.record(stream)
            for i in range(steps):
                self.step(self.sets[i % len(self.sets)], r)
            t_end.record(stream)
            torch.cuda.synchronize()
            total_ms = t_start.elapsed_time(t_end)
            evs = [[torch.cuda.Event(enable_timing=True) for _ in range(4)] for _ in range(steps)]
            for i in range(steps):
                self.step(self.sets[i % len(self.sets)], r, evs[i])
            torch.cuda.synchronize()
            per = np.array([[e[0].elapsed_time(e[1]), e[1].elapsed_time(e[2]), e[2].elapsed_time(e[3])]
                            for e in evs])
            self.step_pct = np.percentile(per.sum(axis=1), [10, 50, 90])
            cu = self.outs["cu_seqlens"].cpu().numpy()
            return total_ms / steps, per.mean(axis=0), cu

        def measure_graph(self, r, steps, warmup):
            """ms per step with each input set's step (its calls) captured
            once in a HIP graph and the graphs replayed in rotation."""
            graphs = []
            for st in self.sets:
                side = torch.cuda.Stream()
                side.wait_stream(torch.cuda.current_stream())
                with torch.cuda.stream(side):
                    self.step(st, r)  # first use of the capture pool and the library on this stream
                torch.cuda.current_stream().wait_stream(side)
                g = torch.cuda.CUDAGraph()
                with torch.cuda.graph(g):
                    self.step(st, r)
                graphs.append(g)
            for i in range(warmup):
                graphs[i % len(graphs)].replay()
            torch.cuda.synchronize()
            t0 = torch.cuda.Event(enable_timing=True)
            t1 = torch.cuda.Event(enable_timing=True)
            t0.record(stream)
            for i in range(steps):
                graphs[i % len(graphs)].replay()
            t1.record(stream)
            torch.cuda.synchronize()
            ms = t0.elapsed_time(t1) / steps
            del graphs
            return ms

    def call_us(rn, p):
        """Per-call durations (us) of a step from measure()'s event pairs: fused,
        the first pair is the whole select call and the second is empty."""
        if rn.fused:
            return {"patch_select_us": None, "select_call_us": round((p[0] + p[1]) * 1e3, 2),
                    "prefill_attn_us": round(p[2] * 1e3, 2)}
        return {"patch_select_us": round(p[0] * 1e3, 2), "select_call_us": round(p[1] * 1e3, 2),
                "prefill_attn_us": round(p[2] * 1e3, 2)}

    def oracle_ms(fn, budget_s=3.0):
        """Median wall time of the CPU oracle call fn() (at least one run, about
        budget_s seconds), in ms; None when the CPU baselines are skipped."""
        if args.no_cpu_baseline:
            return None
        runs, t_begin = [], time.perf_counter()
        while not runs or (time.perf_counter() - t_begin < budget_s and len(runs) < 20):
            t0 = time.perf_counter()
            fn()
            runs.append(time.perf_counter() - t0)
        return round(float(np.median(runs)) * 1e3, 2)

    def measure_decode(runner, r, label, iters=200, warmup=5):
        """One extend-one decode step (litevlm_decode_attn) per sample over the
        compacted KV cache that the runner's last step left, after a step at keep
        ratio r. The cache is cloned into enough copies to exceed the 256 MB
        last-level cache and the timed calls rotate over them (cold reads)."""
        c = runner.case
        runner.step(runner.sets[0], r)
        torch.cuda.synchronize()
        cu = runner.outs["cu_seqlens"]
        cu_h = cu.cpu().numpy()
        total = int(cu_h[-1])
        e = runner.outs["kc"].element_size()
        cache_bytes = 2 * total * c.Hkv * c.D * e
        ncopy = max(2, int(math.ceil(320e6 / max(cache_bytes, 1))))
        caches = [(runner.outs["kc"][:total].clone(), runner.outs["vc"][:total].clone())
                  for _ in range(ncopy)]
        scales = (c.q_scale, c.k_scale, c.v_scale)
        q1, k1, v1, scales = synth.decode_token_inputs(c.B, c.Hq, c.Hkv, c.D, c.dtype, seed=77,
                                                       scales=scales)
        q1_h, k1_h, v1_h = q1, k1, v1
        t = runner.outs["kc"].dtype
        q1, k1, v1 = (up(x, c.dtype) for x in (q1, k1, v1))
        ws = torch.empty((lv.decode_workspace_bytes(t, c.B, c.Hq, c.Hkv, c.D, c.S),), dtype=torch.uint8,
                         device=dev)
        o = torch.empty((c.B, c.Hq, c.D), dtype=torch.bfloat16, device=dev)

        def call(i):
            kc, vc = caches[i % ncopy]
            lv.decode_attn(q1, k1, v1, kc, vc, cu, c.S, q_scale=scales[0], k_scale=scales[1],
                           v_scale=scales[2], out=o, workspace=ws)
        # One call is a few microseconds of GPU work, less than the host needs to
        # issue it, so the calls (one per cache copy) are captured in a HIP graph
        # and the graph is replayed: the timing is the GPU's, not the host's.
        side = torch.cuda.Stream()
        side.wait_stream(torch.cuda.current_stream())
        with torch.cuda.stream(side):
            for i in range(warmup):
                call(i)
        torch.cuda.current_stream().wait_stream(side)
        g = torch.cuda.CUDAGraph()
        with torch.cuda.graph(g):
            for i in range(ncopy):
                call(i)
        reps = max(2, iters // ncopy)
        g.replay()
        torch.cuda.synchronize()
        t0 = torch.cuda.Event(enable_timing=True)
        t1 = torch.cuda.Event(enable_timing=True)
        t0.record(stream)
        for _ in range(reps):
            g.replay()
        t1.record(stream)
        torch.cuda.synchronize()
        us = t0.elapsed_time(t1) / (reps * ncopy) * 1e3
        del g
        moved = cache_bytes + c.B * (c.Hq + 2 * c.Hkv) * c.D * e + c.B * c.Hq * c.D * 2
        del caches
        torch.cuda.empty_cache()
        def dec_oracle():
            import oracle
            from oracle import litevlm as O
            cache = [runner.outs[n][:total].cpu() for n in ("kc", "vc")]
            bits = [t.view(torch.int16).numpy().view(np.uint16) if t.dtype == torch.bfloat16 else t.numpy()
                    for t in cache]
            sc = (c.q_scale, c.k_scale, c.v_scale)
            dq = O.decode_stored(q1_h, c.dtype, sc[0])
            dk, dv = O.decode_stored(k1_h, c.dtype, sc[1]), O.decode_stored(v1_h, c.dtype, sc[2])
            oracle.decode_attention(dq, dk, dv, O.decode_stored(bits[0], c.dtype, sc[1]),
                                    O.decode_stored(bits[1], c.dtype, sc[2]), cu_h, c.Hq, c.Hkv,
                                    1.0 / math.sqrt(c.D))
        cpu_ms = oracle_ms(dec_oracle)
        return {"workload": label, "dtype": c.dtype, "cache_len": np.diff(cu_h).tolist(),
                "cpu_oracle_ms": cpu_ms,
                "decode_us": round(us, 2), "cache_mb": round(cache_bytes / 1e6, 2),
                "algorithmic_mb": round(moved / 1e6, 2), "gbs": round(moved / (us * 1e-6) / 1e9, 1),
                "frac_hbm": round(moved / (us * 1e-6) / 1e9 / PEAK_HBM_GBS, 4),
                "copies_rotated": ncopy, "timing": "HIP graph of one call per cache copy, replayed"}

    def measure_tsm(cfg, label, iters=20, warmup=3):
        """The Token Selection Module front end (litevlm_tsm_qk) on the workload's
        shape with model width Hq*D: scoring keys for every token and queries for
        the text tokens from seeded bf16 hidden states, positions from the
        workload's patch selection. Events around `iters` back-to-back calls."""
        c = synth.config_case(cfg)
        Dm = c.Hq * c.D
        hid, gamma, wq, wk = synth.tsm_inputs(c.B, c.S, Dm, c.Hq, c.Hkv, c.D, seed=31)
        x = up(hid, "bf16")
        g = torch.from_numpy(gamma).to(dev)
        wq_f = lv.tsm_fold_gain(up(wq, "bf16"), g)
        wk_f = lv.tsm_fold_gain(up(wk, "bf16"), g)
        _, tk, nv = lv.patch_select(torch.from_numpy(c.view_logit).to(dev), c.view_offsets, c.S, c.w_lexical,
                                    c.threshold)
        q = torch.empty((c.B, c.S, c.Hq, c.D), dtype=torch.bfloat16, device=dev)
        k = torch.empty((c.B, c.S, c.Hkv, c.D), dtype=torch.bfloat16, device=dev)
        for _ in range(warmup):
            lv.tsm_qk(x, tk, c.V_full, wq_f, wk_f, c.Hq, c.Hkv, c.D, q=q, k=k)
        torch.cuda.synchronize()
        t0 = torch.cuda.Event(enable_timing=True)
        t1 = torch.cuda.Event(enable_timing=True)
        t0.record(stream)
        for _ in range(iters):
            lv.tsm_qk(x, tk, c.V_full, wq_f, wk_f, c.Hq, c.Hkv, c.D, q=q, k=k)
        t1.record(stream)
        torch.cuda.synchronize()
        us = t0.elapsed_time(t1) / iters * 1e3
        # the kept tokens' hidden states gathered for the LLM (selection from this q, k)
        r = HEADLINE_R if cfg == 3 else c.keep_ratio
        sel = lv.token_score_topk(q, k, None, tk, r, c.V_full, gather=False)
        hc = torch.empty((c.B * c.S, Dm), dtype=torch.bfloat16, device=dev)
        for _ in range(warmup):
            lv.gather_hidden(x, sel["kept_index"], sel["cu_seqlens"], out=hc)
        torch.cuda.synchronize()
        t0.record(stream)
        for _ in range(iters):
            lv.gather_hidden(x, sel["kept_index"], sel["cu_seqlens"], out=hc)
        t1.record(stream)
        torch.cuda.synchronize()
        g_us = t0.elapsed_time(t1) / iters * 1e3
        rows = int(sel["cu_seqlens"][-1].item())
        g_bytes = 2.0 * rows * Dm * 2
        T = c.S - c.V_full
        kept = int(nv.sum().item()) + c.B * T
        fl_alg = 2.0 * Dm * (kept * c.Hkv * c.D + c.B * T * c.Hq * c.D)
        # key rows the kernel computes: its row tiles (256 rows when that tile
        # still gives every CU a workgroup, else 128) holding at least one kept token
        mt = 256 if (c.Hkv * c.D) % 256 == 0 and c.B * ((c.S + 255) // 256) * (c.Hkv * c.D // 256) >= 256 else 128
        keep_np = tk.cpu().numpy()
        krows = sum(min(mt, c.S - r0) for bb in range(c.B) for r0 in range(0, c.S, mt)
                    if keep_np[bb, r0:r0 + mt].any())
        fl_done = 2.0 * Dm * (krows * c.Hkv * c.D + c.B * T * c.Hq * c.D)
        cpu_ms = None
        if cfg == 3:
            def tsm_oracle():
                from oracle import litevlm as O
                from oracle import tsm as OT
                keep = tk.cpu().numpy()
                OT.tsm_qk(O.decode_stored(hid, "bf16"), keep, c.V_full, gamma.astype(np.float64),
                          O.decode_stored(wq, "bf16"), O.decode_stored(wk, "bf16"), c.Hq, c.Hkv, c.D, 1e-5, 1e6)
            cpu_ms = oracle_ms(tsm_oracle, budget_s=1.0)
        return {"workload": label, "model_width": Dm, "tsm_us": round(us, 2), "cpu_oracle_ms": cpu_ms,
                "gflop_algorithmic": round(fl_alg / 1e9, 2), "gflop_computed": round(fl_done / 1e9, 2),
                "tflops": round(fl_alg / (us * 1e-6) / 1e12, 1),
                "frac_bf16_peak": round(fl_alg / (us * 1e-6) / 1e12 / PEAK_BF16_TFLOPS, 4),
                "note": "keys of the kept tokens and queries of the text tokens count as algorithmic; "
                        "the kernel skips row tiles of dropped tokens only, so a tile that mixes kept "
                        "and dropped rows is computed whole",
                "gather_hidden": {"keep_ratio": r, "rows": rows, "us": round(g_us, 2),
                                  "gbs": round(g_bytes / (g_us * 1e-6) / 1e9, 1),
                                  "frac_hbm": round(g_bytes / (g_us * 1e-6) / 1e9 / PEAK_HBM_GBS, 4)}}

    def measure_psm(B, label, T=128, d=256, H=4, dff=1024, N=6, L=4, reps=20):
        """The Patch Selection Module forward pass (litevlm_psm_forward) on seeded
        embeddings and parameters; the call's launches captured in a HIP graph and
        replayed (GPU time), and the eager call timed with events (host-bound)."""
        emb, par = synth.psm_inputs(B, T, d, dff, N, L, seed=41)
        e = torch.from_numpy(emb).to(dev)
        p = torch.from_numpy(par).to(dev)
        o = torch.empty((B, N), dtype=torch.float32, device=dev)
        ws = torch.empty((int(lv.load().litevlm_psm_workspace(B, T, d, H, dff)),), dtype=torch.uint8, device=dev)
        for _ in range(3):
            lv.psm_forward(e, p, H, dff, N, L, out=o, workspace=ws)
        torch.cuda.synchronize()
        t0 = torch.cuda.Event(enable_timing=True)
        t1 = torch.cuda.Event(enable_timing=True)
        t0.record(stream)
        for _ in range(reps):
            lv.psm_forward(e, p, H, dff, N, L, out=o, workspace=ws)
        t1.record(stream)
        torch.cuda.synchronize()
        eager_us = t0.elapsed_time(t1) / reps * 1e3
        side = torch.cuda.Stream()
        side.wait_stream(torch.cuda.current_stream())
        with torch.cuda.stream(side):
            lv.psm_forward(e, p, H, dff, N, L, out=o, workspace=ws)
        torch.cuda.current_stream().wait_stream(side)
        g = torch.cuda.CUDAGraph()
        with torch.cuda.graph(g):
            lv.psm_forward(e, p, H, dff, N, L, out=o, workspace=ws)
        g.replay()
        torch.cuda.synchronize()
        t0.record(stream)
        for _ in range(reps):
            g.replay()
        t1.record(stream)
        torch.cuda.synchronize()
        graph_us = t0.elapsed_time(t1) / reps * 1e3
        del g
        M = B * T
        fl = L * (2.0 * M * (3 * d * d + d * d + 2 * d * dff) + 4.0 * B * T * T * d) + 2.0 * M * 2 * d * d \
            + B * N * (2.0 * d * d + 4.0 * T * d)
        def psm_oracle():
            from oracle import psm as OP
            OP.psm_forward(emb.astype(np.float64), par.astype(np.float64), H, dff, N, L)
        cpu_ms = oracle_ms(psm_oracle, budget_s=2.0)
        return {"workload": label, "layers": L, "tokens": T, "width": d, "heads": H, "d_ff": dff, "views": N,
                "cpu_oracle_ms": cpu_ms,
                "graph_us": round(graph_us, 2), "eager_us": round(eager_us, 2), "gflop": round(fl / 1e9, 3),
                "tflops_graph": round(fl / (graph_us * 1e-6) / 1e12, 2),
                "note": "23 dependent launches of a small network: latency-bound, reported for completeness"}

    if args.workload == 3:
        main_runner = Runner([synth.config_case(3, run=run) for run in range(args.sets)])
    else:
        main_runner = Runner([synth.config_case(args.workload)])
    if args.keep_ratio is None:
        args.keep_ratio = HEADLINE_R if args.workload == 3 else main_runner.case.keep_ratio
    case = main_runner.case
    B, S, Hq, Hkv, D, V, T = case.B, case.S, case.Hq, case.Hkv, case.D, case.V_full, case.T
    measure = main_runner.measure

    # Clock settle: the step back to back for about 0.3 s before any timed
    # region, so the headline is taken at the GPU's steady clocks (untimed).
    t_settle = time.perf_counter()
    while time.perf_counter() - t_settle < args.settle_s:
        for i in range(20):
            main_runner.step(main_runner.sets[i % len(main_runner.sets)], args.keep_ratio)
        torch.cuda.synchronize()
    ms_step, per, cu = measure(args.keep_ratio, args.steps, args.warmup)
    step_pct = main_runner.step_pct.copy()
    ms_graph = main_runner.measure_graph(args.keep_ratio, args.steps, args.warmup)
    seqlens = np.diff(cu).tolist()
    fl = attn_flops(seqlens, Hq, D)
    attn_us = per[2] * 1e3
    attn_tflops = fl / (attn_us * 1e-6) / 1e12
    esz = {"f32": 4, "bf16": 2, "fp8": 1}[case.dtype]
    V_b = [V - len(m) * case.Tv for m in case.masked_views]
    sel_flops = score_flops(V_b, T, Hq, D)
    gbytes = gather_bytes(seqlens, Hq, Hkv, D, esz)
    # algorithmic bytes of the select call: the text query rows and the kept
    # keys read by the scoring, the token mask, the scores and packed indices
    # written, and the gather's reads and writes
    sel_bytes = (B * T * Hq * D * esz + sum(v + T for v in V_b) * Hkv * D * esz + B * S
                 + 4 * B * V + 4 * sum(seqlens) + gbytes)
    sel_us = call_us(main_runner, per)["select_call_us"]
    traffic = measured_traffic("attn_bf16_kernel")
    sel_traffic = {k: measured_traffic(k) for k in ("score_rowstats", "score_colmass", "topk_compact",
                                                    "gather_rows")}

    # the same steps with the patch selection as its own call before the scoring
    unfused = None
    if not args.no_sweep:
        rn_u = Runner([st["case"] for st in main_runner.sets], fused=False)
        m_u, p_u, _ = rn_u.measure(args.keep_ratio, args.steps, args.warmup)
        unfused = {"ms_per_step": round(m_u, 4), **call_us(rn_u, p_u),
                   "note": "litevlm_patch_select, litevlm_token_score_topk, litevlm_prefill_attn"}
        del rn_u
        torch.cuda.empty_cache()

    sweep = []
    if not args.no_sweep:
        for r in SWEEP:
            m, p, c = measure(r, max(10, args.steps // 2), 3)
            sl = np.diff(c).tolist()
            f = attn_flops(sl, Hq, D)
            sweep.append({"keep_ratio": r, "compacted_len": sl, "ms_per_step": round(m, 4),
                          **call_us(main_runner, p),
                          "attn_gflop": round(f / 1e9, 2),
                          "attn_tflops": round(f / (p[2] * 1e-3) / 1e12, 1),
                          "attn_frac_bf16_peak": round(f / (p[2] * 1e-3) / 1e12 / PEAK_BF16_TFLOPS, 4)})

    # the same batch-1 shape in E4M3 across the keep ratios (FP8 beside FP16 in
    # the prefill-latency comparison of Figure 3b)
    sweep_fp8 = []
    if not args.no_sweep:
        rn8 = Runner([synth.config_case(3, dtype="fp8")])
        for r in SWEEP:
            m, p, c = rn8.measure(r, max(10, args.steps // 2), 3)
            sl = np.diff(c).tolist()
            f = attn_flops(sl, Hq, D)
            sweep_fp8.append({"keep_ratio": r, "compacted_len": sl, "ms_per_step": round(m, 4),
                              **call_us(rn8, p),
                              "attn_gflop": round(f / 1e9, 2),
                              "attn_tflops": round(f / (p[2] * 1e-3) / 1e12, 1),
                              "attn_frac_fp8_peak": round(f / (p[2] * 1e-3) / 1e12 / PEAK_FP8_TFLOPS, 4)})
        del rn8
        torch.cuda.empty_cache()

    secondary, decode_lines, tsm_lines, psm_lines = [], [], [], []
    if not args.no_sweep:
        psm_lines.append(measure_psm(1, "text query of 128 tokens, batch 1"))
        psm_lines.append(measure_psm(8, "text query of 128 tokens, batch 8"))
        tsm_lines.append(measure_tsm(3, "6 views x 1024 + 128 text, batch 1, GQA 32/8, D=128, model width 4096"))
        tsm_lines.append(measure_tsm(4, "batch 8 ragged (0-4 of 6 views dropped per sample), same shape"))
        torch.cuda.empty_cache()
        decode_lines.append(measure_decode(main_runner, args.keep_ratio,
                                           "decode step after the prefill: the headline workload"))
        for cfg, name, qrows, rr in (
                (4, "batch 8 ragged (0-4 of 6 views masked per sample), bf16, keep ratio 0.3", None, None),
                (5, "batch 8 ragged, fp8 e4m3 Q/K/V with per-tensor scales, bf16 out, keep ratio 0.25", None, None),
                (3, "batch 1, bf16, keep ratio 0.5, scores from the last text token only "
                    "(litevlm_token_score_topk_rows, 1 query row)", 1, HEADLINE_R)):
            rn = Runner([synth.config_case(cfg)], query_rows=qrows)
            c = rn.case
            m, p, cu2 = rn.measure(c.keep_ratio if rr is None else rr, max(10, args.steps // 2), 3)
            sl = np.diff(cu2).tolist()
            f = attn_flops(sl, c.Hq, c.D)
            peak = PEAK_FP8_TFLOPS if c.dtype == "fp8" else PEAK_BF16_TFLOPS
            secondary.append({"workload": "6 views x 1024 + 128 text, GQA 32/8, D=128, " + name,
                              "dtype": c.dtype, "compacted_len": sl, "ms_per_step": round(m, 4),
                              **call_us(rn, p),
                              "attn_gflop": round(f / 1e9, 2),
                              "attn_tflops": round(f / (p[2] * 1e-3) / 1e12, 1),
                              "attn_frac_of_dtype_peak": round(f / (p[2] * 1e-3) / 1e12 / peak, 4)})
            if cfg in (4, 5):
                decode_lines.append(measure_decode(rn, c.keep_ratio, "decode step after the prefill: "
                                                   + secondary[-1]["workload"]))
            del rn
            torch.cuda.empty_cache()

    line = {
        "metric": METRIC,
        "value": round(ms_step, 4),
        "unit": "ms",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms_step, 4),
        "higher_is_better": False,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16",
        "data": "synthetic (seeded multi-camera Q/K/V, N(0,1)/sqrt(D), 5% salient keys +2.5)",
        "config": {"workload": "6 views x 1024 visual + 128 text tokens (S=6272), GQA 32/8 heads, "
                               "head dim 128, bf16, batch 1, one layer, keep ratio %.2f, no views masked"
                               % args.keep_ratio,
                   "global_batch": B, "seq_len": S, "compacted_len": seqlens,
                   "keep_ratio": args.keep_ratio, "parallelism": "none (1 GPU)",
                   "input_sets_rotated": args.sets},
        "step_ms_p10_p50_p90": {"ms": [round(float(x), 4) for x in step_pct],
                                "note": "per-step sums of the calls' event-timed durations "
                                        "(second pass; event records add small gaps)"},
        "hip_graph": {"ms_per_step": round(ms_graph, 4),
                      "note": "the same steps with each input set's calls captured in one HIP graph"},
        "prefill_attn_tflops": round(attn_tflops, 1),
        "calls_us": {**call_us(main_runner, per),
                     "note": "event-timed: litevlm_select_score_topk (view selection inside the scoring "
                             "kernels, score sweeps, top-k, gather), then litevlm_prefill_attn"},
        "unfused": unfused,
        "select_stage": {"call": "litevlm_select_score_topk (view selection, score sweeps, top-k, gather)",
                         "bound": "hbm",
                         "us": round(sel_us, 2), "algorithmic_bytes": sel_bytes,
                         "achieved": round(sel_bytes / (sel_us * 1e-6) / 1e9, 1), "peak": PEAK_HBM_GBS,
                         "unit": "GB/s", "frac": round(sel_bytes / (sel_us * 1e-6) / 1e9 / PEAK_HBM_GBS, 4),
                         "score_gflop": round(sel_flops / 1e9, 3),
                         "score_tflops_over_call": round(sel_flops / (sel_us * 1e-6) / 1e12, 1),
                         "gather_mb": round(gbytes / 1e6, 2),
                         "traffic_per_kernel": sel_traffic,
                         "note": "event-timed whole call; per-kernel durations and counters are in profiles/"},
        "roofline": {"bound": "mfma", "kernel": "attn_bf16_kernel",
                     "achieved": round(attn_tflops, 1), "peak": PEAK_BF16_TFLOPS, "unit": "TFLOP/s",
                     "frac": round(attn_tflops / PEAK_BF16_TFLOPS, 4), "traffic": traffic,
                     "flop_per_launch": fl},
        "sweep": sweep,
        "sweep_fp8": sweep_fp8,
        "secondary": secondary,
        "decode": decode_lines,
        "tsm_front_end": tsm_lines,
        "psm_forward": psm_lines,
    }
    if not args.no_sweep:
        def run_steps(n):
            for i in range(n):
                main_runner.step(main_runner.sets[i % len(main_runner.sets)], args.keep_ratio)
            torch.cuda.synchronize()
        line["gpu_clocks"] = clocks_under_load(run_steps)
    if not args.no_cpu_baseline:
        line["cpu_baseline"] = cpu_baseline(case, args.keep_ratio)
    print(json.dumps(line), flush=True)


if __name__ == "__main__":
    main()
