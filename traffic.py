"""HBM traffic of the attention kernel from rocprofv3 counters, for bench.py's
roofline object.

Two modes:
  python traffic.py copy MB
      runs a plain elementwise copy (y = x + 0, fp32, MB megabytes read and the
      same written) a few times; profiled with --pmc FETCH_SIZE and then
      WRITE_SIZE it calibrates the counters against a known byte count.
  python traffic.py reduce FETCH_ATTN WRITE_ATTN FETCH_COPY WRITE_COPY MB
      reads the four counter_collection.csv files (attention runs of bench.py,
      copy runs of this script), scales each attention counter by the copy's
      known bytes / measured bytes, and writes profiles/attn_bf16_cfg3_traffic.json
      (keyed to a hash of attn.hip, so a changed kernel reads as unmeasured) plus
      a short summary on stdout.
"""
import csv
import json
import os
import re
import sys

ROOT = os.path.dirname(os.path.abspath(__file__))
OUT = os.path.join(ROOT, "profiles", "attn_bf16_cfg3_traffic.json")


def run_copy(mb):
    import torch
    n = int(mb * 1e6) // 4
    x = torch.ones(n, dtype=torch.float32, device="cuda")
    y = torch.empty_like(x)
    for _ in range(5):
        torch.add(x, 0.0, out=y)
    torch.cuda.synchronize()
    print(f"copy {n * 4} bytes read and written per launch, 5 launches", flush=True)


def per_dispatch(path, pattern, counter):
    vals = {}
    for r in csv.DictReader(open(path)):
        if r["Counter_Name"] != counter or not re.search(pattern, r["Kernel_Name"]):
            continue
        key = r.get("Dispatch_Id") or r.get("Correlation_Id")
        vals[key] = vals.get(key, 0.0) + float(r["Counter_Value"])
    if not vals:
        raise SystemExit(f"no {counter} rows for /{pattern}/ in {path}")
    v = sorted(vals.values())
    return v[len(v) // 2], len(v)   # median over dispatches, KiB


def reduce(fa, wa, fc, wc, mb):
    sys.path.insert(0, ROOT)
    from bench import source_hash
    known = int(mb * 1e6) // 4 * 4
    f_attn, n_fa = per_dispatch(fa, r"attn_bf16_kernel", "FETCH_SIZE")
    w_attn, n_wa = per_dispatch(wa, r"attn_bf16_kernel", "WRITE_SIZE")
    f_copy, _ = per_dispatch(fc, r"elementwise", "FETCH_SIZE")
    w_copy, _ = per_dispatch(wc, r"elementwise", "WRITE_SIZE")
    kf = known / (f_copy * 1024.0)
    kw = known / (w_copy * 1024.0)
    fetch = f_attn * 1024.0 * kf
    write = w_attn * 1024.0 * kw
    rec = {"kernel": "attn_bf16_kernel<128, true, 1>",
           "workload": "6x1024+128, GQA 32/8, D=128, bf16, batch 1, keep ratio 0.5 (3200 tokens)",
           "fetch_kib_per_dispatch": f_attn, "write_kib_per_dispatch": w_attn,
           "copy_known_bytes": known, "copy_fetch_kib": f_copy, "copy_write_kib": w_copy,
           "fetch_scale": kf, "write_scale": kw,
           "hbm_bytes_per_launch": round(fetch + write),
           "source_sha256_16": source_hash(os.path.join(ROOT, "paper_2506_07416_amd", "csrc", "attn.hip"))}
    with open(OUT, "w") as f:
        json.dump(rec, f, indent=1)
    print(json.dumps(rec, indent=1))


if __name__ == "__main__":
    if sys.argv[1] == "copy":
        run_copy(float(sys.argv[2]))
    else:
        reduce(*sys.argv[2:6], float(sys.argv[6]))
