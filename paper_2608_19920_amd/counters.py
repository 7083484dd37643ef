"""HBM traffic of the hot kernels from rocprofv3 counter runs.

Two sub-commands:

``run WHAT`` launches one kind of work eagerly, a few times, so that a
``rocprofv3 --pmc FETCH_SIZE`` (or ``WRITE_SIZE``) pass records it per
dispatch:

    decode   one token step (h2o_chunk_step, B8 Hq32 Hkv8 d64 M4096, bf16) on
             each of 8 layer states, 3 times over, so every launch streams
             its cache from HBM
    prefill  the chunk step (attention, accumulate, evict, insert) of one
             chunked-prefill workload (bf16)
    copy     a plain device-to-device copy of 1 GiB, the calibration: its
             algorithmic traffic is exactly 1 GiB read and 1 GiB written

``reduce`` reads the counter CSVs of those runs, scales each kernel's mean
FETCH_SIZE and WRITE_SIZE per dispatch by the copy's factor (known bytes /
counted bytes, one factor per counter), and writes the bytes per launch,
with a hash of the kernel's source so stale figures are not used, to a JSON
file.
"""
from __future__ import annotations

import argparse
import csv
import glob
import hashlib
import json
import os
import sys

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(HERE)
COPY_BYTES = 1 << 30
# kernel label -> (substring of the rocprofv3 kernel name, sources it is built from)
KERNELS = {
    "decode_split": ("decode_split<", ["decode.hip"]),
    "decode_finish": ("decode_finish<", ["decode.hip"]),
    "mfma_lse": ("lse_pass<", ["sdpa_mfma.hip"]),
    "mfma_main": ("main_pass<", ["sdpa_mfma.hip"]),
    "split_reduce": ("split_reduce<", ["sdpa_mfma.hip"]),
    "colsum_reduce": ("colsum_reduce_kernel", ["select.hip"]),
    "bottomk": ("bottomk_kernel<", ["select.hip"]),
    "bottomk_insert": ("bottomk_insert_kernel<", ["select.hip"]),
    "insert": ("::insert_kernel(", ["select.hip"]),
}


def src_hash(names) -> str:
    h = hashlib.sha256()
    for n in names:
        with open(os.path.join(HERE, "csrc", n), "rb") as f:
            h.update(f.read())
    return h.hexdigest()[:16]


def _run(what: str, workload: str) -> None:
    import numpy as np
    import torch

    sys.path.insert(0, ROOT)
    from paper_2608_19920_amd import h2o as H
    from paper_2608_19920_amd import workloads as W

    bf = torch.bfloat16
    to = lambda a, dt=bf: torch.from_numpy(np.ascontiguousarray(a)).to("cuda").to(dt)
    if what == "copy":
        src = torch.ones(COPY_BYTES // 2, dtype=bf, device="cuda")
        dst = torch.empty_like(src)
        torch.cuda.synchronize()
        for _ in range(4):
            dst.copy_(src)
        torch.cuda.synchronize()
        print(f"copy: 4 x {COPY_BYTES} bytes", flush=True)
        return
    w = W.WORKLOADS[workload]
    layers = 8 if what == "decode" else 1
    states = []
    for layer in range(layers):
        x = W.make_inputs(w, seed=layer)
        st = dict(k_cache=to(x["k_cache"]), v_cache=to(x["v_cache"]),
                  scores=to(x["scores"], torch.float32),
                  token_pos=to(x["token_pos"], torch.int32))
        qs = x["q_steps"][0] if "q_steps" in x else x["q"]
        ks = x["k_new_steps"][0] if "k_new_steps" in x else x["k_new"]
        vs = x["v_new_steps"][0] if "v_new_steps" in x else x["v_new"]
        states.append((st, to(qs), to(ks), to(vs), int(x["pos0"]), float(x["scale"]),
                       H.alloc_step(w.B, w.Hq, w.Hkv, w.T, w.M, w.d, bf)))
        del x
    torch.cuda.synchronize()
    for _ in range(3 if what == "decode" else 2):
        for st, q, kn, vn, pos0, scale, bufs in states:
            H.step(st, q, kn, vn, bufs, pos0, scale)
    torch.cuda.synchronize()
    print(f"{what} {w.describe()}: done", flush=True)


def _read(dir_: str, counter: str):
    """{kernel name: [per-dispatch counter values]} from a rocprofv3 CSV run."""
    paths = glob.glob(os.path.join(dir_, "**", "*counter_collection.csv"), recursive=True)
    if not paths:
        raise SystemExit(f"no counter_collection.csv under {dir_}")
    per = {}
    for p in paths:
        with open(p) as f:
            for r in csv.DictReader(f):
                if r["Counter_Name"] != counter:
                    continue
                key = (r["Kernel_Name"], r.get("Dispatch_Id", ""))
                per[key] = per.get(key, 0.0) + float(r["Counter_Value"])
    out = {}
    for (name, _), v in per.items():
        out.setdefault(name, []).append(v)
    return out


def _mean_for(table, needle: str):
    vals = [v for name, vs in table.items() if needle in name for v in vs]
    return (sum(vals) / len(vals), len(vals)) if vals else (None, 0)


def _reduce(a) -> None:
    cf, cw = _read(a.copy_fetch, "FETCH_SIZE"), _read(a.copy_write, "WRITE_SIZE")
    # the copy is the only kernel with a 1 GiB footprint: take the largest dispatches
    copy_f = max(v for vs in cf.values() for v in vs)
    copy_w = max(v for vs in cw.values() for v in vs)
    f_fetch = COPY_BYTES / (copy_f * 1024.0)
    f_write = COPY_BYTES / (copy_w * 1024.0)
    rec = {"_calibration": {"copy_bytes": COPY_BYTES, "fetch_kib": copy_f,
                            "write_kib": copy_w, "fetch_factor": round(f_fetch, 4),
                            "write_factor": round(f_write, 4)}}
    if os.path.exists(a.out):
        with open(a.out) as f:
            old = json.load(f)
        rec.update({k: v for k, v in old.items() if not k.startswith("_")})
    for run in a.runs:
        workload, fdir, wdir = run.split(":")
        tf, tw = _read(fdir, "FETCH_SIZE"), _read(wdir, "WRITE_SIZE")
        for label, (needle, srcs) in KERNELS.items():
            mf, nf = _mean_for(tf, needle)
            mw, nw = _mean_for(tw, needle)
            if mf is None or mw is None:
                continue
            fb, wb = mf * 1024.0 * f_fetch, mw * 1024.0 * f_write
            rec[f"{label}@{workload}"] = {
                "fetch_kib": round(mf, 1), "write_kib": round(mw, 1),
                "dispatches": [nf, nw], "read_bytes": round(fb), "write_bytes": round(wb),
                "bytes_per_launch": round(fb + wb), "src_hash": src_hash(srcs)}
            print(f"{label}@{workload}: read {fb / 1e6:.2f} MB, write {wb / 1e6:.2f} MB "
                  f"per launch ({nf} dispatches)")
    with open(a.out, "w") as f:
        json.dump(rec, f, indent=1, sort_keys=True)
        f.write("\n")
    print(f"fetch factor {f_fetch:.4f}, write factor {f_write:.4f} -> {a.out}")


def main() -> None:
    ap = argparse.ArgumentParser(description=__doc__,
                                 formatter_class=argparse.RawDescriptionHelpFormatter)
    sub = ap.add_subparsers(dest="cmd", required=True)
    r = sub.add_parser("run")
    r.add_argument("what", choices=["decode", "prefill", "copy"])
    r.add_argument("--workload", default=None)
    d = sub.add_parser("reduce")
    d.add_argument("--copy-fetch", required=True)
    d.add_argument("--copy-write", required=True)
    d.add_argument("--out", default=os.path.join(ROOT, "profiles", "traffic.json"))
    d.add_argument("runs", nargs="+", help="WORKLOAD:FETCH_DIR:WRITE_DIR")
    a = ap.parse_args()
    if a.cmd == "run":
        _run(a.what, a.workload or ("decode_bf16" if a.what == "decode" else "prefill_bf16"))
    else:
        _reduce(a)


if __name__ == "__main__":
    main()
