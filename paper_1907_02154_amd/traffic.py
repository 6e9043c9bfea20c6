"""HBM traffic per kernel launch from rocprofv3 counter runs.

Usage (on a machine with the GPU, after four counter runs, see below):

    python -m paper_1907_02154_amd.traffic --fetch DIR --write DIR \
        --copy-fetch DIR --copy-write DIR [--copy-bytes N] > traffic.txt

Each DIR is a ``rocprofv3 --pmc <counter> --kernel-trace -f csv -d DIR -o run``
output directory: FETCH_SIZE and WRITE_SIZE (KiB per dispatch) of the
workload, and the same two counters for a plain device-to-device copy of a
known size (``bench.py --copy-calibration``).  The copy calibrates what the
counters read per byte actually moved: scale = copy bytes / counter bytes.

Output: one tab-separated line per kernel name (template arguments kept,
namespaces and argument list dropped), giving the mean calibrated bytes read
and written per dispatch, the scales, the dispatch count, and the SHA-1 of the
HIP source that defines the kernel, so a reader can tell when the numbers no
longer describe the code.

    python -m paper_1907_02154_amd.traffic --counters DIR [DIR ...] [--match TEXT]

prints, for every kernel whose name contains TEXT, the mean per dispatch of
every counter found in the given counter-run directories (any counters), with
the dispatch count and the source SHA-1.
"""
from __future__ import annotations

import argparse
import csv
import glob
import hashlib
import os
import re
import sys
from collections import defaultdict

CSRC = os.path.join(os.path.dirname(os.path.abspath(__file__)), "csrc")

# kernel name prefix -> the source file that defines it
SOURCES = {
    "igemm_wave_f32_kernel": "conv_wave_f32.hip",
    "igemm_wave_f32_gen_kernel": "conv_wave_f32.hip",
    "igemm_wave_f32_kcrs_kernel": "conv_wave_f32.hip",
    "igemm_bf16_dma_res_kernel": "conv_nhwc_bf16.hip",
    "igemm_bf16_dma_cl_kernel": "conv_nhwc_bf16.hip",
    "igemm_bf16_halo_res_kernel": "conv_nhwc_bf16.hip",
    "igemm_bf16_halo_cl_kernel": "conv_nhwc_bf16.hip",
    "splitk_reduce_cl_kernel": "conv_igemm_f32.hip",
    "maxpool_nhwc_bf16_kernel": "glue.hip",
    "maxpool_kernel": "glue.hip",
    "igemm_f32_kernel": "conv_igemm_f32.hip",
    "splitk_reduce_kernel": "conv_igemm_f32.hip",
    "igemm_bf16_kernel": "conv_igemm_bf16.hip",
    "igemm_bf16_nhwc_kernel": "conv_nhwc_bf16.hip",
    "igemm_bf16_dma_kernel": "conv_nhwc_bf16.hip",
    "igemm_bf16_halo_kernel": "conv_nhwc_bf16.hip",
    "nchw_to_nhwc_bf16_kernel": "conv_nhwc_bf16.hip",
    "nchw_to_nhwc_plane_bf16_kernel": "conv_nhwc_bf16.hip",
    "dw_run_kernel": "dwconv.hip",
    "dw_band_kernel": "dwconv.hip",
    "dw3x3_kernel": "dwconv.hip",
    "dw_generic_kernel": "dwconv.hip",
    "conv_direct_kernel": "conv_direct.hip",
    "pack_krsc_kernel": "pack.hip",
    "pack_wave_kernel": "pack.hip",
    "stem7_bf16_kernel": "conv_stem_bf16.hip",
    "pack_stem_kernel": "conv_stem_bf16.hip",
}


def short_name(full: str) -> str:
    """'void miconv::(anonymous namespace)::k<1, 2>(miconv::ConvArgs)' -> 'k<1, 2>'."""
    s = full.strip()
    if s.startswith("void "):
        s = s[5:]
    depth, cut = 0, len(s)
    for i, ch in enumerate(s):          # drop the argument list: first '(' outside <...>
        if ch == "<":
            depth += 1
        elif ch == ">":
            depth -= 1
        elif ch == "(" and depth == 0 and i > 0 and s[i - 1] != ":":
            cut = i
            break
    s = s[:cut]
    head = s.split("<", 1)
    base = head[0].split("::")[-1]
    return base + ("<" + head[1] if len(head) > 1 else "")


def source_sha(name: str) -> str:
    base = name.split("<", 1)[0]
    src = SOURCES.get(base)
    if not src:
        return "-"
    with open(os.path.join(CSRC, src), "rb") as f:
        return hashlib.sha1(f.read()).hexdigest()[:12]


def read_counter(d: str, counter: str):
    """{kernel short name: [KiB per dispatch, ...]} from one counter run."""
    out = defaultdict(list)
    files = glob.glob(os.path.join(d, "**", "*counter_collection.csv"), recursive=True)
    if not files:
        sys.exit(f"no counter_collection.csv under {d}")
    for p in files:
        with open(p) as f:
            for r in csv.DictReader(f):
                if r["Counter_Name"] != counter:
                    continue
                out[short_name(r["Kernel_Name"])].append(float(r["Counter_Value"]))
    return out


def calibration(d: str, counter: str, nbytes: int) -> float:
    vals = read_counter(d, counter)
    # the copy's kernel: the one whose single dispatch moved the most
    name, v = max(vals.items(), key=lambda kv: max(kv[1]))
    return nbytes / (max(v) * 1024.0)


def counter_means(dirs, match: str):
    """{kernel: {counter: mean per dispatch}} and {kernel: dispatches} over counter runs."""
    vals = defaultdict(lambda: defaultdict(list))
    for d in dirs:
        files = glob.glob(os.path.join(d, "**", "*counter_collection.csv"), recursive=True)
        if not files:
            sys.exit(f"no counter_collection.csv under {d}")
        for p in files:
            with open(p) as f:
                for r in csv.DictReader(f):
                    name = short_name(r["Kernel_Name"])
                    if match in name:
                        vals[name][r["Counter_Name"]].append(float(r["Counter_Value"]))
    means = {k: {c: sum(v) / len(v) for c, v in cs.items()} for k, cs in vals.items()}
    counts = {k: max(len(v) for v in cs.values()) for k, cs in vals.items()}
    return means, counts


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--counters", nargs="+")
    ap.add_argument("--match", default="")
    ap.add_argument("--fetch")
    ap.add_argument("--write")
    ap.add_argument("--copy-fetch")
    ap.add_argument("--copy-write")
    ap.add_argument("--copy-bytes", type=int, default=256 << 20)
    a = ap.parse_args()
    if a.counters:
        means, counts = counter_means(a.counters, a.match)
        for name in sorted(means):
            print(f"{name}\tsource_sha1 {source_sha(name)}\tdispatches {counts[name]}")
            for c in sorted(means[name]):
                print(f"\t{c}\t{means[name][c]:.1f}")
        return
    if not (a.fetch and a.write and a.copy_fetch and a.copy_write):
        ap.error("--fetch, --write, --copy-fetch and --copy-write are required without --counters")
    sf = calibration(a.copy_fetch, "FETCH_SIZE", a.copy_bytes)
    sw = calibration(a.copy_write, "WRITE_SIZE", a.copy_bytes)
    fetch = read_counter(a.fetch, "FETCH_SIZE")
    write = read_counter(a.write, "WRITE_SIZE")
    print("# kernel\tsource_sha1\tfetch_bytes_per_launch\twrite_bytes_per_launch\tfetch_scale\twrite_scale"
          "\tdispatches")
    for name in sorted(set(fetch) & set(write)):
        fv, wv = fetch[name], write[name]
        fb = sum(fv) / len(fv) * 1024.0 * sf
        wb = sum(wv) / len(wv) * 1024.0 * sw
        print(f"{name}\t{source_sha(name)}\t{fb:.0f}\t{wb:.0f}\t{sf:.4f}\t{sw:.4f}\t{len(fv)}")


if __name__ == "__main__":
    main()
