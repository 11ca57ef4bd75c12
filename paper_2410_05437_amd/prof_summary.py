"""Text summaries of rocprofv3 outputs of bench.py (written to profiles/).

    python -m paper_2410_05437_amd.prof_summary stats TRACE_CSV OUT_MD CMD [--steps S --warmup W]
    python -m paper_2410_05437_amd.prof_summary traffic FETCH_CSV WRITE_CSV OUT_MD CMD_FETCH CMD_WRITE

`stats` reads a `--kernel-trace --output-format csv` trace and tabulates
launches per kernel and grid; the 256x256 GEMM launches that serve both the
expand GEMM and the dense baseline are split by their place in bench.py's
launch order.  `traffic` reads two `--pmc FETCH_SIZE` / `--pmc WRITE_SIZE`
runs of `bench.py --kernel-probe` and scales the expand GEMM's counters by
what the same counters read for the 1 GiB elementwise copy of that run.
"""
import argparse
import collections
import csv
import os
import sys

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
EXPAND_KERNEL = "gemm_tn_bf16_v3_kernel<0, 256>"   # the four-wave 256x256 kernel, bf16 output
EXPAND_GRID = 256 * 256                        # one workgroup of 256 threads per CU
COPY_KERNELS = ("AUnaryFunctor<c10::BFloat16", "MulFunctor")   # torch.mul(bf16, 1.0)
COPY_BYTES = 1 << 30


def _short(name):
    return name.replace("espace::(anonymous namespace)::", "").split("(unsigned")[0].split("(float")[0]


def _dur_us(r):
    return (int(r["End_Timestamp"]) - int(r["Start_Timestamp"])) / 1e3


def stats(args):
    rows = sorted(csv.DictReader(open(args.trace)), key=lambda r: int(r["Start_Timestamp"]))
    groups = collections.defaultdict(list)
    for r in rows:
        grid = f'{r["Grid_Size_X"]} x {r.get("Grid_Size_Y", "1")}'
        groups[(_short(r["Kernel_Name"]), grid)].append(_dur_us(r))
    lines = ["# Kernel statistics: projected linear, Llama2-7B fused QKV "
             "(K=4096, M=12288, L=1536, N=4096), bf16", "",
             "Command (from the repository root, on one MI355X):", "", "```", args.cmd, "```", "",
             "Per launch shape (grid in threads x split), durations from the kernel trace:", "",
             "| kernel | grid | launches | average (us) | median (us) |", "|---|---|---|---|---|"]
    other = [0, 0.0]
    for (k, grid), v in sorted(groups.items(), key=lambda kv: -sum(kv[1])):
        if "espace" not in k and "gemm_tn" not in k and "skinny" not in k and "splitk" not in k:
            other[0] += len(v)
            other[1] += sum(v)
            continue
        v = sorted(v)
        lines.append(f"| `{k}` | {grid} | {len(v)} | {sum(v) / len(v):.1f} | {v[len(v) // 2]:.1f} |")
    lines.append(f"| other kernels (input generation, torch copies) | | {other[0]} | "
                 f"{other[1] / max(other[0], 1):.1f} | |")
    big = [r for r in rows if EXPAND_KERNEL in r["Kernel_Name"] and int(r["Grid_Size_X"]) == EXPAND_GRID]
    W, S = args.warmup, args.steps
    seg = [("expand, inside the timed projected-linear steps", big[:W + S]),
           ("expand, back-to-back loop (the roofline kernel; 2 warm-up launches)", big[W + S + 2:W + 2 * S + 2]),
           ("dense baseline", big[W + 2 * S + 2:2 * W + 3 * S + 2])]
    lines += ["", "The 256x256 kernel (one workgroup per CU, 768 tiles) serves both the expand GEMM "
              "(depth L=1536) and the dense baseline (depth K=4096); split by position in bench.py's "
              "launch order:", "", "| launches | count | average (us) | median (us) |",
              "|---|---|---|---|"]
    for name, rs in seg:
        d = sorted(_dur_us(r) for r in rs)
        if d:
            lines.append(f"| {name} | {len(d)} | {sum(d) / len(d):.1f} | {d[len(d) // 2]:.1f} |")
    # decode at N = 1 (Llama2-7B FFN up+gate, K=4096, M=22016, L=1536): each
    # kernel streams one weight-sized operand once; identified by template and grid
    dec = [("projection: Pt, 1536 x 4096", "gemv_tn_bf16_kernel<1, 8>", "98304 x 1", 1536 * 4096 * 2),
           ("expansion: Wf, 22016 x 1536", "gemv_rows_bf16_kernel<1, 3, 2>", "704512 x 1", 22016 * 1536 * 2),
           ("dense: W, 22016 x 4096", "gemv_tn_bf16_kernel<1, 8>", "1409024 x 1", 22016 * 4096 * 2)]
    lines += ["", "Decode kernels at N = 1 (Llama2-7B FFN up+gate), bytes of the streamed operand over the "
              "median duration:", "", "| kernel | streamed bytes | median (us) | GB/s | HBM fraction (8 TB/s) |",
              "|---|---|---|---|---|"]
    for name, k, grid, nbytes in dec:
        v = sorted(d for (gk, gg), ds in groups.items() if gk.endswith(k) and gg == grid for d in ds)
        if v:
            med = v[len(v) // 2]
            lines.append(f"| {name} | {nbytes} | {med:.1f} | {nbytes / med / 1e3:.0f} | "
                         f"{nbytes / med / 1e3 / 8000:.2f} |")
    open(args.out, "w").write("\n".join(lines) + "\n")
    print("\n".join(lines))


def _counter(path, counter):
    """{(kernel name, dispatch id): value} for one counter of a pmc run."""
    vals = {}
    for r in csv.DictReader(open(path)):
        if r["Counter_Name"] != counter:
            continue
        vals[(r["Kernel_Name"], r["Dispatch_Id"], int(r["Grid_Size"]))] = float(r["Counter_Value"])
    return vals


def _select(vals, pred):
    return [v for (name, _, grid), v in vals.items() if pred(name, grid)]


def traffic(args):
    sys.path.insert(0, ROOT)
    import bench                                    # the source hash bench.py checks
    from paper_2410_05437_amd import accounting as acc
    res = {}
    for counter, path in (("FETCH_SIZE", args.fetch), ("WRITE_SIZE", args.write)):
        vals = _counter(path, counter)
        exp = _select(vals, lambda n, g: EXPAND_KERNEL in n and g == EXPAND_GRID)
        cpy = _select(vals, lambda n, g: all(k in n for k in COPY_KERNELS))
        if not exp or len(cpy) != 1:
            raise SystemExit(f"{counter}: expected expand launches and one copy, found {len(exp)} / {len(cpy)}")
        scale = (COPY_BYTES / 1024.0) / cpy[0]     # counters are in KiB
        res[counter] = {"expand_kib": sum(exp) / len(exp), "copy_kib": cpy[0], "scale": scale,
                        "launches": len(exp),
                        "bytes": sum(exp) / len(exp) * scale * 1024.0}
    total = res["FETCH_SIZE"]["bytes"] + res["WRITE_SIZE"]["bytes"]
    alg = acc.gemm_bytes(4096, 12288, 1536)
    lines = ["# HBM traffic: expand GEMM of the Llama2-7B fused QKV layer "
             "(R=N=4096, Cc=M=12288, D=L=1536), bf16", "",
             "Counter runs (from the repository root, on one MI355X), one counter block per run:", "",
             "```", args.cmd_fetch, args.cmd_write, "```", "",
             "Each run launches one elementwise copy of 1 GiB (reads 1 GiB, writes 1 GiB) and then "
             "the expand GEMM; each counter is scaled by the copy's known size over what the same "
             "counter reads for it.", "",
             "| counter | expand launches | expand (KiB/launch) | copy (KiB) | scale | scaled bytes/launch |",
             "|---|---|---|---|---|---|"]
    for c in ("FETCH_SIZE", "WRITE_SIZE"):
        r = res[c]
        lines.append(f"| {c} | {r['launches']} | {r['expand_kib']:.0f} | {r['copy_kib']:.0f} | "
                     f"{r['scale']:.4f} | {r['bytes']:.0f} |")
    lines += ["", f"- hbm_bytes_per_launch: {total:.0f}",
              f"- algorithmic_bytes_per_launch: {alg}",
              f"- ratio_to_algorithmic: {total / alg:.3f}",
              f"- source_sha256: `{bench.traffic_sources()}`", "",
              "Algorithmic bytes: 2·(R·D + Cc·D + R·Cc), each operand read once and the output "
              "written once. bench.py reports `roofline.traffic` from this file only while the "
              "hash of the GEMM kernel, its headers and the tile planner matches."]
    open(args.out, "w").write("\n".join(lines) + "\n")
    print("\n".join(lines))


def main():
    ap = argparse.ArgumentParser()
    sub = ap.add_subparsers(dest="mode", required=True)
    a = sub.add_parser("stats")
    a.add_argument("trace")
    a.add_argument("out")
    a.add_argument("cmd")
    a.add_argument("--steps", type=int, default=50)
    a.add_argument("--warmup", type=int, default=10)
    b = sub.add_parser("traffic")
    b.add_argument("fetch")
    b.add_argument("write")
    b.add_argument("out")
    b.add_argument("cmd_fetch")
    b.add_argument("cmd_write")
    args = ap.parse_args()
    stats(args) if args.mode == "stats" else traffic(args)


if __name__ == "__main__":
    main()
