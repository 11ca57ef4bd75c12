"""Text summaries of rocprofv3 outputs of bench.py (written to profiles/).

    python profile_summary.py stats TRACE_CSV OUT_MD CMD [--steps S --warmup W]
    python profile_summary.py traffic FETCH_CSV WRITE_CSV OUT_MD CMD_FETCH CMD_WRITE
    python profile_summary.py counters OUT_MD --run CSV CMD [--run CSV CMD ...]
    python profile_summary.py loadpath OUT_MD --run CSV CMD [--run CSV CMD ...]

`stats` reads a `--kernel-trace --output-format csv` trace and tabulates
launches per kernel and grid; the 256x256 GEMM launches that serve both the
expand GEMM and the dense baseline are split by their place in bench.py's
launch order.  `traffic` reads two `--pmc FETCH_SIZE` / `--pmc WRITE_SIZE`
runs of `bench.py --kernel-probe` and scales the expand GEMM's counters by
what the same counters read for the 1 GiB elementwise copy of that run.
`counters` reads any number of `--pmc` runs of `bench.py --kernel-probe`,
splits each run's dispatches into the probe's phases at its marker kernels
and tabulates every counter per phase and kernel, with the MFMA busy ratio,
the MFMA flops against the algorithmic flops, and the byte counters scaled
by the copy calibration.  `loadpath` reads `--pmc` runs of the same probe
with the memory-pipeline counters and tabulates, for the tiled GEMMs, how
busy and how stalled the load path of the CUs (TA, TD, TCP) and the L2
channels were, the share of wave time spent in s_waitcnt, and the L2
requests against the operand bytes the tiles read.
"""
import argparse
import collections
import csv
import os
import sys

ROOT = os.path.dirname(os.path.abspath(__file__))
EXPAND_KERNEL = "gemm_tn_bf16_v3_kernel<0, 256, 0>"   # the four-wave 256x256 kernel, bf16 output, plain A
PROJECT_KERNEL = "gemm_tn_bf16_v2_kernel<128, 192"   # the projection's 128x192 tile
EXPAND_GRID = 256 * 256                        # one workgroup of 256 threads per CU
COPY_KERNELS = ("AUnaryFunctor<c10::BFloat16", "MulFunctor")   # torch.mul(bf16, 1.0)
COPY_BYTES = 1 << 30
OWN = ("gemm_tn", "skinny_tn", "gemv_", "splitk_reduce", "espace::")


def _short(name):
    return (name.replace("espace::(anonymous namespace)::", "").split("(unsigned")[0].split("(float")[0]
            .split("(espace::")[0])


def _own(name):
    """A kernel of this library (namespace espace), not torch's."""
    return "espace::" in name


def _dur_us(r):
    return (int(r["End_Timestamp"]) - int(r["Start_Timestamp"])) / 1e3


def stats(args):
    rows = sorted(csv.DictReader(open(args.trace)), key=lambda r: int(r["Start_Timestamp"]))
    groups = collections.defaultdict(list)
    for r in rows:
        grid = f'{r["Grid_Size_X"]} x {r.get("Grid_Size_Y", "1")}'
        groups[(_short(r["Kernel_Name"]), grid, _own(r["Kernel_Name"]))].append(_dur_us(r))
    lines = ["# Kernel statistics: projected linear, Llama2-7B fused QKV "
             "(K=4096, M=12288, L=1536, N=4096), bf16", "",
             "Command (from the repository root, on one MI355X):", "", "```", args.cmd, "```", "",
             "Per launch shape (grid in threads x split), durations from the kernel trace:", "",
             "| kernel | grid | launches | average (us) | median (us) |", "|---|---|---|---|---|"]
    other = [0, 0.0]
    for (k, grid, own), v in sorted(groups.items(), key=lambda kv: -sum(kv[1])):
        if not own:
            other[0] += len(v)
            other[1] += sum(v)
            continue
        v = sorted(v)
        lines.append(f"| `{k}` | {grid} | {len(v)} | {sum(v) / len(v):.1f} | {v[len(v) // 2]:.1f} |")
    lines.append(f"| other kernels (input generation, torch copies) | | {other[0]} | "
                 f"{other[1] / max(other[0], 1):.1f} | |")
    # bench.py's launch order: the layer (project, expand) for the cold timed
    # region, the clock warm-up and the headline timed region (W + S calls
    # each, the warm-up a variable number), then the projection alone and the
    # expansion alone (2 + S launches each), then the dense baseline (W + S)
    own = [r for r in rows if any(k in r["Kernel_Name"] for k in OWN)]
    is_p = [PROJECT_KERNEL in r["Kernel_Name"] for r in own]
    W, S = args.warmup, args.steps
    pb = next(i for i in range(len(own)) if all(is_p[i:i + 2 + S]))      # the projection's own loop
    pe = pb + 2 + S
    layer = own[pb - 2 * S:pb]                                           # headline: S (project, expand) pairs
    p0 = is_p.index(True)                                                # the first layer call (after the fold)
    cold = own[p0 + 2 * W:p0 + 2 * (W + S)]
    seg = [("projection, inside the cold timed region (straight after set-up)", cold[0::2]),
           ("projection, inside the headline timed region (after the clock warm-up)", layer[0::2]),
           ("projection, back-to-back loop", own[pb + 2:pe]),
           ("expand, inside the cold timed region", cold[1::2]),
           ("expand, inside the headline timed region", layer[1::2]),
           ("expand, back-to-back loop (the roofline kernel)", own[pe + 2:pe + 2 + S]),
           ("dense baseline", own[pe + 2 + S + W:pe + 2 + 2 * S + W])]
    lines += ["", "The projection (128x192 tiles) and the 256x256 kernel (one workgroup per CU, 768 "
              "tiles: inside the layer the expand GEMM, depth L=1536, on Z in the workspace's row-pair "
              "layout, `<0, 256, 1>`; the back-to-back expand GEMM on a plain Z and the dense baseline, "
              "depth K=4096, `<0, 256, 0>`), split by position in bench.py's launch order (timed "
              "launches only):", "",
              "| launches | count | average (us) | median (us) |", "|---|---|---|---|"]
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
        v = sorted(d for (gk, gg, _), ds in groups.items() if gk.endswith(k) and gg == grid for d in ds)
        if v:
            med = v[len(v) // 2]
            lines.append(f"| {name} | {nbytes} | {med:.1f} | {nbytes / med / 1e3:.0f} | "
                         f"{nbytes / med / 1e3 / 8000:.2f} |")
    open(args.out, "w").write("\n".join(lines) + "\n")
    print("\n".join(lines))


MARKER = "spin_kernel"           # torch.cuda._sleep, around each of the probe's phases
# the phases of bench.py --kernel-probe, in launch order
PROBE_PHASES = ["project", "expand", "dense", "layer_N1", "dense_N1", "layer_N8", "dense_N8",
                "layer_N16", "dense_N16", "mx_project", "mx_expand", "layer"]


def _dispatches(path):
    """Dispatches of one pmc run in launch order: name, grid, {counter: value}."""
    by = {}
    for r in csv.DictReader(open(path)):
        d = by.setdefault(int(r["Dispatch_Id"]), {"name": r["Kernel_Name"], "grid": int(r["Grid_Size"]), "c": {}})
        d["c"][r["Counter_Name"]] = d["c"].get(r["Counter_Name"], 0.0) + float(r["Counter_Value"])
    return [by[k] for k in sorted(by)]


def _phases(ds, names):
    """{phase: [dispatch]}: phase i lies between markers 2i and 2i + 1."""
    marks = [i for i, d in enumerate(ds) if MARKER in d["name"]]
    if len(marks) < 2 * len(names):
        raise SystemExit(f"{len(marks)} markers for {len(names)} phases")
    return {n: ds[marks[2 * i] + 1:marks[2 * i + 1]] for i, n in enumerate(names)}


def traffic(args):
    sys.path.insert(0, ROOT)
    import bench                                    # the source hash bench.py checks
    from paper_2410_05437_amd import accounting as acc
    res = {}
    for counter, path in (("FETCH_SIZE", args.fetch), ("WRITE_SIZE", args.write)):
        ds = _dispatches(path)
        ph = _phases(ds, PROBE_PHASES)["expand"]
        exp = [d["c"][counter] for d in ph if EXPAND_KERNEL in d["name"] and d["grid"] == EXPAND_GRID]
        cpy = [d["c"][counter] for d in ds if all(k in d["name"] for k in COPY_KERNELS)]
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


def _alg(phase, probe):
    """(algorithmic flops, algorithmic bytes) of one launch of a probe phase."""
    from paper_2410_05437_amd import accounting as acc
    q, d = probe["qkv"], probe["decode"]

    def mx(r, c):   # MX-FP8 matrix bytes: codes, then one scale byte per 32
        cp = (c + 127) // 128 * 128
        return r * cp + r * cp // 32

    if phase == "mx_project":
        return 2 * q["N"] * q["L"] * q["K"], mx(q["N"], q["K"]) + mx(q["L"], q["K"]) + mx(q["N"], q["L"])
    if phase == "mx_expand":
        return 2 * q["N"] * q["M"] * q["L"], mx(q["N"], q["L"]) + mx(q["M"], q["L"]) + 2 * q["N"] * q["M"]
    if phase == "project":
        return acc.gemm_flops(q["N"], q["L"], q["K"]), acc.gemm_bytes(q["N"], q["L"], q["K"])
    if phase == "expand":
        return acc.gemm_flops(q["N"], q["M"], q["L"]), acc.gemm_bytes(q["N"], q["M"], q["L"])
    if phase == "dense":
        return acc.gemm_flops(q["N"], q["M"], q["K"]), acc.gemm_bytes(q["N"], q["M"], q["K"])
    if phase == "layer":
        return (acc.projected_flops(q["K"], q["M"], q["L"], q["N"]),
                acc.projected_bytes(q["K"], q["M"], q["L"], q["N"]))
    n = int(phase.split("_N")[1])
    if phase.startswith("layer"):
        return acc.projected_flops(d["K"], d["M"], d["L"], n), acc.projected_bytes(d["K"], d["M"], d["L"], n)
    return acc.dense_flops(d["K"], d["M"], n), acc.dense_bytes(d["K"], d["M"], n)


def counters(args):
    sys.path.insert(0, ROOT)
    probe = {"qkv": {"K": 4096, "M": 12288, "L": 1536, "N": 4096},
             "decode": {"K": 4096, "M": 22016, "L": 1536, "N": [1, 8, 16]}, "phases": PROBE_PHASES}
    table = collections.OrderedDict()      # (phase, kernel, grid) -> {counter: [values]}
    scale = {}
    for path, _ in args.run:
        ds = _dispatches(path)
        cpy = [d for d in ds if all(k in d["name"] for k in COPY_KERNELS)]
        for c in ("FETCH_SIZE", "WRITE_SIZE"):
            if cpy and c in cpy[0]["c"]:
                scale[c] = (COPY_BYTES / 1024.0) / cpy[0]["c"][c]
        for ph, rows in _phases(ds, probe["phases"]).items():
            for d in rows:
                if not any(k in d["name"] for k in OWN):
                    continue
                key = (ph, _short(d["name"]), d["grid"])
                ent = table.setdefault(key, collections.defaultdict(list))
                for c, v in d["c"].items():
                    ent[c].append(v)
    lines = ["# Hardware counters: the projected linear layer's kernels and the dense layer's", "",
             "Llama2-7B fused QKV (K=4096, M=12288, L=1536, N=4096): project, expand and dense GEMMs; "
             "Llama2-7B FFN up+gate (K=4096, M=22016, L=1536) at decode token counts N = 1, 8, 16: "
             "every kernel of the layer and of the dense layer; the MX-FP8 products of the QKV layer "
             "(mx_project, mx_expand).  bf16 (MX-FP8 in the mx phases), weights rotated over copies "
             "larger than the last-level cache.", "",
             "Counter runs (from the repository root, on one MI355X), one run per counter set:", "", "```"]
    lines += [cmd for _, cmd in args.run] + ["```", ""]
    lines += ["Columns are means per launch.  MFMA busy: the derived `MfmaUtil` (SQ_VALU_MFMA_BUSY_CYCLES "
              "over GRBM_GUI_ACTIVE times the SIMD count).  MFMA flops: (SQ_INSTS_VALU_MFMA_MOPS_BF16 + "
              "SQ_INSTS_VALU_MFMA_MOPS_F8) x 512, against the product's 2·R·C·D.  Bytes: FETCH_SIZE and WRITE_SIZE (KiB) scaled by the "
              "1 GiB copy of the same run "
              + ", ".join(f"({c} x {v:.4f})" for c, v in sorted(scale.items())) + ".", "",
              "| phase | kernel | grid | launches | MFMA busy % | MFMA flops / algorithmic | "
              "fetch MB | write MB | bytes / algorithmic |", "|---|---|---|---|---|---|---|---|---|"]
    phase_bytes = collections.defaultdict(float)
    for (ph, k, grid), ent in table.items():
        mean = {c: sum(v) / len(v) for c, v in ent.items()}
        n = max(len(v) for v in ent.values())
        # a kernel of the layer phase against its own product
        fl, by = _alg(("project" if "v2_kernel" in k else "expand") if ph == "layer" else ph, probe)
        busy = f"{mean['MfmaUtil']:.1f}" if "MfmaUtil" in mean else ""
        mo = [mean[c] for c in ("SQ_INSTS_VALU_MFMA_MOPS_BF16", "SQ_INSTS_VALU_MFMA_MOPS_F8") if c in mean]
        mops = f"{sum(mo) * 512 / fl:.3f}" if mo else ""
        fb = mean.get("FETCH_SIZE", 0.0) * 1024 * scale.get("FETCH_SIZE", 0.0)
        wb = mean.get("WRITE_SIZE", 0.0) * 1024 * scale.get("WRITE_SIZE", 0.0)
        phase_bytes[ph] += fb + wb
        fm = f"{fb / 1e6:.1f}" if "FETCH_SIZE" in mean else ""
        wm = f"{wb / 1e6:.1f}" if "WRITE_SIZE" in mean else ""
        lines.append(f"| {ph} | `{k}` | {grid} | {n} | {busy} | {mops} | {fm} | {wm} | "
                     f"{(fb + wb) / by:.3f} |" if fm and wm else
                     f"| {ph} | `{k}` | {grid} | {n} | {busy} | {mops} | {fm} | {wm} | |")
    if scale:
        lines += ["", "Per phase, all kernels of one call (counter bytes over the call's algorithmic bytes: "
                  "each operand read once, the output written once):", "",
                  "| phase | counter MB per call | algorithmic MB | ratio |", "|---|---|---|---|"]
        for ph in probe["phases"]:
            if ph in phase_bytes:
                _, by = _alg(ph, probe)
                lines.append(f"| {ph} | {phase_bytes[ph] / 1e6:.1f} | {by / 1e6:.1f} | "
                             f"{phase_bytes[ph] / by:.3f} |")
    open(args.out, "w").write("\n".join(lines) + "\n")
    print("\n".join(lines))


# operand bytes the tiles of a tiled GEMM read from L2 per launch: tiles x
# (tile rows + tile columns) x depth x element bytes; per phase, by kernel
# (the layer phase runs the projection, then the expand GEMM on Z in row pairs)
_PROJ = ("4096 x 1536, depth 4096, 128 x 192 tiles", 32 * 8 * (128 + 192) * 4096 * 2)
_EXP = ("4096 x 12288, depth 1536, 256 x 256 tiles", 16 * 48 * 512 * 1536 * 2)
LOADPATH_PHASES = {
    "project": {"gemm_tn_bf16_v2_kernel<128, 192": _PROJ},
    "expand": {"gemm_tn_bf16_v3_kernel<0, 256, 0>": _EXP},
    "dense": {"gemm_tn_bf16_v3_kernel<0, 256, 0>": ("4096 x 12288, depth 4096, 256 x 256 tiles",
                                                    16 * 48 * 512 * 4096 * 2)},
    "layer": {"gemm_tn_bf16_v2_kernel<128, 192": _PROJ,
              "gemm_tn_bf16_v3_kernel<0, 256, 1>": ("expand, Z in row pairs: " + _EXP[0], _EXP[1])},
}


def loadpath(args):
    """Per-CU load path of the tiled GEMMs.  The per-unit counters are sums
    over their instances: TA, TD and TCP one per CU (256), TCC one per L2
    channel (16 per XCD, 128); GRBM_GUI_ACTIVE sums the 8 XCDs' active
    cycles, so one unit's share of the kernel's cycles is counter /
    (GRBM_GUI_ACTIVE / 8 x units)."""
    table = collections.defaultdict(lambda: collections.defaultdict(list))   # (phase, kernel key) -> counters
    kname = {}
    for path, _ in args.run:
        ds = _dispatches(path)
        for ph, rows in _phases(ds, PROBE_PHASES).items():
            for d in rows:
                for key in LOADPATH_PHASES.get(ph, {}):
                    if key in d["name"]:
                        kname[(ph, key)] = _short(d["name"])
                        for c, v in d["c"].items():
                            table[(ph, key)][c].append(v)
    lines = ["# Load-path counters of the tiled GEMMs: Llama2-7B fused QKV (K=4096, M=12288, L=1536, N=4096)", "",
             "The projection, the expand GEMM (on a plain Z) and the dense baseline of `bench.py "
             "--kernel-probe`, and the layer's own two kernels (its expand GEMM reads Z in the workspace's "
             "row-pair layout); bf16, weights rotated over copies larger than the last-level cache.  Counter "
             "runs (from the repository root, on one MI355X):", "", "```"]
    lines += [cmd for _, cmd in args.run] + ["```", ""]
    lines += ["Per launch.  Unit shares: counter / (GRBM_GUI_ACTIVE / 8 x units), units = 256 (TA, TD, "
              "TCP: one per CU) or 128 (TCC: one per L2 channel).  TA busy: the address unit; TA stalled: "
              "cycles the TA could not pass addresses to the TCP (TA_ADDR_STALLED_BY_TC_CYCLES); TD busy / "
              "TD stalled: the data-return unit and its cycles waiting for the TCP (TD_TC_STALL); TCP pending: "
              "cycles the L1 waited for data from L2 (TCP_PENDING_STALL_CYCLES); L2 busy: TCC_BUSY.  "
              "waitcnt: SQ_WAIT_INST_ANY over SQ_WAVE_CYCLES.  Bytes per L2 request: the operand bytes the "
              "tiles read over TCC_HIT + TCC_MISS (which also count the output writes).", "",
              "| phase | kernel | shape | MFMA busy % | waitcnt % | TA busy % | TA stalled % | TD busy % | "
              "TD stalled % | TCP pending % | L2 busy % | L2 hit % | L2 requests (M) | operand B / request |",
              "|---|---|---|---|---|---|---|---|---|---|---|---|---|---|"]
    for ph, kernels in LOADPATH_PHASES.items():
        for key, (shape, opb) in kernels.items():
            if (ph, key) not in table:
                continue
            m = {c: sum(v) / len(v) for c, v in table[(ph, key)].items()}
            cyc = m.get("GRBM_GUI_ACTIVE", 0.0) / 8.0

            def share(c, units):
                return f"{100.0 * m[c] / (cyc * units):.0f}" if c in m and cyc else ""

            busy = f"{100.0 * m['SQ_VALU_MFMA_BUSY_CYCLES'] / (cyc * 1024):.0f}" \
                if "SQ_VALU_MFMA_BUSY_CYCLES" in m and cyc else ""
            wait = f"{100.0 * m['SQ_WAIT_INST_ANY'] / m['SQ_WAVE_CYCLES']:.0f}" \
                if "SQ_WAIT_INST_ANY" in m and m.get("SQ_WAVE_CYCLES") else ""
            req = m.get("TCC_HIT", 0.0) + m.get("TCC_MISS", 0.0)
            hit = f"{100.0 * m['TCC_HIT'] / req:.0f}" if req else ""
            lines.append(f"| {ph} | `{kname[(ph, key)]}` | {shape} | {busy} | {wait} | {share('TA_TA_BUSY', 256)} | "
                         f"{share('TA_ADDR_STALLED_BY_TC_CYCLES', 256)} | {share('TD_TD_BUSY', 256)} | "
                         f"{share('TD_TC_STALL', 256)} | {share('TCP_PENDING_STALL_CYCLES', 256)} | "
                         f"{share('TCC_BUSY', 128)} | {hit} | {req / 1e6:.2f} | "
                         f"{opb / req:.0f} |" if req else "")
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
    c = sub.add_parser("counters")
    c.add_argument("out")
    c.add_argument("--run", nargs=2, action="append", metavar=("CSV", "CMD"), required=True)
    d = sub.add_parser("loadpath")
    d.add_argument("out")
    d.add_argument("--run", nargs=2, action="append", metavar=("CSV", "CMD"), required=True)
    args = ap.parse_args()
    {"stats": stats, "traffic": traffic, "counters": counters, "loadpath": loadpath}[args.mode](args)


if __name__ == "__main__":
    main()
