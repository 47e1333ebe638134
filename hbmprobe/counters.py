"""Summarise rocprofv3 --pmc runs of streaming kernels as one markdown table.

Each --run names a label, a substring of the kernel name, the number of shard
elements one dispatch processes, and the rocprofv3 output directories of the
counter passes taken for it (one counter set per pass; a directory holds
run_counter_collection.csv).  For every run the counters of the matching
dispatches are averaged and these figures derived:

  EA read latency   TCC_EA0_RDREQ_LEVEL_sum / TCC_EA0_RDREQ_sum: the mean time
                    (in GPU clock cycles) a read request from the L2 to the
                    data fabric is outstanding
  reads in flight   TCC_EA0_RDREQ_LEVEL_sum / (GRBM_GUI_ACTIVE / XCDs): the mean
                    number of such requests outstanding over the dispatch
  the same for writes (TCC_EA0_WRREQ_LEVEL_sum, TCC_EA0_WRREQ_sum)
  stall shares      cycles an L2 channel stalled (write requests; out of fabric
                    credits for reads / writes; the tag pipeline) over the
                    dispatch's cycles summed over the 16 channels of each XCD
  VALU figures      VALU instructions per element (all; f64 adds and
                    multiplies), and the share of wave time spent issuing VALU
                    instructions and waiting

GRBM_GUI_ACTIVE is summed over the XCDs by the profiler; it is divided by
their number.  The per-dispatch timestamps of counter runs are not used:
counter collection serialises dispatches and changes their duration.

    python hbmprobe/counters.py --xcds 8 --cmd "..." \\
        --run step_R8 "k_pattern<8, 3, 1, 0, true>" 1003782144 dirA dirB ... \\
        --run ...
"""
import argparse
import csv
import glob
import os

CHANNELS_PER_XCD = 16


def _load(d):
    path = os.path.join(d, "run_counter_collection.csv")
    if not os.path.exists(path):
        hits = glob.glob(os.path.join(d, "**", "*counter_collection.csv"), recursive=True)
        if not hits:
            raise FileNotFoundError(path)
        path = hits[0]
    per = {}
    names = {}
    for r in csv.DictReader(open(path)):
        k = int(r["Dispatch_Id"])
        per.setdefault(k, {})[r["Counter_Name"]] = float(r["Counter_Value"])
        names[k] = r["Kernel_Name"]
    return per, names


def collect(dirs, kernel):
    """Mean of every counter over the dispatches whose name contains
    `kernel`, merged over the passes."""
    out = {}
    for d in dirs:
        per, names = _load(d)
        ks = [k for k in per if kernel in names[k]]
        if not ks:
            raise KeyError("no dispatch of %r in %s" % (kernel, d))
        for c in per[ks[0]]:
            vals = [per[k][c] for k in ks if c in per[k]]
            out.setdefault(c, sum(vals) / len(vals))
        out.setdefault("_dispatches", len(ks))
    return out


def derive(c, elems, xcds):
    d = {}
    cyc = c.get("GRBM_GUI_ACTIVE")
    cyc_xcd = cyc / xcds if cyc else None
    chan_cycles = cyc_xcd * xcds * CHANNELS_PER_XCD if cyc_xcd else None
    rd, wr = c.get("TCC_EA0_RDREQ_sum"), c.get("TCC_EA0_WRREQ_sum")
    if rd and "TCC_EA0_RDREQ_LEVEL_sum" in c:
        d["EA read latency (cycles)"] = c["TCC_EA0_RDREQ_LEVEL_sum"] / rd
        if cyc_xcd:
            d["reads in flight"] = c["TCC_EA0_RDREQ_LEVEL_sum"] / cyc_xcd
    if wr and "TCC_EA0_WRREQ_LEVEL_sum" in c:
        d["EA write latency (cycles)"] = c["TCC_EA0_WRREQ_LEVEL_sum"] / wr
        if cyc_xcd:
            d["writes in flight"] = c["TCC_EA0_WRREQ_LEVEL_sum"] / cyc_xcd
    if rd:
        d["read bytes / element (128 B requests)"] = rd * 128.0 / elems
    if wr and "TCC_EA0_WRREQ_64B_sum" in c:
        w64 = c["TCC_EA0_WRREQ_64B_sum"]
        d["write bytes / element (64 B and 32 B requests)"] = \
            (64.0 * w64 + 32.0 * (wr - w64)) / elems
    if chan_cycles:
        for k, label in (("TCC_EA0_WRREQ_STALL_sum", "write-request stall share"),
                         ("TCC_EA0_RDREQ_DRAM_CREDIT_STALL_sum", "read credit stall share"),
                         ("TCC_EA0_WRREQ_DRAM_CREDIT_STALL_sum", "write credit stall share"),
                         ("TCC_TAG_STALL_sum", "tag stall share")):
            if k in c:
                d[label] = c[k] / chan_cycles
    if "SQ_INSTS_VALU" in c:
        d["VALU instructions / element"] = c["SQ_INSTS_VALU"] * 64.0 / elems
    f64 = sum(c.get(k, 0.0) for k in ("SQ_INSTS_VALU_ADD_F64", "SQ_INSTS_VALU_MUL_F64",
                                       "SQ_INSTS_VALU_FMA_F64"))
    if any(k in c for k in ("SQ_INSTS_VALU_ADD_F64", "SQ_INSTS_VALU_MUL_F64")):
        d["f64 VALU instructions / element"] = f64 * 64.0 / elems
    if c.get("SQ_WAVE_CYCLES"):
        if "SQ_ACTIVE_INST_VALU" in c:
            d["VALU share of wave time"] = c["SQ_ACTIVE_INST_VALU"] / c["SQ_WAVE_CYCLES"]
        if "SQ_WAIT_ANY" in c:
            d["waiting share of wave time"] = c["SQ_WAIT_ANY"] / c["SQ_WAVE_CYCLES"]
    if "SQ_WAVES" in c:
        d["waves"] = c["SQ_WAVES"]
    return d


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--run", nargs="+", action="append", required=True,
                    metavar="LABEL KERNEL ELEMENTS DIR", help="label, kernel-name substring, "
                    "elements per dispatch, then the pass directories")
    ap.add_argument("--xcds", type=int, default=8)
    ap.add_argument("--title", default="Counters of streaming kernels")
    ap.add_argument("--cmd", action="append", default=[], help="command lines quoted")
    a = ap.parse_args()
    rows = []
    for r in a.run:
        label, kernel, elems, dirs = r[0], r[1], int(r[2]), r[3:]
        c = collect(dirs, kernel)
        rows.append((label, kernel, c, derive(c, elems, a.xcds)))
    keys = []
    for _, _, _, d in rows:
        for k in d:
            if k not in keys:
                keys.append(k)
    print("# %s\n" % a.title)
    if a.cmd:
        print("Commands:\n")
        for cmd in a.cmd:
            print("    " + cmd)
        print()
    print("| figure | " + " | ".join(r[0] for r in rows) + " |")
    print("|---|" + "---|" * len(rows))
    for k in keys:
        cells = []
        for _, _, _, d in rows:
            v = d.get(k)
            cells.append("" if v is None else ("%.3f" % v if abs(v) < 10 else "%.0f" % v))
        print("| %s | %s |" % (k, " | ".join(cells)))
    print("\nKernels: " + "; ".join("%s = `%s` (%d dispatches)" % (r[0], r[1],
                                                                  r[2]["_dispatches"])
                                   for r in rows))
    print("\nRaw counters (mean per dispatch):\n")
    names = sorted({k for r in rows for k in r[2] if not k.startswith("_")})
    print("| counter | " + " | ".join(r[0] for r in rows) + " |")
    print("|---|" + "---|" * len(rows))
    for n in names:
        print("| %s | %s |" % (n, " | ".join("%.4g" % r[2][n] if n in r[2] else ""
                                            for r in rows)))


if __name__ == "__main__":
    main()
