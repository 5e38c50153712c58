"""Summaries of rocprofv3 output for profiles/ and bench.py.

  python rocprof_summary.py stats <results.db> <title> <command> > profiles/<name>.md
      per-kernel durations (count, avg/min/max ms, share of GPU time) from a
      --kernel-trace run.

  python rocprof_summary.py counters <config> <trace.db> <fetch.db> <write.db> <sq.db> <tcc.db> <copy_bytes> <command...>
      Counter figures of the score+select kernel of one bench.py workload
      (config 1..5): HBM traffic from a FETCH_SIZE run and a WRITE_SIZE run
      (both in KiB per dispatch), each scaled by what the same counter reads
      for the calibration copy kernel (bench.py --calib-copy), which reads
      and writes copy_bytes; the MFMA work it executed (SQ_INSTS_MFMA; every
      MFMA of the kernel is a 32x32x16 bf16 one, 32768 FLOP); and the busy
      fractions of the units that can bind it: MFMA busy cycles over 1024
      SIMDs, and VALU instructions over one issue per CU per cycle (4 SIMDs,
      each taking a wave64 VALU instruction every 4 cycles), with the
      kernel's cycles from GRBM_GUI_ACTIVE / 8 XCDs.  Stores the entry "c<config>" of
      profiles/select_counters.json (with a hash of the sources the counters
      were taken on; bench.py only reports the figures while the sources are
      unchanged) and prints a markdown summary.

  python rocprof_summary.py pmc <results.db> <command...>
      per-kernel table (mean per dispatch) of every counter of one --pmc run.

  python rocprof_summary.py derived <trace.db> <fetch.db> <write.db> <sq.db> <tcc.db> <copy_bytes>
      per-kernel figures of the kernels above 0.1 ms: average duration (kernel
      trace), calibrated fetch+write bytes, their rate, the L2 hit rate
      (TCC_HIT/(TCC_HIT+TCC_MISS)) and the clock (GRBM_GUI_ACTIVE / 8 XCDs /
      duration); then the MFMA, VALU, SALU and LDS figures of select_kernel.

Reads the SQLite databases rocprofv3 writes by default.
"""
from __future__ import annotations

import hashlib
import json
import os
import sqlite3
import sys

ROOT = os.path.dirname(os.path.abspath(__file__))
COUNTERS_JSON = os.path.join(ROOT, "profiles", "select_counters.json")
# sources whose change invalidates a measured counter figure
SELECT_SOURCES = ["paper_2604_03815_amd/csrc/select.hip", "paper_2604_03815_amd/csrc/group.hip",
                  "paper_2604_03815_amd/csrc/keyorder.hip", "paper_2604_03815_amd/csrc/api.hip",
                  "paper_2604_03815_amd/csrc/kmip_device.h", "paper_2604_03815_amd/csrc/kmip_internal.h"]
MFMA_FLOP = 32 * 32 * 16 * 2


def sources_hash() -> str:
    h = hashlib.sha256()
    for rel in SELECT_SOURCES:
        with open(os.path.join(ROOT, rel), "rb") as f:
            h.update(rel.encode() + b"\0" + f.read() + b"\0")
    return h.hexdigest()


def short(name: str) -> str:
    name = name.replace("kmip::(anonymous namespace)::", "")
    if name.startswith("void "):
        name = name[5:]
    depth, out = 0, []
    for ch in name:
        if ch == "(" and depth == 0:
            break
        depth += ch == "<"
        depth -= ch == ">"
        out.append(ch)
    return "".join(out).strip()


def stats(db: str, title: str, command: str) -> None:
    c = sqlite3.connect(db)
    rows = c.execute("select name, count(*), avg(end-start), min(end-start), max(end-start), "
                     "sum(end-start) from kernels group by name order by sum(end-start) desc").fetchall()
    total = sum(r[5] for r in rows)
    print(f"# Kernel durations: {title}\n")
    print("Command (one MI355X, from the repository root; rocprofv3 writes its database to a "
          "scratch directory):\n")
    print(f"```\n{command}\n```\n")
    print("| kernel | calls | avg ms | min ms | max ms | % of GPU time |")
    print("|---|---|---|---|---|---|")
    for name, n, avg, mn, mx, tot in rows:
        print(f"| `{short(name)}` | {n} | {avg / 1e6:.3f} | {mn / 1e6:.3f} | {mx / 1e6:.3f} | "
              f"{100 * tot / total:.2f} |")


def counter_per_dispatch(db: str, counter: str):
    """{short kernel name: mean over dispatches of the counter summed over its dimensions}."""
    c = sqlite3.connect(db)
    q = ("select kernel_name, dispatch_id, sum(value) from counters_collection "
         "where counter_name = ? group by kernel_name, dispatch_id")
    acc = {}
    for kn, _, v in c.execute(q, (counter,)):
        acc.setdefault(short(kn), []).append(v)
    return {k: sum(v) / len(v) for k, v in acc.items()}


def counters(config: int, trace_db: str, fetch_db: str, write_db: str, sq_db: str, tcc_db: str,
             copy_bytes: int, command: str) -> None:
    c = sqlite3.connect(trace_db)
    dur = {short(n): avg / 1e9 for n, avg in c.execute("select name, avg(end-start) from kernels group by name")}
    fetch = counter_per_dispatch(fetch_db, "FETCH_SIZE")
    write = counter_per_dispatch(write_db, "WRITE_SIZE")
    sq = {n: counter_per_dispatch(sq_db, n) for n in
          ("SQ_INSTS_MFMA", "SQ_VALU_MFMA_BUSY_CYCLES", "SQ_INSTS_VALU", "SQ_INSTS_SALU", "SQ_INSTS_LDS",
           "SQ_WAIT_INST_ANY", "SQ_WAVE_CYCLES")}
    grbm = counter_per_dispatch(tcc_db, "GRBM_GUI_ACTIVE")
    hit = counter_per_dispatch(tcc_db, "TCC_HIT_sum")
    miss = counter_per_dispatch(tcc_db, "TCC_MISS_sum")
    copy = [k for k in fetch if "elementwise" in k.lower()]
    sel = [k for k in fetch if k.startswith("select_kernel")]
    if not copy or not sel:
        raise SystemExit(f"need the calibration copy and select_kernel in the runs, got {sorted(fetch)}")
    ck, sk = copy[0], sel[0]
    f_scale = copy_bytes / (fetch[ck] * 1024.0)
    w_scale = copy_bytes / (write[ck] * 1024.0)
    fetch_b = fetch[sk] * 1024.0 * f_scale
    write_b = write[sk] * 1024.0 * w_scale
    cycles = grbm[sk] / 8.0                       # per XCD, for the counted dispatch
    mfma = sq["SQ_INSTS_MFMA"][sk]
    mfma_busy = sq["SQ_VALU_MFMA_BUSY_CYCLES"][sk] / (1024.0 * cycles)
    valu_issue = sq["SQ_INSTS_VALU"][sk] / (256.0 * cycles)
    entry = {
        "kernel": sk, "sources_sha256": sources_hash(), "trace_ms": dur.get(sk, 0.0) * 1e3,
        "fetch_bytes": fetch_b, "write_bytes": write_b,
        "bytes_per_launch": fetch_b + write_b, "fetch_kib_raw": fetch[sk], "write_kib_raw": write[sk],
        "copy_kernel": ck, "copy_bytes": copy_bytes, "copy_fetch_kib": fetch[ck],
        "copy_write_kib": write[ck], "fetch_scale": f_scale, "write_scale": w_scale,
        "mfma_instructions_per_launch": mfma, "mfma_flop_per_launch": mfma * MFMA_FLOP,
        "valu_instructions_per_launch": sq["SQ_INSTS_VALU"][sk],
        "salu_instructions_per_launch": sq["SQ_INSTS_SALU"][sk],
        "lds_instructions_per_launch": sq["SQ_INSTS_LDS"][sk],
        "kernel_cycles": cycles, "clock_ghz": cycles / dur[sk] / 1e9 if dur.get(sk) else None,
        "mfma_busy_frac": mfma_busy, "valu_issue_frac": valu_issue,
        "wait_frac": sq["SQ_WAIT_INST_ANY"][sk] / max(sq["SQ_WAVE_CYCLES"][sk], 1.0),
        "l2_hit": hit.get(sk, 0.0) / max(hit.get(sk, 0.0) + miss.get(sk, 0.0), 1.0),
        "command": command,
    }
    table = {}
    if os.path.exists(COUNTERS_JSON):
        with open(COUNTERS_JSON) as f:
            table = json.load(f)
        if "kernel" in table:          # a single-workload file of an older layout
            table = {}
    table[f"c{config}"] = entry
    with open(COUNTERS_JSON, "w") as f:
        json.dump(table, f, indent=1, sort_keys=True)
        f.write("\n")
    flop = mfma * MFMA_FLOP
    t = dur.get(sk, 0.0)
    print(f"# Counters of `{sk}`, bench.py workload c{config}\n")
    print(f"Command: `{command}`, one run per counter pass (FETCH_SIZE; WRITE_SIZE; the SQ "
          f"instruction and busy counters; GRBM_GUI_ACTIVE with the L2 hit counters), plus a "
          f"--kernel-trace run of the same command for the duration.\n")
    print("| counter | select_kernel per dispatch | copy kernel | copy bytes | scale | select |")
    print("|---|---|---|---|---|---|")
    print(f"| FETCH_SIZE (KiB) | {fetch[sk]:.4g} | {fetch[ck]:.4g} | {copy_bytes} | {f_scale:.4f} | {fetch_b:.4g} B |")
    print(f"| WRITE_SIZE (KiB) | {write[sk]:.4g} | {write[ck]:.4g} | {copy_bytes} | {w_scale:.4f} | {write_b:.4g} B |")
    print(f"| SQ_INSTS_MFMA | {mfma:.4g} | | | {MFMA_FLOP} FLOP each | {flop:.4g} FLOP |")
    print(f"\n- duration {t * 1e3:.3f} ms (kernel trace), {cycles:.4g} cycles per XCD "
          f"({cycles / t / 1e9 if t else 0:.2f} GHz)")
    if t:
        print(f"- executed MFMA work {flop:.4g} FLOP = {flop / t / 1e12:.0f} TFLOP/s = "
              f"{100 * flop / t / 2.5e15:.1f}% of the 2.5 PFLOP/s bf16 peak")
    print(f"- MFMA busy {100 * mfma_busy:.1f}% of 1024 SIMD-cycles; VALU {sq['SQ_INSTS_VALU'][sk]:.4g} "
          f"instructions = {100 * valu_issue:.1f}% of one issue per CU per cycle; SALU "
          f"{sq['SQ_INSTS_SALU'][sk]:.4g}, LDS {sq['SQ_INSTS_LDS'][sk]:.4g} instructions; "
          f"waiting {100 * entry['wait_frac']:.1f}% of wave cycles; L2 hit {100 * entry['l2_hit']:.0f}%")
    print(f"- HBM traffic {fetch_b + write_b:.4g} B per launch")
    print("\nEvery kernel of the same runs, per dispatch, scaled the same way:\n")
    print("| kernel | fetch bytes | write bytes |")
    print("|---|---|---|")
    for k in sorted(fetch, key=lambda k: -fetch[k] - write.get(k, 0.0)):
        print(f"| `{k}` | {fetch[k] * 1024.0 * f_scale:.4g} | {write.get(k, 0.0) * 1024.0 * w_scale:.4g} |")


def pmc(db: str, command: str) -> None:
    """Per-kernel table of every counter in one --pmc run (mean per dispatch)."""
    c = sqlite3.connect(db)
    names = [r[0] for r in c.execute("select distinct counter_name from counters_collection")]
    table = {n: counter_per_dispatch(db, n) for n in names}
    kernels = sorted({k for t in table.values() for k in t})
    print(f"Command: `{command}`\n")
    print("| kernel | " + " | ".join(names) + " |")
    print("|---|" + "---|" * len(names))
    for k in kernels:
        print(f"| `{k}` | " + " | ".join(f"{table[n].get(k, 0.0):.4g}" for n in names) + " |")


def derived(trace_db: str, fetch_db: str, write_db: str, sq_db: str, tcc_db: str, copy_bytes: int) -> None:
    c = sqlite3.connect(trace_db)
    dur = {}
    for name, avg in c.execute("select name, avg(end-start) from kernels group by name"):
        dur[short(name)] = avg / 1e9
    fetch = counter_per_dispatch(fetch_db, "FETCH_SIZE")
    write = counter_per_dispatch(write_db, "WRITE_SIZE")
    ck = [k for k in fetch if "elementwise" in k.lower()][0]
    f_scale = copy_bytes / (fetch[ck] * 1024.0)
    w_scale = copy_bytes / (write[ck] * 1024.0)
    hit = counter_per_dispatch(tcc_db, "TCC_HIT_sum")
    miss = counter_per_dispatch(tcc_db, "TCC_MISS_sum")
    grbm = counter_per_dispatch(tcc_db, "GRBM_GUI_ACTIVE")
    print("| kernel | avg ms | fetch+write bytes | GB/s | % of 8 TB/s | L2 hit | GPU clock GHz |")
    print("|---|---|---|---|---|---|---|")
    for k in sorted(dur, key=lambda k: -dur[k]):
        if dur[k] < 1e-4 or k not in fetch:
            continue
        b = fetch[k] * 1024.0 * f_scale + write.get(k, 0.0) * 1024.0 * w_scale
        h, m = hit.get(k, 0.0), miss.get(k, 0.0)
        print(f"| `{k}` | {dur[k] * 1e3:.3f} | {b:.4g} | {b / dur[k] / 1e9:.0f} | {b / dur[k] / 8e12 * 100:.1f} | "
              f"{100 * h / max(h + m, 1.0):.0f}% | {grbm.get(k, 0.0) / 8 / dur[k] / 1e9:.2f} |")
    sq = {n: counter_per_dispatch(sq_db, n) for n in
          ("SQ_INSTS_MFMA", "SQ_VALU_MFMA_BUSY_CYCLES", "SQ_INSTS_VALU", "SQ_INSTS_SALU", "SQ_INSTS_LDS",
           "SQ_WAIT_INST_ANY", "SQ_WAVE_CYCLES")}
    sk = [k for k in sq["SQ_INSTS_MFMA"] if k.startswith("select_kernel")][0]
    cycles = grbm[sk] / 8
    flop = sq["SQ_INSTS_MFMA"][sk] * MFMA_FLOP
    print(f"\n`{sk}`: {dur[sk] * 1e3:.3f} ms, {cycles:.4g} cycles per XCD")
    print(f"- MFMA: {sq['SQ_INSTS_MFMA'][sk]:.4g} instructions = {flop:.4g} FLOP executed "
          f"({flop / dur[sk] / 1e12:.0f} TFLOP/s); busy {sq['SQ_VALU_MFMA_BUSY_CYCLES'][sk]:.4g} cycles = "
          f"{100 * sq['SQ_VALU_MFMA_BUSY_CYCLES'][sk] / (1024 * cycles):.1f}% of 1024 SIMDs")
    print(f"- VALU {sq['SQ_INSTS_VALU'][sk]:.4g}, SALU {sq['SQ_INSTS_SALU'][sk]:.4g}, "
          f"LDS {sq['SQ_INSTS_LDS'][sk]:.4g} instructions; waiting "
          f"{100 * sq['SQ_WAIT_INST_ANY'][sk] / sq['SQ_WAVE_CYCLES'][sk]:.1f}% of wave cycles")


def main(argv):
    if len(argv) >= 4 and argv[1] == "stats":
        stats(argv[2], argv[3], " ".join(argv[4:]))
    elif len(argv) >= 9 and argv[1] == "counters":
        counters(int(argv[2]), argv[3], argv[4], argv[5], argv[6], argv[7], int(argv[8]), " ".join(argv[9:]))
    elif len(argv) >= 8 and argv[1] == "derived":
        derived(argv[2], argv[3], argv[4], argv[5], argv[6], int(argv[7]))
    elif len(argv) >= 3 and argv[1] == "pmc":
        pmc(argv[2], " ".join(argv[3:]))
    else:
        raise SystemExit(__doc__)


if __name__ == "__main__":
    main(sys.argv)
