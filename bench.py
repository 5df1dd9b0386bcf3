"""Benchmark of the attention hot path on one MI355X.

One step = one pass over the whole path on resident synthetic inputs:
  * the fused causal attention forward on the long-context workload
    (causal GQA B=1 Hq=32 Hkv=8 S=32768 D=128 bf16, the largest one), then
  * the split-KV decode (equal-work part kernel + LSE merge kernel) on the
    ragged decode batch (B=64 Hq=32 Hkv=8 D=128, lengths in [512, 4096]).
Each workload alternates between two copies of its inputs so the 256 MB
last-level cache cannot hand one launch the previous launch's data.

The K timed steps run as K prefill launches back to back, then K decode
launches back to back, on torch's current stream; HIP events recorded on
that stream before, between and after give each kernel's average launch
duration.  After the step, legs time the other workloads the same way
(each with warm-up launches of its own just before its timed block): the
8k and 2k prefill workloads, the small one, the decode alone over a fixed
number of launches, and the rows built beyond the forward (packed ragged
prefill, paged decode, backward, MLA decode).  Then the CPU oracle is timed
on every workload (a baseline, not a target).  Prints ONE JSON line on
stdout; progress goes to stderr.
"""
from __future__ import annotations

import argparse
import json
import math
import os
import re
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

PEAK_BF16_TFLOPS = 2516.6  # dense bf16 MFMA, 256 CU x 4096 FLOP/clk x 2.4 GHz
PEAK_HBM_GBS = 8000.0      # HBM3E


def log(*a):
    print(*a, file=sys.stderr, flush=True)


def kernel_source_digest() -> str:
    import hashlib
    h = hashlib.sha256()
    csrc = os.path.join(ROOT, "paper_2609_04523_amd", "csrc")
    for name in sorted(os.listdir(csrc)):
        with open(os.path.join(csrc, name), "rb") as fh:
            h.update(name.encode() + b"\0" + fh.read())
    return h.hexdigest()[:16]


def read_traffic(summary_name: str, digest: str):
    """HBM bytes per launch from a committed rocprofv3 counter summary,
    or None when absent or taken on a different kernel source."""
    path = os.path.join(ROOT, "profiles", summary_name)
    if not os.path.exists(path):
        return None
    text = open(path).read()
    m_d = re.search(r"kernel_source_digest:\s*([0-9a-f]+)", text)
    m_t = re.search(r"hbm_bytes_per_launch:\s*([0-9.eE+]+)", text)
    if not m_d or not m_t or m_d.group(1) != digest:
        return None
    return float(m_t.group(1))


# ---------------------------------------------------------------------------
# rocprofv3 summaries (text files committed under profiles/)
# ---------------------------------------------------------------------------
def _find_db(path: str) -> str:
    import glob
    if path.endswith(".db"):
        return path
    hits = sorted(glob.glob(os.path.join(path, "**", "*.db"), recursive=True))
    if not hits:
        raise SystemExit(f"no rocprofv3 database under {path}")
    return hits[0]


def _short(name: str) -> str:
    return name.split("(")[0].replace("void ", "")


def summarize_trace(path: str, command: str, kernels=None) -> str:
    """Markdown table of per-kernel durations from a --kernel-trace run,
    restricted to kernels whose names contain one of `kernels` if given
    (the GPU-time share stays relative to all kernels of the run)."""
    import sqlite3
    db = sqlite3.connect(_find_db(path))
    tags = _dispatch_grids(db)
    try:
        rows = [(n, d, tags.get(i, w)) for i, n, d, w in db.execute(
            "select dispatch_id, name, duration, grid_x / max(workgroup_x, 1) from kernels")]
    except sqlite3.OperationalError:
        try:  # a trace without dispatch ids
            rows = db.execute("select name, duration, grid_x / max(workgroup_x, 1) from kernels"
                              ).fetchall()
        except sqlite3.OperationalError:  # a trace without launch geometry
            rows = [(n, d, 0) for n, d in db.execute("select name, duration from kernels")]
    # launches of one kernel with different grids (one kernel timed on two
    # workloads) get a row per workgroup count
    grids = {}
    for name, _, wgs in rows:
        grids.setdefault(_short(name), set()).add(wgs)
    agg = {}
    for name, dur, wgs in rows:
        key = _short(name)
        if len(grids[key]) > 1:
            key = (f"{key} [after a V^T copy of {wgs[1:]} tiles]" if isinstance(wgs, str)
                   else f"{key} [{wgs} workgroups]")
        agg.setdefault(key, []).append(dur / 1e3)  # ns -> us
    total = sum(sum(v) for v in agg.values())
    if kernels:
        agg = {k: v for k, v in agg.items() if any(f in k for f in kernels)}
    out = ["# rocprofv3 kernel trace", "", f"command: `{command}`", "",
           f"kernel_source_digest: {kernel_source_digest()}", "",
           "| kernel | calls | avg us | min us | max us | % of GPU time |",
           "|---|---|---|---|---|---|"]
    for k, v in sorted(agg.items(), key=lambda kv: -sum(kv[1])):
        out.append(f"| `{k}` | {len(v)} | {sum(v) / len(v):.2f} | {min(v):.2f} | {max(v):.2f} | "
                   f"{100 * sum(v) / total:.1f} |")
    return "\n".join(out) + "\n"


def _dispatch_grids(db):
    """dispatch id -> workgroup count, from the trace tables of a run (empty
    for databases without launch geometry).  The persistent V^T forward
    launches one workgroup per compute unit whatever the workload, so its
    dispatches are told apart by the V^T copy made just before them: 'v'
    and the pack kernel's workgroup count."""
    import sqlite3
    try:
        rows = db.execute("select dispatch_id, name, grid_x / max(workgroup_x, 1) from kernels "
                          "order by dispatch_id").fetchall()
    except sqlite3.OperationalError:
        return {}
    out, last_pack = {}, None
    for d, name, w in rows:
        short = _short(name)
        if "vt_pack_kernel" in short:
            last_pack = int(w)
        if "fwd_kernel" in short and short.endswith("true, true>") and last_pack is not None:
            out[d] = f"v{last_pack}"
        else:
            out[d] = int(w)
    return out


def _pmc_per_kernel(path: str, counter: str):
    """Counter values per dispatch, keyed by kernel name and also by
    'name@N' for the dispatches with N workgroups (one kernel timed on
    several workloads)."""
    import sqlite3
    db = sqlite3.connect(_find_db(path))
    rows = db.execute("select dispatch_id, name, counter_name, counter_value from pmc_events "
                      "where counter_name = ?", (counter,)).fetchall()
    grids = _dispatch_grids(db)
    per_disp = {}
    for disp, name, _, val in rows:
        key = (disp, _short(name))
        per_disp[key] = per_disp.get(key, 0.0) + val
    per_kernel = {}
    for (disp, name), val in per_disp.items():
        per_kernel.setdefault(name, []).append(val)
        if disp in grids:
            per_kernel.setdefault(f"{name}@{grids[disp]}", []).append(val)
    return per_kernel


def _match_kernel(names, frag: str):
    """Kernel key for a fragment 'part' or 'part@N' (N workgroups)."""
    if "@" in frag:
        part, wgs = frag.split("@")
        return [n for n in names if n.endswith(f"@{wgs}") and part in n]
    return [n for n in names if frag in n and "@" not in n]


def summarize_pmc(fetch_path: str, write_path: str, kernels, calib_bytes: int,
                  commands) -> str:
    """Per-launch HBM bytes of `kernels` (summed: one launch of the path)
    from FETCH_SIZE / WRITE_SIZE runs, each scaled by what the counter reads
    for the plain device copy of calib_bytes in the same run."""
    fetch = _pmc_per_kernel(fetch_path, "FETCH_SIZE")
    write = _pmc_per_kernel(write_path, "WRITE_SIZE")
    copy = [k for k in fetch if "copyBuffer" in k and "@" not in k]
    if not copy:
        raise SystemExit("no calibration copy kernel in the FETCH_SIZE run")
    # the calibration copy is the largest copyBuffer dispatch
    f_copy = max(fetch[copy[0]])
    w_copy = max(write[copy[0]])
    f_fac = (calib_bytes / 1024) / f_copy
    w_fac = (calib_bytes / 1024) / w_copy
    out = ["# rocprofv3 HBM traffic counters", ""]
    for c in commands:
        out.append(f"command: `{c}`")
    out += ["", f"kernel_source_digest: {kernel_source_digest()}", "",
            f"calibration: plain device copy of {calib_bytes} bytes reads FETCH_SIZE = "
            f"{f_copy:.1f} KiB and WRITE_SIZE = {w_copy:.1f} KiB per dispatch; "
            f"scale factors fetch x{f_fac:.4f}, write x{w_fac:.4f}", "",
            "| kernel | launches | FETCH_SIZE KiB/launch | WRITE_SIZE KiB/launch | "
            "scaled read bytes | scaled write bytes |", "|---|---|---|---|---|---|"]
    total = 0.0
    for k in kernels:
        name = _match_kernel(list(fetch), k)
        if not name:
            raise SystemExit(f"kernel {k} not in the counter runs")
        fv, wv = fetch[name[0]], write.get(name[0], [])
        if not wv:
            raise SystemExit(f"kernel {k} not in the WRITE_SIZE run")
        f_avg, w_avg = sum(fv) / len(fv), sum(wv) / len(wv)
        rb, wb = f_avg * 1024 * f_fac, w_avg * 1024 * w_fac
        total += rb + wb
        out.append(f"| `{name[0]}` | {len(fv)} | {f_avg:.1f} | {w_avg:.1f} | {rb:.4g} | {wb:.4g} |")
    out += ["", f"hbm_bytes_per_launch: {total:.6g}", ""]
    return "\n".join(out)


def summarize_sq(paths, kernel: str, commands) -> str:
    """Per-dispatch SQ/GRBM counters of the dispatches of `kernel` from one or
    more --pmc runs (one counter pass each), averaged over the dispatches, and
    the ratios derived from them.  SQ_* counters are summed over the chip;
    GRBM_GUI_ACTIVE over the 8 XCDs, so the engine cycles of the kernel are
    GRBM_GUI_ACTIVE / 8; MFMA busy = SQ_VALU_MFMA_BUSY_CYCLES / (1024 SIMDs x
    those cycles); the wave-cycle counters count in units of 4 cycles, so
    their ratios to SQ_WAVE_CYCLES are fractions of wave time."""
    vals = {}
    for path in paths:
        for counter_rows in [_pmc_all(path)]:
            names = sorted({n for n, _ in counter_rows})
            keep = set(_match_kernel(names, kernel))
            for (name, counter), v in counter_rows.items():
                if name in keep:
                    vals.setdefault(counter, []).extend(v)
    avg = {c: sum(v) / len(v) for c, v in vals.items()}
    out = ["# rocprofv3 SQ counters", ""]
    for c in commands:
        out.append(f"command: `{c}`")
    out += ["", f"kernel_source_digest: {kernel_source_digest()}", "",
            f"kernel: `{kernel}`", "", "| counter | per dispatch |", "|---|---|"]
    for c in sorted(avg):
        out.append(f"| {c} | {avg[c]:.4g} |")
    out.append("")
    g = avg.get("GRBM_GUI_ACTIVE")
    if g:
        cyc = g / 8.0
        out.append(f"engine cycles per dispatch (GRBM_GUI_ACTIVE / 8): {cyc:.4g}")
        if "SQ_VALU_MFMA_BUSY_CYCLES" in avg:
            out.append(f"MFMA busy: {100 * avg['SQ_VALU_MFMA_BUSY_CYCLES'] / (1024 * cyc):.1f} % "
                       "of SIMD cycles")
        if "SQ_INSTS_MFMA" in avg:
            out.append(f"MFMA instructions per dispatch: {avg['SQ_INSTS_MFMA']:.4g}")
    w = avg.get("SQ_WAVE_CYCLES")
    if w:
        for c in ("SQ_WAIT_ANY", "SQ_WAIT_INST_ANY", "SQ_WAIT_INST_LDS", "SQ_ACTIVE_INST_VALU",
                  "SQ_ACTIVE_INST_LDS"):
            if c in avg:
                out.append(f"{c} / SQ_WAVE_CYCLES: {100 * avg[c] / w:.1f} %")
    if "SQ_INSTS_VALU" in avg and "SQ_INSTS_MFMA" in avg:
        out.append(f"vector instructions per MFMA (SQ_INSTS_VALU less MFMA): "
                   f"{(avg['SQ_INSTS_VALU'] - avg['SQ_INSTS_MFMA']) / avg['SQ_INSTS_MFMA']:.2f}")
    return "\n".join(out) + "\n"


def _pmc_all(path: str):
    """Every counter per dispatch, keyed (kernel, counter) and also
    (kernel@N, counter) for the dispatches with N workgroups."""
    import sqlite3
    db = sqlite3.connect(_find_db(path))
    rows = db.execute("select dispatch_id, name, counter_name, counter_value from pmc_events"
                      ).fetchall()
    grids = _dispatch_grids(db)
    per_disp = {}
    for disp, name, counter, val in rows:
        key = (disp, _short(name), counter)
        per_disp[key] = per_disp.get(key, 0.0) + val
    out = {}
    for (disp, name, counter), val in per_disp.items():
        out.setdefault((name, counter), []).append(val)
        if disp in grids:
            out.setdefault((f"{name}@{grids[disp]}", counter), []).append(val)
    return out


LEGS_ALL = "c3,c2,c1,decode,varlen,rpa,paged,bwd,mla"


def prefill_alg_bytes(cfg) -> int:
    """Algorithmic HBM bytes of one forward launch: q, k, v read once, o and
    lse written once."""
    q = cfg.B * cfg.Hq * cfg.S * cfg.D * 2
    kv = 2 * cfg.B * cfg.Hkv * cfg.S * cfg.D * 2
    o = cfg.B * cfg.Hq * cfg.S * cfg.D * (4 if cfg.out_fp32 else 2)
    lse = cfg.B * cfg.Hq * cfg.S * 4
    return q + kv + o + lse


def decode_alg_bytes(B, Hq, Hkv, D, sum_l) -> int:
    """Algorithmic HBM bytes of one decode: each valid cached key and value
    row once per kv head, q read, o (bf16) and lse written."""
    return 4 * D * Hkv * sum_l + (B * Hq * D * 2) * 2 + B * Hq * 4


def prefill_record(cfg, us, traffic):
    flops = cfg.flops
    tf = flops / (us * 1e-6) / 1e12
    nbytes = prefill_alg_bytes(cfg)
    gbs = nbytes / (us * 1e-6) / 1e9
    rec = {
        "workload": (f"{cfg.name}: causal attention fwd B={cfg.B} Hq={cfg.Hq} Hkv={cfg.Hkv} "
                     f"S={cfg.S} D={cfg.D} bf16 in, {'fp32' if cfg.out_fp32 else 'bf16'} O"
                     + (f", K x{cfg.k_mult:g}" if cfg.k_mult != 1.0 else "")),
        "us": round(us, 2),
        "tflops": round(tf, 2),
        "frac_mfma_peak": round(tf / PEAK_BF16_TFLOPS, 4),
        "flops": flops,
        "alg_bytes": nbytes,
        "gbs": round(gbs, 1),
        "frac_hbm_peak": round(gbs / PEAK_HBM_GBS, 5),
        "counter_bytes": traffic,
        "counter_gbs": None if traffic is None else round(traffic / (us * 1e-6) / 1e9, 1),
    }
    return rec


def time_block(stream, fn, warmup: int, n: int) -> float:
    """Average duration (ms) of n launches of fn(i) issued back to back after
    `warmup` untimed ones, between two events on `stream`."""
    import torch
    for i in range(warmup):
        fn(i)
    ev = [torch.cuda.Event(enable_timing=True) for _ in range(2)]
    torch.cuda.synchronize()
    ev[0].record(stream)
    for i in range(n):
        fn(i)
    ev[1].record(stream)
    torch.cuda.synchronize()
    return ev[0].elapsed_time(ev[1]) / n


def cpu_baselines(args, dec_sum_l):
    """The oracle as it stands, timed on the host: every workload, the 32k one
    on its 256-row-per-head sample (plus a labelled extrapolation to all
    rows), and single-thread times for the small workloads."""
    import workloads
    from oracle import oracle as orc  # timed CPU baseline only
    threads = orc.default_threads()
    runs = []

    def prefill_run(cfg, nthreads, rows_per_head=0, batches=None):
        q, k, v = workloads.config_inputs(cfg)
        if batches is not None:
            q, k, v = q[:batches], k[:batches], v[:batches]
        B = q.shape[0]
        qb, kb, vb = workloads.bits(q), workloads.bits(k), workloads.bits(v)
        del q, k, v
        if rows_per_head:
            rows = workloads.sample_rows(B, cfg.Hq, cfg.S, rows_per_head, seed=cfg.seed)
            pairs = int((rows.long() + 1).sum())  # causal row i sees i + 1 keys
            rows_np = rows.numpy()
            what = f"{rows_per_head} seeded query rows per head"
        else:
            rows_np = None
            pairs = B * cfg.Hq * cfg.pairs_per_head
            what = "every query row" + (f" of batch entries 0..{B - 1}" if batches else "")
        log(f"[bench] cpu oracle: {cfg.name}, {what}, {nthreads} threads")
        t0 = time.perf_counter()
        orc.attn_fwd(qb, kb, vb, causal=True, scale=cfg.scale, rows=rows_np, threads=nthreads)
        sec = time.perf_counter() - t0
        rec = {"config": cfg.name, "rows": what, "threads": nthreads, "seconds": round(sec, 3),
               "pairs": pairs, "fp64_tflops": 4 * cfg.D * pairs / sec / 1e12}
        full_pairs = cfg.B * cfg.Hq * cfg.pairs_per_head
        if pairs != full_pairs:
            rec["extrapolated_full_seconds"] = round(sec * full_pairs / pairs, 1)
        runs.append(rec)
        return rec

    def decode_run(cfg, nthreads):
        qd, kc, vc, lens = workloads.config_inputs(cfg)
        args_ = (workloads.bits(qd), workloads.bits(kc), workloads.bits(vc), lens.numpy())
        del kc, vc
        log(f"[bench] cpu oracle: {cfg.name}, {nthreads} threads")
        t0 = time.perf_counter()
        orc.decode(*args_, scale=cfg.scale, threads=nthreads)
        sec = time.perf_counter() - t0
        pairs = cfg.Hq * dec_sum_l
        runs.append({"config": cfg.name, "rows": "every sequence", "threads": nthreads,
                     "seconds": round(sec, 3), "pairs": pairs,
                     "fp64_tflops": 4 * cfg.D * pairs / sec / 1e12})

    C = workloads.CONFIGS
    head = prefill_run(C["c4_gqa_s32k"], threads, rows_per_head=C["c4_gqa_s32k"].sample_rows)
    if args.cpu_baseline == "all":
        prefill_run(C["c1_mha_s128_d64"], threads)
        prefill_run(C["c1_mha_s128_d64"], 1)
        prefill_run(C["c2_mha_s2k"], threads)
        prefill_run(C["c2_mha_s2k"], 1, batches=1)
        prefill_run(C["c3_gqa_s8k_k2"], threads)
        decode_run(C["c5_decode_b64"], threads)
        decode_run(C["c5_decode_b64"], 1)
    return {
        "value": round(head["fp64_tflops"], 6),
        "unit": "TFLOP/s",
        "cores": threads,
        "host_cpus": os.cpu_count(),
        "kind": "oracle",
        "sample": (f"{head['rows']} of c4_gqa_s32k ({head['pairs']} query-key pairs, fp64, "
                   f"{head['seconds']:.2f} s on {threads} threads; all rows extrapolate to "
                   f"{head['extrapolated_full_seconds']} s); per_config lists every workload"),
        "per_config": runs,
    }


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--prefill", default="c4_gqa_s32k")
    ap.add_argument("--decode", default="c5_decode_b64")
    ap.add_argument("--parts", type=int, default=0, help="decode parts (0 = library default)")
    ap.add_argument("--legs", default=LEGS_ALL,
                    help="comma-separated legs timed after the step ('' for none): "
                         + LEGS_ALL)
    ap.add_argument("--decode-launches", type=int, default=200,
                    help="launches of the stand-alone decode leg (after 50 warm-up ones)")
    ap.add_argument("--cpu-baseline", choices=("all", "headline", "none"), default="all",
                    help="oracle timing: every workload, the headline sample only, or none")
    ap.add_argument("--page-size", type=int, default=16, help="page size of the paged leg")
    ap.add_argument("--ws-min-seq", type=int, default=8192,
                    help="prefill workloads with at least this many keys run through "
                         "mk_attn_fwd_ws (0: all bf16 ones; a huge value: none)")
    ap.add_argument("--calib-copy-mib", type=int, default=0,
                    help="also run one plain device copy of this size (counter calibration)")
    ap.add_argument("--summarize-trace", metavar="DIR",
                    help="print a summary of a rocprofv3 --kernel-trace output and exit")
    ap.add_argument("--summarize-pmc", nargs=2, metavar=("FETCH_DIR", "WRITE_DIR"),
                    help="print per-launch HBM bytes from FETCH_SIZE / WRITE_SIZE runs and exit")
    ap.add_argument("--summarize-sq", nargs="+", metavar="DIR",
                    help="print SQ/GRBM counters of --kernels (one name) from --pmc runs and exit")
    ap.add_argument("--kernels", default=None,
                    help="semicolon-separated kernel name fragments, each optionally "
                         "'name@N' for its launches with N workgroups, for --summarize-pmc "
                         "(default fwd_kernel) or --summarize-trace (default all)")
    ap.add_argument("--command", action="append", default=[],
                    help="command line(s) recorded in a summary")
    args = ap.parse_args()
    args.kernels_given = args.kernels is not None
    if args.kernels is None:
        args.kernels = "fwd_kernel"

    if args.summarize_trace:
        kern = args.kernels.split(";") if args.kernels_given else None
        print(summarize_trace(args.summarize_trace, "; ".join(args.command), kern), end="")
        return
    if args.summarize_sq:
        print(summarize_sq(args.summarize_sq, args.kernels, args.command), end="")
        return
    if args.summarize_pmc:
        print(summarize_pmc(args.summarize_pmc[0], args.summarize_pmc[1],
                            args.kernels.split(";"), args.calib_copy_mib << 20, args.command),
              end="")
        return

    if args.gpus != 1:
        print(f"bench.py runs on one GPU only; --gpus {args.gpus} is not supported "
              "(the path would shard by (batch, kv head) groups, one group set per GPU)",
              file=sys.stderr)
        sys.exit(2)
    legs = [x for x in args.legs.split(",") if x]
    unknown = set(legs) - set(LEGS_ALL.split(","))
    if unknown:
        raise SystemExit(f"unknown legs {sorted(unknown)}")

    import torch

    import paper_2609_04523_amd as mk
    import workloads

    if not os.path.exists(mk.LIB_PATH):
        from paper_2609_04523_amd import build as hip_build
        hip_build.build()
    mk.lib()
    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    stream = torch.cuda.current_stream()
    digest = kernel_source_digest()

    def prefill_inputs_on_device(cfg):
        """Two copies of a prefill workload's tensors, used alternately."""
        q, k, v = workloads.config_inputs(cfg)
        out = []
        for _ in range(2):
            o = torch.empty(q.shape, device=dev,
                            dtype=torch.float32 if cfg.out_fp32 else torch.bfloat16)
            lse = torch.empty(q.shape[:3], device=dev, dtype=torch.float32)
            out.append((q.to(dev), k.to(dev), v.to(dev), o, lse))
        return out

    def prefill_entry(cfg):
        """The entry point a workload runs through: mk_attn_fwd_ws (V^T tiles
        written by the call, then the forward) where the copy pays for itself
        (keys re-read by many query tiles: S >= --ws-min-seq), else mk_attn_fwd."""
        if cfg.out_fp32:
            return "mk_attn_fwd_o32"
        return "mk_attn_fwd_ws" if cfg.S >= args.ws_min_seq else "mk_attn_fwd"

    def prefill_fn(cfg, bufs):
        name = prefill_entry(cfg)
        if name == "mk_attn_fwd_ws":
            wsb = mk.mk_attn_fwd_workspace_bytes(cfg.B, cfg.Hkv, cfg.S, cfg.D)
            wsp = torch.empty(wsb, device=dev, dtype=torch.uint8)

            def run(i):
                q, k, v, o, lse = bufs[i & 1]
                mk.mk_attn_fwd_ws(q, k, v, o, lse, cfg.B, cfg.Hq, cfg.Hkv, cfg.S, cfg.S, cfg.D,
                                  1, cfg.scale, None, wsp, wsb, stream)
            return run
        entry = getattr(mk, name)

        def run(i):
            q, k, v, o, lse = bufs[i & 1]
            entry(q, k, v, o, lse, cfg.B, cfg.Hq, cfg.Hkv, cfg.S, cfg.S, cfg.D, 1, cfg.scale,
                  None, stream)
        return run

    pcfg = workloads.CONFIGS[args.prefill]
    dcfg = workloads.CONFIGS[args.decode]
    log(f"[bench] inputs: prefill {pcfg.name}, decode {dcfg.name}")
    pre = prefill_inputs_on_device(pcfg)
    prefill = prefill_fn(pcfg, pre)
    qd, kc, vc, lens = workloads.config_inputs(dcfg)
    caches = [(kc.to(dev), vc.to(dev)), (kc.to(dev), vc.to(dev))]
    qd = qd.to(dev)
    lens_d = lens.to(dev)
    B, Hq, D = qd.shape
    Hkv, Smax = dcfg.Hkv, dcfg.Smax
    ws_bytes = mk.mk_attn_decode_workspace_bytes(Hq, Hkv, D, args.parts)
    ws = torch.empty(ws_bytes, device=dev, dtype=torch.uint8)
    od = torch.empty((B, Hq, D), device=dev, dtype=torch.bfloat16)
    lsed = torch.empty((B, Hq), device=dev, dtype=torch.float32)
    sum_l = int(lens.clamp(0, Smax).sum())
    dec_bytes = decode_alg_bytes(B, Hq, Hkv, D, sum_l)

    def decode(i):
        kcc, vcc = caches[i & 1]
        mk.mk_attn_decode(qd, kcc, vcc, od, lsed, B, Hq, Hkv, Smax, D, dcfg.scale, lens_d,
                          args.parts, ws, ws_bytes, stream)

    if args.calib_copy_mib:
        n = args.calib_copy_mib << 20
        src = torch.empty(n, device=dev, dtype=torch.uint8).fill_(1)
        dst = torch.empty_like(src)
        torch.cuda.synchronize()
        dst.copy_(src)
        torch.cuda.synchronize()
        log(f"[bench] calibration copy of {n} bytes done")
        del src, dst

    # ---- the step: K prefill launches, then K decode launches ----
    log(f"[bench] warmup {args.warmup}")
    for i in range(args.warmup):
        prefill(i)
        decode(i)
    torch.cuda.synchronize()
    K = args.steps
    # One event before, between and after: a marker between two kernels
    # costs the command processor several microseconds, which per-launch
    # events would add to every launch's measured duration.
    ev = [torch.cuda.Event(enable_timing=True) for _ in range(3)]
    log(f"[bench] timing {K} steps")
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    ev[0].record(stream)
    for i in range(K):
        prefill(i)
    ev[1].record(stream)
    for i in range(K):
        decode(i)
    ev[2].record(stream)
    torch.cuda.synchronize()
    t1 = time.perf_counter()
    ms_step = (t1 - t0) * 1e3 / K
    pre_ms = ev[0].elapsed_time(ev[1]) / K
    dec_step_ms = ev[1].elapsed_time(ev[2]) / K
    del pre
    torch.cuda.empty_cache()
    log(f"[bench] step: prefill {pcfg.name} {pre_ms * 1e3:.1f} us, decode {dec_step_ms * 1e3:.1f} "
        f"us, {ms_step:.3f} ms per step")

    def traffic_of(cfg_name, kernel="fwd_kernel"):
        return read_traffic(f"{kernel}_{cfg_name}_counters.md", digest)

    configs = {pcfg.name: prefill_record(pcfg, pre_ms * 1e3, traffic_of(pcfg.name))}
    configs[pcfg.name]["entry"] = prefill_entry(pcfg)

    # ---- legs ----
    dec_ms = None
    if "decode" in legs:
        # the decode alone, its figure independent of --steps: a fixed number
        # of launches right after warm-up launches of its own
        dec_ms = time_block(stream, decode, 50, args.decode_launches)
        log(f"[bench] decode leg: {dec_ms * 1e3:.1f} us over {args.decode_launches} launches")
    for leg, cname, warm, n in (("c3", "c3_gqa_s8k_k2", 10, 20), ("c2", "c2_mha_s2k", 20, 100),
                                ("c1", "c1_mha_s128_d64", 20, 100)):
        if leg not in legs or cname == pcfg.name:
            continue
        cfg = workloads.CONFIGS[cname]
        bufs = prefill_inputs_on_device(cfg)
        ms = time_block(stream, prefill_fn(cfg, bufs), warm, n)
        configs[cname] = prefill_record(cfg, ms * 1e3, traffic_of(cname))
        configs[cname]["entry"] = prefill_entry(cfg)
        log(f"[bench] {cname}: {ms * 1e3:.1f} us ({configs[cname]['tflops']} TFLOP/s)")
        del bufs
        torch.cuda.empty_cache()
    d_us = (dec_ms if dec_ms is not None else dec_step_ms) * 1e3
    d_gbs = dec_bytes / (d_us * 1e-6) / 1e9
    d_traffic = read_traffic(f"dec_part_kernel_{dcfg.name}_counters.md", digest)
    configs[dcfg.name] = {
        "workload": (f"{dcfg.name}: decode B={B} Hq={Hq} Hkv={Hkv} D={D} Smax={Smax} lengths "
                     f"U[{dcfg.lmin},{dcfg.lmax}] (sum {sum_l}), split-KV in equal-work parts "
                     "+ LSE merge"),
        "us": round(d_us, 2),
        "us_in_step": round(dec_step_ms * 1e3, 2),
        "launches": args.decode_launches if dec_ms is not None else K,
        "gbs": round(d_gbs, 1),
        "frac_hbm_peak": round(d_gbs / PEAK_HBM_GBS, 4),
        "alg_bytes": dec_bytes,
        "tflops": round(16384 * sum_l / (d_us * 1e-6) / 1e12, 3),
        "counter_bytes": d_traffic,
        "counter_gbs": None if d_traffic is None else round(d_traffic / (d_us * 1e-6) / 1e9, 1),
    }

    extra = {}
    if "varlen" in legs:
        VL = dict(B=16, Hq=32, Hkv=8, D=128, lmin=256, lmax=8192, seed=1006)
        vq, vk, vv, vcu = workloads.varlen_inputs(**VL)
        vlens = (vcu[1:] - vcu[:-1]).tolist()
        vb = [(vq.to(dev), vk.to(dev), vv.to(dev), vcu.to(dev),
               torch.empty(vq.shape, device=dev, dtype=torch.bfloat16),
               torch.empty((VL["Hq"], vq.shape[0]), device=dev, dtype=torch.float32))
              for _ in range(2)]

        def prefill_varlen(i):
            q_, k_, v_, cu_, o_, l_ = vb[i & 1]
            mk.mk_attn_fwd_varlen(q_, k_, v_, o_, l_, cu_, cu_, VL["B"], VL["Hq"], VL["Hkv"],
                                  max(vlens), q_.shape[0], k_.shape[0], VL["D"], 1,
                                  VL["D"] ** -0.5, stream)
        ms = time_block(stream, prefill_varlen, 5, 20)
        v_flops = 4 * VL["D"] * VL["Hq"] * sum(L * (L + 1) // 2 for L in vlens)
        v_tf = v_flops / (ms * 1e-3) / 1e12
        extra["varlen_prefill"] = {
            "workload": (f"packed ragged causal prefill: B={VL['B']} sequences, lengths "
                         f"U[{VL['lmin']},{VL['lmax']}] (total {sum(vlens)} tokens), "
                         f"Hq={VL['Hq']} Hkv={VL['Hkv']} D={VL['D']}"),
            "value": round(v_tf, 2), "unit": "TFLOP/s", "us": round(ms * 1e3, 2),
            "flops": v_flops,
            "roofline": {"bound": "mfma", "achieved": round(v_tf, 2), "peak": PEAK_BF16_TFLOPS,
                         "unit": "TFLOP/s", "frac": round(v_tf / PEAK_BF16_TFLOPS, 4),
                         "traffic": None},
        }
        log(f"[bench] varlen prefill: {ms * 1e3:.1f} us")
        del vb, vq, vk, vv
    if "rpa" in legs:
        # prefill chunks and decode tokens over a paged cache in one call,
        # against the packed forward on the same keys gathered contiguously
        RP = workloads.RPA
        rseqs = workloads.ragged_paged_mix(RP["n_prefill"], RP["n_decode"], RP["seed"])
        rq, rkp, rvp, rbt, rcu, rlens, rkc, rvc = workloads.ragged_paged_inputs(
            rseqs, RP["Hq"], RP["Hkv"], RP["D"], RP["page_size"], RP["seed"], extra_pages=64)
        rk = torch.cat([rkc[b, :, :L].permute(1, 0, 2) for b, (_, L) in enumerate(rseqs)])
        rv = torch.cat([rvc[b, :, :L].permute(1, 0, 2) for b, (_, L) in enumerate(rseqs)])
        rck = torch.zeros(len(rseqs) + 1, dtype=torch.int32)
        rck[1:] = torch.cumsum(rlens, 0)
        del rkc, rvc
        max_sq = max(a for a, _ in rseqs)
        tq = int(rcu[-1])
        rb = [(rq.to(dev), rkp.to(dev), rvp.to(dev), rbt.to(dev), rcu.to(dev), rlens.to(dev),
               rk.contiguous().to(dev), rv.contiguous().to(dev), rck.to(dev),
               torch.empty(rq.shape, device=dev, dtype=torch.bfloat16),
               torch.empty((RP["Hq"], tq), device=dev, dtype=torch.float32)) for _ in range(2)]
        del rq, rkp, rvp, rk, rv

        def rpa(i):
            q_, kp_, vp_, bt_, cu_, ln_, _, _, _, o_, l_ = rb[i & 1]
            mk.mk_attn_fwd_ragged_paged(q_, kp_, vp_, bt_, o_, l_, cu_, ln_, len(rseqs), RP["Hq"],
                                        RP["Hkv"], max_sq, tq, RP["page_size"], bt_.shape[1],
                                        kp_.shape[0], RP["D"], 1, RP["D"] ** -0.5, stream)

        def rpa_gathered(i):
            q_, _, _, _, cu_, _, k_, v_, ck_, o_, l_ = rb[i & 1]
            mk.mk_attn_fwd_varlen(q_, k_, v_, o_, l_, cu_, ck_, len(rseqs), RP["Hq"], RP["Hkv"],
                                  max_sq, tq, k_.shape[0], RP["D"], 1, RP["D"] ** -0.5, stream)
        ms = time_block(stream, rpa, 5, 20)
        ms_g = time_block(stream, rpa_gathered, 5, 20)
        r_pairs = sum(sq * (L - sq) + sq * (sq + 1) // 2 for sq, L in rseqs)
        r_flops = 4 * RP["D"] * RP["Hq"] * r_pairs
        r_tf = r_flops / (ms * 1e-3) / 1e12
        extra["ragged_paged"] = {
            "workload": (f"{RP['name']}: {RP['n_prefill']} prefill chunks U[512,2048] after "
                         f"U[0,4096] context keys + {RP['n_decode']} decode tokens over U[512,4096] "
                         f"keys, {tq} query tokens, Hq={RP['Hq']} Hkv={RP['Hkv']} D={RP['D']}, "
                         f"{RP['page_size']}-key pages in a seeded random order, causal"),
            "value": round(r_tf, 2), "unit": "TFLOP/s", "us": round(ms * 1e3, 2),
            "us_packed_contiguous": round(ms_g * 1e3, 2), "flops": r_flops,
            "roofline": {"bound": "mfma", "achieved": round(r_tf, 2), "peak": PEAK_BF16_TFLOPS,
                         "unit": "TFLOP/s", "frac": round(r_tf / PEAK_BF16_TFLOPS, 4),
                         "traffic": None},
        }
        log(f"[bench] ragged paged: {ms * 1e3:.1f} us (packed contiguous {ms_g * 1e3:.1f} us)")
        del rb
        torch.cuda.empty_cache()
    if "paged" in legs:
        # the decode's keys scattered over pages in a seeded random order
        kp, vp, bt = workloads.paged_layout(kc, vc, args.page_size, seed=dcfg.seed + 7,
                                            extra_pages=64)
        pg = [(kp.to(dev), vp.to(dev), bt.to(dev)) for _ in range(2)]
        del kp, vp, bt

        def decode_paged(i):
            kp_, vp_, bt_ = pg[i & 1]
            mk.mk_attn_decode_paged(qd, kp_, vp_, bt_, od, lsed, B, Hq, Hkv, args.page_size,
                                    bt_.shape[1], kp_.shape[0], D, dcfg.scale, lens_d,
                                    args.parts, ws, ws_bytes, stream)
        ms = time_block(stream, decode_paged, 20, 100)
        p_gbs = dec_bytes / (ms * 1e-3) / 1e9
        extra["paged_decode"] = {
            "workload": (f"{dcfg.name} with its cache in {args.page_size}-key pages "
                         "in a seeded random order (block table)"),
            "value": round(p_gbs, 1), "unit": "GB/s", "us": round(ms * 1e3, 2),
            "roofline": {"bound": "hbm", "achieved": round(p_gbs, 1), "peak": PEAK_HBM_GBS,
                         "unit": "GB/s", "frac": round(p_gbs / PEAK_HBM_GBS, 4),
                         "traffic": None},
        }
        log(f"[bench] paged decode: {ms * 1e3:.1f} us")
        del pg
    del caches
    torch.cuda.empty_cache()
    if "bwd" in legs:
        # backward on the 2k workload's shape: the forward's bf16 O and LSE
        # (computed once, untimed), a seeded dO, two input copies
        bcfg = workloads.CONFIGS["c2_mha_s2k"]
        gb = torch.Generator().manual_seed(bcfg.seed + 11)
        dout = torch.randn((bcfg.B, bcfg.Hq, bcfg.S, bcfg.D), generator=gb).to(torch.bfloat16)
        bws_bytes = mk.mk_attn_bwd_workspace_bytes(bcfg.B, bcfg.Hq, bcfg.S)
        bb = []
        for q_, k_, v_, _, _ in prefill_inputs_on_device(bcfg):
            o_, lse_ = mk.fwd(q_, k_, v_, causal=True, scale=bcfg.scale)
            bb.append((q_, k_, v_, o_, lse_, dout.to(dev), torch.empty_like(q_),
                       torch.empty_like(k_), torch.empty_like(v_),
                       torch.empty(bws_bytes, device=dev, dtype=torch.uint8)))

        def backward(i):
            q_, k_, v_, o_, lse_, do_, dq_, dk_, dv_, bws_ = bb[i & 1]
            mk.mk_attn_bwd(q_, k_, v_, o_, do_, lse_, dq_, dk_, dv_, bcfg.B, bcfg.Hq, bcfg.Hkv,
                           bcfg.S, bcfg.S, bcfg.D, 1, bcfg.scale, None, bws_, bws_.numel(),
                           stream)
        ms = time_block(stream, backward, 10, 50)
        # the usual convention: 2.5 times the forward's FLOPs (five products
        # of the forward's size: S, dP, dV, dK, dQ)
        b_flops = 5 * bcfg.flops // 2
        b_tf = b_flops / (ms * 1e-3) / 1e12
        extra["backward"] = {
            "workload": (f"{bcfg.name} backward: dQ, dK, dV from O, LSE and a seeded dO, causal "
                         f"B={bcfg.B} Hq={bcfg.Hq} Hkv={bcfg.Hkv} S={bcfg.S} D={bcfg.D} bf16"),
            "value": round(b_tf, 2), "unit": "TFLOP/s", "us": round(ms * 1e3, 2),
            "flops": b_flops,
            "roofline": {"bound": "mfma", "achieved": round(b_tf, 2), "peak": PEAK_BF16_TFLOPS,
                         "unit": "TFLOP/s", "frac": round(b_tf / PEAK_BF16_TFLOPS, 4),
                         "traffic": read_traffic(f"bwd_kernels_{bcfg.name}_counters.md",
                                                 digest)},
        }
        log(f"[bench] backward: {ms * 1e3:.1f} us")
        del bb, dout
        torch.cuda.empty_cache()
    if "mla" in legs:
        MW = workloads.MLA
        mq, mckv, mlens = workloads.mla_inputs(MW["B"], MW["H"], MW["Dc"], MW["Dr"], MW["Smax"],
                                               MW["seed"], MW["lmin"], MW["lmax"])
        mws_bytes = mk.mk_attn_mla_decode_workspace_bytes(MW["H"], MW["Dc"], 0)
        mla_bytes = (int(mlens.clamp(0, MW["Smax"]).sum()) * (MW["Dc"] + MW["Dr"]) * 2
                     + MW["B"] * MW["H"] * ((MW["Dc"] + MW["Dr"]) * 2 + MW["Dc"] * 2 + 4))
        mb = [(mq.to(dev), mckv.to(dev), mlens.to(dev),
               torch.empty((MW["B"], MW["H"], MW["Dc"]), device=dev, dtype=torch.bfloat16),
               torch.empty((MW["B"], MW["H"]), device=dev, dtype=torch.float32),
               torch.empty(mws_bytes, device=dev, dtype=torch.uint8)) for _ in range(2)]
        del mq, mckv

        def mla_decode(i):
            mq_, mc_, ml_, mo_, mlse_, mws_ = mb[i & 1]
            mk.mk_attn_mla_decode(mq_, mc_, mo_, mlse_, MW["B"], MW["H"], MW["Dc"], MW["Dr"],
                                  MW["Smax"], MW["scale"], ml_, 0, mws_, mws_.numel(), stream)
        ms = time_block(stream, mla_decode, 20, 100)
        m_gbs = mla_bytes / (ms * 1e-3) / 1e9
        extra["mla_decode"] = {
            "workload": (f"{MW['name']}: MLA decode B={MW['B']} H={MW['H']} latent {MW['Dc']} + "
                         f"rotary {MW['Dr']}, lengths U[{MW['lmin']},{MW['lmax']}], shared "
                         "latent cache, split-KV (equal-work parts) + LSE merge"),
            "value": round(m_gbs, 1), "unit": "GB/s", "us": round(ms * 1e3, 2),
            "bytes": mla_bytes,
            "roofline": {"bound": "hbm", "achieved": round(m_gbs, 1), "peak": PEAK_HBM_GBS,
                         "unit": "GB/s", "frac": round(m_gbs / PEAK_HBM_GBS, 4),
                         "traffic": read_traffic(f"mla_part_kernel_{MW['name']}_counters.md",
                                                 digest)},
        }
        log(f"[bench] MLA decode: {ms * 1e3:.1f} us")
        del mb

    head = configs[pcfg.name]
    result = {
        "metric": "attention fwd TFLOP/s and % bf16 MFMA peak (prefill); HBM GB/s (decode)",
        "value": head["tflops"],
        "unit": "TFLOP/s",
        "n_gpus": 1,
        "steps": K,
        "warmup": args.warmup,
        "ms_per_step": round(ms_step, 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16",
        "data": "synthetic (seeded N(0,1) bf16, generated on the host, resident in HBM)",
        "config": {
            "workload": (f"{head['workload']} + fp32 LSE; then {configs[dcfg.name]['workload']}"),
            "prefill_entry": configs[pcfg.name]["entry"],
            "prefill_flops_per_step": pcfg.flops,
            "decode_bytes_per_step": dec_bytes,
            "decode_sum_kv_len": sum_l,
            "kernel_source_digest": digest,
        },
        "prefill_us": head["us"],
        "roofline": {
            "bound": "mfma",
            "achieved": head["tflops"],
            "peak": PEAK_BF16_TFLOPS,
            "unit": "TFLOP/s",
            "frac": head["frac_mfma_peak"],
            "traffic": head["counter_bytes"],
        },
        "decode": {
            "value": configs[dcfg.name]["gbs"],
            "unit": "GB/s",
            "us": configs[dcfg.name]["us"],
            "roofline": {
                "bound": "hbm",
                "achieved": configs[dcfg.name]["gbs"],
                "peak": PEAK_HBM_GBS,
                "unit": "GB/s",
                "frac": configs[dcfg.name]["frac_hbm_peak"],
                "traffic": d_traffic,
            },
        },
        "configs": configs,
        "cpu_baseline": None,
    }
    result.update(extra)
    if args.cpu_baseline != "none":
        result["cpu_baseline"] = cpu_baselines(args, sum_l)
    print(json.dumps(result), flush=True)


if __name__ == "__main__":
    main()
