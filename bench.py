"""Benchmark of the attention hot path on one MI355X.

One step = one pass over the whole path on resident synthetic inputs:
  * the fused causal attention forward on the prefill workload
    (causal MHA B=4 H=16 S=2048 D=128 bf16 by default), then
  * the split-KV decode (equal-work part kernel + LSE merge kernel) on the
    ragged decode batch (B=64 Hq=32 Hkv=8 D=128, lengths in [512, 4096]).
Each workload alternates between two copies of its inputs so the 256 MB
last-level cache cannot hand one launch the previous launch's data.

The K timed steps run as K prefill launches back to back, then K decode
launches back to back, on torch's current stream; HIP events recorded on
that stream before, between and after give each kernel's average launch
duration.  Prints ONE JSON line on stdout; progress goes to stderr.
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
    try:
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
            key = f"{key} [{wgs} workgroups]"
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


def _pmc_per_kernel(path: str, counter: str):
    import sqlite3
    db = sqlite3.connect(_find_db(path))
    rows = db.execute("select dispatch_id, name, counter_name, counter_value from pmc_events "
                      "where counter_name = ?", (counter,)).fetchall()
    per_disp = {}
    for disp, name, _, val in rows:
        key = (disp, _short(name))
        per_disp[key] = per_disp.get(key, 0.0) + val
    per_kernel = {}
    for (disp, name), val in per_disp.items():
        per_kernel.setdefault(name, []).append(val)
    return per_kernel


def summarize_pmc(fetch_path: str, write_path: str, kernels, calib_bytes: int,
                  commands) -> str:
    """Per-launch HBM bytes of `kernels` (summed: one launch of the path)
    from FETCH_SIZE / WRITE_SIZE runs, each scaled by what the counter reads
    for the plain device copy of calib_bytes in the same run."""
    fetch = _pmc_per_kernel(fetch_path, "FETCH_SIZE")
    write = _pmc_per_kernel(write_path, "WRITE_SIZE")
    copy = [k for k in fetch if "copyBuffer" in k]
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
        name = [n for n in fetch if k in n]
        if not name:
            raise SystemExit(f"kernel {k} not in the counter runs")
        fv, wv = fetch[name[0]], write[name[0]]
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
            for (name, counter), v in counter_rows.items():
                if kernel in name:
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
    import sqlite3
    db = sqlite3.connect(_find_db(path))
    rows = db.execute("select dispatch_id, name, counter_name, counter_value from pmc_events"
                      ).fetchall()
    per_disp = {}
    for disp, name, counter, val in rows:
        key = (disp, _short(name), counter)
        per_disp[key] = per_disp.get(key, 0.0) + val
    out = {}
    for (disp, name, counter), val in per_disp.items():
        out.setdefault((name, counter), []).append(val)
    return out


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=100)
    ap.add_argument("--warmup", type=int, default=20)
    ap.add_argument("--prefill", default="c2_mha_s2k")
    ap.add_argument("--decode", default="c5_decode_b64")
    ap.add_argument("--parts", type=int, default=0, help="decode parts (0 = library default)")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--page-size", type=int, default=16,
                    help="page size of the paged-decode leg (0 skips the leg)")
    ap.add_argument("--no-varlen", action="store_true",
                    help="skip the packed ragged prefill leg")
    ap.add_argument("--no-bwd", action="store_true",
                    help="skip the backward leg (dQ, dK, dV on the prefill shape)")
    ap.add_argument("--no-mla", action="store_true", help="skip the MLA decode leg")
    ap.add_argument("--long", default="c4_gqa_s32k",
                    help="workload of the long-context prefill leg ('' skips the leg)")
    ap.add_argument("--cpu-rows", type=int, default=0,
                    help="query rows per head timed for the CPU oracle baseline (0: all)")
    ap.add_argument("--calib-copy-mib", type=int, default=0,
                    help="also run one plain device copy of this size (counter calibration)")
    ap.add_argument("--summarize-trace", metavar="DIR",
                    help="print a summary of a rocprofv3 --kernel-trace output and exit")
    ap.add_argument("--summarize-pmc", nargs=2, metavar=("FETCH_DIR", "WRITE_DIR"),
                    help="print per-launch HBM bytes from FETCH_SIZE / WRITE_SIZE runs and exit")
    ap.add_argument("--summarize-sq", nargs="+", metavar="DIR",
                    help="print SQ/GRBM counters of --kernels (one name) from --pmc runs and exit")
    ap.add_argument("--kernels", default=None,
                    help="semicolon-separated kernel name fragments for --summarize-pmc "
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

    import numpy as np
    import torch

    import paper_2609_04523_amd as mk
    import workloads

    if not os.path.exists(mk.LIB_PATH):
        from paper_2609_04523_amd import build as hip_build
        hip_build.build()
    mk.lib()
    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)

    pcfg = workloads.CONFIGS[args.prefill]
    dcfg = workloads.CONFIGS[args.decode]
    log(f"[bench] inputs: prefill {pcfg.name}, decode {dcfg.name}")
    q, k, v = workloads.config_inputs(pcfg)
    # two copies of the prefill tensors, used alternately, so that the
    # 256 MB last-level cache cannot hand one launch the previous one's data
    pre = []
    for _ in range(2):
        o = torch.empty(q.shape, device=dev,
                        dtype=torch.float32 if pcfg.out_fp32 else torch.bfloat16)
        lse = torch.empty(q.shape[:3], device=dev, dtype=torch.float32)
        pre.append((q.to(dev), k.to(dev), v.to(dev), o, lse))
    del q, k, v
    qd, kc, vc, lens = workloads.config_inputs(dcfg)
    caches = [(kc.to(dev), vc.to(dev)), (kc.to(dev).clone(), vc.to(dev).clone())]
    # packed ragged prefill batch: 16 causal sequences, lengths U{256..8192}
    VL = dict(B=16, Hq=32, Hkv=8, D=128, lmin=256, lmax=8192, seed=1006)
    varlen = []
    if not args.no_varlen:
        vq, vk, vv, vcu = workloads.varlen_inputs(**VL)
        vlens = (vcu[1:] - vcu[:-1]).tolist()
        varlen = [(vq.to(dev), vk.to(dev), vv.to(dev), vcu.to(dev),
                   torch.empty(vq.shape, device=dev, dtype=torch.bfloat16),
                   torch.empty((VL["Hq"], vq.shape[0]), device=dev, dtype=torch.float32))
                  for _ in range(2)]
        del vq, vk, vv
    paged = []
    if args.page_size:
        # the same keys scattered over pages in a seeded random order (two
        # copies of the pools, used alternately like the caches above)
        kp, vp, bt = workloads.paged_layout(kc, vc, args.page_size, seed=dcfg.seed + 7,
                                            extra_pages=64)
        paged = [(kp.to(dev), vp.to(dev), bt.to(dev)) for _ in range(2)]
        del kp, vp, bt
    bwd = []
    if not args.no_bwd:
        # backward on the prefill shape: the forward's bf16 O and LSE
        # (computed once, untimed), a seeded dO, two input copies
        gb = torch.Generator().manual_seed(pcfg.seed + 11)
        dout = torch.randn((pcfg.B, pcfg.Hq, pcfg.S, pcfg.D), generator=gb).to(torch.bfloat16)
        bws_bytes = mk.mk_attn_bwd_workspace_bytes(pcfg.B, pcfg.Hq, pcfg.S)
        for i in range(2):
            q_, k_, v_ = pre[i][:3]
            o_, lse_ = mk.fwd(q_, k_, v_, causal=pcfg.causal, scale=pcfg.scale)
            bwd.append((q_, k_, v_, o_, lse_, dout.to(dev), torch.empty_like(q_),
                        torch.empty_like(k_), torch.empty_like(v_),
                        torch.empty(bws_bytes, device=dev, dtype=torch.uint8)))
        del dout
    mla = []
    MW = workloads.MLA
    if not args.no_mla:
        # MLA decode: 64 sequences, 16 heads, latent 512 + rotary 64; two
        # copies of the latent cache, used alternately
        mq, mckv, mlens = workloads.mla_inputs(MW["B"], MW["H"], MW["Dc"], MW["Dr"], MW["Smax"],
                                               MW["seed"], MW["lmin"], MW["lmax"])
        mws_bytes = mk.mk_attn_mla_decode_workspace_bytes(MW["H"], MW["Dc"], 0)
        mla_bytes = (int(mlens.clamp(0, MW["Smax"]).sum()) * (MW["Dc"] + MW["Dr"]) * 2
                     + MW["B"] * MW["H"] * ((MW["Dc"] + MW["Dr"]) * 2 + MW["Dc"] * 2 + 4))
        mla = [(mq.to(dev), mckv.to(dev) if i == 0 else mckv.to(dev).clone(), mlens.to(dev),
                torch.empty((MW["B"], MW["H"], MW["Dc"]), device=dev, dtype=torch.bfloat16),
                torch.empty((MW["B"], MW["H"]), device=dev, dtype=torch.float32),
                torch.empty(mws_bytes, device=dev, dtype=torch.uint8)) for i in range(2)]
        del mq, mckv
    del kc, vc
    qd = qd.to(dev)
    lens_d = lens.to(dev)
    B, Hq, D = qd.shape
    Hkv, Smax = dcfg.Hkv, dcfg.Smax
    ws_bytes = mk.mk_attn_decode_workspace_bytes(Hq, Hkv, D, args.parts)
    ws = torch.empty(ws_bytes, device=dev, dtype=torch.uint8)
    od = torch.empty((B, Hq, D), device=dev, dtype=torch.bfloat16)
    lsed = torch.empty((B, Hq), device=dev, dtype=torch.float32)
    torch.cuda.synchronize()

    fwd_entry = mk.mk_attn_fwd_o32 if pcfg.out_fp32 else mk.mk_attn_fwd
    stream = torch.cuda.current_stream()

    def prefill(i):
        q, k, v, o, lse = pre[i & 1]
        fwd_entry(q, k, v, o, lse, pcfg.B, pcfg.Hq, pcfg.Hkv, pcfg.S, pcfg.S, pcfg.D, 1,
                  pcfg.scale, None, stream)

    def decode(i):
        kcc, vcc = caches[i & 1]
        mk.mk_attn_decode(qd, kcc, vcc, od, lsed, B, Hq, Hkv, Smax, D, dcfg.scale, lens_d,
                          args.parts, ws, ws_bytes, stream)

    def prefill_varlen(i):
        vq_, vk_, vv_, vcu_, vo_, vl_ = varlen[i & 1]
        mk.mk_attn_fwd_varlen(vq_, vk_, vv_, vo_, vl_, vcu_, vcu_, VL["B"], VL["Hq"], VL["Hkv"],
                              max(vlens), vq_.shape[0], vk_.shape[0], VL["D"], 1,
                              VL["D"] ** -0.5, stream)

    def backward(i):
        q_, k_, v_, o_, lse_, do_, dq_, dk_, dv_, bws_ = bwd[i & 1]
        mk.mk_attn_bwd(q_, k_, v_, o_, do_, lse_, dq_, dk_, dv_, pcfg.B, pcfg.Hq, pcfg.Hkv,
                       pcfg.S, pcfg.S, pcfg.D, int(pcfg.causal), pcfg.scale, None, bws_,
                       bws_.numel(), stream)

    def mla_decode(i):
        mq_, mc_, ml_, mo_, mlse_, mws_ = mla[i & 1]
        mk.mk_attn_mla_decode(mq_, mc_, mo_, mlse_, MW["B"], MW["H"], MW["Dc"], MW["Dr"],
                              MW["Smax"], MW["scale"], ml_, 0, mws_, mws_.numel(), stream)

    def decode_paged(i):
        kp_, vp_, bt_ = paged[i & 1]
        mk.mk_attn_decode_paged(qd, kp_, vp_, bt_, od, lsed, B, Hq, Hkv, args.page_size,
                                bt_.shape[1], kp_.shape[0], D, dcfg.scale, lens_d, args.parts,
                                ws, ws_bytes, stream)

    if args.calib_copy_mib:
        n = args.calib_copy_mib << 20
        src = torch.empty(n, device=dev, dtype=torch.uint8).fill_(1)
        dst = torch.empty_like(src)
        torch.cuda.synchronize()
        dst.copy_(src)
        torch.cuda.synchronize()
        log(f"[bench] calibration copy of {n} bytes done")
        del src, dst

    log(f"[bench] warmup {args.warmup}")
    for i in range(args.warmup):
        prefill(i)
        decode(i)
    torch.cuda.synchronize()

    K = args.steps
    # The K steps run as K prefill launches back to back, then K decode
    # launches back to back (each alternating its two input copies), with
    # one event before, between and after: a marker between two kernels
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
    varlen_ms = None
    if varlen:
        # the packed ragged prefill leg, timed after the step the same way
        for i in range(args.warmup):
            prefill_varlen(i)
        evv = [torch.cuda.Event(enable_timing=True) for _ in range(2)]
        torch.cuda.synchronize()
        evv[0].record(stream)
        for i in range(K):
            prefill_varlen(i)
        evv[1].record(stream)
        torch.cuda.synchronize()
        varlen_ms = evv[0].elapsed_time(evv[1]) / K
    paged_ms = None
    if paged:
        # the paged-decode leg, timed after the step the same way
        for i in range(args.warmup):
            decode_paged(i)
        evp = [torch.cuda.Event(enable_timing=True) for _ in range(2)]
        torch.cuda.synchronize()
        evp[0].record(stream)
        for i in range(K):
            decode_paged(i)
        evp[1].record(stream)
        torch.cuda.synchronize()
        paged_ms = evp[0].elapsed_time(evp[1]) / K
    bwd_ms = None
    if bwd:
        # the backward leg, timed after the step the same way
        for i in range(args.warmup):
            backward(i)
        evb = [torch.cuda.Event(enable_timing=True) for _ in range(2)]
        torch.cuda.synchronize()
        evb[0].record(stream)
        for i in range(K):
            backward(i)
        evb[1].record(stream)
        torch.cuda.synchronize()
        bwd_ms = evb[0].elapsed_time(evb[1]) / K
    mla_ms = None
    if mla:
        # the MLA decode leg, timed after the step the same way
        for i in range(args.warmup):
            mla_decode(i)
        evm = [torch.cuda.Event(enable_timing=True) for _ in range(2)]
        torch.cuda.synchronize()
        evm[0].record(stream)
        for i in range(K):
            mla_decode(i)
        evm[1].record(stream)
        torch.cuda.synchronize()
        mla_ms = evm[0].elapsed_time(evm[1]) / K
    long_ms, lcfg = None, None
    if args.long:
        # the long-context prefill leg: the same kernel on a long causal
        # workload (two input copies alternating), a few launches after two
        # untimed ones, timed after the step the same way
        lcfg = workloads.CONFIGS[args.long]
        lq, lk, lv = workloads.config_inputs(lcfg)
        lin = []
        for _ in range(2):
            lin.append((lq.to(dev), lk.to(dev), lv.to(dev),
                        torch.empty(lq.shape, device=dev,
                                    dtype=torch.float32 if lcfg.out_fp32 else torch.bfloat16),
                        torch.empty(lq.shape[:3], device=dev, dtype=torch.float32)))
        del lq, lk, lv
        lentry = mk.mk_attn_fwd_o32 if lcfg.out_fp32 else mk.mk_attn_fwd

        def long_prefill(i):
            q_, k_, v_, o_, l_ = lin[i & 1]
            lentry(q_, k_, v_, o_, l_, lcfg.B, lcfg.Hq, lcfg.Hkv, lcfg.S, lcfg.S, lcfg.D, 1,
                   lcfg.scale, None, stream)
        for i in range(2):
            long_prefill(i)
        KL = max(2, min(K, 10))
        evl = [torch.cuda.Event(enable_timing=True) for _ in range(2)]
        torch.cuda.synchronize()
        evl[0].record(stream)
        for i in range(KL):
            long_prefill(i)
        evl[1].record(stream)
        torch.cuda.synchronize()
        long_ms = evl[0].elapsed_time(evl[1]) / KL
        del lin
        torch.cuda.empty_cache()
    ms_step = (t1 - t0) * 1e3 / K
    pre_ms = ev[0].elapsed_time(ev[1]) / K  # average launch duration
    dec_ms = ev[1].elapsed_time(ev[2]) / K
    flops = pcfg.flops
    tflops = flops / (pre_ms * 1e-3) / 1e12
    sum_l = int(lens.clamp(0, Smax).sum())
    dec_bytes = 4 * D * Hkv * sum_l + (B * Hq * D * 2) * 2 + B * Hq * 4  # K+V, q, o, lse
    dec_gbs = dec_bytes / (dec_ms * 1e-3) / 1e9
    log(f"[bench] prefill {pre_ms * 1e3:.1f} us ({tflops:.1f} TFLOP/s), "
        f"decode {dec_ms * 1e3:.1f} us ({dec_gbs:.1f} GB/s), step {ms_step:.3f} ms"
        + (f", varlen prefill {varlen_ms * 1e3:.1f} us" if varlen_ms is not None else "")
        + (f", paged decode {paged_ms * 1e3:.1f} us" if paged_ms is not None else "")
        + (f", backward {bwd_ms * 1e3:.1f} us" if bwd_ms is not None else "")
        + (f", MLA decode {mla_ms * 1e3:.1f} us" if mla_ms is not None else "")
        + (f", long prefill {long_ms * 1e3:.1f} us" if long_ms is not None else ""))

    digest = kernel_source_digest()
    traffic_pre = read_traffic(f"fwd_kernel_{pcfg.name}_counters.md", digest)
    traffic_dec = read_traffic(f"dec_part_kernel_{dcfg.name}_counters.md", digest)

    result = {
        "metric": "attention fwd TFLOP/s and % bf16 MFMA peak (prefill); HBM GB/s (decode)",
        "value": round(tflops, 2),
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
            "workload": (f"{pcfg.name}: causal attention fwd B={pcfg.B} Hq={pcfg.Hq} "
                         f"Hkv={pcfg.Hkv} S={pcfg.S} D={pcfg.D} bf16 in, "
                         f"{'fp32' if pcfg.out_fp32 else 'bf16'} O + fp32 LSE; then "
                         f"{dcfg.name}: decode B={B} Hq={Hq} Hkv={Hkv} D={D} "
                         f"lengths U[{dcfg.lmin},{dcfg.lmax}] split-KV (equal-work parts) + LSE merge"),
            "prefill_flops_per_step": flops,
            "decode_bytes_per_step": dec_bytes,
            "decode_sum_kv_len": sum_l,
            "kernel_source_digest": digest,
        },
        "prefill_us": round(pre_ms * 1e3, 2),
        "roofline": {
            "bound": "mfma",
            "achieved": round(tflops, 2),
            "peak": PEAK_BF16_TFLOPS,
            "unit": "TFLOP/s",
            "frac": round(tflops / PEAK_BF16_TFLOPS, 4),
            "traffic": traffic_pre,
        },
        "decode": {
            "value": round(dec_gbs, 1),
            "unit": "GB/s",
            "us": round(dec_ms * 1e3, 2),
            "roofline": {
                "bound": "hbm",
                "achieved": round(dec_gbs, 1),
                "peak": PEAK_HBM_GBS,
                "unit": "GB/s",
                "frac": round(dec_gbs / PEAK_HBM_GBS, 4),
                "traffic": traffic_dec,
            },
        },
        "cpu_baseline": None,
    }
    if varlen_ms is not None:
        # causal pairs counted exactly: S (S + 1) / 2 per sequence and head
        v_flops = 4 * VL["D"] * VL["Hq"] * sum(L * (L + 1) // 2 for L in vlens)
        v_tf = v_flops / (varlen_ms * 1e-3) / 1e12
        result["varlen_prefill"] = {
            "workload": (f"packed ragged causal prefill: B={VL['B']} sequences, lengths "
                         f"U[{VL['lmin']},{VL['lmax']}] (total {sum(vlens)} tokens), "
                         f"Hq={VL['Hq']} Hkv={VL['Hkv']} D={VL['D']}"),
            "value": round(v_tf, 2),
            "unit": "TFLOP/s",
            "us": round(varlen_ms * 1e3, 2),
            "flops": v_flops,
            "roofline": {"bound": "mfma", "achieved": round(v_tf, 2), "peak": PEAK_BF16_TFLOPS,
                         "unit": "TFLOP/s", "frac": round(v_tf / PEAK_BF16_TFLOPS, 4),
                         "traffic": None},
        }
    if paged_ms is not None:
        p_gbs = dec_bytes / (paged_ms * 1e-3) / 1e9
        result["paged_decode"] = {
            "workload": (f"{dcfg.name} with its cache in {args.page_size}-key pages "
                         "in a seeded random order (block table)"),
            "value": round(p_gbs, 1),
            "unit": "GB/s",
            "us": round(paged_ms * 1e3, 2),
            "roofline": {"bound": "hbm", "achieved": round(p_gbs, 1), "peak": PEAK_HBM_GBS,
                         "unit": "GB/s", "frac": round(p_gbs / PEAK_HBM_GBS, 4),
                         "traffic": None},
        }

    if bwd_ms is not None:
        # the usual convention for attention backward: 2.5 times the
        # forward's FLOPs (five products of the forward's size: S, dP, dV,
        # dK, dQ); the dQ kernel recomputes S and dP, which is not counted
        b_flops = 5 * pcfg.flops // 2
        b_tf = b_flops / (bwd_ms * 1e-3) / 1e12
        result["backward"] = {
            "workload": (f"{pcfg.name} backward: dQ, dK, dV from O, LSE and a seeded dO, "
                         f"{'causal' if pcfg.causal else 'non-causal'} B={pcfg.B} Hq={pcfg.Hq} "
                         f"Hkv={pcfg.Hkv} S={pcfg.S} D={pcfg.D} bf16"),
            "value": round(b_tf, 2),
            "unit": "TFLOP/s",
            "us": round(bwd_ms * 1e3, 2),
            "flops": b_flops,
            "roofline": {"bound": "mfma", "achieved": round(b_tf, 2), "peak": PEAK_BF16_TFLOPS,
                         "unit": "TFLOP/s", "frac": round(b_tf / PEAK_BF16_TFLOPS, 4),
                         "traffic": None},
        }

    if mla_ms is not None:
        m_gbs = mla_bytes / (mla_ms * 1e-3) / 1e9
        result["mla_decode"] = {
            "workload": (f"{MW['name']}: MLA decode B={MW['B']} H={MW['H']} latent {MW['Dc']} + "
                         f"rotary {MW['Dr']}, lengths U[{MW['lmin']},{MW['lmax']}], shared "
                         "latent cache, split-KV (equal-work parts) + LSE merge"),
            "value": round(m_gbs, 1),
            "unit": "GB/s",
            "us": round(mla_ms * 1e3, 2),
            "bytes": mla_bytes,
            "roofline": {"bound": "hbm", "achieved": round(m_gbs, 1), "peak": PEAK_HBM_GBS,
                         "unit": "GB/s", "frac": round(m_gbs / PEAK_HBM_GBS, 4),
                         "traffic": None},
        }

    if long_ms is not None:
        l_tf = lcfg.flops / (long_ms * 1e-3) / 1e12
        result["long_prefill"] = {
            "workload": (f"{lcfg.name}: causal attention fwd B={lcfg.B} Hq={lcfg.Hq} "
                         f"Hkv={lcfg.Hkv} S={lcfg.S} D={lcfg.D} bf16"),
            "value": round(l_tf, 2),
            "unit": "TFLOP/s",
            "us": round(long_ms * 1e3, 1),
            "roofline": {"bound": "mfma", "achieved": round(l_tf, 2), "peak": PEAK_BF16_TFLOPS,
                         "unit": "TFLOP/s", "frac": round(l_tf / PEAK_BF16_TFLOPS, 4),
                         "traffic": None},
        }

    if not args.no_cpu_baseline:
        from oracle import oracle as orc  # timed CPU baseline only
        qh, kh, vh = workloads.config_inputs(pcfg)
        qb, kb, vb = workloads.bits(qh), workloads.bits(kh), workloads.bits(vh)
        threads = orc.default_threads()
        if args.cpu_rows and args.cpu_rows < pcfg.S:
            rows = workloads.sample_rows(pcfg.B, pcfg.Hq, pcfg.S, args.cpu_rows,
                                         seed=pcfg.seed + 7)
            pairs = int((rows.long() + 1).sum())  # causal row i sees i+1 keys
            rows_np, what = rows.numpy(), f"{args.cpu_rows} seeded query rows per head"
        else:
            rows_np, what = None, "every query row"
            pairs = pcfg.B * pcfg.Hq * pcfg.pairs_per_head
        log(f"[bench] cpu oracle baseline: {what} on {threads} threads")
        c0 = time.perf_counter()
        orc.attn_fwd(qb, kb, vb, causal=True, scale=pcfg.scale, rows=rows_np, threads=threads)
        c1 = time.perf_counter()
        cpu_tflops = 4 * pcfg.D * pairs / (c1 - c0) / 1e12
        result["cpu_baseline"] = {
            "value": cpu_tflops,
            "unit": "TFLOP/s",
            "cores": threads,
            "kind": "oracle",
            "sample": (f"{what} of {pcfg.name} ({pairs} query-key pairs, fp64, "
                       f"{c1 - c0:.2f} s)"),
        }
    print(json.dumps(result), flush=True)


if __name__ == "__main__":
    main()
