#!/usr/bin/env python3
"""Benchmark of the dataset-decomposition attention hot path on one MI355X.

A bench step runs causal attention forward + backward (through the C ABI)
over every launch group of the chosen workload; each group is one
65,536-token training step, so per group B * L = 65536.

Workloads (``--workload``):
  dd_sweep_d64   (default) buckets L = 256 .. 8192, B = 65536 / L, H = 16, D = 64
  dd_sweep_d128  the same with D = 128
  chunk_vs_dd    8 x 8192 chunks of log-normal documents: dense causal,
                 document-masked, the DD buckets of the same documents (one
                 launch per bucket), and the same DD pieces packed into one
                 document-masked launch
  stream         64 steps with L drawn from 256 .. 16384, weights 1/L, D = 128
  curriculum     48 steps of the length curriculum of Algorithm 1 ("Grow-P2"
                 odds, 8 cycles, equal tokens from buckets 256 .. 8192), D = 128
  rope_d128      dd_sweep_d128 with rotary position embedding (base 100,000):
                 q and k rotated by dd_rope before the forward, dq and dk
                 rotated back in the backward kernels
  rope_d128_fused  the same, with q rotated inside the forward as it is
                 loaded (dd_attn_fwd_rope, which also writes the rotated q
                 for the backward); k still by dd_rope
  layer_1b       one OpenLM-1B block (d 2048, 16 heads, SwiGLU 5632, RoPE)
                 forward + backward per bucket L = 256 .. 8192 at 65,536
                 tokens: step time, attention's share of it, and the fit
                 t(L) = alpha + beta * L (value: block TFLOP/s)
  gemm_1b        the bf16 GEMMs of one OpenLM-1B block step at 65,536 tokens
                 (forward, input-gradient and weight-gradient shapes), the
                 library's dd_gemm timed beside torch.matmul (the vendor
                 library) on the same operands
  tiny           B = 4, L = 256, H = 4, D = 64

Prints ONE JSON line on stdout: the metric is useful attention TFLOP/s
(forward 4*D and backward 10*D FLOPs per allowed (query, key) pair and head)
over the whole bench step, with per-group times, tokens/s and per-kernel
launch times, per-length efficiency where lengths repeat (stream,
curriculum), the roofline of the dominant kernel launch (the kernel and
group with the largest total time in the timed region, timed with HIP events
on the kernel's own stream) and the fp64 CPU oracle timed on a bounded
sample of every group of the workload.

The default run (dd_sweep_d64 over every bucket) also times, after its own
timed region, the D = 128 sweep and the concat-and-chunk vs DD comparison
(``extra_workloads``; ``--no-extras`` skips them), and reports the L = 8192
buckets of both sweeps in ``roofline.bucket_8192``.

``--traffic-summary FETCH_DIR WRITE_DIR`` instead turns two rocprofv3 counter
runs of this script (``--pmc FETCH_SIZE``, then ``--pmc WRITE_SIZE``, each
with ``--copy-calibration``) into the HBM traffic per (kernel, group) that
``profiles/traffic_<workload>.txt`` holds.
"""
from __future__ import annotations

import argparse
import ctypes
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

ROPE_BASE = 100000.0
TOKENS = 65536
BF16_PEAK_TFLOPS = 2500.0   # MI355X dense bf16 matrix-core peak
HBM_PEAK_GBS = 8000.0       # MI355X HBM3E
METRIC = "attention fwd+bwd TFLOP/s and tokens/s per bucket at 65,536 tokens/step"
BUCKETS = [256, 512, 1024, 2048, 4096, 8192]
# D = 64 rows of at most this many tokens (without RoPE) run the one-kernel
# backward.
SHORT_MAX_ROW = 256


def log(msg):
    print(msg, file=sys.stderr, flush=True)


def kernel_source_hash():
    """sha256 of the HIP sources and the build script, with comments and
    white space removed: counter-based traffic is void once the code or its
    compile flags change (comment edits leave it valid)."""
    import glob
    import hashlib
    import re
    h = hashlib.sha256()
    csrc = os.path.join(ROOT, "paper_2405_13226_amd", "csrc")
    build = os.path.join(ROOT, "paper_2405_13226_amd", "build.py")
    for f in sorted(glob.glob(os.path.join(csrc, "*.hip")) + glob.glob(os.path.join(csrc, "*.hpp"))) \
            + [build]:
        with open(f, encoding="utf-8") as fh:
            code = fh.read()
        if f == build:
            code = re.sub(r"#[^\n]*", " ", code)
        else:
            code = re.sub(r"/\*.*?\*/", " ", code, flags=re.S)
            code = re.sub(r"//[^\n]*", " ", code)
        code = " ".join(code.split())
        h.update(os.path.basename(f).encode() + b"\0" + code.encode())
    return h.hexdigest()[:16]


class SclkSampler:
    """Samples the GPU shader clock's current DPM level (sysfs pp_dpm_sclk,
    the line marked '*') every 10 ms while the timed region runs; summary()
    is {mean, min, max, samples} in MHz, or None where sysfs is unavailable."""

    def __init__(self, period=0.01):
        import glob
        import threading
        self.paths = sorted(glob.glob("/sys/class/drm/card*/device/pp_dpm_sclk"))
        self.period, self.samples = period, []
        self.stop = threading.Event()
        self.thread = threading.Thread(target=self._run, daemon=True)

    def _read(self):
        for path in self.paths:
            try:
                with open(path) as fh:
                    for line in fh:
                        if line.rstrip().endswith("*"):
                            return float(line.split()[1].lower().rstrip("mhz"))
            except (OSError, ValueError, IndexError):
                continue
        return None

    def _run(self):
        while not self.stop.wait(self.period):
            v = self._read()
            if v is not None:
                self.samples.append(v)

    def __enter__(self):
        if self.paths:
            self.thread.start()
        return self

    def __exit__(self, *exc):
        self.stop.set()
        if self.paths:
            self.thread.join()

    def summary(self):
        if not self.samples:
            return None
        v = self.samples
        return dict(mean=round(sum(v) / len(v), 1), min=min(v), max=max(v), samples=len(v))


def measured_traffic(workload, kernel, group=None):
    """HBM bytes per launch of `kernel` (in `group`, if given) from
    profiles/traffic_<workload>.txt (key = value lines), or None if absent,
    for another kernel or group, or taken on other kernel sources."""
    path = os.path.join(ROOT, "profiles", f"traffic_{workload}.txt")
    if not os.path.exists(path):
        return None
    kv = {}
    with open(path) as f:
        for line in f:
            if "=" in line and not line.lstrip().startswith("#"):
                k, v = line.rsplit("=", 1)  # group names may hold "=" ("L=8192")
                kv[k.strip()] = v.strip()
    if kv.get("source_hash") != kernel_source_hash():
        return None
    key = f"bytes_per_launch.{kernel}" + (f".{group}" if group else "")
    return int(float(kv[key])) if key in kv else None


def parse():
    ap = argparse.ArgumentParser(description=__doc__.splitlines()[0])
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=10)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--workload", default="dd_sweep_d64",
                    choices=["dd_sweep_d64", "dd_sweep_d128", "chunk_vs_dd", "stream",
                             "curriculum", "rope_d128", "rope_d128_fused", "layer_1b", "gemm_1b",
                             "tiny"])
    ap.add_argument("--buckets", default=None,
                    help="comma-separated subset of bucket lengths (sweeps only)")
    ap.add_argument("--seed", type=int, default=0)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--cpu-seconds", type=float, default=15.0,
                    help="target CPU time of the oracle sample")
    ap.add_argument("--events", default="inline", choices=["inline", "separate"],
                    help="time groups/kernels with events inside the timed region, or in "
                         "a second pass after a clean one")
    ap.add_argument("--copy-calibration", action="store_true",
                    help="before warmup, copy 1 GiB on the device 3 times (a kernel of known "
                         "traffic that scales FETCH_SIZE / WRITE_SIZE counter runs)")
    ap.add_argument("--no-extras", action="store_true",
                    help="default run only: skip the D=128 sweep and chunk_vs_dd extras")
    ap.add_argument("--sq-summary", nargs=2, metavar=("PASS1_DIR", "PASS2_DIR"),
                    help="print the SQ counter table of two rocprofv3 counter runs and exit")
    ap.add_argument("--traffic-summary", nargs=2, metavar=("FETCH_DIR", "WRITE_DIR"),
                    help="summarise two rocprofv3 counter runs of this script (no GPU use)")
    return ap.parse_args()


# ---------------------------------------------------------------------------
# workloads: a list of launch groups {name, B, L, cu (host int32 or None)}
# ---------------------------------------------------------------------------
def workload(name, seed, buckets=None):
    import numpy as np
    import synth
    from paper_2405_13226_amd import dd

    if name in ("dd_sweep_d64", "dd_sweep_d128"):
        H, D = 16, 64 if name.endswith("64") else 128
        lens = buckets or BUCKETS
        groups = [dict(name=f"L={L}", B=TOKENS // L, L=L, cu=None) for L in lens]
        desc = dict(workload=name, tokens_per_group=TOKENS, buckets=lens, H=H, D=D,
                    causal=True)
    elif name in ("rope_d128", "rope_d128_fused"):
        # The D=128 sweep with rotary position embedding (base 100,000, the
        # paper's curriculum runs): the forward rotates q and k (two dd_rope
        # launches) before attention; the backward rotates dq and dk back in
        # its kernels' epilogues (dd_attn_bwd_rope).
        H, D = 16, 128
        lens = buckets or BUCKETS
        fused = name.endswith("fused")
        groups = [dict(name=f"L={L}", B=TOKENS // L, L=L, cu=None, rope=ROPE_BASE,
                       rope_fused=fused) for L in lens]
        desc = dict(workload=name, tokens_per_group=TOKENS, buckets=lens, H=H, D=D,
                    causal=True, rope_base=ROPE_BASE,
                    q_rotation="inside the forward" if fused else "dd_rope pass")
    elif name == "tiny":
        H, D = 4, 64
        groups = [dict(name="L=256", B=4, L=256, cu=None)]
        desc = dict(workload=name, tokens_per_group=1024, buckets=[256], H=H, D=D, causal=True)
    elif name == "chunk_vs_dd":
        H, D = 16, 64
        docs = synth.lognormal_doc_lengths(seed, TOKENS)
        cu = dd.chunk_doclens(docs, TOKENS)
        groups = [dict(name="dense 8x8192", B=8, L=8192, cu=None, variant="dense"),
                  dict(name="masked 8x8192", B=8, L=8192, cu=cu, variant="masked")]
        for n, b in dd.decompose(docs, min_len=256, max_len=8192).items():
            groups.append(dict(name=f"DD L={n}", B=b.count, L=n, cu=None, variant="dd"))
        packed = dd.pack_step(docs, min_len=256, max_len=8192)
        groups.append(dict(name="DD packed 1x", B=1, L=packed.tokens, cu=packed.cu_doclens,
                           variant="dd_packed"))
        desc = dict(workload=name, tokens_per_group=TOKENS, H=H, D=D, causal=True,
                    documents=int(len(docs)), doc_seed=seed,
                    dd_tokens_kept=int(sum(g["B"] * g["L"] for g in groups
                                           if g.get("variant") == "dd")),
                    note="one bench step runs every variant once; compare the variants' "
                         "ms (dense, masked, the sum of the dd buckets, dd_packed)")
    elif name == "curriculum":
        from paper_2405_13226_amd import sampler
        H, D, cycles = 16, 128, 8
        lens_all = list(sampler.CURRICULUM_LENGTHS)
        n = {L: cycles * TOKENS for L in lens_all}            # one step per bucket per cycle
        rows = {L: n[L] // L for L in lens_all}
        steps = sampler.curriculum_steps(rows, n, sampler.preset_odds("grow_p2"), cycles, TOKENS,
                                         np.random.default_rng(seed))
        lens = [st.length for st in steps]
        groups = [dict(name=f"step{i} L={L}", B=TOKENS // L, L=L, cu=None)
                  for i, L in enumerate(lens)]
        desc = dict(workload=name, tokens_per_group=TOKENS, steps_per_stream=len(lens), H=H,
                    D=D, causal=True, odds="grow_p2", cycles=cycles,
                    order=[int(L) for L in lens])
    else:  # stream
        H, D = 16, 128
        lens = synth.length_stream(seed, steps=64)
        groups = [dict(name=f"step{i} L={int(L)}", B=TOKENS // int(L), L=int(L), cu=None)
                  for i, L in enumerate(lens)]
        desc = dict(workload=name, tokens_per_group=TOKENS, steps_per_stream=64, H=H, D=D,
                    causal=True, lengths={int(k): int(v) for k, v in
                                          zip(*np.unique(lens, return_counts=True))})
    for g in groups:
        g["H"], g["D"] = H, D
        f, b = dd.attention_flops(g["B"], g["L"], H, D, True, g["cu"])
        g["flops_fwd"], g["flops_bwd"] = f, b
        g["pairs"] = dd.useful_pairs(g["B"], g["L"], True, g["cu"]) * H
        g["tokens"] = g["B"] * g["L"]
    return groups, desc


# ---------------------------------------------------------------------------
# per-launch attribution
# ---------------------------------------------------------------------------
# Library kernel ids (dd_prof_kernel_name) and the algorithmic FLOPs per
# allowed (query, key) pair, per head dim, of each: the forward forms S and
# O (4); dK/dV forms S, dP, dV and dK (8); dQ forms dQ (2: its S and dP are
# recomputation); the one-kernel backward of D = 64 rows of at most 256
# tokens without RoPE forms S, dP, dV, dK and dQ once (10).
PER_PAIR = {"forward": 4, "backward_dkdv": 8, "backward_dq": 2, "backward_short": 10}


def split_by_group(launches, names, n_groups):
    """[(kernel name, ms)] in launch order -> per group {kernel: [ms, ...]}.
    Every group launches exactly one forward per step, preceded by its RoPE
    launches (if any) and followed by its backward kernels."""
    out = [dict() for _ in range(n_groups)]
    gi = -1
    for kid, ms in launches:
        name = names[kid]
        if name == "forward":
            gi = (gi + 1) % n_groups
            target = gi
        elif name == "rope":
            target = (gi + 1) % n_groups
        else:
            target = gi
        out[target].setdefault(name, []).append(ms)
    return out


def kernel_alg(name, g):
    """Algorithmic work of one launch of kernel `name` in group g: (amount,
    'flop' or 'byte')."""
    if name == "rope":  # reads and writes one [tokens, H, D] bf16 tensor
        return 2 * g["tokens"] * g["H"] * g["D"] * 2, "byte"
    return PER_PAIR[name] * g["D"] * g["pairs"], "flop"


def roofline_of(name, g, avg_ms, workload):
    amount, kind = kernel_alg(name, g)
    if kind == "byte":
        achieved = amount / (avg_ms * 1e-3) / 1e9
        bound, peak, unit = "hbm", HBM_PEAK_GBS, "GB/s"
    else:
        achieved = amount / (avg_ms * 1e-3) / 1e12
        bound, peak, unit = "mfma", BF16_PEAK_TFLOPS, "TFLOP/s"
    return dict(bound=bound, kernel=name, group=g["name"], achieved=round(achieved, 2), peak=peak,
                unit=unit, frac=round(achieved / peak, 4),
                traffic=measured_traffic(workload, name, g["name"]),
                avg_ms=round(avg_ms, 5), algorithmic_per_launch=int(amount))


# ---------------------------------------------------------------------------
def run_workload(name, args, buckets, dev, seed):
    """Warm up, time `args.steps` bench steps of workload `name` and return
    the result dict (without cpu_baseline)."""
    import numpy as np
    import torch
    import paper_2405_13226_amd as ddlib
    from paper_2405_13226_amd import _lib

    lib = ddlib.lib()
    groups, desc = workload(name, seed, buckets)
    H, D = desc["H"], desc["D"]
    ntok = max(g["tokens"] for g in groups)

    # Resident inputs (seeded N(0,1) bf16) and outputs, sized for the largest group.
    gen = torch.Generator(device=dev)
    gen.manual_seed(seed)
    shape = (ntok, H, D)
    q, k, v, do = (torch.randn(shape, generator=gen, device=dev, dtype=torch.float32)
                   .to(torch.bfloat16) for _ in range(4))
    o = torch.empty_like(q)
    dq, dk, dv = torch.empty_like(q), torch.empty_like(q), torch.empty_like(q)
    use_rope = any(g.get("rope") for g in groups)
    qr = torch.empty_like(q) if use_rope else q
    kr = torch.empty_like(q) if use_rope else k
    lse = torch.empty((ntok, H), dtype=torch.float32, device=dev)
    ws_bytes = max(ddlib.workspace_bytes(g["B"], g["L"], H, D) for g in groups)
    ws = torch.empty(ws_bytes, dtype=torch.uint8, device=dev)
    for g in groups:
        g["docs"] = ddlib.DocLens(g["cu"], g["tokens"], dev) if g["cu"] is not None else None
    P = ctypes.c_void_p
    ptr = {n: P(t.data_ptr()) for n, t in dict(q=q, k=k, v=v, do=do, o=o, dq=dq, dk=dk, dv=dv,
                                                lse=lse, ws=ws, qr=qr, kr=kr).items()}
    stream = torch.cuda.current_stream(dev)
    sptr = P(stream.cuda_stream)

    def run_group(g, mark=False):
        B, L = g["B"], g["L"]
        cu = P(g["docs"].dev.data_ptr()) if g["docs"] else None
        nd = g["docs"].n_docs if g["docs"] else 0
        base = g.get("rope")
        if base and g.get("rope_fused"):
            st = lib.dd_rope(ptr["k"], ptr["kr"], B, L, H, D, base, 0, cu, nd, 0, sptr)
            _lib.check(st, "dd_rope")
            st = lib.dd_attn_fwd_rope(ptr["q"], ptr["kr"], ptr["v"], ptr["o"], ptr["lse"],
                                      ptr["qr"], B, L, H, D, 1, cu, nd, base, 0, sptr)
            _lib.check(st, "dd_attn_fwd_rope")
        else:
            if base:
                for src, dst in (("q", "qr"), ("k", "kr")):
                    st = lib.dd_rope(ptr[src], ptr[dst], B, L, H, D, base, 0, cu, nd, 0, sptr)
                    _lib.check(st, "dd_rope")
            st = lib.dd_attn_fwd(ptr["qr"], ptr["kr"], ptr["v"], ptr["o"], ptr["lse"], B, L, H,
                                 D, 1, cu, nd, sptr)
            _lib.check(st, "dd_attn_fwd")
        if mark:
            g["ev"][1].record(stream)
        if base:
            st = lib.dd_attn_bwd_rope(ptr["qr"], ptr["kr"], ptr["v"], ptr["o"], ptr["do"],
                                      ptr["lse"], ptr["dq"], ptr["dk"], ptr["dv"], B, L, H, D, 1,
                                      cu, nd, base, 0, ptr["ws"], ws_bytes, sptr)
            _lib.check(st, "dd_attn_bwd_rope")
        else:
            st = lib.dd_attn_bwd(ptr["qr"], ptr["kr"], ptr["v"], ptr["o"], ptr["do"], ptr["lse"],
                                 ptr["dq"], ptr["dk"], ptr["dv"], B, L, H, D, 1, cu, nd,
                                 ptr["ws"], ws_bytes, sptr)
            _lib.check(st, "dd_attn_bwd")

    def new_events():
        return [torch.cuda.Event(enable_timing=True) for _ in range(3)]

    log(f"workload {desc['workload']}: {len(groups)} groups, H={H} D={D}")
    if args.copy_calibration:
        src = torch.empty(1 << 30, dtype=torch.uint8, device=dev)
        dst = torch.empty_like(src)
        for _ in range(3):
            dst.copy_(src)
        torch.cuda.synchronize(dev)
        del src, dst
    for g in groups:
        g["ev"] = new_events()
    for _ in range(args.warmup):
        for g in groups:
            run_group(g)
    torch.cuda.synchronize(dev)

    def timed(with_events):
        """K bench steps; returns wall seconds.  With events, every group is
        bracketed by torch events and every library kernel by the library's
        own HIP event pair on the same stream."""
        if with_events:
            for g in groups:
                g["evs"] = [new_events() for _ in range(args.steps)]
            _lib.prof_enable(True)
        torch.cuda.synchronize(dev)
        t0 = time.perf_counter()
        for s in range(args.steps):
            for g in groups:
                if with_events:
                    g["ev"] = g["evs"][s]
                    g["ev"][0].record(stream)
                run_group(g, with_events)
                if with_events:
                    g["ev"][2].record(stream)
        torch.cuda.synchronize(dev)
        wall = time.perf_counter() - t0
        if with_events:
            _lib.prof_enable(False)
        return wall

    with SclkSampler() as sclk:
        wall = timed(args.events == "inline")
    if args.events == "separate":
        wall_ev = timed(True)
        log(f"wall per step: {wall * 1e3 / args.steps:.3f} ms clean, "
            f"{wall_ev * 1e3 / args.steps:.3f} ms with events")

    ms_per_step = wall * 1e3 / args.steps
    flops_step = sum(g["flops_fwd"] + g["flops_bwd"] for g in groups)
    tokens_step = sum(g["tokens"] for g in groups)
    value = flops_step / (ms_per_step * 1e-3) / 1e12

    # Every library launch of the timed region, attributed to its group.
    names = {kid: n for n, kid in _lib.KERNELS.items()}
    launches = _lib.prof_launches()
    by_group = split_by_group(launches, names, len(groups))

    per_group, pairs_ms = [], []
    for g, kl in zip(groups, by_group):
        f = [e[0].elapsed_time(e[1]) for e in g["evs"]]
        b = [e[1].elapsed_time(e[2]) for e in g["evs"]]
        fm, bm = float(np.mean(f)), float(np.mean(b))
        tot = fm + bm
        fb, bb = ddlib.dd.attention_bytes(g["B"], g["L"], H, D)
        rec = dict(name=g["name"], B=g["B"], L=g["L"], fwd_ms=round(fm, 4), bwd_ms=round(bm, 4),
                   ms=round(tot, 4), ms_std=round(float(np.std(np.add(f, b))), 4),
                   ms_median=round(float(np.median(np.add(f, b))), 4),
                   tflops=round((g["flops_fwd"] + g["flops_bwd"]) / (tot * 1e-3) / 1e12, 2),
                   fwd_tflops=round(g["flops_fwd"] / (fm * 1e-3) / 1e12, 2),
                   bwd_tflops=round(g["flops_bwd"] / (bm * 1e-3) / 1e12, 2),
                   tokens_per_s=round(g["tokens"] / (tot * 1e-3)),
                   mfma_frac=round((g["flops_fwd"] + g["flops_bwd"]) / (tot * 1e-3) / 1e12
                                   / BF16_PEAK_TFLOPS, 4),
                   hbm_frac=round((fb + bb) / (tot * 1e-3) / 1e9 / HBM_PEAK_GBS, 4))
        kern = {}
        for kname, mss in kl.items():
            avg = float(np.mean(mss))
            r = roofline_of(kname, g, avg, desc["workload"])
            kern[kname] = dict(launches=len(mss), avg_ms=round(avg, 5), achieved=r["achieved"],
                               unit=r["unit"], frac=r["frac"])
            pairs_ms.append((sum(mss), kname, g, avg))
        rec["kernels"] = kern
        if "variant" in g:
            rec["variant"] = g["variant"]
        per_group.append(rec)
        log(f"  {g['name']:>16s}  fwd {fm:8.3f} ms  bwd {bm:8.3f} ms  "
            f"{rec['tflops']:8.1f} TFLOP/s  {rec['tokens_per_s'] / 1e6:8.2f} Mtok/s  " +
            " ".join(f"{k}={v['avg_ms']:.3f}ms/{v['frac']:.3f}" for k, v in kern.items()))

    # Per-kernel totals over the whole timed region.
    kern_all = {}
    for kname in _lib.KERNELS:
        mss = [m for kid, m in launches if names[kid] == kname]
        kern_all[kname] = dict(total_ms=round(float(sum(mss)), 3), launches=len(mss),
                               avg_ms=round(float(np.mean(mss)), 5) if mss else 0.0)
    # Dominant kernel launch: the (kernel, group) with the largest total time.
    _, dname, dg, davg = max(pairs_ms, key=lambda x: x[0])
    roofline = roofline_of(dname, dg, davg, desc["workload"])
    roofline["launches"] = len(by_group[groups.index(dg)][dname])
    log(f"dominant kernel launch {dname} in {dg['name']}: {roofline}")

    result = {
        "metric": METRIC, "value": round(value, 2), "unit": "TFLOP/s", "n_gpus": 1,
        "steps": args.steps, "warmup": args.warmup, "ms_per_step": round(ms_per_step, 4),
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None, "dtype": "bf16",
        "data": "synthetic (seeded N(0,1) bf16 on device; log-normal document lengths)",
        "config": desc,
        "tokens_per_s": round(tokens_step / (ms_per_step * 1e-3)),
        "groups": per_group, "kernels": kern_all, "roofline": roofline,
        "sclk_mhz": sclk.summary(),
    }
    # Streams repeat lengths: per-L efficiency over the steps of each length.
    lens = [g["L"] for g in groups]
    if len(set(lens)) < len(lens):
        per_l = {}
        for g, rec in zip(groups, per_group):
            a = per_l.setdefault(g["L"], dict(steps=0, ms=0.0, flops=0.0, bytes=0.0))
            a["steps"] += 1
            a["ms"] += rec["ms"]
            a["flops"] += g["flops_fwd"] + g["flops_bwd"]
            a["bytes"] += sum(ddlib.dd.attention_bytes(g["B"], g["L"], H, D))
        result["per_L"] = {
            str(n): dict(steps=a["steps"], ms_mean=round(a["ms"] / a["steps"], 4),
                         share_of_stream=round(a["ms"] / sum(r["ms"] for r in per_group), 4),
                         tflops=round(a["flops"] / (a["ms"] * 1e-3) / 1e12, 2),
                         mfma_frac=round(a["flops"] / (a["ms"] * 1e-3) / 1e12 / BF16_PEAK_TFLOPS, 4),
                         hbm_frac=round(a["bytes"] / (a["ms"] * 1e-3) / 1e9 / HBM_PEAK_GBS, 4))
            for n, a in sorted(per_l.items())}
    del q, k, v, do, o, dq, dk, dv, qr, kr, lse, ws
    torch.cuda.empty_cache()
    return result, groups


def bucket_summary(result, L=8192):
    """Fwd+bwd fraction of the bf16 peak of the bucket of length L and the
    roofline of its dominant kernel launch."""
    for g in result["groups"]:
        if g["L"] == L and g["B"] * g["L"] == TOKENS and "variant" not in g:
            dom = max(g["kernels"].items(), key=lambda kv: kv[1]["avg_ms"] * kv[1]["launches"])
            return dict(ms=g["ms"], fwd_ms=g["fwd_ms"], bwd_ms=g["bwd_ms"], tflops=g["tflops"],
                        mfma_frac=g["mfma_frac"], dominant_kernel=dom[0],
                        dominant_avg_ms=dom[1]["avg_ms"], dominant_frac=dom[1]["frac"])
    return None


def chunk_summary(result):
    """Step times of the concat-and-chunk vs DD comparison (ms per variant)."""
    g = result["groups"]
    dd_ms = sum(r["ms"] for r in g if r.get("variant") == "dd")
    pick = {r.get("variant"): r["ms"] for r in g if r.get("variant") in
            ("dense", "masked", "dd_packed")}
    return dict(dense_ms=pick.get("dense"), masked_ms=pick.get("masked"),
                dd_per_bucket_ms=round(dd_ms, 4), dd_packed_ms=pick.get("dd_packed"),
                dd_tokens_kept=result["config"]["dd_tokens_kept"], step_tokens=TOKENS)


def main():
    args = parse()
    if args.traffic_summary:
        return traffic_summary(args)
    if args.sq_summary:
        return sq_summary(args)
    if args.gpus != 1:
        print(f"bench.py runs on one GPU only (got --gpus {args.gpus}): every (b, h) slice "
              "of the attention path is independent, so there is no cross-GPU exchange to "
              "measure; the figure is one MI355X's throughput.", file=sys.stderr)
        sys.exit(2)

    import torch
    import paper_2405_13226_amd as ddlib

    ddlib.lib()  # raises if the HIP library is missing
    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    buckets = [int(x) for x in args.buckets.split(",")] if args.buckets else None
    if args.workload == "layer_1b":
        return run_layer(args, buckets, dev)
    if args.workload == "gemm_1b":
        return run_gemm(args, dev)
    result, groups = run_workload(args.workload, args, buckets, dev, args.seed)

    extras = {}
    if args.workload == "dd_sweep_d64" and buckets is None and not args.no_extras:
        # Every target configuration in one run, after the headline's timed
        # region: the D = 128 sweep and the concat-and-chunk vs DD step.
        for name in ("dd_sweep_d128", "chunk_vs_dd"):
            r, _ = run_workload(name, args, None, dev, args.seed)
            keep = ("value", "unit", "ms_per_step", "tokens_per_s", "config", "roofline",
                    "sclk_mhz", "groups")
            extras[name] = {k: r[k] for k in keep}
            if name == "chunk_vs_dd":
                extras[name]["step_ms"] = chunk_summary(r)
                log(f"chunk_vs_dd step ms: {extras[name]['step_ms']}")
        result["extra_workloads"] = extras
    b8 = {}
    for key, r in (("d%d" % result["config"]["D"], result),
                   ("d128", extras.get("dd_sweep_d128"))):
        if r is not None and bucket_summary(r) is not None:
            b8[key] = bucket_summary(r)
    if b8:
        result["roofline"]["bucket_8192"] = b8
        log(f"L=8192 buckets: {b8}")
    if "chunk_vs_dd" in extras:
        result["chunk_vs_dd_step_ms"] = extras["chunk_vs_dd"]["step_ms"]
    if not args.no_cpu_baseline:
        result["cpu_baseline"] = cpu_baseline(groups, result, args)
    print(json.dumps(result), flush=True)


def run_layer(args, buckets, dev):
    """One OpenLM-1B block fwd+bwd per bucket (one autograd node; every step in
    the library's kernels: GEMMs, LayerNorms, SwiGLU, RoPE and attention)."""
    import numpy as np
    import torch
    from paper_2405_13226_amd import _lib, dd
    from paper_2405_13226_amd.layer import OPENLM_1B, OpenLMBlock

    d, H, hidden = OPENLM_1B["d"], OPENLM_1B["H"], OPENLM_1B["hidden"]
    D = d // H
    lens = buckets or BUCKETS
    blk = OpenLMBlock(d, H, hidden, ROPE_BASE, device=dev, seed=args.seed)
    gen = torch.Generator(device=dev)
    gen.manual_seed(args.seed)
    x_all = torch.randn((TOKENS, d), generator=gen, device=dev).to(torch.bfloat16)
    dy_all = torch.randn((TOKENS, d), generator=gen, device=dev).to(torch.bfloat16)
    attn_kernels = ("forward", "rope", "backward_dkdv", "backward_dq", "backward_short")
    log(f"workload layer_1b: d={d} H={H} hidden={hidden} rope_base={ROPE_BASE:g}")

    def step(L):
        B = TOKENS // L
        x = x_all.view(B, L, d).detach().requires_grad_(True)
        blk.zero_grad(set_to_none=True)
        y = blk(x)
        y.backward(dy_all.view(B, L, d))

    per = []
    total_ms = 0.0
    total_flops = 0.0
    for L in lens:
        B = TOKENS // L
        for _ in range(args.warmup):
            step(L)
        torch.cuda.synchronize(dev)
        _lib.prof_enable(True)
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record()
        for _ in range(args.steps):
            step(L)
        e1.record()
        torch.cuda.synchronize(dev)
        _lib.prof_enable(False)
        ms = e0.elapsed_time(e1) / args.steps
        attn_ms = sum(_lib.prof_read(_lib.KERNELS[k])[0] for k in attn_kernels) / args.steps
        gemm = 3 * blk.gemm_flops(TOKENS)
        af, ab = dd.attention_flops(B, L, H, D, True, None)
        flops = gemm + af + ab
        per.append(dict(name=f"L={L}", B=B, L=L, ms=round(ms, 4), attention_ms=round(attn_ms, 4),
                        attention_share=round(attn_ms / ms, 4),
                        tflops=round(flops / (ms * 1e-3) / 1e12, 2),
                        tokens_per_s=round(TOKENS / (ms * 1e-3))))
        total_ms += ms
        total_flops += flops
        log(f"  L={L:5d}  {ms:8.3f} ms  attention {attn_ms:7.3f} ms ({100 * attn_ms / ms:5.1f}%)  "
            f"{per[-1]['tflops']:7.1f} TFLOP/s")
    Ls = np.array([g["L"] for g in per], dtype=np.float64)
    ts = np.array([g["ms"] for g in per])
    beta, alpha = np.polyfit(Ls, ts, 1)
    resid = float(np.max(np.abs(alpha + beta * Ls - ts)))
    log(f"fit t(L) = {alpha:.3f} ms + {beta * 1e3:.4f} us * L (max residual {resid:.3f} ms)")
    result = {
        "metric": "OpenLM-1B block fwd+bwd TFLOP/s (GEMM + useful attention FLOPs) at 65,536 tokens/step",
        "value": round(total_flops / (total_ms * 1e-3) / 1e12, 2), "unit": "TFLOP/s", "n_gpus": 1,
        "steps": args.steps, "warmup": args.warmup, "ms_per_step": round(total_ms, 4),
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None, "dtype": "bf16",
        "data": "synthetic (seeded N(0,1) bf16 activations, random-init weights)",
        "config": dict(workload="layer_1b", tokens_per_group=TOKENS, buckets=lens, d=d, H=H,
                       D=D, hidden=hidden, rope_base=ROPE_BASE, causal=True),
        "groups": per,
        "fit": dict(alpha_ms=round(float(alpha), 4), beta_us_per_token=round(float(beta) * 1e3, 5),
                    max_residual_ms=round(resid, 4)),
    }
    print(json.dumps(result), flush=True)


def run_gemm(args, dev):
    """dd_gemm on the block's shapes at 65,536 tokens, timed with events
    beside torch.matmul (vendor library) on the same operands."""
    import torch
    from paper_2405_13226_amd import block_ops
    from paper_2405_13226_amd.layer import OPENLM_1B

    T, d, hid = TOKENS, OPENLM_1B["d"], OPENLM_1B["hidden"]
    # (name, M, N, K, trans_a, trans_b): y = x (W^T)^T (the block's forward
    # reads transposed weight copies), dx = dy W^T, dW = x^T dy
    shapes = [("qkv fwd", T, 3 * d, d, 0, 1), ("out fwd", T, d, d, 0, 1),
              ("w1 fwd", T, hid, d, 0, 1), ("w2 fwd", T, d, hid, 0, 1),
              ("qkv dx", T, d, 3 * d, 0, 1), ("w1 dx", T, d, hid, 0, 1),
              ("w2 dx", T, hid, d, 0, 1), ("qkv dW", d, 3 * d, T, 1, 0),
              ("w1 dW", d, hid, T, 1, 0), ("w2 dW", hid, d, T, 1, 0)]
    gen = torch.Generator(device=dev)
    gen.manual_seed(args.seed)
    per, tot_ms, tot_fl, tot_ms_t = [], 0.0, 0.0, 0.0
    for name, M, N, K, ta, tb in shapes:
        a = torch.randn((K, M) if ta else (M, K), generator=gen, device=dev).to(torch.bfloat16)
        b = torch.randn((N, K) if tb else (K, N), generator=gen, device=dev).to(torch.bfloat16)
        c = torch.empty((M, N), dtype=torch.bfloat16, device=dev)
        at, bt = (a.t() if ta else a), (b.t() if tb else b)
        fns = {"dd": lambda: block_ops.gemm(a, b, bool(ta), bool(tb), out=c),
               "torch": lambda: torch.matmul(at, bt)}
        ms = {}
        for key, fn in fns.items():
            for _ in range(args.warmup):
                fn()
            e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            torch.cuda.synchronize(dev)
            e0.record()
            for _ in range(args.steps):
                fn()
            e1.record()
            torch.cuda.synchronize(dev)
            ms[key] = e0.elapsed_time(e1) / args.steps
        fl = 2.0 * M * N * K
        rec = dict(name=name, M=M, N=N, K=K, trans_a=ta, trans_b=tb, ms=round(ms["dd"], 4),
                   tflops=round(fl / (ms["dd"] * 1e-3) / 1e12, 1),
                   torch_ms=round(ms["torch"], 4),
                   torch_tflops=round(fl / (ms["torch"] * 1e-3) / 1e12, 1))
        per.append(rec)
        tot_ms += ms["dd"]
        tot_ms_t += ms["torch"]
        tot_fl += fl
        log(f"  {name:8s} M={M} N={N} K={K}: dd {rec['ms']:.3f} ms {rec['tflops']:7.1f} TFLOP/s"
            f" | torch {rec['torch_ms']:.3f} ms {rec['torch_tflops']:7.1f}")
        del a, b, c
    value = tot_fl / (tot_ms * 1e-3) / 1e12
    result = {
        "metric": "OpenLM-1B block GEMM TFLOP/s (dd_gemm) at 65,536 tokens",
        "value": round(value, 2), "unit": "TFLOP/s", "n_gpus": 1, "steps": args.steps,
        "warmup": args.warmup, "ms_per_step": round(tot_ms, 4), "higher_is_better": True,
        "scaling": "weak", "vs_baseline": None, "dtype": "bf16",
        "data": "synthetic (seeded N(0,1) bf16 on device)",
        "config": dict(workload="gemm_1b", tokens=T, d=d, hidden=hid),
        "groups": per,
        "roofline": dict(bound="mfma", kernel="gemm", achieved=round(value, 2),
                         peak=BF16_PEAK_TFLOPS, unit="TFLOP/s",
                         frac=round(value / BF16_PEAK_TFLOPS, 4), traffic=None),
        "torch_value": round(tot_fl / (tot_ms_t * 1e-3) / 1e12, 2),
    }
    print(json.dumps(result), flush=True)


def row_pairs(B, L, cu=None):
    """Allowed causal (query, key) pairs of each of the B rows (one head)."""
    import numpy as np
    from paper_2405_13226_amd import dd as ddh
    seg = ddh.segments(B, L, cu)
    starts = np.concatenate([[0], np.cumsum(seg)[:-1]])
    out = np.zeros(B, dtype=np.int64)
    np.add.at(out, starts // L, seg * (seg + 1) // 2)
    return out


def sample_flops(pairs, B, L, D, cu=None):
    """Useful forward + backward FLOPs (14 D per allowed pair) of the listed
    (b, h) slices of a [B, L] batch."""
    rp = row_pairs(B, L, cu)
    return 14 * D * sum(int(rp[b]) for b, _ in pairs)


def cpu_baseline(groups, result, args):
    """The fp64 oracle timed on a bounded sample of every distinct group of
    the workload: as many (b, h) pairs as the oracle has threads (all of
    them, for smaller groups), on rows of the group's shape and document
    layout, extrapolated to the whole group by its useful FLOPs (the
    oracle's work per pair follows the allowed pairs).  Timing does not
    depend on the values, so each sample draws only the rows it times."""
    import numpy as np
    import oracle
    import synth

    cores = oracle.threads()
    seen, per_group = {}, []
    t_all = 0.0
    for g, rec in zip(groups, result["groups"]):
        B, L, H, D = g["B"], g["L"], g["H"], g["D"]
        key = (B, L, H, D, g.get("rope"), None if g["cu"] is None else g["cu"].tobytes())
        if key not in seen:
            n = min(B * H, cores)
            for _ in range(2):  # a second, larger sample if the first took < 0.5 s
                Bs = -(-n // H)
                pairs = [(b, h) for b in range(Bs) for h in range(H)][:n]
                cu = None
                if g["cu"] is not None:
                    c = np.asarray(g["cu"], dtype=np.int64)
                    c = c[c < Bs * L]
                    cu = np.concatenate([c, [Bs * L]]).astype(np.int32)
                x = {nm: synth.normal_bf16((Bs, L, H, D), args.seed, i + 1)
                     for i, nm in enumerate(("q", "k", "v", "do"))}
                t = time.perf_counter()
                if g.get("rope"):
                    from oracle import rope as orope
                    orope.attn_fwd(x["q"], x["k"], x["v"], g["rope"], True, cu, bh=pairs)
                    orope.attn_bwd(x["q"], x["k"], x["v"], x["do"], g["rope"], True, cu,
                                   bh=pairs)
                else:
                    oracle.attn_fwd(x["q"], x["k"], x["v"], causal=True, cu_doclens=cu, bh=pairs)
                    oracle.attn_bwd(x["q"], x["k"], x["v"], x["do"], causal=True,
                                    cu_doclens=cu, bh=pairs)
                secs = time.perf_counter() - t
                t_all += secs
                grow = min(B * H // n, int(np.ceil(0.5 / max(secs, 1e-3))))
                if secs >= 0.5 or grow < 2:
                    break
                n *= grow
            rate = sample_flops(pairs, Bs, L, D, cu) / secs
            seen[key] = dict(pairs_timed=len(pairs), seconds=round(secs, 3), rate=rate)
            log(f"cpu oracle: {len(pairs)} (b,h) pairs of {g['name']} in {secs:.2f} s")
        m = seen[key]
        flops = g["flops_fwd"] + g["flops_bwd"]
        ext = flops / m["rate"]
        per_group.append(dict(name=g["name"], B=B, L=L, pairs_timed=m["pairs_timed"],
                              pairs_total=B * H, seconds=m["seconds"],
                              tflops=round(m["rate"] / 1e12, 6),
                              extrapolated_seconds=round(ext, 2),
                              tokens_per_s=round(g["tokens"] / ext, 1),
                              gpu_ms=rec["ms"], gpu_speedup=round(ext / (rec["ms"] * 1e-3), 1)))
    flops_step = sum(g["flops_fwd"] + g["flops_bwd"] for g in groups)
    ext_step = sum(r["extrapolated_seconds"] for r in per_group)
    return {"value": round(flops_step / ext_step / 1e12, 6), "unit": "TFLOP/s",
            "cores": cores, "kind": "oracle",
            "sample": f"fp64 fwd+bwd of up to {cores} (b, h) pairs of every distinct group "
                      f"of {result['config']['workload']}, extrapolated by useful FLOPs to the "
                      "whole step (per_group)",
            "seconds": round(t_all, 2), "extrapolated_seconds_per_step": round(ext_step, 1),
            "per_group": per_group}


def traffic_summary(args):
    """profiles/traffic_<workload>.txt text (stdout) from two rocprofv3 counter
    runs of this script: FETCH_SIZE / WRITE_SIZE (KiB per dispatch) of the
    last bench step's library launches, per (kernel, group), scaled by what
    the counters read for the 1 GiB copies of --copy-calibration."""
    import csv
    import glob
    import re

    import numpy as np

    fam = {"fwd_kernel": "forward", "dq_kernel": "backward_dq", "dkdv1_kernel": "backward_dkdv",
           "dkdv_kernel": "backward_dkdv", "bwd_short_kernel": "backward_short",
           "bwd_short_persist_kernel": "backward_short", "rope_kernel": "rope"}

    def read(d, counter):
        f = glob.glob(os.path.join(d, "**", "*counter_collection.csv"), recursive=True)
        if not f:
            raise SystemExit(f"no counter_collection.csv under {d}")
        disp = {}
        for r in csv.DictReader(open(f[0])):
            if r["Counter_Name"] != counter:
                continue
            did = int(r["Dispatch_Id"])
            name = r["Kernel_Name"]
            d0 = disp.setdefault(did, [name, 0.0])
            d0[1] += float(r["Counter_Value"]) * 1024.0
        return [disp[k] for k in sorted(disp)]

    out = {}
    for counter, d in (("FETCH_SIZE", args.traffic_summary[0]),
                       ("WRITE_SIZE", args.traffic_summary[1])):
        rows = read(d, counter)
        # the three 1 GiB copies of --copy-calibration run right before the
        # first library launch
        first = next(i for i, (n, _) in enumerate(rows) if "dd::" in n)
        copies = [v for n, v in rows[max(first - 3, 0):first] if "copy" in n.lower()]
        if len(copies) != 3 or min(copies) < 2 ** 28:
            raise SystemExit(f"{counter}: no copy-calibration dispatches before the first launch")
        scale = float(2 ** 30) / float(np.median(copies))
        lib_rows = []
        for n, v in rows:
            m = re.search(r"dd::(\w+)", n)
            if m and m.group(1) in fam:
                lib_rows.append((fam[m.group(1)], v * scale))
        out[counter] = (scale, lib_rows)
    groups, desc = workload(args.workload, args.seed,
                            [int(x) for x in args.buckets.split(",")] if args.buckets else None)
    lines = [f"# HBM traffic per launch, workload {desc['workload']}, from rocprofv3 counter runs",
             f"# command: rocprofv3 --pmc FETCH_SIZE (then WRITE_SIZE) --output-format csv -d <dir> "
             f"-o run -- python3 -u bench.py --workload {desc['workload']}"
             + (f" --buckets {args.buckets}" if args.buckets else "") +
             " --copy-calibration --steps 1 --warmup 1 --no-cpu-baseline --no-extras",
             "# summary:  python3 bench.py --workload " + desc["workload"]
             + (f" --buckets {args.buckets}" if args.buckets else "")
             + " --traffic-summary <fetch dir> <write dir>",
             "# FETCH_SIZE and WRITE_SIZE are KiB per dispatch; each is scaled by 2^30 / what it",
             "# reads for a plain 1 GiB device copy (bytes of the last bench step's launches).",
             f"workload = {desc['workload']}", f"source_hash = {kernel_source_hash()}",
             f"fetch_scale = {out['FETCH_SIZE'][0]:.6f}", f"write_scale = {out['WRITE_SIZE'][0]:.6f}"]
    for counter, key in (("FETCH_SIZE", "fetch"), ("WRITE_SIZE", "write")):
        lib_rows = out[counter][1]
        names = [n for n, _ in lib_rows]
        n_fwd = sum(1 for n in names if n == "forward")
        if n_fwd % len(groups):
            raise SystemExit("launch count does not match the workload's groups")
        # index of the first launch of the last step: the (len(groups))-th
        # forward from the end, with its preceding RoPE launches
        fwd_idx = [i for i, n in enumerate(names) if n == "forward"]
        start = fwd_idx[-len(groups)]
        while start > 0 and names[start - 1] == "rope":
            start -= 1
        tail = lib_rows[start:]
        kid = {"forward": 0, "rope": 4, "backward_dq": 3, "backward_dkdv": 2, "backward_short": 1}
        nm = {v: k for k, v in kid.items()}
        by = split_by_group([(kid[n], v) for n, v in tail], nm, len(groups))
        for g, kl in zip(groups, by):
            for kname, vals in kl.items():
                out.setdefault("_bytes", {}).setdefault((kname, g["name"]), {})[key] = \
                    float(np.mean(vals))
    for (kname, gname), v in out["_bytes"].items():
        lines.append(f"fetch_bytes_per_launch.{kname}.{gname} = {int(v['fetch'])}")
        lines.append(f"write_bytes_per_launch.{kname}.{gname} = {int(v['write'])}")
        lines.append(f"bytes_per_launch.{kname}.{gname} = {int(v['fetch'] + v['write'])}")
    print("\n".join(lines))


def sq_summary(args):
    """Markdown table (stdout) of SQ counters per (group, kernel) of the last
    bench step, from two rocprofv3 counter runs of this script (pass 1:
    SQ_VALU_MFMA_BUSY_CYCLES SQ_VALU_MFMA_COEXEC_CYCLES SQ_WAVE_CYCLES
    SQ_WAIT_ANY SQ_WAIT_INST_ANY ... GRBM_GUI_ACTIVE; pass 2: SQ_WAIT_INST_LDS
    SQ_INSTS_VALU SQ_INSTS_MFMA SQ_INSTS_LDS ... GRBM_GUI_ACTIVE), each with
    --steps 1 --warmup 1.  GRBM_GUI_ACTIVE is summed over the 8 XCDs; the
    matrix-pipe shares are over (GUI / 8) * 1024 SIMD-cycles, the wait shares
    over SQ_WAVE_CYCLES."""
    import csv
    import glob
    import re

    fam = {"fwd_kernel": "forward", "dq_kernel": "backward_dq", "dkdv1_kernel": "backward_dkdv",
           "dkdv_kernel": "backward_dkdv", "bwd_short_kernel": "backward_short",
           "bwd_short_persist_kernel": "backward_short", "rope_kernel": "rope"}
    kid = {"forward": 0, "rope": 4, "backward_dq": 3, "backward_dkdv": 2, "backward_short": 1}

    def read(d):
        f = glob.glob(os.path.join(d, "**", "*counter_collection.csv"), recursive=True)
        if not f:
            raise SystemExit(f"no counter_collection.csv under {d}")
        disp = {}
        for r in csv.DictReader(open(f[0])):
            m = re.search(r"dd::(\w+)(<[^>]*>)?", r["Kernel_Name"])
            if not m or m.group(1) not in fam:
                continue
            did = int(r["Dispatch_Id"])
            e = disp.setdefault(did, {"kernel": m.group(1) + (m.group(2) or ""),
                                      "fam": fam[m.group(1)],
                                      "ms": (int(r["End_Timestamp"]) - int(r["Start_Timestamp"])) / 1e6})
            e[r["Counter_Name"]] = e.get(r["Counter_Name"], 0.0) + float(r["Counter_Value"])
        return [disp[k] for k in sorted(disp)]

    groups, desc = workload(args.workload, args.seed,
                            [int(x) for x in args.buckets.split(",")] if args.buckets else None)
    passes = []
    for d in args.sq_summary:
        rows = read(d)
        names = [r["fam"] for r in rows]
        fwd_idx = [i for i, n in enumerate(names) if n == "forward"]
        if len(fwd_idx) < len(groups):
            raise SystemExit("fewer forward launches than groups")
        start = fwd_idx[-len(groups)]
        while start > 0 and names[start - 1] == "rope":
            start -= 1
        passes.append(rows[start:])
    if len(passes[0]) != len(passes[1]):
        raise SystemExit("the two passes hold different launch sequences")
    merged = []
    for a, b in zip(*passes):
        if a["kernel"] != b["kernel"]:
            raise SystemExit("the two passes hold different launch sequences")
        merged.append({**b, **a})
    nm = {v: k for k, v in kid.items()}
    by = split_by_group([(kid[m["fam"]], m) for m in merged], nm, len(groups))
    lines = ["| L | kernel | ms | SCLK GHz | MFMA busy % | MFMA+VALU co-issue % | waves waiting % "
             "| waiting to issue % | waiting on LDS issue % | VALU / MFMA instr | LDS / MFMA instr |",
             "|---|---|---|---|---|---|---|---|---|---|---|"]
    for g, kl in zip(groups, by):
        for fname in ("rope", "forward", "backward_short", "backward_dq", "backward_dkdv"):
            for m in kl.get(fname, []):
                gui = m["GRBM_GUI_ACTIVE"] / 8.0
                simd = gui * 1024.0
                wave = m["SQ_WAVE_CYCLES"]
                mf = max(m["SQ_INSTS_MFMA"], 1.0)
                lines.append(
                    f"| {g['L']} | `{m['kernel']}` | {m['ms']:.3f} | {gui / (m['ms'] * 1e-3) / 1e9:.2f} "
                    f"| {100 * m['SQ_VALU_MFMA_BUSY_CYCLES'] / simd:.0f} "
                    f"| {100 * m['SQ_VALU_MFMA_COEXEC_CYCLES'] / simd:.0f} "
                    f"| {100 * m['SQ_WAIT_ANY'] / wave:.0f} | {100 * m['SQ_WAIT_INST_ANY'] / wave:.0f} "
                    f"| {100 * m['SQ_WAIT_INST_LDS'] / wave:.0f} "
                    f"| {m['SQ_INSTS_VALU'] / mf:.1f} | {m['SQ_INSTS_LDS'] / mf:.2f} |")
    print("\n".join(lines))


if __name__ == "__main__":
    main()
