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
                 q and k rotated before the forward, dq and dk rotated back in
                 the backward kernels
  layer_1b       one OpenLM-1B block (d 2048, 16 heads, SwiGLU 5632, RoPE)
                 forward + backward per bucket L = 256 .. 8192 at 65,536
                 tokens: step time, attention's share of it, and the fit
                 t(L) = alpha + beta * L (value: block TFLOP/s)
  tiny           B = 4, L = 256, H = 4, D = 64

Prints ONE JSON line on stdout: the metric is useful attention TFLOP/s
(forward 4*D and backward 10*D FLOPs per allowed (query, key) pair and head)
over the whole bench step, with per-group times, tokens/s, per-length
efficiency where lengths repeat (stream, curriculum), the roofline of the
dominant kernel (timed with HIP events on its own stream) and the fp64 CPU
oracle timed on a bounded sample of the same workload.
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


def measured_traffic(workload, kernel):
    """HBM bytes per launch of `kernel` from profiles/traffic_<workload>.txt
    (key = value lines), or None if absent, for another kernel, or taken on
    other kernel sources."""
    path = os.path.join(ROOT, "profiles", f"traffic_{workload}.txt")
    if not os.path.exists(path):
        return None
    kv = {}
    with open(path) as f:
        for line in f:
            if "=" in line and not line.lstrip().startswith("#"):
                k, v = line.split("=", 1)
                kv[k.strip()] = v.strip()
    if kv.get("source_hash") != kernel_source_hash():
        return None
    key = f"bytes_per_launch.{kernel}"
    return int(float(kv[key])) if key in kv else None


def parse():
    ap = argparse.ArgumentParser(description=__doc__.splitlines()[0])
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=10)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--workload", default="dd_sweep_d64",
                    choices=["dd_sweep_d64", "dd_sweep_d128", "chunk_vs_dd", "stream",
                             "curriculum", "rope_d128", "layer_1b", "tiny"])
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
    elif name == "rope_d128":
        # The D=128 sweep with rotary position embedding (base 100,000, the
        # paper's curriculum runs): the forward rotates q and k (two dd_rope
        # launches) before attention; the backward rotates dq and dk back in
        # its kernels' epilogues (dd_attn_bwd_rope).
        H, D = 16, 128
        lens = buckets or BUCKETS
        groups = [dict(name=f"L={L}", B=TOKENS // L, L=L, cu=None, rope=ROPE_BASE)
                  for L in lens]
        desc = dict(workload=name, tokens_per_group=TOKENS, buckets=lens, H=H, D=D,
                    causal=True, rope_base=ROPE_BASE)
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
def main():
    args = parse()
    if args.gpus != 1:
        print(f"bench.py runs on one GPU only (got --gpus {args.gpus}): every (b, h) slice "
              "of the attention path is independent, so there is no cross-GPU exchange to "
              "measure; the figure is one MI355X's throughput.", file=sys.stderr)
        sys.exit(2)

    import numpy as np
    import torch
    import paper_2405_13226_amd as ddlib
    from paper_2405_13226_amd import _lib

    lib = ddlib.lib()  # raises if the HIP library is missing
    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    buckets = [int(x) for x in args.buckets.split(",")] if args.buckets else None
    if args.workload == "layer_1b":
        return run_layer(args, buckets, dev)
    groups, desc = workload(args.workload, args.seed, buckets)
    H, D = desc["H"], desc["D"]
    ntok = max(g["tokens"] for g in groups)

    # Resident inputs (seeded N(0,1) bf16) and outputs, sized for the largest group.
    gen = torch.Generator(device=dev)
    gen.manual_seed(args.seed)
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
        if base:
            for src, dst in (("q", "qr"), ("k", "kr")):
                st = lib.dd_rope(ptr[src], ptr[dst], B, L, H, D, base, 0, cu, nd, 0, sptr)
                _lib.check(st, "dd_rope")
        st = lib.dd_attn_fwd(ptr["qr"], ptr["kr"], ptr["v"], ptr["o"], ptr["lse"], B, L, H, D,
                             1, cu, nd, sptr)
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

    per_group = []
    for g in groups:
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
        if "variant" in g:
            rec["variant"] = g["variant"]
        per_group.append(rec)
        log(f"  {g['name']:>16s}  fwd {fm:8.3f} ms  bwd {bm:8.3f} ms  "
            f"{rec['tflops']:8.1f} TFLOP/s  {rec['tokens_per_s'] / 1e6:8.2f} Mtok/s")

    # Per-kernel durations from the library's event pairs (the kernel's stream).
    kern = {}
    for name, kid in _lib.KERNELS.items():
        ms, n = _lib.prof_read(kid)
        kern[name] = dict(total_ms=ms, launches=n, avg_ms=ms / n if n else 0.0)
    # Algorithmic FLOPs per (query, key) pair and head dim: the forward forms
    # S and O (4); dK/dV forms S, dP, dV and dK (8); dQ forms dQ (2, its S and
    # dP are recomputation); the one-kernel backward of D = 64 rows of at most
    # 256 tokens without RoPE forms S, dP, dV, dK and dQ once (10).
    def fused(g):
        return D == 64 and g["L"] <= SHORT_MAX_ROW and not g.get("rope")

    per_pair = {"forward": 4, "backward_dkdv": 8, "backward_dq": 2, "backward_short": 10}
    alg = {name: sum(per_pair[name] * D * g["pairs"] for g in groups
                     if name == "forward" or (name == "backward_short") == fused(g))
           * args.steps for name in per_pair}
    # rope: each launch reads and writes one [tokens, H, D] bf16 tensor
    alg["rope"] = sum(2 * 2 * g["tokens"] * H * D * 2 for g in groups if g.get("rope")) \
        * args.steps
    dom = max(kern, key=lambda n: kern[n]["total_ms"])
    kd = kern[dom]
    launches = max(kd["launches"], 1)
    if dom == "rope":
        achieved = alg[dom] / launches / (kd["avg_ms"] * 1e-3) / 1e9
        roof = dict(bound="hbm", unit="GB/s", peak=HBM_PEAK_GBS)
    else:
        achieved = alg[dom] / launches / (kd["avg_ms"] * 1e-3) / 1e12
        roof = dict(bound="mfma", unit="TFLOP/s", peak=BF16_PEAK_TFLOPS)
    traffic = measured_traffic(desc["workload"], dom)
    roofline = dict(bound=roof["bound"], kernel=dom, achieved=round(achieved, 2),
                    peak=roof["peak"], unit=roof["unit"], frac=round(achieved / roof["peak"], 4),
                    traffic=traffic, launches=kd["launches"], avg_ms=round(kd["avg_ms"], 5),
                    algorithmic_per_launch=alg[dom] // launches)
    for name in kern:
        kern[name]["avg_ms"] = round(kern[name]["avg_ms"], 5)
        kern[name]["total_ms"] = round(kern[name]["total_ms"], 3)
    log(f"dominant kernel {dom}: {roofline}")

    result = {
        "metric": METRIC, "value": round(value, 2), "unit": "TFLOP/s", "n_gpus": 1,
        "steps": args.steps, "warmup": args.warmup, "ms_per_step": round(ms_per_step, 4),
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None, "dtype": "bf16",
        "data": "synthetic (seeded N(0,1) bf16 on device; log-normal document lengths)",
        "config": desc,
        "tokens_per_s": round(tokens_step / (ms_per_step * 1e-3)),
        "groups": per_group, "kernels": kern, "roofline": roofline,
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
    if not args.no_cpu_baseline:
        result["cpu_baseline"] = cpu_baseline(groups, desc, args)
    print(json.dumps(result), flush=True)


def run_layer(args, buckets, dev):
    """One OpenLM-1B block fwd+bwd per bucket (torch autograd; attention and RoPE
    in the library's kernels, projections and MLP as vendor GEMMs)."""
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


def cpu_baseline(groups, desc, args):
    """The fp64 oracle on a bounded sample: (b, h) pairs of one group."""
    import numpy as np
    import oracle
    import synth

    # The middle group of the workload, its sampled (b, h) pairs.
    g = groups[len(groups) // 2]
    B, L, H, D = g["B"], g["L"], g["H"], g["D"]
    rng = np.random.default_rng(args.seed)
    per_pair_flops = (g["flops_fwd"] + g["flops_bwd"]) / (B * H)
    x = {n: synth.normal_bf16((B, L, H, D), args.seed, i + 1) for i, n in enumerate("qkv")}
    x["do"] = synth.normal_bf16((B, L, H, D), args.seed, 4)

    def run(pairs):
        t = time.perf_counter()
        if g.get("rope"):
            from oracle import rope as orope
            orope.attn_fwd(x["q"], x["k"], x["v"], g["rope"], True, g["cu"], bh=pairs)
            orope.attn_bwd(x["q"], x["k"], x["v"], x["do"], g["rope"], True, g["cu"], bh=pairs)
        else:
            oracle.attn_fwd(x["q"], x["k"], x["v"], causal=True, cu_doclens=g["cu"], bh=pairs)
            oracle.attn_bwd(x["q"], x["k"], x["v"], x["do"], causal=True, cu_doclens=g["cu"],
                            bh=pairs)
        return time.perf_counter() - t

    all_pairs = [(b, h) for b in range(B) for h in range(H)]
    order = rng.permutation(len(all_pairs))
    first = [all_pairs[order[0]]]
    t1 = run(first)
    n = int(min(len(all_pairs), max(1, args.cpu_seconds / max(t1, 1e-3))))
    pairs = [all_pairs[i] for i in order[:n]]
    secs = run(pairs) if n > 1 else t1
    flops = per_pair_flops * n
    log(f"cpu oracle: {n} (b,h) pairs of {g['name']} in {secs:.2f} s")
    return {"value": round(flops / secs / 1e12, 6), "unit": "TFLOP/s",
            "cores": oracle.threads(), "kind": "oracle",
            "sample": f"{g['name']} (B={B}, L={L}, H={H}, D={D}): fwd+bwd of {n} of the "
                      f"{B * H} (b, h) pairs, fp64",
            "seconds": round(secs, 3),
            "tokens_per_s": round(n * L / secs, 1)}


if __name__ == "__main__":
    main()
