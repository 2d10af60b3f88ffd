#!/usr/bin/env python3
"""Benchmark of one layer of RcLLM's selective prefill (arXiv 2605.07443) on
one MI355X.

A step is one pass of the whole path over one batch of synthetic
recommendation prompts already resident in HBM, on one stream:
  rc_kv_assemble          gather of history/item KV blocks + fused RoPE
                          re-alignment + K deviation score
  rc_select_tokens        top-k, heavy-hitter patch
  rc_selective_attention  causal GQA attention of the fresh + selected rows
Batches rotate (default 4 independent draws over one shared pool) so the
working set exceeds the 256 MB Infinity Cache.

Prints ONE JSON line: selected-query tokens/s/layer (whole job), ms per step,
microseconds per request, the roofline of the dominant kernel (measured with
HIP events on the launch stream in a second timed pass over the same steps,
with events between the kernels; the step time comes from a pass without
them), every kernel's achieved rate, the same figures for the rest of the
15% headline (workloads 5 and 4) and for workload 4's recompute-ratio sweep
(0-100%), context legs (Full-Recompute, standalone re-alignment, zero-copy,
Eq. (3) selection, host-resident pool, layer stack), and the CPU oracle timed
on a bounded sample of the same workload.
"""
from __future__ import annotations

import argparse
import hashlib
import json
import os
import re
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

HBM_PEAK_GBS = 8000.0          # MI355X HBM3E
BF16_PEAK_TFLOPS = 2500.0      # MI355X dense bf16 matrix
F32_PEAK_TFLOPS = 157.3        # MI355X fp32 vector
PROFILES = os.path.join(ROOT, "profiles")


def parse_args():
    ap = argparse.ArgumentParser(description=__doc__.splitlines()[0])
    ap.add_argument("--gpus", type=int, default=1)
    # The shader clock rises over the first tens of milliseconds of sustained
    # load: 500 untimed steps (about 90 ms on workload 2) reach the sustained
    # clock before the 1000 timed ones (about 0.2 s).
    ap.add_argument("--steps", type=int, default=1000)
    ap.add_argument("--warmup", type=int, default=500)
    ap.add_argument("--config", type=int, default=2, help="workload 1..5 (default 2)")
    ap.add_argument("--pct", type=int, default=None, help="recompute ratio in percent")
    ap.add_argument("--batches", type=int, default=4, help="independent batches rotated")
    ap.add_argument("--cpu-requests", type=int, default=None,
                    help="requests of batch 0 in the CPU oracle's sample (default: all; 0 = skip)")
    ap.add_argument("--cpu-seconds", type=float, default=10.0,
                    help="repeat the CPU oracle's sample until this much time has passed")
    ap.add_argument("--no-paged", action="store_true",
                    help="skip timing the zero-copy (paged attention) variant")
    ap.add_argument("--no-host-pool", action="store_true",
                    help="skip timing the token-granular gather from a pinned host pool")
    ap.add_argument("--stack-layers", type=int, default=4,
                    help="layers of the multi-layer leg (0 skips it)")
    ap.add_argument("--no-eq3", action="store_true",
                    help="skip timing the selection by the full Eq. (3) score")
    ap.add_argument("--no-workloads", action="store_true",
                    help="skip the other workloads (5 and 4 at 15%%, the ratio sweep on 4, 3 at 10%%, 1)")
    ap.add_argument("--no-full-prefill", action="store_true",
                    help="skip timing the Full-Recompute baseline")
    ap.add_argument("--chain", choices=("auto", "copy", "vref"), default="auto",
                    help="value rows: copied into the assembled V (copy) or read through a table "
                         "of row addresses (vref); auto: vref where the library supports it "
                         "(bf16, D = 128, at most 64 segments per request), else copy")
    ap.add_argument("--no-two-streams", action="store_true",
                    help="skip the two-stream pipelined context leg (its kernels overlap, so a "
                         "kernel-trace profile would mix their durations into the headline's)")
    ap.add_argument("--copy-calibration", action="store_true",
                    help="only run a plain 1 GiB device copy (HBM counter calibration)")
    return ap.parse_args()


def code_text(text: str) -> str:
    """A source file without comments and whitespace: edits to comments or
    layout do not change the digest of the code they describe."""
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    text = re.sub(r"//[^\n]*", "", text)
    return re.sub(r"\s+", "", text)


def source_digest(*names) -> str:
    h = hashlib.sha256()
    for n in names:
        with open(os.path.join(ROOT, "paper_2605_07443_amd", "csrc", n), encoding="utf-8") as f:
            h.update(code_text(f.read()).encode())
    return h.hexdigest()[:16]


def load_traffic(config: int, pct: int):
    """Measured HBM bytes per launch from committed rocprofv3 counter runs, if
    they were taken on the current kernel sources; else None."""
    path = os.path.join(PROFILES, f"traffic_config{config}_pct{pct}.md")
    if not os.path.exists(path):
        return None
    m = re.search(r"```json\n(.*?)\n```", open(path).read(), re.S)
    if not m:
        return None
    return json.loads(m.group(1))


def copy_calibration():
    import torch
    n = 1 << 30
    a = torch.empty(n, dtype=torch.uint8, device="cuda")
    a.random_()
    b = torch.empty_like(a)
    for _ in range(5):
        b.copy_(a)
    torch.cuda.synchronize()
    print(json.dumps({"copy_bytes_read": n, "copy_bytes_written": n, "launches": 5}), flush=True)


def use_vref(cfg, batches, chain: str) -> bool:
    """Whether a workload runs the value-reference chain (see --chain)."""
    ok = cfg.dtype == "bf16" and cfg.D == 128 and all(segs.S <= 64 for (_, segs, _) in batches)
    if chain == "vref" and not ok:
        raise SystemExit(f"--chain vref: workload {cfg.name} is outside the value-reference chain")
    return chain == "vref" or (chain == "auto" and ok)


def kern(kernels: dict, name: str) -> dict:
    """Per-kernel figures by base name, whichever chain produced them."""
    return kernels[name] if name in kernels else kernels[name + "_vref"]


def make_batches(cfg, config_id: int, R: int, n_batches: int, dev):
    """`n_batches` independent request batches over one shared pool (so the
    working set exceeds the 256 MB Infinity Cache), each with its buffers."""
    from paper_2605_07443_amd import inputs, ops
    base = 1000 * config_id
    batches, pools = [], None
    for i in range(n_batches):
        w = inputs.make(cfg, base + i, device=dev, pool_seed=base, pools=pools)
        pools = w.pools
        segs = ops.prepare_segments(w.segs, cfg.N, w.pools, dev)
        bufs = ops.PrefillBuffers.alloc(cfg.B, cfg.N, cfg.Hq, cfg.Hkv, cfg.D, R, cfg.torch_dtype, dev,
                                        v_ref=True)
        batches.append((w, segs, bufs))
    return batches


def time_selective(cfg, k: int, batches, cos, sin, steps: int, warmup: int, stream,
                   vref: bool = False) -> dict:
    """Per-kernel durations first: max(steps, 400) steps (gather + score ->
    top-k + patch -> attention, rotating over the batches) with HIP events on
    the launch stream between the kernels (each event record adds a gap to the
    stream, about 20 us per step for four of them, so they stay out of the
    timed loop). Then `warmup` steps and `steps` timed steps in a loop with
    nothing but the steps in it, which give the step time. The events pass
    coming first also keeps a short timed region in the state a long run
    reaches: right after the Full-Recompute leg's matrix work the shader
    clock is lower for some tens of milliseconds (20 timed steps measured
    2.5% slower there). The host synchronises after the warm-up steps and
    after the timed ones (that gap measured no slower than none).
    vref: the value-reference chain (K gathered and aligned, V read through a
    table of row addresses) instead of the assembled copy."""
    import torch
    from paper_2605_07443_amd import ops
    B, N, Hq, Hkv, D = cfg.B, cfg.N, cfg.Hq, cfg.Hkv, cfg.D
    R = cfg.n_fresh + k
    row = Hkv * D * (2 if cfg.dtype == "bf16" else 4)

    def step(i, ev=None):
        w, segs, bufs = batches[i % len(batches)]
        if ev is not None:
            ev[0].record(stream)
        if vref:
            ops.kv_assemble_vref(w.pools, segs, w.k_fresh, w.v_fresh, cos, sin, bufs.k_asm,
                                 bufs.v_ref, scores_out=bufs.scores)
        else:
            ops.kv_assemble(w.pools, segs, w.k_fresh, w.v_fresh, cos, sin, bufs.k_asm, bufs.v_asm,
                            scores_out=bufs.scores)
        if ev is not None:
            ev[1].record(stream)
        if vref:
            ops.select_tokens_vref(segs, k, w.k_fresh, w.v_fresh, bufs.k_asm, bufs.v_ref,
                                   scores_in=bufs.scores, rows_out=bufs.rows)
        else:
            ops.select_tokens(segs, k, w.k_fresh, w.v_fresh, bufs.k_asm, bufs.v_asm,
                              scores_in=bufs.scores, rows_out=bufs.rows, patch=True)
        if ev is not None:
            ev[2].record(stream)
        if R > 0 and vref:
            ops.selective_attention_vref(w.q, bufs.k_asm, bufs.v_ref, bufs.rows, None, bufs.out)
        elif R > 0:
            ops.selective_attention(w.q, bufs.k_asm, bufs.v_asm, bufs.rows, None, bufs.out)
        if ev is not None:
            ev[3].record(stream)

    n_inst = max(steps, 400)
    evs = [[torch.cuda.Event(enable_timing=True) for _ in range(4)] for _ in range(n_inst)]
    t_start = torch.cuda.Event(enable_timing=True)
    t_end = torch.cuda.Event(enable_timing=True)
    i_start = torch.cuda.Event(enable_timing=True)
    i_end = torch.cuda.Event(enable_timing=True)
    i_start.record(stream)
    for i in range(n_inst):
        step(i, evs[i])
    i_end.record(stream)
    for i in range(warmup):
        step(i)
    torch.cuda.synchronize()   # the timed steps are bracketed by synchronisations
    t_start.record(stream)
    for i in range(steps):
        step(warmup + i)
    t_end.record(stream)
    torch.cuda.synchronize()
    total_ms = t_start.elapsed_time(t_end)
    steps_i = n_inst
    # attention work of each batch from its actual rows (unmasked causal work;
    # the selection of a batch is the same in every step)
    att_flops = []
    for (w, segs, bufs) in batches:
        r = bufs.rows.to(torch.int64).cpu()
        att_flops.append(4.0 * D * Hq * float((r + 1).sum()) if R > 0 else 0.0)
    asm_ms = sum(e[0].elapsed_time(e[1]) for e in evs) / steps_i
    sel_ms = sum(e[1].elapsed_time(e[2]) for e in evs) / steps_i
    att_ms = sum(e[2].elapsed_time(e[3]) for e in evs) / steps_i
    flops = sum(att_flops[i % len(batches)] for i in range(steps_i)) / steps_i

    # assemble: read K,V rows, write K,V rows, read the fresh K row of every
    # cached position and write its score; select: read scores, write rows,
    # patch k rows of K and V (read fresh, write assembled). With value
    # references the V rows are neither read nor written by these two: the
    # gather writes one 8-byte address per position instead, the patch one
    # per patched row.
    if vref:
        gather_bytes = 2.0 * B * N * row + 1.0 * B * (N - cfg.n_fresh) * row + 4.0 * B * N + 8.0 * B * N
        select_bytes = 4.0 * B * N + 4.0 * B * R + 2.0 * B * k * row + 8.0 * B * k
    else:
        gather_bytes = 4.0 * B * N * row + 1.0 * B * (N - cfg.n_fresh) * row + 4.0 * B * N
        select_bytes = 4.0 * B * N + 4.0 * B * R + 4.0 * B * k * row
    mfma_peak = BF16_PEAK_TFLOPS if cfg.dtype == "bf16" else F32_PEAK_TFLOPS

    def hbm(bytes_, ms):
        a = bytes_ / (ms * 1e-3) / 1e9 if ms > 0 else 0.0
        return {"bound": "hbm", "achieved": round(a, 1), "peak": HBM_PEAK_GBS, "unit": "GB/s",
                "frac": round(a / HBM_PEAK_GBS, 4), "bytes_per_launch": bytes_}

    att_tf = flops / (att_ms * 1e-3) / 1e12 if att_ms > 0 else 0.0
    sfx = "_vref" if vref else ""
    kernels = {
        "rc_kv_assemble" + sfx: dict(us=round(asm_ms * 1e3, 2), **hbm(gather_bytes, asm_ms)),
        "rc_select_tokens" + sfx: dict(us=round(sel_ms * 1e3, 2), **hbm(select_bytes, sel_ms)),
        "rc_selective_attention" + sfx: {
            "us": round(att_ms * 1e3, 2), "bound": "mfma" if cfg.dtype == "bf16" else "alu",
            "achieved": round(att_tf, 2), "peak": mfma_peak, "unit": "TFLOP/s",
            "frac": round(att_tf / mfma_peak, 4), "flops_per_launch": flops},
    }
    ms_per_step = total_ms / steps
    return {"ms_per_step": round(ms_per_step, 5),
            "ms_per_step_with_kernel_events": round(i_start.elapsed_time(i_end) / steps_i, 5),
            "total_ms": total_ms, "att_flops": att_flops, "kernels": kernels,
            "R": R, "selected_tokens_per_s": round(B * R / (ms_per_step * 1e-3), 1),
            "us_per_request": round(ms_per_step * 1e3 / B, 3)}


def time_two_streams(cfg, k: int, batches, cos, sin, steps: int, warmup: int, vref: bool) -> dict:
    """Context for serving: the same steps with consecutive batches on two
    streams (batch i on stream i % 2; the rotated batches keep their buffers
    on one stream), so that one batch's gather and selection can run beside
    the previous batch's attention. Timed from an event on stream 0 that
    stream 1 waits for, to an event on stream 0 after it has waited for
    stream 1's last step."""
    import torch
    from paper_2605_07443_amd import ops
    if len(batches) % 2:
        return None
    ss = [torch.cuda.Stream(), torch.cuda.Stream()]   # default priority

    def step(i):
        w, segs, bufs = batches[i % len(batches)]
        s = ss[i % 2]
        if vref:
            ops.kv_assemble_vref(w.pools, segs, w.k_fresh, w.v_fresh, cos, sin, bufs.k_asm,
                                 bufs.v_ref, scores_out=bufs.scores, stream=s)
            ops.select_tokens_vref(segs, k, w.k_fresh, w.v_fresh, bufs.k_asm, bufs.v_ref,
                                   scores_in=bufs.scores, rows_out=bufs.rows, stream=s)
            ops.selective_attention_vref(w.q, bufs.k_asm, bufs.v_ref, bufs.rows, None, bufs.out,
                                         stream=s)
        else:
            ops.kv_assemble(w.pools, segs, w.k_fresh, w.v_fresh, cos, sin, bufs.k_asm, bufs.v_asm,
                            scores_out=bufs.scores, stream=s)
            ops.select_tokens(segs, k, w.k_fresh, w.v_fresh, bufs.k_asm, bufs.v_asm,
                              scores_in=bufs.scores, rows_out=bufs.rows, patch=True, stream=s)
            ops.selective_attention(w.q, bufs.k_asm, bufs.v_asm, bufs.rows, None, bufs.out,
                                    stream=s)

    torch.cuda.synchronize()
    for i in range(warmup):
        step(i)
    torch.cuda.synchronize()
    a = torch.cuda.Event(enable_timing=True)
    z = torch.cuda.Event(enable_timing=True)
    e1 = torch.cuda.Event()
    a.record(ss[0])
    ss[1].wait_event(a)
    for i in range(steps):
        step(warmup + i)
    e1.record(ss[1])
    ss[0].wait_event(e1)
    z.record(ss[0])
    torch.cuda.synchronize()
    ms = a.elapsed_time(z) / steps
    B, R = cfg.B, cfg.n_fresh + k
    return {"streams": 2, "ms_per_step": round(ms, 5), "value": round(B * R / (ms * 1e-3), 1)}


def other_workloads(args, dev, stream) -> dict:
    """The rest of the 15% headline (workload 5, the gather-bound case, and
    workload 4), workload 4's recompute-ratio sweep (the kernel-level
    analogue of the paper's ratio study), the long-prompt workload 3 at 10%
    and the tiny fp32 workload 1: step time, selected tok/s, microseconds per
    request, and the gather and attention roofline fractions of each,
    measured as the headline is."""
    import torch
    from paper_2605_07443_amd import inputs, ops
    out = {}
    # lightest first: the headline is timed right after these legs, so the last
    # one keeps the GPU at its sustained clock
    for cid, pcts in ((1, (15,)), (3, (10,)), (4, inputs.SWEEP_PCTS), (5, (15,))):
        if cid == args.config:
            continue
        cfg = inputs.WORKLOADS[cid]
        cos, sin = ops.rope_table(cfg.N, cfg.D, cfg.rope_base, dev)
        batches = make_batches(cfg, cid, cfg.n_fresh, args.batches, dev)
        rows = {}
        for pct in pcts:
            k = cfg.k_for(pct)
            R = cfg.n_fresh + k
            for (_, _, bufs) in batches:   # row and output buffers of this ratio
                bufs.rows = torch.empty((cfg.B, R), dtype=torch.int32, device=dev)
                bufs.out = torch.empty((cfg.B, R, cfg.Hq, cfg.D), dtype=cfg.torch_dtype, device=dev)
            vr = use_vref(cfg, batches, args.chain)
            r = time_selective(cfg, k, batches, cos, sin, args.steps, args.warmup, stream, vref=vr)
            kk = r["kernels"]
            rows[str(pct)] = {
                "chain": "vref" if vr else "copy",
                "R": r["R"], "ms_per_step": r["ms_per_step"],
                "selected_tokens_per_s": r["selected_tokens_per_s"],
                "us_per_request": r["us_per_request"],
                "gather_us": kern(kk, "rc_kv_assemble")["us"],
                "gather_frac": kern(kk, "rc_kv_assemble")["frac"],
                "select_us": kern(kk, "rc_select_tokens")["us"],
                "attention_us": kern(kk, "rc_selective_attention")["us"],
                "attention_frac": kern(kk, "rc_selective_attention")["frac"]}
        name = f"config{cid}:{cfg.name}"
        out[name] = rows if len(pcts) > 1 else rows[str(pcts[0])]
        del batches
        torch.cuda.empty_cache()
    return out


def main():
    args = parse_args()
    world = int(os.environ.get("WORLD_SIZE", "1"))
    if args.gpus != 1 or world != 1:
        print("bench.py measures one GPU only: the library has no multi-GPU path "
              "(requests are independent and would be split across GPUs by request)",
              file=sys.stderr)
        sys.exit(2)
    if args.copy_calibration:
        copy_calibration()
        return

    import numpy as np
    import torch

    from paper_2605_07443_amd import _lib, inputs, ops

    _lib.load()  # fails loudly when the HIP library is not built
    dev = torch.device("cuda:0")
    cfg = inputs.WORKLOADS[args.config]
    pct = cfg.pct if args.pct is None else args.pct
    k = cfg.k_for(pct)
    R = cfg.n_fresh + k
    B, N, Hq, Hkv, D = cfg.B, cfg.N, cfg.Hq, cfg.Hkv, cfg.D
    es = 2 if cfg.dtype == "bf16" else 4
    row = Hkv * D * es

    base = 1000 * args.config   # seed base of this workload's draws
    batches = make_batches(cfg, args.config, R, args.batches, dev)
    cos, sin = ops.rope_table(N, D, cfg.rope_base, dev)
    torch.cuda.synchronize()
    stream = torch.cuda.current_stream()

    mfma_peak = BF16_PEAK_TFLOPS if cfg.dtype == "bf16" else F32_PEAK_TFLOPS

    def hbm(bytes_, ms):
        a = bytes_ / (ms * 1e-3) / 1e9 if ms > 0 else 0.0
        return {"bound": "hbm", "achieved": round(a, 1), "peak": HBM_PEAK_GBS, "unit": "GB/s",
                "frac": round(a / HBM_PEAK_GBS, 4), "bytes_per_launch": bytes_}

    # ---- standalone re-alignment (rc_rerope) of the reused rows of one batch,
    # in place on a copy of its assembled K: delta = dst_start on pool rows
    rerope = None
    w0, segs0, bufs0 = batches[0]
    ops.kv_assemble(w0.pools, segs0, w0.k_fresh, w0.v_fresh, cos, sin, bufs0.k_asm, bufs0.v_asm)
    delta = torch.zeros((B, N), dtype=torch.int32)
    for b in range(B):
        for dst, ln, pool, _blk in w0.segs[b].tolist():
            if pool >= 0:
                delta[b, dst:dst + ln] = dst
    n_reused = int((delta != 0).sum())
    delta = delta.to(dev)
    kk = bufs0.k_asm.clone()
    reps = max(5, min(50, args.steps // 2))
    ops.rerope(kk, delta, cos, sin)
    torch.cuda.synchronize()
    r0, r1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    r0.record(stream)
    for _ in range(reps):
        ops.rerope(kk, delta, cos, sin)
    r1.record(stream)
    torch.cuda.synchronize()
    r_ms = r0.elapsed_time(r1) / reps
    rerope = dict(us=round(r_ms * 1e3, 2), reused_rows=n_reused, **hbm(2.0 * n_reused * row, r_ms))
    del kk, delta

    # ---- zero-copy variant: score-only alignment pass, top-k, paged attention
    paged = None
    if not args.no_paged and cfg.dtype == "bf16" and R > 0:
        pbuf = ops.PrefillBuffers.alloc(B, N, Hq, Hkv, D, R, cfg.torch_dtype, dev)

        def stepp(i, ev=None):
            w, segs, _ = batches[i % len(batches)]
            if ev is not None:
                ev[0].record(stream)
            ops.kv_assemble(w.pools, segs, w.k_fresh, w.v_fresh, cos, sin, scores_out=pbuf.scores,
                            score_only=True)
            if ev is not None:
                ev[1].record(stream)
            ops.select_tokens(segs, k, w.k_fresh, w.v_fresh, None, None, scores_in=pbuf.scores,
                              rows_out=pbuf.rows, patch=False)
            if ev is not None:
                ev[2].record(stream)
            ops.paged_attention(w.q, w.k_fresh, w.v_fresh, w.pools, segs, pbuf.rows, cos, sin,
                                None, pbuf.out)
            if ev is not None:
                ev[3].record(stream)

        for i in range(3):
            stepp(i)
        torch.cuda.synchronize()
        reps = max(5, min(50, args.steps // 2))
        # step time from a bare loop, kernel split from a pass with events
        p0, p1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        p0.record(stream)
        for i in range(reps):
            stepp(i)
        p1.record(stream)
        torch.cuda.synchronize()
        p_ms = p0.elapsed_time(p1) / reps
        evp = [[torch.cuda.Event(enable_timing=True) for _ in range(4)] for _ in range(reps)]
        for i in range(reps):
            stepp(i, evp[i])
        torch.cuda.synchronize()
        pp = [sum(e[j].elapsed_time(e[j + 1]) for e in evp) / reps for j in range(3)]
        p_rows = []
        for i in range(len(batches)):
            stepp(i)
            p_rows.append(4.0 * D * Hq * float((pbuf.rows.to(torch.int64).cpu() + 1).sum()))
        p_flops = sum(p_rows[i % len(batches)] for i in range(reps)) / reps
        score_bytes = 2.0 * B * (N - cfg.n_fresh) * row + 4.0 * B * N
        pa_tf = p_flops / (pp[2] * 1e-3) / 1e12
        paged = {"ms": round(p_ms, 4), "selected_tokens_per_s": round(B * R / (p_ms * 1e-3), 1),
                 "kernels": {
                     "rc_kv_assemble_score_only": dict(us=round(pp[0] * 1e3, 2), **hbm(score_bytes, pp[0])),
                     "rc_select_tokens_no_patch": {"us": round(pp[1] * 1e3, 2)},
                     "rc_paged_attention": {"us": round(pp[2] * 1e3, 2), "bound": "mfma",
                                            "achieved": round(pa_tf, 2), "peak": mfma_peak,
                                            "unit": "TFLOP/s", "frac": round(pa_tf / mfma_peak, 4),
                                            "flops_per_launch": p_flops}}}
        del pbuf

    # ---- selection by the full Eq. (3) score: the first layer in full (with
    # log-sum-exp), attention mass, assembly, score, history/item top-k, patch
    eq3 = None
    if not args.no_eq3 and cfg.dtype == "bf16":
        kh, ki = cfg.k_split(pct)
        lam = 0.5
        R3 = cfg.n_fresh + kh + ki
        ebuf = ops.Eq3Buffers.alloc(B, N, Hq, Hkv, D, R3, cfg.torch_dtype, dev)
        mask = inputs.ITEM_POOL_MASK

        def step3(i, ev=None):
            w, segs, _ = batches[i % len(batches)]
            if ev is not None:
                ev[0].record(stream)
            ops.selective_attention_lse(w.q, w.k_fresh, w.v_fresh, None, None, ebuf.out_full,
                                        ebuf.lse)
            if ev is not None:
                ev[1].record(stream)
            ops.attention_mass(w.q, w.k_fresh, ebuf.lse, None, ebuf.mass)
            if ev is not None:
                ev[2].record(stream)
            ops.kv_assemble(w.pools, segs, w.k_fresh, w.v_fresh, cos, sin, ebuf.k_asm, ebuf.v_asm)
            if ev is not None:
                ev[3].record(stream)
            ops.select_tokens_eq3(segs, mask, lam, kh, ki, w.k_fresh, w.v_fresh, ebuf.k_asm,
                                  ebuf.v_asm, mass=ebuf.mass, scores_out=ebuf.scores,
                                  rows_out=ebuf.rows, patch=True)
            if ev is not None:
                ev[4].record(stream)

        for i in range(3):
            step3(i)
        torch.cuda.synchronize()
        reps = max(3, min(20, args.steps // 5))
        ev3 = [[torch.cuda.Event(enable_timing=True) for _ in range(5)] for _ in range(reps)]
        for i in range(reps):
            step3(i, ev3[i])
        torch.cuda.synchronize()
        part = [sum(e[j].elapsed_time(e[j + 1]) for e in ev3) / reps for j in range(4)]
        e3_ms = sum(e[0].elapsed_time(e[4]) for e in ev3) / reps
        causal = B * N * (N + 1) / 2.0
        att_f, mass_f = 4.0 * D * Hq * causal, 2.0 * D * Hq * causal
        n_div = cfg.n_fresh + cfg.n_hist_reused   # positions whose K/V divergence is read
        sel3_bytes = (4.0 * B * n_div * row + 4.0 * B * Hkv * N + 4.0 * B * N + 4.0 * B * N
                      + 4.0 * B * R3 + 4.0 * B * (kh + ki) * row)

        def mf(fl, ms):
            a = fl / (ms * 1e-3) / 1e12
            return {"bound": "mfma", "achieved": round(a, 2), "peak": BF16_PEAK_TFLOPS,
                    "unit": "TFLOP/s", "frac": round(a / BF16_PEAK_TFLOPS, 4), "flops_per_launch": fl}

        eq3 = {"ms": round(e3_ms, 4), "lambda": lam, "budgets": [kh, ki],
               "selected_rows_per_request": R3,
               "selected_tokens_per_s": round(B * R3 / (e3_ms * 1e-3), 1),
               "kernels": {
                   "rc_selective_attention_lse": dict(us=round(part[0] * 1e3, 2), **mf(att_f, part[0])),
                   "rc_attention_mass": dict(us=round(part[1] * 1e3, 2), **mf(mass_f, part[1])),
                   "rc_kv_assemble": dict(us=round(part[2] * 1e3, 2),
                                          **hbm(4.0 * B * N * row, part[2])),
                   "rc_select_tokens_eq3": dict(us=round(part[3] * 1e3, 2), **hbm(sel3_bytes, part[3]))}}
        del ebuf

    # ---- token-granular history (single-token prototypes) with the prototype
    # pool in pinned host memory: PCIe-inclusive gather, and the Eq. (3)
    # selection with that gather overlapped with the first layer
    host = None
    if not args.no_host_pool and cfg.dtype == "bf16":
        tw = inputs.make_prototypes(cfg, base + 7, device=dev, n_protos=65536)
        tmap = tw.token_map.to(dev)
        dev_pools = tw.w.pools
        host_pools = [ops.pin_pool(dev_pools[0]), dev_pools[1]]
        status = ops.prepare_segments(tw.status_segs, N, dev_pools, dev, check_blocks=False)
        kh, ki = cfg.k_split(pct)
        hb = ops.Eq3Buffers.alloc(B, N, Hq, Hkv, D, cfg.n_fresh + kh + ki, cfg.torch_dtype, dev)
        ww = tw.w
        side = torch.cuda.Stream()

        def timeit(fn, reps):
            fn()
            torch.cuda.synchronize()
            a, z = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            a.record(stream)
            for _ in range(reps):
                fn()
            z.record(stream)
            torch.cuda.synchronize()
            return a.elapsed_time(z) / reps

        def gather(pools_, wgs=0):
            return lambda: ops.kv_gather_tokens(pools_, tmap, ww.k_fresh, ww.v_fresh, cos, sin,
                                                hb.k_asm, hb.v_asm, hb.scores, max_workgroups=wgs)

        def eq3_path(pools_, gs):
            return lambda: ops.eq3_select_tokens_path(ww.q, ww.k_fresh, ww.v_fresh, pools_, tmap,
                                                      status, inputs.ITEM_POOL_MASK, 0.5, kh, ki,
                                                      cos, sin, bufs=hb, gather_stream=gs)

        reps = max(3, min(10, args.steps // 10))
        g_dev = timeit(gather(dev_pools), reps * 3)
        g_host = timeit(gather(host_pools), reps * 3)
        g_host_b = timeit(gather(host_pools, ops.OVERLAP_GATHER_WORKGROUPS), reps * 3)
        # The three Eq. (3) variants alternate over five rounds and each keeps
        # its median: timed one after another, the shader clock's drift
        # between them is as large as the overlap being measured.
        variants = (eq3_path(dev_pools, None), eq3_path(host_pools, None), eq3_path(host_pools, side))
        runs = [[], [], []]
        for _ in range(5):
            for i, fn in enumerate(variants):
                runs[i].append(timeit(fn, reps))
        e_dev, e_seq, e_ovl = (float(np.median(r)) for r in runs)
        pcie_bytes = 2.0 * B * cfg.hist_len * row   # K and V rows of the history, from host memory
        host = {"n_protos": 65536, "history_bytes_from_host": pcie_bytes,
                "gather_device_pool_us": round(g_dev * 1e3, 2),
                "gather_host_pool_us": round(g_host * 1e3, 2),
                "gather_host_pool_bounded_us": round(g_host_b * 1e3, 2),
                "gather_bounded_workgroups": ops.OVERLAP_GATHER_WORKGROUPS,
                "host_read_GBps": round(pcie_bytes / ((g_host - g_dev) * 1e-3) / 1e9, 1)
                if g_host > g_dev else None,
                "eq3_device_pool_ms": round(e_dev, 4),
                "eq3_host_pool_sequential_ms": round(e_seq, 4),
                "eq3_host_pool_overlapped_ms": round(e_ovl, 4),
                "overlap_hidden_fraction": round((e_seq - e_ovl) / (e_seq - e_dev), 3)
                if e_seq > e_dev else None,
                "overlapped_over_device_pool": round(e_ovl / e_dev, 4)}
        del tw, ww, hb, host_pools, dev_pools, tmap

    # ---- several layers (Llama-3-8B layer dimensions, random weights): the
    # first layer for every row picks the rows, later layers recompute only
    # them; against the full recompute of every row of every layer
    stack = None
    if args.stack_layers > 0 and cfg.dtype == "bf16":
        Hd, I, nl = 4096, 14336, args.stack_layers
        sx, slayers, spools, ssegs = inputs.make_stack(cfg, base + 11, nl, Hd, I, device=dev)
        W = 16
        sseg = ops.prepare_segments(ops.segments_with_window(ssegs.numpy(), N, W), N, spools[0], dev)
        sk = (sseg.n_reused * pct + 99) // 100
        scos, ssin = cos, sin

        def run_sel():
            return ops.stack_prefill(sx, slayers, spools, sseg, sk, scos, ssin)

        def run_full():
            return ops.stack_full(sx, slayers, Hq, Hkv, D, scos, ssin)

        def timeit2(fn, reps):
            fn()
            torch.cuda.synchronize()
            a, z = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            a.record(stream)
            for _ in range(reps):
                fn()
            z.record(stream)
            torch.cuda.synchronize()
            return a.elapsed_time(z) / reps

        reps = max(2, min(5, args.steps // 20))
        t_sel = timeit2(run_sel, reps)
        t_full = timeit2(run_full, reps)
        R2 = sseg.n_fresh + sk
        per_row = 2.0 * Hd * ((Hq + 2 * Hkv) * D + Hq * D + 3 * I)      # projection FLOPs of one row
        sel_flops = B * N * 2.0 * Hd * (Hq + 2 * Hkv) * D + (B * R2) * (per_row - 2.0 * Hd * (Hq + 2 * Hkv) * D) \
            + (nl - 1) * B * R2 * per_row
        stack = {"layers": nl, "hidden": Hd, "intermediate": I, "window": W,
                 "rows_per_request": R2, "selective_ms": round(t_sel, 3), "full_ms": round(t_full, 3),
                 "speedup": round(t_full / t_sel, 2),
                 "selective_projection_tflops": round(sel_flops / (t_sel * 1e-3) / 1e12, 1)}
        del sx, slayers, spools

    # ---- the rest of the 15% headline and the recompute-ratio sweep
    workloads = None
    if not args.no_workloads:
        workloads = other_workloads(args, dev, stream)

    # ---- Full-Recompute baseline on the same batch (context), enqueued right
    # before the headline: about 60 ms of matrix work without a host gap, so
    # that the headline starts at the GPU's sustained clock (from idle the
    # clock rises over the first tens of milliseconds of load, and a short
    # timed region would measure that ramp)
    full = None
    if not args.no_full_prefill and cfg.dtype == "bf16":
        w0 = batches[0][0]
        fout = torch.empty((B, N, Hq, D), dtype=cfg.torch_dtype, device=dev)
        ops.full_prefill(w0.q, w0.k_fresh, w0.v_fresh, out=fout)
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        ops.full_prefill(w0.q, w0.k_fresh, w0.v_fresh, out=fout)
        torch.cuda.synchronize()
        f_reps = max(3, min(200, int(0.06 / max(time.perf_counter() - t0, 1e-4))))
        f_ev = (torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))
        f_ev[0].record(stream)
        for _ in range(f_reps):
            ops.full_prefill(w0.q, w0.k_fresh, w0.v_fresh, out=fout)
        f_ev[1].record(stream)

    # ---- the headline, timed last, right after the Full-Recompute work
    vref = use_vref(cfg, batches, args.chain)
    head = time_selective(cfg, k, batches, cos, sin, args.steps, args.warmup, stream, vref=vref)
    ms_per_step = head["ms_per_step"]
    total_ms = head["total_ms"]
    kernels = head["kernels"]
    dominant = max(kernels, key=lambda n: kernels[n]["us"])
    dk = kernels[dominant]
    # context: the chain that copies V into the assembled tensor, same batches
    copy_chain = None
    if vref:
        c = time_selective(cfg, k, batches, cos, sin, args.steps, args.warmup, stream, vref=False)
        copy_chain = {"ms_per_step": c["ms_per_step"],
                      "value": round(B * R / (c["ms_per_step"] * 1e-3), 1),
                      "kernels": c["kernels"],
                      "vref_speedup": round(c["ms_per_step"] / ms_per_step, 3)}
    two = None
    if not args.no_two_streams:
        try:   # context only: a failure here must not cost the headline line
            two = time_two_streams(cfg, k, batches, cos, sin, args.steps, args.warmup, vref)
            if two is not None:
                two["vs_one_stream"] = round(ms_per_step / two["ms_per_step"], 3)
        except Exception as e:  # noqa: BLE001
            two = {"error": f"{type(e).__name__}: {e}"}
            print(f"two-stream leg failed: {two['error']}", file=sys.stderr)
    traffic = None
    tr = load_traffic(args.config, pct)
    digest = {"rc_kv_assemble": source_digest("assemble.hip"),
              "rc_select_tokens": source_digest("select.hip"),
              "rc_selective_attention": source_digest("attention.hip"),
              "rc_attention_mass": source_digest("mass.hip"),
              "rc_gemm_bf16": source_digest("gemm.hip")}
    base_name = dominant[:-len("_vref")] if dominant.endswith("_vref") else dominant
    if tr and tr.get("source_digest", {}).get(base_name) == digest[base_name]:
        traffic = tr.get("kernels", {}).get(dominant, {}).get("hbm_bytes")
    roofline = {"kernel": dominant, "bound": dk["bound"], "achieved": dk["achieved"],
                "peak": dk["peak"], "unit": dk["unit"], "frac": dk["frac"], "traffic": traffic}
    if not args.no_full_prefill and cfg.dtype == "bf16":
        fms = f_ev[0].elapsed_time(f_ev[1]) / f_reps
        fflops = 4.0 * D * Hq * B * N * (N + 1) / 2
        full = {"ms": round(fms, 4), "reps": f_reps, "tflops": round(fflops / (fms * 1e-3) / 1e12, 2),
                "frac_of_bf16_peak": round(fflops / (fms * 1e-3) / 1e12 / BF16_PEAK_TFLOPS, 4),
                "selective_speedup": round(fms / ms_per_step, 3)}
        del fout
    if paged is not None:
        paged["vs_headline_step"] = round(ms_per_step / paged["ms"], 3)

    # ---- CPU oracle on a bounded sample of the same workload
    cpu = None
    if args.cpu_requests is None or args.cpu_requests > 0:
        from oracle import oracle as O
        w0 = batches[0][0]
        n = B if args.cpu_requests is None else min(args.cpu_requests, B)
        H = inputs.to_host_bits
        sub = inputs.Workload(cfg=cfg, seed=w0.seed, q=w0.q[:n], k_fresh=w0.k_fresh[:n],
                              v_fresh=w0.v_fresh[:n], pools=w0.pools, segs=w0.segs[:n].clone(),
                              item_ids=w0.item_ids[:n], hist_ids=w0.hist_ids[:n])
        subpools, segs_sub = inputs.referenced_subpools(sub)
        qh, kh, vh = H(sub.q), H(sub.k_fresh), H(sub.v_fresh)
        ocos, osin = O.rope_table(N, D, cfg.rope_base)
        reps = 0
        t0 = time.perf_counter()
        while True:
            O.selective_prefill(qh, kh, vh, subpools, segs_sub, k, ocos, osin)
            reps += 1
            dt = time.perf_counter() - t0
            if dt >= args.cpu_seconds or reps >= 50:
                break
        cpu = {"value": round(reps * n * R / dt, 1), "unit": "tokens/s/layer",
               "cores": O.num_threads(), "kind": "oracle", "seconds": round(dt, 2),
               "sample": f"{reps} pass(es) over {n} of {B} requests of one batch: the whole oracle "
                         f"pipeline (assemble, rerope, deviation, top-k, patch, attention of {R} "
                         f"rows each), fp64 accumulation"}

    value = B * R * args.steps / (total_ms * 1e-3)
    result = {
        "metric": "selected-query tokens/s/layer at 15% recompute (one attention layer)"
                  if pct == 15 else f"selected-query tokens/s/layer at {pct}% recompute",
        "value": round(value, 1),
        "unit": "tokens/s/layer",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms_per_step, 5),
        "ms_per_step_with_kernel_events": head["ms_per_step_with_kernel_events"],
        "us_per_request": round(ms_per_step * 1e3 / B, 3),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": cfg.dtype,
        "data": "synthetic",
        "config": {"workload": f"config{args.config}:{cfg.name}",
                   "chain": "vref" if vref else "copy", "B": B, "N": N,
                   "recompute_pct": pct, "selected_rows_per_request": R, "Hq": Hq, "Hkv": Hkv,
                   "D": D, "pools": [[cfg.hist_pool, cfg.hist_len], [cfg.item_pool, cfg.item_len]],
                   "batches_rotated": args.batches},
        "roofline": roofline,
        "kernels": kernels,
        "assembled_copy_chain": copy_chain,
        "pipelined_two_streams": two,
        "full_prefill": full,
        "rerope_standalone": rerope,
        "paged_prefill": paged,
        "eq3_selection": eq3,
        "token_history_host_pool": host,
        "layer_stack": stack,
        "workloads": workloads,
        "cpu_baseline": cpu,
        "source_digest": digest,
    }
    print(json.dumps(result), flush=True)


if __name__ == "__main__":
    main()
