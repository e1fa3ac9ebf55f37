#!/usr/bin/env python3
"""Throughput of the target verification step on one MI355X.

A step is one verification call (Section 4.2; Appendix C.2): one forward
pass of the 7B-shaped target over the pending root and k candidates against
the prefilled audio + instruction + committed KV cache, greedy acceptance,
correction and KV rollback.  The default workload is the Qwen2-7B-shaped
decoder (28 layers, hidden 3584, 28/4 heads, FFN 18944, vocab 152064, bf16,
random weights) with a 750-row audio + 32-token instruction prefix, a
256-token reply verified at k = 8 with candidate corruption p = 0.3.

Printed: one JSON line with committed tokens/s (`value`), ms per step, the
step's algorithmic HBM bandwidth and its fraction of the 8 TB/s peak, the
roofline of the dominant kernel (gate/up GEMM) from HIP events on the
library's stream, and the float64 CPU oracle timed on a bounded sample.

The K timed steps start at the beginning of the replies (so a given K
always covers the same stream positions); `full_pass` gives the tokens per
step of one whole pass over the replies, which a K-step window samples.
"""
import argparse
import json
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

from workload import configs as wc            # noqa: E402
from workload import gen                      # noqa: E402

PEAK_HBM_GBPS = 8000.0
METRIC = "committed tokens/sec and verify-step HBM GB/s (% peak), 7B-shape k=8, 1 GPU"
PROFILES = os.path.join(ROOT, "profiles")


def log(*a):
    print(*a, file=sys.stderr, flush=True)


def parse():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=60)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--workload", type=int, default=2, help="index of workload.configs.workload")
    ap.add_argument("--k", type=int, default=None)
    ap.add_argument("--p", type=float, default=None)
    ap.add_argument("--layers", type=int, default=None, help="(tuning only) override layer count")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-kernel-timing", action="store_true")
    ap.add_argument("--no-align", action="store_true", help="skip the candidate-buffer decoding measurement")
    ap.add_argument("--no-decoupled", action="store_true", help="skip the concurrent-drafter measurement")
    ap.add_argument("--no-width-profile", action="store_true",
                    help="skip the per-k step times (single-request workloads with a k sweep)")
    ap.add_argument("--passes", type=int, default=5, help="whole-reply passes behind `value` (median)")
    ap.add_argument("--no-configs", action="store_true", help="skip the 3B, long-audio and mixed-batch workloads")
    ap.add_argument("--trace-window", action="store_true",
                    help="profiling run: reference streams and every timed call at the workload's width, "
                         "nothing else (no passes, extras or back-to-back GEMM timing)")
    ap.add_argument("--library-gemm", action="store_true",
                    help="also time the vendor library's bf16 GEMM (torch.nn.functional.linear, i.e. "
                         "hipBLASLt/rocBLAS) on the verification GEMM shapes at W = 1 and the timed width")
    ap.add_argument("--calib-copy-mib", type=int, default=0,
                    help="also run one device-to-device copy of this many MiB (a plain copy kernel "
                         "of known size, for scaling hardware byte counters)")
    return ap.parse_args()


def traffic_from_profiles():
    """HBM bytes per gate/up launch from the committed rocprofv3 counter
    summary (profiles/gemm_gate_up_qwen7b_k8_pmc.md), if it was taken on
    the current library sources (its `library_source_sha` line)."""
    p = os.path.join(PROFILES, "gemm_gate_up_qwen7b_k8_pmc.md")
    if not os.path.exists(p):
        return None
    fields = {}
    for line in open(p):
        if ":" in line and line.startswith("- "):
            k, v = line[2:].split(":", 1)
            fields[k.strip()] = v.strip().strip("`")
    if fields.get("library_source_sha") != library_source_sha():
        return None
    try:
        return int(fields["traffic_bytes_per_launch"])
    except (KeyError, ValueError):
        return None


def library_source_sha():
    """Hash of the HIP library sources (a counter summary is valid only for
    the sources it was taken on)."""
    import hashlib
    h = hashlib.sha256()
    d = os.path.join(ROOT, "paper_2609_37617_amd", "csrc")
    for f in sorted(os.listdir(d)):
        h.update(f.encode())
        h.update(open(os.path.join(d, f), "rb").read())
    return h.hexdigest()[:16]


def copy_calibration(mib):
    """One device-to-device copy of `mib` MiB through the HIP runtime (its
    plain copy kernel reads and writes exactly that many bytes), so that
    hardware byte counters can be scaled by what they report for it."""
    import ctypes
    hip = ctypes.CDLL("libamdhip64.so")
    n = ctypes.c_size_t(mib << 20)
    src, dst = ctypes.c_void_p(), ctypes.c_void_p()
    assert hip.hipMalloc(ctypes.byref(src), n) == 0 and hip.hipMalloc(ctypes.byref(dst), n) == 0
    assert hip.hipMemset(src, 1, n) == 0
    assert hip.hipDeviceSynchronize() == 0
    assert hip.hipMemcpy(dst, src, n, 3) == 0      # hipMemcpyDeviceToDevice
    assert hip.hipDeviceSynchronize() == 0
    hip.hipFree(src)
    hip.hipFree(dst)
    log(f"[bench] calibration copy: {mib} MiB read + {mib} MiB written")


def library_gemm_us(n, k, rows, reps=40):
    """The vendor library's bf16 product y = x W^T (x [rows, k], W [n, k],
    float32 accumulation, bf16 output) through torch, back to back over
    enough weight copies that no launch finds its matrix in the 256 MB
    memory-side cache: the comparison for a matrix-core GEMM at small
    widths (a GEMV-style kernel at rows = 1)."""
    import torch
    import torch.nn.functional as F
    dev = torch.device("cuda", 0)
    copies = max(1, -(-(600 << 20) // (2 * n * k)))
    ws = [torch.randn(n, k, device=dev, dtype=torch.bfloat16) for _ in range(copies)]
    x = torch.randn(rows, k, device=dev, dtype=torch.bfloat16)
    for w in ws:
        F.linear(x, w)
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    e0.record()
    for i in range(reps):
        F.linear(x, ws[i % copies])
    e1.record()
    e1.synchronize()
    us = e0.elapsed_time(e1) * 1e3 / reps
    del ws, x
    torch.cuda.empty_cache()
    return us


def cpu_baseline(shape, n_audio, n_instr, k, mean_committed, seed=0, min_seconds=10.0, max_reps=400):
    """The float64 oracle on a bounded sample of the same workload: prefix
    of n_audio + n_instr rows through the first 2 of the layers (setup, not
    timed), then verify steps of k candidates through those 2 layers and the
    LM head, repeated from the same cache state until about min_seconds of
    CPU work are timed; the mean step is scaled to all layers."""
    from oracle import OracleModel
    n_sample = 2
    sub = shape.with_layers(n_sample)
    t0 = time.time()
    w = gen.weights_dict(sub, gen.make_weights(sub, seed))
    om = OracleModel(sub, w)
    audio = gen.audio_embeddings(sub, n_audio, seed)
    instr = gen.instruction_tokens(sub, n_instr, seed)
    om.prefill(audio, instr)
    setup = time.time() - t0
    cands = gen.uniform_int(gen.stream_key(seed, "bench-cpu-cands"), shape.vocab, k)
    x = om.embed_tokens([om.root] + list(cands))
    L0, root = om.kv_len, om.root
    t_layers = t_full = 0.0
    reps = 0
    while reps < max_reps and (reps == 0 or t_layers + t_full < min_seconds):
        # layers only (logits of no row), then the whole step with the LM head on all k + 1 rows
        t0 = time.perf_counter()
        om.forward(x, L0, logit_rows=np.array([], dtype=np.int64))
        t_layers += time.perf_counter() - t0
        om.rollback(L0, root)
        t0 = time.perf_counter()
        om.verify(cands, k)
        t_full += time.perf_counter() - t0
        om.rollback(L0, root)
        reps += 1
    t_layers /= reps
    t_full /= reps
    t_head = max(t_full - t_layers, 0.0)
    t_step = t_layers * shape.n_layers / n_sample + t_head
    try:
        cores = len(os.sched_getaffinity(0))
    except AttributeError:
        cores = os.cpu_count()
    threads = int(os.environ.get("OPENBLAS_NUM_THREADS", os.environ.get("OMP_NUM_THREADS", cores)))
    return {"value": mean_committed / t_step, "unit": "tokens/s", "cores": min(cores, threads),
            "kind": "oracle",
            "sample": (f"k={k} verify steps of the {shape.name} workload ({n_audio}+{n_instr} prefix) "
                       f"through {n_sample} of {shape.n_layers} layers plus the LM head, float64 numpy, "
                       f"{reps} repetitions from the same cache state; layer time scaled "
                       f"x{shape.n_layers}/{n_sample}; committed per step taken from the GPU run "
                       f"({mean_committed:.2f}); setup {setup:.1f}s untimed"),
            "step_seconds": t_step}


class Runner:
    """One library context with its requests prefilled: the greedy
    reference stream of every request (committed by the GPU itself; by the
    Proposition any proposal stream commits exactly it) and the seeded
    corrupted candidates drawn from it.  A step is one verification call
    over every request whose reply is not finished (one fused pass when
    there are several)."""

    def __init__(self, model, shape, reqs, seed, ref_width=1):
        self.model, self.shape, self.reqs, self.seed = model, shape, reqs, seed
        self.starts, self.refs, self.srcs = [], [], []
        self.prefill_info = None
        for i, r in enumerate(reqs):
            audio = gen.audio_embeddings(shape, r.n_audio, seed, i, fmt="device")
            instr = gen.instruction_tokens(shape, r.n_instr, seed, i)
            t0 = time.perf_counter()
            first, L = model.prefill(i, audio, instr)
            dt = time.perf_counter() - t0
            if self.prefill_info is None:
                self.prefill_info = {"rows": L, "ms": round(dt * 1e3, 2), "rows_per_s": round(L / dt, 1)}
            self.starts.append((L, first))
        t0 = time.perf_counter()
        self.refs = self._references(ref_width)
        log(f"[bench] {len(reqs)} request(s) prefilled; reference streams in {time.perf_counter() - t0:.1f}s")
        self.set_p(None)
        self.done = [0] * len(reqs)

    def _references(self, width):
        """[first root, y_1, ..., y_N] per request, committed by the GPU in
        fused passes over the unfinished requests; width - 1 zero tokens
        are proposed per call (width 1: target-only steps)."""
        refs = [[st[1]] for st in self.starts]
        for i in range(len(self.reqs)):
            self.model.rollback(i, *self.starts[i])
        while True:
            ids = [i for i, r in enumerate(self.reqs) if len(refs[i]) - 1 < r.reply_len]
            if not ids:
                break
            # width > 1: every call at the full width (the stream may run a
            # few tokens past the reply; it is cut below)
            cands = [[0] * (width - 1 if width > 1 else 0) for i in ids]
            outs = self.model.verify_batch(ids, cands)
            for i, c, o in zip(ids, cands, outs):
                refs[i] += c[:o["accepted_len"]] + [o["correction_token"]]
        for i in range(len(self.reqs)):
            refs[i] = refs[i][:self.reqs[i].reply_len + 1]
            self.model.rollback(i, *self.starts[i])
        return refs

    def set_p(self, p):
        """Candidate sources of corruption p (None: each request's own)."""
        self.srcs = [gen.CandidateSource(self.refs[i], self.shape.vocab, r.p if p is None else p,
                                         seed=self.seed, req=i) for i, r in enumerate(self.reqs)]

    def restart(self):
        for i in range(len(self.reqs)):
            self.model.rollback(i, *self.starts[i])
        self.done = [0] * len(self.reqs)

    def finished(self):
        return all(d >= r.reply_len for d, r in zip(self.done, self.reqs))

    def step(self, k_force=None):
        """One verification call; returns (tokens committed, rows, KV
        positions attended before the call)."""
        if self.finished():
            self.restart()
        ids, cands = [], []
        for i, r in enumerate(self.reqs):
            if self.done[i] >= r.reply_len:
                continue
            k = min(r.k if k_force is None else k_force, r.reply_len - self.done[i] - 1)
            ids.append(i)
            cands.append(self.srcs[i].block(self.done[i], k))
        kv = sum(self.starts[i][0] + self.done[i] for i in ids)
        m = self.model
        outs = m.verify_batch(ids, cands) if len(ids) > 1 else [m.verify(ids[0], cands[0])]
        got = 0
        for i, c, o in zip(ids, cands, outs):
            assert c[:o["accepted_len"]] == self.srcs[i].ref[self.done[i] + 1:self.done[i] + 1 + o["accepted_len"]].tolist()
            self.done[i] += o["accepted_len"] + 1
            got += o["accepted_len"] + 1
        return got, sum(len(c) + 1 for c in cands), kv

    def full_passes(self, n_passes):
        """n_passes whole passes over every reply (from the end of the
        prefix to the last token), each timed on its own."""
        out = []
        for _ in range(n_passes):
            self.restart()
            sync()
            steps = tok = rows = kv = 0
            t0 = time.perf_counter()
            while not self.finished():
                c, w, kk = self.step()
                steps += 1
                tok += c
                rows += w
                kv += kk
            sync()
            out.append({"s": time.perf_counter() - t0, "steps": steps, "tokens": tok, "rows": rows, "kv": kv})
        self.restart()
        return out

    def near_ties(self, margin=0.05):
        """One untimed pass counting verified rows whose device-side top-2
        logit margin is at most `margin`."""
        self.restart()
        n = rows = 0
        while not self.finished():
            before = [d for d in self.done]
            self.step()
            for i, r in enumerate(self.reqs):
                if self.done[i] != before[i]:
                    mg = self.model.row_margins(i)
                    n += int(np.sum(mg <= margin))
                    rows += len(mg)
        self.restart()
        return {"rows": rows, "near_tie_rows": n, "margin": margin}


_hip = None


def sync():
    global _hip
    if _hip is None:
        import ctypes
        _hip = ctypes.CDLL("libamdhip64.so")
    assert _hip.hipDeviceSynchronize() == 0


def kv_bytes(shape, rows, kv_keys, elem):
    """KV bytes of a pass: reads of the attended keys plus the appended rows."""
    return elem * shape.n_layers * 2 * shape.n_kv_heads * shape.head_dim * (kv_keys + rows)


def summarize(model, shape, passes):
    """Whole-reply throughput from timed passes: median tokens/s and the
    step's algorithmic bytes (float32 KV as stored, and with the KV counted
    in bf16 as a bf16 cache would hold it) over the median step time."""
    tps = sorted(p["tokens"] / p["s"] for p in passes)
    med = passes[[p["tokens"] / p["s"] for p in passes].index(tps[len(tps) // 2])]
    steps, s = med["steps"], med["s"]
    rows, kv = med["rows"] / steps, med["kv"] / steps
    b32 = model.step_bytes(int(round(rows)), int(round(kv)))
    b16 = b32 - kv_bytes(shape, rows, kv, 4) + kv_bytes(shape, rows, kv, 2)
    ms = s * 1e3 / steps
    return {"tokens_per_s": round(tps[len(tps) // 2], 2), "passes": len(passes),
            "tokens_per_s_min_max": [round(tps[0], 2), round(tps[-1], 2)],
            "verify_steps_per_s": round(steps / s, 2), "ms_per_step": round(ms, 4),
            "mean_committed_per_step": round(med["tokens"] / steps, 3), "mean_rows_per_step": round(rows, 2),
            "step_bytes": int(b32), "step_gbps": round(b32 / ms / 1e6, 1),
            "step_hbm_frac": round(b32 / ms / 1e6 / PEAK_HBM_GBPS, 4),
            "step_bytes_bf16_kv": int(b16), "step_hbm_frac_bf16_kv": round(b16 / ms / 1e6 / PEAK_HBM_GBPS, 4)}


def measure_config(index, shape_dev=None, seed=0, n_passes=3):
    """Whole-reply throughput of workload `index` in a context of its own
    (weights from shape_dev when given: the same model)."""
    from paper_2609_37617_amd import as2d
    wl = wc.workload(index)
    shape, reqs = wl.shape, wl.requests
    t0 = time.time()
    dev = shape_dev if shape_dev is not None else gen.make_weights(shape, wl.seed, fmt="device")
    max_k = max(max(r.k for r in reqs), 1)
    max_kv = (max(r.n_audio + r.n_instr + r.reply_len for r in reqs) + max_k + 2 + 63) // 64 * 64
    model = as2d.Model(shape, dev, max_requests=len(reqs), max_kv_len=max_kv, max_k=max_k)
    del dev
    run = Runner(model, shape, reqs, wl.seed)
    for _ in range(3):
        run.step()
    res = summarize(model, shape, run.full_passes(n_passes))
    res.update({"workload": wl.name, "layers": shape.n_layers, "requests": len(reqs),
                "prefix": [r.n_audio + r.n_instr for r in reqs] if len(reqs) > 1 else reqs[0].n_audio + reqs[0].n_instr,
                "reply_tokens": [r.reply_len for r in reqs] if len(reqs) > 1 else reqs[0].reply_len,
                "k": [r.k for r in reqs] if len(reqs) > 1 else reqs[0].k,
                "p": [round(r.p, 3) for r in reqs] if len(reqs) > 1 else reqs[0].p,
                "prefill_first_request": run.prefill_info})
    model.close()
    log(f"[bench] {wl.name}: {res['tokens_per_s']} tok/s, {res['ms_per_step']} ms/step, "
        f"{res['step_hbm_frac']:.1%} of peak ({time.time() - t0:.1f}s)")
    return res


def main():
    args = parse()
    if args.gpus != 1:
        print(f"bench.py runs on exactly one GPU: the library has no multi-GPU path "
              f"(--gpus {args.gpus} requested)", file=sys.stderr)
        sys.exit(2)
    from paper_2609_37617_amd import as2d
    if not os.path.exists(as2d.LIB_PATH):
        from paper_2609_37617_amd import build
        build.build()
    wl = wc.workload(args.workload)
    shape = wl.shape if args.layers is None else wl.shape.with_layers(args.layers)
    reqs = wl.requests
    if args.k is not None or args.p is not None:
        reqs = [wc.Request(r.n_audio, r.n_instr, r.reply_len, args.k if args.k is not None else r.k,
                           args.p if args.p is not None else r.p) for r in reqs]
    max_k = max(max(r.k for r in reqs), max(wl.k_sweep, default=0) if len(reqs) == 1 else 0, 1)
    max_kv = max(r.n_audio + r.n_instr + r.reply_len for r in reqs) + max_k + 2
    max_kv = (max_kv + 63) // 64 * 64
    trace = args.trace_window
    extras = not trace
    log(f"[bench] workload {wl.name}: {len(reqs)} request(s), shape {shape.name} L={shape.n_layers}")
    t0 = time.time()
    weights = gen.make_weights(shape, wl.seed, fmt="device")
    log(f"[bench] weights generated in {time.time() - t0:.1f}s")
    t0 = time.time()
    model = as2d.Model(shape, weights, max_requests=len(reqs), max_kv_len=max_kv, max_k=max_k)
    keep_dev = extras and not args.no_configs and args.layers is None and wl.shape.name == wc.QWEN7B.name
    if not keep_dev:
        del weights
    log(f"[bench] weights loaded and packed in {time.time() - t0:.1f}s")

    # prefill every request; reference streams committed by the GPU (with
    # --trace-window in passes of the timed width, so that a kernel trace of
    # the run holds verification launches of that width only)
    run = Runner(model, shape, reqs, wl.seed, ref_width=(reqs[0].k + 1) if trace else 1)
    srcs, starts, prefill_info = run.srcs, run.starts, run.prefill_info
    step, restart = run.step, run.restart

    if args.calib_copy_mib:
        copy_calibration(args.calib_copy_mib)
    for _ in range(args.warmup):
        step()
    # the driver's window: K steps from the beginning of the replies
    restart()
    sync()
    committed = rows = kvsum = 0
    t0 = time.perf_counter()
    for _ in range(args.steps):
        c, w, kv = step()
        committed += c
        rows += w
        kvsum += kv
    sync()
    elapsed = time.perf_counter() - t0
    ms = elapsed * 1e3 / args.steps
    mean_rows = rows / args.steps
    mean_kv = kvsum / args.steps
    step_bytes = model.step_bytes(int(round(mean_rows)), int(mean_kv))
    gbps = step_bytes / (elapsed / args.steps) / 1e9
    log(f"[bench] {args.steps} steps in {elapsed:.3f}s: {ms:.3f} ms/step, {committed / elapsed:.1f} tok/s in the window, "
        f"{gbps:.0f} GB/s ({gbps / PEAK_HBM_GBPS:.1%} of peak)")

    # the headline: whole replies, median of n passes
    whole = ties = None
    if extras:
        whole = summarize(model, shape, run.full_passes(args.passes))
        log(f"[bench] whole replies ({args.passes} passes): {whole['tokens_per_s']} tok/s, "
            f"{whole['mean_committed_per_step']} tokens per step, {whole['ms_per_step']} ms/step")
        ties = run.near_ties()
        log(f"[bench] near ties (device top-2 margin <= 0.05): {ties}")

    # the same window through the persistent step kernel (one launch per
    # pass; opt-in, reported beside the headline, which is the graph mode)
    exec_modes = {"graph_ms_per_step": round(ms, 4)}
    if extras and model.exec_info()[1] > 0:
        restart()
        model.set_exec_mode(as2d.EXEC_PERSISTENT)
        for _ in range(2):
            step()
        restart()
        sync()
        t1 = time.perf_counter()
        for _ in range(args.steps):
            step()
        sync()
        exec_modes["persistent_ms_per_step"] = round((time.perf_counter() - t1) * 1e3 / args.steps, 4)
        model.set_exec_mode(as2d.EXEC_GRAPH)
        restart()
        log(f"[bench] persistent step kernel: {exec_modes['persistent_ms_per_step']:.3f} ms/step")

    # p-sweep of the k = 8 workload: whole-reply throughput per corruption rate
    p_sweep = None
    if extras and len(reqs) == 1 and wl.p_sweep:
        p_sweep = {}
        for p in wl.p_sweep:
            run.set_p(p)
            for _ in range(2):
                step()
            p_sweep[str(p)] = summarize(model, shape, run.full_passes(3))
        run.set_p(None)
        restart()
        log("[bench] p-sweep: " + ", ".join(f"p={p} {v['tokens_per_s']} tok/s ({v['mean_committed_per_step']}/step)"
                                             for p, v in p_sweep.items()))

    roof = None
    kernel_ms = {}
    if extras and not args.no_kernel_timing:
        model.set_timing(True)
        model.timing_reset()
        n_t = max(10, args.steps // 2)
        sync()
        t1 = time.perf_counter()
        for _ in range(n_t):
            step()
        sync()
        t_evt = (time.perf_counter() - t1) * 1e3 / n_t
        model.set_timing(False)
        for name, (tot, cnt) in model.timing().items():
            if cnt:
                kernel_ms[name] = {"avg_us": tot * 1e3 / cnt, "launches": cnt, "total_ms_per_step": tot / n_t}
        # the dominant kernel, gate/up, timed over back-to-back launches
        # (events around a batch, so their own overhead is amortised)
        rows0 = reqs[0].k + 1 if len(reqs) == 1 else int(round(mean_rows))
        gu_us = model.time_gemm(2, rows0, 4 * shape.n_layers)
        gu_bytes = 2 * shape.ffn * shape.hidden * (2 if shape.dtype == wc.BF16 else 4)
        achieved = gu_bytes / (gu_us * 1e-6) / 1e9
        roof = {"bound": "hbm", "achieved": round(achieved, 1), "peak": PEAK_HBM_GBPS, "unit": "GB/s",
                "frac": round(achieved / PEAK_HBM_GBPS, 4), "traffic": traffic_from_profiles(),
                "kernel": "gemm_gate_up", "rows": rows0, "bytes_per_launch": gu_bytes,
                "avg_launch_us": round(gu_us, 2), "ms_per_step_with_events": round(t_evt, 3)}
        log("[bench] per-kernel: " + ", ".join(f"{k} {v['avg_us']:.1f}us x{v['launches'] // n_t}"
                                               for k, v in kernel_ms.items()))

    # achievable read bandwidth of the device (plain streaming kernel, 1 GiB)
    stream_gbps = model.stream_bandwidth(1 << 30, 10)
    log(f"[bench] stream-read ceiling {stream_gbps:.0f} GB/s")
    if roof is not None:
        roof["stream_ceiling_gbps"] = round(stream_gbps, 1)
        roof["frac_of_stream_ceiling"] = round(roof["achieved"] / stream_gbps, 4)

    # width-cost profile: step time per k (the paper's R(K) curve, one request)
    width = None
    if extras and not args.no_width_profile and len(reqs) == 1 and wl.k_sweep:
        width = {}
        for kk in wl.k_sweep:
            for _ in range(2):
                step(kk)
            sync()
            n_w = 10
            t1 = time.perf_counter()
            for _ in range(n_w):
                step(kk)
            sync()
            width[str(kk)] = round((time.perf_counter() - t1) * 1e3 / n_w, 4)
        log("[bench] ms per step by k: " + ", ".join(f"k={kk} {v}" for kk, v in width.items()))

    # verification width profile (the paper's protocol: known-reference
    # continuations at prefix offsets 0, 64 and 128 after prefill, 5 timed
    # calls per width and offset) and the offline budget choice from it
    vprof = budget_sel = None
    if extras and not args.no_width_profile and len(reqs) == 1:
        from paper_2609_37617_amd import budget as bsel
        r0 = reqs[0]
        y = srcs[0].ref.tolist()                    # [first root, y_1, y_2, ...]
        L0, root0 = starts[0]
        Ks = [K for K in range(1, max_k + 2) if 128 + K <= r0.reply_len]
        samples = {K: [] for K in Ks}
        model.rollback(0, L0, root0)
        for off in (0, 64, 128):
            # commit the reference up to off + max K (rollback only shortens)
            while model.state(0)[0] < L0 + off + Ks[-1]:
                n = model.state(0)[2]
                kk = min(max_k, L0 + off + Ks[-1] - model.state(0)[0])
                assert model.verify(0, y[n + 1:n + 1 + kk])["accepted_len"] == kk
            for K in Ks:
                cands = y[off + 1:off + K]
                for rep in range(6):
                    model.rollback(0, L0 + off, y[off])
                    t1 = time.perf_counter()
                    r = model.verify(0, cands)
                    dt = time.perf_counter() - t1
                    assert r["accepted_len"] == K - 1
                    if rep:
                        samples[K].append(dt * 1e3)
            model.rollback(0, L0 + off, y[off])
            n = off
            while model.state(0)[0] < L0 + off + Ks[-1]:      # back to off + max K for the next offset
                n = model.state(0)[2]
                kk = min(max_k, L0 + off + Ks[-1] - model.state(0)[0])
                assert model.verify(0, y[n + 1:n + 1 + kk])["accepted_len"] == kk
        vbar = {K: float(np.mean(v)) for K, v in samples.items()}
        sd = {K: float(np.std(v, ddof=1)) for K, v in samples.items()}
        R = bsel.cost_reduction(vbar)
        vprof = {"K": Ks, "vbar_ms": [round(vbar[K], 4) for K in Ks], "sd_ms": [round(sd[K], 4) for K in Ks],
                 "R_percent": [round(R[K], 2) for K in Ks],
                 "R_err_pp": [round(100 * sd[K] / (K * vbar[1]), 2) for K in Ks], "calls_per_width": 15}
        log("[bench] R(K) %: " + ", ".join(f"K={K} {R[K]:.1f}" for K in Ks))
        # budget choice: development drafts replayed and priced with V(K);
        # then the choice and its neighbours measured on a validation draft
        target = y[1:]
        n_tok = r0.reply_len - 1
        edits = (0.2, 0.05, 0.05)
        dev = [(gen.edited_stream(target, shape.vocab, *edits, seed=wl.seed + 100 + i), target, n_tok) for i in range(3)]
        budgets = [b for b in range(0, max_k + 1) if b + 1 in vbar]
        best, est = bsel.select_budget(vbar, dev, budgets)
        val = gen.edited_stream(target, shape.vocab, *edits, seed=wl.seed + 200)
        measured = {}
        for b in sorted({best, 1, 3, 7, max(budgets)} & set(budgets)):
            buf = as2d.CandidateBuffer(len(val))
            for i in range(0, len(val), 8):
                buf.publish(val[i:i + 8])
            cur = as2d.ReadCursor(8)
            model.rollback(0, L0, root0)
            got = 0
            t1 = time.perf_counter()
            while got < r0.reply_len:
                rr, _ = cur.verify_from_buffer(model, 0, buf, b, r0.reply_len - got)
                got += rr["accepted_len"] + 1
            measured[b] = round(got / (time.perf_counter() - t1), 1)
            buf.close()
        restart()
        budget_sel = {"draft_edits": {"sub": edits[0], "ins": edits[1], "del": edits[2]}, "dev_traces": len(dev),
                      "selected_budget": best,
                      "estimated_tokens_per_s": {str(b): round(1e3 * v, 1) for b, v in est.items()},
                      "measured_tokens_per_s_validation": {str(b): v for b, v in measured.items()}}
        log(f"[bench] budget: selected {best}; measured on validation {measured}")

    # target-decoupled decoding with a drafter on the same GPU (3B- and 0.5B-shaped):
    # serial comparator and concurrent run, with the stage accounting
    decoupled = None
    if extras and not args.no_decoupled and len(reqs) == 1 and wl.shape.name == wc.QWEN7B.name and args.layers is None:
        from paper_2609_37617_amd import overlap as ovl
        r0 = reqs[0]
        y = srcs[0].ref.tolist()
        n_tok = r0.reply_len - 1
        draft = gen.edited_stream(y[1:], shape.vocab, 0.2, 0.05, 0.05, seed=wl.seed + 300)
        b = budget_sel["selected_budget"] if budget_sel else r0.k
        decoupled = {"draft_edits": {"sub": 0.2, "ins": 0.05, "del": 0.05}, "budget": b, "tokens": n_tok}
        for dshape in (wc.QWEN3B, wc.QWEN05B):
            t_load = time.time()
            d_dev = gen.make_weights(dshape, wl.seed + 1, fmt="device")
            d_max_kv = (r0.n_audio + r0.n_instr + 2 * r0.reply_len + 63) // 64 * 64
            drafter = as2d.Model(dshape, d_dev, max_requests=1, max_kv_len=d_max_kv, max_k=1)
            del d_dev
            d_first, d_L = drafter.prefill(0, gen.audio_embeddings(dshape, r0.n_audio, wl.seed + 1, 0, fmt="device"),
                                           gen.instruction_tokens(dshape, r0.n_instr, wl.seed + 1, 0))
            log(f"[bench] drafter {dshape.name} loaded and prefilled in {time.time() - t_load:.1f}s")
            def warm():
                # capture every graph the runs launch, one thread at a time
                for kk in range(0, b + 1):
                    restart()
                    model.verify(0, y[1:1 + kk])
                restart()
                drafter.rollback(0, d_L, d_first)
                drafter.decode_one(0)
                drafter.rollback(0, d_L, d_first)

            def one(conc):
                restart()
                drafter.rollback(0, d_L, d_first)
                r = as2d.run_decoupled(model, 0, drafter, 0, draft, b, n_tok, conc)
                assert r["committed"] == y[1:1 + n_tok]
                acc = ovl.accounting(r["intervals"], r["total_ns"])
                steps = [iv for iv in r["intervals"] if iv[2] == 0]
                return acc, {"T_ms": round(acc["T"] / 1e6, 3), "D_ms": round(acc["D"] / 1e6, 3),
                             "V_ms": round(acc["V"] / 1e6, 3), "O_ms": round(acc["O"] / 1e6, 3),
                             "H_ms": round(acc["H"] / 1e6, 3), "rounds": acc["R"],
                             "tokens_per_s": round(n_tok / (acc["T"] / 1e9), 1),
                             "mean_committed_per_round": round(acc["N"] / acc["R"], 3),
                             "verifier_ms_per_round": round(acc["V"] / acc["R"] / 1e6, 4),
                             "producer_steps": len(steps),
                             "producer_ms_per_step": round(sum(e - s for s, e, _, _ in steps) / max(1, len(steps)) / 1e6, 4)}

            res, accs = {}, {}
            warm()
            accs["serial"], res["serial"] = one(False)
            accs["concurrent"], res["concurrent"] = one(True)
            # CU budgets: the drafter's GEMMs on `dc` workgroups, the target's on the rest
            res["concurrent_cu_budget"] = {}
            best = None
            for dc in ((32, 64, 96) if dshape.name == wc.QWEN05B.name else (64,)):
                model.set_cu_budget(256 - dc)
                drafter.set_cu_budget(dc)
                warm()
                acc, row = one(True)
                row["speedup_vs_serial"] = round(accs["serial"]["T"] / acc["T"], 4)
                res["concurrent_cu_budget"][str(dc)] = row
                if best is None or acc["T"] < accs[best]["T"]:
                    best = f"budget{dc}"
                accs[f"budget{dc}"] = acc
                model.set_cu_budget(0)
                drafter.set_cu_budget(0)
            res["best_concurrent"] = best if accs[best]["T"] < accs["concurrent"]["T"] else "concurrent"
            c = ovl.compare(accs["serial"], accs[res["best_concurrent"]])
            res["compare"] = {"speedup": round(c["speedup"], 4), "O_a_ms": round(c["O_a"] / 1e6, 3),
                              "added_ms": round(c["added"] / 1e6, 3), "dD_ms": round(c["dD"] / 1e6, 3),
                              "dV_ms": round(c["dV"] / 1e6, 3), "dH_ms": round(c["dH"] / 1e6, 3),
                              "break_even_holds": bool(c["break_even_holds"]),
                              "bottleneck_bound": round(c["bound"], 4)}
            decoupled[dshape.name] = res
            drafter.close()
            restart()
            log(f"[bench] decoupled with {dshape.name}: serial {res['serial']['T_ms']} ms, concurrent "
                f"{res['concurrent']['T_ms']} ms, with CU budgets " +
                ", ".join(f"{k}: {v['T_ms']} ms ({v['speedup_vs_serial']}x)" for k, v in res["concurrent_cu_budget"].items()) +
                f" | best {res['best_concurrent']}: {res['compare']}")

    # decoding from the candidate buffer with an edited draft (substitutions,
    # insertions, deletions): with the bounded realignment, and with the
    # search turned off (radius 0: every mismatch read as a substitution)
    aligned = None
    if extras and not args.no_align and len(reqs) == 1:
        r0 = reqs[0]
        edits = (0.2, 0.05, 0.05)
        draft = gen.edited_stream(srcs[0].ref[1:].tolist(), shape.vocab, *edits, seed=wl.seed)
        aligned = {"draft": {"sub": edits[0], "ins": edits[1], "del": edits[2], "tokens": len(draft)},
                   "budget": r0.k, "reply_tokens": r0.reply_len}
        for name, radius in (("with_alignment", 8), ("without_search", 0)):
            buf = as2d.CandidateBuffer(len(draft))
            for i in range(0, len(draft), 8):
                buf.publish(draft[i:i + 8], offset=i)
            cur = as2d.ReadCursor(radius)
            restart()
            calls = got = 0
            t1 = time.perf_counter()
            while got < r0.reply_len:
                r, _ = cur.verify_from_buffer(model, 0, buf, r0.k, r0.reply_len - got)
                got += r["accepted_len"] + 1
                calls += 1
            dt = time.perf_counter() - t1
            aligned[name] = {"calls": calls, "tokens_per_s": round(got / dt, 1),
                             "mean_committed_per_call": round(got / calls, 3), "ms_per_call": round(dt * 1e3 / calls, 4)}
            buf.close()
        restart()
        log(f"[bench] buffer decoding, edited draft: {aligned['with_alignment']} | radius 0: {aligned['without_search']}")

    cpu = None
    if extras and not args.no_cpu_baseline:
        r0 = reqs[0]
        t0 = time.time()
        cpu = cpu_baseline(shape, r0.n_audio, r0.n_instr, r0.k, whole["mean_committed_per_step"])
        log(f"[bench] cpu baseline {cpu['value']:.3f} tok/s ({time.time() - t0:.1f}s)")

    # every verification GEMM back to back at W = 1 and at the timed width
    # (last use of this context: the QKV launches overwrite cache rows of slot 0)
    if roof is not None:
        gemms = {}
        H, F, V = shape.hidden, shape.ffn, shape.vocab
        es = 2 if shape.dtype == wc.BF16 else 4
        nbytes = {"gemm_qkv": es * H * shape.qkv_out, "gemm_o": es * H * shape.n_q_heads * shape.head_dim,
                  "gemm_gate_up": es * 2 * F * H, "gemm_down": es * F * H, "gemm_lm_head": es * V * H}
        for which, name in enumerate(nbytes):
            for w in sorted({1, roof["rows"]}):
                us = model.time_gemm(which, w, 4 * shape.n_layers if which < 4 else 8)
                gemms[f"{name}_w{w}"] = {"us": round(us, 2), "gbps": round(nbytes[name] / us / 1e3, 1),
                                         "frac": round(nbytes[name] / us / 1e3 / PEAK_HBM_GBPS, 4)}
        roof["gemms_back_to_back"] = gemms
        log("[bench] GEMMs back to back: " + ", ".join(f"{k} {v['us']}us {v['frac']:.0%}" for k, v in gemms.items()))
        if args.library_gemm and shape.dtype == wc.BF16:
            shapes = {"gemm_qkv": shape.qkv_out, "gemm_o": H, "gemm_gate_up": 2 * F, "gemm_down": H,
                      "gemm_lm_head": V}
            kdim = {"gemm_qkv": H, "gemm_o": shape.n_q_heads * shape.head_dim, "gemm_gate_up": H,
                    "gemm_down": F, "gemm_lm_head": H}
            lib = {}
            for name, n in shapes.items():
                for w in sorted({1, roof["rows"]}):
                    us = library_gemm_us(n, kdim[name], w)
                    lib[f"{name}_w{w}"] = {"us": round(us, 2), "frac": round(nbytes[name] / us / 1e3 / PEAK_HBM_GBPS, 4)}
            roof["library_gemm_back_to_back"] = lib
            log("[bench] library bf16 GEMM back to back: "
                + ", ".join(f"{k} {v['us']}us {v['frac']:.0%}" for k, v in lib.items()))

    # the other workloads, each in a context of its own: the 3B shape, the
    # long-audio prefix and the mixed batch (the same 7B weights)
    configs = None
    if keep_dev:
        model.close()
        configs = {}
        for idx in (1, 3, 4):
            same = wc.workload(idx).shape.name == shape.name
            configs[wc.workload(idx).name] = measure_config(idx, weights if same else None,
                                                            n_passes=3 if idx != 4 else 2)
        del weights

    r0 = reqs[0]
    out = {
        "metric": METRIC,
        "value": whole["tokens_per_s"] if whole else round(committed / elapsed, 2),
        "unit": "tokens/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms, 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16" if shape.dtype == wc.BF16 else "f32",
        "data": "synthetic",
        "config": {"workload": wl.name, "layers": shape.n_layers, "hidden": shape.hidden,
                   "ffn": shape.ffn, "vocab": shape.vocab, "heads": f"{shape.n_q_heads}/{shape.n_kv_heads}",
                   "requests": len(reqs), "prefix": r0.n_audio + r0.n_instr, "reply_tokens": r0.reply_len,
                   "k": r0.k, "p": r0.p},
        "verify_steps_per_s": round(args.steps / elapsed, 2),
        "window": {"steps": args.steps, "committed": committed, "tokens_per_s": round(committed / elapsed, 2),
                   "mean_committed_per_step": round(committed / args.steps, 3)},
        "whole_replies": whole,
        "near_ties": ties,
        "trace_window": bool(trace),
        "step_hbm_bytes": step_bytes,
        "step_hbm_bytes_bf16_kv": int(step_bytes - kv_bytes(shape, mean_rows, mean_kv, 4)
                                      + kv_bytes(shape, mean_rows, mean_kv, 2)),
        "step_hbm_gbps": round(gbps, 1),
        "step_hbm_frac": round(gbps / PEAK_HBM_GBPS, 4),
        "roofline": roof,
        "cpu_baseline": cpu,
        "stream_ceiling_gbps": round(stream_gbps, 1),
        "exec_modes": exec_modes,
        "p_sweep": p_sweep,
        "configs": configs,
        "ms_per_step_by_k": width,
        "buffer_decoding": aligned,
        "prefill_first_request": prefill_info,
        "verification_profile": vprof,
        "budget_selection": budget_sel,
        "decoupled": decoupled,
        "kernels": {k: round(v["avg_us"], 2) for k, v in kernel_ms.items()},
    }
    print(json.dumps(out), flush=True)
    if not keep_dev:
        model.close()


if __name__ == "__main__":
    main()
