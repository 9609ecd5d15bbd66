#!/usr/bin/env python3
"""Benchmark of the DO-loss hot path on one MI355X.

One step = one do_fused call over the whole workload already resident in HBM:
router Top-K -> signatures (written out) -> E x E Hamming -> loss, for every
layer.  Prints ONE JSON line (rank 0, one GPU).

Default workload: 8 layers x 4,194,304 tokens, 256 experts, top-8, fp32
scores drawn as a per-token softmax with clustered expert preferences.  The
default run also times the streaming history (16 micro-batches of 65,536
bf16 tokens, 128 experts, top-8, appended into one 1,048,576-token history,
then finalised) and reports it as the "stream" sub-record; ``--workload 3``
makes it the headline instead.
"""
from __future__ import annotations

import argparse
import glob
import hashlib
import json
import os
import re
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

HBM_PEAK_GBS = 8000.0  # MI355X HBM3E, published

# Sources whose hash identifies the score-streaming kernel; HBM byte counts
# recorded under profiles/ are reported only while they still match.
KERNEL_SOURCES = ["paper_2609_32398_amd/csrc/topk.hip", "paper_2609_32398_amd/csrc/common.h",
                  "paper_2609_32398_amd/hipbuild.py"]


def log(msg: str):
    print(f"[bench] {msg}", file=sys.stderr, flush=True)


def parse():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--settle", type=float, default=0.5,
                    help="seconds of untimed steps before the warm-up steps (the GPU leaves its idle clock)")
    ap.add_argument("--workload", type=int, default=4, choices=[1, 2, 3, 4])
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--cpu-seconds", type=float, default=10.0,
                    help="oracle time to accumulate for cpu_baseline (whole layers, at least one)")
    ap.add_argument("--layers", type=int, default=None, help="override the layer count (testing only)")
    ap.add_argument("--gram", choices=["mfma", "popc"], default="mfma",
                    help="co-occurrence Gram inside k_topk for E <= 256: fp4 MFMA (default) or VALU popcount")
    ap.add_argument("--calibrate-copy", action="store_true",
                    help="only run a plain 4 GiB device copy (calibrates the HBM byte counters)")
    return ap.parse_args()


def ensure_built():
    import paper_2609_32398_amd.hipbuild as hb

    if not os.path.exists(hb.LIB_PATH):
        import __graft_entry__

        __graft_entry__.build()


def pinned_host(n, E, dtype_code):
    import torch

    tdt = torch.float32 if dtype_code == 0 else torch.int16
    return torch.empty((n, E), dtype=tdt, pin_memory=True)


def upload_workload(cfg: int, layers: int):
    """Generate the workload layer by layer on the host and copy it into one device buffer."""
    import numpy as np
    import torch

    import synth

    w = synth.WORKLOADS[cfg]
    N, E = w["n"], w["E"]
    tdt = torch.float32 if w["dtype"] == 0 else torch.bfloat16
    dev = torch.empty((layers, N, E), dtype=tdt, device="cuda")
    host = pinned_host(N, E, w["dtype"])
    hview = host.numpy() if w["dtype"] == 0 else host.numpy().view(np.uint16)
    t0 = time.time()
    for l in range(layers):
        synth.workload_fill(cfg, l, out=hview)
        dev[l].copy_(host.view(tdt) if w["dtype"] == 1 else host)
        log(f"generated layer {l + 1}/{layers} ({time.time() - t0:.1f} s)")
    torch.cuda.synchronize()
    return dev


def _code_only(text: str, py: bool) -> str:
    """The source without comments and blank lines (comments do not change the kernel)."""
    if py:
        text = re.sub(r'"""(?:.|\n)*?"""', "", text)
        text = re.sub(r"(?m)#.*$", "", text)
    else:
        text = re.sub(r"/\*(?:.|\n)*?\*/", "", text)
        text = re.sub(r"(?m)//.*$", "", text)
    return "\n".join(l.rstrip() for l in text.splitlines() if l.strip())


def kernel_source_digest() -> str:
    """sha256 over the code of KERNEL_SOURCES (comments and blank lines removed)."""
    h = hashlib.sha256()
    for p in KERNEL_SOURCES:
        with open(os.path.join(ROOT, p), encoding="utf-8") as f:
            h.update(_code_only(f.read(), p.endswith(".py")).encode())
    return h.hexdigest()


def recorded_traffic(workload: str):
    """HBM bytes per launch of k_topk from the rocprofv3 counter summaries, or
    None when no summary was taken with the current kernel sources."""
    digest = kernel_source_digest()
    for path in sorted(glob.glob(os.path.join(ROOT, "profiles", "*.md"))):
        with open(path) as f:
            for line in f:
                if not line.startswith("traffic:"):
                    continue
                kv = dict(item.split("=", 1) for item in line.split()[1:])
                if kv.get("workload") == workload and kv.get("source_sha256") == digest:
                    return float(kv["bytes_per_launch"]), os.path.relpath(path, ROOT)
    return None, None


def host_cpu():
    """CPU model and the CPUs this process may run on (the host of the GPU)."""
    model = "unknown"
    ids = {}
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                key = line.split(":", 1)[0].strip()
                if key == "model name" and model == "unknown":
                    model = line.split(":", 1)[1].strip()
                elif key in ("cpu family", "model") and key not in ids:
                    ids[key] = line.split(":", 1)[1].strip()
                if model != "unknown" and len(ids) == 2:
                    break
    except OSError:
        pass
    if ids:  # a virtualised host may name only the brand: add the family / model numbers
        model = f"{model} (family {ids.get('cpu family', '?')}, model {ids.get('model', '?')})"
    try:
        avail = len(os.sched_getaffinity(0))
    except AttributeError:  # pragma: no cover
        avail = os.cpu_count() or 1
    return model, os.cpu_count() or 1, avail


def cpu_baseline(cfg: int, seconds: float):
    """The oracle as it stands, on rank 0, over whole layers of the same workload
    (workload 3: the whole 16-micro-batch history) until about `seconds` of
    oracle time have accumulated.  Input generation is not timed."""
    import oracle
    import synth

    w = synth.WORKLOADS[cfg]
    th = oracle.threads()
    spent, tokens, units = 0.0, 0, 0
    while spent < seconds:
        if cfg == 3:
            mbs = [synth.workload_fill(cfg, b) for b in range(w["layers"])]
            t0 = time.perf_counter()
            oracle.run_stream(mbs, w["k"], th)
            spent += time.perf_counter() - t0
            tokens += w["layers"] * w["n"]
        else:
            x = synth.workload_fill(cfg, units % w["layers"])
            t0 = time.perf_counter()
            oracle.run(x, w["k"], th)
            spent += time.perf_counter() - t0
            tokens += w["n"]
        units += 1
    what = (f"{units} pass(es) over the whole 16 x {w['n']}-token history" if cfg == 3
            else f"{units} whole layer(s) of {w['n']} tokens")
    model, ncpu, avail = host_cpu()
    return dict(value=tokens / spent, unit="tokens/s", cores=th, kind="oracle",
                sample=f"{what}: top-k, XOR-count Hamming, loss; {spent:.1f} s of oracle time, generation excluded",
                threads_used=th, host_cpus=ncpu, cpus_available=avail, cpu_model=model,
                build="gcc " + " ".join(oracle.CFLAGS))


def roofline(alg_bytes: float, kern_ms: float, workload: str, kernel: str, bytes_per_token: int,
             gram: str = "mfma") -> dict:
    achieved = alg_bytes / (kern_ms / 1e3) / 1e9
    # recorded counters cover the default (MFMA Gram) kernel only
    traffic, source = recorded_traffic(workload) if gram == "mfma" else (None, None)
    return dict(bound="hbm", achieved=achieved, peak=HBM_PEAK_GBS, unit="GB/s", frac=achieved / HBM_PEAK_GBS,
                traffic=traffic, traffic_source=source, kernel=kernel, kernel_ms=kern_ms,
                algorithmic_bytes=alg_bytes, bytes_per_token=bytes_per_token)


def settle(step, seconds: float) -> int:
    """Runs step(i) untimed for about `seconds` of wall time and returns the count.

    Launches of 0.1-6 ms timed right after an idle period run at a lower clock:
    at workload 2 the first 30 launches measure 3-4 % slower than later ones.
    """
    import torch

    t0 = time.perf_counter()
    n = 0
    while True:
        step(n)
        n += 1
        if n % 4 == 0:
            torch.cuda.synchronize()
            if time.perf_counter() - t0 >= seconds:
                return n


def bench_layers(args, cfg):
    import torch

    import paper_2609_32398_amd as dl
    import synth

    w = synth.WORKLOADS[cfg]
    L = args.layers or w["layers"]
    N, E, k = w["n"], w["E"], w["k"]
    scores = upload_workload(cfg, L)
    bits = dl.alloc_bits(L, N, E, scores.device)
    D = dl.alloc_D(L, E, scores.device)
    out = dl.alloc_out(L, scores.device)

    def step():
        dl.do_fused(scores, k, bits=bits, D=D, out=out)

    n_settle = settle(lambda i: step(), args.settle)
    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()
    ks = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)) for _ in range(args.steps)]
    for a, b in ks:  # materialise the events so their handles exist
        a.record()
        b.record()
    torch.cuda.synchronize()
    t_start = torch.cuda.Event(enable_timing=True)
    t_stop = torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    wall0 = time.perf_counter()
    t_start.record()
    for _ in range(args.steps):
        step()
    t_stop.record()
    torch.cuda.synchronize()
    wall = time.perf_counter() - wall0
    total_ms = t_start.elapsed_time(t_stop)
    ms_per_step = total_ms / args.steps
    # the Top-K kernel's own duration: the same steps again, each with a pair
    # of events bound to its dispatch (the binding costs a few us per step)
    for a, b in ks:
        dl.do_profile_next(a, b)
        step()
    torch.cuda.synchronize()
    kern_ms = sum(a.elapsed_time(b) for a, b in ks) / len(ks)
    tokens = L * N
    elem = 4 if w["dtype"] == 0 else 2
    bytes_per_token = E * elem + E // 8
    alg_bytes = tokens * bytes_per_token
    rec = dl.loss_records(out)
    # the same pass without writing the signatures out (D and the loss only),
    # timed separately after the headline steps
    nb = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)) for _ in range(args.steps)]
    for a, b in nb:
        a.record()
        b.record()
    for _ in range(max(args.warmup, 3)):  # the library settles this launch shape's schedule here
        dl.do_fused(scores, k, D=D, out=out)
    torch.cuda.synchronize()
    for a, b in nb:
        dl.do_profile_next(a, b)
        dl.do_fused(scores, k, D=D, out=out)
    torch.cuda.synchronize()
    nb_ms = sum(a.elapsed_time(b) for a, b in nb) / len(nb)
    nb_bytes = tokens * E * elem
    # the surrogate loss (Eq. 7) and its gradient on the same tokens: the scores
    # of this workload are per-token probabilities; signatures and distances
    # from the headline pass
    dl.do_fused(scores, k, bits=bits, D=D, out=out)
    sloss = torch.empty(L, dtype=torch.float64, device=scores.device)
    sgrad = torch.empty((L, N, E), dtype=torch.float32, device=scores.device)
    dl.do_surrogate(scores, k, bits, D, loss=sloss, grad=sgrad)
    torch.cuda.synchronize()
    sv = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)) for _ in range(args.steps)]
    for a, b in sv:
        a.record()
        b.record()
    torch.cuda.synchronize()
    for a, b in sv:
        dl.do_profile_next(a, b)
        dl.do_surrogate(scores, k, bits, D, loss=sloss, grad=sgrad)
    torch.cuda.synchronize()
    s_ms = sum(a.elapsed_time(b) for a, b in sv) / len(sv)
    s_bytes = tokens * (2 * E * 4 + E // 8) if w["dtype"] == 0 else tokens * (E * 2 + E * 4 + E // 8)
    del sgrad
    # load statistics (loads, Local-LBL with the scores as probabilities, MaxVio
    # over 8 ranks of E/8 consecutive experts) on the same signatures
    ranks = [i * 8 // E for i in range(E)]
    ls_loads, ls_out = dl.do_load_stats(bits, N, k, p=scores, expert_rank=ranks, R=8)
    torch.cuda.synchronize()
    lv = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)) for _ in range(args.steps)]
    for a, b in lv:
        a.record()
        b.record()
    torch.cuda.synchronize()
    for a, b in lv:
        a.record()
        dl.do_load_stats(bits, N, k, p=scores, expert_rank=ranks, R=8, loads=ls_loads, out=ls_out)
        b.record()
    torch.cuda.synchronize()
    ls_ms = sum(a.elapsed_time(b) for a, b in lv) / len(lv)
    ls_bytes = tokens * (E * elem + E // 8)
    ls_rec = dl.load_stats_records(ls_out)[0]
    assert ls_rec["total"] == N * k
    res = dict(
        metric="DO-loss tokens/s per layer (top-k→signature→E×E Hamming→loss); % of HBM peak",
        value=tokens / (ms_per_step / 1e3),
        unit="tokens/s",
        n_gpus=1,
        steps=args.steps,
        warmup=args.warmup,
        clock_settle=dict(seconds=args.settle, steps=n_settle),
        ms_per_step=ms_per_step,
        higher_is_better=True,
        scaling="weak",
        vs_baseline=None,
        dtype="i32",
        data="synthetic",
        config=dict(workload=w["name"], layers=L, tokens_per_layer=N, experts=E, k=k,
                    score_dtype="f32" if w["dtype"] == 0 else "bf16", signatures_written=True,
                    gram=args.gram),
        roofline=roofline(alg_bytes, kern_ms, w["name"], "k_topk (fused top-k, signatures, "
                          + ("fp4 MFMA Gram)" if args.gram == "mfma" else "popcount Gram)"),
                          bytes_per_token, args.gram),
        step_gbs=alg_bytes / (ms_per_step / 1e3) / 1e9,
        without_signature_output=dict(kernel_ms=nb_ms, algorithmic_bytes=nb_bytes,
                                      achieved_gbs=nb_bytes / (nb_ms / 1e3) / 1e9,
                                      frac=nb_bytes / (nb_ms / 1e3) / 1e9 / HBM_PEAK_GBS),
        surrogate=dict(kernel="k_surrogate (Eq. 7 loss and dloss/dp)", kernel_ms=s_ms, algorithmic_bytes=s_bytes,
                       bytes_per_token=s_bytes // tokens, achieved_gbs=s_bytes / (s_ms / 1e3) / 1e9,
                       frac=s_bytes / (s_ms / 1e3) / 1e9 / HBM_PEAK_GBS,
                       tokens_per_s=tokens / (s_ms / 1e3)),
        load_stats=dict(kernels="k_unit_loads + " + ("k_lbl_sums_vec" if w["dtype"] == 0 else "k_lbl_sums")
                        + " + k_load_finalize (loads, Local-LBL, MaxVio)",
                        ms=ls_ms, algorithmic_bytes=ls_bytes, bytes_per_token=ls_bytes // tokens,
                        achieved_gbs=ls_bytes / (ls_ms / 1e3) / 1e9,
                        frac=ls_bytes / (ls_ms / 1e3) / 1e9 / HBM_PEAK_GBS,
                        layer0=dict(lbl=ls_rec["lbl"], maxvio_8_ranks=ls_rec["maxvio"], max_load=ls_rec["max_load"],
                                    min_load=ls_rec["min_load"])),
        wall_s_timed=wall,
        check=dict(layer0_sum=rec[0]["sum"], expected_sum=2 * N * k * (E - k)),
    )
    assert rec[0]["sum"] == 2 * N * k * (E - k), "zero-sum identity (Eq. 2) violated"
    return res


def bench_stream(args):
    import numpy as np
    import torch

    import paper_2609_32398_amd as dl
    import synth

    cfg = 3
    w = synth.WORKLOADS[cfg]
    nmb, N, E, k = w["layers"], w["n"], w["E"], w["k"]
    copies = 2  # two distinct sets of 16 buffers defeat the 256 MB last-level cache
    host = pinned_host(N, E, 1)
    hview = host.numpy().view(np.uint16)
    bufs = []
    for c in range(copies):
        row = []
        for b in range(nmb):
            synth.workload_fill(cfg, b, out=hview)
            t = torch.empty((N, E), dtype=torch.bfloat16, device="cuda")
            t.copy_(host.view(torch.bfloat16))
            row.append(t)
        bufs.append(row)
    log("streaming micro-batches uploaded")
    s = dl.DoStream(E, k, nmb * N)
    D = torch.empty((E, E), dtype=torch.int32, device="cuda")
    out = dl.alloc_out(1, "cuda")

    def step(i):
        s.reset()
        s.append_many(bufs[i % copies])
        s.finalize(D, out)

    n_settle = settle(step, args.settle)
    for i in range(args.warmup):
        step(i)
    torch.cuda.synchronize()
    ks = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)) for _ in range(args.steps)]
    for a, b in ks:
        a.record()
        b.record()
    t_start = torch.cuda.Event(enable_timing=True)
    t_stop = torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    t_start.record()
    for i in range(args.steps):
        step(i)
    t_stop.record()
    torch.cuda.synchronize()
    ms_per_step = t_start.elapsed_time(t_stop) / args.steps
    # the append kernel's own duration: the same steps again, with a pair of
    # events bound to each append's dispatch (the binding costs a few us per step)
    for i, (a, b) in enumerate(ks):
        s.reset()
        dl.do_profile_next(a, b)
        s.append_many(bufs[i % copies])
        s.finalize(D, out)
    torch.cuda.synchronize()
    kern_ms = sum(a.elapsed_time(b) for a, b in ks) / len(ks)
    tokens = nmb * N
    bytes_per_token = E * 2 + E // 8
    alg = tokens * bytes_per_token
    rec = dl.loss_records(out)[0]
    assert rec["sum"] == 2 * tokens * k * (E - k)
    s.close()
    return dict(
        metric="DO-loss tokens/s per layer (top-k→signature→E×E Hamming→loss); % of HBM peak",
        value=tokens / (ms_per_step / 1e3), unit="tokens/s", n_gpus=1, steps=args.steps, warmup=args.warmup,
        clock_settle=dict(seconds=args.settle, steps=n_settle), ms_per_step=ms_per_step, higher_is_better=True,
        scaling="weak", vs_baseline=None, dtype="i32", data="synthetic",
        config=dict(workload=w["name"], micro_batches=nmb, tokens_per_micro_batch=N, experts=E, k=k,
                    score_dtype="bf16", buffer_sets=copies, gram=args.gram),
        roofline=roofline(alg, kern_ms, w["name"], "k_topk (stream append, 16 micro-batches per launch, "
                          + ("fp4 MFMA Gram)" if args.gram == "mfma" else "popcount Gram)"),
                          bytes_per_token, args.gram),
        step_gbs=alg / (ms_per_step / 1e3) / 1e9,
        step_frac=alg / (ms_per_step / 1e3) / 1e9 / HBM_PEAK_GBS,
        check=dict(sum=rec["sum"], expected_sum=2 * tokens * k * (E - k)),
    )


def main():
    args = parse()
    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) != 1:
        print("bench.py runs on exactly one GPU: there is no multi-GPU path. The distances are additive "
              "over token shards, so N GPUs would each run this pass on their shard and sum the counters "
              "with one all-reduce; that path is not built.", file=sys.stderr)
        sys.exit(2)
    ensure_built()
    import torch

    assert torch.cuda.is_available(), "bench.py needs a GPU"
    import paper_2609_32398_amd as dl

    dl.lib()
    if args.gram == "popc":
        dl.set_option(dl.DO_OPT_GRAM, 1)
    if args.calibrate_copy:
        n = 1 << 30  # 4 GiB of fp32
        src = torch.ones(n, dtype=torch.float32, device="cuda")
        dst = torch.empty_like(src)
        for _ in range(3):
            dst.copy_(src)
        torch.cuda.synchronize()
        print(json.dumps(dict(calibration="device copy", bytes_read=4 * n, bytes_written=4 * n, launches=3)))
        return
    cfg = args.workload
    res = bench_stream(args) if cfg == 3 else bench_layers(args, cfg)
    if cfg == 4:
        # the streaming history (the other large workload) beside the headline
        log("timing the streaming history")
        st = bench_stream(args)
        res["stream"] = {key: st[key] for key in ("value", "unit", "ms_per_step", "steps", "warmup", "clock_settle",
                                                  "config", "roofline", "step_gbs", "step_frac", "check")}
    if not args.no_cpu_baseline:
        log("timing the oracle on the host")
        res["cpu_baseline"] = cpu_baseline(cfg, args.cpu_seconds)
    print(json.dumps(res), flush=True)


if __name__ == "__main__":
    main()
