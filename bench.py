#!/usr/bin/env python3
"""Benchmark of the batched verification step on one MI355X.

One step = the whole hot path on one batch: hardware-aware prefix scheduling
(dspark_schedule) -> ragged paged verify attention for one attention layer
(dspark_verify_attn) -> speculative acceptance over the vocabulary
(dspark_accept), all enqueued on one stream with inputs resident in HBM.

The default workload is the 128-request serving shape (64 query / 8 KV heads,
head dim 128, log-normal contexts 2048..16384, draft block 16, vocabulary
129280, bf16, stochastic acceptance).  Inputs are seeded and synthetic.
Three copies of every input are rotated so that no step finds its inputs in
the 256 MB last-level cache from the step before.

Prints ONE JSON line on stdout: verified tokens/s (sum of q_len over the step
time), the per-stage times measured with HIP events on the launch stream, the
achieved HBM bandwidth of attention + acceptance, a roofline entry for the
dominant kernel (verify attention) and the oracle timed on the host cores on a
bounded sample of the same workload.  Progress goes to stderr.
"""
from __future__ import annotations

import argparse
import json
import os
import sys
import time

import numpy as np

HBM_PEAK_GBPS = 8000.0  # MI355X HBM3E
MFMA_BF16_PEAK_TFLOPS = 2500.0  # MI355X dense bf16 matrix peak
NCOPY = 3


def log(*a):
    print("[bench]", *a, file=sys.stderr, flush=True)


def parse():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--workload", default="serving")
    ap.add_argument("--stage", default="step", choices=["step", "draft"],
                    help="step: the verification step (schedule, attention, acceptance); "
                         "draft: the draft block that produces its inputs")
    ap.add_argument("--head", default="markov", choices=["markov", "rnn"],
                    help="the draft block's sequential head (--stage draft)")
    ap.add_argument("--seed", type=int, default=0)
    ap.add_argument("--cpu-seconds", type=float, default=15.0,
                    help="target CPU time of the oracle baseline sample")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--graph", action="store_true",
                    help="time the steps as replays of one captured HIP graph per input copy "
                         "instead of direct launches (--stage step; measured slower on this stack)")
    ap.add_argument("--rate", action="store_true",
                    help="also time dspark_accept with the analytic acceptance-rate output "
                         "(stochastic workloads) and report its extra time and bytes")
    ap.add_argument("--identity-pages", action="store_true",
                    help="also time attention on a copy of the KV pool laid out in request and "
                         "page order (identity block table) beside the shuffled pages")
    ap.add_argument("--copy-probe", action="store_true",
                    help="only run a plain 1 GiB device copy 10 times (calibrates the HBM counters)")
    ap.add_argument("--traffic-from", nargs=4, metavar=("FETCH_CSV", "WRITE_CSV", "COPY_FETCH_CSV",
                                                        "COPY_WRITE_CSV"),
                    help="turn four rocprofv3 --pmc counter files (FETCH_SIZE and WRITE_SIZE of a bench "
                         "run, then of a --copy-probe run) into the committed traffic summary")
    ap.add_argument("--traffic-group", default="attention", choices=["attention", "accept"],
                    help="which launches --traffic-from summarises: one dspark_verify_attn call "
                         "(or draft block with --stage draft), or one dspark_accept call")
    return ap.parse_args()


def attention_bytes(w, kv_len: np.ndarray, q_len: np.ndarray) -> int:
    """Algorithmic HBM bytes of one verify-attention launch."""
    s = w.kv_elem_bytes
    per_tok = w.Hkv * (w.Dqk if w.mla else (w.Dqk + w.Dv)) * s
    kv = int(kv_len.astype(np.int64).sum()) * per_tok
    qo = int(q_len.sum()) * w.Hq * (w.Dqk + w.Dv) * s
    bt = int(((kv_len + w.page - 1) // w.page).sum()) * 4
    return kv + qo + bt


def attention_flop(w, kv_len: np.ndarray, q_len: np.ndarray) -> int:
    """Algorithmic FLOP of one verify-attention launch: query t of request r
    scores and mixes kv_len - q_len + t + 1 keys (causal), Dqk + Dv MACs each."""
    kv = kv_len.astype(np.int64)
    ql = q_len.astype(np.int64)
    keys = int((ql * (kv - ql) + ql * (ql + 1) // 2).sum())
    return 2 * keys * w.Hq * (w.Dqk + w.Dv)


def accept_bytes(w, q_len: np.ndarray, accepted: np.ndarray) -> int:
    """Algorithmic HBM bytes of one acceptance call: every verified logit row
    once, plus the draft row at the first rejection (stochastic)."""
    rows = int(q_len.sum()) * w.V * w.logit_elem_bytes
    if w.greedy:
        return rows
    rejected = int((accepted < (q_len - 1)).sum())
    return rows + rejected * w.V * 4


HERE = os.path.dirname(os.path.abspath(__file__))
CSRC = os.path.join(HERE, "paper_2607_05147_amd", "csrc")
# The launches of one dspark_verify_attn call per attention path, the source
# they come from and the roofline that bounds the main kernel.
ATTN_PATHS = {
    "gqa": {"src": "attn_mfma.hip", "kernels": ("mf_plan", "attn_mfma_kernel", "attn_mfma_merge"),
            "bound": "hbm"},
    "latent": {"src": "attn_mla.hip", "kernels": ("mla_plan", "mla_kernel", "mla_merge"),
               "bound": "mfma"},
    "generic": {"src": "attn_generic.hip", "kernels": ("attn_generic_kernel", "attn_generic_merge"),
                "bound": "hbm"},
    # not attention: the draft blocks' launches
    "draft": {"src": "markov.hip", "kernels": ("md_hidden", "md_first", "md_coop", "md_check", "md_tile",
                                              "md_stats", "md_norm"),
              "bound": "hbm"},
    "rnn_draft": {"src": "markov.hip", "kernels": ("md_hidden", "rnn_hproj", "md_first", "rnn_state",
                                                   "md_coop", "md_check", "md_tile", "md_stats", "md_norm"),
                  "bound": "hbm"},
    # not attention: the acceptance launches of one dspark_accept call (the
    # resolve kernel runs once per call)
    "accept": {"src": "accept.hip", "kernels": ("acc_resolve", "acc_rowpass", "acc_resid", "acc_draw"),
               "bound": "hbm"},
}


def attn_path(w, bf16: bool) -> str:
    """Which kernels dspark_verify_attn runs for the workload (the library's
    own dispatch conditions; the bench's V aliases K on latent shapes)."""
    pow2 = w.page >= 64 and (w.page & (w.page - 1)) == 0
    if bf16 and w.Dqk == 128 and w.Dv == 128 and pow2:
        return "gqa"
    if bf16 and w.mla and w.Dqk == 576 and w.Dv == 512 and pow2:
        return "latent"
    return "generic"


def path_of_workload(name: str) -> str:
    if name in ("draft", "rnn_draft"):
        return name
    import paper_2607_05147_amd.synth as synth
    w = synth.WORKLOADS[name]
    return attn_path(w, w.kv_elem_bytes == 2)


def traffic_file(workload: str, group: str = "attention") -> str:
    if group == "accept":
        return os.path.join(HERE, "profiles", f"accept_{workload}_traffic.json")
    if workload == "draft":
        return os.path.join(HERE, "profiles", "markov_draft_serving_traffic.json")
    if workload == "rnn_draft":
        return os.path.join(HERE, "profiles", "rnn_draft_serving_traffic.json")
    return os.path.join(HERE, "profiles", f"verify_attn_{workload}_traffic.json")


def source_sha(path: str) -> str:
    import hashlib
    with open(path, "rb") as f:
        return hashlib.sha256(f.read()).hexdigest()


def _counter_rows(path: str):
    """(kernel name, value) per dispatch of a rocprofv3 counter_collection.csv."""
    import csv
    per = {}
    with open(path) as f:
        for row in csv.DictReader(f):
            key = (row["Dispatch_Id"], row["Kernel_Name"])
            per[key] = per.get(key, 0.0) + float(row["Counter_Value"])
    return [(k[1], v) for k, v in per.items()]


def traffic_from(fetch_csv, write_csv, copy_fetch_csv, copy_write_csv, workload="serving",
                 group="attention"):
    """Per-call HBM traffic of dspark_verify_attn (or a draft block, or with
    group "accept" of dspark_accept) from FETCH_SIZE / WRITE_SIZE (KiB per
    dispatch), each scaled by what the same counter reads for a plain 1 GiB
    device copy; written next to the other profile summaries."""
    path = ATTN_PATHS["accept" if group == "accept" else path_of_workload(workload)]
    kernels = path["kernels"]
    first = kernels[0] if group == "accept" else kernels[1]  # launched once per call
    def copy_scale(path):
        vals = [v for name, v in _counter_rows(path) if "copyBuffer" in name or "copy" in name.lower()]
        vals = [v for v in vals if v > 1e5]  # the 1 GiB copies
        return (float(1 << 30) / 1024.0) / (sum(vals) / len(vals))

    def per_call(path):
        rows = _counter_rows(path)
        calls = sum(1 for name, _ in rows if first in name)
        if workload in ("draft", "rnn_draft"):  # one md_first launch per call
            calls = sum(1 for name, _ in rows if "md_first" in name)
        tot = {k: sum(v for name, v in rows if k in name) for k in kernels}
        return {k: tot[k] / calls * 1024.0 for k in kernels}, calls

    sel = {"draft": "--stage draft", "rnn_draft": "--stage draft --head rnn"}.get(
        workload, f"--workload {workload}")
    sf, sw = copy_scale(copy_fetch_csv), copy_scale(copy_write_csv)
    fetch, calls = per_call(fetch_csv)
    write, _ = per_call(write_csv)
    out = {
        "workload": workload,
        "group": group,
        "kernels": list(kernels),
        "calls": calls,
        "copy_scale": {"FETCH_SIZE": sf, "WRITE_SIZE": sw},
        "fetch_bytes_per_call": {k: v * sf for k, v in fetch.items()},
        "write_bytes_per_call": {k: v * sw for k, v in write.items()},
        "bytes_per_call": sum(fetch.values()) * sf + sum(write.values()) * sw,
        "source_sha256": source_sha(os.path.join(CSRC, path["src"])),
        "commands": [
            f"rocprofv3 --pmc FETCH_SIZE --output-format csv -d <dir> -o pmc -- python bench.py "
            f"{sel} --steps 2 --warmup 1 --no-cpu-baseline",
            f"rocprofv3 --pmc WRITE_SIZE --output-format csv -d <dir> -o pmc -- python bench.py "
            f"{sel} --steps 2 --warmup 1 --no-cpu-baseline",
            "rocprofv3 --pmc FETCH_SIZE --output-format csv -d <dir> -o pmc -- python bench.py --copy-probe",
            "rocprofv3 --pmc WRITE_SIZE --output-format csv -d <dir> -o pmc -- python bench.py --copy-probe",
            f"python bench.py {sel} --traffic-group {group} --traffic-from <the four "
            "pmc_counter_collection.csv files>",
        ],
    }
    dest = traffic_file(workload, group)
    os.makedirs(os.path.dirname(dest), exist_ok=True)
    with open(dest, "w") as f:
        json.dump(out, f, indent=1)
    log(f"traffic: {out['bytes_per_call'] / 1e9:.3f} GB per call (copy scale fetch {sf:.3f}, "
        f"write {sw:.3f}) -> {dest}")


def measured_traffic(workload: str):
    """HBM bytes per verify-attention call from the committed counter summary,
    or None when there is none or the kernel source changed since."""
    try:
        with open(traffic_file(workload)) as f:
            t = json.load(f)
    except (OSError, ValueError):
        return None
    src = os.path.join(CSRC, ATTN_PATHS[path_of_workload(workload)]["src"])
    if t.get("source_sha256") != source_sha(src):
        return None
    return t["bytes_per_call"]


def copy_probe():
    """A plain device copy of 1 GiB, ten times: the known byte count against
    which rocprofv3's FETCH_SIZE / WRITE_SIZE counters are scaled."""
    import torch
    n = 1 << 30
    a = torch.empty(n, dtype=torch.uint8, device="cuda:0")
    b = torch.empty_like(a)
    a.fill_(1)
    torch.cuda.synchronize()
    for _ in range(10):
        b.copy_(a)
    torch.cuda.synchronize()
    log(f"copy probe: 10 copies of {n} bytes")


def device_copy_gbps():
    """Bandwidth of a plain device-to-device copy (1 GiB, read + write bytes,
    best of ten), measured after the timed steps.  A reference point for a
    streaming kernel that reads and writes equal amounts, not a ceiling: a
    read-mostly kernel such as attention can exceed it."""
    import torch
    n = 1 << 30
    a = torch.empty(n, dtype=torch.uint8, device="cuda:0")
    b = torch.empty_like(a)
    a.fill_(1)
    b.copy_(a)
    best = 0.0
    for _ in range(10):
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record()
        b.copy_(a)
        e1.record()
        e1.synchronize()
        best = max(best, 2 * n / (e0.elapsed_time(e1) / 1e3) / 1e9)
    del a, b
    return best


def main():
    args = parse()
    if args.traffic_from:
        traffic_from(*args.traffic_from,
                     workload=draft_key(args) if args.stage == "draft" else args.workload,
                     group=args.traffic_group)
        return
    if args.copy_probe:
        copy_probe()
        return
    if args.gpus != 1:
        print(f"bench.py measures one GPU (--gpus {args.gpus} requested): the verify step "
              "shards by request across GPUs with no exchange, so N GPUs run N copies of "
              "this step", file=sys.stderr)
        sys.exit(2)

    import torch
    from paper_2607_05147_amd import dspark, synth

    if not torch.cuda.is_available():
        print("bench.py: no ROCm GPU visible", file=sys.stderr)
        sys.exit(1)
    if args.stage == "draft":
        draft_bench(args)
        return
    dev = torch.device("cuda:0")
    w = synth.WORKLOADS[args.workload]
    seed = args.seed
    bf16 = w.dtype == "bf16"

    def to_dev(a, as_bf16=False):
        a = np.ascontiguousarray(a)
        if as_bf16 or a.dtype == np.uint16:
            return torch.from_numpy(a.view(np.int16)).to(dev).view(torch.bfloat16)
        return torch.from_numpy(a).to(dev)

    t0 = time.time()
    conf = synth.confidences(w, seed)
    sps = synth.sps_table(w)
    conf_d, sps_d = to_dev(conf), to_dev(sps)
    # schedule once (untimed) to lay out the flattened verify rows
    ln_d, cu_d, _ = dspark.dspark_schedule(conf_d, sps_d, 0)
    torch.cuda.synchronize()
    ln = ln_d.cpu().numpy()
    q_len = 1 + ln.astype(np.int64)
    keys = synth.flat_keys(q_len)
    total_q = len(keys)
    log(f"workload {w.name}: R={w.R} total_q={total_q} mean q_len={q_len.mean():.2f}")
    kv = synth.paged_kv(w, seed)
    q = synth.query_rows(w, seed, keys)
    logits = synth.logit_rows(w, seed, keys)
    needed = np.arange(w.K)[None, :] < ln[:, None]
    dr = synth.drafts(w, seed, conf, needed=needed)
    log(f"inputs generated in {time.time() - t0:.1f}s: KV {kv.k.nbytes * (1 if w.mla else 2) / 1e9:.2f} GB, "
        f"logits {logits.nbytes / 1e6:.0f} MB")

    # device copies (rotated)
    copies = []
    k0 = to_dev(kv.k.reshape(-1), bf16)
    v0 = k0 if w.mla else to_dev(kv.v.reshape(-1), bf16)
    base = dict(conf=conf_d, sps=sps_d, k=k0, v=v0, bt=to_dev(kv.block_table),
                kv_len=to_dev(kv.kv_len), q=to_dev(q, bf16),
                logits=to_dev(logits, w.logit_dtype == "bf16"), tok=to_dev(dr.draft_tok),
                dp=None if dr.draft_p is None else to_dev(dr.draft_p),
                u=None if dr.u is None else to_dev(dr.u))
    del kv.k, kv.v
    for c in range(NCOPY):
        d = {k: (None if v is None else (v if c == 0 else v.clone())) for k, v in base.items()}
        if w.mla:
            d["v"] = d["k"]
        d["len"] = torch.empty(w.R, dtype=torch.int32, device=dev)
        d["cu"] = torch.empty(w.R + 1, dtype=torch.int32, device=dev)
        d["out"] = torch.empty((total_q, w.Hq, w.Dv), dtype=base["q"].dtype, device=dev)
        d["acc"] = torch.empty(w.R, dtype=torch.int32, device=dev)
        d["nxt"] = torch.empty(w.R, dtype=torch.int32, device=dev)
        copies.append(d)
    ws_attn = torch.empty(dspark.dspark_verify_attn_workspace_size(
        w.R, w.max_q, w.Hq, w.Hkv, w.Dqk, w.Dv, kv.max_pages, w.page, base["q"].dtype),
        dtype=torch.uint8, device=dev)
    ws_acc = torch.empty(dspark.dspark_accept_workspace_size(w.R, w.K, w.V), dtype=torch.uint8,
                         device=dev)
    ws_sched = torch.empty(dspark.dspark_schedule_workspace_size(w.R, w.K), dtype=torch.uint8,
                           device=dev)
    torch.cuda.synchronize()
    log(f"device inputs ready ({NCOPY} copies), {time.time() - t0:.1f}s")

    stream = torch.cuda.current_stream()

    def step(d, ev=None):
        if ev is not None:
            ev[0].record(stream)
        dspark.dspark_schedule(d["conf"], d["sps"], 0, len_out=d["len"], cu_q=d["cu"],
                               ws=ws_sched)
        if ev is not None:
            ev[1].record(stream)
        dspark.dspark_verify_attn(d["q"], d["k"], d["v"], kv.k_strides, kv.v_strides, d["bt"],
                                  d["kv_len"], d["cu"], w.max_q, w.Hkv, w.Dv, w.page, w.scale,
                                  out=d["out"], ws=ws_attn)
        if ev is not None:
            ev[2].record(stream)
        dspark.dspark_accept(d["tok"], d["logits"], d["cu"], draft_p=d["dp"], u=d["u"],
                             accepted_len=d["acc"], next_tok=d["nxt"], ws=ws_acc)
        if ev is not None:
            ev[3].record(stream)

    for i in range(args.warmup):
        step(copies[i % NCOPY])
    torch.cuda.synchronize()
    accepted = copies[0]["acc"].cpu().numpy()

    # one captured step per input copy: a replay enqueues the whole step at once
    graphs = []
    if args.graph:
        for c in range(NCOPY):
            g = torch.cuda.CUDAGraph()
            with torch.cuda.graph(g):
                step(copies[c])
            graphs.append(g)
        torch.cuda.synchronize()
        for i in range(args.warmup):
            graphs[i % NCOPY].replay()
        torch.cuda.synchronize()

    # the timed region: exactly K steps and nothing else on the stream
    torch.cuda.synchronize()
    t_start = time.perf_counter()
    for i in range(args.steps):
        if graphs:
            graphs[i % NCOPY].replay()
        else:
            step(copies[i % NCOPY])
    torch.cuda.synchronize()
    wall = time.perf_counter() - t_start
    # per-stage times from a second, separate pass with events between the
    # stages (each event record leaves the GPU idle for a few microseconds,
    # so these passes are kept out of the timed region)
    evs = [[torch.cuda.Event(enable_timing=True) for _ in range(4)] for _ in range(args.steps)]
    for i in range(args.steps):
        step(copies[i % NCOPY], evs[i])
    torch.cuda.synchronize()
    sched_ms = np.array([e[0].elapsed_time(e[1]) for e in evs])
    attn_ms = np.array([e[1].elapsed_time(e[2]) for e in evs])
    acc_ms = np.array([e[2].elapsed_time(e[3]) for e in evs])
    ms_per_step = wall * 1e3 / args.steps
    # per-step times from a third pass with one event at each step boundary
    # (one event record per step, so each includes one record's idle gap)
    bnd = [torch.cuda.Event(enable_timing=True) for _ in range(args.steps + 1)]
    bnd[0].record(stream)
    for i in range(args.steps):
        step(copies[i % NCOPY])
        bnd[i + 1].record(stream)
    torch.cuda.synchronize()
    step_ms = np.array([bnd[i].elapsed_time(bnd[i + 1]) for i in range(args.steps)])

    ab = attention_bytes(w, kv.kv_len, q_len)
    path = attn_path(w, bf16)
    af = attention_flop(w, kv.kv_len, q_len)
    cb = accept_bytes(w, q_len, accepted)
    attn_s = attn_ms.mean() / 1e3
    acc_s = acc_ms.mean() / 1e3
    attn_gbps = ab / attn_s / 1e9
    both_gbps = (ab + cb) / (attn_s + acc_s) / 1e9
    attn_tflops = af / attn_s / 1e12
    log(f"step: {ms_per_step * 1e3:.1f} us (wall mean), median {np.median(step_ms) * 1e3:.1f} us "
        f"over {args.steps} event-bounded steps")
    log(f"per step: schedule {sched_ms.mean() * 1e3:.1f} us, attention {attn_ms.mean() * 1e3:.1f} us "
        f"({attn_gbps:.0f} GB/s, {attn_tflops:.1f} TFLOP/s), accept {acc_ms.mean() * 1e3:.1f} us; "
        f"attention+accept {both_gbps:.0f} GB/s = {both_gbps / HBM_PEAK_GBPS:.1%} of peak")

    result = {
        "metric": "verified tokens/s and achieved HBM GB/s (% of peak), verify step on 1 MI355X",
        "value": total_q / (ms_per_step / 1e3),
        "unit": "verified tokens/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": ms_per_step,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16" if bf16 else "f32",
        "data": "synthetic (seeded; shapes and distributions of the workload)",
        "config": {
            "workload": f"{w.name}: R={w.R} requests, Hq={w.Hq}/Hkv={w.Hkv}, head dim {w.Dqk}/{w.Dv}, "
                        f"page {w.page}, K={w.K}, V={w.V}, "
                        f"{'greedy' if w.greedy else 'stochastic'} acceptance, one attention layer",
            "seed": seed,
            "total_q": total_q,
            "mean_q_len": float(q_len.mean()),
            "kv_tokens": int(kv.kv_len.sum()),
        },
        "ms_per_step_median": float(np.median(step_ms)),
        "timing": f"ms_per_step: wall clock over exactly {args.steps} steps / {args.steps}; "
                  f"ms_per_step_median: median of {args.steps} steps bounded by HIP events "
                  "(one event record per step); stages: HIP events between the stages in a "
                  "separate pass, mean and median",
        "stages_us": {"schedule": float(sched_ms.mean() * 1e3),
                      "verify_attn": float(attn_ms.mean() * 1e3),
                      "accept": float(acc_ms.mean() * 1e3)},
        "stages_us_median": {"schedule": float(np.median(sched_ms) * 1e3),
                             "verify_attn": float(np.median(attn_ms) * 1e3),
                             "accept": float(np.median(acc_ms) * 1e3)},
        "attn_accept_hbm": {"bytes": ab + cb, "achieved_gbps": both_gbps,
                            "frac_of_peak": both_gbps / HBM_PEAK_GBPS},
        "emitted_tokens_per_s": float((accepted + 1).sum()) / (ms_per_step / 1e3),
        "launch": "HIP graph replay (one captured step per input copy)" if args.graph else "direct launches",
        # the dominant kernel: one dspark_verify_attn call (plan, attention and
        # split-merge launches, bracketed together by the events)
        "roofline": roofline_entry(w.name, path, ab, af, attn_s),
    }
    if args.rate and not w.greedy:
        result["accept_rate"] = rate_timing(args, w, copies, ws_acc, stream, q_len, cb, acc_ms)
    if args.identity_pages:
        result["page_layout"] = page_layout_timing(args, w, kv, copies, ws_attn, stream, ab)
    cp = device_copy_gbps()
    result["device_copy"] = {"what": "device-to-device copy of 1 GiB, read + write bytes, best "
                                     "of 10 (a reference point, not a ceiling)",
                             "gbps": cp, "attn_ratio": attn_gbps / cp,
                             "attn_accept_ratio": both_gbps / cp}
    log(f"device copy {cp:.0f} GB/s: attention at {attn_gbps / cp:.2f}x of it, "
        f"attention+accept at {both_gbps / cp:.2f}x")

    if not args.no_cpu_baseline:
        result["cpu_baseline"] = cpu_baseline(w, seed, conf, sps, ln, kv, q, logits, dr,
                                              args.cpu_seconds)
    print(json.dumps(result), flush=True)


def rate_timing(args, w, copies, ws_acc, stream, q_len, accept_nbytes, acc_ms):
    """dspark_accept with the analytic acceptance-rate output (sum_v min(p_t,
    p_d) of every tested row): its time beside the plain call, and the bytes
    of the rate pass (it reads every tested logit row and its draft row
    again, after the row statistics are known)."""
    import torch
    from paper_2607_05147_amd import dspark
    rates = [torch.empty(int(q_len.sum()), dtype=torch.float32, device="cuda:0") for _ in copies]
    evs = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))
           for _ in range(args.steps)]
    for i in range(args.warmup + args.steps):
        d = copies[i % NCOPY]
        if i >= args.warmup:
            evs[i - args.warmup][0].record(stream)
        dspark.dspark_accept(d["tok"], d["logits"], d["cu"], draft_p=d["dp"], u=d["u"],
                             accepted_len=d["acc"], next_tok=d["nxt"],
                             accept_rate=rates[i % NCOPY], ws=ws_acc)
        if i >= args.warmup:
            evs[i - args.warmup][1].record(stream)
    torch.cuda.synchronize()
    ms = np.array([e[0].elapsed_time(e[1]) for e in evs])
    tested = int((q_len - 1).sum())
    rate_bytes = tested * w.V * (w.logit_elem_bytes + 4)
    extra_us = (np.median(ms) - np.median(acc_ms)) * 1e3
    out = {"accept_with_rate_us_median": float(np.median(ms) * 1e3),
           "accept_us_median": float(np.median(acc_ms) * 1e3),
           "extra_us": float(extra_us),
           "rate_pass_bytes": rate_bytes,
           "rate_pass_gbps": rate_bytes / max(extra_us, 1e-3) / 1e3,
           "tested_rows": tested}
    log(f"accept with rate: {out['accept_with_rate_us_median']:.1f} us vs "
        f"{out['accept_us_median']:.1f} us; rate pass {rate_bytes / 1e6:.0f} MB in "
        f"{extra_us:.1f} us")
    return out


def page_layout_timing(args, w, kv, copies, ws_attn, stream, nbytes):
    """Attention on the shuffled page pool against a copy laid out in request
    and page order with an identity block table: the cost of page scatter."""
    import torch
    from paper_2607_05147_amd import dspark
    bt = kv.block_table
    npg = (kv.kv_len.astype(np.int64) + w.page - 1) // w.page
    perm = np.concatenate([bt[r, :npg[r]] for r in range(w.R)]).astype(np.int64)
    offs = np.concatenate([[0], np.cumsum(npg)])
    bt_id = np.zeros_like(bt)
    for r in range(w.R):
        bt_id[r, :npg[r]] = np.arange(offs[r], offs[r + 1])
    d0 = copies[0]
    pages = int(d0["k"].numel() // kv.k_strides[0])
    idx = torch.from_numpy(perm).to("cuda:0")
    k_id = d0["k"].view(pages, -1).index_select(0, idx).reshape(-1)
    v_id = k_id if w.mla else d0["v"].view(pages, -1).index_select(0, idx).reshape(-1)
    bt_d = torch.from_numpy(bt_id).to("cuda:0")

    def timed(k, v, btab):
        evs = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))
               for _ in range(args.steps)]
        for i in range(args.warmup + args.steps):
            if i >= args.warmup:
                evs[i - args.warmup][0].record(stream)
            dspark.dspark_verify_attn(d0["q"], k, v, kv.k_strides, kv.v_strides, btab,
                                      d0["kv_len"], d0["cu"], w.max_q, w.Hkv, w.Dv, w.page,
                                      w.scale, out=d0["out"], ws=ws_attn)
            if i >= args.warmup:
                evs[i - args.warmup][1].record(stream)
        torch.cuda.synchronize()
        return float(np.median([e[0].elapsed_time(e[1]) for e in evs]) * 1e3)

    sh = timed(d0["k"], d0["v"], d0["bt"])
    ident = timed(k_id, v_id, bt_d)
    del k_id, v_id
    out = {"note": "one input copy in both runs (the KV is ~9x the 256 MB last-level cache)",
           "shuffled_us_median": sh, "identity_us_median": ident,
           "shuffled_gbps": nbytes / sh / 1e3, "identity_gbps": nbytes / ident / 1e3}
    log(f"page layout: shuffled {sh:.1f} us, identity {ident:.1f} us")
    return out


def draft_bytes(w, rank: int, d: int, base_bytes: int) -> int:
    """Algorithmic HBM bytes of one draft-block call: per position the base
    logits and the projection read once and the draft distribution written
    once, plus the embedding rows, hidden states and small per-row values."""
    per_pos = w.R * w.V * base_bytes + w.V * rank * 2 + w.R * w.V * 4
    return w.K * per_pos + w.R * w.K * (d * 2 + rank * 2 + 16) + (d + rank) * 4


def rnn_draft_bytes(w, rank: int, d: int, base_bytes: int) -> int:
    """Algorithmic HBM bytes of one RNN-head draft-block call: the Markov
    head's, plus the projection's hidden columns read once and its product
    written once, and per position the state and embedding columns of the
    projection, that product's row, and the state read and written."""
    once = 3 * rank * d * 2 + w.R * w.K * 3 * rank * 4
    per_pos = 3 * rank * 2 * rank * 2 + w.R * 3 * rank * 4 + 2 * w.R * rank * 4
    return draft_bytes(w, rank, d, base_bytes) + once + w.K * per_pos


def draft_key(args) -> str:
    return "rnn_draft" if args.head == "rnn" else "draft"


def draft_bench(args):
    """Times the draft block (dspark_markov_draft, or dspark_rnn_draft with
    --head rnn) on the workload's shape (R requests, K draft positions, its
    vocabulary and logit dtype, rank 256, 4096-wide hidden states) and prints
    one JSON line."""
    import torch
    import oracle
    from paper_2607_05147_amd import dspark, synth

    dev = torch.device("cuda:0")
    w = synth.WORKLOADS[args.workload]
    rank, d = synth.MARKOV_RANK, synth.MARKOV_HIDDEN
    rnn = args.head == "rnn"
    t0 = time.time()
    inp = synth.markov_inputs(w, args.seed, rank=rank, d=d, rnn=rnn)

    def to_dev(a):
        a = np.ascontiguousarray(a)
        if a.dtype == np.uint16:
            return torch.from_numpy(a.view(np.int16)).to(dev).view(torch.bfloat16)
        return torch.from_numpy(a).to(dev)

    args_d = dict(anchor=to_dev(inp.anchor), base=to_dev(inp.base), W1=to_dev(inp.W1),
                  W2t=to_dev(inp.W2t), w_conf=to_dev(inp.w_conf), u=to_dev(inp.u),
                  hidden=to_dev(inp.hidden), sts=to_dev(inp.sts_temp),
                  Wrnn=to_dev(inp.Wrnn) if rnn else None)
    tok = torch.empty((w.R, w.K), dtype=torch.int32, device=dev)
    dp = torch.empty((w.R, w.K, w.V), dtype=torch.float32, device=dev)
    conf = torch.empty((w.R, w.K), dtype=torch.float32, device=dev)
    ws_size = (dspark.dspark_rnn_draft_workspace_size if rnn else
               dspark.dspark_markov_draft_workspace_size)(w.R, w.K, w.V, rank)
    ws = torch.empty(ws_size, dtype=torch.uint8, device=dev)
    torch.cuda.synchronize()
    log(f"draft inputs ready in {time.time() - t0:.1f}s: base logits {inp.base.nbytes / 1e6:.0f} MB, "
        f"W1 + W2t {2 * inp.W1.nbytes / 1e6:.0f} MB")

    def call():
        if rnn:
            dspark.dspark_rnn_draft(args_d["anchor"], args_d["base"], args_d["W1"], args_d["W2t"],
                                    args_d["Wrnn"], args_d["w_conf"], args_d["u"], w.K,
                                    hidden=args_d["hidden"], sts_temp=args_d["sts"], draft_tok=tok,
                                    draft_p=dp, conf=conf, ws=ws)
        else:
            dspark.dspark_markov_draft(args_d["anchor"], args_d["base"], args_d["W1"], args_d["W2t"],
                                       args_d["w_conf"], args_d["u"], w.K, hidden=args_d["hidden"],
                                       sts_temp=args_d["sts"], draft_tok=tok, draft_p=dp, conf=conf,
                                       ws=ws)

    for _ in range(args.warmup):
        call()
    torch.cuda.synchronize()
    # the timed region: exactly the calls; events in a second pass
    t_start = time.perf_counter()
    for _ in range(args.steps):
        call()
    torch.cuda.synchronize()
    wall = time.perf_counter() - t_start
    stream = torch.cuda.current_stream()
    evs = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))
           for _ in range(args.steps)]
    for e in evs:
        e[0].record(stream)
        call()
        e[1].record(stream)
    torch.cuda.synchronize()
    ms = np.array([e[0].elapsed_time(e[1]) for e in evs])
    ms_per = wall * 1e3 / args.steps
    nbytes = (rnn_draft_bytes if rnn else draft_bytes)(w, rank, d, w.logit_elem_bytes)
    gbps = nbytes / (ms.mean() / 1e3) / 1e9
    head = "RNN-head" if rnn else "Markov-head"
    log(f"{head} draft block: {ms.mean() * 1e3:.1f} us per call ({ms.mean() * 1e3 / w.K:.1f} us per "
        f"position), {gbps:.0f} GB/s = {gbps / HBM_PEAK_GBPS:.1%} of HBM peak")
    kernels = ("dspark_rnn_draft: md_hidden + rnn_hproj + md_first, then rnn_state + md_coop per "
               "position, md_check" if rnn else
               "dspark_markov_draft: md_hidden + md_first, then md_coop per position, md_check")
    result = {
        "metric": f"draft tokens/s and achieved HBM GB/s (% of peak), {head} draft block on 1 MI355X",
        "value": w.R * w.K / (ms_per / 1e3),
        "unit": "draft tokens/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": ms_per,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16",
        "data": "synthetic (seeded; shapes and distributions of the workload)",
        "config": {"workload": f"{args.head} draft ({w.name} shape): R={w.R} requests, K={w.K} "
                               f"positions, V={w.V}, rank {rank}, hidden {d}, {w.logit_dtype} base logits",
                   "seed": args.seed},
        "roofline": {"kernel": kernels,
                     "bound": "hbm", "achieved": gbps, "peak": HBM_PEAK_GBPS, "unit": "GB/s",
                     "frac": gbps / HBM_PEAK_GBPS, "bytes_per_launch": nbytes,
                     "traffic": measured_traffic(draft_key(args))},
    }
    if not args.no_cpu_baseline:
        # the oracle on the first n requests, n sized to about --cpu-seconds
        base = inp.base.reshape(w.R, w.K, -1)

        def run(n):
            s = time.perf_counter()
            if rnn:
                oracle.rnn_draft(inp.anchor[:n], base[:n].reshape(n * w.K, -1), w.logit_dtype, inp.W1,
                                 inp.W2t, inp.Wrnn, inp.w_conf, inp.u[:n], w.K, w.V,
                                 hidden=inp.hidden[:n], sts_temp=inp.sts_temp, want_p=False)
            else:
                oracle.markov_draft(inp.anchor[:n], base[:n].reshape(n * w.K, -1), w.logit_dtype,
                                    inp.W1, inp.W2t, inp.w_conf, inp.u[:n], w.K, w.V,
                                    hidden=inp.hidden[:n], sts_temp=inp.sts_temp, want_p=False)
            return time.perf_counter() - s

        th = oracle.threads()
        t1 = run(min(th, w.R))
        n = int(min(w.R, max(th, th * round(args.cpu_seconds / max(t1, 1e-3)))))
        tn = run(n) if n > min(th, w.R) else t1
        n = max(n, min(th, w.R))
        reps = 1
        while tn * reps < 0.66 * args.cpu_seconds:  # the whole block is quick: repeat it
            tn += run(n)
            reps += 1
        # one thread, one request
        oracle.set_threads(1)
        try:
            t_one = run(1)
        finally:
            oracle.set_threads(th)
        result["cpu_baseline"] = {"value": reps * n * w.K / tn, "unit": "draft tokens/s", "cores": th,
                                  "kind": "oracle", "sample": f"requests 0..{n - 1} of the same block "
                                  f"({n * w.K} draft tokens), {reps} times", "seconds": tn,
                                  "cpu_model": cpu_model(),
                                  "one_thread": {"value": w.K / t_one, "sample": f"request 0 ({w.K} draft tokens)",
                                                 "seconds": t_one}}
        log(f"oracle baseline: {n} requests x {reps} in {tn:.1f}s on {th} threads; "
            f"one request on 1 thread in {t_one:.1f}s")
    print(json.dumps(result), flush=True)


def roofline_entry(workload: str, path: str, nbytes: int, flop: int, seconds: float) -> dict:
    """Roofline of one dspark_verify_attn call (its plan, attention and merge
    launches, bracketed together by the events): HBM-bound paths report
    algorithmic bytes per second against the HBM peak, the latent path FLOP per
    second against the dense bf16 matrix peak."""
    info = ATTN_PATHS[path]
    out = {"kernel": "dspark_verify_attn: " + " + ".join(info["kernels"]), "bound": info["bound"]}
    if info["bound"] == "mfma":
        achieved = flop / seconds / 1e12
        out.update({"achieved": achieved, "peak": MFMA_BF16_PEAK_TFLOPS, "unit": "TFLOP/s",
                    "frac": achieved / MFMA_BF16_PEAK_TFLOPS, "flop_per_launch": flop})
    else:
        achieved = nbytes / seconds / 1e9
        out.update({"achieved": achieved, "peak": HBM_PEAK_GBPS, "unit": "GB/s",
                    "frac": achieved / HBM_PEAK_GBPS, "bytes_per_launch": nbytes})
    out["traffic"] = measured_traffic(workload) if path != "generic" else None
    return out


def cpu_baseline(w, seed, conf, sps, ln, kv, q, logits, dr, target_s):
    """The oracle on a bounded sample of the same step: the schedule over all
    requests, then attention and acceptance for the first n requests (all of
    their verify tokens); n grows until the sample costs about target_s."""
    import oracle
    from paper_2607_05147_amd import synth

    cu = oracle.cu_from_len(ln)
    kvk = synth.paged_kv(w, seed)  # the device copy freed the host arrays

    def run(n):
        t = time.perf_counter()
        oracle.schedule(conf, sps, 0)
        sub_cu = cu[: n + 1]
        rows = int(sub_cu[-1])
        oracle.verify_attn(q[:rows], kvk.k, kvk.v, kvk.k_strides, kvk.v_strides,
                           kvk.block_table[:n], kvk.kv_len[:n], sub_cu, w.Hq, w.Hkv, w.Dqk, w.Dv,
                           w.page, w.scale, w.dtype)
        oracle.accept(dr.draft_tok[:n], None if dr.draft_p is None else dr.draft_p[:n],
                      logits[:rows], w.logit_dtype, sub_cu, w.K, w.V,
                      u=None if dr.u is None else dr.u[:n])
        return time.perf_counter() - t, rows

    n = 1
    el, rows = run(n)
    while el < target_s / 4 and n < w.R:
        n = min(w.R, max(n + 1, int(n * min(8.0, target_s / max(el, 1e-3)))))
        el, rows = run(n)
    # a whole step that is quicker than the target is repeated up to it
    reps = 1
    while n == w.R and el < target_s * 0.7:
        e2, _ = run(n)
        el += e2
        reps += 1
    nthreads = oracle.threads()
    log(f"oracle baseline: {n} requests, {rows} verify tokens x {reps} in {el:.1f}s "
        f"on {nthreads} threads")
    # the same oracle on one thread, over a smaller sample (a few seconds)
    oracle.set_threads(1)
    try:
        n1 = 1
        el1, rows1 = run(n1)
        while el1 < target_s / 8 and n1 < n:
            n1 = min(n, max(n1 + 1, int(n1 * min(4.0, target_s / 6 / max(el1, 1e-3)))))
            el1, rows1 = run(n1)
    finally:
        oracle.set_threads(nthreads)
    log(f"oracle on 1 thread: {n1} requests, {rows1} verify tokens in {el1:.1f}s")
    return {"value": rows * reps / el, "unit": "verified tokens/s", "cores": nthreads,
            "kind": "oracle",
            "sample": f"schedule over all {w.R} requests; attention + acceptance for requests "
                      f"0..{n - 1} ({rows} verify tokens, {int(kvk.kv_len[:n].sum())} context tokens)"
                      + (f", repeated {reps} times" if reps > 1 else ""),
            "seconds": el,
            "cpu_model": cpu_model(),
            "one_thread": {"value": rows1 / el1, "sample": f"requests 0..{n1 - 1} ({rows1} verify tokens)",
                           "seconds": el1}}


def cpu_model() -> str:
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return "unknown"


if __name__ == "__main__":
    main()
