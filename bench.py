"""Benchmark of the FastEagle single-pass cascaded drafter on one MI355X.

One step = one whole drafting pass (feature fusion, input FC, N cascade
layers, LM head with fused softmax/top-k) plus the Backbone Expansion tree,
over one batch of synthetic, seeded, paper-shaped inputs that are resident in
HBM before timing starts.  Prints ONE JSON line.

    python bench.py [--steps K] [--warmup W] [--workload NAME] [--no-cpu-baseline]
"""
from __future__ import annotations

import argparse
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

METRIC = "µs per N-token cascaded draft pass and drafts/s, 8B-shaped bf16, batch 1 / 32"
HBM_PEAK_GBS = 8000.0          # MI355X HBM3E, vendor figure
MFMA_PEAK_TFS = {"bf16": 2500.0, "f32": 157.3}  # dense matrix-core peaks (fp32: the vector figure)
TRAFFIC_FILE = os.path.join(ROOT, "profiles", "traffic_gateup_llama8b_bf16_b1.txt")


def log(*a):
    print("[bench]", *a, file=sys.stderr, flush=True)


def gateup_bytes(cfg, batch):
    """Algorithmic bytes of one gate/up + SwiGLU launch: both weight matrices
    once, the normed input rows and the SwiGLU output rows."""
    es = 2 if cfg.dtype == "bf16" else 4
    d, I = cfg.hidden, cfg.intermediate
    return 2 * I * d * es + batch * d * es + batch * I * es


def pass_bytes(cfg, plens):
    """Algorithmic bytes of one pass: every weight once, each layer's prefix K/V once."""
    es = 2 if cfg.dtype == "bf16" else 4
    kv = cfg.n_layers * 2 * int(sum(plens)) * cfg.n_kv_heads * cfg.head_dim * es
    emb = len(plens) * cfg.hidden * es
    feats = len(plens) * cfg.n_feat_levels * cfg.hidden * es
    return cfg.weight_bytes() + kv + emb + feats


def pass_flops(cfg, plens):
    """Algorithmic FLOPs of one pass (2 per multiply-add): q, O and the MLP at
    B rows, layer i's K/V over its context rows (B*i under the cascade context,
    B otherwise), the LM head over all B*N rows, and per layer the attention's
    two contractions over P_b + nctx keys."""
    B, d, N = len(plens), cfg.hidden, cfg.n_layers
    qd, kvd, I, V = cfg.n_q_heads * cfg.head_dim, cfg.n_kv_heads * cfg.head_dim, cfg.intermediate, cfg.draft_vocab
    f = 2 * B * cfg.n_feat_levels * d * d + 2 * B * 2 * d * d
    for i in range(1, N + 1):
        nctx = i if cfg.cascade_ctx == "cascade" else 1
        f += 2 * B * d * qd + 2 * B * nctx * d * 2 * kvd + 2 * B * qd * d
        f += 2 * B * d * 2 * I + 2 * B * I * d
        f += sum(4 * qd * (int(p) + nctx) for p in plens)
    return f + 2 * B * N * d * V


def gemm_source_sha1():
    import hashlib
    h = hashlib.sha1()
    for f in ("fe_gemm.hip", "fe_internal.h"):
        with open(os.path.join(ROOT, "paper_2509_20416_amd", "csrc", f), "rb") as fh:
            h.update(fh.read())
    return h.hexdigest()


def kernel_source_sha1():
    """Digest of every kernel source of the library (a counter summary is valid
    only for the kernels it was taken from)."""
    import glob
    import hashlib
    h = hashlib.sha1()
    for f in sorted(glob.glob(os.path.join(ROOT, "paper_2509_20416_amd", "csrc", "*"))):
        with open(f, "rb") as fh:
            h.update(fh.read())
    return h.hexdigest()


def read_traffic():
    """HBM bytes per gate/up launch from the committed rocprofv3 counter summary
    (FETCH_SIZE + WRITE_SIZE, scaled by the copy-kernel factor); None when the
    summary is missing or was taken from other kernel sources than these."""
    vals = {}
    try:
        for line in open(TRAFFIC_FILE):
            if ":" in line and not line.startswith(("#", " ", "|")):
                k, v = line.split(":", 1)
                vals[k.strip()] = v.strip()
    except OSError:
        return None
    if vals.get("source_sha1") != gemm_source_sha1():
        log("traffic summary was taken from other GEMM sources; reporting traffic null")
        return None
    try:
        return float(vals["traffic_bytes_per_launch"])
    except (KeyError, ValueError):
        return None


def read_pass_traffic(name):
    """HBM bytes of one whole pass (FETCH_SIZE + WRITE_SIZE over every launch of
    one eager pass, scaled by the copy-kernel factors) from the committed
    counter summary of that workload; None when missing or taken from other
    kernel sources than these."""
    vals = {}
    try:
        for line in open(os.path.join(ROOT, "profiles", f"traffic_pass_{name}.txt")):
            if ":" in line and not line.startswith(("#", " ", "|")):
                k, v = line.split(":", 1)
                vals[k.strip()] = v.strip()
    except OSError:
        return None
    if vals.get("source_sha1") != kernel_source_sha1():
        log(f"pass traffic summary of {name} was taken from other kernel sources; reporting null")
        return None
    try:
        return float(vals["traffic_bytes_per_pass"])
    except (KeyError, ValueError):
        return None


def read_mfma_counters(name):
    """Matrix-core FLOPs counted by rocprofv3 (SQ_INSTS_VALU_MFMA_MOPS_BF16 x 512)
    for one pass and one max_prefix-row cache update of the workload, from the
    committed counter summary; None when missing or taken from other kernel
    sources than these."""
    vals = {}
    try:
        for line in open(os.path.join(ROOT, "profiles", f"mfma_{name}.txt")):
            if ":" in line and not line.startswith(("#", " ", "|")):
                k, v = line.split(":", 1)
                vals[k.strip()] = v.strip()
    except OSError:
        return None
    if vals.get("source_sha1") != kernel_source_sha1():
        log(f"MFMA counter summary of {name} was taken from other kernel sources; reporting null")
        return None
    try:
        return {"pass_flops": float(vals["pass_counter_mfma_flops"]),
                "kv_update_rows": int(vals["kv_update_rows"]),
                "kv_update_flops": float(vals["kv_update_counter_mfma_flops"]),
                "kv_update_busy": float(vals["kv_update_mfma_busy"]),
                "file": f"profiles/mfma_{name}.txt"}
    except (KeyError, ValueError):
        return None


def counter_mfma(ctr, ms, peak):
    """The pass's matrix-core rate from counted FLOPs over the measured pass time."""
    if ctr is None:
        return None
    return {"flops_per_pass": ctr["pass_flops"],
            "TFLOPs": ctr["pass_flops"] / (ms * 1e-3) / 1e12,
            "frac": ctr["pass_flops"] / (ms * 1e-3) / 1e12 / peak, "source": ctr["file"]}


def counter_update(ctr, upd, peak):
    """A cache update's matrix-core use from the counter summary (same row count only)."""
    if ctr is None or ctr["kv_update_rows"] != upd["rows"]:
        return None
    return {"flops": ctr["kv_update_flops"], "flops_vs_algorithmic": ctr["kv_update_flops"] / upd["flops"],
            "frac": ctr["kv_update_flops"] / (upd["us_per_call"] * 1e-6) / 1e12 / peak,
            "mfma_busy": ctr["kv_update_busy"], "source": ctr["file"]}


def cpu_baseline(cfg, w, inp, budget_s):
    """The oracle, as it stands, on the machine's host cores: whole passes (+ tree)
    of the same workload until about budget_s seconds have been spent, a third
    of the budget on one thread and the rest on all the threads it may use."""
    from oracle import feo
    affinity = len(os.sched_getaffinity(0))
    threads = max(1, min(16, affinity))

    def run(nthreads, budget):
        feo.set_threads(nthreads)
        n, t0 = 0, time.time()
        while True:
            ref = feo.draft_forward(cfg, w, inp, want_logits=False)
            feo.build_tree(cfg.n_layers, cfg.topk, inp.next_tokens, ref["topk_ids"], inp.prefix_lens)
            n += 1
            el = time.time() - t0
            if el >= budget:
                return n, el

    n1, el1 = run(1, budget_s / 3)
    n, el = run(threads, budget_s * 2 / 3)
    B = len(inp.prefix_lens)
    return {"value": n * B / el, "unit": "drafts/s", "cores": threads, "kind": "oracle",
            "ms_per_pass": el / n * 1e3, "ms_per_pass_1_thread": el1 / n1 * 1e3,
            "nproc": os.cpu_count(), "affinity": affinity,
            "sample": f"{n} full pass(es) + tree of the {cfg.name} workload "
                      f"(batch {B}) in {el:.1f} s on {threads} OpenMP threads, and "
                      f"{n1} in {el1:.1f} s on 1 thread; fp64"}


def kv_update_cost(cfg, M):
    """Algorithmic FLOPs and bytes of one cache update of M rows: the fusion
    and input FCs and every layer's K/V projection per row; every weight
    matrix read once, each row's features and embedding row read, its K/V rows
    written."""
    es = 2 if cfg.dtype == "bf16" else 4
    d, F, N = cfg.hidden, cfg.n_feat_levels, cfg.n_layers
    kvd = cfg.n_kv_heads * cfg.head_dim
    per_row_mac = F * d * d + 2 * d * d + N * d * 2 * kvd
    wbytes = per_row_mac * es
    rbytes = M * (F * d + d + N * 2 * kvd) * es
    return 2 * M * per_row_mac, wbytes + rbytes


def kv_update_cost_self(cfg, positions):
    """Algorithmic FLOPs and bytes of one cache update under the self context
    (the N layers run over the rows): per row the fusion and input FCs and per
    layer Q/K/V, O, gate/up and down, plus the attention's two contractions
    over the row's p earlier keys and its own; every weight matrix the layers
    use read once, each row's features, embedding row and written K/V rows."""
    es = 2 if cfg.dtype == "bf16" else 4
    d, F, N, I = cfg.hidden, cfg.n_feat_levels, cfg.n_layers, cfg.intermediate
    qd, kvd = cfg.n_q_heads * cfg.head_dim, cfg.n_kv_heads * cfg.head_dim
    M = len(positions)
    per_row_mac = F * d * d + 2 * d * d + N * (d * (qd + 2 * kvd) + qd * d + 3 * d * I)
    attn = sum(N * 4 * qd * (int(p) + 1) for p in positions)
    wbytes = (F * d * d + 2 * d * d + N * (d * (qd + 2 * kvd) + qd * d + 3 * d * I)) * es
    rbytes = M * (F * d + d + N * 2 * kvd) * es
    return 2 * M * per_row_mac + attn, wbytes + rbytes


def time_kv_update(dr, cfg, positions, reps=20, warmup=3, chunk_rows=1024):
    """fe_kv_update of len(positions) rows into fresh caches (rows written in
    order), eager launches on the current stream, mean per call."""
    import numpy as np
    import torch
    from fe_synth.gen import float_tensor, int_rng
    from paper_2509_20416_amd.drafter import to_device
    M = len(positions)
    dev = dr.device
    feats = to_device(float_tensor("bench.update.features", (M, cfg.n_feat_levels * cfg.hidden),
                                   7, cfg.dtype), cfg.dtype, dev)
    toks = to_device(int_rng("bench.update.tokens", 7).integers(0, cfg.target_vocab, M)
                     .astype(np.int32), "i32", dev)
    pos = to_device(np.asarray(positions, np.int32), "i32", dev)
    dst = to_device(np.arange(M, dtype=np.int32), "i32", dev)
    tdt = torch.bfloat16 if cfg.dtype == "bf16" else torch.float32
    shape = (M, cfg.n_kv_heads, cfg.head_dim)
    ks = [torch.zeros(shape, dtype=tdt, device=dev) for _ in range(cfg.n_layers)]
    vs = [torch.zeros(shape, dtype=tdt, device=dev) for _ in range(cfg.n_layers)]
    for _ in range(warmup):
        dr.kv_update(feats, toks, pos, dst, ks, vs, chunk_rows=chunk_rows)
    torch.cuda.synchronize()
    stream = torch.cuda.current_stream()
    ev0, ev1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    ev0.record(stream)
    for _ in range(reps):
        dr.kv_update(feats, toks, pos, dst, ks, vs, chunk_rows=chunk_rows)
    ev1.record(stream)
    torch.cuda.synchronize()
    ms = ev0.elapsed_time(ev1) / reps
    if cfg.cascade_ctx == "self":
        flops, nbytes = kv_update_cost_self(cfg, positions)
    else:
        flops, nbytes = kv_update_cost(cfg, M)
    tfs = flops / (ms * 1e-3) / 1e12
    peak = MFMA_PEAK_TFS[cfg.dtype]
    return {"rows": M, "us_per_call": ms * 1000.0, "flops": flops, "bytes": nbytes,
            "achieved_TFLOPs": tfs, "mfma_frac": tfs / peak,
            "hbm_frac": nbytes / (ms * 1e-3) / 1e9 / HBM_PEAK_GBS,
            "bound": "mfma" if flops / nbytes > peak * 1e3 / HBM_PEAK_GBS else "hbm",
            "issue": "eager, from Python"}


def device_weights(cfg, seed, device):
    """Seeded synthetic weights drawn on the device (timing of the larger
    configurations only; parity uses fe_synth.make_weights): the same shapes and
    distributions -- N(0, 0.02) matrices, 1 + N(0, 0.02) gains, a sorted random
    draft->target map -- from torch's device generator, so a 10 GB weight set
    takes milliseconds instead of a minute of host time."""
    import numpy as np
    import torch
    from fe_synth.gen import LayerWeights, Weights, int_rng
    g = torch.Generator(device=device).manual_seed(int(seed))
    tdt = torch.bfloat16 if cfg.dtype == "bf16" else torch.float32
    d, I, D = cfg.hidden, cfg.intermediate, cfg.head_dim
    qd, kvd = cfg.n_q_heads * D, cfg.n_kv_heads * D

    def lin(*shape):
        return (torch.randn(shape, generator=g, device=device) * 0.02).to(tdt)

    def gain():
        return (1.0 + torch.randn((d,), generator=g, device=device) * 0.02).to(tdt)

    layers = [LayerWeights(attn_norm=gain(), wq=lin(qd, d), wk=lin(kvd, d), wv=lin(kvd, d),
                           wo=lin(d, qd), mlp_norm=gain(), w_gate=lin(I, d), w_up=lin(I, d),
                           w_down=lin(d, I)) for _ in range(cfg.n_layers)]
    if cfg.draft_vocab == cfg.target_vocab:
        d2t = np.arange(cfg.draft_vocab, dtype=np.int32)
    else:
        d2t = np.sort(int_rng("d2t", seed).choice(cfg.target_vocab, size=cfg.draft_vocab,
                                                  replace=False)).astype(np.int32)
    return Weights(w_fuse=lin(d, cfg.n_feat_levels * d), w_in=lin(d, 2 * d),
                   embed=lin(cfg.target_vocab, d), final_norm=gain(),
                   lm_head=lin(cfg.draft_vocab, d), d2t=d2t, layers=layers)


def time_config(name, seed, steps, warmup, pass_mode=None):
    """One more configuration (tiny, 13B-, 70B-shaped): passes (forward + tree,
    graph replays) timed like the primary workload, weights drawn on the device."""
    import numpy as np
    import torch
    from fe_synth import NAMED, make_inputs
    from paper_2509_20416_amd import Drafter
    cfg = NAMED[name]
    inp = make_inputs(cfg, seed)
    plens = np.asarray(inp.prefix_lens)
    w = device_weights(cfg, seed, "cuda")
    dr = Drafter(cfg, w, max_batch=cfg.batch, max_prefix=int(plens.max()), graph=True)
    del w
    if pass_mode is not None:
        dr.set_pass_mode(pass_mode)
    di = dr.upload_inputs(inp)
    out = dr.alloc_outputs(cfg.batch, cfg.topk, draft=False)
    tree = dr.alloc_tree(cfg.batch, cfg.topk)
    for _ in range(warmup):
        dr.forward(di, out=out, tree=tree)
    torch.cuda.synchronize()
    stream = torch.cuda.current_stream()
    ev0, ev1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    ev0.record(stream)
    for _ in range(steps):
        dr.forward(di, out=out, tree=tree)
    ev1.record(stream)
    torch.cuda.synchronize()
    ms = ev0.elapsed_time(ev1) / steps
    dr.close()
    pbytes = pass_bytes(cfg, plens)
    log(f"{name}: {ms * 1000:.1f} us/pass")
    return {"batch": cfg.batch, "dtype": cfg.dtype, "hidden": cfg.hidden,
            "cascade_layers": cfg.n_layers, "prefix": int(plens.max()), "topk": cfg.topk,
            "steps": steps, "us_per_pass": ms * 1000.0, "drafts_per_s": cfg.batch * 1000.0 / ms,
            "bytes_per_pass": pbytes,
            "hbm_frac": pbytes / (ms * 1e-3) / 1e9 / HBM_PEAK_GBS,
            "weights": "seeded, drawn on the device"}


def time_second(name, seed, steps, warmup):
    """The other half of the metric (by default the batch-32 workload): passes
    (forward + tree, graph replays) timed the same way as the primary one."""
    import numpy as np
    import torch
    from fe_synth import NAMED, make_inputs, make_weights
    from paper_2509_20416_amd import Drafter
    cfg = NAMED[name]
    w = make_weights(cfg, seed)
    inp = make_inputs(cfg, seed)
    plens = np.asarray(inp.prefix_lens)
    dr = Drafter(cfg, w, max_batch=cfg.batch, max_prefix=int(plens.max()), graph=True)
    di = dr.upload_inputs(inp)
    out = dr.alloc_outputs(cfg.batch, cfg.topk, draft=False)
    tree = dr.alloc_tree(cfg.batch, cfg.topk)
    for _ in range(warmup):
        dr.forward(di, out=out, tree=tree)
    torch.cuda.synchronize()
    stream = torch.cuda.current_stream()
    ev0, ev1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    ev0.record(stream)
    for _ in range(steps):
        dr.forward(di, out=out, tree=tree)
    ev1.record(stream)
    torch.cuda.synchronize()
    ms = ev0.elapsed_time(ev1) / steps
    # stochastic drafting at this batch: uniforms read from HBM, or drawn in the pass
    from fe_synth import make_uniforms
    ud = torch.from_numpy(make_uniforms((cfg.batch, cfg.n_layers, cfg.draft_vocab),
                                        seed=seed + 1)).to(dr.device)
    so = torch.tensor([seed + 1, 0], dtype=torch.int64, device=dr.device)
    samp = {}
    for source, kw in (("uniforms_array", dict(uniforms=ud)), ("seeded", dict(seed_offset=so))):
        dr.forward(di, out=out, tree=tree, temperature=1.0, **kw)
        torch.cuda.synchronize()
        ev0.record(stream)
        for _ in range(steps):
            dr.forward(di, out=out, tree=tree, temperature=1.0, **kw)
        ev1.record(stream)
        torch.cuda.synchronize()
        samp[source + "_us_per_pass"] = ev0.elapsed_time(ev1) / steps * 1000.0
    samp["uniform_bytes"] = cfg.batch * cfg.n_layers * cfg.draft_vocab * 4
    # NEXT-1 for this batch: every sequence appends N+1 verified positions
    # (the most one cycle accepts) after its prefix
    upd_pos = np.concatenate([np.arange(p - cfg.n_layers - 1, p) for p in plens])
    upd = time_kv_update(dr, cfg, upd_pos)
    dr.close()
    pbytes, pflops = pass_bytes(cfg, plens), pass_flops(cfg, plens)
    peak = MFMA_PEAK_TFS[cfg.dtype]
    ctr = read_mfma_counters(name)
    log(f"{name}: {ms * 1000:.1f} us/pass")
    return {"workload": name, "batch": cfg.batch, "steps": steps, "warmup": warmup,
            "traffic_per_pass": read_pass_traffic(name),
            "counter_mfma": counter_mfma(ctr, ms, peak),
            "us_per_pass": ms * 1000.0, "drafts_per_s": cfg.batch * 1000.0 / ms,
            "hbm_frac": pbytes / (ms * 1e-3) / 1e9 / HBM_PEAK_GBS,
            "mfma_frac": pflops / (ms * 1e-3) / 1e12 / peak,
            "mfma_ceiling_frac": min(1.0, pflops / pbytes * HBM_PEAK_GBS / 1e3 / peak),
            "sampled_drafting": samp,
            "next_kv_update_cycle": upd}


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=200)
    ap.add_argument("--warmup", type=int, default=20)
    ap.add_argument("--workload", default="llama8b_bf16_b1")
    ap.add_argument("--seed", type=int, default=0)
    ap.add_argument("--eager", action="store_true", help="launch kernels one by one, no HIP graph")
    ap.add_argument("--pass-mode", type=int, default=None, choices=[0, 1],
                    help="batch-1 pass launches: 0 persistent stage launches, 1 one launch "
                         "per stage (default: the library's)")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--cpu-budget", type=float, default=12.0)
    ap.add_argument("--prof-repeats", type=int, default=8)
    ap.add_argument("--second", default="llama8b_bf16_b32",
                    help="second workload timed in the same run and reported in its own "
                         "object ('' = none; the batch-32 half of the metric by default)")
    ap.add_argument("--configs", default="tiny_fp32_b1,vicuna13b_bf16_b1,llama70b_bf16_b1",
                    help="further workloads timed in the same run ('' = none)")
    ap.add_argument("--device-weights", action="store_true",
                    help="draw the workload's weights on the device (seeded; for timing the large "
                         "configurations without a minute of host-side generation; implies "
                         "--no-cpu-baseline)")
    ap.add_argument("--counter-probe", action="store_true",
                    help="for rocprofv3 --pmc runs: two eager passes and two cache updates of "
                         "max_prefix rows, separated by fill kernels, then a plain 512 MiB "
                         "device copy as the counter scale reference; prints what ran")
    ap.add_argument("--traffic-probe", action="store_true",
                    help="for rocprofv3 --pmc runs: a few eager passes, one round of the gate/up "
                         "launches, then a plain 512 MiB device copy as the counter scale "
                         "reference; prints what ran, no benchmark line")
    args = ap.parse_args()
    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) != 1:
        print("bench.py measures one GPU only: the drafter pass runs on a single MI355X "
              "(multi-GPU sharding is a design note, not built).", file=sys.stderr)
        sys.exit(2)

    import numpy as np
    import torch
    from fe_synth import NAMED, make_inputs, make_weights
    from paper_2509_20416_amd import Drafter, fe

    cfg = NAMED[args.workload]
    t0 = time.time()
    w = device_weights(cfg, args.seed, "cuda") if args.device_weights else make_weights(cfg, args.seed)
    inp = make_inputs(cfg, args.seed)
    log(f"{cfg.name}: inputs generated in {time.time() - t0:.1f}s")
    plens = np.asarray(inp.prefix_lens)
    probe = args.traffic_probe or args.counter_probe
    dr = Drafter(cfg, w, max_batch=cfg.batch, max_prefix=int(plens.max()), graph=not (args.eager or probe))
    if args.pass_mode is not None:
        dr.set_pass_mode(args.pass_mode)
    di = dr.upload_inputs(inp)
    out = dr.alloc_outputs(cfg.batch, cfg.topk, draft=False)
    tree = dr.alloc_tree(cfg.batch, cfg.topk)

    def step():  # one pass: forward + tree, one graph replay
        dr.forward(di, out=out, tree=tree)

    if args.traffic_probe:
        for _ in range(3):
            step()
        torch.cuda.synchronize()
        _, per_pass = fe.fe_time_stage(dr.handle, fe.FE_STAGE["gateup"], 1, dr.stream())
        copy_bytes = 512 << 20
        src = torch.ones(copy_bytes // 4, dtype=torch.float32, device="cuda")
        dst = torch.empty_like(src)
        torch.cuda.synchronize()
        dst.copy_(src)
        torch.cuda.synchronize()
        print(json.dumps({"traffic_probe": cfg.name, "gateup_launches": per_pass,
                          "gateup_algorithmic_bytes": gateup_bytes(cfg, cfg.batch),
                          "copy_bytes_read": copy_bytes, "copy_bytes_written": copy_bytes}),
              flush=True)
        dr.close()
        return
    if args.counter_probe:
        # segments: [pass][fill][pass][fill][update][fill][update][fill][copy]
        marker = torch.zeros(1, device=dr.device)
        P = int(plens.max())
        for i in range(2):
            step()
            marker.fill_(float(i + 1))
        upd_pos = np.arange(P)
        for i in range(2):
            time_kv_update(dr, cfg, upd_pos, reps=1, warmup=0)
            marker.fill_(float(i + 3))
        torch.cuda.synchronize()
        copy_bytes = 512 << 20
        src = torch.ones(copy_bytes // 4, dtype=torch.float32, device="cuda")
        dst = torch.empty_like(src)
        torch.cuda.synchronize()
        dst.copy_(src)
        torch.cuda.synchronize()
        uflops, ubytes = kv_update_cost(cfg, P)
        print(json.dumps({"counter_probe": cfg.name, "passes": 2, "pass_bytes": pass_bytes(cfg, plens),
                          "pass_flops": pass_flops(cfg, plens), "kv_update_rows": P,
                          "kv_update_calls": 2, "kv_update_flops": uflops,
                          "kv_update_bytes": ubytes, "copy_bytes": copy_bytes}), flush=True)
        dr.close()
        return
    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()
    log("warmup done")
    stream = torch.cuda.current_stream()
    ev0, ev1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    ev0.record(stream)
    for _ in range(args.steps):
        step()
    ev1.record(stream)
    torch.cuda.synchronize()
    ms = ev0.elapsed_time(ev1) / args.steps
    # Dominant kernel: the gate/up + SwiGLU launches of the last timed pass
    # (one per cascade layer, each its own weights) replayed back to back on
    # the same stream between two HIP events; mean duration per launch.
    gu_avg, per_pass = fe.fe_time_stage(dr.handle, fe.FE_STAGE["gateup"], args.prof_repeats,
                                        dr.stream())
    n_timed = per_pass * args.prof_repeats
    log(f"{ms * 1000:.1f} us/pass; gate/up: {n_timed} launches, mean {gu_avg * 1000:.1f} us")

    # NEXT-2, greedy acceptance of the cycle's tree (after verification, not
    # part of the drafting pass): target predictions that follow the backbone
    # for half the levels; mean launch time over back-to-back calls
    T = 1 + cfg.n_layers * cfg.topk
    tok = tree["tokens"].cpu().numpy()
    nx = np.full((cfg.batch, T), -7, np.int32)
    for b in range(cfg.batch):
        cur = 0
        for lvl in range(cfg.n_layers // 2):
            child = 1 + lvl * cfg.topk          # rank-0 node of the level: the backbone
            nx[b, cur] = tok[b, child]
            cur = child
    nx_d = torch.from_numpy(nx).cuda()
    acc = dr.accept_greedy(tree, nx_d, cfg.topk)
    torch.cuda.synchronize()
    accept_len0 = int(acc["accept_len"][0].item())
    ev0.record(stream)
    for _ in range(100):
        dr.accept_greedy(tree, nx_d, cfg.topk, out=acc)
    ev1.record(stream)
    torch.cuda.synchronize()
    accept_us = ev0.elapsed_time(ev1) * 1000.0 / 100

    # NEXT-3, stochastic drafting at T = 1: the same pass with k candidates
    # sampled without replacement (uniforms resident on the device), graph replays
    from fe_synth import make_uniforms
    ud = torch.from_numpy(make_uniforms((cfg.batch, cfg.n_layers, cfg.draft_vocab),
                                        seed=args.seed + 1)).to(dr.device)
    dr.forward(di, out=out, tree=tree, temperature=1.0, uniforms=ud)
    torch.cuda.synchronize()
    ev0.record(stream)
    for _ in range(args.steps):
        dr.forward(di, out=out, tree=tree, temperature=1.0, uniforms=ud)
    ev1.record(stream)
    torch.cuda.synchronize()
    sms = ev0.elapsed_time(ev1) / args.steps
    log(f"sampled drafting: {sms * 1000:.1f} us/pass")
    # ... and with the uniforms drawn inside the pass (counter-based stream,
    # (seed, offset) in device memory, a new offset per pass)
    so = torch.tensor([args.seed + 1, 0], dtype=torch.int64, device=dr.device)
    dr.forward(di, out=out, tree=tree, temperature=1.0, seed_offset=so)
    torch.cuda.synchronize()
    seeded = []
    for advance in (False, True):   # replays as they are; then a new offset per pass
        ev0.record(stream)
        for i in range(args.steps):
            if advance:
                so[1:].fill_(i)
            dr.forward(di, out=out, tree=tree, temperature=1.0, seed_offset=so)
        ev1.record(stream)
        torch.cuda.synchronize()
        seeded.append(ev0.elapsed_time(ev1) / args.steps)
    seeded_ms = seeded[0]
    log(f"seeded sampled drafting: {seeded[0] * 1000:.1f} us/pass, "
        f"{seeded[1] * 1000:.1f} with the offset advanced per pass")
    # ... and its speculative-sampling acceptance against synthetic target
    # distributions over the target vocabulary (one per tree node)
    sout = dr.alloc_outputs(cfg.batch, cfg.topk, logits=True)
    stree = dr.alloc_tree(cfg.batch, cfg.topk)
    dr.forward(di, out=sout, tree=stree, temperature=1.0, uniforms=ud)
    gen = torch.Generator(device=dr.device).manual_seed(args.seed)
    tprobs = torch.rand((cfg.batch, 1 + cfg.n_layers * cfg.topk, cfg.target_vocab),
                        generator=gen, device=dr.device)
    tprobs /= tprobs.sum(-1, keepdim=True)
    ua = torch.rand((cfg.batch, cfg.n_layers * cfg.topk + 1), generator=gen,
                    device=dr.device).clamp_(2.0 ** -24, 1 - 2.0 ** -24)
    acc_s = dr.accept_sample(stree, sout["topk_draft"], sout["logits"], tprobs, ua,
                             temperature=1.0, draft_uniforms=ud)
    torch.cuda.synchronize()
    ev0.record(stream)
    for _ in range(50):
        dr.accept_sample(stree, sout["topk_draft"], sout["logits"], tprobs, ua, temperature=1.0,
                         draft_uniforms=ud, out=acc_s)
    ev1.record(stream)
    torch.cuda.synchronize()
    accept_s_us = ev0.elapsed_time(ev1) * 1000.0 / 50

    # NEXT-1, the drafter cache update: one cycle's N+1 verified positions,
    # and a whole prefix of max_prefix positions (the prompt's cache, the
    # shape where the update becomes matrix-core bound)
    P = int(plens.max())
    upd_cycle = time_kv_update(dr, cfg, np.arange(max(0, P - cfg.n_layers - 1), P))
    upd_prefill = time_kv_update(dr, cfg, np.arange(P), reps=10)
    # ... and under the self context, where the update is a prefill of the N
    # layers over the rows (same weights, a drafter of its own)
    sdr = Drafter(cfg.with_(cascade_ctx="self"), w, max_batch=cfg.batch, max_prefix=P,
                  max_topk=cfg.topk)
    upd_self_cycle = time_kv_update(sdr, sdr.cfg, np.arange(max(0, P - cfg.n_layers - 1), P))
    upd_self_prefill = time_kv_update(sdr, sdr.cfg, np.arange(P), reps=5, warmup=1)
    sdr.close()
    log(f"self-context update: {upd_self_cycle['us_per_call']:.1f} us cycle, "
        f"{upd_self_prefill['us_per_call']:.1f} us for {P} rows")
    log(f"kv update: {upd_cycle['rows']} rows {upd_cycle['us_per_call']:.1f} us, "
        f"{upd_prefill['rows']} rows {upd_prefill['us_per_call']:.1f} us "
        f"({upd_prefill['mfma_frac'] * 100:.1f}% of the MFMA peak)")

    B = cfg.batch
    gbytes = gateup_bytes(cfg, B)
    achieved = gbytes / (gu_avg * 1e-3) / 1e9
    traffic = read_traffic()
    pass_traffic = read_pass_traffic(cfg.name)
    ctr = read_mfma_counters(cfg.name)
    if ctr is not None:
        upd_prefill["counter"] = counter_update(ctr, upd_prefill, MFMA_PEAK_TFS[cfg.dtype])
    pbytes = pass_bytes(cfg, plens)
    pflops = pass_flops(cfg, plens)
    res = {
        "metric": METRIC,
        "value": B * 1000.0 / ms,
        "unit": "drafts/s",
        "n_gpus": 1, "steps": args.steps, "warmup": args.warmup,
        "ms_per_step": ms,
        "us_per_pass": ms * 1000.0,
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None,
        "dtype": cfg.dtype, "data": "synthetic (seeded N(0,0.02) weights, N(0,1) features and KV)",
        "config": {"workload": cfg.name, "batch": B, "hidden": cfg.hidden,
                   "q_heads": cfg.n_q_heads, "kv_heads": cfg.n_kv_heads,
                   "head_dim": cfg.head_dim, "intermediate": cfg.intermediate,
                   "cascade_layers": cfg.n_layers, "draft_vocab": cfg.draft_vocab,
                   "target_vocab": cfg.target_vocab, "prefix": cfg.prefix, "topk": cfg.topk,
                   "tree_nodes": cfg.tree_nodes, "cascade_ctx": cfg.cascade_ctx,
                   "graph": not args.eager,
                   "pass_launches": "persistent" if args.pass_mode == 0 else "one per stage"},
        # the whole pass as the unit: every weight and each layer's prefix K/V
        # once, over the time of one graph replay (all of its launches)
        "roofline": {"kernel": "whole drafting pass (one graph replay)",
                     "bound": "hbm", "achieved": pbytes / (ms * 1e-3) / 1e9,
                     "peak": HBM_PEAK_GBS, "unit": "GB/s",
                     "frac": pbytes / (ms * 1e-3) / 1e9 / HBM_PEAK_GBS,
                     "traffic": pass_traffic, "bytes_per_pass": pbytes,
                     "avg_pass_ms": ms},
        # the dominant kernel alone
        "roofline_dominant_kernel": {
            "kernel": "gate/up projections + SwiGLU (one per cascade layer)",
            "bound": "hbm", "achieved": achieved, "peak": HBM_PEAK_GBS,
            "unit": "GB/s", "frac": achieved / HBM_PEAK_GBS,
            "traffic": traffic, "bytes_per_launch": gbytes,
            "avg_launch_ms": gu_avg, "launches_timed": n_timed},
        # host-issued launches back to back: the rate is bound by the Python
        # call, the kernel itself is a few microseconds
        "next_accept_greedy": {"us_per_call": accept_us, "batch": B,
                               "accept_len_seq0": accept_len0, "issue": "eager, from Python"},
        "next_kv_update": {"cycle": upd_cycle, "prefill": upd_prefill,
                           "self_context": {"cycle": upd_self_cycle, "prefill": upd_self_prefill}},
        "next_sampled_drafting": {"temperature": 1.0, "steps": args.steps,
                                  "us_per_pass": sms * 1000.0,
                                  "drafts_per_s": cfg.batch * 1000.0 / sms,
                                  "uniform_bytes": cfg.batch * cfg.n_layers * cfg.draft_vocab * 4,
                                  "vs_greedy": ms / sms,
                                  "seeded_us_per_pass": seeded_ms * 1000.0,
                                  "seeded_advancing_us_per_pass": seeded[1] * 1000.0,
                                  "seeded_note": "uniforms drawn in the pass (Philox4x64-10); "
                                                 "advancing: one torch fill launch per pass "
                                                 "writes the next offset",
                                  "accept_sample_us_per_call": accept_s_us,
                                  "accept_sample_issue": "eager, from Python"},
        # matrix-core use over the whole pass, against the most that an
        # HBM-bound pass of this arithmetic intensity could reach
        "pass_mfma": {"flops_per_pass": pflops,
                      "achieved_TFLOPs": pflops / (ms * 1e-3) / 1e12,
                      "peak_TFLOPs": MFMA_PEAK_TFS[cfg.dtype],
                      "frac": pflops / (ms * 1e-3) / 1e12 / MFMA_PEAK_TFS[cfg.dtype],
                      "ceiling_frac": min(1.0, pflops / pbytes * HBM_PEAK_GBS / 1e3
                                          / MFMA_PEAK_TFS[cfg.dtype]),
                      # FLOPs the matrix cores executed (padding included), counted
                      "counter": counter_mfma(ctr, ms, MFMA_PEAK_TFS[cfg.dtype])},
    }
    dr.close()
    # NEXT-4, the ablation without the cascade: every layer reads x_0 (same
    # weights, same bytes), timed like the primary pass
    if cfg.cascade_ctx == "cascade":
        pcfg = cfg.with_(cascade_ctx="parallel")
        pdr = Drafter(pcfg, w, max_batch=cfg.batch, max_prefix=int(plens.max()),
                      graph=not args.eager)
        pdi = pdr.upload_inputs(inp)
        pout = pdr.alloc_outputs(cfg.batch, cfg.topk, draft=False)
        ptree = pdr.alloc_tree(cfg.batch, cfg.topk)
        for _ in range(max(3, args.warmup // 4)):
            pdr.forward(pdi, out=pout, tree=ptree)
        torch.cuda.synchronize()
        psteps = max(10, args.steps // 2)
        ev0.record(stream)
        for _ in range(psteps):
            pdr.forward(pdi, out=pout, tree=ptree)
        ev1.record(stream)
        torch.cuda.synchronize()
        pms = ev0.elapsed_time(ev1) / psteps
        pdr.close()
        log(f"parallel heads: {pms * 1000:.1f} us/pass")
        res["next_parallel_heads"] = {
            "workload": cfg.name, "cascade_ctx": "parallel", "steps": psteps,
            "us_per_pass": pms * 1000.0, "drafts_per_s": B * 1000.0 / pms,
            "bytes_per_pass": pass_bytes(pcfg, plens),
            "hbm_frac": pass_bytes(pcfg, plens) / (pms * 1e-3) / 1e9 / HBM_PEAK_GBS,
            "vs_cascade": ms / pms}
    if args.second and args.second != cfg.name:
        res["second_workload"] = time_second(args.second, args.seed, max(10, args.steps // 4),
                                             max(3, args.warmup // 4))
    if args.configs:
        res["other_configs"] = {}
        for name in [n for n in args.configs.split(",") if n and n != cfg.name]:
            res["other_configs"][name] = time_config(name, args.seed, max(20, args.steps // 2),
                                                     max(3, args.warmup // 4), args.pass_mode)
    if not (args.no_cpu_baseline or args.device_weights):
        log("timing the oracle on the host cores ...")
        res["cpu_baseline"] = cpu_baseline(cfg, w, inp, args.cpu_budget)
    print(json.dumps(res), flush=True)


if __name__ == "__main__":
    main()
