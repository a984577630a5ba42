"""Throughput of batched VLA rollout inference on one MI355X.

A step is one environment step of VLA-RL's rollout phase for a batch of
environments: prefill of [256 visual embeddings ; prompt] through the
OpenVLA-7B-shaped decoder, then the KV-cached decode of the 7 action tokens
with Gumbel-max sampling over the 256 action bins and per-token log-probs.
Inputs are synthetic and seeded (random-init bf16 weights, N(0,1) visual
embeddings, uniform prompt ids, ragged prompt lengths), resident in HBM
before the timed region.  The teacher-forced log-prob pass is timed in the
same run and reported beside the step.

Prints ONE JSON line.  `roofline` is the prefill GEMM (the dominant kernel),
measured with HIP events on the launch stream during the timed steps;
`roofline_decode` the decode GEMM, measured on a separate profiled decode.
"""
import argparse
import json
import os
import re
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

PEAK_BF16_TFLOPS = 2500.0   # MI355X dense bf16 MFMA
PEAK_HBM_GBS = 8000.0       # MI355X HBM3E


# Fields of the printed line and their types; `check_line` rejects a line that
# lacks one or whose headline figures are not numbers.
LINE_FIELDS = {"metric": str, "value": float, "unit": str, "n_gpus": int, "steps": int, "warmup": int,
               "ms_per_step": float, "higher_is_better": bool, "scaling": str, "dtype": str, "data": str,
               "config": dict, "roofline": dict}
ROOFLINE_FIELDS = {"bound": str, "achieved": float, "peak": float, "unit": str, "frac": float}


def pass_flops(d, F, L, Lb, n_out):
    """Algorithmic flops of one forward pass over sequences of Lb rows: every
    layer's QKV projection and every layer but the last over all rows; the last
    layer's attention, O projection and MLP over the n_out rows per sequence
    whose output is read (the last prefix row, or the scoring rows)."""
    Lb = np.asarray(Lb, dtype=np.float64)
    rows = Lb.sum()
    last = np.concatenate([np.arange(lb - n_out, lb) for lb in Lb.astype(np.int64)]).astype(np.float64)
    gemm = 2 * 3 * d * d * L * rows + 2 * (d * d + 3 * d * F) * ((L - 1) * rows + n_out * len(Lb))
    attn = 2 * d * (L - 1) * (Lb * (Lb + 1)).sum() + 4 * d * (last + 1).sum()
    return gemm + attn


def check_line(result):
    for key, t in LINE_FIELDS.items():
        if not isinstance(result.get(key), t) or (t is not bool and isinstance(result.get(key), bool)):
            raise ValueError(f"bench line field {key!r} must be {t.__name__}, got {result.get(key)!r:.80}")
    for key, t in ROOFLINE_FIELDS.items():
        if not isinstance(result["roofline"].get(key), t):
            raise ValueError(f"roofline field {key!r} must be {t.__name__}")
    if "cpu_baseline" in result and not isinstance(result["cpu_baseline"].get("value"), float):
        raise ValueError("cpu_baseline value must be a number")
    if "workload" not in result["config"]:
        raise ValueError("config must name the workload")
    return result


# HBM traffic (rocprofv3 FETCH_SIZE / WRITE_SIZE, scaled by a plain streaming
# kernel of known size) is kept in a profile summary together with hashes of
# the kernel sources it was taken on; it is reported only while they match.
TRAFFIC_FILE = os.path.join(ROOT, "profiles", "hbm_traffic_openvla7b_b64.md")
TRAFFIC_SOURCES = {"prefill_gemm": ["gemm_prefill.hip", "common.h"],
                   "decode_gemm": ["gemm_decode.hip", "skinny_dev.h", "common.h"],
                   "decode_layer": ["decode_layer.hip", "skinny_dev.h", "common.h"]}
TRAFFIC_KERNELS = {"prefill_gemm": "gemm_bf16_kernel", "decode_gemm": "skinny_kernel",
                   "decode_layer": "decode_layer_kernel"}
CALIB_ELEMS = 1 << 28       # bf16 elements of the calibration kernel: reads and writes 512 MiB


def source_hash(names):
    import hashlib
    h = hashlib.sha256()
    for n in names:
        with open(os.path.join(ROOT, "paper_2505_18719_amd", "csrc", n), "rb") as f:
            h.update(f.read())
    return h.hexdigest()[:16]


def load_traffic():
    """Measured HBM bytes per launch for each kernel whose sources are unchanged."""
    try:
        text = open(TRAFFIC_FILE).read()
    except OSError:
        return {}
    m = re.search(r"^traffic_json: (\{.*\})$", text, re.M)
    if not m:
        return {}
    rec = json.loads(m.group(1))
    return {k: v["bytes_per_launch"] for k, v in rec.items()
            if k in TRAFFIC_SOURCES and v.get("source") == source_hash(TRAFFIC_SOURCES[k])}


def summarise_traffic(fetch_dir, write_dir):
    """Markdown summary of a FETCH_SIZE run and a WRITE_SIZE run (KiB per
    dispatch), each scaled by what the counter reads for the calibration
    kernel (torch.neg over CALIB_ELEMS bf16 elements)."""
    import csv
    import glob

    def per_dispatch(d, counter):
        rows = {}
        for path in glob.glob(os.path.join(d, "**", "*counter_collection.csv"), recursive=True):
            for r in csv.DictReader(open(path)):
                if r["Counter_Name"] == counter:
                    key = r["Dispatch_Id"]
                    name, val = rows.get(key, (r["Kernel_Name"], 0.0))
                    rows[key] = (name, val + float(r["Counter_Value"]))
        return list(rows.values())

    true_kib = CALIB_ELEMS * 2 / 1024.0
    out, rec = [], {}
    scale = {}
    for counter, d in (("FETCH_SIZE", fetch_dir), ("WRITE_SIZE", write_dir)):
        rows = per_dispatch(d, counter)
        calib = [v for n, v in rows if "neg" in n]
        if len(calib) != 1:
            raise SystemExit(f"expected one calibration dispatch in {d}, found {len(calib)}")
        scale[counter] = true_kib / calib[0]
        out.append(f"| {counter} | calibration kernel reads {calib[0]:.0f} KiB for {true_kib:.0f} KiB | "
                   f"scale {scale[counter]:.4f} |")
        for k, kname in TRAFFIC_KERNELS.items():
            vals = [v for n, v in rows if kname in n]
            rec.setdefault(k, {"launches": len(vals), "source": source_hash(TRAFFIC_SOURCES[k])})
            rec[k][counter] = float(np.mean(vals)) * scale[counter] * 1024.0 if vals else None
    lines = ["| counter | calibration | factor |", "|---|---|---|"] + out + ["",
             "| kernel | launches | fetch MB / launch | write MB / launch | HBM MB / launch |", "|---|---|---|---|---|"]
    for k, v in rec.items():
        if v["FETCH_SIZE"] is None or v["WRITE_SIZE"] is None:
            continue
        v["bytes_per_launch"] = v["FETCH_SIZE"] + v["WRITE_SIZE"]
        lines.append(f"| {TRAFFIC_KERNELS[k]} | {v['launches']} | {v['FETCH_SIZE'] / 1e6:.2f} | "
                     f"{v['WRITE_SIZE'] / 1e6:.2f} | {v['bytes_per_launch'] / 1e6:.2f} |")
    rec = {k: v for k, v in rec.items() if "bytes_per_launch" in v}
    lines += ["", "traffic_json: " + json.dumps(rec)]
    return "\n".join(lines)


def log(*a):
    print(*a, file=sys.stderr, flush=True)


def cpu_baseline(cfg, w, inp, layers, T):
    """The oracle on the host cores: one environment (the shortest prefix of
    the batch), prefill + 7-token KV-cached decode + log-probs over the first
    `layers` decoder layers, scaled to all layers."""
    import oracle
    from paper_2505_18719_amd import inputs as I
    try:
        from threadpoolctl import threadpool_info
        cores = max([p.get("num_threads", 0) for p in threadpool_info()] + [1])
    except Exception:  # pragma: no cover
        cores = os.cpu_count()
    b = int(np.argmin(inp.prompt_lens))
    sub = cfg.replace(n_layers=layers)
    wc = {k: w[k].cpu() for k in ("embed", "lm_head", "final_norm")}
    wc["layers"] = [{k: t.cpu() for k, t in w["layers"][l].items()} for l in range(layers)]
    W = oracle.as_weights(wc, sub, cache_layers=False)
    t0 = time.perf_counter()
    oracle.rollout(sub, W, inp.vis[b:b + 1].cpu(), inp.env_prompt(b), inp.prompt_lens[b:b + 1],
                   inp.gumbel[b:b + 1], T, mode="bf16")
    dt = time.perf_counter() - t0
    t_env = dt * cfg.n_layers / layers
    cpu = "unknown"
    try:
        for line in open("/proc/cpuinfo"):
            if line.startswith("model name"):
                cpu = line.split(":", 1)[1].strip()
                break
    except OSError:
        pass
    return {"value": 1.0 / t_env, "unit": "actions/s", "cores": int(cores), "kind": "oracle",
            "cpu": cpu, "extrapolated": True,
            "sample": f"1 environment (prefix {int(inp.prefix_lens[b])} tokens), prefill + 7-token decode + "
                      f"log-probs over {layers} of {cfg.n_layers} layers in {dt:.1f} s; the rate is extrapolated "
                      f"to all layers (x{cfg.n_layers / layers:g}: every layer does the same work)"}


def step_work(cfg, inp):
    """Algorithmic work of one rollout step on its own inputs: prefill flops
    (the GEMMs and causal attention actually run, plus the action head) and
    decode HBM bytes (every 7B weight once per decode pass, the action rows of
    the LM head, the KV cache read and appended, the embedding rows)."""
    d, F, L, B = cfg.d_model, cfg.d_ffn, cfg.n_layers, inp.batch
    layer_params = 4 * d * d + 3 * d * F
    Lb = inp.prefix_lens.astype(np.float64)
    flops = pass_flops(d, F, L, Lb, 1) + 2 * d * cfg.action_bins * B
    nbytes = 0.0
    for t in range(1, cfg.n_actions):
        nbytes += 2 * layer_params * L + 2 * cfg.action_bins * d + 4 * d * L * (Lb + t).sum() + 2 * d * B
    return flops, nbytes


def measure_rollout(model, cfg, sets, steps, warmup, T, dev):
    """Rollout steps (vla_prefill + vla_decode_actions) over device-resident
    input sets, step k on sets[k % len(sets)]: `warmup` untimed steps, then
    `steps` timed ones between two synchronisations, with HIP events around
    each step's prefill and decode and the library's per-launch events on the
    prefill GEMM and attention; then one separately profiled decode (decode
    GEMM and attention launches), since events between the ~10^3 decode
    launches would perturb the timed region."""
    import torch
    B = sets[0][0].batch
    logits = torch.empty(B, cfg.action_bins, dtype=torch.float32, device=dev)
    out = {"tokens": torch.empty(B, cfg.n_actions, dtype=torch.int32, device=dev),
           "logp": torch.empty(B, cfg.n_actions, dtype=torch.float32, device=dev),
           "entropy": torch.empty(B, cfg.n_actions, dtype=torch.float32, device=dev)}
    stream = torch.cuda.current_stream(dev)
    n = len(sets)

    def step(k, ev=None):
        inp, ids, g = sets[k % n]
        if ev:
            ev[0].record(stream)
        model.prefill(inp.vis, ids, inp.prompt_lens, out=logits)
        if ev:
            ev[1].record(stream)
        model.decode_actions(g, T, batch=B, out=out)
        if ev:
            ev[2].record(stream)

    for k in range(warmup):
        step(k)
    torch.cuda.synchronize()
    evs = [[torch.cuda.Event(enable_timing=True) for _ in range(3)] for _ in range(steps)]
    model.profile_begin(("prefill_gemm", "prefill_attn"))
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for k in range(steps):
        step(warmup + k, evs[k])
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    prof = model.profile_end()
    inp0, ids0, g0 = sets[0]
    model.prefill(inp0.vis, ids0, inp0.prompt_lens, out=logits)
    model.profile_begin(("decode_gemm", "decode_attn", "decode_layer"))
    model.decode_actions(g0, T, batch=B, out=out)
    dprof = model.profile_end()
    flops = nbytes = 0.0
    for k in range(steps):
        f, b = step_work(cfg, sets[(warmup + k) % n][0])
        flops += f / steps
        nbytes += b / steps
    prefill_ms = float(np.mean([e[0].elapsed_time(e[1]) for e in evs]))
    decode_ms = float(np.mean([e[1].elapsed_time(e[2]) for e in evs]))
    pg = prof["prefill_gemm"]
    # the decode's weight-streaming kernel: the persistent layer kernel where it runs, else the projections
    layer = dprof["decode_layer"]["launches"] > 0
    dg = dprof["decode_layer"] if layer else dprof["decode_gemm"]
    g_tflops = pg["work"] / (pg["ms"] * 1e-3) / 1e12
    dg_gbs = dg["work"] / (dg["ms"] * 1e-3) / 1e9
    return {
        "ms_per_step": wall * 1e3 / steps, "prefill_ms": prefill_ms, "decode_ms": decode_ms,
        "prefill_mfma_frac": flops / (prefill_ms * 1e-3) / 1e12 / PEAK_BF16_TFLOPS,
        "decode_hbm_gbs": nbytes / (decode_ms * 1e-3) / 1e9,
        "decode_hbm_frac": nbytes / (decode_ms * 1e-3) / 1e9 / PEAK_HBM_GBS,
        "roofline": {"kernel": "gemm_bf16_kernel (prefill QKV/O/gate-up/down)", "bound": "mfma",
                     "achieved": g_tflops, "peak": PEAK_BF16_TFLOPS, "unit": "TFLOP/s",
                     "frac": g_tflops / PEAK_BF16_TFLOPS, "avg_launch_ms": pg["ms"] / max(pg["launches"], 1),
                     "launches": pg["launches"]},
        "roofline_decode": {"kernel": ("decode_layer_kernel (per layer and step: O, gate/up, down and the next QKV "
                                       "projection with their norms, one persistent launch)") if layer else
                                      "skinny_kernel (decode QKV/O/gate-up/down)", "bound": "hbm", "key": ("decode_layer" if layer else "decode_gemm"),
                            "achieved": dg_gbs, "peak": PEAK_HBM_GBS, "unit": "GB/s",
                            "frac": dg_gbs / PEAK_HBM_GBS, "avg_launch_ms": dg["ms"] / max(dg["launches"], 1),
                            "launches": dg["launches"]},
        "prof": prof, "dprof": dprof,
    }


def teacher_forced_pass(model, cfg, inp, ids, acts, T, dev, reps=2):
    """Mean time of `reps` teacher-forced passes (vla_token_logprobs) after an untimed one."""
    import torch
    stream = torch.cuda.current_stream(dev)
    model.token_logprobs(inp.vis, ids, inp.prompt_lens, acts, T)
    torch.cuda.synchronize()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record(stream)
    for _ in range(reps):
        model.token_logprobs(inp.vis, ids, inp.prompt_lens, acts, T)
    e1.record(stream)
    torch.cuda.synchronize()
    tf_ms = e0.elapsed_time(e1) / reps
    d, F, L, B = cfg.d_model, cfg.d_ffn, cfg.n_layers, inp.batch
    Lb = inp.prefix_lens.astype(np.float64) + cfg.n_actions
    tf_flops = pass_flops(d, F, L, Lb, cfg.n_actions) + 2 * d * cfg.action_bins * B * cfg.n_actions
    return {"ms": tf_ms, "rows": int(Lb.sum()),
            "mfma_frac": tf_flops / (tf_ms * 1e-3) / 1e12 / PEAK_BF16_TFLOPS,
            "log_probs_per_s": B * cfg.n_actions / (tf_ms * 1e-3)}


def secondary_configs(model, w, T, dev, steps):
    """The other 7B-shape workloads, on the same handle and weights:
    batch 8 (prompt 32) rollout steps, and the PPO-update workload at batch
    128: a 10-step rollout loop in which every environment keeps its 32-token
    prompt and sees fresh visual embeddings each step (the KV cache is rebuilt
    every step), then a teacher-forced pass over 128 x 295 rows."""
    import torch
    from paper_2505_18719_amd import inputs as I
    res = {}
    cfg = I.L7B_B8
    sets = []
    for k in range(4):
        inp = I.make_inputs(cfg, seed=0, step=k, device=dev)
        sets.append((inp, torch.from_numpy(inp.prompt_ids).to(dev), torch.from_numpy(inp.gumbel).to(dev)))
    r = measure_rollout(model, cfg, sets, max(steps, 10), 3, T, dev)
    res[cfg.name] = {"actions_per_s": cfg.batch / (r["ms_per_step"] * 1e-3),
                     **{k: v for k, v in r.items() if k not in ("prof", "dprof")}}
    log(f"[bench] {cfg.name}: {r['ms_per_step']:.2f} ms/step (prefill {r['prefill_ms']:.2f}, "
        f"decode {r['decode_ms']:.2f})")
    cfg = I.L7B_B128
    base = I.make_inputs(cfg, seed=0, step=0, device=dev)
    ids = torch.from_numpy(base.prompt_ids).to(dev)
    sets = []
    for k in range(10):
        vis = base.vis if k == 0 else I.make_inputs(cfg, seed=0, step=k, device=dev).vis
        inp = I.RolloutInputs(vis=vis, prompt_lens=base.prompt_lens, prompt_ids=base.prompt_ids,
                              gumbel=I.gumbel_noise(cfg, cfg.batch, seed=0, step=k))
        sets.append((inp, ids, torch.from_numpy(inp.gumbel).to(dev)))
    r = measure_rollout(model, cfg, sets, 10, 1, T, dev)
    acts = torch.from_numpy(I.stored_actions(cfg, cfg.batch, seed=0)).to(dev)
    tf = teacher_forced_pass(model, cfg, base, ids, acts, T, dev)
    res[cfg.name] = {"rollout_loop_steps": 10, "actions_per_s": cfg.batch / (r["ms_per_step"] * 1e-3),
                     **{k: v for k, v in r.items() if k not in ("prof", "dprof")}, "teacher_forced": tf}
    log(f"[bench] {cfg.name}: rollout loop {r['ms_per_step']:.2f} ms/step (prefill {r['prefill_ms']:.2f}, "
        f"decode {r['decode_ms']:.2f}); teacher-forced pass over {tf['rows']} rows {tf['ms']:.2f} ms")
    return res


def main():
    ap = argparse.ArgumentParser(description=__doc__.split("\n")[0])
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=5)
    ap.add_argument("--warmup", type=int, default=2)
    ap.add_argument("--config", default="openvla7b_b64_ragged")
    ap.add_argument("--temperature", type=float, default=1.5)
    ap.add_argument("--cpu-layers", type=int, default=8, help="decoder layers in the oracle's timed sample")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-teacher-forced", action="store_true")
    ap.add_argument("--no-configs", action="store_true", help="skip the batch-8 and batch-128 7B workloads")
    ap.add_argument("--no-value", action="store_true")
    ap.add_argument("--no-learning", action="store_true")
    ap.add_argument("--no-lora-merge", action="store_true")
    ap.add_argument("--no-backward", action="store_true")
    ap.add_argument("--copy-calibration", action="store_true",
                    help="run one plain streaming kernel of known size before timing (HBM counter calibration)")
    ap.add_argument("--traffic-from", nargs=2, metavar=("FETCH_DIR", "WRITE_DIR"),
                    help="summarise two rocprofv3 --pmc runs (FETCH_SIZE, WRITE_SIZE) as markdown and exit")
    args = ap.parse_args()
    if args.traffic_from:
        print(summarise_traffic(*args.traffic_from))
        return
    world = int(os.environ.get("WORLD_SIZE", "1"))
    if args.gpus != 1 or world != 1:
        print("bench.py: the library runs on one GPU only (no multi-GPU path); use --gpus 1", file=sys.stderr)
        sys.exit(2)

    import torch
    from paper_2505_18719_amd import inputs as I
    from paper_2505_18719_amd.vla import VlaModel

    cfg = I.PRESETS[args.config]
    B, T = cfg.batch, args.temperature
    torch.cuda.set_device(0)
    dev = torch.device("cuda:0")
    log(f"[bench] {cfg.name}: building weights and inputs")
    w = I.make_weights(cfg, seed=0, device=dev)
    # one handle serves every 7B-shape workload (batch 8, 64 and 128; sequences up to 311 rows)
    model = VlaModel(cfg, w, max_batch=max(B, 128), max_seq=max(cfg.max_seq, I.L7B_B64.max_seq), device=dev)
    n_sets = max(1, min(args.steps + args.warmup, 4))
    sets = []
    for k in range(n_sets):
        inp = I.make_inputs(cfg, seed=0, step=k, device=dev)
        sets.append((inp, torch.from_numpy(inp.prompt_ids).to(dev), torch.from_numpy(inp.gumbel).to(dev)))
    stream = torch.cuda.current_stream(dev)
    if args.copy_calibration:
        src = torch.ones(CALIB_ELEMS, dtype=torch.bfloat16, device=dev)
        dst = torch.empty_like(src)
        torch.cuda.synchronize()
        torch.neg(src, out=dst)
        del src, dst
    log(f"[bench] timing {args.steps} steps after {args.warmup} warm-up steps")
    r = measure_rollout(model, cfg, sets, args.steps, args.warmup, T, dev)
    ms_per_step = r["ms_per_step"]
    log(f"[bench] {ms_per_step:.2f} ms/step (prefill {r['prefill_ms']:.2f} ms, decode {r['decode_ms']:.2f} ms)")
    d, F, L = cfg.d_model, cfg.d_ffn, cfg.n_layers
    layer_params = 4 * d * d + 3 * d * F
    traffic = load_traffic()
    prof, dprof = r["prof"], r["dprof"]
    pg, da, pa, dg = prof["prefill_gemm"], dprof["decode_attn"], prof["prefill_attn"], dprof["decode_gemm"]

    result = {
        "metric": "VLA actions/sec at 7B shape, batch 64; decode HBM GB/s; prefill MFMA util",
        "value": B / (ms_per_step * 1e-3),
        "unit": "actions/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": ms_per_step,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16",
        "data": "synthetic (seeded random-init bf16 weights ~N(0,0.02), N(0,1) visual embeddings, "
                "uniform prompt ids, supplied Gumbel noise)",
        "config": {"workload": f"{cfg.name}: OpenVLA-7B-shaped decoder (32 layers, d 4096, 32 heads, FFN 11008, "
                               f"vocab 32064), batch {B}, 256 visual + prompt U[{cfg.prompt_min},{cfg.prompt_max}] "
                               f"tokens, 7-token action decode with log-probs, T={T}",
                   "global_batch": B, "seq_len": int(cfg.n_visual + cfg.prompt_max + cfg.n_actions),
                   "parallelism": "single GPU"},
        "action_tokens_per_s": B * cfg.n_actions / (ms_per_step * 1e-3),
        "prefill_ms": r["prefill_ms"],
        "decode_ms": r["decode_ms"],
        "prefill_mfma_frac": r["prefill_mfma_frac"],
        "decode_hbm_gbs": r["decode_hbm_gbs"],
        "decode_hbm_frac": r["decode_hbm_frac"],
        "roofline": {**r["roofline"], "traffic": traffic.get("prefill_gemm")},
        "roofline_decode": {**r["roofline_decode"], "traffic": traffic.get(r["roofline_decode"]["key"])},
        "kernels": {"prefill_attn_tflops": pa["work"] / max(pa["ms"], 1e-9) / 1e9,
                    "prefill_attn_ms_per_step": pa["ms"] / args.steps,
                    "prefill_gemm_ms_per_step": pg["ms"] / args.steps,
                    "decode_attn_gbs": da["work"] / max(da["ms"], 1e-9) / 1e6,
                    "decode_attn_ms": da["ms"], "decode_gemm_ms": dg["ms"],
                    "decode_layer_ms": dprof["decode_layer"]["ms"]},
    }

    if not args.no_teacher_forced:
        inp, ids, _ = sets[0]
        acts = torch.from_numpy(I.stored_actions(cfg, B, seed=0)).to(dev)
        result["teacher_forced"] = teacher_forced_pass(model, cfg, inp, ids, acts, T, dev)

    if not args.no_configs:
        result["configs"] = secondary_configs(model, w, T, dev, args.steps)

    if not args.no_value:
        # value estimate of every environment's prefix (Alg. 1), a value model of
        # the policy's architecture: here the policy's trunk with a seeded head
        inp, ids, _ = sets[0]
        g = torch.Generator(device=dev)
        g.manual_seed(0)
        head = (torch.randn(d, generator=g, device=dev) * 0.02).to(torch.bfloat16)
        vals = model.value(inp.vis, ids, inp.prompt_lens, head)
        torch.cuda.synchronize()
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record(stream)
        for _ in range(2):
            model.value(inp.vis, ids, inp.prompt_lens, head, out=vals)
        e1.record(stream)
        torch.cuda.synchronize()
        v_ms = e0.elapsed_time(e1) / 2
        Lp = inp.prefix_lens.astype(np.float64)
        v_flops = pass_flops(d, F, L, Lp, 1) + 2 * d * B
        result["value_model"] = {"ms": v_ms, "rows": int(Lp.sum()),
                                 "mfma_frac": v_flops / (v_ms * 1e-3) / 1e12 / PEAK_BF16_TFLOPS,
                                 "values_per_s": B / (v_ms * 1e-3)}
        log(f"[bench] value pass over {B} prefixes: {v_ms:.2f} ms")

    if not args.no_learning:
        # learning-phase kernels (Alg. 1 after the rollout, Eq. 2): GAE over a
        # 512-step window of the 64 environments, PPO-clip and the logits
        # gradient over a minibatch of 128 stored actions (7 tokens, 256 bins)
        from paper_2505_18719_amd import vla as V
        Ng, Mg, nb = B, 512, 128
        r, vv, dd = (torch.from_numpy(x).to(dev) for x in I.rollout_window(Ng, Mg, seed=0))
        old, new, adv = (torch.from_numpy(x).to(dev) for x in I.ppo_minibatch(nb, cfg.n_actions, seed=0))
        zb = torch.randn(nb * cfg.n_actions, cfg.action_bins, device=dev)
        tb = torch.randint(cfg.action_begin, cfg.action_begin + cfg.action_bins, (nb * cfg.n_actions,),
                           device=dev, dtype=torch.int32)
        adv_o, ret_o = V.gae(r, vv, dd, 0.99, 0.95)
        st, gl = V.ppo_clip(new, old, adv, 0.2)
        dzb = V.logprob_backward(zb, tb, cfg.action_begin, T, gl.reshape(-1))
        reps = 50
        times = {}
        for name, fn in (("gae", lambda: V.gae(r, vv, dd, 0.99, 0.95, adv_o, ret_o)),
                         ("ppo_clip", lambda: V.ppo_clip(new, old, adv, 0.2, gl, st)),
                         ("logprob_backward", lambda: V.logprob_backward(zb, tb, cfg.action_begin, T,
                                                                         gl.reshape(-1), dzb))):
            torch.cuda.synchronize()
            e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            e0.record(stream)
            for _ in range(reps):
                fn()
            e1.record(stream)
            torch.cuda.synchronize()
            times[name] = e0.elapsed_time(e1) / reps * 1e3
        # action extraction f of Alg. 1 on the batch's 7 tokens per environment
        tok_e = torch.randint(cfg.action_begin, cfg.action_begin + cfg.action_bins, (B, cfg.n_actions),
                              device=dev, dtype=torch.int32)
        lo_e = torch.full((cfg.n_actions,), -1.0, device=dev)
        hi_e = torch.full((cfg.n_actions,), 1.0, device=dev)
        act_e = V.extract_actions(tok_e, cfg.action_begin, cfg.action_bins, lo_e, hi_e)
        torch.cuda.synchronize()
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record(stream)
        for _ in range(reps):
            V.extract_actions(tok_e, cfg.action_begin, cfg.action_bins, lo_e, hi_e, act_e)
        e1.record(stream)
        torch.cuda.synchronize()
        result["action_extraction"] = {"us": e0.elapsed_time(e1) / reps * 1e3, "environments": B,
                                       "dims": cfg.n_actions}
        gae_bytes = 4 * Mg * Ng + 4 * (Mg + 1) * Ng + (Mg + 1) * Ng + 8 * Mg * Ng
        result["learning"] = {"gae_us": times["gae"], "gae_envs": Ng, "gae_steps": Mg,
                              "gae_gbs": gae_bytes / (times["gae"] * 1e-6) / 1e9,
                              "ppo_clip_us": times["ppo_clip"], "ppo_actions": nb,
                              "logprob_backward_us": times["logprob_backward"],
                              "logprob_backward_rows": nb * cfg.n_actions}
        log(f"[bench] learning kernels (us): " + ", ".join(f"{k} {v:.1f}" for k, v in times.items()))

    if not args.no_lora_merge:
        # LoRA merge before a rollout (Sec. 3.3): every projection of every layer,
        # rank 32, from the original checkpoint; timed after the rollout figures
        rank = 32
        adapters = I.make_lora(cfg, rank, seed=0, device=dev)
        def merge_all():  # every projection of a layer in one launch (vla_lora_merge_layer)
            for li, ad in enumerate(adapters):
                model.lora_merge_layer(li, w["layers"][li], ad, 0.5)
        merge_all()
        torch.cuda.synchronize()
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record(stream)
        for _ in range(3):
            merge_all()
        e1.record(stream)
        torch.cuda.synchronize()
        merge_ms = e0.elapsed_time(e1) / 3
        Fp = (F + 255) // 256 * 256
        # algorithmic bytes: the original weights read, the packed weights written, the adapters read
        merge_bytes = L * 2.0 * (4 * d * d + 3 * d * F                # W0
                                 + 4 * d * d + 2 * Fp * d + d * Fp    # packed (gate/up rows and down columns padded to Fp)
                                 + rank * (4 * d + 2 * d + F)         # A factors [rank, in]
                                 + rank * (4 * d + 2 * F + d))        # B factors [out, rank]
        result["lora_merge"] = {"ms": merge_ms, "rank": rank, "projections": 7 * L, "launches": L,
                                "achieved": merge_bytes / (merge_ms * 1e-3) / 1e9, "peak": PEAK_HBM_GBS,
                                "unit": "GB/s", "frac": merge_bytes / (merge_ms * 1e-3) / 1e9 / PEAK_HBM_GBS,
                                "bytes": merge_bytes}
        log(f"[bench] LoRA merge of all {7 * L} projections: {merge_ms:.2f} ms")

    if not args.no_lora_merge and not args.no_backward:
        # PPO update gradient (Eq. 2 through the teacher-forced pass) w.r.t. the
        # rank-32 adapters just merged, over the same batch with stored actions
        inp, ids, _ = sets[0]
        acts = torch.from_numpy(I.stored_actions(cfg, B, seed=0)).to(dev)
        old = model.token_logprobs(inp.vis, ids, inp.prompt_lens, acts, T)["logp"].contiguous()
        adv_b = torch.from_numpy(I.ppo_minibatch(B, seed=0)[2]).to(dev)
        model.ppo_lora_grads(inp.vis, ids, inp.prompt_lens, acts, old, adv_b, 0.2, T, adapters, 0.5)
        torch.cuda.synchronize()
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record(stream)
        st_b, _, _ = model.ppo_lora_grads(inp.vis, ids, inp.prompt_lens, acts, old, adv_b, 0.2, T, adapters, 0.5)
        e1.record(stream)
        torch.cuda.synchronize()
        bwd_ms = e0.elapsed_time(e1)
        Lt = inp.prefix_lens.astype(np.float64) + cfg.n_actions
        # algorithmic work: the forward, the input gradients (the GEMMs' flops again;
        # dV, dP, dQ and dK of attention, twice its forward), and the four rank-32
        # products of each adapted projection (X A^T, dY B, dY^T T1, T2^T X); no
        # weight gradient is formed and the per-layer recompute is not counted
        fwd_gemm = 2 * layer_params * L * Lt.sum()
        fwd_attn = 2 * d * L * (Lt * (Lt + 1)).sum()
        lora_flops = 4 * Lt.sum() * 32 * (11 * d + 3 * F) * L
        work = 2 * fwd_gemm + 3 * fwd_attn + lora_flops
        result["lora_backward"] = {"ms": bwd_ms, "rows": int(Lt.sum()), "projections": 7 * L, "rank": 32,
                                   "mfma_frac": work / (bwd_ms * 1e-3) / 1e12 / PEAK_BF16_TFLOPS,
                                   "loss": float(st_b[0])}
        log(f"[bench] PPO LoRA gradient (teacher-forced pass + backward): {bwd_ms:.1f} ms")

    if not args.no_cpu_baseline:
        log(f"[bench] oracle CPU baseline ({args.cpu_layers} layers of one environment)")
        result["cpu_baseline"] = cpu_baseline(cfg, w, sets[0][0], args.cpu_layers, T)
    model.close()
    print(json.dumps(check_line(result)), flush=True)


if __name__ == "__main__":
    main()
