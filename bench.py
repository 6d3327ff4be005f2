"""Benchmark of the DraftAttention2 hot path on one MI355X.

One step = the four library calls (draft_map, rank_assign, prep_operands,
mixed_attn) over one attention layer of the mid video-DiT workload: B=1,
12 heads, d=128, latent grid 21x30x52 = 32,760 tokens, 8x8 tiles, budgets
10% 8-bit / 30% 4-bit / 60% skip, head-scope ranking, bf16 synthetic
Q/K/V already resident in HBM (--workload picks another configured layer).

Prints one JSON line. Times are medians over the timed steps, each step
run after a 512 MiB device write that evicts the 256 MB Infinity Cache and
timed with HIP events on the stream the calls run on; the warm (back to
back) numbers are reported beside them. ``value`` is the dense-equivalent
throughput of the whole step, 4*B*H*N^2*d flops per step; mixed_attn alone
is reported too. The roofline object covers mixed_attn, the dominant
kernel: algorithmic flops = retained tiles x 4*64*64*d, with a peak that
weights 8-bit tiles at the int8/fp8 peak and 4-bit tiles at the fp4 peak
(``frac``), and beside it at the peak of the MFMA the kernel issues for the
4-bit tiles (fp16 for NVFP4, ``frac_issued_dtype``). Its ``traffic`` is the
HBM bytes per launch that rocprofv3 counted for the same kernel source
(profiles/mixed_attn_traffic.json, FETCH_SIZE and WRITE_SIZE scaled by a
plain-copy calibration), or null when the source has changed since. The
``hbm`` object rates draft_map and prep_operands against HBM bandwidth with
the bytes each call must move: draft_map reads Q and K and writes A;
prep_operands reads Q, K and V (V twice: the per-channel scales come first)
and writes the operand sections the run uses.
"""
import argparse
import hashlib
import json
import os
import re
import sys
import time

from dataclasses import replace

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

PEAK_8BIT = 5.0e15      # MI355X dense int8 / fp8 MFMA (published)
PEAK_FP16 = 2.5e15      # MI355X dense fp16 / bf16 MFMA (published)
PEAK_FP4 = 10.1e15      # MI355X dense fp4 / fp6 MFMA (published)
PEAK_HBM = 8.0e12       # bytes/s
TRAFFIC = os.path.join(ROOT, "profiles", "mixed_attn_traffic.json")
ATTN_SOURCES = [os.path.join(ROOT, "paper_2609_32628_amd", "csrc", f) for f in ("attn.hip", "common.hpp", "launch.hpp")]


def attn_source_hash():
    """SHA-256 of the attention kernel's sources without comments and blank
    lines (a comment edit does not change the kernel)."""
    h = hashlib.sha256()
    for f in ATTN_SOURCES:
        with open(f) as fh:
            for line in fh:
                code = re.sub(r"//.*", "", line).strip()
                if code:
                    h.update(code.encode() + b"\n")
    return h.hexdigest()


def recorded_traffic(workload):
    """HBM bytes per mixed_attn launch recorded for this kernel source and
    workload, or None."""
    try:
        with open(TRAFFIC) as fh:
            rec = json.load(fh)
    except (OSError, ValueError):
        return None
    if rec.get("source_sha256") != attn_source_hash() or rec.get("workload") != workload:
        return None
    return rec.get("read_bytes", 0) + rec.get("write_bytes", 0)


# ---- operator error-vs-latency sweep (attention error analysis) -------------
# Precision mixes as percentages of the retained pairs on the (16, 8, 4)-bit
# paths, and the retained fractions swept at each mix (1.0 = no sparsity).
SWEEP_MIXES = {"4": (0, 0, 100), "8": (0, 100, 0), "16": (100, 0, 0),
               "8/16": (10, 90, 0), "4/8": (0, 25, 75), "4/8/16": (10, 30, 60)}
SWEEP_RETAINED = (0.05, 0.1, 0.2, 0.3, 0.5, 0.7, 1.0)
SWEEP_DEN = 1000


def sweep_points():
    """(lambda, mix, retained, fmt4) of every sweep point: all mixes with the
    max-pooled draft (lambda = 0.2), the 8-bit and 8/16 mixes also with average
    pooling alone (lambda = 0), and the mixes with a 4-bit share also with MXFP4."""
    pts = [(0.2, m, r, "nvfp4") for m in SWEEP_MIXES for r in SWEEP_RETAINED]
    pts += [(0.0, m, r, "nvfp4") for m in ("8", "8/16") for r in SWEEP_RETAINED]
    pts += [(0.2, m, r, "mxfp4") for m in ("4", "4/8", "4/8/16") for r in SWEEP_RETAINED]
    return pts


def sweep_budgets(mix, retained):
    """(num16, num8, num4) out of SWEEP_DEN for a mix at a retained fraction."""
    return tuple(int(retained * pct * SWEEP_DEN / 100 + 0.5) for pct in SWEEP_MIXES[mix])


def _sweep_head(h):
    from synth import configs, gen
    Q, K, V = gen.generate(configs.FIG4, heads=[h])
    return Q[0, 0], K[0, 0], V[0, 0]


def dense_rows(q, K, V):
    """Textbook softmax(q K^T / sqrt d) V in float64 for a few query rows: the
    dense output the error metric compares against."""
    S = q.astype(np.float64) @ K.astype(np.float64).T / np.sqrt(K.shape[1])
    P = np.exp(S - S.max(axis=1, keepdims=True))
    return (P / P.sum(axis=1, keepdims=True)) @ V.astype(np.float64)


def run_sweep(args):
    """Relative L2 error against dense attention versus the latency of the whole
    operator (draft map, ranking, operand preparation, attention), one JSON line
    per point. Latency: median of three timed steps after one warm-up. Error:
    over a seeded sample of query rows (8 heads x 64 tokens) whose dense output
    is computed in float64 on the host."""
    from multiprocessing import get_context

    from synth import configs
    w = configs.FIG4
    # inputs drawn head by head in worker processes, before the GPU is touched
    workers = min(16, os.cpu_count() or 1)
    heads = []
    with get_context("fork").Pool(workers) as pool:
        for i, hv in enumerate(pool.imap(_sweep_head, range(w.H))):
            heads.append(hv)
            if (i + 1) % 8 == 0:
                print(f"sweep inputs: {i + 1}/{w.H} heads", file=sys.stderr, flush=True)
    rng = np.random.default_rng(7)
    ref_heads = sorted(rng.choice(w.H, 8, replace=False))
    ref_rows = {h: np.sort(rng.choice(w.N, 64, replace=False)) for h in ref_heads}
    ref = {h: dense_rows(heads[h][0][ref_rows[h]], heads[h][1], heads[h][2]) for h in ref_heads}
    print("sweep dense reference rows ready", file=sys.stderr, flush=True)

    import torch

    from paper_2609_32628_amd import api
    dev = []
    for t in range(3):
        X = torch.empty((1, w.H, w.N, w.d), dtype=torch.bfloat16, device="cuda")
        for h in range(w.H):
            X[0, h].copy_(torch.from_numpy(heads[h][t]).to(torch.bfloat16))
        dev.append(X)
    del heads
    p = api.problem(w.B, w.H, w.d, w.T, w.Hg, w.Wg, w.partition)
    buf = api.alloc(p, "head", with16=True)
    # the operand buffer of each 4-bit encoding (sized for the 16-bit path too)
    ops_of = {"nvfp4": buf.ops,
              "mxfp4": torch.empty(api.da2_sizes(p, "head", "mxfp4", True)["ops_bytes"], dtype=torch.uint8,
                                   device="cuda")}
    O = torch.empty(dev[0].shape, dtype=torch.bfloat16, device="cuda")
    stream = torch.cuda.current_stream()
    idx_h = torch.tensor(ref_heads, device="cuda")
    for lam, mix, rho, fmt4 in sweep_points():
        n16, n8, n4 = sweep_budgets(mix, rho)

        def step(ev=None):
            api.da2_draft_map(dev[0], dev[1], buf.layout, p, lam, buf.A, buf.stats, buf.ws_draft)
            api.da2_rank_assign(buf.A, p, n16, n8, n4, SWEEP_DEN, "head", buf.cls, buf.lists, buf.ws_rank)
            api.da2_prep_operands(dev[0], dev[1], dev[2], buf.layout, p, int(n16 > 0), fmt4, buf.stats,
                                  ops_of[fmt4], None)
            if ev is not None:
                ev[0].record(stream)
            api.da2_mixed_attn(ops_of[fmt4], buf.lists, buf.layout, p, O, fmt4=fmt4)
            if ev is not None:
                ev[1].record(stream)

        step()
        torch.cuda.synchronize()
        total, attn = [], []
        for _ in range(3):
            e = [torch.cuda.Event(enable_timing=True) for _ in range(4)]
            e[0].record(stream)
            step(e[2:])
            e[1].record(stream)
            torch.cuda.synchronize()
            total.append(e[0].elapsed_time(e[1]))
            attn.append(e[2].elapsed_time(e[3]))
        Os = O[0].index_select(0, idx_h).float().cpu().numpy()
        num = den = 0.0
        for i, h in enumerate(ref_heads):
            diff = Os[i][ref_rows[h]].astype(np.float64) - ref[h]
            num += float((diff ** 2).sum())
            den += float((ref[h] ** 2).sum())
        cls = buf.cls
        rec = {"sweep": "operator error vs latency", "workload": w.name, "lambda": lam, "mix_16_8_4_pct": mix,
               "retained": rho, "fmt4": fmt4, "budgets_16_8_4_of_1000": [n16, n8, n4],
               "ms_median": float(np.median(total)), "mixed_attn_ms_median": float(np.median(attn)),
               "rel_l2_pct": 100.0 * float(np.sqrt(num / den)),
               "tiles": {str(c): int((cls == c).sum().item()) for c in (16, 8, 4)},
               "error_sample": f"{len(ref_heads)} heads x 64 query tokens"}
        print(json.dumps(rec), flush=True)


def parse():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--workload", default="mid-21x30x52-h12-d128")
    ap.add_argument("--partition", choices=("tiles8", "ragged"), default=None,
                    help="region partition (the configured workloads use 8x8 tiles)")
    ap.add_argument("--num16", type=int, default=None,
                    help="num16/den of the region pairs on the 16-bit path (the hot path uses 0)")
    ap.add_argument("--fmt4", choices=("nvfp4", "mxfp4"), default="nvfp4",
                    help="encoding of the 4-bit path: the paper's NVFP4 (default) or gfx950's native MXFP4")
    ap.add_argument("--sweep", action="store_true",
                    help="operator error-vs-latency sweep over sparsity, precision mixes and lambda on the "
                         "109,368-token x 56-head shape (one JSON line per point) instead of the benchmark")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--copy-calibration", action="store_true",
                    help="also run a plain 512 MiB device copy (HBM counter calibration)")
    return ap.parse_args()


def _cpu_model():
    """Model name of the host CPU (lscpu), for the baseline record."""
    try:
        import subprocess
        out = subprocess.run(["lscpu"], capture_output=True, text=True, timeout=10).stdout
        for line in out.splitlines():
            if line.startswith("Model name:"):
                return line.split(":", 1)[1].strip()
    except (OSError, ValueError, subprocess.SubprocessError):
        pass
    return "unknown"


def _oracle_head_task(task):
    """One oracle task (runs in a spawned worker on one BLAS thread): the
    head-level steps (draft map, ranking, encodings) of head h, then the
    attention of the query blocks in ``rows``. Returns the two times."""
    from threadpoolctl import threadpool_limits
    threadpool_limits(1)
    from oracle import attention, draft, encode, partition, rank
    from synth import configs, gen
    wd, h, rows = task
    w = configs.Workload(**wd)
    Q, K, V = gen.generate(w, heads=[h])
    q, k, v = Q[0, 0], K[0, 0], V[0, 0]
    slot2tok, n_a, _ = partition.make_partition(w.partition, w.T, w.Hg, w.Wg)
    t0 = time.perf_counter()
    A32, _ = draft.draft_head(q, k, slot2tok, n_a, w.lam)
    cls = rank.rank_head(A32, *w.budgets, w.scope, num16=w.num16)
    enc = encode.encode_head(q, k, v, slot2tok, n_a)
    ops = attention.Operands.quantized(encode.reconstruct(enc), n_a)
    t1 = time.perf_counter()
    for a in rows:
        attention.attend(ops, a, *rank.key_lists_all(cls[a]))
    t2 = time.perf_counter()
    return t1 - t0, t2 - t1


def cpu_baseline(w, rows_per_head=32):
    """The oracle as it stands, timed on the host's cores: a process pool
    (spawned workers, one BLAS thread each, one worker per core) runs, for
    every head, the head-level steps (draft map, ranking, encodings) and the
    attention of a seeded sample of query blocks. The whole job's time is
    extrapolated to every query block of every head and divided over the
    workers (the (head, block) tasks are independent)."""
    from dataclasses import asdict
    from multiprocessing import get_context

    from oracle import partition
    R = partition.make_partition(w.partition, w.T, w.Hg, w.Wg)[1].size
    cores = max(1, min(os.cpu_count() or 1, 64))
    rows = sorted(int(a) for a in np.random.default_rng(13).choice(R, min(rows_per_head, R), replace=False))
    tasks = [(asdict(w), h, rows) for h in range(w.H)]
    t0 = time.perf_counter()
    with get_context("spawn").Pool(min(cores, len(tasks))) as pool:
        res = pool.map_async(_oracle_head_task, tasks, chunksize=1).get(1200)
    wall = time.perf_counter() - t0
    fixed = sum(r[0] for r in res)
    per_row = sum(r[1] for r in res) / (len(res) * len(rows))
    cpu_job = w.B * (fixed + per_row * R * w.H)       # single-core seconds for the whole job
    t_job = cpu_job / cores
    flops = 4.0 * w.B * w.H * w.N ** 2 * w.d
    return {"value": flops / t_job / 1e12, "unit": "TFLOP/s (dense-equivalent)", "cores": cores,
            "kind": "oracle", "cpu_model": _cpu_model(),
            "seconds_measured_cpu": round(fixed + per_row * len(rows) * len(res), 1),
            "seconds_measured_wall": round(wall, 1),
            "seconds_job_extrapolated": round(t_job, 1),
            "sample": f"all {w.H} heads' draft map, ranking and encodings, and the attention of {len(rows)} seeded "
                      f"query blocks per head (of {R}); process pool of {cores} single-threaded workers; the whole "
                      f"job extrapolated to all query blocks and divided over the workers"}


def main():
    args = parse()
    if args.gpus != 1:
        print(f"bench.py runs on one GPU only (asked for --gpus {args.gpus}); "
              "the path shards by head with no exchange, so multi-GPU numbers are not produced.", file=sys.stderr)
        sys.exit(2)
    if args.sweep:
        run_sweep(args)
        return
    import torch

    from paper_2609_32628_amd import api
    from synth import configs, gen

    w = configs.BY_NAME[args.workload]
    if args.num16 is not None:
        w = replace(w, num16=args.num16)
    if args.partition is not None:
        w = replace(w, partition=args.partition)
    Q, K, V = gen.generate(w)
    dev = [torch.from_numpy(x).to(torch.bfloat16).cuda() for x in (Q, K, V)]
    p = api.problem(w.B, w.H, w.d, w.T, w.Hg, w.Wg, w.partition)
    buf = api.alloc(p, w.scope, fmt4=args.fmt4, with16=w.num16 > 0)
    O = torch.empty(dev[0].shape, dtype=torch.bfloat16, device="cuda")
    stream = torch.cuda.current_stream()
    torch.cuda.synchronize()

    stages = ("draft_map", "rank_assign", "prep_operands", "mixed_attn")

    def step(ev=None):
        calls = (lambda: api.da2_draft_map(dev[0], dev[1], buf.layout, p, w.lam, buf.A, buf.stats, buf.ws_draft),
                 lambda: api.da2_rank_assign(buf.A, p, w.num16, *w.budgets, w.scope, buf.cls, buf.lists, buf.ws_rank),
                 lambda: api.da2_prep_operands(dev[0], dev[1], dev[2], buf.layout, p, int(w.num16 > 0), args.fmt4,
                                               buf.stats, buf.ops, None),
                 lambda: api.da2_mixed_attn(buf.ops, buf.lists, buf.layout, p, O, fmt4=args.fmt4))
        for i, c in enumerate(calls):
            if ev is not None:
                ev[i][0].record(stream)
            c()
            if ev is not None:
                ev[i][1].record(stream)

    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()

    def ms_of(evs):
        return [[evs[s][i][0].elapsed_time(evs[s][i][1]) for i in range(len(stages))] for s in range(len(evs))]

    # Primary: K steps, each after a 512 MiB device write that evicts the
    # 256 MB Infinity Cache, each step and stage timed with HIP events on the
    # stream; the median over the K steps.
    scratch = torch.empty(512 << 20, dtype=torch.uint8, device="cuda")
    evs = [[[torch.cuda.Event(enable_timing=True) for _ in range(2)] for _ in stages] for _ in range(args.steps)]
    torch.cuda.synchronize()
    t_wall0 = time.perf_counter()
    for s_ in range(args.steps):
        scratch.fill_(s_ & 0xFF)
        step(evs[s_])
    torch.cuda.synchronize()
    wall_flushed = time.perf_counter() - t_wall0
    flushed = np.array(ms_of(evs))                      # [K, stages]
    step_flushed = flushed.sum(axis=1)
    # Beside it: K steps back to back without flushing (warm caches).
    evw = [[[torch.cuda.Event(enable_timing=True) for _ in range(2)] for _ in stages] for _ in range(args.steps)]
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record(stream)
    for s_ in range(args.steps):
        step(evw[s_])
    e1.record(stream)
    torch.cuda.synchronize()
    ms_step_warm_mean = e0.elapsed_time(e1) / args.steps
    warm = np.array(ms_of(evw))
    del scratch
    ms_step = float(np.median(step_flushed))
    stage_ms = {name: float(np.median(flushed[:, i])) for i, name in enumerate(stages)}
    stage_ms_warm = {name: float(np.median(warm[:, i])) for i, name in enumerate(stages)}
    cache_study = {"step_ms_flushed_median": ms_step, "step_ms_flushed_min": float(step_flushed.min()),
                   "step_ms_warm_median": float(np.median(warm.sum(axis=1))),
                   "step_ms_warm_back_to_back_mean": ms_step_warm_mean,
                   "stage_ms_warm_median": stage_ms_warm,
                   "wall_s_flushed_loop": wall_flushed,
                   "note": f"median over {args.steps} steps; flushed = a 512 MiB device write before each step "
                           "(outside the events), warm = steps back to back"}
    if args.copy_calibration:
        src = torch.empty(512 << 20, dtype=torch.uint8, device="cuda")
        dst = torch.empty_like(src)
        for _ in range(3):
            dst.copy_(src)
        torch.cuda.synchronize()

    counts = buf.cls.view(w.B * w.H, -1)
    n8 = int((counts == 8).sum().item())
    n4 = int((counts == 4).sum().item())
    n16 = int((counts == 16).sum().item())
    tile_flops = 4.0 * 64 * 64 * w.d
    F8, F4, F16 = n8 * tile_flops, n4 * tile_flops, n16 * tile_flops
    # flops of the retained tiles counted on valid tokens only (sum of 4 n_a n_b d)
    n_a = buf.layout[:buf.sizes["R"]].to(torch.float64)
    kept = (buf.cls.view(w.B * w.H, buf.sizes["R"], buf.sizes["R"]) != 0).to(torch.float64)
    valid_flops = float(4.0 * w.d * (kept * n_a[None, :, None] * n_a[None, None, :]).sum().item())
    # transcendental-issue floor: 64 x 64 exponentials per retained tile at one
    # v_exp_f32 wave instruction per 8 clocks per SIMD (the half rate measured
    # on gfx950 with independent chains), 256 CUs x 4 SIMDs x 64 lanes / 8 at 2.4 GHz
    exp_floor_ms = (n8 + n4 + n16) * 4096 / (256 * 4 * 64 / 8 * 2.4e9) * 1e3
    t_attn = stage_ms["mixed_attn"] * 1e-3
    # the roofline rates the average launch: the mean over the flushed steps
    t_attn_mean = float(flushed[:, stages.index("mixed_attn")].mean()) * 1e-3
    achieved = (F8 + F4 + F16) / t_attn_mean
    mx = args.fmt4 == "mxfp4"
    # budget-weighted peak: 8-bit tiles at the int8/fp8 peak, 4-bit tiles at
    # the fp4 peak (the 4-bit format's own MFMA rate), 16-bit tiles at fp16
    peak_eff = (F8 + F4 + F16) / (F8 / PEAK_8BIT + F4 / PEAK_FP4 + F16 / PEAK_FP16)
    # the same with 4-bit tiles at the peak of the dtype the kernel issues for
    # them (fp16 MFMA on the exact NVFP4 values, or the scaled fp4 MFMA)
    peak_issued = (F8 + F4 + F16) / (F8 / PEAK_8BIT + F4 / (PEAK_FP4 if mx else PEAK_FP16) + F16 / PEAK_FP16)
    dense_flops = 4.0 * w.B * w.H * w.N ** 2 * w.d
    # bytes each preparation call must move (bf16 inputs)
    sizes = buf.sizes
    e_in = w.B * w.H * w.N * w.d * 2
    draft_bytes = 2 * e_in + sizes["A_bytes"]
    # the ops buffer holds exactly the sections prep_operands writes: 8-bit
    # operands and scales, the 4-bit encoding in use, and the 16-bit operands
    # only when that path is on
    # reads: Q, K, V, and V once more for the per-channel E4M3 scales, which
    # must exist before any V block is encoded
    prep_bytes = 4 * e_in + sizes["ops_bytes"]
    t_draft, t_prep = stage_ms["draft_map"] * 1e-3, stage_ms["prep_operands"] * 1e-3
    hbm = {"draft_map": {"bytes": draft_bytes, "GB/s": draft_bytes / t_draft / 1e9,
                         "frac": draft_bytes / t_draft / PEAK_HBM},
           "prep_operands": {"bytes": prep_bytes, "GB/s": prep_bytes / t_prep / 1e9,
                             "frac": prep_bytes / t_prep / PEAK_HBM},
           "combined_frac": (draft_bytes + prep_bytes) / (t_draft + t_prep) / PEAK_HBM,
           "peak_GB/s": PEAK_HBM / 1e9}
    rec = {
        "metric": "mixed_attn ms + dense-equiv TFLOP/s @32760 tok×12 heads, % MFMA roofline",
        "value": dense_flops / (ms_step * 1e-3) / 1e12,
        "unit": "TFLOP/s (dense-equivalent, whole step)",
        "n_gpus": 1, "steps": args.steps, "warmup": args.warmup,
        "ms_per_step": ms_step,
        "ms_per_step_note": "median over the timed steps, each with the Infinity Cache flushed first",
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None,
        "dtype": ("mixed: int8/fp8 + scaled fp4 (mxfp4) MFMA" if mx else
                  "mixed: int8/fp8 + fp16(nvfp4-exact) MFMA") + ", fp32 softmax state; bf16 in/out",
        "data": "synthetic",
        "config": {"workload": w.name, "B": w.B, "heads": w.H, "tokens": w.N, "d": w.d,
                   "grid": [w.T, w.Hg, w.Wg], "budgets_8_4_skip": [w.budgets[0], w.budgets[1],
                                                                   w.budgets[2] - w.budgets[0] - w.budgets[1] - w.num16],
                   "scope": w.scope, "lambda": w.lam, "num16": w.num16, "partition": w.partition,
                   "fmt4": args.fmt4,
                   "parallelism": "single GPU"},
        "stage_ms": stage_ms,
        "mixed_attn_ms": stage_ms["mixed_attn"],
        "mixed_attn_dense_equiv_tflops": dense_flops / t_attn / 1e12,
        "tiles": {"8bit": n8, "4bit": n4, "16bit": n16},
        "valid_token_flops_frac": valid_flops / (F8 + F4 + F16) if (n8 + n4 + n16) else None,
        "mixed_attn_valid_token_tflops": valid_flops / t_attn / 1e12,
        "exp_floor_ms": exp_floor_ms,
        "cache_study": cache_study,
        "roofline": {"bound": "mfma", "kernel": "mixed_attn_kernel", "achieved": achieved / 1e12,
                     "limiter": "vector ALU: the softmax of every phase and, for NVFP4, the decode of the packed "
                                "K/V tiles issue more VALU cycles than the tiles' MFMAs (per-phase counters in "
                                "profiles/mixed_attn_phases_mid-21x30x52-h12-d128.md)",
                     "peak": peak_eff / 1e12, "unit": "TFLOP/s", "frac": achieved / peak_eff,
                     # recorded for the workload's own configuration only
                     "traffic": recorded_traffic(w.name) if args.partition is None and args.num16 is None
                     and not mx else None,
                     "peak_note": "budget-weighted: 8-bit tiles at 5.0 PF (int8/fp8), 4-bit tiles at 10.1 PF "
                                  "(fp4), 16-bit tiles at 2.5 PF; achieved = retained tiles x 4*64*64*d flop over "
                                  "the mean mixed_attn launch duration of the flushed steps",
                     "launch_ms_mean": t_attn_mean * 1e3,
                     "frac_issued_dtype": achieved / peak_issued,
                     "peak_issued_dtype": peak_issued / 1e12,
                     "issued_note": "4-bit tiles at the peak of the MFMA the kernel issues for them: " +
                                    ("10.1 PF (scaled fp4, MXFP4)" if mx else
                                     "2.5 PF (fp16 MFMA on the exact NVFP4 values; gfx950 has no MFMA that applies "
                                     "E4M3 scales per 16 elements)")},
        "hbm": hbm,
    }
    if not args.no_cpu_baseline:
        rec["cpu_baseline"] = cpu_baseline(w)
    print(json.dumps(rec), flush=True)


if __name__ == "__main__":
    main()
