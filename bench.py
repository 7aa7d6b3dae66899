"""Benchmark of one verify step on one MI355X: tree build -> cascade verify
attention -> accept path, on a seeded synthetic batch resident in HBM.

    python bench.py [--steps K] [--warmup W] [--config 5] [--kv-split S]
                    [--cpu-seconds 15] [--no-cpu-baseline] [--noncascade]
                    [--tree canonical|third_level|resample] [--graph]
                    [--temperature 1.0] [--sample-vocab 32000]
    python bench.py --profile-stage tree|prefix|cascade   (attention calls of one stage only, for counters)
    python bench.py --copy-probe       (HBM counter calibration copy)

Prints one JSON line. Default workload: 64 requests x 32768-token contexts,
64 query / 8 KV heads, bf16 (the largest one-GPU workload). The K timed steps
each follow a 512 MiB cache-evicting write (outside the step's own event
pair), so every input comes from HBM; ms_per_step is their median and value =
verified tree tokens per second of the whole step (tree nodes / ms_per_step).
The roofline object describes the cascade attention operation (its main
kernel plus the split merge when the context is split), timed with HIP events
that the library records on its launch stream over the timed steps. `timing`
adds the same steps back to back (warm) beside the cold ones.
"""

from __future__ import annotations

import argparse
import hashlib
import json
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

HBM_PEAK_GBPS = 8000.0          # MI355X HBM3E
MFMA_PEAK_TFLOPS = {"bf16": 2500.0, "f32": 157.3}   # dense matrix peaks
METRIC = "verified tree tokens/sec + prefix-KV HBM GB/s (% of peak), cascade verify attn"
FLUSH_BYTES = 512 << 20         # larger than the 256 MB Infinity Cache and every L2


def percentiles(v) -> dict:
    """Median, 10th and 90th percentile of a list of times (ms)."""
    a = np.asarray(v, np.float64)
    return {"median": round(float(np.median(a)), 4), "p10": round(float(np.percentile(a, 10)), 4),
            "p90": round(float(np.percentile(a, 90)), 4)}
KERNEL_SRCS = [os.path.join(ROOT, "paper_2606_04446_amd", "csrc", f) for f in ("attention.hip", "common.h")]
TRAFFIC_FILE = os.path.join(ROOT, "profiles", "cascade_attention_traffic.json")


def parse():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--config", type=int, default=5)
    ap.add_argument("--kv-split", type=int, default=0)
    ap.add_argument("--row-group", type=int, default=0, choices=[0, 128, 384],
                    help="bf16 query rows per workgroup (0: the library's choice)")
    ap.add_argument("--packed", type=int, default=0, choices=[0, 1, 2],
                    help="384-row workgroups over all streams' tiles: 0 the library's choice, 1 off, 2 on")
    ap.add_argument("--cpu-seconds", type=float, default=15.0)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--noncascade", action="store_true",
                    help="also time the non-cascade baseline kernel (always on for workload 5)")
    ap.add_argument("--profile-stage", choices=["cascade", "prefix", "tree"],
                    help="only run W + K attention calls of this stage on the workload (no step, no oracle), "
                         "e.g. the tree-suffix tiles alone for MFMA counters; prints a short JSON line")
    ap.add_argument("--prefix-stage", action="store_true",
                    help="also time the attention call with the context keys only (STAGE_PREFIX)")
    ap.add_argument("--tree", choices=["canonical", "third_level", "resample"], default="canonical",
                    help="tree shape: the canonical chain-plus-branches tree (default), the third-level cascade "
                         "(a sub-branch inside every branch) or K+1 resampled chains, the latter two built from "
                         "parent arrays")
    ap.add_argument("--temperature", type=float, default=1.0,
                    help="temperature of the separately timed sampling-verification draws")
    ap.add_argument("--sample-vocab", type=int, default=32000,
                    help="vocabulary of the target logits for the sampling draws")
    ap.add_argument("--graph", action="store_true",
                    help="also capture the step in a HIP graph and take `value` from graph replays "
                         "(measured no faster than eager launches: the step is not launch-bound)")
    ap.add_argument("--copy-probe", action="store_true",
                    help="only run a plain 1 GiB device copy three times (HBM counter calibration)")
    ap.add_argument("--trace-summary", metavar="DIR",
                    help="host only: average duration of the attention kernel and the split merge per bench phase "
                         "(warm-up, cold, warm, back to back; --warmup/--steps of the traced run) from a rocprofv3 "
                         "kernel trace under DIR")
    ap.add_argument("--record-traffic", metavar="DIR",
                    help="host only: derive the attention kernel's HBM bytes per launch from rocprofv3 counter "
                         "CSVs under DIR (fetch/, write/, copy_fetch/, copy_write/, and fetch.log holding the "
                         "profiled bench line) and write them to the traffic record read by later runs")
    return ap.parse_args()


def copy_probe():
    """A device copy of known size: its FETCH_SIZE / WRITE_SIZE counters give
    the factor between those counters and the bytes actually moved."""
    import torch

    n = 1 << 30
    src = torch.ones(n, dtype=torch.uint8, device="cuda")
    dst = torch.empty_like(src)
    torch.cuda.synchronize()
    for _ in range(3):
        dst.copy_(src)
    torch.cuda.synchronize()
    print(json.dumps({"copy_probe_bytes": n, "copies": 3}), flush=True)


def kernel_sha() -> str:
    """Hash of the attention kernel sources with comments and blank lines
    removed (a comment edit does not invalidate recorded counters)."""
    h = hashlib.sha256()
    for path in KERNEL_SRCS:
        with open(path) as f:
            for line in f:
                code = line.split("//", 1)[0].rstrip()
                if code:
                    h.update(code.encode() + b"\n")
    return h.hexdigest()[:16]


def measured_traffic(config: int, kv_split: int, resolved_split: int):
    """HBM bytes per launch from committed rocprofv3 counters, if they were taken
    on the current kernel source and the same launch configuration."""
    try:
        with open(TRAFFIC_FILE) as f:
            rec = json.load(f)
    except (OSError, ValueError):
        return None
    key = f"config{config}"
    r = rec.get(key)
    if not r or r.get("kernel_sha") != kernel_sha() or r.get("kv_split") != kv_split \
            or r.get("resolved_kv_split") != resolved_split:
        return None
    return r.get("hbm_bytes_per_launch")


def kernel_name_matches(name: str, kernel: str) -> bool:
    """Whether a demangled kernel name is `kernel` (as a whole identifier:
    "cascade_bf16_kernel" does not match "noncascade_bf16_kernel")."""
    import re
    return re.search(r"(?<![A-Za-z0-9_])" + re.escape(kernel) + r"(?![A-Za-z0-9_])", name) is not None


def _counter_per_dispatch(csv_dir: str, kernel: str, counter: str) -> float:
    """Mean over dispatches of `kernel` of the counter's value (summed over the
    rows of each dispatch) in a rocprofv3 counter-collection CSV."""
    import csv
    import glob

    paths = glob.glob(os.path.join(csv_dir, "**", "*counter_collection.csv"), recursive=True)
    if not paths:
        raise FileNotFoundError(f"no counter_collection.csv under {csv_dir}")
    per = {}
    for path in paths:
        with open(path) as f:
            for r in csv.DictReader(f):
                if kernel_name_matches(r["Kernel_Name"], kernel) and r["Counter_Name"] == counter:
                    per[r["Dispatch_Id"]] = per.get(r["Dispatch_Id"], 0.0) + float(r["Counter_Value"])
    if not per:
        raise ValueError(f"no {counter} rows for {kernel} under {csv_dir}")
    return sum(per.values()) / len(per)


def trace_summary(d: str, warmup: int, steps: int) -> dict:
    """Mean duration (us) of every attention kernel and split merge in a
    rocprofv3 kernel trace, per phase of a default bench run: `warmup`
    warm-up steps, then `steps` cold, `steps` warm and `steps` back-to-back
    steps, each with one attention call (dispatches in start order)."""
    import csv
    import glob

    paths = glob.glob(os.path.join(d, "**", "*kernel_trace.csv"), recursive=True)
    if not paths:
        raise FileNotFoundError(f"no kernel_trace.csv under {d}")
    names = ["cascade_bf16_packed_kernel", "cascade_bf16_wide_kernel", "cascade_bf16_kernel",
             "cascade_attention_kernel", "split_merge_kernel"]
    per = {}
    for path in paths:
        with open(path) as f:
            for r in csv.DictReader(f):
                for k in names:
                    if kernel_name_matches(r["Kernel_Name"], k):
                        per.setdefault(k, []).append((int(r["Start_Timestamp"]), int(r["End_Timestamp"])))
    bounds = {"warmup": (0, warmup), "cold": (warmup, warmup + steps),
              "warm": (warmup + steps, warmup + 2 * steps), "backtoback": (warmup + 2 * steps, warmup + 3 * steps)}
    out = {}
    for k, ev in per.items():
        dur = [(e - s_) / 1e3 for s_, e in sorted(ev)]
        out[k] = {"dispatches": len(dur), "all": round(float(np.mean(dur)), 1)}
        for ph, (a, b) in bounds.items():
            if len(dur) >= b:
                out[k][ph] = round(float(np.mean(dur[a:b])), 1)
    return out


def attention_kernel_name(line: dict) -> str:
    """The attention kernel a bench line's launch ran: by dtype and
    workgroup shape (config.row_group, config.packed)."""
    if line.get("dtype") != "bf16":
        return "cascade_attention_kernel"
    cfg = line.get("config", {})
    if cfg.get("packed"):
        return "cascade_bf16_packed_kernel"
    if cfg.get("row_group") == 384:
        return "cascade_bf16_wide_kernel"
    return "cascade_bf16_kernel"


def record_traffic(d: str):
    """Write the attention kernel's measured HBM bytes per launch. FETCH_SIZE and
    WRITE_SIZE (KiB per dispatch) are scaled by what they read for a 1 GiB
    device copy (--copy-probe), so the factors come from the same counters."""
    with open(os.path.join(d, "fetch.log")) as f:
        line = [ln for ln in f.read().splitlines() if ln.startswith("{")][-1]
    bench = json.loads(line)
    kern = attention_kernel_name(bench)
    fetch = _counter_per_dispatch(os.path.join(d, "fetch"), kern, "FETCH_SIZE")
    write = _counter_per_dispatch(os.path.join(d, "write"), kern, "WRITE_SIZE")
    if bench.get("roofline", {}).get("splits", 1) > 1:
        # the split merge reads the partial states back: part of the same operation
        fetch += _counter_per_dispatch(os.path.join(d, "fetch"), "split_merge_kernel", "FETCH_SIZE")
        write += _counter_per_dispatch(os.path.join(d, "write"), "split_merge_kernel", "WRITE_SIZE")
    copy_kib = (1 << 30) / 1024.0
    f_fac = copy_kib / _counter_per_dispatch(os.path.join(d, "copy_fetch"), "__amd_rocclr_copyBuffer", "FETCH_SIZE")
    w_fac = copy_kib / _counter_per_dispatch(os.path.join(d, "copy_write"), "__amd_rocclr_copyBuffer", "WRITE_SIZE")
    cfg = bench["config"]
    cfg_num = next(k for k, v in _workload_names().items() if v == cfg["workload"])
    rec = {}
    if os.path.exists(TRAFFIC_FILE):
        with open(TRAFFIC_FILE) as f:
            rec = json.load(f)
    rec[f"config{cfg_num}"] = {
        "workload": cfg["workload"], "kernel_sha": kernel_sha(), "kv_split": bench.get("requested_kv_split", 0),
        "resolved_kv_split": cfg["kv_split"], "kernel": kern, "fetch_kib_per_dispatch": round(fetch, 1),
        "write_kib_per_dispatch": round(write, 1), "fetch_factor": round(f_fac, 4), "write_factor": round(w_fac, 4),
        "hbm_bytes_per_launch": int(round((fetch * f_fac + write * w_fac) * 1024)),
        "summary": f"profiles/cascade_attention_{cfg['workload']}.md",
    }
    with open(TRAFFIC_FILE, "w") as f:
        json.dump(rec, f, indent=1)
        f.write("\n")
    print(json.dumps(rec[f"config{cfg_num}"]), flush=True)


def _workload_names() -> dict:
    from paper_2606_04446_amd import workload as wl
    return {k: v.name for k, v in wl.WORKLOADS.items()}


def bench_parent_array(B: int, p_row, q_row=None, chains: int = 0) -> np.ndarray:
    """Parent array (local indices, node 0 the anchor) of one request's tree:
    the input of the parent-array tree builder for the --tree shapes (the
    third-level cascade of sec. 4.3 and resampled chains):
      chains > 0  `chains` independent chains of B-1 drafts under the anchor;
      otherwise   the first-draft chain, one branch per re-anchor position p
                  (ascending) hanging under the chain node at p - 1, and, when
                  q_row is given, per branch a sub-branch hanging under the
                  branch node at q - 1 (q > p; 0 = none), after all branches."""
    par = [-1]
    if chains > 0:
        for _ in range(chains):
            prev = 0
            for _ in range(B - 1):
                par.append(prev)
                prev = len(par) - 1
        return np.asarray(par, np.int32)
    for j in range(1, B):
        par.append(j - 1)
    order = sorted(range(len(p_row)), key=lambda k: p_row[k])
    at = {}                                     # (branch, position) -> node
    for k in order:
        pk = int(p_row[k])
        prev = pk - 1
        for pos in range(pk, B):
            par.append(prev)
            prev = len(par) - 1
            at[(k, pos)] = prev
    if q_row is not None:
        for k in order:
            qk = int(q_row[k])
            if qk <= 0:
                continue
            prev = at[(k, qk - 1)] if qk - 1 >= int(p_row[k]) else qk - 1
            for _ in range(qk, B):
                par.append(prev)
                prev = len(par) - 1
    return np.asarray(par, np.int32)


def cpu_model() -> str:
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return "unknown"


def cpu_baseline(x, layout, node_indptr, parent_host, budget_s: float, parents=None):
    """The oracle, as it stands, on whole requests until the time budget is spent."""
    import torch
    from threadpoolctl import threadpool_info

    from oracle.attention import gather_context, request_attention
    from oracle.tree import build_tree, tree_from_parents

    done_nodes, done_req = 0, 0
    t_total = 0.0
    for b in range(layout.batch):
        s, e = int(node_indptr[b]), int(node_indptr[b + 1])
        C = int(layout.ctx_len[b])
        npg = (C + 15) // 16
        pages = torch.from_numpy(layout.page_table[b, :npg].astype(np.int64)).to(x["k_cache"].device)
        kc = x["k_cache"].index_select(0, pages).float().cpu().numpy()
        vc = x["v_cache"].index_select(0, pages).float().cpu().numpy()
        q = x["q"][s:e].float().cpu().numpy()
        kt = x["k_tree"][s:e].float().cpu().numpy()
        vt = x["v_tree"][s:e].float().cpu().numpy()
        def run_oracle():
            tree = (build_tree(layout.spec.B, layout.p[b, :layout.K[b]]) if parents is None
                    else tree_from_parents(parents[b], layout.spec.B))
            kcb, vcb = gather_context(kc, vc, np.arange(npg), C, 16)
            request_attention(q.astype(np.float64), kcb, vcb, kt.astype(np.float64), vt.astype(np.float64), tree)

        t0 = time.perf_counter()
        run_oracle()
        t_total += time.perf_counter() - t0
        done_nodes += e - s
        done_req += 1
        if layout.batch == 1:
            # a single request: the same oracle call with one BLAS thread
            from threadpoolctl import threadpool_limits
            with threadpool_limits(limits=1):
                t1 = time.perf_counter()
                run_oracle()
                one_thread = (e - s) / (time.perf_counter() - t1)
        if t_total >= budget_s:
            break
    blas = [i for i in threadpool_info() if i.get("user_api") == "blas"]
    cores = max([i.get("num_threads", 1) for i in blas] or [1])
    blas_name = ", ".join(sorted({f"{i.get('internal_api')} {i.get('version')}" for i in blas})) or "unknown"
    res = {
        "value": done_nodes / t_total, "unit": "tokens/s", "cores": cores, "kind": "oracle",
        "sample": f"{done_req} of {layout.batch} requests (tree build + float64 attention of every node "
                  f"and query head over the full context and its ancestors), {t_total:.1f} s, "
                  f"{len(os.sched_getaffinity(0))} host cores visible",
        "cpu_model": cpu_model(), "blas": blas_name,
    }
    if layout.batch == 1:
        res["value_1_thread"] = one_thread
    return res


def main():
    args = parse()
    world = int(os.environ.get("WORLD_SIZE", "1"))
    if args.gpus > 1 or world > 1:
        print(f"bench.py measures one GPU only (the verify path is built and measured on a single "
              f"MI355X); --gpus {args.gpus} / WORLD_SIZE {world} is not supported", file=sys.stderr)
        sys.exit(2)
    if args.copy_probe:
        copy_probe()
        return
    if args.record_traffic:
        record_traffic(args.record_traffic)
        return
    if args.trace_summary:
        print(json.dumps(trace_summary(args.trace_summary, args.warmup, args.steps)), flush=True)
        return

    import torch

    from paper_2606_04446_amd import d2sd
    from paper_2606_04446_amd import workload as wl

    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    layout = wl.draw_layout(args.config)
    spec = layout.spec
    B = spec.B
    parents = None
    if args.tree == "canonical":
        node_indptr, W = d2sd.tree_plan(B, layout.K, layout.p)
    else:
        q_sub = wl.draw_sub_branch_positions(layout)
        parents = [bench_parent_array(B, layout.p[b, :layout.K[b]], q_sub[b, :layout.K[b]])
                   if args.tree == "third_level" else bench_parent_array(B, [], chains=int(layout.K[b]) + 1)
                   for b in range(layout.batch)]
        node_indptr = np.concatenate([[0], np.cumsum([len(pa) for pa in parents])]).astype(np.int32)
        W = (int(np.diff(node_indptr).max()) + 31) // 32
    total = int(node_indptr[-1])
    max_nodes = int(np.diff(node_indptr).max())
    max_ctx = int(layout.ctx_len.max())
    t = lambda a: torch.from_numpy(np.ascontiguousarray(a)).to(dev)
    d_K, d_p, d_ip = t(layout.K), t(layout.p), t(node_indptr)
    d_ctx, d_pt = t(layout.ctx_len), t(layout.page_table)
    x = wl.draw_tensors(layout, total, device=dev)

    if parents is None:
        build = lambda out=None: d2sd.tree_build(B, d_K, d_p, d_ip, total, W, out=out)
    else:
        d_par = t(np.concatenate(parents))
        build = lambda out=None: d2sd.tree_from_parents(d_ip, total, max_nodes, d_par, W, out=out)
    tree = build()
    torch.cuda.synchronize()
    parent_host = tree["parent"].cpu().numpy()
    draft, argmax = wl.draw_tokens(layout, node_indptr, parent_host)
    d_draft, d_argmax = t(draft), t(argmax)
    out = torch.empty_like(x["q"])
    lse = torch.empty(x["q"].shape[:2], dtype=torch.float32, device=dev)
    a = d2sd.attn_args(x["q"], x["k_cache"], x["v_cache"], d_pt, d_ctx, x["k_tree"], x["v_tree"], d_ip,
                       tree["anc_mask"], out, lse, total_nodes=total, max_nodes=max_nodes, max_ctx_len=max_ctx,
                       kv_split=args.kv_split, node_indptr_host=node_indptr, row_group=args.row_group,
                       packed=args.packed)
    ws_bytes = d2sd.cascade_workspace_size(a)
    kv_split = d2sd.cascade_kv_split(a)
    row_group, packed = d2sd.cascade_shape(a)
    n_splits = -(-max_ctx // kv_split) if max_ctx > 0 else 1
    ws = torch.empty(max(ws_bytes, 1), dtype=torch.uint8, device=dev)
    acc = d2sd.accept_path(B, d_ip, total, tree["parent"], tree["depth"], tree["path_id"], d_draft, d_argmax)

    def attention(stage=d2sd.STAGE_CASCADE, o=out, l=lse):
        d2sd.cascade_verify_attention(x["q"], x["k_cache"], x["v_cache"], d_pt, d_ctx, x["k_tree"], x["v_tree"],
                                      d_ip, tree["anc_mask"], total_nodes=total, max_nodes=max_nodes,
                                      max_ctx_len=max_ctx, stage=stage, kv_split=args.kv_split, out=o, lse=l,
                                      workspace=ws, node_indptr_host=node_indptr, row_group=args.row_group,
                                      packed=args.packed)

    if args.profile_stage:
        # Attention calls of one stage only (e.g. the tree-suffix tiles alone),
        # for counter runs that must see nothing else.
        stage = {"cascade": d2sd.STAGE_CASCADE, "prefix": d2sd.STAGE_PREFIX, "tree": d2sd.STAGE_TREE}[args.profile_stage]
        for _ in range(args.warmup):
            attention(stage)
        torch.cuda.synchronize()
        d2sd.kernel_timing_collect_parts()
        d2sd.kernel_timing_enable(True)
        for _ in range(args.steps):
            attention(stage)
        torch.cuda.synchronize()
        d2sd.kernel_timing_enable(False)
        kern, merge = d2sd.kernel_timing_collect_parts()
        depth = tree["depth"].cpu().numpy().astype(np.int64)
        tree_keys = float((depth + 1).sum())                       # visible tree keys per (node, query head)
        flops = 4.0 * spec.hq * spec.head_dim * (tree_keys if stage == d2sd.STAGE_TREE else
                                                 float(np.repeat(layout.ctx_len.astype(np.int64),
                                                                 np.diff(node_indptr)).sum())
                                                 + (tree_keys if stage == d2sd.STAGE_CASCADE else 0.0))
        k_ms = float(np.mean(kern))
        splits = n_splits if stage != d2sd.STAGE_TREE else 1
        # the keys read by --record-traffic: dtype, config, requested_kv_split, roofline.splits
        print(json.dumps({"profile_stage": args.profile_stage, "dtype": spec.dtype, "calls": len(kern),
                          "config": {"workload": spec.name, "kv_split": kv_split, "row_group": row_group,
                                     "packed": packed, "tree": args.tree},
                          "requested_kv_split": args.kv_split, "roofline": {"splits": splits},
                          "kernel_ms": round(k_ms, 4), "merge_ms": round(float(np.mean(merge)), 4),
                          "algorithmic_flop_per_call": flops, "tflops": round(flops / (k_ms / 1e3) / 1e12, 3)}),
              flush=True)
        return

    def step():
        build(out=tree)
        attention()
        d2sd.accept_path(B, d_ip, total, tree["parent"], tree["depth"], tree["path_id"], d_draft, d_argmax,
                         out=acc)

    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()
    flush_buf = torch.empty(FLUSH_BYTES, dtype=torch.uint8, device=dev)

    def timed_steps(reps, flush):
        """reps steps, each bracketed by its own event pair; with flush, a
        512 MiB write before each step (outside its pair) evicts the L2
        caches and the 256 MB Infinity Cache, so every input comes from HBM.
        Returns the per-step times and the library's per-call attention
        kernel and split-merge times (ms)."""
        evs = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)) for _ in range(reps)]
        d2sd.kernel_timing_collect_parts()
        d2sd.kernel_timing_enable(True)
        torch.cuda.synchronize()
        for i, (e_a, e_b) in enumerate(evs):
            if flush:
                flush_buf.fill_(i & 0xff)
            e_a.record()
            step()
            e_b.record()
        torch.cuda.synchronize()
        d2sd.kernel_timing_enable(False)
        kern, merge = d2sd.kernel_timing_collect_parts()
        return [e_a.elapsed_time(e_b) for e_a, e_b in evs], kern, merge

    # The timed region: K cold steps (the headline), bracketed by synchronisations.
    step_cold, kern_cold, merge_cold = timed_steps(args.steps, True)
    # The same steps back to back (warm), and K back-to-back steps between one event pair.
    step_warm, kern_warm, merge_warm = timed_steps(args.steps, False)
    ev0, ev1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    ev0.record()
    for _ in range(args.steps):
        step()
    ev1.record()
    torch.cuda.synchronize()
    step_ms_backtoback = ev0.elapsed_time(ev1) / args.steps
    del flush_buf

    op_cold = [k + m for k, m in zip(kern_cold, merge_cold)]
    timing = {"reps": args.steps, "flush_bytes": FLUSH_BYTES,
              "cold": {"step_ms": percentiles(step_cold), "attn_ms": percentiles(op_cold),
                       "attn_kernel_ms": percentiles(kern_cold), "merge_ms": percentiles(merge_cold)},
              "warm": {"step_ms": percentiles(step_warm),
                       "attn_ms": percentiles([k + m for k, m in zip(kern_warm, merge_warm)]),
                       "attn_kernel_ms": percentiles(kern_warm), "merge_ms": percentiles(merge_warm)},
              "backtoback_step_ms": round(step_ms_backtoback, 4)}
    step_ms_cold = float(np.median(step_cold))
    op_ms = float(np.mean(op_cold))                 # attention operation: kernel + split merge
    kern_ms = float(np.mean(kern_cold))
    merge_ms = float(np.mean(merge_cold))

    # The prefix stage alone (context keys only, no tree tiles), on request:
    # the time that the prefix K/V bandwidth can also be quoted against.
    prefix_ms = None
    if args.prefix_stage:
        out_p, lse_p = torch.empty_like(out), torch.empty_like(lse)
        for _ in range(args.warmup):
            attention(d2sd.STAGE_PREFIX, out_p, lse_p)
        torch.cuda.synchronize()
        d2sd.kernel_timing_collect_parts()
        d2sd.kernel_timing_enable(True)
        for _ in range(args.steps):
            attention(d2sd.STAGE_PREFIX, out_p, lse_p)
        torch.cuda.synchronize()
        d2sd.kernel_timing_enable(False)
        pk, pm = d2sd.kernel_timing_collect_parts()
        prefix_ms = float(np.mean(pk)) + float(np.mean(pm))
        del out_p, lse_p

    # The same step captured once in a HIP graph and replayed (the step
    # allocates nothing and issues no memset, so it can be captured as it is).
    step_ms = step_ms_cold
    graph_ms = None
    if args.graph:
        side = torch.cuda.Stream()
        side.wait_stream(torch.cuda.current_stream())
        with torch.cuda.stream(side):
            step()
        torch.cuda.current_stream().wait_stream(side)
        torch.cuda.synchronize()
        graph = torch.cuda.CUDAGraph()
        with torch.cuda.graph(graph):
            step()
        for _ in range(args.warmup):
            graph.replay()
        torch.cuda.synchronize()
        ev0.record()
        for _ in range(args.steps):
            graph.replay()
        ev1.record()
        torch.cuda.synchronize()
        graph_ms = ev0.elapsed_time(ev1) / args.steps

    # algorithmic work of one attention operation
    esz = 2 if spec.dtype == "bf16" else 4
    D, Hq, Hkv = spec.head_dim, spec.hq, spec.hkv
    ctx = layout.ctx_len.astype(np.int64)
    prefix_bytes = int(ctx.sum()) * Hkv * D * 2 * esz
    depth = tree["depth"].cpu().numpy().astype(np.int64)
    n_per_req = np.diff(node_indptr).astype(np.int64)
    visible = np.repeat(ctx, n_per_req) + depth + 1          # keys each node attends to
    flops = 4.0 * Hq * D * float(visible.sum())
    t_s = op_ms / 1e3
    gbps = prefix_bytes / t_s / 1e9
    tflops = flops / t_s / 1e12
    t_hbm = prefix_bytes / (HBM_PEAK_GBPS * 1e9)
    t_mfma = flops / (MFMA_PEAK_TFLOPS[spec.dtype] * 1e12)
    traffic = measured_traffic(args.config, args.kv_split, kv_split) if args.tree == "canonical" else None
    parts = {"kernel_ms": round(kern_ms, 4), "merge_ms": round(merge_ms, 4), "splits": n_splits}
    if t_mfma > t_hbm:
        roof = {"bound": "mfma", "achieved": round(tflops, 2), "peak": MFMA_PEAK_TFLOPS[spec.dtype],
                "unit": "TFLOP/s", "frac": round(tflops / MFMA_PEAK_TFLOPS[spec.dtype], 4), "traffic": traffic,
                **parts}
    else:
        roof = {"bound": "hbm", "achieved": round(gbps, 1), "peak": HBM_PEAK_GBPS, "unit": "GB/s",
                "frac": round(gbps / HBM_PEAK_GBPS, 4), "traffic": traffic, **parts}

    res = {
        "metric": METRIC,
        "value": round(total / (step_ms / 1e3), 1),
        "unit": "tokens/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(step_ms, 4),
        "ms_per_step_timing": "median of the K timed steps, each after a 512 MiB cache-evicting write",
        "graph": bool(args.graph),
        "graph_replay_ms_per_step": round(graph_ms, 4) if graph_ms is not None else None,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": spec.dtype,
        "data": "synthetic",
        "config": {"workload": spec.name, "batch": layout.batch,
                   "ctx_len": [int(ctx.min()), int(ctx.max())], "q_heads": Hq, "kv_heads": Hkv,
                   "head_dim": D, "block": B, "branches": spec.K, "tree_nodes": total,
                   "page_size": spec.page_size, "kv_split": kv_split, "row_group": row_group, "packed": packed,
                   "tree": args.tree},
        "roofline": roof,
        "roofline_note": ("mfma-bound: the workload's algorithmic flops at the bf16 dense peak take longer "
                          "than its prefix K/V bytes at the HBM peak" if roof["bound"] == "mfma" else
                          "hbm-bound: the prefix K/V bytes at the HBM peak take longer than the flops at the "
                          "MFMA peak"),
        "prefix_kv_gbps": round(gbps, 1),
        "prefix_kv_hbm_frac": round(gbps / HBM_PEAK_GBPS, 4),
        "prefix_stage": None if prefix_ms is None else {
            "ms": round(prefix_ms, 4), "prefix_kv_gbps": round(prefix_bytes / (prefix_ms / 1e3) / 1e9, 1),
            "prefix_kv_hbm_frac": round(prefix_bytes / (prefix_ms / 1e3) / 1e9 / HBM_PEAK_GBPS, 4)},
        "attn_tflops": round(tflops, 2),
        "attn_mfma_frac": round(tflops / MFMA_PEAK_TFLOPS[spec.dtype], 4),
        "attn_ms": round(op_ms, 4),
        "attn_tokens_per_s": round(total / t_s, 1),
        "kernel_sha": kernel_sha(),
        "requested_kv_split": args.kv_split,
        "timing": timing,
    }
    if args.noncascade or args.config == 5:
        out2 = torch.empty_like(out)
        lse2 = torch.empty_like(lse)
        reps = 3
        d2sd.noncascade_verify_attention(x["q"], x["k_cache"], x["v_cache"], d_pt, d_ctx, x["k_tree"], x["v_tree"],
                                         d_ip, tree["anc_mask"], total_nodes=total, max_nodes=max_nodes,
                                         max_ctx_len=max_ctx, out=out2, lse=lse2)
        torch.cuda.synchronize()
        d2sd.kernel_timing_enable(True)
        for _ in range(reps):
            d2sd.noncascade_verify_attention(x["q"], x["k_cache"], x["v_cache"], d_pt, d_ctx, x["k_tree"],
                                             x["v_tree"], d_ip, tree["anc_mask"], total_nodes=total,
                                             max_nodes=max_nodes, max_ctx_len=max_ctx, out=out2, lse=lse2)
        torch.cuda.synchronize()
        d2sd.kernel_timing_enable(False)
        n, ms = d2sd.kernel_timing_collect()
        nc_ms = ms / max(n, 1)
        res["noncascade"] = {"kernel_ms": round(nc_ms, 3), "speedup_of_cascade": round(nc_ms / op_ms, 2),
                             "requested_prefix_bytes": int((np.repeat(ctx, n_per_req)).sum()) * Hkv * D * 2 * esz,
                             "max_abs_diff_vs_cascade": float((out2.float() - out.float()).abs().max())}
    # Device re-anchor selection (Eq. 4-5) and node offsets for the same batch,
    # the steps that precede the verify path when boundaries come from the
    # drafter's confidences; timed on their own (they are not in `value`).
    conf = t(wl.draw_confidences(layout))
    kmax = max(int(layout.K.max(initial=0)), 1)
    p_sel = torch.empty((layout.batch, kmax), dtype=torch.int32, device=dev)
    ip_sel = torch.empty(layout.batch + 1, dtype=torch.int32, device=dev)
    for _ in range(3):
        d2sd.select_reanchor(B, conf, d_K, kmax, p_out=p_sel)
        d2sd.tree_indptr(B, d_K, p_sel, out=ip_sel)
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    e0.record()
    for _ in range(args.steps):
        d2sd.select_reanchor(B, conf, d_K, kmax, p_out=p_sel)
        d2sd.tree_indptr(B, d_K, p_sel, out=ip_sel)
    e1.record()
    torch.cuda.synchronize()
    res["device_reanchor_us"] = round(e0.elapsed_time(e1) * 1e3 / args.steps, 2)

    # Commit of the accepted paths into the paged cache (the step after the
    # path): pages for every position below C + B are appended to the pool.
    acc_c = d2sd.accept_path(B, d_ip, total, tree["parent"], tree["depth"], tree["path_id"], d_draft, d_argmax)
    C = layout.ctx_len.astype(np.int64)
    have = (C + 15) // 16
    need = (C + B + 15) // 16
    table2 = np.zeros((layout.batch, int(need.max())), np.int32)
    table2[:, :layout.page_table.shape[1]] = layout.page_table
    nxt = x["k_cache"].shape[0]
    for b_ in range(layout.batch):
        for j in range(int(have[b_]), int(need[b_])):
            table2[b_, j] = nxt
            nxt += 1
    grow = nxt - x["k_cache"].shape[0]
    kc2 = torch.cat([x["k_cache"], torch.zeros((grow,) + tuple(x["k_cache"].shape[1:]), dtype=x["k_cache"].dtype, device=dev)])
    vc2 = torch.cat([x["v_cache"], torch.zeros((grow,) + tuple(x["v_cache"].shape[1:]), dtype=x["v_cache"].dtype, device=dev)])
    d_t2 = t(table2)
    ctx2 = d_ctx.clone()
    commit = lambda: d2sd.commit_accepted_kv(B, d_ip, total, acc_c["path_nodes"], acc_c["accept_len"], x["k_tree"],
                                             x["v_tree"], d_t2, ctx2, kc2, vc2, max_ctx_len=max_ctx)
    for _ in range(3):
        commit()
    torch.cuda.synchronize()
    e0.record()
    for _ in range(args.steps):
        commit()                      # context lengths are clamped to max_ctx: same work every call
    e1.record()
    torch.cuda.synchronize()
    commit_s = e0.elapsed_time(e1) / 1e3 / args.steps
    n_tok = int((acc_c["accept_len"].cpu().numpy().astype(np.int64) + 1).sum())
    commit_bytes = 2 * 2 * n_tok * Hkv * D * esz          # K and V rows, read and written
    res["commit"] = {"us": round(commit_s * 1e6, 2), "tokens": n_tok,
                     "gbps": round(commit_bytes / commit_s / 1e9, 1)}
    del kc2, vc2

    # Sampling verification (T > 0): a target draw at every node from its
    # logits row (bf16 [nodes, vocab]), one draw per distinct context, then the
    # accept path on the drawn tokens; timed on its own (not in `value`).
    Vs = args.sample_vocab
    logits = wl.draw_logits(layout, argmax, vocab=Vs, device=dev, dtype="bf16")
    d_u = t(wl.draw_uniforms(layout, total))
    toks = torch.empty(total, dtype=torch.int32, device=dev)
    draw = lambda: d2sd.sample_targets(d_ip, total, max_nodes, tree["parent"], d_draft, logits, args.temperature,
                                       d_u, out=toks)
    for _ in range(3):
        draw()
    torch.cuda.synchronize()
    e0.record()
    for _ in range(args.steps):
        draw()
    e1.record()
    torch.cuda.synchronize()
    draw_s = e0.elapsed_time(e1) / 1e3 / args.steps
    # cold: each draw after a 512 MiB write, so the logits come from HBM and
    # not from the Infinity Cache, which holds the whole batch's rows when
    # they fit (167 MB on the bench workload)
    flush_buf = torch.empty(FLUSH_BYTES, dtype=torch.uint8, device=dev)
    evs = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)) for _ in range(args.steps)]
    for i, (e_a, e_b) in enumerate(evs):
        flush_buf.fill_(i & 0xff)
        e_a.record()
        draw()
        e_b.record()
    torch.cuda.synchronize()
    cold_s = float(np.median([e_a.elapsed_time(e_b) for e_a, e_b in evs])) / 1e3
    del flush_buf
    acc_t = d2sd.accept_path(B, d_ip, total, tree["parent"], tree["depth"], tree["path_id"], d_draft, toks)
    draw_bytes = total * Vs * 2                            # every node streams one logits row once
    draw_gbps = draw_bytes / draw_s / 1e9
    cold_gbps = draw_bytes / cold_s / 1e9
    res["sampling"] = {"temperature": args.temperature, "vocab": Vs, "rows": total, "us": round(draw_s * 1e6, 2),
                       "gbps": round(draw_gbps, 1), "hbm_frac": round(draw_gbps / HBM_PEAK_GBPS, 4),
                       "us_cold": round(cold_s * 1e6, 2), "gbps_cold": round(cold_gbps, 1),
                       "hbm_frac_cold": round(cold_gbps / HBM_PEAK_GBPS, 4),
                       "mean_accept_len": round(float(acc_t["accept_len"].float().mean()), 3),
                       "greedy_mean_accept_len": round(float(acc["accept_len"].float().mean()), 3)}
    del logits
    if not args.no_cpu_baseline:
        res["cpu_baseline"] = cpu_baseline(x, layout, node_indptr, parent_host, args.cpu_seconds, parents)
    print(json.dumps(res), flush=True)


if __name__ == "__main__":
    main()
