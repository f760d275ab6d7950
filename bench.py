"""Benchmark: shared-prefix decode attention on one MI355X.

One step is one call of parrot_shared_prefix_decode (partial-result kernel
with its prefix-group and split-KV roles, then the merge kernel) for one layer
of a decode batch.  The headline workload is the full-depth mixed serving
step: 32 LLaMA-7B layers (32 heads x 128, bf16 KV in 16-token blocks with
permuted block tables), 256 requests in 8 Zipf(1.1) prefix groups plus 32
ungrouped requests.  All 32 layers are resident in HBM with their own KV and
the steps cycle through them, so a layer's KV is never still in the 256 MB
Infinity Cache when it is read again.  A one-layer workload cycles `--layers`
distinct-KV copies instead.

The line carries, besides the headline: the same measurements for the other
decode workloads (`workloads`), the prefix-length sweep of the shared path
against the per-request path (`sweep`), a prefill leg (`prefill`: the Fill of
64 contexts forked from a 6000-token system prompt, with an MFMA roofline),
the device's read-bandwidth ceiling measured in the same process by the
library's read probe (`ceilings`), and the float64 CPU oracle timed on a
bounded sample of the headline workload (`cpu_baseline`).  `--mode prefill`
prints only the prefill leg as the line.

`value` is requests per second per layer (R / seconds per step).  The
`roofline` object describes the dominant kernel (the partial-result kernel)
from HIP events attached to its launches on the launch stream during the
timed steps.
"""
from __future__ import annotations

import argparse
import hashlib
import json
import os
import re
import subprocess
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

HBM_PEAK_GBPS = 8000.0          # MI355X HBM3E
MFMA_F16_PEAK_TFLOPS = 2500.0   # dense fp16/bf16 MFMA
ELT_BYTES = {"float32": 4, "float16": 2, "bfloat16": 2}
DTYPE_TAG = {"float32": "f32", "float16": "f16", "bfloat16": "bf16"}
COUNTERS_FILE = os.path.join(ROOT, "profiles", "partials_counters.json")
KERNEL_SOURCES = ["paper_2405_19888_amd/csrc/partials.hip", "paper_2405_19888_amd/csrc/prefix_role.h",
                  "paper_2405_19888_amd/csrc/splitkv_role.h", "paper_2405_19888_amd/csrc/common.h"]
PREFILL_COUNTERS_FILE = os.path.join(ROOT, "profiles", "prefill_counters.json")
PREFILL_SOURCES = ["paper_2405_19888_amd/csrc/prefill.hip", "paper_2405_19888_amd/csrc/prefill_tile.h",
                   "paper_2405_19888_amd/csrc/prefill_shape.h", "paper_2405_19888_amd/csrc/prefill_args.h",
                   "paper_2405_19888_amd/csrc/prefix_role.h", "paper_2405_19888_amd/csrc/common.h"]
SWEEP_DEFAULT = "256,512,1024,2048,4096,8192,16384"


def kernel_source_hash(sources=KERNEL_SOURCES) -> str:
    """Hash of a kernel's code with comments and blank space removed, so that
    counters taken on it stay attached until the code itself changes."""
    h = hashlib.sha256()
    for rel in sources:
        with open(os.path.join(ROOT, rel), encoding="utf-8") as f:
            src = f.read()
        src = re.sub(r"/\*.*?\*/", " ", src, flags=re.S)
        src = re.sub(r"//[^\n]*", " ", src)
        h.update(" ".join(src.split()).encode())
    return h.hexdigest()[:16]


def traffic_from_counters(workload: str, path: str = COUNTERS_FILE, sources=KERNEL_SOURCES):
    """HBM bytes per launch of the dominant kernel from committed rocprofv3
    counter runs on `workload`, only if they were taken on the current kernel
    source."""
    if not os.path.exists(path):
        return None
    with open(path) as f:
        rec = json.load(f)
    if rec.get("source_hash") != kernel_source_hash(sources):
        return None
    w = rec.get("workloads", {}).get(workload)
    return None if w is None else w.get("bytes_per_launch")


def algorithmic_bytes(plan):
    """Bytes the method must move, per layer (no partials, no re-reads)."""
    elt = ELT_BYTES[plan.dtype]
    kv_tok = 2 * plan.heads * plan.head_dim * elt
    R = plan.num_requests
    q = R * plan.heads * plan.head_dim * elt
    out = q
    lse = R * plan.heads * 4
    prefix_kv = int(plan.prefix_lens.sum()) * kv_tok
    suffix_kv = int(plan.suffix_lens.sum()) * kv_tok
    naive_kv = int(plan.context_lens().sum()) * kv_tok
    sizes = plan.reader_counts()      # requests that read each group's prefix
    prefix_flops = sum(4 * plan.head_dim * plan.heads * sizes[g] * int(plan.prefix_lens[g])
                       for g in range(plan.num_groups))
    return dict(prefix_kv=prefix_kv, suffix_kv=suffix_kv, q=q, out=out, lse=lse,
                shared_total=prefix_kv + suffix_kv + q + out + lse,
                splitkv=suffix_kv + q,
                naive_total=naive_kv + q + out + lse,
                prefix_flops=prefix_flops)


# ------------------------------------------------------------------ CPU side
def cpu_model() -> str | None:
    """lscpu's model name with the vendor, family, model and stepping numbers
    (a virtualised host may report only a generic name)."""
    try:
        out = subprocess.run(["lscpu"], capture_output=True, text=True, timeout=10).stdout
        f = {}
        for line in out.splitlines():
            if ":" in line:
                k, v = line.split(":", 1)
                f[k.strip().lower()] = v.strip()
        if "model name" in f:
            ids = ", ".join(f"{k} {f[k]}" for k in ("vendor id", "cpu family", "model", "stepping")
                            if k in f)
            return f"{f['model name']} ({ids})" if ids else f["model name"]
    except (OSError, subprocess.SubprocessError):
        pass
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return None


def host_info() -> dict:
    """The host CPU model and the BLAS numpy links against."""
    blas = None
    try:
        import numpy as np
        deps = np.show_config(mode="dicts").get("Build Dependencies", {})
        blas = deps.get("blas", {}).get("name")
    except Exception:
        pass
    return {"cpu_model": cpu_model(), "numpy_blas": blas}


class pinned_host_threads:
    """BLAS / OpenMP pools and torch's intra-op pool pinned to the CPUs this
    process may run on, for the duration of the block."""

    def __enter__(self):
        import torch
        from threadpoolctl import threadpool_limits
        self.n = len(os.sched_getaffinity(0))
        self.prev = torch.get_num_threads()
        self.limits = threadpool_limits(limits=self.n)
        torch.set_num_threads(self.n)
        return self.n

    def __exit__(self, *exc):
        import torch
        torch.set_num_threads(self.prev)
        self.limits.restore_original_limits()
        return False


def cpu_baseline(plan, layer_dev, budget_s: float):
    """The oracle on host copies of one layer, request by request, for ~budget_s."""
    import numpy as np
    import oracle

    q = layer_dev["q"].cpu()
    kp = layer_dev["k_pool"].cpu()
    vp = layer_dev["v_pool"].cpu()
    order = np.random.default_rng(0).permutation(plan.num_requests)
    with pinned_host_threads() as n:
        t_wall0, t_cpu0 = time.perf_counter(), time.process_time()
        done = 0
        while True:
            r = int(order[done % plan.num_requests])
            oracle.shared_prefix_decode(q, kp, vp, kp, vp, plan.prefix_tables, plan.prefix_lens,
                                        plan.suffix_tables, plan.suffix_lens, plan.group_ids,
                                        plan.sm_scale, requests=[r],
                                        prefix_parents=plan.prefix_parents if plan.nested else None)
            done += 1
            wall = time.perf_counter() - t_wall0
            if wall >= budget_s:
                break
        cpu = time.process_time() - t_cpu0
    return {
        "value": round(done / wall, 3),
        "unit": "req/s per layer",
        "cores": n,
        "threads_note": "BLAS/OpenMP and torch thread pools pinned to the process's CPU affinity",
        "cpu_time_per_wall": round(cpu / wall, 2),
        **host_info(),
        "kind": "oracle",
        "sample": f"{done} random requests of layer 0 of the same workload, one oracle call each, "
                  f"{wall:.1f} s wall, {cpu:.1f} s CPU",
    }


def prefill_work(plan, query_rows):
    """Keys seen by all rows of a prefill call, split into prefix and own keys.
    Row j of request r sits at own position p = S_r - Q_r + j and sees the
    chain's prefix tokens plus own tokens 0..p."""
    pre = own = 0
    for r in range(plan.num_requests):
        g = int(plan.group_ids[r])
        P = plan.chain_prefix_len(g) if g >= 0 else 0
        S, Q = int(plan.suffix_lens[r]), int(query_rows[r])
        pre += Q * P
        own += S * (S + 1) // 2 - (S - Q) * (S - Q + 1) // 2
    return pre, own


def cpu_prefill_baseline(plan, q_rows, offsets, layer_dev, budget_s: float):
    """The oracle on host copies of one layer, one prefill row at a time, for
    ~budget_s (rows drawn at random over the whole batch)."""
    import numpy as np
    import oracle

    q = q_rows.cpu()
    kp = layer_dev["k_pool"].cpu()
    vp = layer_dev["v_pool"].cpu()
    T = int(offsets[-1])
    order = np.random.default_rng(0).permutation(T)
    with pinned_host_threads() as n:
        t_wall0, t_cpu0 = time.perf_counter(), time.process_time()
        done = 0
        while True:
            t = int(order[done % T])
            oracle.shared_prefix_prefill(q, offsets, kp, vp, kp, vp, plan.prefix_tables,
                                         plan.prefix_lens, plan.suffix_tables, plan.suffix_lens,
                                         plan.group_ids, plan.sm_scale, rows=[t],
                                         prefix_parents=plan.prefix_parents if plan.nested else None)
            done += 1
            wall = time.perf_counter() - t_wall0
            if wall >= budget_s:
                break
        cpu = time.process_time() - t_cpu0
    return {
        "value": round(done / wall, 3),
        "unit": "rows/s per layer",
        "cores": n,
        "cpu_time_per_wall": round(cpu / wall, 2),
        **host_info(),
        "kind": "oracle",
        "sample": f"{done} random query rows of one layer of the same workload, one oracle "
                  f"call each, {wall:.1f} s wall, {cpu:.1f} s CPU",
    }


# ------------------------------------------------------------------ ceilings
def read_ceiling(torch, gib: int = 4, reps: int = 3) -> dict:
    """Read-only HBM bandwidth from the library's read probe (16-byte
    nontemporal loads over a buffer 16x the Infinity Cache), best over its
    access orders and a few launch shapes."""
    from paper_2405_19888_amd import parrot_hbm_read_ceiling
    nbytes = gib << 30
    buf = torch.ones(nbytes // 4, dtype=torch.int32, device="cuda")
    sink = torch.zeros(1, dtype=torch.int32, device="cuda")
    cus = torch.cuda.get_device_properties(0).multi_processor_count
    stream = torch.cuda.current_stream()
    best, trials = None, []
    for spans in (True, False):
        for wpc in (1, 2, 4, 8):
            for unroll in (4, 8, 16):
                parrot_hbm_read_ceiling(buf, sink, cus * wpc, unroll, spans, stream=stream)
                e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
                e0.record(stream)
                for _ in range(reps):
                    parrot_hbm_read_ceiling(buf, sink, cus * wpc, unroll, spans, stream=stream)
                e1.record(stream)
                e1.synchronize()
                gbps = reps * nbytes / (e0.elapsed_time(e1) * 1e-3) / 1e9
                trials.append({"order": "wave_spans" if spans else "grid_stride",
                               "workgroups_per_cu": wpc, "loads_per_thread": unroll,
                               "gbps": round(gbps, 1)})
                if best is None or gbps > best["gbps"]:
                    best = trials[-1]
    del buf
    torch.cuda.empty_cache()
    return {"read_gbps": best["gbps"], "read_best_shape": best, "read_trials": trials,
            "read_note": f"parrot_hbm_read_ceiling over {gib} GiB, {reps} passes per shape, "
                         f"HIP events on the launch stream"}


def read_probe_same_bytes(torch, nbytes: int, steps: int = 48) -> dict:
    """The read probe over exactly ``nbytes`` (a stream's own byte count),
    cycling distinct cold buffers, each launch timed with events attached to
    it as the decode kernels are; best shape.  A short stream pays its start
    and drain once per launch whatever reads it, so this is the read ceiling
    at that size."""
    import numpy as np
    from paper_2405_19888_amd import ParrotTrace, parrot_hbm_read_ceiling
    n = nbytes // 4096 * 4096
    copies = max(2, min(8, (1536 << 20) // max(n, 1)))
    bufs = [torch.ones(n // 4, dtype=torch.int32, device="cuda") for _ in range(copies)]
    sink = torch.zeros(1, dtype=torch.int32, device="cuda")
    cus = torch.cuda.get_device_properties(0).multi_processor_count
    stream = torch.cuda.current_stream()
    best = None
    for spans in (True, False):
        for wpc in (1, 2):
            for unroll in (8, 16):
                evs = [[torch.cuda.Event(enable_timing=True) for _ in range(4)] for _ in range(steps)]
                for e in evs:
                    for x in e:
                        x.record(stream)
                torch.cuda.synchronize()
                trs = [ParrotTrace(*[x.cuda_event for x in e]) for e in evs]
                for i in range(copies):
                    parrot_hbm_read_ceiling(bufs[i], sink, cus * wpc, unroll, spans, stream=stream)
                for i in range(steps):
                    parrot_hbm_read_ceiling(bufs[i % copies], sink, cus * wpc, unroll, spans,
                                            stream=stream, trace=trs[i])
                torch.cuda.synchronize()
                us = float(np.median([e[0].elapsed_time(e[1]) * 1e3 for e in evs]))
                if best is None or us < best["us"]:
                    best = {"us": round(us, 3), "order": "wave_spans" if spans else "grid_stride",
                            "workgroups_per_cu": wpc, "loads_per_thread": unroll}
    del bufs
    torch.cuda.empty_cache()
    best["bytes"] = n
    best["gbps"] = round(n / (best["us"] * 1e-6) / 1e9, 1)
    best["note"] = (f"parrot_hbm_read_ceiling over {n} bytes ({copies} cold buffers cycled), "
                    "median launch time by attached events, best shape")
    return best


def mfma_issue_ceiling(torch, vx4_list=(0, 11), waves_per_simd: int = 3, iters: int = 12000,
                       reps: int = 5) -> dict:
    """The matrix cores' issue rate from the library's register-only probe
    (16x16x32 fp16 MFMAs, with vx4 / 4 vector instructions issued per MFMA),
    on every SIMD at the prefill tile's occupancy; median of `reps` launches
    of about the prefill kernel's length (so the clock is the one a sustained
    matrix-core load holds), each timed by events attached to it."""
    from paper_2405_19888_amd import ParrotTrace, parrot_mfma_issue_ceiling
    cus = torch.cuda.get_device_properties(0).multi_processor_count
    wgs = cus * waves_per_simd                   # 4 waves per workgroup, one per SIMD
    sink = torch.zeros(1, dtype=torch.int32, device="cuda")
    stream = torch.cuda.current_stream()
    out = {}
    for vx4 in vx4_list:
        parrot_mfma_issue_ceiling(sink, wgs, iters, vx4, stream=stream)   # clocks up
        times = []
        for _ in range(reps):
            e = [torch.cuda.Event(enable_timing=True) for _ in range(4)]
            for x in e:
                x.record(stream)
            torch.cuda.synchronize()
            parrot_mfma_issue_ceiling(sink, wgs, iters, vx4, stream=stream,
                                      trace=ParrotTrace(*[x.cuda_event for x in e]))
            torch.cuda.synchronize()
            times.append(e[0].elapsed_time(e[1]))
        ms = sorted(times)[len(times) // 2]
        flops = wgs * 4 * iters * 8 * 16384
        out[f"vector_per_mfma_{vx4 / 4:g}"] = round(flops / (ms * 1e-3) / 1e12, 1)
    return out


def copy_ceiling(torch, mib: int = 1024, reps: int = 5) -> float:
    """Read + write GB/s of a plain device-to-device copy (measured in the
    same process; a copy both reads and writes, so it is not the read
    ceiling)."""
    src = torch.ones(mib << 19, dtype=torch.float16, device="cuda")
    dst = torch.empty_like(src)
    dst.copy_(src)
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record()
    for _ in range(reps):
        dst.copy_(src)
    e1.record()
    e1.synchronize()
    gbps = 2 * reps * src.numel() * 2 / (e0.elapsed_time(e1) * 1e-3) / 1e9
    del src, dst
    torch.cuda.empty_cache()
    return gbps


# ------------------------------------------------------------------ decode
def problem_of(plan, flat=None):
    from paper_2405_19888_amd import problem_from_host
    from workloads.gen import TORCH_DTYPES
    p = flat or plan
    return problem_from_host(
        num_heads=p.heads, head_dim=p.head_dim, block_size=p.block_size,
        dtype=TORCH_DTYPES[p.dtype], sm_scale=p.sm_scale, group_ids=p.group_ids,
        prefix_lens=p.prefix_lens, suffix_lens=p.suffix_lens,
        prefix_table_stride=p.prefix_tables.shape[1],
        suffix_table_stride=p.suffix_tables.shape[1],
        num_prefix_blocks=p.num_blocks, num_suffix_blocks=p.num_blocks,
        prefix_parents=p.prefix_parents if (flat is None and p.nested) else None)


def decode_leg(cfg_name: str, steps: int, warmup: int, one_layer_copies: int, trace_every: int,
               baselines: bool, read_gbps: float | None, trace: bool = True, keep_layers=False):
    """Time parrot_shared_prefix_decode on a decode workload.  Returns (the
    leg's JSON object, the plan, the device layers if `keep_layers`)."""
    import numpy as np
    import torch
    from paper_2405_19888_amd import (Decoder, ParrotTrace, parrot_validate_inputs,
                                      parrot_validate_nested_inputs)
    from workloads import get_config, make_device_layer, make_plan

    cfg = get_config(cfg_name)
    plan = make_plan(cfg)
    dev = "cuda"
    # A multi-layer workload cycles through all of its layers (each with its
    # own KV, all resident); a one-layer workload cycles distinct-KV copies so
    # that every call reads cold HBM.
    n_layers = cfg.layers if cfg.layers > 1 else one_layer_copies
    layers = [make_device_layer(plan, l, dev, seed=cfg.seed) for l in range(n_layers)]
    prob = problem_of(plan)
    scratch = torch.zeros(16, dtype=torch.int32, device=dev)
    t0 = layers[0]
    if plan.nested:
        parrot_validate_nested_inputs(prob, t0["prefix_tables"], t0["prefix_lens"],
                                      t0["prefix_parents"], t0["suffix_tables"], t0["suffix_lens"],
                                      t0["group_ids"], scratch)
    else:
        parrot_validate_inputs(prob, t0["prefix_tables"], t0["prefix_lens"], t0["suffix_tables"],
                               t0["suffix_lens"], t0["group_ids"], scratch)
    dec = Decoder(prob, device=dev)
    stream = torch.cuda.current_stream()
    ab = algorithmic_bytes(plan)
    K, W, L = steps, warmup, n_layers
    names = ("partials", "merge")
    nested = plan.nested
    flat = flat_layers = flat_dec = None
    new_kv = None
    if nested:
        # baselines for nested groups: the flat entry points on the same blocks,
        # each group's chain of prefixes laid end to end as one flat prefix
        from workloads.gen import flatten_nested
        flat = flatten_nested(plan)
        ints = {k: torch.from_numpy(np.ascontiguousarray(v)).to(dev)
                for k, v in (("prefix_tables", flat.prefix_tables), ("prefix_lens", flat.prefix_lens),
                             ("group_ids", flat.group_ids))}
        flat_layers = [dict(t, **ints) for t in layers]
        flat_dec = Decoder(problem_of(plan, flat), device=dev)

    def run(shared: bool, trace: bool, flat_baseline: bool = False, append: bool = False,
            inputs=None, steps=None, every=None):
        """W untimed steps, then K timed steps; every `every`-th timed step
        carries per-kernel (start, stop) event pairs when `trace` is set."""
        K = steps or K_default
        if inputs is not None:
            calls = [dec.bind(t, shared=shared, stream=stream, nested=nested) for t in inputs]
        elif nested and (flat_baseline or not shared):
            calls = [flat_dec.bind(flat_layers[l], shared=shared, stream=stream) for l in range(L)]
        elif append:
            calls = [dec.bind(dict(layers[l], k_new=new_kv[l][0], v_new=new_kv[l][1]),
                              stream=stream, append=True) for l in range(L)]
        else:
            calls = [dec.bind(layers[l], shared=shared, stream=stream, nested=nested)
                     for l in range(L)]
        every = max(1, every or trace_every)
        traced = list(range(0, K, every)) if trace else []
        events = {i: [torch.cuda.Event(enable_timing=True) for _ in range(4)] for i in traced}
        for evs in events.values():       # materialise the events outside the timed region
            for e in evs:
                e.record(stream)
        torch.cuda.synchronize()
        traces = {i: ParrotTrace(*[e.cuda_event for e in evs]) for i, evs in events.items()}
        n = len(calls)
        for i in range(W):
            calls[i % n]()
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        for i in range(K):
            calls[i % n](traces.get(i))
        torch.cuda.synchronize()
        wall = time.perf_counter() - t0
        per = None
        if trace:
            per = {}
            for k, name in enumerate(names):
                us = np.array([evs[2 * k].elapsed_time(evs[2 * k + 1]) * 1e3 for evs in events.values()])
                per[name + "_us"] = float(us.mean())
                per[name + "_pct"] = [round(float(x), 3) for x in np.percentile(us, [10, 50, 90])]
            per["traced_steps"] = len(events)
        return wall, per

    K_default = K
    wall, per = run(shared=True, trace=trace)
    R = plan.num_requests
    result = {
        "value": round(R / (wall / K), 1),
        "unit": "req/s",
        "steps": K,
        "warmup": W,
        "ms_per_step": round(wall / K * 1e3, 5),
        "dtype": DTYPE_TAG[plan.dtype],
        "config": {
            "workload": cfg.name, "requests": R, "heads": plan.heads, "head_dim": plan.head_dim,
            "prefix_groups": plan.num_groups, "group_sizes": plan.group_sizes(),
            **({"prefix_parents": [int(x) for x in plan.prefix_parents]} if nested else {}),
            "prefix_lens": [int(x) for x in plan.prefix_lens],
            "suffix_len_mean": round(float(plan.suffix_lens.mean()), 1),
            "ungrouped": int((plan.group_ids < 0).sum()),
            "kv_block": plan.block_size, "kv_dtype": DTYPE_TAG[plan.dtype],
            "layers": cfg.layers, "layers_cycled": L,
            "timing": "HBM-resident inputs, distinct KV per cycled layer",
        },
        "algorithmic_bytes_per_step": ab["shared_total"],
        "hbm_gbps": round(ab["shared_total"] / (wall / K) / 1e9, 1),
    }
    result["hbm_frac"] = round(result["hbm_gbps"] / HBM_PEAK_GBPS, 4)
    if per is not None:
        # dominant kernel: the partial-result kernel (prefix-group and split-KV roles)
        part_bytes = ab["prefix_kv"] + ab["suffix_kv"] + ab["q"]
        achieved = part_bytes / (per["partials_us"] * 1e-6) / 1e9
        result["roofline"] = {
            "kernel": "k_partials (prefix-group MFMA role + split-KV role)",
            "bound": "hbm", "achieved": round(achieved, 1), "peak": HBM_PEAK_GBPS,
            "unit": "GB/s", "frac": round(achieved / HBM_PEAK_GBPS, 4),
            "traffic": traffic_from_counters(cfg.name),
            "algorithmic_bytes": part_bytes,
            "avg_us": round(per["partials_us"], 3),
        }
        if read_gbps:
            result["roofline"]["frac_of_read_ceiling"] = round(achieved / read_gbps, 4)
        result["kernels_us"] = {k: round(v, 3) for k, v in per.items() if k.endswith("_us")}
        result["kernels_us"].update({k.replace("_pct", "_p10_p50_p90_us"): v
                                     for k, v in per.items() if k.endswith("_pct")})
        result["kernels_us"]["traced_steps"] = per["traced_steps"]
        if ab["prefix_flops"] > 0:
            intensity = ab["prefix_flops"] / ab["prefix_kv"]
            result["prefix_mfma"] = {
                "flops": ab["prefix_flops"],
                "flop_per_byte": round(intensity, 2),
                "util_over_partials_kernel": round(ab["prefix_flops"] / (per["partials_us"] * 1e-6) / 1e12
                                                   / MFMA_F16_PEAK_TFLOPS, 5),
                "util_ceiling_at_hbm_peak": round(min(1.0, intensity * HBM_PEAK_GBPS / 1e3
                                                      / MFMA_F16_PEAK_TFLOPS), 5),
            }
    if baselines and per is not None and int(plan.suffix_lens.min()) > 0:
        # The roles one at a time, on the same blocks (the kernel runs both
        # roles side by side, so its events cannot split them):
        #  * suffix + merge: every request ungrouped, so the partial-result
        #    kernel streams only the own tokens, then the merge;
        #  * prefix: grouped requests with no own tokens (ungrouped ones keep
        #    one), so the kernel is the prefix-group role.
        ungrouped = torch.full((R,), -1, dtype=torch.int32, device=dev)
        slen_p = torch.from_numpy(np.where(plan.group_ids >= 0, 0, 1).astype(np.int32)).to(dev)
        n_roles = min(K, 400)
        _, per_s = run(shared=True, trace=True, steps=n_roles, every=4,
                       inputs=[dict(t, group_ids=ungrouped) for t in layers])
        _, per_p = run(shared=True, trace=True, steps=n_roles, every=4,
                       inputs=[dict(t, suffix_lens=slen_p) for t in layers])
        suffix_bytes = ab["suffix_kv"] + ab["q"] + ab["out"] + ab["lse"]
        sm_us = per_s["partials_us"] + per_s["merge_us"]
        sm_gbps = suffix_bytes / (sm_us * 1e-6) / 1e9
        roles = {
            "suffix_merge": {
                "partials_us": round(per_s["partials_us"], 3), "merge_us": round(per_s["merge_us"], 3),
                "algorithmic_bytes": suffix_bytes,
                "gbps": round(sm_gbps, 1),
                "frac_of_hbm_peak": round(sm_gbps / HBM_PEAK_GBPS, 4),
                "partials_frac_of_hbm_peak": round((ab["suffix_kv"] + ab["q"]) / (per_s["partials_us"] * 1e-6)
                                                   / 1e9 / HBM_PEAK_GBPS, 4),
                "note": "the same call with every request ungrouped (own tokens only): "
                        "partial-result kernel + merge, kernel events",
            },
        }
        if read_gbps:
            roles["suffix_merge"]["frac_of_read_ceiling"] = round(sm_gbps / read_gbps, 4)
        # the same own-token bytes read by the read probe: what a plain read
        # of that size achieves, start and drain included
        probe = read_probe_same_bytes(torch, ab["suffix_kv"])
        probe["partials_speed_vs_probe"] = round(probe["us"] / per_s["partials_us"], 4)
        roles["suffix_merge"]["read_probe_same_bytes"] = probe
        if ab["prefix_flops"] > 0:
            pre_us = per_p["partials_us"]
            roles["prefix"] = {
                "partials_us": round(pre_us, 3),
                "algorithmic_bytes": ab["prefix_kv"] + ab["q"],
                "gbps": round((ab["prefix_kv"] + ab["q"]) / (pre_us * 1e-6) / 1e9, 1),
                "mfma_util": round(ab["prefix_flops"] / (pre_us * 1e-6) / 1e12 / MFMA_F16_PEAK_TFLOPS, 5),
                "mfma_util_ceiling_at_hbm_peak": round(min(1.0, ab["prefix_flops"] / ab["prefix_kv"]
                                                           * HBM_PEAK_GBPS / 1e3 / MFMA_F16_PEAK_TFLOPS), 5),
                "note": "the same call with grouped requests holding no own tokens: the "
                        "prefix-group role alone, kernel events",
            }
        result["roles"] = roles
        # warm: one layer's KV reused by every call (it stays partly in the
        # 256 MB Infinity Cache); the headline cycles distinct-KV layers
        wall_w, _ = run(shared=True, trace=False, steps=n_roles, inputs=[layers[0]])
        result["warm"] = {"ms_per_step": round(wall_w / n_roles * 1e3, 5),
                          "value": round(R / (wall_w / n_roles), 1),
                          "note": "one layer's KV reused by every call"}

    if baselines:
        if nested:
            wall_f, _ = run(shared=True, trace=False, flat_baseline=True)
            flat_bytes = (int(flat.prefix_lens.sum()) * 2 * plan.heads * plan.head_dim
                          * ELT_BYTES[plan.dtype] + ab["shared_total"] - ab["prefix_kv"])
            result["flat_sharing_baseline"] = {
                "value": round(R / (wall_f / K), 1), "unit": "req/s",
                "ms_per_step": round(wall_f / K * 1e3, 5),
                "speedup_of_nested": round(wall_f / wall, 3),
                "hbm_gbps": round(flat_bytes / (wall_f / K) / 1e9, 1),
                "note": "parrot_shared_prefix_decode with each group's prefix chain as one flat prefix",
            }
        else:
            # decode with append: the same step, with this step's K/V written
            # into the cache by the partial-result kernel (the values equal
            # what the slots already hold, so later steps see the same data)
            last = [(r, int(plan.suffix_tables[r][(int(plan.suffix_lens[r]) - 1) // plan.block_size]),
                     (int(plan.suffix_lens[r]) - 1) % plan.block_size)
                    for r in range(R) if plan.suffix_lens[r] > 0]
            rows = torch.tensor([x[0] for x in last], device=dev, dtype=torch.long)
            blks = torch.tensor([x[1] for x in last], device=dev, dtype=torch.long)
            slots = torch.tensor([x[2] for x in last], device=dev, dtype=torch.long)
            new_kv = []
            for t in layers:
                pair = []
                for name in ("k_pool", "v_pool"):
                    x = torch.zeros((R, plan.heads, plan.head_dim), dtype=t["q"].dtype, device=dev)
                    x[rows] = t[name][blks, :, slots]
                    pair.append(x)
                new_kv.append(pair)
            wall_a, _ = run(shared=True, trace=False, append=True)
            result["append_step"] = {
                "ms_per_step": round(wall_a / K * 1e3, 5),
                "overhead_vs_plain": round(wall_a / wall - 1.0, 4),
                "note": "parrot_shared_prefix_decode_append on the same workload",
            }
            del new_kv
        wall_n, _ = run(shared=False, trace=False)
        result["per_request_baseline"] = {
            "value": round(R / (wall_n / K), 1), "unit": "req/s",
            "ms_per_step": round(wall_n / K * 1e3, 5),
            "speedup_of_shared": round(wall_n / wall, 3),
            "hbm_gbps": round(ab["naive_total"] / (wall_n / K) / 1e9, 1),
            "byte_ratio": round(ab["naive_total"] / ab["shared_total"], 3),
        }
    kept = layers if keep_layers else None
    del dec, flat_dec, flat_layers
    if not keep_layers:
        del layers
        torch.cuda.empty_cache()
    return result, plan, kept


def sweep_leg(lens, steps: int, warmup: int, copies: int) -> dict:
    """Shared path against the per-request path on the LLaMA-7B one-group
    shape for each prefix length (speedup as a function of prefix length)."""
    import torch
    from paper_2405_19888_amd import Decoder
    from workloads import get_config, make_device_layer, make_plan

    out = {}
    stream = torch.cuda.current_stream()
    for P in lens:
        cfg = get_config(f"sweep_p{P}")
        plan = make_plan(cfg)
        layers = [make_device_layer(plan, l, "cuda", seed=cfg.seed) for l in range(copies)]
        dec = Decoder(problem_of(plan))
        ab = algorithmic_bytes(plan)
        times = {}
        for shared in (True, False):
            calls = [dec.bind(t, shared=shared, stream=stream) for t in layers]
            for i in range(warmup):
                calls[i % copies]()
            torch.cuda.synchronize()
            t0 = time.perf_counter()
            for i in range(steps):
                calls[i % copies]()
            torch.cuda.synchronize()
            times[shared] = (time.perf_counter() - t0) / steps
        out[str(P)] = {"shared_us": round(times[True] * 1e6, 2),
                       "per_request_us": round(times[False] * 1e6, 2),
                       "speedup": round(times[False] / times[True], 3),
                       "byte_ratio": round(ab["naive_total"] / ab["shared_total"], 3),
                       "shared_hbm_frac": round(ab["shared_total"] / times[True] / 1e9 / HBM_PEAK_GBPS, 4)}
        del layers, dec
        torch.cuda.empty_cache()
    sp = [out[str(P)]["speedup"] for P in lens]
    return {"workload": "llama7b_g32_p<P>: 32 heads x 128, fp16, 1 group of 32, own U[64,512]",
            "steps": steps, "layers_cycled": copies, "points": out,
            "speedup_monotonic_in_prefix_len": all(b > a for a, b in zip(sp, sp[1:]))}


# ------------------------------------------------------------------ prefill
def prefill_leg(cfg_name: str, steps: int, warmup: int, n_layers: int, baselines: bool,
                cpu_budget: float) -> dict:
    """Time parrot_shared_prefix_prefill on a prefill workload: `steps` calls,
    each one layer's Fill of every request's new rows, cycling `n_layers`
    distinct-KV layers.  Returns the leg's JSON object."""
    import numpy as np
    import torch
    from paper_2405_19888_amd import (ParrotTrace, Prefiller, parrot_prefill_single_pass,
                                      parrot_validate_prefill_inputs)
    from paper_2405_19888_amd import prefill_rows_from_host
    from workloads import (get_config, make_device_layer, make_device_prefill_queries, make_plan,
                           one_group_per_request, prefill_rows)

    cfg = get_config(cfg_name)
    if cfg.prefill_rows is None:
        raise SystemExit(f"{cfg_name} is not a prefill workload")
    plan = make_plan(cfg)
    qr = prefill_rows(plan, cfg.prefill_rows, None)
    dev = "cuda"
    layers = []
    for l in range(n_layers):
        t = make_device_layer(plan, l, dev, seed=cfg.seed)
        t["q_rows"], t["query_offsets"] = make_device_prefill_queries(plan, qr, dev, cfg.seed, l)
        layers.append(t)
    offsets = layers[0]["query_offsets"].cpu().numpy()

    def setup(p):
        rows = prefill_rows_from_host(offsets, p.group_ids, p.num_groups,
                                      p.prefix_parents if p.nested else None)
        return problem_of(p), rows

    prob, rows = setup(plan)
    scratch = torch.zeros(16, dtype=torch.int32, device=dev)
    t0 = layers[0]
    parrot_validate_prefill_inputs(prob, rows, t0["query_offsets"], t0["prefix_tables"],
                                   t0["prefix_lens"], t0["prefix_parents"] if plan.nested else None,
                                   t0["suffix_tables"], t0["suffix_lens"], t0["group_ids"], scratch)
    pre = Prefiller(prob, rows, device=dev)
    single = parrot_prefill_single_pass(prob, rows, nested=plan.nested)
    stream = torch.cuda.current_stream()

    def timed(calls, trace: bool):
        events = [[torch.cuda.Event(enable_timing=True) for _ in range(4)] for _ in range(steps)] \
            if trace else []
        for evs in events:
            for e in evs:
                e.record(stream)
        torch.cuda.synchronize()
        traces = [ParrotTrace(*[e.cuda_event for e in evs]) for evs in events]
        for i in range(warmup):
            calls[i % len(calls)]()
        torch.cuda.synchronize()
        w0 = time.perf_counter()
        for i in range(steps):
            calls[i % len(calls)](traces[i] if trace else None)
        torch.cuda.synchronize()
        wall = time.perf_counter() - w0
        per = None
        if trace:
            per = {"prefill_us": sum(e[0].elapsed_time(e[1]) for e in events) * 1e3 / steps}
            if not single:
                per["merge_us"] = sum(e[2].elapsed_time(e[3]) for e in events) * 1e3 / steps
        return wall, per

    calls = [pre.bind(t, stream=stream, nested=plan.nested) for t in layers]
    wall, per = timed(calls, trace=False)
    _, per = timed(calls, trace=True)
    T = int(offsets[-1])
    pre_keys, own_keys = prefill_work(plan, qr)
    flops = 4 * plan.head_dim * plan.heads * (pre_keys + own_keys)
    achieved = flops / (per["prefill_us"] * 1e-6) / 1e12
    out = {
        "metric": "prefill query rows/sec per layer",
        "value": round(T / (wall / steps), 1), "unit": "rows/s",
        "steps": steps, "warmup": warmup, "ms_per_step": round(wall / steps * 1e3, 5),
        "dtype": DTYPE_TAG[plan.dtype],
        "config": {"workload": cfg.name, "requests": plan.num_requests, "rows": T,
                   "heads": plan.heads, "head_dim": plan.head_dim,
                   "prefix_lens": [int(x) for x in plan.prefix_lens],
                   "rows_per_request_mean": round(float(np.mean(qr)), 1),
                   "own_len_mean": round(float(plan.suffix_lens.mean()), 1),
                   "layers_cycled": n_layers},
        "plan": ("single pass: one kernel, no partial results, no merge" if single else
                 "split: prefix and own partial results, then the merge kernel"),
        "roofline": {
            "kernel": ("k_prefill single pass (group tiles: the prefix, then their rows' own "
                       "tokens; MFMA)" if single else
                       "k_prefill (prefix items + causal own items, MFMA)"),
            "bound": "mfma", "achieved": round(achieved, 1), "peak": MFMA_F16_PEAK_TFLOPS,
            "unit": "TFLOP/s", "frac": round(achieved / MFMA_F16_PEAK_TFLOPS, 4),
            "traffic": traffic_from_counters(cfg.name, PREFILL_COUNTERS_FILE, PREFILL_SOURCES),
            "algorithmic_flops": flops,
            "avg_us": round(per["prefill_us"], 3),
        },
        "kernels_us": {k: round(v, 3) for k, v in per.items()},
        "tflops_step": round(flops / (wall / steps) / 1e12, 1),
    }
    # what the matrix cores issue on this box alone and with the tile's share
    # of vector work (about 2.75 vector instructions per MFMA: the softmax)
    issue = mfma_issue_ceiling(torch)
    mixed = issue["vector_per_mfma_2.75"]
    out["roofline"]["issue_ceiling_tflops"] = issue
    out["roofline"]["frac_of_issue_ceiling"] = round(achieved / mixed, 4)
    out["roofline"]["issue_note"] = ("parrot_mfma_issue_ceiling: registers only, 3 waves per SIMD "
                                     "(the tile's occupancy), 16x16x32 fp16 MFMAs alone and with "
                                     "2.75 vector instructions per MFMA between them")
    if baselines:
        # no sharing: each request its own group (same kernels and blocks)
        solo = one_group_per_request(plan)
        sprob, srows = setup(solo)
        spre = Prefiller(sprob, srows, device=dev)
        ints = {k: torch.from_numpy(np.ascontiguousarray(v)).to(dev)
                for k, v in (("prefix_tables", solo.prefix_tables), ("prefix_lens", solo.prefix_lens),
                             ("group_ids", solo.group_ids))}
        scalls = [spre.bind(dict(t, **ints), stream=stream) for t in layers]
        wall_s, _ = timed(scalls, trace=False)
        out["per_request_baseline"] = {
            "value": round(T / (wall_s / steps), 1), "unit": "rows/s",
            "ms_per_step": round(wall_s / steps * 1e3, 5),
            "speedup_of_shared": round(wall_s / wall, 3),
            "note": "the same entry point with one group per request (prefix rows not stacked "
                    "across requests)",
        }
        if cpu_budget > 0:
            out["cpu_baseline"] = cpu_prefill_baseline(plan, layers[0]["q_rows"], offsets,
                                                       layers[0], cpu_budget)
    del layers, pre
    torch.cuda.empty_cache()
    return out


SUB_KEYS = ("value", "unit", "ms_per_step", "dtype", "hbm_gbps", "hbm_frac", "roofline",
            "kernels_us", "prefix_mfma", "roles", "per_request_baseline", "flat_sharing_baseline",
            "append_step", "warm", "algorithmic_bytes_per_step")


def main():
    ap = argparse.ArgumentParser(description=__doc__.split("\n")[0])
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=1000)
    ap.add_argument("--warmup", type=int, default=50)
    ap.add_argument("--config", default="c5", help="headline decode workload (default: the "
                                                   "32-layer mixed serving step)")
    ap.add_argument("--layers", type=int, default=8,
                    help="distinct-KV copies cycled by one-layer workloads")
    ap.add_argument("--cpu-budget", type=float, default=15.0, help="seconds of oracle timing")
    ap.add_argument("--no-baselines", action="store_true",
                    help="skip the per-request, role, append and CPU legs")
    ap.add_argument("--no-trace", action="store_true", help="time without per-kernel events")
    ap.add_argument("--copy-mib", type=int, default=0,
                    help="first run three plain device copies of this many MiB (a known-size "
                         "kernel for scaling rocprofv3 FETCH_SIZE / WRITE_SIZE counters)")
    ap.add_argument("--trace-every", type=int, default=16,
                    help="attach per-kernel HIP events to every N-th timed step (each traced "
                         "launch costs a few microseconds of stream time)")
    ap.add_argument("--workloads", default="c2,c3,c4,nested",
                    help="other decode workloads measured after the headline ('none' to skip)")
    ap.add_argument("--sub-steps", type=int, default=400, help="timed steps per other workload")
    ap.add_argument("--sweep", default=SWEEP_DEFAULT,
                    help="prefix lengths of the sweep ('none' to skip)")
    ap.add_argument("--prefill", default="prefill",
                    help="prefill workload timed after the decode legs ('none' to skip)")
    ap.add_argument("--prefill-steps", type=int, default=20)
    ap.add_argument("--no-ceilings", action="store_true", help="skip the read and copy ceilings")
    ap.add_argument("--mode", choices=("decode", "prefill"), default="decode",
                    help="prefill: time only the prefill workload (--prefill) and print its line")
    args = ap.parse_args()

    if args.gpus != 1:
        print(json.dumps({"error": "this benchmark measures one GPU: run with --gpus 1 "
                                   "(no multi-GPU path exists)"}))
        sys.exit(2)

    import torch
    if args.copy_mib > 0:
        n = args.copy_mib << 19                      # fp16 elements in that many MiB
        src = torch.ones(n, dtype=torch.float16, device="cuda")
        dst = torch.empty_like(src)
        for _ in range(3):
            dst.copy_(src)
        torch.cuda.synchronize()
        del src, dst
        torch.cuda.empty_cache()

    if args.mode == "prefill":
        leg = prefill_leg(args.prefill, args.steps, args.warmup, min(args.layers, 4),
                          not args.no_baselines, args.cpu_budget)
        leg.update(n_gpus=1, higher_is_better=True, scaling="weak", vs_baseline=None,
                   data="synthetic")
        print(json.dumps(leg), flush=True)
        return

    ceilings = {}
    if not args.no_ceilings:
        ceilings = read_ceiling(torch)
        ceilings["copy_gbps"] = round(copy_ceiling(torch), 1)
        ceilings["copy_note"] = "device-to-device copy of 1 GiB, read + write bytes per second"
    read_gbps = ceilings.get("read_gbps")

    head, plan, layers = decode_leg(args.config, args.steps, args.warmup, args.layers,
                                    args.trace_every, not args.no_baselines, read_gbps,
                                    trace=not args.no_trace, keep_layers=True)
    result = {
        "metric": "decode-attention requests/sec per layer",
        "value": head["value"], "unit": "req/s", "n_gpus": 1,
        "steps": args.steps, "warmup": args.warmup, "ms_per_step": head["ms_per_step"],
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None,
        "dtype": head["dtype"], "data": "synthetic", "config": head["config"],
    }
    result.update({k: head[k] for k in SUB_KEYS if k in head and k not in result})
    if ceilings:
        result["ceilings"] = ceilings
    if not args.no_baselines and args.cpu_budget > 0:
        result["cpu_baseline"] = cpu_baseline(plan, layers[0], args.cpu_budget)
    del layers
    torch.cuda.empty_cache()

    if args.workloads != "none":
        result["workloads"] = {}
        for name in [w for w in args.workloads.split(",") if w]:
            leg, _, _ = decode_leg(name, args.sub_steps, min(args.warmup, 20), args.layers,
                                   args.trace_every, not args.no_baselines, read_gbps,
                                   trace=not args.no_trace)
            sub = {k: leg[k] for k in SUB_KEYS if k in leg}
            sub["config"] = leg["config"]
            result["workloads"][leg["config"]["workload"]] = sub
    if args.sweep != "none":
        result["sweep"] = sweep_leg([int(x) for x in args.sweep.split(",")], 300, 20, args.layers)
    if args.prefill != "none":
        # the Fill step of the same kind of batch: every forked context's own
        # prompt rows against the shared prefix (its own line object)
        result["prefill"] = prefill_leg(args.prefill, args.prefill_steps, 3, 2,
                                        not args.no_baselines, min(args.cpu_budget, 10.0))
    print(json.dumps(result), flush=True)


if __name__ == "__main__":
    main()
