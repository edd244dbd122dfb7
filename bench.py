#!/usr/bin/env python3
"""Decode throughput of the benchmarked workload on one MI355X.

Workload (synthetic, seeded): Llama-2-7B shape, bf16 weights and KV cache,
a closed batch of 32 requests with lognormal prompt lengths (median 200), a
directive level per request (prefix 0 / 8 / 12 tokens) and lognormal
generation lengths by level (medians 400 / 120 / 40); each request retires at
its own stop length.  One bench step is one full ragged decode of that batch
-- every decode step from the prefilled cache until the last request retires
-- so a step's tokens are sum(L_i - 1).  Inputs (weights, KV cache, first
tokens) are resident in HBM when the timed region starts; prefill is outside
it.

Prints one JSON line on stdout (progress goes to stderr).
"""
import argparse
import hashlib
import json
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

METRIC = "decode tokens/s + achieved HBM GB/s, Llama-2-7B-shape bf16, ragged batch 32"
PEAK_HBM_GBPS = 8000.0          # MI355X HBM3E
PEAK_BF16_TFLOPS = 2500.0       # MI355X dense bf16 MFMA
DOMINANT = "k_stream_gemm<BF16, 1, 1, EpiSwiGLU<BF16>, 2, 8, true, true>"
TRAFFIC_PROFILE = os.path.join(ROOT, "profiles", "gate_up_gemm_pmc_llama2_7b_b8.txt")


def log(*a):
    print(*a, file=sys.stderr, flush=True)


# The sources that define the dominant kernel (its template arguments fix its launch shape).
DOMINANT_SOURCES = ("device_common.h", "gemm_kernels.h")


def kernel_source_hash() -> str:
    h = hashlib.sha256()
    for f in (os.path.join(ROOT, "paper_2403_12900_amd", "csrc", n) for n in DOMINANT_SOURCES):
        with open(f, "rb") as fh:
            h.update(os.path.basename(f).encode())
            h.update(fh.read())
    return h.hexdigest()[:16]


def measured_traffic(bytes_per_launch: float):
    """HBM bytes per launch of the dominant kernel from the committed PMC summary,
    or None when its sources (DOMINANT_SOURCES) changed since the counters were taken."""
    if not os.path.exists(TRAFFIC_PROFILE):
        return None
    vals = {}
    for line in open(TRAFFIC_PROFILE):
        if "=" in line and not line.startswith("#"):
            k, v = line.split("=", 1)
            vals[k.strip()] = v.strip()
    if vals.get("kernel_source_hash") != kernel_source_hash():
        return None
    try:
        return float(vals["hbm_bytes_per_launch"])
    except (KeyError, ValueError):
        return None


PMC_COPY_BYTES = 256 << 20     # calibration copy of --traffic-probe


def traffic_probe():
    """Launches exactly what the roofline line times -- the gate/up projection at
    8 rows, rotating through the 32 layers -- plus a plain device copy of known
    size, for two rocprofv3 --pmc passes (FETCH_SIZE, then WRITE_SIZE)."""
    import torch
    from paper_2403_12900_amd.binding import DecodeModel
    from paper_2403_12900_amd.configs import CONFIGS
    m = CONFIGS["c3"].model
    torch.cuda.set_device(0)
    model = DecodeModel(m, CONFIGS["c3"].weight_seed, max_slots=8, max_ctx=64, kv_blocks=32)
    us = model.time_projection("gate_up", 8, 64)
    log(f"traffic probe: 64 gate/up launches, {us:.2f} us each")
    model.close()
    x = torch.ones(PMC_COPY_BYTES, dtype=torch.uint8, device="cuda")
    y = torch.empty_like(x)
    for _ in range(4):
        y.copy_(x)
    torch.cuda.synchronize()
    log(f"traffic probe: 4 device copies of {PMC_COPY_BYTES} bytes")


def pmc_probe():
    """Kernels for a rocprofv3 --pmc diagnosis of the projections' memory path: the dominant gate/up
    kernel, the O projection (fewest row tiles) and the plain weight stream of the read ceiling."""
    import torch
    from paper_2403_12900_amd.binding import DecodeModel
    from paper_2403_12900_amd.configs import CONFIGS
    cfg = CONFIGS["c3"]
    model = DecodeModel(cfg.model, cfg.weight_seed, max_slots=32, max_ctx=256, kv_blocks=64)
    model.time_projection("gate_up", 8, 32)
    model.time_projection("o", 8, 32)
    model.read_ceiling(2)
    torch.cuda.synchronize()
    log("pmc probe: 32 gate/up, 32 O, 2 read-ceiling passes")
    model.close()


def prefill_probe():
    """The c3 batch's prefill (8427 prompt tokens: chunks of 4096, 4096 and 235 rows), run twice,
    for a rocprofv3 --pmc diagnosis of the prefill GEMMs."""
    import torch
    from paper_2403_12900_amd.binding import DecodeModel
    from paper_2403_12900_amd.configs import CONFIGS
    from paper_2403_12900_amd.workload import make_workload
    cfg = CONFIGS["c3"]
    wl = make_workload(cfg)
    seq = [int(x) for x in wl.seq_lens]
    stops = [int(x) for x in wl.stop_lens]
    max_ctx = max(s + L - 1 for s, L in zip(seq, stops))
    blocks = sum((s + L - 1 + 15) // 16 for s, L in zip(seq, stops))
    model = DecodeModel(cfg.model, cfg.weight_seed, max_slots=wl.batch, max_ctx=max_ctx, kv_blocks=blocks)
    tok = model.new_token_buffer()
    for k in range(2):
        if k:
            for i in range(wl.batch):
                model.free_slot(i)
        model.prefill(list(range(wl.batch)), wl.tokens, stops, tok)
    torch.cuda.synchronize()
    log(f"prefill probe: 2 prefills of {sum(seq)} prompt tokens")
    model.close()


def decode_probe():
    """The c3 prefill, then one ragged decode of the batch (no timing), for a rocprofv3 --kernel-trace
    that --trace-summary breaks down by active rows."""
    import torch
    from paper_2403_12900_amd.binding import DecodeModel
    from paper_2403_12900_amd.configs import CONFIGS
    from paper_2403_12900_amd.workload import make_workload
    cfg = CONFIGS["c3"]
    wl = make_workload(cfg)
    seq = [int(x) for x in wl.seq_lens]
    stops = [int(x) for x in wl.stop_lens]
    max_ctx = max(s + L - 1 for s, L in zip(seq, stops))
    blocks = sum((s + L - 1 + 15) // 16 for s, L in zip(seq, stops))
    model = DecodeModel(cfg.model, cfg.weight_seed, max_slots=wl.batch, max_ctx=max_ctx, kv_blocks=blocks)
    tok = model.new_token_buffer()
    model.prefill(list(range(wl.batch)), wl.tokens, stops, tok)
    for act, lens in _decode_schedule(seq, stops):
        model.decode_step(act, lens, tok)
    torch.cuda.synchronize()
    log(f"decode probe: {len(_decode_schedule(seq, stops))} decode steps after the prefill")
    model.close()


def _decode_schedule(seq, stops):
    """(active requests, their cached lengths) of every decode step of a closed ragged batch."""
    return [([i for i in range(len(seq)) if stops[i] > s], [seq[i] + s - 1 for i in range(len(seq)) if stops[i] > s])
            for s in range(1, max(stops))]


def trace_summary(trace_dir: str) -> None:
    """Prints the c3 decode's kernel time by active rows from the kernel_trace.csv that rocprofv3
    wrote under trace_dir for `bench.py --decode-probe`.  Steps are split at each embedding launch;
    per launch, the algorithmic bytes are the weights (projections) or the KV read of every active
    row's cached positions and the new one (attention)."""
    import csv
    import glob
    import re
    from paper_2403_12900_amd.configs import CONFIGS
    from paper_2403_12900_amd.workload import make_workload
    paths = glob.glob(os.path.join(trace_dir, "**", "*kernel_trace.csv"), recursive=True)
    if len(paths) != 1:
        raise SystemExit(f"{trace_dir}: expected one kernel_trace.csv, found {len(paths)}")
    cfg = CONFIGS["c3"]
    m = cfg.model
    wl = make_workload(cfg)
    sched = _decode_schedule([int(x) for x in wl.seq_lens], [int(x) for x in wl.stop_lens])
    rows = []
    with open(paths[0]) as fh:
        for r in csv.DictReader(fh):
            rows.append((int(r["Start_Timestamp"]), int(r["End_Timestamp"]), r["Kernel_Name"]))
    rows.sort()
    starts = [i for i, r in enumerate(rows) if re.search(r"\bk_embed<", r[2])]
    if len(starts) < len(sched):
        raise SystemExit(f"{len(starts)} embedding launches for {len(sched)} decode steps")
    starts = starts[-len(sched):] + [len(rows)]
    d, hd, f, wb = m.d_model, m.head_dim, m.d_ff, m.weight_bytes
    wbytes = {"QKV": m.qkv_rows * d * wb, "O": d * m.n_heads * hd * wb, "gate/up": 2 * f * d * wb, "down": d * f * wb}
    kv_layer = m.kv_bytes_per_token() // m.n_layers
    roles = ["QKV", "attention", "O", "gate/up", "down"]
    bins = [("1", 1, 1), ("2-8", 2, 8), ("9-16", 9, 16), ("17-32", 17, 32)]
    acc = {b[0]: {"steps": 0, "wall": 0.0, "busy": 0.0, "kv": 0, **{r: 0.0 for r in roles}, "launches": 0}
           for b in bins}
    for k, (act, lens) in enumerate(sched):
        n = len(act)
        a = next(acc[name] for name, lo, hi in bins if lo <= n <= hi)
        step = rows[starts[k]:starts[k + 1]]
        a["steps"] += 1
        a["wall"] += (step[-1][1] - step[0][0]) / 1e3
        a["busy"] += sum(s1 - s0 for s0, s1, _ in step) / 1e3
        a["kv"] += (sum(lens) + n) * kv_layer
        resid = 0
        for s0, s1, name in step:
            us = (s1 - s0) / 1e3
            if "EpiQKV" in name:
                a["QKV"] += us
                a["launches"] += 1
            elif "k_attn_decode" in name:
                a["attention"] += us
            elif "EpiSwiGLU" in name:
                a["gate/up"] += us
            elif "EpiResid" in name:
                a["O" if resid % 2 == 0 else "down"] += us
                resid += 1
    total = sum(a["wall"] for a in acc.values())
    busy = sum(a["busy"] for a in acc.values())
    launches = len(rows) - starts[0]
    print("| active rows | steps | wall ms | " + " | ".join(roles) + " |")
    print("|---|---:|---:|" + "---|" * len(roles))
    for name, _, _ in bins:
        a = acc[name]
        if a["steps"] == 0:
            continue
        L = a["launches"]
        cells = []
        for r in roles:
            us = a[r] / L
            byts = a["kv"] / a["steps"] if r == "attention" else wbytes[r]
            cells.append(f"{us:.1f} us, {byts / us / 1e3:.0f} GB/s")
        print(f"| {name} | {a['steps']} | {a['wall'] / 1e3:.1f} | " + " | ".join(cells) + " |")
    print(f"\nAll steps: {total / 1e3:.1f} ms from each step's first launch start to its last launch end, "
          f"{busy / 1e3:.1f} ms of it in kernels: {(total - busy) / 1e3:.1f} ms between the decode's "
          f"{launches} launches ({(total - busy) / launches:.2f} us each). Per launch in the table: mean "
          f"kernel time and algorithmic GB/s.")


def stats_summary(csv_path: str, top: int = 24) -> None:
    """Prints a rocprofv3 kernel_stats.csv (--kernel-trace --stats) as a markdown table: total and
    average kernel time per kernel, the `top` kernels by total time."""
    import csv
    import re
    rows = []
    with open(csv_path) as fh:
        for r in csv.DictReader(fh):
            name = re.sub(r"\(.*", "", r["Name"]).replace("sprk::", "").strip()
            rows.append((float(r["TotalDurationNs"]), int(r["Calls"]), float(r["AverageNs"]), float(r["MinNs"]),
                         float(r["MaxNs"]), float(r["Percentage"]), name))
    rows.sort(reverse=True)
    total = sum(r[0] for r in rows)
    print(f"Total kernel time {total / 1e6:.1f} ms over {sum(r[1] for r in rows)} launches.\n")
    print("| total ms | % | calls | avg us | min us | max us | kernel |")
    print("|---:|---:|---:|---:|---:|---:|---|")
    for tot, calls, avg, mn, mx, pct, name in rows[:top]:
        print(f"| {tot / 1e6:.1f} | {pct:.2f} | {calls} | {avg / 1e3:.2f} | {mn / 1e3:.2f} | {mx / 1e3:.2f} | `{name}` |")


def step_sweep(key: str, steps: int = 12):
    """Decode-step time and algorithmic GB/s of one configuration's model at 1, 8, 16 and 32 rows of
    about 512 cached positions: the weights of every layer and the LM head, plus each row's KV read
    (its cached positions and the new one) and write."""
    import torch
    from paper_2403_12900_amd.binding import DecodeModel
    from paper_2403_12900_amd.configs import CONFIGS
    cfg = CONFIGS[key]
    m = cfg.model
    dm = DecodeModel(m, cfg.weight_seed, max_slots=32, max_ctx=512 + steps + 2, kv_blocks=32 * 34)
    tok = dm.new_token_buffer()
    rng = np.random.default_rng(0)
    wbytes = m.weight_elements_per_step() * m.weight_bytes
    kv_tok = m.kv_bytes_per_token()
    for rows in (1, 8, 16, 32):
        slots = list(range(rows))
        dm.prefill(slots, [rng.integers(0, m.vocab, size=512).astype(np.int32) for _ in range(rows)],
                   [steps + 2] * rows, tok)
        lens = [512] * rows
        dm.decode_step(slots, lens, tok)
        lens = [x + 1 for x in lens]
        torch.cuda.synchronize()
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record()
        for _ in range(steps):
            dm.decode_step(slots, lens, tok)
            lens = [x + 1 for x in lens]
        e1.record()
        torch.cuda.synchronize()
        ms = e0.elapsed_time(e1) / steps
        cached = 513 + (steps - 1) / 2         # mean cached positions per row over the timed steps
        byts = wbytes + rows * (cached + 2) * kv_tok
        log(f"{cfg.name} rows {rows:2d}: {ms:.3f} ms/step, {rows / ms * 1e3:.0f} tokens/s, "
            f"{byts / ms / 1e6:.0f} GB/s algorithmic ({byts / ms / 1e6 / PEAK_HBM_GBPS * 100:.1f}% of 8 TB/s)")
        for sl in slots:
            dm.free_slot(sl)
    dm.close()


def _pmc_rows(path: str, counter: str):
    """(kernel name, value) per dispatch from a rocprofv3 counter_collection.csv."""
    import csv
    out = []
    with open(path) as fh:
        for r in csv.DictReader(fh):
            if r.get("Counter_Name") == counter:
                out.append((r["Kernel_Name"], float(r["Counter_Value"])))
    return out


def traffic_summary(fetch_csv: str, write_csv: str) -> None:
    """Writes the committed PMC summary that measured_traffic() reads."""
    import re
    import statistics

    def norm(name):
        return re.sub(r"\(.*", "", name).replace("sprk::", "").replace("void ", "").strip()

    res = {}
    for counter, path in (("FETCH_SIZE", fetch_csv), ("WRITE_SIZE", write_csv)):
        rows = _pmc_rows(path, counter)
        k = [v for n, v in rows if norm(n) == DOMINANT]
        c = sorted((v for n, v in rows if "copy" in n.lower()), reverse=True)[:4]
        if not k or len(c) < 4:
            raise SystemExit(f"{path}: {len(k)} dispatches of {DOMINANT}, {len(c)} copies")
        res[counter] = (statistics.mean(k), len(k), statistics.mean(c))
    m_fetch, n_fetch, c_fetch = res["FETCH_SIZE"]
    m_write, n_write, c_write = res["WRITE_SIZE"]
    true_kib = PMC_COPY_BYTES / 1024.0
    s_fetch, s_write = true_kib / c_fetch, true_kib / c_write
    fetch_b = m_fetch * s_fetch * 1024.0
    write_b = m_write * s_write * 1024.0
    with open(TRAFFIC_PROFILE, "w") as fh:
        fh.write(f"""# rocprofv3 PMC summary: HBM traffic of {DOMINANT}
# (gate/up projection with SwiGLU, Llama-2-7B shape, 8 rows; each launch streams one layer's
# 180.4 MB gate/up matrix, rotating through all 32 layers).
# Commands (one MI355X; the repository at /root/repo; `cd /tmp && export TMPDIR=/tmp` first):
#   rocprofv3 --pmc FETCH_SIZE --output-format csv -d /tmp/pmc_fetch -o probe -- python3 /root/repo/bench.py --traffic-probe
#   rocprofv3 --pmc WRITE_SIZE --output-format csv -d /tmp/pmc_write -o probe -- python3 /root/repo/bench.py --traffic-probe
#   python3 /root/repo/bench.py --traffic-summary /tmp/pmc_fetch/probe_counter_collection.csv /tmp/pmc_write/probe_counter_collection.csv
# Each counter (KiB per dispatch) is scaled by the ratio true/measured of the same counter on a
# plain device copy of {PMC_COPY_BYTES} bytes (reads and writes that many bytes).
# kernel_source_hash covers the kernel's sources: csrc/{' and csrc/'.join(DOMINANT_SOURCES)}.
kernel = {DOMINANT}
dispatches_fetch = {n_fetch}
dispatches_write = {n_write}
fetch_kib_per_dispatch = {m_fetch:.1f}
write_kib_per_dispatch = {m_write:.1f}
copy_fetch_kib = {c_fetch:.1f}
copy_write_kib = {c_write:.1f}
fetch_scale = {s_fetch:.4f}
write_scale = {s_write:.4f}
hbm_fetch_bytes_per_launch = {fetch_b:.0f}
hbm_write_bytes_per_launch = {write_b:.0f}
hbm_bytes_per_launch = {fetch_b + write_b:.0f}
kernel_source_hash = {kernel_source_hash()}
""")
    print(open(TRAFFIC_PROFILE).read())


def time_prefill(model, m, wl, stops, reps: int = 3):
    """Prefill of the whole batch (every prompt, chunks of up to 4096 rows),
    re-run on freed slots.  Algorithmic flops: 2 x weight elements of the layer
    stack per prompt token, 4 x hd x H x (positions attended) per token and layer
    for attention, and the LM head for each prompt's last row; bf16 models issue
    twice that MFMA work (hi + lo activation parts), and three times it for the
    QKV projection (hi + mid + lo: its keys and values are rounded into the bf16
    cache)."""
    import torch
    B = wl.batch
    tokens = int(sum(len(t) for t in wl.tokens))
    layer_w = m.weight_elements_per_step() - m.vocab * m.d_model     # projections of all layers
    att = sum(n * (n + 1) // 2 for n in (len(t) for t in wl.tokens)) * 4 * m.head_dim * m.n_heads * m.n_layers
    flops = 2.0 * layer_w * tokens + att + 2.0 * m.vocab * m.d_model * B
    tok = model.new_token_buffer()
    times = []
    for _ in range(reps + 1):
        for i in range(B):
            model.free_slot(i)
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        model.prefill(list(range(B)), wl.tokens, stops, tok)   # synchronous
        times.append(time.perf_counter() - t0)
    ms = 1e3 * min(times[1:])
    tflops = flops / (ms * 1e-3) / 1e12
    qkv_flops = 2.0 * tokens * m.n_layers * m.d_model * (m.n_heads + 2 * m.n_kv_heads) * m.head_dim
    issue = (2.0 * flops + qkv_flops) / flops if m.bf16 else 1.0
    # mfma_frac counts the method's own 2 M N K flops; the MFMA work actually issued is `issued_factor`
    # times that (bf16 activations go in as hi + lo parts, the QKV input as hi + mid + lo), reported
    # separately.
    return {"tokens": tokens, "ms": round(ms, 2), "tokens_per_s": round(tokens / (ms * 1e-3), 1),
            "algorithmic_tflops": round(tflops, 1), "peak_tflops": PEAK_BF16_TFLOPS,
            "mfma_frac": round(tflops / PEAK_BF16_TFLOPS, 4), "issued_factor": round(issue, 3),
            "mfma_issued_tflops": round(tflops * issue, 1),
            "mfma_issued_frac": round(tflops * issue / PEAK_BF16_TFLOPS, 4)}


def gpu_energy_reader():
    """A function returning GPU 0's accumulated energy in joules (amd-smi energy counter), or None
    when amd-smi cannot read it here."""
    try:
        import amdsmi
        amdsmi.amdsmi_init()
        handle = amdsmi.amdsmi_get_processor_handles()[0]

        def read():
            c = amdsmi.amdsmi_get_energy_count(handle)
            return c["energy_accumulator"] * c["counter_resolution"] * 1e-6

        read()
        return read
    except Exception as exc:  # no amd-smi, no permission, or no counter on this device
        log(f"energy counter unavailable: {exc}")
        return None


def time_serving(cfg, n_req: int = 96, max_active: int = 32):
    """Continuous batching (spr_serve) against closed batches, on the same
    requests: n_req requests drawn with the workload's recipe, all waiting at
    the start, at most max_active in flight.  Closed batches take max_active
    requests at a time and drain each batch before the next starts; continuous
    batching refills a slot as soon as its request retires.  Both include
    prefill.  Tokens = every generated token (the prefill's first ones too)."""
    import dataclasses
    import torch
    from paper_2403_12900_amd.binding import DecodeModel
    from paper_2403_12900_amd.workload import make_workload
    m = cfg.model
    c2 = dataclasses.replace(cfg, workload=dataclasses.replace(cfg.workload, batch=n_req))
    wl = make_workload(c2, seed=cfg.workload_seed + 7919)
    prompts = [np.asarray(t) for t in wl.tokens]
    stops = [int(x) for x in wl.stop_lens]
    need = sorted(((len(p) + s - 1 + 15) // 16 for p, s in zip(prompts, stops)), reverse=True)
    max_ctx = max(len(p) + s - 1 for p, s in zip(prompts, stops))
    model = DecodeModel(m, cfg.weight_seed, max_slots=max_active, max_ctx=max_ctx, kv_blocks=sum(need[:max_active]))
    model.serve(prompts[:4], [min(s, 4) for s in stops[:4]], max_active)          # warm-up
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    n_lv = len(cfg.workload.prefix_lens)
    energy = gpu_energy_reader()
    j0 = energy() if energy else None
    _, st = model.serve(prompts, stops, max_active, levels=[int(x) for x in wl.levels])
    cont = time.perf_counter() - t0
    joules = energy() - j0 if energy else None
    tok = model.new_token_buffer()
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for b0 in range(0, n_req, max_active):
        idx = list(range(b0, min(n_req, b0 + max_active)))
        slots = list(range(len(idx)))
        _, retired = model.prefill(slots, [prompts[i] for i in idx], [stops[i] for i in idx], tok)
        lens = [len(prompts[i]) for i in idx]
        active = [k for k in slots if not retired[k]]
        while active:
            _, r = model.decode_step(active, [lens[k] for k in active], tok)
            for k in active:
                lens[k] += 1
            active = [k for j, k in enumerate(active) if not r[j]]
        for k in slots:
            model.free_slot(k)
    torch.cuda.synchronize()
    closed = time.perf_counter() - t0
    model.close()
    total = sum(stops)
    return {"requests": n_req, "max_active": max_active, "generated_tokens": total,
            "continuous_tokens_per_s": round(total / cont, 1), "closed_batches_tokens_per_s": round(total / closed, 1),
            "continuous_s": round(cont, 3), "closed_batches_s": round(closed, 3),
            "continuous_mean_batch": round(st["mean_batch"], 2), "continuous_decode_steps": st["decode_steps"],
            # Eq. 2's per-level p: mean device seconds per request of each directive level, each
            # iteration's time shared equally by the requests it served.
            "level_requests": st["level_requests"][:n_lv],
            "level_mean_tokens": [round(x, 1) for x in st["level_tokens"][:n_lv]],
            "level_seconds_per_request": [round(x, 4) for x in st["level_seconds"][:n_lv]],
            # Eq. 2's per-level e: the amd-smi energy of the whole serving run, attributed to each
            # request in proportion to its share of device time (the same sharing as p).
            "energy_joules": None if joules is None else round(joules, 2),
            "level_joules_per_request": None if joules is None or st["device_seconds"] <= 0 else
            [round(joules * x / st["device_seconds"], 3) for x in st["level_seconds"][:n_lv]]}


ROW_BINS = (("1", 1, 1), ("2-8", 2, 8), ("9-16", 9, 16), ("17-32", 17, 32))


def cpu_baseline(cfg, wl, per_bin: int = 3):
    """The CPU oracle's KV-cache decode on the same ragged batch, timed on a bounded sample of its
    decode steps: the schedule's steps fall into active-row bins (1, 2-8, 9-16, 17-32 rows); per_bin
    steps spread evenly over each bin are run with the caches at their real lengths, and each bin's
    mean step time is weighted by the bin's step count.  tokens/s = the batch's decode tokens / that
    estimated whole-decode time."""
    import numpy as np
    from threadpoolctl import threadpool_info
    from oracle import llama_ref as R
    m = cfg.model
    sh = R.Shape(m.n_layers, m.d_model, m.n_heads, m.n_kv_heads, m.head_dim, m.d_ff, m.vocab,
                 m.rope_base, m.rms_eps, m.bf16, kv_bf16=m.kv_is_bf16)
    t0 = time.perf_counter()
    w = R.Weights(sh, cfg.weight_seed, resident=True)
    for l in range(sh.n_layers):
        w.layer(l)
    w.matrix("embed")
    w.matrix("lm_head")
    log(f"cpu baseline: oracle weights drawn in {time.perf_counter() - t0:.1f} s")
    seq = [int(x) for x in wl.seq_lens]
    stops = [int(x) for x in wl.stop_lens]
    sched = _decode_schedule(seq, stops)
    rng = np.random.default_rng(0)
    bins, est, sampled_s, n_sampled = {}, 0.0, 0.0, 0
    for name, lo, hi in ROW_BINS:
        idx = [k for k, (act, _) in enumerate(sched) if lo <= len(act) <= hi]
        if not idx:
            continue
        pick = sorted({idx[int(round(j * (len(idx) - 1) / max(per_bin - 1, 1)))] for j in range(per_bin)})
        times = []
        for k in pick:
            act, lens = sched[k]
            dec = R.KVCacheDecoder(w)
            for i, L in zip(act, lens):
                dec.attach_cache(i, L + 1, L)
            toks = [int(x) for x in rng.integers(0, m.vocab, size=len(act))]
            t1 = time.perf_counter()
            dec.step(act, toks)
            times.append(time.perf_counter() - t1)
            del dec
        mean = float(np.mean(times))
        bins[name] = {"steps": len(idx), "sampled": len(pick), "s_per_step": round(mean, 3)}
        est += mean * len(idx)
        sampled_s += sum(times)
        n_sampled += len(pick)
    tokens = sum(L - 1 for L in stops)
    blas = [p for p in threadpool_info() if p.get("user_api") == "blas"]
    cores = max((p.get("num_threads", 1) for p in blas), default=1)
    return {"value": tokens / est, "unit": "tokens/s", "cores": int(cores), "kind": "oracle",
            "estimated_decode_s": round(est, 1), "bins": bins,
            "sample": f"{n_sampled} decode steps of the same batch ({sampled_s:.1f} s of CPU time), {per_bin} "
                      f"spread over each active-row bin, caches at their real lengths; whole-decode time = "
                      f"sum over bins of steps x mean sampled step time; fp64 numpy KV-cache decode with "
                      f"resident weights"}


def main():
    ap = argparse.ArgumentParser(description=__doc__, formatter_class=argparse.RawDescriptionHelpFormatter)
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=5)
    ap.add_argument("--warmup", type=int, default=1)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--cpu-steps-per-bin", type=int, default=3)
    ap.add_argument("--no-serving", action="store_true", help="skip the continuous-batching measurement")
    ap.add_argument("--pmc-probe", action="store_true",
                    help="run 32 gate/up and 32 O projections at 8 rows and 2 read-ceiling passes, for rocprofv3 --pmc")
    ap.add_argument("--step-sweep", metavar="CONFIG", default=None,
                    help="decode-step GB/s of one configuration's model (c2..c5) at 1-32 rows of ~512 positions")
    ap.add_argument("--prefill-probe", action="store_true",
                    help="only run the c3 prefill twice (for rocprofv3 --pmc of the prefill GEMMs)")
    ap.add_argument("--decode-probe", action="store_true",
                    help="only run the c3 prefill and one ragged decode (for rocprofv3 --kernel-trace)")
    ap.add_argument("--stats-summary", metavar="STATS_CSV", default=None,
                    help="print a rocprofv3 kernel_stats.csv as the markdown table kept under profiles/")
    ap.add_argument("--trace-summary", metavar="TRACE_DIR", default=None,
                    help="print the decode's kernel time by active rows from a --decode-probe kernel trace")
    ap.add_argument("--traffic-probe", action="store_true",
                    help="only launch the dominant kernel and a calibration copy (for rocprofv3 --pmc)")
    ap.add_argument("--traffic-summary", nargs=2, metavar=("FETCH_CSV", "WRITE_CSV"),
                    help="write the PMC traffic summary from two rocprofv3 counter_collection.csv files")
    args = ap.parse_args()
    if args.traffic_summary:
        traffic_summary(*args.traffic_summary)
        return
    if args.pmc_probe:
        pmc_probe()
        return
    if args.traffic_probe:
        traffic_probe()
        return
    if args.prefill_probe:
        prefill_probe()
        return
    if args.decode_probe:
        decode_probe()
        return
    if args.trace_summary:
        trace_summary(args.trace_summary)
        return
    if args.stats_summary:
        stats_summary(args.stats_summary)
        return
    if args.step_sweep:
        step_sweep(args.step_sweep)
        return
    if args.gpus != 1:
        print(f"bench.py measures one GPU only (asked for {args.gpus}): the decode path runs one model "
              "replica per GPU with no exchange between GPUs, and this build has no multi-GPU mode.",
              file=sys.stderr)
        sys.exit(2)

    import torch
    from paper_2403_12900_amd.binding import DecodeModel
    from paper_2403_12900_amd.configs import CONFIGS
    from paper_2403_12900_amd.workload import make_workload, workload_stats

    cfg = CONFIGS["c3"]
    m = cfg.model
    wl = make_workload(cfg)
    st = workload_stats(cfg, wl)
    B = wl.batch
    seq = [int(x) for x in wl.seq_lens]
    stops = [int(x) for x in wl.stop_lens]
    max_ctx = max(s + L - 1 for s, L in zip(seq, stops))
    blocks = sum((s + L - 1 + 15) // 16 for s, L in zip(seq, stops))
    torch.cuda.set_device(0)
    t0 = time.perf_counter()
    model = DecodeModel(m, cfg.weight_seed, max_slots=B, max_ctx=max_ctx, kv_blocks=blocks)
    tok = model.new_token_buffer()
    model.prefill(list(range(B)), wl.tokens, stops, tok)
    tok0 = tok.clone()
    torch.cuda.synchronize()
    log(f"init + prefill {time.perf_counter() - t0:.1f} s; {st['steps']} decode steps, "
        f"{st['decode_tokens']} tokens, avg active {st['avg_active']:.2f}")

    schedule = _decode_schedule(seq, stops)
    active_bins = {name: sum(1 for act, _ in schedule if lo <= len(act) <= hi) for name, lo, hi in ROW_BINS}

    def one_step():
        for i in range(B):
            if stops[i] > 1:
                model.rewind(i, seq[i], 1)
        tok.copy_(tok0)
        for act, lens in schedule:
            model.decode_step(act, lens, tok)

    for _ in range(args.warmup):
        one_step()
    torch.cuda.synchronize()
    # Each slot's last token ends its greedy chain: repeated decodes must leave the same ones.
    tok_ref = tok.clone() if args.warmup > 0 else None
    # One event pair brackets all timed steps (the reported mean); events between steps give each
    # step's own time for the median.
    marks = [torch.cuda.Event(enable_timing=True) for _ in range(args.steps + 1)]
    wall0 = time.perf_counter()
    marks[0].record()
    for k in range(args.steps):
        one_step()
        marks[k + 1].record()
    torch.cuda.synchronize()
    wall = time.perf_counter() - wall0
    checks = {"tokens_repeat_exactly": None if tok_ref is None else bool(torch.equal(tok, tok_ref)),
              "all_retired_at_stop": all(model.slot_info(i)[1] == stops[i] for i in range(B))}
    if not all(v is not False for v in checks.values()):
        log(f"WARNING: decode checks failed: {checks}")
    ms = marks[0].elapsed_time(marks[-1]) / args.steps
    per_step = [marks[k].elapsed_time(marks[k + 1]) for k in range(args.steps)]
    ms_median = float(np.median(per_step))
    tokens = st["decode_tokens"]
    value = tokens / (ms / 1e3)
    gbps = st["bytes"] / (ms / 1e3) / 1e9
    log(f"decode: {ms:.1f} ms per ragged batch (wall {1e3 * wall / args.steps:.1f} ms), {value:.0f} tokens/s, "
        f"{gbps:.0f} GB/s algorithmic")

    # Dominant kernel: the gate/up projection with SwiGLU (largest weight stream of a layer).
    n_probe = 8
    reps = 200
    us = model.time_projection("gate_up", n_probe, reps)
    elem = 2 * m.d_ff * m.d_model
    per_launch = elem * 2 + n_probe * m.d_model * 2 * 2 + n_probe * m.d_ff * 2 * 2
    achieved = per_launch / (us * 1e-6) / 1e9
    others = {}
    for name, el in (("o", m.d_model * m.n_heads * m.head_dim), ("down", m.d_model * m.d_ff),
                     ("lm_head", m.vocab * m.d_model)):
        u = model.time_projection(name, n_probe, 50)
        others[name] = {"us": round(u, 2), "gbps": round(el * 2 / (u * 1e-6) / 1e9, 1)}
    ceiling, ceiling_bytes = model.read_ceiling(5)
    log(f"read ceiling: {ceiling:.0f} GB/s over {ceiling_bytes / 1e9:.2f} GB of weights")
    traffic = measured_traffic(per_launch)
    log(f"gate/up kernel: {us:.2f} us per launch, {achieved:.0f} GB/s; others {others}")

    out = {
        "metric": METRIC,
        "value": round(value, 2),
        "unit": "tokens/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms, 3),
        "ms_per_step_median": round(ms_median, 3),
        "ms_per_step_runs": [round(x, 1) for x in per_step],
        "checks": checks,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16",
        "data": "synthetic",
        "achieved_hbm_gbps": round(gbps, 1),
        "hbm_frac": round(gbps / PEAK_HBM_GBPS, 4),
        # The measured read ceiling: every weight matrix streamed with the projections' load form
        # (16-byte nontemporal loads, 8 in flight per thread) and no arithmetic.
        "read_ceiling_gbps": round(ceiling, 1),
        "frac_of_read_ceiling": round(gbps / ceiling, 4),
        # One bench step = one full ragged decode of the batch (decode_steps_per_batch model steps).
        "config": {"workload": cfg.name, "batch": B, "decode_steps_per_batch": st["steps"],
                   "decode_tokens_per_batch": tokens, "avg_active": round(st["avg_active"], 3),
                   "active_row_bins": active_bins,
                   "algorithmic_bytes_per_batch": st["bytes"], "parallelism": "none (1 GPU)"},
        "roofline": {"bound": "hbm", "kernel": DOMINANT, "rows": n_probe, "achieved": round(achieved, 1),
                     "peak": PEAK_HBM_GBPS, "unit": "GB/s", "frac": round(achieved / PEAK_HBM_GBPS, 4),
                     "traffic": traffic, "bytes_per_launch": per_launch, "us_per_launch": round(us, 3),
                     "other_projections": others},
    }
    out["prefill"] = time_prefill(model, m, wl, stops)
    log(f"prefill: {out['prefill']}")
    model.close()
    del model
    torch.cuda.empty_cache()
    if not args.no_serving:
        out["serving"] = time_serving(cfg)
        log(f"serving: {out['serving']}")
        torch.cuda.empty_cache()
    if not args.no_cpu_baseline:
        out["cpu_baseline"] = cpu_baseline(cfg, wl, args.cpu_steps_per_bin)
        log(f"cpu baseline: {out['cpu_baseline']}")
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
