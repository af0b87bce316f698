"""Benchmark: full-model VaSE-AttnV eviction rounds on one MI355X.

One step is one eviction round over every (layer, batch, KV head) instance of
the workload -- score, select, compact -- plus one decode-attention step over
the compacted cache (fused with the compaction), all through the C ABI on the
current HIP stream.  Before each round the B token rows that the decoder
appended since the previous round are copied into the buffer slots, and the
round uses that period's window and decode queries: both are drawn ahead of
the timed region, distinct for every round.  Inputs are synthetic and already
resident in HBM when the timed region starts.

    python bench.py [--gpus 1] [--steps 20] [--warmup 5] [--config qwen3-8b]

Prints one JSON line.  ``value`` is rounds per second; ``roofline`` describes
the dominant kernel; ``round_hbm`` gives the step's algorithmic bytes (score +
select + compact + decode) against the HBM peak; ``score_select_compact`` times
the round alone (score, select and the compaction without a decode step, with
the value scores carried from round to round where the layout allows) and
gives its bytes against the HBM peak, ``score_select_compact_reading_v`` the
same round with the score reading V every round; ``cpu_baseline`` is the CPU oracle on the
same workload, scaled to rounds per second.
"""
import argparse
import hashlib
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

HBM_PEAK_GBS = 8000.0          # MI355X HBM3E, datasheet
MFMA_BF16_PEAK_TFS = 2500.0    # MI355X dense bf16 MFMA, datasheet
FP32_VECTOR_PEAK_TFS = 157.3   # MI355X fp32 vector, datasheet (packed fp32, which this build does not emit)
# VALU issue peak without packed fp32: 256 CUs x 4 SIMDs x 16 lanes x 2.4 GHz, in
# tera lane-operations per second; v_exp_f32 runs at half that rate on this part
# (measured with bench.py --peaks), so it counts as 2
VALU_PEAK_TOPS = 256 * 4 * 16 * 2.4e9 / 1e12
EXP_SLOTS = 2


VALUE_KINDS = {"range": 0, "l2": 1, "var": 2, "random": 3}
PEAKS_JSON = os.path.join(ROOT, "profiles", "measured_peaks.json")


def parse():
    p = argparse.ArgumentParser()
    p.add_argument("--gpus", type=int, default=1)
    p.add_argument("--steps", type=int, default=20)
    p.add_argument("--warmup", type=int, default=5)
    p.add_argument("--config", default="qwen3-8b")
    p.add_argument("--method", choices=("attnv", "dkv"), default="attnv",
                   help="VaSE-AttnV (default) or VaSE-DKV (Gaussian-projection scores, "
                        "deterministic selection)")
    p.add_argument("--value", choices=tuple(VALUE_KINDS), default="range",
                   help="VaSE-AttnV value score: Range (the method), or the L2 / Var / random "
                        "reservation variants")
    p.add_argument("--seed", type=int, default=0)
    p.add_argument("--cpu-sample", type=int, default=0,
                   help="instances for the CPU-oracle baseline (0 = pick ~10-30 s of work)")
    p.add_argument("--no-cpu-baseline", action="store_true")
    p.add_argument("--copy-probe", type=int, default=0, metavar="MIB",
                   help="only run a plain device copy of MIB MiB three times (the reference "
                        "for scaling HBM traffic counters) and exit")
    p.add_argument("--write-traffic", nargs=4, metavar=("FETCH_CSV", "WRITE_CSV", "COPY_FETCH_CSV",
                                                         "COPY_WRITE_CSV"),
                   help="only turn rocprofv3 --pmc FETCH_SIZE / WRITE_SIZE counter files (of this "
                        "benchmark, then of --copy-probe 1024) into profiles/traffic.json")
    p.add_argument("--carry", choices=("on", "off"), default="on",
                   help="on: each round's compaction also computes the value scores of the rows "
                        "it writes, which are the next round's candidates, and the next round's "
                        "score kernel does not read V (the first round computes them itself); "
                        "off: every round's score kernel computes them from V")
    p.add_argument("--sustained", action="store_true",
                   help="sustained decode: one step is a period of B decode steps (append, window "
                        "ring, attention, persistent-slot LSE) followed by one round whose score "
                        "is the one-pass score over the decode steps' LSEs")
    p.add_argument("--quant", default="", metavar="bBgG",
                   help="time the Range-based quantiser instead (e.g. b4g32: 4-bit codes in "
                        "groups of 32) on the value cache's K rows, with the N_v reserve")
    p.add_argument("--layout", choices=("map", "stable"), default="map",
                   help="map: survivors stay in their slots and an order map keeps the temporal "
                        "order (compaction moves the B buffer rows into the evicted slots); "
                        "stable: compaction moves every survivor into temporal slot order")
    p.add_argument("--dec-logits", choices=("on", "off"), default="on",
                   help="order map, bf16, G <= 8: on: the score's pass over every key also "
                        "writes the decode queries' logits, and the compaction's decode step "
                        "reads them instead of K; off: the decode reads K")
    p.add_argument("--group", type=int, default=0,
                   help="instances per call (0 = all in one call); calls run in instance order")
    p.add_argument("--no-target", action="store_true",
                   help="skip the score+select+compact timing (the round without the decode step)")
    p.add_argument("--peaks", action="store_true",
                   help="only measure the chip's copy, read, bf16 MFMA, exp2 and fp32 fma rates with "
                        "the probes of libvase_peaks.so and print them as one JSON line")
    return p.parse_args()


def source_digest(files):
    h = hashlib.sha256()
    for f in files:
        with open(os.path.join(ROOT, f), "rb") as fh:
            h.update(fh.read())
    return h.hexdigest()[:16]


def algorithmic_bytes(cfg, moved_rows, reads_values=True, layout="stable", dec_logits=False):
    """Bytes the method must move per round (one read of K over N slots, one read of
    V over K slots unless the value score is random, the window, the score/select
    arrays, and the moved rows).  Under the order map the pooling also reads the
    map (4 bytes per candidate) and the compaction reads the survivor map and
    reads and writes the order map (12 bytes per candidate).  With the decode
    logits left by the score (fp32, G per slot: written for all N slots, read for
    the K decoded ones) the decode reads no K row; the K rows that move are still
    read."""
    e = cfg.elem_bytes
    n, N, K, d, R = cfg.n_inst, cfg.N, cfg.K, cfg.d, cfg.R
    score = n * (N * d * e + (K * d * e if reads_values else 0) + R * d * e + 2 * K * 4)
    select = n * (2 * K * 4 + K * 4)
    # compaction fused with one decode step: every survivor row of K and V is read once
    # (the decode needs all of them), the rows that move are written, plus q and o
    compact_decode = n * (2 * K * d * e + 2 * cfg.G * d * e) + 2 * d * e * moved_rows
    if layout == "map":
        score += n * K * 4          # the map, read by the pooling
        compact_decode += n * K * 12
    if dec_logits:
        score += n * cfg.G * (N * 4 + d * e)
        compact_decode += n * (cfg.G * K * 4 - K * d * e) + d * e * moved_rows
    return {"score": score, "select": select, "compact_decode": compact_decode}


def carried_bytes(cfg, moved_rows, carry, args, reads_values):
    """Algorithmic bytes of a timed step when the compaction carries the value scores:
    the score reads no V, except in a first round that nothing carried into (a timed
    region with no warm-up), and the compaction writes one fp32 score per row."""
    ab = algorithmic_bytes(cfg, moved_rows, reads_values=reads_values and not carry,
                           layout=getattr(args, "layout", "stable"),
                           dec_logits=uses_dec_logits(args, cfg))
    if carry:
        ab["compact_decode"] += cfg.n_inst * cfg.K * 4
        if reads_values and args.warmup == 0:
            ab["score"] += cfg.n_inst * cfg.K * cfg.d * cfg.elem_bytes / args.steps
    return ab


DKV_RANK = 20


def dkv_score_bytes(cfg):
    """DKV scoring: the K candidate rows of K and V once, G written and read, scores out."""
    e = cfg.elem_bytes
    return cfg.n_inst * (2 * cfg.K * cfg.d * e + 2 * cfg.d * DKV_RANK * 4 + cfg.K * 4)


def score_flops(cfg):
    """Useful QK^T flops of one round (one pass over the window)."""
    return 2.0 * cfg.n_inst * cfg.R * cfg.N * cfg.d


def score_valu_ops(cfg, passes=2, supplied_lse=False):
    """VALU lane-operations of the score's per-element work: each (row, slot) score
    costs an fma (scale and offset), an exp2 (a half-rate instruction, counted
    as EXP_SLOTS) and an add, 2 + EXP_SLOTS issue slots.  passes=1 counts the work
    the method needs (every window score once, over all N slots); passes=2 the
    kernel's two passes (pass 1 over all N slots, or only the B buffer slots with a
    supplied normaliser; pass 2 over the K candidates)."""
    per = 2 + EXP_SLOTS
    if passes == 1:
        return float(per) * cfg.n_inst * cfg.R * cfg.N
    p1 = cfg.B if supplied_lse else cfg.N
    return float(per) * cfg.n_inst * cfg.R * (p1 + cfg.K)


def _oracle_step(cfg, x, sl, seed, method="attnv", value="range", chunk=256):
    """score + Range + select + compact + decode on instances `sl`, by the oracle
    (for VaSE-DKV: projection + score + deterministic select + compact + decode),
    in chunks of `chunk` instances; returns the oracle's own time in seconds
    (host copies of the inputs are not counted)."""
    import torch
    import oracle
    total = 0.0
    for c0 in range(sl.start, sl.stop, chunk):
        c = slice(c0, min(sl.stop, c0 + chunk))
        k = x["k"][c].cpu()
        v = x["v"][c].cpu()
        qw = x["q_win"][c].cpu()
        qd = x["q_dec"][c].cpu()
        bf = k.dtype == torch.bfloat16
        t0 = time.perf_counter()
        if method == "dkv":
            _, src = oracle.dkv_round(k, v, cfg.K, cfg.B, seed, 0, inst_base=c.start, r=DKV_RANK)
        elif value == "range":
            attn, vr, src = oracle.round_(qw, k, v, cfg.K, cfg.B, cfg.Nv, cfg.pool, seed=seed,
                                          rnd=0, inst_base=c.start)
        else:
            kind = VALUE_KINDS[value]
            attn = oracle.score(qw, k, cfg.K, cfg.pool)
            vr = oracle.value_score(None if value == "random" else v, cfg.K, kind, seed, 0,
                                    inst_base=c.start, n_inst=k.shape[0])
            src = oracle.select(attn, vr, cfg.K, cfg.B, cfg.Nv, seed, 0, inst_base=c.start)
        kb = k.view(torch.int16).numpy().copy() if bf else k.numpy().copy()
        vb = v.view(torch.int16).numpy().copy() if bf else v.numpy().copy()
        oracle.compact(kb, vb, src)
        kk = torch.from_numpy(kb).view(k.dtype) if bf else torch.from_numpy(kb)
        vv = torch.from_numpy(vb).view(v.dtype) if bf else torch.from_numpy(vb)
        oracle.decode(qd, kk, vv, cfg.K)
        total += time.perf_counter() - t0
    return total


def cpu_model() -> str:
    """The host CPU's model name (from /proc/cpuinfo)."""
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    return line.split(":", 1)[1].strip()
    except OSError:
        pass
    import platform
    return platform.processor() or "unknown"


def cpu_baseline(cfg, x, sample_n, seed, max_s=45.0, method="attnv", value="range"):
    """The oracle, as it stands, timed on the host's cores, scaled to rounds/s.
    With sample_n = 0 it runs every instance of the workload when a 32-instance
    probe predicts at most `max_s` seconds, and otherwise the prefix of
    instances that takes about `max_s` / 3."""
    import oracle
    oracle.build(force=False)
    if not sample_n:
        probe = min(32, cfg.n_inst)
        t_probe = _oracle_step(cfg, x, slice(0, probe), seed, method, value)
        full = t_probe * cfg.n_inst / probe
        sample_n = cfg.n_inst if full <= max_s else int(max(probe, probe * (max_s / 3) / t_probe))
    sample_n = min(sample_n, cfg.n_inst)
    dt = _oracle_step(cfg, x, slice(0, sample_n), seed, method, value)
    threads = int(os.environ.get("OMP_NUM_THREADS", "0")) or len(os.sched_getaffinity(0))
    what = "projection+DKV score" if method == "dkv" else "score+" + value
    if sample_n == cfg.n_inst:
        sample = "all %d instances (%.1f s for %s+select+compact+decode)" % (cfg.n_inst, dt, what)
    else:
        sample = ("first %d of %d instances (%.1f s for %s+select+compact+decode, scaled by %d/%d)"
                  % (sample_n, cfg.n_inst, dt, what, sample_n, cfg.n_inst))
    return {"value": (sample_n / cfg.n_inst) / dt, "unit": "rounds/s", "cores": threads,
            "kind": "oracle", "cpu_model": cpu_model(), "sample": sample}


_SRC = "paper_2606_03928_amd/csrc/"
TRAFFIC_KERNELS = {
    # kernel: sources whose digest keys its entry (the trace name is matched as
    # "::<kernel><" so that, e.g., dequant_rows_kernel is not quant_rows_kernel)
    "score_mfma_kernel": [_SRC + "score.hip", _SRC + "vase_internal.hpp"],
    "compact_decode_kernel": [_SRC + "compact.hip", _SRC + "vase_internal.hpp"],
    "compact_map_decode_kernel": [_SRC + "order.hip", _SRC + "vase_internal.hpp"],
    "compact_map_mfma_kernel": [_SRC + "order.hip", _SRC + "vase_internal.hpp"],
    "order_scores_kernel": [_SRC + "order.hip", _SRC + "vase_internal.hpp"],
    "decode_mfma_kernel": [_SRC + "decode.hip", _SRC + "vase_internal.hpp"],
    "dkv_score_mfma_kernel": [_SRC + "dkv.hip", _SRC + "vase_internal.hpp"],
    "quant_rows_kernel": [_SRC + "quant.hip", _SRC + "vase_internal.hpp"],
    "dequant_rows_kernel": [_SRC + "quant.hip", _SRC + "vase_internal.hpp"],
}


def uses_dec_logits(args, cfg):
    """Whether the default round runs its decode from the score's logits."""
    from paper_2606_03928_amd.vase import dec_logits_fit
    return (getattr(args, "dec_logits", "off") == "on" and getattr(args, "layout", "") == "map"
            and not args.sustained and not args.quant and cfg.dtype == "bf16" and cfg.G <= 8
            and dec_logits_fit(cfg.N, cfg.d, cfg.G))


def workload_tag(args, cfg):
    """Key of a benchmark mode's entries in profiles/traffic.json."""
    if args.sustained:
        return (cfg.name + "/sustained" + ("/no-carry" if args.carry == "off" else "") +
                ("/map" if args.layout == "map" else ""))
    if args.quant:
        return cfg.name + "/quant-" + args.quant
    if args.method == "dkv":
        tag = cfg.name + "/dkv"
        if args.layout == "map":
            tag += "/map"
            if args.dec_logits == "off" and cfg.dtype == "bf16" and cfg.G <= 8:
                tag += "/no-dl"
        return tag
    tag = cfg.name
    if args.value != "range":
        tag += "/value-" + args.value
    if args.carry == "off" and args.value != "random":
        tag += "/no-carry"
    if args.layout == "map":
        tag += "/map"
        if args.dec_logits == "off" and cfg.dtype == "bf16" and cfg.G <= 8:
            tag += "/no-dl"
    return tag


def traffic_for(kernel, workload, inst=None):
    """Measured HBM bytes per launch of `kernel` (its template instantiation `inst`,
    e.g. "<128, 8, 2, 1, false>", when several run in one benchmark) on `workload` from
    profiles/traffic.json, or None when absent or taken on sources that have
    changed since."""
    tpath = os.path.join(ROOT, "profiles", "traffic.json")
    if not os.path.exists(tpath):
        return None
    with open(tpath) as f:
        db = json.load(f)
    ent = db.get("%s%s@%s" % (kernel, inst or "", workload)) or db.get("%s@%s" % (kernel, workload))
    if ent and ent.get("source_digest") == source_digest(ent["sources"]):
        return ent["bytes_per_launch"]
    return None


def score_instantiation(cfg, dec_logits):
    """Template arguments of the fused score kernel a benchmark step launches:
    <d, waves (4 for at most 256 window rows, else 8), fused, decode-logit mode,
    whether the last row slab has waves without rows>."""
    n_slab = (cfg.R + 511) // 512
    waves = 4 if (cfg.R + 64 * n_slab - 1) // (64 * n_slab) <= 4 else 8
    rows = 64 * waves
    partial = ((cfg.R + rows - 1) // rows) * rows - cfg.R >= 64
    return "<%d, %d, 2, %d, %s>" % (cfg.d, waves, 1 if dec_logits else 0,
                                    "true" if partial else "false")


def _counter_per_dispatch(path, counter):
    """{kernel name: [value per dispatch]} for one counter of a rocprofv3 --pmc csv."""
    import collections
    import csv
    per = collections.defaultdict(float)
    names = {}
    with open(path) as f:
        for r in csv.DictReader(f):
            if r["Counter_Name"] != counter:
                continue
            per[r["Dispatch_Id"]] += float(r["Counter_Value"])      # summed over instances
            names[r["Dispatch_Id"]] = r["Kernel_Name"]
    out = collections.defaultdict(list)
    for d, v in per.items():
        out[names[d]].append(v)
    return out


def write_traffic(paths, workload):
    """HBM bytes per launch of the kernels in TRAFFIC_KERNELS found in one benchmark's
    FETCH_SIZE and WRITE_SIZE runs (KiB per dispatch, medians over dispatches), each
    scaled by what that counter reads on a plain 1 GiB device copy; merged into
    profiles/traffic.json under "<kernel>@<workload>"."""
    import statistics
    fetch, write, cfetch, cwrite = (p for p in paths)

    def copy_kib(path, counter):
        vals = [v for n, vs in _counter_per_dispatch(path, counter).items()
                if "copy" in n.lower() for v in vs]
        return statistics.median(vals)

    gib_kib = float(1 << 20)
    f_scale = gib_kib / copy_kib(cfetch, "FETCH_SIZE")
    w_scale = gib_kib / copy_kib(cwrite, "WRITE_SIZE")
    fk = _counter_per_dispatch(fetch, "FETCH_SIZE")
    wk = _counter_per_dispatch(write, "WRITE_SIZE")
    path = os.path.join(ROOT, "profiles", "traffic.json")
    out = {}
    if os.path.exists(path):
        with open(path) as f:
            out = {k_: v_ for k_, v_ in json.load(f).items() if "@" in k_}
    out["_calibration"] = {"copy_bytes": 1 << 30, "fetch_scale": round(f_scale, 4),
                           "write_scale": round(w_scale, 4)}
    import re
    for name, sources in TRAFFIC_KERNELS.items():
        pat = "::%s<" % name
        # one entry per template instantiation found (several may run in one benchmark)
        insts = sorted({re.search(r"::%s(<[^>(]*>)" % name, n).group(1) for n in fk if pat in n})
        for inst in insts:
            fv = [v for n, vs in fk.items() if pat in n and ("::%s%s" % (name, inst)) in n for v in vs]
            wv = [v for n, vs in wk.items() if pat in n and ("::%s%s" % (name, inst)) in n for v in vs]
            if not fv or not wv:
                continue
            rb = statistics.median(fv) * 1024 * f_scale
            wb = statistics.median(wv) * 1024 * w_scale
            ent = {"sources": sources, "source_digest": source_digest(sources), "dispatches": len(fv),
                   "read_bytes_per_launch": round(rb), "write_bytes_per_launch": round(wb),
                   "bytes_per_launch": round(rb + wb)}
            out["%s%s@%s" % (name, inst, workload)] = ent
            if len(insts) == 1:
                out["%s@%s" % (name, workload)] = ent
    with open(path, "w") as f:
        json.dump(dict(sorted(out.items())), f, indent=1)
    print(json.dumps(out))


def decode_step_bytes(cfg, pos):
    """One decode step at buffer position pos: K + pos + 1 rows of K and V read, the
    new (k, v) rows and the G queries written and cached, q read, out written."""
    e = cfg.elem_bytes
    n, d, G = cfg.n_inst, cfg.d, cfg.G
    return n * (2 * (cfg.K + pos + 1) * d * e + 2 * d * e + 3 * G * d * e + G * 4)


def quant_bytes(cfg, bits, group, Nv):
    """Quantise: read K rows, write codes, (Delta, z), Range and MSE, then the reserve
    reads the Ranges and copies N_v rows.  Dequantise: read codes and params, write
    K rows, then write the N_v reserved rows."""
    e = cfg.elem_bytes
    n, K, d = cfg.n_inst, cfg.K, cfg.d
    codes = K * d * bits // 8
    params = K * (d // group) * 8
    reserve = (K * 4 + 2 * Nv * d * e + Nv * 4) if Nv else 0
    q = n * (K * d * e + codes + params + 2 * K * 4 + reserve)
    dq = n * (codes + params + K * d * e + ((Nv * d * e * 2 + Nv * 4) if Nv else 0))
    return q, dq


def run_quant(args, cfg, x, dev):
    import re
    import torch
    from paper_2606_03928_amd import vase
    m = re.fullmatch(r"b(\d+)g(\d+)", args.quant)
    if not m:
        print("--quant takes bBgG, e.g. b4g32", file=sys.stderr)
        sys.exit(2)
    bits, group = int(m.group(1)), int(m.group(2))
    n, K, B, Nv = cfg.n_inst, cfg.K, cfg.B, cfg.Nv
    stream = torch.cuda.current_stream(dev)
    v = x["v"]
    q = vase.quantize(v, K, B, bits, group, Nv=Nv, stream=stream)
    out = torch.empty_like(v)
    for _ in range(args.warmup):
        vase.quantize(v, K, B, bits, group, Nv=Nv, out=q, stream=stream)
        vase.dequantize(q, K, B, bits, group, v.dtype, out=out, stream=stream)
    torch.cuda.synchronize()
    ev = [[torch.cuda.Event(enable_timing=True) for _ in range(3)] for _ in range(args.steps)]
    t0 = time.perf_counter()
    for s_ in range(args.steps):
        ev[s_][0].record(stream)
        vase.quantize(v, K, B, bits, group, Nv=Nv, out=q, stream=stream)
        ev[s_][1].record(stream)
        vase.dequantize(q, K, B, bits, group, v.dtype, out=out, stream=stream)
        ev[s_][2].record(stream)
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    q_ms = sum(e[0].elapsed_time(e[1]) for e in ev) / args.steps
    dq_ms = sum(e[1].elapsed_time(e[2]) for e in ev) / args.steps
    qb, dqb = quant_bytes(cfg, bits, group, Nv)
    q_gbs = qb / (q_ms * 1e-3) / 1e9
    dq_gbs = dqb / (dq_ms * 1e-3) / 1e9
    line = {
        "metric": "Range-based quantisation of the value cache, K rows of every instance, "
                  "quantise + dequantise per step (GB/s vs HBM peak)",
        "value": round(1000.0 * args.steps / (wall * 1e3), 3),
        "unit": "caches/s",
        "n_gpus": 1, "steps": args.steps, "warmup": args.warmup,
        "ms_per_step": round(wall * 1e3 / args.steps, 4),
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None,
        "dtype": "bf16" if cfg.dtype == "bf16" else "f32",
        "data": "synthetic (seeded Qwen3-shaped value cache with log-uniform outlier rows)",
        "config": {"workload": "Eq. 6 per-token asymmetric quantisation, %s value cache: %d "
                               "instances x K=%d rows x d=%d, %d-bit codes in groups of %d, "
                               "N_v=%d rows kept in full precision"
                               % (cfg.name, n, K, cfg.d, bits, group, Nv),
                   "bits": bits, "group": group, "N_v": Nv, "n_inst": n, "K": K, "d": cfg.d},
        "stage_ms": {"quantize": round(q_ms, 4), "dequantize": round(dq_ms, 4)},
        "quantize_hbm": {"bytes": qb, "GB/s": round(q_gbs, 1),
                         "frac_of_peak": round(q_gbs / HBM_PEAK_GBS, 4)},
        "dequantize_hbm": {"bytes": dqb, "GB/s": round(dq_gbs, 1),
                           "frac_of_peak": round(dq_gbs / HBM_PEAK_GBS, 4)},
        "roofline": {"bound": "hbm", "kernel": "quant_rows_kernel (+ quant_reserve_kernel)",
                     "achieved": round(q_gbs, 1), "peak": HBM_PEAK_GBS, "unit": "GB/s",
                     "frac": round(q_gbs / HBM_PEAK_GBS, 4),
                     "traffic": traffic_for("quant_rows_kernel", workload_tag(args, cfg))},
        "cpu_baseline": None,
    }
    print(json.dumps(line), flush=True)


def run_sustained(args, cfg, x, dev):
    """Periods of B decode steps followed by one round (one-pass score, select,
    compaction fused with a decode step), timed period by period."""
    import torch
    from paper_2606_03928_amd import vase
    n, K, B, d, G, w = cfg.n_inst, cfg.K, cfg.B, cfg.d, cfg.G, cfg.w
    stream = torch.cuda.current_stream(dev)
    rb = vase.Round(n, K, B, d, G, w, cfg.torch_dtype, dev, layout=args.layout)
    q_win = torch.zeros_like(x["q_win"])
    lse_win = torch.zeros((n, G, w), dtype=torch.float32, device=dev)
    dec_out = torch.empty((n, G, d), dtype=cfg.torch_dtype, device=dev)
    # the B new tokens of a period (drawn once, reused every period)
    gen = torch.Generator(device=dev)
    gen.manual_seed(args.seed + 17)
    kn = torch.randn((B, n, d), generator=gen, device=dev).to(cfg.torch_dtype)
    vn = torch.randn((B, n, d), generator=gen, device=dev).to(cfg.torch_dtype)
    qn = torch.randn((B, n, G, d), generator=gen, device=dev).to(cfg.torch_dtype)

    carry = args.carry == "on"
    carried = [False]

    def period(p, ev=None):
        if ev: ev[0].record(stream)
        for pos in range(B):
            vase.decode_step(x["k"], x["v"], kn[pos], vn[pos], qn[pos], K, B, pos, q_win, lse_win,
                             out=dec_out, ws=rb.ws, stream=stream)
        if ev: ev[1].record(stream)
        vase.score(x["k"], x["v"], q_win, K, B, cfg.pool, attn=rb.attn, vrange=rb.vrange,
                   ws=rb.ws, stream=stream, lse_win=lse_win, ord=rb.ord,
                   value_kind=vase.VALUE_SKIP if carried[0] else vase.VALUE_RANGE)
        if ev: ev[2].record(stream)
        vase.select(rb.attn, rb.vrange, K, B, cfg.Nv, args.seed, p, src=rb.src, stream=stream)
        if ev: ev[3].record(stream)
        if rb.ord is not None:
            vase.compact_decode_map(x["k"], x["v"], rb.src, rb.ord, K, B, q=x["q_dec"], out=rb.out,
                                    stream=stream, vrange_out=rb.vrange if carry else None,
                                    vrange_in=rb.vrange if carry else None)
        else:
            vase.compact_decode(x["k"], x["v"], rb.src, x["q_dec"], K, B, out=rb.out, ws=rb.ws,
                                stream=stream, vrange_out=rb.vrange if carry else None)
        if ev: ev[4].record(stream)
        carried[0] = carry

    for p in range(args.warmup):
        period(p)
    torch.cuda.synchronize()
    events = [[torch.cuda.Event(enable_timing=True) for _ in range(5)] for _ in range(args.steps)]
    ar = torch.arange(K, device=dev, dtype=torch.int32)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for s in range(args.steps):
        period(args.warmup + s, events[s])
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    moved = n * B if rb.ord is not None else int((rb.src != ar).sum().item())
    names = ["decode_steps", "score_one_pass", "select", "compact_decode"]
    stage_ms = {nm: sum(ev[i].elapsed_time(ev[i + 1]) for ev in events) / args.steps
                for i, nm in enumerate(names)}
    period_ms = wall * 1e3 / args.steps
    dec_bytes = sum(decode_step_bytes(cfg, pos) for pos in range(B))
    dec_gbs = dec_bytes / (stage_ms["decode_steps"] * 1e-3) / 1e9
    ab = carried_bytes(cfg, moved, carry, args, reads_values=True)
    round_ms = stage_ms["score_one_pass"] + stage_ms["select"] + stage_ms["compact_decode"]
    round_bytes = ab["score"] + ab["select"] + ab["compact_decode"]
    line = {
        "metric": "eviction rounds/sec (all layers x heads, 1 GPU) + achieved HBM GB/s vs peak",
        "value": round(1000.0 / period_ms, 3),
        "unit": "rounds/s",
        "n_gpus": 1, "steps": args.steps, "warmup": args.warmup,
        "ms_per_step": round(period_ms, 4),
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None,
        "dtype": "bf16" if cfg.dtype == "bf16" else "f32",
        "data": "synthetic (seeded Qwen3-shaped caches; B fresh N(0,1) token rows per period)",
        "config": {
            "workload": "VaSE-AttnV sustained decode, %s: %d instances, G=%d, d=%d, K=%d, B=%d, "
                        "w=%d, N_v=%d, P=%d; one step = one period: B decode steps (append, "
                        "window ring, attention over K+pos+1 slots, persistent-slot LSE) then one "
                        "round with the one-pass score, select, compaction + decode%s%s"
                        % (cfg.name, n, G, d, K, B, w, cfg.Nv, cfg.pool,
                           "; value scores computed by each round's compaction for the rows it "
                           "writes, the next round's candidates" if carry else "",
                           LAYOUT_NOTE[args.layout]),
            "layout": args.layout, "method": "attnv", "sustained": True, "value_scores_carried": carry, "n_inst": n, "K": K, "B": B, "w": w,
            "N_v": cfg.Nv, "d": d, "G": G, "pool": cfg.pool,
        },
        "stage_ms": {k_: round(v_, 4) for k_, v_ in stage_ms.items()},
        "decode_step_ms": round(stage_ms["decode_steps"] / B, 4),
        "decode_hbm": {"bytes_per_period": dec_bytes, "GB/s": round(dec_gbs, 1),
                       "frac_of_peak": round(dec_gbs / HBM_PEAK_GBS, 4)},
        "round_hbm": {"bytes": round_bytes, "ms": round(round_ms, 4),
                      "GB/s": round(round_bytes / (round_ms * 1e-3) / 1e9, 1),
                      "frac_of_peak": round(round_bytes / (round_ms * 1e-3) / 1e9 / HBM_PEAK_GBS, 4),
                      "moved_rows": moved},
        "roofline": {"bound": "hbm", "kernel": "decode_mfma_kernel (+ combine, append)",
                     "achieved": round(dec_gbs, 1), "peak": HBM_PEAK_GBS, "unit": "GB/s",
                     "frac": round(dec_gbs / HBM_PEAK_GBS, 4),
                     "traffic": traffic_for("decode_mfma_kernel", workload_tag(args, cfg)),
                     "note": "achieved: the period's decode-step bytes over the decode-step "
                             "time; traffic: median HBM bytes of one decode_mfma_kernel launch"},
        "cpu_baseline": None,
    }
    print(json.dumps(line), flush=True)


LAYOUT_NOTE = {
    "map": "; cache layout: order map (survivors keep their slots, the B buffer rows move into "
           "the evicted slots, scores pooled and selected in temporal order)",
    "stable": "; cache layout: stable (compaction moves the survivors into temporal order)",
}


def main():
    args = parse()
    if args.write_traffic:
        from paper_2606_03928_amd import synth as _synth
        write_traffic(args.write_traffic, workload_tag(args, _synth.CONFIGS[args.config]))
        return
    if args.gpus != 1:
        print("bench.py measures one GPU only: the eviction round has no cross-GPU work "
              "(head instances are independent); run with --gpus 1", file=sys.stderr)
        sys.exit(2)
    import torch
    from paper_2606_03928_amd import synth, vase

    if not torch.cuda.is_available():
        print("bench.py needs a GPU", file=sys.stderr)
        sys.exit(2)
    dev = torch.device("cuda:0")
    if args.copy_probe:
        n = args.copy_probe << 20
        a = torch.empty(n, dtype=torch.uint8, device=dev).fill_(1)
        b = torch.empty_like(a)
        torch.cuda.synchronize()
        for _ in range(3):
            b.copy_(a)
        torch.cuda.synchronize()
        print(json.dumps({"copy_probe_bytes": n, "copies": 3}), flush=True)
        return
    if args.peaks:
        run_peaks(dev)
        return
    vase.load()
    cfg = synth.CONFIGS[args.config]
    x = synth.make_round_inputs(cfg, dev, seed=args.seed)
    if args.sustained:
        run_sustained(args, cfg, x, dev)
        return
    if args.quant:
        run_quant(args, cfg, x, dev)
        return
    rb = vase.Round(cfg.n_inst, cfg.K, cfg.B, cfg.d, cfg.G, cfg.w, cfg.torch_dtype, dev,
                    layout=args.layout, dec_logits=uses_dec_logits(args, cfg))
    stream = torch.cuda.current_stream(dev)
    K, B = cfg.K, cfg.B
    omap = rb.ord is not None
    dls = rb.dec_logits

    dkv = args.method == "dkv"
    value_kind = VALUE_KINDS[args.value]
    g_buf = (torch.empty((cfg.n_inst, cfg.d, DKV_RANK), dtype=torch.float32, device=dev)
             if dkv else None)
    # VaSE-DKV under the order map: per-slot scores here, then into temporal order
    phys_a = torch.empty((cfg.n_inst, K), dtype=torch.float32, device=dev) if omap and dkv else None
    if dkv:
        rb.vrange.zero_()      # DKV reserves nothing: the selection's value scores are unused
    grp = args.group if args.group > 0 else cfg.n_inst
    groups = [(g0, min(cfg.n_inst, g0 + grp)) for g0 in range(0, cfg.n_inst, grp)]

    # the tokens of each period (B appended rows, the window, the decode queries),
    # drawn before the timed region and distinct for every round
    pool = token_pool(cfg, dev, args.warmup + args.steps, args.seed)

    def views_for(tok):
        out = []
        for g0, g1 in groups:
            out.append(dict(k=x["k"][g0:g1], v=x["v"][g0:g1], q_win=tok["q_win"][g0:g1],
                            q_dec=tok["q_dec"][g0:g1], attn=rb.attn[g0:g1], vrange=rb.vrange[g0:g1],
                            src=rb.src[g0:g1], out=rb.out[g0:g1], base=g0, n=g1 - g0,
                            g=g_buf[g0:g1] if dkv else None,
                            ord=rb.ord[g0:g1] if omap else None,
                            dl=dls[g0:g1] if dls is not None else None,
                            pa=phys_a[g0:g1] if phys_a is not None else None))
        return out
    views = [views_for(tok) for tok in pool]

    def append(tok):
        # the B rows the decoder appended since the previous round
        x["k"][:, K:, :].copy_(tok["k_new"])
        x["v"][:, K:, :].copy_(tok["v_new"])

    # value scores carried from one round's compaction to the next (Range, L2, Var)
    carry = args.carry == "on" and not dkv and value_kind != VALUE_KINDS["random"]
    carried = [False]
    # the data-fault word that score and select OR their status bits into
    st_word = torch.zeros(1, dtype=torch.int32, device=dev)

    def step(rnd, ev=None):
        # one full-model round: every group runs score -> select -> compact + decode
        p = rnd % len(pool)
        if ev: ev[0][5].record(stream)
        append(pool[p])
        for gi, gv in enumerate(views[p]):
            e = ev[gi] if ev else None
            if e: e[0].record(stream)
            if dkv:
                vase.dkv_projection(gv["n"], cfg.d, args.seed, rnd, r=DKV_RANK,
                                    inst_base=gv["base"], out=gv["g"], stream=stream)
                vase.dkv_score(gv["k"], gv["v"], gv["g"], K, B,
                               out=gv["pa"] if omap else gv["attn"], stream=stream,
                               q_dec=gv["q_dec"] if gv["dl"] is not None else None,
                               dec_logits=gv["dl"])
                if e: e[1].record(stream)
                if omap:      # into temporal order (DKV does not pool)
                    vase.order_scores(gv["pa"], gv["ord"], 1, attn=gv["attn"], stream=stream)
            elif omap:
                # vase_score_map: when one workgroup holds each instance (the Qwen3-8B
                # shape) the score kernel pools through the map itself
                vk = vase.VALUE_SKIP if carried[0] else value_kind
                vase.score(gv["k"], gv["v"], gv["q_win"], K, B, cfg.pool, attn=gv["attn"],
                           vrange=gv["vrange"], ws=rb.ws, stream=stream, value_kind=vk,
                           seed=args.seed, round=rnd, inst_base=gv["base"], ord=gv["ord"],
                           q_dec=gv["q_dec"] if gv["dl"] is not None else None,
                           dec_logits=gv["dl"], status=st_word)
                if e: e[1].record(stream)
            else:
                vk = vase.VALUE_SKIP if carried[0] else value_kind
                vase.score(gv["k"], gv["v"], gv["q_win"], K, B, cfg.pool, attn=gv["attn"],
                           vrange=gv["vrange"], ws=rb.ws, stream=stream, value_kind=vk,
                           seed=args.seed, round=rnd, inst_base=gv["base"], status=st_word)
                if e: e[1].record(stream)
            if e: e[2].record(stream)
            vase.select(gv["attn"], gv["vrange"], K, B, 0 if dkv else cfg.Nv, args.seed, rnd,
                        inst_base=gv["base"], flags=vase.DETERMINISTIC if dkv else 0,
                        src=gv["src"], stream=stream, status=st_word)
            if e: e[3].record(stream)
            if omap:
                vase.compact_decode_map(gv["k"], gv["v"], gv["src"], gv["ord"], K, B,
                                        q=gv["q_dec"], out=gv["out"], stream=stream,
                                        vrange_out=gv["vrange"] if carry else None,
                                        vrange_in=gv["vrange"] if carry else None,
                                        value_kind=value_kind, dec_logits=gv["dl"])
            else:
                vase.compact_decode(gv["k"], gv["v"], gv["src"], gv["q_dec"], K, B,
                                    out=gv["out"], ws=rb.ws, stream=stream,
                                    vrange_out=gv["vrange"] if carry else None,
                                    value_kind=value_kind)
            if e: e[4].record(stream)
        carried[0] = carry

    for r in range(args.warmup):
        step(r)
    torch.cuda.synchronize()
    # per group: [score start, score end, select start, select end, compact end, append start]
    events = [[[torch.cuda.Event(enable_timing=True) for _ in range(6)] for _ in groups]
              for _ in range(args.steps)]
    ar = torch.arange(K, device=dev, dtype=torch.int32)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for s in range(args.steps):
        step(args.warmup + s, events[s])
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    # rows that moved in the last round (counted outside the timed region); under
    # the order map exactly the B buffer rows of every instance move
    moved = cfg.n_inst * B if omap else int((rb.src != ar).sum().item())
    stage_ms = {"append": 0.0, "score": 0.0, "order": 0.0, "select": 0.0, "compact_decode": 0.0}
    for evs in events:
        stage_ms["append"] += evs[0][5].elapsed_time(evs[0][0])
        for ev in evs:
            for i, nme in enumerate(["score", "order", "select", "compact_decode"]):
                stage_ms[nme] += ev[i].elapsed_time(ev[i + 1])
    for nme in stage_ms:
        stage_ms[nme] /= args.steps
    step_ms = wall * 1e3 / args.steps
    event_step_ms = sum(events[s][0][5].elapsed_time(events[s][-1][4])
                        for s in range(args.steps)) / args.steps
    ab = carried_bytes(cfg, moved, carry, args, reads_values=args.value != "random")
    if dkv:
        ab["score"] = dkv_score_bytes(cfg) + (cfg.n_inst * K * 12 if omap else 0)
        if dls is not None:
            # the decode queries in, their logits over all N slots out, and the B
            # buffer rows of K and V read as well
            e_ = cfg.elem_bytes
            ab["score"] += cfg.n_inst * (cfg.G * (cfg.N * 4 + cfg.d * e_) + 2 * B * cfg.d * e_)
    round_ms = stage_ms["score"] + stage_ms["order"] + stage_ms["select"] + stage_ms["compact_decode"]
    round_bytes = ab["score"] + ab["select"] + ab["compact_decode"]
    round_gbs = round_bytes / (round_ms * 1e-3) / 1e9

    # dominant kernel: the score kernel (at this size one launch: both passes, Range
    # and pooling) or the fused compaction + decode kernel (one launch)
    # the map compaction runs its MFMA kernel for bf16 caches (GQA groups up to 8)
    map_kernel = ("compact_map_mfma_kernel" if cfg.dtype == "bf16" and cfg.G <= 8
                  else "compact_map_decode_kernel")
    cand = {
        (map_kernel if omap else "compact_decode_kernel"):
            ("hbm", ab["compact_decode"], stage_ms["compact_decode"], "GB/s", HBM_PEAK_GBS,
             ab["compact_decode"]),
    }
    if dkv:
        cand["dkv_score (projection + score)"] = ("hbm", ab["score"], stage_ms["score"], "GB/s",
                                                  HBM_PEAK_GBS, ab["score"])
    elif cfg.dtype == "bf16":
        cand["score_mfma_kernel"] = ("mfma", score_flops(cfg), stage_ms["score"], "TFLOP/s",
                                     MFMA_BF16_PEAK_TFS, ab["score"])
    else:
        # fp32 caches score on the VALU (one thread per row, then per slot)
        cand["score_rows_valu + score_cols_valu"] = ("alu", score_flops(cfg), stage_ms["score"],
                                                     "TFLOP/s", FP32_VECTOR_PEAK_TFS, ab["score"])
    dom = max(cand, key=lambda c: cand[c][2])
    roofline = roofline_entry(dom, cand[dom], cfg, args)

    target = target_v = None
    if not dkv and not args.no_target:
        # the steady-state round carries the value scores (as the step does) where
        # the layout and the value score allow; the round that reads V beside it
        can_carry = omap and args.carry == "on" and value_kind != VALUE_KINDS["random"]
        target = time_score_select_compact(args, cfg, x, rb, pool, append, stream, dev,
                                           carried=can_carry)
        if can_carry:
            target_v = time_score_select_compact(args, cfg, x, rb, pool, append, stream, dev,
                                                 carried=False)

    cpu = None
    if not args.no_cpu_baseline:
        cpu = cpu_baseline(cfg, x, args.cpu_sample, args.seed, method=args.method,
                           value=args.value)

    value = 1000.0 / step_ms
    line = {
        "metric": "eviction rounds/sec (all layers x heads, 1 GPU) + achieved HBM GB/s vs peak",
        "value": round(value, 3),
        "unit": "rounds/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(step_ms, 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16" if cfg.dtype == "bf16" else "f32",
        "data": "synthetic (seeded Qwen3-shaped caches: N(0,1) keys with 4 sink rows x10, "
                "N(0,1) values with log-uniform outlier rows, N(0,1) queries; fresh buffer rows, "
                "window and decode queries for every round)",
        "config": {
            "workload": (("VaSE-DKV (r=%d), " % DKV_RANK) if dkv else
                         "VaSE-AttnV, " if args.value == "range" else
                         "VaSE-AttnV with %s value score, " % args.value) +
                        "%s: %d layers x batch %d x %d KV heads (%d instances), G=%d, d=%d, "
                        "K=%d, B=%d, w=%d, N_v=%d, P=%d; one step = the B appended token rows "
                        "copied into the buffer, then score+select+compact on every instance + "
                        "one decode-attention step (fused with compaction)%s"
                        % (cfg.name, cfg.layers, cfg.batch, cfg.h_kv, cfg.n_inst, cfg.G, cfg.d,
                           cfg.K, cfg.B, cfg.w, 0 if dkv else cfg.Nv, cfg.pool,
                           "; value scores computed by each round's compaction for the rows it "
                           "writes, the next round's candidates" if carry else "") +
                        LAYOUT_NOTE[args.layout] +
                        ("; the score's pass over the keys also writes the decode queries' "
                         "logits, so the decode step reads V but not K" if dls is not None else ""),
            "layout": args.layout,
            "decode_logits_from_score": dls is not None,
            "method": args.method,
            "value_score": None if dkv else args.value,
            "value_scores_carried": carry,
            "n_inst": cfg.n_inst, "K": K, "B": B, "w": cfg.w, "N_v": cfg.Nv, "d": cfg.d,
            "G": cfg.G, "pool": cfg.pool, "instances_per_call": grp,
            "distinct_token_sets": len(pool),
        },
        "stage_ms": {k_: round(v_, 4) for k_, v_ in stage_ms.items()},
        "round_hbm": {"bytes": round_bytes, "ms": round(round_ms, 4), "GB/s": round(round_gbs, 1),
                      "frac_of_peak": round(round_gbs / HBM_PEAK_GBS, 4),
                      "moved_rows": moved,
                      "note": "score+select+compact+decode algorithmic bytes"},
        "dev_status": int(st_word.item()),
        "score_select_compact": target,
        "score_select_compact_reading_v": target_v,
        "event_ms_per_step": round(event_step_ms, 4),
        "roofline": roofline,
        "cpu_baseline": cpu,
    }
    print(json.dumps(line), flush=True)


def token_pool(cfg, dev, count, seed, budget_bytes=24e9):
    """Per-period token sets (appended rows, window, decode queries), one per round
    up to `count`, or as many as fit `budget_bytes` (then reused in turn)."""
    from paper_2606_03928_amd import synth
    e = cfg.elem_bytes
    per = cfg.n_inst * cfg.d * e * (2 * cfg.B + cfg.G * cfg.w + cfg.G)
    n = max(1, min(count, int(budget_bytes // per)))
    return [synth.draw_round_tokens(cfg, dev, cfg.n_inst, 7919 * (seed + 1) + i) for i in range(n)]


def read_peaks():
    """The measured peaks that `bench.py --peaks` wrote under profiles/, or None."""
    if not os.path.exists(PEAKS_JSON):
        return None
    with open(PEAKS_JSON) as f:
        return json.load(f)


def roofline_entry(dom, cand, cfg, args):
    """The dominant kernel against its roofline.  For the score kernel: the
    useful work is one pass of QK^T on bf16 MFMA (the method computes every
    window score once); its VALU work (one pass, and the two passes the kernel
    runs) and the measured traffic against the algorithmic bytes sit beside it."""
    bound, amount, ms, unit, peak, alg_bytes = cand
    achieved = amount / (ms * 1e-3) / (1e9 if unit == "GB/s" else 1e12)
    traffic = traffic_for("dkv_score_mfma_kernel" if dom.startswith("dkv_score") else dom,
                          workload_tag(args, cfg),
                          score_instantiation(cfg, uses_dec_logits(args, cfg))
                          if dom == "score_mfma_kernel" else None)
    out = {"bound": bound, "kernel": dom, "achieved": round(achieved, 1), "peak": peak,
           "unit": unit, "frac": round(achieved / peak, 4), "traffic": traffic,
           "algorithmic_bytes": int(alg_bytes), "kernel_ms": round(ms, 4),
           "traffic_ratio": round(traffic / alg_bytes, 3) if traffic else None}
    peaks = read_peaks()
    if dom == "score_mfma_kernel":
        executed = 2.0 * cfg.n_inst * cfg.R * (cfg.N + cfg.K) * cfg.d / (ms * 1e-3) / 1e12
        one = score_valu_ops(cfg, passes=1) / (ms * 1e-3) / 1e12
        two = score_valu_ops(cfg, passes=2) / (ms * 1e-3) / 1e12
        out["mfma_executed_TFLOP/s"] = round(executed, 1)
        out["alu_one_pass"] = {"achieved": round(one, 2), "peak": round(VALU_PEAK_TOPS, 2),
                               "unit": "TOP/s", "frac": round(one / VALU_PEAK_TOPS, 4)}
        out["alu_kernel_two_pass"] = {"achieved": round(two, 2), "peak": round(VALU_PEAK_TOPS, 2),
                                      "unit": "TOP/s", "frac": round(two / VALU_PEAK_TOPS, 4)}
        out["note"] = ("achieved: one pass of QK^T (2 G w N d flops per instance) over the "
                       "kernel's average launch time; alu: VALU lane-operations per window score "
                       "(fma, exp2 at half rate, add), one pass and the kernel's two, against "
                       "256 CUs x 4 SIMDs x 16 lanes x 2.4 GHz")
        if peaks:
            out["frac_of_measured_peak"] = round(achieved / peaks["mfma_bf16_TFLOP/s"], 4)
        st = (peaks or {}).get("score_step", {}).get("dma_from_hbm")
        if st and cfg.R == 512 and cfg.d == 128 and cfg.n_inst >= 512:
            # one workgroup of 8 waves per instance: each wave runs one step per
            # 32-key chunk of pass 1 (N slots) and of pass 2 (K candidates)
            steps = cfg.n_inst * 8 * (-(-cfg.N // 32) - (-cfg.K // 32)) / 1024.0
            k_ns = ms * 1e6 / steps
            p_ns = st["ms"] * 1e6 / st.get("wave_steps_per_simd", 2 * 8000)
            out["step_probe"] = {
                "kernel_ns_per_wave_step": round(k_ns, 1), "probe_ns_per_wave_step": round(p_ns, 1),
                "frac": round(p_ns / k_ns, 3),
                "note": "the kernel's launch time over its wave-steps per SIMD (instances x 8 "
                        "waves x (N/32 + K/32 chunks) / 1024 SIMDs) against the score-step probe "
                        "with the ring DMA from HBM (bench.py --peaks: the same per-step MFMA, "
                        "LDS, VALU, barrier and DMA stream on N(0,1) bf16 operands)"}
    elif unit == "GB/s" and peaks:
        out["frac_of_measured_peak"] = round(achieved / peaks["copy_GB/s"], 4)
    if peaks:
        out["measured_peaks"] = {k_: peaks[k_] for k_ in ("copy_GB/s", "read_GB/s",
                                                          "mfma_bf16_TFLOP/s", "exp2_T/s",
                                                          "fma_T/s") if k_ in peaks}
    return out


def compact_only_bytes(cfg, moved_rows, layout):
    """The compaction without a decode step: under the order map the survivor map
    and the order map are read, the new map written, and the B buffer rows of K
    and V read and written into the evicted slots; in the stable layout every row
    that moves is read and written."""
    e = cfg.elem_bytes
    if layout == "map":
        return cfg.n_inst * (12 * cfg.K + 4 * cfg.B * cfg.d * e)
    return cfg.n_inst * 4 * cfg.K + 4 * cfg.d * e * moved_rows


def time_score_select_compact(args, cfg, x, rb, pool, append, stream, dev, carried):
    """The round on its own: score, select, and the compaction without a decode
    step, every instance in one call each; same token sets as the main loop.
    carried: the compaction also leaves the next round's candidate value scores
    (the survivors keep theirs, the moved buffer rows are scored from the rows it
    copies), so the score reads no V after the first warm-up round; else every
    round's score reads V for them."""
    import torch
    from paper_2606_03928_amd import vase
    K, B = cfg.K, cfg.B
    omap = rb.ord is not None
    value_kind = VALUE_KINDS[args.value]
    base = 10000

    def one(rnd, ev=None):
        tok = pool[rnd % len(pool)]
        append(tok)
        vk = vase.VALUE_SKIP if carried and rnd > base else value_kind
        if ev: ev[0].record(stream)
        vase.score(x["k"], x["v"], tok["q_win"], K, B, cfg.pool, attn=rb.attn, vrange=rb.vrange,
                   ws=rb.ws, stream=stream, value_kind=vk, seed=args.seed, round=rnd,
                   ord=rb.ord)
        if ev: ev[1].record(stream)
        vase.select(rb.attn, rb.vrange, K, B, cfg.Nv, args.seed, rnd, src=rb.src, stream=stream)
        if ev: ev[2].record(stream)
        if omap:
            vase.compact_decode_map(x["k"], x["v"], rb.src, rb.ord, K, B, stream=stream,
                                    vrange_out=rb.vrange if carried else None,
                                    vrange_in=rb.vrange if carried else None,
                                    value_kind=value_kind)
        else:
            vase.compact(x["k"], x["v"], rb.src, K, B, ws=rb.ws, stream=stream)
        if ev: ev[3].record(stream)

    # a carried round needs one earlier round to have scored V
    w = max(args.warmup, 1) if carried else args.warmup
    for r in range(w):
        one(base + r)
    torch.cuda.synchronize()
    events = [[torch.cuda.Event(enable_timing=True) for _ in range(4)] for _ in range(args.steps)]
    for s_ in range(args.steps):
        one(base + w + s_, events[s_])
    torch.cuda.synchronize()
    ar = torch.arange(K, device=dev, dtype=torch.int32)
    moved = cfg.n_inst * B if omap else int((rb.src != ar).sum().item())
    st = {nm: sum(ev[i].elapsed_time(ev[i + 1]) for ev in events) / args.steps
          for i, nm in enumerate(["score", "select", "compact"])}
    ms = st["score"] + st["select"] + st["compact"]
    ab = algorithmic_bytes(cfg, moved, reads_values=args.value != "random" and not carried,
                           layout=args.layout)
    nbytes = ab["score"] + ab["select"] + compact_only_bytes(cfg, moved, args.layout)
    if carried:
        nbytes += cfg.n_inst * cfg.K * 8     # the value scores gathered by rank and written
    gbs = nbytes / (ms * 1e-3) / 1e9
    note = ("score (K over N slots twice in the kernel, counted once; no V: the value scores "
            "come from the previous round's compaction, which scores the B rows it moves) + "
            "select + compaction alone, no decode step" if carried else
            "score (K over N slots twice in the kernel, counted once; V over the K candidates) "
            "+ select + compaction alone, no decode step")
    return {"rounds_per_s": round(1000.0 / ms, 3), "ms": round(ms, 4),
            "stage_ms": {k_: round(v_, 4) for k_, v_ in st.items()},
            "bytes": int(nbytes), "GB/s": round(gbs, 1), "frac_of_peak": round(gbs / HBM_PEAK_GBS, 4),
            "moved_rows": moved, "value_scores_carried": carried,
            "note": note + "; event time of the three calls per round, the appends excluded"}


def run_peaks(dev):
    """Measured copy, read, MFMA, exp2 and fma rates (medians of 5 timed launches)."""
    import ctypes
    import statistics
    import torch
    from paper_2606_03928_amd import build as hb
    if not os.path.exists(hb.PEAKS_PATH):
        print("libvase_peaks.so is missing: run the build first", file=sys.stderr)
        sys.exit(2)
    lib = ctypes.CDLL(hb.PEAKS_PATH)
    P, I, SZ = ctypes.c_void_p, ctypes.c_int, ctypes.c_size_t
    lib.peaks_copy.argtypes = [P, P, SZ, I, I, P]
    lib.peaks_read.argtypes = [P, SZ, I, I, P, P]
    lib.peaks_mfma.argtypes = [I, I, P, P]
    lib.peaks_exp2.argtypes = [I, I, P, P]
    lib.peaks_fma.argtypes = [I, I, P, P]
    lib.peaks_coexec.argtypes = [I, I, I, P, P]
    lib.peaks_score_step.argtypes = [I, P, SZ, I, I, P, P, P]
    stream = torch.cuda.current_stream(dev)
    sp = ctypes.c_void_p(stream.cuda_stream)

    def timed(launch, reps=5):
        launch()
        torch.cuda.synchronize()
        ts = []
        for _ in range(reps):
            a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            a.record(stream)
            assert launch() == 0
            b.record(stream)
            torch.cuda.synchronize()
            ts.append(a.elapsed_time(b) * 1e-3)
        return statistics.median(ts)

    nbytes = 4 << 30
    src = torch.ones(nbytes // 4, dtype=torch.int32, device=dev)
    dst = torch.empty_like(src)
    n16 = nbytes // 16
    out = torch.empty(n16, dtype=torch.float32, device=dev)    # one word per thread of any launch
    sweep = {}
    for blocks in (256 * 8, 256 * 32):
        for unroll in (1, 4, 8):
            tc = timed(lambda: lib.peaks_copy(P(src.data_ptr()), P(dst.data_ptr()), n16, blocks,
                                              unroll, sp))
            tr = timed(lambda: lib.peaks_read(P(src.data_ptr()), n16, blocks, unroll,
                                              P(out.data_ptr()), sp))
            sweep["copy b%d u%d" % (blocks, unroll)] = round(2 * nbytes / tc / 1e9, 1)
            sweep["read b%d u%d" % (blocks, unroll)] = round(nbytes / tr / 1e9, 1)
    # one 16-byte piece per thread, the grid covering the buffer
    full = n16 // 256
    tc = timed(lambda: lib.peaks_copy(P(src.data_ptr()), P(dst.data_ptr()), n16, full, 1, sp))
    tr = timed(lambda: lib.peaks_read(P(src.data_ptr()), n16, full, 1, P(out.data_ptr()), sp))
    sweep["copy one piece per thread"] = round(2 * nbytes / tc / 1e9, 1)
    sweep["read one piece per thread"] = round(nbytes / tr / 1e9, 1)
    t_torch = timed(lambda: (dst.copy_(src), 0)[1])
    sweep["copy torch"] = round(2 * nbytes / t_torch / 1e9, 1)
    del src, dst
    it = 4096
    for mb in (256 * 2, 256 * 4, 256 * 8):      # 2, 4, 8 waves per SIMD
        t = timed(lambda: lib.peaks_mfma(mb, it, P(out.data_ptr()), sp))
        sweep["mfma %dw/SIMD" % (mb // 256)] = round(mb * 4 * it * 4 * 2.0 * 32 * 32 * 16 / t / 1e12, 1)
    eb = 256 * 16
    t_exp = timed(lambda: lib.peaks_exp2(eb, it, P(out.data_ptr()), sp))
    t_fma = timed(lambda: lib.peaks_fma(eb, it, P(out.data_ptr()), sp))
    ops = eb * 256 * it * 8.0
    # MFMA and VALU co-execution at 2 waves per SIMD (512 workgroups of 4 waves)
    coexec = {}
    for w_, nm in enumerate(("mfma_only_ms", "valu_only_ms", "interleaved_in_each_wave_ms",
                             "split_over_two_waves_ms")):
        coexec[nm] = round(timed(lambda: lib.peaks_coexec(w_, 512, 2000, P(out.data_ptr()), sp)) * 1e3, 3)
    # the score kernel's key-loop step (256 workgroups of 8 waves, one per CU, 8000
    # steps per wave, about 6 ms per launch so that the clock settles): time,
    # shader clock (the last launch's shader cycles over its 100 MHz reference
    # cycles) and cycles per wave-step, without data movement, with the ring
    # DMA served from L2 or from HBM, and without the epilogue
    # N(0, 1) bf16 operands, as the synthetic keys and queries
    src2 = torch.randn((2 << 30) // 2, dtype=torch.bfloat16, device=dev)
    clk = torch.zeros(2 * 256, dtype=torch.int64, device=dev)
    score_step = {}
    for which, nm in enumerate(("no_memory", "dma_from_l2", "dma_from_hbm", "no_epilogue",
                                "no_memory_patterned_operands")):
        t = timed(lambda: lib.peaks_score_step(which, P(src2.data_ptr()), src2.numel() * 2, 256, 1000,
                                               P(out.data_ptr()), P(clk.data_ptr()), sp))
        ck = clk.view(256, 2).double().sum(0)
        ghz = float(ck[0] / ck[1]) * 0.1
        score_step[nm] = {"ms": round(t * 1e3, 4), "GHz": round(ghz, 3),
                          "wave_steps_per_simd": 2 * 8000,
                          "cycles_per_wave_step": round(t * ghz * 1e9 / (2 * 8000), 1)}
    del src2
    best = lambda pre: max(v_ for k_, v_ in sweep.items() if k_.startswith(pre))
    res = {"copy_GB/s": best("copy"),
           "read_GB/s": best("read"),
           "mfma_bf16_TFLOP/s": best("mfma"),
           "exp2_T/s": round(ops / t_exp / 1e12, 3),
           "fma_T/s": round(ops / t_fma / 1e12, 3),
           "sweep": sweep,
           "coexec": coexec,
           "score_step": score_step,
           "datasheet": {"hbm_GB/s": HBM_PEAK_GBS, "mfma_bf16_TFLOP/s": MFMA_BF16_PEAK_TFS,
                         "valu_fp32_lane_ops_T/s": round(VALU_PEAK_TOPS, 2)},
           "method": "median of 5 launches each, HIP events on the launch stream; each peak is "
                     "the best of its sweep: copy (read + write bytes) and read of 4 GiB with "
                     "2048 or 8192 workgroups of 256 threads and 1, 4 or 8 16-byte pieces in "
                     "flight per thread, one piece per thread over the whole buffer, and torch's "
                     "device copy; 4 independent "
                     "v_mfma_f32_32x32x16_bf16 chains per wave, 4096 steps, at 2, 4 and 8 "
                     "waves per SIMD; 4096 workgroups x 256 threads x 8 independent v_exp_f32 "
                     "(or fp32 fma) chains, 4096 steps; coexec: 512 workgroups of 4 waves (2 per "
                     "SIMD), 2000 steps of 16 v_mfma_f32_32x32x16_bf16 and/or 32 x (fma, exp2, add) "
                     "per wave, interleaved in every wave or split over even and odd waves; "
                     "score_step: the score kernel's key-loop step on synthetic operands (8 waves "
                     "per workgroup, 256 workgroups, 8000 steps per wave of 16 MFMAs with LDS "
                     "B operands and 32 x (fma, exp2, add), a barrier every 2 steps), without data "
                     "movement, with one 1 KB global->LDS DMA per wave and step from a 2 MiB (L2) "
                     "or 2 GiB (HBM) window of N(0, 1) bf16 data (the operands come from it too), "
                     "without the epilogue, and on a few repeated small operand values; clock "
                     "from s_memtime over "
                     "s_memrealtime",
           "gpu": torch.cuda.get_device_name(dev)}
    print(json.dumps(res), flush=True)


if __name__ == "__main__":
    main()
