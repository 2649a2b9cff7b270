#!/usr/bin/env python3
"""Throughput of the bucket reducer on one MI355X.

One step = one call of nf_route_buckets over every bucket of the workload:
pass 1 (sign payload, health statistics, FP32 sums at routed positions),
the per-bucket decision, and pass 2 (sign counts and decode, or the FP32
fallback), for all W stacked workers.  Inputs are generated on the device
before the timed region and stay resident in HBM.

Metric: FP32-equivalent input GB/s = 4 * W * n_total / step time, and its
fraction of the 8 TB/s HBM peak, over the timed steps, which record four
HIP events each for the phase split.  The JSON line also carries
  without_phase_events  the same number of steps timed again without those
                events (their records cost a few microseconds per step,
                which shows only on the small workloads)
  roofline      the dominant kernel (pass 1): algorithmic bytes per launch
                over its average launch time, from HIP events the library
                records on its own launch stream; `traffic` is the counter-
                measured HBM bytes per launch from a committed rocprofv3 run
                of the current kernel source (else null)
  cpu_baseline  the oracle, single-threaded on one pinned host core, on a
                bounded sample of the same workload
  achievable    a plain streaming read of the same input (reference rate)
  configs       (default run) every other workload: G-Ternary at GPT scale,
                GPT scale in DDP's buckets, ViT-B/16 and ResNet-50 scale, the tiny bucket, the stress
                bucket, the W = 255 pair; each with its pass-1 roofline
                (`traffic` from that workload's committed counters) and the
                counter bytes per dispatch of every kernel of its step

  python bench.py [--gpus 1] [--steps 20] [--warmup 3] [--workload gpt1p3b]
  python bench.py --calibrate-copy     (copy kernel of known size, for counters)
"""
import argparse
import ctypes
import hashlib
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

HBM_PEAK_GBS = 8000.0  # MI355X HBM3E, AMD specification
COPY_CAL_BYTES = 4 << 30  # bytes read (and written) by the calibration copy


def parse():
    ap = argparse.ArgumentParser(description=__doc__, formatter_class=argparse.RawDescriptionHelpFormatter)
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--workload", default=None,
                    choices=["tiny", "resnet50", "vitb16", "gpt1p3b", "stress", "fanin255"],
                    help="measure this workload only (default: the GPT-1.3B-scale headline, then a few "
                         "steps of every other workload in the JSON line's `configs`)")
    ap.add_argument("--force-lowbit", action="store_true", help="guard disabled (forced low-bit)")
    ap.add_argument("--ddp-buckets", action="store_true",
                    help="buckets cut as DDP cuts the model (25 MiB capacity, closed at tensor boundaries) "
                         "through the bucket-table driver, instead of equal 25 MiB buckets")
    ap.add_argument("--no-counts", action="store_true", help="do not write the uint8 counts")
    ap.add_argument("--cold", action="store_true",
                    help="overwrite 1 GiB before every step so the caches hold none of the input; value "
                         "then comes from the per-step device events, which exclude the overwrite")
    ap.add_argument("--format", default="binary", choices=["binary", "ternary"],
                    help="low-bit payload: G-Binary sign counts or G-Ternary two-plane counts")
    ap.add_argument("--tau", type=float, default=0.5, help="G-Ternary gate (units of mean |g|)")
    ap.add_argument("--cpu-buckets", type=int, default=None,
                    help="buckets of the oracle's CPU sample (default: about 15 s of work)")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-probe", action="store_true", help="skip the streaming-read reference")
    ap.add_argument("--no-split", action="store_true", help="skip the standalone entry points on one bucket")
    ap.add_argument("--calibrate-copy", action="store_true",
                    help="only run the copy kernel of known traffic (counter calibration)")
    ap.add_argument("--contrast", action="store_true",
                    help="only time hierarchical vs stock vs direct sign counting (one JSON line per shape)")
    ap.add_argument("--sliced", action="store_true",
                    help="only time the compacted payload and per-slice scale kernels on the workload")
    ap.add_argument("--controller", type=int, default=0, metavar="STEPS",
                    help="only run STEPS controller-driven reducer steps (Supervisor + endpoint guard feeding "
                         "the route policy) on the chosen workload and report route evidence")
    return ap.parse_args()


class HipEvents:
    """hipEvent_t handles from the HIP runtime torch has loaded."""

    def __init__(self):
        self.rt = ctypes.CDLL("libamdhip64.so.7")
        self.rt.hipEventCreate.argtypes = [ctypes.POINTER(ctypes.c_void_p)]
        self.rt.hipEventElapsedTime.argtypes = [ctypes.POINTER(ctypes.c_float), ctypes.c_void_p,
                                                ctypes.c_void_p]
        self.rt.hipEventDestroy.argtypes = [ctypes.c_void_p]

    def create(self):
        ev = ctypes.c_void_p()
        if self.rt.hipEventCreate(ctypes.byref(ev)) != 0:
            raise RuntimeError("hipEventCreate failed")
        return ev.value

    def elapsed_ms(self, a, b):
        ms = ctypes.c_float()
        if self.rt.hipEventElapsedTime(ctypes.byref(ms), a, b) != 0:
            raise RuntimeError("hipEventElapsedTime failed")
        return ms.value

    def destroy(self, ev):
        self.rt.hipEventDestroy(ev)


def kernel_source_sha():
    """Hash of the pass-1 kernel source, its device helpers and the geometry that shapes its launches."""
    h = hashlib.sha256()
    for name in ("nf_pass1.hip", "nf_device.h", "nf_internal.h"):
        h.update(open(os.path.join(ROOT, "paper_2606_25759_amd", "csrc", name), "rb").read())
    return h.hexdigest()[:16]


def all_kernels_sha():
    """Hash of every kernel source of the library and the geometry header."""
    h = hashlib.sha256()
    csrc = os.path.join(ROOT, "paper_2606_25759_amd", "csrc")
    for name in sorted(os.listdir(csrc)):
        if name.endswith((".hip", ".h")):
            h.update(name.encode())
            h.update(open(os.path.join(csrc, name), "rb").read())
    return h.hexdigest()[:16]


def counter_traffic(workload):
    """HBM bytes per pass-1 launch from committed rocprofv3 counters, if they
    were taken on the current kernel source; else None."""
    path = os.path.join(ROOT, "profiles", f"pass1_{workload}_counters.json")
    if not os.path.exists(path):
        return None
    rec = json.load(open(path))
    if rec.get("kernel_sha") != kernel_source_sha():
        return None
    return rec.get("hbm_bytes_per_launch")


def host_cpu():
    model = "unknown"
    try:
        for line in open("/proc/cpuinfo"):
            if line.startswith("model name"):
                model = line.split(":", 1)[1].strip()
                break
    except OSError:
        pass
    return model, os.cpu_count()


def calibrate_copy():
    import torch
    import synth
    n = COPY_CAL_BYTES // 4
    src = torch.ones(n, dtype=torch.float32, device="cuda:0")
    dst = torch.empty_like(src)
    for _ in range(3):
        synth.copy(src, dst)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    reps = 5
    for _ in range(reps):
        synth.copy(src, dst)
    torch.cuda.synchronize()
    ms = (time.perf_counter() - t0) * 1e3 / reps
    print(json.dumps({"kernel": "k_copy", "bytes_read_per_dispatch": COPY_CAL_BYTES,
                      "bytes_written_per_dispatch": COPY_CAL_BYTES, "ms": round(ms, 4),
                      "gbs_each_way": round(COPY_CAL_BYTES / ms / 1e6, 1)}), flush=True)
    return 0


# (nodes, GPUs per node, elements): the paper's local-count logical buckets (8 workers x 131K and
# x 524K elements, 2 nodes x 4 GPUs), and one 25 MiB bucket at 4 x 4 and 8 x 8 workers.
CONTRAST_SHAPES = [(2, 4, 131_072), (2, 4, 524_288), (4, 4, 6_553_600), (8, 8, 6_553_600)]
# Context only (another machine): mean local-count route times of the paper's reducer check on
# 2 nodes x 4 A100 (its Table 9): 8 x 131K -> 260 us, 8 x 524K -> 570 us.
PAPER_LOCAL_COUNT_US = {131_072: 260.0, 524_288: 570.0}


def contrast(reps=50):
    """Kernel time of three ways to turn W sign bitmaps into counts and the decoded aggregate:
    direct (one bit-sliced count over all W rows), hierarchical (node-local partial counts over
    each node's P rows, then the partial-count sum and decode), and stock (every one of the W
    workers counts all W rows and decodes itself: W replicas)."""
    import torch
    import paper_2606_25759_amd as nf

    dev = torch.device("cuda:0")
    gen = torch.Generator(device=dev)
    gen.manual_seed(11)

    def timed(fn):
        fn()
        torch.cuda.synchronize()
        a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        a.record()
        for _ in range(reps):
            fn()
        b.record()
        torch.cuda.synchronize()
        return a.elapsed_time(b) * 1e3 / reps  # us per call

    for nodes, per, n in CONTRAST_SHAPES:
        W = nodes * per
        nw = (n + 63) // 64
        bits = torch.randint(-2 ** 62, 2 ** 62, (W, nw), dtype=torch.int64, device=dev, generator=gen)
        mask = torch.full((nw,), -1, dtype=torch.int64, device=dev)
        scale = torch.full((1,), 1e-3, dtype=torch.float32, device=dev)
        counts = torch.empty(n, dtype=torch.uint8, device=dev)
        out = torch.empty(n, dtype=torch.float32, device=dev)
        stride = (n + 15) // 16 * 16
        partial = torch.empty((nodes, stride), dtype=torch.uint8, device=dev)
        sc = torch.empty(W * stride, dtype=torch.uint8, device=dev)
        so = torch.empty(W * stride, dtype=torch.float32, device=dev)
        t_direct = timed(lambda: nf.nf_signcount_reduce(bits, W, n, mask, scale, 0, counts, out))
        t_local = timed(lambda: nf.nf_partial_counts(bits, W, per, n, partial))
        t_exch = timed(lambda: nf.nf_partial_count_reduce(partial, W, n, mask, scale, 0, counts, out))
        t_hier = timed(lambda: (nf.nf_partial_counts(bits, W, per, n, partial),
                                nf.nf_partial_count_reduce(partial, W, n, mask, scale, 0, counts, out)))
        t_stock = timed(lambda: nf.nf_stock_signcount(bits, W, n, mask, scale, 0, W, sc, so, stride))
        torch.cuda.synchronize()
        ok = bool(torch.equal(sc[:n], counts))
        rec = {"metric": "sign-count kernel time, hierarchical vs stock (one GPU)", "unit": "us",
               "config": {"nodes": nodes, "gpus_per_node": per, "W": W, "n": n},
               "direct_us": round(t_direct, 2), "hier_local_us": round(t_local, 2),
               "hier_exchange_return_us": round(t_exch, 2), "hier_total_us": round(t_hier, 2),
               "stock_total_us": round(t_stock, 2), "stock_per_worker_us": round(t_stock / W, 2),
               "stock_over_hier": round(t_stock / t_hier, 2), "replica_parity": "ok" if ok else "MISMATCH",
               "bits_read_gb_direct": round(8 * W * nw / 1e9, 4),
               "paper_local_count_us_a100": PAPER_LOCAL_COUNT_US.get(n) if W == 8 else None}
        print(json.dumps(rec), flush=True)
        del bits, sc, so, partial
    return 0


def controller_run(args):
    """A synthetic training run in which the host controller supplies each step's route policy:
    Commander admission, Supervisor CUSUM recovery and the route-use budget from a loss trace,
    and the endpoint-capacity guard from a cost model.  Every step runs the reducer on the GPU;
    its route decisions go back to the controller (L/F/P events, MGTR)."""
    import numpy as np
    import torch
    import paper_2606_25759_amd as nf
    import synth

    dev = torch.device("cuda:0")
    lay = synth.CONFIGS[args.workload]()
    W, n, bn, nb = lay.W, lay.n_total, lay.bucket_n, lay.nb
    nw = (n + 63) // 64
    grads = torch.empty((W, lay.stride), dtype=torch.float32, device=dev)
    synth.generate_device(lay, grads)
    off, ln, el = synth.mask_segments(lay)
    mask_h = nf.nf_mask_from_segments(off, ln, el, n)
    mask = torch.from_numpy(mask_h.view(np.int64)).to(dev)
    ternary = args.format == "ternary"
    planes = 2 if ternary else 1
    bits = torch.empty((planes * W, nw), dtype=torch.int64, device=dev)
    out = torch.empty(n, dtype=torch.float32, device=dev)
    stats = torch.empty(nb * W * nf.STATS_BYTES, dtype=torch.uint8, device=dev)
    dec = torch.empty(nb * nf.DECISION_BYTES, dtype=torch.uint8, device=dev)
    ws = nf.empty_workspace(nf.nf_workspace_bytes_buckets(W, n, bn), dev)

    # Operating profile in the style of the paper's Transformer row (Table 2: slack 2.11e-4, threshold
    # 1.01e-2, one-epoch cooldown, a post-recovery guard); an epoch is 50 steps here, the guard lasts
    # two cooldowns with the threshold halved, admission after a 40-step warm-up, a 0.8 route-use target.
    T = args.controller
    prof = nf.supervisor_profile(admit_step=40, cooldown_steps=50, guard_steps=100, short_cooldown_steps=5,
                                 ema_alpha=0.1, slack=2.11e-4, threshold=1.01e-2, guard_scale=0.5,
                                 near_band=0.25, small_move=5e-3, target_share=0.8, share_margin=0.03)
    state = nf.nf_supervisor_init(prof)
    # Endpoint guard for a full bucket: 2 nodes x (W/2) GPUs, 25 GB/s links, 100 GB/s endpoint counting.
    elig = np.unpackbits(mask_h[: bn // 64].view(np.uint8), bitorder="little").sum()
    model = nf.nf_endpoint_model(2, max(1, W // 2), planes, 0, 25e9, 100e9, 20e-6, 30e-6)
    t_fp32, t_low, guard_ok = nf.nf_endpoint_guard(model, min(bn, n), int(elig))
    # Synthetic loss: a decaying curve with noise and two degradation episodes.
    rng = np.random.default_rng(17)
    t = np.arange(T)
    loss = 0.7 * np.exp(-t / 300.0) + 0.3 + rng.normal(0, 2e-3, T)
    for a in (T // 3, (2 * T) // 3):
        loss[a:a + 30] += np.linspace(0.0, 0.05, 30)[: len(loss[a:a + 30])]
    routes_per_step = []
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for k in range(T):
        pol = nf.nf_supervisor_policy(prof, state, nf.policy(guard_ok=int(guard_ok), format=int(ternary)))
        nf.nf_route_buckets(grads, n, bn, mask, pol, bits, None, out, stats, dec, ws)
        d = nf.decisions_host(dec, nb)  # synchronises the stream
        nf.nf_supervisor_update(prof, state, d, float(loss[k]))
        routes_per_step.append((int((d["route"] == 0).sum()), int((d["route"] == 1).sum()),
                                int((d["route"] == 2).sum())))
    wall = time.perf_counter() - t0
    rec = {"metric": "controller-driven reducer run (route evidence)", "config": {
               "workload": lay.name, "W": W, "buckets": nb, "steps": T, "format": args.format},
           "endpoint_guard": {"t_fp32_us": round(t_fp32 * 1e6, 2), "t_lowbit_us": round(t_low * 1e6, 2),
                              "guard_ok": guard_ok},
           "events": {"L": state.events_l, "F": state.events_f, "P": state.events_p},
           "lowbit_share": round(state.events_l / max(1, state.events_l + state.events_f + state.events_p), 4),
           "mgtr": round(state.bytes_route / state.bytes_fp32, 4),
           "alarms": state.alarms, "short_recoveries": state.short_recoveries,
           "readmissions": state.readmissions, "budget_vetoes": state.budget_vetoes,
           "ms_per_step_wall": round(wall * 1e3 / T, 3),
           "first_lowbit_step": next((i for i, r in enumerate(routes_per_step) if r[0]), None)}
    print(json.dumps(rec), flush=True)
    return 0


def sliced_run(args, reps=5):
    """Kernel times of the compacted eligible-only payload and per-slice scales over the whole
    workload (every eligible tensor of the binding is one slice): compaction of the positional sign
    rows, the per-slice statistics and scales (with a second read of the gradients, and from pass
    1's chunk partials), the count + decode from the compacted rows, and the whole sliced step:
    pass 1 over the buffer as one bucket, compaction, scales from pass 1, count + decode."""
    import numpy as np
    import torch
    import paper_2606_25759_amd as nf
    import synth

    dev = torch.device("cuda:0")
    lay = synth.CONFIGS[args.workload]()
    W, n, bn, nb = lay.W, lay.n_total, lay.bucket_n, lay.nb
    nw = (n + 63) // 64
    grads = torch.empty((W, lay.stride), dtype=torch.float32, device=dev)
    synth.generate_device(lay, grads)
    off, ln, el = synth.mask_segments(lay)
    e = np.asarray(el, bool)
    sl = nf.SlicedLayout(np.asarray(off)[e], np.asarray(ln)[e], n, device=dev)
    mask = sl.d_mask
    bits = torch.empty((W, nw), dtype=torch.int64, device=dev)
    out = torch.empty(n, dtype=torch.float32, device=dev)
    stats = torch.empty(nb * W * nf.STATS_BYTES, dtype=torch.uint8, device=dev)
    dec = torch.empty(nb * nf.DECISION_BYTES, dtype=torch.uint8, device=dev)
    ws = nf.empty_workspace(nf.nf_workspace_bytes_buckets(W, n, bn), dev)
    nf.nf_route_buckets(grads, n, bn, mask, nf.policy(force_lowbit=1), bits, None, out, stats, dec, ws)
    nwc = (sl.n_eligible + 63) // 64
    cbits = torch.empty((W, nwc), dtype=torch.int64, device=dev)
    sums = torch.empty((sl.S, W), dtype=torch.float64, device=dev)
    scales = torch.empty(sl.S, dtype=torch.float32, device=dev)
    ws2 = nf.empty_workspace(nf.nf_slice_workspace_bytes(W, sl.segments), dev)
    counts_c = torch.empty(sl.n_eligible, dtype=torch.uint8, device=dev)

    def timed(fn):
        fn()
        torch.cuda.synchronize()
        a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        a.record()
        for _ in range(reps):
            fn()
        b.record()
        torch.cuda.synchronize()
        return a.elapsed_time(b) / reps  # ms per call

    # pass 1 over the whole buffer as one bucket, whose chunk partials give the slice statistics
    ws1 = nf.empty_workspace(nf.nf_workspace_bytes(W, n), dev)
    stats1 = torch.empty(W * nf.STATS_BYTES, dtype=torch.uint8, device=dev)
    t_pack = timed(lambda: nf.nf_pack_signs(grads, n, mask, bits, stats1, ws1))
    t_from1 = timed(lambda: nf.nf_slice_scales_from_pass1(grads, n, sl, sums, scales, ws1))

    def chain():
        nf.nf_pack_signs(grads, n, mask, bits, stats1, ws1)
        nf.nf_compact_signs(bits, W, n, sl, cbits)
        nf.nf_slice_scales_from_pass1(grads, n, sl, sums, scales, ws1)
        nf.nf_compact_signcount_reduce(cbits, W, sl, scales, 0, counts_c, out)
    t_chain = timed(chain)
    t_compact = timed(lambda: nf.nf_compact_signs(bits, W, n, sl, cbits))
    t_scales = timed(lambda: nf.nf_slice_scales(grads, sl, sums, scales, ws2))
    t_reduce = timed(lambda: nf.nf_compact_signcount_reduce(cbits, W, sl, scales, 0, counts_c, out))
    t_count = timed(lambda: nf.nf_compact_signcount_reduce(cbits, W, sl, scales, 0, counts_c, None))
    nE, S = sl.n_eligible, sl.S
    b_compact = 8 * W * nw + 16 * nw + 8 * W * nwc          # positional rows, mask + prefix, compacted rows
    b_scales = 4 * W * nE                                  # the eligible gradients once
    b_reduce = 8 * W * nwc + nE + nE + 20 * nw + 4 * nE    # rows, counts out and in, tables, decoded values
    gbs = lambda b, t: round(b / (t * 1e-3) / 1e9, 1)
    rec = {"metric": "compacted payload and per-slice scales, kernel times", "unit": "ms",
           "config": {"workload": lay.name, "W": W, "n": n, "n_eligible": nE, "slices": S},
           "compact_ms": round(t_compact, 4), "compact_gbs": gbs(b_compact, t_compact),
           "slice_scales_ms": round(t_scales, 4), "slice_scales_gbs": gbs(b_scales, t_scales),
           "slice_scales_from_pass1_ms": round(t_from1, 4),
           "pack_one_bucket_ms": round(t_pack, 4),
           "sliced_step_ms": round(t_chain, 4),
           "sliced_step_gbs_fp32_equiv": gbs(lay.input_bytes(), t_chain),
           "compact_reduce_ms": round(t_reduce, 4), "compact_reduce_gbs": gbs(b_reduce, t_reduce),
           "of_which_count_ms": round(t_count, 4),
           "payload_bytes_per_worker": {"positional": 8 * nw, "compacted": 8 * nwc},
           "mgtr_sliced_compacted": round((nE / 8 + 4 * S + 4 * (n - nE)) / (4 * n), 5),
           "mgtr_bucket_scale_positional_bits": round((nw * 8 + 4 * nb + 4 * (n - nE)) / (4 * n), 5)}
    print(json.dumps(rec), flush=True)
    return 0


def pattern_probe(synth, torch, wl, reps=3):
    """The first pass's read schedule without its arithmetic (16 rows in
    chunks of 16 x 16,384 elements, launches of 256 chunks), alone and with
    1/32 of the bytes read written back as 2 KiB rows at each chunk's end
    (the sign words' share and layout), or 2/32 (two planes, the G-Ternary
    pack's share): the rates the reducer's first pass and the pack are
    bounded by on this machine."""
    n = wl.n // 16384 * 16384
    res = {"elements_per_row": n}
    dst = torch.empty((32, n // 64), dtype=torch.int64, device=wl.dev)  # not the reducer's outputs
    for store in (0, 1, 2):
        synth.pattern_probe(wl.grads, dst, n, store)
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        for _ in range(reps):
            launches = synth.pattern_probe(wl.grads, dst, n, store)
        torch.cuda.synchronize()
        ms = (time.perf_counter() - t0) * 1e3 / reps
        nbytes = 4 * 16 * n + 2 * n * store
        res[("read_only", "read_write", "read_write_two_planes")[store]] = {
            "ms": round(ms, 3), "gbs": round(nbytes / ms / 1e6, 1), "bytes": nbytes, "launches": launches}
    del dst
    print(f"[bench] first-pass pattern probe: reads only {res['read_only']['ms']:.3f} ms "
          f"({res['read_only']['gbs']} GB/s), with the 1/32 writes {res['read_write']['ms']:.3f} ms "
          f"({res['read_write']['gbs']} GB/s), with 2/32 {res['read_write_two_planes']['ms']:.3f} ms "
          f"({res['read_write_two_planes']['gbs']} GB/s)", file=sys.stderr, flush=True)
    return res


def split_one_bucket(nf, torch, grads, mask, W, n, n_e, reps=10):
    """Device time of each standalone entry point on one bucket of n elements
    (the first), with the algorithmic bytes each one moves."""
    dev = grads.device
    nw = (n + 63) // 64
    g0, m0 = grads[:, :n], mask[:nw]
    bits = torch.empty((W, nw), dtype=torch.int64, device=dev)
    counts = torch.empty(n, dtype=torch.uint8, device=dev)
    out = torch.empty(n, dtype=torch.float32, device=dev)
    stats = torch.empty(W * nf.STATS_BYTES, dtype=torch.uint8, device=dev)
    ws = nf.empty_workspace(nf.nf_workspace_bytes(W, n), dev)
    scale = torch.full((1,), 1e-4, dtype=torch.float32, device=dev)
    calls = {
        "nf_bucket_health": (lambda: nf.nf_bucket_health(g0, n, m0, stats, ws), 4 * W * n + 8 * nw),
        "nf_pack_signs": (lambda: nf.nf_pack_signs(g0, n, m0, bits, stats, ws), 4 * W * n + 8 * nw + 8 * W * nw),
        # the FP32 path at every position (route F/P's full-precision sum of the bucket)
        "nf_fp32_reduce": (lambda: nf.nf_fp32_reduce(g0, n, m0, nf.NF_SEL_ALL, nf.NF_FP32_SUM, out),
                           4 * W * n + 8 * nw + 4 * n),
        "nf_signcount_reduce": (lambda: nf.nf_signcount_reduce(bits, W, n, m0, scale, nf.NF_DECODE_SOFT, counts, out),
                                8 * W * nw + 8 * nw + n + 4 * n_e),
    }
    res = {"bucket_elements": n, "eligible": n_e}
    for name, (fn, nbytes) in calls.items():
        fn()
        torch.cuda.synchronize()
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record()
        for _ in range(reps):
            fn()
        e1.record()
        torch.cuda.synchronize()
        ms = e0.elapsed_time(e1) / reps
        res[name] = {"ms": round(ms, 4), "algorithmic_gbs": round(nbytes / ms / 1e6, 1)}
    return res


class Workload:
    """One workload's device buffers, generated once, and measurements of
    one driver call over all of its buckets under a given policy: equal
    buckets (nf_route_buckets) or, after set_buckets(offsets), the buckets of
    a bucket table (nf_route_bucket_table)."""

    def __init__(self, nf, torch, name, planes=1, ddp=False):
        import numpy as np
        import synth
        self.nf, self.torch, self.np = nf, torch, np
        self.dev = torch.device("cuda:0")
        self.lay = lay = synth.CONFIGS[name]()
        self.W, self.n = lay.W, lay.n_total
        W, n = self.W, self.n
        self.nw = (n + 63) // 64
        self.grads = torch.empty((W, lay.stride), dtype=torch.float32, device=self.dev)
        synth.generate_device(lay, self.grads)
        self.segs = synth.mask_segments(lay)
        self.mask_h = nf.nf_mask_from_segments(*self.segs, n)
        self.mask = torch.from_numpy(self.mask_h.view(np.int64)).to(self.dev)
        self.planes = planes  # 2: room for G-Ternary's positive and negative planes
        self.bits = torch.empty((planes * W, self.nw), dtype=torch.int64, device=self.dev)
        self.counts = torch.empty(planes * n, dtype=torch.uint8, device=self.dev)
        self.out = torch.empty(n, dtype=torch.float32, device=self.dev)
        self.set_buckets(synth.ddp_offsets(lay) if ddp else None)
        print("[bench] inputs resident", file=sys.stderr, flush=True)

    def set_buckets(self, off=None):
        """Equal buckets of the layout's bucket_n (off None), or the buckets
        [off[b], off[b+1]) through a device bucket table."""
        nf, torch, np = self.nf, self.torch, self.np
        W, n, lay = self.W, self.n, self.lay
        self.table = self.stats = self.dec = self.ws = None
        if off is None:
            self.bn = lay.bucket_n
            self.off = np.array(list(range(0, n, self.bn)) + [n], np.int64)
            ws = nf.nf_workspace_bytes_buckets(W, n, self.bn)
        else:
            self.bn = None
            self.off = np.asarray(off, np.int64)
            self.table = torch.empty(nf.nf_bucket_table_bytes(W, self.off), dtype=torch.uint8, device=self.dev)
            nf.nf_bucket_table_init(W, self.off, self.table)
            ws = nf.nf_workspace_bytes_table(W, self.off)
        self.nb = nb = len(self.off) - 1
        self.stats = torch.empty(nb * W * nf.STATS_BYTES, dtype=torch.uint8, device=self.dev)
        self.dec = torch.empty(nb * nf.DECISION_BYTES, dtype=torch.uint8, device=self.dev)
        self.ws = nf.empty_workspace(ws, self.dev)
        torch.cuda.synchronize()
        sizes = np.diff(self.off)
        print(f"[bench] {lay.name}: W={W} n={n:,} buckets={nb} "
              + (f"bucket_n={self.bn:,}" if self.bn else f"DDP cut, {sizes.min():,} to {sizes.max():,} elements")
              + f" input={lay.input_bytes() / 1e9:.2f} GB", file=sys.stderr, flush=True)

    def buckets_desc(self):
        """The config's bucket fields: equal buckets or the DDP cut."""
        if self.bn:
            return {"buckets": self.nb, "bucket_n": self.bn}
        sizes = self.np.diff(self.off)
        return {"buckets": self.nb, "bucket_n": None,
                "bucket_cut": f"DDP: 25 MiB capacity (first bucket 1 MiB), closed at tensor boundaries; "
                              f"{int(sizes.min()):,} to {int(sizes.max()):,} elements"}

    def release(self):
        del self.grads, self.mask, self.bits, self.counts, self.out, self.stats, self.dec, self.ws, self.table
        self.torch.cuda.synchronize()
        self.torch.cuda.empty_cache()

    def step(self, pol, counts=True):
        ternary = pol.format == self.nf.NF_FORMAT_TERNARY
        cnt = self.counts[: (2 if ternary else 1) * self.n] if counts else None
        if self.table is not None:
            self.nf.nf_route_bucket_table(self.grads, self.off, self.table, self.mask, pol, self.bits, cnt,
                                          self.out, self.stats, self.dec, self.ws)
        else:
            self.nf.nf_route_buckets(self.grads, self.n, self.bn, self.mask, pol, self.bits, cnt, self.out,
                                     self.stats, self.dec, self.ws)

    def measure(self, pol, steps, warmup, cold=False, counts=True):
        """Wall and device time of `steps` steps; algorithmic bytes and rates per phase."""
        nf, torch, np = self.nf, self.torch, self.np
        W, n, nb = self.W, self.n, self.nb
        ternary = pol.format == nf.NF_FORMAT_TERNARY
        for _ in range(warmup):
            self.step(pol, counts)
        torch.cuda.synchronize()
        hip = HipEvents()
        evs = [[hip.create() for _ in range(4)] for _ in range(steps)]
        scrub = torch.zeros(1 << 28, dtype=torch.float32, device=self.dev) if cold else None
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        for k in range(steps):
            if scrub is not None:
                scrub.add_(1.0)
            nf.nf_set_phase_events(*evs[k])
            self.step(pol, counts)
        torch.cuda.synchronize()
        t1 = time.perf_counter()
        nf.nf_set_phase_events()
        del scrub
        ms_per_step = (t1 - t0) * 1e3 / steps
        # The same steps again without the four phase events per step: each
        # event record costs a few microseconds on the stream, which shows on
        # the small workloads (about 13 us of the 1M-element bucket's step).
        plain_ms = None
        if not cold:
            torch.cuda.synchronize()
            p0 = time.perf_counter()
            for k in range(steps):
                self.step(pol, counts)
            torch.cuda.synchronize()
            plain_ms = (time.perf_counter() - p0) * 1e3 / steps
        ph = np.array([[hip.elapsed_ms(e[0], e[1]), hip.elapsed_ms(e[1], e[2]), hip.elapsed_ms(e[2], e[3]),
                        hip.elapsed_ms(e[0], e[3])] for e in evs])
        for e in evs:
            for x in e:
                hip.destroy(x)
        pass1_ms, decide_ms, pass2_ms, device_ms = (float(v) for v in ph.mean(axis=0))
        dev_med, dev_min = float(np.median(ph[:, 3])), float(ph[:, 3].min())
        d = nf.decisions_host(self.dec, nb)
        routes = {"L": int((d["route"] == 0).sum()), "F": int((d["route"] == 1).sum()),
                  "P": int((d["route"] == 2).sum())}
        nbs = np.diff(self.off)
        ne = d["n_eligible"].astype(np.int64)
        nwb = (nbs + 63) // 64
        # pass 1: gradients once, mask once, sign words out (G-Binary only), FP32 sums at routed positions out
        pass1_bytes = float((4 * W * nbs + 8 * nwb + (0 if ternary else 8 * W * nwb) + 4 * (nbs - ne)).sum())
        is_l, is_f = d["route"] == 0, d["route"] == 1
        cbytes = (2 if ternary else 1) * nbs if counts else 0
        if ternary:
            # second read of the eligible elements, two planes out and back in, mask, counts, decode
            l_bytes = 4 * W * ne + 8 * nwb + 16 * W * nwb + 16 * W * nwb + 8 * nwb + cbytes + 4 * ne
        else:
            l_bytes = 8 * W * nwb + 8 * nwb + cbytes + 4 * ne
        pass2_bytes = float((l_bytes * is_l).sum() + ((4 * W * ne + 8 * nwb + 4 * ne) * is_f).sum())
        launches = (nf.nf_pass1_launches(W, n, self.bn, sign_words=not ternary) if self.bn else
                    nf.nf_pass1_launches_table(W, self.off, sign_words=not ternary))
        # a cold run's wall clock includes the overwrites: its value comes from the device events
        value = self.lay.input_bytes() / ((device_ms if cold else ms_per_step) * 1e-3) / 1e9
        plain_value = None if plain_ms is None else self.lay.input_bytes() / (plain_ms * 1e-3) / 1e9
        achieved = pass1_bytes / (pass1_ms * 1e-3) / 1e9
        print(f"[bench] {self.lay.name} {'ternary' if ternary else 'binary'}"
              f"{' forced' if pol.force_lowbit else ''}{' cold' if cold else ''}"
              f"{'' if self.bn else ' DDP buckets'}: {steps} steps, "
              f"{ms_per_step:.4f} ms/step wall, device {device_ms:.4f} (pass1 {pass1_ms:.4f}, decide "
              f"{decide_ms:.4f}, pass2 {pass2_ms:.4f}), {value:.1f} GB/s"
              + ("" if plain_ms is None else f"; without phase events {plain_ms:.4f} ms/step, {plain_value:.1f} GB/s"),
              file=sys.stderr, flush=True)
        return {
            "steps": steps, "warmup": warmup, "ms_per_step": round(ms_per_step, 4),
            "value": round(value, 2), "pct_hbm_peak": round(100 * value / HBM_PEAK_GBS, 2),
            "without_phase_events": None if plain_ms is None else {
                "ms_per_step": round(plain_ms, 4), "value": round(plain_value, 2),
                "pct_hbm_peak": round(100 * plain_value / HBM_PEAK_GBS, 2)},
            "device_ms": {"mean": round(device_ms, 4), "median": round(dev_med, 4), "min": round(dev_min, 4)},
            "phases_ms": {"pass1": round(pass1_ms, 4), "decide": round(decide_ms, 4),
                          "pass2": round(pass2_ms, 4), "device_total": round(device_ms, 4),
                          "pass2_algorithmic_gbs": round(pass2_bytes / max(pass2_ms, 1e-9) / 1e6, 1)},
            "pass1": {"kernel": "k_pass1", "bound": "hbm", "achieved": round(achieved, 1), "peak": HBM_PEAK_GBS,
                      "unit": "GB/s", "frac": round(achieved / HBM_PEAK_GBS, 4), "launches_per_step": launches,
                      "algorithmic_bytes_per_launch": round(pass1_bytes / launches),
                      "avg_launch_ms": round(pass1_ms / launches, 5)},
            "routes": routes,
            "mgtr": round(float(d["bytes_route"].sum() / d["bytes_fp32"].sum()), 4),
            "eligible_frac": round(float(ne.sum()) / n, 4),
        }

    def cpu_baseline(self, pol, seconds):
        """The oracle, single-threaded and pinned to one host core, on the first
        buckets (or, for a one-bucket workload, a leading range) of the data the
        GPU just reduced, with the oracle's own mask; its results are checked
        against the GPU's on the sample."""
        import oracle as nfo
        nf, np = self.nf, self.np
        W, n, nb, off = self.W, self.n, self.nb, self.off
        ternary = pol.format == nf.NF_FORMAT_TERNARY
        opol = nfo.policy(admitted=pol.admitted, veto=pol.veto, guard_ok=pol.guard_ok,
                          force_lowbit=pol.force_lowbit, decode_mode=pol.decode_mode, fp32_op=pol.fp32_op,
                          kappa=pol.kappa, format=pol.format, tau=pol.tau)
        mask_o = nfo.mask_from_segments(*self.segs, n)
        rate_guess = 0.55e9  # bytes per second of the single-threaded oracle
        one_bucket = nb == 1 and n * 4 * W > rate_guess * seconds
        if one_bucket:
            # a leading 64-aligned range of the one bucket, reduced by the oracle as a bucket of its own:
            # its decision is not the GPU's, so only the element-wise results are compared
            span = max(64, int(rate_guess * seconds / (4 * W)) // 64 * 64)
            ranges = [(0, min(span, n))]
        else:
            # leading buckets while they fit the budget (at least one)
            k = 1
            while k < nb and 4 * W * (off[k + 1] - off[0]) <= rate_guess * seconds:
                k += 1
            ranges = [(int(off[b]), int(off[b + 1])) for b in range(k)]
        model, ncpu = host_cpu()
        old_aff = os.sched_getaffinity(0)
        core = min(old_aff)
        dh = nf.decisions_host(self.dec, nb)
        sh = nf.stats_host(self.stats, W, nb)
        # a sample far below a second of oracle work (the tiny bucket) is reduced several times over
        reps = max(1, int(1.0 / (4 * W * sum(e - a for a, e in ranges) / rate_guess)))
        t_cpu, nbytes, bad = 0.0, 0, []
        try:
            os.sched_setaffinity(0, {core})
            for b, (a, e) in enumerate(ranges):
                gh = self.grads[:, a:e].cpu().numpy()
                mh = np.ascontiguousarray(mask_o[a // 64:(e + 63) // 64])
                c0 = time.perf_counter()
                for _ in range(reps):
                    ref = (nfo.reduce_bucket_ternary if ternary else nfo.reduce_bucket)(gh, mh, opol)
                t_cpu += time.perf_counter() - c0
                nbytes += reps * 4 * W * (e - a)
                bad += sample_mismatches(nf, np, self, ref, b, a, e, mh, ternary, whole_bucket=not one_bucket)
        finally:
            os.sched_setaffinity(0, old_aff)
        what = (f"elements 0..{ranges[0][1] - 1} of the one bucket, reduced as a bucket of their own"
                if one_bucket else f"buckets 0..{len(ranges) - 1} ({off[len(ranges)] - off[0]:,} elements)")
        if reps > 1:
            what += f", reduced {reps} times"
        rec = {"value": round(nbytes / t_cpu / 1e9, 4), "unit": "GB/s", "cores": 1, "kind": "oracle",
               "sample": f"{self.lay.name} {what} x {W} workers, single-threaded C++ oracle pinned to core "
                         f"{core} of {ncpu} ({model}), {t_cpu:.1f} s",
               "sample_parity": "ok" if not bad else "MISMATCH: " + "; ".join(bad[:4]),
               "sample_parity_checks": (("FP32 values (the planes' thresholds need the whole bucket)" if ternary
                                         else "bits, counts, FP32 values") if one_bucket else
                                        ("planes" if ternary else "bits") +
                                        ", counts, outputs, statistics, route, reasons, n_E, modeled bytes")}
        print(f"[bench] oracle on {self.lay.name}: {rec['value']} GB/s ({t_cpu:.1f} s), sample parity "
              f"{rec['sample_parity']}", file=sys.stderr, flush=True)
        return rec


def sample_mismatches(nf, np, wl, ref, b, a, e, mh, ternary, whole_bucket):
    """What differs between the GPU's results and the oracle's on elements
    [a, e) (bucket b when whole_bucket).  Bars as in the parity tests: bit-exact
    integers, FP32 sums and modeled bytes; statistics, scale and decoded values
    within 1e-6 relative."""
    W, n = wl.W, wl.n
    bad = []
    m = np.unpackbits(mh.view(np.uint8), bitorder="little")[: e - a].astype(bool)
    got_bits = wl.bits[: (2 if ternary else 1) * W, a // 64:(e + 63) // 64].cpu().numpy().view(np.uint64)
    out = wl.out[a:e].cpu().numpy()

    def close(x, y, tol=1e-6):
        x, y = np.asarray(x, np.float64), np.asarray(y, np.float64)
        same = (x == y) | (np.isnan(x) & np.isnan(y))
        with np.errstate(invalid="ignore"):
            return bool(np.all(same | (np.abs(x - y) <= tol * np.abs(y))))

    def same32(x, y):
        x, y = np.asarray(x, np.float32), np.asarray(y, np.float32)
        nx, ny = np.isnan(x), np.isnan(y)
        return bool(np.array_equal(nx, ny) and np.array_equal(x[~nx].view(np.uint32), y[~ny].view(np.uint32)))

    if whole_bucket:
        d, rd, st = wl.nf.decisions_host(wl.dec, wl.nb)[b], ref["decision"], nf.stats_host(wl.stats, W, wl.nb)[b]
        if (int(d["route"]), int(d["reasons"]), int(d["n_eligible"])) != (rd.route, rd.reasons, rd.n_eligible):
            bad.append(f"bucket {b} decision")
        if float(d["bytes_route"]) != rd.bytes_route or float(d["bytes_fp32"]) != rd.bytes_fp32:
            bad.append(f"bucket {b} modeled bytes")
        if not close(d["scale"], rd.scale):
            bad.append(f"bucket {b} scale")
        if not (np.array_equal(st["nonfinite"], ref["stats"]["nonfinite"]) and
                close(st["sum_abs_elig"], ref["stats"]["sum_abs_elig"]) and close(st["sum_sq"], ref["stats"]["sum_sq"])):
            bad.append(f"bucket {b} statistics")
        route, scale = int(d["route"]), np.float32(d["scale"])
    else:
        route, scale = int(wl.nf.decisions_host(wl.dec, 1)[0]["route"]), None
    if ternary:
        # the planes' thresholds come from the whole bucket's statistics: a leading range reduced as a
        # bucket of its own has other thresholds, so there only its FP32 values are compared
        if whole_bucket and route == 0 and not (np.array_equal(got_bits[:W], ref["pos"]) and
                                                np.array_equal(got_bits[W:], ref["neg"])):
            bad.append(f"bucket {b} planes")
    elif not np.array_equal(got_bits, ref["bits"]):
        bad.append(f"range {b} bits")
    if route == 0 and (whole_bucket or not ternary):
        cnt = wl.counts[a:e].cpu().numpy()
        want_c = ref["cpos"] if ternary else ref["counts"]
        if not np.array_equal(cnt, want_c):
            bad.append(f"range {b} counts")
    if route != 0 or not whole_bucket:
        # the FP32 path: every position off route L, the routed positions on it
        sel = np.ones(e - a, bool) if route != 0 else ~m
        if whole_bucket and not same32(out[sel], ref["out"][sel]):
            bad.append(f"range {b} FP32 values")
        if not whole_bucket:
            import oracle as nfo
            y = nfo.fp32_path(wl.grads[:, a:e].cpu().numpy(), 0)
            if not same32(out[sel], y[sel]):
                bad.append(f"range {b} FP32 values")
    if ternary and not whole_bucket and route == 0:
        return bad  # routed positions were compared above
    if whole_bucket and route == 0:
        if not same32(out[~m], ref["out"][~m]):
            bad.append(f"bucket {b} routed values")
        if not close(out[m], ref["out"][m]):
            bad.append(f"bucket {b} decoded values")
    return bad


def main():
    args = parse()
    if args.gpus != 1:
        print(f"bench.py measures one GPU: the reducer simulates the W workers as stacked buffers on "
              f"one device and this build has no multi-GPU path (asked for --gpus {args.gpus}).",
              file=sys.stderr)
        return 2

    import numpy as np
    import torch

    assert torch.cuda.is_available(), "bench.py needs a GPU"
    torch.cuda.init()
    if args.calibrate_copy:
        return calibrate_copy()
    if args.contrast:
        return contrast()
    if args.controller or args.sliced:
        args.workload = args.workload or "gpt1p3b"
    if args.controller:
        return controller_run(args)
    if args.sliced:
        return sliced_run(args)

    import paper_2606_25759_amd as nf
    import synth

    sweep = args.workload is None
    name = args.workload or "gpt1p3b"
    ternary = args.format == "ternary"
    pol = nf.policy(force_lowbit=int(args.force_lowbit), format=int(ternary), tau=args.tau)
    # the headline workload, with room for the G-Ternary planes when the sweep measures them too
    wl = Workload(nf, torch, name, planes=2 if (ternary or sweep) else 1, ddp=args.ddp_buckets)
    m = wl.measure(pol, args.steps, args.warmup, cold=args.cold, counts=not args.no_counts)

    split = None
    if not ternary and not args.no_split:
        split = split_one_bucket(nf, torch, wl.grads, wl.mask, wl.W, int(wl.off[1]),
                                 int(nf.decisions_host(wl.dec, wl.nb)["n_eligible"][0]))
        print(f"[bench] standalone, first bucket: " + ", ".join(f"{k} {v['ms']:.3f} ms" for k, v in split.items()
                                                            if isinstance(v, dict)), file=sys.stderr, flush=True)
    achievable = pattern = None
    if not args.no_probe:
        sink = torch.zeros(1024, dtype=torch.float32, device=wl.dev)
        synth.read_probe(wl.grads, sink)
        torch.cuda.synchronize()
        a0 = time.perf_counter()
        for _ in range(3):
            synth.read_probe(wl.grads, sink)
        torch.cuda.synchronize()
        probe_ms = (time.perf_counter() - a0) * 1e3 / 3
        achievable = round(4 * wl.grads.numel() / (probe_ms * 1e-3) / 1e9, 1)
        print(f"[bench] streaming read of the input: {achievable} GB/s", file=sys.stderr, flush=True)
        if wl.W == 16:
            pattern = pattern_probe(synth, torch, wl)
    cpu = None if args.no_cpu_baseline else wl.cpu_baseline(pol, 10.0)

    # HBM bytes per pass-1 launch from the committed counters (null unless taken on this kernel source)
    if args.ddp_buckets:
        traffic = None if ternary else pass1_traffic(committed_counters(name, "ddp"))
    else:
        traffic = counter_traffic(name) if not ternary else None
    roofline = dict(m["pass1"])
    roofline["traffic"] = traffic
    roofline["traffic_gbs"] = (None if traffic is None else
                               round(traffic / (m["phases_ms"]["pass1"] / roofline["launches_per_step"]) / 1e6, 1))
    rec = {
        "metric": "reducer FP32-equiv input GB/s (pack+signcount+fp32) and % of HBM peak",
        "value": m["value"],
        "unit": "GB/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": m["ms_per_step"],
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "f32",
        "data": "synthetic",
        "pct_hbm_peak": m["pct_hbm_peak"],
        "without_phase_events": m["without_phase_events"],
        "config": {"workload": wl.lay.name, "W": wl.W, "n_total": wl.n, **wl.buckets_desc(),
                   "eligible_frac": m["eligible_frac"],
                   "policy": "forced low-bit" if args.force_lowbit else "admitted, guard ok",
                   "format": args.format, "counts_written": not args.no_counts,
                   "caches": "cold (1 GiB overwritten before each step)" if args.cold else "warm"},
        "device_ms": m["device_ms"],
        "roofline": roofline,
        "phases_ms": m["phases_ms"],
        "achievable_read_gbs": achievable,
        "pass1_pattern_probe": pattern,
        "split_one_bucket": split,
        "routes": m["routes"],
        "mgtr": m["mgtr"],
        "cpu_baseline": cpu,
    }
    if sweep:
        rec["configs"] = sweep_configs(nf, torch, wl, args)
    else:
        wl.release()
    print(json.dumps(rec), flush=True)
    return 0


def config_record(wl, m, pol, cold, cpu, counters):
    """One row of the per-workload list: rate, share of peak, the pass-1
    roofline, the oracle's sample and the committed counter bytes."""
    ternary = pol.format == 1
    row = {"workload": wl.lay.name, "W": wl.W, "n_total": wl.n, **wl.buckets_desc(),
           "format": "ternary" if ternary else "binary",
           "policy": "forced low-bit" if pol.force_lowbit else "admitted, guard ok",
           "caches": "cold (1 GiB overwritten before each step)" if cold else "warm",
           "input_gb": round(wl.lay.input_bytes() / 1e9, 4)}
    row.update({k: m[k] for k in ("value", "pct_hbm_peak", "ms_per_step", "without_phase_events", "steps",
                                  "device_ms", "phases_ms", "routes", "mgtr")})
    row["unit"] = "GB/s"
    roof = dict(m["pass1"])
    roof["traffic"] = pass1_traffic(counters)
    roof["traffic_gbs"] = (None if roof["traffic"] is None else
                           round(roof["traffic"] / (roof["avg_launch_ms"] * 1e-3) / 1e9, 1))
    row["roofline_pass1"] = roof
    row["cpu_baseline"] = cpu
    row["counter_bytes"] = counters
    return row


def committed_counters(workload, fmt):
    """Counter-measured HBM bytes per dispatch of the step's kernels from the
    committed rocprofv3 summaries of this workload, where the kernel source is
    the one they were taken on; else None."""
    path = os.path.join(ROOT, "profiles", f"counters_{workload}_{fmt}.json")
    if not os.path.exists(path):
        return None
    rec = json.load(open(path))
    if rec.get("kernel_sha") != all_kernels_sha():
        return None
    return rec.get("kernels")


def pass1_traffic(counters):
    """HBM bytes per pass-1 launch in a workload's committed counters (the
    pass-1 instantiation the step ran), or None."""
    if not counters:
        return None
    names = [k for k in counters if k.startswith("k_pass1<")]
    if not names:
        return None
    return counters[max(names, key=lambda k: counters[k]["dispatches"])]["hbm_bytes_per_dispatch"]


def sweep_configs(nf, torch, gpt, args):
    """Every workload of the sweep after the headline: G-Ternary on the same
    GPT-scale buffer, the same buffer cut into DDP's buckets (bucket table),
    then ViT-B/16 scale, ResNet-50 scale, the tiny bucket
    (warm and cold caches), the stress bucket (route F, forced low-bit,
    forced low-bit G-Ternary) and the W = 255 fan-in bucket pair (G-Binary
    and G-Ternary).  Each row is a few timed steps and a bounded oracle
    sample."""
    rows = []
    tern = nf.policy(format=nf.NF_FORMAT_TERNARY, tau=args.tau)
    m = gpt.measure(tern, 10, 2)
    rows.append(config_record(gpt, m, tern, False, None if args.no_cpu_baseline else gpt.cpu_baseline(tern, 3.0),
                              committed_counters(gpt.lay.name, "ternary")))
    # the same buffer cut as DDP cuts the model, through the bucket-table driver
    import synth
    gpt.set_buckets(synth.ddp_offsets(gpt.lay))
    m = gpt.measure(nf.policy(), 10, 2)
    rows.append(config_record(gpt, m, nf.policy(), False,
                              None if args.no_cpu_baseline else gpt.cpu_baseline(nf.policy(), 3.0),
                              committed_counters(gpt.lay.name, "ddp")))
    gpt.release()
    plan = [("vitb16", [(nf.policy(), False, 20)]),
            ("resnet50", [(nf.policy(), False, 50)]),
            ("tiny", [(nf.policy(), False, 200), (nf.policy(), True, 50)]),
            ("stress", [(nf.policy(), False, 10), (nf.policy(force_lowbit=1), False, 10),
                        (nf.policy(force_lowbit=1, format=nf.NF_FORMAT_TERNARY, tau=args.tau), False, 10)]),
            ("fanin255", [(nf.policy(), False, 10),
                          (nf.policy(format=nf.NF_FORMAT_TERNARY, tau=args.tau), False, 10)])]
    for name, runs in plan:
        wl = Workload(nf, torch, name, planes=2 if any(p.format for p, _, _ in runs) else 1)
        for pol, cold, steps in runs:
            m = wl.measure(pol, steps, 3, cold=cold)
            cpu = None if (args.no_cpu_baseline or cold) else wl.cpu_baseline(pol, 3.0)
            fmt = "ternary" if pol.format else ("forced" if pol.force_lowbit else "binary")
            rows.append(config_record(wl, m, pol, cold, cpu, committed_counters(name, fmt)))
        wl.release()
    return rows


if __name__ == "__main__":
    sys.exit(main())
