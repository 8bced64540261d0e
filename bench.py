#!/usr/bin/env python3
"""Benchmark of the H-Scale hot path on one MI355X.

One step = one pass of the whole path over one workload:
  hdiag  (h = diag(X^T X)) over each calibration activation tensor, then
  search (the E4M3 scale search of every 16-weight group of each weight
          matrix, scored with its input's h, writing scale codes and packed
          E2M1 codes).
Inputs are resident in HBM before the timed region starts.  The default
workload is the Llama-3-8B-shaped MLP down_proj: W 4096 x 14336 bf16 and
X 262144 x 14336 bf16 (128 sequences x 2048 tokens), window +-4.  Other
workloads: attn_proj (4096 x 4096), down_proj_70b (8192 x 28672, +-8) and
block (an 8B-class decoder block: q/k/v/o and gate/up/down with three shared
activation tensors of 262144 tokens).

Timing: W untimed warm-up steps, then K timed steps bracketed by device
synchronisation; each kernel call is bracketed by HIP events recorded on the
stream the library launches on (torch's current stream, passed through the C
ABI).  The multi-GB reads of X in each step evict W from the 256 MB Infinity
Cache, so the search reads W from HBM.

Prints one JSON line.  `value` is the search throughput in Gweights/s (the
metric's first figure); `hdiag` carries the second figure (HBM GB/s and its
fraction of the 8 TB/s peak).  `ceilings` holds what the chip sustains in the
same run for the same kinds of work (a streaming read, VALU issue of the
search's instruction stream), measured by the probes of libhscale_probes.so
after the timed steps; the rooflines carry each kernel's fraction of them.  `cpu_baseline` is the CPU oracle timed on this
host's cores over the same workload's last layer (its whole W and X by
default); the same rows and tokens are checked for parity against the
benchmarked outputs.
"""
from __future__ import annotations

import argparse
import hashlib
from concurrent.futures import ThreadPoolExecutor
import json
import os
import sys
import time

import numpy as np

METRIC = "H-Scale search Gweights/s + hdiag HBM GB/s (fraction of peak), 1 MI355X"
HBM_PEAK_GBS = 8000.0
BF16_MFMA_PEAK_TFLOPS = 2500.0  # dense bf16 matrix-core peak
# fp32 VALU issue ceiling: 256 CU x 4 SIMD x 32 lanes/clk (one wave64 fp32
# op per 2 clocks) x 2.4 GHz = 78.64 T lane-ops/s = 157.3 TFLOP/s of FMA.
VALU_PEAK_TOPS = 256 * 4 * 32 * 2.4e9 / 1e12
SEARCH_BYTES_PER_WEIGHT = 2 + 0.5 + 1.0 / 16  # read W, write codes and scales
HERE = os.path.dirname(os.path.abspath(__file__))
PROBE_LIB = os.path.join(HERE, "paper_2608_28113_amd", "libhscale_probes.so")
# Sources of the hot-path kernels (hdiag, search): the committed HBM-traffic
# figures are valid only for the source they were measured on.
HOT_SOURCES = ("common.h", "hdiag.hip", "search.hip")
DIAG_SOURCES = ("common.h", "diag.hip")


def source_hash(names=HOT_SOURCES) -> str:
    h = hashlib.sha256()
    for name in names:
        with open(os.path.join(HERE, "paper_2608_28113_amd", "csrc", name), "rb") as f:
            h.update(f.read())
    return h.hexdigest()[:16]


def diag_traffic(workload: str):
    """HBM bytes of one output-error call (dW split + tile kernel) from the
    committed rocprofv3 summary, or None when absent or stale."""
    path = os.path.join(HERE, "profiles", f"output_error_{workload}.json")
    if not os.path.exists(path):
        return None
    with open(path) as f:
        prof = json.load(f)
    if prof.get("kernel_source_sha256_16") != source_hash(DIAG_SOURCES):
        return None
    t = prof.get("traffic", {})
    names = ("delta_split_kernel", "lfull_tile_kernel")
    if not all(n in t for n in names):
        return None
    return sum(t[n]["read_bytes"] + t[n]["write_bytes"] for n in names), os.path.relpath(path, HERE)


def search_ops_per_weight(K: int, init: str) -> int:
    # 5 per weight-candidate (scale product, grid rounding, residual,
    # square, weighted accumulate) + 3 per weight (max, encode, pack); the
    # 4over6 initial code adds two anchor evaluations of 4 ops per weight
    # (scale product, rounding, residual, square-accumulate).
    return 5 * K + 3 + (8 if init == "4over6" else 0)


def profile_json(workload: str) -> str:
    return os.path.join(HERE, "profiles", f"{workload}.json")


def measured_traffic(workload: str):
    """HBM bytes per step from the committed rocprofv3 FETCH_SIZE/WRITE_SIZE
    summary of this workload (copy-calibrated), or None when there is none or
    it was taken before the kernels last changed."""
    path = profile_json(workload)
    if not os.path.exists(path):
        return None
    with open(path) as f:
        prof = json.load(f)
    if prof.get("kernel_source_sha256_16") != source_hash(HOT_SOURCES):
        return None
    t = prof.get("traffic", {})
    steps = prof.get("steps_profiled")

    def per_step(name):
        # mean bytes per dispatch x dispatches per step (several hdiag
        # calls in a multi-layer step)
        k = t[name]
        n = k["dispatches"] / steps if steps and "dispatches" in k else 1.0
        return (k["read_bytes"] + k["write_bytes"]) * n

    def tot(*names):
        if not all(n in t for n in names):
            return None
        return sum(per_step(n) for n in names)
    search = "search_layers_kernel" if "search_layers_kernel" in t else "search_kernel"
    return {"hdiag": tot("hdiag_partial", "hdiag_tree"), "search": tot(search),
            "valu": prof.get("valu", {}).get(search), "source": os.path.relpath(path, HERE)}


def parse():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--workload", default="down_proj",
                    choices=["tiny", "attn_proj", "down_proj", "down_proj_70b", "block"])
    ap.add_argument("--window", type=int, default=None, help="symmetric shift set -w..+w")
    ap.add_argument("--down", type=int, default=None, help="asymmetric shift set -down..+up")
    ap.add_argument("--up", type=int, default=None)
    ap.add_argument("--init", default="maxabs", choices=["maxabs", "4over6"])
    ap.add_argument("--cpu-rows", type=int, default=None,
                    help="rows of W in the CPU oracle leg (default: all; also checked for parity)")
    ap.add_argument("--cpu-tokens", type=int, default=None,
                    help="tokens of X in the CPU oracle hdiag leg (default: all)")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-ceilings", action="store_true",
                    help="skip the measured read and VALU ceilings (probe kernels run after the timed steps)")
    ap.add_argument("--no-diagnostics", action="store_true",
                    help="skip the quality-diagnostics leg (shift statistics, Eq. 3 output error)")
    ap.add_argument("--diag-profile", action="store_true",
                    help="run only the diagnostics kernels on the workload's last layer (for rocprofv3)")
    ap.add_argument("--profile-mode", action="store_true",
                    help="only warm-up and timed steps (for rocprofv3 runs)")
    ap.add_argument("--copy-calibration", action="store_true",
                    help="also run one plain 1 GiB device copy, a kernel of known traffic "
                         "for scaling the HBM byte counters")
    return ap.parse_args()


def build_workload(name, dev, window_override):
    """Returns (activations {key: X}, layers [(label, W, x_key, s_g, window)], description)."""
    from synth.workloads import CONFIGS, block_workloads, harness_global_scale, make_activations, make_weight
    if name != "block":
        wl = CONFIGS[name]
        w = wl.window if window_override is None else window_override
        X = make_activations(wl, dev)
        W = make_weight(wl, dev)
        desc = f"{wl.name}: W {wl.out}x{wl.inp} bf16 ({wl.w_dist}), X {wl.tokens}x{wl.inp} bf16"
        return {"x": X}, [(wl.name, W, "x", harness_global_scale(W), w)], desc
    wls = block_workloads(window=4 if window_override is None else window_override)
    xkey = {"q_proj": "attn", "k_proj": "attn", "v_proj": "attn", "o_proj": "attn",
            "gate_proj": "mlp", "up_proj": "mlp", "down_proj": "down"}
    acts = {"attn": make_activations(wls["q_proj"], dev), "mlp": make_activations(wls["gate_proj"], dev),
            "down": make_activations(wls["down_proj"], dev)}
    layers = []
    for lname, wl in wls.items():
        W = make_weight(wl, dev)
        layers.append((lname, W, xkey[lname], harness_global_scale(W), wl.window))
    desc = ("8B-class decoder block: q/o 4096x4096, k/v 1024x4096, gate/up 14336x4096, down 4096x14336 bf16; "
            "X_attn and X_mlp 262144x4096, X_down 262144x14336 bf16")
    return acts, layers, desc


def progress(msg: str) -> None:
    """A progress line on stderr (stdout carries only the JSON line)."""
    print(f"[bench] {msg}", file=sys.stderr, flush=True)


def main():
    args = parse()
    world = int(os.environ.get("WORLD_SIZE", "1"))
    if args.gpus != 1 or world != 1:
        print("bench.py runs on one GPU only: the H-Scale hot path has no cross-GPU "
              "communication (rows shard with no exchange; see the sharding notes). "
              "Run with --gpus 1.", file=sys.stderr)
        sys.exit(2)
    if (args.down is None) != (args.up is None) or (args.window is not None and args.down is not None):
        print("give --window, or both --down and --up", file=sys.stderr)
        sys.exit(2)

    import torch
    import paper_2608_28113_amd as hs
    from paper_2608_28113_amd import _lib

    _lib.load()
    if not torch.cuda.is_available():
        print("no GPU visible", file=sys.stderr)
        sys.exit(1)
    dev = "cuda"
    torch.cuda.set_device(0)

    progress(f"generating the {args.workload} workload")
    acts, layers, desc = build_workload(args.workload, dev, args.window)
    if args.down is not None:
        layers = [(l, W, xk, s, None) for (l, W, xk, s, _) in layers]
    if args.diag_profile:
        diag = diag_leg(args, acts, layers, repeats=2)
        if args.copy_calibration:
            copy_calibration(dev)
        print(json.dumps({"diag_profile": True, "diagnostics": diag}), flush=True)
        return
    hbuf = {k: torch.empty(X.shape[1], dtype=torch.float32, device=dev) for k, X in acts.items()}
    ws = torch.empty(max(max(hs.hdiag_workspace_bytes(*X.shape) for X in acts.values()), 16),
                     dtype=torch.uint8, device=dev)
    outs = [(torch.empty((W.shape[0], W.shape[1] // 16), dtype=torch.uint8, device=dev),
             torch.empty((W.shape[0], W.shape[1] // 2), dtype=torch.uint8, device=dev)) for (_, W, _, _, _) in layers]
    torch.cuda.synchronize()
    stream = torch.cuda.current_stream()

    def window_args(w):
        return dict(window=w) if w is not None else dict(down=args.down, up=args.up)

    def run_search():
        # Several layers (the decoder block) are searched by one batched
        # launch; a single layer by the plain search.
        if len(layers) > 1:
            hs.search_layers([(W, hbuf[xk], s_g) for (_, W, xk, s_g, _) in layers], init=args.init,
                             outputs=outs, stream=stream, **window_args(layers[0][4]))
        else:
            (lname, W, xk, s_g, w), (codes, packed) = layers[0], outs[0]
            hs.search(W, hbuf[xk], s_g, init=args.init, scale_codes=codes, packed_e2m1=packed, stream=stream,
                      **window_args(w))

    def step(evs=None):
        k = 0
        for key, X in acts.items():
            if evs is not None:
                evs[k].record(stream)
            hs.hdiag(X, h=hbuf[key], workspace=ws, stream=stream)
            k += 1
        if evs is not None:
            evs[k].record(stream)
        run_search()
        if evs is not None:
            evs[k + 1].record(stream)

    n_ev = len(acts) + 2
    progress(f"{args.warmup} warm-up and {args.steps} timed steps")
    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()
    events = [[torch.cuda.Event(enable_timing=True) for _ in range(n_ev)] for _ in range(args.steps)]
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for k in range(args.steps):
        step(events[k])
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0

    nh = len(acts)
    t_h = np.array([e[0].elapsed_time(e[nh]) for e in events]) * 1e-3  # all hdiag calls of a step
    t_s = np.array([e[nh].elapsed_time(e[-1]) for e in events]) * 1e-3  # all search calls of a step
    t_step = np.array([e[0].elapsed_time(e[-1]) for e in events]) * 1e-3
    iso = None if args.profile_mode else isolated_search(run_search, stream)
    if args.copy_calibration:
        copy_calibration(dev)
    if args.profile_mode:
        print(json.dumps({"profile_mode": True, "hdiag_ms": float(t_h.mean() * 1e3),
                          "search_ms": float(t_s.mean() * 1e3)}), flush=True)
        return

    weights = sum(W.numel() for (_, W, _, _, _) in layers)
    hd_bytes = float(sum(2.0 * X.numel() + 4.0 * X.shape[1] for X in acts.values()))
    hd_gbs = hd_bytes / t_h.mean() / 1e9
    search_gws = weights / t_s.mean() / 1e9
    ops = 0
    windows = []
    for (_, W, _, _, w) in layers:
        K = 2 * w + 1 if w is not None else args.down + args.up + 1
        windows.append(w if w is not None else [args.down, args.up])
        ops += search_ops_per_weight(K, args.init) * W.numel()
    search_tops = ops / t_s.mean() / 1e12
    search_gbs = SEARCH_BYTES_PER_WEIGHT * weights / t_s.mean() / 1e9

    rl_hdiag = {"bound": "hbm", "achieved": round(hd_gbs, 1), "peak": HBM_PEAK_GBS, "unit": "GB/s",
                "frac": round(hd_gbs / HBM_PEAK_GBS, 4), "traffic": None,
                "kernel": "hscale_hdiag (hdiag_partial + hdiag_tree)",
                "algorithmic_bytes_per_step": hd_bytes, "avg_ms_per_step": round(t_h.mean() * 1e3, 4),
                "launches_per_step": nh}
    # The model's bound: VALU for windows of a few candidates and up, HBM for
    # the smallest (window 0, the RTN baseline, moves 2.56 bytes but issues
    # only 8 ops per weight).
    valu_bound = ops / (VALU_PEAK_TOPS * 1e12) >= SEARCH_BYTES_PER_WEIGHT * weights / (HBM_PEAK_GBS * 1e9)
    rl_search = {"bound": "alu", "achieved": round(search_tops, 3), "peak": round(VALU_PEAK_TOPS, 2),
                 "unit": "T lane-ops/s", "frac": round(search_tops / VALU_PEAK_TOPS, 4), "traffic": None,
                 "kernel": "hscale_search (search_kernel)",
                 "algorithmic_ops_per_step": ops, "hbm_GBps": round(search_gbs, 1),
                 "hbm_frac": round(search_gbs / HBM_PEAK_GBS, 4), "valu_frac": round(search_tops / VALU_PEAK_TOPS, 4),
                 "avg_ms_per_step": round(t_s.mean() * 1e3, 4),
                 "launches_per_step": 1 if len(layers) <= 32 else (len(layers) + 31) // 32,
                 "layers": len(layers)}
    if not valu_bound:
        rl_search.update({"bound": "hbm", "achieved": round(search_gbs, 1), "peak": HBM_PEAK_GBS, "unit": "GB/s",
                          "frac": round(search_gbs / HBM_PEAK_GBS, 4)})
    ceil = None
    if not args.no_ceilings:
        progress("measured ceilings (streaming read, VALU issue)")
        ceil = ceilings_leg(max(acts.values(), key=lambda X: X.numel()), stream)
        rl_hdiag["frac_of_stream_read"] = round(hd_gbs / ceil["stream_read"]["GBps"], 4)
        Ks = [2 * w + 1 if w is not None else args.down + args.up + 1 for (_, _, _, _, w) in layers]
        wc = sum(W.numel() * K for (_, W, _, _, _), K in zip(layers, Ks))
        rl_search["weight_candidates_per_s"] = wc / t_s.mean()
        walk = ("class" if all(CLASS_WALK_K[0] <= K <= CLASS_WALK_K[1] for K in Ks)
                else "plain" if all(K < CLASS_WALK_K[0] for K in Ks) else None)
        if walk is not None and valu_bound:
            probe = "search_class_pair" if walk == "class" else "search_pair"
            mix = ceil["valu"][f"{probe}_weight_candidates_per_s"]
            rl_search["search_mix_probe"] = probe
            rl_search["frac_of_search_mix"] = round(wc / t_s.mean() / mix, 4)
            if iso is not None:
                rl_search["frac_of_search_mix_isolated"] = round(wc / iso / mix, 4)
    default_shape = args.init == "maxabs" and args.down is None and args.window is None
    traffic = measured_traffic(args.workload) if default_shape else None
    if traffic:
        rl_hdiag["traffic"] = traffic["hdiag"]
        rl_search["traffic"] = traffic["search"]
        rl_hdiag["traffic_source"] = rl_search["traffic_source"] = traffic["source"]
        if traffic["valu"]:
            # VALU issue counters of the search kernel from the same summary
            rl_search["valu_counters"] = dict(traffic["valu"], source=traffic["source"])
    dominant = rl_hdiag if t_h.mean() >= t_s.mean() else rl_search

    out = {
        "metric": METRIC,
        "value": round(search_gws, 2),
        "unit": "Gweights/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(float(t_step.mean() * 1e3), 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "f32",
        "data": "synthetic",
        "config": {"workload": desc, "name": args.workload, "layers": [l for (l, _, _, _, _) in layers],
                   "weights": weights, "tokens": [X.shape[0] for X in acts.values()],
                   "windows": windows, "init": args.init},
        "hdiag": {"GBps": round(hd_gbs, 1), "frac_of_peak": round(hd_gbs / HBM_PEAK_GBS, 4),
                  "ms": round(t_h.mean() * 1e3, 4)},
        "search": {"Gweights_per_s": round(search_gws, 2), "ms": round(t_s.mean() * 1e3, 4),
                   "frac_of_valu_roofline": round(search_tops / VALU_PEAK_TOPS, 4)},
        "search_isolated": None if iso is None else {
            "Gweights_per_s": round(weights / iso / 1e9, 2), "ms": round(iso * 1e3, 4),
            "frac_of_valu_roofline": round(ops / iso / 1e12 / VALU_PEAK_TOPS, 4),
            "protocol": "the step's search call alone: 3 warm-ups, then the median of 20 runs, a 1 GiB device "
                        "buffer overwritten before each run; not the headline (the step runs the search right "
                        "after the hdiag read, at a lower engine clock)"},
        "step_Gweights_per_s": round(weights / t_step.mean() / 1e9, 3),
        "wall_s_timed": round(wall, 4),
        "roofline": dominant,
        "rooflines": {"hdiag": rl_hdiag, "search": rl_search},
        "ceilings": ceil,
    }
    if not args.no_cpu_baseline:
        progress("CPU oracle leg and parity")
        out.update(cpu_leg(args, acts, layers))
    if not args.no_diagnostics:
        progress("diagnostics leg")
        out["diagnostics"] = diag_leg(args, acts, layers)
    print(json.dumps(out), flush=True)


def isolated_search(run_search, stream):
    """Seconds of one search pass over the workload's layers timed alone: 3
    warm-ups, then the median of 20 runs with a 1 GiB buffer overwritten
    before every run so that W is not served from the Infinity Cache."""
    import torch

    flush = torch.empty(1 << 30, dtype=torch.uint8, device="cuda")
    for _ in range(3):
        flush.fill_(1)
        run_search()
    evs = []
    for _ in range(20):
        flush.fill_(1)
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record(stream)
        run_search()
        e1.record(stream)
        evs.append((e0, e1))
    torch.cuda.synchronize()
    del flush
    return float(np.median([a.elapsed_time(b) for a, b in evs])) * 1e-3


def load_probes():
    """libhscale_probes.so: the measurement probes (built beside libhscale.so)."""
    import ctypes

    if not os.path.exists(PROBE_LIB):
        raise RuntimeError(f"{PROBE_LIB} is not built: run `python __graft_entry__.py build`")
    lib = ctypes.CDLL(PROBE_LIB)
    P, i32, i64 = ctypes.c_void_p, ctypes.c_int32, ctypes.c_int64
    lib.hsprobe_stream_read.argtypes = [P, i64, i32, P, P]
    lib.hsprobe_stream_read.restype = i64
    lib.hsprobe_valu.argtypes = [i32, i32, i32, P, P, P]
    lib.hsprobe_valu.restype = ctypes.c_int
    lib.hsprobe_wall_clock_khz.argtypes = []
    lib.hsprobe_wall_clock_khz.restype = ctypes.c_int
    return lib


# hsprobe_valu kinds: (name, loop iterations, VALU instructions per iteration)
VALU_PROBES = {0: ("fma", 1024, 64), 1: ("pack_cvt", 256, 64), 2: ("unpack_cvt", 512, 64),
               3: ("search_pair", 512, None), 4: ("search_class_pair", 512, None)}
# Windows of this many candidates take the search's residue-class walk (when
# every lane of a wave has only normal, unclipped candidates); fewer take the
# plain walk.  Each is set against the probe of its own instruction stream.
CLASS_WALK_K = (16, 24)
READ_PROBE_BLOCKS = 1792  # as many blocks as the chip keeps resident (256 CUs x 7)


def ceilings_leg(X, stream):
    """What this MI355X sustains, measured in the same run, for the two kinds
    of work on the path:
      stream_read  a read of the largest activation tensor with 16-byte
                   non-temporal loads (the median of 5), against which hdiag's
                   rate is set (frac_of_stream_read);
      valu         VALU issue from registers with no memory traffic: plain fp32
                   FMAs, the FP4 pack and unpack conversions (cycles per wave64
                   instruction per SIMD at the clock read from s_memtime /
                   s_memrealtime), and the scale search's per-candidate
                   instruction stream (two candidates of a 16-weight group per
                   iteration; and the residue-class walk's stream for two
                   members of one class), whose weight-candidates per second
                   the search's own rate is set against (frac_of_search_mix,
                   against the stream of the walk its windows take; max-abs
                   and 4over6 initial codes alike, so 4over6's extra per-group
                   work shows as a lower fraction).  7 waves per SIMD, the
                   search kernel's occupancy."""
    import torch

    lib = load_probes()
    cus = torch.cuda.get_device_properties(0).multi_processor_count
    simds = 4 * cus

    def timed(fn, runs):
        # A warm-up run, then `runs` runs queued back to back with an event
        # between each two: the GPU is busy when each event is reached, so an
        # interval holds one kernel and none of the host's launch latency.
        statuses = [fn()]
        evs = [torch.cuda.Event(enable_timing=True) for _ in range(runs + 1)]
        evs[0].record(stream)
        for i in range(runs):
            statuses.append(fn())
            evs[i + 1].record(stream)
        torch.cuda.synchronize()
        ts = [evs[i].elapsed_time(evs[i + 1]) * 1e-3 for i in range(runs)]
        bad = [s for s in statuses if s < 0]
        return float(np.median(ts)), (bad[0] if bad else statuses[-1])

    sums = torch.empty(READ_PROBE_BLOCKS * 256, dtype=torch.int32, device=X.device)
    t_read, nread = timed(lambda: lib.hsprobe_stream_read(X.data_ptr(), X.numel() * X.element_size(),
                                                          READ_PROBE_BLOCKS, sums.data_ptr(), stream.cuda_stream), 5)
    if nread <= 0:
        raise RuntimeError("hsprobe_stream_read failed")
    read_gbs = nread / t_read / 1e9

    wall_hz = lib.hsprobe_wall_clock_khz() * 1e3
    blocks = 7 * cus
    sink = torch.empty(blocks * 256, dtype=torch.float32, device=X.device)
    clocks = torch.zeros(blocks * 4 * 4, dtype=torch.int64, device=X.device)
    valu = {"blocks": blocks, "waves_per_simd": 7}
    ghz = []
    for kind, (name, iters, per_iter) in VALU_PROBES.items():
        t, st = timed(lambda: lib.hsprobe_valu(kind, blocks, iters, sink.data_ptr(), clocks.data_ptr(),
                                               stream.cuda_stream), 3)
        if st != 0:
            raise RuntimeError(f"hsprobe_valu({kind}) failed")
        c = clocks.view(-1, 4).cpu().numpy().astype(np.float64)
        clock = float(np.median((c[:, 1] - c[:, 0]) / (c[:, 3] - c[:, 2]))) * wall_hz
        ghz.append(clock / 1e9)
        valu[f"{name}_ms"] = round(t * 1e3, 4)
        if per_iter is not None:
            instr_per_simd = blocks * 4 * iters * per_iter / simds
            valu[f"{name}_cycles_per_instr_per_simd"] = round(t * clock / instr_per_simd, 3)
            if name == "fma":
                valu["fma_T_lane_ops_per_s"] = round(blocks * 256 * iters * per_iter / t / 1e12, 2)
        else:
            valu[f"{name}_weight_candidates_per_s"] = blocks * 256 * iters * 2 * 16 / t
    valu["clock_GHz"] = [round(g, 3) for g in ghz]
    valu["clock_source"] = "median over waves of the s_memtime / s_memrealtime ratio, per probe"
    del sink, clocks, sums
    return {"stream_read": {"GBps": round(read_gbs, 1), "frac_of_peak": round(read_gbs / HBM_PEAK_GBS, 4),
                            "ms": round(t_read * 1e3, 4), "bytes": nread, "blocks": READ_PROBE_BLOCKS, "loads_in_flight_per_lane": 16},
            "valu": valu}


def copy_calibration(dev):
    """One plain 1 GiB device-to-device copy: a kernel of known traffic for
    scaling the HBM byte counters."""
    import torch
    src = torch.empty(1 << 30, dtype=torch.uint8, device=dev)
    src.fill_(1)
    dst = torch.empty_like(src)
    torch.cuda.synchronize()
    dst.copy_(src)
    torch.cuda.synchronize()
    del src, dst


def diag_leg(args, acts, layers, repeats=5):
    """Quality diagnostics of the paper's appendix on the workload's last
    layer, outside the timed hot-path steps: the search with per-group
    statistics and their per-shift summary (selected-shift figure), and the
    Eq. 3 layer-output error L_full of the initial codes, of the searched
    codes and of the full-ladder search, with the share of the full-ladder
    gain this window recovers (the window-sweep metric).  The output-error kernel is timed with HIP
    events on the stream it runs on and priced against the bf16 matrix-core
    peak with its algorithmic 2 T n m flops (it issues twice that: the
    rounding error enters as two bf16 parts)."""
    import torch
    import paper_2608_28113_amd as hs

    lname, W, xk, s_g, w = layers[-1]
    X = acts[xk]
    down, up = (w, w) if w is not None else (args.down, args.up)
    stream = torch.cuda.current_stream()
    T, n = X.shape
    m = W.shape[0]
    h = hs.hdiag(X)

    def timed(fn):
        ts, res = [], None
        for _ in range(repeats):
            e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            e0.record(stream)
            res = fn()
            e1.record(stream)
            torch.cuda.synchronize()
            ts.append(e0.elapsed_time(e1))
        return res, float(np.median(ts))

    st, t_stats = timed(lambda: hs.search_stats(W, h, s_g, down, up, init=args.init, stream=stream))
    summ, t_summ = timed(lambda: hs.shift_summary(st["shift"], st["err_best"], st["err_init"], down, up,
                                                   stream=stream))
    count = summ["count"].cpu().numpy().astype(np.float64)
    si, sb = summ["sum_init"].cpu().numpy(), summ["sum_best"].cpu().numpy()
    frac = count / count.sum()
    ws = torch.empty(max(hs.output_error_workspace_bytes(T, n, m), 256), dtype=torch.uint8, device=X.device)
    row = torch.zeros(m, dtype=torch.float64, device=X.device)

    def lfull(codes, packed):
        row.zero_()
        hs.output_error(X, W, s_g, codes, packed, row_err=row, workspace=ws, stream=stream)
        return row

    L_search, t_lf = timed(lambda: lfull(st["scale_codes"], st["packed_e2m1"]))
    L_search = float(L_search.sum().item())
    c0, p0 = hs.search(W, h, s_g, window=0, init=args.init, stream=stream)
    L_init = float(lfull(c0, p0).sum().item())
    # The window sweep's score (App. "Candidate-Window Width"): the share of
    # the max-abs -> full-ladder L_full gain that this window recovers; the
    # full ladder is every positive E4M3 code (window 125 from any start).
    cf, pf = hs.search(W, h, s_g, window=125, init=args.init, stream=stream)
    L_full_grid = float(lfull(cf, pf).sum().item())
    gain = L_init - L_full_grid
    flops = 2.0 * T * n * m
    tf = flops / (t_lf * 1e-3) / 1e12
    traffic = diag_traffic(args.workload) if (args.workload, down, up, args.init) == ("down_proj", 4, 4, "maxabs") \
        else None
    return {
        "layer": lname, "window": [down, up], "init": args.init, "tokens": T,
        "shift_fractions": {"keep": round(float(frac[down]), 4), "larger": round(float(frac[down + 1:].sum()), 4),
                            "smaller": round(float(frac[:down].sum()), 4)},
        "shift_histogram": {str(d): int(c) for d, c in zip(range(-down, up + 1), count)},
        "surrogate_error_removed": round(float(1.0 - sb.sum() / si.sum()), 4),
        "L_full_init": L_init, "L_full_search": L_search, "L_full_full_grid": L_full_grid,
        "L_full_reduction": round(1.0 - L_search / L_init, 4),
        "full_grid_gain_recovered": round((L_init - L_search) / gain, 4) if gain > 0 else None,
        "search_stats_ms": round(t_stats, 4), "shift_summary_ms": round(t_summ, 4),
        "output_error_ms": round(t_lf, 3),
        "roofline": {"bound": "mfma", "achieved": round(tf, 1), "peak": BF16_MFMA_PEAK_TFLOPS, "unit": "TFLOP/s",
                     "frac": round(tf / BF16_MFMA_PEAK_TFLOPS, 4), "traffic": traffic[0] if traffic else None,
                     "traffic_source": traffic[1] if traffic else None,
                     "kernel": "hscale_output_error (delta_split_kernel + lfull_tile_kernel + hdiag_tree)",
                     "algorithmic_flops": flops, "issued_mfma_flops": 2 * flops},
    }


def cpu_leg(args, acts, layers):
    """The oracle on this host's cores, on the workload's last layer: by
    default its whole W and whole X (the full configuration), else the first
    --cpu-rows rows and --cpu-tokens tokens.

    All cores: the rows (tokens) split into one contiguous chunk per core,
    one unmodified oracle call per chunk on its own thread (the oracle's C
    code shares no state between calls and ctypes releases the GIL), timed
    wall-clock.  One thread: a fixed 256-row search slice and an 8192-token
    hdiag slice, extrapolated linearly to the same size and labelled so.

    Parity: h for the check is the oracle's, over the same tokens, rounded
    to fp32 (no oracle input comes from the HIP path).  The HIP search runs
    again, untimed, on the whole last layer in the launch configuration the
    timed steps use, with that h; every checked row must match the oracle's
    search.  The HIP hdiag of the same tokens is checked against the
    oracle's h."""
    import torch
    import paper_2608_28113_amd as hs
    import oracle
    from synth.workloads import tensor_bits
    from tests import parity

    lname, W, xk, s_g, w = layers[-1]
    X = acts[xk]
    rows = W.shape[0] if args.cpu_rows is None else min(args.cpu_rows, W.shape[0])
    tok = X.shape[0] if args.cpu_tokens is None else min(args.cpu_tokens, X.shape[0])
    full = rows == W.shape[0] and tok == X.shape[0]
    down, up = (w, w) if w is not None else (args.down, args.up)
    init = "4over6" if args.init == "4over6" else "rtn"
    Wb = tensor_bits(W[:rows])
    Xb = tensor_bits(X[:tok])
    oracle._load()
    cores = _host_cores()

    # one thread, fixed slices
    r1, t1 = min(256, rows), min(8192, tok)
    t0 = time.perf_counter()
    h1 = oracle.hdiag(Xb[:t1])
    t_hd1 = time.perf_counter() - t0
    t0 = time.perf_counter()
    oracle.search(Wb[:r1], h1.astype(np.float32), s_g, down=down, up=up, init=init)
    t_s1 = time.perf_counter() - t0

    # all cores, the whole sample
    row_sl = [sl for sl in np.array_split(np.arange(rows), cores) if len(sl)]
    tok_sl = [sl for sl in np.array_split(np.arange(tok), cores) if len(sl)]
    with ThreadPoolExecutor(max_workers=cores) as ex:
        t0 = time.perf_counter()
        parts = list(ex.map(lambda sl: oracle.hdiag(Xb[sl[0]:sl[-1] + 1]), tok_sl))
        t_hd = time.perf_counter() - t0
        href = np.sum(parts, axis=0)  # fp64 sum of the chunk sums
        h_in = href.astype(np.float32)
        t0 = time.perf_counter()
        res = list(ex.map(lambda sl: oracle.search(Wb[sl[0]:sl[-1] + 1], h_in, s_g, down=down, up=up,
                                                   init=init), row_sl))
        t_search = time.perf_counter() - t0
    ref = {k: np.concatenate([r[k] for r in res]) for k in res[0]}

    codes, packed = hs.search(W, torch.from_numpy(h_in).to(W.device), s_g, down=down, up=up, init=args.init)
    rep = parity.compare_search(Wb, h_in, s_g, down, up, codes[:rows].cpu().numpy(), packed[:rows].cpu().numpy(),
                                init=init, oracle_result=ref)
    h_gpu = hs.hdiag(X if tok == X.shape[0] else X[:tok].contiguous()).cpu().numpy()
    hrep = parity.compare_h(h_gpu, href)
    what = (f"the full {lname} configuration: search of all {rows} rows ({Wb.size} weights, shifts -{down}..+{up}, "
            f"init {init}), hdiag of all {tok} tokens of its X ({Xb.nbytes / 1e9:.2f} GB)") if full else (
            f"rows 0..{rows - 1} of {lname} ({Wb.size} weights, shifts -{down}..+{up}, init {init}); "
            f"tokens 0..{tok - 1} of its X ({Xb.nbytes / 1e9:.2f} GB)")
    return {
        "cpu_baseline": {
            "value": round(Wb.size / t_search / 1e9, 6), "unit": "Gweights/s", "cores": len(row_sl),
            "kind": "oracle",
            "sample": f"{what}; {len(row_sl)} threads, one oracle call per contiguous chunk; search "
                      f"{t_search:.2f} s, hdiag {t_hd:.2f} s",
            "full_config": full,
            "hdiag_GBps": round(Xb.nbytes / t_hd / 1e9, 3),
            "search_s": round(t_search, 3), "hdiag_s": round(t_hd, 3),
            "cpu_model": _cpu_model(),
            "host_cpus": os.cpu_count(),
            "one_thread": {
                "value": round(r1 * Wb.shape[1] / t_s1 / 1e9, 6), "unit": "Gweights/s", "cores": 1,
                "hdiag_GBps": round(t1 * Xb.shape[1] * 2 / t_hd1 / 1e9, 3),
                "extrapolated": True,
                "search_s_extrapolated": round(t_s1 * rows / r1, 2),
                "hdiag_s_extrapolated": round(t_hd1 * tok / t1, 2),
                "sample": f"rows 0..{r1 - 1} ({t_s1:.2f} s) and tokens 0..{t1 - 1} ({t_hd1:.3f} s) on one "
                          f"thread, extrapolated linearly to the {rows} rows and {tok} tokens above"},
        },
        "parity": {"layer": lname, "h_source": f"oracle hdiag of tokens 0..{tok - 1} (chunk sums in fp64), fp32",
                   "search_rows_checked": rows, "groups": rep["groups"],
                   "near_ties": rep["near_ties"], "init_ties": rep["init_ties"], "mismatches": rep["mismatches"],
                   "ok": rep["ok"], "hdiag_tokens_checked": tok, "hdiag_max_rel": hrep["max_rel"],
                   "hdiag_ok": hrep["ok"]},
    }


def _host_cores() -> int:
    """Cores this process may use: the cgroup CPU quota when one is set,
    else the CPU affinity set."""
    n = len(os.sched_getaffinity(0))
    try:
        with open("/sys/fs/cgroup/cpu.max") as f:
            quota, period = f.read().split()[:2]
        if quota != "max":
            n = min(n, max(1, int(int(quota) // int(period))))
    except (OSError, ValueError):
        pass
    return n


def _cpu_model() -> str:
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
