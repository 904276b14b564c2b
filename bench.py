#!/usr/bin/env python3
"""Throughput of the bit-packed LUT-network forward pass on one MI355X.

One step = one whole forward (encode -> LUT layers -> GroupSum head + argmax)
over one batch already resident in HBM, through the C-ABI entry point
bitlogic_forward.  Default workload: the CIFAR-100-shaped wide network
(2^18 samples x 3072 uint8 features, 7 uniform thresholds = 21504 wires,
2 x 64000 nodes with k = 6, 100 classes x 640), synthetic seeded data.

Prints ONE JSON line.  Besides the driver's fields it carries
  roofline      the dominant kernel (the stage of the forward with the longest
                launch; on C4 a k = 6 LUT layer, which the roofline model puts
                on the integer VALU) against the chip's published peak for its
                bound, from per-launch HIP-event times
                that the library records between the stages of the same
                forward (bitlogic_forward_timed);
  cpu_baseline  the CPU oracle timed on a bounded sample of the same
                workload on this host (and its agreement with the GPU there);
  detail        per-stage times, algorithmic bytes/ops and roofline fractions,
                and the peaks measured on this device by the library's probes
                (integer VALU rate, HBM copy rate) with the dominant kernel's
                fraction of them.

Algorithmic work follows the path the library takes (bitlogic_forward_plan):
when the last LUT layer is fused with the GroupSum head its output bits are
never stored, so that stage's compulsory bytes are its input only and the
head's counting is charged to it; a layer that the node-per-wave kernel runs
(table-selected 3-input leaves, plan "jump_layers") is charged its 15
lane-ops per node and 32 samples instead of the 2^k - 1 multiplexers, which
puts it on its byte roofline.
"""
from __future__ import annotations

import argparse
import hashlib
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

# MI355X peaks (published): HBM3E bandwidth; 32-bit VALU lane-ops from
# 256 CUs x 4 SIMDs x 32 lanes a clock x 2.4 GHz (the published fp32 vector
# peak, 157.3 TFLOP/s, counts an FMA as two operations; the integer
# v_bitop3_b32 of the LUT layers issues at the same 32 lanes a clock)
PEAK_HBM_GBS = 8000.0
PEAK_VALU_TOPS = 256 * 4 * 32 * 2.4e9 / 1e12      # 78.64 T lane-ops/s

TRAFFIC_FILE = os.path.join(ROOT, "profiles", "forward_c4_traffic.json")

# The paper's own throughput for its deployed network (Sec. 7 hardware table),
# on an NVIDIA RTX 3090: MSamples/s by batch.  Context only (other hardware).
PAPER_MSAMPLES = {("paper_mnist_w4000", 1024): 8.6637, ("paper_mnist_w4000", 64): 0.5500}
CSRC = os.path.join(ROOT, "paper_2602_07400_amd", "csrc")


def parse():
    ap = argparse.ArgumentParser(description=__doc__.splitlines()[0])
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=50)
    ap.add_argument("--warmup", type=int, default=20)
    ap.add_argument("--config", default="c4_cifar100_wide")
    ap.add_argument("--seed", type=int, default=0)
    ap.add_argument("--cpu-seconds", type=float, default=15.0,
                    help="target CPU time of the oracle baseline sample")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-peaks", action="store_true",
                    help="skip the on-device peak probes (integer VALU rate, HBM copy rate)")
    ap.add_argument("--stage-steps", type=int, default=None,
                    help="steps of the per-kernel (staged) timing loop; default = --steps")
    ap.add_argument("--batch", type=int, default=None,
                    help="samples per forward (default: the configuration's batch)")
    ap.add_argument("--head", choices=["groupsum", "dsp"], default="groupsum",
                    help="class head of the timed forward: the popcount GroupSum, or the "
                         "quantized c x c head on the group sums (bitlogic_forward_grouped_dsp)")
    ap.add_argument("--encoder", choices=["thermometer", "binary"], default="thermometer",
                    help="input encoder: the configuration's thermometer, or the binary-coded "
                         "uniform fixed-point code (layer 1 is redrawn if the wire count changes)")
    ap.add_argument("--bits", type=int, default=None,
                    help="code width of the binary encoder (default: the configuration's b)")
    ap.add_argument("--specialize", action="store_true",
                    help="evaluate the network from its specialized tables (tied and "
                         "ignored inputs removed, nodes ordered by effective fan-in)")
    ap.add_argument("--power-seconds", type=float, default=0.0,
                    help="also run forwards back to back for this long while amd-smi samples "
                         "the board's socket power and engine clocks (detail.power)")
    ap.add_argument("--calibrate-copy-mib", type=int, default=0,
                    help="also run a write-only fill and a read-only sum over this many MiB "
                         "(reference kernels for scaling rocprofv3 FETCH_SIZE/WRITE_SIZE)")
    return ap.parse_args()


def algorithmic(cfg, n, fused_head, binary_bits=0, fanin_hist=None, jump_layers=()):
    """Compulsory bytes and algorithmic 32-bit lane-ops per stage of one forward.
    fanin_hist: per layer, None or the node count per effective fan-in 0..6 of
    a specialized layer (its multiplexers: 2^k' - 1 per node).
    jump_layers: layers the node-per-wave kernel evaluates with table-selected
    3-input leaves: 8 leaves + 7 multiplexers = 15 lane-ops per node and 32
    samples instead of 2^k - 1, which leaves such a layer bound by its bytes."""
    W = (n + 63) // 64
    D0 = cfg.d * (binary_bits or cfg.b)
    st = {"encode": {"bytes": n * cfg.d + D0 * W * 8, "ops": n * D0}}
    w_in = D0
    L = len(cfg.widths)
    for l, w in enumerate(cfg.widths):
        last_fused = fused_head and l == L - 1
        h = fanin_hist[l] if fanin_hist else None
        muxes = (((1 << cfg.k) - 1) * w if h is None else
                 sum(int(c) * ((1 << q) - 1) for q, c in enumerate(h)))
        if l in jump_layers:
            muxes = JUMP_OPS_PER_NODE * w
        st[f"layer{l + 1}"] = {
            # a fused last layer reads its input and hands counts to the head
            "bytes": (w_in + (0 if last_fused else w)) * W * 8,
            "ops": 2 * muxes * W + (n * w // 32 if last_fused else 0)}
        w_in = w
    out_bytes = 4 * n * cfg.n_classes + 4 * n
    if fused_head:
        st["head"] = {"bytes": out_bytes, "ops": n * cfg.n_classes}
    else:
        st["head"] = {"bytes": w_in * W * 8 + out_bytes, "ops": n * w_in // 32}
    for v in st.values():
        t_mem = v["bytes"] / (PEAK_HBM_GBS * 1e9)
        t_alu = v["ops"] / (PEAK_VALU_TOPS * 1e12)
        v["roof_ms"] = max(t_mem, t_alu) * 1e3
        v["bound"] = "hbm" if t_mem >= t_alu else "alu"
    return st


def cpu_model() -> str:
    """The host CPU's model name, from /proc/cpuinfo (empty if unreadable)."""
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return ""


def _smi_sample():
    """One amd-smi reading: (socket power W, [engine clock MHz per XCD], memory clock MHz)."""
    import subprocess
    r = subprocess.run(["amd-smi", "metric", "--power", "--clock", "--json"],
                       capture_output=True, text=True, timeout=20)
    g = json.loads(r.stdout)["gpu_data"][0]

    def num(v):
        v = v.get("value") if isinstance(v, dict) else v
        return float(v) if isinstance(v, (int, float)) else None

    clk = g["clock"]
    gfx = [num(clk[k]["clk"]) for k in sorted(clk) if k.startswith("gfx_")]
    mem = num(clk["mem_0"]["clk"]) if "mem_0" in clk else None
    return num(g["power"]["socket_power"]), [c for c in gfx if c is not None], mem


def power_under_load(step, seconds):
    """Run step() back to back for `seconds` while a thread samples amd-smi."""
    import threading
    samples, errors = [], []
    stop = threading.Event()

    def sampler():
        while not stop.is_set():
            try:
                samples.append((time.perf_counter(),) + _smi_sample())
            except Exception as e:            # tool missing or output not understood
                errors.append(repr(e))
                return
            stop.wait(0.2)

    import numpy as np
    import torch
    th = threading.Thread(target=sampler, daemon=True)
    t0 = time.perf_counter()
    th.start()
    n = 0
    while time.perf_counter() - t0 < seconds:
        for _ in range(50):
            step()
        torch.cuda.synchronize()
        n += 50
    t1 = time.perf_counter()
    stop.set()
    th.join()
    use = [s for s in samples if t0 + 1.0 <= s[0] <= t1]      # after a second of load
    if not use:
        return {"error": errors[0] if errors else "no amd-smi sample under load"}
    watts = [s[1] for s in use if s[1] is not None]
    gfx = [c for s in use for c in s[2]]
    mem = [s[3] for s in use if s[3] is not None]
    return {"seconds": round(t1 - t0, 2), "forwards": n,
            "ms_per_forward": round((t1 - t0) / n * 1e3, 4), "samples": len(use),
            "socket_power_W_median": float(np.median(watts)) if watts else None,
            "socket_power_W_range": [min(watts), max(watts)] if watts else None,
            "gfx_clock_MHz_median": float(np.median(gfx)) if gfx else None,
            "gfx_clock_MHz_range": [min(gfx), max(gfx)] if gfx else None,
            "mem_clock_MHz_median": float(np.median(mem)) if mem else None,
            "source": "amd-smi metric --power --clock --json, every ~0.2 s after the first "
                      "second of back-to-back forwards; engine clocks of all XCDs"}


def measured_traffic(stage):
    """HBM bytes per launch of `stage` from the committed rocprofv3 counter
    summary (FETCH_SIZE + WRITE_SIZE, scaled), or None when a kernel source
    changed since the counters were taken or the stage was not measured."""
    try:
        with open(TRAFFIC_FILE) as f:
            rec = json.load(f)
        sources = {n for n in os.listdir(CSRC) if n.endswith((".hip", ".h"))}
        if sources != set(rec["sources_sha256"]):
            return None
        for name, digest in rec["sources_sha256"].items():
            with open(os.path.join(CSRC, name), "rb") as f:
                if hashlib.sha256(f.read()).hexdigest() != digest:
                    return None
        return rec["stages"][stage]["bytes"]
    except (OSError, ValueError, KeyError):
        return None


JUMP_OPS_PER_NODE = 15      # 8 table-selected v_bitop3_b32 leaves + 7 multiplexers
STAGE_KERNELS = {"encode": "k_encode_t / k_encode_ballot (encoder + bit-pack)",
                 "layer": "k_lut_slab (LUT layer)",
                 "layer_jump": "k_jump_prep + k_jump_layer (LUT layer, a node per wave, "
                               "table-selected bitop3 leaves)",
                 "layer_fused": "k_lut_slab_head (last LUT layer fused with GroupSum counting)",
                 "head_fused": "k_head_finish (counts -> scores, argmax)",
                 "head": "k_head_planes + k_head_finish (GroupSum head, argmax)"}


def main():
    args = parse()
    if args.gpus != 1:
        print(f"bench.py runs on one GPU only: the path shards by samples with no exchange, and "
              f"this library has no multi-GPU driver; got --gpus {args.gpus}", file=sys.stderr)
        sys.exit(2)

    import numpy as np
    import torch

    from paper_2602_07400_amd import bitlogic as bl
    from paper_2602_07400_amd.workloads import CONFIGS, make_workload

    assert torch.cuda.is_available(), "bench.py needs a GPU"
    dev = torch.device("cuda:0")
    cfg = CONFIGS[args.config]
    t0 = time.time()
    wl = make_workload(cfg, seed=args.seed, n=args.batch)
    print(f"[bench] {cfg.name}: generated inputs in {time.time() - t0:.1f}s", file=sys.stderr,
          flush=True)
    n = wl.n
    binary_bits = 0
    if args.encoder == "binary":
        binary_bits = args.bits or cfg.b
        if cfg.d * binary_bits != cfg.wires:
            # another wire count: layer 1 reads the binary wires (seeded redraw)
            from paper_2602_07400_amd.workloads import draw_connectivity
            rng = np.random.default_rng([args.seed, binary_bits, 1])
            conn0, tab0 = wl.layers[0]
            wl.layers[0] = (draw_connectivity(rng, conn0.shape[0], cfg.k, cfg.d * binary_bits),
                            tab0)
    dsp_np = wl.dsp_weights if args.head == "dsp" else None
    model = bl.BitlogicModel.from_numpy(None if binary_bits else wl.thresholds, wl.layers,
                                        wl.n_classes, device=dev,
                                        encoder="binary" if binary_bits else "thermometer",
                                        n_features=cfg.d, n_bits=binary_bits or None,
                                        head_weights=dsp_np, specialize=args.specialize)
    dsp_w = model.head_weights
    x = torch.from_numpy(wl.x).to(dev)
    ws = torch.empty(model.workspace_bytes(n), dtype=torch.uint8, device=dev)
    scores = torch.empty((n, cfg.n_classes), dtype=torch.int32, device=dev)
    argmax = torch.empty((n,), dtype=torch.int32, device=dev)
    stream = torch.cuda.current_stream(dev)

    def step(events=None):
        model.forward(x, out=scores, argmax=argmax, workspace=ws, stream=stream, events=events)

    if args.calibrate_copy_mib:
        # reference kernels of known traffic for scaling rocprofv3's
        # FETCH_SIZE / WRITE_SIZE: a read-only reduction and a write-only fill
        nbytes = args.calibrate_copy_mib << 20
        buf = torch.empty(nbytes // 8, dtype=torch.int64, device=dev)
        for _ in range(2):
            buf.fill_(1)
        torch.cuda.synchronize()
        for _ in range(2):
            total = buf.sum()
        torch.cuda.synchronize()
        del buf, total
        print(f"[bench] calibration: fill_ writes and sum reads {nbytes} bytes, twice each",
              file=sys.stderr, flush=True)

    # ---- warmup, then exactly K timed steps
    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()
    t_start = time.perf_counter()
    for _ in range(args.steps):
        step()
    torch.cuda.synchronize()
    elapsed = time.perf_counter() - t_start
    ms_per_step = elapsed / args.steps * 1e3
    value = n * args.steps / elapsed / 1e6
    print(f"[bench] timed {args.steps} steps: {ms_per_step:.3f} ms/step, {value:.2f} MSamples/s",
          file=sys.stderr, flush=True)

    # ---- per-kernel times: the same forward with HIP events recorded by the
    # library at its stage boundaries, on the stream its kernels run on
    layer_names = [f"layer{l + 1}" for l in range(len(cfg.widths))]
    names = ["encode"] + layer_names + ["head"]
    ksteps = args.stage_steps or args.steps
    sums = np.zeros(len(names))
    for it in range(ksteps + 2):
        ev = [torch.cuda.Event(enable_timing=True) for _ in range(len(names) + 1)]
        for e in ev:
            e.record(stream)          # creates the HIP event handles
        step(ev)
        torch.cuda.synchronize()
        if it >= 2:                   # two untimed passes first
            sums += [ev[i].elapsed_time(ev[i + 1]) for i in range(len(names))]
    stage_ms = dict(zip(names, (sums / ksteps).tolist()))
    plan = model.plan(n)

    # ---- board power and engine clocks under a sustained load of the forward
    power = None
    if args.power_seconds > 0:
        power = power_under_load(step, args.power_seconds)
        print(f"[bench] power under load: {power}", file=sys.stderr, flush=True)

    # ---- on-device peaks, after the timed work: probes with the hot path's
    # instruction and access types (v_bitop3_b32 chains; 16-byte non-temporal
    # copies), giving measured roofline denominators beside the published ones
    peaks = None
    if not args.no_peaks:
        def span(fn, reps):
            e0 = torch.cuda.Event(enable_timing=True)
            e1 = torch.cuda.Event(enable_timing=True)
            for r in range(2):
                fn(r)
            e0.record(stream)
            for r in range(reps):
                work = fn(r)
            e1.record(stream)
            torch.cuda.synchronize()
            return work * reps / (e0.elapsed_time(e1) * 1e-3)
        pblocks = 256 * 256                    # 256 blocks a CU: enough waves to saturate
        pout = torch.empty(pblocks * bl.PROBE_THREADS, dtype=torch.int32, device=dev)
        valu = span(lambda r: bl.bitlogic_probe_valu(pout, pblocks, 1024, r, stream), 5) / 1e12
        # HBM streams of 4 GiB: read-only, write-only and copy, each at a few
        # loads-in-flight depths and grid sizes; the best of each is reported
        cbytes = 4 << 30
        csrc = torch.ones(cbytes, dtype=torch.uint8, device=dev)
        cdst = torch.empty_like(csrc)
        hbm = {}
        for mode, tag in ((bl.PROBE_HBM_READ, "read"), (bl.PROBE_HBM_WRITE, "write"),
                          (bl.PROBE_HBM_COPY, "copy")):
            best = None
            for unroll, blocks in ((4, 256 * 8), (8, 256 * 4), (8, 256 * 8), (2, 256 * 16)):
                src = None if mode == bl.PROBE_HBM_WRITE else csrc
                rate = span(lambda r: bl.bitlogic_probe_hbm(mode, src, cdst, cbytes, unroll,
                                                            blocks, stream), 5) / 1e9
                if best is None or rate > best[0]:
                    best = (rate, unroll, blocks)
            hbm[tag] = best
        # instruction rates of the multiplexer (three source banks, and two
        # sources in one bank) and of the table-bit mask extraction, in cycles
        # per wave instruction per SIMD at the measured engine clock span
        ops = {}
        for op, tag in ((bl.PROBE_OP_MUX, "mux_3banks"), (bl.PROBE_OP_MUX_BANK, "mux_2banks"),
                        (bl.PROBE_OP_BFE, "bfe_mask")):
            rate = span(lambda r: bl.bitlogic_probe_valu_op(op, pout, pblocks // 4, 64, r,
                                                            stream), 5)
            ops[tag] = round(rate * 64 / 1e12, 3)          # T lane-ops/s
        # the layers' row gathers alone (no multiplexers) and with 512 VALU
        # instructions per pass, at 4 waves per SIMD as the layer kernels run:
        # 16 rows per load instruction in two halves (lanes_per_row 4) or whole
        # lines (8), over an L2-resident 2.75 MB set (C4's layer-1 slab) and an
        # 8.2 MB set (its layer-2 slab), with and without the output stores
        gather = {}
        gblocks, gpasses = 256 * 16, 8
        gout = torch.empty(gblocks * 256, dtype=torch.int32, device=dev)
        gsink = torch.empty(gblocks * gpasses * 8192, dtype=torch.uint8, device=dev)
        for mb, nrow in (("2.75MB", 21504), ("8.2MB", 64000)):
            grows = torch.ones(nrow * 128, dtype=torch.uint8, device=dev)
            for lpr, v, sk in ((4, 0, False), (8, 0, False), (4, 512, False), (4, 0, True),
                               (4, 512, True)):
                rate = span(lambda r: bl.bitlogic_probe_gather(
                    grows, lpr, v, gblocks, gpasses, gout, gsink if sk else None,
                    waves_per_simd=4, seed=r, stream=stream), 5)
                gather[f"{mb} lanes/row {lpr} valu {v}{' +stores' if sk else ''}"] = round(
                    rate * 128 / 1e12, 2)                  # TB/s of gathered lines
            del grows
        del pout, csrc, cdst, gout, gsink
        peaks = {"valu_TOPs": round(valu, 3),
                 "valu_frac_of_published": round(valu / PEAK_VALU_TOPS, 4),
                 "hbm_read_GBs": round(hbm["read"][0], 1),
                 "hbm_write_GBs": round(hbm["write"][0], 1),
                 "hbm_copy_GBs": round(hbm["copy"][0], 1),
                 "hbm_read_frac_of_published": round(hbm["read"][0] / PEAK_HBM_GBS, 4),
                 "valu_op_T_lane_ops": ops,
                 "gather_TBs": gather,
                 "probes": "bitlogic_probe_valu (65536 x 256 lanes, 1024 rounds of 8 v_bitop3_b32); "
                           "bitlogic_probe_valu_op (16384 x 256 lanes, 64 rounds of 64); "
                           "bitlogic_probe_gather (4096 blocks x 8 passes, 4 waves per SIMD); "
                           "bitlogic_probe_hbm over 4 GiB, best of (unroll, blocks) in "
                           "(4, 2048), (8, 1024), (8, 2048), (2, 4096): "
                           + ", ".join(f"{t} unroll {u} blocks {b}" for t, (_, u, b) in hbm.items())
                           + " (copy counts read + write)"}
        print(f"[bench] measured peaks: {valu:.2f} T int32 lane-ops/s, HBM read "
              f"{hbm['read'][0]:.0f} / write {hbm['write'][0]:.0f} / copy {hbm['copy'][0]:.0f} GB/s",
              file=sys.stderr, flush=True)

    dsp_detail = None
    if dsp_w is not None:
        # the quantized head alone, on the group sums of this batch: HIP events
        # on the launch stream around repeated calls
        counts = torch.empty((n, cfg.n_classes), dtype=torch.int32, device=dev)
        plain = bl.BitlogicModel(model.thresholds, model.layers, model.n_classes, model.n_features,
                                 model.encoder, model.n_bits, pass_fanin=model.pass_fanin,
                                 fanin_histogram=model.fanin_histogram, order=model.order)
        plain.forward(x, out=counts, argmax=argmax, workspace=ws, stream=stream)
        lg = torch.empty_like(counts)
        reps = max(ksteps, 10)
        for _ in range(3):
            bl.bitlogic_grouped_dsp_head(counts, dsp_w, logits=lg, argmax=argmax, stream=stream)
        e0 = torch.cuda.Event(enable_timing=True)
        e1 = torch.cuda.Event(enable_timing=True)
        e0.record(stream)
        for _ in range(reps):
            bl.bitlogic_grouped_dsp_head(counts, dsp_w, logits=lg, argmax=argmax, stream=stream)
        e1.record(stream)
        torch.cuda.synchronize()
        t_ms = e0.elapsed_time(e1) / reps
        c = cfg.n_classes
        hb = 8 * n * c + 4 * n + c * c            # counts in, logits + argmax out, weights
        hops = 2 * n * c * c                      # int8 MACs on the matrix cores, x2 ops
        dsp_detail = {"kernel": "k_grouped_dsp (bitlogic_grouped_dsp_head, 8-bit MFMA)",
                      "ms": round(t_ms, 4), "bytes": hb, "int8_ops": hops,
                      "bound": "hbm", "achieved_GBs": round(hb / (t_ms * 1e-3) / 1e9, 1),
                      "frac_of_hbm_peak": round(hb / (t_ms * 1e-3) / 1e9 / PEAK_HBM_GBS, 4),
                      "achieved_int8_TOPs": round(hops / (t_ms * 1e-3) / 1e12, 3)}

    # quantile-threshold fitting on the device over this batch: HBM-bound
    # (reads N*d pixel bytes); per-channel groups for 3-channel images
    groups = cfg.channels if cfg.d % max(cfg.channels, 1) == 0 else 1
    th_fit = torch.empty((cfg.d, cfg.b), dtype=torch.uint8, device=dev)
    fit_ws = torch.empty(max(8, groups * 256 * 8), dtype=torch.uint8, device=dev)
    for _ in range(2):
        bl.bitlogic_fit_quantile_thresholds(x, cfg.b, groups, out=th_fit, workspace=fit_ws,
                                            stream=stream)
    f0 = torch.cuda.Event(enable_timing=True)
    f1 = torch.cuda.Event(enable_timing=True)
    f0.record(stream)
    for _ in range(5):
        bl.bitlogic_fit_quantile_thresholds(x, cfg.b, groups, out=th_fit, workspace=fit_ws,
                                            stream=stream)
    f1.record(stream)
    torch.cuda.synchronize()
    fit_ms = f0.elapsed_time(f1) / 5
    fit_detail = {"kernels": "k_fit_clear + k_fit_hist + k_fit_select "
                             "(bitlogic_fit_quantile_thresholds)",
                  "groups": groups, "thresholds": cfg.b, "ms": round(fit_ms, 4),
                  "bytes": n * cfg.d,
                  "achieved_GBs": round(n * cfg.d / (fit_ms * 1e-3) / 1e9, 1),
                  "frac_of_hbm_peak": round(n * cfg.d / (fit_ms * 1e-3) / 1e9 / PEAK_HBM_GBS, 4)}

    fused = plan["fused_head"]
    jump = plan.get("jump_layers", [])
    alg = algorithmic(cfg, n, fused, binary_bits, model.fanin_histogram, jump)
    roof_sum = sum(v["roof_ms"] for v in alg.values())
    # dominant kernel: the stage with the longest launch
    dom = max(names, key=lambda k: stage_ms[k])
    a = alg[dom]
    if a["bound"] == "alu":
        achieved = a["ops"] / (stage_ms[dom] * 1e-3) / 1e12
        peak, unit, per = PEAK_VALU_TOPS, "TOP/s", f"{a['ops']} int32 lane-ops"
    else:
        achieved = a["bytes"] / (stage_ms[dom] * 1e-3) / 1e9
        peak, unit, per = PEAK_HBM_GBS, "GB/s", f"{a['bytes']} bytes"
    if dom == "encode":
        kname = STAGE_KERNELS["encode"]
    elif dom == "head":
        kname = STAGE_KERNELS["head_fused" if fused else "head"]
    elif dom == layer_names[-1] and fused:
        kname = STAGE_KERNELS["layer_fused"]
    elif layer_names.index(dom) in jump:
        kname = STAGE_KERNELS["layer_jump"]
    else:
        kname = STAGE_KERNELS["layer"]
    if model.pass_fanin and dom in layer_names:
        kname += ", specialized (one fan-in per pass)"
    roofline = {"bound": a["bound"], "achieved": round(achieved, 3), "peak": round(peak, 3),
                "unit": unit, "frac": round(achieved / peak, 4),
                "traffic": measured_traffic(dom) if cfg.name == "c4_cifar100_wide" else None,
                "kernel": f"{kname}; stage {dom}",
                "per_launch": per}

    detail = {
        "stage_ms": {k: round(v, 4) for k, v in stage_ms.items()},
        "stage_roofline_ms": {k: round(v["roof_ms"], 4) for k, v in alg.items()},
        "stage_bound": {k: v["bound"] for k, v in alg.items()},
        "stage_achieved_GBs": {k: round(alg[k]["bytes"] / (stage_ms[k] * 1e-3) / 1e9, 1)
                               for k in names},
        "stage_achieved_TOPs": {k: round(alg[k]["ops"] / (stage_ms[k] * 1e-3) / 1e12, 3)
                                for k in names},
        "forward_roofline_ms": round(roof_sum, 4),
        "forward_roofline_frac": round(roof_sum / ms_per_step, 4),
        "staged_sum_ms": round(sum(stage_ms.values()), 4),
        "fused_head": fused,
        "jump_layers": [layer_names[l] for l in jump],
        "specialized": bool(args.specialize),
        "fanin_histogram": ([None if h is None else [int(v) for v in h]
                             for h in model.fanin_histogram]
                            if model.fanin_histogram else None),
        "head": args.head,
        "encoder": args.encoder + (f" ({binary_bits} bits)" if binary_bits else ""),
        "grouped_dsp_head": dsp_detail,
        "fit_quantile_thresholds": fit_detail,
        "layer_frac_of_valu_peak": {k: round(alg[k]["ops"] / (stage_ms[k] * 1e-3) / 1e12
                                             / PEAK_VALU_TOPS, 4) for k in layer_names},
        # the row segments the layers gather (k per node, each read whole), and
        # the rate at which each layer moves them from the caches: the path that
        # binds the k = 6 layers (compare measured_peaks.gather_TBs)
        "layer_gathered_GB": {k: round(cfg.k * w * n / 8 / 1e9, 3)
                              for k, w in zip(layer_names, cfg.widths)},
        "layer_gather_TBs": {k: round(cfg.k * w * n / 8 / (stage_ms[k] * 1e-3) / 1e12, 2)
                             for k, w in zip(layer_names, cfg.widths)},
        "measured_peaks": peaks,
        "dominant_frac_of_measured_peak": (
            None if peaks is None else
            round(achieved / (peaks["valu_TOPs"] if a["bound"] == "alu" else
                              max(peaks["hbm_read_GBs"], peaks["hbm_write_GBs"],
                                  peaks["hbm_copy_GBs"])), 4)),
        "gpu": torch.cuda.get_device_name(dev),
        "hip": torch.version.hip,
    }
    if power is not None:
        detail["power"] = power

    # ---- CPU oracle on a bounded sample of the same workload
    cpu = None
    if not args.no_cpu_baseline:
        import oracle
        step()                        # outputs of the timed forward itself
        torch.cuda.synchronize()
        threads = oracle.max_threads()
        probe = min(n, 2048)
        t0 = time.perf_counter()
        oracle.forward(wl.x[:probe], wl.thresholds, wl.layers, wl.n_classes,
                       binary_bits=binary_bits)
        per = (time.perf_counter() - t0) / probe
        m = int(min(n, max(probe, args.cpu_seconds / max(per, 1e-9))))
        idx = np.random.default_rng(1).choice(n, size=m, replace=False)
        idx.sort()
        xs = np.ascontiguousarray(wl.x[idx])
        t0 = time.perf_counter()
        rs, rp = oracle.forward(xs, wl.thresholds, wl.layers, wl.n_classes,
                                binary_bits=binary_bits)
        if dsp_w is not None:
            rs, rp = oracle.grouped_dsp(rs, wl.dsp_weights)
        cpu_s = time.perf_counter() - t0
        agree = bool(np.array_equal(scores.cpu().numpy()[idx].astype(np.int64), rs) and
                     np.array_equal(argmax.cpu().numpy()[idx], rp))
        # one thread on a smaller sample (about a tenth of the time budget)
        m1 = int(min(m, max(64, args.cpu_seconds / 10 / max(per * threads, 1e-9))))
        t0 = time.perf_counter()
        oracle.forward(xs[:m1], wl.thresholds, wl.layers, wl.n_classes, n_threads=1,
                       binary_bits=binary_bits)
        cpu1_s = time.perf_counter() - t0
        cpu = {"value": round(m / cpu_s / 1e6, 6), "unit": "MSamples/s", "cores": threads,
               "kind": "oracle",
               "sample": f"{m} random samples of the {n}-sample batch, whole forward, "
                         f"{cpu_s:.1f} s on {threads} OpenMP threads",
               "gpu_agrees_on_sample": agree,
               "single_thread_value": round(m1 / cpu1_s / 1e6, 6),
               "single_thread_sample": f"the first {m1} of those samples, {cpu1_s:.1f} s",
               "cpu_model": cpu_model()}
        print(f"[bench] oracle: {m} samples in {cpu_s:.1f}s on {threads} threads; "
              f"GPU agrees: {agree}", file=sys.stderr, flush=True)

    out = {
        "metric": "MSamples/s end-to-end LUT-net inference at 1 GPU; % of HBM/int-VALU roofline",
        "value": round(value, 3),
        "unit": "MSamples/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms_per_step, 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": (round(value / PAPER_MSAMPLES[(cfg.name, n)], 3)
                        if (cfg.name, n) in PAPER_MSAMPLES and args.encoder == "thermometer"
                        and args.head == "groupsum" else None),
        "dtype": "u64 (bitwise on packed 64-sample words; u8 pixels, i32 scores)",
        "data": "synthetic",
        "config": {"workload": cfg.description
                   + ("" if not binary_bits else
                      f"; binary-coded {binary_bits}-bit encoder instead of the thermometer")
                   + ("" if dsp_w is None else "; quantized c x c head on the group sums")
                   + ("" if not args.specialize else "; table-specialized layers"),
                   "name": cfg.name, "head": args.head, "encoder": args.encoder,
                   "n_samples": n,
                   "features": cfg.d, "thresholds": cfg.b, "widths": list(cfg.widths),
                   "k": cfg.k, "classes": cfg.n_classes, "seed": args.seed},
        "roofline": roofline,
        "cpu_baseline": cpu,
        "detail": detail,
    }
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
