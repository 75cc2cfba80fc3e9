"""Benchmark of the shard halo-convolution hot path on one MI355X.

One step = one pass of the whole per-shard hot path over one synthetic shard:
pack the boundary faces this shard sends (both faces of an axis in one launch),
unpack the received slabs into its margins (both margins of an axis in one
launch), forward convolution, weight gradient. All inputs are resident in HBM
before the timed region. Geometry and slab shapes come from the library
itself; the CPU oracle is used only by the cpu_baseline leg. Prints ONE JSON
line on stdout (progress goes to stderr).

    python bench.py [--steps K] [--warmup W] [--workload c3] [--no-cpu-baseline] [--copy-calibration]
                    [--no-backward]

The ops beyond the step on the same shard - the backward pass (input gradient
onto the padded tile, reverse halo), group normalisation with statistics over
all shards (the shard's sums, then the interior normalised), the forward with
the halo folded into its loads (whole, interior, boundary) and one ring-attention
block step - are timed after the step and reported under "next_rows"; they are
not part of `value`.

Beside the published peaks the line carries the part's measured ceilings: a
device-to-device copy of the halo launch's bytes ("measured_copy_ceiling"), and a
matrix-instruction-only kernel with the shader clock it ran at plus hipBLASLt on
a large square bf16 GEMM ("measured_mfma_ceiling"; bf16 workloads, skipped with
--no-backward).

The roofline's "traffic" field is the HBM traffic of the dominant kernel measured
with rocprofv3 counters (FETCH_SIZE and WRITE_SIZE, each scaled by what it reads
for a plain device copy of known size) and recorded in
profiles/<op>_<workload>_traffic.txt together with a hash of that kernel's sources;
it is reported only while the sources still hash the same, else null.
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

PEAK = {"bf16": 2516.6, "f32": 157.3}   # dense MFMA TFLOP/s, MI355X (AMD spec)
HBM_PEAK = 8000.0                        # GB/s
# Targets of the hot path: the convolutions at half the bf16 MFMA peak on the
# bf16 workloads; the halo copies at 70 % of the HBM peak on the two largest
# shards (the smaller ones are launch-bound and not held to it).
CONV_TARGET = 0.50
HALO_TARGET = 0.70
HALO_TARGET_WORKLOADS = ("c3", "c5")

DESCR = {
    "c1": "2d_fp32_c8_64x64_split2H_shard0_k3",
    "c2": "2d_bf16_c64_4096x4096_split4H_shard1_k3",
    "c3": "3d_bf16_c32_512cube_split4D_shard1_k3_smooth",
    "c4": "3d_bf16_c16to64_256cube_split2x2DH_corner_k5",
    "c5": "3d_fp32_c64to128_384cube_split8D_shard3_k3_s2",
}


def log(msg):
    print(msg, file=sys.stderr, flush=True)


def geometry(sc, w, idx):
    off, ext = w.interior(idx)
    sharded = [1 if p > 1 else 0 for p in w.parts]
    g = sc.shard_conv_geometry(w.G, off, ext, w.K, w.S, sharded)
    g["off"], g["ext"] = off, ext
    return g


def margin_box(g, axis, side):
    """Tile-coordinate box of the margin on (axis, side): the slab layout of the
    library (padded extent on earlier axes, interior on later ones)."""
    lo, ext, hi = g["halo_lo"], g["ext"], g["halo_hi"]
    b0, b1 = [], []
    for b in range(len(ext)):
        if b == axis:
            r = (0, lo[b]) if side == 0 else (lo[b] + ext[b], lo[b] + ext[b] + hi[b])
        elif b < axis:
            r = (0, lo[b] + ext[b] + hi[b])
        else:
            r = (lo[b], lo[b] + ext[b])
        b0.append(r[0])
        b1.append(r[1])
    return b0, b1


def dev(arr):
    import numpy as np
    import torch
    if arr.dtype == np.uint16:
        return torch.from_numpy(np.ascontiguousarray(arr).view(np.int16)).view(torch.bfloat16).cuda()
    return torch.from_numpy(np.ascontiguousarray(arr)).cuda()


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=10)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--workload", default="c3", choices=sorted(DESCR))
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--copy-calibration", action="store_true",
                    help="run one 64 MiB device-to-device copy first (reference for counter scaling)")
    ap.add_argument("--no-backward", action="store_true",
                    help="skip the ops beyond the step (input gradient, reverse halo, group normalisation, "
                         "folded forward, attention) and the measured MFMA ceiling")
    args = ap.parse_args()
    if args.gpus != 1:
        print(f"bench.py measures one GPU's shard; --gpus {args.gpus} is not supported: shardconv has no "
              "multi-GPU path (no collectives or sharding across devices)", file=sys.stderr)
        sys.exit(2)

    import numpy as np
    import torch

    import synth
    from synth.workloads import SHORT
    from paper_2605_11111_amd import shardconv as sc

    w = SHORT[args.workload]
    torch.cuda.set_device(0)
    g = geometry(sc, w, w.shard)
    lo, hi, ext = g["halo_lo"], g["halo_hi"], g["ext"]
    tile_lo = [o - h for o, h in zip(g["off"], lo)]
    tile_hi = [o + e + h for o, e, h in zip(g["off"], ext, hi)]
    t0 = time.time()
    full_h = w.x_box(tile_lo, tile_hi)
    log(f"generated padded box {full_h.shape} in {time.time() - t0:.1f}s ({synth.threads()} threads)")
    tile = dev(full_h)
    desc = sc.tile_desc(w.N, w.cin, ext, lo, hi)
    tdt = torch.float32 if w.dtype == "f32" else torch.bfloat16

    recv, send = [], []
    for axis in range(w.nd):
        for side in (0, 1):
            width = lo[axis] if side == 0 else hi[axis]
            if width > 0:
                b0, b1 = margin_box(g, axis, side)
                box = (slice(None),) + tuple(slice(a, b) for a, b in zip(b0, b1)) + (slice(None),)
                nbytes = full_h[box].size * full_h.itemsize
                slab = dev(full_h[box]) if w.neighbour_exists(w.shard, axis, side) else None
                recv.append((axis, side, slab, nbytes))
            if w.neighbour_exists(w.shard, axis, side):
                nb = list(w.shard)
                nb[axis] += 1 if side else -1
                ng = geometry(sc, w, tuple(nb))
                nwidth = ng["halo_lo"][axis] if side == 1 else ng["halo_hi"][axis]
                if nwidth > 0:
                    buf = torch.empty(sc.shard_halo_slab_shape(desc, axis, nwidth), dtype=tdt, device="cuda")
                    send.append((axis, side, nwidth, buf, buf.numel() * buf.element_size()))
    del full_h
    O = g["out_ext"]
    wt = dev(w.weights_host())
    full_out = sc.shard_conv_geometry(w.G, [0] * w.nd, list(w.G), w.K, w.S, [0] * w.nd)["out_ext"]
    t0 = time.time()
    dyh = w.dy_field(full_out).box((0, 0, *g["out_off"]), (w.N, w.cout, *[o + e for o, e in zip(g["out_off"], O)]),
                                   out=w.out)
    dy = dev(dyh)
    del dyh
    log(f"generated dy in {time.time() - t0:.1f}s")
    y = torch.empty([w.N] + list(O) + [w.cout], dtype=tdt, device="cuda")
    dw = torch.empty((w.cout, w.cin) + tuple(w.K), dtype=torch.float32, device="cuda")
    code = sc.SHARD_F32 if w.dtype == "f32" else sc.SHARD_BF16
    wsf = torch.empty(max(16, sc.shard_conv_workspace_bytes(0, desc, code, w.cout, w.K, w.S, O)),
                      dtype=torch.uint8, device="cuda")
    wsw = torch.empty(max(16, sc.shard_conv_workspace_bytes(1, desc, code, w.cout, w.K, w.S, O)),
                      dtype=torch.uint8, device="cuda")
    stream = torch.cuda.current_stream()

    # the exchange along an axis: both faces packed by one launch before the
    # sends, both margins filled by one launch after the receives
    ops = []
    for axis in range(w.nd):
        sends = {side: (nwidth, buf, nbytes) for (a_, side, nwidth, buf, nbytes) in send if a_ == axis}
        if sends:
            wl, bl, nl = sends.get(0, (0, None, 0))
            wh, bh, nh = sends.get(1, (0, None, 0))
            ops.append((f"pack_a{axis}", "pack", 2 * (nl + nh),
                        lambda axis=axis, wl=wl, bl=bl, wh=wh, bh=bh:
                        sc.shard_halo_pack_pair(desc, tile, axis, wl, bl, wh, bh)))
        recvs = {side: (slab, nbytes) for (a_, side, slab, nbytes) in recv if a_ == axis}
        if recvs:
            sl, nl = recvs.get(0, (None, 0))
            sh, nh = recvs.get(1, (None, 0))
            moved = (2 if sl is not None else 1) * nl + (2 if sh is not None else 1) * nh
            ops.append((f"unpack_a{axis}", "unpack", moved,
                        lambda axis=axis, sl=sl, sh=sh: sc.shard_halo_unpack_pair(desc, tile, axis, sl, sh)))
    flops = 2.0 * w.N * int(np.prod(O)) * w.cout * w.cin * int(np.prod(w.K))
    ops.append(("conv_fwd", "fwd", flops,
                lambda: sc.shard_conv_fwd(desc, tile, wt, w.cout, w.K, w.S, g["pad_lo"], O, y, wsf)))
    ops.append(("conv_wgrad", "wgrad", flops,
                lambda: sc.shard_conv_wgrad(desc, tile, dy, w.cout, w.K, w.S, g["pad_lo"], O, dw, wsw)))

    def step(events=None):
        for i, op in enumerate(ops):
            if events is not None:
                events[i][0].record(stream)
            op[3]()
            if events is not None:
                events[i][1].record(stream)

    if args.copy_calibration:
        src = torch.empty(64 << 20, dtype=torch.uint8, device="cuda")
        src.fill_(1)
        torch.cuda.synchronize()
        torch.empty_like(src).copy_(src)
        torch.cuda.synchronize()
        del src
    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()
    log("warmup done")
    ev = [[[torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)] for _ in ops]
          for _ in range(args.steps)]
    start, stop = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    start.record(stream)
    for k in range(args.steps):
        step(ev[k])
    stop.record(stream)
    torch.cuda.synchronize()
    ms_step = start.elapsed_time(stop) / args.steps
    # the weight gradient's status word (0 unless a bounded wait inside the
    # kernel gave up, which would also have made dw NaN)
    if int(wsw[:4].view(torch.int32).item()) != 0 or not bool(torch.isfinite(dw).all()):
        log("weight gradient reported a failed hand-off wait")
        sys.exit(3)
    per_op = {}
    for i, (label, kind, work, _) in enumerate(ops):
        per_op[label] = (kind, work, float(np.mean([ev[k][i][0].elapsed_time(ev[k][i][1])
                                                     for k in range(args.steps)])))
    log("timed region done")

    # the halo launches again, cold: 8 launches on 8 rotating buffer sets
    cold = time_halo_cold(sc, w, desc, tile, ops, send, recv, args, stream)

    next_rows = None
    if not args.no_backward:
        next_rows = time_backward(sc, w, g, desc, wt, dy, send, flops, args, stream)
        next_rows.update(time_group_norm(sc, w, g, desc, tile, args, stream))
        next_rows.update(time_folded(sc, w, g, desc, tile, wt, dy, recv, args, stream))
        next_rows.update(time_attention(sc, args, stream))

    dt = w.dtype
    value = 2 * flops / (ms_step * 1e-3) / 1e12
    halo_kernel = measured_halo_kernel(args.workload)
    detail = {}
    for label, (kind, work, ms) in per_op.items():
        if kind in ("fwd", "wgrad"):
            tf = work / (ms * 1e-3) / 1e12
            detail[label] = {"ms": round(ms, 4), "tflops": round(tf, 2), "frac_mfma_peak": round(tf / PEAK[dt], 4)}
            if dt == "bf16":
                # the stated target for the convolutions on the bf16 workloads
                detail[label]["target_frac_mfma_peak"] = CONV_TARGET
                detail[label]["meets_target"] = bool(tf / PEAK[dt] >= CONV_TARGET)
            ctr = measured_counters(label, args.workload)
            if ctr:
                detail[label]["mfma_busy_frac"] = ctr["mfma_busy_frac"]
                detail[label]["counters"] = ctr
        else:
            # the gated figures are the cold ones; the launch inside the step
            # (event pair around one launch, caches as the step left them) beside them
            cms = cold[label]
            gbs = work / (cms * 1e-3) / 1e9
            detail[label] = {"ms": round(cms, 4), "gbs": round(gbs, 1), "frac_hbm_peak": round(gbs / HBM_PEAK, 4),
                             "bytes": int(work), "in_step_ms": round(ms, 4),
                             "protocol": "cold: 8 consecutive launches on 8 buffer sets (tile and slabs, 8 x the bytes "
                                         "> the 256 MB last-level cache), replayed from a captured graph between "
                                         "one event pair, per launch; median of the repeats"}
            hk = halo_kernel.get(kind) if halo_kernel and label.endswith("_a0") else None
            if hk:
                # the same launches' kernel time from the committed rocprofv3 trace
                # (the event-timed figure adds the gaps between graph nodes)
                detail[label]["kernel_ms_rocprof"] = round(hk * 1e-3, 4)
                detail[label]["frac_hbm_peak_kernel"] = round(work / (hk * 1e-6) / 1e9 / HBM_PEAK, 4)
                detail[label]["kernel_source"] = halo_kernel["source"]
            if args.workload in HALO_TARGET_WORKLOADS:
                # the stated target for the halo copies on the largest shards
                detail[label]["target_frac_hbm_peak"] = HALO_TARGET
                detail[label]["meets_target"] = bool(gbs / HBM_PEAK >= HALO_TARGET)
    dom = max(("conv_fwd", "conv_wgrad"), key=lambda k: per_op[k][2])
    ach = per_op[dom][1] / (per_op[dom][2] * 1e-3) / 1e12
    roofline = {"kernel": dom, "bound": "mfma", "achieved": round(ach, 2), "peak": PEAK[dt], "unit": "TFLOP/s",
                "frac": round(ach / PEAK[dt], 4), "traffic": measured_traffic(dom, args.workload),
                "work_per_launch": f"{flops:.4e} flop: 2*Cout*Cin*prod(K) per output voxel x {int(np.prod(O))} voxels"}

    halo_bytes = max((work for (label, kind, work, _) in ops if kind in ("pack", "unpack")), default=0)
    ceiling = measured_ceiling(args, stream, int(halo_bytes)) if halo_bytes else None
    mfma_ceiling = measured_mfma_ceiling(stream) if dt == "bf16" and not args.no_backward else None
    cpu = None if args.no_cpu_baseline else cpu_baseline(w, g, tile_lo)
    line = {
        "metric": "shard conv fwd+wgrad TFLOP/s (% MFMA peak); halo pack/unpack GB/s (% HBM)",
        "value": round(value, 3), "unit": "TFLOP/s", "n_gpus": 1, "steps": args.steps, "warmup": args.warmup,
        "ms_per_step": round(ms_step, 4), "higher_is_better": True, "scaling": "weak", "vs_baseline": None,
        "dtype": "bf16" if dt == "bf16" else "f32", "data": "synthetic (seeded counter-based generator)",
        "config": {"workload": DESCR[args.workload],
                   "tile_padded": [w.N] + [l + e + h for l, e, h in zip(lo, ext, hi)] + [w.cin],
                   "out": [w.N] + list(O) + [w.cout], "kernel": list(w.K), "stride": list(w.S),
                   "accumulate": "f32"},
        "ops": detail, "roofline": roofline, "measured_copy_ceiling": ceiling,
        "measured_mfma_ceiling": mfma_ceiling, "cpu_baseline": cpu,
        "next_rows": next_rows,
    }
    print(json.dumps(line), flush=True)


def time_halo_cold(sc, w, desc, tile, ops, send, recv, args, stream):
    """Per-launch time of every halo op of the step on cold data: 8 copies of
    the tile and of every slab, used in turn by 8 consecutive launches between
    one event pair (each set was last touched 7 launches earlier, 7 x its bytes
    ago: more than the last-level cache holds at the workloads' sizes), median
    over `steps` repeats. The launches are replayed from a captured graph and
    one event pair spans all 8, so neither host call overhead nor the event
    overhead enters the figure, which is close to the kernel time."""
    import numpy as np
    import torch
    NS = 8
    halo = [(label, kind) for (label, kind, _, _) in ops if kind in ("pack", "unpack")]
    if not halo:
        return {}
    tiles = [tile] + [tile.clone() for _ in range(NS - 1)]
    out = {}
    for label, kind in halo:
        axis = int(label.split("_a")[1])
        calls, outs = [], []
        for k in range(NS):
            if kind == "pack":
                sends = {side: (nwidth, buf) for (a_, side, nwidth, buf, _) in send if a_ == axis}
                wl, bl = sends.get(0, (0, None))
                wh, bh = sends.get(1, (0, None))
                bl = torch.empty_like(bl) if bl is not None else None
                bh = torch.empty_like(bh) if bh is not None else None
                outs += [b for b in (bl, bh) if b is not None]
                calls.append(lambda t=tiles[k], wl=wl, bl=bl, wh=wh, bh=bh:
                             sc.shard_halo_pack_pair(desc, t, axis, wl, bl, wh, bh))
            else:
                rv = {side: slab for (a_, side, slab, _) in recv if a_ == axis}
                sl = rv.get(0)
                sh = rv.get(1)
                sl = sl.clone() if sl is not None else None
                sh = sh.clone() if sh is not None else None
                calls.append(lambda t=tiles[k], sl=sl, sh=sh: sc.shard_halo_unpack_pair(desc, t, axis, sl, sh))
        for c in calls:
            c()
        torch.cuda.synchronize()
        # the 8 launches are replayed from a captured graph, so that the host's
        # per-call cost (argument checks, the binding) cannot leave the GPU idle
        # between kernels of ~10 us; the graph's first replay is checked bit for
        # bit against the eager calls' result
        ref = [t.clone() for t in outs] if outs else None
        graph = torch.cuda.CUDAGraph()
        with torch.cuda.graph(graph):
            for c in calls:
                c()
        for t in outs:
            t.zero_()
        graph.replay()
        torch.cuda.synchronize()
        if ref is not None and not all(torch.equal(a, b) for a, b in zip(ref, outs)):
            raise RuntimeError(f"{label}: graph replay differs from the eager launches")
        times = []
        for _ in range(max(3, args.steps)):
            e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            e0.record(stream)
            graph.replay()
            e1.record(stream)
            torch.cuda.synchronize()
            times.append(e0.elapsed_time(e1) / NS)
        out[label] = float(np.median(times))
        del calls, graph, ref
    del tiles
    torch.cuda.empty_cache()
    log("cold halo launches timed")
    return out


def time_backward(sc, w, g, desc, wt, dy, send, flops, args, stream):
    """The backward-pass ops of the same shard, timed after the step (they are not
    part of `value`): the input gradient onto the padded tile, then the reverse
    halo per axis - the margins' gradients packed for the neighbours they came
    from (both sides in one launch), and the received gradient slabs added onto
    the interior faces (one launch; the slabs the forward pack filled stand in
    for the neighbours' gradients: same shapes)."""
    import numpy as np
    import torch
    tdt = torch.float32 if w.dtype == "f32" else torch.bfloat16
    code = sc.SHARD_F32 if w.dtype == "f32" else sc.SHARD_BF16
    O = g["out_ext"]
    P = [l + e + h for l, e, h in zip(g["halo_lo"], g["ext"], g["halo_hi"])]
    dtile = torch.empty([w.N] + P + [w.cin], dtype=tdt, device="cuda")
    wsd = torch.empty(max(16, sc.shard_conv_workspace_bytes(2, desc, code, w.cout, w.K, w.S, O)),
                      dtype=torch.uint8, device="cuda")
    ops = [("conv_dgrad", "dgrad", flops,
            lambda: sc.shard_conv_dgrad(desc, dy, wt, w.cout, w.K, w.S, g["pad_lo"], O, dtile, wsd))]
    # the reverse exchange runs the axes in descending order; both sides of an
    # axis go out in one launch and come back in one launch
    for axis in reversed(range(w.nd)):
        bufs, moved = [None, None], 0
        for side in (0, 1):
            width = g["halo_lo"][axis] if side == 0 else g["halo_hi"][axis]
            if width > 0 and w.neighbour_exists(w.shard, axis, side):
                bufs[side] = torch.empty(sc.shard_halo_slab_shape(desc, axis, width), dtype=tdt, device="cuda")
                moved += 2 * bufs[side].numel() * bufs[side].element_size()
        if moved:
            ops.append((f"pack_margin_a{axis}", "halo", moved,
                        lambda axis=axis, b=bufs: sc.shard_halo_pack_margin_pair(desc, dtile, axis, b[0], b[1])))
        recv = {side: (nwidth, buf, nbytes) for (a_, side, nwidth, buf, nbytes) in send if a_ == axis}
        if recv:
            wl, bl, nl = recv.get(0, (0, None, 0))
            wh, bh, nh = recv.get(1, (0, None, 0))
            # read slab + read and write the face rows
            ops.append((f"accumulate_a{axis}", "halo", 3 * (nl + nh),
                        lambda axis=axis, wl=wl, bl=bl, wh=wh, bh=bh:
                        sc.shard_halo_accumulate_pair(desc, dtile, axis, wl, bl, wh, bh)))
    for _ in range(args.warmup):
        for op in ops:
            op[3]()
    torch.cuda.synchronize()
    ev = [[[torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)] for _ in ops]
          for _ in range(args.steps)]
    for k in range(args.steps):
        for i, op in enumerate(ops):
            ev[k][i][0].record(stream)
            op[3]()
            ev[k][i][1].record(stream)
    torch.cuda.synchronize()
    out = {}
    for i, (label, kind, work, _) in enumerate(ops):
        ms = _median_ms(label, [ev[k][i][0].elapsed_time(ev[k][i][1]) for k in range(args.steps)])
        if kind == "dgrad":
            tf = work / (ms * 1e-3) / 1e12
            out[label] = {"ms": round(ms, 4), "tflops": round(tf, 2), "frac_mfma_peak": round(tf / PEAK[w.dtype], 4)}
        else:
            gbs = work / (ms * 1e-3) / 1e9
            out[label] = {"ms": round(ms, 4), "gbs": round(gbs, 1), "frac_hbm_peak": round(gbs / HBM_PEAK, 4),
                          "bytes": int(work)}
    log("backward ops timed")
    return out


def _median_ms(label, times):
    """Median of the event-timed repeats of a side op (the step's own ops are
    averaged). A repeat far above the median is reported on stderr: one-off
    stalls outside the kernels (seen as a single slow repeat) then cannot move
    the reported figure."""
    import numpy as np
    med = float(np.median(times))
    if max(times) > 1.5 * med:
        log(f"{label}: repeats {', '.join(f'{t:.3f}' for t in times)} ms (median {med:.3f})")
    return med


def _time_ops(ops, args, stream):
    import numpy as np
    import torch
    for _ in range(args.warmup):
        for op in ops:
            op[3]()
    torch.cuda.synchronize()
    ev = [[[torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)] for _ in ops]
          for _ in range(args.steps)]
    for k in range(args.steps):
        for i, op in enumerate(ops):
            ev[k][i][0].record(stream)
            op[3]()
            ev[k][i][1].record(stream)
    torch.cuda.synchronize()
    out = {}
    for i, (label, kind, work, _) in enumerate(ops):
        ms = _median_ms(label, [ev[k][i][0].elapsed_time(ev[k][i][1]) for k in range(args.steps)])
        if kind.startswith("mfma:"):
            tf = work / (ms * 1e-3) / 1e12
            out[label] = {"ms": round(ms, 4), "tflops": round(tf, 2),
                          "frac_mfma_peak": round(tf / PEAK[kind[5:]], 4)}
        else:
            gbs = work / (ms * 1e-3) / 1e9
            out[label] = {"ms": round(ms, 4), "gbs": round(gbs, 1), "frac_hbm_peak": round(gbs / HBM_PEAK, 4),
                          "bytes": int(work)}
    return out


def time_folded(sc, w, g, desc, tile, wt, dy, recv, args, stream):
    """The forward with the halo folded into its loads (margins never read; the
    received slabs serve the margin rows), whole and as the interior / boundary
    pair that lets the exchange overlap the interior (timed after the step, not
    part of `value`; flops of each part are those of its outputs)."""
    import numpy as np
    import torch
    tdt = torch.float32 if w.dtype == "f32" else torch.bfloat16
    code = sc.SHARD_F32 if w.dtype == "f32" else sc.SHARD_BF16
    O = g["out_ext"]
    y = torch.empty([w.N] + list(O) + [w.cout], dtype=tdt, device="cuda")
    ws = torch.empty(max(16, sc.shard_conv_workspace_bytes(0, desc, code, w.cout, w.K, w.S, O)),
                     dtype=torch.uint8, device="cuda")
    slabs = {(axis, side): slab for (axis, side, slab, _) in recv}
    lo, hi = sc.shard_conv_interior(desc, w.K, w.S, g["pad_lo"], O)
    per_vox = 2.0 * w.N * w.cout * w.cin * int(np.prod(w.K))
    n_all = int(np.prod(O))
    n_int = int(np.prod([b - a for a, b in zip(lo, hi)]))

    def call(region, sl):
        return lambda: sc.shard_conv_fwd_folded(desc, tile, sl, region, wt, w.cout, w.K, w.S, g["pad_lo"], O, y, ws)
    dw = torch.empty((w.cout, w.cin) + tuple(w.K), dtype=torch.float32, device="cuda")
    wsw = torch.empty(max(16, sc.shard_conv_workspace_bytes(1, desc, code, w.cout, w.K, w.S, O)), dtype=torch.uint8,
                      device="cuda")
    ops = [("conv_fwd_folded", "mfma:" + w.dtype, per_vox * n_all, call(sc.SHARD_REGION_ALL, slabs)),
           ("conv_wgrad_folded", "mfma:" + w.dtype, per_vox * n_all,
            lambda: sc.shard_conv_wgrad_folded(desc, tile, slabs, dy, w.cout, w.K, w.S, g["pad_lo"], O, dw, wsw)),
           ("conv_fwd_interior", "mfma:" + w.dtype, per_vox * n_int, call(sc.SHARD_REGION_INTERIOR, None)),
           ("conv_fwd_boundary", "mfma:" + w.dtype, per_vox * (n_all - n_int), call(sc.SHARD_REGION_BOUNDARY, slabs))]
    res = _time_ops(ops, args, stream)
    log("folded forward timed")
    return res


def measured_ceiling(args, stream, nbytes):
    """The part's own copy rate at the halo's size: a device-to-device copy
    (torch's copy_, the runtime's blit kernel) of nbytes / 2 read + nbytes / 2
    written, over 8 buffer pairs in turn, event-timed like the halo launches."""
    import numpy as np
    import torch
    half = nbytes // 2
    pairs = [(torch.empty(half, dtype=torch.uint8, device="cuda").fill_(1),
              torch.empty(half, dtype=torch.uint8, device="cuda")) for _ in range(8)]
    flush = torch.empty(512 << 20, dtype=torch.uint8, device="cuda")
    times = []
    for k in range(max(8, args.steps)):
        src, dst = pairs[k % 8]
        flush.fill_(k & 255)      # evict the last-level cache between copies
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record(stream)
        dst.copy_(src)
        e1.record(stream)
        torch.cuda.synchronize()
        times.append(e0.elapsed_time(e1))
    ms = float(np.median(times))
    gbs = nbytes / (ms * 1e-3) / 1e9
    del pairs, flush
    return {"ms": round(ms, 4), "gbs": round(gbs, 1), "frac_hbm_peak": round(gbs / HBM_PEAK, 4), "bytes": int(nbytes),
            "what": "device-to-device copy of the same bytes (torch copy_), median of event-timed launches"}


def measured_mfma_ceiling(stream):
    """The part's sustained bf16 matrix rate and shader clock: a kernel of
    nothing but v_mfma_f32_32x32x16_bf16 (one 4-wave workgroup per compute unit,
    4 independent chains per wave, libshardprobe.so), on constant operands and
    on random ones that change every instruction (the part is power-limited and
    toggling operands lower its clock), median of 3 launches each; and the rate
    hipBLASLt reaches on a large square bf16 GEMM of N(0, 1) operands
    (torch.matmul), the vendor library's own figure for a plain contraction.
    Context beside the published peak, not a bound of the path."""
    import numpy as np
    import torch
    from paper_2605_11111_amd import probe
    cus = torch.cuda.get_device_properties(0).multi_processor_count
    iters = 20000
    out = torch.empty(cus * 256, dtype=torch.float32, device="cuda")
    clk = torch.empty(2 * cus, dtype=torch.int64, device="cuda")
    res = {}
    for random in (False, True):
        runs = []
        for k in range(4):
            e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            e0.record(stream)
            probe.shard_probe_mfma_bf16(iters, cus, random, out, clk)
            e1.record(stream)
            torch.cuda.synchronize()
            c = clk.cpu().numpy().reshape(-1, 2).astype(np.float64)
            mhz = float(np.mean(c[:, 0] / (c[:, 1] / 100.0)))
            if k > 0:
                runs.append((e0.elapsed_time(e1), mhz))
        ms, mhz = sorted(runs)[len(runs) // 2]
        tf = 2.0 * 32 * 32 * 16 * 4 * iters * cus * 4 / (ms * 1e-3) / 1e12
        res["mfma_only_random" if random else "mfma_only_constant"] = {
            "tflops": round(tf, 1), "frac_mfma_peak": round(tf / PEAK["bf16"], 4), "shader_clock_mhz": round(mhz),
            "ms": round(ms, 4),
            "what": "v_mfma_f32_32x32x16_bf16 only, 4 chains per wave, 1 wave per SIMD, "
                    + ("random N(0,1) operands changing every instruction" if random else "constant operands")}
    n = 8192
    a = torch.randn(n, n, device="cuda", dtype=torch.bfloat16)
    b = torch.randn(n, n, device="cuda", dtype=torch.bfloat16)
    for _ in range(3):
        torch.matmul(a, b)
    torch.cuda.synchronize()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record(stream)
    for _ in range(10):
        torch.matmul(a, b)
    e1.record(stream)
    torch.cuda.synchronize()
    gms = e0.elapsed_time(e1) / 10
    gtf = 2.0 * n ** 3 / (gms * 1e-3) / 1e12
    del a, b
    res["gemm"] = {"tflops": round(gtf, 1), "frac_mfma_peak": round(gtf / PEAK["bf16"], 4), "ms": round(gms, 4),
                   "what": "torch.matmul bf16 8192x8192x8192, N(0,1) operands (hipBLASLt)"}
    return res


def time_attention(sc, args, stream):
    """One ring-attention block step on a sequence shard: 16 heads of dim 128,
    16384 local queries against a 16384-key block (a 131072-token sequence over
    8 devices), merged into a running state (4 * heads * Sq * Sk * D flops)."""
    import torch
    B, H, S, D = 1, 16, 16384, 128
    g = torch.Generator(device="cuda").manual_seed(0)
    q = torch.randn((B, H, S, D), generator=g, device="cuda").to(torch.bfloat16)
    k = torch.randn((B, H, S, D), generator=g, device="cuda").to(torch.bfloat16)
    v = torch.randn((B, H, S, D), generator=g, device="cuda").to(torch.bfloat16)
    o = torch.zeros((B, H, S, D), device="cuda")
    lse = torch.zeros((B, H, S), device="cuda")
    scale = D ** -0.5
    sc.shard_attn_block(q, k, v, o, lse, scale, True)
    flops = 4.0 * B * H * S * S * D
    ops = [("attn_block", "mfma:bf16", flops, lambda: sc.shard_attn_block(q, k, v, o, lse, scale, False))]
    res = _time_ops(ops, args, stream)
    res["attn_block"]["shape"] = f"B{B} H{H} Sq{S} Sk{S} D{D}"
    log("attention block step timed")
    return res


def time_group_norm(sc, w, g, desc, tile, args, stream):
    """Group normalisation of the shard's interior (c / 8 groups): its sums (reads
    the interior once) and the normalisation with those sums standing for the
    totals over all shards (reads and writes the interior), into a second tile."""
    import numpy as np
    import torch
    code = sc.SHARD_F32 if w.dtype == "f32" else sc.SHARD_BF16
    groups = max(1, w.cin // 8)
    ws = torch.empty(max(16, sc.shard_norm_workspace_bytes(desc, code, groups)), dtype=torch.uint8, device="cuda")
    sums = torch.empty((w.N, groups, 2), dtype=torch.float64, device="cuda")
    out = torch.empty_like(tile)
    gamma = torch.ones(w.cin, device="cuda")
    beta = torch.zeros(w.cin, device="cuda")
    inner_bytes = w.N * int(np.prod(g["ext"])) * w.cin * tile.element_size()
    count = int(np.prod(w.G)) * (w.cin // groups)
    sc.shard_norm_stats(desc, tile, groups, sums, ws)
    torch.cuda.synchronize()
    ops = [("norm_stats", "norm", inner_bytes, lambda: sc.shard_norm_stats(desc, tile, groups, sums, ws)),
           ("norm_apply", "norm", 2 * inner_bytes,
            lambda: sc.shard_norm_apply(desc, tile, sums, count, 1e-5, groups, gamma, beta, out, ws))]
    res = _time_ops(ops, args, stream)
    log("group normalisation timed")
    return res


# The source files each measured kernel is built and launched from: the kernel
# itself, its host-side launcher and the shared headers.
KERNEL_SOURCES = {
    "conv_fwd": ["conv_fwd.hip", "conv_fwd_rows.hip", "common.h", "internal.h"],
    "conv_wgrad": ["conv_wgrad.hip", "conv_wgrad_xm.hip", "common.h", "internal.h"],
    "halo": ["halo.hip", "common.h", "internal.h"],
}


def source_hash(op):
    """sha256 over the sources of `op`'s kernel (any change to them invalidates
    the recorded counters)."""
    h = hashlib.sha256()
    files = [os.path.join(ROOT, "paper_2605_11111_amd", "csrc", f) for f in KERNEL_SOURCES[op]]
    for f in files:
        h.update(os.path.basename(f).encode())
        with open(f, "rb") as fh:
            h.update(fh.read())
    return h.hexdigest()


def measured_counters(op, workload):
    """Matrix-core utilisation of `op`'s main kernel from the committed counter
    summary (rocprofv3 --pmc: SQ_VALU_MFMA_BUSY_CYCLES over the SIMD cycles the
    kernel ran, at the clock it ran at), or None when there is none or the
    kernel sources changed since it was taken."""
    path = os.path.join(ROOT, "profiles", f"{op}_{workload}_counters.txt")
    if not os.path.exists(path):
        return None
    rec = {}
    with open(path) as fh:
        for line in fh:
            if ":" in line and not line.startswith("#"):
                k, v = line.split(":", 1)
                rec[k.strip()] = v.strip()
    if rec.get("source_sha256") != source_hash(op):
        return None
    out = {}
    for k in ("mfma_busy_frac", "valu_per_mfma", "salu_per_mfma", "lds_bank_conflict_per_lds_cycle", "clock_mhz"):
        try:
            out[k] = float(rec[k])
        except (KeyError, ValueError):
            pass
    if "mfma_busy_frac" not in out:
        return None
    out["kernel"] = rec.get("kernel")
    out["source"] = f"profiles/{op}_{workload}_counters.txt"
    return out


def measured_halo_kernel(workload):
    """rocprofv3 kernel durations (µs, medians) of the cold graph-replayed pack
    and unpack launches from the committed kernel trace summary, or None when
    there is none or the halo sources changed since it was taken."""
    path = os.path.join(ROOT, "profiles", f"halo_{workload}_kernel_trace.txt")
    if not os.path.exists(path):
        return None
    rec = {}
    with open(path) as fh:
        for line in fh:
            if ":" in line and not line.startswith("#"):
                k, v = line.split(":", 1)
                rec[k.strip()] = v.strip()
    if rec.get("source_sha256") != source_hash("halo"):
        return None
    try:
        return {"pack": float(rec["pack_cold_kernel_us"]), "unpack": float(rec["unpack_cold_kernel_us"]),
                "source": f"profiles/halo_{workload}_kernel_trace.txt"}
    except (KeyError, ValueError):
        return None


def measured_traffic(op, workload):
    """HBM bytes per launch of `op` from the committed counter summary, or None
    when there is none or the kernel sources changed since it was taken."""
    path = os.path.join(ROOT, "profiles", f"{op}_{workload}_traffic.txt")
    if not os.path.exists(path):
        return None
    rec = {}
    with open(path) as fh:
        for line in fh:
            if ":" in line and not line.startswith("#"):
                k, v = line.split(":", 1)
                rec[k.strip()] = v.strip()
    if rec.get("source_sha256") != source_hash(op):
        return None
    try:
        return int(float(rec["traffic_bytes_per_launch"]))
    except (KeyError, ValueError):
        return None


def cpu_baseline(w, g, tile_lo):
    """The oracle (float64 NumPy) timed on a bounded sample of the same shard:
    forward and weight gradient over a few output planes along axis 0."""
    import numpy as np
    from oracle import conv as oconv
    from synth.workloads import as_f64
    try:
        from threadpoolctl import threadpool_info
        cores = max([i.get("num_threads", 1) for i in threadpool_info()] + [1])
    except Exception:
        cores = os.cpu_count()
    L = g["out_ext"][0]
    sharded = [p > 1 for p in w.parts]
    pad = [0 if sharded[a] else (w.K[a] - 1) // 2 for a in range(w.nd)]
    full_out = [(G + 2 * ((K - 1) // 2) - K) // S + 1 for G, K, S in zip(w.G, w.K, w.S)]
    w64 = as_f64(w.weights_host())
    dyf = w.dy_field(full_out)
    budget = 12.0          # seconds of oracle time
    sec, planes = 0.0, 0
    p0 = L // 2
    while sec < budget and planes < L:
        p = (p0 + planes) % L
        r0 = p * w.S[0] - g["pad_lo"][0]
        r1 = p * w.S[0] - g["pad_lo"][0] + w.K[0]
        lo_t = [tile_lo[0] + r0] + [0 - pad[a] if not sharded[a] else tile_lo[a] for a in range(1, w.nd)]
        hi_t = [tile_lo[0] + r1] + [w.G[a] + pad[a] if not sharded[a] else
                                    tile_lo[a] + g["halo_lo"][a] + g["ext"][a] + g["halo_hi"][a]
                                    for a in range(1, w.nd)]
        xw = np.moveaxis(as_f64(w.x_box(lo_t, hi_t)), -1, 1)
        lo = list(g["out_off"])
        hi = [o + e for o, e in zip(g["out_off"], g["out_ext"])]
        lo[0], hi[0] = lo[0] + p, lo[0] + p + 1
        dy64 = np.moveaxis(as_f64(dyf.box((0, 0, *lo), (w.N, w.cout, *hi), out=w.out)), -1, 1)
        t0 = time.time()
        oconv.conv_forward_window(xw, lo_t, w.G, w64, w.S, lo, hi)
        oconv.conv_wgrad_window(xw, lo_t, w.G, dy64, w.K, w.S, lo, hi)
        sec += time.time() - t0
        planes += 1
    plane_vox = w.N * int(np.prod(g["out_ext"][1:]))
    fl = 2 * 2.0 * planes * plane_vox * w.cout * w.cin * int(np.prod(w.K))
    return {"value": round(fl / sec / 1e12, 6), "unit": "TFLOP/s", "cores": int(cores), "kind": "oracle",
            "sample": f"fwd+wgrad over {planes} of {L} output planes along axis 0 of the same shard, "
                      f"one plane per call ({sec:.1f}s of oracle time, float64 NumPy; input generation excluded)"}


if __name__ == "__main__":
    main()
