"""Device helpers for the GPU parity tests: upload/download of channels-last
buffers, and running one shard's hot path through the C-ABI binding."""
from __future__ import annotations

import sys

import numpy as np

import synth
import shard_cases as cases

CANARY_BF16 = np.uint16(0x7FC1)             # a NaN pattern never produced by the generator
CANARY_F32 = np.array([0x7FC00001], dtype=np.uint32).view(np.float32)[0]


def log(msg: str):
    print(msg, flush=True)
    sys.stdout.flush()


def dev(arr: np.ndarray):
    import torch
    if arr.dtype == np.uint16:
        return torch.from_numpy(np.ascontiguousarray(arr).view(np.int16)).view(torch.bfloat16).cuda()
    return torch.from_numpy(np.ascontiguousarray(arr)).cuda()


def host(t) -> np.ndarray:
    import torch
    t = t.detach().cpu().contiguous()
    if t.dtype == torch.bfloat16:
        return t.view(torch.int16).numpy().view(np.uint16)
    return t.numpy()


def canary_for(w):
    return CANARY_BF16 if w.dtype == "bf16" else CANARY_F32


def empty_like_dtype(shape, w):
    import torch
    return torch.empty(tuple(shape), dtype=cases.torch_dtype(w), device="cuda")


def build_tile(sc, w, idx, dist=None, keep_host=False):
    """Upload the shard's interior (margins poisoned), then fill every margin with
    the library's unpack (received slabs cut from the seeded full domain; zero
    fill at the global boundary). The zero-extended domain over the padded-tile
    box is generated once; the interior and the slabs are slices of it.
    Returns (desc, device tile, geometry, host padded box or None)."""
    from oracle import halo as ohalo
    sg = cases.shard_geom(w, idx)
    out = cases.out_code(w)
    full_h = cases.x_box(w, sg.tile_lo, sg.tile_hi, out, dist)
    lo, hi = sg.g["halo_lo"], sg.g["halo_hi"]
    tile_h = np.full_like(full_h, canary_for(w))
    inner = (slice(None),) + tuple(slice(l, l + e) for l, e in zip(lo, sg.ext)) + (slice(None),)
    tile_h[inner] = full_h[inner]
    tile = dev(tile_h)
    del tile_h
    desc = sc.tile_desc(w.N, w.cin, sg.ext, lo, hi)
    for axis in range(w.nd):
        for side in (0, 1):
            width = lo[axis] if side == 0 else hi[axis]
            if width == 0:
                continue
            if cases.neighbour_exists(w, idx, axis, side):
                b0, b1 = ohalo.face_box(axis, ohalo.margin_rows(axis, side, lo, sg.ext, hi), lo, sg.ext, hi)
                box = (slice(None),) + tuple(slice(a, b) for a, b in zip(b0, b1)) + (slice(None),)
                slab = dev(np.ascontiguousarray(full_h[box]))
                sc.shard_halo_unpack(desc, tile, axis, side, slab)
                del slab
            else:
                sc.shard_halo_unpack(desc, tile, axis, side, None)
    return desc, tile, sg, (full_h if keep_host else None)


def run_fwd(sc, w, desc, tile, sg, wt):
    import torch
    O = sg.g["out_ext"]
    y = empty_like_dtype([w.N] + list(O) + [w.cout], w)
    code = sc.SHARD_F32 if w.dtype == "f32" else sc.SHARD_BF16
    nbytes = sc.shard_conv_workspace_bytes(0, desc, code, w.cout, w.K, w.S, O)
    ws = torch.empty(max(nbytes, 16), dtype=torch.uint8, device="cuda")
    sc.shard_conv_fwd(desc, tile, wt, w.cout, w.K, w.S, sg.g["pad_lo"], O, y, ws)
    return y


def run_wgrad(sc, w, desc, tile, sg, dy):
    import torch
    O = sg.g["out_ext"]
    dw = torch.empty((w.cout, w.cin) + tuple(w.K), dtype=torch.float32, device="cuda")
    code = sc.SHARD_F32 if w.dtype == "f32" else sc.SHARD_BF16
    nbytes = sc.shard_conv_workspace_bytes(1, desc, code, w.cout, w.K, w.S, O)
    ws = torch.empty(max(nbytes, 16), dtype=torch.uint8, device="cuda")
    sc.shard_conv_wgrad(desc, tile, dy, w.cout, w.K, w.S, sg.g["pad_lo"], O, dw, ws)
    # the call's status word (first word of the workspace): 0 unless a bounded
    # wait inside the kernel gave up
    assert int(ws[:4].view(torch.int32).item()) == 0, "weight gradient reported a wait that gave up"
    return dw


def weights(w, dist=None):
    logical = w.weights_host(dist)               # [co][ci][k...]
    return logical, cases.as_f64(logical, w)


def dy_box(w, sg, dist=None):
    lo, hi = cases.owned_box(sg)
    f = cases.field(w, "dy", dist)
    return f.box((0, 0, *lo), (w.N, w.cout, *hi), out=cases.out_code(w))


def window_from_tile(w, sg, tile_cl, planes_in=None):
    """Logical float64 oracle window sliced from a host padded tile (channels-last),
    grown with zeros by P on unsharded axes (outside the domain)."""
    pads = [(0, 0)]
    for a in range(w.nd):
        p = 0 if sg.sharded[a] else (w.K[a] - 1) // 2
        pads.append((p, p))
    pads.append((0, 0))
    t64 = cases.as_f64(tile_cl if planes_in is None else tile_cl[:, planes_in[0]:planes_in[1]], w)
    t64 = np.pad(t64, pads)
    origin = [sg.tile_lo[a] - pads[1 + a][0] for a in range(w.nd)]
    if planes_in is not None:
        origin[0] = sg.tile_lo[0] + planes_in[0]
    return cases.to_ncdhw(t64), origin
