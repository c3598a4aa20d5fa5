"""Where a tile's time goes: per-phase clock stamps of the tile kernel.

A diagnostic build of the library (``python -m paper_2607_29678_amd._build
--phases``, or ``--build`` here; compile it on the build host, not on the GPU
host) has thread 0 of every tile write the 100 MHz wall clock at each phase
boundary of the tile kernel (the slots are listed in ``csrc/tt_tile.hip``).
This script encodes seeded device-resident requests (``--host``: requests in
pageable host arrays through ``tt_encode``) through that build and prints, per
workload, one JSON line: the mean and maximum time of every phase
over the tiles, the phases of the critical tiles (the last to finish their
placement look-back) and of the tiles that publish their token count last
(which every later tile's placement waits for), when tiles start and publish
their counts (also by the number of tiles on the tile's compute unit), the
split of the dispatch phase and, for the walked patterns, of the predicate
phase.  Times are in microseconds; the kernel time
from HIP events is printed beside the stamps' span.

    python -m paper_2607_29678_amd.phase_timeline --build
    python -m paper_2607_29678_amd.phase_timeline --runs C3:gpt2:3,C4:cl100k:4
"""

import argparse
import ctypes
import json
import os
import sys

import numpy as np

from . import _build, _lib

SLOTS, MAX_TILES, PT_OWN = 32, 8192, 1984
PHASES = ["ticket and tables", "window staging", "decode and classify", "cl100k scan and carries", "predicate",
          "units and dispatch", "thread and wave engines", "block engine", "placement look-back", "writing tokens"]
DISPATCH = ["unit scan", "unit starts listed", "incoming unit and dictionaries", "length lists", "to the engines",
            "incoming unit's start known (after the listing)"]
WALK = ["bitmaps", "extra starts and first wait", "walks", "flags"]
PRED = ["per-position rules (wave 0)", "read past the window, vocabulary probes", "junction cuts (wave 0)",
        "predicate, slowest wave"]


def _summary(rows, names):
    a = np.concatenate(rows)
    return {"mean": {k: round(float(a[:, j].mean()), 2) for j, k in enumerate(names)},
            "max": {k: round(float(a[:, j].max()), 2) for j, k in enumerate(names)}}


def _spread(rows):
    a = np.concatenate(rows)
    return {"p50": round(float(np.percentile(a, 50)), 2), "p90": round(float(np.percentile(a, 90)), 2),
            "max": round(float(a.max()), 2)}


def timeline(workload, pattern, table, samples=8, reps=2, host=False):
    import torch
    from workloads import textgen
    from workloads.tables import load_table
    from .tokenizer import Tokenizer

    lib = _lib.load()
    if not hasattr(lib, "tt_phase_stamps"):
        raise RuntimeError("the loaded library has no phase stamps (not the --phases build)")
    lib.tt_phase_stamps.restype = ctypes.c_int
    lib.tt_phase_stamps.argtypes = [ctypes.c_void_p, ctypes.c_int]
    k = int(workload.lstrip("Cc"))
    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    stream = torch.cuda.current_stream(dev)
    m, vb, vo = load_table(table)
    tok = Tokenizer(m, vb, vo, pattern)
    texts = [textgen.latency_sample(k, s).encode() for s in range(samples)]
    d_in = [torch.from_numpy(np.frombuffer(t, dtype=np.uint8).copy()).to(dev) for t in texts]
    d_out = torch.empty(max(len(t) for t in texts), dtype=torch.int32, device=dev)
    d_len = torch.zeros(1, dtype=torch.int64, device=dev)
    # host delivery: tt_encode from pageable arrays (the kernel reads the request
    # from pinned staging and writes the IDs into pinned memory over the bus)
    h_in = [np.frombuffer(t, dtype=np.uint8).copy() for t in texts]
    h_out = np.empty(max(len(t) for t in texts), dtype=np.int32)

    def call(i):
        if host:
            tok.encode_into(h_in[i], h_out, stream.cuda_stream)
        else:
            tok.encode_device(d_in[i], len(texts[i]), d_out, d_len, stream.cuda_stream)

    for i in range(2):
        call(i)
    torch.cuda.synchronize()
    buf = np.zeros(MAX_TILES * SLOTS, dtype=np.uint64)
    phases, disp, walk, pred, crit, spans, late, starts, counts = [], [], [], [], [], [], [], [], []
    by_cu = {}  # tiles on a compute unit -> times at which such tiles publish their counts
    tok.set_profiling(samples * reps)
    for _ in range(reps):
        for i, t in enumerate(texts):
            nt = (len(t) + PT_OWN - 1) // PT_OWN
            assert nt <= MAX_TILES
            call(i)
            stream.synchronize()
            _lib.check(lib.tt_phase_stamps(buf.ctypes.data, nt), "tt_phase_stamps")
            a = buf[: nt * SLOTS].reshape(nt, SLOTS).astype(np.int64)
            rel = (a - a[:, 0].min()) * 0.01  # 100 MHz ticks -> microseconds
            phases.append(np.diff(rel[:, :11], axis=1))
            inc = np.where(a[:, 20] > 0, rel[:, 20] - rel[:, 12], 0.0)  # (0: no incoming unit)
            disp.append(np.stack([rel[:, 11] - rel[:, 5], rel[:, 12] - rel[:, 11], rel[:, 13] - rel[:, 12],
                                  rel[:, 14] - rel[:, 13], rel[:, 6] - rel[:, 14], inc], axis=1))
            pred.append(np.stack([rel[:, 21] - rel[:, 4], rel[:, 22] - rel[:, 21], rel[:, 5] - rel[:, 22],
                                  rel[:, 24:32].max(axis=1) - rel[:, 4]], axis=1))
            if pattern in ("o200k", "deepseek"):
                walk.append(np.stack([rel[:, 16] - rel[:, 4], rel[:, 17] - rel[:, 16], rel[:, 18] - rel[:, 17],
                                      rel[:, 19] - rel[:, 18]], axis=1))
            c = int(np.argmax(rel[:, 9]))
            crit.append({"tile": c, "of": nt, "phases": [round(float(x), 2) for x in phases[-1][c]]})
            # the tile whose count is published last (the end of its engines):
            # every later tile's placement waits for it
            # the compute unit of each tile (XCD, then bits 8-15 of the hardware
            # ID: unit, shader array, engine) and how many tiles it holds
            cu = (a[:, 15] >> 32) * 256 + ((a[:, 15] >> 8) & 255)
            _, inv, per = np.unique(cu, return_inverse=True, return_counts=True)
            on_cu = per[inv]
            for k in np.unique(on_cu):
                by_cu.setdefault(int(k), []).append(rel[on_cu == k, 8])
            b = int(np.argmax(rel[:, 8]))
            late.append({"tile": b, "of": nt, "starts_at": round(float(rel[b, 0]), 2),
                         "count_at": round(float(rel[b, 8]), 2),
                         "phases": [round(float(x), 2) for x in phases[-1][b]],
                         "incoming_start_wait": round(float(inc[b]), 2), "tiles_on_its_unit": int(on_cu[b])})
            starts.append(rel[:, 0])
            counts.append(rel[:, 8])
            spans.append(float(rel[:, 10].max()))
    kernel_us = [x["tile"] * 1e3 for x in tok.stage_times(stream.cuda_stream)]
    tok.set_profiling(0)
    tok.close()
    out = {"workload": workload, "pattern": pattern, "table": table, "calls": samples * reps,
           "delivery": "tt_encode from pageable host arrays" if host else "device-resident (tt_encode_device)",
           "kernel_us_p50_hip_events": round(float(np.median(kernel_us)), 2),
           "stamp_span_us_p50": round(float(np.median(spans)), 2),
           "phases": _summary(phases, PHASES), "dispatch": _summary(disp, DISPATCH),
           "predicate_split": _summary(pred, PRED),
           "critical_tiles": crit[:4],
           "tile_start_us": _spread(starts), "count_published_us": _spread(counts),
           "last_count_tiles": late[:4],
           "count_published_us_by_tiles_on_unit": {str(k): dict(_spread(v), tiles=int(sum(len(x) for x in v)))
                                                   for k, v in sorted(by_cu.items())}}
    if walk:
        out["walked_predicate"] = _summary(walk, WALK)
    return out


def main(argv=None):
    ap = argparse.ArgumentParser(description=__doc__.split("\n\n")[0])
    ap.add_argument("--build", action="store_true", help="compile the phase-stamp build and exit")
    ap.add_argument("--runs", default="C3:gpt2:3,C4:cl100k:4",
                    help="comma-separated WORKLOAD:PATTERN:TABLE (tables as in workloads.tables)")
    ap.add_argument("--samples", type=int, default=8)
    ap.add_argument("--host", action="store_true", help="time tt_encode from host arrays instead of device-resident calls")
    args = ap.parse_args(argv)
    if args.build:
        print(_build.build(verbose=True, phases=True))
        return 0
    if not os.path.exists(_build.PHASES_LIB):
        raise SystemExit("the phase-stamp build is missing: run with --build first (on the build host)")
    _lib.LIB_PATH = _build.PHASES_LIB  # this process loads the diagnostic build instead of the product
    for run in args.runs.split(","):
        w, p, t = run.split(":")
        print(json.dumps(timeline(w, p, int(t), samples=args.samples, host=args.host)), flush=True)
    return 0


if __name__ == "__main__":
    sys.exit(main())
