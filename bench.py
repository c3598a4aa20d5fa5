"""Benchmark: exact tokenization of 1M-character requests on one MI355X.

    python bench.py [--gpus 1] [--steps K] [--warmup W] [--config 3|4] [--no-cpu] [--calibrate-copy]

A step is one full-request tokenization (pre-tokenization, BPE, compaction)
of one distinct seeded 1,000,000-character sample whose bytes are already in
HBM; the IDs stay in HBM.  W warm-up requests use other samples.  The K timed
requests run back to back between two stream synchronisations:
value = K * 1e6 chars / elapsed.  During the timed region the library records
HIP events between its stages on the same stream; their average gives the
duration of the dominant kernel (the tile kernel) for the roofline.
Per-request latencies (enqueue to completion, input in HBM) give P50/P90/P99
in a second pass; the host-to-host latency through ``tt_encode`` (PCIe copies
included), a steady-state P50 (100 re-encodes of one sample), the P50 of the
same requests with span export (IDs plus byte and character spans, device
resident), the P50 of all timed samples joined into one request (many tiles
per resident slot: the throughput with the chip full) and the host-to-host
time of a 64 x 16,384-char document batch are reported separately, and so
are the append latency of incremental-repair sessions at 100,000 and
1,000,000 characters and the latency of the two front-end options
(ignore_merges, added-token literals) and of the o200k-style and
DeepSeek-style patterns.  The CPU oracle is timed on the same timed samples,
one thread pinned to one core, and its IDs are compared with the GPU's.

``--calibrate-copy`` first runs a plain int32 copy kernel of 64 MiB read +
64 MiB written, so that a hardware-counter profile of this command can scale
the tile kernel's FETCH_SIZE / WRITE_SIZE to bytes.

Prints one JSON line.
"""

import argparse
import hashlib
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

HBM_PEAK_GBS = 8000.0
TRAFFIC_FILE = os.path.join(ROOT, "profiles", "tile_kernel_traffic.json")
CSRC = os.path.join(ROOT, "paper_2607_29678_amd", "csrc")


def percentile(xs, q):
    xs = sorted(xs)
    if not xs:
        return None
    k = (len(xs) - 1) * q / 100.0
    lo = int(k)
    hi = min(lo + 1, len(xs) - 1)
    return xs[lo] + (xs[hi] - xs[lo]) * (k - lo)


def kernel_source_sha():
    """SHA-256 over the library sources (the counters are void once these change)."""
    h = hashlib.sha256()
    for name in sorted(os.listdir(CSRC)):
        if name.endswith((".hip", ".h", ".inc")):
            with open(os.path.join(CSRC, name), "rb") as f:
                h.update(name.encode() + b"\0" + f.read())
    return h.hexdigest()


def measured_traffic(config):
    """HBM bytes per tile-kernel launch from the committed counter profile, if still valid."""
    try:
        with open(TRAFFIC_FILE) as f:
            rec = json.load(f)
    except (OSError, ValueError):
        return None
    if rec.get("source_sha256") != kernel_source_sha() or rec.get("config") != config:
        return None
    return rec.get("traffic_bytes_per_launch")


def incremental_repair(tok, k, sid, n_appends=24):
    """Append latency of a session (window re-tokenization and splice, host to
    host) against re-tokenizing the whole text through tt_encode, at two
    context sizes; appends are seeded lognormal sizes around 1,500 characters
    (the paper's median append), cut from a separate sample."""
    import random

    import numpy as np

    from paper_2607_29678_amd import Session
    from workloads import textgen

    feed = textgen.latency_sample(k, 30)
    rows = []
    for ctx_chars, ctx_seed in ((100_000, 28), (1_000_000, 29)):
        base = textgen.latency_sample(k, ctx_seed)[:ctx_chars]
        rng = random.Random(0xA5 + ctx_chars)
        sess = Session(tok)
        sess.append(base.encode("utf-8"), sid)
        text = base.encode("utf-8")
        pos = 0
        rep, full, sizes, first, fallbacks, same = [], [], [], 0, 0, True
        for _ in range(n_appends):
            n = max(1, min(20000, int(rng.lognormvariate(np.log(1500.0), 0.8))))
            piece = feed[pos:pos + n].encode("utf-8")
            pos += n
            a = time.perf_counter()
            info = sess.append(piece, sid)
            rep.append((time.perf_counter() - a) * 1e3)
            text += piece
            a = time.perf_counter()
            want = tok.encode(text, sid)
            full.append((time.perf_counter() - a) * 1e3)
            sizes.append(n)
            first += info["windows"] == 1 and not info["full"]
            fallbacks += info["full"]
            same &= np.array_equal(sess.ids(), want)
        sess.close()
        rows.append({"ctx_chars": ctx_chars, "appends": n_appends, "append_chars_p50": int(percentile(sizes, 50)),
                     "repair_p50_ms": round(percentile(rep, 50), 4), "repair_p90_ms": round(percentile(rep, 90), 4),
                     "full_reencode_p50_ms": round(percentile(full, 50), 4),
                     "first_window_admitted": int(first), "full_fallbacks": int(fallbacks),
                     "ids_identical_to_full_encode": bool(same)})
    return {"window_chars": 512, "shapes": rows,
            "context": {"paper_repair_p50_ms_1M": 1.23, "paper_hardware": "CPU session store (Qwen3 real text)"}}


def front_end_options(sid, n=10):
    """ignore_merges and added tokens (Sec. 4.2, Sec. 4.5) on 1,000,000-character
    requests.  ignore_merges: the multilingual samples with the cl100k-style
    table, device-resident P50 with and without the option.  Added tokens: the
    transcript samples with a chat-template literal before every turn (about
    one per 1,400 characters), host to host through tt_encode, against the same
    text on a handle without literals."""
    import numpy as np
    import torch

    from paper_2607_29678_amd import Tokenizer
    from workloads import textgen
    from workloads.tables import load_table

    dev = torch.device("cuda:0")
    stream = torch.cuda.current_stream(dev)
    out = {}
    m, vb, vo = load_table(4)
    texts = [textgen.latency_sample(4, s).encode("utf-8") for s in range(n)]
    d_in = [torch.from_numpy(np.frombuffer(t, dtype=np.uint8).copy()).to(dev) for t in texts]
    d_out = torch.empty(max(len(t) for t in texts), dtype=torch.int32, device=dev)
    d_len = torch.zeros(1, dtype=torch.int64, device=dev)
    for ignore in (False, True):
        tok = Tokenizer(m, vb, vo, "cl100k", ignore_merges=ignore)
        lat = []
        for i in range(n + 2):
            j = i % n
            torch.cuda.synchronize()
            a = time.perf_counter()
            tok.encode_device(d_in[j], len(texts[j]), d_out, d_len, sid)
            stream.synchronize()
            if i >= 2:
                lat.append((time.perf_counter() - a) * 1e3)
        out["ignore_merges" if ignore else "plain"] = round(percentile(lat, 50), 4)
        tok.close()
    ign = {"workload": "C4 samples (1,000,000 chars, cl100k-style, 100,000 merges)", "p50_ms_plain": out["plain"],
           "p50_ms_ignore_merges": out["ignore_merges"]}

    m, vb, vo = load_table(3)
    lits = [("<|im_start|>", 50300), ("<|im_end|>", 50301), ("<|endoftext|>", 50302)]
    texts = []
    for s in range(n):
        t = textgen.latency_sample(3, s)
        parts, pos, k = [], 0, 0
        while pos < len(t):
            parts.append(lits[k % 2][0] + t[pos:pos + 1400])
            pos += 1400
            k += 1
        texts.append("".join(parts).encode("utf-8"))
    res = {}
    for name, added in (("no_literals", None), ("literals", lits)):
        tok = Tokenizer(m, vb, vo, "gpt2", added=added)
        tok.encode(texts[0], sid)
        lat = []
        for t in texts:
            a = time.perf_counter()
            tok.encode(t, sid)
            lat.append((time.perf_counter() - a) * 1e3)
        res[name] = round(percentile(lat, 50), 4)
        tok.close()
    lit = {"workload": "C3 samples with a literal before every 1,400 characters (%d literals, %d bytes)"
                       % (len(texts[0].split(b"<|im_")) - 1, len(texts[0])),
           "host_to_host_p50_ms_literal_handle": res["literals"],
           "host_to_host_p50_ms_same_text_plain_handle": res["no_literals"]}
    # the o200k-style and DeepSeek-style patterns (no table of their own: the
    # multilingual table serves them), against cl100k-style on the same
    # samples and table
    m, vb, vo = load_table(4)
    o2 = {}
    for k in (3, 4):
        texts = [textgen.latency_sample(k, s).encode("utf-8") for s in range(n)]
        d_in = [torch.from_numpy(np.frombuffer(t, dtype=np.uint8).copy()).to(dev) for t in texts]
        d_out = torch.empty(max(len(t) for t in texts), dtype=torch.int32, device=dev)
        row = {}
        for pat in ("cl100k", "o200k", "deepseek"):
            tok = Tokenizer(m, vb, vo, pat)
            lat = []
            for i in range(n + 2):
                j = i % n
                torch.cuda.synchronize()
                a = time.perf_counter()
                tok.encode_device(d_in[j], len(texts[j]), d_out, d_len, sid)
                stream.synchronize()
                if i >= 2:
                    lat.append((time.perf_counter() - a) * 1e3)
            row["p50_ms_" + pat] = round(percentile(lat, 50), 4)
            tok.close()
        o2["C%d_samples" % k] = row
    o2["table"] = "C4 (100,000 merges)"
    return {"ignore_merges": ign, "added_tokens": lit, "other_patterns": o2}


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--config", type=int, default=3, choices=(3, 4))
    ap.add_argument("--no-cpu", action="store_true", help="skip the CPU oracle baseline")
    ap.add_argument("--calibrate-copy", action="store_true", help="run the counter-calibration copy kernel first")
    args = ap.parse_args()
    if args.gpus != 1:
        print("bench.py measures one GPU only: the tokenizer runs on a single MI355X "
              "(--gpus %d requested)" % args.gpus, file=sys.stderr)
        sys.exit(2)

    import numpy as np
    import torch

    from paper_2607_29678_amd import Tokenizer
    from workloads import textgen
    from workloads.tables import load_table

    k = args.config
    cfg = textgen.CONFIGS[k]
    merges, vb, vo = load_table(k)
    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    stream = torch.cuda.current_stream(dev)
    sid = stream.cuda_stream
    tok = Tokenizer(merges, vb, vo, cfg["pattern"])

    if args.calibrate_copy:
        src = torch.arange(16 << 20, dtype=torch.int32, device=dev)
        dst = torch.empty_like(src)
        torch.add(src, 0, out=dst)  # reads 64 MiB, writes 64 MiB
        torch.cuda.synchronize()
        del src, dst

    # seeded samples: warm-up samples are distinct from the timed ones
    n_total = args.warmup + args.steps
    texts = [textgen.latency_sample(k, s % 32).encode("utf-8") for s in range(n_total)]
    d_in = [torch.from_numpy(np.frombuffer(t, dtype=np.uint8).copy()).to(dev) for t in texts]
    cap = max(len(t) for t in texts)
    d_out = torch.empty((len(texts), cap), dtype=torch.int32, device=dev)
    d_len = torch.zeros(len(texts), dtype=torch.int64, device=dev)
    n_chars = [len(t.decode("utf-8")) for t in texts]
    torch.cuda.synchronize()

    def run(i):
        tok.encode_device(d_in[i], len(texts[i]), d_out[i], d_len[i:i + 1], sid)

    for i in range(args.warmup):
        run(i)
    torch.cuda.synchronize()

    # --- timed region: K requests back to back, stage events recorded -------
    timed = list(range(args.warmup, n_total))
    tok.set_profiling(len(timed))
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for i in timed:
        run(i)
    torch.cuda.synchronize()
    elapsed = time.perf_counter() - t0
    stage_calls = tok.stage_times(sid)
    tok.set_profiling(0)
    chars = sum(n_chars[i] for i in timed)
    value = chars / elapsed
    lens = d_len.cpu().numpy()
    if (lens[timed] <= 0).any():
        raise SystemExit("tokenizer reported an error: %s" % lens[timed])
    stage_avg = {s: sum(c[s] for c in stage_calls) / len(stage_calls) for s in stage_calls[0]}

    # --- per-request latency (enqueue to completion, input in HBM) -----------
    lat = []
    for i in timed:
        torch.cuda.synchronize()
        a = time.perf_counter()
        run(i)
        stream.synchronize()
        lat.append((time.perf_counter() - a) * 1e3)

    # --- host-to-host latency through tt_encode (PCIe copies included) --------
    host_lat = []
    for i in timed[: min(10, len(timed))]:
        a = time.perf_counter()
        tok.encode(texts[i], sid)
        host_lat.append((time.perf_counter() - a) * 1e3)

    # --- steady state: 100 re-encodes of one sample (input in HBM) --------------
    steady = []
    for _ in range(100):
        torch.cuda.synchronize()
        a = time.perf_counter()
        run(timed[0])
        stream.synchronize()
        steady.append((time.perf_counter() - a) * 1e3)

    # --- span export: IDs with byte and character spans (device-resident) -----
    d_spans = torch.empty((cap, 4), dtype=torch.int32, device=dev)
    d_sids = torch.empty(cap, dtype=torch.int32, device=dev)
    d_slen = torch.zeros(1, dtype=torch.int64, device=dev)
    span_lat = []
    for i in timed:
        torch.cuda.synchronize()
        a = time.perf_counter()
        tok.encode_spans_device(d_in[i], len(texts[i]), d_sids, d_spans, d_slen, sid)
        stream.synchronize()
        span_lat.append((time.perf_counter() - a) * 1e3)
    if int(d_slen.item()) != int(lens[timed[-1]]):
        raise SystemExit("span export returned a different token count")

    # --- shape of the work: pieces of one sample (split-level export) ----------
    starts = tok.pretokenize(texts[timed[0]], sid)
    n_pieces = len(starts)
    longest_piece = int(np.max(np.diff(np.append(starts, len(texts[timed[0]]))))) if n_pieces else 0

    # --- throughput with the chip full: the timed samples as one request -------
    # (a 1,000,000-char request fills about two thirds of the resident tile
    # slots once, so its time is one tile's latency; a request of all timed
    # samples runs many tiles per slot)
    big = b"".join(texts[i] for i in timed)
    d_big = torch.from_numpy(np.frombuffer(big, dtype=np.uint8).copy()).to(dev)
    d_bout = torch.empty(len(big), dtype=torch.int32, device=dev)
    d_blen = torch.zeros(1, dtype=torch.int64, device=dev)
    tok.encode_device(d_big, len(big), d_bout, d_blen, sid)
    torch.cuda.synchronize()
    big_lat = []
    for _ in range(10):
        a = time.perf_counter()
        tok.encode_device(d_big, len(big), d_bout, d_blen, sid)
        stream.synchronize()
        big_lat.append((time.perf_counter() - a) * 1e3)
    big_T = int(d_blen.item())
    if big_T <= 0:
        raise SystemExit("tokenizer reported an error on the joined request: %d" % big_T)
    big_chars = sum(n_chars[i] for i in timed)
    big_ms = percentile(big_lat, 50)
    large_request = {"chars": big_chars, "bytes": len(big), "tokens": big_T, "p50_ms": round(big_ms, 4),
                     "chars_per_s": round(big_chars / (big_ms * 1e-3), 1),
                     "hbm_frac": round((len(big) + 4.0 * big_T) / (big_ms * 1e-3) / 1e9 / HBM_PEAK_GBS, 6)}
    del d_big, d_bout

    # --- a batch of 64 independent 16,384-char documents (the stress config's
    # batch, its own tokenizer), host to host through tt_encode_batch -----------
    bmerges, bvb, bvo = load_table(5)
    btok = Tokenizer(bmerges, bvb, bvo, textgen.CONFIGS[5]["pattern"])
    docs = [d.encode("utf-8") for d in textgen.batch_docs()]
    btok.encode_batch(docs, sid)
    blat = []
    for _ in range(10):
        a = time.perf_counter()
        btok.encode_batch(docs, sid)
        blat.append((time.perf_counter() - a) * 1e3)
    bchars = sum(len(d.decode("utf-8")) for d in docs)
    batch = {"docs": len(docs), "chars": bchars, "bytes": sum(len(d) for d in docs),
             "p50_ms_host_to_host": round(percentile(blat, 50), 4),
             "chars_per_s": round(bchars / (percentile(blat, 50) * 1e-3), 1)}
    btok.close()

    # --- incremental repair: appends to a stored session (Sec. 3.2) ------------
    repair = incremental_repair(tok, k, sid)

    # --- front-end options: ignore_merges and added-token literals ----------------
    options = front_end_options(sid)

    # --- roofline of the dominant kernel -------------------------------------
    # algorithmic bytes of one tile-kernel launch: the request's bytes are
    # read once and its token IDs written once (merge-table probes are L2
    # traffic, not HBM traffic, for tables of a few MB)
    B_avg = sum(len(texts[i]) for i in timed) / len(timed)
    T_avg = float(np.mean(lens[timed]))
    tile_ms = stage_avg["tile"]
    alg = B_avg + 4.0 * T_avg
    achieved = alg / (tile_ms * 1e-3) / 1e9
    roofline = {"kernel": "tile_kernel", "bound": "hbm", "achieved": round(achieved, 2), "peak": HBM_PEAK_GBS,
                "unit": "GB/s", "frac": round(achieved / HBM_PEAK_GBS, 6),
                "traffic": measured_traffic(k), "algorithmic_bytes": int(alg),
                "kernel_ms": round(tile_ms, 4)}

    # --- CPU oracle baseline on the timed samples --------------------------------
    cpu = None
    if not args.no_cpu:
        from oracle.bpe import MergeTable
        from oracle.tokenizer import encode as oracle_encode
        from workloads.tables import vocab_list

        table = MergeTable(merges.tolist(), vocab_list(vb, vo))
        host_ids = d_out.cpu().numpy()
        same = True
        dt = 0.0
        # one process pinned to one core, timing the tokenize call only
        affinity = os.sched_getaffinity(0)
        core = min(affinity)
        os.sched_setaffinity(0, {core})
        try:
            for i in timed:
                a = time.perf_counter()
                ids = oracle_encode(texts[i], table, cfg["pattern"])
                dt += time.perf_counter() - a
                same &= host_ids[i, : int(lens[i])].tolist() == ids
        finally:
            os.sched_setaffinity(0, affinity)
        model = ""
        try:
            with open("/proc/cpuinfo") as f:
                model = next((ln.split(":", 1)[1].strip() for ln in f if ln.startswith("model name")), "")
        except OSError:
            pass
        cpu = {"value": round(sum(n_chars[i] for i in timed) / dt, 1), "unit": "chars/s", "cores": 1,
               "kind": "oracle",
               "sample": "the %d timed 1,000,000-char samples, one after another, one thread pinned to core %d, "
                         "pure Python" % (len(timed), core),
               "seconds": round(dt, 2), "ids_identical_to_gpu": bool(same),
               "host": {"cpu_model": model, "cores_visible": len(affinity), "python": sys.version.split()[0]}}

    out = {
        "metric": "exact-tokenization chars/sec and P50 latency for a 1M-char request, 1 MI355X",
        "value": round(value, 1),
        "unit": "chars/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(elapsed * 1e3 / len(timed), 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "int32",
        "data": "synthetic",
        "config": {"workload": "C%d: 1,000,000-char seeded %s request, %s-style pattern, %d merges"
                               % (k, "agent-transcript" if k == 3 else "multilingual agent-transcript",
                                  cfg["pattern"], cfg["merges"]),
                   "chars": 1_000_000, "bytes_avg": int(B_avg), "tokens_avg": int(T_avg), "samples": len(timed),
                   "pieces_sample0": n_pieces, "longest_piece_bytes_sample0": longest_piece},
        "p50_ms": round(percentile(lat, 50), 4),
        "p90_ms": round(percentile(lat, 90), 4),
        "p99_ms": round(percentile(lat, 99), 4),
        "host_to_host_p50_ms": round(percentile(host_lat, 50), 4),
        "steady_state_p50_ms": round(percentile(steady, 50), 4),
        "span_export_p50_ms": round(percentile(span_lat, 50), 4),
        "large_request": large_request,
        "batch_64x16k": batch,
        "incremental_repair": repair,
        "front_end_options": options,
        "stage_ms": {s: round(v, 4) for s, v in stage_avg.items()},
        "roofline": roofline,
        "cpu_baseline": cpu,
        "context": {"paper_p50_ms_1M_chars": 0.87, "paper_hardware": "RTX PRO 6000 Blackwell (Qwen3 real text)"},
    }
    print(json.dumps(out))


if __name__ == "__main__":
    main()
