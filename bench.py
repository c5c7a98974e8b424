#!/usr/bin/env python3
"""Benchmark: the PULSESync patch codec over a whole synthetic parameter set on one MI355X.

One step = one pass of the hot path over every tensor of the parameter set
(default: the 32B-shaped set, 32,763,417,600 FP32 parameters in 579 tensors):
the fused encode, which casts the FP32 masters to BF16 (RNE), compares them
bitwise with the previous BF16 snapshot, compacts the changed positions into
an index-ordered (uint32 index, bf16 value) patch with its device-side count,
and writes the changed values into the inference-side BF16 copy in the same
pass.  That step is the headline.

Also measured, outside the headline: the unfused form (encode, then the
standalone scatter apply of the patch into the inference copy) and the
PULSELoCo rounds over the 7B-shaped set (10 rounds, fixed threshold): the
error-feedback sparsification and the outer step that consumes its patch;
the patch's delta-varint index stream; and the weight hash (a SHA-256 tree)
of the refreshed inference copy that a receiver checks.  All inputs are
generated on the GPU before timing and stay resident in HBM.

Prints ONE JSON line on stdout; progress goes to stderr.

    python bench.py [--steps K] [--warmup W] [--workload 32b|7b|0.5b] [--no-cpu-baseline] [--no-loco]
"""
from __future__ import annotations

import argparse
import json
import os
import platform
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

METRIC = "encode+apply GB/s of weights scanned, % of MI355X HBM peak; patch density"
HBM_PEAK_GBS = 8000.0
WORKLOAD_IDS = {"0.5b": 2, "7b": 3, "32b": 4}
CHUNK = 64  # tensors per launch (the library's batch limit)
TRAFFIC_FILE = os.path.join(ROOT, "profiles", "encode_fused_32b_traffic.txt")
CALIB_WORDS = 1 << 28  # int32 words of the plain copy kernel run for counter calibration
# Vector-ALU peak for 32-bit integer work: 256 CUs x 4 SIMDs x 16 lanes, one
# operation per lane per clock, at 2.4 GHz (lane-operations per second).
ALU_PEAK_TOPS = 256 * 64 * 2.4e9 / 1e12
# VALU instructions of one SHA-256 compression in the leaf kernel: per round 6
# rotates, 4 three-input bitwise ops (two XOR3, Ch, Maj) and 4 adds; per
# schedule step 4 rotates, 2 shifts, 2 XOR3 and 2 adds; 8 adds into the state;
# 16 byte permutes assembling the message words; 3 of loop control.
SHA_VALU_PER_BLOCK = 64 * 14 + 48 * 10 + 8 + 16 + 3


def log(*a):
    print(*a, file=sys.stderr, flush=True)


def cpu_model() -> str:
    try:
        with open("/proc/cpuinfo") as fh:
            for line in fh:
                if line.startswith("model name"):
                    return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return platform.processor() or "unknown"


class ParamSet:
    """Flat FP32 master, BF16 snapshot and BF16 inference copy, with per-tensor views."""

    def __init__(self, key: str, lr: float, device):
        import torch
        from paper_2602_03839_amd import pulse
        from paper_2602_03839_amd import workloads as wl

        self.key = key
        self.specs = wl.SHAPES[key].tensors()
        self.sizes = [s.numel for s in self.specs]
        self.offsets = []
        o = 0
        for n in self.sizes:
            self.offsets.append(o)
            o += n
        self.N = o
        self.flat_index = self.N < (1 << 32)
        cfg = WORKLOAD_IDS[key]
        free, total = torch.cuda.mem_get_info(device)
        log(f"[bench] {key}: {self.N:,} params in {len(self.specs)} tensors; "
            f"device memory free {free / 1e9:.1f} / {total / 1e9:.1f} GB")
        self.w = torch.empty(self.N, dtype=torch.float32, device=device)
        self.S = torch.empty(self.N, dtype=torch.int16, device=device)
        t0 = time.perf_counter()
        for i, (spec, off, n) in enumerate(zip(self.specs, self.offsets, self.sizes)):
            wv = self.w[off:off + n]
            wl.init_weights_(wv, spec, cfg, 0, i)
            pulse.cast_bf16(wv, out=self.S[off:off + n])
            wl.adam_step_(wv, lr, cfg, 1, i)
            if i % 64 == 0:
                log(f"[bench] generated {i + 1}/{len(self.specs)} tensors")
        torch.cuda.synchronize()
        torch.cuda.empty_cache()
        log(f"[bench] generation {time.perf_counter() - t0:.1f}s")
        self.R = self.S.clone()

    def view(self, buf, i):
        return buf[self.offsets[i]:self.offsets[i] + self.sizes[i]]

    def base(self, i):
        return self.offsets[i] if self.flat_index else 0


def chunks(n, k):
    return [(a, min(a + k, n)) for a in range(0, n, k)]


def event_pair():
    import torch
    return torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)


def main():
    ap = argparse.ArgumentParser(description=__doc__, formatter_class=argparse.RawDescriptionHelpFormatter)
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=10)
    ap.add_argument("--warmup", type=int, default=2)
    ap.add_argument("--workload", default="32b", choices=sorted(WORKLOAD_IDS))
    ap.add_argument("--lr", type=float, default=1e-6)
    ap.add_argument("--capacity-frac", type=float, default=0.05)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--cpu-sample", type=float, default=1.0e9,
                    help="elements of the parameter set the oracle baseline encodes")
    ap.add_argument("--refresh", default="mirror", choices=["mirror", "sparse"],
                    help="fused refresh form: whole 128-byte runs of the inference copy, which mirrors "
                         "the snapshot (mirror), or one 2-byte write per change (sparse)")
    ap.add_argument("--no-loco", action="store_true", help="skip the PULSELoCo leg")
    ap.add_argument("--loco-rounds", type=int, default=10)
    ap.add_argument("--no-varint", action="store_true", help="skip the wire-format (delta-varint) leg")
    ap.add_argument("--no-hash", action="store_true", help="skip the weight-hash leg")
    ap.add_argument("--no-receivers", action="store_true",
                    help="skip the FP8/MXFP4-receiver and k-step legs (7B set)")
    args = ap.parse_args()

    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) != 1:
        print("bench.py measures one GPU only: the patch codec needs no collectives; across GPUs "
              "each rank would run it on its own shard of the tensors, with no cross-GPU traffic.",
              file=sys.stderr)
        sys.exit(2)

    import numpy as np
    import torch
    from paper_2602_03839_amd import pulse

    device = torch.device("cuda:0")
    torch.cuda.set_device(device)
    pulse.lib()
    stream = torch.cuda.current_stream()

    # A plain copy kernel of known size (bitwise_not over 1 GiB of int32 reads
    # 1 GiB and writes 1 GiB), run once so that a counter-collection run of this
    # script can calibrate the HBM byte counters against it.
    calib = torch.empty(CALIB_WORDS, dtype=torch.int32, device=device).random_()
    torch.bitwise_not(calib, out=torch.empty_like(calib))
    torch.cuda.synchronize()
    del calib
    torch.cuda.empty_cache()

    ps = ParamSet(args.workload, args.lr, device)
    T = len(ps.specs)
    cap = int(args.capacity_frac * ps.N)
    idx = torch.empty(cap, dtype=torch.int32, device=device)
    val = torch.empty(cap, dtype=torch.int16, device=device)
    count = torch.zeros(1, dtype=torch.int64, device=device)
    seg = torch.zeros(T, dtype=torch.int64, device=device)
    ws = pulse.workspace(device)
    log(f"[bench] patch capacity {cap:,} entries ({cap * 6 / 1e9:.2f} GB)")

    parts = chunks(T, CHUNK)
    n_launch = len(parts)
    # The inference copy starts as a copy of the snapshot and only ever receives
    # bf16(w') at the positions the step changes, so it equals the snapshot
    # everywhere else: the whole-run refresh (PULSE_REFRESH_MIRRORS_SNAP) applies.
    mirror = args.refresh == "mirror"
    enc_fused = [pulse.EncodeBatch([pulse.EncodeTensor(ps.view(ps.w, i), ps.view(ps.S, i),
                                                       ps.view(ps.R, i), ps.base(i), mirror)
                                    for i in range(a, b)]) for a, b in parts]
    enc_plain = [pulse.EncodeBatch([pulse.EncodeTensor(ps.view(ps.w, i), ps.view(ps.S, i), None, ps.base(i))
                                    for i in range(a, b)]) for a, b in parts]
    app = pulse.ApplyBatch([pulse.ApplyTensor(ps.view(ps.R, i), ps.base(i)) for i in range(T)])

    def encode_pass(batches, ev=None):
        """One pass over all tensors; `ev` = (start, end) HIP events around its launches."""
        count.zero_()
        if ev:
            ev[0].record(stream)
        for (a, _b), b in zip(parts, batches):
            b(idx, val, count, ws, seg_begin=seg[a:])
        if ev:
            ev[1].record(stream)

    def timed_steps(step_fn, make_events):
        for _ in range(args.warmup):
            step_fn(None)
        torch.cuda.synchronize()
        evs = [make_events() for _ in range(args.steps)]
        t0 = time.perf_counter()
        for k in range(args.steps):
            step_fn(evs[k])
        torch.cuda.synchronize()
        return (time.perf_counter() - t0) * 1e3 / args.steps, evs

    # ---- headline: fused encode + refresh of the inference copy.  Events
    # bracket each step's launches (one pair per step: an event between
    # back-to-back launches would itself add a gap); the average launch
    # duration is the bracketed time over the launches of the step.
    fused_ms, fused_ev = timed_steps(lambda ev: encode_pass(enc_fused, ev), event_pair)
    nnz = int(count.item())
    sent = min(nnz, cap)
    if nnz > cap:
        log(f"[bench] WARNING: patch overflow ({nnz:,} > capacity {cap:,})")
    step_kernel_ms = np.array([s.elapsed_time(e) for s, e in fused_ev])
    fused_kernel_ms = float(step_kernel_ms.mean())
    fused_avg_launch_ms = fused_kernel_ms / n_launch
    value = 6.0 * ps.N / (fused_ms * 1e-3) / 1e9
    fused_bytes = 6.0 * ps.N + 8.0 * sent  # FP32 + BF16 read; idx + val + refresh written per entry
    achieved = fused_bytes / n_launch / (fused_avg_launch_ms * 1e-3) / 1e9
    log(f"[bench] fused encode+refresh {fused_ms:.3f} ms/step ({value:.0f} GB/s scanned); "
        f"kernels {fused_kernel_ms:.3f} ms over {n_launch} launches; nnz {nnz:,} density {nnz / ps.N:.4%}")
    seg_fused = seg.clone()
    idx_head = idx[: min(sent, 1 << 24)].clone()
    val_head = val[: min(sent, 1 << 24)].clone()

    # ---- encode, then the standalone scatter apply (receiver side)
    def unfused(ev):
        encode_pass(enc_plain, ev[0] if ev else None)
        if ev:
            ev[1][0].record(stream)
        app(idx, val, seg, count)
        if ev:
            ev[1][1].record(stream)

    unf_ms, unf_ev = timed_steps(unfused, lambda: (event_pair(), event_pair()))
    enc_ms = float(np.mean([ev[0][0].elapsed_time(ev[0][1]) for ev in unf_ev]))
    app_ms = float(np.mean([ev[1][0].elapsed_time(ev[1][1]) for ev in unf_ev]))
    log(f"[bench] encode then apply {unf_ms:.3f} ms/step: encode {enc_ms:.3f} ms, apply {app_ms:.3f} ms")

    # ---- sanity: both forms give the same patch; the inference copy equals bf16(w')
    assert int(count.item()) == nnz, "fused and plain encode disagree on the count"
    assert torch.equal(seg, seg_fused), "fused and plain encode disagree on the segments"
    assert torch.equal(idx[: idx_head.numel()], idx_head) and torch.equal(val[: val_head.numel()], val_head)
    check = pulse.cast_bf16(ps.w[: min(ps.N, 1 << 28)])
    assert torch.equal(check, ps.R[: check.numel()]), "inference copy differs from bf16(w')"
    del check, idx_head, val_head

    # ---- the patch's wire format: delta-varint index stream, encoded and decoded
    varint = None if args.no_varint else varint_leg(args, ps, idx, count, seg, sent, ws, stream)

    # ---- the weight hash a receiver checks after applying the patch
    whash = None if args.no_hash else hash_leg(args, ps, stream)

    cpu = None
    if not args.no_cpu_baseline:
        cpu = cpu_baseline(ps, args.cpu_sample, idx, val, seg, nnz, cap)

    from paper_2602_03839_amd.traffic import read_summary  # noqa: E402
    traffic = read_summary(TRAFFIC_FILE) if args.workload == "32b" else None
    out = {
        "metric": METRIC,
        "value": round(value, 2),
        "unit": "GB/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(fused_ms, 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16",
        "data": "synthetic",
        "config": {
            "workload": f"pulsesync-{args.workload}-shaped fused encode+refresh",
            "params": ps.N,
            "tensors": T,
            "lr": args.lr,
            "nnz": nnz,
            "patch_density": round(nnz / ps.N, 6),
            "hbm_frac_of_peak": round(fused_bytes / (fused_ms * 1e-3) / 1e9 / HBM_PEAK_GBS, 4),
            "index_form": "flat uint32" if ps.flat_index else "per-tensor uint32 + segment offsets",
            "patch_capacity": cap,
            "launches_per_step": n_launch,
        },
        "roofline": {
            "bound": "hbm",
            "kernel": "encode_kernel (refresh form)",
            "achieved": round(achieved, 2),
            "peak": HBM_PEAK_GBS,
            "unit": "GB/s",
            "frac": round(achieved / HBM_PEAK_GBS, 4),
            "traffic": None if traffic is None else round(traffic, 0),
            "bytes_per_launch": fused_bytes / n_launch,
            "avg_launch_ms": round(fused_avg_launch_ms, 5),
        },
        "cpu_baseline": cpu,
        "legs": {
            "varint_patch": varint,
            "weight_hash": whash,
            "encode_then_apply": {
                "ms_per_step": round(unf_ms, 4),
                "GBps_scanned": round(6.0 * ps.N / (unf_ms * 1e-3) / 1e9, 2),
                "encode_ms": round(enc_ms, 4),
                "apply_ms": round(app_ms, 4),
                "hbm_frac_of_peak": round((6.0 * ps.N + 14.0 * sent) / (unf_ms * 1e-3) / 1e9 / HBM_PEAK_GBS, 4),
            },
        },
    }
    del enc_fused, enc_plain, app, idx, val, ps
    torch.cuda.empty_cache()
    if not args.no_loco:
        out["legs"]["loco_7b"] = loco_leg(args, device, stream)
    if not args.no_receivers:
        out["legs"]["receivers_7b"] = receivers_leg(args, device, stream)
    print(json.dumps(out), flush=True)


def varint_leg(args, ps, idx, count, seg, sent, ws, stream):
    """The patch's index stream in the paper's wire format (App. H.2 / F.3): the
    per-tensor segments of the last encode pass, delta-varint encoded and decoded."""
    import numpy as np
    import torch
    from paper_2602_03839_amd import pulse

    # App. F.3 bound per segment: nnz + (N - nnz)/127 bytes; N = tensor length
    segs = seg.cpu().numpy().tolist() + [sent]
    bound = sum((segs[i + 1] - segs[i]) + (n - (segs[i + 1] - segs[i])) // 127
                for i, n in enumerate(ps.sizes))
    out = torch.empty(bound + 64, dtype=torch.uint8, device=idx.device)
    total = torch.zeros(1, dtype=torch.int64, device=idx.device)
    back = torch.empty(sent + 1, dtype=torch.int32, device=idx.device)
    got = torch.zeros(1, dtype=torch.int64, device=idx.device)
    end = torch.tensor([sent], dtype=torch.int64, device=idx.device)
    reps = max(3, args.steps)
    te, td = [], []
    for r in range(reps + 1):
        a, b = event_pair()
        c, d = event_pair()
        a.record(stream)
        pulse.varint_encode(idx, end, out, total, ws, seg_begin=seg, capacity=sent)
        b.record(stream)
        c.record(stream)
        pulse.varint_decode(out, total, back, got, ws, seg_begin=seg)
        d.record(stream)
        d.synchronize()
        if r:
            te.append(a.elapsed_time(b))
            td.append(c.elapsed_time(d))
    nbytes = int(total.item())
    assert nbytes <= bound, (nbytes, bound)
    assert int(got.item()) == sent
    assert torch.equal(back[:sent], idx[:sent]), "varint round trip differs from the patch"
    enc_ms, dec_ms = float(np.median(te)), float(np.median(td))
    coo = coo_leg(args, ps, idx, end, seg, sent, ws, stream)
    enc_bytes = 4.0 * sent + nbytes          # indices read, stream written
    dec_bytes = nbytes + 4.0 * sent * 3      # stream read, differences written, re-read, indices written
    log(f"[bench] varint: {sent:,} indices -> {nbytes / 1e6:.1f} MB ({nbytes / sent:.3f} B/index, "
        f"bound {bound / 1e6:.1f} MB); encode {enc_ms:.3f} ms, decode {dec_ms:.3f} ms")
    del out, back
    return {
        "entries": sent,
        "stream_bytes": nbytes,
        "bytes_per_index": round(nbytes / max(sent, 1), 4),
        "paper_bound_bytes": bound,
        "encode_ms": round(enc_ms, 4),
        "decode_ms": round(dec_ms, 4),
        "encode_GBps_algorithmic": round(enc_bytes / enc_ms / 1e6, 2),
        "decode_GBps_algorithmic": round(dec_bytes / dec_ms / 1e6, 2),
        "kernels": "varint_encode_kernel; varint_gaps_kernel + varint_sums_kernel",
        "coo_downcast": coo,
    }


def coo_leg(args, ps, idx, end, seg, sent, ws, stream):
    """The same patch's indices as the paper's 2-D COO delta downcast (App. H.2
    step 4, App. H.4.1): per tensor the first index, then (uint8 row, uint16
    column) pairs with (255, 0) escapes for row gaps over 255."""
    import numpy as np
    import torch
    from paper_2602_03839_amd import pulse

    dev = idx.device
    T = len(ps.specs)
    if ps.flat_index:  # the 2-D view needs indices local to each tensor
        return None
    cols = torch.tensor([s.shape[-1] for s in ps.specs], dtype=torch.int32, device=dev)
    first = torch.empty(T, dtype=torch.int32, device=dev)
    sp = torch.empty(T, dtype=torch.int64, device=dev)
    total = torch.zeros(1, dtype=torch.int64, device=dev)
    cap_p = sent + sent // 8 + 64 * T
    drow = torch.empty(cap_p, dtype=torch.uint8, device=dev)
    dcol = torch.empty(cap_p, dtype=torch.int16, device=dev)
    times = []
    for r in range(max(3, args.steps) + 1):
        a, b = event_pair()
        a.record(stream)
        pulse.coo_encode(idx, end, seg, cols, first, drow, dcol, sp, total, ws, capacity=sent)
        b.record(stream)
        b.synchronize()
        if r:
            times.append(a.elapsed_time(b))
    P = int(total.item())
    assert P <= cap_p
    esc = int(((drow[:P] == 255) & (dcol[:P] == 0)).sum().item())
    nbytes = 3 * P + 4 * T
    ms = float(np.median(times))
    # decode (the receiver's Upcast + DeltaDecode) and check the round trip
    back = torch.empty(sent + 1, dtype=torch.int32, device=dev)
    npairs = torch.tensor([P], dtype=torch.int64, device=dev)
    td = []
    for r in range(max(3, args.steps) + 1):
        a, b = event_pair()
        a.record(stream)
        pulse.coo_decode(drow[:P], dcol[:P], npairs, seg, sp, cols, first, end, back[:sent], ws)
        b.record(stream)
        b.synchronize()
        if r:
            td.append(a.elapsed_time(b))
    assert torch.equal(back[:sent], idx[:sent]), "COO round trip differs from the patch"
    ms_d = float(np.median(td))
    del back
    log(f"[bench] coo downcast: {sent:,} indices -> {P:,} pairs ({esc:,} escapes), "
        f"{nbytes / 1e6:.1f} MB ({nbytes / max(sent, 1):.3f} B/index); encode {ms:.3f} ms, "
        f"decode {ms_d:.3f} ms")
    return {"pairs": P, "escapes": esc, "stream_bytes": nbytes,
            "bytes_per_index": round(nbytes / max(sent, 1), 4), "encode_ms": round(ms, 4),
            "decode_ms": round(ms_d, 4),
            "encode_GBps_algorithmic": round((4.0 * sent + nbytes) / ms / 1e6, 2),
            "kernels": "coo_encode_kernel; coo_decode_kernel"}


def hash_leg(args, ps, stream):
    """Weight hash (App. J.4) of the refreshed BF16 inference copy: a SHA-256 tree
    over 16 KiB chunks of its bytes, the check a receiver runs after a patch."""
    import numpy as np
    import torch
    from paper_2602_03839_amd import pulse

    batch = pulse.HashBatch([ps.view(ps.R, i) for i in range(len(ps.specs))])
    reps = max(3, args.steps)
    times, roots = [], set()
    for r in range(reps + 1):
        a, b = event_pair()
        a.record(stream)
        batch(stream)
        b.record(stream)
        b.synchronize()
        roots.add(bytes(batch.root.cpu().numpy()))
        if r:
            times.append(a.elapsed_time(b))
    assert len(roots) == 1, "the weight hash changed between calls on unchanged weights"
    ms = float(np.median(times))
    blocks = batch.nleaves * ((pulse.HASH_LEAF_BYTES + 1 + 1 + 8 + 63) // 64)
    tops = blocks * SHA_VALU_PER_BLOCK / (ms * 1e-3) / 1e12
    log(f"[bench] weight hash: {batch.nleaves:,} leaves of 16 KiB in {ms:.3f} ms "
        f"({2.0 * ps.N / ms / 1e6:.0f} GB/s of BF16; {tops:.1f} T lane-ops/s = "
        f"{tops / ALU_PEAK_TOPS:.1%} of the vector-ALU peak)")
    nleaves = batch.nleaves
    del batch
    return {
        "leaves": nleaves,
        "root": roots.pop().hex(),
        "ms": round(ms, 4),
        "GBps_bf16_hashed": round(2.0 * ps.N / ms / 1e6, 2),
        "roofline": {"bound": "alu", "achieved": round(tops, 3), "peak": round(ALU_PEAK_TOPS, 3),
                     "unit": "T lane-ops/s", "frac": round(tops / ALU_PEAK_TOPS, 4),
                     "valu_per_64B_block": SHA_VALU_PER_BLOCK},
        "kernels": "hash_setup_kernel + hash_leaf_kernel + hash_tree_kernel (whole call timed)",
    }


def loco_leg(args, device, stream):
    """PULSELoCo rounds over the 7B-shaped set at a fixed threshold: the error-feedback
    sparsification (Alg. 2, one worker) and the outer step that consumes its patch
    (SparseSync average over R = 1 worker, outer Nesterov, mu 0.9, alpha 0.7)."""
    import numpy as np
    import torch
    from paper_2602_03839_amd import pulse
    from paper_2602_03839_amd import workloads as wl

    specs = wl.SHAPES["7b"].tensors()
    sizes = [s.numel for s in specs]
    offs = np.concatenate([[0], np.cumsum(sizes)]).tolist()
    N = offs[-1]
    T = len(sizes)
    tau = wl.loco_tau()
    delta = torch.empty(N, dtype=torch.float32, device=device)
    resid = torch.zeros(N, dtype=torch.float32, device=device)
    theta = torch.empty(N, dtype=torch.float32, device=device).normal_(0.0, 0.02 ** 0.5)
    mom = torch.zeros(N, dtype=torch.float32, device=device)
    cap = N // 10
    idx = torch.empty(cap, dtype=torch.int32, device=device)
    val = torch.empty(cap, dtype=torch.float32, device=device)
    count = torch.zeros(1, dtype=torch.int64, device=device)
    seg = torch.zeros(T, dtype=torch.int64, device=device)
    ws = pulse.workspace(device)
    parts = chunks(T, CHUNK)
    view = lambda b, i: b[offs[i]:offs[i + 1]]
    batches = [pulse.LocoBatch([pulse.LocoTensor(view(delta, i), view(resid, i), None, 0)
                                for i in range(a, b)]) for a, b in parts]
    outer = pulse.OuterBatch([pulse.OuterTensor(view(theta, i), view(mom, i), 0) for i in range(T)])
    lists = [pulse.SparseList(idx, val, seg, count, capacity=cap)]
    ms, ms_outer, dens = [], [], []
    for r in range(args.loco_rounds):
        for i in range(T):
            wl.loco_delta_(view(delta, i), 5, r, i)
        count.zero_()
        torch.cuda.synchronize()
        a, e = event_pair()
        c, d = event_pair()
        a.record(stream)
        for (t0, _t1), b in zip(parts, batches):
            b(tau, idx, val, count, ws, seg_begin=seg[t0:])
        e.record(stream)
        c.record(stream)
        outer(lists, mu=0.9, alpha=0.7)
        d.record(stream)
        d.synchronize()
        ms.append(a.elapsed_time(e))
        ms_outer.append(c.elapsed_time(d))
        dens.append(int(count.item()) / N)
    skip = 1 if len(ms) > 1 else 0
    med = float(np.median(ms[skip:]))
    med_outer = float(np.median(ms_outer[skip:]))
    nnz_mean = float(np.mean(dens[skip:])) * N
    outer_bytes = 16.0 * N + 8.0 * nnz_mean
    log(f"[bench] loco 7b: sparsify median {med:.3f} ms/round ({12.0 * N / med / 1e6:.0f} GB/s at 12 B/param); "
        f"outer step median {med_outer:.3f} ms ({outer_bytes / med_outer / 1e6:.0f} GB/s); "
        f"density {dens[0]:.4%} -> {dens[-1]:.4%}")
    return {
        "params": N,
        "tau": tau,
        "rounds": args.loco_rounds,
        "ms_per_round_median": round(med, 4),
        "GBps_12B_per_param": round(12.0 * N / med / 1e6, 2),
        "kernel": "loco_kernel (threshold form)",
        "density_first_last": [round(dens[0], 6), round(dens[-1], 6)],
        "outer_step": {
            "kernel": "outer_kernel (SparseSync average over 1 worker + outer Nesterov)",
            "ms_per_round_median": round(med_outer, 4),
            "GBps_algorithmic": round(outer_bytes / med_outer / 1e6, 2),
            "hbm_frac_of_peak": round(outer_bytes / med_outer / 1e6 / HBM_PEAK_GBS, 4),
            "bytes_per_round": outer_bytes,
        },
        "round_ms_median": round(med + med_outer, 4),
    }


def receivers_leg(args, device, stream):
    """Receivers below BF16 (App. D) and k-step patches (App. A.1) on the 7B-shaped set.

    From w_0 (the workload's init) the leg keeps the BF16 snapshot, the FP8 E4M3
    view (per-tensor scale 448 / max|w_0|) and the MXFP4 view.  After one Adam
    step at the bench lr it times the FP8 and MXFP4 encode against their views
    and the apply of each patch into a receiver copy; then it continues the
    chain and reports the k-step BF16 density against w_0's snapshot for
    k = 1, 8, 16, 32 (the same encode, an older snapshot).
    """
    import numpy as np
    import torch
    from paper_2602_03839_amd import pulse
    from paper_2602_03839_amd import workloads as wl

    specs = wl.SHAPES["7b"].tensors()
    sizes = [s.numel for s in specs]
    offs = np.concatenate([[0], np.cumsum(sizes)]).tolist()
    N, T = offs[-1], len(sizes)
    cfg = WORKLOAD_IDS["7b"]
    view = lambda b, i: b[offs[i]:offs[i + 1]]
    mx_offs = [0]
    for n in sizes:  # each tensor's packed codes start 16-byte aligned
        mx_offs.append(mx_offs[-1] + ((n + 1) // 2 + 15) // 16 * 16)
    sc_offs = [0]
    for n in sizes:
        sc_offs.append(sc_offs[-1] + (n + 31) // 32)
    w = torch.empty(N, dtype=torch.float32, device=device)
    S0 = torch.empty(N, dtype=torch.int16, device=device)
    F0 = torch.empty(N, dtype=torch.uint8, device=device)
    Mc = torch.empty(mx_offs[-1], dtype=torch.uint8, device=device)
    Ms = torch.empty(sc_offs[-1], dtype=torch.uint8, device=device)
    inv = []
    for i, spec in enumerate(specs):
        wv = view(w, i)
        wl.init_weights_(wv, spec, cfg, 0, i)
        pulse.cast_bf16(wv, out=view(S0, i))
        inv.append(float(448.0 / float(wv.abs().max().item())))
        pulse.cast_lowp(pulse.FP8_E4M3, wv, inv[i], codes=view(F0, i))
        pulse.cast_lowp(pulse.MXFP4, wv, codes=Mc[mx_offs[i]:mx_offs[i + 1]],
                        scales=Ms[sc_offs[i]:sc_offs[i + 1]])
    for i in range(T):
        wl.adam_step_(view(w, i), args.lr, cfg, 1, i)
    cap = N // 10
    idx = torch.empty(cap, dtype=torch.int32, device=device)
    val8 = torch.empty(cap, dtype=torch.uint8, device=device)
    val16 = torch.empty(cap, dtype=torch.int16, device=device)
    count = torch.zeros(1, dtype=torch.int64, device=device)
    seg = torch.zeros(T, dtype=torch.int64, device=device)
    ws = pulse.workspace(device)
    parts = chunks(T, CHUNK)
    mcv = lambda i: Mc[mx_offs[i]:mx_offs[i + 1]]
    msv = lambda i: Ms[sc_offs[i]:sc_offs[i + 1]]
    enc = {
        "fp8_e4m3": [pulse.EncodeLowpBatch(pulse.FP8_E4M3, [
            pulse.LowpTensor(view(w, i), view(F0, i), None, 0, inv[i]) for i in range(a, b)])
            for a, b in parts],
        "mxfp4": [pulse.EncodeLowpBatch(pulse.MXFP4, [
            pulse.LowpTensor(view(w, i), mcv(i), msv(i), 0) for i in range(a, b)])
            for a, b in parts],
    }
    F1, Mc1, Ms1 = F0.clone(), Mc.clone(), Ms.clone()
    app = {
        "fp8_e4m3": pulse.ApplyLowpBatch(pulse.FP8_E4M3, [
            pulse.LowpApplyTensor(view(F1, i), None, sizes[i], 0) for i in range(T)]),
        "mxfp4": pulse.ApplyLowpBatch(pulse.MXFP4, [
            pulse.LowpApplyTensor(Mc1[mx_offs[i]:mx_offs[i + 1]], Ms1[sc_offs[i]:sc_offs[i + 1]],
                                  sizes[i], 0) for i in range(T)]),
    }
    per_param = {"fp8_e4m3": 5.0, "mxfp4": 4.5 + 1.0 / 32}
    per_entry = {"fp8_e4m3": 5.0, "mxfp4": 6.0}
    out = {"params": N, "lr": args.lr, "scale": "fp8: 448 / max|w_0| per tensor"}
    reps = max(3, args.steps)
    for name, batches in enc.items():
        val = val8 if name == "fp8_e4m3" else val16
        te, ta = [], []
        for r in range(reps + 1):
            count.zero_()
            a, e = event_pair()
            c, d = event_pair()
            a.record(stream)
            for (t0, _t1), b in zip(parts, batches):
                b(idx, val, count, ws, seg_begin=seg[t0:])
            e.record(stream)
            c.record(stream)
            app[name](idx, val, seg, count)
            d.record(stream)
            d.synchronize()
            if r:
                te.append(a.elapsed_time(e))
                ta.append(c.elapsed_time(d))
        nnz = int(count.item())
        assert nnz <= cap, f"{name} patch overflow"
        ms_e, ms_a = float(np.median(te)), float(np.median(ta))
        gbs = (per_param[name] * N + per_entry[name] * nnz) / ms_e / 1e6
        log(f"[bench] {name} receiver 7b: encode {ms_e:.3f} ms ({gbs:.0f} GB/s, "
            f"{gbs / HBM_PEAK_GBS:.1%} of HBM), apply {ms_a:.3f} ms, density {nnz / N:.5%}")
        out[name] = {"encode_ms": round(ms_e, 4), "apply_ms": round(ms_a, 4), "nnz": nnz,
                     "density": round(nnz / N, 7), "encode_GBps_algorithmic": round(gbs, 2),
                     "encode_hbm_frac_of_peak": round(gbs / HBM_PEAK_GBS, 4),
                     "bytes_per_param": per_param[name], "bytes_per_entry": per_entry[name]}
    # the receiver copies now hold cast_D(w_1)
    chk = torch.empty(sizes[0], dtype=torch.uint8, device=device)
    pulse.cast_lowp(pulse.FP8_E4M3, view(w, 0), inv[0], codes=chk)
    assert torch.equal(chk, view(F1, 0)), "FP8 receiver copy differs from the cast"
    del F1, Mc1, Ms1, chk, enc, app

    # k-step: BF16 patches against w_0's snapshot
    plain = [pulse.EncodeBatch([pulse.EncodeTensor(view(w, i), view(S0, i), None, 0)
                                for i in range(a, b)]) for a, b in parts]
    dens, kms = {}, None
    for t in range(1, 33):
        if t > 1:
            for i in range(T):
                wl.adam_step_(view(w, i), args.lr, cfg, t, i)
        if t in (1, 8, 16, 32):
            times = []
            for r in range(3 if t == 32 else 1):
                count.zero_()
                a, e = event_pair()
                a.record(stream)
                for (t0, _t1), b in zip(parts, plain):
                    b(idx, val16, count, ws, seg_begin=seg[t0:])
                e.record(stream)
                e.synchronize()
                times.append(a.elapsed_time(e))
            dens[t] = int(count.item()) / N
            kms = float(np.median(times))
    log(f"[bench] k-step BF16 density vs w_0 (7b): " +
        ", ".join(f"k={k}: {d:.4%}" for k, d in dens.items()) + f"; k=32 encode {kms:.3f} ms")
    out["kstep_bf16"] = {"density": {str(k): round(d, 6) for k, d in dens.items()},
                         "sparsity": {str(k): round(1 - d, 6) for k, d in dens.items()},
                         "encode_ms_k32": round(kms, 4)}
    return out


def cpu_baseline(ps, sample_elems, idx, val, seg, nnz, cap):
    """The oracle (single-threaded C) on a bounded sample of the same step: encode with refresh."""
    import numpy as np
    import oracle

    oracle.build()
    take, tot = [], 0
    for i, n in enumerate(ps.sizes):
        if tot >= sample_elems:
            break
        take.append(i)
        tot += n
    segs = seg.cpu().numpy().tolist() + [min(nnz, cap)]
    t_enc = 0.0
    parity = True
    for i in take:
        w = ps.view(ps.w, i).cpu().numpy()
        s = ps.view(ps.S, i).cpu().numpy().view(np.uint16)
        r = s.copy()
        c0 = time.perf_counter_ns()
        cnt, o_idx, o_val = oracle.encode(w, s, index_base=ps.base(i), refresh=r)
        t_enc += (time.perf_counter_ns() - c0) * 1e-9
        b, e = segs[i], segs[i + 1]
        if e <= cap:
            g_idx = idx[b:e].cpu().numpy().view(np.uint32)
            g_val = val[b:e].cpu().numpy().view(np.uint16)
            parity &= (e - b == cnt and np.array_equal(g_idx, o_idx[:cnt])
                       and np.array_equal(g_val, o_val[:cnt]))
        parity &= np.array_equal(r, ps.view(ps.R, i).cpu().numpy().view(np.uint16))
        log(f"[bench] cpu baseline: tensor {i} ({ps.sizes[i]:,} elems) done")
    return {
        "value": round(6.0 * tot / t_enc / 1e9, 4),
        "unit": "GB/s",
        "cores": 1,
        "kind": "oracle",
        "sample": f"first {len(take)} tensors in model order ({tot:,} of {ps.N:,} params): "
                  f"oracle fused encode + refresh, single-threaded C",
        "seconds": round(t_enc, 3),
        "host_cpu": cpu_model(),
        "host_nproc": os.cpu_count(),
        "sample_parity_with_gpu": bool(parity),
    }


if __name__ == "__main__":
    main()
