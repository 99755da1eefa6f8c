#!/usr/bin/env python3
"""Restore+verify throughput of one GPU's engine state (libgms on MI355X).

A step is one fused restore+verify of the Llama-style 8B bf16 weight set
(291 tensors, 16.06 GB) from a device-resident packed image: every tensor is
rewritten from the image and every 4 KiB block is hashed in registers and
compared with the hashes recorded at snapshot time.  ``value`` is payload
bytes restored and verified per second (GB/s, 1e9).  The same run also
measures the other rows of the path (snapshot, plain restore, verify alone,
pinned-host restore through the staging ring and zero-copy, the 8 GiB KV pool
with live-block restore and a planted corruption), the host-link and plain
copy references, the roofline of the fused restore kernel and the CPU oracle
on a bounded sample.  Prints one JSON line on stdout; progress goes to stderr.

    python bench.py [--gpus 1] [--steps 20] [--warmup 3] [--rows all|main,cpu,...]
"""
from __future__ import annotations

import argparse
import hashlib
import json
import os
import statistics
import sys
import threading
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

METRIC = "restore+verify GB/s on 1 GPU; seconds to restore a 16 GB weight shard"
HBM_PEAK_GBS = 8000.0
ALL_ROWS = ["main", "snapshot", "plain", "verify", "sequential", "unaligned", "tiny", "mixed", "h2d", "file", "kv",
            "kv_vmm", "store", "owner", "recovery", "copy", "cpu", "shards"]
# What shapes the measured kernel's accesses: the kernel and its launch code, the
# header's block and default chunk sizes and the chunking in manifest creation.
KERNEL_SOURCES = ["paper_2609_25451_amd/csrc/gms_kernels.hip", "paper_2609_25451_amd/csrc/gms_internal.h"]
HEADER = "include/gms.h"
# the host code that decides what the measured kernel is launched over: the chunking, the launch
# groups and the launch itself (function bodies), and the grouping threshold (a line)
CHUNKING = ("paper_2609_25451_amd/csrc/gms_api.hip",
            ["int gms_manifest_create(", "uint32_t unit_class(", "void plan_launch_groups(", "hipError_t launch_all("],
            ["constexpr uint64_t kSplitUnits"])
TRAFFIC_FILE = os.path.join(ROOT, "profiles", "traffic_restore_verify_llama8b.json")


def log(*a):
    print("[bench]", *a, file=sys.stderr, flush=True)


def _code(text: str) -> str:
    """C/C++ source without comments or blank lines (comments do not change a kernel)."""
    import re

    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    text = re.sub(r"//[^\n]*", "", text)
    return "\n".join(l.rstrip() for l in text.splitlines() if l.strip())


def kernel_source_digest() -> str:
    h = hashlib.sha256()
    for p in KERNEL_SOURCES:
        with open(os.path.join(ROOT, p)) as f:
            h.update(_code(f.read()).encode())
    with open(os.path.join(ROOT, HEADER)) as f:
        h.update("".join(l for l in f if l.startswith(("#define GMS_BLOCK_BYTES", "#define GMS_DEFAULT_CHUNK_BYTES")))
                 .encode())
    with open(os.path.join(ROOT, CHUNKING[0])) as f:
        src = f.read()
    for marker in CHUNKING[1]:
        start = src.index(marker)
        h.update(_code(src[start:src.index("\n}\n", start)]).encode())
    for prefix in CHUNKING[2]:
        h.update("".join(l for l in src.splitlines(True) if l.startswith(prefix)).encode())
    return h.hexdigest()[:16]


def parse():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--rows", default="all", help="comma list of " + ",".join(ALL_ROWS) + " or 'all'")
    ap.add_argument("--calib-copy", action="store_true",
                    help="also run one plain 1 GiB torch copy (counter calibration)")
    return ap.parse_args()


class Timer:
    """HIP events on the stream the library launches on (torch's current stream)."""

    def __init__(self, torch):
        self.torch = torch

    def run(self, fn, reps: int):
        t = self.torch
        s = t.cuda.current_stream()
        out = []
        for _ in range(reps):
            a, b = t.cuda.Event(enable_timing=True), t.cuda.Event(enable_timing=True)
            a.record(s)
            fn()
            b.record(s)
            b.synchronize()
            out.append(a.elapsed_time(b) / 1e3)
        return out


class GpuSampler:
    """Polls the card's clock levels, junction and HBM temperatures and power from sysfs
    on a thread while a row runs (every 5 ms); the summary is empty where the files are absent."""

    def __init__(self, period: float = 0.005):
        import glob

        cards = sorted(glob.glob("/sys/class/drm/card*/device/pp_dpm_sclk"))
        self.dev = os.path.dirname(cards[0]) if cards else None
        hw = sorted(glob.glob(os.path.join(self.dev, "hwmon", "hwmon*"))) if self.dev else []
        self.hwmon = hw[0] if hw else None
        self.period = period
        self.samples = []
        self._stop = threading.Event()
        self._t = None

    @staticmethod
    def _read(path):
        try:
            with open(path) as f:
                return f.read()
        except OSError:
            return None

    def _sample(self):
        s = {}
        for clk in ("sclk", "mclk", "fclk", "socclk"):
            txt = self._read(os.path.join(self.dev, "pp_dpm_" + clk))
            for line in (txt or "").splitlines():
                if line.rstrip().endswith("*"):
                    s[clk + "_mhz"] = int(line.split(":")[1].strip().split("Mhz")[0].split("MHz")[0])
        if self.hwmon:
            for key, name, scale in (("junction_c", "temp2_input", 1e3), ("mem_c", "temp3_input", 1e3),
                                     ("power_w", "power1_input", 1e6)):
                v = self._read(os.path.join(self.hwmon, name))
                if v and v.strip().lstrip("-").isdigit():
                    s[key] = int(v) / scale
        return s

    def _run(self):
        while not self._stop.is_set():
            self.samples.append(self._sample())
            self._stop.wait(self.period)

    def __enter__(self):
        if self.dev:
            self._t = threading.Thread(target=self._run, daemon=True)
            self._t.start()
        return self

    def __exit__(self, *exc):
        self._stop.set()
        if self._t:
            self._t.join()

    def summary(self):
        out = {}
        for key in ("sclk_mhz", "mclk_mhz", "fclk_mhz", "socclk_mhz", "power_w"):
            v = [s[key] for s in self.samples if key in s]
            if v:
                out[key + "_median"] = statistics.median(v)
        for key in ("junction_c", "mem_c"):
            v = [s[key] for s in self.samples if key in s]
            if v:
                out[key + "_max"] = max(v)
        if out:
            out["samples"] = len(self.samples)
        return out


def settled(timer, fn, warm: int = 3, reps: int = 20):
    """Median launch time after `warm` untimed launches.  Switching between rows of different
    VALU load moves the shader clock (about 2.37 GHz under the copy, 2.19 GHz under verify),
    and the first launches after a switch run at neither."""
    for _ in range(warm):
        fn()
    return statistics.median(timer.run(fn, reps))


def build_weights(torch, synth, name):
    seed, specs = synth.weight_set(name)
    tensors = [torch.empty(sp.shape, dtype=torch.bfloat16, device="cuda") for sp in specs]
    torch.cuda.synchronize()
    synth.dev_fill_tensors(tensors, seed)  # one launch for the whole set
    return seed, specs, tensors


def main():
    args = parse()
    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) > 1:
        print("bench.py measures one GPU only: the restore path is per-GPU and independent "
              "(each rank restores its own shard); run with --gpus 1", file=sys.stderr)
        sys.exit(2)
    rows = ALL_ROWS if args.rows == "all" else [r.strip() for r in args.rows.split(",") if r.strip()]

    import numpy as np
    import torch

    import paper_2609_25451_amd as gms
    import synth

    if not torch.cuda.is_available():
        print("bench.py needs a GPU", file=sys.stderr)
        sys.exit(1)
    torch.cuda.set_device(0)
    timer = Timer(torch)
    result_rows = {}

    # ---------------------------------------------------------------- workload
    t0 = time.time()
    seed, specs, tensors = build_weights(torch, synth, "llama8b")
    tm = time.perf_counter()
    m = gms.Manifest(tensors, device=0)
    manifest_s = time.perf_counter() - tm
    P, nb, n, nchunks = m.payload_bytes, m.num_blocks, m.num_entries, m.num_chunks
    image = torch.empty(m.image_bytes, dtype=torch.uint8, device="cuda")
    expected = torch.zeros(nb, dtype=torch.int64, device="cuda")
    ten_hash = torch.zeros(n, dtype=torch.int64, device="cuda")
    gms.snapshot(m, image, m.image_bytes, gms.MEM_DEVICE, blk_hash=expected, ten_hash=ten_hash)
    torch.cuda.synchronize()
    log(f"llama8b: {n} tensors, {P} B, {nb} blocks, {nchunks} chunks; setup {time.time() - t0:.1f}s")
    pinned_reserved = reserve_pinned(torch, synth, rows, m.image_bytes)

    cnt = torch.zeros(1, dtype=torch.int64, device="cuda")
    mlist = torch.zeros(64, dtype=torch.int64, device="cuda")

    def fused_restore():
        gms.restore(m, image, m.image_bytes, gms.MEM_DEVICE, expected=expected, mismatch_count=cnt,
                    mismatch_list=mlist, mismatch_cap=64)

    # correctness gate for the timed configuration: poison, restore, compare a sample
    for t in tensors:
        t.view(torch.uint8).fill_(0xA5)
    fused_restore()
    torch.cuda.synchronize()
    assert int(cnt.item()) == 0, "fused restore reported mismatches on a clean image"
    for i in (0, 1, 7, len(tensors) - 1):
        k = min(tensors[i].numel(), 1 << 16)
        got = tensors[i].reshape(-1)[:k].view(torch.int16).cpu().numpy().view(np.uint16)
        assert np.array_equal(got, synth.bf16_bits(k, seed, i)), f"tensor {i} restored wrong"

    # ---------------------------------------------------------------- main step
    main_times = []
    gpu_main = None
    if "main" in rows:
        for _ in range(args.warmup):
            fused_restore()
        torch.cuda.synchronize()
        s = torch.cuda.current_stream()
        evs = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))
               for _ in range(args.steps)]
        torch.cuda.synchronize()
        with GpuSampler() as gpu_main:
            w0 = time.perf_counter()
            for a, b in evs:
                a.record(s)
                fused_restore()
                b.record(s)
            torch.cuda.synchronize()
            wall = time.perf_counter() - w0
        main_times = [a.elapsed_time(b) / 1e3 for a, b in evs]
        assert int(cnt.item()) == 0
        log(f"fused restore+verify: wall {wall * 1e3 / args.steps:.3f} ms/step, "
            f"kernel avg {statistics.mean(main_times) * 1e3:.3f} ms")
    else:
        wall = float("nan")

    # ---------------------------------------------------------------- other rows
    if "snapshot" in rows:
        blk2 = torch.zeros(nb, dtype=torch.int64, device="cuda")
        with GpuSampler() as gs:
            t = settled(timer, lambda: gms.snapshot(m, image, m.image_bytes, gms.MEM_DEVICE, blk_hash=blk2))
        assert torch.equal(blk2, expected)
        tp = settled(timer, lambda: gms.snapshot(m, image, m.image_bytes, gms.MEM_DEVICE))  # no hashes
        result_rows["snapshot_d2d_hash"] = {"s": t, "GB_s": P / t / 1e9,
                                            "hbm_frac": (2 * P + 8 * nb) / t / 1e9 / HBM_PEAK_GBS,
                                            "unhashed_s": tp, "unhashed_hbm_frac": 2 * P / tp / 1e9 / HBM_PEAK_GBS,
                                            "gpu": gs.summary()}
    if "plain" in rows:
        with GpuSampler() as gs:
            t = settled(timer, lambda: gms.restore(m, image, m.image_bytes, gms.MEM_DEVICE))
        result_rows["restore_d2d_plain"] = {"s": t, "GB_s": P / t / 1e9, "hbm_frac": 2 * P / t / 1e9 / HBM_PEAK_GBS,
                                            "gpu": gs.summary()}
    if "verify" in rows:
        vc = torch.zeros(1, dtype=torch.int64, device="cuda")
        with GpuSampler() as gs:  # verify needs about eight launches to reach its rate after other work
            t = settled(timer, lambda: gms.verify(m, expected=expected, mismatch_count=vc), warm=10)
        assert int(vc.item()) == 0
        result_rows["verify_only"] = {"s": t, "GB_s": P / t / 1e9,
                                      "hbm_frac": (P + 8 * nb) / t / 1e9 / HBM_PEAK_GBS, "gpu": gs.summary()}
    if "sequential" in rows:  # restore, then a separate verify pass: 3P bytes against the fused 2P
        vc = torch.zeros(1, dtype=torch.int64, device="cuda")

        def seq():
            gms.restore(m, image, m.image_bytes, gms.MEM_DEVICE)
            gms.verify(m, expected=expected, mismatch_count=vc)

        t = settled(timer, seq, reps=10)
        assert int(vc.item()) == 0
        result_rows["restore_then_verify_sequential"] = {
            "s": t, "GB_s": P / t / 1e9, "hbm_frac": (3 * P + 8 * nb) / t / 1e9 / HBM_PEAK_GBS,
            "fused_speedup": t / statistics.median(main_times) if main_times else None}
    if "unaligned" in rows:
        result_rows["unaligned"] = bench_unaligned(torch, gms, timer, tensors)
    if "tiny" in rows:
        result_rows["tiny"] = bench_tiny(torch, gms, synth, timer)
    if "mixed" in rows:
        result_rows["mixed"] = bench_mixed(torch, gms, synth, timer, tensors,
                                           statistics.median(main_times) if main_times else None)
    if "copy" in rows:
        a = torch.empty(4 << 30, dtype=torch.uint8, device="cuda")
        b = torch.empty_like(a)
        t = settled(timer, lambda: b.copy_(a))
        result_rows["torch_copy_4GiB_reference"] = {"s": t, "hbm_GB_s": 2 * a.numel() / t / 1e9,
                                                    "hbm_frac": 2 * a.numel() / t / 1e9 / HBM_PEAK_GBS}
        del a, b
    if args.calib_copy:
        a = torch.ones(1 << 30, dtype=torch.uint8, device="cuda")
        b = torch.empty_like(a)
        b.copy_(a)
        torch.cuda.synchronize()
        del a, b

    if "h2d" in rows:
        pinned = pinned_view(m.image_bytes)
        # link peak: 1 GiB pinned -> device copies
        gib = pinned[: 1 << 30]
        dst = torch.empty(1 << 30, dtype=torch.uint8, device="cuda")
        lt = timer.run(lambda: dst.copy_(gib, non_blocking=True), 20)
        link = (1 << 30) / statistics.median(lt) / 1e9
        lt = timer.run(lambda: gib.copy_(dst, non_blocking=True), 20)
        link_d2h = (1 << 30) / statistics.median(lt) / 1e9
        del dst
        gms.snapshot(m, pinned, m.image_bytes, gms.MEM_HOST_PINNED)  # allocates the ring, untimed

        def snap():
            gms.snapshot(m, pinned, m.image_bytes, gms.MEM_HOST_PINNED)

        snap_warm = settle_link(timer, snap, P, link_d2h)  # as for the restore leg below
        snap_h = statistics.median(timer.run(snap, 3))
        hc = torch.zeros(1, dtype=torch.int64, device="cuda")

        def h2d():
            gms.restore(m, pinned, m.image_bytes, gms.MEM_HOST_PINNED, expected=expected, mismatch_count=hc)

        h2d_warm = settle_link(timer, h2d, P, link)
        th = statistics.median(timer.run(h2d, 3))
        link_after = link_now(torch, timer)
        assert int(hc.item()) == 0

        def h2d_noalloc():  # the same restore with no allocation: fixed staging area, one stream
            gms.restore_pinned_noalloc(m, pinned, m.image_bytes, expected=expected, mismatch_count=hc)

        h2d_noalloc()
        tna = statistics.median(timer.run(h2d_noalloc, 3))
        assert int(hc.item()) == 0
        m.set_staging(0, 0)
        tz = statistics.median(timer.run(h2d, 2))
        assert int(hc.item()) == 0
        snap_z = statistics.median(timer.run(lambda: gms.snapshot(m, pinned, m.image_bytes, gms.MEM_HOST_PINNED), 2))
        m.set_staging(gms.DEFAULT_SLICE_BYTES, gms.DEFAULT_SLOTS)
        result_rows["h2d"] = {
            "pinned_buffer": pinned_reserved,
            "link_peak_GB_s": link,
            "restore_verify_ring_s": th, "restore_verify_ring_GB_s": P / th / 1e9,
            "restore_untimed_calls_s": h2d_warm, "link_right_after_GB_s": link_after,
            "link_frac": P / th / 1e9 / link,
            "restore_verify_zero_copy_s": tz, "restore_verify_zero_copy_GB_s": P / tz / 1e9,
            "restore_verify_noalloc_s": tna, "restore_verify_noalloc_GB_s": P / tna / 1e9,
            "noalloc_link_frac": P / tna / 1e9 / link,
            "link_peak_d2h_GB_s": link_d2h,
            "snapshot_to_pinned_s": snap_h, "snapshot_to_pinned_GB_s": P / snap_h / 1e9,
            "snapshot_untimed_calls_s": snap_warm,
            "snapshot_link_frac": P / snap_h / 1e9 / link_d2h,
            "snapshot_to_pinned_zero_copy_GB_s": P / snap_z / 1e9,
        }
        del pinned
        result_rows["h2d"]["pageable"] = pageable_leg(torch, np, gms, timer, m, expected, link, link_d2h)
        assert result_rows["h2d"]["pageable"]["mismatches"] == 0

    if "file" in rows:
        result_rows["file"] = bench_file(torch, gms, m, expected)

    link = result_rows.get("h2d", {}).get("link_peak_GB_s")
    if "kv" in rows:
        result_rows["kv_pool"] = bench_kv(torch, np, gms, synth, timer, link)
    if "kv_vmm" in rows:
        result_rows["kv_pool_vmm"] = bench_kv_vmm(torch, np, gms, synth, timer)
    if "store" in rows:
        result_rows["store"] = bench_store(torch, gms, m, image, expected)
    if "owner" in rows:
        result_rows["owner"] = bench_owner(torch, gms, timer, m, image, expected)
    if "recovery" in rows:
        result_rows["recovery"] = bench_recovery(torch, np, gms, synth, m, image, expected)

    # ---------------------------------------------------------------- roofline
    roof = None
    if main_times:
        kt = statistics.mean(main_times)
        alg = 2 * P + 8 * nb  # read image + write entries + read expected hashes
        achieved = alg / kt / 1e9
        traffic = None
        if os.path.exists(TRAFFIC_FILE):
            with open(TRAFFIC_FILE) as f:
                tr = json.load(f)
            if tr.get("kernel_digest") == kernel_source_digest():
                traffic = tr.get("hbm_bytes_per_launch")
        roof = {"bound": "hbm", "kernel": "gms::k_stream<restore,hash>", "achieved": round(achieved, 1),
                "peak": HBM_PEAK_GBS, "unit": "GB/s", "frac": round(achieved / HBM_PEAK_GBS, 4),
                "traffic": traffic, "algorithmic_bytes_per_launch": alg,
                "avg_launch_ms": round(kt * 1e3, 4),
                "gpu_during_timed_steps": gpu_main.summary() if gpu_main else {}}

    # ---------------------------------------------------------------- CPU oracle
    cpu = None
    if "cpu" in rows:
        cpu = bench_cpu(torch, np, image, m, specs, expected)

    if "shards" in rows:  # last: frees the llama8b buffers to make room for the 122 GB MoE shard
        del tensors, image, expected, ten_hash, cnt, mlist
        m.close()
        torch.cuda.synchronize()
        torch.cuda.empty_cache()
        result_rows["shards"] = {name: bench_shard(torch, gms, synth, timer, name, link)
                                 for name in ("llama70b_tp8", "moe")}

    # release the pinned and device buffers and join helper threads before the result line,
    # so that the process has nothing left to tear down once it has reported
    t_rel = time.perf_counter()
    _PINNED["buf"] = None
    if "shards" not in rows:  # the shard rows freed these already
        del tensors, image, expected, ten_hash, cnt, mlist
        m.close()
    import gc

    gc.collect()
    torch.cuda.synchronize()
    torch.cuda.empty_cache()
    for t in threading.enumerate():
        if t is not threading.current_thread() and not t.daemon:
            t.join(timeout=30)
    log(f"buffers released in {time.perf_counter() - t_rel:.2f} s")

    value = P * args.steps / wall / 1e9 if main_times else None
    out = {
        "metric": METRIC,
        "value": round(value, 2) if value else None,
        "unit": "GB/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(wall * 1e3 / args.steps, 4) if main_times else None,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "u64",
        "data": "synthetic (seeded Philox bf16 ~N(0,0.02), generated on the GPU)",
        "config": {
            "workload": "llama8b bf16 weight set: 32 layers, d_model 4096, GQA 32q/8kv x 128, SwiGLU ffn 14336, "
                        "vocab 128256; 291 tensors; device-resident image; fused restore+verify",
            "payload_bytes": P, "entries": n, "blocks": nb, "chunks": nchunks, "block_bytes": 4096,
            "manifest_create_s": round(manifest_s, 4),
        },
        "seconds_to_restore_16GB": {
            "device_image_restore_verify": round(statistics.mean(main_times), 6) if main_times else None,
            "device_image_plain": round(result_rows["restore_d2d_plain"]["s"], 6) if "restore_d2d_plain" in result_rows else None,
            "host_pinned_restore_verify": round(result_rows["h2d"]["restore_verify_ring_s"], 4) if "h2d" in result_rows else None,
        },
        "roofline": roof,
        "cpu_baseline": cpu,
        "rows": result_rows,
    }
    print(json.dumps(out), flush=True)


def bench_file(torch, gms, m, expected):
    """Cold repopulation from storage: the image written to a file, then streamed back."""
    import shutil
    import tempfile

    d = tempfile.gettempdir()
    free = shutil.disk_usage(d).free
    if free < m.image_bytes + (2 << 30):
        return {"skipped": f"{free} bytes free in {d}, need {m.image_bytes + (2 << 30)}"}
    path = os.path.join(d, f"gms_bench_image_{os.getpid()}.bin")
    cnt = torch.zeros(1, dtype=torch.int64, device="cuda")
    out = {"dir": d, "bytes": m.image_bytes}
    try:
        t0 = time.perf_counter()
        gms.snapshot_to_file(m, path, flags=gms.FILE_DIRECT | gms.FILE_SYNC)
        torch.cuda.synchronize()
        out["snapshot_direct_sync_s"] = time.perf_counter() - t0
        def restore(flags):
            torch.cuda.synchronize()
            t0 = time.perf_counter()
            gms.restore_from_file(m, path, flags=flags, expected=expected, mismatch_count=cnt)
            torch.cuda.synchronize()
            t = time.perf_counter() - t0
            assert int(cnt.item()) == 0, "file restore reported mismatches"
            return m.payload_bytes / t / 1e9

        # The shared disk's speed drifts within a run (it is slow right after the write), so raw
        # O_DIRECT reads and direct restores alternate and the best of each is compared.
        raw, direct = [], []
        for _ in range(3):
            raw.append(raw_direct_read(path, m.image_bytes) / 1e9)
            direct.append(restore(gms.FILE_DIRECT))
        cold = restore(0)    # buffered; O_DIRECT reads left the page cache cold
        cached = restore(0)  # buffered, now from the page cache
        out.update({
            "restore_verify_direct_GB_s": max(direct), "restore_verify_direct_s": m.payload_bytes / max(direct) / 1e9,
            "restore_verify_direct_runs_GB_s": direct, "storage_read_direct_GB_s": max(raw),
            "storage_read_direct_runs_GB_s": raw, "storage_frac": max(direct) / max(raw),
            "restore_verify_buffered_cold_GB_s": cold, "restore_verify_buffered_cached_GB_s": cached,
        })
        log(f"file restore+verify: direct {out['restore_verify_direct_GB_s']:.1f} GB/s "
            f"(raw direct read {out['storage_read_direct_GB_s']:.1f} GB/s), "
            f"cached {out['restore_verify_buffered_cached_GB_s']:.1f} GB/s")
    finally:
        if os.path.exists(path):
            os.remove(path)
    return out


def raw_direct_read(path, nbytes, threads=16, piece=16 << 20):
    """Bytes/s of plain parallel O_DIRECT reads of the file (the storage side alone), in the
    library's own request shape: `threads` workers taking `piece`-byte reads in file order."""
    import mmap
    import threading

    fd = os.open(path, os.O_RDONLY | getattr(os, "O_DIRECT", 0))
    try:
        npieces = -(-nbytes // piece)

        def work(t):
            buf = mmap.mmap(-1, piece)
            for i in range(t, npieces, threads):
                lo = i * piece
                want = min(piece, nbytes - lo)
                n = os.preadv(fd, [memoryview(buf)[:want]], lo)
                if n != want:
                    raise OSError("short read")
            buf.close()

        t0 = time.perf_counter()
        ts = [threading.Thread(target=work, args=(t,)) for t in range(threads)]
        for t in ts:
            t.start()
        for t in ts:
            t.join()
        return nbytes / (time.perf_counter() - t0)
    finally:
        os.close(fd)


def bench_unaligned(torch, gms, timer, tensors, offset: int = 2):
    """The llama8b tensors as entries 2 bytes past their start (each tensor minus its first
    bf16 element), so every entry address is off a 16-byte boundary: the kernels' shifted
    path.  Snapshot with hashes into an image of its own, then fused restore+verify (which
    rewrites the same bytes) and verify alone."""
    ents = [(t.data_ptr() + offset, t.numel() * t.element_size() - offset) for t in tensors]
    mu = gms.Manifest(ents, device=0)
    Pu, nbu = mu.payload_bytes, mu.num_blocks
    img = torch.empty(mu.image_bytes, dtype=torch.uint8, device="cuda")
    exp = torch.zeros(nbu, dtype=torch.int64, device="cuda")
    c = torch.zeros(1, dtype=torch.int64, device="cuda")
    with GpuSampler() as gs:
        ts = settled(timer, lambda: gms.snapshot(mu, img, mu.image_bytes, blk_hash=exp))
        tr = settled(timer, lambda: gms.restore(mu, img, mu.image_bytes, expected=exp, mismatch_count=c))
    assert int(c.item()) == 0
    tv = settled(timer, lambda: gms.verify(mu, expected=exp, mismatch_count=c), warm=10)
    assert int(c.item()) == 0
    out = {"entry_offset_bytes": offset, "payload_bytes": Pu, "launch_groups": mu.num_launch_groups,
           "restore_verify_s": tr, "restore_verify_GB_s": Pu / tr / 1e9,
           "restore_verify_hbm_frac": (2 * Pu + 8 * nbu) / tr / 1e9 / HBM_PEAK_GBS,
           "snapshot_hash_s": ts, "snapshot_hbm_frac": (2 * Pu + 8 * nbu) / ts / 1e9 / HBM_PEAK_GBS,
           "verify_s": tv, "verify_hbm_frac": (Pu + 8 * nbu) / tv / 1e9 / HBM_PEAK_GBS, "gpu": gs.summary()}
    log(f"unaligned (+{offset} B) llama8b: restore+verify {tr * 1e3:.2f} ms "
        f"({out['restore_verify_hbm_frac'] * 100:.1f}% of HBM peak), snapshot {ts * 1e3:.2f} ms, "
        f"verify {tv * 1e3:.2f} ms")
    mu.close()
    del img, exp
    torch.cuda.synchronize()
    torch.cuda.empty_cache()
    return out


def bench_tiny(torch, gms, synth, timer):
    """The tiny 21-tensor set (8.4 MB): it fits in the 256 MB last-level cache, so it is
    reported as latency, not against the HBM roofline."""
    seed, specs, tensors = build_weights(torch, synth, "tiny")
    m = gms.Manifest(tensors, device=0)
    img = torch.empty(m.image_bytes, dtype=torch.uint8, device="cuda")
    exp = torch.zeros(m.num_blocks, dtype=torch.int64, device="cuda")
    gms.snapshot(m, img, m.image_bytes, blk_hash=exp)
    cnt = torch.zeros(1, dtype=torch.int64, device="cuda")
    fused = lambda: gms.restore(m, img, m.image_bytes, expected=exp, mismatch_count=cnt)
    for _ in range(3):
        fused()
    t = statistics.median(timer.run(fused, 20))
    assert int(cnt.item()) == 0
    ts = statistics.median(timer.run(lambda: gms.snapshot(m, img, m.image_bytes, blk_hash=exp), 20))
    # the same fused call captured once into a HIP graph and replayed
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        fused()
    for _ in range(3):
        g.replay()
    tg = statistics.median(timer.run(g.replay, 20))
    assert int(cnt.item()) == 0
    del g
    out = {"tensors": len(tensors), "payload_bytes": m.payload_bytes, "restore_verify_us": round(t * 1e6, 1),
           "restore_verify_graph_replay_us": round(tg * 1e6, 1), "snapshot_us": round(ts * 1e6, 1)}
    m.close()
    return out


def bench_mixed(torch, gms, synth, timer, tensors, weights_s=None, n_small=200_000, small_bytes=256):
    """The llama8b weights plus 200,000 small runtime buffers of 256 bytes (seeded bytes), restored
    and verified in one call.  A small buffer's chunk needs one work unit where a 64 KiB chunk
    needs eight; the manifest launches them apart (launch groups), so the buffers should cost what
    they cost alone.  Reported beside the weights-only step and the buffers alone."""
    small = torch.empty(n_small * 512, dtype=torch.uint8, device="cuda")
    synth.dev_fill_bf16(small.data_ptr(), small.numel() // 2, 4242, 0)
    bufs = [(small.data_ptr() + i * 512, small_bytes) for i in range(n_small)]

    def one(entries):
        m = gms.Manifest(entries, device=0)
        img = torch.empty(m.image_bytes, dtype=torch.uint8, device="cuda")
        exp = torch.zeros(m.num_blocks, dtype=torch.int64, device="cuda")
        gms.snapshot(m, img, m.image_bytes, blk_hash=exp)
        cnt = torch.zeros(1, dtype=torch.int64, device="cuda")
        t = settled(timer, lambda: gms.restore(m, img, m.image_bytes, expected=exp, mismatch_count=cnt))
        assert int(cnt.item()) == 0
        out = (t, m.num_launch_groups, m.num_chunks)
        m.close()
        del img, exp
        return out

    t_mixed, groups, chunks = one(list(tensors) + bufs)
    t_small, _, _ = one(bufs)
    del small
    torch.cuda.empty_cache()
    out = {"entries": len(tensors) + n_small, "small_buffers": n_small, "small_bytes": small_bytes, "chunks": chunks,
           "launch_groups": groups, "restore_verify_s": t_mixed, "small_buffers_alone_s": t_small}
    if weights_s:
        out["weights_only_s"] = weights_s
        out["added_by_small_buffers_s"] = t_mixed - weights_s
    return out


def host_info():
    """The measuring host: the CPU as /proc/cpuinfo and lscpu describe it (a virtual machine may
    show only a family name as the model), the CPUs this process may run on and NUMA nodes."""
    info = {}
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                key, _, val = line.partition(":")
                key = key.strip()
                if key in ("model name", "vendor_id", "cpu family", "model", "stepping", "cpu MHz", "cache size"):
                    info.setdefault(key.replace(" ", "_"), val.strip())
                if not line.strip() and info:
                    break
    except OSError:
        pass
    try:
        import subprocess

        out = subprocess.run(["lscpu"], capture_output=True, text=True, timeout=10).stdout
        for line in out.splitlines():
            key, _, val = line.partition(":")
            if key.strip() in ("Model name", "BIOS Model name", "Socket(s)", "Core(s) per socket",
                               "Thread(s) per core", "Hypervisor vendor", "L3 cache"):
                info["lscpu_" + key.strip().replace(" ", "_").replace("(s)", "s")] = val.strip()
    except (OSError, ValueError):
        pass
    nodes = 0
    try:
        nodes = len([d for d in os.listdir("/sys/devices/system/node") if d.startswith("node") and d[4:].isdigit()])
    except OSError:
        pass
    return {"cpu_model": info.get("model_name", ""), "cpu": info, "cores_available": len(os.sched_getaffinity(0)),
            "os_cpu_count": os.cpu_count(), "numa_nodes": nodes}


def bench_kv(torch, np, gms, synth, timer, link=None):
    """8 GiB paged KV pool: restore only the live blocks + verify, one planted bit flip."""
    p = synth.kv_pool()
    pool = [torch.empty(p.layer_bytes, dtype=torch.uint8, device="cuda") for _ in range(p.layers)]
    for l, t in enumerate(pool):
        synth.dev_fill_bf16(t.data_ptr(), p.layer_bytes // 2, p.seed, l)
    live = synth.live_map(p.blocks, p.n_live, p.map_seed, p.map_stream)
    ents = [(pool[l].data_ptr() + int(b) * p.unit_bytes, p.unit_bytes) for l in range(p.layers) for b in live]
    m = gms.Manifest(ents, device=0)
    P, nb = m.payload_bytes, m.num_blocks
    img = torch.empty(m.image_bytes, dtype=torch.uint8, device="cuda")
    exp = torch.zeros(nb, dtype=torch.int64, device="cuda")
    gms.snapshot(m, img, m.image_bytes, blk_hash=exp)
    # planted corruption: one bit of one live unit in the image
    e = synth.u64(p.corrupt_seed, p.corrupt_stream, 0) % m.num_entries
    blk = synth.u64(p.corrupt_seed, p.corrupt_stream, 1) % (p.unit_bytes // 4096)
    bit = synth.u64(p.corrupt_seed, p.corrupt_stream, 2) % (4096 * 8)
    off, base = m.layout()
    byte = off[e] + blk * 4096 + bit // 8
    img[byte] ^= 1 << (bit % 8)
    for t in pool:
        t.fill_(0xA5)
    cnt = torch.zeros(1, dtype=torch.int64, device="cuda")
    lst = torch.zeros(8, dtype=torch.int64, device="cuda")

    def run():
        gms.restore(m, img, m.image_bytes, expected=exp, mismatch_count=cnt, mismatch_list=lst, mismatch_cap=8)

    t = settled(timer, run)
    c = int(cnt.item())
    flagged = sorted(int(v) for v in lst[:min(c, 8)].cpu().tolist())
    # dead units keep the poison
    dead = np.setdiff1d(np.arange(p.blocks), live)
    dead_ok = all(bool((u.view(p.blocks, p.unit_bytes)[torch.from_numpy(dead).cuda()] == 0xA5).all()) for u in pool[:4])
    h2d = h2d_leg(torch, gms, timer, m, img, exp, link)  # the same planted flip, through the host link
    return {"entries": m.num_entries, "payload_bytes": P, "s": t, "GB_s": P / t / 1e9,
            "hbm_frac": 2 * P / t / 1e9 / HBM_PEAK_GBS, "mismatches": c, "flagged": flagged,
            "planted_block": int(base[e] + blk), "dead_units_untouched_first4_layers": dead_ok, "h2d": h2d}


H2D_MAX_PINNED = 64 << 30  # the measuring host cannot pin the 122 GB MoE image
# One pinned host buffer serves every pinned-image leg.  It is allocated once, before the rows
# run, so no leg pins (0.3 s per 16 GB) or re-allocates pinned memory inside its own timing.
_PINNED = {"buf": None}


def link_now(torch, timer, reps: int = 3):
    """A plain 1 GiB pinned-to-device copy, to put a leg's rate beside what the link gives at that
    moment (the host link of the measuring machine sometimes runs at half its rate for seconds)."""
    buf = _PINNED["buf"]
    if buf is None or buf.numel() < (1 << 30):
        return None
    dst = torch.empty(1 << 30, dtype=torch.uint8, device="cuda")
    t = statistics.median(timer.run(lambda: dst.copy_(buf[: 1 << 30], non_blocking=True), reps))
    del dst
    return round((1 << 30) / t / 1e9, 2)


def settle_link(timer, run, payload, link, max_calls: int = 10):
    """Untimed calls until one reaches 90% of `link` (or, with no link figure, until two in a
    row agree within 2%), at most `max_calls`; returns every call time."""
    calls = [statistics.median(timer.run(run, 1))]
    while len(calls) < max_calls:
        if link and payload / calls[-1] / 1e9 >= 0.9 * link:
            break
        calls += timer.run(run, 1)
        if not link and abs(calls[-1] - calls[-2]) <= 0.02 * calls[-1]:
            break
    return [round(x, 4) for x in calls]


def image_bytes_of(sizes):
    return sum((n + 4095) // 4096 * 4096 for n in sizes)


def reserve_pinned(torch, synth, rows, llama_image_bytes):
    """Allocates the pinned buffer for the largest image a pinned leg of `rows` will copy."""
    need = [llama_image_bytes] if "h2d" in rows else []
    if "kv" in rows:
        p = synth.kv_pool()
        need.append(p.layers * p.n_live * p.unit_bytes)
    if "shards" in rows:
        need += [image_bytes_of(sp.nbytes for sp in synth.weight_set(n)[1]) for n in ("llama70b_tp8", "moe")]
    need = [n for n in need if n <= H2D_MAX_PINNED]
    if not need:
        return None
    t0 = time.perf_counter()
    _PINNED["buf"] = torch.empty(max(need), dtype=torch.uint8, pin_memory=True)
    dt = time.perf_counter() - t0
    log(f"pinned {max(need)} B for the pinned-image legs in {dt:.1f}s")
    return {"bytes": max(need), "alloc_s": round(dt, 3)}


def pinned_view(nbytes):
    buf = _PINNED["buf"]
    if buf is None or buf.numel() < nbytes:
        raise RuntimeError("no pinned buffer reserved for this image")
    return buf[:nbytes]


def pageable_leg(torch, np, gms, timer, m, exp, link=None, link_d2h=None, reps=3):
    """Snapshot into and restore+verify from an image in ordinary pageable host memory (a numpy
    buffer the library never pins), through the staging rings and the worker pool.  The first
    snapshot also faults the buffer's pages in and is reported apart; then the median of `reps`
    synchronous snapshots (wall clock) and of `reps` restores (HIP events around the call,
    which returns once the image is copied out; the last kernel ends the interval)."""
    P = m.payload_bytes
    t0 = time.perf_counter()
    host = np.empty(m.image_bytes, dtype=np.uint8)
    gms.snapshot_to_host(m, host)
    first = time.perf_counter() - t0
    ts = []
    for _ in range(reps):
        t0 = time.perf_counter()
        gms.snapshot_to_host(m, host)
        ts.append(time.perf_counter() - t0)
    snap = statistics.median(ts)
    cnt = torch.zeros(1, dtype=torch.int64, device="cuda")
    run = lambda: gms.restore_from_host(m, host, expected=exp, mismatch_count=cnt)
    tr = statistics.median(timer.run(run, reps))
    out = {"first_snapshot_with_page_faults_s": round(first, 3), "snapshot_s": snap, "snapshot_GB_s": P / snap / 1e9,
           "restore_verify_s": tr, "restore_verify_GB_s": P / tr / 1e9, "mismatches": int(cnt.item())}
    if link:
        out["restore_link_frac"] = P / tr / 1e9 / link
    if link_d2h:
        out["snapshot_link_frac"] = P / snap / 1e9 / link_d2h
    del host
    return out


def h2d_leg(torch, gms, timer, m, img, exp, link=None, reps=3, cap=8):
    """The same restore+verify from a pinned host copy of the image (in the buffer reserved at
    start-up), through the staging ring: rate, and the mismatches it reports.  One untimed call
    first allocates the manifest's staging ring.  An image this host cannot pin is restored from
    pageable host memory instead."""
    if m.image_bytes > H2D_MAX_PINNED:
        import numpy as np

        out = pageable_leg(torch, np, gms, timer, m, exp, link)
        out["source"] = f"pageable host memory: this host cannot pin an image of {m.image_bytes} B"
        return out
    pinned = pinned_view(m.image_bytes)
    pinned.copy_(img)
    cnt = torch.zeros(1, dtype=torch.int64, device="cuda")
    lst = torch.zeros(cap, dtype=torch.int64, device="cuda")
    run = lambda: gms.restore(m, pinned, m.image_bytes, gms.MEM_HOST_PINNED, expected=exp, mismatch_count=cnt,
                              mismatch_list=lst, mismatch_cap=cap)
    warm = settle_link(timer, run, m.payload_bytes, link)
    t = statistics.median(timer.run(run, reps))
    c = int(cnt.item())
    out = {"restore_verify_s": t, "restore_verify_GB_s": m.payload_bytes / t / 1e9,
           "untimed_calls_s": warm, "link_right_after_GB_s": link_now(torch, timer),
           "mismatches": c, "flagged": sorted(int(v) for v in lst[:min(c, cap)].cpu().tolist())}
    if link:
        out["link_frac"] = m.payload_bytes / t / 1e9 / link
    return out


def bench_shard(torch, gms, synth, timer, name, link=None):
    """Fused restore+verify of another weight workload from a device-resident image."""
    _, specs = synth.weight_set(name)
    P = sum(sp.nbytes for sp in specs)
    free, _ = torch.cuda.mem_get_info()
    if free < 2 * P + (4 << 30):
        return {"skipped": f"needs {2 * P} bytes of device memory, {free} free"}
    seed, specs, tensors = build_weights(torch, synth, name)
    m = gms.Manifest(tensors, device=0)
    img = torch.empty(m.image_bytes, dtype=torch.uint8, device="cuda")
    exp = torch.zeros(m.num_blocks, dtype=torch.int64, device="cuda")
    gms.snapshot(m, img, m.image_bytes, blk_hash=exp)
    cnt = torch.zeros(1, dtype=torch.int64, device="cuda")
    t = settled(timer, lambda: gms.restore(m, img, m.image_bytes, expected=exp, mismatch_count=cnt))
    assert int(cnt.item()) == 0
    out = {"tensors": len(tensors), "payload_bytes": P, "chunks": m.num_chunks, "restore_verify_s": t,
           "restore_verify_GB_s": P / t / 1e9, "hbm_frac": (2 * P + 8 * m.num_blocks) / t / 1e9 / HBM_PEAK_GBS}
    log(f"{name}: restore+verify {t * 1e3:.2f} ms, {out['hbm_frac'] * 100:.1f}% of HBM peak")
    out["h2d"] = h2d_leg(torch, gms, timer, m, img, exp, link)
    if "skipped" not in out["h2d"]:
        assert out["h2d"]["mismatches"] == 0
        log(f"{name}: H2D restore+verify {out['h2d']['restore_verify_s']:.3f} s")
    m.close()
    del tensors, img, exp
    torch.cuda.synchronize()
    torch.cuda.empty_cache()
    return out


def bench_store(torch, gms, m, image, expected):
    """The lease protocol on the llama8b set in a store of its own: a writer populates the
    store's allocations from the device image with a fused restore+verify and commits them
    (hashing every block, mapping the pool read-only); a replacement then attaches read-only
    after re-hashing the committed state.  Wall times of the synchronous calls."""
    sizes = list(m.sizes)
    P = m.payload_bytes
    store = gms.Store(va_bytes=P + (8 << 30), slab_bytes=2 << 30)
    try:
        w = store.connect_rw()
        addrs = [w.alloc(n) for n in sizes]
        sm = gms.Manifest(list(zip(addrs, sizes)), device=0)
        cnt = torch.zeros(1, dtype=torch.int64, device="cuda")
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        gms.restore(sm, image, sm.image_bytes, expected=expected, mismatch_count=cnt)
        torch.cuda.synchronize()
        populate = time.perf_counter() - t0
        assert int(cnt.item()) == 0
        t0 = time.perf_counter()
        w.commit(list(zip(addrs, sizes)), expected=expected)
        commit = time.perf_counter() - t0
        attach = []
        for _ in range(5):
            t0 = time.perf_counter()
            r = store.connect_ro(verify=True)
            attach.append(time.perf_counter() - t0)
            r.close()
        t0 = time.perf_counter()
        w2 = store.connect_rw()  # the writer reacquires: the pool becomes writable again
        reacquire = time.perf_counter() - t0
        w2.commit(list(zip(addrs, sizes)))
        sm.close()
        out = {"payload_bytes": P, "populate_restore_verify_s": populate, "commit_s": commit,
               "attach_ro_verified_s": statistics.median(attach), "writer_reacquire_s": reacquire,
               "mappings": store.pool_info()["mappings"]}
        log(f"store: commit {commit * 1e3:.1f} ms, verified read-only attach {out['attach_ro_verified_s'] * 1e3:.2f} ms")
        return out
    finally:
        store.close()


def bench_owner(torch, gms, timer, m, image, expected):
    """The lease protocol across processes on the llama8b set: an owner process holds the
    allocations; this process, as the writer, populates them from the device image with a fused
    restore+verify and commits; then, as a replacement engine, attaches read-only after
    re-hashing all of it.  Wall times of the synchronous calls; the restore and the re-verify
    are also timed as kernels on the owner's memory (mapped here as external memory)."""
    import signal
    import subprocess
    import tempfile

    sizes = list(m.sizes)
    P, nb = m.payload_bytes, m.num_blocks
    sock = os.path.join(tempfile.mkdtemp(prefix="gms-"), "owner.sock")
    t0 = time.perf_counter()
    p = subprocess.Popen([sys.executable, "-m", "paper_2609_25451_amd.owner", sock, "--device", "0"], cwd=ROOT,
                         stdout=subprocess.PIPE, stderr=subprocess.PIPE, text=True)
    try:
        line = p.stdout.readline()
        assert line.startswith("owner ready"), line + p.stderr.read()
        start = time.perf_counter() - t0
        cnt = torch.zeros(1, dtype=torch.int64, device="cuda")
        t0 = time.perf_counter()
        w = gms.Client(sock, gms.LEASE_RW)
        addrs = [w.alloc(n) for n in sizes]
        alloc = time.perf_counter() - t0
        entries = list(zip(addrs, sizes))
        wm = w.manifest_over(entries)
        tr = settled(timer, lambda: gms.restore(wm, image, expected=expected, mismatch_count=cnt), warm=2, reps=5)
        assert int(cnt.item()) == 0
        wm.close()
        t0 = time.perf_counter()
        w.commit(entries, expected=expected)
        commit = time.perf_counter() - t0
        w.close()
        attach = []
        for _ in range(3):
            t0 = time.perf_counter()
            r = gms.Client(sock, gms.LEASE_RO, verify=True)
            attach.append(time.perf_counter() - t0)
            rm = r.manifest()
            tv = settled(timer, lambda: gms.verify(rm, expected=expected, mismatch_count=cnt), warm=2, reps=5)
            assert int(cnt.item()) == 0
            r.close()
        state, readers, invalid, allocs = gms.owner_query(sock)
        assert (state, readers, invalid) == ("COMMITTED", 0, False)
        out = {"payload_bytes": P, "owner_start_s": start, "allocations": allocs, "writer_alloc_s": alloc,
               "populate_restore_verify_s": tr, "populate_hbm_frac": (2 * P + 8 * nb) / tr / 1e9 / HBM_PEAK_GBS,
               "commit_s": commit, "attach_ro_verified_s": statistics.median(attach),
               "attach_runs_s": [round(a, 4) for a in attach], "reverify_s": tv,
               "reverify_hbm_frac": (P + 8 * nb) / tv / 1e9 / HBM_PEAK_GBS}
        log(f"owner process: {allocs} allocations, populate {tr * 1e3:.2f} ms "
            f"({out['populate_hbm_frac'] * 100:.1f}% of HBM peak), commit {commit * 1e3:.1f} ms, "
            f"verified attach from another lease {out['attach_ro_verified_s'] * 1e3:.1f} ms")
        return out
    finally:
        p.send_signal(signal.SIGTERM)
        try:
            p.wait(timeout=60)
        except subprocess.TimeoutExpired:
            p.kill()
            p.wait()


def bench_recovery(torch, np, gms, synth, m, image, expected):
    """The recovery data path as the paper composes it: the llama8b weights stay resident in a
    committed store, the engine's live KV blocks were saved to a pageable host image (a process
    snapshot's staged device state) and its KV pages released.  Recovery, timed step by step
    (wall clock, each step synchronous): a verified read-only attach to the weights (re-hashed in
    place), the KV pages remapped at their retained addresses, and the live KV blocks restored
    from the host image with fused verification.  The failure and the recovery repeat three
    times; every run is reported with the median (the host link can run at half rate for about
    two seconds after earlier rows free device memory)."""
    sizes = list(m.sizes)
    p = synth.kv_pool()
    store = gms.Store(va_bytes=m.payload_bytes + (8 << 30), slab_bytes=2 << 30)
    pool = gms.Pool(va_bytes=p.layers * p.layer_bytes + (1 << 30), slab_bytes=p.layer_bytes)
    try:
        # the weights, committed (the engine's first start)
        w = store.connect_rw()
        addrs = [w.alloc(n) for n in sizes]
        sm = gms.Manifest(list(zip(addrs, sizes)), device=0)
        gms.restore(sm, image, sm.image_bytes)
        torch.cuda.synchronize()
        w.commit(list(zip(addrs, sizes)), expected=expected)
        sm.close()
        engine = store.connect_ro()
        # the KV pool and its live blocks, saved with their block hashes to pageable host memory
        kv = [pool.alloc(p.layer_bytes) for _ in range(p.layers)]
        for l, a in enumerate(kv):
            synth.dev_fill_bf16(a, p.layer_bytes // 2, p.seed, l)
        live = synth.live_map(p.blocks, p.n_live, p.map_seed, p.map_stream)
        km = gms.Manifest([(kv[l] + int(b) * p.unit_bytes, p.unit_bytes) for l in range(p.layers) for b in live],
                          device=0)
        kv_exp = torch.zeros(km.num_blocks, dtype=torch.int64, device="cuda")
        host = np.empty(km.image_bytes, dtype=np.uint8)
        gms.snapshot_to_host(km, host, blk_hash=kv_exp)
        cnt = torch.zeros(1, dtype=torch.int64, device="cuda")
        runs = []
        for _ in range(3):
            # the failure: the engine's lease ends and its KV pages are released
            engine.close()
            for a in kv:  # one mapping per layer; mappings need not be contiguous
                pool.release(a, p.layer_bytes)
            torch.cuda.synchronize()
            # the recovery
            t0 = time.perf_counter()
            engine = store.connect_ro(verify=True)
            t1 = time.perf_counter()
            for a in kv:
                pool.remap(a, p.layer_bytes)
            t2 = time.perf_counter()
            gms.restore_from_host(km, host, expected=kv_exp, mismatch_count=cnt)
            torch.cuda.synchronize()
            t3 = time.perf_counter()
            assert int(cnt.item()) == 0
            # the same restore again, into pages it has now touched
            gms.restore_from_host(km, host, expected=kv_exp, mismatch_count=cnt)
            torch.cuda.synchronize()
            t4 = time.perf_counter()
            runs.append((t1 - t0, t2 - t1, t3 - t2, t3 - t0, t4 - t3))
        engine.close()
        kv_live = km.payload_bytes
        km.close()
        med = sorted(runs, key=lambda r: r[3])[1]
        out = {"weights_resident_bytes": m.payload_bytes, "kv_live_bytes": kv_live,
               "attach_weights_verified_s": med[0], "remap_kv_pages_s": med[1],
               "restore_kv_from_host_verified_s": med[2], "total_s": med[3],
               "runs_total_s": [round(r[3], 4) for r in runs],
               "restore_kv_repeated_s": statistics.median(r[4] for r in runs)}
        log(f"recovery: {out['total_s'] * 1e3:.1f} ms (attach {med[0] * 1e3:.1f}, remap {med[1] * 1e3:.1f}, "
            f"KV restore {med[2] * 1e3:.1f}); runs {out['runs_total_s']}")
        return out
    finally:
        pool.close()
        store.close()


def bench_kv_vmm(torch, np, gms, synth, timer):
    """The 8 GiB KV pool in VMM slabs: pages released and remapped at the same
    addresses, then the live blocks restored (and verified) into the fresh pages."""
    p = synth.kv_pool()
    pool = gms.Pool(va_bytes=p.layers * p.layer_bytes + (1 << 30), slab_bytes=p.layer_bytes)
    try:
        kv = [pool.alloc(p.layer_bytes) for _ in range(p.layers)]
        for l, a in enumerate(kv):
            synth.dev_fill_bf16(a, p.layer_bytes // 2, p.seed, l)
        live = synth.live_map(p.blocks, p.n_live, p.map_seed, p.map_stream)
        ents = [(kv[l] + int(b) * p.unit_bytes, p.unit_bytes) for l in range(p.layers) for b in live]
        m = gms.Manifest(ents, device=0)
        img = torch.empty(m.image_bytes, dtype=torch.uint8, device="cuda")
        exp = torch.zeros(m.num_blocks, dtype=torch.int64, device="cuda")
        gms.snapshot(m, img, m.image_bytes, blk_hash=exp)
        torch.cuda.synchronize()
        span = p.layers * p.layer_bytes
        t0 = time.perf_counter()
        for a in kv:  # one mapping per layer; mappings need not be contiguous
            pool.release(a, p.layer_bytes)
        t_rel = time.perf_counter() - t0
        t0 = time.perf_counter()
        for a in kv:
            pool.remap(a, p.layer_bytes)
        t_map = time.perf_counter() - t0
        cnt = torch.zeros(1, dtype=torch.int64, device="cuda")
        t = settled(timer, lambda: gms.restore(m, img, m.image_bytes, expected=exp, mismatch_count=cnt))
        assert int(cnt.item()) == 0
        payload = m.payload_bytes
        m.close()
        return {"pool_bytes": span, "release_s": t_rel, "remap_s": t_map, "restore_verify_s": t,
                "restore_verify_GB_s": payload / t / 1e9, "hbm_frac": 2 * payload / t / 1e9 / HBM_PEAK_GBS,
                "mappings": pool.info()["mappings"]}
    finally:
        pool.close()


# Worker threads for the CPU oracle: the box grants each GPU a share of 16 CPUs, whatever
# the affinity mask or os.cpu_count() show there.
CPU_SHARE = 16


def bench_cpu(torch, np, image, m, specs, expected):
    """The CPU oracle, as it stands, over the whole llama8b set (291 tensors, 16.06 GB): a
    snapshot (pack + block hashes of every tensor) and a restore+verify (unpack, then
    block-hash compare against the snapshot's hashes), each timed as the median of 3 passes
    on one thread and on the CPU share's threads, the tensors spread over a thread pool
    largest first; the oracle's C calls release the interpreter lock.  The oracle's block
    hashes of the whole set are also compared with the GPU snapshot's."""
    from concurrent.futures import ThreadPoolExecutor

    import oracle

    off, _ = m.layout()
    pad = lambda n: -(-n // 4096) * 4096  # noqa: E731
    img = image.cpu().numpy()
    total = sum(sp.nbytes for sp in specs)
    jobs = [[img[off[i]:off[i] + pad(sp.nbytes)], np.empty(sp.nbytes, dtype=np.uint8), None]
            for i, sp in enumerate(specs)]
    order = sorted(range(len(jobs)), key=lambda i: -jobs[i][1].nbytes)
    threads = max(1, min(CPU_SHARE, len(os.sched_getaffinity(0))))

    def expect(j):
        oracle.unpack_into(j[0], [j[1]])
        j[2] = oracle.hashes([j[1]])[0]

    def restore_verify(j):
        oracle.unpack_into(j[0], [j[1]])
        return oracle.verify([j[1]], j[2])[0]

    def snapshot(j):
        packed = oracle.pack([j[1]])
        blk, _ = oracle.hashes([j[1]])
        return int(packed.nbytes != j[0].nbytes or not np.array_equal(blk, j[2]))

    def passes(fn, nthreads, reps=3):
        out = []
        for _ in range(reps):
            t0 = time.perf_counter()
            if nthreads == 1:
                bad = sum(fn(jobs[i]) for i in order)
            else:
                with ThreadPoolExecutor(nthreads) as ex:
                    bad = sum(ex.map(fn, [jobs[i] for i in order]))
            out.append(time.perf_counter() - t0)
            assert bad == 0
        return statistics.median(out)

    with ThreadPoolExecutor(threads) as ex:
        list(ex.map(expect, [jobs[i] for i in order]))
    o_blk = np.concatenate([j[2] for j in jobs])
    assert np.array_equal(o_blk, expected.cpu().numpy().view(np.uint64)), "oracle block hashes != GPU snapshot"
    rv_n = passes(restore_verify, threads)
    sn_n = passes(snapshot, threads)
    rv_1 = passes(restore_verify, 1)
    sn_1 = passes(snapshot, 1)
    log(f"cpu oracle over {total} B: restore+verify {rv_1:.2f} s on 1 thread, {rv_n:.2f} s on {threads}; "
        f"snapshot {sn_1:.2f} s / {sn_n:.2f} s")
    del img, jobs
    return {"value": round(total / rv_n / 1e9, 4), "unit": "GB/s", "cores": threads, "kind": "oracle",
            "sample": f"restore+verify (unpack + block-hash compare) of the whole llama8b set ({len(specs)} tensors, "
                      f"{total} B), {threads} threads over tensors, median of 3 passes",
            "seconds": round(rv_n, 3), "single_thread_value": round(total / rv_1 / 1e9, 4),
            "single_thread_seconds": round(rv_1, 3),
            "snapshot": {"what": "pack + block hashes of every tensor", "seconds": round(sn_n, 3),
                         "GB_s": round(total / sn_n / 1e9, 4), "single_thread_seconds": round(sn_1, 3),
                         "single_thread_GB_s": round(total / sn_1 / 1e9, 4)},
            "block_hashes_equal_gpu": True, "host": host_info()}


if __name__ == "__main__":
    main()
