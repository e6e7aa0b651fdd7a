#!/usr/bin/env python3
"""Benchmark of the DAMP decode-step state update on one MI355X.

Workload (the headline): GDN decode, one layer, B = 256 requests, 16 key /
32 value heads, d_k = d_v = 128, the state pre-warmed over 512 FP32 tokens
with 8 outlier key channels per head scaled by 10, 16 protected channels per
head chosen by the channel selection from 64 stride-8 samples; bf16 inputs
and bf16 output. One step = one launch of the fused update over the batch.

Timing: W untimed steps, then exactly K steps between two synchronisations
(ms_per_step = wall time / K). The pool holds `--rotations` disjoint copies
of the batch's slots and consecutive steps use different copies, so the
state (158 MB per copy) is not served from the 256 MB last-level cache.
Each copy holds the batch in consecutive slots, as a [B, HV, d, d] state
would be; the same workload with the batch scattered over the whole pool
in random order is reported beside it (`headline_random_slots`). A HIP
event pair on the launch stream brackets the timed region; its duration
over K is the kernel duration the roofline uses.

Also reported: the FP32-state and uniform-INT8 kernels on the same workload,
KDA decode (B = 256, 32 heads, per-channel decay, selection from a
2048-token calibration run), and the CPU oracle timed on the host.

    python bench.py [--steps K] [--warmup W] [--gpus 1] [--quick]
"""
from __future__ import annotations

import argparse
import hashlib
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

HBM_PEAK_GBS = 8000.0  # MI355X HBM3E
PROFILE = os.path.join(ROOT, "profiles", "update_gdn_mixed_b256.txt")
KERNEL_SOURCES = ["paper_2608_27513_amd/csrc/update_stream.hip", "paper_2608_27513_amd/csrc/update.hpp",
                  "paper_2608_27513_amd/csrc/device.hpp"]
# the sources each profiled kernel is built from (the hash in its summary)
PROFILED_SOURCES = {
    "update_stream128": KERNEL_SOURCES,
    "update_fp32_128": ["paper_2608_27513_amd/csrc/update_fp32.hip", "paper_2608_27513_amd/csrc/update.hpp",
                        "paper_2608_27513_amd/csrc/device.hpp"],
    "prefill_blk128": ["paper_2608_27513_amd/csrc/prefill.hip", "paper_2608_27513_amd/csrc/device.hpp"],
    "pack_unpack": ["paper_2608_27513_amd/csrc/pack.hip", "paper_2608_27513_amd/csrc/device.hpp"],
    "copy_inplace_nt": ["paper_2608_27513_amd/bench_csrc/copy_ceiling.hip"],
    "copy_tiles_nt": ["paper_2608_27513_amd/bench_csrc/copy_ceiling.hip"],
}


# --only: one measurement of the full run (same set-up and timing), so that a
# profiler run covers a single kernel on a single workload
FP16_, U8_ = 2, 3
ONLY = {
    "gdn_mixed": ("gdn", 1, 16, None), "gdn_int8": ("gdn", 1, 0, None), "gdn_fp32": ("gdn", 0, 0, None),
    "gdn_mixed_scattered": ("gdn", 1, 16, None),  # the headline batch at random slots of the pool
    "gdn_int8_h32": ("gdn", 1, 16, (FP16_, 32, FP16_, 1, U8_)),
    "gdn_int8_g32": ("gdn", 1, 16, (FP16_, 32, FP16_, 0, U8_)),
    "gdn_int4_h32": ("gdn", 1, 16, (FP16_, 32, FP16_, 1, 4)),
    "gdn_int4_g32": ("gdn", 1, 16, (FP16_, 32, FP16_, 0, 4)),
    "gdn_fp8": ("gdn", 1, 16, (FP16_, 32, 0, 0, 5)), "gdn_nvfp4": ("gdn", 1, 16, (FP16_, 16, 5, 0, 6)),
    "kda_mixed": ("kda", 1, 16, None), "kda_fp32": ("kda", 0, 0, None),
    "prefill_gdn": None, "prefill_kda": None, "pack_unpack": None, "copy": ("gdn", None, None, None),
    "copy_tiles": ("gdn", None, None, None), "copy_tiles_scattered": ("gdn", None, None, None),
}


def parse():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=200)
    ap.add_argument("--warmup", type=int, default=20)
    ap.add_argument("--rotations", type=int, default=8)
    ap.add_argument("--prewarm", type=float, default=PREWARM_S,
                    help="seconds of launches before the warm-up steps of each measurement")
    ap.add_argument("--quick", action="store_true", help="headline only: no baselines, no CPU")
    ap.add_argument("--no-cpu", action="store_true")
    ap.add_argument("--cpu-seconds", type=float, default=10.0)
    ap.add_argument("--no-sweep", action="store_true")
    ap.add_argument("--no-multilayer", action="store_true")
    ap.add_argument("--copy-calibration", action="store_true",
                    help="only run a plain 1 GiB device copy (counter calibration)")
    ap.add_argument("--cpu-only", type=float, default=0.0, metavar="SECONDS",
                    help="only time the CPU oracle for SECONDS and print its JSON (no GPU)")
    ap.add_argument("--only", choices=sorted(ONLY), default=None,
                    help="run one measurement (for per-kernel profiles) and print its JSON")
    return ap.parse_args()


def copy_calibration(torch, reps: int = 5):
    """A plain device-to-device copy of exactly 1 GiB, `reps` times: the known
    byte count that HBM counters (FETCH_SIZE, WRITE_SIZE) are scaled by."""
    n = 1 << 30
    src = torch.ones(n, dtype=torch.uint8, device="cuda")
    dst = torch.empty_like(src)
    torch.cuda.synchronize()
    for _ in range(reps):
        dst.copy_(src)
    torch.cuda.synchronize()
    print(json.dumps({"copy_bytes_read": n, "copy_bytes_written": n, "reps": reps}), flush=True)


def kernel_source_hash(paths=None) -> str:
    h = hashlib.sha256()
    for p in (KERNEL_SOURCES if paths is None else paths):
        h.update(open(os.path.join(ROOT, p), "rb").read())
    return h.hexdigest()[:16]


def algorithmic_bytes(tile_bytes: int, B: int, HK: int, HV: int, d: int, kda: bool,
                      o_bytes: int = 2) -> int:
    """Bytes one launch must move: every tile read and written once, plus
    q, k per key head, v, o per value head, the decay (per head or per
    channel), beta, the slot ids and the permutation."""
    state = 2 * tile_bytes * B * HV
    qk = 2 * B * HK * d * 2
    vo = B * HV * d * (2 + o_bytes)
    g = B * HV * (d if kda else 1) * 2
    beta = B * HV * 2
    return state + qk + vo + g + beta + 4 * B + HV * d


def profile_traffic():
    """(fetch + write bytes per launch, scale note) from the committed counter
    summary, or None when the kernel sources changed since it was taken."""
    if not os.path.exists(PROFILE):
        return None
    kv = {}
    for line in open(PROFILE):
        if ":" in line and not line.startswith("#"):
            k, v = line.split(":", 1)
            kv[k.strip()] = v.strip()
    if kv.get("kernel_source_sha256") != kernel_source_hash():
        return None
    try:
        return float(kv["hbm_bytes_per_launch"])
    except (KeyError, ValueError):
        return None


class Workload:
    """Pools, inputs and prepared launches of one decode configuration."""

    def __init__(self, torch, D, inputs, *, kda: bool, B: int, HK: int, HV: int, d: int,
                 k_hi: int, rotations: int, seed: int, log=print):
        self.torch, self.D, self.inputs = torch, D, inputs
        self.kda, self.B, self.HK, self.HV, self.d, self.k_hi = kda, B, HK, HV, d, k_hi
        self.rotations = rotations
        dev = "cuda"
        gen = torch.Generator(device=dev)
        gen.manual_seed(seed)
        self.mu = None
        if kda:
            self.mu = torch.from_numpy(inputs.kda_mu(seed, HV, d)).to(dev)

        # 1. FP32 warm-up of every request over 512 tokens from the zero state
        t0 = time.time()
        fp_layout = D.damp_layout_init(d, d, 0, D.DAMP_STATE_FP32)
        warm = D.Pool(fp_layout, 1, B, HV)
        slots = torch.arange(B, dtype=torch.int32, device=dev)
        D.damp_pool_reset_slots(warm, 0, slots)
        o = torch.empty((B, HV, d), dtype=torch.float32, device=dev)
        samples, logs = [], []
        for t in range(512):
            x = inputs.decode_inputs_device(gen, B, HK, HV, d, kda=kda, mu=self.mu)
            fn = D.damp_state_update_kda if kda else D.damp_state_update_gdn
            fn(warm, 0, slots, x["q"], x["k"], x["v"], x["g"], x["beta"], o=o)
            if not kda and (t + 1) % 8 == 0:  # calibration samples of request 0
                samples.append(D.damp_state_unpack(warm, 0, slots[:1])[0])
                logs.append(x["g"][0].float())
        S = D.damp_state_unpack(warm, 0, slots)
        del warm
        # 2. outlier channels (GDN): 8 key channels per head scaled by 10
        if not kda:
            ch = torch.from_numpy(inputs.outlier_channels(seed, HV, d, 8)).long().to(dev)
            rows = torch.zeros((HV, d), dtype=torch.float32, device=dev)
            rows.scatter_(1, ch, 9.0)
            scale = (1.0 + rows)[None, :, :, None]
            S *= scale
            cal = torch.stack(samples) * scale
            cal_logs = torch.stack(logs)
        else:
            # separate 2048-token calibration sequence (one request), stride 8
            cg = torch.Generator(device=dev)
            cg.manual_seed(seed + 1)
            cpool = D.Pool(fp_layout, 1, 1, HV)
            one = slots[:1]
            D.damp_pool_reset_slots(cpool, 0, one)
            o1 = torch.empty((1, HV, d), dtype=torch.float32, device=dev)
            cs, cl = [], []
            for t in range(2048):
                x = inputs.decode_inputs_device(cg, 1, HK, HV, d, kda=True, mu=self.mu)
                D.damp_state_update_kda(cpool, 0, one, x["q"], x["k"], x["v"], x["g"], x["beta"],
                                        o=o1)
                if (t + 1) % 8 == 0:
                    cs.append(D.damp_state_unpack(cpool, 0, one)[0])
                    cl.append(x["g"][0].float())
            cal = torch.stack(cs)
            cal_logs = torch.stack(cl)
        # 3. channel selection (Alg. 1) on the device-resident samples
        _, perm, _ = D.damp_select_channels(cal.contiguous(), cal_logs.contiguous(), k_hi, kda=kda)
        self.perm = perm.to(dev)
        self.n_cal = cal.shape[0]
        del cal, cal_logs
        self.S = S
        self.setup_s = time.time() - t0
        log(f"  warm-up, calibration (N={self.n_cal}) and selection in {self.setup_s:.1f} s")

        # per-step inputs (a few distinct sets, cycled)
        self.step_inputs = [inputs.decode_inputs_device(gen, B, HK, HV, d, kda=kda, mu=self.mu)
                            for _ in range(4)]

    def make_pool(self, kind: int, k_hi: int, rotations: int, scattered: bool = False,
                  tiers=None):
        """A pool with `rotations` disjoint slot sets, each packed with the
        warm state (permuted by the selection). Set r is slots r*B .. r*B+B-1
        in order, or with `scattered` B slots drawn at random from the whole
        pool, in random order. `tiers` = (hi_dtype, group, meta_dtype,
        hadamard[, code_dtype]) selects another storage format than the default."""
        torch, D = self.torch, self.D
        B, HV, d = self.B, self.HV, self.d
        layout = D.damp_layout_init(d, d, k_hi, kind)
        if tiers is not None:
            (layout.hi_dtype, layout.group, layout.meta_dtype, layout.hadamard,
             layout.code_dtype) = (tuple(tiers) + (D.DAMP_DT_U8,))[:5]
        pool = D.Pool(layout, 1, B * rotations, HV)
        if scattered:
            order = torch.from_numpy(self.inputs.slot_order(7, B * rotations, B * rotations)).cuda()
        else:
            order = torch.arange(B * rotations, dtype=torch.int32, device="cuda")
        slot_sets = [order[r * B:(r + 1) * B].contiguous() for r in range(rotations)]
        for s in slot_sets:
            D.damp_state_pack(pool, 0, s, self.S, self.perm)
        torch.cuda.synchronize()
        return pool, slot_sets, layout

    def prepared(self, pool, slot_sets, o_dtype):
        torch, D = self.torch, self.D
        o = torch.empty((self.B, self.HV, self.d), dtype=o_dtype, device="cuda")
        calls = []
        for r, s in enumerate(slot_sets):
            for x in self.step_inputs:
                calls.append(D.PreparedUpdate(self.kda, pool, 0, s, x["q"], x["k"], x["v"],
                                              x["g"], x["beta"], self.perm, 1.0, o))
        # interleave so consecutive steps use different slot sets
        n_in = len(self.step_inputs)
        return [calls[(i % len(slot_sets)) * n_in + (i // len(slot_sets)) % n_in]
                for i in range(len(calls))]


PREWARM_S = 0.5


def time_steps(torch, calls, warmup: int, steps: int, prewarm_s: float = None):
    """`steps` back-to-back launches between two synchronisations: wall time,
    and the HIP-event time over the same region on the launch stream (its
    mean per launch is the kernel duration the roofline uses). Before the
    `warmup` untimed launches the same calls run for `prewarm_s` seconds, so
    that the GPU has left its idle clocks: a decode loop runs the kernel back
    to back, and the first ~50 ms of launches after idle run up to 10% slower."""
    n = len(calls)
    t_end = time.perf_counter() + (PREWARM_S if prewarm_s is None else prewarm_s)
    i = 0
    while time.perf_counter() < t_end:
        for _ in range(32):
            calls[i % n]()
            i += 1
        torch.cuda.synchronize()
    for i in range(warmup):
        calls[i % n]()
    torch.cuda.synchronize()
    start, end = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    t0 = time.perf_counter()
    start.record()
    for i in range(steps):
        calls[(warmup + i) % n]()
    end.record()
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    ev = start.elapsed_time(end) * 1e-3
    return dict(wall_s=wall, mean_launch_s=ev / steps)


def measure(torch, D, wl: Workload, kind: int, k_hi: int, rotations: int, warmup: int,
            steps: int, o_dtype, scattered: bool = False, tiers=None, per_launch: bool = False):
    pool, sets, layout = wl.make_pool(kind, k_hi, rotations, scattered, tiers)
    calls = wl.prepared(pool, sets, o_dtype)
    t = time_steps(torch, calls, warmup, steps)
    stats = launch_stats(torch, calls) if per_launch else None
    tb = D.damp_tile_bytes(layout)
    nbytes = algorithmic_bytes(tb, wl.B, wl.HK, wl.HV, wl.d, wl.kda,
                               2 if o_dtype == torch.bfloat16 else 4)
    res = dict(
        us_per_step=1e6 * t["wall_s"] / steps,
        kernel_us=1e6 * t["mean_launch_s"],
        bytes_per_step=nbytes,
        gbs=nbytes * steps / t["wall_s"] / 1e9,
        kernel_gbs=nbytes / t["mean_launch_s"] / 1e9,
        tile_bytes=tb,
        bits_per_value=D.damp_bits_per_value(layout),
    )
    res["kernel_frac_peak"] = res["kernel_gbs"] / HBM_PEAK_GBS
    if stats is not None:
        stats["frac_hbm_peak_at_median"] = round(nbytes / (stats["median_us"] * 1e-6) / 1e9 /
                                                 HBM_PEAK_GBS, 4)
        res["launch_stats"] = stats
    del pool, calls
    torch.cuda.empty_cache()
    return res


def sweep(torch, D, inputs, steps: int, log=print):
    """B x high-precision rows x state layout, GDN (16 key heads) and KDA, 32
    value heads, d = 128. States are random packed tiles (timing does not
    depend on their values); pools span >= 1 GB so they are not cache
    resident. Returns one record per point."""
    out = []
    d, HV = 128, 32
    for kda in (False, True):
        HK = HV if kda else 16
        for B in (1, 16, 64, 256, 1024):
            gen = torch.Generator(device="cuda")
            gen.manual_seed(B)
            mu = torch.from_numpy(inputs.kda_mu(1, HV, d)).cuda() if kda else None
            x = inputs.decode_inputs_device(gen, B, HK, HV, d, kda=kda, mu=mu)
            perm = torch.from_numpy(inputs.random_perms(B, HV, d)).cuda()
            S = torch.randn((B, HV, d, d), generator=gen, device="cuda") * 0.1
            o = torch.empty((B, HV, d), dtype=torch.bfloat16, device="cuda")
            for kind, k_hi in ((D.DAMP_STATE_FP32, 0), (D.DAMP_STATE_MIXED, 0),
                               (D.DAMP_STATE_MIXED, 8), (D.DAMP_STATE_MIXED, 16),
                               (D.DAMP_STATE_MIXED, 32)):
                layout = D.damp_layout_init(d, d, k_hi, kind)
                tb = D.damp_tile_bytes(layout)
                rot = max(1, min(16, -(-(1 << 30) // (tb * B * HV))))
                pool = D.Pool(layout, 1, B * rot, HV)
                sets = [torch.arange(r * B, (r + 1) * B, dtype=torch.int32, device="cuda")
                        for r in range(rot)]
                for sl in sets:
                    D.damp_state_pack(pool, 0, sl, S, perm)
                calls = [D.PreparedUpdate(kda, pool, 0, sl, x["q"], x["k"], x["v"], x["g"],
                                          x["beta"], perm, 1.0, o) for sl in sets]
                t = time_steps(torch, calls, 10, steps, prewarm_s=0.1)
                nbytes = algorithmic_bytes(tb, B, HK, HV, d, kda, 2)
                out.append(dict(model="KDA" if kda else "GDN", B=B,
                                layout="fp32" if kind == D.DAMP_STATE_FP32 else
                                ("int8" if k_hi == 0 else "mixed"), k_hi=k_hi,
                                kernel_us=round(1e6 * t["mean_launch_s"], 2),
                                GBs=round(nbytes / t["mean_launch_s"] / 1e9, 1)))
                del pool, calls
            del S
            torch.cuda.empty_cache()
        log(f"  sweep {'KDA' if kda else 'GDN'} done")
    return out


def copy_ceiling(torch, D, wl, rotations: int, steps: int, log=print, linear: bool = True,
                 walks=("consecutive", "scattered")):
    """The practical ceiling of the update's state traffic: an in-place copy
    (every 16-byte piece read and written back, non-temporal, like the
    update's tile accesses; `libcopyceiling.so`, built beside libdamp) over
    the same rotated pool regions the headline updates, timed like the update
    (steady clock, HIP events around `steps` launches); the fastest of a few
    grid sizes. Then the tile-walk copies (`walks`): the tiles of each step
    copied in place in the update's own order and launch shape, at the
    batch's consecutive slots and at slots scattered over the pool."""
    import ctypes

    from paper_2608_27513_amd import build as B

    lib = ctypes.CDLL(B.BENCH_LIB)
    lib.copy_ceiling_inplace.restype = ctypes.c_int
    lib.copy_ceiling_inplace.argtypes = [ctypes.c_void_p, ctypes.c_size_t, ctypes.c_int,
                                         ctypes.c_int, ctypes.c_void_p]
    pool, sets, layout = wl.make_pool(D.DAMP_STATE_MIXED, wl.k_hi, rotations)
    region = wl.B * wl.HV * pool.tile_stride  # one rotation's slots are contiguous
    base = pool.buffer.data_ptr()
    stream = ctypes.c_void_p(torch.cuda.current_stream().cuda_stream)
    best = None
    for grid, unroll in ((1024, 1), (512, 2), (768, 2), (256, 4)) if linear else ():  # ~4 MB in flight
        def call(r, grid=grid, unroll=unroll):
            rc = lib.copy_ceiling_inplace(ctypes.c_void_p(base + r * region), region, grid, unroll,
                                          stream)
            if rc != 0:
                raise RuntimeError(f"copy_ceiling_inplace returned {rc}")
        calls = [lambda r=r: call(r) for r in range(rotations)]
        t = time_steps(torch, calls, 20, steps, prewarm_s=0.1)
        if best is None or t["mean_launch_s"] < best[1]:
            best = ((grid, unroll), t["mean_launch_s"])
    res = dict(bytes=2 * region)
    if linear:
        sec = best[1]
        res.update(grid=best[0][0], unroll=best[0][1], copy_us=round(1e6 * sec, 2),
                   copy_gbs=round(2 * region / sec / 1e9, 1),
                   copy_frac_hbm_peak=round(2 * region / sec / 1e9 / HBM_PEAK_GBS, 4),
                   kernel="in-place 16-byte non-temporal copy of the rotated pool regions")
        log(f"  in-place copy of the same state bytes: {res['copy_us']} us, {res['copy_gbs']} GB/s "
            f"(grid {best[0][0]}, {best[0][1]} per thread)")
    # the same tiles copied in the update's own walk and launch shape, with the
    # batch at consecutive slots and at slots scattered over the whole pool
    lib.copy_tiles_inplace.restype = ctypes.c_int
    lib.copy_tiles_inplace.argtypes = [ctypes.c_void_p, ctypes.c_void_p, ctypes.c_int, ctypes.c_int,
                                       ctypes.c_uint64, ctypes.c_uint64, ctypes.c_int, ctypes.c_int,
                                       ctypes.c_int, ctypes.c_void_p]
    cus = torch.cuda.get_device_properties(0).multi_processor_count
    per_head = max(1, min((3 * cus) // wl.HV, wl.B))  # the update's three workgroups per CU
    tb = D.damp_tile_bytes(layout)
    n = wl.B * rotations
    order = torch.from_numpy(wl.inputs.slot_order(7, n, n)).cuda()
    all_walks = {"consecutive": sets, "scattered": [order[r * wl.B:(r + 1) * wl.B].contiguous()
                                                    for r in range(rotations)]}
    walks = {k: all_walks[k] for k in walks}
    res["tile_walk"] = dict(grid=per_head * wl.HV, tile_bytes=tb,
                            kernel="in-place copy of each step's tiles in the update's order")
    for name, slot_sets in walks.items():
        def tcall(sl):
            rc = lib.copy_tiles_inplace(ctypes.c_void_p(base), ctypes.c_void_p(sl.data_ptr()), wl.B,
                                        wl.HV, wl.HV * pool.tile_stride, pool.tile_stride, tb, n,
                                        per_head * wl.HV, stream)
            if rc != 0:
                raise RuntimeError(f"copy_tiles_inplace returned {rc}")
        calls = [lambda sl=sl: tcall(sl) for sl in slot_sets]
        t = time_steps(torch, calls, 20, steps, prewarm_s=0.1)
        res["tile_walk"][f"{name}_us"] = round(1e6 * t["mean_launch_s"], 2)
        log(f"  tile-walk copy, {name} slots: {res['tile_walk'][f'{name}_us']} us")
    del pool
    torch.cuda.empty_cache()
    return res


def launch_stats(torch, calls, groups: int = 10, per_group: int = 20):
    """Kernel duration over groups x per_group launches (after the calls have
    run at the steady clock): each group of back-to-back launches is
    bracketed by its own HIP event pair on the launch stream, and the
    duration per launch of each group is reported as the median, minimum and
    maximum over the groups. An event pair around every single launch would
    break the back-to-back stream and add each launch's own ramp."""
    import statistics

    evs = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))
           for _ in range(groups)]
    i = 0
    for a, b in evs:
        a.record()
        for _ in range(per_group):
            calls[i % len(calls)]()
            i += 1
        b.record()
    torch.cuda.synchronize()
    d = [1e3 * a.elapsed_time(b) / per_group for a, b in evs]
    return dict(launches=groups * per_group, groups=groups, median_us=round(statistics.median(d), 3),
                min_us=round(min(d), 3), max_us=round(max(d), 3))


def pack_unpack_bench(torch, D, steps: int, log=print):
    """Pack (natural-order FP32 state -> packed tiles, Eq. (3)) and unpack
    (packed -> FP32) of the B=256, 32-head, d=128 GDN state with 16 BF16
    rows, each launch moving the FP32 state (537 MB) one way and the packed
    tiles (158 MB) the other; two FP32 buffers and two pool halves alternate
    so that no launch is served from the last-level cache."""
    B, HV, d, k_hi = 256, 32, 128, 16
    gen = torch.Generator(device="cuda")
    gen.manual_seed(21)
    S = [torch.randn((B, HV, d, d), generator=gen, device="cuda") * 0.1 for _ in range(2)]
    from paper_2608_27513_amd import inputs
    perm = torch.from_numpy(inputs.random_perms(21, HV, d)).cuda()
    layout = D.damp_layout_init(d, d, k_hi)
    pool = D.Pool(layout, 1, 2 * B, HV)
    sets = [torch.arange(r * B, (r + 1) * B, dtype=torch.int32, device="cuda") for r in range(2)]
    tb = D.damp_tile_bytes(layout)
    nbytes = B * HV * (d * d * 4 + tb)
    out = {}
    for name, calls in (
            ("pack", [lambda i=i: D.damp_state_pack(pool, 0, sets[i], S[i], perm) for i in range(2)]),
            ("unpack", [lambda i=i: D.damp_state_unpack(pool, 0, sets[i], perm, S[i])
                        for i in range(2)])):
        t = time_steps(torch, calls, 5, steps, prewarm_s=0.1)
        sec = t["mean_launch_s"]
        out[name] = dict(kernel_us=round(1e6 * sec, 1), GBs=round(nbytes / sec / 1e9, 1),
                         frac_hbm_peak=round(nbytes / sec / 1e9 / HBM_PEAK_GBS, 4))
    out["bytes_per_launch"] = nbytes
    log(f"  pack {out['pack']['kernel_us']} us ({out['pack']['GBs']} GB/s), "
        f"unpack {out['unpack']['kernel_us']} us ({out['unpack']['GBs']} GB/s)")
    del S, pool
    torch.cuda.empty_cache()
    return out


def tp_share(torch, D, inputs, steps: int, log=print):
    """One GPU's share of an 8-way tensor-parallel deployment: B = 256 with 4
    of the 32 value heads (and 2 of 16 key heads for GDN), d = 128, 16
    high-precision rows, against the FP32 state: 1024 tiles, four per CU."""
    out = []
    d, HV, B = 128, 4, 256
    for kda in (False, True):
        HK = HV if kda else 2
        gen = torch.Generator(device="cuda")
        gen.manual_seed(8)
        mu = torch.from_numpy(inputs.kda_mu(1, HV, d)).cuda() if kda else None
        x = inputs.decode_inputs_device(gen, B, HK, HV, d, kda=kda, mu=mu)
        perm = torch.from_numpy(inputs.random_perms(8, HV, d)).cuda()
        S = torch.randn((B, HV, d, d), generator=gen, device="cuda") * 0.1
        o = torch.empty((B, HV, d), dtype=torch.bfloat16, device="cuda")
        for kind, k_hi in ((D.DAMP_STATE_FP32, 0), (D.DAMP_STATE_MIXED, 16)):
            layout = D.damp_layout_init(d, d, k_hi, kind)
            tb = D.damp_tile_bytes(layout)
            rot = max(1, min(64, -(-(1 << 30) // (tb * B * HV))))
            pool = D.Pool(layout, 1, B * rot, HV)
            sets = [torch.arange(r * B, (r + 1) * B, dtype=torch.int32, device="cuda")
                    for r in range(rot)]
            for sl in sets:
                D.damp_state_pack(pool, 0, sl, S, perm)
            calls = [D.PreparedUpdate(kda, pool, 0, sl, x["q"], x["k"], x["v"], x["g"],
                                      x["beta"], perm, 1.0, o) for sl in sets]
            t = time_steps(torch, calls, 10, steps, prewarm_s=0.1)
            nbytes = algorithmic_bytes(tb, B, HK, HV, d, kda, 2)
            out.append(dict(model="KDA" if kda else "GDN", B=B, HK=HK, HV=HV,
                            layout="fp32" if kind == D.DAMP_STATE_FP32 else "mixed", k_hi=k_hi,
                            kernel_us=round(1e6 * t["mean_launch_s"], 2),
                            GBs=round(nbytes / t["mean_launch_s"] / 1e9, 1)))
            del pool, calls
        del S
        torch.cuda.empty_cache()
    log("  TP=8 share: " + ", ".join(f"{r['model']} {r['layout']} {r['kernel_us']} us"
                                      for r in out))
    return out


def multilayer(torch, D, inputs, steps: int, log=print):
    """48 GDN layers over one slot-indexed pool of 512 requests, 384 of them
    active in random non-contiguous order (32 value / 16 key heads, d = 128,
    16 BF16 rows). One decode step = 48 launches, captured once as a HIP
    graph and replayed; two input sets alternate between steps. Reports the
    per-step latency for the mixed pool and the FP32-state pool."""
    L, slots_total, B, HK, HV, d, k_hi = 48, 512, 384, 16, 32, 128, 16
    gen = torch.Generator(device="cuda")
    gen.manual_seed(5)
    active = torch.from_numpy(inputs.slot_order(5, slots_total, B)).cuda()
    perms = [torch.from_numpy(inputs.random_perms(100 + l, HV, d)).cuda() for l in range(L)]
    sets = [[inputs.decode_inputs_device(gen, B, HK, HV, d) for _ in range(L)] for _ in range(2)]
    o = torch.empty((B, HV, d), dtype=torch.bfloat16, device="cuda")
    res = {}
    for name, kind, kh in (("mixed", D.DAMP_STATE_MIXED, k_hi), ("fp32_state", D.DAMP_STATE_FP32, 0)):
        layout = D.damp_layout_init(d, d, kh, kind)
        pool = D.Pool(layout, L, slots_total, HV)
        for l in range(L):  # random warm states for the active slots of every layer
            S = torch.randn((B, HV, d, d), generator=gen, device="cuda") * 0.1
            D.damp_state_pack(pool, l, active, S, perms[l])
            del S
        def step(s_):
            for l, x in enumerate(sets[s_]):  # launches go to the current stream
                D.damp_state_update_gdn(pool, l, active, x["q"], x["k"], x["v"], x["g"],
                                        x["beta"], perm=perms[l], o=o)

        graphs = []
        for s_ in range(2):
            step(s_)  # warm the launch path before capture
            torch.cuda.synchronize()
            g = torch.cuda.CUDAGraph()
            with torch.cuda.graph(g):
                step(s_)
            graphs.append((g, s_))
        t_end = time.perf_counter() + PREWARM_S  # leave the idle clocks (time_steps)
        i = 0
        while time.perf_counter() < t_end or i < 4:
            graphs[i % 2][0].replay()
            i += 1
            if i % 8 == 0:
                torch.cuda.synchronize()
        torch.cuda.synchronize()
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        t0 = time.perf_counter()
        e0.record()
        for i in range(steps):
            graphs[i % 2][0].replay()
        e1.record()
        torch.cuda.synchronize()
        wall = time.perf_counter() - t0
        step_s = e0.elapsed_time(e1) * 1e-3 / steps
        nbytes = L * algorithmic_bytes(D.damp_tile_bytes(layout), B, HK, HV, d, False, 2)
        res[name] = dict(ms_per_step=round(1e3 * step_s, 4), wall_ms_per_step=round(1e3 * wall / steps, 4),
                         GBs=round(nbytes / step_s / 1e9, 1), pool_bytes=pool.buffer.numel(),
                         launches_per_step=L)
        del graphs, pool
        torch.cuda.empty_cache()
        log(f"  48-layer step ({name}): {res[name]['ms_per_step']:.3f} ms")
    res["speedup_vs_fp32_state"] = round(res["fp32_state"]["ms_per_step"] / res["mixed"]["ms_per_step"], 3)
    res["config"] = dict(layers=L, pool_slots=slots_total, active=B, HK=HK, HV=HV, d=d, k_hi=k_hi,
                         steps=steps)
    return res


def prefill_bench(torch, D, inputs, steps: int, log=print, T: int = 64, kda: bool = False):
    """Prefill of one T-token chunk per request (App. A.5, prefill path) on
    the B=256 GDN workload (16 key / 32 value heads, d=128, 16 BF16 rows) or
    the KDA one (32 heads, per-channel decay):
    decode the stored state once, T fp32 steps, store once. Reports tokens per
    second and the fp32 rate (7 flops per state value and token: decay, two
    read-outs, the update), against the vector fp32 peak."""
    B, HV, d, k_hi = 256, 32, 128, 16
    HK = HV if kda else 16
    gen = torch.Generator(device="cuda")
    gen.manual_seed(11)
    mu = torch.from_numpy(inputs.kda_mu(1, HV, d)).cuda() if kda else None
    steps_in = [inputs.decode_inputs_device(gen, B, HK, HV, d, kda=kda, mu=mu) for _ in range(T)]
    x = {name: torch.stack([s_[name] for s_ in steps_in], dim=1).contiguous()
         for name in steps_in[0]}
    del steps_in
    perm = torch.from_numpy(inputs.random_perms(12, HV, d)).cuda()
    layout = D.damp_layout_init(d, d, k_hi)
    rot = 2
    pool = D.Pool(layout, 1, B * rot, HV)
    S = torch.randn((B, HV, d, d), generator=gen, device="cuda") * 0.1
    sets = [torch.arange(r * B, (r + 1) * B, dtype=torch.int32, device="cuda") for r in range(rot)]
    for sl in sets:
        D.damp_state_pack(pool, 0, sl, S, perm)
    del S
    o = torch.empty((B, T, HV, d), dtype=torch.bfloat16, device="cuda")
    fn = D.damp_state_prefill_kda if kda else D.damp_state_prefill_gdn
    calls = [lambda sl=sl: fn(pool, 0, sl, x["q"], x["k"], x["v"], x["g"], x["beta"], perm=perm,
                              o=o) for sl in sets]
    t = time_steps(torch, calls, 3, steps)
    sec = t["mean_launch_s"]
    flops = 7.0 * d * d * B * HV * T
    res = dict(B=B, T=T, HK=HK, HV=HV, d=d, k_hi=k_hi, chunk_us=round(1e6 * sec, 1),
               tokens_per_s=round(B * T / sec), tflops=round(flops / sec / 1e12, 2),
               frac_fp32_vector_peak=round(flops / sec / 157.3e12, 4))
    log(f"  prefill {'KDA' if kda else 'GDN'} T={T}: {res['chunk_us']} us per chunk, "
        f"{res['tokens_per_s']:.3g} tokens/s, {res['tflops']} TFLOP/s")
    del pool, x, o
    torch.cuda.empty_cache()
    return res


def calibration_bench(torch, D, inputs, log=print, T: int = 2048, stride: int = 8):
    """On-device calibration on the KDA workload (App. A.2-A.4): a T-token
    FP32 calibration sequence per split (one request, 32 heads, d=128), the
    state write after every `stride` tokens folded into the accumulators,
    then Alg. 1. Two disjoint splits (different sequences) give the
    calibration-split agreement of App. B: mean top-16 overlap and mean
    Spearman correlation of the scores over heads."""
    HV, d, k_hi = 32, 128, 16
    dev = "cuda"
    mu = torch.from_numpy(inputs.kda_mu(1, HV, d)).to(dev)
    res = {}
    for name, tiers in (("int8_h32", (D.DAMP_DT_FP16, 32, D.DAMP_DT_FP16, 1)),
                        ("int8_rows", None)):
        lo = D.damp_layout_init(d, d, 0)
        if tiers is not None:
            lo.hi_dtype, lo.group, lo.meta_dtype, lo.hadamard = tiers
        picks, scores, times = [], [], []
        for split in range(2):
            gen = torch.Generator(device=dev)
            gen.manual_seed(100 + split)
            steps = [inputs.decode_inputs_device(gen, 1, HV, HV, d, kda=True, mu=mu)
                     for _ in range(T)]
            x = {n: torch.stack([st[n] for st in steps], dim=1).contiguous() for n in steps[0]}
            del steps
            pool = D.Pool(D.damp_layout_init(d, d, 0, D.DAMP_STATE_FP32), 1, 1, HV)
            slots = torch.zeros(1, dtype=torch.int32, device=dev)
            cal = D.Calib(lo, kda=True, num_heads=HV)
            D.damp_pool_reset_slots(pool, 0, slots)
            torch.cuda.synchronize()
            t0 = time.perf_counter()
            D.damp_calibrate_sequence(cal, 0, pool, 0, slots, x["q"], x["k"], x["v"], x["g"],
                                      x["beta"], stride=stride)
            r = D.damp_calib_finalize(cal, k_hi)  # synchronises
            times.append(time.perf_counter() - t0)
            picks.append(r["sel"].numpy())
            scores.append(r["score"].numpy())
            del pool, cal, x
        overlap = float(sum(D.damp_topk_overlap(picks[0][h], picks[1][h]) for h in range(HV)) / HV)
        rho = float(sum(D.damp_spearman(scores[0][h], scores[1][h]) for h in range(HV)) / HV)
        res[name] = dict(T=T, stride=stride, samples=T // stride, heads=HV, d=d,
                         ms=round(1e3 * min(times), 2), split_overlap=round(overlap, 4),
                         split_spearman=round(rho, 4))
        log(f"  calibration ({name}): {res[name]['ms']} ms for {T} tokens x {HV} heads, "
            f"split overlap {overlap:.3f}, Spearman {rho:.3f}")
    torch.cuda.empty_cache()
    return res


def accuracy_bench(torch, log=print):
    """Held-out trajectory accuracy (App. E's state and output RRMSE against
    the FP32 state) of uniform INT8 and of 16 protected rows chosen by a
    random, an E-only and the C = E P selector, in the default and the
    paper's INT8+H32 tiers, on the GDN and KDA decode workloads (B = 64, 512
    warm-up tokens, selection from a separate 2048-token calibration
    sequence, 256 held-out decode steps), with the benchmark's isotropic keys
    and with keys whose energy concentrates in 8 channels per key head (x4
    before normalization). The paper's figures are context: real model
    trajectories, INT8+H32 with 16 FP16 rows (App. E)."""
    from paper_2608_27513_amd import accuracy as A

    out = {}
    t0 = time.time()
    for name, kda, kc in (("gdn", False, 0), ("kda", True, 0), ("gdn_key8x4", False, 8),
                          ("kda_key8x4", True, 8)):
        out[name] = A.study(kda=kda, B=64, steps=256, seed=0, key_channels=kc, key_factor=4.0,
                            log=log)
        torch.cuda.empty_cache()
    out["seconds"] = round(time.time() - t0, 1)
    out["paper_context"] = {"gdn_common_16_16": {"state_rrmse": 8.748e-3, "output_rrmse": 2.256e-3},
                            "source": "App. E, held-out Qwen3.6 trajectories, INT8+H32 + 16 FP16 rows"}
    out["parity"] = "unpinned (no printed value for synthetic inputs)"
    return out


def cpu_baseline(seconds: float, log=print):
    """The CPU oracle on the GDN workload (B=256, 16/32 heads, d=128, 16 BF16 rows),
    timed on the host: as many whole decode steps as fit in `seconds`."""
    import numpy as np

    from oracle import oracle as orc
    from paper_2608_27513_amd import inputs

    B, HK, HV, d, k_hi = 256, 16, 32, 128, 16
    S = inputs.synthetic_states(0, B, HV, d)
    inputs.scale_channels(S, inputs.outlier_channels(0, HV, d, 8), 10.0)
    perm = inputs.random_perms(0, HV, d)
    ref = orc.Pool(orc.KIND_MIXED, d, d, k_hi, 1, B, HV)
    slots = np.arange(B, dtype=np.int32)
    orc.pack(ref, 0, slots, S, perm)
    del S
    inp = inputs.step(inputs.decode_inputs(0, 1, B, HK, HV, d), 0)
    n = 0
    t0 = time.perf_counter()
    while True:
        orc.update(ref, 0, slots, kda=False, perm=perm, **inp)
        n += 1
        el = time.perf_counter() - t0
        if el >= seconds or n >= 1000:
            break
    nbytes = algorithmic_bytes(orc.tile_bytes(orc.KIND_MIXED, d, d, k_hi), B, HK, HV, d, False, 4)
    log(f"  cpu oracle: {n} steps in {el:.1f} s")
    return dict(value=nbytes * n / el / 1e9, unit="GB/s", cores=orc.max_threads(), kind="oracle",
                sample=f"{n} whole decode steps of the B=256, 32-head, d=128 GDN workload "
                       f"(fp32 o), {el:.1f} s", ms_per_step=1e3 * el / n)


def cpu_single_thread(seconds: float, log=print):
    """The same oracle timing on one host thread, in a child process started
    with OMP_NUM_THREADS=1 (the oracle's thread count is fixed when it loads)."""
    import subprocess

    env = dict(os.environ, OMP_NUM_THREADS="1")
    r = subprocess.run([sys.executable, os.path.abspath(__file__), "--cpu-only", str(seconds)],
                       env=env, capture_output=True, text=True, timeout=300)
    if r.returncode != 0:
        log(f"  cpu oracle, one thread: failed ({r.stderr.strip()[-200:]})")
        return None
    res = json.loads(r.stdout.strip().splitlines()[-1])
    log(f"  cpu oracle, one thread: {res['ms_per_step']:.0f} ms per step")
    return res


def run_only(args, torch, D, inputs, log):
    name = args.only
    spec = ONLY[name]
    if name in ("prefill_gdn", "prefill_kda"):
        res = prefill_bench(torch, D, inputs, args.steps, log=log, kda=name == "prefill_kda")
    elif name == "pack_unpack":
        res = pack_unpack_bench(torch, D, args.steps, log=log)
    else:
        kda = spec[0] == "kda"
        wl = Workload(torch, D, inputs, kda=kda, B=256, HK=32 if kda else 16, HV=32, d=128,
                      k_hi=16, rotations=args.rotations, seed=1 if kda else 0, log=log)
        if name == "copy":
            res = copy_ceiling(torch, D, wl, args.rotations, args.steps, log=log, walks=())
        elif name.startswith("copy_tiles"):
            res = copy_ceiling(torch, D, wl, args.rotations, args.steps, log=log, linear=False,
                               walks=("scattered",) if name.endswith("_scattered") else ("consecutive",))
        else:
            _, kind, k_hi, tiers = spec
            rot = args.rotations if kind == D.DAMP_STATE_MIXED else max(2, args.rotations // 2)
            res = measure(torch, D, wl, kind, k_hi, rot, args.warmup, args.steps, torch.bfloat16,
                          tiers=tiers, scattered=name.endswith("_scattered"))
            log(f"  {name}: kernel {res['kernel_us']:.2f} us, {res['kernel_gbs']:.0f} GB/s "
                f"({100 * res['kernel_frac_peak']:.1f}% of peak)")
    print(json.dumps({"only": name, "steps": args.steps, "warmup": args.warmup, **res}), flush=True)


def main():
    args = parse()
    if args.cpu_only > 0:  # child of cpu_single_thread: no GPU work
        print(json.dumps(cpu_baseline(args.cpu_only, log=lambda *a: None)), flush=True)
        return
    global PREWARM_S
    PREWARM_S = args.prewarm
    if args.gpus != 1:
        print(f"bench.py measures one GPU only (got --gpus {args.gpus}): the state update has no "
              "cross-GPU step (tiles shard by value heads or request slots with no collective).", file=sys.stderr)
        sys.exit(2)
    log = lambda *a: print(*a, file=sys.stderr, flush=True)
    import torch

    from paper_2608_27513_amd import damp as D
    from paper_2608_27513_amd import inputs

    if not torch.cuda.is_available():
        raise SystemExit("no GPU visible")
    if args.copy_calibration:
        copy_calibration(torch)
        return
    D.lib()
    B, HK, HV, d, k_hi = 256, 16, 32, 128, 16
    if args.only is not None:
        run_only(args, torch, D, inputs, log)
        return
    log("setting up GDN B=256 HK=16 HV=32 d=128 K_hi=16")
    gdn = Workload(torch, D, inputs, kda=False, B=B, HK=HK, HV=HV, d=d, k_hi=k_hi,
                   rotations=args.rotations, seed=0, log=log)
    head = measure(torch, D, gdn, D.DAMP_STATE_MIXED, k_hi, args.rotations, args.warmup,
                   args.steps, torch.bfloat16, per_launch=True)
    log(f"  mixed: {head['us_per_step']:.1f} us/step, kernel {head['kernel_us']:.1f} us, "
        f"{head['kernel_gbs']:.0f} GB/s ({100 * head['kernel_frac_peak']:.1f}% of peak)")
    extra = {}
    if not args.quick:
        cop = copy_ceiling(torch, D, gdn, args.rotations, max(args.steps, 100), log=log)
        cop["update_frac_of_copy"] = round(cop["copy_us"] / head["kernel_us"], 4)
        extra["practical_ceiling"] = cop
        scat = measure(torch, D, gdn, D.DAMP_STATE_MIXED, k_hi, args.rotations, args.warmup,
                       args.steps, torch.bfloat16, scattered=True)
        log(f"  mixed, slots scattered over the pool: kernel {scat['kernel_us']:.1f} us, "
            f"{scat['kernel_gbs']:.0f} GB/s")
        scat["frac_of_tile_walk_copy"] = round(cop["tile_walk"]["scattered_us"] / scat["kernel_us"], 4)
        cop["update_frac_of_tile_walk_copy"] = round(cop["tile_walk"]["consecutive_us"] /
                                                     head["kernel_us"], 4)
        extra["headline_random_slots"] = scat
        rot_fp = max(2, args.rotations // 2)
        fp = measure(torch, D, gdn, D.DAMP_STATE_FP32, 0, rot_fp, args.warmup, args.steps,
                     torch.bfloat16)
        log(f"  fp32 state: {fp['us_per_step']:.1f} us/step, kernel {fp['kernel_us']:.1f} us, "
            f"{fp['kernel_gbs']:.0f} GB/s")
        i8 = measure(torch, D, gdn, D.DAMP_STATE_MIXED, 0, args.rotations, args.warmup,
                     args.steps, torch.bfloat16)
        log(f"  uniform int8: {i8['us_per_step']:.1f} us/step, kernel {i8['kernel_us']:.1f} us")
        extra["baselines_gdn"] = {"fp32_state": fp, "uniform_int8": i8,
                                  "speedup_vs_fp32_state": fp["kernel_us"] / head["kernel_us"]}
        # the paper's own tiers (FP16 rows, INT8 groups of 32 with FP16 (s, z))
        # and the other rows of its format table
        paper = {}
        fp16, u8 = D.DAMP_DT_FP16, D.DAMP_DT_U8
        for name, tiers in (("int8_h32", (fp16, 32, fp16, 1, u8)), ("int8_g32", (fp16, 32, fp16, 0, u8)),
                            ("int4_h32", (fp16, 32, fp16, 1, D.DAMP_DT_U4)),
                            ("int4_g32", (fp16, 32, fp16, 0, D.DAMP_DT_U4)),
                            ("fp8_e4m3", (fp16, 32, D.DAMP_DT_FP32, 0, D.DAMP_DT_E4M3)),
                            ("nvfp4", (fp16, 16, D.DAMP_DT_E4M3, 0, D.DAMP_DT_E2M1))):
            r = measure(torch, D, gdn, D.DAMP_STATE_MIXED, k_hi, args.rotations, args.warmup,
                        args.steps, torch.bfloat16, tiers=tiers)
            log(f"  paper tiers ({name}): kernel {r['kernel_us']:.1f} us, "
                f"{r['kernel_gbs']:.0f} GB/s, {r['bits_per_value']} bits/value")
            paper[name] = r
        extra["paper_tiers_gdn"] = paper
        del gdn
        torch.cuda.empty_cache()
        log("setting up KDA B=256 H=32 d=128 K_hi=16")
        kda = Workload(torch, D, inputs, kda=True, B=B, HK=32, HV=32, d=d, k_hi=k_hi,
                       rotations=args.rotations, seed=1, log=log)
        km = measure(torch, D, kda, D.DAMP_STATE_MIXED, k_hi, args.rotations, args.warmup,
                     args.steps, torch.bfloat16, per_launch=True)
        kf = measure(torch, D, kda, D.DAMP_STATE_FP32, 0, max(2, args.rotations // 2),
                     args.warmup, args.steps, torch.bfloat16)
        log(f"  kda mixed: kernel {km['kernel_us']:.1f} us ({100 * km['kernel_frac_peak']:.1f}%),"
            f" fp32 state kernel {kf['kernel_us']:.1f} us")
        extra["kda_b256"] = {"mixed": km, "fp32_state": kf,
                             "speedup_vs_fp32_state": kf["kernel_us"] / km["kernel_us"]}
        del kda
        torch.cuda.empty_cache()

        if not args.no_sweep:
            extra["sweep"] = sweep(torch, D, inputs, 50, log=log)
            extra["tp8_share"] = tp_share(torch, D, inputs, 100, log=log)
        if not args.no_multilayer:
            extra["multilayer_48"] = multilayer(torch, D, inputs, 64, log=log)
        extra["prefill_gdn"] = prefill_bench(torch, D, inputs, 10, log=log)
        extra["prefill_kda"] = prefill_bench(torch, D, inputs, 10, log=log, kda=True)
        extra["pack_unpack_gdn"] = pack_unpack_bench(torch, D, 20, log=log)
        extra["calibration_kda"] = calibration_bench(torch, D, inputs, log=log)
        extra["accuracy"] = accuracy_bench(torch, log=log)

    cpu = None
    if not args.quick and not args.no_cpu:
        cpu = cpu_baseline(args.cpu_seconds, log=log)
        one = cpu_single_thread(min(args.cpu_seconds, 10.0), log=log)
        if cpu is not None and one is not None:
            cpu["one_thread"] = {"value": one["value"], "unit": one["unit"],
                                 "cores": one["cores"], "ms_per_step": one["ms_per_step"]}

    traffic = profile_traffic()
    out = {
        "metric": "mixed-precision state-update µs/step + achieved HBM GB/s (% peak), B=256",
        "value": round(head["gbs"], 1),
        "unit": "GB/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(head["us_per_step"] / 1e3, 5),
        "us_per_step": round(head["us_per_step"], 2),
        "frac_of_hbm_peak": round(head["gbs"] / HBM_PEAK_GBS, 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16/u8 state, f32 compute",
        "data": "synthetic (seeded; FP32 warm-up over 512 tokens on the GPU)",
        "config": {"workload": "GDN decode, 1 layer: B=256, 16 key / 32 value heads, "
                               "d_k=d_v=128, 16 of 128 key channels BF16, rest INT8 rows "
                               "with fp32 (s, z); bf16 q/k/v/g/beta in, bf16 o out",
                   "global_batch": B, "layers": 1, "rotations": args.rotations,
                   "slots": "consecutive per rotation",
                   "bytes_per_step": head["bytes_per_step"]},
        "roofline": {"bound": "hbm", "achieved": round(head["kernel_gbs"], 1),
                     "peak": HBM_PEAK_GBS, "unit": "GB/s",
                     "frac": round(head["kernel_frac_peak"], 4),
                     "traffic": traffic,
                     "kernel_us": round(head["kernel_us"], 2),
                     "launch_stats": head.get("launch_stats")},
        "cpu_baseline": cpu,
        "storage": {"tile_bytes": head["tile_bytes"], "bits_per_value": head["bits_per_value"],
                    "reduction_vs_fp32_pct": round(100 * (1 - head["bits_per_value"] / 32), 2)},
    }
    out.update(extra)
    # the paper's own figures (section 1 and section 6, an unnamed NVIDIA GPU
    # running its CUDA executor in SGLang), reported beside ours as context
    out["paper_context"] = {
        "state_update_speedup_vs_fp32_state": {"gdn": "1.46-1.65x", "kda": "1.81-2.01x",
                                               "batch": "32-256", "format": "INT8+H32, 16 FP16 rows"},
        "storage_cut_pct": 69.1,
        "tpot_gain_pct_bs256": {"gdn": 10.9, "kda": 9.6},
        "hardware": "unnamed NVIDIA GPU (CUDA executor in SGLang)",
    }
    if "baselines_gdn" in extra and "paper_tiers_gdn" in extra:
        fp = extra["baselines_gdn"]["fp32_state"]["kernel_us"]
        out["paper_context"]["this_build_gdn_speedup_vs_fp32_state"] = {
            "default_tiers": round(fp / head["kernel_us"], 2),
            "paper_tiers_int8_h32": round(fp / extra["paper_tiers_gdn"]["int8_h32"]["kernel_us"], 2)}
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
