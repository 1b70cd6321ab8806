"""Throughput of the GIFT codec hot path on one MI355X.

One step = one pass of the whole per-layer hot path over a full synthetic
gradient set: the factor refresh of every GIFT matrix (statistics, rank-r
transform), the encode of every matrix (transform + amax + FP8 E4M3 for the
GIFT matrices, amax + FP8 for the Euclidean ones), the local rank sum and the
inverse transform.  Inputs are resident in HBM before the timed region.

Default workload: the Llama-600M-like gradient set, the largest of the five
workloads (24 layers, hidden 1536, MLP 4096; 16 simulated ranks; the GIFT
transform with rank 128 on every projection; per-128-column-block FP8 scales;
factors from 32768 bf16 tokens refreshed every 50 steps, Sec. V-E).
``--config 4`` is the Llama-300M-like set (8 ranks, rank 64 on gate/up/down,
Euclidean with a shared scale on q/k/v/o, embedding and LM head; refresh
every step), ``--config 1..3`` the single-matrix and MLP-pair workloads.

Refresh cadence: a step refreshes the factors iff its index is a multiple of
the cadence K.  Steps with and without a refresh are timed apart (HIP events
around each step), and ``ms_per_step`` / ``value`` are the cadence's average
``(t_refresh + (K - 1) t_codec) / K`` whatever ``--steps`` is;
``ms_per_step_raw`` is the plain mean over the timed steps.

Independent matrices are spread over several HIP streams (one library
context each; for the Llama-600M set 6 streams over 8 hardware queues, each
bucket to the stream with the fewest gradient bytes so far; otherwise 4
streams dealt in turn): a matrix's encode, rank sum and decode stay in
order on its stream, and each stream decodes its same-shape matrices in one
grouped call after their rank sums.  The factor refresh runs once per factor shape (the smallest group on
the main stream, the others on further streams), and a GIFT matrix's encode
waits only for its own group's refresh; the Euclidean matrices run beside the
refresh.

Prints one JSON line (metric: gradient GB/s through encode+decode; transform
TFLOP/s; % of roofline).  ``--gpus N`` with N > 1 is not supported: this codec runs
its N data-parallel ranks locally on one GPU.
"""

from __future__ import annotations

import argparse
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

# Source file of each kernel family: a measured HBM traffic figure (profiles/,
# rocprofv3 FETCH_SIZE / WRITE_SIZE) is reported only while this file is
# unchanged since the counters were taken.
FAMILY_SOURCE = {
    "syrk": "paper_2607_07494_amd/csrc/k_syrk.hip",
    "amax": "paper_2607_07494_amd/csrc/k_stream.hip",
    "quant": "paper_2607_07494_amd/csrc/k_stream.hip",
    "reduce": "paper_2607_07494_amd/csrc/k_stream.hip",
    "project": "paper_2607_07494_amd/csrc/k_lowrank.hip",
    "update_amax": "paper_2607_07494_amd/csrc/k_lowrank.hip",
    "update_quant": "paper_2607_07494_amd/csrc/k_lowrank.hip",
    "update_store": "paper_2607_07494_amd/csrc/k_update.hip",
    "decode_project": "paper_2607_07494_amd/csrc/k_update.hip",
    "chol_transform": "paper_2607_07494_amd/csrc/k_chol.hip",
    "mxfp4": "paper_2607_07494_amd/csrc/k_mx.hip",
}
TRAFFIC_GLOB = os.path.join(ROOT, "profiles", "*_hbm-traffic-per-kernel.md")

HBM_PEAK_GBS = 8000.0
FP32_MFMA_TFLOPS = 157.3
BF16_MFMA_TFLOPS = 2500.0


def parse():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=None,
                    help="timed steps (default 10; 20 when the factors are refreshed less often "
                         "than every step: step 0 refreshes, the others reuse the factors)")
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--config", type=int, default=5, choices=[1, 2, 3, 4, 5])
    ap.add_argument("--sides", choices=["input", "both"], default="input")
    ap.add_argument("--iters", type=int, default=1, help="subspace iterations per warm refresh")
    ap.add_argument("--cold-iters", type=int, default=6, help="subspace iterations of the first refresh")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--cpu-seconds", type=float, default=20.0)
    ap.add_argument("--issue", choices=["euclid-first", "interleave", "euclid-after-refresh",
                                        "euclid-after-statistics"],
                    default="euclid-after-statistics",
                    help="host issue order of the matrices within a step; euclid-after-refresh "
                         "also holds the Euclidean matrices until the largest factor group's "
                         "refresh is done, euclid-after-statistics only until its statistics "
                         "kernel is done (the compute-bound part that cannot share CUs)")
    ap.add_argument("--streams", type=int, default=None,
                    help="HIP streams (one library context each); each matrix's encode -> rank sum "
                         "-> decode stays on its stream (default 6 for the Llama-600M set, 8 "
                         "with error feedback there, 4 otherwise)")
    ap.add_argument("--assign", choices=["round-robin", "balance"], default=None,
                    help="GIFT buckets to streams: dealt in turn (in layer order, each layer's "
                         "buckets land on the same streams), or each to the stream with the fewest "
                         "gradient bytes so far (default balance for the Llama-600M set, "
                         "round-robin otherwise)")
    ap.add_argument("--hw-queues", type=int, default=None,
                    help="hardware queues of this process (GPU_MAX_HW_QUEUES, set before the HIP "
                         "runtime starts; 0 keeps the environment's value; default 8 for the "
                         "Llama-600M set, 4 (HIP's own) otherwise). Measured on the Llama-600M "
                         "set (codec-only step): 4 queues, 4 streams dealt in turn 37.1-38.1 ms "
                         "(the best with 4 queues; 2, 3, 6 streams and the balanced assignment "
                         "slower); 8 queues, 6 streams balanced 33.1-34.2 ms over seven runs on "
                         "three boxes (against 37.9-38.1 for the former on the same box), 5 / 7 / 8 "
                         "streams 51.1 / 42.5 / 35.3-36.6 ms, 6 streams in turn 48.2 ms; 16 queues, "
                         "6 / 8 / 12 streams balanced 33.2 / 33.8-34.9 / 50.8 ms. The Llama-300M "
                         "set keeps 4 streams in turn: 13.0 ms per step, 16.9 with 6 balanced on "
                         "8 queues. With error feedback (Llama-600M) 8 balanced streams on 8 "
                         "queues: 44.2-46.7 ms per codec step, 6: 55.0-55.3, 4 in turn on 4 "
                         "queues: 52.5")
    ap.add_argument("--breakdown-steps", type=int, default=2,
                    help="untimed steps with every kernel family bracketed by events")
    ap.add_argument("--format", choices=["fp8", "mxfp4"], default="fp8",
                    help="communication format: FP8 E4M3 (the paper's) or OCP MXFP4 (E2M1 with an "
                         "E8M0 scale per 32 elements of a row, per-rank scales for every matrix)")
    ap.add_argument("--no-bucket", dest="bucket", action="store_false",
                    help="one call per gradient matrix instead of one per bucket of same-shape "
                         "matrices stacked by rows (same results)")
    ap.add_argument("--fidelity", action="store_true",
                    help="only run the transform-variant fidelity study (one-step FP8 round trip "
                         "of one layer's gradient per transform, Tables I-II's metrics) and print "
                         "its table")
    ap.add_argument("--fid-shape", type=int, nargs=2, default=[1024, 2816], metavar=("M", "N"),
                    help="layer of the fidelity study (d_out d_in; default the MLP down projection)")
    ap.add_argument("--fid-tokens", type=int, default=8192)
    ap.add_argument("--decode", choices=["batch", "each"], default="batch",
                    help="batch: each stream decodes its same-shape buckets in one gift_decode_batch call "
                         "after their rank sums; each: one gift_decode per bucket right after its rank sum")
    ap.add_argument("--ef", action="store_true",
                    help="error feedback on the GIFT matrices (Algorithm 1: U~ = U + R, R <- U~ - Deq(Q(U~))), "
                         "a float32 residual per rank and element kept across steps")
    ap.add_argument("--no-embed", action="store_true",
                    help="leave the embedding and LM head out of the Llama-300M set")
    ap.add_argument("--flush-mall", action="store_true",
                    help="overwrite a 512 MiB scratch buffer before every timed step (outside the "
                         "step's events), so that each step starts with a cold 256 MB Infinity Cache")
    ap.add_argument("--calibrate", action="store_true",
                    help="only measure the achievable peaks the roofline is compared with: the "
                         "library's float32 copy kernel over 1 GiB (HBM read + write) and matrix-core "
                         "loops with no memory traffic (bf16 16x16x32 and float32 16x16x4 MFMA)")
    ap.add_argument("--copy-calibration", action="store_true",
                    help="only run the library's plain copy kernel on 256 MiB (5 launches), "
                         "the known-size reference for the HBM byte counters")
    args = ap.parse_args()
    # the schedule measured best for each workload (see --hw-queues)
    big = args.config == 5
    if args.streams is None:
        args.streams = (8 if args.ef else 6) if big else 4
    if args.assign is None:
        args.assign = "balance" if big else "round-robin"
    if args.hw_queues is None:
        args.hw_queues = 8 if big else 4
    return args


def source_sha256(rel):
    import hashlib
    with open(os.path.join(ROOT, rel), "rb") as fh:
        return hashlib.sha256(fh.read()).hexdigest()


def measured_traffic(family, workload):
    """HBM bytes per launch of `family` on `workload` from the committed
    counter summary, or None when there is none or the kernel's source has
    changed since it was taken.  Lines look like
    `traffic: family=F workload=W bytes_per_launch=B sha256=H`."""
    import glob
    if family not in FAMILY_SOURCE:
        return None
    sha = source_sha256(FAMILY_SOURCE[family])
    for path in sorted(glob.glob(TRAFFIC_GLOB)):
        for line in open(path):
            if not line.startswith("traffic:"):
                continue
            kv = dict(item.split("=", 1) for item in line.split()[1:])
            if kv.get("family") == family and kv.get("workload") == workload and kv.get("sha256") == sha:
                return float(kv["bytes_per_launch"])
    return None


def copy_calibration():
    """Five launches of the library's float32 copy kernel (decode with no
    factor) over 256 MiB: FETCH_SIZE and WRITE_SIZE of these dispatches give
    the counters' scale against exactly 256 MiB read and 256 MiB written."""
    import torch
    import paper_2607_07494_amd as gift

    dev = torch.device("cuda", 0)
    torch.cuda.set_device(dev)
    ctx = gift.Context()
    count = 64 * 1024 * 1024
    src = torch.rand(count, device=dev).reshape(8192, 8192)
    dst = torch.empty_like(src)
    for _ in range(5):
        gift.decode(ctx, None, src, dst)
    torch.cuda.synchronize()
    assert torch.equal(src, dst)
    ctx.close()
    print(json.dumps({"copy_calibration": {"bytes_read": count * 4, "bytes_written": count * 4,
                                           "launches": 5}}), flush=True)


def calibrate():
    """Achievable peaks on this GPU, reported beside the vendor figures."""
    import ctypes
    import torch
    import paper_2607_07494_amd as gift

    dev = torch.device("cuda", 0)
    torch.cuda.set_device(dev)
    ctx = gift.Context()
    out = {}
    ev = lambda: torch.cuda.Event(enable_timing=True)
    for mib in (1024, 4096):
        count = mib * 1024 * 1024 // 4
        src = torch.rand(count, device=dev).reshape(-1, 4096)
        dst = torch.empty_like(src)
        for _ in range(3):
            gift.decode(ctx, None, src, dst)
        e0, e1 = ev(), ev()
        reps = 10
        e0.record()
        for _ in range(reps):
            gift.decode(ctx, None, src, dst)
        e1.record()
        torch.cuda.synchronize()
        ms = e0.elapsed_time(e1) / reps
        out[f"copy_{mib}mib_gbs"] = round(2 * count * 4 / (ms * 1e-3) / 1e9, 1)
        del src, dst
    lib = ctypes.CDLL(os.path.join(ROOT, "paper_2607_07494_amd", "libgift_calib.so"))
    lib.gift_calib_mfma.argtypes = [ctypes.c_void_p, ctypes.c_int, ctypes.c_void_p, ctypes.c_int, ctypes.c_int]
    chains = lib.gift_calib_chains()
    blocks = 256 * 8                       # 8 waves per SIMD
    buf = torch.empty(blocks * 256, dtype=torch.float32, device=dev)
    stream = ctypes.c_void_p(torch.cuda.current_stream().cuda_stream)
    for kind, name, flops_per, iters in ((0, "mfma_bf16_tflops", 16384, 2000), (1, "mfma_f32_tflops", 2048, 1000),
                                         (2, "mfma_bf16_32x32x16_tflops", 32768, 1000),
                                         (3, "mfma_f32_32x32x2_tflops", 4096, 500)):
        for _ in range(2):
            assert lib.gift_calib_mfma(stream, kind, ctypes.c_void_p(buf.data_ptr()), blocks, 50) == 0
        e0, e1 = ev(), ev()
        e0.record()
        assert lib.gift_calib_mfma(stream, kind, ctypes.c_void_p(buf.data_ptr()), blocks, iters) == 0
        e1.record()
        torch.cuda.synchronize()
        ms = e0.elapsed_time(e1)
        flops = blocks * 4.0 * iters * chains * flops_per
        out[name] = round(flops / (ms * 1e-3) / 1e12, 1)
    # streaming reads of 4 GiB (far past the 256 MB Infinity Cache) and of
    # 128 MiB (held by it), cached and non-temporal loads
    lib.gift_calib_read.argtypes = [ctypes.c_void_p, ctypes.c_int, ctypes.c_void_p, ctypes.c_int64,
                                    ctypes.c_void_p, ctypes.c_int]
    rblocks = 256 * 16
    rout = torch.empty(rblocks * 256, dtype=torch.float32, device=dev)
    for mib in (4096, 128):
        src = torch.zeros(mib * 1024 * 1024 // 4, dtype=torch.float32, device=dev)
        nbytes = src.numel() * 4
        for kind, name in ((0, "cached"), (1, "nontemporal")):
            for _ in range(3):
                assert lib.gift_calib_read(stream, kind, ctypes.c_void_p(src.data_ptr()), nbytes,
                                           ctypes.c_void_p(rout.data_ptr()), rblocks) == 0
            reps = 20
            e0, e1 = ev(), ev()
            e0.record()
            for _ in range(reps):
                assert lib.gift_calib_read(stream, kind, ctypes.c_void_p(src.data_ptr()), nbytes,
                                           ctypes.c_void_p(rout.data_ptr()), rblocks) == 0
            e1.record()
            torch.cuda.synchronize()
            ms = e0.elapsed_time(e1) / reps
            out[f"read_{mib}mib_{name}_gbs"] = round(nbytes / (ms * 1e-3) / 1e9, 1)
        del src
    ctx.close()
    out.update({"hbm_spec_gbs": HBM_PEAK_GBS, "mfma_bf16_spec_tflops": BF16_MFMA_TFLOPS,
                "mfma_f32_spec_tflops": FP32_MFMA_TFLOPS})
    print(json.dumps({"calibration": out}), flush=True)


class Job:
    """Device buffers of one bucket: gradient matrices of one shape stacked by
    rows in every rank's buffer (``[N, count*m, n]``), encoded in one call.
    Each matrix keeps its own scale blocks (block rows never cross a matrix),
    so the codes, scales, rank mean and decode equal per-matrix calls."""

    def __init__(self, mats, wl, sides_flag, dev, torch, gift, fmt="fp8"):
        self.mats = mats
        layer, mat = mats[0]
        self.layer, self.mat = layer, mat
        N, m, n = wl.N, sum(mt.m for _, mt in mats), mat.n
        self.N, self.m, self.n = N, m, n
        self.gift_branch = mat.gift
        self.br, self.bc = wl.block_rows, wl.block_cols
        if len(mats) > 1 and self.br == 0:
            self.br = mat.m        # the whole of each matrix
        nbr, nbc = gift.scale_grid(m, n, self.br, self.bc)
        self.grads = torch.empty((N, m, n), dtype=torch.float32, device=dev)
        if fmt == "mxfp4":
            self.codes = torch.empty((N, m, n // 2), dtype=torch.uint8, device=dev)
            self.scales = torch.empty((N, m, n // 32), dtype=torch.uint8, device=dev)
        else:
            self.codes = torch.empty((N, m, n), dtype=torch.uint8, device=dev)
            self.scales = torch.empty((N, nbr, nbc), dtype=torch.float32, device=dev)
        self.mean = torch.empty((m, n), dtype=torch.float32, device=dev)
        self.out = torch.empty((m, n), dtype=torch.float32, device=dev) if mat.gift else None
        self.ef = None
        self.factor = None
        self.sides = sides_flag if mat.gift else 0
        self.acts = self.dgrads = None
        self.owns_factor = False   # the matrix whose refresh updates a shared factor


BUCKET_ELEMS = 1 << 26   # per rank: 256 MB of float32 gradient per bucket


def buckets(wl, sides, gift, enable):
    """Matrices grouped into buckets of one shape, in step order.

    Euclidean matrices of one shape share buckets of up to BUCKET_ELEMS
    elements per rank; with the input-side transform alone the GIFT matrices
    that read the same layer input (gate, up) share a bucket, since their
    common factor acts on rows independently; everything else is a bucket of
    one.  Block rows must tile each matrix exactly."""
    mats = wl.all_matrices()
    if not enable:
        return [[x] for x in mats]
    aligned = lambda mt: wl.block_rows == 0 or mt.m % wl.block_rows == 0
    out, open_eu = [], {}
    for layer, mt in mats:
        if not mt.gift and aligned(mt):
            key = (mt.m, mt.n)
            b = open_eu.get(key)
            if b is None or (len(b) + 1) * mt.m * mt.n > BUCKET_ELEMS:
                b = []
                open_eu[key] = b
                out.append(b)
            b.append((layer, mt))
        elif mt.gift and sides == gift.SIDE_INPUT and aligned(mt):
            for b in out:
                l0, m0 = b[0]
                if m0.gift and l0 == layer and m0.act == mt.act and (m0.m, m0.n) == (mt.m, mt.n):
                    b.append((layer, mt))
                    break
            else:
                out.append([(layer, mt)])
        else:
            out.append([(layer, mt)])
    return out


def build_workload(args, torch, gift, synth, dev):
    from synth.configs import WORKLOADS
    wl = WORKLOADS[args.config]
    if args.no_embed:
        import dataclasses
        wl = dataclasses.replace(wl, name=wl.name + "-no-embedding", extra=())
    sides = gift.SIDE_INPUT if args.sides == "input" else gift.SIDE_BOTH
    jobs = [Job(b, wl, sides, dev, torch, gift, args.format) for b in buckets(wl, sides, gift, args.bucket)]
    # one random set per distinct shape, copied into every matrix's rows
    cache = {}
    for jb in jobs:
        off = 0
        for _, mt in jb.mats:
            key = (mt.m, mt.n)
            if key not in cache:
                cache[key] = synth.gradient_set_torch(synth.seed_for(wl.cfg, 0, 0, mt.kind),
                                                      wl.N, mt.m, mt.n, dev)
            jb.grads[:, off:off + mt.m].copy_(cache[key])
            off += mt.m
    del cache
    if args.ef:
        for jb in jobs:
            if jb.gift_branch:
                jb.ef = torch.zeros_like(jb.grads)
    # factor inputs: per layer, one activation stream per layer input and one
    # output-gradient stream per GIFT matrix (copies of one draw per shape)
    xcache = {}

    def stream(dim, role):
        key = (dim, role)
        if key not in xcache:
            xcache[key] = synth.factor_inputs_torch(synth.seed_for(wl.cfg, role, 0, dim % 97), wl.T,
                                                    dim, dev, dtype=wl.act_dtype)
        return xcache[key]

    # K-FAC's input factor A = E[a a^T] belongs to a layer input: matrices that
    # read the same input (gate and up) have the same A and, with the input
    # side alone, the same transform, so they share one factor (refreshed
    # once).  With the output side each matrix keeps its own factor.
    per_layer_acts, shared = {}, {}
    for jb in jobs:
        if not jb.gift_branch:
            continue
        akey = (jb.layer, jb.mat.act)
        if akey not in per_layer_acts:
            per_layer_acts[akey] = stream(jb.n, 1).clone()
        jb.acts = per_layer_acts[akey]
        if jb.sides & gift.SIDE_OUTPUT:
            jb.dgrads = stream(jb.m, 2).clone()
        fkey = (akey, jb.m, jb.n) if jb.sides == gift.SIDE_INPUT else (akey, jb.mat.kind)
        if fkey not in shared:
            shared[fkey] = gift.Factor(ctx_holder["ctx"], jb.m, jb.n, wl.rank, jb.sides,
                                       seed=synth.seed_for(wl.cfg, 50, jb.layer, jb.mat.kind))
            jb.owns_factor = True
        jb.factor = shared[fkey]
    del xcache
    return wl, jobs


ctx_holder = {}


def algorithmic_work(wl, jobs, args):
    """Algorithmic flops / bytes per step for each kernel family."""
    r = wl.rank
    fam = {}

    def add(name, flops=0.0, bytes_=0.0):
        f, b = fam.get(name, (0.0, 0.0))
        fam[name] = (f + flops, b + bytes_)

    refresh = 1.0 / wl.refresh
    mxb = 0.5 + 1.0 / 32.0     # MXFP4 bytes per element: a 4-bit code and 1/32 of a scale
    for jb in jobs:
        N, m, n = jb.N, jb.m, jb.n
        e = float(N) * m * n
        mn = float(m) * n
        ra = r if jb.gift_branch and jb.sides & 1 else 0
        rg = r if jb.gift_branch and jb.sides & 2 else 0
        proj_flops = 2 * e * (ra + rg) + (4 * N * rg * ra * m if ra and rg else 0)
        proj_bytes = 4 * e * ((ra > 0) + (rg > 0))
        if args.format == "mxfp4":
            # the MXFP4 pass (on the GIFT branch fused with the rank-r update:
            # 2r flops/elem), the rank sum; the projections and the decode as
            # in FP8
            add("mxfp4", 2 * e * (ra + rg), (4 + mxb) * e)
            add("reduce", 0, mn * (N * mxb + 4))
            if jb.gift_branch:
                add("project", proj_flops, proj_bytes)
                add("update_store", 2 * mn * (ra + rg), 8 * mn)
                add("decode_project", 2 * mn * (ra + rg), 4 * mn * ((ra > 0) + (rg > 0)))
        elif not jb.gift_branch:
            add("amax", 0, 4 * e)
            add("quant", 0, 5 * e)
            add("reduce", 0, mn * (N + 4))
        else:
            # encode: projections (2r flops/elem per side), the rank-r update
            # fused with the block maxima, then scale + FP8 pack of W~
            # (error feedback: the AMAX pass reads R, the QUANT pass reads
            # and rewrites it, since both form W~ + R)
            efb = 1.0 if jb.ef is not None else 0.0
            add("project", proj_flops, proj_bytes)
            add("update_amax", 2 * e * (ra + rg), (4 + 4 * efb) * e)
            add("update_quant", 0, (5 + 8 * efb) * e)
            add("reduce", 0, mn * (N + 4))
            add("decode_project", 2 * mn * (ra + rg), 4 * mn * ((ra > 0) + (rg > 0)))
            add("update_store", 2 * mn * (ra + rg), 8 * mn)
        if not jb.gift_branch:
            continue
        # factor refresh (amortised by the cadence), once per distinct factor
        for dim, on in ((n, ra), (m, rg)):
            if not on or not jb.owns_factor:
                continue
            T = wl.T
            k = min(dim, 2 * r)
            add("syrk", refresh * T * dim * (dim + 1), refresh * T * dim * 2)
            q = args.iters
            sub = 8 * dim * k * k + q * (2 * dim * dim * k + 8 * dim * k * k) + \
                2 * dim * dim * k + 2 * dim * k * k + 2 * dim * k * r
            add("factor", refresh * sub, 0)
            # the k x k Cholesky factorisations and the eigensolver are
            # latency-bound single-workgroup kernels: timed, no roofline
    return fam


def cpu_baseline(wl, jobs, seconds):
    """The oracle on a bounded sample of the workload, timed on the host cores.

    Sample: the first ``rows`` rows of the first GIFT matrix, all N ranks
    (the input-side transform acts on each row alone, so a row slice is a
    proper part of the encode / rank sum / decode), plus the full factor
    refresh of that matrix's input side (statistics from all T tokens, exact
    eigendecomposition).  Inputs are the benchmark's own device inputs copied
    to the host.  Each part is timed up to three times (median), bounded by
    ``seconds``; the refresh is charged to the sample in the proportion the
    GPU metric charges it: divided by the cadence K and by the rows that share
    the factor.  A single-thread time of the codec sample is reported too.
    """
    import numpy as np
    from threadpoolctl import threadpool_info, threadpool_limits
    from oracle import codec

    jb = next(j for j in jobs if j.gift_branch and j.owns_factor)
    mat = jb.mats[0][1]
    N, n, r = jb.N, jb.n, wl.rank
    rows = min(512, mat.m)
    grads = jb.grads[:, :rows, :].float().cpu().numpy()
    X = jb.acts.float().cpu().numpy()
    shared_rows = sum(j.m for j in jobs if j.factor is jb.factor)
    cores = max([i.get("num_threads", 1) for i in threadpool_info()] + [1])

    def timed(fn, budget):
        ts = []
        t_start = time.perf_counter()
        while len(ts) < 3:
            t0 = time.perf_counter()
            out = fn()
            ts.append(time.perf_counter() - t0)
            if time.perf_counter() - t_start >= budget:
                break
        return float(np.median(ts)), len(ts), out

    t_ref, n_ref, fA = timed(lambda: codec.lowrank_factor(codec.factor_statistics(X), r).to_f32(),
                             0.25 * seconds)
    br, bc = wl.block_rows, wl.block_cols
    codec_fn = lambda: codec.round_trip(grads, fA, None, br, bc, False)
    t_codec, n_codec, _ = timed(codec_fn, 0.5 * seconds)
    with threadpool_limits(1):
        t1 = time.perf_counter()
        codec_fn()
        t_codec_1 = time.perf_counter() - t1
    share = rows / shared_rows / wl.refresh
    per = t_codec + share * t_ref
    by = N * rows * n * 4
    return {"value": round(by / per / 1e9, 5), "unit": "GB/s", "cores": int(cores), "kind": "oracle",
            "single_thread_value": round(by / (t_codec_1 + share * t_ref) / 1e9, 5),
            "sample": f"rows 0..{rows - 1} of one {mat.name} matrix ({mat.m}x{n}, N={N} ranks, r={r}, "
                      f"input side, block ({br},{bc})): encode + rank sum + decode, median of {n_codec} "
                      f"({t_codec:.2f} s; one thread {t_codec_1:.2f} s), plus the factor refresh from "
                      f"{X.shape[0]} tokens (statistics + exact eigendecomposition, median of {n_ref}: "
                      f"{t_ref:.2f} s) charged x {share:.2e} (the sample's rows of the {shared_rows} rows "
                      f"sharing the factor, over the cadence {wl.refresh})"}


# Transform variants of the fidelity study: (label, kind, size, sides); kind
# "chol" takes a block size (0 = the full factor, 1 = the diagonal), "lowrank"
# a rank.
FIDELITY_METHODS = [
    ("Euclidean baseline", None, 0, 0),
    ("Output-side only (full)", "chol", 0, 2),
    ("Input-side only (full-A)", "chol", 0, 1),
    ("K-FAC (both sides, full)", "chol", 0, 3),
    ("Input-side diag-A", "chol", 1, 1),
    ("Input-side block-A-32", "chol", 32, 1),
    ("Input-side block-A-64", "chol", 64, 1),
    ("Input-side block-A-128", "chol", 128, 1),
    ("Input-side low-rank-A-8", "lowrank", 8, 1),
    ("Input-side low-rank-A-16", "lowrank", 16, 1),
    ("Input-side low-rank-A-32", "lowrank", 32, 1),
]
FIDELITY_REGIMES = [
    ("gaussian tokens", {}),
    ("spiked tokens (1/512 of the tokens x20 in inputs and output gradients)",
     {"spike_frac": 1.0 / 512.0, "spike": 20.0}),
]


def recon_metrics(ghat, g):
    """RelL2, Cos, MaxErr, MSE of a reconstruction (eq. recon_metrics)."""
    import numpy as np
    gh = ghat.astype(np.float64).ravel()
    g = g.astype(np.float64).ravel()
    d = gh - g
    return {"RelL2": float(np.linalg.norm(d) / np.linalg.norm(g)),
            "Cos": float(gh @ g / (np.linalg.norm(gh) * np.linalg.norm(g))),
            "MaxErr": float(np.abs(d).max()), "MSE": float(d @ d / d.size)}


def fidelity_study(args):
    """One-step FP8 round trip (transform, per-tensor amax E4M3, rank sum of
    one rank, inverse) of one layer's gradient for every transform variant,
    and the same with MXFP4 (per-32-element E8M0 scales) in place of FP8,
    factors refreshed on the GPU from the layer's own inputs; plus the time of
    one refresh and of encode + rank sum + decode of 8 ranks of that shape."""
    import numpy as np
    import torch
    import paper_2607_07494_amd as gift
    import synth

    dev = torch.device("cuda", 0)
    torch.cuda.set_device(dev)
    ctx = gift.Context()
    m, n = args.fid_shape
    T = args.fid_tokens
    N8 = 8
    ev = lambda: torch.cuda.Event(enable_timing=True)
    rows = []
    for regime, kw in FIDELITY_REGIMES:
        g, xa, xg = synth.layer_gradients(4242, 1, T, m, n, **kw)
        print(f"[fidelity] {regime}: layer {m}x{n}, {T} tokens", file=sys.stderr, flush=True)
        gt = torch.from_numpy(g).to(dev)
        g8 = gt.expand(N8, m, n).contiguous()
        at = torch.from_numpy(xa).to(dev)
        ot = torch.from_numpy(xg).to(dev)
        codes = torch.empty((N8, m, n), dtype=torch.uint8, device=dev)
        scales = torch.empty((N8, 1, 1), dtype=torch.float32, device=dev)
        mxc = torch.empty((1, m, n // 2), dtype=torch.uint8, device=dev)
        mxs = torch.empty((1, m, n // 32), dtype=torch.uint8, device=dev)
        mean = torch.empty((m, n), dtype=torch.float32, device=dev)
        out = torch.empty((m, n), dtype=torch.float32, device=dev)
        for label, kind, size, sides in FIDELITY_METHODS:
            f = None
            refresh_ms = 0.0
            if kind is not None:
                f = (gift.CholFactor(ctx, m, n, size, sides, 1e-6) if kind == "chol"
                     else gift.Factor(ctx, m, n, size, sides, 1e-6, seed=11))
                a_in = at if sides & gift.SIDE_INPUT else None
                o_in = ot if sides & gift.SIDE_OUTPUT else None
                f.update(acts=a_in, out_grads=o_in, iters=8)   # cold start
                torch.cuda.synchronize()
                e0, e1 = ev(), ev()
                e0.record()
                f.update(acts=a_in, out_grads=o_in, iters=2)   # a warm refresh
                e1.record()
                torch.cuda.synchronize()
                refresh_ms = e0.elapsed_time(e1)
            # the round trip of the one gradient
            gift.encode(ctx, f, gt, codes[:1], scales[:1])
            gift.reduce_local(ctx, codes[:1], scales[:1], mean)
            gift.decode(ctx, f, mean, out)
            torch.cuda.synchronize()
            met = recon_metrics(out.cpu().numpy(), g[0])
            gift.encode_mxfp4(ctx, f, gt, mxc, mxs)
            gift.reduce_local_mxfp4(ctx, mxc, mxs, mean)
            gift.decode(ctx, f, mean, out)
            torch.cuda.synchronize()
            met_mx = recon_metrics(out.cpu().numpy(), g[0])
            # encode + rank sum + decode of 8 ranks
            for _ in range(2):
                gift.encode(ctx, f, g8, codes, scales)
            reps = 5
            e0, e1 = ev(), ev()
            e0.record()
            for _ in range(reps):
                gift.encode(ctx, f, g8, codes, scales)
                gift.reduce_local(ctx, codes, scales, mean)
                gift.decode(ctx, f, mean, out)
            e1.record()
            torch.cuda.synchronize()
            codec_ms = e0.elapsed_time(e1) / reps
            row = {"regime": regime, "method": label, **met, "refresh_ms": refresh_ms,
                   "codec_ms_8ranks": codec_ms, "mxfp4": met_mx}
            rows.append(row)
            print(f"[fidelity] {label}: RelL2 {met['RelL2']:.4e}  refresh {refresh_ms:.2f} ms  "
                  f"codec {codec_ms:.3f} ms", file=sys.stderr, flush=True)
            if f is not None:
                f.close()
    ctx.close()
    print(f"| regime | method | RelL2 | Cos | MaxErr | MSE | refresh ms | encode+sum+decode ms (8 ranks) |")
    print("|---|---|---|---|---|---|---|---|")
    for r in rows:
        print(f"| {r['regime'].split(' (')[0]} | {r['method']} | {r['RelL2']:.4e} | {r['Cos']:.7f} | "
              f"{r['MaxErr']:.4e} | {r['MSE']:.4e} | {r['refresh_ms']:.2f} | {r['codec_ms_8ranks']:.3f} |")
    print()
    print("| regime | method | MXFP4 RelL2 | Cos | MaxErr | MSE |")
    print("|---|---|---|---|---|---|")
    for r in rows:
        x = r["mxfp4"]
        print(f"| {r['regime'].split(' (')[0]} | {r['method']} | {x['RelL2']:.4e} | {x['Cos']:.7f} | "
              f"{x['MaxErr']:.4e} | {x['MSE']:.4e} |")
    print(json.dumps({"fidelity": rows, "layer": [m, n], "tokens": T}), flush=True)


def main():
    args = parse()
    if args.gpus != 1:
        print(f"bench.py runs on one GPU: the codec simulates its N data-parallel ranks locally "
              f"and has no multi-GPU path (asked for --gpus {args.gpus}).", file=sys.stderr)
        sys.exit(2)
    if args.hw_queues > 0:
        # read by the HIP runtime when it starts (nothing above has touched it)
        os.environ["GPU_MAX_HW_QUEUES"] = str(args.hw_queues)
    if args.copy_calibration:
        copy_calibration()
        return
    if args.calibrate:
        calibrate()
        return
    if args.fidelity:
        fidelity_study(args)
        return
    import torch
    import paper_2607_07494_amd as gift
    import synth

    dev = torch.device("cuda", 0)
    torch.cuda.set_device(dev)
    ctx = gift.Context()
    ctx_holder["ctx"] = ctx
    wl, jobs = build_workload(args, torch, gift, synth, dev)
    if args.steps is None:
        args.steps = 10 if wl.refresh <= 1 else 20
    torch.cuda.synchronize()
    print(f"[bench] workload {wl.name}: {sum(len(j.mats) for j in jobs)} matrices in "
          f"{len(jobs)} buckets, "
          f"{sum(j.N * j.m * j.n for j in jobs) * 4 / 1e9:.2f} GB of rank gradients", file=sys.stderr,
          flush=True)

    fjobs = [jb for jb in jobs if jb.owns_factor]
    # independent matrices on several streams (default priority), one library
    # context per stream.  The factor refresh runs per factor shape (one call
    # per group, the smallest first on the main stream, the others on the
    # next streams), so a GIFT matrix waits only for its own group's refresh.
    main = torch.cuda.current_stream()
    nstreams = max(args.streams, 1)
    streams = [main] + [torch.cuda.Stream() for _ in range(nstreams - 1)]
    ctxs = [ctx] + [gift.Context(stream=st.cuda_stream) for st in streams[1:]]

    def fkey(jb):
        return (jb.n, jb.m if jb.sides & gift.SIDE_OUTPUT else 0)

    groups = {}
    for jb in fjobs:
        groups.setdefault(fkey(jb), []).append(jb)
    gorder = sorted(groups, key=lambda k: sum(jb.n * jb.n + (jb.m * jb.m if k[1] else 0)
                                             for jb in groups[k]))
    gsid = {k: (i if i < nstreams else 0) for i, k in enumerate(gorder)}
    for jb in jobs:
        jb.group = fkey(jb) if jb.gift_branch else None
    # Euclidean matrices first, on streams that host no refresh (they run
    # beside it); then each group's GIFT matrices, a group's matrices avoiding
    # the streams of the groups refreshed after it
    eu = [jb for jb in jobs if not jb.gift_branch]
    free = [s for s in range(nstreams) if s not in gsid.values()] or list(range(1, nstreams)) or [0]
    for i, jb in enumerate(eu):
        jb.sid = free[i % len(free)]
    gift_order = []
    load = [0] * nstreams       # gradient bytes dealt to each stream
    for jb in eu:
        load[jb.sid] += jb.N * jb.m * jb.n
    for gi, k in enumerate(gorder):
        later = {gsid[k2] for k2 in gorder[gi + 1:]}
        ok = [s for s in range(nstreams) if s not in later] or [0]
        gjobs = [jb for jb in jobs if jb.gift_branch and jb.group == k]
        for i, jb in enumerate(gjobs):
            if args.assign == "balance":
                # the least loaded allowed stream
                jb.sid = min(ok, key=lambda s: (load[s], s))
            else:
                jb.sid = ok[i % len(ok)]
            load[jb.sid] += jb.N * jb.m * jb.n
        gift_order += gjobs
    stream_load = load
    stats_ev = None
    if args.issue == "euclid-after-statistics" and gorder:
        stats_ev = torch.cuda.Event()
        ctxs[gsid[gorder[-1]]].set_statistics_event(stats_ev)
    if args.issue in ("euclid-first", "euclid-after-refresh", "euclid-after-statistics"):
        order = list(eu) + gift_order
    else:   # alternate, so that every stream's queue holds both kinds early
        order, a, b = [], list(eu), list(gift_order)
        while a or b:
            if b:
                order.append(b.pop(0))
            if a:
                order.append(a.pop(0))

    def join_into_main():
        for st in streams[1:]:
            ev = torch.cuda.Event()
            ev.record(st)
            main.wait_event(ev)

    def step(iters, serial=False, refresh=True, codec=True):
        """One step; refresh=False reuses the factors of the last refresh
        (the cadence's other steps), codec=False runs the refresh alone."""
        join_into_main()           # the refresh rewrites factors the last step's encodes read
        joined = torch.cuda.Event()
        joined.record(main)
        ready = {}
        for k in (gorder if refresh else ()):
            sid = 0 if serial else gsid[k]
            if sid != 0:
                streams[sid].wait_event(joined)
            g = groups[k]
            gift.factor_update_batch(ctxs[sid], [jb.factor for jb in g], [jb.acts for jb in g],
                                     [jb.dgrads for jb in g], iters=iters)
            ready[k] = (sid, torch.cuda.Event())
            ready[k][1].record(streams[sid])
        waited = set()
        pending = {}   # (stream, shape) -> buckets whose decode is grouped
        for jb in (order if codec else ()):
            sid = 0 if serial else jb.sid
            if not jb.gift_branch and args.issue == "euclid-after-refresh" and not serial and ready:
                rsid, ev = ready[gorder[-1]]
                if rsid != sid and (sid, None) not in waited:
                    streams[sid].wait_event(ev)
                    waited.add((sid, None))
            if not jb.gift_branch and stats_ev is not None and not serial and ready:
                if gsid[gorder[-1]] != sid and (sid, None) not in waited:
                    streams[sid].wait_event(stats_ev)
                    waited.add((sid, None))
            if jb.gift_branch and jb.group in ready:
                rsid, ev = ready[jb.group]
                if rsid != sid and (sid, jb.group) not in waited:
                    streams[sid].wait_event(ev)    # GIFT encodes need the refreshed factor
                    waited.add((sid, jb.group))
            c = ctxs[sid]
            if args.format == "mxfp4":
                gift.encode_mxfp4(c, jb.factor, jb.grads, jb.codes, jb.scales, ef=jb.ef)
                gift.reduce_local_mxfp4(c, jb.codes, jb.scales, jb.mean)
            else:
                gift.encode(c, jb.factor, jb.grads, jb.codes, jb.scales, jb.br, jb.bc,
                            gift.SCALE_LOCAL if jb.gift_branch else gift.SCALE_SHARED, ef=jb.ef)
                gift.reduce_local(c, jb.codes, jb.scales, jb.mean, jb.br, jb.bc)
            if jb.gift_branch:
                if args.decode == "batch":
                    # (buckets are issued in layer order, so the streams run a
                    # mix of shapes at any time; each stream decodes its
                    # buckets of a shape together once it has summed them all)
                    pending.setdefault((sid, jb.m, jb.n), []).append(jb)
                else:
                    gift.decode(c, jb.factor, jb.mean, jb.out)
        for (sid, _, _), jbs in pending.items():
            gift.decode_batch(ctxs[sid], [jb.factor for jb in jbs], [jb.mean for jb in jbs],
                              [jb.out for jb in jbs])

    for w in range(max(args.warmup, 1)):
        step(args.cold_iters if w == 0 else args.iters)
        join_into_main()
        torch.cuda.synchronize()
        print(f"[bench] warmup step {w} done", file=sys.stderr, flush=True)

    def profile_all(enable, families=None, reset=False):
        for c in ctxs:
            if reset:
                c.profile_reset()
            c.profile_select(families)
            c.profile(enable)

    def read_all(name):
        tot_l, tot_ms = 0, 0.0
        for c in ctxs:
            launches, ms = c.profile_read(name)
            tot_l += launches
            tot_ms += ms
        return tot_l, tot_ms

    # untimed breakdown with every launch on the main stream (isolated,
    # non-overlapping kernel times): every kernel family bracketed by events;
    # the refresh and the codec passes are timed apart and the refresh is
    # amortised over its cadence.  The largest family per amortised step is
    # the dominant kernel; its roofline comes from these isolated launches.
    nb = max(args.breakdown_steps, 1)
    fam_ms = {}
    fam_raw = {}     # family -> (launches, ms) per isolated step of its kind
    for refresh, codec, weight in ((True, False, 1.0 / wl.refresh), (False, True, 1.0)):
        profile_all(True, None, reset=True)
        for s in range(nb):
            step(args.iters, serial=True, refresh=refresh, codec=codec)
        for name in gift.KERNELS:
            launches, ms = read_all(name)
            if launches:
                l0, m0 = fam_ms.get(name, (0.0, 0.0))
                fam_ms[name] = (l0 + weight * launches / nb, m0 + weight * ms / nb)
                r0, q0 = fam_raw.get(name, (0, 0.0))
                fam_raw[name] = (r0 + launches, q0 + ms)
    profile_all(False)
    # the dominant kernel: the family with the most time per step among
    # those with a roofline (algorithmic bytes or flops); the refresh's
    # one-workgroup-per-factor k x k kernels (chol, eig) are latency-bound
    work = algorithmic_work(wl, jobs, args)
    with_roof = [k for k in fam_ms if sum(work.get(k, (0.0, 0.0))) > 0]
    dom = max(with_roof or list(fam_ms), key=lambda k: fam_ms[k][1])
    latency_ms = {k: round(fam_ms[k][1], 4) for k in fam_ms if k not in with_roof}

    # timed region: events around every step (refresh steps and codec-only
    # steps are timed apart), and around the dominant family's launches
    profile_all(True, [dom], reset=True)
    K = max(wl.refresh, 1)
    nsteps = args.steps
    ev_s = [torch.cuda.Event(enable_timing=True) for _ in range(nsteps)]
    ev_e = [torch.cuda.Event(enable_timing=True) for _ in range(nsteps)]
    flush = torch.empty(128 * 1024 * 1024, dtype=torch.float32, device=dev) if args.flush_mall else None
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for s in range(nsteps):
        if flush is not None:
            join_into_main()
            flush.fill_(float(s))
        join_into_main()
        ev_s[s].record(main)
        step(args.iters, refresh=s % K == 0)
        join_into_main()
        ev_e[s].record(main)
    enqueue = time.perf_counter() - t0   # host time to issue the timed steps
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    step_ms = [ev_s[s].elapsed_time(ev_e[s]) for s in range(nsteps)]
    ms_raw = sum(step_ms) / nsteps
    ref_ms = [step_ms[s] for s in range(nsteps) if s % K == 0]
    cod_ms = [step_ms[s] for s in range(nsteps) if s % K != 0]
    import statistics
    t_ref = statistics.median(ref_ms)
    t_cod = statistics.median(cod_ms) if cod_ms else None
    if K > 1 and t_cod is not None:
        ms_step = (t_ref + (K - 1) * t_cod) / K
    else:
        ms_step = statistics.median(step_ms)
    dom_launches, dom_ms_total = read_all(dom)
    profile_all(False)
    print(f"[bench] timed {nsteps} steps: {ms_step:.3f} ms/step at the refresh cadence {K} "
          f"(refresh step {t_ref:.3f} ms, codec-only step "
          f"{t_cod if t_cod is None else round(t_cod, 3)} ms, raw mean {ms_raw:.3f} ms; wall "
          f"{wall:.2f} s, host issue {enqueue / nsteps * 1e3:.3f} ms/step)", file=sys.stderr, flush=True)

    grad_bytes = sum(j.N * j.m * j.n * 4 for j in jobs)
    value = grad_bytes / (ms_step * 1e-3) / 1e9
    kernels = {}
    for name, (launches, ms) in fam_ms.items():
        fl, by = work.get(name, (0.0, 0.0))
        kernels[name] = {"ms_per_step": round(ms, 4), "launches_per_step": round(launches, 2),
                         "tflops": round(fl / (ms * 1e-3) / 1e12, 3) if ms > 0 else None,
                         "gbs": round(by / (ms * 1e-3) / 1e9, 2) if ms > 0 else None}
    # roofline of the dominant kernel from its isolated launches: algorithmic
    # work per launch (per step / launches per step) over the average
    # isolated launch duration
    fl, by = work.get(dom, (0.0, 0.0))
    per_step_launches, per_step_ms = fam_ms[dom]
    iso_launches, iso_ms = fam_raw[dom]
    avg_ms = iso_ms / iso_launches
    fl_l, by_l = fl / per_step_launches, by / per_step_launches
    # matrix-core basis: the statistics from bf16 tokens on BF16 MFMA; the
    # encode's projections and rank-r update as three bf16 products of the
    # split float32 operands (hi hi + hi lo + lo hi) on BF16 MFMA, so 3x the
    # float32 flops against the bf16 peak; the rest on FP32 MFMA
    if dom == "syrk" and wl.act_dtype == "bf16":
        peak_f, mult, basis = BF16_MFMA_TFLOPS, 1, "bf16 MFMA"
    elif dom in ("project", "update_amax", "update_quant"):
        peak_f, mult, basis = BF16_MFMA_TFLOPS, 3, "3 bf16 MFMA products per float32 product (split operands)"
    else:
        peak_f, mult, basis = FP32_MFMA_TFLOPS, 1, "FP32 MFMA"
    frac_f = mult * fl_l / (avg_ms * 1e-3) / 1e12 / peak_f if fl else 0.0
    frac_b = by_l / (avg_ms * 1e-3) / 1e9 / HBM_PEAK_GBS if by else 0.0
    if frac_f >= frac_b:
        roof = {"bound": "mfma", "achieved": round(mult * fl_l / (avg_ms * 1e-3) / 1e12, 3),
                "peak": peak_f, "unit": "TFLOP/s", "frac": round(frac_f, 4), "mfma_basis": basis}
    else:
        roof = {"bound": "hbm", "achieved": round(by_l / (avg_ms * 1e-3) / 1e9, 2),
                "peak": HBM_PEAK_GBS, "unit": "GB/s", "frac": round(frac_b, 4)}
    wl_key = f"config{wl.cfg}-{args.sides}" + ("-ef" if args.ef else "")
    traffic = measured_traffic(dom, wl_key)
    timed_avg = dom_ms_total / dom_launches if dom_launches else None
    roof.update({"kernel": dom, "avg_launch_ms": round(avg_ms, 5),
                 "launch_source": "isolated launches (untimed pass, every launch on one stream)",
                 "timed_region_avg_launch_ms": round(timed_avg, 5) if timed_avg else None,
                 "algorithmic_gb_per_launch": round(by_l / 1e9, 4),
                 "algorithmic_tflop_per_launch": round(fl_l / 1e12, 4),
                 "traffic": round(traffic / 1e9, 4) if traffic is not None else None})
    if traffic is not None:
        roof["traffic_unit"] = "GB per launch (rocprofv3 FETCH_SIZE + WRITE_SIZE, copy-calibrated)"
    tf_fams = ("project", "update_amax", "update_quant", "decode_project", "update_store")
    tf_ms = sum(fam_ms[k][1] for k in tf_fams if k in fam_ms)
    tf_flops = sum(work[k][0] for k in tf_fams if k in work)
    line = {
        "metric": "gradient GB/s through GIFT encode+decode; transform TFLOP/s; % of roofline",
        "value": round(value, 3),
        "unit": "GB/s",
        "n_gpus": 1,
        "steps": nsteps,
        "warmup": args.warmup,
        "ms_per_step": round(ms_step, 4),
        "ms_per_step_raw": round(ms_raw, 4),
        "ms_refresh_step": round(t_ref, 4),
        "ms_codec_step": round(t_cod, 4) if t_cod is not None else None,
        "host_issue_ms_per_step": round(enqueue / nsteps * 1e3, 3),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "f32",
        "dtype_detail": "float32 gradients, transforms and accumulation; the forward transform's "
                        "products as three bf16 MFMA products of hi/lo splits of both float32 operands "
                        "(within 1e-5 of float64); the inverse on FP32 MFMA; statistics from bf16 "
                        "inputs on BF16 MFMA with float32 sums; FP8 E4M3 codes",
        "data": "synthetic",
        "config": {"workload": f"{wl.name} (config {wl.cfg})", "ranks": wl.N, "rank": wl.rank,
                   "sides": args.sides, "tokens": wl.T,
                   "matrices": sum(len(jb.mats) for jb in jobs), "buckets": len(jobs),
                   "format": args.format, "error_feedback": bool(args.ef),
                   "factors": sum(1 for jb in jobs if jb.owns_factor), "streams": nstreams,
                   "grad_gb": round(grad_bytes / 1e9, 3), "factor_refresh_every": wl.refresh,
                   "refreshes_timed": len(ref_ms), "subspace_iters": args.iters,
                   "mall_flushed": bool(args.flush_mall), "decode": args.decode,
                   "assign": args.assign, "hw_queues": int(os.environ.get("GPU_MAX_HW_QUEUES", "0") or 0),
                   "stream_gb": [round(x * 4 / 1e9, 2) for x in stream_load]},
        "transform_tflops": round(tf_flops / (tf_ms * 1e-3) / 1e12, 3) if tf_ms else None,
        "roofline": roof,
        "kernels": kernels,
        "kernels_note": "per-family time per step (refresh amortised over the cadence) from an untimed "
                        "pass with every launch on one stream",
        "latency_bound_ms_per_step": latency_ms,
    }
    if not args.no_cpu_baseline:
        print("[bench] timing the oracle on the host", file=sys.stderr, flush=True)
        line["cpu_baseline"] = cpu_baseline(wl, jobs, args.cpu_seconds)
    torch.cuda.synchronize()
    for jb in jobs:
        if jb.owns_factor:
            jb.factor.close()
    for c in ctxs[1:]:
        c.close()
    ctx.close()
    print(json.dumps(line), flush=True)


if __name__ == "__main__":
    main()
