"""Benchmark: one step = forward + backward of every CoLA projection of a
LLaMA-shaped decoder block (q, k, v, o, gate, up, down), all through the
C ABI of libcola.so on one MI355X.

Default workload: the LLaMA-1B-shaped block (d = 2048, ffn = 5461, r = 512,
T = 128 x 256 = 32768 tokens), bf16 storage with fp32 accumulation, SiLU.
Reported value: algorithmic TFLOP/s = sum over projections of
6 T r (d_in + d_out) per step (Sec. 3.4: 2MNK per GEMM, sigma excluded),
divided by the measured step time.  Inputs are resident in HBM before the
timed region, which records no event between launches; a second pass of the
same K steps with a HIP event pair around every launch gives the per-kernel
durations (roofline of the dominant kernel).  Also measured on the same harness: the CoLA-M step and the
dense full-rank step (6 T d_in d_out), for tokens/s and the speedup; the
block with same-input projections grouped (q+k+v and gate+up share one
input: one GEMM for their Z, dX and dA each); and the inference forward of
that block (nothing kept for a backward pass) against the dense forward.

Prints ONE JSON line.
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

import numpy as np  # noqa: E402

BF16_PEAK_TFLOPS = 2516.6     # MI355X dense bf16 MFMA: 256 CU x 4096 flop/clk x 2.4 GHz
FP32_PEAK_TFLOPS = 157.3
HBM_PEAK_GBS = 8000.0


def parse():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1, help="GPUs (one only: the library runs on a single GPU)")
    ap.add_argument("--steps", type=int, default=20, help="timed steps of the headline pass")
    ap.add_argument("--warmup", type=int, default=5, help="untimed steps before them")
    ap.add_argument("--workload", type=int, default=4, help="1..5 (default 4: LLaMA-1B-shaped block)")
    ap.add_argument("--no-cpu-baseline", action="store_true", help="skip timing the fp64 oracle on the host")
    ap.add_argument("--streams", type=int, default=2,
                    help="HIP streams the independent projections (or groups) of every step are spread over")
    ap.add_argument("--no-dense", action="store_true", help="skip the dense-layer baseline")
    ap.add_argument("--no-cola-m", action="store_true", help="skip the CoLA-M mode")
    ap.add_argument("--cpu-tokens", type=int, default=8192,
                    help="tokens per projection in the oracle's CPU sample")
    ap.add_argument("--no-fused", action="store_true",
                    help="skip the block with same-input projections grouped (q,k,v and gate,up)")
    ap.add_argument("--only", choices=["cola", "cola_m", "dense", "block"], default=None,
                    help="run only one mode (profiling)")
    ap.add_argument("--no-block", action="store_true", help="skip the decoder-block record")
    ap.add_argument("--no-workloads", action="store_true", help="skip the records of the other workloads")
    ap.add_argument("--sub-steps", type=int, default=50, help="timed steps of the block and workload records")
    ap.add_argument("--sub-warmup", type=int, default=10, help="untimed steps before them")
    ap.add_argument("--per-projection", action="store_true",
                    help="per-projection kernel-class durations of the workload (event-timed, one stream) and exit")
    ap.add_argument("--library-baseline", action="store_true",
                    help="time hipBLASLt (torch.matmul) on the workload's GEMM shapes and exit")
    ap.add_argument("--hbm-ceilings", action="store_true",
                    help="time plain read / write / copy / add passes over 1 GiB and exit")
    ap.add_argument("--copy-calibration", action="store_true",
                    help="run only a plain 1 GiB device copy (3 times), for scaling HBM counters")
    ap.add_argument("--traffic-from", nargs=4, metavar=("FETCH_CSV", "WRITE_CSV", "COPY_FETCH_CSV",
                                                         "COPY_WRITE_CSV"),
                    help="summarise rocprofv3 --pmc FETCH_SIZE / WRITE_SIZE runs into "
                         "profiles/traffic.json and exit (no GPU use)")
    return ap.parse_args()


COPY_BYTES = 1 << 30
# the workload of the headline line (LLaMA-1B-shaped block); its counter readings sit at the
# top level of profiles/traffic.json
HEADLINE_WORKLOAD = 4
KERNEL_TAGS = {0: "fwd_z_sigma", 1: "fwd_y", 2: "bwd_dz", 3: "bwd_dx", 4: "bwd_da", 5: "bwd_db",
               7: "dense_fwd", 8: "dense_dx", 9: "dense_dw"}


def copy_calibration():
    """Dispatches of known HBM traffic for scaling the counters: a plain 1 GiB
    device copy (reads and writes COPY_BYTES), then a read-only pass, a sum
    over the same 1 GiB (reads COPY_BYTES, writes a few bytes), 3 times each."""
    import torch
    src = torch.empty(COPY_BYTES, dtype=torch.uint8, device="cuda:0").fill_(1)
    dst = torch.empty_like(src)
    torch.cuda.synchronize()
    for _ in range(3):
        dst.copy_(src)
    torch.cuda.synchronize()
    f = src.view(torch.float32)
    for _ in range(3):
        f.sum()
    torch.cuda.synchronize()
    print(json.dumps({"copy_calibration_bytes": COPY_BYTES, "repeats": 3, "read_only_pass": "sum"}), flush=True)


def hbm_ceilings(nbytes=COPY_BYTES, reps=10):
    """What this machine's HBM sustains for plain streaming patterns over nbytes
    buffers (torch's own kernels, the median of `reps` event-timed launches
    after two warm-up ones): a read-only pass (row sums), a write-only pass (a
    fill), a copy (one read and one write stream) and two reads with one
    write (an add): the practical ceilings for kernels that read and write,
    beside the nominal 8 TB/s."""
    import torch
    n = nbytes // 4
    a = torch.ones(n, dtype=torch.float32, device="cuda:0")
    b = torch.ones(n, dtype=torch.float32, device="cuda:0")
    c = torch.empty(n, dtype=torch.float32, device="cuda:0")
    # read-only: row sums over 65536 rows of 16 KB (a single full reduction
    # keeps too few loads in flight: 3.9 against 6.1 TB/s, measured)
    pats = {"read": (lambda: a.view(65536, -1).sum(1), 1), "write": (lambda: c.fill_(2.0), 1),
            "copy": (lambda: c.copy_(a), 2), "read2_write1": (lambda: torch.add(a, b, out=c), 3)}
    out = {"buffer_bytes": nbytes}
    for name, (fn, streams) in pats.items():
        for _ in range(2):
            fn()
        times = []
        for _ in range(reps):
            s = torch.cuda.Event(enable_timing=True)
            e = torch.cuda.Event(enable_timing=True)
            s.record()
            fn()
            e.record()
            torch.cuda.synchronize()
            times.append(s.elapsed_time(e))
        ms = sorted(times)[len(times) // 2]
        out[name + "_gbs"] = round(streams * nbytes / (ms * 1e6), 1)
    del a, b, c
    torch.cuda.empty_cache()
    return out


def _pmc_rows(path, counter):
    import csv
    rows = []
    for r in csv.DictReader(open(path)):
        if r.get("Counter_Name") != counter:
            continue
        rows.append((r["Kernel_Name"], int(r["Dispatch_Id"]), float(r["Counter_Value"])))
    return rows


def traffic_summary(fetch_csv, write_csv, copy_fetch_csv, copy_write_csv, workload=4):
    """HBM bytes per launch for each GEMM kernel class, from rocprofv3 --pmc
    FETCH_SIZE and WRITE_SIZE (KiB per dispatch), each scaled by the ratio of
    the known bytes of a plain 1 GiB copy to what the same counter reads for
    that copy.  The headline workload's classes sit at the top level of
    profiles/traffic.json, another workload's under "workload_<n>"; the other
    sections of the file are kept."""
    import hashlib
    import re

    def copy_factor(path, counter):
        vals = [v for name, _, v in _pmc_rows(path, counter) if "copy" in name.lower()
                or "elementwise" in name.lower()]
        big = [v for v in vals if v * 1024 > 0.5 * COPY_BYTES]
        if not big:
            raise SystemExit(f"no copy dispatch found in {path}")
        return COPY_BYTES / (sorted(big)[len(big) // 2] * 1024.0)

    ff = copy_factor(copy_fetch_csv, "FETCH_SIZE")
    fw = copy_factor(copy_write_csv, "WRITE_SIZE")
    # cross-check of the fetch factor: the read-only pass (a reduction over the
    # same 1 GiB) in the same counter run
    ro = [v for name, _, v in _pmc_rows(copy_fetch_csv, "FETCH_SIZE") if "reduce" in name.lower()
          and v * 1024 > 0.25 * COPY_BYTES]
    ff_ro = COPY_BYTES / (sorted(ro)[len(ro) // 2] * 1024.0) if ro else None
    per = {}
    for path, counter, scale, key in ((fetch_csv, "FETCH_SIZE", ff, "fetch"),
                                      (write_csv, "WRITE_SIZE", fw, "write")):
        for name, _, v in _pmc_rows(path, counter):
            m = re.search(r"gemm_\w+_kernel<[^>]*, (\d+)>", name)
            if not m:
                continue
            # the launch of both weight gradients carries the dA tag
            cls = "bwd_da_db" if "pair_kernel" in name else KERNEL_TAGS.get(int(m.group(1)))
            per.setdefault(cls, {}).setdefault(key, []).append(v * 1024.0 * scale)
    h = kernel_source_hash()
    sec = {"_note": "HBM bytes per launch from rocprofv3 FETCH_SIZE + WRITE_SIZE, scaled by a "
                    "1 GiB copy (fetch factor %.4f, write factor %.4f; a read-only 1 GiB pass gives fetch "
                    "factor %s)" % (ff, fw, "%.4f" % ff_ro if ff_ro else "n/a"),
           "_fetch_factor": ff, "_write_factor": fw, "_fetch_factor_read_only": ff_ro}
    for cls, d in per.items():
        f = d.get("fetch", [])
        w = d.get("write", [])
        if not f or not w:
            continue
        sec[cls] = {"bytes_per_launch": sum(f) / len(f) + sum(w) / len(w),
                    "fetch_bytes_per_launch": sum(f) / len(f),
                    "write_bytes_per_launch": sum(w) / len(w),
                    "launches": len(f), "source_sha256_16": h}
    path = os.path.join(ROOT, "profiles", "traffic.json")
    out = {}
    if os.path.exists(path):
        try:
            out = json.load(open(path))
        except (OSError, ValueError):
            out = {}
    if workload == HEADLINE_WORKLOAD:
        out = {k: v for k, v in out.items() if k.startswith("workload_")}
        out.update(sec)
    else:
        out["workload_%d" % workload] = sec
    with open(path, "w") as fh:
        json.dump(out, fh, indent=1, sort_keys=True)
    print(json.dumps(sec), flush=True)


def algo_flops_cola(T, d_in, d_out, r):
    """fwd + bwd of one CoLA layer: 6 GEMMs of 2 T r d each (Sec. 3.4)."""
    return 6.0 * T * r * (d_in + d_out)


def algo_flops_cola_fwd(T, d_in, d_out, r):
    """forward only (inference): the two GEMMs of Eq. main-fwd, 2 T r d each."""
    return 2.0 * T * r * (d_in + d_out)


def algo_flops_dense(T, d_in, d_out):
    """fwd + bwd of one dense layer: 3 GEMMs of 2 T d_in d_out each."""
    return 6.0 * T * d_in * d_out


class Projection:
    def __init__(self, cfg, name, idx, d_in, d_out, r, T, dtype, dense: bool, recompute_too: bool):
        import torch
        from paper_2502_10940_amd import cola
        from paper_2502_10940_amd import inputs as I
        self.name, self.T, self.d_in, self.d_out, self.r = name, T, d_in, d_out, r
        self.dtype = dtype
        tdt = torch.bfloat16 if dtype == "bf16" else torch.float32
        dev = "cuda:0"
        self.ldx = I.padded_ld(d_in, dtype)
        self.ldy = I.padded_ld(d_out, dtype)
        self.ldz = I.padded_ld(r, dtype)
        ins = I.layer_inputs(cfg, idx, d_in, d_out, r, T, dtype, with_dense=dense)
        self.host = ins

        def put(t, ld=None):
            a = t.store
            if ld is not None and ld != a.shape[1]:
                a = I.with_pitch(a, ld, 0)
            if dtype == "bf16":
                x = torch.from_numpy(np.ascontiguousarray(a).view(np.int16)).to(dev).view(torch.bfloat16)
            else:
                x = torch.from_numpy(np.ascontiguousarray(a)).to(dev)
            return x

        self.X = put(ins["X"], self.ldx)
        self.A = put(ins["A"])
        self.B = put(ins["B"])
        self.dY = put(ins["dY"], self.ldy)
        self.W = put(ins["W"]) if dense else None
        self.Y = torch.empty((T, self.ldy), dtype=tdt, device=dev)
        self.Z = torch.empty((T, self.ldz), dtype=tdt, device=dev)
        self.H = torch.empty((T, self.ldz), dtype=tdt, device=dev)
        self.dX = torch.empty((T, self.ldx), dtype=tdt, device=dev)
        self.dA = torch.empty((r, d_in), dtype=torch.float32, device=dev)
        self.dB = torch.empty((d_out, r), dtype=torch.float32, device=dev)
        self.dW = torch.empty((d_out, d_in), dtype=torch.float32, device=dev) if dense else None
        self.desc = cola.desc(T, d_in, d_out, r, dtype, "silu", False, self.ldx, self.ldy, self.ldz)
        self.desc_m = cola.desc(T, d_in, d_out, r, dtype, "silu", True, self.ldx, self.ldy, self.ldz)
        self.ddesc = cola.dense_desc(T, d_in, d_out, dtype, self.ldx, self.ldy)
        self.ws_need = max(cola.workspace_bytes(self.desc, 0), cola.workspace_bytes(self.desc, 1),
                           cola.workspace_bytes(self.desc, 2),
                           cola.workspace_bytes(self.desc_m, 0) if recompute_too else 0,
                           cola.workspace_bytes(self.desc_m, 1) if recompute_too else 0,
                           cola.dense_workspace_bytes(self.ddesc, 0) if dense else 0,
                           cola.dense_workspace_bytes(self.ddesc, 1) if dense else 0)

    def fwd(self, ws, recompute=False):
        from paper_2502_10940_amd import cola
        if recompute:
            cola.fwd(self.desc_m, self.X, self.A, self.B, self.Y, self.Z, None, ws)
        else:
            cola.fwd(self.desc, self.X, self.A, self.B, self.Y, self.Z, self.H, ws)

    def bwd(self, ws, recompute=False):
        from paper_2502_10940_amd import cola
        if recompute:
            cola.bwd(self.desc_m, self.dY, self.X, self.Z, None, self.A, self.B, self.dX, self.dA,
                     self.dB, ws)
        else:
            cola.bwd(self.desc, self.dY, self.X, self.Z, self.H, self.A, self.B, self.dX, self.dA,
                     self.dB, ws)

    def infer(self, ws):
        from paper_2502_10940_amd import cola
        cola.infer(self.desc, self.X, self.A, self.B, self.Y, ws)

    def dense_fwd(self, ws):
        from paper_2502_10940_amd import cola
        cola.dense_fwd(self.ddesc, self.X, self.W, self.Y, ws)

    def dense_step(self, ws):
        from paper_2502_10940_amd import cola
        cola.dense_fwd(self.ddesc, self.X, self.W, self.Y, ws)
        cola.dense_bwd(self.ddesc, self.dY, self.X, self.W, self.dX, self.dW, ws)


class Group:
    """Projections that read the same input (q, k, v; gate, up) run through the
    grouped entry points: the first member's X is the shared input; the members'
    weights, output and gradient buffers are reused."""

    def __init__(self, members, dtype):
        import torch
        from paper_2502_10940_amd import cola
        from paper_2502_10940_amd import inputs as I
        self.m = members
        p0 = members[0]
        T, d_in = p0.T, p0.d_in
        ranks = [p.r for p in members]
        self.R = sum(ranks)
        tdt = torch.bfloat16 if dtype == "bf16" else torch.float32
        dev = "cuda:0"
        self.ldz = I.padded_ld(self.R, dtype)
        self.A_all = torch.cat([p.A for p in members], dim=0).contiguous()
        self.Z = torch.empty((T, self.ldz), dtype=tdt, device=dev)
        self.H = torch.empty((T, self.ldz), dtype=tdt, device=dev)
        self.dA = torch.empty((self.R, d_in), dtype=torch.float32, device=dev)
        self.desc = cola.group_desc(T, d_in, ranks, [p.d_out for p in members], dtype, "silu", False,
                                    ldx=p0.ldx, ldz=self.ldz, ldy=[p.ldy for p in members])
        self.ws_need = max(cola.group_workspace_bytes(self.desc, p) for p in (0, 1, 2))

    def fwd(self, ws):
        from paper_2502_10940_amd import cola
        p0 = self.m[0]
        cola.group_fwd(self.desc, p0.X, self.A_all, [p.B for p in self.m], [p.Y for p in self.m], self.Z, self.H, ws)

    def infer(self, ws):
        from paper_2502_10940_amd import cola
        cola.group_infer(self.desc, self.m[0].X, self.A_all, [p.B for p in self.m], [p.Y for p in self.m], ws)

    def bwd(self, ws):
        from paper_2502_10940_amd import cola
        p0 = self.m[0]
        cola.group_bwd(self.desc, [p.dY for p in self.m], p0.X, self.Z, self.H, self.A_all, [p.B for p in self.m],
                       p0.dX, self.dA, [p.dB for p in self.m], ws)


def proj_work(item, dense=False):
    """Relative work of a projection (a group: the sum over its members):
    T d_in d_out for the dense layer, T r (d_in + d_out) for CoLA."""
    if isinstance(item, Group):
        return sum(proj_work(m, dense) for m in item.m)
    return item.T * (item.d_in * item.d_out if dense else item.r * (item.d_in + item.d_out))


def assign_streams(works, nstreams):
    """Stream index of each item: largest work first, each to the stream with
    the least work so far (ties to the lowest index, stream 0 being the
    caller's current stream)."""
    load = [0.0] * nstreams
    out = [0] * len(works)
    for i in sorted(range(len(works)), key=lambda i: -works[i]):
        k = min(range(nstreams), key=lambda k: load[k])
        out[i] = k
        load[k] += works[i]
    return out


def timed_steps(step, steps, warmup):
    import torch
    for _ in range(warmup):
        step()
    torch.cuda.synchronize()
    s = torch.cuda.Event(enable_timing=True)
    e = torch.cuda.Event(enable_timing=True)
    s.record()
    for _ in range(steps):
        step()
    e.record()
    torch.cuda.synchronize()
    return s.elapsed_time(e) / steps


def timed_steps_median(step, steps, warmup):
    """Median of per-step times (HIP events around each step): the secondary
    measurements, robust to a stall of the host or the box in one step."""
    import torch
    for _ in range(warmup):
        step()
    torch.cuda.synchronize()
    ev = [torch.cuda.Event(enable_timing=True) for _ in range(steps + 1)]
    ev[0].record()
    for i in range(steps):
        step()
        ev[i + 1].record()
    torch.cuda.synchronize()
    t = sorted(ev[i].elapsed_time(ev[i + 1]) for i in range(steps))
    return t[len(t) // 2]


def kernel_table(cola):
    out = {}
    for k, name in enumerate(cola.KERNEL_CLASSES):
        n, ms, fl, by = cola.timing_read(k)
        if n == 0:
            continue
        out[name] = {"launches": n, "avg_us": 1000.0 * ms / n, "total_ms": ms,
                     "tflops": fl / (ms * 1e9) if ms > 0 else 0.0,
                     "gbs": by / (ms * 1e6) if ms > 0 else 0.0,
                     "flops_per_launch": fl / n, "bytes_per_launch": by / n}
    return out


# the sources the layer's GEMM kernels and their launch plans are built from
GEMM_SOURCES = ("cola_abi.hip", "device_math.hpp", "epilogue.hpp", "gemm_dispatch.hip", "gemm_f32.hip",
                "gemm_pp.hip", "gemm_stream.hip", "internal.hpp", "lds_tile.hpp")


def kernel_source_hash():
    """sha256 (first 16 hex digits) over the sources of the layer's GEMM kernels
    and their launch plans, so a stored counter reading is dropped as soon as
    any of them changes."""
    import hashlib
    d = os.path.join(ROOT, "paper_2502_10940_amd", "csrc")
    h = hashlib.sha256()
    for name in GEMM_SOURCES:
        h.update(name.encode())
        h.update(open(os.path.join(d, name), "rb").read())
    return h.hexdigest()[:16]


def load_traffic(kernel, workload=4):
    """HBM bytes per launch measured by rocprofv3 counters (profiles/traffic.json),
    or None when absent or taken on a different kernel source."""
    path = os.path.join(ROOT, "profiles", "traffic.json")
    if not os.path.exists(path):
        return None
    try:
        rec = json.load(open(path))
    except (OSError, ValueError):
        return None
    if workload != HEADLINE_WORKLOAD:
        rec = rec.get("workload_%d" % workload, {})
    ent = rec.get(kernel)
    if not ent:
        return None
    if ent.get("source_sha256_16") != kernel_source_hash():
        return None
    return ent.get("bytes_per_launch")


def cpu_baseline(projs, cfg_T, tokens):
    """The fp64 oracle (test infrastructure, untuned) on a bounded sample: the
    first ``tokens`` tokens of each projection, forward + backward."""
    import oracle
    from paper_2502_10940_amd import inputs as I
    t_total = 0.0
    flops = 0.0
    for p in projs:
        X = I.Tensor(p.host["X"].store[:tokens], p.dtype).f64
        A = p.host["A"].f64
        B = p.host["B"].f64
        dY = I.Tensor(p.host["dY"].store[:tokens], p.dtype).f64
        t0 = time.perf_counter()
        Z, _, _ = oracle.cola_fwd(X, A, B, "silu")
        oracle.cola_bwd(X, Z, A, B, dY, "silu")
        t_total += time.perf_counter() - t0
        flops += algo_flops_cola(tokens, p.d_in, p.d_out, p.r)
    return {"value": flops / t_total / 1e12, "unit": "TFLOP/s", "cores": oracle.num_threads(),
            "kind": "oracle",
            "sample": f"first {tokens} of {cfg_T} tokens of each of the {len(projs)} projections, "
                      f"fwd+bwd in fp64 ({t_total:.1f} s)",
            "seconds": t_total, "tokens_per_s": tokens / t_total}


class Harness:
    """The projections of one workload on the device, their grouping, the
    streams they are spread over and one workspace per stream; the step
    functions of every measured mode."""

    def __init__(self, cfg, dense, cola_m, fused, nstreams):
        import torch
        from paper_2502_10940_amd import inputs as I
        w = I.WORKLOADS[cfg]
        self.cfg, self.w = cfg, w
        self.dtype = w["dtype"]
        self.T, self.r = w["T"], w["r"]
        self.projs = [Projection(cfg, name, idx, d_in, d_out, self.r, self.T, self.dtype, dense, cola_m)
                      for name, idx, d_in, d_out in I.projections(cfg)]
        self.units = []     # the grouped block: groups for same-input projections, single layers otherwise
        if fused and cfg != 1:
            by = {p.name: p for p in self.projs}
            self.units = [Group([by["q"], by["k"], by["v"]], self.dtype), by["o"],
                          Group([by["gate"], by["up"]], self.dtype), by["down"]]
        ws_need = max([p.ws_need for p in self.projs] + [u.ws_need for u in self.units if isinstance(u, Group)])
        # independent projections spread over several HIP streams (default
        # priority), each with its own workspace, balanced by work: a
        # projection runs its forward and backward on one stream, and one
        # kernel's ramp-up overlaps another stream's drain.  The step still
        # starts and ends on the current stream.
        self.nstreams = max(1, nstreams)
        self.streams = [None] + [torch.cuda.Stream() for _ in range(self.nstreams - 1)]
        self.wss = [torch.empty(ws_need, dtype=torch.uint8, device="cuda:0") for _ in range(self.nstreams)]
        self.flops_cola = sum(algo_flops_cola(self.T, p.d_in, p.d_out, self.r) for p in self.projs)
        self.flops_dense = sum(algo_flops_dense(self.T, p.d_in, p.d_out) for p in self.projs)
        self.flops_infer = sum(algo_flops_cola_fwd(self.T, p.d_in, p.d_out, self.r) for p in self.projs)

    def spread(self, items, fwd, bwd=None, dense=False):
        """fwd over items in order, then bwd in reverse order; each item on
        the stream `assign_streams` gives it, with that stream's workspace."""
        import torch
        main = torch.cuda.current_stream()
        for st in self.streams[1:]:
            st.wait_stream(main)
        where = assign_streams([proj_work(x, dense) for x in items], self.nstreams)
        order = list(enumerate(items))
        phases = [(fwd, order)] + ([(bwd, order[::-1])] if bwd is not None else [])
        for phase, seq in phases:
            for i, p in seq:
                k = where[i]
                if k == 0:
                    phase(p, self.wss[0])
                else:
                    with torch.cuda.stream(self.streams[k]):
                        phase(p, self.wss[k])
        for st in self.streams[1:]:
            main.wait_stream(st)

    def step(self, mode):
        if mode == "cola":
            return lambda: self.spread(self.projs, lambda p, w: p.fwd(w), lambda p, w: p.bwd(w))
        if mode == "cola_1s":           # one stream: the pass whose launches carry events
            def run():
                for p in self.projs:
                    p.fwd(self.wss[0])
                for p in reversed(self.projs):
                    p.bwd(self.wss[0])
            return run
        if mode == "cola_m":
            return lambda: self.spread(self.projs, lambda p, w: p.fwd(w, True), lambda p, w: p.bwd(w, True))
        if mode == "fused":
            return lambda: self.spread(self.units, lambda u, w: u.fwd(w), lambda u, w: u.bwd(w))
        if mode == "dense":
            return lambda: self.spread(self.projs, lambda p, w: p.dense_step(w), dense=True)
        if mode == "infer":
            return lambda: self.spread(self.units, lambda u, w: u.infer(w))
        if mode == "dense_infer":
            return lambda: self.spread(self.projs, lambda p, w: p.dense_fwd(w), dense=True)
        raise ValueError(mode)


class SclkSampler:
    """The GPU's current shader clock (MHz) and board power (W), sampled from
    the driver's sysfs DPM table and power sensor while a measurement runs;
    None where they are not readable."""

    def __init__(self):
        import glob
        self.files = sorted(glob.glob("/sys/class/drm/card*/device/pp_dpm_sclk"))
        self.pfiles = sorted(glob.glob("/sys/class/drm/card*/device/hwmon/hwmon*/power1_input"))
        self.vals = []
        self.pvals = []
        self._stop = None

    @staticmethod
    def _microwatts(path):
        try:
            with open(path) as fh:
                return int(fh.read().strip())
        except (OSError, ValueError):
            return None

    def read_power(self):
        """Board power in W (the sum over the cards the sensors list), or None."""
        vals = [self._microwatts(f) for f in self.pfiles]
        vals = [v for v in vals if v is not None]
        return sum(vals) / 1e6 if vals else None

    def power(self):
        """Median and maximum of the sampled board power and the power cap (W)."""
        if not self.pvals:
            return None
        v = sorted(self.pvals)
        caps = [self._microwatts(f.replace("power1_input", "power1_cap")) for f in self.pfiles]
        caps = [c for c in caps if c]
        return {"median": round(v[len(v) // 2], 1), "max": round(v[-1], 1),
                "cap": round(sum(caps) / 1e6, 1) if caps else None, "samples": len(v)}

    def read(self):
        import re
        best = None
        for f in self.files:
            try:
                with open(f) as fh:
                    for line in fh:
                        if line.rstrip().endswith("*"):
                            m = re.search(r"(\d+)\s*mhz", line, re.I)
                            if m:
                                best = max(best or 0, int(m.group(1)))
            except OSError:
                continue
        return best

    def __enter__(self):
        import threading
        self._stop = threading.Event()

        def loop():
            while not self._stop.is_set():
                v = self.read()
                if v is not None:
                    self.vals.append(v)
                w = self.read_power()
                if w is not None:
                    self.pvals.append(w)
                self._stop.wait(0.01)

        self._t = threading.Thread(target=loop, daemon=True)
        self._t.start()
        return self

    def __exit__(self, *exc):
        self._stop.set()
        self._t.join()

    def median(self):
        if not self.vals:
            return None
        v = sorted(self.vals)
        return v[len(v) // 2]


# shader clock (MHz) at which the nominal MFMA peaks are quoted
NOMINAL_SCLK_MHZ = 2400.0


def at_clock(roofline, sclk_mhz):
    """Beside the fraction of the nominal peak (quoted at 2.4 GHz), an
    MFMA-bound kernel's fraction of the peak at the shader clock sampled during
    the run (the clock falls to 1.4-2.1 GHz under sustained load on MI355X)."""
    if roofline.get("bound") != "mfma" or not sclk_mhz:
        return
    p = roofline["peak"] * sclk_mhz / NOMINAL_SCLK_MHZ
    roofline["peak_at_sclk"] = round(p, 1)
    roofline["frac_at_sclk"] = round(roofline["achieved"] / p, 4)


def roofline_of(kernels, peak):
    """The dominant kernel class (largest total time) against its roofline:
    MFMA-bound when its algorithmic intensity is above the ridge point, else
    HBM-bound."""
    dom = max(kernels, key=lambda k: kernels[k]["total_ms"])
    kd = kernels[dom]
    ai = kd["flops_per_launch"] / kd["bytes_per_launch"] if kd["bytes_per_launch"] > 0 else float("inf")
    ridge = peak * 1e12 / (HBM_PEAK_GBS * 1e9)
    if ai >= ridge:
        achieved = kd["flops_per_launch"] / (kd["avg_us"] * 1e6)        # TFLOP/s
        out = {"kernel": dom, "bound": "mfma", "achieved": round(achieved, 2), "peak": peak, "unit": "TFLOP/s",
               "frac": round(achieved / peak, 4)}
    else:
        achieved = kd["bytes_per_launch"] / (kd["avg_us"] * 1e3)        # GB/s
        out = {"kernel": dom, "bound": "hbm", "achieved": round(achieved, 1), "peak": HBM_PEAK_GBS,
               "unit": "GB/s", "frac": round(achieved / HBM_PEAK_GBS, 4)}
    out.update({"avg_us": round(kd["avg_us"], 2), "flops_per_launch": kd["flops_per_launch"],
                "bytes_per_launch": kd["bytes_per_launch"], "intensity": round(ai, 1), "ridge": round(ridge, 1)})
    return dom, out


def events_pass(cola, step, steps):
    """`steps` steps with a HIP event pair around every launch (recorded on its
    launch stream): per-kernel-class durations."""
    cola.timing_reset()
    cola.timing_enable(True)
    try:
        for _ in range(steps):
            step()
    finally:
        cola.timing_enable(False)
    table = kernel_table(cola)
    cola.timing_reset()
    return table


# modes measured per workload (as the configuration list names them; the
# headline workload measures every mode)
WORKLOAD_MODES = {1: ("cola", "cola_m"), 2: ("cola", "cola_m"), 3: ("cola", "cola_m", "dense"),
                  5: ("cola_m", "cola", "dense")}


def workload_record(cfg, args):
    """Compact record of one workload: median step time over `--sub-steps`
    steps after `--sub-warmup`, per mode, with TFLOP/s, tokens/s, the speedup
    over dense, the dominant kernel against its roofline, and the clock."""
    import torch
    from paper_2502_10940_amd import cola
    from paper_2502_10940_amd import inputs as I
    modes = WORKLOAD_MODES[cfg]
    t0 = time.time()
    h = Harness(cfg, dense="dense" in modes, cola_m="cola_m" in modes, fused=False, nstreams=args.streams)
    setup = time.time() - t0
    peak = BF16_PEAK_TFLOPS if h.dtype == "bf16" else FP32_PEAK_TFLOPS
    rec = {"workload": h.w["name"], "dtype": h.dtype, "tokens": h.T, "steps": args.sub_steps,
           "warmup": args.sub_warmup, "timing": "median per-step HIP events", "modes": {}}
    with SclkSampler() as sc:
        for mode in modes:
            ms = timed_steps_median(h.step(mode), args.sub_steps, args.sub_warmup)
            fl = h.flops_dense if mode == "dense" else h.flops_cola
            rec["modes"][mode] = {"ms_per_step": round(ms, 4), "tflops": round(fl / (ms * 1e9), 2),
                                  "pct_of_peak": round(100.0 * fl / (ms * 1e9) / peak, 2),
                                  "tokens_per_s": round(h.T / (ms / 1e3), 1)}
    rec["sclk_mhz"] = sc.median()
    rec["power_w"] = sc.power()
    if "dense" in rec["modes"]:
        for mode in modes:
            if mode != "dense":
                rec["modes"][mode]["speedup_vs_dense"] = round(rec["modes"]["dense"]["ms_per_step"] /
                                                               rec["modes"][mode]["ms_per_step"], 3)
    main_mode = modes[0]
    kern = events_pass(cola, h.step("cola_1s") if main_mode == "cola" else h.step(main_mode), 3)
    if kern:
        dom, rec["roofline"] = roofline_of(kern, peak)
        rec["roofline"]["traffic"] = load_traffic(dom, cfg)
        at_clock(rec["roofline"], rec["sclk_mhz"])
    rec["setup_s"] = round(setup, 1)
    del h
    torch.cuda.empty_cache()
    return rec


def block_record(cfg, args):
    """The decoder block (cola_block_fwd + cola_block_bwd: norms, attention,
    gated product and the seven CoLA projections) at the workload's shape, in
    CoLA and in CoLA-M: median step time, tokens/s, the saved bytes of each
    mode and the recompute overhead."""
    import torch
    from paper_2502_10940_amd import cola
    from paper_2502_10940_amd import inputs as I
    w = I.WORKLOADS[cfg]
    L = I.SEQ_LEN
    n_seq, d, ffn, r, heads = w["T"] // L, w["d"], w["ffn"], w["r"], I.HEADS[cfg]
    T = n_seq * L
    ins = I.block_inputs(cfg, n_seq, L, d, ffn, r)
    dev = lambda a: torch.from_numpy(np.ascontiguousarray(a).view(np.int16)).to("cuda:0").view(torch.bfloat16)
    wts = {k: dev(ins[k].store) for k in cola.BLOCK_PARAMS}
    x0, dx2 = dev(ins["x0"].store), dev(ins["dx2"].store)
    x2 = torch.empty_like(x0)
    dx0 = torch.empty_like(x0)
    grads = {k: torch.empty(v.shape, dtype=torch.float32, device="cuda:0") for k, v in wts.items()}
    descs = {m: cola.block_desc(n_seq, L, d, ffn, heads, r, "silu", m == "cola_m") for m in ("cola", "cola_m")}
    saved_b = {m: cola.block_saved_bytes(descs[m]) for m in descs}
    ws_b = max(cola.block_workspace_bytes(descs[m], p) for m in descs for p in (0, 1))
    saved = torch.empty(max(saved_b.values()), dtype=torch.uint8, device="cuda:0")
    ws = torch.empty(ws_b, dtype=torch.uint8, device="cuda:0")

    def step(m):
        def run():
            cola.block_fwd(descs[m], wts, x0, x2, saved, ws, saved_b[m], ws_b)
            cola.block_bwd(descs[m], wts, x0, saved, dx2, dx0, grads, ws, saved_b[m], ws_b)
        return run

    shapes = [(d, d)] * 4 + [(d, ffn)] * 2 + [(ffn, d)]
    lin = sum(algo_flops_cola(T, a, b, r) for a, b in shapes)
    pairs = L * (L + 1) / 2
    attn = 12.0 * pairs * d * n_seq                     # causal: 4 (fwd) + 8 (bwd) flops per pair and element
    rec = {"workload": f"decoder block at the {w['name']}, heads={heads}, seq_len={L}",
           "tokens": T, "steps": args.sub_steps, "warmup": args.sub_warmup,
           "flops_per_step": {"projections": lin, "attention_causal": attn},
           "saved_bytes": dict(saved_b), "input_bytes": 2 * T * d, "modes": {}}
    with SclkSampler() as sc:
        for m in ("cola", "cola_m"):
            ms = timed_steps_median(step(m), args.sub_steps, args.sub_warmup)
            rec["modes"][m] = {"ms_per_step": round(ms, 4), "tokens_per_s": round(T / (ms / 1e3), 1),
                               "tflops": round((lin + attn) / (ms * 1e9), 2)}
    rec["sclk_mhz"] = sc.median()
    rec["power_w"] = sc.power()
    # CoLA-M's activation memory against CoLA's, the caller's x0 counted in both
    rec["cola_m_memory_ratio"] = round((saved_b["cola_m"] + 2 * T * d) / (saved_b["cola"] + 2 * T * d), 4)
    rec["cola_m_overhead"] = round(rec["modes"]["cola_m"]["ms_per_step"] / rec["modes"]["cola"]["ms_per_step"] - 1,
                                   4)
    kern = events_pass(cola, step("cola_m"), 2)
    rec["cola_m_kernels_ms_per_step"] = {k: round(v["total_ms"] / 2, 4) for k, v in kern.items()}
    del saved, ws
    torch.cuda.empty_cache()
    return rec


def library_baseline(args):
    """hipBLASLt through torch.matmul (bf16 in, fp32 accumulate) on the GEMM
    shapes of the headline workload's CoLA steps and dense layers, for
    comparison with the library's own kernels: median of 20 launches each."""
    import torch
    from paper_2502_10940_amd import inputs as I
    w = I.WORKLOADS[args.workload]
    T, r = w["T"], w["r"]
    shapes = {}
    for name, idx, d_in, d_out in I.projections(args.workload):
        # (M, N, K): the six CoLA GEMMs and the three dense ones
        for step, mnk in (("K1 Z=X A^T", (T, r, d_in)), ("K2 Y=H B^T", (T, d_out, r)),
                          ("K3 dH=dY B", (T, r, d_out)), ("K4 dX=dZ A", (T, d_in, r)),
                          ("K5 dA=dZ^T X", (r, d_in, T)), ("K6 dB=dY^T H", (d_out, r, T)),
                          ("D1 Y=X W^T", (T, d_out, d_in)), ("D2 dX=dY W", (T, d_in, d_out)),
                          ("D3 dW=dY^T X", (d_out, d_in, T))):
            shapes.setdefault((step, mnk), 0)
            shapes[(step, mnk)] += 1
    out = {"library": "hipBLASLt (torch.matmul, bf16)", "workload": w["name"], "shapes": []}
    for (step, (M, N, K)), count in sorted(shapes.items()):
        a = torch.randn(M, K, device="cuda:0", dtype=torch.bfloat16)
        b = torch.randn(K, N, device="cuda:0", dtype=torch.bfloat16)
        ms = timed_steps_median(lambda: torch.matmul(a, b), 20, 5)
        out["shapes"].append({"step": step, "M": M, "N": N, "K": K, "projections": count, "ms": round(ms, 4),
                              "tflops": round(2.0 * M * N * K / (ms * 1e9), 1)})
        del a, b
    print(json.dumps(out), flush=True)


def vendor_dense_step_ms(workload, reps=20, warmup=5):
    """The dense layer's step on hipBLASLt (torch.matmul, bf16 in, fp32
    accumulate): the median time of each of its GEMM shapes (Y = X W^T,
    dX = dY W, dW = dY^T X per projection), summed over the step.  Context for
    the speedup, which the bench line quotes against the dense layer on this
    library's own kernels."""
    import torch
    from paper_2502_10940_amd import inputs as I
    T = I.WORKLOADS[workload]["T"]
    count = {}
    for _, _, d_in, d_out in I.projections(workload):
        for mnk in ((T, d_out, d_in), (T, d_in, d_out), (d_out, d_in, T)):
            count[mnk] = count.get(mnk, 0) + 1
    total = 0.0
    for (M, N, K), n in sorted(count.items()):
        a = torch.randn(M, K, device="cuda:0", dtype=torch.bfloat16)
        b = torch.randn(K, N, device="cuda:0", dtype=torch.bfloat16)
        total += n * timed_steps_median(lambda: torch.matmul(a, b), reps, warmup)
        del a, b
    return total


def per_projection(args):
    """Kernel-class durations per projection: after 3 warm-up steps, each
    projection's forward and backward 5 times with an event pair around every
    launch (one stream).  One JSON line per projection."""
    import torch
    from paper_2502_10940_amd import cola
    h = Harness(args.workload, dense=False, cola_m=False, fused=False, nstreams=1)
    ws = h.wss[0]
    step = h.step("cola_1s")
    for _ in range(3):
        step()
    torch.cuda.synchronize()
    for p in h.projs:
        cola.timing_reset()
        cola.timing_enable(True)
        for _ in range(5):
            p.fwd(ws)
            p.bwd(ws)
        cola.timing_enable(False)
        t = kernel_table(cola)
        print(json.dumps({"projection": p.name, "d_in": p.d_in, "d_out": p.d_out, "r": p.r, "T": p.T,
                          "avg_us": {k: round(v["avg_us"], 1) for k, v in t.items()},
                          "tflops": {k: round(v["tflops"], 1) for k, v in t.items()}}), flush=True)
    cola.timing_reset()


def main():
    args = parse()
    if args.traffic_from:
        traffic_summary(*args.traffic_from, workload=args.workload)
        return
    if args.gpus != 1:
        print(f"bench.py measures one GPU only (got --gpus {args.gpus}); the library runs on a single GPU "
              "and has no multi-GPU path", file=sys.stderr)
        sys.exit(2)
    import torch
    from paper_2502_10940_amd import cola
    from paper_2502_10940_amd import inputs as I

    if args.copy_calibration:
        copy_calibration()
        return
    if args.hbm_ceilings:
        print(json.dumps({"hbm_ceilings": hbm_ceilings()}), flush=True)
        return
    cola.lib()
    if args.library_baseline:
        library_baseline(args)
        return
    if args.per_projection:
        per_projection(args)
        return
    if args.only == "block":
        # the decoder-block record alone (profiling)
        print(json.dumps({"block": block_record(args.workload, args)}), flush=True)
        return
    w = I.WORKLOADS[args.workload]
    dtype = w["dtype"]
    T, r = w["T"], w["r"]
    do_dense = not args.no_dense and args.only in (None, "dense")
    do_m = not args.no_cola_m and args.only in (None, "cola_m")
    do_cola = args.only in (None, "cola")
    do_fused = not args.no_fused and args.only is None and args.workload != 1
    t0 = time.time()
    h = Harness(args.workload, do_dense, do_m, do_fused, args.streams)
    setup_s = time.time() - t0
    projs = h.projs
    flops_cola, flops_dense = h.flops_cola, h.flops_dense
    peak = BF16_PEAK_TFLOPS if dtype == "bf16" else FP32_PEAK_TFLOPS

    res = {}
    kernels = {}
    sampler = SclkSampler()
    with sampler:
        if do_cola:
            # the headline: exactly K steps as a caller runs them, no per-kernel events
            cola.timing_enable(False)
            res["cola"] = timed_steps(h.step("cola"), args.steps, args.warmup)
            # the median of per-step times over max(K, 50) steps after 10 warm-up
            res["cola_median"] = timed_steps_median(h.step("cola"), max(args.steps, 50), 10)
            # then K more steps with a HIP event pair around every launch (recorded on the
            # launch stream): per-kernel durations for the roofline and the table
            cola.timing_reset()
            cola.timing_enable(True)
            res["cola_events"] = timed_steps(h.step("cola_1s"), args.steps, 0)
            cola.timing_enable(False)
            kernels = kernel_table(cola)
        # the headline mode: total time of exactly K steps / K; the others: median step
        if do_m:
            res["cola_m"] = (timed_steps if not do_cola else timed_steps_median)(h.step("cola_m"), args.steps,
                                                                                 args.warmup)
        if do_dense:
            res["dense"] = (timed_steps if not (do_cola or do_m) else timed_steps_median)(h.step("dense"),
                                                                                         args.steps, args.warmup)
        if do_fused:
            res["fused"] = timed_steps_median(h.step("fused"), args.steps, args.warmup)
            res["infer"] = timed_steps_median(h.step("infer"), args.steps, args.warmup)
            if do_dense:
                res["dense_infer"] = timed_steps_median(h.step("dense_infer"), args.steps, args.warmup)

    main_mode = "cola" if do_cola else ("cola_m" if do_m else "dense")
    ms = res[main_mode]
    flops_main = flops_dense if main_mode == "dense" else flops_cola
    value = flops_main / (ms * 1e9)

    out = {
        "metric": ("CoLA layer fwd+bwd TFLOP/s (algorithmic) on a LLaMA-1B-shaped block, 7 projections"
                   if args.workload == 4 else "CoLA layer fwd+bwd TFLOP/s (algorithmic) on a " + w["name"]),
        "value": round(value, 2),
        "unit": "TFLOP/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms, 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": dtype,
        "data": "synthetic",
        "config": {"workload": w["name"], "tokens": T, "d": w["d"], "ffn": w["ffn"], "rank": r,
                   "projections": [p.name for p in projs], "act": "silu", "mode": main_mode,
                   "step": "fwd of all projections, then bwd in reverse order",
                   "streams": h.nstreams},
        "pct_of_bf16_mfma_peak": round(100.0 * value / peak, 2),
        "tokens_per_s": round(T / (ms / 1e3), 1),
        "sclk_mhz": sampler.median(),
        "power_w": sampler.power(),
    }
    if dtype == "bf16" and not args.only:
        # the box's streaming ceilings, for the HBM-bound records below
        out["hbm_ceilings"] = hbm_ceilings()
    if args.workload == 4 and main_mode == "cola":
        # the target: 60 % of the bf16 dense MFMA peak on this block; how far
        # the step is from it, as a time ratio and in ms
        target_ms = flops_cola / (0.6 * peak * 1e9)
        out["target"] = {"pct_of_peak": 60.0, "ms_per_step": round(target_ms, 4),
                         "step_over_target": round(ms / target_ms, 3), "ms_above_target": round(ms - target_ms, 4)}
    if "cola_median" in res:
        out["median_ms_per_step"] = {"steps": max(args.steps, 50), "warmup": 10,
                                     "ms": round(res["cola_median"], 4),
                                     "tflops": round(flops_cola / (res["cola_median"] * 1e9), 2)}
    if "cola_events" in res:
        out["cola_with_kernel_events"] = {"ms_per_step": round(res["cola_events"], 4),
                                          "tflops": round(flops_cola / (res["cola_events"] * 1e9), 2),
                                          "streams": 1}
    if "cola_m" in res:
        out["cola_m"] = {"ms_per_step": round(res["cola_m"], 4),
                         "tflops": round(flops_cola / (res["cola_m"] * 1e9), 2),
                         "tokens_per_s": round(T / (res["cola_m"] / 1e3), 1)}
    if "dense" in res:
        out["dense"] = {"ms_per_step": round(res["dense"], 4),
                        "tflops": round(flops_dense / (res["dense"] * 1e9), 2),
                        "tokens_per_s": round(T / (res["dense"] / 1e3), 1)}
        if "cola" in res:
            out["speedup_vs_dense"] = round(res["dense"] / res["cola"], 3)
        if "cola_m" in res:
            out["cola_m"]["speedup_vs_dense"] = round(res["dense"] / res["cola_m"], 3)
        if dtype == "bf16" and "cola" in res and not args.only:
            # the same dense step on the vendor library, as context
            vms = vendor_dense_step_ms(args.workload)
            out["dense_hipblaslt"] = {"ms_per_step": round(vms, 4),
                                      "tflops": round(flops_dense / (vms * 1e9), 2),
                                      "speedup_cola_vs_it": round(vms / res["cola"], 3),
                                      "how": "sum of per-shape medians of torch.matmul, 20 launches each"}
    if "fused" in res:
        # same algorithmic flops; q, k, v read one X and gate, up another
        out["fused_block"] = {"ms_per_step": round(res["fused"], 4),
                              "tflops": round(flops_cola / (res["fused"] * 1e9), 2),
                              "tokens_per_s": round(T / (res["fused"] / 1e3), 1),
                              "groups": ["q+k+v", "o", "gate+up", "down"]}
        if "dense" in res:
            out["fused_block"]["speedup_vs_dense"] = round(res["dense"] / res["fused"], 3)
    if "infer" in res:
        # forward only, nothing kept for a backward pass; grouped as fused_block
        out["inference"] = {"ms_per_step": round(res["infer"], 4),
                            "tflops": round(h.flops_infer / (res["infer"] * 1e9), 2),
                            "tokens_per_s": round(T / (res["infer"] / 1e3), 1)}
        if "dense_infer" in res:
            out["inference"]["dense_tokens_per_s"] = round(T / (res["dense_infer"] / 1e3), 1)
            out["inference"]["speedup_vs_dense"] = round(res["dense_infer"] / res["infer"], 3)
    if kernels:
        dom, out["roofline"] = roofline_of(kernels, peak)
        out["roofline"]["traffic"] = load_traffic(dom)
        at_clock(out["roofline"], out["sclk_mhz"])
        out["kernels"] = {k: {kk: (round(vv, 3) if isinstance(vv, float) else vv)
                              for kk, vv in v.items()} for k, v in kernels.items()}
    if not args.no_cpu_baseline and main_mode != "dense":
        out["cpu_baseline"] = cpu_baseline(projs, T, min(args.cpu_tokens, T))
        out["cpu_baseline"]["value"] = round(out["cpu_baseline"]["value"], 6)
    out["setup_s"] = round(setup_s, 1)
    del h, projs
    torch.cuda.empty_cache()
    if not args.no_block and args.only is None and args.workload != 1:
        out["block"] = block_record(args.workload, args)
    if not args.no_workloads and args.only is None:
        out["workloads"] = {str(c): workload_record(c, args) for c in (1, 2, 3, 5) if c != args.workload}
        box_relative(out["workloads"], out.get("hbm_ceilings"))
    print(json.dumps(out), flush=True)


def box_relative(records, ceilings):
    """HBM-bound dominant kernels of the workload records against what this
    box's HBM sustains for a read-only pass and for a copy (hbm_ceilings), beside
    their fraction of the nominal 8 TB/s: achieved GB/s of the algorithmic
    bytes, and of the measured traffic where the counters are stored."""
    if not ceilings:
        return
    for rec in records.values():
        rl = rec.get("roofline")
        if not rl or rl.get("bound") != "hbm":
            continue
        meas = rl.get("traffic")
        gbs = {"algorithmic": rl["achieved"]}
        if meas:
            gbs["measured_traffic"] = round(meas / (rl["avg_us"] * 1e3), 1)
        rl["vs_box"] = {k: {"gbs": v, "of_read_only": round(v / ceilings["read_gbs"], 3),
                            "of_copy": round(v / ceilings["copy_gbs"], 3)} for k, v in gbs.items()}


if __name__ == "__main__":
    main()
