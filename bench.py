#!/usr/bin/env python3
"""Benchmark of the LittleBit linear-layer forward on one MI355X.

Default workload (one "step" = one full forward of the layer through the C ABI,
both paths, all scalings): a Llama2-7B q_proj-shaped LittleBit linear,
d_in = d_out = 4096 at 0.1 bits per weight (rank r = 80 per path), T = 1
token (decode), bf16 activations, fp16 scales, signs Bernoulli(1/2), inputs
resident in HBM.  Prints ONE JSON line:
  value      tokens/s over the timed steps
  roofline   algorithmic bytes per launch / average launch duration vs 8 TB/s
  cpu_baseline  the fp64 oracle timed on this host's cores on the same inputs

--sweep FILE additionally writes one JSON line per (configuration, linear, T)
for the other benchmark configurations (Llama2-7B block at 0.1/0.55 BPW and
T in {1,16,64}; Llama2-13B prefill at T=2048; Llama2-70B 80-layer decode sweep).
"""
from __future__ import annotations

import argparse
import ctypes
import hashlib
import json
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

PEAK_HBM_GBS = 8000.0
PEAK_BF16_TFLOPS = 2500.0
PEAK_FP64_TFLOPS = 78.6


def log(*a):
    print(*a, file=sys.stderr, flush=True)


# ----------------------------------------------------------------------------
# algorithmic cost model (per call)
# ----------------------------------------------------------------------------
def alg_bytes(T, d_in, d_out, r, e_act=2, e_scale=2):
    signs = 2 * r * (d_in + d_out) / 8.0               # both paths, 1 bit per sign
    scales = 2 * e_scale * (d_in + d_out + r)           # h, g, l for both paths
    acts = T * d_in * e_act + T * d_out * e_act         # x read once, y written once
    return signs + scales + acts, signs + scales


def alg_flops(T, d_in, d_out, r):
    return 2.0 * 2 * T * r * (d_in + d_out)            # two paths, multiply-add counted as 2


# ----------------------------------------------------------------------------
# device setup
# ----------------------------------------------------------------------------
class Layer:
    """One LittleBit linear resident on the GPU, plus a pre-marshalled C-ABI call."""

    def __init__(self, li, device, kernel=0, pack_on_gpu=True):
        import torch
        import paper_2506_13771_amd as lb
        self.li = li
        self.T, self.d_in, self.d_out, self.r = li.T, li.d_in, li.d_out, li.r
        tdt = {"f32": torch.float32, "f16": torch.float16, "bf16": torch.bfloat16}

        def dev(raw, code):
            if code == "f32":
                return torch.from_numpy(np.ascontiguousarray(raw, np.float32)).to(device)
            return torch.from_numpy(np.ascontiguousarray(raw).view(np.int16)).to(device).view(tdt[code])

        self.paths = []
        for p in range(2):
            if li.U_latent is not None and pack_on_gpu:
                ub = lb.lb_pack_signs(torch.from_numpy(li.U_latent[p]).to(device), lb.LB_ROLE_U)
                vb = lb.lb_pack_signs(torch.from_numpy(li.V_latent[p]).to(device), lb.LB_ROLE_V)
            else:
                ub = torch.from_numpy(li.U_words[p]).to(device)
                vb = torch.from_numpy(li.V_words[p]).to(device)
            self.paths.append(lb.LittleBitPath(U=ub, V=vb, h=dev(li.h[p], li.scale_dtype),
                                               g=dev(li.g[p], li.scale_dtype), l=dev(li.l[p], li.scale_dtype)))
        self.x = dev(li.x, li.act_dtype)
        self.y = torch.empty((li.T, li.d_out), dtype=self.x.dtype, device=device)
        self.ws = lb.alloc_workspace(li.T, li.d_in, li.d_out, li.r, device=device)
        arr, sc = lb._paths_struct(self.paths)
        self._arr = arr
        self.lib = lb.load_library()
        self.kernel = kernel
        self.stream = torch.cuda.current_stream().cuda_stream
        self.argv = (ctypes.c_void_p(self.x.data_ptr()), lb._dtype_code(self.x), li.T, li.d_in, li.d_out, li.r,
                     arr, sc, ctypes.c_void_p(self.y.data_ptr()), ctypes.c_void_p(self.ws.data_ptr()),
                     self.ws.numel(), kernel, ctypes.c_void_p(self.stream))

    def set_stream(self, handle):
        self.argv = self.argv[:-1] + (ctypes.c_void_p(handle),)

    def weight_copies(self, n):
        """n - 1 more instances of the same layer whose packed signs and scales live in fresh
        device memory (x, y and the workspace are shared): a cold-cache rotation.  All copies
        sit in one allocation filled by one broadcast copy per tensor."""
        import copy
        import torch
        import paper_2506_13771_amd as lb
        tensors = [getattr(p, f) for p in self.paths for f in ("U", "V", "h", "g", "l")]
        sizes = [t.numel() * t.element_size() for t in tensors]
        offs = np.concatenate([[0], np.cumsum([(b + 255) // 256 * 256 for b in sizes])]).astype(int)
        big = torch.empty((n - 1, int(offs[-1])), dtype=torch.uint8, device=tensors[0].device)
        for t, o, b in zip(tensors, offs[:-1], sizes):
            big[:, o:o + b] = t.contiguous().view(torch.uint8).reshape(1, b).expand(n - 1, b)
        out = [self]
        for c in range(n - 1):
            views = [big[c, o:o + b].view(t.dtype) for t, o, b in zip(tensors, offs[:-1], sizes)]
            L = copy.copy(self)
            L.paths = [lb.LittleBitPath(*views[5 * p:5 * p + 5]) for p in range(2)]
            L._arr, _ = lb._paths_struct(L.paths)
            L.argv = self.argv[:6] + (L._arr,) + self.argv[7:]
            L._big = big
            out.append(L)
        return out

    def call(self):
        st = self.lib.lb_linear_forward_kernel(*self.argv)
        if st != 0:
            raise RuntimeError(f"lb_linear_forward failed with status {st}")

    @property
    def e_act(self):
        return 4 if self.li.act_dtype == "f32" else 2

    @property
    def e_scale(self):
        return 4 if self.li.scale_dtype == "f32" else 2


class LayerList:
    """Resident layers run by one lb_linear_forward_many call (pre-marshalled descriptors and
    one workspace with a slice per layer); times like a Layer."""

    def __init__(self, layers):
        import torch
        import paper_2506_13771_amd as lb
        self.layers = layers
        self.arr, _ = lb.make_descs([(L.x, L.paths, L.r, L.y) for L in layers])
        need = lb.lb_forward_many_workspace_bytes(self.arr, len(layers))
        self.ws = lb.lb_workspace_init(torch.empty(max(need, 256), dtype=torch.uint8, device=layers[0].x.device))
        self.lib = lb.load_library()
        self.argv = (self.arr, len(layers), ctypes.c_void_p(self.ws.data_ptr()), self.ws.numel(),
                     ctypes.c_void_p(torch.cuda.current_stream().cuda_stream))

    def set_stream(self, handle):
        self.argv = self.argv[:-1] + (ctypes.c_void_p(handle),)

    def call(self):
        st = self.lib.lb_linear_forward_many(*self.argv)
        if st != 0:
            raise RuntimeError(f"lb_linear_forward_many failed with status {st}")


class LatentCall:
    """A layer's latent-cache call, pre-marshalled: "latent" writes the cache [T, 2, r] (bf16) of
    the layer's x, "from" computes y from that cache; times like a Layer."""

    def __init__(self, layer, mode):
        import torch
        import paper_2506_13771_amd as lb
        L = layer
        self.layer, self.mode = L, mode
        self.lib = lb.load_library()
        self.cache = torch.zeros((L.T, 2, L.r), dtype=torch.bfloat16, device=L.x.device)
        stream = ctypes.c_void_p(torch.cuda.current_stream().cuda_stream)
        if mode == "latent":
            n = lb.lb_latent_workspace_bytes(L.T, L.d_in, L.r)
            self.ws = torch.empty(max(n, 256), dtype=torch.uint8, device=L.x.device)
            self.fn = self.lib.lb_linear_latent
            self.argv = (ctypes.c_void_p(L.x.data_ptr()), lb._dtype_code(L.x), L.T, L.d_in, L.r, L._arr,
                         lb._dtype_code(L.paths[0].h), ctypes.c_void_p(self.cache.data_ptr()), lb.LB_BF16,
                         ctypes.c_void_p(self.ws.data_ptr()), self.ws.numel(), stream)
        else:
            n = lb.lb_from_latent_workspace_bytes(L.T, L.r)
            self.ws = torch.empty(max(n, 256), dtype=torch.uint8, device=L.x.device)
            self.fn = self.lib.lb_linear_from_latent
            self.argv = (ctypes.c_void_p(self.cache.data_ptr()), lb.LB_BF16, L.T, L.d_out, L.r, L._arr,
                         lb._dtype_code(L.paths[0].h), ctypes.c_void_p(L.y.data_ptr()), lb._dtype_code(L.y),
                         ctypes.c_void_p(self.ws.data_ptr()), self.ws.numel(), stream)

    def set_stream(self, handle):
        self.argv = self.argv[:-1] + (ctypes.c_void_p(handle),)

    def call(self):
        st = self.fn(*self.argv)
        if st != 0:
            raise RuntimeError(f"latent-cache call ({self.mode}) failed with status {st}")


class BackwardCall:
    """A layer's backward (lb_linear_backward, dx included) for x and a random upstream gradient,
    pre-marshalled; times like a Layer."""

    def __init__(self, layer, kappa=100.0):
        import torch
        import paper_2506_13771_amd as lb
        L = layer
        self.layer = L
        self.lib = lb.load_library()
        g = torch.Generator(device=L.x.device).manual_seed(7)
        self.dy = torch.randn((L.T, L.d_out), generator=g, device=L.x.device).to(L.x.dtype)
        self.dx = torch.empty_like(L.x)
        self.train = []
        tarr = (lb.lb_path_train * 2)()
        for p in range(2):
            U_lat = torch.randn((L.d_out, L.r), generator=g, device=L.x.device) / kappa
            V_lat = torch.randn((L.d_in, L.r), generator=g, device=L.x.device) / kappa
            q = lb.LittleBitPathTrain(U_latent=U_lat, V_latent=V_lat,
                                      Ut=lb.lb_pack_signs(U_lat, lb.LB_ROLE_V), Vt=lb.lb_pack_signs(V_lat, lb.LB_ROLE_U))
            for name, shape in (("dU", (L.d_out, L.r)), ("dV", (L.d_in, L.r)), ("dh", (L.d_out,)),
                                ("dg", (L.d_in,)), ("dl", (L.r,))):
                setattr(q, name, torch.empty(shape, dtype=torch.float32, device=L.x.device))
            tarr[p] = lb.lb_path_train(*[getattr(q, f).data_ptr() for f in ("U_latent", "V_latent", "Ut", "Vt", "dU",
                                                                            "dV", "dh", "dg", "dl")])
            self.train.append(q)
        self._tarr = tarr
        n = lb.lb_backward_workspace_bytes(L.T, L.d_in, L.d_out, L.r)
        self.ws = torch.empty(max(n, 256), dtype=torch.uint8, device=L.x.device)
        self.argv = (ctypes.c_void_p(L.x.data_ptr()), ctypes.c_void_p(self.dy.data_ptr()), lb._dtype_code(L.x), L.T,
                     L.d_in, L.d_out, L.r, L._arr, lb._dtype_code(L.paths[0].h), tarr, ctypes.c_float(kappa),
                     ctypes.c_void_p(self.dx.data_ptr()), ctypes.c_void_p(self.ws.data_ptr()), self.ws.numel(),
                     ctypes.c_void_p(torch.cuda.current_stream().cuda_stream))

    def set_stream(self, handle):
        self.argv = self.argv[:-1] + (ctypes.c_void_p(handle),)

    def call(self):
        st = self.lib.lb_linear_backward(*self.argv)
        if st != 0:
            raise RuntimeError(f"lb_linear_backward failed with status {st}")


def time_calls(layers, steps, warmup, use_graph=True, per_graph=None):
    """Run every layer's forward `steps` times (after `warmup`) on the current stream, timed
    with HIP events recorded on that stream.  With use_graph the launches of `per_graph`
    steps are captured once into a HIP graph that is replayed.  Returns (ms per step, steps)."""
    import torch
    stream = torch.cuda.current_stream()
    for L in layers:
        L.set_stream(stream.cuda_stream)
    fns = [L.call for L in layers]
    for _ in range(warmup):
        for f in fns:
            f()
    torch.cuda.synchronize()
    graph = None
    reps = steps
    if use_graph:
        per_graph = per_graph or max(1, min(steps, 100))
        graph = torch.cuda.CUDAGraph()
        with torch.cuda.graph(graph):
            cap = torch.cuda.current_stream().cuda_stream
            for L in layers:
                L.set_stream(cap)
            for _ in range(per_graph):
                for f in fns:
                    f()
        for L in layers:
            L.set_stream(stream.cuda_stream)
        graph.replay()
        torch.cuda.synchronize()
        reps = max(1, steps // per_graph)
        steps = reps * per_graph
    e0 = torch.cuda.Event(enable_timing=True)
    e1 = torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    e0.record(stream)
    if graph is not None:
        for _ in range(reps):
            graph.replay()
    else:
        for _ in range(steps):
            for f in fns:
                f()
    e1.record(stream)
    torch.cuda.synchronize()
    return e0.elapsed_time(e1) / steps, steps


def cache_flush(nbytes=1 << 30):
    """Evict the caches (every L2 and the 256 MB Infinity Cache): read and write a buffer of
    `nbytes` on the current stream.  Also keeps the GPU busy while the host submits whatever
    is enqueued next, so that a timed region that starts after it has no submission gap."""
    import torch
    buf = getattr(cache_flush, "_buf", None)
    if buf is None or buf.numel() != nbytes // 4:
        buf = torch.empty(nbytes // 4, dtype=torch.float32, device="cuda")
        buf.zero_()
        cache_flush._buf = buf
    buf.add_(1.0)


def time_rotation(copies, steps, warmup):
    """Cold-cache timing: `steps` calls on distinct weight buffers of one layer (the
    `copies`, together larger than twice the Infinity Cache), captured into one HIP graph.
    The timed calls start at copy len(copies) // 2 and cycle; the untimed warm-up calls use
    copies 0, 1, ...; before the timed replay the caches are flushed (cache_flush), so no
    timed call finds its weights in a cache.  Returns (ms per call, calls timed, distinct
    copies the timed calls touched)."""
    import torch
    n = len(copies)
    c0 = n // 2
    order = [copies[(c0 + i) % n] for i in range(steps)]
    stream = torch.cuda.current_stream()
    for L in copies:
        L.set_stream(stream.cuda_stream)
    for i in range(warmup):
        copies[i % max(1, c0)].call()
    torch.cuda.synchronize()
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph):
        cap = torch.cuda.current_stream().cuda_stream
        for L in order:
            L.set_stream(cap)
        for L in order:
            L.call()
    for L in copies:
        L.set_stream(stream.cuda_stream)
    graph.replay()  # untimed: first replay (graph upload)
    torch.cuda.synchronize()
    e0 = torch.cuda.Event(enable_timing=True)
    e1 = torch.cuda.Event(enable_timing=True)
    cache_flush()
    e0.record(stream)
    graph.replay()
    e1.record(stream)
    torch.cuda.synchronize()
    return e0.elapsed_time(e1) / steps, steps, len({id(L) for L in order})


def source_digest(files):
    h = hashlib.sha256()
    for f in files:
        with open(os.path.join(ROOT, f), "rb") as fh:
            h.update(fh.read())
    return h.hexdigest()[:16]


DECODE_SOURCES = ["paper_2506_13771_amd/csrc/decode.hip", "paper_2506_13771_amd/csrc/lb_internal.h",
                  "paper_2506_13771_amd/csrc/device_common.h"]


def copy_probe(mib):
    """A plain device-to-device copy of `mib` MiB, five times: the reference kernel whose
    FETCH_SIZE / WRITE_SIZE counters calibrate those of the decode kernel."""
    import torch
    n = int(mib) << 20
    src = torch.ones(n, dtype=torch.uint8, device="cuda")
    dst = torch.empty_like(src)
    torch.cuda.synchronize()
    for _ in range(5):
        dst.copy_(src)
    torch.cuda.synchronize()
    log(f"copy probe: 5 copies of {n} bytes")


def _pmc_rows(path, counter):
    import csv
    rows = []
    with open(path, newline="") as fh:
        for row in csv.DictReader(fh):
            if row.get("Counter_Name") == counter:
                rows.append((row.get("Kernel_Name", ""), float(row["Counter_Value"])))
    return rows


def ingest_pmc(fetch_csv, write_csv, copy_mib, workload_key, commands):
    """Per-launch HBM bytes of the decode kernel from two rocprofv3 --pmc runs (FETCH_SIZE,
    then WRITE_SIZE, KiB per dispatch), each scaled by what the same counter reads for the
    plain copy of copy_mib MiB made by --copy-probe in the same run.  Writes
    profiles/traffic.json."""
    n = float(int(copy_mib) << 20)
    out = {}
    for name, path in (("fetch", fetch_csv), ("write", write_csv)):
        counter = "FETCH_SIZE" if name == "fetch" else "WRITE_SIZE"
        rows = _pmc_rows(path, counter)
        dec = [v for k, v in rows if "decode_kernel" in k]
        # the probe's five copies are the five largest copy-kernel dispatches of the run
        cop = sorted((v for k, v in rows if "copyBuffer" in k), reverse=True)[:5]
        if not dec or not cop:
            raise SystemExit(f"{path}: no {counter} rows for the decode kernel or the copy probe")
        dec_kib = float(np.mean(dec))
        cop_kib = float(np.median(cop))
        factor = n / (cop_kib * 1024.0)
        out[name] = {"dispatches": len(dec), "kib_per_dispatch": dec_kib, "kib_min": float(np.min(dec)),
                     "kib_max": float(np.max(dec)), "copy_kib_per_dispatch": cop_kib, "copy_bytes": n,
                     "factor": factor, "bytes_per_launch": dec_kib * 1024.0 * factor}
    path = os.path.join(ROOT, "profiles", "traffic.json")
    d = json.load(open(path)) if os.path.exists(path) else {}
    d[workload_key] = {"bytes_per_launch": out["fetch"]["bytes_per_launch"] + out["write"]["bytes_per_launch"],
                       "fetch": out["fetch"], "write": out["write"], "sources": DECODE_SOURCES,
                       "source_digest": source_digest(DECODE_SOURCES), "commands": commands}
    with open(path, "w") as fh:
        json.dump(d, fh, indent=1)
        fh.write("\n")
    print(json.dumps(d[workload_key], indent=1))


LIST_SOURCES = ["paper_2506_13771_amd/csrc/stream.hip", "paper_2506_13771_amd/csrc/stream_mma.hip",
                "paper_2506_13771_amd/csrc/stream_plan.h", "paper_2506_13771_amd/csrc/lut_common.h",
                "paper_2506_13771_amd/csrc/device_common.h", "paper_2506_13771_amd/csrc/lb_internal.h"]


def sweep70b_alg_bytes(T):
    """Algorithmic bytes of one 70B list sweep at T tokens (bf16 x, fp16 scales)."""
    from paper_2506_13771_amd import synth
    return sum(alg_bytes(T, d_in, d_out, RANKS_70B[(d_in, d_out)])[0] for _ in range(80)
               for (_, d_in, d_out) in synth.LLAMA2_70B)


def ingest_pmc_list(fetch_csv, write_csv, copy_mib, T, commands):
    """HBM bytes of one lb_list_forward call of the 70B sweep at T tokens from two rocprofv3 --pmc
    runs (FETCH_SIZE, then WRITE_SIZE) of `bench.py --sweep70b-tokens T --copy-probe MIB`: the list
    kernels' counters summed per call (one stage-2 launch per call), scaled by the copy probe's
    factor; beside the algorithmic bytes.  Writes profiles/traffic.json key list_llama2_70b_T<T>."""
    n = float(int(copy_mib) << 20)
    out = {"per_kernel": {}}
    for name, path in (("fetch", fetch_csv), ("write", write_csv)):
        counter = "FETCH_SIZE" if name == "fetch" else "WRITE_SIZE"
        rows = _pmc_rows(path, counter)
        lst = [(k, v) for k, v in rows if "stream_" in k or "sm_" in k]
        calls = sum(1 for k, _ in lst if "stream_s2_kernel" in k or "sm_s2_kernel" in k)
        cop = sorted((v for k, v in rows if "copyBuffer" in k), reverse=True)[:5]
        if not lst or not calls or not cop:
            raise SystemExit(f"{path}: no {counter} rows for the list kernels or the copy probe")
        factor = n / (float(np.median(cop)) * 1024.0)
        per_call = sum(v for _, v in lst) * 1024.0 * factor / calls
        for k, v in lst:
            short = k.replace("void lb::(anonymous namespace)::", "").replace("lb::(anonymous namespace)::", "")
            short = short.split("(")[0]
            d = out["per_kernel"].setdefault(short, {})
            d[name + "_bytes_per_call"] = d.get(name + "_bytes_per_call", 0.0) + v * 1024.0 * factor / calls
        out[name] = {"calls": calls, "factor": factor, "bytes_per_call": per_call}
    alg = sweep70b_alg_bytes(T)
    total = out["fetch"]["bytes_per_call"] + out["write"]["bytes_per_call"]
    path = os.path.join(ROOT, "profiles", "traffic.json")
    d = json.load(open(path)) if os.path.exists(path) else {}
    d[f"list_llama2_70b_T{T}"] = {"bytes_per_call": total, "alg_bytes_per_call": alg, "ratio": total / alg,
                                   "fetch": out["fetch"], "write": out["write"], "per_kernel": out["per_kernel"],
                                   "sources": LIST_SOURCES, "source_digest": source_digest(LIST_SOURCES),
                                   "commands": commands}
    with open(path, "w") as fh:
        json.dump(d, fh, indent=1)
        fh.write("\n")
    print(json.dumps(d[f"list_llama2_70b_T{T}"], indent=1))


def summarize_pmc(paths, name_filter):
    """Per-kernel means of every counter in rocprofv3 --pmc counter_collection.csv files (kernels
    whose name contains name_filter), one line per kernel."""
    import csv
    import collections
    vals = collections.defaultdict(lambda: collections.defaultdict(list))
    for path in paths:
        with open(path, newline="") as fh:
            for row in csv.DictReader(fh):
                k = row.get("Kernel_Name", "")
                if name_filter in k:
                    vals[k][row["Counter_Name"]].append(float(row["Counter_Value"]))
    for k, cs in sorted(vals.items()):
        short = k.replace("void lb::(anonymous namespace)::", "").replace("lb::(anonymous namespace)::", "")
        short = short.split("(")[0]
        n = max(len(v) for v in cs.values())
        print(f"{short} dispatches={n} " + " ".join(f"{c}={np.mean(v):.4g}" for c, v in sorted(cs.items())))


def measured_traffic(workload_key):
    """HBM bytes per launch from committed rocprofv3 counter runs, or None if the kernel
    source changed since they were taken."""
    path = os.path.join(ROOT, "profiles", "traffic.json")
    if not os.path.exists(path):
        return None
    try:
        d = json.load(open(path))
    except Exception:
        return None
    ent = d.get(workload_key)
    if not ent or ent.get("source_digest") != source_digest(ent.get("sources", DECODE_SOURCES)):
        return None
    return ent.get("bytes_per_launch")


# ----------------------------------------------------------------------------
# CPU baseline: the oracle as it stands, on this host
# ----------------------------------------------------------------------------
def cpu_model() -> str:
    try:
        with open("/proc/cpuinfo") as fh:
            for line in fh:
                if line.startswith("model name"):
                    return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return "unknown"


def host_threads() -> int:
    """Threads for the all-core oracle: the cores this process may run on, capped by
    OMP_NUM_THREADS when that is set."""
    n = len(os.sched_getaffinity(0))
    env = os.environ.get("OMP_NUM_THREADS", "")
    if env.isdigit() and int(env) > 0:
        n = min(n, int(env))
    return max(1, n)


def cpu_baseline(li, seconds):
    """The fp64 oracle O1 (as it stands) on this host, on the headline layer and inputs:
    single-threaded, and the same loops on every available core (OpenMP over (path, token,
    latent) and (token, row)).  Each variant runs for about `seconds`."""
    import oracle as O
    Us, Vs = [], []
    for p in range(2):
        ub, _ = O.pack(li.U_latent[p].astype(np.float64), O.ROLE_U)
        vb, _ = O.pack(li.V_latent[p].astype(np.float64), O.ROLE_V)
        Us.append(O.unpack(ub, li.d_out, li.r, O.ROLE_U))
        Vs.append(O.unpack(vb, li.d_in, li.r, O.ROLE_V))
    x = O.to_f64(li.x, li.act_dtype)
    h = [O.to_f64(a, li.scale_dtype) for a in li.h]
    g = [O.to_f64(a, li.scale_dtype) for a in li.g]
    l = [O.to_f64(a, li.scale_dtype) for a in li.l]
    nthr = host_threads()

    def timed(fn):
        fn()
        n = 0
        t0 = time.perf_counter()
        while True:
            fn()
            n += 1
            el = time.perf_counter() - t0
            if el >= seconds:
                return n, el

    n1, el1 = timed(lambda: O.forward_factored(x, Us, Vs, h, g, l))
    nm, elm = timed(lambda: O.forward_factored_par(x, Us, Vs, h, g, l, nthr))
    y1 = O.forward_factored(x, Us, Vs, h, g, l)
    ym = O.forward_factored_par(x, Us, Vs, h, g, l, nthr)
    return {"value": nm * li.T / elm, "unit": "tokens/s", "cores": nthr, "kind": "oracle",
            "cpu_model": cpu_model(), "omp_threads": nthr,
            "single_thread_value": n1 * li.T / el1,
            "identical_results": bool(np.array_equal(y1, ym)),
            "sample": f"full fp64 oracle forwards of the headline layer and inputs ({li.d_in}x{li.d_out}, "
                      f"r={li.r}, T={li.T}): {nm} on {nthr} threads in {elm:.1f} s (value), "
                      f"{n1} on one thread in {el1:.1f} s (single_thread_value)"}


# ----------------------------------------------------------------------------
# sweep of the other configurations (diagnostic lines written to a file)
# ----------------------------------------------------------------------------
def run_sweep(path, steps, warmup, only=("7b", "13b", "kv", "train", "70b", "svid")):
    import torch
    from paper_2506_13771_amd import synth
    out = open(path, "w")

    def emit(rec):
        out.write(json.dumps(rec) + "\n")
        out.flush()
        log(json.dumps(rec))

    ranks_7b = {0.1: {4096: 80, 11008: 128}, 0.55: {4096: 544, 11008: 800}}
    for bpw in ((0.1, 0.55) if "7b" in only else ()):
        for T in (1, 16, 64):
            for idx, (name, d_in, d_out) in enumerate(synth.LLAMA2_7B):
                r = ranks_7b[bpw][max(d_in, d_out)]
                L = Layer(synth.make_linear(d_in, d_out, r, T, cfg=2, linear=idx), "cuda")
                ms, n = time_calls([L], steps, warmup)
                b, bw = alg_bytes(T, d_in, d_out, r)
                emit({"config": "llama2-7b-block", "linear": name, "bpw": bpw, "T": T, "d_in": d_in,
                      "d_out": d_out, "r": r, "us_per_call": ms * 1e3, "tokens_per_s": T / (ms * 1e-3),
                      "alg_bytes": b, "GBps": b / (ms * 1e-3) / 1e9, "hbm_frac": b / (ms * 1e-3) / 1e9 / PEAK_HBM_GBS,
                      "weights_GBps": bw / (ms * 1e-3) / 1e9,
                      "mfma_frac": alg_flops(T, d_in, d_out, r) / (ms * 1e-3) / 1e12 / PEAK_BF16_TFLOPS})
                del L
    ranks_13b = {(5120, 5120): 96, (5120, 13824): 160, (13824, 5120): 160}
    for idx, (name, d_in, d_out) in enumerate(synth.LLAMA2_13B if "13b" in only else ()):
        r = ranks_13b[(d_in, d_out)]
        T = 2048
        L = Layer(synth.make_linear(d_in, d_out, r, T, cfg=3, linear=idx), "cuda")
        ms, n = time_calls([L], max(10, steps // 20), max(3, warmup // 20))
        b, bw = alg_bytes(T, d_in, d_out, r)
        f = alg_flops(T, d_in, d_out, r)
        emit({"config": "llama2-13b-prefill", "linear": name, "bpw": 0.1, "T": T, "d_in": d_in, "d_out": d_out,
              "r": r, "us_per_call": ms * 1e3, "tokens_per_s": T / (ms * 1e-3), "alg_bytes": b,
              "GBps": b / (ms * 1e-3) / 1e9, "hbm_frac": b / (ms * 1e-3) / 1e9 / PEAK_HBM_GBS,
              "mfma_tflops": f / (ms * 1e-3) / 1e12, "mfma_frac": f / (ms * 1e-3) / 1e12 / PEAK_BF16_TFLOPS})
        del L
    # latent K/V cache on the Llama2-7B k_proj shape: the cache write (x -> bf16 latents of both
    # paths) and the output from the cache, beside the forward of the same tokens
    for bpw, r in ((0.1, 80), (0.55, 544)) if "kv" in only else ():
        for T in (1, 64, 2048):
            d_in = d_out = 4096
            L = Layer(synth.make_linear(d_in, d_out, r, T, cfg=5, linear=1), "cuda")
            n_st, n_wu = (steps, warmup) if T < 2048 else (max(10, steps // 20), max(3, warmup // 20))
            ms_f, _ = time_calls([L], n_st, n_wu)
            lat, frm = LatentCall(L, "latent"), LatentCall(L, "from")
            ms_l, _ = time_calls([lat], n_st, n_wu)
            ms_u, _ = time_calls([frm], n_st, n_wu)
            e = L.e_act
            b_l = 2 * r * d_in / 8.0 + 2 * (d_in + r) * L.e_scale + T * d_in * e + 2 * T * r * 2
            b_u = 2 * r * d_out / 8.0 + 2 * d_out * L.e_scale + 2 * T * r * 2 + T * d_out * e
            emit({"config": "llama2-7b-kv-cache", "linear": "k_proj", "bpw": bpw, "T": T, "d_in": d_in,
                  "d_out": d_out, "r": r, "cache_values_per_token": 2 * r, "cache_reduction": d_out / (2 * r),
                  "us_latent": ms_l * 1e3, "us_from_latent": ms_u * 1e3, "us_forward": ms_f * 1e3,
                  "latent_GBps": b_l / (ms_l * 1e-3) / 1e9, "from_latent_GBps": b_u / (ms_u * 1e-3) / 1e9,
                  "latent_tflops": 4 * T * d_in * r / (ms_l * 1e-3) / 1e12,
                  "from_latent_tflops": 4 * T * r * d_out / (ms_u * 1e-3) / 1e12})
            del L, lat, frm
    # training step of one layer (QAT backward with SmoothSign) on the Llama2-7B block shapes at
    # 0.1 BPW, 2048 tokens (the paper's training sequence length), beside the forward
    for idx, (name, d_in, d_out) in enumerate(synth.LLAMA2_7B if "train" in only else ()):
        if name not in ("q", "gate", "down"):
            continue
        r = ranks_7b[0.1][max(d_in, d_out)]
        T = 2048
        L = Layer(synth.make_linear(d_in, d_out, r, T, cfg=6, linear=idx), "cuda")
        n_st, n_wu = max(10, steps // 20), max(3, warmup // 20)
        ms_f, _ = time_calls([L], n_st, n_wu)
        B = BackwardCall(L)
        ms_b, _ = time_calls([B], n_st, n_wu)
        fl = 2.0 * 2 * T * r * (2 * d_out + 3 * d_in)
        emit({"config": "llama2-7b-train-step", "linear": name, "bpw": 0.1, "T": T, "d_in": d_in, "d_out": d_out,
              "r": r, "us_backward": ms_b * 1e3, "us_forward": ms_f * 1e3, "backward_flops": fl,
              "backward_tflops": fl / (ms_b * 1e-3) / 1e12,
              "backward_mfma_frac": fl / (ms_b * 1e-3) / 1e12 / PEAK_BF16_TFLOPS})
        del L, B
    if "svid" in only:
        for rec in run_svid(((4096, 4096), (11008, 4096), (4096, 11008)))["per_shape"]:
            emit({"config": "llama2-7b-dual-svid", **rec})
    # 70B sweep: 80 layers x 7 linears resident, back-to-back on one stream
    ranks_70b = {(8192, 8192): 176, (8192, 1024): 16, (8192, 28672): 288, (28672, 8192): 288}
    for T in ((1, 8, 64) if "70b" in only else ()):
        layers = []
        tot_b = 0.0
        tot_w = 0.0
        for layer in range(80):
            for idx, (name, d_in, d_out) in enumerate(synth.LLAMA2_70B):
                r = ranks_70b[(d_in, d_out)]
                li = synth.make_linear(d_in, d_out, r, T, cfg=4, linear=layer * 7 + idx, direct_words=True)
                layers.append(Layer(li, "cuda", pack_on_gpu=False))
                b, bw = alg_bytes(T, d_in, d_out, r)
                tot_b += b
                tot_w += bw
        # one lb_linear_forward_many call for the whole sweep (list launches of up to 16
        # look-up-table decode linears where T <= 2), and one call per linear beside it
        ms, n = time_calls([LayerList(layers)], max(3, steps // 100), 2, use_graph=True, per_graph=1)
        ms1, _ = time_calls(layers, max(3, steps // 100), 2, use_graph=True, per_graph=1)
        emit({"config": "llama2-70b-sweep", "T": T, "linears": len(layers), "launch": "lb_linear_forward_many",
              "ms_per_sweep": ms, "tokens_per_s": T / (ms * 1e-3), "alg_bytes": tot_b, "weights_bytes": tot_w,
              "GBps": tot_b / (ms * 1e-3) / 1e9, "hbm_frac": tot_b / (ms * 1e-3) / 1e9 / PEAK_HBM_GBS,
              "us_per_linear": ms * 1e3 / len(layers), "ms_per_sweep_single_calls": ms1,
              "us_per_linear_single_calls": ms1 * 1e3 / len(layers)})
        del layers
        torch.cuda.empty_cache()
    out.close()


class ListCall:
    """One lb_linear_forward_many call over pre-marshalled descriptors, timed like a Layer."""

    def __init__(self, descs, n, device="cuda"):
        import torch
        import paper_2506_13771_amd as lb
        self.arr, self.n = descs, n
        need = lb.lb_forward_many_workspace_bytes(descs, n)
        self.ws = lb.lb_workspace_init(torch.empty(max(need, 256), dtype=torch.uint8, device=device))
        self.lib = lb.load_library()
        self.argv = (self.arr, n, ctypes.c_void_p(self.ws.data_ptr()), self.ws.numel(),
                     ctypes.c_void_p(torch.cuda.current_stream().cuda_stream))

    def set_stream(self, handle):
        self.argv = self.argv[:-1] + (ctypes.c_void_p(handle),)

    def call(self):
        st = self.lib.lb_linear_forward_many(*self.argv)
        if st != 0:
            raise RuntimeError(f"lb_linear_forward_many failed with status {st}")


class ResidentLinears:
    """Linears resident on the GPU (packed signs, fp16 scales) with bf16 inputs of up to
    t_max tokens each; desc(T) gives lb_linear_desc entries over the first T tokens."""

    def __init__(self, shapes, t_max, cfg, direct_words, device="cuda"):
        import torch
        import paper_2506_13771_amd as lb
        from paper_2506_13771_amd import synth
        self.shapes = shapes
        self.items = []
        self.alg = {}
        for idx, (name, d_in, d_out, r) in enumerate(shapes):
            li = synth.make_linear(d_in, d_out, r, t_max, cfg=cfg, linear=idx, direct_words=direct_words)
            L = Layer(li, device, pack_on_gpu=not direct_words)
            del L.ws
            self.items.append(L)
        self.lb = lb

    def descs(self, T):
        arr, ys = self.lb.make_descs([(L.x[:T], L.paths, L.r, L.y[:T]) for L in self.items])
        return arr

    def bytes_and_flops(self, T):
        b = w = f = 0.0
        for L in self.items:
            bb, ww = alg_bytes(T, L.d_in, L.d_out, L.r, L.e_act, L.e_scale)
            b += bb
            w += ww
            f += alg_flops(T, L.d_in, L.d_out, L.r)
        return b, w, f


class StreamListCall:
    """The streaming list forward (lb_list_init once, then lb_list_forward: three launches for the
    whole list) over pre-marshalled descriptors, timed like a Layer."""

    def __init__(self, descs, n, device="cuda"):
        import torch
        import paper_2506_13771_amd as lb
        self.arr, self.n = descs, n
        self.lib = lb.load_library()
        need = lb.lb_list_workspace_bytes(descs, n)
        if need == 0:
            raise RuntimeError("list out of the streaming forward's scope")
        self.ws = torch.empty(need, dtype=torch.uint8, device=device)
        st = self.lib.lb_list_init(descs, n, ctypes.c_void_p(self.ws.data_ptr()), need,
                                   ctypes.c_void_p(torch.cuda.current_stream().cuda_stream))
        if st != 0:
            raise RuntimeError(f"lb_list_init failed with status {st}")
        self.argv = (self.arr, n, ctypes.c_void_p(self.ws.data_ptr()), need,
                     ctypes.c_void_p(torch.cuda.current_stream().cuda_stream))

    def set_stream(self, handle):
        self.argv = self.argv[:-1] + (ctypes.c_void_p(handle),)

    def call(self):
        st = self.lib.lb_list_forward(*self.argv)
        if st != 0:
            raise RuntimeError(f"lb_list_forward failed with status {st}")


def list_timing(res, T, steps, warmup):
    """ms per list call over every linear of `res` at T tokens, graph-replayed, with the derived
    rates: the streaming list forward (lb_list_forward: look-up-table kernels for T <= 2,
    matrix-core kernels up to 64 tokens) where the list is in its scope, else
    lb_linear_forward_many; at T = 1 lb_linear_forward_many is timed beside it."""
    import torch
    import paper_2506_13771_amd as lb
    n = len(res.items)
    descs = res.descs(T)
    extra = {}
    if lb.lb_list_workspace_bytes(descs, n) > 0:
        call = StreamListCall(descs, n)
        api = "lb_list_forward"
        if T == 1:
            many = ListCall(descs, n)
            ms_many, _ = time_calls([many], steps, warmup, use_graph=True, per_graph=1)
            extra["ms_per_call_forward_many"] = ms_many
            del many
    else:
        call = ListCall(descs, n)
        api = "lb_linear_forward_many"
    ms, k = time_calls([call], steps, warmup, use_graph=True, per_graph=1)
    b, w, f = res.bytes_and_flops(T)
    t_att = max(b / (PEAK_HBM_GBS * 1e9), f / (PEAK_BF16_TFLOPS * 1e12))
    del call
    torch.cuda.synchronize()
    return {"T": T, "api": api, "ms_per_call": ms, "calls_timed": k, "us_per_linear": ms * 1e3 / n, **extra,
            "tokens_per_s": T / (ms * 1e-3), "alg_bytes": b, "weights_bytes": w,
            "GBps": b / (ms * 1e-3) / 1e9, "hbm_frac": b / (ms * 1e-3) / 1e9 / PEAK_HBM_GBS,
            "weights_GBps": w / (ms * 1e-3) / 1e9, "alg_flops": f,
            "attainable_us": t_att * 1e6, "attainable_frac": t_att / (ms * 1e-3)}


RANKS_70B = {(8192, 8192): 176, (8192, 1024): 16, (8192, 28672): 288, (28672, 8192): 288}
RANKS_7B = {0.1: {4096: 80, 11008: 128}, 0.55: {4096: 544, 11008: 800}}


def run_sweep70b(ts, steps, warmup):
    """The Llama2-70B-shaped decode sweep: 80 layers x 7 linears at 0.1 BPW resident in HBM
    (about 0.81 GB of packed signs and scales, more than three times the Infinity Cache, so
    every call streams its weights from HBM), all 560 linears in one list call, T tokens per
    linear."""
    import torch
    from paper_2506_13771_amd import synth
    t0 = time.perf_counter()
    shapes = [(f"L{layer}.{name}", d_in, d_out, RANKS_70B[(d_in, d_out)])
              for layer in range(80) for (name, d_in, d_out) in synth.LLAMA2_70B]
    res = ResidentLinears(shapes, max(ts), cfg=4, direct_words=True)
    setup_s = time.perf_counter() - t0
    out = {"workload": "Llama2-70B shapes, 80 layers x (q,k,v,o,gate,up,down) at 0.1 BPW, bf16 x, fp16 scales, "
                       "one lb_list_forward call per sweep (look-up-table kernels for T <= 2, matrix-core "
                       "kernels for larger T)",
           "linears": len(shapes), "weights_bytes": res.bytes_and_flops(1)[1], "setup_s": setup_s, "per_T": []}
    for T in ts:
        rec = list_timing(res, T, steps, warmup)
        out["per_T"].append(rec)
        log(f"sweep70b T={T}: {rec['ms_per_call']:.3f} ms, {rec['GBps']:.0f} GB/s ({100 * rec['hbm_frac']:.1f}% of HBM peak)")
    del res
    torch.cuda.empty_cache()
    return out


def svid_gemm_flops(m, n, r, b, iters):
    """Flops of the fp64 matrix-core products of one lb_dual_svid call (both paths): per path the
    2 iters + 2 multiplications by W or W^T, the Gram matrices and basis changes of 2 iters + 1
    orthonormalisations, the Rayleigh-Ritz products, the rank-1 Gram matrices; W_res once."""
    mul = (2 * iters + 2) * 2.0 * m * n * b
    orth = iters * (4.0 * m * b * b + 4.0 * n * b * b) + 4.0 * m * b * b
    rr = 2.0 * n * b * b + 2.0 * m * b * r + 2.0 * n * b * r
    rank1 = 2.0 * (m + n) * r * r + 2.0 * (m + n) * r
    return 2 * (mul + orth + rr + rank1) + 2.0 * m * n * r


def run_svid(shapes=((4096, 4096), ), reps=3):
    """Dual-SVID conversion (lb_dual_svid) of dense Llama2-7B-shaped weights at 0.1 BPW: ms per
    conversion (both paths, default block and rounds) and the rate of its fp64 matrix-core
    products against the fp64 peak (78.6 TFLOP/s)."""
    import torch
    import paper_2506_13771_amd as lb
    from paper_2506_13771_amd import synth
    out = {"workload": "Dual-SVID of a dense weight (synthetic: rank-2r part with linearly falling scales plus "
                       "N(0, 0.05^2) noise), both paths, default block and rounds", "per_shape": []}
    for d_out, d_in in shapes:
        r = lb.lb_rank_for_bpw(d_in, d_out, 0.1)
        over, iters = lb.svid_defaults(r, d_out, d_in)
        W = torch.from_numpy(synth.dense_weight(d_out, d_in, 2 * r, 0.05, cfg=73)).cuda()
        ws = torch.empty(lb.lb_dual_svid_workspace_bytes(d_out, d_in, r, over), dtype=torch.uint8, device="cuda")
        lb.lb_dual_svid(W, r, workspace=ws)
        torch.cuda.synchronize()
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record()
        for _ in range(reps):
            lb.lb_dual_svid(W, r, workspace=ws)
        e1.record()
        torch.cuda.synchronize()
        ms = e0.elapsed_time(e1) / reps
        b = min(r + over, d_out, d_in)
        f = svid_gemm_flops(d_out, d_in, r, b, iters)
        out["per_shape"].append({"d_out": d_out, "d_in": d_in, "r": r, "block": b, "iters": iters,
                                 "ms_per_conversion": ms, "gemm_flops": f, "gemm_tflops": f / (ms * 1e-3) / 1e12,
                                 "fp64_peak_frac": f / (ms * 1e-3) / 1e12 / PEAK_FP64_TFLOPS})
        log(f"svid {d_out}x{d_in} r={r}: {ms:.1f} ms per conversion")
        del W, ws
    torch.cuda.empty_cache()
    return out


def run_block7b(ts, steps, warmup, bpw=0.1):
    """The 7 linears of one Llama2-7B block (q,k,v,o 4096x4096; gate, up 4096->11008; down
    11008->4096) in one lb_linear_forward_many call (weights warm: one block is about 2 MB)."""
    import torch
    from paper_2506_13771_amd import synth
    shapes = [(name, d_in, d_out, RANKS_7B[bpw][max(d_in, d_out)]) for (name, d_in, d_out) in synth.LLAMA2_7B]
    res = ResidentLinears(shapes, max(ts), cfg=2, direct_words=False)
    out = {"workload": f"Llama2-7B block, 7 linears at {bpw} BPW, bf16 x, fp16 scales, one lb_list_forward "
                       "call (look-up-table kernels for T <= 2, matrix-core kernels for larger T; weights warm in "
                       "the caches)",
           "bpw": bpw, "per_T": []}
    for T in ts:
        rec = list_timing(res, T, max(steps, 50), max(warmup, 10))
        out["per_T"].append(rec)
        log(f"block7b T={T}: {rec['us_per_linear']:.2f} us per linear")
    del res
    torch.cuda.empty_cache()
    return out


# The paper's kernel-level latencies of one linear at batch 1 (Appendix "Inference Efficiency
# Analysis", Table tab:latency_appendix_full): NVIDIA A100, FP16 inputs and FP16 accumulation,
# cuBLAS FP16 torch.matmul as the baseline.  Context only: other hardware, other precision.
PAPER_CONTEXT = {
    "source": "Appendix Inference Efficiency Analysis, Table tab:latency_appendix_full",
    "hardware": "NVIDIA A100, FP16 activations and accumulation, batch size 1",
    "rows": [
        {"shape": "Llama2-7B MLP-like, out 4096 x in 11008", "bpw": 0.1, "littlebit_ms": 0.0190, "fp16_ms": 0.0620,
         "speedup_vs_fp16": 3.26},
        {"shape": "Llama2-70B ATTN-like, 8192 x 8192", "bpw": 0.1, "littlebit_ms": 0.0207, "fp16_ms": 0.0896,
         "speedup_vs_fp16": 4.33},
        {"shape": "Llama2-70B MLP-like, out 8192 x in 28672", "bpw": 0.1, "littlebit_ms": 0.0249, "fp16_ms": 0.2882,
         "speedup_vs_fp16": 11.57},
    ],
    "note": "no row has the 4096x4096 headline shape; the closest is the 7B MLP-like row",
}


def main():
    ap = argparse.ArgumentParser(description=__doc__, formatter_class=argparse.RawDescriptionHelpFormatter)
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=5000)
    ap.add_argument("--warmup", type=int, default=500)
    ap.add_argument("--launch", choices=["graph", "stream"], default="graph")
    ap.add_argument("--cpu-seconds", type=float, default=8.0)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-sweep70b", action="store_true", help="skip the 70B 560-linear list sweep")
    ap.add_argument("--sweep70b-tokens", default="1,8,64", help="token counts of the 70B list sweep")
    ap.add_argument("--no-block7b", action="store_true", help="skip the 7B block list timing")
    ap.add_argument("--no-svid", action="store_true", help="skip the Dual-SVID conversion timing")
    ap.add_argument("--sweep", default=None, help="write per-configuration JSON lines to this file")
    ap.add_argument("--sweep-only", default="7b,13b,kv,train,70b,svid",
                    help="comma list of the sweep's parts to run (7b block, 13b prefill, 7b latent K/V cache, "
                         "7b training-step backward, 70b decode sweep, 7b Dual-SVID conversions)")
    ap.add_argument("--no-warm", action="store_true",
                    help="skip the warm-cache measurements (counter runs: every decode dispatch is then a "
                         "cold-rotation one)")
    ap.add_argument("--copy-probe", type=int, default=0, metavar="MIB",
                    help="after the run, copy MIB MiB device-to-device five times (counter calibration)")
    ap.add_argument("--ingest-pmc", nargs=2, metavar=("FETCH_CSV", "WRITE_CSV"), default=None,
                    help="no GPU: turn two rocprofv3 --pmc counter_collection.csv files (FETCH_SIZE, "
                         "WRITE_SIZE) of runs with --copy-probe into profiles/traffic.json")
    ap.add_argument("--ingest-pmc-list", nargs=3, metavar=("FETCH_CSV", "WRITE_CSV", "T"), default=None,
                    help="no GPU: the same for the list kernels of a --sweep70b-tokens T run")
    ap.add_argument("--summarize-pmc", nargs="+", metavar="CSV", default=None,
                    help="no GPU: per-kernel means of the counters in rocprofv3 --pmc CSV files")
    ap.add_argument("--pmc-kernel", default="", help="with --summarize-pmc: kernel name filter")
    ap.add_argument("--pmc-command", action="append", default=[],
                    help="with --ingest-pmc: the command lines that produced the files (recorded)")
    args = ap.parse_args()

    if args.ingest_pmc:
        ingest_pmc(args.ingest_pmc[0], args.ingest_pmc[1], args.copy_probe or 64,
                   "decode_q_proj_4096_r80_T1", args.pmc_command)
        return
    if args.ingest_pmc_list:
        ingest_pmc_list(args.ingest_pmc_list[0], args.ingest_pmc_list[1], args.copy_probe or 64,
                        int(args.ingest_pmc_list[2]), args.pmc_command)
        return
    if args.summarize_pmc:
        summarize_pmc(args.summarize_pmc, args.pmc_kernel)
        return

    world = int(os.environ.get("WORLD_SIZE", "1"))
    if args.gpus != 1 or world != 1:
        print(json.dumps({"error": "this benchmark runs on exactly one GPU: the LittleBit linear forward is "
                                   "measured on one MI355X (multi-GPU sharding is a design note, not a run)",
                          "n_gpus": args.gpus}))
        sys.exit(2)

    import torch
    import paper_2506_13771_amd as lb
    from paper_2506_13771_amd import synth
    lb.load_library()
    assert torch.cuda.is_available(), "bench.py needs a GPU"
    torch.cuda.set_device(0)

    d_in, d_out, r, T = 4096, 4096, 80, 1
    assert lb.lb_rank_for_bpw(d_in, d_out, 0.1, 16) == r
    li = synth.make_linear(d_in, d_out, r, T, act_dtype="bf16", scale_dtype="f16", cfg=1, linear=0)
    L = Layer(li, "cuda")
    b, bw = alg_bytes(T, d_in, d_out, r, L.e_act, L.e_scale)
    # headline: weights cold in HBM -- the calls rotate over copies of the layer's packed signs
    # and scales that together exceed twice the 256 MB Infinity Cache (and every L2)
    ncopies = int(np.ceil(2 * 256e6 / bw))
    copies = L.weight_copies(ncopies)
    # every copy computes the same output (bitwise: same inputs, deterministic kernel)
    copies[0].call()
    y0 = L.y.clone()
    copies[-1].call()
    torch.cuda.synchronize()
    assert torch.equal(y0, L.y), "a weight copy of the rotation differs from the original layer"
    distinct = None
    if args.launch == "graph":
        ms, steps, distinct = time_rotation(copies, args.steps, args.warmup)
    else:
        ms, steps = time_calls(copies, max(1, args.steps // ncopies), max(1, args.warmup // ncopies),
                               use_graph=False)
        ms, steps = ms / ncopies, steps * ncopies
        distinct = ncopies
    # the same layer called repeatedly (weights warm in the caches), graph-replayed and stream-issued
    ms_warm = ms_stream = None
    if not args.no_warm:
        ms_warm, _ = time_calls([L], args.steps, args.warmup, use_graph=True)
        ms_stream, _ = time_calls([L], min(args.steps, 2000), 100, use_graph=False)
    del copies
    achieved = b / (ms * 1e-3) / 1e9
    traffic = measured_traffic("decode_q_proj_4096_r80_T1")
    rec = {
        "metric": "tokens/s + HBM GB/s (% peak) per LittleBit linear, Llama2-7B shapes @0.1 BPW",
        "value": T / (ms * 1e-3),
        "unit": "tokens/s",
        "n_gpus": 1,
        "steps": steps,
        "warmup": args.warmup,
        "ms_per_step": ms,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "f32",
        "data": "synthetic",
        "config": {"workload": "LittleBit linear forward, Llama2-7B q_proj shape 4096x4096, 0.1 BPW (r=80 per "
                               "path, 2 paths), T=1 decode, bf16 x, fp16 scales, Bernoulli(1/2) signs",
                   "d_in": d_in, "d_out": d_out, "r": r, "T": T, "bpw": round(lb.lb_bits_per_weight(d_in, d_out, r), 5),
                   "kernel": "decode", "launch": args.launch,
                   "weights": f"cold: {ncopies} copies ({ncopies * bw / 1e6:.0f} MB), the timed calls on copies "
                              f"the warm-up did not touch, caches flushed before the timed replay",
                   "distinct_copies_touched": distinct},
        "roofline": {"bound": "hbm", "achieved": achieved, "peak": PEAK_HBM_GBS, "unit": "GB/s",
                     "frac": achieved / PEAK_HBM_GBS, "traffic": traffic,
                     "alg_bytes_per_launch": b, "weights_bytes_per_launch": bw,
                     "avg_launch_us": ms * 1e3,
                     "avg_launch_us_warm": ms_warm * 1e3 if ms_warm is not None else None,
                     "avg_launch_us_warm_stream_issued": ms_stream * 1e3 if ms_stream is not None else None},
    }
    if not args.no_sweep70b:
        ts = tuple(int(t) for t in args.sweep70b_tokens.split(","))
        rec["sweep70b"] = run_sweep70b(ts, args.steps, args.warmup)
    if not args.no_block7b:
        rec["block7b"] = run_block7b((1, 16, 64), args.steps, args.warmup)
    if not args.no_svid:
        rec["svid7b"] = run_svid()
    rec["paper_context"] = PAPER_CONTEXT
    if not args.no_cpu_baseline:
        rec["cpu_baseline"] = cpu_baseline(li, args.cpu_seconds)
    print(json.dumps(rec), flush=True)
    if args.copy_probe:
        copy_probe(args.copy_probe)
    if args.sweep:
        run_sweep(args.sweep, min(args.steps, 1000), min(args.warmup, 100), tuple(args.sweep_only.split(",")))


if __name__ == "__main__":
    main()
