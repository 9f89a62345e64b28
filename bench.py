"""Benchmark of the UltraMem memory-layer forward on one MI355X.

A step is one whole forward of the layer (axis scoring, per-axis top-k, grid top-m, gather-sum)
over one batch of the 20.07M-slot decode workload: 32 tokens, 2 heads, dk 128, 4480 x 4480
keys, a 20,070,400 x 512 bf16 value table (20.55 GB), k = m = 32.  Inputs are resident in HBM
before timing starts.  Steps take distinct query batches from a rotating set (512 batches, over
1 GiB of distinct value rows), and a 1 GiB device copy runs between the untimed and the timed
replay, so every timed step gathers rows that are in no cache (the keys, the same every step,
stay cached from one step to the next, as they would in decoding).

Prints one JSON line (stdout): the headline, the roofline of the dominant kernel (its average
duration over launches replayed back to back from a HIP graph, between two HIP events on the
launch stream; bytes and flops are the method's own, not the intermediates the kernels pass
between them), the decode forward's value-gather rate beside two measured read ceilings of this
GPU, a decode batch sweep, a summary of the other layer shapes, and the CPU oracle's throughput.
The full per-workload reports (every kernel's roofline, backward, overlap, front-end) go to
stderr and, with --details, to a JSON file.
"""
from __future__ import annotations

import argparse
import ctypes
import hashlib
import json
import math
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

HBM_PEAK_GBS = 8000.0          # MI355X HBM3E, vendor figure
FP32_PEAK_TFLOPS = 157.3       # MI355X dense fp32 matrix
BF16_PEAK_TFLOPS = 2500.0      # MI355X dense bf16 matrix
F16_PEAK_TFLOPS = 2500.0       # MI355X dense fp16 matrix
# Vector lane-operations per second: 256 CUs x 4 SIMDs x 16 lanes per clock (a wave64 instruction
# every 4 cycles) x 2.4 GHz.  The selection is compare/select work, one lane-op per element
# examined at the least.
ALU_PEAK_TOPS = 256 * 4 * 16 * 2.4e9 / 1e12
METRIC = "memory-layer tokens/sec + value-gather HBM GB/s (% of peak), 20M-slot decode"
INPUTS = ("seeded counter-based SplitMix64 draws; 'normal' = Irwin-Hall(4) of four 16-bit fields "
          "(bounded at 3.46 sd), std 1/sqrt(dim); decode queries i.i.d.")
KERNEL_SOURCES = {
    "axis_scores_kernel": "score.hip",
    "select_kernel": "select.hip",
    "gather_kernel": "gather.hip",
}
FLUSH_BYTES = 1 << 30
# Untimed replays of each timed graph before its cache flush and timed replay: short timed regions
# (20 decode steps are 0.37 ms) otherwise run before the GPU's clocks reach the state sustained
# work holds them in (measured: the batched decode gather 95.8 us right after other work, 92.3 us
# after 0.3 s of reads).
WARM_SECONDS = 0.25


def warm(replay, torch, seconds=None):
    """Calls ``replay`` (one untimed pass of the work about to be timed) until ``seconds`` of wall
    time have passed, at least once."""
    seconds = WARM_SECONDS if seconds is None else seconds
    t0 = time.perf_counter()
    while True:
        replay()
        torch.cuda.synchronize()
        if time.perf_counter() - t0 >= seconds:
            return


def parse():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=2000)
    ap.add_argument("--warmup", type=int, default=100)
    ap.add_argument("--batches", type=int, default=512, help="distinct query batches rotated")
    ap.add_argument("--no-sweep", action="store_true")
    ap.add_argument("--no-workloads", action="store_true",
                    help="skip the prefill, Tucker + IVE (one and two cores) and 1.6B-x12 forwards")
    ap.add_argument("--only-workload", default=None,
                    help="time only this layer's forward (prefill-1M, tucker-ive-4M, "
                         "tucker-ive-mcs-4M, ultramem-1.6B-x12) and print its report as the "
                         "JSON line")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--warm-seconds", type=float, default=WARM_SECONDS,
                    help="untimed replays of each timed graph before its flush and timed replay")
    ap.add_argument("--cpu-seconds", type=float, default=10.0,
                    help="oracle seconds per leg (one thread, then every worker)")
    ap.add_argument("--cpu-workers", type=int, default=16, help="at most this many oracle processes")
    ap.add_argument("--details", default=None, help="write the full reports to this JSON file")
    ap.add_argument("--copy-calibration", action="store_true",
                    help="first run a plain 256 MiB device copy three times (a known-size kernel "
                         "for scaling HBM traffic counters)")
    ap.add_argument("--eager", action="store_true",
                    help="launch each step from Python instead of replaying a captured HIP graph")
    return ap.parse_args()


def log(msg):
    print(f"[bench] {msg}", file=sys.stderr, flush=True)


# ---------------------------------------------------------------- byte and flop accounting

def kernel_work(cfg, T, fused=False):
    """The method's work per launch of each kernel at T tokens: ``bytes`` counts what the layer
    must read or write (keys, queries, value rows, the selection, outputs), ``intermediate`` the
    scratch one kernel of this build writes for the next (the selection scores), which is not the
    method's.  With ``fused`` the selection kernel also reads the value rows and writes the pooled
    rows."""
    H, n, dk, m = cfg.heads, cfg.n_keys, cfg.dk, cfg.topm
    keys = 2 * H * n * dk * 4
    q = 2 * T * H * dk * 4
    sel = 2 * T * H * n * 4
    sel_out = T * H * m * 4 * (1 + cfg.cores)                 # idx and the weights
    rows = T * cfg.bag * cfg.dv * cfg.vbytes
    cand = (cfg.topk * cfg.topk if cfg.grid else additive_candidates(cfg.topk, m))
    return {
        "axis_scores_kernel": dict(bytes=keys + q, flops=2 * 2 * T * H * n * dk, intermediate=sel),
        "select_kernel": dict(bytes=sel_out + (rows + T * cfg.dv * 4 if fused else 0), flops=0,
                              intermediate=sel, row_bytes=rows if fused else 0,
                              elements=T * H * (2 * n + cand)),
        "gather_kernel": dict(bytes=rows + T * cfg.bag * 4 * (1 + cfg.cores) + T * cfg.expand * cfg.dv * 4,
                              flops=2 * T * cfg.bag * cfg.dv, row_bytes=rows, intermediate=0),
        # the IVE projection and the output linear: two bf16 GEMMs with fp32 accumulation
        "project_kernels": dict(bytes=T * cfg.expand * cfg.dv * 4 + cfg.expand * cfg.dv * cfg.dv_virt * 2
                                + cfg.dv_virt * cfg.d_out * 2 + T * max(cfg.d_out, cfg.dv_virt) * 4,
                                flops=2 * T * cfg.expand * cfg.dv * cfg.dv_virt
                                + 2 * T * cfg.dv_virt * cfg.d_out, intermediate=0),
    }


def additive_candidates(k, m):
    """Grid candidates (a, b) of the additive grid with (a+1)(b+1) <= m."""
    return sum(min(k, m // (a + 1)) for a in range(min(k, m)))


def source_digest(name):
    path = os.path.join(ROOT, "paper_2411_12364_amd", "csrc", KERNEL_SOURCES[name])
    with open(path, "rb") as f:
        return hashlib.sha256(f.read()).hexdigest()[:16]


def measured_traffic(name, workload):
    """HBM bytes per launch from the committed rocprofv3 counter summary, if it was taken on the
    kernel source as it is now; else None."""
    path = os.path.join(ROOT, "profiles", "traffic.json")
    if name not in KERNEL_SOURCES or not os.path.exists(path):
        return None
    with open(path) as f:
        rec = json.load(f).get(workload, {}).get(name)
    if not rec or rec.get("source_sha256_16") != source_digest(name):
        return None
    return rec.get("hbm_bytes_per_launch")


def layer_rules(cfg):
    """(project, fused) as the library decides them: a projection runs when D'v or d_out is set;
    the selection pools the rows itself for layers without expansion or projection, at most two
    heads, topm <= 64, rows of 1 or 2 KiB and T <= 128."""
    project = bool(cfg.dv_virt or cfg.d_out)
    fused = (not project and cfg.expand == 1 and cfg.heads <= 2 and cfg.topm <= 64
             and cfg.dv * cfg.vbytes in (1024, 2048) and cfg.T <= 128)
    return project, fused


# ---------------------------------------------------------------- GPU measurement

class Flusher:
    """A 1 GiB device copy (1 GiB read, 1 GiB written) run outside every timed region: it evicts
    the 256 MB last-level cache and the L2s, so that the timed launches find no value row there."""

    def __init__(self, torch):
        self.torch = torch
        self.src = torch.empty(FLUSH_BYTES, dtype=torch.uint8, device="cuda").fill_(1)
        self.dst = torch.empty_like(self.src)

    def __call__(self):
        self.dst.copy_(self.src)
        self.torch.cuda.synchronize()


class Probe:
    """The read-bandwidth probes of libumem_probe.so (sequential runs; whole rows of a bag)."""

    def __init__(self, torch):
        import paper_2411_12364_amd as U
        path = os.path.join(os.path.dirname(U.LIB_PATH), "libumem_probe.so")
        if not os.path.exists(path):
            raise ImportError(f"{path} is not built; run __graft_entry__.build() first")
        self.lib = ctypes.CDLL(path)
        P = ctypes.c_void_p
        self.lib.umem_probe_read_rows.argtypes = [P, ctypes.c_int, P, ctypes.c_int64, P, P]
        self.lib.umem_probe_read_seq.argtypes = [P, ctypes.c_int64, ctypes.c_int, P, P]
        self.torch = torch
        self.sink = torch.zeros(1024, dtype=torch.int32, device="cuda")

    def read_rows(self, table, row_bytes, rows):
        st = self.lib.umem_probe_read_rows(table.data_ptr(), row_bytes, rows.data_ptr(), rows.numel(),
                                           self.sink.data_ptr(), self.torch.cuda.current_stream().cuda_stream)
        assert st == 0, st

    def read_seq(self, buf, nbytes, blocks=4096):
        st = self.lib.umem_probe_read_seq(buf.data_ptr(), nbytes, blocks, self.sink.data_ptr(),
                                          self.torch.cuda.current_stream().cuda_stream)
        assert st == 0, st


class Runner:
    def __init__(self, cfg, batches, values=None, flusher=None):
        import torch

        import paper_2411_12364_amd as U
        from synth import device as SD
        self.U, self.torch, self.cfg = U, torch, cfg
        t0 = time.time()
        self.dl = SD.make_layer(cfg, batches=batches, values=values)
        torch.cuda.synchronize()
        log(f"inputs for {cfg.name} T={cfg.T} ({batches} query batches) ready in {time.time() - t0:.1f}s")
        self.flush = flusher or Flusher(torch)
        self.desc = self._desc()
        T = cfg.T
        st, nbytes = U.umem_workspace_size(self.desc, T)
        U.check(st)
        self.ws = torch.empty(max(nbytes, 256), dtype=torch.uint8, device="cuda")
        self.project, self.fused = layer_rules(cfg)
        # the forward's output: the projected rows, else the pooled rows [T, E, Dv]
        width = (cfg.d_out or cfg.dv_virt) if self.project else cfg.expand * cfg.dv
        self.out = torch.empty((T, width), dtype=torch.float32, device="cuda")
        self.pooled = torch.empty((T, cfg.expand, cfg.dv), dtype=torch.float32, device="cuda")
        self.idx = torch.empty((T, cfg.heads, cfg.topm), dtype=torch.int32, device="cuda")
        wshape = (T, cfg.heads, cfg.topm) + ((cfg.cores,) if cfg.cores > 1 else ())
        self.w = torch.empty(wshape, dtype=torch.float32, device="cuda")
        self.sel = torch.empty((2, T, cfg.heads, cfg.n_keys), dtype=torch.float32, device="cuda")
        self.R = batches

    def _desc(self):
        c, d = self.cfg, self.U.umem_desc()
        d.heads, d.dk, d.n_keys, d.rank = c.heads, c.dk, c.n_keys, c.rank
        d.topk, d.topm, d.grid, d.weight = c.topk, c.topm, c.grid, c.weight
        d.n_values, d.dv, d.vdtype, d.expand = c.n_values, c.dv, c.vdtype, c.expand
        d.dv_virt, d.d_out, d.cores = c.dv_virt, c.d_out, c.cores
        return d

    def forward(self, b):
        U, dl, c = self.U, self.dl, self.cfg
        st = U.umem_forward(self.desc, c.T, dl.q_row[b], dl.q_col[b], dl.k_row, dl.k_col, dl.core,
                            dl.values, dl.perm, dl.w_proj, dl.w_out, self.out, self.idx, self.w,
                            self.ws, self.ws.numel())
        if st:
            U.check(st, "umem_forward")

    def scores(self, b):
        U, dl, c = self.U, self.dl, self.cfg
        st = U.umem_axis_scores(self.desc, c.T, dl.q_row[b], dl.q_col[b], dl.k_row, dl.k_col,
                                dl.core, self.sel, self.ws, self.ws.numel())
        if st:
            U.check(st, "umem_axis_scores")

    def select(self, sel, idx, w, b=0):
        """The selection as umem_forward launches it: pooling the rows itself where it can."""
        U, dl, c = self.U, self.dl, self.cfg
        pool = self.fused
        st = U.umem_select(self.desc, c.T, sel, dl.q_row[b], dl.q_col[b], dl.k_row, dl.k_col,
                           dl.core, idx, w, None, dl.values if pool else None,
                           self.out if pool else None)
        if st:
            U.check(st, "umem_select")

    def gather(self, idx, w):
        U, dl, c = self.U, self.dl, self.cfg
        st = U.umem_gather_sum(c.n_values, c.dv, c.vdtype, dl.values, c.T, c.bag, idx, w, dl.perm,
                               c.expand, c.cores, self.pooled)
        if st:
            U.check(st, "umem_gather_sum")

    def project_rows(self):
        U, dl, c = self.U, self.dl, self.cfg
        st = U.umem_project(c.T, c.expand, c.dv, c.dv_virt, c.d_out, self.pooled, dl.w_proj,
                            dl.w_out, self.out, self.ws, self.ws.numel())
        if st:
            U.check(st, "umem_project")

    def _graph_time(self, launches):
        """Average seconds per call of ``launches`` (a list of thunks) replayed from a HIP graph,
        between two events on the replay stream, after the cache flush."""
        torch = self.torch
        for f in launches[:8]:
            f()
        torch.cuda.synchronize()
        g = torch.cuda.CUDAGraph()
        with torch.cuda.graph(g):
            for f in launches:
                f()
        g.replay()
        torch.cuda.synchronize()
        warm(g.replay, torch)
        self.flush()
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record()
        g.replay()
        e1.record()
        torch.cuda.synchronize()
        return e0.elapsed_time(e1) * 1e-3 / len(launches)

    def time_forward(self, steps, warmup, graph=True):
        """Wall time of exactly ``steps`` forwards (inputs rotating over the query batches),
        between two device synchronisations, after the cache flush."""
        torch = self.torch
        for s in range(warmup):
            self.forward(s % self.R)
        torch.cuda.synchronize()
        if graph:
            g = torch.cuda.CUDAGraph()
            with torch.cuda.graph(g):
                for s in range(steps):
                    self.forward(s % self.R)
            g.replay()                              # untimed replay: graph upload
            torch.cuda.synchronize()
            warm(g.replay, torch)
            self.flush()
            t0 = time.perf_counter()
            g.replay()
            torch.cuda.synchronize()
            return time.perf_counter() - t0, steps
        warm(lambda: [self.forward(s % self.R) for s in range(steps)], torch)
        self.flush()
        t0 = time.perf_counter()
        for s in range(steps):
            self.forward(s % self.R)
        torch.cuda.synchronize()
        return time.perf_counter() - t0, steps

    def _unique_rows(self, idxs):
        """Distinct physical value rows one step gathers (averaged over the query batches)."""
        c, dl = self.cfg, self.dl
        tot = 0
        for b in range(self.R):
            flat = idxs[b].reshape(-1).long()
            rows = flat if dl.perm is None else dl.perm[flat].long() % c.n_values
            tot += int(self.torch.unique(rows).numel())
        return tot / self.R

    def time_probe_rows(self, probe, launches=64):
        """Average seconds per launch of the read probe over exactly the rows the selections of
        the rotating query batches gather (one launch per batch, T x bag rows), for comparison
        with the gather kernel on the same rows (kept from time_kernels)."""
        idxs, _ = self.queue_inputs
        c = self.cfg
        return self._graph_time([lambda b=b: probe.read_rows(self.dl.values, c.dv * c.vbytes,
                                                              idxs[b % self.R]) for b in range(launches)])

    def time_kernels(self, launches_per_kernel, queue=False):
        """Average duration (us) of each kernel of the forward, launched back to back from a HIP
        graph with distinct inputs per launch: the scoring over the rotating query batches, the
        selection over the score sets of all of them, the gather over their selections."""
        torch = self.torch
        c, n = self.cfg, launches_per_kernel
        sels = torch.empty((self.R,) + tuple(self.sel.shape), dtype=torch.float32, device="cuda")
        idxs = torch.empty((self.R,) + tuple(self.idx.shape), dtype=torch.int32, device="cuda")
        ws_ = torch.empty((self.R,) + tuple(self.w.shape), dtype=torch.float32, device="cuda")
        for b in range(self.R):
            self.scores(b)
            sels[b].copy_(self.sel)
            self.select(self.sel, idxs[b], ws_[b], b)
        torch.cuda.synchronize()
        out = {
            "axis_scores_kernel": self._graph_time([lambda b=b: self.scores(b % self.R) for b in range(n)]),
            "select_kernel": self._graph_time([lambda b=b: self.select(sels[b % self.R], self.idx, self.w, b % self.R)
                                               for b in range(n)]),
            "gather_kernel": self._graph_time([lambda b=b: self.gather(idxs[b % self.R], ws_[b % self.R])
                                               for b in range(n)]),
        }
        if self.project:
            out["project_kernels"] = self._graph_time([self.project_rows] * n)
        self.queue_inputs = (idxs, ws_) if queue else None
        self.unique_rows = self._unique_rows(idxs)
        del sels
        if not queue:
            del idxs, ws_
        return {k: v * 1e6 for k, v in out.items()}

    def time_gather_queue(self, probe):
        """The gather of many queued decode steps in one launch: the selections of R/2 distinct
        query batches (R/2 * T tokens) pooled by one umem_gather_sum, alternating between the two
        halves of the R batches; beside it, the probe reading exactly the same rows."""
        torch, U, dl, c = self.torch, self.U, self.dl, self.cfg
        idxs, ws_ = self.queue_inputs
        half = self.R // 2
        if half < 2:
            return None
        Tq = half * c.T
        stacks = [(idxs[i * half:(i + 1) * half].reshape(Tq, c.bag).contiguous(),
                   ws_[i * half:(i + 1) * half].reshape((Tq, c.bag) + tuple(ws_.shape[4:])).contiguous())
                  for i in (0, 1)]
        outq = torch.empty((Tq, c.expand, c.dv), dtype=torch.float32, device="cuda")

        def launch(i):
            st = U.umem_gather_sum(c.n_values, c.dv, c.vdtype, dl.values, Tq, c.bag, stacks[i][0],
                                   stacks[i][1], dl.perm, c.expand, c.cores, outq)
            if st:
                U.check(st, "umem_gather_sum")
        secs = self._graph_time([lambda i=i: launch(i % 2) for i in range(16)])
        probe_secs = self._graph_time([lambda i=i: probe.read_rows(dl.values, c.dv * c.vbytes,
                                                                    stacks[i % 2][0]) for i in range(16)])
        rows = Tq * c.bag * c.dv * c.vbytes
        algo = kernel_work(c.with_tokens(Tq), Tq)["gather_kernel"]["bytes"]   # + bag, + output
        uniq = int(torch.unique(stacks[0][0]).numel())
        del outq, stacks
        self.queue_inputs = None
        return dict(what=f"batched proxy: the bags of {half} distinct {c.T}-token decode steps "
                         f"pooled by one gather launch ({Tq} tokens)",
                    row_bytes=rows, unique_row_bytes=uniq * c.dv * c.vbytes,
                    avg_us=round(secs * 1e6, 2), GBps=round(rows / secs / 1e9, 1),
                    frac_of_peak=round(rows / secs / 1e9 / HBM_PEAK_GBS, 4),
                    probe_same_rows_GBps=round(rows / probe_secs / 1e9, 1),
                    frac_of_probe=round(probe_secs / secs, 4),
                    algorithmic_GBps=round(algo / secs / 1e9, 1),
                    algorithmic_frac_of_peak=round(algo / secs / 1e9 / HBM_PEAK_GBS, 4))


def scores_on_planes(cfg, T):
    """Whether the scoring of T tokens takes the fp16-plane kernel (the library's own rule)."""
    return T > 64 and cfg.dk % 32 == 0 and cfg.n_keys % 4 == 0 and (cfg.dk // cfg.rank) % 8 == 0


def roofline_for(cfg, T, name, avg_us, workload, fused, unique_row_bytes=None):
    """The roofline of one kernel on the method's work (kernel_work).  The gather of a layer whose
    rows repeat within a launch is priced on its distinct rows (what HBM must deliver) when
    ``unique_row_bytes`` is given."""
    work = kernel_work(cfg, T, fused)[name]
    base = dict(kernel=name, avg_us=round(avg_us, 3))
    if name == "project_kernels":
        achieved = work["flops"] / (avg_us * 1e-6) / 1e12
        return dict(base, bound="mfma", achieved=round(achieved, 2), peak=BF16_PEAK_TFLOPS,
                    unit="TFLOP/s", frac=round(achieved / BF16_PEAK_TFLOPS, 4), traffic=None)
    if name == "axis_scores_kernel":
        tr = measured_traffic(name, workload)
        if work["flops"] / work["bytes"] > FP32_PEAK_TFLOPS * 1e3 / HBM_PEAK_GBS:
            # the method's flops at fp32 accuracy.  The fp32-MFMA kernel is priced on the fp32
            # peak; the fp16-plane kernel computes on fp16 MFMA and is priced on that dtype's peak
            # (the same as bf16's), with its three issued fp16 products per method flop and the
            # fp32 peak's fraction reported beside.
            achieved = work["flops"] / (avg_us * 1e-6) / 1e12
            planes = scores_on_planes(cfg, T)
            peak = F16_PEAK_TFLOPS if planes else FP32_PEAK_TFLOPS
            r = dict(base, bound="mfma", achieved=round(achieved, 2), peak=peak,
                     unit="TFLOP/s", frac=round(achieved / peak, 4), traffic=tr,
                     mfma_dtype="f16 (two parts per fp32 operand)" if planes else "f32",
                     intermediate_bytes=work["intermediate"])
            if planes:
                issued = 3 * achieved
                r.update(issued_fp16_TFLOPs=round(issued, 1),
                         issued_frac_of_fp16_peak=round(issued / F16_PEAK_TFLOPS, 4),
                         frac_of_fp32_peak=round(achieved / FP32_PEAK_TFLOPS, 4))
            return r
        achieved = work["bytes"] / (avg_us * 1e-6) / 1e9
        return dict(base, bound="hbm", achieved=round(achieved, 1), peak=HBM_PEAK_GBS, unit="GB/s",
                    frac=round(achieved / HBM_PEAK_GBS, 4), traffic=tr, algorithmic_bytes=work["bytes"],
                    intermediate_bytes=work["intermediate"])
    if name == "select_kernel" and not fused:
        achieved = work["elements"] / (avg_us * 1e-6) / 1e12
        return dict(base, bound="alu", achieved=round(achieved, 4), peak=round(ALU_PEAK_TOPS, 2),
                    unit="T element-ops/s", frac=round(achieved / ALU_PEAK_TOPS, 5), traffic=None,
                    elements=work["elements"], intermediate_bytes=work["intermediate"])
    nbytes = work["bytes"]
    if name == "gather_kernel" and unique_row_bytes is not None:
        nbytes = nbytes - work["row_bytes"] + int(unique_row_bytes)
    achieved = nbytes / (avg_us * 1e-6) / 1e9
    return dict(base, bound="hbm", achieved=round(achieved, 1), peak=HBM_PEAK_GBS, unit="GB/s",
                frac=round(achieved / HBM_PEAK_GBS, 4), traffic=measured_traffic(name, workload),
                algorithmic_bytes=int(nbytes), intermediate_bytes=work["intermediate"])


def workload_report(cfg, flusher, steps=50, warmup=5):
    """The whole forward of another layer shape (graph-replayed, distinct query batches, cold
    caches) and the roofline of each of its kernels.  The gather is priced on the distinct rows of
    a step (what HBM must deliver); its rate on the logical rows of its bag (eq. (1)) is given
    beside."""
    R = max(2, distinct_batches(cfg.T, cfg.bag * cfg.dv * cfg.vbytes))
    r = Runner(cfg, R, flusher=flusher)
    secs, n = r.time_forward(steps, warmup)
    st = r.time_kernels(min(steps, 64))
    kernels = ["axis_scores_kernel", "select_kernel"] + ([] if r.fused else ["gather_kernel"])
    if r.project:
        kernels.append("project_kernels")
    g = kernel_work(cfg, cfg.T)["gather_kernel"]
    uniq = r.unique_rows * cfg.dv * cfg.vbytes
    rep = dict(workload=cfg.name, tokens=cfg.T, heads=cfg.heads, n_keys=cfg.n_keys,
               slots=cfg.n_slots, rank=cfg.rank, grid="tucker" if cfg.grid else "additive",
               expand=cfg.expand, cores=cfg.cores, topk=cfg.topk, topm=cfg.topm, dv=cfg.dv,
               query_batches=R, us_per_step=round(secs / n * 1e6, 2),
               tokens_per_s=round(cfg.T * n / secs, 1),
               kernel_us={k: round(v, 3) for k, v in st.items()}, forward_kernels=kernels,
               rooflines={k: roofline_for(cfg, cfg.T, k, st[k], cfg.name, r.fused,
                                          uniq if k == "gather_kernel" else None) for k in kernels},
               gather_unique_row_bytes=int(uniq),
               gather_unique_GBps=round(uniq / (st["gather_kernel"] * 1e-6) / 1e9, 1),
               gather_logical_GBps=round(g["row_bytes"] / (st["gather_kernel"] * 1e-6) / 1e9, 1))
    rep["backward"] = backward_report(r)
    if cfg.name in overlap_stand_ins():
        rep["overlap"] = overlap_report(r, *overlap_stand_ins()[cfg.name])
    fe = front_ends().get(cfg.name)
    if fe is not None:
        rep["front_end"] = front_end_report(fe)
        rep["tokens_per_s_with_front_end"] = round(
            cfg.T / ((secs / n) + rep["front_end"]["avg_us"] * 1e-6), 1)
    log(f"workload {cfg.name}: {json.dumps(rep)}")
    del r
    import torch
    torch.cuda.empty_cache()
    return rep


def front_end_report(fe, launches=200):
    """The query front-end (convolution, query linear, LayerNorm) of ``fe``: the average
    duration of ``launches`` umem_query calls replayed from a HIP graph, and its roofline."""
    import numpy as np
    import torch

    import paper_2411_12364_amd as U
    from synth import configs as CF
    inp = CF.front_end_inputs(fe)
    qd = U.umem_query_desc()
    qd.d_model, qd.conv_k, qd.heads, qd.dk, qd.shared, qd.eps = (fe.d_model, fe.conv_k, fe.heads,
                                                                  fe.dk, int(fe.shared), fe.eps)
    st, nws = U.umem_query_workspace_size(qd, fe.B, fe.L)
    U.check(st)
    ws = torch.empty(max(nws, 256), dtype=torch.uint8, device="cuda")
    dev = lambda a: None if a is None else torch.from_numpy(np.ascontiguousarray(a)).cuda()
    x, hist, cw = dev(inp["x"]), dev(inp["hist"]), dev(inp["conv_w"])
    wq, g, b = dev(CF.output_major(inp["w_q"]).view(np.int16)), dev(inp["gamma"]), dev(inp["beta"])
    q_row = torch.empty((fe.T, fe.heads, fe.dk), dtype=torch.float32, device="cuda")
    q_col = None if fe.shared else torch.empty_like(q_row)

    def call():
        st = U.umem_query(qd, fe.B, fe.L, x, hist, cw, wq, g, b, q_row, q_col, ws, ws.numel())
        if st:
            U.check(st, "umem_query")
    for _ in range(3):
        call()
    torch.cuda.synchronize()
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph):
        for _ in range(launches):
            call()
    graph.replay()
    torch.cuda.synchronize()
    warm(graph.replay, torch)
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record()
    graph.replay()
    e1.record()
    torch.cuda.synchronize()
    us = e0.elapsed_time(e1) * 1e3 / launches
    A = 1 if fe.shared else 2
    hist_rows = fe.B * (fe.conv_k - 1) if fe.history else 0
    algo = (4 * (fe.T + hist_rows + fe.conv_k) * fe.d_model + 2 * fe.d_model * fe.n_queries
            + 4 * 2 * A * fe.heads * fe.dk + 4 * fe.T * fe.n_queries)
    flops = 2 * fe.T * fe.d_model * fe.n_queries
    achieved = algo / (us * 1e-6) / 1e9
    return dict(front_end=fe.name, tokens=fe.T, d_model=fe.d_model, conv_k=fe.conv_k,
                shared=fe.shared, avg_us=round(us, 3), algorithmic_bytes=algo,
                roofline=dict(kernel="query_front_end", bound="hbm", achieved=round(achieved, 1),
                              peak=HBM_PEAK_GBS, unit="GB/s", frac=round(achieved / HBM_PEAK_GBS, 4),
                              traffic=None, avg_us=round(us, 3)),
                gemm_TFLOPs=round(flops / (us * 1e-6) / 1e12, 2))


def backward_report(r, launches=20):
    """The backward of one step of runner ``r``'s layer at its forward's selection: the gather
    backward (value-row and weight gradients) and the score backward (query, key and core
    gradients), each replayed ``launches`` times from a HIP graph."""
    torch, U, dl, c = r.torch, r.U, r.dl, r.cfg
    r.forward(0)
    T = c.T
    idx, w = r.idx.reshape(T, c.bag), r.w.reshape((T, c.bag) + tuple(r.w.shape[3:]))
    dp = torch.randn((T, c.expand, c.dv), dtype=torch.float32, device="cuda")
    dV = torch.zeros((c.n_values, c.dv), dtype=torch.float32, device="cuda")
    dw = torch.empty_like(w)
    st, n1 = U.umem_gather_backward_workspace_size(T, c.bag, c.dv)
    U.check(st)
    ws1 = torch.empty(max(n1, 256), dtype=torch.uint8, device="cuda")
    st, n2 = U.umem_score_backward_workspace_size(r.desc, T)
    U.check(st)
    ws2 = torch.empty(max(n2, 256), dtype=torch.uint8, device="cuda")
    dq_r, dq_c = torch.empty_like(dl.q_row[0]), torch.empty_like(dl.q_col[0])
    dk_r, dk_c = torch.zeros_like(dl.k_row), torch.zeros_like(dl.k_col)
    dcore = None if dl.core is None else torch.zeros_like(dl.core)

    def gb():
        st = U.umem_gather_backward(c.n_values, c.dv, c.vdtype, dl.values, T, c.bag, idx, w, dl.perm,
                                    c.expand, c.cores, dp, dV, dw, ws1, ws1.numel())
        if st:
            U.check(st, "umem_gather_backward")

    def sb():
        st = U.umem_score_backward(r.desc, T, dl.q_row[0], dl.q_col[0], dl.k_row, dl.k_col, dl.core,
                                   r.idx, r.w, dw.reshape(r.w.shape), dq_r, dq_c, dk_r, dk_c, dcore,
                                   ws2, ws2.numel())
        if st:
            U.check(st, "umem_score_backward")
    # the compact form: one gradient row per distinct row, written (the dense row is not read)
    M = T * c.bag
    rows = torch.empty((M,), dtype=torch.int32, device="cuda")
    d_rows = torch.empty((M, c.dv), dtype=torch.float32, device="cuda")
    n_rows = torch.empty((1,), dtype=torch.int32, device="cuda")

    def gr():
        st = U.umem_gather_backward_rows(c.n_values, c.dv, c.vdtype, dl.values, T, c.bag, idx, w,
                                         dl.perm, c.expand, c.cores, dp, rows, d_rows, n_rows, dw,
                                         ws1, ws1.numel())
        if st:
            U.check(st, "umem_gather_backward_rows")
    g_us = r._graph_time([gb] * launches) * 1e6
    gr_us = r._graph_time([gr] * launches) * 1e6
    s_us = r._graph_time([sb] * launches) * 1e6
    uniq = r.unique_rows
    # value row read and fp32 gradient row read and written per distinct row (the compact form:
    # written only, plus its row number), d_pooled once, idx, w and dw per entry
    per_entry = T * c.expand * c.dv * 4 + T * c.bag * 4 * (2 + c.cores)
    algo = int(uniq * c.dv * (c.vbytes + 8) + per_entry)
    algo_rows = int(uniq * (c.dv * (c.vbytes + 4) + 4) + per_entry)

    def roof(kernel, us, nbytes):
        achieved = nbytes / (us * 1e-6) / 1e9
        return dict(kernel=kernel, bound="hbm", achieved=round(achieved, 1), peak=HBM_PEAK_GBS,
                    unit="GB/s", frac=round(achieved / HBM_PEAK_GBS, 4), traffic=None,
                    avg_us=round(us, 3), algorithmic_bytes=nbytes)
    out = dict(gather_backward_us=round(g_us, 3), gather_backward_rows_us=round(gr_us, 3),
               score_backward_us=round(s_us, 3),
               tokens_per_s=round(T / ((g_us + s_us) * 1e-6), 1),
               gather_backward_roofline=roof("gather_backward", g_us, algo),
               gather_backward_rows_roofline=roof("gather_backward_rows", gr_us, algo_rows))
    del dV, ws1, ws2, d_rows
    return out


def overlap_stand_ins():
    """Layer name -> (hidden width, MLP width, transformer layers spanned) of the dense work the
    memory layer can run beside: in UltraMem-1.6B each memory layer takes layer 3's output and
    adds into layer 7's (insertion 3:7/8:12/...), so it spans four layers of hidden 2048, MLP
    8192."""
    from synth import configs as CF
    return {CF.C6.name: (2048, 8192, 4)}


def overlap_report(r, d_model, d_ff, layers, launches=10):
    """The memory layer beside the dense layers (the skip-layer structure of Sec. 3.2 and the
    asynchronous execution of the appendix): ``launches`` forwards of runner ``r``'s layer on one
    stream and ``launches`` passes of a stand-in for the dense layers it spans on another, each
    replayed from its own HIP graph, timed alone and concurrently.  The stand-in is the bf16
    GEMMs of ``layers`` transformer layers over the layer's tokens (QKV and output projections,
    MLP up and down; random weights, distinct per layer); attention's own softmax and cache reads
    are left out."""
    torch, c = r.torch, r.cfg
    x = torch.randn((c.T, d_model), dtype=torch.bfloat16, device="cuda")
    ws = [(torch.randn((d_model, 3 * d_model), dtype=torch.bfloat16, device="cuda") / d_model ** 0.5,
           torch.randn((d_model, d_model), dtype=torch.bfloat16, device="cuda") / d_model ** 0.5,
           torch.randn((d_model, d_ff), dtype=torch.bfloat16, device="cuda") / d_model ** 0.5,
           torch.randn((d_ff, d_model), dtype=torch.bfloat16, device="cuda") / d_ff ** 0.5)
          for _ in range(layers)]

    def dense():
        for wqkv, wo, w1, w2 in ws:
            torch.mm(x, wqkv)
            torch.mm(x, wo)
            torch.mm(torch.mm(x, w1), w2)

    def capture(fns):
        for f in fns[:2]:
            f()
        torch.cuda.synchronize()
        g = torch.cuda.CUDAGraph()
        with torch.cuda.graph(g):
            for f in fns:
                f()
        return g
    g_mem = capture([lambda b=b: r.forward(b % r.R) for b in range(launches)])
    g_dense = capture([dense] * launches)
    s_mem, s_dense = torch.cuda.Stream(), torch.cuda.Stream()     # default priority

    def timed(which):
        main = torch.cuda.current_stream()
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        done = []
        e0.record(main)
        for g, s in which:
            s.wait_event(e0)
            with torch.cuda.stream(s):
                g.replay()
            ev = torch.cuda.Event()
            ev.record(s)
            done.append(ev)
        for ev in done:
            main.wait_event(ev)
        e1.record(main)
        torch.cuda.synchronize()
        return e0.elapsed_time(e1) * 1e3 / launches
    warm(lambda: timed([(g_mem, s_mem), (g_dense, s_dense)]), torch)
    mem_us = timed([(g_mem, s_mem)])
    dense_us = timed([(g_dense, s_dense)])
    both_us = timed([(g_mem, s_mem), (g_dense, s_dense)])
    dense_flops = layers * 2 * c.T * (4 * d_model * d_model + 2 * d_model * d_ff)
    del g_mem, g_dense, ws
    return dict(dense_stand_in=(f"bf16 GEMMs of {layers} transformer layers (hidden {d_model}, MLP "
                                f"{d_ff}) over {c.T} tokens"),
                memory_layer_us=round(mem_us, 2), dense_us=round(dense_us, 2),
                dense_TFLOPs=round(dense_flops / (dense_us * 1e-6) / 1e12, 1),
                sequential_us=round(mem_us + dense_us, 2), concurrent_us=round(both_us, 2),
                memory_layer_hidden_frac=round((mem_us + dense_us - both_us) / mem_us, 3))


def front_ends():
    """Layer name -> the query front-end timed beside that layer's forward."""
    from synth import configs as CF
    return {CF.C6.name: CF.FE6}


def extra_workloads(CF):
    """The layer shapes reported beside the decode headline."""
    import dataclasses
    return (CF.C2, CF.C5, dataclasses.replace(CF.C5, cores=2, name="tucker-ive-mcs-4M"), CF.C6)


def distinct_batches(T, row_bytes_per_token):
    """Enough query batches that one rotation touches over 1 GiB of value rows (capped)."""
    return int(min(4096, max(1, math.ceil((1 << 30) / (T * row_bytes_per_token)))))


def gather_figure(cfg, T, st, fused):
    """The value gather of the decode forward as it runs: inside the selection kernel where that
    pools the rows, else the gather kernel; its row bytes over that kernel's time."""
    name = "select_kernel" if fused else "gather_kernel"
    rows = kernel_work(cfg, T)["gather_kernel"]["row_bytes"]
    gbps = rows / (st[name] * 1e-6) / 1e9
    return dict(kernel=name + (" (pools the rows)" if fused else ""), row_bytes=rows,
                avg_us=round(st[name], 3), GBps=round(gbps, 1), frac_of_peak=round(gbps / HBM_PEAK_GBS, 4))


def sweep(base_cfg, values, flusher, probe, steps=512, warmup=30):
    """The decode forward at T = 1 ... 1024 on the same table; the gather figure is taken from
    the kernel that pools the rows in that forward.  Where that is the gather kernel, the read
    probe over exactly the same rows is timed beside it: the ceiling of one launch of that size."""
    res = []
    for T in (1, 4, 16, 64, 256, 1024):
        cfg = base_cfg.with_tokens(T)
        R = distinct_batches(T, cfg.bag * cfg.dv * cfg.vbytes)
        r = Runner(cfg, R, values, flusher)
        secs, n = r.time_forward(steps, warmup)
        st = r.time_kernels(min(steps, 512), queue=not r.fused)
        gf = gather_figure(cfg, T, st, r.fused)
        row = dict(tokens=T, query_batches=R, us_per_step=round(secs / n * 1e6, 2),
                   tokens_per_s=round(T * n / secs, 1),
                   kernel_us={k: round(v, 2) for k, v in st.items()},
                   gather_kernel=gf["kernel"], gather_GBps=gf["GBps"],
                   gather_frac=gf["frac_of_peak"])
        if not r.fused:
            p_us = r.time_probe_rows(probe) * 1e6
            row.update(probe_same_rows_us=round(p_us, 2),
                       probe_same_rows_GBps=round(gf["row_bytes"] / (p_us * 1e-6) / 1e9, 1),
                       gather_frac_of_probe=round(p_us / st["gather_kernel"], 4))
            r.queue_inputs = None
        res.append(row)
        log(f"sweep T={T}: {res[-1]}")
        del r
        import torch
        torch.cuda.empty_cache()
    return res


# ---------------------------------------------------------------- CPU oracle baseline

def _oracle_batches(cfg, seconds, first_batch, max_batches=400):
    """The oracle (unchanged) on successive query batches of ``cfg`` until ``seconds`` of its own
    time have elapsed: (tokens, seconds).  Value rows are drawn before each timed call (a first,
    untimed call learns which rows are gathered), so input generation is excluded."""
    import numpy as np
    from threadpoolctl import threadpool_limits

    import oracle.umem_oracle as O
    from synth import configs as CF

    kr, kc = CF.keys(cfg)
    tokens, spent, b = 0, 0.0, 0
    with threadpool_limits(limits=1):
        while spent < seconds and b < max_batches:
            qr, qc = CF.queries(cfg, batch=first_batch + b)
            sel = O.score_topk(qr, qc, kr, kc, cfg.topk, cfg.topm, cfg.grid, cfg.weight)
            rows = np.unique(sel["idx"].reshape(-1))
            table = dict(zip(rows.tolist(), CF.value_rows_f32(cfg, rows)))
            fetch = lambda r: np.stack([table[int(x)] for x in r])
            t0 = time.perf_counter()
            O.forward(qr, qc, kr, kc, fetch, cfg.topk, cfg.topm, cfg.grid, cfg.weight)
            spent += time.perf_counter() - t0
            tokens += cfg.T
            b += 1
    return tokens, spent


def _oracle_worker(args):
    name, seconds, first = args
    from synth import configs as CF
    return _oracle_batches(CF.CONFIGS[name], seconds, first)


def cpu_baseline(cfg, seconds, max_workers):
    """The oracle on the host cores: one thread alone, then one process per core (at most
    ``max_workers``, each single-threaded, on distinct batches, all at once); the all-core
    throughput is the sum of the workers' own rates.  Runs before the GPU is touched, so the
    worker processes are forked from a process without GPU state."""
    import multiprocessing as mp
    cpu_model = "unknown"
    try:
        with open("/proc/cpuinfo") as f:
            cpu_model = next((l.split(":", 1)[1].strip() for l in f if l.startswith("model name")), cpu_model)
    except OSError:
        pass
    avail = len(os.sched_getaffinity(0))
    workers = max(1, min(avail, max_workers))
    tok1, sec1 = _oracle_batches(cfg, seconds, 1000)
    with mp.get_context("fork").Pool(workers) as pool:
        parts = pool.map(_oracle_worker, [(cfg.name, seconds, 2000 + 400 * i) for i in range(workers)])
    rate = sum(t / s for t, s in parts)
    return dict(value=round(rate, 1), unit="tokens/s", cores=workers, kind="oracle",
                single_thread=round(tok1 / sec1, 1),
                host=f"{cpu_model}; {avail} cores available to the process, {os.cpu_count()} online",
                sample=(f"fp64 numpy oracle on successive {cfg.T}-token batches of {cfg.name}: "
                        f"{tok1 // cfg.T} batches in {sec1:.1f} s on 1 thread; then {workers} "
                        f"single-threaded processes at once, {sum(t for t, _ in parts) // cfg.T} "
                        f"batches, about {seconds:.0f} s each"))


# ---------------------------------------------------------------- main

def main():
    global WARM_SECONDS
    args = parse()
    WARM_SECONDS = args.warm_seconds
    if args.gpus != 1:
        print(f"bench.py runs on one GPU only (asked for {args.gpus}); the memory layer is not "
              "sharded across GPUs.", file=sys.stderr)
        sys.exit(2)
    from synth import configs as CF
    cfg = CF.C3
    # the oracle first, before this process touches the GPU (its worker processes are forked)
    cpu = None
    if not args.no_cpu_baseline and not args.only_workload:
        cpu = cpu_baseline(cfg, args.cpu_seconds, args.cpu_workers)
        log(f"cpu baseline: {cpu}")
    import torch
    torch.cuda.set_device(0)
    if args.copy_calibration:
        a = torch.empty(256 << 20, dtype=torch.uint8, device="cuda").fill_(1)
        b = torch.empty_like(a)
        for _ in range(3):
            b.copy_(a)
        torch.cuda.synchronize()
        log("copy calibration: 3 x 256 MiB device copies done")
        del a, b
    flusher = Flusher(torch)
    if args.only_workload:
        layers = {c.name: c for c in extra_workloads(CF)}
        if args.only_workload not in layers:
            print(f"unknown workload {args.only_workload}; one of {sorted(layers)}", file=sys.stderr)
            sys.exit(2)
        print(json.dumps(workload_report(layers[args.only_workload], flusher, args.steps,
                                         args.warmup)), flush=True)
        return
    r = Runner(cfg, args.batches, flusher=flusher)
    secs, n = r.time_forward(args.steps, args.warmup, graph=not args.eager)
    ms = secs / n * 1e3
    log(f"forward: {n} steps in {secs:.4f}s = {ms * 1e3:.2f} us/step")
    e_secs, e_n = r.time_forward(min(args.steps, 1000), 10, graph=False)
    eager_us = e_secs / e_n * 1e6
    log(f"eager forward (one launch sequence per step from Python): {eager_us:.2f} us/step")
    stage_us = r.time_kernels(512, queue=True)
    log(f"per-kernel (graph replay, events, cold rows): {stage_us}")
    # the kernels umem_forward launches: the standalone gather only where the selection does not
    # pool the rows itself
    fused = r.fused
    fwd_kernels = ["axis_scores_kernel", "select_kernel"] + ([] if fused else ["gather_kernel"])
    dominant = max(fwd_kernels, key=stage_us.get)
    probe = Probe(torch)
    queue = r.time_gather_queue(probe)
    log(f"gather of queued decode steps: {queue}")
    # the ceilings: a sequential read of 4 GiB of the table, and the random rows of the queue
    nseq = min(4 << 30, r.dl.values.numel() * r.dl.values.element_size()) // 16 * 16
    seq_s = r._graph_time([lambda: probe.read_seq(r.dl.values, nseq)] * 4)
    probe_rep = dict(sequential_read_GBps=round(nseq / seq_s / 1e9, 1),
                     random_1KiB_rows_GBps=queue["probe_same_rows_GBps"] if queue else None,
                     what="libumem_probe.so: 16-byte nontemporal loads folded by XOR, no stores; "
                          "4 GiB of the table in order, and the queued bags' rows")
    gather = gather_figure(cfg, cfg.T, stage_us, fused)
    if queue:
        gather["frac_of_probe_rows"] = round(gather["GBps"] / queue["probe_same_rows_GBps"], 4)
        queue["frac_of_sequential_probe"] = round(queue["GBps"] / probe_rep["sequential_read_GBps"], 4)
    step_bytes = sum(kernel_work(cfg, cfg.T, fused)[k]["bytes"] for k in fwd_kernels)
    values = r.dl.values
    del r
    sw = None if args.no_sweep else sweep(cfg, values, flusher, probe)
    del values
    torch.cuda.empty_cache()
    wl = None if args.no_workloads else [workload_report(c, flusher) for c in extra_workloads(CF)]
    line = {
        "metric": METRIC, "value": round(cfg.T * n / secs, 1), "unit": "tokens/s", "n_gpus": 1,
        "steps": n, "warmup": args.warmup, "ms_per_step": round(ms, 5), "higher_is_better": True,
        "scaling": "weak", "vs_baseline": None, "dtype": "f32", "data": "synthetic",
        "config": {"workload": cfg.name, "tokens": cfg.T, "heads": cfg.heads, "dk": cfg.dk,
                   "n_keys": cfg.n_keys, "slots": cfg.n_slots, "dv": cfg.dv, "values": "bf16",
                   "topk": cfg.topk, "topm": cfg.topm, "query_batches": args.batches,
                   "launch": "eager" if args.eager else "hip-graph",
                   "timed_region": (f"{WARM_SECONDS:g} s of untimed replays of the same steps, then "
                                    "cold rows: 1 GiB device copy before the timed replay, a "
                                    "distinct query batch per step"),
                   "inputs": INPUTS},
        "roofline": roofline_for(cfg, cfg.T, dominant, stage_us[dominant], cfg.name, fused),
        "step_roofline": dict(algorithmic_bytes=step_bytes, GBps=round(step_bytes / (ms * 1e-3) / 1e9, 1),
                              frac=round(step_bytes / (ms * 1e-3) / 1e9 / HBM_PEAK_GBS, 4)),
        "cpu_baseline": cpu,
        "kernel_us": {k: round(v, 3) for k, v in stage_us.items()},
        "forward_kernels": fwd_kernels,
        "eager_us_per_step": round(eager_us, 3),
        "gather": gather,
        "gather_queue": queue,
        "probe": probe_rep,
        "batch_sweep": None if sw is None else [
            {k: s[k] for k in ("tokens", "us_per_step", "tokens_per_s", "gather_GBps", "gather_frac",
                               "probe_same_rows_GBps", "gather_frac_of_probe") if k in s}
            for s in sw],
        "workloads": None if wl is None else {
            w["workload"]: dict(us_per_step=w["us_per_step"], tokens_per_s=w["tokens_per_s"],
                                kernel_us={k: round(v, 1) for k, v in w["kernel_us"].items()},
                                gather_frac_unique=w["rooflines"].get("gather_kernel", {}).get("frac"),
                                backward_us=round(w["backward"]["gather_backward_us"]
                                                  + w["backward"]["score_backward_us"], 1))
            for w in wl},
    }
    if args.details:
        with open(args.details, "w") as f:
            json.dump(dict(line, batch_sweep_full=sw, workloads_full=wl), f, indent=1)
    print(json.dumps(line), flush=True)


if __name__ == "__main__":
    main()
