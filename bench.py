#!/usr/bin/env python3
"""Benchmark of the MASW hot path on one MI355X (gfx950).

    python bench.py [--gpus 1] [--steps 64] [--warmup 8] [--no-cpu-baseline]

Headline workload: draft decode at a 32K prefix -- batch 1, 16 layers, 32
query / 8 KV heads, head_dim 64, bf16, a compact memory of 2048 slots (slot
interval 16, no sinks) plus a 1024-token exact window.  One step is one draft
token through all 16 layers:
  * per layer, the fused draft decode attention over [memory | window ring]
    with the current token's K/V appended to the ring in the same launch;
  * when a sequence crosses a 64-token boundary, per layer the memory update
    (mirrored projection of 4 slot rows + RoPE + append) and then one launch
    for the raw query and the four new slots' write scopes (five rows aliasing
    one sequence's buffers).
Six independent sequences are decoded round-robin so that each layer's data
(6.3 MB, 100 MB per sequence) has left the 256 MB Infinity Cache before it is
read again: the timed reads come from HBM.  The timed steps are captured in
one HIP graph and replayed, so the clock measures GPU work, not Python.

Reported in the same run (sub-objects of the JSON line):
  full_kv        the same draft step over the uncompressed 32768-token KV
  batched_decode the same kernel on 16 sequences per launch (50 MB of K/V)
  memory_update  the adaptor alone at 4 rows (32K) and 64 rows (16 sequences)
  verify         the target's 5-query verify attention, 8B- and 70B-shaped
                 layers at a 32768-token prefix
  accept         greedy accept on [B, 5, 128256] fp32 logits, and the stochastic
                 accept/reject rule on probabilities with caller uniforms
  draft_layer    whole draft steps through 16 random-init decoder layers
                 (RMSNorm, Q/K/V + RoPE, attention, projections, SwiGLU) with
                 the compact memory and with the full KV, and the weight
                 stream of the linear maps alone
  memory_prefill the draft's masked prefill attention over a 32K prefix (32768
                 raw tokens + 2048 slots, 32/8 heads, d 64 and d 128), TFLOP/s
                 against the bf16 matrix-core peak
  draft_8k       the 8K-prefix draft: 512 slots + 512-token window, 64 steps
                 per sequence with its memory update, beside the full 8K KV
  batched_drafting  16 ragged sequences drafting 4 tokens per iteration for
                 128 iterations with staggered memory updates (one graph)
  probes         the device's own figures: streaming read bandwidth (the
                 measured peak the fractions are also reported against), the
                 empty-launch floor, hand-off primitive latencies
  roofline       the dominant kernel (draft decode attention): algorithmic
                 bytes per launch / mean launch duration from HIP events, its
                 fraction of 8 TB/s and of the streaming probe, and the
                 per-launch p10 / median / p90
  cpu_baseline   the fp64 oracle on the host cores (a bounded sample), with
                 the full-KV layer, both verify layers and a memory update
                 on all threads and on one
Inputs are synthetic N(0, 1) activations and N(0, 0.02^2) adaptor weights.
"""
import argparse
import hashlib
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

METRIC = "draft-step attn latency (µs/layer) + achieved HBM TB/s at 32K prefix, 1 GPU"
PEAK_HBM = 8.0e12          # B/s, MI355X HBM3E
PEAK_BF16 = 2.5e15         # dense MFMA bf16 FLOP/s
GAMMA, ROLLBACK = 4, 16


def log(msg):
    print(f"[bench] {msg}", file=sys.stderr, flush=True)


def parse():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=64)
    ap.add_argument("--warmup", type=int, default=8)
    ap.add_argument("--sets", type=int, default=6, help="sequences decoded round-robin (cold HBM reads)")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--cpu-seconds", type=float, default=8.0)
    ap.add_argument("--summarize-trace", metavar="CSV",
                    help="print per-(kernel, grid) durations of a rocprofv3 kernel_trace.csv and exit")
    ap.add_argument("--pmc-workload", choices=("decode", "copy", "update", "verify", "prefill"),
                    help="run only a counter workload (under rocprofv3 --pmc): 'decode' = the headline's "
                         "compact-memory decode launches, 'copy' = a streaming copy of known size, "
                         "'update' / 'verify' / 'prefill' = the matrix-core kernels at the benchmark's shapes")
    ap.add_argument("--summarize-counters", metavar="CSV",
                    help="print per-(kernel, grid) mean counter values of a rocprofv3 counter_collection.csv")
    return ap.parse_args()


COPY_FLOATS = 64 << 20   # the calibration copy: 256 MiB read + 256 MiB written


def pmc_workload(kind):
    """Kernels whose hardware counters calibrate or measure HBM traffic."""
    import torch
    import paper_2608_30252_amd as mad
    if kind == "copy":
        src = torch.ones(COPY_FLOATS, dtype=torch.float32, device="cuda")
        dst = torch.empty_like(src)
        torch.cuda.synchronize()
        for _ in range(4):
            torch.mul(src, 1.0, out=dst)   # one elementwise kernel: 4 B read + 4 B written per element
        torch.cuda.synchronize()
        print(f"copy: 4 launches of {COPY_FLOATS * 4} B read + {COPY_FLOATS * 4} B written", flush=True)
        return
    if kind in ("update", "verify", "prefill"):
        mfma_workload(torch, mad, kind)
        return
    model = DraftModel(torch, mad, 6)
    n = 0
    for k in range(4):
        for i in range(model.n_sets):
            view = model.lay.decode_view(model.prefix + k)
            for l in range(model.layers):
                mad.draft_decode_attn(model.q[l], mad.KV(model.mem_k[i][l], model.mem_v[i][l], [view.mem_len]),
                                      mad.KV(model.ring_k[i][l], model.ring_v[i][l], [view.win_len],
                                             [view.win_start]),
                                      model.kn[l], model.vn[l], model.out[l], model.lse[l], ws=model.ws)
                n += 1
    torch.cuda.synchronize()
    print(f"decode: {n} compact-memory launches, {kv_bytes(3073, model.Hkv, model.d)} B of K/V each", flush=True)


def mfma_workload(torch, mad, kind):
    """Launches of the matrix-core kernels at the benchmark's shapes, for the
    MFMA counters: the memory update of 64 rows (16 sequences x 4 slots) and of
    4 rows; verify at the 8B-layer (B4, 32/8) and 70B-layer (B1, 64/8) shapes;
    the memory prefill over a 32K prefix at d 64 and d 128."""
    bf = torch.bfloat16
    rn = lambda *s_: torch.randn(*s_, device="cuda").to(bf)
    if kind == "update":
        Hkv, d, D = 8, 64, 2048
        for B, n_new in ((16, 4), (1, 4)):
            x, w = rn(B, n_new, D), (torch.randn(2 * Hkv * d, D, device="cuda") * 0.02).to(bf)
            mk, mv = rn(B, Hkv, 1088, d), rn(B, Hkv, 1088, d)
            pos = [[16 * (2048 + 4 * b + i) for i in range(n_new)] for b in range(B)]
            for _ in range(8):
                mad.memory_update(x, w, pos, mad.KV(mk, mv, [1024] * B))
            torch.cuda.synchronize()
            print(f"update: 8 launches of {B * n_new} rows, {2 * B * n_new * D * 2 * Hkv * d} flop each", flush=True)
    elif kind == "verify":
        Hkv, d, T = 8, 128, 5
        L = 32768 + T
        for B, Hq in ((4, 32), (1, 64)):
            k, v = rn(B, Hkv, 32776, d), rn(B, Hkv, 32776, d)
            q = rn(B, T, Hq, d)
            out, lse = torch.empty_like(q), torch.empty(B, T, Hq, device="cuda")
            ws = torch.zeros(mad.workspace_bytes(mad.MAD_OP_VERIFY, B, Hq, Hkv, d, T), dtype=torch.uint8,
                             device="cuda")
            for _ in range(4):
                mad.verify_attn(q, mad.KV(k, v, [L] * B), out, lse, ws=ws)
            torch.cuda.synchronize()
            print(f"verify: 4 launches, B{B} {Hq}/{Hkv}, {4 * B * Hq * T * L * d} flop each", flush=True)
    else:
        P, S_, W_, r_, u_ = 32768, 0, 1024, 16, 4
        M = mad.slots_after(P, S_, r_, u_)
        for Hq, Hkv, d in ((32, 8, 64), (32, 8, 128)):
            qr, qs_ = rn(1, P, Hq, d), rn(1, M, Hq, d)
            rk, rv = rn(1, Hkv, P, d), rn(1, Hkv, P, d)
            mk, mv = rn(1, Hkv, S_ + M, d), rn(1, Hkv, S_ + M, d)
            for _ in range(2):
                mad.memory_prefill_attn(qr, qs_, mad.KV(mk, mv, [S_ + M]), mad.KV(rk, rv, [P]), [P], S_, W_, r_, u_)
            torch.cuda.synchronize()
            print(f"prefill: 2 launches, d{d}, {prefill_flops(P, S_, W_, r_, u_, Hq, d)} flop each", flush=True)


def summarize_counters(path):
    """Mean value per dispatch of each counter in a rocprofv3 --pmc counter_collection.csv,
    grouped by the library's kernel (or any kernel for the copy) and grid."""
    import csv
    groups = {}
    with open(path, newline="") as f:
        for row in csv.DictReader(f):
            name = row["Kernel_Name"].replace("void ", "").split("(")[0]
            grid = row.get("Grid_Size") or row.get("Grid_Size_X") or "?"
            key = (name[:60], grid, row["Counter_Name"])
            groups.setdefault(key, []).append(float(row["Counter_Value"]))
    for (name, grid, ctr), v in sorted(groups.items()):
        print(f"{name:60s} grid {grid:>8s} {ctr:12s} n {len(v):4d} mean {sum(v) / len(v):14.1f}")


def summarize_trace(path):
    """Durations of the library's kernels in a rocprofv3 --kernel-trace CSV,
    grouped by kernel and launch shape (grid and workgroup size)."""
    import csv
    import statistics
    groups = {}
    with open(path, newline="") as f:
        for row in csv.DictReader(f):
            name = row["Kernel_Name"]
            if "mad::" not in name:
                continue
            short = name.split("(")[0].replace("void ", "")
            # workgroups over all three grid dimensions (the sizes are in work-items)
            ext = [(int(row.get(f"Grid_Size_{a}") or 1), int(row.get(f"Workgroup_Size_{a}") or 1)) for a in "XYZ"]
            dims = tuple(g // w for g, w in ext)
            wgs, wg = dims[0] * dims[1] * dims[2], ext[0][1] * ext[1][1] * ext[2][1]
            key = (short, wgs, "x".join(str(n) for n in dims), wg)
            groups.setdefault(key, []).append((int(row["End_Timestamp"]) - int(row["Start_Timestamp"])) / 1e3)
    print(f"{'kernel':48s} {'grid':>8s} {'shape':>10s} {'wg':>5s} {'calls':>6s} {'mean_us':>8s} {'p10':>8s} {'median':>8s} "
          f"{'p90':>8s}")
    for (short, wgs, shape, wg), d in sorted(groups.items()):
        d.sort()
        print(f"{short:48s} {wgs:8d} {shape:>10s} {wg:5d} {len(d):6d} {sum(d) / len(d):8.2f} {d[len(d) // 10]:8.2f} "
              f"{statistics.median(d):8.2f} {d[9 * len(d) // 10]:8.2f}")


def kv_bytes(keys, hkv, d, esz=2):
    return keys * hkv * d * 2 * esz


class FullKVLayout:
    """The uncompressed draft: raw position x at row x, all earlier tokens attended."""

    def __init__(self, ring_cap):
        self.ring_cap = ring_cap

    def decode_view(self, p):
        from paper_2608_30252_amd.state import DecodeView
        if p + 1 > self.ring_cap:
            raise ValueError("full-KV capacity exceeded")
        return DecodeView(0, 0, p)


class DraftModel:
    """Buffers and host bookkeeping of the 16-layer compact draft memory for
    `n_sets` independent batch-1 sequences at a 32K prefix."""

    def __init__(self, torch, mad, n_sets, layers=16, Hq=32, Hkv=8, d=64, W=1024, r=16, u=4,
                 prefix=32768, full_kv=False, dev="cuda"):
        from paper_2608_30252_amd.state import MemoryLayout
        self.torch, self.mad = torch, mad
        self.layers, self.Hq, self.Hkv, self.d = layers, Hq, Hkv, d
        self.D = Hq * d
        self.full_kv = full_kv
        self.n_sets = n_sets
        self.prefix = prefix
        ring_extra = r * u + GAMMA + ROLLBACK
        if full_kv:
            # the uncompressed draft: no memory, every earlier token in the window
            self.lay = FullKVLayout(ring_cap=prefix + 256)
        else:
            ring_cap = (W + ring_extra + 7) // 8 * 8
            n_mem = (prefix // (r * u)) * u
            self.lay = MemoryLayout(0, W, r, ring_cap=ring_cap, mem_cap=n_mem + 64, slots_per_update=u)
        bf = torch.bfloat16
        L = layers
        mk = lambda *s: torch.randn(*s, device=dev, dtype=torch.float32).to(bf)
        if not full_kv:
            self.mem_k = [[mk(1, Hkv, self.lay.mem_cap, d) for _ in range(L)] for _ in range(n_sets)]
            self.mem_v = [[mk(1, Hkv, self.lay.mem_cap, d) for _ in range(L)] for _ in range(n_sets)]
        self.ring_k = [[mk(1, Hkv, self.lay.ring_cap, d) for _ in range(L)] for _ in range(n_sets)]
        self.ring_v = [[mk(1, Hkv, self.lay.ring_cap, d) for _ in range(L)] for _ in range(n_sets)]
        self.q = [mk(1, Hq, d) for _ in range(L)]
        self.kn = [mk(1, Hkv, d) for _ in range(L)]
        self.vn = [mk(1, Hkv, d) for _ in range(L)]
        self.out = [torch.empty(1, Hq, d, device=dev, dtype=bf) for _ in range(L)]
        self.lse = [torch.empty(1, Hq, device=dev, dtype=torch.float32) for _ in range(L)]
        if not full_kv:
            self.u = u
            self.x = [mk(1, u, self.D) for _ in range(L)]
            self.w_g = [(torch.randn(2 * Hkv * d, self.D, device=dev) * 0.02).to(bf) for _ in range(L)]
            # boundary steps: one launch for the raw query (row 0) and the u new
            # slots' write scopes (rows 1..u), all rows aliasing the sequence
            self.qf = [mk(1 + u, Hq, d) for _ in range(L)]
            self.knf = [self.kn[l].expand(1 + u, Hkv, d).contiguous() for l in range(L)]
            self.vnf = [self.vn[l].expand(1 + u, Hkv, d).contiguous() for l in range(L)]
            self.outf = [torch.empty(1 + u, Hq, d, device=dev, dtype=bf) for _ in range(L)]
            self.lsef = [torch.empty(1 + u, Hq, device=dev, dtype=torch.float32) for _ in range(L)]
        self.ws = torch.zeros(mad.workspace_bytes(mad.MAD_OP_DECODE, 1 + u if not full_kv else 1, Hq, Hkv, d),
                              dtype=torch.uint8, device=dev)
        self.decode_calls = []   # keys the raw query attends, per layer-step (slot-scope rows not counted)
        self.n_updates = 0

    def step(self, set_idx, p):
        """One draft step of sequence `set_idx` at raw position p through all layers.
        A step whose pass materialises memory slots runs, per layer, the memory
        update and then one launch for the raw query and the slots' write scopes."""
        mad, lay = self.mad, self.lay
        view = lay.decode_view(p)
        upd = None if self.full_kv else lay.update_in_pass_of(p)
        fused = None if upd is None else lay.step_views(p)
        for l in range(self.layers):
            rk, rv = self.ring_k[set_idx][l], self.ring_v[set_idx][l]
            if upd is None:
                mem = None if self.full_kv else mad.KV(self.mem_k[set_idx][l], self.mem_v[set_idx][l],
                                                       [view.mem_len])
                mad.draft_decode_attn(self.q[l], mem, mad.KV(rk, rv, [view.win_len], [view.win_start]),
                                      self.kn[l], self.vn[l], self.out[l], self.lse[l], ws=self.ws)
                self.decode_calls.append(view.mem_len + view.win_len + 1)
                continue
            mk, mv = self.mem_k[set_idx][l], self.mem_v[set_idx][l]
            mad.memory_update(self.x[l], self.w_g[l], [upd.positions], mad.KV(mk, mv, [upd.mem_row]))
            views, modes = fused
            mad.draft_step_attn(self.qf[l], mad.KV(mk, mv, [v.mem_len for v in views]),
                                mad.KV(rk, rv, [v.win_len for v in views], [v.win_start for v in views]),
                                self.knf[l], self.vnf[l], modes, self.outf[l], self.lsef[l], ws=self.ws)
            self.decode_calls.append(view.mem_len + view.win_len + 1)
        if upd is not None:
            self.n_updates += 1


def graph_of(torch, fn):
    """Capture fn() into a HIP graph on a side stream; return the graph."""
    s = torch.cuda.Stream()
    s.wait_stream(torch.cuda.current_stream())
    g = torch.cuda.CUDAGraph()
    with torch.cuda.stream(s):
        with torch.cuda.graph(g, stream=s):
            fn()
    torch.cuda.current_stream().wait_stream(s)
    torch.cuda.synchronize()
    return g


def time_graph(torch, g, reps=1):
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    e0.record()
    for _ in range(reps):
        g.replay()
    e1.record()
    torch.cuda.synchronize()
    return e0.elapsed_time(e1) * 1e-3 / reps   # seconds per replay


def time_cycled(torch, fns, launches=64, reps=5):
    """Median device time per launch of `launches` calls cycling through fns
    (one call per rotated buffer set), captured in one graph so that the
    graph's own launch cost is spread over many kernels, as in a decode loop."""
    g = graph_of(torch, lambda: [fns[i % len(fns)]() for i in range(launches)])
    g.replay()
    ts = sorted(time_graph(torch, g) for _ in range(reps))
    return ts[len(ts) // 2] / launches


def mean_launch_seconds(torch, launches, reps=3):
    """Mean device time per launch: the launches are captured in one HIP graph
    and replayed back to back between two HIP events on the replaying stream.
    The figure includes the graph's gaps between kernels, so it bounds the
    profiler's per-kernel duration from above."""
    g = graph_of(torch, lambda: [fn() for fn in launches])
    g.replay()
    return time_graph(torch, g, reps=reps) / len(launches)


def source_digest(*names):
    h = hashlib.sha256()
    for n in names:
        with open(os.path.join(ROOT, "paper_2608_30252_amd", "csrc", n), "rb") as f:
            h.update(f.read())
    return h.hexdigest()


DECODE_SOURCES = ("decode.hip", "mad_device.h", "mad_internal.h")   # what the decode kernel is built from


def traffic_from_profile(sources, bytes_default=None):
    """HBM bytes per launch from the committed counter summary, if it was
    taken on the current kernel sources; else None."""
    path = os.path.join(ROOT, "profiles", "decode_32k_compressed_traffic.json")
    if not os.path.exists(path):
        return None
    with open(path) as f:
        t = json.load(f)
    if t.get("source_sha256") != source_digest(*sources):
        return None
    return t.get("traffic_bytes_per_launch")


def trace_percentiles(sources, kernel="mad::decode_kernel<mad::bf16_t, 64, 4, 1>", grid=192):
    """The headline kernel's row of the committed rocprofv3 trace summary
    (per-kernel start/end timestamps, no inter-kernel gaps), if that trace was
    taken on the current kernel sources; else None."""
    path = os.path.join(ROOT, "profiles", "bench_kernel_trace.md")
    if not os.path.exists(path):
        return None
    text = open(path).read()
    if f"source_sha256: {source_digest(*sources)}" not in text:
        return None
    for line in text.splitlines():
        if not line.startswith(kernel):
            continue
        f = line[len(kernel):].split()   # grid, shape, wg, calls, mean, p10, median, p90
        if len(f) == 8 and int(f[0]) == grid:
            return {"calls": int(f[3]), "mean_us": float(f[4]), "p10_us": float(f[5]), "median_us": float(f[6]),
                    "p90_us": float(f[7]), "source": "profiles/bench_kernel_trace.md (rocprofv3 kernel trace)"}
    return None


def main():
    args = parse()
    if args.summarize_trace:
        summarize_trace(args.summarize_trace)
        return
    if args.summarize_counters:
        summarize_counters(args.summarize_counters)
        return
    if args.pmc_workload:
        pmc_workload(args.pmc_workload)
        return
    if args.gpus != 1:
        print(f"bench.py measures one GPU: the library has no multi-GPU path (asked for --gpus {args.gpus}).",
              file=sys.stderr)
        sys.exit(2)
    import torch
    import paper_2608_30252_amd as mad

    if not torch.cuda.is_available():
        print("bench.py needs a GPU", file=sys.stderr)
        sys.exit(3)
    torch.manual_seed(0)
    K, Wm = max(args.steps, 1), max(args.warmup, 0)
    n_sets = max(args.sets, 1)
    log(f"device {torch.cuda.get_device_name(0)}; {mad.version()}")

    # -------------------------------------------------------------- probes ----
    probes, stream_peak = device_probes(torch, mad)
    torch.cuda.empty_cache()

    # ------------------------------------------------------------ headline ----
    model = DraftModel(torch, mad, n_sets)
    # positions: every sequence starts at the 32K prefix; sequence 0 starts a few
    # tokens before a 64-token boundary so that one memory update falls in the
    # timed steps (one per 64 tokens of one sequence)
    uses_before = -(-(Wm + 1) // n_sets)
    pos = [model.prefix] * n_sets
    pos[0] = model.prefix + 64 - 1 - uses_before
    schedule = []
    for s in range(Wm + K):
        i = s % n_sets
        schedule.append((i, pos[i]))
        pos[i] += 1
    warm, timed = schedule[:Wm], schedule[Wm:]
    log(f"headline: {K} timed steps x {model.layers} layers, {n_sets} sequences round-robin")
    g_warm = graph_of(torch, lambda: [model.step(i, p) for i, p in warm]) if warm else None
    model.decode_calls.clear()
    model.n_updates = 0
    g_timed = graph_of(torch, lambda: [model.step(i, p) for i, p in timed])
    keys_per_call = list(model.decode_calls)
    n_updates = model.n_updates
    if g_warm is not None:
        g_warm.replay()
    torch.cuda.synchronize()
    t_step_total = time_graph(torch, g_timed)
    ms_per_step = t_step_total * 1e3 / K
    us_per_layer = ms_per_step * 1e3 / model.layers
    decode_bytes = [kv_bytes(k, model.Hkv, model.d) for k in keys_per_call]
    step_tbps = sum(decode_bytes) / t_step_total / 1e12
    log(f"headline: {ms_per_step:.4f} ms/step, {us_per_layer:.2f} us/layer, {n_updates} boundary step(s)")

    # dominant kernel: mean duration of the draft decode launches of the timed steps
    launches = []
    for i, p in timed[: min(len(timed), 8)]:
        view = model.lay.decode_view(p)
        for l in range(model.layers):
            def fn(i=i, l=l, view=view):
                mad.draft_decode_attn(model.q[l], mad.KV(model.mem_k[i][l], model.mem_v[i][l], [view.mem_len]),
                                      mad.KV(model.ring_k[i][l], model.ring_v[i][l], [view.win_len],
                                             [view.win_start]),
                                      model.kn[l], model.vn[l], model.out[l], model.lse[l], ws=model.ws)
            launches.append((fn, view.mem_len + view.win_len + 1))
    t_launch = mean_launch_seconds(torch, [f for f, _ in launches])
    bytes_launch = sum(kv_bytes(k, model.Hkv, model.d) for _, k in launches) / len(launches)
    achieved = bytes_launch / t_launch
    log(f"decode launch: {t_launch * 1e6:.2f} us mean over {len(launches)}, {bytes_launch:,.0f} B -> "
        f"{achieved / 1e12:.2f} TB/s")
    dist = launch_distribution(torch, mad, [f for f, _ in launches])
    log(f"decode launch distribution: {dist}")
    roofline = {"bound": "hbm", "achieved": round(achieved / 1e9, 1), "peak": PEAK_HBM / 1e9, "unit": "GB/s",
                "frac": round(achieved / PEAK_HBM, 4), "traffic": traffic_from_profile(DECODE_SOURCES),
                "kernel": "mad::decode_kernel<bf16_t, 64, 4, 1>", "bytes_per_launch": int(bytes_launch),
                "mean_launch_us": round(t_launch * 1e6, 3),
                "frac_of_stream_probe": round(achieved / stream_peak, 4),
                "stream_probe_gbps": round(stream_peak / 1e9, 1), "launch_distribution": dist,
                "trace_distribution": trace_percentiles(DECODE_SOURCES)}
    del model
    torch.cuda.empty_cache()

    # ------------------------------- one sequence: compact memory stays cached ----
    # The 16 layers' compact memory of one 32K sequence is ~100 MB, which fits the
    # 256 MB Infinity Cache: decoding a single sequence re-reads it from there,
    # not from HBM.  Reported beside the cold headline, labelled as such.
    one = DraftModel(torch, mad, 1)
    sched1 = [(0, one.prefix + s) for s in range(Wm + K)]
    g1_w = graph_of(torch, lambda: [one.step(i, p) for i, p in sched1[:Wm]]) if Wm else None
    g1 = graph_of(torch, lambda: [one.step(i, p) for i, p in sched1[Wm:]])
    if g1_w is not None:
        g1_w.replay()
    t1 = time_graph(torch, g1)
    one_launch = []
    for i, p in sched1[Wm:Wm + 4]:
        view = one.lay.decode_view(p)
        for l in range(one.layers):
            one_launch.append(lambda l=l, view=view: mad.draft_decode_attn(
                one.q[l], mad.KV(one.mem_k[0][l], one.mem_v[0][l], [view.mem_len]),
                mad.KV(one.ring_k[0][l], one.ring_v[0][l], [view.win_len], [view.win_start]),
                one.kn[l], one.vn[l], one.out[l], one.lse[l], ws=one.ws))
    t1_launch = mean_launch_seconds(torch, one_launch)
    cache_resident = {"workload": "the headline step on one sequence (its 16 layers' compact memory, ~100 MB, "
                                  "stays in the 256 MB Infinity Cache between steps): not an HBM figure",
                      "us_per_layer": round(t1 * 1e6 / (K * one.layers), 3),
                      "mean_launch_us": round(t1_launch * 1e6, 3),
                      "effective_tbps": round(bytes_launch / t1_launch / 1e12, 3), "steps": K}
    log(f"cache-resident: {t1 * 1e6 / (K * one.layers):.2f} us/layer, launch {t1_launch * 1e6:.2f} us")
    del one, g1, g1_w
    torch.cuda.empty_cache()

    # ------------------------------------------------------- full-KV draft ----
    K2 = min(K, 16)
    full = DraftModel(torch, mad, 1, full_kv=True)
    sched = [(0, full.prefix + s) for s in range(K2 + 2)]
    g_full_w = graph_of(torch, lambda: [full.step(i, p) for i, p in sched[:2]])
    full.decode_calls.clear()
    g_full = graph_of(torch, lambda: [full.step(i, p) for i, p in sched[2:]])
    g_full_w.replay()
    t_full = time_graph(torch, g_full)
    full_bytes = sum(kv_bytes(k, full.Hkv, full.d) for k in full.decode_calls)
    full_us_layer = t_full * 1e6 / (K2 * full.layers)
    f_launch = []
    for i, p in sched[2:4]:
        view = full.lay.decode_view(p)
        for l in range(full.layers):
            f_launch.append(lambda l=l, view=view: mad.draft_decode_attn(
                full.q[l], None, mad.KV(full.ring_k[0][l], full.ring_v[0][l], [view.win_len], [view.win_start]),
                full.kn[l], full.vn[l], full.out[l], full.lse[l], ws=full.ws))
    t_full_launch = mean_launch_seconds(torch, f_launch)
    full_launch_bytes = kv_bytes(full.prefix + 1, full.Hkv, full.d)
    full_kv = {"workload": "draft decode over the full 32768-token KV: B1, 16 layers, 32/8 heads, d64, bf16",
               "us_per_layer": round(full_us_layer, 3), "ms_per_step": round(t_full * 1e3 / K2, 4),
               "tbps": round(full_bytes / t_full / 1e12, 3),
               "mean_launch_us": round(t_full_launch * 1e6, 3),
               "launch_frac_of_hbm_peak": round(full_launch_bytes / t_full_launch / PEAK_HBM, 4),
               "bytes_per_launch": full_launch_bytes, "steps": K2}
    log(f"full KV: {full_us_layer:.2f} us/layer, launch {t_full_launch * 1e6:.2f} us "
        f"({full_launch_bytes / t_full_launch / 1e12:.2f} TB/s)")
    del full
    torch.cuda.empty_cache()

    # ------------------------------------- batched draft decode (16 sequences) ----
    # 16 sequences, 1024 slots + 511 window tokens + the new token each (50 MB per
    # launch), the same kernel with enough work per launch to leave the latency floor
    Bb, Lb, setsb = 16, 16, 4
    mkb = [torch.randn(Bb, 8, 1024, 64, device="cuda").to(torch.bfloat16) for _ in range(setsb * 2)]
    rkb = [torch.randn(Bb, 8, 576, 64, device="cuda").to(torch.bfloat16) for _ in range(setsb * 2)]
    qb = torch.randn(Bb, 32, 64, device="cuda").to(torch.bfloat16)
    knb = torch.randn(Bb, 8, 64, device="cuda").to(torch.bfloat16)
    vnb = torch.randn_like(knb)
    ob = torch.empty_like(qb)
    lb = torch.empty(Bb, 32, device="cuda")
    wsb = torch.zeros(mad.workspace_bytes(mad.MAD_OP_DECODE, Bb, 32, 8, 64), dtype=torch.uint8, device="cuda")
    starts = [(37 * i) % 64 for i in range(Bb)]
    fns = [lambda j=j: mad.draft_decode_attn(qb, mad.KV(mkb[2 * j], mkb[2 * j + 1], [1024] * Bb),
                                             mad.KV(rkb[2 * j], rkb[2 * j + 1], [511] * Bb, starts), knb, vnb, ob,
                                             lb, ws=wsb) for j in range(setsb)]
    g = graph_of(torch, lambda: [fns[i % setsb]() for i in range(Lb)])
    g.replay()
    t = time_graph(torch, g, reps=3) / Lb
    nb = kv_bytes(1024 + 511 + 1, 8, 64) * Bb
    batched = {"workload": "B16, 32/8 heads, d64, 1024 slots + 512-token window per sequence, bf16",
               "us_per_launch": round(t * 1e6, 2), "bytes_per_launch": nb, "tbps": round(nb / t / 1e12, 3),
               "hbm_frac": round(nb / t / PEAK_HBM, 4)}
    log(f"batched decode B16: {t * 1e6:.2f} us/launch, {nb / t / 1e12:.2f} TB/s")
    del mkb, rkb, fns, g
    torch.cuda.empty_cache()

    # ------------------------------------------- 8K-prefix draft, and C4 loop ----
    c2 = c2_leg(torch, mad)
    c4 = c4_loop(torch, mad)

    # ------------------------------------------------------- memory update ----
    upd_res = {}
    for name, B, n_new, sets in (("32k_4_rows", 1, 4, 8), ("batched_64_rows", 16, 4, 8)):
        Hkv, d, D = 8, 64, 2048
        xs = [torch.randn(B, n_new, D, device="cuda").to(torch.bfloat16) for _ in range(sets)]
        ws_ = [(torch.randn(2 * Hkv * d, D, device="cuda") * 0.02).to(torch.bfloat16) for _ in range(sets)]
        mks = [torch.randn(B, Hkv, 1088, d, device="cuda").to(torch.bfloat16) for _ in range(sets)]
        mvs = [torch.randn(B, Hkv, 1088, d, device="cuda").to(torch.bfloat16) for _ in range(sets)]
        posl = [[16 * (2048 + 4 * b + i) for i in range(n_new)] for b in range(B)]
        fns = [lambda j=j: mad.memory_update(xs[j], ws_[j], posl, mad.KV(mks[j], mvs[j], [1024] * B))
               for j in range(sets)]
        t = time_cycled(torch, fns)
        nbytes = 2 * Hkv * d * D * 2 + B * n_new * D * 2 + B * n_new * 2 * Hkv * d * 2
        flops = 2.0 * B * n_new * D * 2 * Hkv * d
        upd_res[name] = {"rows": B * n_new, "us": round(t * 1e6, 3), "tbps": round(nbytes / t / 1e12, 3),
                         "hbm_frac": round(nbytes / t / PEAK_HBM, 4), "tflops": round(flops / t / 1e12, 3),
                         "mfma_frac_of_bf16_peak": round(flops / t / PEAK_BF16, 6), "bytes": nbytes}
        log(f"memory update {name}: {t * 1e6:.2f} us, {nbytes / t / 1e12:.3f} TB/s")
        del xs, ws_, mks, mvs, fns
    torch.cuda.empty_cache()

    # -------------------------------------------------------------- verify ----
    # the verifier's cache in its natural layout (rows of d, mad_verify_attn), and
    # the same kernels over a transposed V cache (mad_verify_attn_vt)
    ver_res = {}
    for name, B, Hq, sets in (("8b_layer_b4", 4, 32, 1), ("70b_layer_b1", 1, 64, 3)):
        Hkv, d, T, cap = 8, 128, 5, 32776
        L = 32768 + T
        ks = [torch.randn(B, Hkv, cap, d, device="cuda").to(torch.bfloat16) for _ in range(sets)]
        vs = [torch.randn(B, Hkv, cap, d, device="cuda").to(torch.bfloat16) for _ in range(sets)]
        qv = torch.randn(B, T, Hq, d, device="cuda").to(torch.bfloat16)
        ov = torch.empty_like(qv)
        lv = torch.empty(B, T, Hq, device="cuda")
        wsv = torch.zeros(mad.workspace_bytes(mad.MAD_OP_VERIFY, B, Hq, Hkv, d, T), dtype=torch.uint8,
                          device="cuda")
        reps = max(3, 6 // sets) * sets
        nbytes = kv_bytes(L, Hkv, d) * B
        flops = 4.0 * B * Hq * T * L * d
        res = {}
        for layout in ("natural", "transposed_v"):
            if layout == "natural":
                fns = [lambda j=j: mad.verify_attn(qv, mad.KV(ks[j % sets], vs[j % sets], [L] * B), ov, lv, ws=wsv)
                       for j in range(reps)]
            else:
                vts = [v_.transpose(2, 3).contiguous() for v_ in vs]
                fns = [lambda j=j: mad.verify_attn_vt(qv, ks[j % sets], vts[j % sets], [L] * B, ov, lv, ws=wsv)
                       for j in range(reps)]
            t = time_cycled(torch, fns, launches=24)
            res[layout] = {"us": round(t * 1e6, 2), "tbps": round(nbytes / t / 1e12, 3),
                           "hbm_frac": round(nbytes / t / PEAK_HBM, 4), "mfma_tflops": round(flops / t / 1e12, 2)}
            log(f"verify {name} ({layout} V): {t * 1e6:.2f} us, {nbytes / t / 1e12:.3f} TB/s")
            del fns
        ver_res[name] = dict(res["natural"], bytes=nbytes, transposed_v=res["transposed_v"])
        del ks, vs, vts
    torch.cuda.empty_cache()

    # -------------------------------------------------------------- accept ----
    acc_res = {}
    for name, B in (("8b_b4", 4), ("70b_b1", 1)):
        T, V = 5, 128256
        lg = [torch.randn(B, T, V, device="cuda") for _ in range(4)]
        dr = torch.randint(0, V, (B, T - 1), device="cuda", dtype=torch.int32)
        na = torch.empty(B, dtype=torch.int32, device="cuda")
        nx = torch.empty(B, dtype=torch.int32, device="cuda")
        wsa = torch.zeros(mad.workspace_bytes(mad.MAD_OP_ACCEPT, B, 1, 1, 64, T, V), dtype=torch.uint8,
                          device="cuda")
        fns = [lambda j=j: mad.accept_greedy(lg[j], dr, na, nx, ws=wsa) for j in range(4)]
        t = time_cycled(torch, fns)
        nbytes = B * T * V * 4
        acc_res[name] = {"us": round(t * 1e6, 2), "tbps": round(nbytes / t / 1e12, 3), "bytes": nbytes}
        log(f"accept {name}: {t * 1e6:.2f} us")
        del lg, fns
        # stochastic accept/reject with caller uniforms: reads the drafted tokens'
        # probabilities, then one target row (and one draft row) of the vocabulary
        ps = [torch.softmax(torch.randn(B, T, V, device="cuda"), -1) for _ in range(4)]
        qs = [torch.softmax(torch.randn(B, T - 1, V, device="cuda"), -1) for _ in range(4)]
        uu = torch.rand(B, T, device="cuda")
        wss = torch.zeros(mad.workspace_bytes(mad.MAD_OP_ACCEPT_STOCH, B, 1, 1, 64, T, V), dtype=torch.uint8,
                          device="cuda")
        fns = [lambda j=j: mad.accept_stochastic(ps[j], qs[j], dr, uu, na, nx, ws=wss) for j in range(4)]
        t = time_cycled(torch, fns)
        acc_res[name + "_stochastic"] = {"us": round(t * 1e6, 2), "bytes_max": B * 2 * V * 4}
        log(f"accept {name} stochastic: {t * 1e6:.2f} us")
        del ps, qs, fns

    # ------------------------------------------------ draft layer, end to end ----
    lay_res = draft_layer_bench(torch, mad, K)
    torch.cuda.empty_cache()

    # --------------------------------------------------------- prefix sweep ----
    sweep = prefix_sweep(torch, mad)

    # ------------------------------------------------------ memory prefill ----
    pre_res = {}
    P, S_, W_, r_, u_ = 32768, 0, 1024, 16, 4
    M = mad.slots_after(P, S_, r_, u_)
    for name, Hq, Hkv, d in (("32k_d64_32_8", 32, 8, 64), ("32k_d128_32_8", 32, 8, 128)):
        qr = torch.randn(1, P, Hq, d, device="cuda").to(torch.bfloat16)
        qs_ = torch.randn(1, M, Hq, d, device="cuda").to(torch.bfloat16)
        rk = torch.randn(1, Hkv, P, d, device="cuda").to(torch.bfloat16)
        rv = torch.randn(1, Hkv, P, d, device="cuda").to(torch.bfloat16)
        mk = torch.randn(1, Hkv, S_ + M, d, device="cuda").to(torch.bfloat16)
        mv = torch.randn(1, Hkv, S_ + M, d, device="cuda").to(torch.bfloat16)
        outs = mad.memory_prefill_attn(qr, qs_, mad.KV(mk, mv, [S_ + M]), mad.KV(rk, rv, [P]), [P], S_, W_, r_, u_)
        fn = lambda: mad.memory_prefill_attn(qr, qs_, mad.KV(mk, mv, [S_ + M]), mad.KV(rk, rv, [P]), [P],
                                             S_, W_, r_, u_, *outs)
        g = graph_of(torch, lambda: [fn() for _ in range(3)])
        # ~60-100 ms of the same work first: the first few replays after the
        # host-side setup run 10-25 % slower while the clocks come up
        for _ in range(20):
            g.replay()
        t = time_graph(torch, g, reps=5) / 3
        flops = prefill_flops(P, S_, W_, r_, u_, Hq, d)
        pre_res[name] = {"us": round(t * 1e6, 1), "tflops": round(flops / t / 1e12, 1),
                         "mfma_frac_of_bf16_peak": round(flops / t / PEAK_BF16, 4), "flops": flops,
                         "queries": P + M}
        log(f"memory prefill {name}: {t * 1e6:.1f} us, {flops / t / 1e12:.1f} TFLOP/s")
        del qr, qs_, rk, rv, mk, mv, outs, g
    torch.cuda.empty_cache()

    # --------------------------------------------------------- CPU baseline ----
    cpu = None
    if not args.no_cpu_baseline:
        cpu = cpu_baseline(args.cpu_seconds)
        log(f"cpu baseline: {cpu['value']:.1f} us/layer on {cpu['cores']} threads")

    result = {
        "metric": METRIC, "value": round(us_per_layer, 3), "unit": "us/layer", "n_gpus": 1, "steps": K,
        "warmup": Wm, "ms_per_step": round(ms_per_step, 5), "higher_is_better": False, "scaling": "weak",
        "vs_baseline": None, "dtype": "bf16", "data": "synthetic",
        "config": {"workload": "draft decode at a 32K prefix: batch 1, 16 layers, 32 query / 8 KV heads, "
                               "head_dim 64, 2048 memory slots + 1024-token window, bf16",
                   "batch": 1, "prefix": 32768, "layers": 16, "memory_slots": 2048, "window": 1024,
                   "slot_interval": 16, "slots_per_update": 4, "sequences_round_robin": n_sets,
                   "parallelism": "none"},
        "step_tbps": round(step_tbps, 3),
        "tokens_per_s": round(1.0 / (ms_per_step * 1e-3), 1),
        "boundary_steps_timed": n_updates,
        "roofline": roofline,
        "full_kv": full_kv,
        "cache_resident": cache_resident,
        "speedup_vs_full_kv": round(full_us_layer / us_per_layer, 3),
        "batched_decode": batched,
        "draft_8k": c2,
        "batched_drafting": c4,
        "probes": probes,
        "prefix_sweep": sweep,
        "memory_update": upd_res,
        "verify": ver_res,
        "accept": acc_res,
        "memory_prefill": pre_res,
        "draft_layer": lay_res,
        "cpu_baseline": cpu,
    }
    print(json.dumps(result), flush=True)


def draft_layer_bench(torch, mad, K):
    """Whole draft steps through 16 random-init decoder layers of the 32K draft
    (D 2048, 32/8 heads, d 64, SwiGLU FFN 8192: the attention shapes of the
    headline): RMSNorm + Q/K/V + RoPE, attention, output projection, RMSNorm +
    SwiGLU, down projection, per layer, with the compact memory and with the
    full 32768-token KV.  The layers' 1.9 GB of weights are streamed from HBM
    every step.  A step crossing a 64-token boundary carries four slot rows
    through every layer (memory update + fused attention)."""
    from paper_2608_30252_amd.layer import DraftLayer, LayerWeights
    L, D, Hq, Hkv, d, F = 16, 2048, 32, 8, 64, 8192
    dev = torch.device("cuda")
    bf = torch.bfloat16

    def rnd(*shape, std=0.02):
        return (torch.randn(*shape, device=dev) * std).to(bf)
    layers = []
    for _ in range(L):
        w = LayerWeights(gamma1=(1 + rnd(D, std=0.1).float()).to(bf), w_qkv=rnd((Hq + 2 * Hkv) * d, D),
                         w_kv_g=rnd(2 * Hkv * d, D), w_o=rnd(D, Hq * d), gamma2=(1 + rnd(D, std=0.1).float()).to(bf),
                         w_gate_up=rnd(2 * F, D), w_down=rnd(D, F))
        layers.append(DraftLayer(w, D, Hq, Hkv, d, F, device=dev))
    wbytes = layers[0].w.weight_bytes()
    out = {"workload": "16 random-init layers, D 2048, 32/8 heads, d 64, FFN 8192, bf16, batch 1, 32K prefix",
           "weight_bytes_per_layer": wbytes}
    emb = rnd(5, D, std=1.0)   # row 0: the raw token entering layer 0; rows 1..4: slot tokens
    for name, full in (("compact", False), ("full_kv", True)):
        m = DraftModel(torch, mad, 1, layers=L, full_kv=full)
        ws = m.ws
        if full:
            start = m.prefix
        else:   # a few steps before a 64-token boundary, so one materialisation step is timed
            start = m.prefix + 64 - 3

        def step(p):
            upd = None if full else m.lay.update_in_pass_of(p)
            x = emb[:1] if upd is None else emb[:1 + len(upd.positions)]
            for l in range(L):
                x = layers[l].step(x, p, m.lay, None if full else m.mem_k[0][l], None if full else m.mem_v[0][l],
                                   m.ring_k[0][l], m.ring_v[0][l], ws=ws, full_kv=full)
        nsteps = min(K, 16)
        warm = graph_of(torch, lambda: step(start))
        g = graph_of(torch, lambda: [step(start + 1 + i) for i in range(nsteps)])
        warm.replay()
        t = time_graph(torch, g, reps=2) / nsteps
        out[name] = {"ms_per_step": round(t * 1e3, 4), "us_per_layer": round(t * 1e6 / L, 2),
                     "tokens_per_s": round(1.0 / t, 1), "steps": nsteps}
        log(f"draft layer {name}: {t * 1e6 / L:.2f} us/layer, {t * 1e3:.3f} ms per 16-layer step")
        del m, warm, g
        torch.cuda.empty_cache()
    # the weight stream alone: the four linear maps of one decode row per layer
    x1 = emb[:1]

    def maps():
        for lyr in layers:
            w = lyr.w
            mad.rmsnorm_qkv_rope(x1, w.gamma1, w.w_qkv, [40000], Hq, Hkv, d, lyr.q[:1], lyr.k[:1], lyr.v[:1])
            h = mad.linear_residual(lyr.o[:1].view(1, Hq * d), w.w_o, x1, out=lyr.h[:1])
            a = mad.rmsnorm_swiglu(h, w.gamma2, w.w_gate_up, out=lyr.a[:1])
            mad.linear_residual(a, w.w_down, h, out=lyr.y[:1])
    g = graph_of(torch, maps)
    g.replay()
    t = time_graph(torch, g, reps=4)
    out["linear_maps"] = {"us_per_layer": round(t * 1e6 / L, 2), "tbps": round(wbytes * L / t / 1e12, 3),
                          "hbm_frac": round(wbytes * L / t / PEAK_HBM, 4)}
    out["speedup_vs_full_kv"] = round(out["full_kv"]["us_per_layer"] / out["compact"]["us_per_layer"], 3)
    log(f"draft layer linear maps: {t * 1e6 / L:.2f} us/layer, {wbytes * L / t / 1e12:.2f} TB/s")
    return out


def decode_launch_cold(torch, mad, mem_len, win_len, Hq=32, Hkv=8, d=64, cold_bytes=640 << 20):
    """Mean duration of one batch-1 draft decode launch over mem_len memory rows,
    win_len ring rows and the new token, the launches rotating through enough
    independent buffers (>= 640 MB, over twice the L2 and Infinity Cache) that
    every launch reads its K/V from HBM.  Returns (seconds, algorithmic bytes)."""
    keys = mem_len + win_len + 1
    nbytes = kv_bytes(keys, Hkv, d)
    n = max(2, min(256, -(-cold_bytes // nbytes)))
    mcap, rcap = max(mem_len, 1), (win_len + 1 + 63) // 64 * 64
    bf = torch.bfloat16
    mem = torch.randn(n, 2, Hkv, mcap, d, device="cuda").to(bf) if mem_len else None
    ring = torch.randn(n, 2, Hkv, rcap, d, device="cuda").to(bf)
    q = torch.randn(1, Hq, d, device="cuda").to(bf)
    kn, vn = torch.randn(1, Hkv, d, device="cuda").to(bf), torch.randn(1, Hkv, d, device="cuda").to(bf)
    out, lse = torch.empty_like(q), torch.empty(1, Hq, device="cuda")
    ws = torch.zeros(mad.workspace_bytes(mad.MAD_OP_DECODE, 1, Hq, Hkv, d), dtype=torch.uint8, device="cuda")

    def launch(j):
        m = mad.KV(mem[j, 0:1], mem[j, 1:2], [mem_len]) if mem_len else None
        mad.draft_decode_attn(q, m, mad.KV(ring[j, 0:1], ring[j, 1:2], [win_len], [0]), kn, vn, out, lse, ws=ws)

    t = mean_launch_seconds(torch, [lambda j=j: launch(j) for j in range(n)])
    del mem, ring
    return t, nbytes


def prefix_sweep(torch, mad):
    """Draft decode latency against the prefix length L (8K..32K), compact memory
    beside the full KV, with the least-squares fit t = alpha + beta * L of the
    per-layer cost model (Eq. 2); and the paper's own memory shapes at 32K
    (S = 128 sinks, W = 128, slot interval r = 4 and 8)."""
    import numpy as np
    from paper_2608_30252_amd.state import MemoryLayout
    pts = []
    for P in (8192, 16384, 24576, 32768):
        lay = MemoryLayout(0, 1024, 16, ring_cap=1024 + 128, mem_cap=P // 16 + 64, slots_per_update=4)
        v = lay.decode_view(P)
        tc, bc = decode_launch_cold(torch, mad, v.mem_len, v.win_len)
        tf, bf_ = decode_launch_cold(torch, mad, 0, P)
        pts.append({"prefix": P, "compact_keys": v.mem_len + v.win_len + 1, "compact_us": round(tc * 1e6, 3),
                    "compact_tbps": round(bc / tc / 1e12, 3), "full_keys": P + 1, "full_us": round(tf * 1e6, 3),
                    "full_tbps": round(bf_ / tf / 1e12, 3), "speedup": round(tf / tc, 2)})
        log(f"prefix {P}: compact {tc * 1e6:.2f} us ({bc / tc / 1e12:.2f} TB/s), full {tf * 1e6:.2f} us "
            f"({bf_ / tf / 1e12:.2f} TB/s)")
    Ls = np.array([p["prefix"] for p in pts], dtype=np.float64)

    def fit(key):
        beta, alpha = np.polyfit(Ls, np.array([p[key] for p in pts]), 1)
        return {"alpha_us": round(float(alpha), 3), "beta_ns_per_token": round(float(beta) * 1e3, 4)}
    full_fit, compact_fit = fit("full_us"), fit("compact_us")
    # one token of the full KV costs 8 KV heads x 64 x 2 (K, V) x 2 B = 2048 B
    full_fit["beta_tbps"] = round(2048 / (full_fit["beta_ns_per_token"] * 1e-9) / 1e12, 3)
    paper = []
    for r in (4, 8):
        lay = MemoryLayout(128, 128, r, ring_cap=256, mem_cap=128 + 32768 // r, slots_per_update=4)
        v = lay.decode_view(32768)
        t, b = decode_launch_cold(torch, mad, v.mem_len, v.win_len)
        paper.append({"sinks": 128, "window": 128, "slot_interval": r, "keys": v.mem_len + v.win_len + 1,
                      "us": round(t * 1e6, 3), "tbps": round(b / t / 1e12, 3)})
        log(f"paper-shaped S = W = 128, r = {r}: {v.mem_len + v.win_len + 1} keys, {t * 1e6:.2f} us")
    torch.cuda.empty_cache()
    return {"workload": "batch-1 draft decode launch, 32/8 heads, d64, bf16, cold (buffers rotated over >= 640 MB); "
                        "compact = L/16 slots + 1024-token window, full = L + 1 keys",
            "points": pts, "full_fit": full_fit, "compact_fit": compact_fit, "paper_shaped_32k": paper}


def device_probes(torch, mad):
    """What the device itself delivers, measured in the same run: the read
    bandwidth of a plain streaming kernel over 256 MiB buffers rotated through
    1 GiB (cold: four times the Infinity Cache), the cost of an empty launch in a
    replayed graph, and the latency of the hand-off primitives (one thread)."""
    import numpy as np
    size, nbuf = 256 << 20, 4
    bufs = [torch.empty(size, dtype=torch.uint8, device="cuda") for _ in range(nbuf)]
    sink = torch.zeros(1, dtype=torch.int32, device="cuda")
    stream = {}
    for nwg in (1024, 2048):
        g = graph_of(torch, lambda: [mad.probe_stream_read(bufs[j % nbuf], sink, nwg) for j in range(8)])
        g.replay()
        t = time_graph(torch, g, reps=3) / 8
        stream[nwg] = size / t
        log(f"stream probe ({nwg} workgroups): {size / t / 1e12:.3f} TB/s")
    del bufs
    # one CU reading L2-resident data: 256 workgroups (one per CU) all read the
    # same 128 KB or 512 KB; the difference of the two launch times over the
    # difference of bytes is the per-CU rate, by waves per workgroup
    shr = torch.empty(512 << 10, dtype=torch.uint8, device="cuda")
    l2 = {}
    for threads in (256, 512, 1024):
        ts = {}
        for kb in (128, 512):
            src = shr[:kb << 10]
            ts[kb] = time_cycled(torch, [lambda s_=src, t_=threads: mad.probe_shared_read(s_, sink, 256, t_)])
        l2[str(threads // 64)] = {"us_128k": round(ts[128] * 1e6, 2), "us_512k": round(ts[512] * 1e6, 2),
                                  "cu_gbps": round((384 << 10) / (ts[512] - ts[128]) / 1e9, 1)}
    del shr
    log(f"L2-resident read per CU (by waves per workgroup): {l2}")
    g = graph_of(torch, lambda: [mad.probe_empty(256, 256) for _ in range(64)])
    g.replay()
    t_empty = time_graph(torch, g, reps=3) / 64
    reps = 64
    hb = torch.zeros(reps * 256 + 4096, dtype=torch.uint8, device="cuda")
    cyc = torch.zeros(8, reps, dtype=torch.int64, device="cuda")
    mad.probe_handoff_latency(hb, cyc, reps)
    torch.cuda.synchronize()
    c = cyc.cpu().numpy().astype(np.float64)
    ghz = (c[7, -1] - c[7, 1]) / ((c[6, -1] - c[6, 1]) * 10.0)
    names = ["plain_store_ack", "device_store_ack", "device_atomic", "device_load_written", "load_l2_hit",
             "load_miss"]
    lat = {n: round(float(np.median(c[k, 8:]) / ghz), 1) for k, n in enumerate(names)}
    log(f"empty launch {t_empty * 1e6:.2f} us; hand-off latencies (ns) {lat}")
    peak = max(stream.values())
    return {"stream_read_tbps": round(peak / 1e12, 3),
            "stream_read_by_workgroups": {str(k): round(v / 1e12, 3) for k, v in stream.items()},
            "stream_workload": "nontemporal 16-byte loads, 8 in flight per thread, 256 threads per workgroup, "
                               "256 MiB per launch over four buffers (1 GiB)",
            "l2_resident_read_per_cu": l2,
            "empty_launch_us": round(t_empty * 1e6, 3), "handoff_latency_ns": lat,
            "shader_clock_ghz": round(float(ghz), 3)}, peak


def launch_distribution(torch, mad, fns, n=256):
    """Per-launch device time from a pair of HIP events around each launch:
    p10 / median / p90 in us.  A streaming read of ~1 GiB per launch keeps the
    device busy while the host enqueues every (event, launch, event) triple, so
    the launches run back to back and each interval is the kernel plus the
    two event packets, not the host's submission time."""
    import numpy as np
    busy = torch.empty(1 << 30, dtype=torch.uint8, device="cuda")
    evs = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)) for _ in range(n)]
    for i in range(8):
        fns[i % len(fns)]()
    torch.cuda.synchronize()
    for _ in range(60):                    # ~12 ms of device work ahead of the timed launches
        mad.probe_stream_read(busy, None, 1024)
    for i in range(n):
        evs[i][0].record()
        fns[i % len(fns)]()
        evs[i][1].record()
    torch.cuda.synchronize()
    del busy
    t = np.array([a.elapsed_time(b) * 1e3 for a, b in evs])
    return {"p10_us": round(float(np.percentile(t, 10)), 3), "median_us": round(float(np.median(t)), 3),
            "p90_us": round(float(np.percentile(t, 90)), 3), "launches": n,
            "method": "HIP events around each launch, enqueued behind ~12 ms of device work (kernel + event packets)"}


def c2_leg(torch, mad, K=64):
    """The 8K-prefix draft: 16 layers, 512 slots + a 512-token window, every
    sequence decoding 64 steps (its memory update fires at the 64th, when its
    64-token block ends); ten sequences round-robin keep the reads in HBM
    (16 layers x 2 MB x 10 > 256 MB).  Beside it the same steps over the full
    8192-token KV."""
    n_sets = 10
    model = DraftModel(torch, mad, n_sets, prefix=8192, W=512)
    sched = [(i, model.prefix + s) for s in range(K) for i in range(n_sets)]
    g = graph_of(torch, lambda: [model.step(i, p) for i, p in sched])
    calls = list(model.decode_calls)
    n_upd = model.n_updates
    g.replay()
    t = time_graph(torch, g)
    steps = len(sched)
    us_layer = t * 1e6 / (steps * model.layers)
    nbytes = sum(kv_bytes(k, model.Hkv, model.d) for k in calls)
    del model, g
    torch.cuda.empty_cache()
    full = DraftModel(torch, mad, 2, prefix=8192, full_kv=True)
    fs = [(i, full.prefix + s) for s in range(16) for i in range(2)]
    gf = graph_of(torch, lambda: [full.step(i, p) for i, p in fs])
    fcalls = list(full.decode_calls)
    gf.replay()
    tf = time_graph(torch, gf)
    f_us = tf * 1e6 / (len(fs) * full.layers)
    fbytes = sum(kv_bytes(k, full.Hkv, full.d) for k in fcalls)
    del full, gf
    torch.cuda.empty_cache()
    log(f"8K draft: {us_layer:.2f} us/layer ({nbytes / t / 1e12:.2f} TB/s), {n_upd} updates; full KV "
        f"{f_us:.2f} us/layer")
    return {"workload": "draft decode at an 8K prefix: B1, 16 layers, 32/8 heads, d64, bf16, 512 slots + 512-token "
                        "window (1024 keys), 64 steps per sequence with the memory update at the 64th, 10 sequences "
                        "round-robin",
            "us_per_layer": round(us_layer, 3), "ms_per_step": round(t * 1e3 / steps, 4),
            "tbps": round(nbytes / t / 1e12, 3), "bytes_per_layer": kv_bytes(1024, 8, 64), "steps": steps,
            "updates": n_upd, "full_kv_us_per_layer": round(f_us, 3),
            "full_kv_tbps": round(fbytes / tf / 1e12, 3), "speedup_vs_full_kv": round(f_us / us_layer, 3)}


def c4_loop(torch, mad, layers=16, gamma=4, iters=128, seed=44):
    """Batched drafting with continuous memory updates: 16 sequences with
    prefixes drawn uniformly in [8192, 32768), 1024 memory slots and a 512-token
    window each, 32/8 heads, d 64, bf16, `layers` layers; gamma = 4 tokens per
    iteration for 128 iterations (512 tokens).  Per token and layer one decode
    launch for the 16 sequences; a sequence's update fires when its own 64-token
    block ends (slot interval 16, 4 slots per update), all firing sequences of a
    token in one update launch with per-sequence fire flags.  Whole run captured
    in one graph."""
    import numpy as np
    from paper_2608_30252_amd.state import MemoryLayout
    B, Hq, Hkv, d, W, r, u, base_slots = 16, 32, 8, 64, 512, 16, 4, 1024
    D = Hq * d
    N = gamma * iters
    rng = np.random.default_rng(seed)
    P = rng.integers(8192, 32768, B).tolist()
    ring_cap = (W + r * u + gamma + ROLLBACK + 7) // 8 * 8
    lays = [MemoryLayout(0, W, r, ring_cap=ring_cap, mem_cap=1 << 20, slots_per_update=u) for _ in range(B)]
    made0 = [lays[b].slots_materialised(P[b]) for b in range(B)]
    mem_cap = base_slots + (N // (r * u) + 2) * u
    bf = torch.bfloat16
    mk = lambda *sh: torch.randn(*sh, device="cuda").to(bf)
    mem_k = [mk(B, Hkv, mem_cap, d) for _ in range(layers)]
    mem_v = [mk(B, Hkv, mem_cap, d) for _ in range(layers)]
    ring_k = [mk(B, Hkv, ring_cap, d) for _ in range(layers)]
    ring_v = [mk(B, Hkv, ring_cap, d) for _ in range(layers)]
    q, kn, vn = mk(B, Hq, d), mk(B, Hkv, d), mk(B, Hkv, d)
    out, lse = torch.empty_like(q), torch.empty(B, Hq, device="cuda")
    x = mk(B, u, D)
    w_g = [(torch.randn(2 * Hkv * d, D, device="cuda") * 0.02).to(bf) for _ in range(layers)]
    ws = torch.zeros(mad.workspace_bytes(mad.MAD_OP_DECODE, B, Hq, Hkv, d), dtype=torch.uint8, device="cuda")
    keys, n_upd_launch, n_fired = [], 0, 0

    def run():
        nonlocal n_upd_launch, n_fired
        for t in range(N):
            pos = [P[b] + t for b in range(B)]
            views = [lays[b].decode_view(pos[b]) for b in range(B)]
            mlen = [base_slots + views[b].mem_len - made0[b] for b in range(B)]
            upds = [lays[b].update_in_pass_of(pos[b]) for b in range(B)]
            fire = [1 if x_ is not None else 0 for x_ in upds]
            for l in range(layers):
                mad.draft_decode_attn(q, mad.KV(mem_k[l], mem_v[l], mlen),
                                      mad.KV(ring_k[l], ring_v[l], [v.win_len for v in views],
                                             [v.win_start for v in views]), kn, vn, out, lse, ws=ws)
                keys.append(sum(mlen) + sum(v.win_len for v in views) + B)
                if any(fire):
                    posl = [x_.positions if x_ is not None else [0] * u for x_ in upds]
                    rows = [base_slots + x_.mem_row - made0[b] if x_ is not None else mlen[b]
                            for b, x_ in enumerate(upds)]
                    mad.memory_update(x, w_g[l], posl, mad.KV(mem_k[l], mem_v[l], rows), fire=fire)
                    n_upd_launch += 1
            n_fired += sum(fire)

    g = graph_of(torch, run)
    g.replay()
    t = time_graph(torch, g)
    nbytes = sum(kv_bytes(k, Hkv, d) for k in keys)
    del mem_k, mem_v, ring_k, ring_v, g
    torch.cuda.empty_cache()
    log(f"batched drafting B16: {t * 1e3 / iters:.3f} ms per gamma-{gamma} iteration, {nbytes / t / 1e12:.2f} TB/s, "
        f"{n_upd_launch} update launches")
    return {"workload": f"16 ragged sequences (prefixes U[8192, 32768), seed {seed}), 1024 slots + 512-token window, "
                        f"32/8 heads, d64, bf16, {layers} layers, gamma {gamma} x {iters} iterations ({N} tokens), "
                        "staggered memory updates (4 slots per 64-token block, per-sequence fire flags)",
            "ms_per_iteration": round(t * 1e3 / iters, 4), "us_per_token_layer": round(t * 1e6 / (N * layers), 3),
            "tokens_per_s": round(B * N / t, 1), "tbps_decode_bytes": round(nbytes / t / 1e12, 3),
            "update_launches": n_upd_launch // max(layers, 1), "slot_updates_per_layer": n_fired,
            "prefixes": P}


def prefill_flops(P, S, W, r, u, Hq, d):
    """Multiply-adds x 2 of both attention products over every query's visible
    keys in the memory-prefill pass: a raw token at p sees min(S, p+1) sinks,
    the slots materialised before it and its window; slot m sees S sinks, m
    slots and the W raw tokens before its position id."""
    import numpy as np
    p = np.arange(P, dtype=np.int64)
    seen_slots = np.where(p <= S, 0, (p - S) // (r * u) * u)
    window = np.where(p < S, 0, p - np.maximum(S, p - W + 1) + 1)
    raw = np.minimum(S, p + 1) + seen_slots + window
    M = 0 if P <= S else (P - S) // (r * u) * u
    m = np.arange(1, M + 1, dtype=np.int64)
    bm = S + m * r
    slot = S + m + (bm - np.maximum(S, bm - W))
    return int((raw.sum() + slot.sum()) * Hq * d * 4)


def _cpu_model():
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return "unknown"


def _time_calls(fn, seconds, min_calls=1, warm=True):
    """Mean wall time of fn() over about `seconds` (at least min_calls calls, after one warm call)."""
    if warm:
        fn()
    t0 = time.perf_counter()
    calls = 0
    while calls < min_calls or time.perf_counter() - t0 < seconds:
        fn()
        calls += 1
    return (time.perf_counter() - t0) / calls, calls


def cpu_baseline(seconds):
    """The fp64 oracle on the host, a bounded sample of the workloads.

    value: the 32K compact-memory layer attention (8 KV heads x 3072 keys x 4
    query heads, head_dim 64) on every host thread OpenMP uses, repeated for
    about `seconds`.  breadth: the same layer over the full 32769-token KV, the
    verify attention of both target layers (B4 32/8 heads and B1 64/8 heads,
    d 128, 32768 + 5 keys, 5 queries) and one memory update of 4 slot rows
    (D 2048 -> 8 KV heads x 64), each timed on all threads and on one thread
    (one or a few calls each; the verify layers dominate the few seconds)."""
    import numpy as np
    import oracle
    from paper_2608_30252_amd import synth
    Hq, Hkv, d, n = 32, 8, 64, 3072
    q = synth.normal((1, Hq, d), 1).double().numpy()
    k = synth.normal((1, Hkv, n, d), 2).double().numpy()
    v = synth.normal((1, Hkv, n, d), 3).double().numpy()
    nn = np.array([n])
    threads = oracle.num_threads()
    t, calls = _time_calls(lambda: oracle.attend_batched(q, k, v, nn, d ** -0.5), seconds)
    res = {"value": round(t * 1e6, 1), "unit": "us/layer", "cores": threads, "kind": "oracle",
           "cpu_model": _cpu_model(),
           "sample": f"{calls} calls of one 32K compact-memory layer attention (8 KV heads x 3072 keys x 4 "
                     f"query heads, d 64, fp64)"}
    # breadth: full KV, verify (both target layers), one memory update; all threads and one thread
    nf = 32769
    kf = synth.normal((1, Hkv, nf, d), 4).double().numpy()
    vf = synth.normal((1, Hkv, nf, d), 5).double().numpy()
    items = [("32k_full_kv_layer", lambda: oracle.attend_batched(q, kf, vf, np.array([nf]), d ** -0.5), 1.0)]
    T, L = 5, 32768 + 5
    for name, B, Hq_v in (("verify_8b_layer_b4", 4, 32), ("verify_70b_layer_b1", 1, 64)):
        qv = synth.normal((B, T, Hq_v, 128), 6).double().numpy()
        kv_ = synth.normal((B, 8, L, 128), 7).double().numpy()
        vv_ = synth.normal((B, 8, L, 128), 8).double().numpy()
        items.append((name, lambda qv=qv, kv_=kv_, vv_=vv_, B=B: oracle.verify(qv, kv_, vv_, np.array([L] * B),
                                                                               128 ** -0.5), 0.5))
    x = synth.normal((4, 2048), 9).double().numpy()
    w = synth.normal((2 * 8 * 64, 2048), 10, std=0.02).double().numpy()
    items.append(("memory_update_4_rows", lambda: oracle.memory_update(x, w, np.array([32768, 32784, 32800, 32816]),
                                                                       8, 64, 500000.0), 1.0))
    breadth = {}
    for name, fn, secs in items:
        heavy = name.startswith("verify")   # seconds per call: one call each, no warm call
        tm, cm = _time_calls(fn, secs, warm=not heavy)
        oracle.set_threads(1)
        t1, c1 = _time_calls(fn, secs / 4, warm=not heavy)
        oracle.set_threads(threads)
        breadth[name] = {"us_all_threads": round(tm * 1e6, 1), "us_one_thread": round(t1 * 1e6, 1),
                         "calls": [cm, c1]}
        log(f"cpu baseline {name}: {tm * 1e6:.0f} us on {threads} threads, {t1 * 1e6:.0f} us on one")
    oracle.set_threads(1)
    t1, c1 = _time_calls(lambda: oracle.attend_batched(q, k, v, nn, d ** -0.5), seconds / 6)
    oracle.set_threads(threads)
    breadth["32k_compact_layer_one_thread"] = {"us": round(t1 * 1e6, 1), "calls": c1}
    res["breadth"] = breadth
    return res


if __name__ == "__main__":
    main()
