"""Where a launch's time goes: per-workgroup phase marks of the library's kernels.

    python -m paper_2608_30252_amd.build --trace        # builds libmad_trace.so
    python -m paper_2608_30252_amd.phase_trace [--launches N]

A diagnostic, not part of the product path.  It loads libmad_trace.so, which
is built from the same sources with MAD_PHASE_TRACE defined: thread 0 of every
workgroup then stores the device's 100 MHz constant counter (s_memrealtime) at
named phases of the kernel, and its XCC id.  The counter has its own origin on
each XCD, so every time below is measured from the earliest start of a
workgroup on the same XCD and then averaged over the XCDs and launches.  Every
split of a decode unit runs on one XCD (the unit count is a multiple of 8), so
a unit's whole hand-off is timed on one counter.

Workloads (the benchmark's shapes, random inputs, buffer sets rotated so the
key/value reads come from HBM):
  decode_compact  32K compact-memory layer: 2048 slots + 1023-token window + the
                  new token, 32/8 heads, d 64, bf16 (192 workgroups)
  decode_full     the full 32769-key KV of the same layer
  decode_batched  16 sequences, 1024 slots + 511-token window each
  update_64       memory update of 64 rows (16 sequences x 4 slots), D 2048,
                  8 KV heads x d 64 (update_rows_kernel)
  verify_70b      verify attention, B1, 64/8 heads, d 128, 32768 + 5 keys, T 5
                  (split kernel; the merge is a separate launch)
"""
import argparse
import ctypes
import os

import numpy as np
import torch

import paper_2608_30252_amd as mad
from paper_2608_30252_amd import build as _build

SLOTS, WGS = 16, 4096   # kTraceSlots, kTraceWGs of the trace build
TICK_US = 0.01         # one tick of the 100 MHz counter


class Trace:
    def __init__(self, lib, name):
        self.read = getattr(lib, f"mad_trace_{name}_read")
        self.clear = getattr(lib, f"mad_trace_{name}_clear")
        self.buf = np.zeros(SLOTS * WGS, dtype=np.uint64)
        assert self.clear() == 0

    def grab(self):
        """Marks of the last launch: rows [workgroup][slot], workgroups that marked entry."""
        torch.cuda.synchronize()
        assert self.read(self.buf.ctypes.data_as(ctypes.c_void_p), ctypes.c_size_t(self.buf.nbytes)) == 0
        assert self.clear() == 0
        e = self.buf.reshape(WGS, SLOTS).astype(np.int64)
        return e[e[:, 0] != 0]


def per_xcd(e):
    """(xcd, its rows, its origin) for each XCD present."""
    xcc = (e[:, SLOTS - 1] >> 32) & 0xF
    for x in np.unique(xcc):
        rows = e[xcc == x]
        yield x, rows, rows[:, 0].min()


def us(t, t0):
    return (t - t0) * TICK_US


def report_decode(name, runs):
    st, arr, atom, loads, head, rest, done, iss, land, args = [], [], [], [], [], [], [], [], [], []
    for e in runs:
        for _, r, t0 in per_xcd(e):
            st.append(us(r[:, 0].max(), t0))
            iss.append(np.mean(r[:, 6] - r[:, 0]) * TICK_US)
            land.append(np.mean(r[:, 7] - r[:, 0]) * TICK_US)
            args.append(np.mean(r[:, 8] - r[:, 0]) * TICK_US)
            arr.append(np.percentile(us(r[:, 1], t0), [0, 50, 100]))
            m = r[r[:, 5] != 0]
            for w in m:
                atom.append(us(w[2], w[1])); loads.append(us(w[3], w[2])); head.append(us(w[4], w[3]))
                rest.append(us(w[5], w[4])); done.append(us(w[5], t0))
    a = np.mean(arr, axis=0)
    print(f"{name}: {len(runs[0])} workgroups, {len(runs)} launches (times from the XCD's first start)")
    print(f"  workgroup starts spread over {np.mean(st):.2f} us; per workgroup, after its start: kernel "
          f"arguments read {np.mean(args):.2f}, first loads issued {np.mean(iss):.2f}, first tile landed "
          f"{np.mean(land):.2f} us")
    print(f"  split partials stored and acknowledged: {a[0]:.2f} / {a[1]:.2f} / {a[2]:.2f} us (min / median / max)")
    print(f"  merging workgroups ({len(done) // len(runs)} a launch): arrival atomic {np.mean(atom):.2f}, "
          f"partials into LDS {np.mean(loads):.2f}, first head merged {np.mean(head):.2f}, "
          f"other heads and stores {np.mean(rest):.2f} us")
    print(f"  merge done {np.mean(done):.2f} us (latest {np.max(done):.2f})")


def report_update(name, runs):
    st, rows, prod, epi, end, acc, red, bar, sto = [], [], [], [], [], [], [], [], []
    for e in runs:
        for _, r, t0 in per_xcd(e):
            st.append(us(r[:, 0].max(), t0))
            rows.append(np.mean(r[:, 1] - r[:, 0]) * TICK_US)
            prod.append(np.mean(r[:, 2] - r[:, 1]) * TICK_US)
            epi.append(np.mean(r[:, 3] - r[:, 2]) * TICK_US)
            acc.append(np.mean(r[:, 4] - r[:, 2]) * TICK_US)
            red.append(np.mean(r[:, 5] - r[:, 4]) * TICK_US)
            bar.append(np.mean(r[:, 6] - r[:, 5]) * TICK_US)
            sto.append(np.mean(r[:, 3] - r[:, 6]) * TICK_US)
            end.append(us(r[:, 3].max(), t0))
    print(f"{name}: {len(runs[0])} workgroups, {len(runs)} launches")
    print(f"  workgroup starts spread over {np.mean(st):.2f} us; per workgroup: first rows in LDS "
          f"{np.mean(rows):.2f}, products {np.mean(prod):.2f}, reduction and stores {np.mean(epi):.2f} us; "
          f"last store {np.mean(end):.2f} us")
    print(f"  reduction and stores: partial tiles in LDS {np.mean(acc):.2f}, summed {np.mean(red):.2f}, "
          f"second barrier {np.mean(bar):.2f}, store issued {np.mean(sto):.2f} us")


def report_verify(name, runs):
    st, ends, dur = [], [], []
    for e in runs:
        for _, r, t0 in per_xcd(e):
            st.append(us(r[:, 0].max(), t0))
            ends.append(np.percentile(us(r[:, 1], t0), [0, 50, 100]))
            dur.append(np.mean(r[:, 1] - r[:, 0]) * TICK_US)
    a = np.mean(ends, axis=0)
    print(f"{name}: {len(runs[0])} workgroups, {len(runs)} launches")
    print(f"  workgroup starts spread over {np.mean(st):.2f} us; partials written {a[0]:.2f} / {a[1]:.2f} / "
          f"{a[2]:.2f} us (min / median / max); mean workgroup {np.mean(dur):.2f} us")


def gen(shape, g, dev):
    return torch.randn(shape, generator=g, device=dev).to(torch.bfloat16)


def decode_sets(wl, n, dev):
    Hq, Hkv, d = 32, 8, 64
    B, mlen, wlen, wcap = {"decode_compact": (1, 2048, 1023, 1088), "decode_full": (1, 0, 32768, 32832),
                           "decode_batched": (16, 1024, 511, 576)}[wl]
    out = []
    for i in range(n):
        g = torch.Generator(device=dev).manual_seed(100 + i)
        s = dict(B=B, q=gen((B, Hq, d), g, dev), kn=gen((B, Hkv, d), g, dev), vn=gen((B, Hkv, d), g, dev),
                 rk=gen((B, Hkv, wcap, d), g, dev), rv=gen((B, Hkv, wcap, d), g, dev), mlen=mlen, wlen=wlen,
                 starts=[(37 * b + 5) % wcap for b in range(B)])
        if mlen:
            s["mk"], s["mv"] = gen((B, Hkv, mlen, d), g, dev), gen((B, Hkv, mlen, d), g, dev)
        out.append(s)
    ws = torch.zeros(mad.workspace_bytes(mad.MAD_OP_DECODE, B, Hq, Hkv, d), dtype=torch.uint8, device=dev)

    def call(s):
        mem = mad.KV(s["mk"], s["mv"], [s["mlen"]] * s["B"]) if s["mlen"] else None
        win = mad.KV(s["rk"], s["rv"], [s["wlen"]] * s["B"], s["starts"])
        # mode 1: the new token is attended but not appended, so every set stays as generated
        mad.draft_step_attn(s["q"], mem, win, s["kn"], s["vn"], [1] * s["B"], ws=ws)
    return out, call


def update_sets(n, dev):
    B, n_new, D, Hkv, d = 16, 4, 2048, 8, 64
    out = []
    for i in range(n):
        g = torch.Generator(device=dev).manual_seed(200 + i)
        out.append(dict(x=gen((B, n_new, D), g, dev), w=(gen((2 * Hkv * d, D), g, dev).float() * 0.02).to(torch.bfloat16),
                        mk=torch.zeros(B, Hkv, 1088, d, dtype=torch.bfloat16, device=dev),
                        mv=torch.zeros(B, Hkv, 1088, d, dtype=torch.bfloat16, device=dev),
                        pos=[[16 * (2048 + 4 * b + j) for j in range(n_new)] for b in range(B)]))

    def call(s):
        mad.memory_update(s["x"], s["w"], s["pos"], mad.KV(s["mk"], s["mv"], [1024] * B))
    return out, call


def verify_sets(n, dev):
    B, Hq, Hkv, d, T, cap = 1, 64, 8, 128, 5, 32776
    L = 32768 + T
    out = []
    for i in range(n):
        g = torch.Generator(device=dev).manual_seed(300 + i)
        out.append(dict(q=gen((B, T, Hq, d), g, dev), k=gen((B, Hkv, cap, d), g, dev), v=gen((B, Hkv, cap, d), g, dev)))
    ws = torch.zeros(mad.workspace_bytes(mad.MAD_OP_VERIFY, B, Hq, Hkv, d, T), dtype=torch.uint8, device=dev)

    def call(s):
        mad.verify_attn(s["q"], mad.KV(s["k"], s["v"], [L] * B), ws=ws)
    return out, call


def run(trace, sets, call, launches):
    for s in sets + sets:
        call(s)
    trace.grab()
    runs = []
    for j in range(launches):
        call(sets[j % len(sets)])
        runs.append(trace.grab())
    return runs


def main():
    ap = argparse.ArgumentParser(description=__doc__, formatter_class=argparse.RawDescriptionHelpFormatter)
    ap.add_argument("--launches", type=int, default=12, help="traced launches per workload")
    ap.add_argument("--lib", default=_build.TRACE_LIB, help="the trace build of the library")
    args = ap.parse_args()
    if not os.path.exists(args.lib):
        raise SystemExit(f"{args.lib} is missing: build it with `python -m paper_2608_30252_amd.build --trace`")
    assert torch.cuda.is_available(), "the phase trace needs a GPU"
    dev = torch.device("cuda")
    mad._LIB = None
    mad.LIB_PATH = args.lib
    lib = mad._load_library()
    for wl, n in (("decode_compact", 48), ("decode_full", 6), ("decode_batched", 8)):
        sets, call = decode_sets(wl, n, dev)
        report_decode(wl, run(Trace(lib, "decode"), sets, call, args.launches))
        del sets
        torch.cuda.empty_cache()
    sets, call = update_sets(8, dev)
    report_update("update_64", run(Trace(lib, "update"), sets, call, args.launches))
    del sets
    sets, call = verify_sets(3, dev)
    report_verify("verify_70b", run(Trace(lib, "verify"), sets, call, args.launches))


if __name__ == "__main__":
    main()
