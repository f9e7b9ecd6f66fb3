"""Benchmark of the ArborKV eviction hot path on one MI355X.

One step = one eviction event on the Llama-3-8B-shaped synthetic tree (32
layers, 8 KV heads, head_dim 128, bf16; root 1024 tokens, branching 4, depth 3,
256 tokens per node; 4 active leaves; budget 25 % of all tokens):

    arbor_score -> arbor_allocate -> arbor_select -> arbor_compact
    -> arbor_tree_decode_attn (all 32 layers, the 4 active leaves)

on inputs already resident in HBM.  Before every step the pristine pool and
tree state are restored with an untimed device copy, and a 512 MiB buffer is
then read (untimed) so that the 256 MB last-level cache holds only clean lines:
otherwise the write-back of the restore copy's dirty lines would be charged to
the timed kernels.  Write-backs of what the step itself writes (the compaction)
stay inside the step.  `value` is resident KV tokens per second of step time
(tokens scored as keys, then kept or evicted, compacted, then decoded).

Lazy rehydration reads the token-span record from pinned host memory, so its
rate includes the host link; it is timed in the same run as a separate
backtracking transition leg and reported under "rehydrate", never in `value`.

Per-entry-point times come from HIP events recorded on the stream the kernels
run on.  The CPU oracle is timed on a bounded sample of the same workload and
reported as "cpu_baseline".
"""
from __future__ import annotations

import argparse
import json
import math
import os
import sys
import time

import numpy as np
import torch

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

from paper_2605_22106_amd import _lib as L  # noqa: E402
from paper_2605_22106_amd import synth  # noqa: E402

HBM_PEAK_GBS = 8000.0
BF16_PEAK_TFLOPS = 2500.0
METRIC = "KV tokens scored+evicted+compacted/s; tree-decode attn HBM GB/s (% of peak)"


CSRC = os.path.join(ROOT, "paper_2605_22106_amd", "csrc")
# kernels of each entry point (name prefix) and the source file that defines them
ENTRY_KERNELS = {
    "arbor_score": ("score_", "score.hip"),
    "arbor_allocate": ("allocate_", "allocate.hip"),
    "arbor_select": ("select_", "select.hip"),
    "arbor_compact": ("compact_", "compact.hip"),
    "arbor_select_compact": ("select_plan", "compact.hip"),
    "arbor_tree_decode_attn": ("decode_", "decode.hip"),
    "arbor_rehydrate": ("rehyd_", "rehydrate.hip"),
    "arbor_uncertainty": ("uncert_", "uncertainty.hip"),
}


def short_kernel_name(name: str) -> str:
    """'arbor::(anonymous namespace)::compact_move(...)' -> 'compact_move';
    '_ZN5arbor12_GLOBAL__N_110score_passILi0EDF16bLi128ELi2ELi2EEEv...' -> 'score_pass<0,bf16,128,2,2>'."""
    import re
    m = re.search(r"_GLOBAL__N_1(\d+)", name)
    if m and name.startswith("_Z"):
        k = int(m.group(1))
        start = m.end()
        ident = name[start:start + k]
        rest = name[start + k:]
        if rest.startswith("I"):
            args = []
            for tok in re.finditer(r"Li(\d+)E|Lb([01])E|DF16b|(?<=[IE])f(?=[LE])",
                                   rest[:rest.find("EEv") + 1]):
                t = tok.group(0)
                if tok.group(1):
                    args.append(tok.group(1))
                elif tok.group(2):
                    args.append("true" if tok.group(2) == "1" else "false")
                else:
                    args.append("bf16" if t == "DF16b" else "f32")
            return f"{ident}<{','.join(args)}>"
        return ident
    m = re.search(r"arbor::\(anonymous namespace\)::(?:void )?([A-Za-z_0-9]+(?:<[^>(]*>)?)\(", name)
    if m:
        return m.group(1)
    m = re.search(r"void arbor::\(anonymous namespace\)::([A-Za-z_0-9]+(?:<[^>(]*>)?)\(", name)
    return m.group(1) if m else name[:80]


def source_sha256(fname: str) -> str:
    import hashlib
    with open(os.path.join(CSRC, fname), "rb") as f:
        return hashlib.sha256(f.read()).hexdigest()[:16]


def summarize_trace(db: str, title: str, command: str) -> str:
    """Per-kernel calls / avg / min / max / total (us) of a rocprofv3 kernel-trace database."""
    import collections
    import sqlite3
    c = sqlite3.connect(db)
    d = collections.defaultdict(list)
    for name, dur in c.execute("select name, duration from kernels"):
        d[name].append(dur / 1000.0)
    lines = [f"# {title}", f"# command: {command}",
             "# durations from rocprofv3 --kernel-trace, microseconds",
             f"{'calls':>5} {'avg_us':>9} {'min_us':>9} {'max_us':>9} {'total_us':>10}  kernel"]
    rows = sorted(((short_kernel_name(n), v) for n, v in d.items() if "arbor" in n),
                  key=lambda kv: -sum(kv[1]))
    for name, v in rows:
        lines.append(f"{len(v):5d} {sum(v) / len(v):9.2f} {min(v):9.2f} {max(v):9.2f} "
                     f"{sum(v):10.1f}  {name}")
    return "\n".join(lines) + "\n"


def summarize_traffic(fetch_csv: str, write_csv: str, title: str, command: str,
                      copy_bytes: int) -> str:
    """HBM bytes per dispatch from FETCH_SIZE / WRITE_SIZE (KiB), each scaled by what the
    counter reads for a plain device copy of `copy_bytes` (the last dispatches of the run)."""
    import collections
    import csv

    def per_kernel(path, counter):
        agg = collections.defaultdict(list)
        copies = []
        for r in csv.DictReader(open(path)):
            if r["Counter_Name"] != counter:
                continue
            v = float(r["Counter_Value"])
            if "arbor" in r["Kernel_Name"]:
                agg[short_kernel_name(r["Kernel_Name"])].append(v)
            elif "copyBuffer" in r["Kernel_Name"] or "copy" in r["Kernel_Name"].lower():
                copies.append((int(r["Dispatch_Id"]), v))
        copies.sort()
        return agg, copies

    fk, fcopy = per_kernel(fetch_csv, "FETCH_SIZE")
    wk, wcopy = per_kernel(write_csv, "WRITE_SIZE")
    kib = copy_bytes / 1024.0
    # the calibration copies are the last three copy dispatches of the run
    f_cal = float(np.mean([v for _, v in fcopy[-3:]]))
    w_cal = float(np.mean([v for _, v in wcopy[-3:]]))
    ff, wf = kib / f_cal, kib / w_cal
    lines = [f"# {title}", f"# command (FETCH_SIZE): {command.format(counter='FETCH_SIZE')}",
             f"# command (WRITE_SIZE): {command.format(counter='WRITE_SIZE')}",
             f"# calibration: a plain device copy of {copy_bytes} bytes reads FETCH_SIZE "
             f"{f_cal:.1f} KiB and WRITE_SIZE {w_cal:.1f} KiB; factors {ff:.4f} (fetch), "
             f"{wf:.4f} (write)",
             "# one JSON object per kernel: average counters per dispatch and scaled HBM bytes"]
    src_of = {pre: src for pre, src in ENTRY_KERNELS.values()}
    for name in sorted(set(fk) | set(wk)):
        fkib = float(np.mean(fk.get(name, [0.0])))
        wkib = float(np.mean(wk.get(name, [0.0])))
        # the longest matching prefix ("select_plan" of arbor_select_compact
        # lives in compact.hip, the other "select_" kernels in select.hip)
        pres = sorted((pre for pre in src_of if name.startswith(pre)), key=len)
        src = src_of[pres[-1]] if pres else None
        lines.append(json.dumps({
            "kernel": name, "fetch_kib": round(fkib, 3), "write_kib": round(wkib, 3),
            "hbm_read_bytes": round(fkib * ff * 1024), "hbm_write_bytes": round(wkib * wf * 1024),
            "source": src, "source_sha256": source_sha256(src) if src else None}))
    lines.append(json.dumps({"calibration": {"copy_bytes": copy_bytes, "fetch_kib": f_cal,
                                             "write_kib": w_cal, "fetch_factor": ff,
                                             "write_factor": wf}}))
    return "\n".join(lines) + "\n"


# the kernel of each rated stage whose launches are timed on their own
# (a per-call timing request, arbor_timing_t) and rated against its roofline
STAGE_KERNEL = {"score": (L.KERNEL_SCORE_ATTN, "score_attn", "score.hip"),
                "compact": (L.KERNEL_COMPACT_MOVE, "compact_move", "compact.hip"),
                "decode": (L.KERNEL_DECODE_ATTN, "decode_attn", "decode.hip")}


def stored_kernel_traffic(workload: str, prefix: str, src: str):
    """HBM bytes per launch of the kernels named `prefix*` from the committed counter
    summary, or None when it is missing or their source changed since."""
    path = os.path.join(ROOT, "profiles", f"{workload}_hbm_traffic.txt")
    if not os.path.exists(path):
        return None
    rows = [json.loads(line) for line in open(path) if line.startswith("{")]
    # (the attention of a scored decode keeps its logits: a kernel of its own,
    # never launched by the plain decode that the stage times)
    rows = [r for r in rows if r.get("kernel", "").startswith(prefix)
            and not r["kernel"].endswith(",true>")]
    if not rows or any(r["source_sha256"] != source_sha256(src) for r in rows):
        return None
    return {"read_bytes": sum(r["hbm_read_bytes"] for r in rows),
            "write_bytes": sum(r["hbm_write_bytes"] for r in rows),
            "kernels": [r["kernel"] for r in rows], "source": os.path.relpath(path, ROOT)}


def parse():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=10)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--config", default="llama8b")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-rehydrate-leg", action="store_true")
    ap.add_argument("--no-uncertainty-leg", action="store_true")
    ap.add_argument("--no-credit-leg", action="store_true",
                    help="skip timing arbor_tree_decode_attn_scored (decode + A credit)")
    ap.add_argument("--legs", default="dpts,llama70b,deep",
                    help="other configurations measured after the headline one")
    ap.add_argument("--no-legs", action="store_true")
    ap.add_argument("--walk-only", action="store_true",
                    help="run only the deep-tree walk leg and print its record")
    ap.add_argument("--no-graph", action="store_true",
                    help="launch the timed steps eagerly instead of replaying a captured HIP graph")
    ap.add_argument("--summarize-trace", metavar="DB",
                    help="write a per-kernel summary of a rocprofv3 kernel-trace database and exit")
    ap.add_argument("--summarize-traffic", nargs=2, metavar=("FETCH_CSV", "WRITE_CSV"),
                    help="write per-kernel HBM bytes from FETCH_SIZE / WRITE_SIZE counter CSVs")
    ap.add_argument("--title", default="")
    ap.add_argument("--command", default="")
    ap.add_argument("--out", default=None)
    ap.add_argument("--copy-calibration-mib", type=int, default=0,
                    help="after the run, copy a buffer of this many MiB device to device with "
                         "a plain copy kernel (a known-size reference for HBM byte counters)")
    return ap.parse_args()


class Event:
    def __init__(self, kv, st, cfg):
        self.kv = kv
        self.st = st
        self.cfg = cfg
        V, N = kv.num_nodes, kv.num_tokens
        dev = "cuda"
        self.observers = st["observers"].to(dev)
        self.q_win = st["q_win"].to(dev).contiguous()
        self.v_sig = st["v_sig"].to(dev)
        self.u_sig = st["u_sig"].to(dev)
        self.A = torch.zeros(N, device=dev)
        self.rows = torch.zeros(V, dtype=torch.int64, device=dev)
        self.a = torch.empty(V, device=dev)
        self.s = torch.empty(V, device=dev)
        self.k = torch.empty(V, dtype=torch.int32, device=dev)
        self.delta = torch.empty_like(self.k)
        self.on_path = torch.empty(V, dtype=torch.uint8, device=dev)
        self.sel = torch.empty(N, dtype=torch.int32, device=dev)
        self.status = torch.zeros(1, dtype=torch.int32, device=dev)
        self.q_dec = st["q_dec"].to(dev).contiguous()
        Hq = kv.kv_heads * kv.q_per_kv
        self.out = torch.empty((st["active"].numel(), kv.layers, Hq, kv.head_dim),
                               dtype=torch.bfloat16, device=dev)
        self.lse = torch.empty((st["active"].numel(), kv.layers, Hq), device=dev)
        chain_max = max(sum(int(st["n_full"][a]) for a in _chain(st["parent"].tolist(), j))
                        for j in range(V))
        nbytes = L.arbor_workspace_size(kv, max_context=chain_max,
                                        max_observers=self.observers.numel(),
                                        window=st["window"], n_slice=len(st["slice_layers"]),
                                        max_leaves=max(4, st["active"].numel()),
                                        max_layers=kv.layers)
        self.ws = torch.empty(nbytes, dtype=torch.uint8, device=dev)
        self.params = dict(st["params"])

    def check(self, rc):
        if rc != L.OK:
            raise RuntimeError(f"arbor call failed on the host: {L.arbor_strerror(rc)}")

    def reset_scores(self):
        self.A.zero_()
        self.rows.zero_()
        self.status.zero_()

    def run(self, active, marks=None, timings=None, decode=True):
        """score -> allocate -> select + compact (arbor_select_compact) -> decode;
        `marks` records events between the entry points, `timings` ({stage:
        L.Timing}) asks each call to time its rated kernel; decode=False stops
        after the compaction."""
        tm = timings or {}
        kv, st = self.kv, self.st
        ev = (lambda: marks.append(torch.cuda.Event(enable_timing=True))) if marks is not None else None

        def mark():
            if ev is not None:
                ev()
                marks[-1].record()

        mark()
        self.check(L.arbor_score(kv, self.observers, self.q_win, st["window"], st["slice_layers"],
                                 self.v_sig, self.u_sig, self.A, self.rows, self.a, self.s,
                                 self.params, self.status, self.ws, timing=tm.get("score")))
        mark()
        self.check(L.arbor_allocate(kv, active, st["budget"], self.s, self.params, self.k,
                                    self.delta, self.on_path, self.status, self.ws))
        mark()
        self.check(L.arbor_select_compact(kv, self.A, self.k, self.params, self.sel,
                                          self.status, self.ws, timing=tm.get("compact")))
        mark()
        if not decode:
            return
        self.check(L.arbor_tree_decode_attn(kv, active, 0, kv.layers, self.q_dec, self.out,
                                            self.lse, 0.0, self.status, self.ws,
                                            timing=tm.get("decode")))
        mark()


def _chain(parent, j):
    out = []
    while j >= 0:
        out.append(j)
        j = parent[j]
    return out


def algorithmic_work(st, kv, k_after, n_kept_before, active):
    """Bytes / flops each entry point must move or compute on this instance."""
    parent = st["parent"].tolist()
    n_full = st["n_full"].tolist()
    Hkv, G, d, Lyr = kv.kv_heads, kv.q_per_kv, kv.head_dim, kv.layers
    esz = 2 if kv.dtype == L.BF16 else 4
    row_all_layers = Lyr * Hkv * d * esz * 2            # K + V of one token, all layers
    S = len(st["slice_layers"])
    W = st["window"]
    # score: every (window row, context key) pair once
    pairs = 0
    for j in range(len(parent)):
        ch = _chain(parent, j)
        anc = sum(n_kept_before[a] for a in ch[1:])
        wj = min(W, n_full[j])
        own = sum(n_full[j] - wj + t + 1 for t in range(wj))
        pairs += (anc * wj + own) * S * Hkv * G
    score_flops = 2.0 * d * pairs
    score_bytes = (sum(n_kept_before) * S * Hkv * d * esz + st["q_win"].numel() * esz
                   + 4 * kv.num_tokens)
    # compact: rows whose slot changes, read + write, every layer and KV head
    moved = 0
    sel = st.get("_sel_cpu")
    tok_off = st["tok_off"].tolist()
    for i in range(len(parent)):
        if k_after[i] < n_kept_before[i]:
            keep = sel[tok_off[i]:tok_off[i] + k_after[i]]
            moved += int(np.sum(keep != np.arange(k_after[i])))
    compact_bytes = 2.0 * moved * row_all_layers
    # select: A of every candidate + one position per kept token
    cand = sum(n_kept_before[i] for i in range(len(parent)) if k_after[i] < n_kept_before[i])
    kept = sum(k_after[i] for i in range(len(parent)) if k_after[i] < n_kept_before[i])
    select_bytes = 4.0 * cand + 4.0 * kept
    # decode: K + V of the union of the active chains, every layer, + Q + O
    union = set()
    for l in active:
        union.update(_chain(parent, l))
    union_tok = sum(k_after[a] for a in union)
    naive_tok = sum(k_after[a] for l in active for a in _chain(parent, l))
    qo = 2 * len(active) * Lyr * Hkv * G * d * 2
    decode_bytes = union_tok * row_all_layers + qo
    decode_naive = naive_tok * row_all_layers + qo
    # decode-time credit: K of the slice layers and A (read + write) for every
    # key of a proper ancestor of an active leaf, + the slice-layer queries
    anc = set()
    for l in active:
        anc.update(_chain(parent, l)[1:])
    anc_tok = sum(k_after[a] for a in anc)
    credit_bytes = (anc_tok * S * Hkv * d * esz + 8 * anc_tok
                    + len(active) * S * Hkv * G * d * esz)
    return dict(score_flops=score_flops, score_bytes=score_bytes, score_pairs=pairs,
                compact_bytes=compact_bytes, moved_rows=moved, select_bytes=select_bytes,
                decode_bytes=decode_bytes, decode_naive_bytes=decode_naive,
                union_tokens=union_tok, credit_bytes=credit_bytes)


def cpu_baseline(st, kv_cpu_state, sel_budget_active, work, reps=2):
    """Time the oracle on the host cores: `reps` whole steps of the same event (every
    observer window scored, allocate, select, compact, decode of every active leaf over all
    layers), on the same input bytes; the value is the mean over the reps."""
    from oracle import arbor_oracle as O

    def np_float(t):
        return t.detach().to("cpu", torch.float32).numpy()

    def oracle_state(d):
        out = {key: d[key].cpu().numpy().astype(np.int64) for key in
               ("parent", "n_full", "tok_off", "page_off", "n_kept", "page_table", "slot_pos",
                "free_stack")}
        out.update(free_top=np.int64(int(d["free_top"].reshape(-1)[0])), k=np_float(d["k"]),
                   v=np_float(d["v"]), page_size=int(d["page_size"]))
        return out

    # the oracle's numpy products run on as many BLAS threads as the process
    # has cores
    cores = len(os.sched_getaffinity(0))
    blas_threads = None
    try:
        from threadpoolctl import threadpool_limits
        limiter = threadpool_limits(limits=cores, user_api="blas")
        blas_threads = cores
    except Exception:       # threadpoolctl missing: numpy's own default
        limiter = None
    t0 = time.perf_counter()
    ost = oracle_state(kv_cpu_state)
    t_conv = time.perf_counter() - t0
    parent = st["parent"].numpy()
    V = len(parent)
    obs = st["observers"].tolist()
    q = np_float(st["q_win"])
    qd = np_float(st["q_dec"])
    active, budget, params = sel_budget_active
    Lyr = st["layers"]
    stage = {"score": 0.0, "allocate": 0.0, "select": 0.0, "compact": 0.0, "decode": 0.0}
    for _ in range(reps):
        t0 = time.perf_counter()
        A, _, _, s = O.score(ost, obs, q, st["window"], st["slice_layers"], st["q_per_kv"],
                             st["v_sig"].numpy(), st["u_sig"].numpy(),
                             np.zeros(st["num_tokens"], np.float32), np.zeros(V, np.int64),
                             theta=st["params"]["theta"])
        t1 = time.perf_counter()
        k, _, _, _ = O.allocate(parent, ost["n_full"], ost["n_kept"], active, budget, s, params)
        t2 = time.perf_counter()
        sel, _ = O.select(ost, A, k, params["l_tail"])
        t3 = time.perf_counter()
        new = O.compact(ost, k, sel)
        t4 = time.perf_counter()
        O.tree_decode_attn(new, active, 0, Lyr, qd, st["q_per_kv"])
        t5 = time.perf_counter()
        for name, dt in zip(stage, (t1 - t0, t2 - t1, t3 - t2, t4 - t3, t5 - t4)):
            stage[name] += dt / reps
    if limiter is not None:
        limiter.unregister()
    total = sum(stage.values())
    return {"value": st["num_tokens"] / total, "unit": "tokens/s", "cores": cores, "kind": "oracle",
            "cpu_model": cpu_model(), "blas_threads": blas_threads,
            "sample": (f"{reps} whole steps of the same event on the same inputs (all "
                       f"{len(obs)} observer windows scored, allocate, select, compact, decode of "
                       f"the {len(active)} active leaves over all {Lyr} layers), "
                       f"{total:.1f} s per step, {reps * total:.1f} s in all"),
            "stage_s": dict(stage, state_to_numpy=t_conv)}


def cpu_model() -> str:
    try:
        for line in open("/proc/cpuinfo"):
            if line.startswith("model name"):
                return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return "unknown"


def copy_rate_gbs(mib=1024, reps=5):
    """Read+write GB/s of a plain device-to-device copy of `mib` MiB (a
    reference for what a data-moving kernel can reach on this GPU)."""
    src = torch.ones(mib << 20, dtype=torch.uint8, device="cuda")
    dst = torch.empty_like(src)
    dst.copy_(src)
    torch.cuda.synchronize()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record()
    for _ in range(reps):
        dst.copy_(src)
    e1.record()
    torch.cuda.synchronize()
    ms = e0.elapsed_time(e1) / reps
    del src, dst
    return 2.0 * (mib << 20) / (ms * 1e-3) / 1e9


def config_label(cfg, kv):
    return (f"{cfg.name}: {cfg.layers} layers, {cfg.kv_heads} KV heads, {cfg.q_heads} q heads, "
            f"head_dim {cfg.head_dim}, {cfg.dtype}; root {cfg.root_tokens}, branching "
            f"{cfg.branching}, depth {cfg.depth}, {cfg.node_tokens} tokens/node "
            f"({kv.num_nodes} nodes, {kv.num_tokens} tokens); {cfg.n_active} active leaves; "
            f"budget {cfg.rho:.0%}; window {cfg.window}")


def measure_event(cfg, steps, warmup, use_graph=True, copy_gbs=None, rehydrate_leg=True):
    """One eviction event on configuration `cfg` (score -> allocate -> select ->
    compact -> tree decode of the active leaves over every layer) on inputs
    resident in HBM: the whole step and the event without the decode, each
    captured once as a HIP graph and replayed, then a breakdown pass with the
    rated kernels timed on their own.  Returns (result dict, objects the
    caller may reuse)."""
    st = synth.build_config(cfg, device="cuda", host_store=rehydrate_leg)
    kv = L.kv_state_from(st, "cuda")
    del st["k"], st["v"]                            # the pool lives in kv
    pristine = kv.clone()
    ev = Event(kv, st, cfg)
    active = st["active"].cuda()
    flush = torch.ones(128 << 20, dtype=torch.int32, device="cuda")  # 512 MiB

    def restore():
        kv.copy_from(pristine)
        ev.reset_scores()
        flush.sum()  # reads only: leaves the last-level cache clean

    def raise_on_status():
        code = int(ev.status)
        if code < 0:
            raise RuntimeError(f"device status {code}: {L.arbor_strerror(code)}")
        return code

    for _ in range(warmup):
        restore()
        ev.run(active)
    torch.cuda.synchronize()
    raise_on_status()

    # the step (and the event without the decode) captured once as HIP graphs:
    # their launches replay without per-launch host work (the library only
    # enqueues kernels: no host synchronisation, allocation or memset inside
    # an entry point)
    graphs = {}
    if use_graph:
        for name, dec in (("step", True), ("event", False)):
            restore()
            torch.cuda.synchronize()
            g = torch.cuda.CUDAGraph()
            with torch.cuda.graph(g):
                ev.run(active, decode=dec)
            torch.cuda.synchronize()
            graphs[name] = g

    def timed(n, name):
        times, wall = [], 0.0
        for _ in range(n):
            restore()
            torch.cuda.synchronize()
            e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            t0 = time.perf_counter()
            e0.record()
            if name in graphs:
                graphs[name].replay()
            else:
                ev.run(active, decode=name == "step")
            e1.record()
            torch.cuda.synchronize()
            wall += time.perf_counter() - t0
            times.append(e0.elapsed_time(e1))
        return times, wall

    if graphs:
        timed(warmup, "step")
        raise_on_status()
    step_ms, wall = timed(steps, "step")
    event_ms, _ = timed(steps, "event")
    eager_ms = None
    if graphs:
        saved = graphs
        graphs = {}
        eager_ms = float(np.mean(timed(steps, "step")[0]))
        graphs = saved
    status = raise_on_status()

    # breakdown pass: events between the entry points and around the rated
    # kernels' launches (one timing request per call); kept apart from the
    # timed steps because every recorded event costs the stream a little time
    kevents = {}
    for name in STAGE_KERNEL:
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record()
        e1.record()
        kevents[name] = (e0, e1)
    ktiming = {name: L.timing(STAGE_KERNEL[name][0], *kevents[name]) for name in STAGE_KERNEL}
    stages = ["score", "allocate", "select+compact", "decode"]
    per_stage = {x: [] for x in stages}
    per_kernel = {x: [] for x in STAGE_KERNEL}
    for _ in range(steps):
        restore()
        torch.cuda.synchronize()
        marks = []
        ev.run(active, marks, ktiming)
        torch.cuda.synchronize()
        for si, x in enumerate(stages):
            per_stage[x].append(marks[si].elapsed_time(marks[si + 1]))
        for x, (e0, e1) in kevents.items():
            per_kernel[x].append(e0.elapsed_time(e1))
    raise_on_status()
    ms = float(np.mean(step_ms))
    ems = float(np.mean(event_ms))
    N_event = int(pristine.n_kept.sum())
    k_after = ev.k.cpu().tolist()
    st["_sel_cpu"] = ev.sel.cpu().numpy()
    work = algorithmic_work(st, kv, k_after, pristine.n_kept.cpu().tolist(), st["active"].tolist())
    mean = {x: float(np.mean(v)) for x, v in per_stage.items()}
    kmean = {x: float(np.mean(v)) for x, v in per_kernel.items()}
    rates = {
        "score": {"bound": "mfma", "achieved": work["score_flops"] / (kmean["score"] * 1e-3) / 1e12,
                  "peak": BF16_PEAK_TFLOPS, "unit": "TFLOP/s"},
        "compact": {"bound": "hbm",
                    "achieved": work["compact_bytes"] / (kmean["compact"] * 1e-3) / 1e9,
                    "peak": HBM_PEAK_GBS, "unit": "GB/s"},
        "decode": {"bound": "hbm", "achieved": work["decode_bytes"] / (kmean["decode"] * 1e-3) / 1e9,
                   "peak": HBM_PEAK_GBS, "unit": "GB/s"},
    }
    entry = {"score": "arbor_score", "compact": "arbor_select_compact",
             "decode": "arbor_tree_decode_attn"}
    for st_name, r in rates.items():
        _, kname, ksrc = STAGE_KERNEL[st_name]
        r["frac"] = r["achieved"] / r["peak"]
        if copy_gbs and r["unit"] == "GB/s":
            r["frac_of_copy"] = r["achieved"] / copy_gbs
        r["kernel"] = kname
        r["entry_point"] = entry[st_name]
        r["ms_per_launch"] = kmean[st_name]
        r["stage_ms"] = mean["select+compact" if st_name == "compact" else st_name]
        tr = stored_kernel_traffic(cfg.name, kname, ksrc)
        r["traffic"] = None if tr is None else tr["read_bytes"] + tr["write_bytes"]
        if tr is not None:
            r["traffic_kernels"] = tr["kernels"]
    # the entry points rated on their whole time: select + compact (one entry
    # point: the eviction and compaction of the event), the decode entry point
    sc_ms = mean["select+compact"]
    entry_rates = {
        "select+compact": {"ms": sc_ms, "bytes": work["compact_bytes"] + work["select_bytes"],
                           "achieved": (work["compact_bytes"] + work["select_bytes"])
                           / (sc_ms * 1e-3) / 1e9},
        "decode": {"ms": mean["decode"], "bytes": work["decode_bytes"],
                   "achieved": work["decode_bytes"] / (mean["decode"] * 1e-3) / 1e9},
    }
    for r in entry_rates.values():
        r.update(peak=HBM_PEAK_GBS, unit="GB/s", frac=r["achieved"] / HBM_PEAK_GBS)
        if copy_gbs:
            r["frac_of_copy"] = r["achieved"] / copy_gbs
    res = {
        "workload": config_label(cfg, kv), "tokens_per_step": N_event, "ms_per_step": ms,
        "value": N_event / (ms * 1e-3),
        "event_ms": ems, "event_tokens_per_s": N_event / (ems * 1e-3),
        "stages_ms": mean, "rates": rates, "entry_rates": entry_rates,
        "decode_union_vs_naive_bytes": [work["decode_bytes"], work["decode_naive_bytes"]],
        "compact_moved_rows": work["moved_rows"], "wall_ms_per_step": wall / steps * 1e3,
        "launch": "hip graph replay of the captured step" if graphs else "eager",
        "eager_ms_per_step": eager_ms, "status": status,
    }
    env = dict(st=st, kv=kv, pristine=pristine, ev=ev, active=active, flush=flush,
               restore=restore, work=work)
    if rehydrate_leg:
        res["rehydrate"] = rehydrate_leg_of(env)
    return res, env


def rehydrate_leg_of(env):
    """A transition to other leaves after the event: lazy rehydration of the
    new Path* from the pinned-host token store (PCIe-inclusive)."""
    st, kv, ev, restore = env["st"], env["kv"], env["ev"], env["restore"]
    restore()
    ev.run(env["active"])
    parent = st["parent"].tolist()
    leaves = [i for i in range(kv.num_nodes) if i not in parent]
    a0 = set(st["active"].tolist())
    alt = [l for l in leaves if l not in a0]
    a1 = torch.tensor([alt[(j * len(alt)) // len(a0) + 3] for j in range(len(a0))],
                      dtype=torch.int32, device="cuda")
    torch.cuda.synchronize()
    n_kept_before = kv.n_kept.cpu().numpy()
    e = [torch.cuda.Event(enable_timing=True) for _ in range(3)]
    e[0].record()
    ev.check(L.arbor_allocate(kv, a1, st["budget"], ev.s, ev.params, ev.k, ev.delta,
                              ev.on_path, ev.status, ev.ws))
    e[1].record()
    ev.check(L.arbor_rehydrate(kv, ev.on_path, st["host_k"], st["host_v"], ev.status, ev.ws))
    e[2].record()
    torch.cuda.synchronize()
    onp = ev.on_path.cpu().numpy().astype(bool)
    nf = st["n_full"].numpy()
    restored = int(np.sum((nf - n_kept_before)[onp]))
    row_bytes = kv.layers * kv.kv_heads * kv.head_dim * 2 * 2
    t_re = e[1].elapsed_time(e[2])
    return {"ms": t_re, "tokens_from_host": restored,
            "host_link_gbs": restored * row_bytes / (t_re * 1e-3) / 1e9,
            "nodes": int(np.sum(onp & (n_kept_before < nf))), "status": int(ev.status),
            "note": "pinned host -> HBM, PCIe-inclusive; not part of value"}


def walk_leg(steps_cap=None):
    """The deep backtracking tree (9,841 nodes, 82.7 GB of pool, budget 20 %):
    a 256-event random walk with 30 % backtracking run by arbor_walk (Alg. 2 on
    the device: Transition, lazy rehydration, scoring of each new leaf's
    window, eviction, Pressure at B - delta).  The first event (from full
    retention down to the budget) is timed on its own, then the other 255 in
    one call.  The token-span record stays in device memory: the 2 x 82.7 GB
    record exceeds the host memory the box can pin."""
    cfg = synth.CONFIGS["deep"]
    st = synth.build_config(cfg, device="cuda", decode_queries=False, host_store="device",
                            observers=[0])
    kv = L.kv_state_from(st, "cuda")
    del st["k"], st["v"], st["q_win"]
    V, N = kv.num_nodes, kv.num_tokens
    parent = st["parent"].tolist()
    n_ev = cfg.walk_steps if steps_cap is None else min(cfg.walk_steps, steps_cap)
    targets = synth.walk_targets(parent, n_ev, cfg.walk_backtrack, cfg.seed, int(st["active"][0]))
    Hq = kv.kv_heads * kv.q_per_kv
    g = torch.Generator(device="cuda").manual_seed(cfg.seed)
    q = torch.randn((len(targets), len(st["slice_layers"]), Hq, cfg.window, kv.head_dim),
                    generator=g, device="cuda").to(torch.bfloat16)
    rng = np.random.default_rng(cfg.seed)
    s = torch.tensor(rng.random(V).astype(np.float32), device="cuda")
    A = torch.zeros(N, device="cuda")
    rows = torch.zeros(V, dtype=torch.int64, device="cuda")
    a = torch.empty(V, device="cuda")
    k = torch.empty(V, dtype=torch.int32, device="cuda")
    delta = torch.empty_like(k)
    on_path = torch.empty(V, dtype=torch.uint8, device="cuda")
    sel = torch.empty(N, dtype=torch.int32, device="cuda")
    stats = torch.zeros((len(targets), 4), dtype=torch.int64, device="cuda")
    ws = torch.empty(L.arbor_workspace_size(kv, max_context=cfg.root_tokens
                                            + cfg.depth * cfg.node_tokens, max_observers=1,
                                            window=cfg.window, n_slice=len(st["slice_layers"])),
                     dtype=torch.uint8, device="cuda")
    stt = torch.zeros(1, dtype=torch.int32, device="cuda")
    tg = torch.tensor(targets, dtype=torch.int32, device="cuda")
    margin = 2048
    p = dict(st["params"])
    v_in, u_in = st["v_sig"].cuda(), st["u_sig"].cuda()

    def run(lo, hi):
        rc = L.arbor_walk(kv, tg[lo:hi], st["budget"], p, A, s, k, delta, on_path, sel, stt, ws,
                          host_k=st["host_k"], host_v=st["host_v"], pressure_margin=margin,
                          q_win=q[lo:hi], window=cfg.window, slice_layers=st["slice_layers"],
                          v_in=v_in, u_in=u_in, rows_seen=rows, a_out=a, stats=stats[lo:hi])
        if rc != L.OK:
            raise RuntimeError(f"arbor_walk failed on the host: {L.arbor_strerror(rc)}")

    torch.cuda.synchronize()
    e = [torch.cuda.Event(enable_timing=True) for _ in range(3)]
    e[0].record()
    run(0, 1)
    e[1].record()
    run(1, len(targets))
    e[2].record()
    torch.cuda.synchronize()
    code = int(stt)
    if code < 0:
        raise RuntimeError(f"device status {code}: {L.arbor_strerror(code)}")
    t = stats.cpu().numpy()
    first_ms = e[0].elapsed_time(e[1])
    rest_ms = e[1].elapsed_time(e[2])
    row_bytes = kv.layers * kv.kv_heads * kv.head_dim * 2 * 2
    restored = int(t[1:, 1].sum())
    res = {
        "workload": config_label(cfg, kv) + f"; {len(targets)}-event walk, backtrack "
                    f"{cfg.walk_backtrack:.0%}, pressure margin {margin} tokens",
        "events": len(targets), "first_event_ms": first_ms,
        "first_event_evicted_tokens": int(t[0, 2]),
        "ms_per_transition": rest_ms / max(1, len(targets) - 1),
        "transitions_per_s": (len(targets) - 1) / (rest_ms * 1e-3),
        "tokens_restored": restored, "bytes_restored": restored * row_bytes,
        "restore_gbs": restored * row_bytes / (rest_ms * 1e-3) / 1e9,
        "tokens_evicted": int(t[1:, 2].sum()), "pressure_events": int(t[:, 3].sum()),
        "resident_tokens_after": int(t[-1, 0]), "budget": st["budget"], "status": code,
        "note": ("token-span record in device memory (2 x 82.7 GB exceeds the pinnable host "
                 "memory): restore_gbs is HBM to HBM; the host-link rate is the pinned-host "
                 "rehydrate leg of llama8b and dpts"),
    }
    del kv, st, q, A, sel
    return res


def main():
    args = parse()
    if args.summarize_trace or args.summarize_traffic:
        if args.summarize_trace:
            text = summarize_trace(args.summarize_trace, args.title, args.command)
        else:
            text = summarize_traffic(args.summarize_traffic[0], args.summarize_traffic[1],
                                     args.title, args.command, args.copy_calibration_mib << 20)
        if args.out:
            with open(args.out, "w") as f:
                f.write(text)
        print(text, end="")
        return
    if args.gpus != 1:
        print(f"bench.py runs on one GPU only (asked for --gpus {args.gpus}); the multi-GPU "
              "subtree sharding of this path is a design note, not a measured configuration.",
              file=sys.stderr)
        sys.exit(2)
    cfg = synth.CONFIGS[args.config]
    torch.cuda.init()
    if args.walk_only:
        print(json.dumps({"deep_walk": walk_leg()}))
        return
    copy_gbs = copy_rate_gbs()
    head, env = measure_event(cfg, args.steps, args.warmup, use_graph=not args.no_graph,
                              copy_gbs=copy_gbs, rehydrate_leg=not args.no_rehydrate_leg)
    rates = head["rates"]
    dominant = max(STAGE_KERNEL, key=lambda x: rates[x]["ms_per_launch"])
    result = {
        "metric": METRIC, "value": head["value"], "unit": "tokens/s", "n_gpus": 1,
        "steps": args.steps, "warmup": args.warmup, "ms_per_step": head["ms_per_step"],
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None, "dtype": "bf16",
        "data": "synthetic",
        "config": {"workload": head["workload"], "tokens_per_step": head["tokens_per_step"],
                   "parallelism": "single GPU"},
        "roofline": dict(rates[dominant]),
        "metric1": {"what": "resident KV tokens scored + evicted + compacted per second "
                            "(score, allocate, select, compact; no decode)",
                    "value": head["event_tokens_per_s"], "unit": "tokens/s",
                    "ms": head["event_ms"]},
        "copy_gbs": copy_gbs,
    }
    for key in ("stages_ms", "rates", "entry_rates", "decode_union_vs_naive_bytes",
                "compact_moved_rows", "wall_ms_per_step", "launch", "eager_ms_per_step",
                "status", "rehydrate"):
        if key in head:
            result[key] = head[key]
    result["decode_hbm_gbs"] = rates["decode"]["achieved"]
    result["decode_hbm_frac"] = rates["decode"]["frac"]
    st, kv, ev, active, flush, restore = (env[x] for x in ("st", "kv", "ev", "active", "flush",
                                                          "restore"))
    work = env["work"]

    # decode that also credits its slice-layer attention weights to A, on the
    # state the step leaves behind, beside the plain decode timed the same way
    if not args.no_credit_leg:
        restore()
        ev.run(active)
        torch.cuda.synchronize()
        ce = (torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))
        for e in ce:
            e.record()          # torch refuses elapsed_time on events it never recorded
        ctm = L.timing(L.KERNEL_DECODE_CREDIT, *ce)
        t_sc, t_pl, t_k = [], [], []
        # the scored and plain calls carry no timing hooks of their own; the
        # merge-and-credit kernel is timed on a third call, so its events do
        # not bias the comparison
        for rep in range(args.warmup + args.steps):
            for leg in ("scored", "plain", "kernel"):
                flush.sum()
                e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
                e0.record()
                if leg != "plain":
                    ev.check(L.arbor_tree_decode_attn_scored(
                        kv, active, 0, kv.layers, ev.q_dec, ev.out, ev.lse, 0.0,
                        st["slice_layers"], 0, ev.A, ev.rows, ev.status, ev.ws,
                        timing=ctm if leg == "kernel" else None))
                else:
                    ev.check(L.arbor_tree_decode_attn(kv, active, 0, kv.layers, ev.q_dec, ev.out,
                                                      ev.lse, 0.0, ev.status, ev.ws))
                e1.record()
                torch.cuda.synchronize()
                if rep >= args.warmup:
                    if leg == "kernel":
                        t_k.append(ce[0].elapsed_time(ce[1]))
                    else:
                        (t_sc if leg == "scored" else t_pl).append(e0.elapsed_time(e1))
        if int(ev.status) < 0:
            raise RuntimeError(f"device status {int(ev.status)}")
        tk = float(np.mean(t_k))
        result["decode_scored"] = {
            "ms": float(np.mean(t_sc)), "plain_decode_ms": float(np.mean(t_pl)),
            "overhead_ms": float(np.mean(t_sc)) - float(np.mean(t_pl)),
            "merge_credit_kernel_ms": tk, "credit_bytes": work["credit_bytes"],
            "slice_layers": list(st["slice_layers"]),
            "note": "arbor_tree_decode_attn_scored (decode + decode-time credit of A); "
                    "not part of value"}

    # Eq. 1 uncertainty at the block boundaries: one logit row per block
    if not args.no_uncertainty_leg:
        vocab = 128256
        z = synth.boundary_logits(kv.num_nodes, vocab, seed=11, dtype="bf16", device="cuda")
        u = torch.empty(kv.num_nodes, device="cuda")
        st_u = torch.zeros(1, dtype=torch.int32, device="cuda")
        ws_u = torch.empty(L.arbor_uncertainty_workspace_size(kv.num_nodes, vocab, L.BF16),
                           dtype=torch.uint8, device="cuda")
        leg = {}
        for top_k in (0, 40):
            ts = []
            for rep in range(args.warmup + args.steps):
                flush.sum()
                e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
                e0.record()
                ev.check(L.arbor_uncertainty(z, top_k, u, st_u, ws_u))
                e1.record()
                torch.cuda.synchronize()
                if rep >= args.warmup:
                    ts.append(e0.elapsed_time(e1))
            t = float(np.mean(ts))
            nbytes = z.numel() * 2
            gbs = nbytes / (t * 1e-3) / 1e9
            leg["full" if top_k == 0 else f"top{top_k}"] = {
                "ms": t, "rows": kv.num_nodes, "vocab": vocab, "bytes": nbytes,
                "achieved": gbs, "peak": HBM_PEAK_GBS, "unit": "GB/s", "frac": gbs / HBM_PEAK_GBS}
        leg["status"] = int(st_u)
        leg["note"] = "arbor_uncertainty over one bf16 logit row per block; not part of value"
        result["uncertainty"] = leg

    if not args.no_cpu_baseline:
        pristine = env["pristine"]
        cpu_state = {k_: (v_.cpu() if isinstance(v_, torch.Tensor) else v_) for k_, v_ in st.items()
                     if k_ not in ("host_k", "host_v")}
        cpu_state.update(k=pristine.k.cpu(), v=pristine.v.cpu(), n_kept=pristine.n_kept.cpu(),
                         page_table=pristine.page_table.cpu(), slot_pos=pristine.slot_pos.cpu(),
                         free_stack=pristine.free_stack.cpu(), free_top=pristine.free_top.cpu())
        result["cpu_baseline"] = cpu_baseline(st, cpu_state, (st["active"].tolist(), st["budget"],
                                                                st["params"]), work)
    del env, st, kv, ev, active, flush, restore
    torch.cuda.empty_cache()

    # the other configurations: extra keys, never part of value
    legs = {}
    names = [] if args.no_legs else [x for x in args.legs.split(",") if x]
    for name in names:
        if name == "deep":
            legs[name] = walk_leg()
        else:
            leg, env = measure_event(synth.CONFIGS[name], min(args.steps, 5),
                                     min(args.warmup, 2), use_graph=not args.no_graph,
                                     copy_gbs=copy_gbs, rehydrate_leg=(name == "dpts"))
            legs[name] = leg
            del env
        torch.cuda.empty_cache()
    if legs:
        result["legs"] = legs
    if args.copy_calibration_mib > 0:
        n = args.copy_calibration_mib << 20
        src = torch.ones(n, dtype=torch.uint8, device="cuda")
        dst = torch.empty_like(src)
        for _ in range(3):
            dst.copy_(src)
        torch.cuda.synchronize()
        result["copy_calibration_bytes"] = n
    print(json.dumps(result))


if __name__ == "__main__":
    main()
