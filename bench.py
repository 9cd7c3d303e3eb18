"""Throughput of shared-prompt group attention (forward + backward) on one MI355X.

    python bench.py [--gpus 1] [--steps K] [--warmup W] [--workload prompt]

One step = one pass of the whole hot path over one batch of synthetic input
already resident in HBM: prefill_fwd, replay_fwd, replay_bwd, prefill_bwd and
the Eq. 2 prompt_grad_reduce. The value is counted fwd+bwd TFLOP/s with the
FlashAttention-2 convention 14 * d * Hq * (valid query-key pairs of the shared
form: prefill + replay prompt column + replay own-branch blocks); the
flattened baseline's recomputed prompt and masked-out pairs are never counted.

Also reported on the same JSON line: % of the bf16 dense MFMA peak, the
wall-time speedup over the flattened per-branch baseline built from the same
kernels, a roofline entry for the dominant kernel (per-launch HIP-event
durations taken around each launch by the library's launch hook, on the
stream the kernel runs on), and the fp64 CPU oracle timed on a bounded sample
of the same workload (cpu_baseline).
"""
from __future__ import annotations

import argparse
import csv
import ctypes
import glob
import hashlib
import json
import math
import os
import re
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

PEAK_BF16_TFLOPS = 2500.0   # MI355X dense bf16 MFMA
PEAK_HBM_GBS = 8000.0       # MI355X HBM3E
METRIC = "shared-prompt attn fwd+bwd TFLOP/s, % bf16 MFMA peak, speedup vs flattened"

WORKLOAD_TEXT = {
    "tiny": "tiny group: 1 prompt, P=256, G=2, R=128, Hq=Hkv=4, d=64, seed 0",
    "balanced": "balanced: 4 groups x (P=4096, G=8, R=4096), Hq=32, Hkv=8, d=128, seed 0",
    "prompt": "prompt-dominant: 1 group, P=32768, G=8, R=2048, Hq=32, Hkv=8, d=128, seed 0",
    "response": "response-dominant: 1 group, P=2048, G=16, R=16384, Hq=32, Hkv=8, d=128, seed 0",
    "ragged": "ragged: 16 groups, P log-uniform [512,65536], G in {4,8,16}, R log-uniform [256,32768], "
              "<=1,048,576 tokens, Hq=32, Hkv=8, d=128, seed 7",
    **{f"gsweep{g}": f"group-size sweep: 1 group, P=8192, G={g}, R={65536 // g} (65,536 response tokens), "
                     f"Hq=32, Hkv=8, d=128, seed 0" for g in (8, 16, 32, 64)},
    "prompt_gqa7": "prompt-dominant, 7B-model heads: 1 group, P=32768, G=8, R=2048, Hq=28, Hkv=4 (g=7), d=128, seed 0",
    "short_resp": "short answers: 1 group, P=16384, G=32, R=64, Hq=32, Hkv=8, d=128, seed 0",
}

# launch role -> compiled kernel (template instantiation) it runs
ROLE_KERNEL = {
    "fwd_prefill": "attn_fwd_kernel<bf16 out>", "fwd_replay": "attn_fwd_kernel<bf16 out>",
    "fwd_tree": "attn_fwd_kernel<bf16 out>", "fwd_replay_split": "attn_fwd_kernel<fp32 out>",
    "dkv_prefill": "attn_dkv_kernel", "dkv_replay": "attn_dkv_kernel", "dkv_tree": "attn_dkv_kernel",
    "dq_prefill": "attn_dq_kernel", "dq_replay": "attn_dq_kernel", "dq_tree": "attn_dq_kernel",
    "lse_merge": "lse_merge_kernel", "grad_reduce": "grad_reduce_kernel", "reduce_tree": "grad_reduce_kernel",
}
# launch role -> step of the method (the prefill / replay time breakdown of the
# six-call path; the two-call path's launches hold both)
ROLE_STEP = {
    "fwd_prefill": "prefill_fwd", "fwd_replay": "replay_fwd", "fwd_replay_split": "replay_fwd",
    "lse_merge": "replay_fwd", "dkv_replay": "replay_bwd", "dq_replay": "replay_bwd",
    "dkv_prefill": "prefill_bwd", "dq_prefill": "prefill_bwd", "grad_reduce": "prompt_grad_reduce",
    "fwd_tree": "tree_fwd", "dq_tree": "tree_bwd", "dkv_tree": "tree_bwd", "reduce_tree": "tree_bwd",
}
# flops per (valid pair, query head) each attention role performs
ROLE_FLOPS_PER_PAIR_D = {"fwd": 4, "dkv": 8, "dq": 6}


def tree_chunk_rows(shape, chunk_blocks: int) -> int:
    """fp32 partial rows of the tree backward's chunked prompt-key sweeps:
    sum over groups of chunks x P when any group is cut into chunks of at most
    `chunk_blocks` query blocks (64 rows x one query head), else 0."""
    g = shape.num_q_heads // shape.num_kv_heads
    n = [min(64, max(1, -(-(-(-sum(rs) // 64) * g) // chunk_blocks))) for rs in shape.branch_lens]
    if max(n) == 1:
        return 0
    return sum(c * p for c, p in zip(n, shape.prompt_lens))


def role_work(role: str, shape, n_seed: int, split=None, chunk_blocks: int = 1024):
    """Algorithmic work of one step's launches of a role: ('flop', F) for
    contractions, ('byte', B) for the HBM-bound kernels. `split` flags the
    groups whose replay forward runs SPLIT (None: none of them)."""
    vp = shape.valid_pairs()
    hq, d = shape.num_q_heads, shape.head_dim
    rp_split = rr_split = rows_split = 0
    if split is not None:
        for g, on in enumerate(split):
            if on:
                P, rs = shape.prompt_lens[g], shape.branch_lens[g]
                rp_split += sum(r * P for r in rs)
                rr_split += sum(r * (r + 1) // 2 for r in rs)
                rows_split += sum(rs)
    replay = vp["replay_prompt"] + vp["replay_resp"]
    pairs = {
        "fwd_prefill": vp["prefill"], "fwd_replay": replay - rp_split - rr_split,
        "fwd_tree": vp["prefill"] + replay - rp_split - rr_split, "fwd_replay_split": rp_split + rr_split,
        "dkv_prefill": vp["prefill"], "dkv_replay": replay, "dkv_tree": vp["shared"],
        "dq_prefill": vp["prefill"], "dq_replay": replay, "dq_tree": vp["shared"],
    }
    if role in pairs:
        per = ROLE_FLOPS_PER_PAIR_D[role.split("_")[0]]
        return "flop", float(per * d * hq * pairs[role])
    tp, hkv = shape.total_prompt, shape.num_kv_heads
    if role == "grad_reduce":
        e = 2 * tp * hkv * d
        return "byte", float(e * 4 * (1 + n_seed) + e * 2)
    if role == "lse_merge":
        return "byte", float(rows_split * hq * (2 * d * 4 + 2 * 4 + d * 2 + 4))
    if role == "reduce_tree":   # the chunks' fp32 partials in, bf16 dK_P / dV_P out
        v = tree_chunk_rows(shape, chunk_blocks)
        parts = max(1, -(-v // max(tp, 1)))
        return "byte", float(2 * v * hkv * d * 4 + parts * tp * 4 + 2 * tp * hkv * d * 2)
    raise KeyError(role)


# profiles/ file names per workload
WORKLOAD_SLUG = {"tiny": "tiny_P256_G2", "balanced": "balanced_4groups_P4096_G8", "prompt": "prompt_P32768_G8",
                 "response": "response_P2048_G16", "ragged": "ragged_16groups",
                 **{f"gsweep{g}": f"gsweep_P8192_G{g}" for g in (8, 16, 32, 64)},
                 "prompt_gqa7": "prompt_P32768_G8_H28_4", "short_resp": "short_P16384_G32_R64"}


def kernel_source_hash() -> str:
    """Hash of the code (comments and whitespace removed) of every native
    source the kernels and their schedules are built from, and of the
    compile flags: HBM counters recorded under one hash do not describe
    another."""
    h = hashlib.sha256()
    for path in sorted(glob.glob(os.path.join(ROOT, "paper_2609_33133_amd", "csrc", "*"))):
        if path.endswith((".hip", ".h", ".cpp")):
            with open(path) as f:
                code = f.read()
            code = re.sub(r"/\*.*?\*/", " ", code, flags=re.S)
            code = re.sub(r"//[^\n]*", " ", code)
            h.update(os.path.basename(path).encode())
            h.update(" ".join(code.split()).encode())
    from paper_2609_33133_amd import build as _build
    for src in ("attn_fwd.hip", "attn_bwd.hip", "elementwise.hip"):
        h.update(" ".join(_build.hip_flags(src)).encode())
    return h.hexdigest()[:16]


_KNAME = re.compile(r"(attn_fwd_kernel|attn_dkv_kernel|attn_dq_kernel|bwd_dsum_kernel|lse_merge_kernel|"
                    r"grad_reduce_kernel)(<([^>]*)>)?")


def bench_kernel_name(rocprof_name: str):
    """rocprofv3 kernel name -> the name used in the bench line (None for
    kernels that are not the library's, e.g. runtime copies)."""
    m = _KNAME.search(rocprof_name)
    if not m:
        return None
    base, targs = m.group(1), (m.group(3) or "")
    if base == "attn_fwd_kernel":
        return base + ("<fp32 out>" if "true" in targs else "<bf16 out>")
    return base


def _counter_rows(path: str, counter: str):
    out = []
    with open(path) as f:
        for r in csv.DictReader(f):
            if r["Counter_Name"] == counter:
                out.append((r["Kernel_Name"], float(r["Counter_Value"])))
    return out


def algorithmic_bytes(role: str, shape, flat_rows: int = 0):
    """Minimum HBM bytes of one launch of an attention role: every input read
    once and every output written once (the prompt KV counted once). For the
    flattened baseline's roles (tag "flattened") the inputs are its private
    copies, `flat_rows` rows in all."""
    hq, hkv, d = shape.num_q_heads, shape.num_kv_heads, shape.head_dim
    tp, tr = shape.total_prompt, shape.total_resp
    qrow, kvrow = hq * d * 2, hkv * d * 2
    if role.startswith("flattened:"):
        role, tp, tr = role.split(":", 1)[1], flat_rows, 0
    role = role.split(":", 1)[-1]
    if role == "fwd_prefill":      # Q_P, K_P, V_P -> O_P, LSE_P
        return tp * (qrow + 2 * kvrow), tp * (qrow + hq * 4)
    if role == "fwd_replay":       # Q_R, K_P, V_P, K_R, V_R -> O_R, LSE_R
        return tr * qrow + (tp + tr) * 2 * kvrow, tr * (qrow + hq * 4)
    if role == "fwd_tree":
        return (tp + tr) * (qrow + 2 * kvrow), (tp + tr) * (qrow + hq * 4)
    if role in ("dq_prefill", "dq_replay", "dq_tree"):   # Q, dO, O, LSE, K, V -> dQ, D
        rows = {"dq_prefill": tp, "dq_replay": tr, "dq_tree": tp + tr}[role]
        kv = tp if role == "dq_prefill" else tp + tr
        return rows * (3 * qrow + hq * 4) + kv * 2 * kvrow, rows * (qrow + hq * 4)
    if role in ("dkv_prefill", "dkv_replay", "dkv_tree"):  # Q, dO, LSE, D, K, V -> dK, dV (fp32 slabs or bf16)
        rows = {"dkv_prefill": tp, "dkv_replay": tr, "dkv_tree": tp + tr}[role]
        kv = {"dkv_prefill": tp, "dkv_replay": tp + tr, "dkv_tree": tp + tr}[role]
        out = {"dkv_prefill": tp * 2 * hkv * d * 4, "dkv_replay": tp * 2 * hkv * d * 4 + tr * 2 * kvrow,
               "dkv_tree": (tp + tr) * 2 * kvrow}[role]
        return rows * (2 * qrow + hq * 8) + kv * 2 * kvrow, out
    return None


def summarize_pmc(d: str, workload: str, roles_file: str = None) -> str:
    """Markdown summary (with a machine-readable line) of the FETCH_SIZE and
    WRITE_SIZE passes in d/{fetch,write} and of the 1 GiB copy calibration
    passes in d/{cfetch,cwrite} (rocprofv3 -f csv, file run_counter_collection.csv).
    With `roles_file` (the launch roles of the profiled run in launch order,
    written by --profile-roles), the library's dispatches are attributed to
    their roles as well: per-role bytes against the role's algorithmic bytes."""
    def rows(sub, counter):
        return _counter_rows(os.path.join(d, sub, "run_counter_collection.csv"), counter)
    copy_bytes = 1 << 30
    cf = max(v for _, v in rows("cfetch", "FETCH_SIZE"))
    cw = max(v for _, v in rows("cwrite", "WRITE_SIZE"))
    f_scale = copy_bytes / (cf * 1024.0)
    w_scale = copy_bytes / (cw * 1024.0)
    roles = None
    if roles_file:
        with open(roles_file) as f:
            roles = json.load(f)
    per, per_role = {}, {}
    for sub, counter, scale, key in (("fetch", "FETCH_SIZE", f_scale, "fetch"), ("write", "WRITE_SIZE", w_scale, "write")):
        lib_rows = [(name, v) for name, v in rows(sub, counter) if bench_kernel_name(name) is not None]
        if roles is not None and len(lib_rows) != len(roles["launches"]):
            raise ValueError(f"{sub}: {len(lib_rows)} library dispatches but {len(roles['launches'])} logged launches")
        for i, (name, v) in enumerate(lib_rows):
            k = bench_kernel_name(name)
            r = None if roles is None else roles["launches"][i]
            if r is not None:
                if ROLE_KERNEL[r.split(":", 1)[-1]] != k:
                    raise ValueError(f"dispatch {i}: kernel {k} but logged role {r}")
                per_role.setdefault(r, {"fetch": [], "write": []})[key].append(v * 1024.0 * scale)
            # the per-kernel figures (the bench line's roofline traffic) cover
            # the shared step only, not the flattened baseline's launches
            if r is None or r.startswith("shared:"):
                per.setdefault(k, {"fetch": [], "write": []})[key].append(v * 1024.0 * scale)

    def avg(e):
        n = len(e["fetch"])
        fb = sum(e["fetch"]) / max(n, 1)
        wb = sum(e["write"]) / max(len(e["write"]), 1)
        return {"launches": n, "fetch_bytes_per_launch": round(fb), "write_bytes_per_launch": round(wb),
                "bytes_per_launch": round(fb + wb)}
    kernels = {k: avg(e) for k, e in per.items()}
    roles_out = {r: avg(e) for r, e in per_role.items()}
    data = {"workload": workload, "source_hash": kernel_source_hash(),
            "path": None if roles is None else roles.get("path"),
            "calibration": {"copy_bytes": copy_bytes, "copy_fetch_kib": cf, "copy_write_kib": cw,
                            "fetch_scale": round(f_scale, 4), "write_scale": round(w_scale, 4)},
            "kernels": kernels}
    if roles is not None:
        data["roles"] = roles_out
    lines = [("Shared step only (" + str(data["path"]) + " path):" if roles is not None else "Every library dispatch:"),
             "", "| kernel | launches | HBM read GB / launch | HBM write GB / launch |", "|---|---|---|---|"]
    for k, v in sorted(kernels.items(), key=lambda kv: -kv[1]["bytes_per_launch"]):
        lines.append(f"| {k} | {v['launches']} | {v['fetch_bytes_per_launch'] / 1e9:.3f} | "
                     f"{v['write_bytes_per_launch'] / 1e9:.3f} |")
    if roles is not None:
        from paper_2609_33133_amd import inputs as I
        shape = I.config_shape(workload)
        lines += ["", "Per launch role (tag: the step that launched it):", "",
                  "| role | launches | HBM read GB / launch | algorithmic read GB | HBM write GB / launch | "
                  "algorithmic write GB |", "|---|---|---|---|---|---|"]
        for r, v in sorted(roles_out.items()):
            alg = algorithmic_bytes(r, shape, roles.get("flattened_rows", 0))
            ar, aw = ("-", "-") if alg is None else (f"{alg[0] / 1e9:.3f}", f"{alg[1] / 1e9:.3f}")
            lines.append(f"| {r} | {v['launches']} | {v['fetch_bytes_per_launch'] / 1e9:.3f} | {ar} | "
                         f"{v['write_bytes_per_launch'] / 1e9:.3f} | {aw} |")
    lines.append("")
    lines.append(f"Copy calibration: a 1 GiB device copy reads {cf:.1f} KiB of FETCH_SIZE and writes {cw:.1f} KiB of "
                 f"WRITE_SIZE per dispatch, so the factors are {f_scale:.4f} (read) and {w_scale:.4f} (write).")
    lines.append("")
    lines.append("<!-- traffic-json " + json.dumps(data, sort_keys=True) + " -->")
    return "\n".join(lines)


def summarize_counters(d: str, roles_file: str = None) -> str:
    """Markdown table per kernel: MFMA busy % (SQ_VALU_MFMA_BUSY_CYCLES over
    GRBM_GUI_ACTIVE / 8 x 1024 SIMDs, pass d/sq) and achieved HBM read / write
    GB/s (copy-calibrated FETCH_SIZE / WRITE_SIZE over the dispatch time,
    passes d/{fetch,write,cfetch,cwrite}). With `roles_file` (the
    --profile-roles log of the same command as every pass) only the shared
    step's dispatches are counted."""
    def load(sub):
        rows = {}
        with open(os.path.join(d, sub, "run_counter_collection.csv")) as f:
            for r in csv.DictReader(f):
                e = rows.setdefault(int(r["Dispatch_Id"]), {"name": r["Kernel_Name"]})
                e[r["Counter_Name"]] = float(r["Counter_Value"])
                e["ns"] = int(r["End_Timestamp"]) - int(r["Start_Timestamp"])
        return [rows[i] for i in sorted(rows)]
    roles = None
    if roles_file:
        with open(roles_file) as f:
            roles = json.load(f)["launches"]
    cf = max(e["FETCH_SIZE"] for e in load("cfetch"))
    cw = max(e["WRITE_SIZE"] for e in load("cwrite"))
    f_scale, w_scale = (1 << 30) / (cf * 1024.0), (1 << 30) / (cw * 1024.0)
    acc = {}
    for sub in ("sq", "fetch", "write"):
        lib = [e for e in load(sub) if bench_kernel_name(e["name"]) is not None]
        if roles is not None:
            if len(lib) != len(roles):
                raise ValueError(f"{sub}: {len(lib)} library dispatches but {len(roles)} logged launches")
            lib = [e for e, r in zip(lib, roles) if r.startswith("shared:")]
        for e in lib:
            k = bench_kernel_name(e["name"])
            a = acc.setdefault(k, {"sq_ns": 0, "busy": 0.0, "gui": 0.0, "f_ns": 0, "fb": 0.0, "w_ns": 0, "wb": 0.0,
                                   "n": 0})
            if sub == "sq":
                a["busy"] += e["SQ_VALU_MFMA_BUSY_CYCLES"]
                a["gui"] += e["GRBM_GUI_ACTIVE"] / 8.0 * 1024.0
                a["sq_ns"] += e["ns"]
                a["n"] += 1
            elif sub == "fetch":
                a["fb"] += e["FETCH_SIZE"] * 1024.0 * f_scale
                a["f_ns"] += e["ns"]
            else:
                a["wb"] += e["WRITE_SIZE"] * 1024.0 * w_scale
                a["w_ns"] += e["ns"]
    lines = ["| kernel | launches | avg ms | MFMA busy % | HBM read GB/s | HBM write GB/s |", "|---|---|---|---|---|---|"]
    for k, a in sorted(acc.items(), key=lambda kv: -kv[1]["sq_ns"]):
        busy = 100.0 * a["busy"] / a["gui"] if a["gui"] else 0.0
        rd = a["fb"] / a["f_ns"] if a["f_ns"] else 0.0
        wr = a["wb"] / a["w_ns"] if a["w_ns"] else 0.0
        lines.append(f"| {k} | {a['n']} | {a['sq_ns'] / max(a['n'], 1) / 1e6:.3f} | {busy:.1f} | {rd:.0f} | {wr:.0f} |")
    return "\n".join(lines)


def summarize_trace(stats_csv: str) -> str:
    """Markdown table of a rocprofv3 --kernel-trace --stats kernel_stats.csv."""
    lines = ["| kernel | calls | total ms | avg ms | % |", "|---|---|---|---|---|"]
    with open(stats_csv) as f:
        for r in csv.DictReader(f):
            name = r["Name"].replace("void ", "").replace("augtree::(anonymous namespace)::", "").split("(")[0]
            lines.append(f"| {name} | {r['Calls']} | {int(r['TotalDurationNs']) / 1e6:.2f} | "
                         f"{float(r['AverageNs']) / 1e6:.4f} | {float(r['Percentage']):.2f} |")
    return "\n".join(lines)


def recorded_traffic(workload: str, kernel: str, path: str = "tree"):
    """HBM bytes per launch of `kernel` from the committed counter summary of
    this workload and step path, or None when there is none or the kernel
    sources changed since the counters were taken."""
    fname = os.path.join(ROOT, "profiles", f"hbm_traffic_{WORKLOAD_SLUG[workload]}.md")
    if not os.path.exists(fname):
        return None
    with open(fname) as f:
        m = re.search(r"<!-- traffic-json (\{.*\}) -->", f.read())
    if not m:
        return None
    data = json.loads(m.group(1))
    if (data.get("source_hash") != kernel_source_hash() or data.get("workload") != workload
            or data.get("path") != path):
        return None
    k = data["kernels"].get(kernel)
    return None if k is None else k["bytes_per_launch"]


class KernelTimer:
    """Records a HIP event pair around every library kernel launch (through
    augtree_set_launch_hook) on the stream the kernel goes to."""

    def __init__(self, lib):
        import torch
        self.torch = torch
        self.lib = lib
        self.events = []        # (role, start, end)
        self._open = {}
        from paper_2609_33133_amd._lib import LAUNCH_HOOK
        self._cb = LAUNCH_HOOK(self._hook)

    def _hook(self, role, phase, stream, user):
        torch = self.torch
        ext = torch.cuda.ExternalStream(stream) if stream else torch.cuda.default_stream()
        ev = torch.cuda.Event(enable_timing=True)
        ev.record(ext)
        r = role.decode()
        if phase == 0:
            self._open[r] = ev
        else:
            self.events.append((r, self._open.pop(r), ev))

    def __enter__(self):
        self.lib.augtree_set_launch_hook(self._cb, None)
        return self

    def __exit__(self, *a):
        self.lib.augtree_set_launch_hook(ctypes.cast(None, type(self._cb)), None)

    def summary(self):
        out = {}
        for role, a, b in self.events:
            out.setdefault(role, []).append(a.elapsed_time(b))
        return out


def time_steps(fn, steps: int, warmup: int):
    """Mean ms per step over `steps` back-to-back steps between two events,
    host wall ms per step, and the per-step times (an event between steps)."""
    import torch
    for _ in range(warmup):
        fn()
    torch.cuda.synchronize()
    ev = [torch.cuda.Event(enable_timing=True) for _ in range(steps + 1)]
    t0 = time.perf_counter()
    ev[0].record()
    for i in range(steps):
        fn()
        ev[i + 1].record()
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    per = [ev[i].elapsed_time(ev[i + 1]) for i in range(steps)]
    return ev[0].elapsed_time(ev[steps]) / steps, wall / steps * 1e3, per


_ORACLE_UNITS = None


def _oracle_unit(i):
    """Worker: one flattened (group, query head, branch) unit of the oracle,
    single-threaded BLAS; returns its wall seconds (input decoding included)."""
    from threadpoolctl import threadpool_limits

    from oracle import attention as A
    from paper_2609_33133_amd import inputs as I
    gi, spec = _ORACLE_UNITS[0], _ORACLE_UNITS[1][i]
    _, g, h, br, p0, p1, r0, r1, G = spec
    s = gi.shape
    c = I.bf16_bits_to_f64
    kh = h // (s.num_q_heads // s.num_kv_heads)
    with threadpool_limits(1):
        t0 = time.perf_counter()
        unit = (c(gi.q_p[p0:p1, h]), c(gi.k_p[p0:p1, kh]), c(gi.v_p[p0:p1, kh]), c(gi.q_r[r0:r1, h]),
                c(gi.k_r[r0:r1, kh]), c(gi.v_r[r0:r1, kh]), c(gi.do_p[p0:p1, h]), c(gi.do_r[r0:r1, h]),
                1.0 / G, s.scale)
        A._flat_unit(unit)
        return time.perf_counter() - t0


def cpu_baseline(gi, shared_flops: float, budget_s: float = 20.0, max_workers: int = 16):
    """The fp64 oracle (unchanged) timed on the host: its flattened units
    (group, query head, branch), largest first, on a process pool with one
    single-threaded worker per core (at most `max_workers`: the CPU share of
    one GPU). Units are started until `budget_s` has passed; the ones started
    are waited for. The whole job's time is extrapolated from the measured
    wall time by the flattened pairs of the measured units."""
    import multiprocessing as mp

    global _ORACLE_UNITS
    s = gi.shape
    specs = []
    for g in range(s.num_groups):
        p0, p1 = int(s.cu_prompt[g]), int(s.cu_prompt[g + 1])
        G = int(s.cu_branch[g + 1] - s.cu_branch[g])
        for h in range(s.num_q_heads):
            for br in range(int(s.cu_branch[g]), int(s.cu_branch[g + 1])):
                r0, r1 = int(s.cu_resp[br]), int(s.cu_resp[br + 1])
                L = (p1 - p0) + (r1 - r0)
                specs.append((L * (L + 1) // 2, g, h, br, p0, p1, r0, r1, G))
    specs.sort(key=lambda u: -u[0])
    total_pairs = sum(u[0] for u in specs)
    affinity = len(os.sched_getaffinity(0))
    workers = max(1, min(affinity, max_workers))
    units = specs                     # decoded inside the workers (forked: the inputs are shared)
    _ORACLE_UNITS = (gi, specs)
    done_pairs, done, unit_s = 0, 0, []
    t0 = time.perf_counter()
    with mp.get_context("fork").Pool(workers) as pool:
        pending = []
        nxt = 0
        while nxt < len(units) and (nxt < workers or time.perf_counter() - t0 < budget_s):
            # keep at most `workers` units in flight
            while nxt < len(units) and len([x for x in pending if not x[1].ready()]) < workers and \
                    (nxt < workers or time.perf_counter() - t0 < budget_s):
                pending.append((nxt, pool.apply_async(_oracle_unit, (nxt,))))
                nxt += 1
            time.sleep(0.05)
        for i, r in pending:
            unit_s.append(r.get())
            done_pairs += specs[i][0]
            done += 1
    wall = time.perf_counter() - t0
    _ORACLE_UNITS = None
    est_job_s = wall * total_pairs / done_pairs
    return {"value": round(shared_flops / est_job_s / 1e12, 6), "unit": "TFLOP/s", "cores": workers,
            "kind": "oracle",
            "sample": f"fp64 oracle (flattened per-branch units: group, query head, branch), largest first, on "
                      f"{workers} single-threaded workers ({affinity} cores in the affinity mask): {done} of "
                      f"{len(specs)} units measured in {wall:.1f} s wall (unit times {min(unit_s):.1f}-"
                      f"{max(unit_s):.1f} s); job time extrapolated by flattened pairs x{total_pairs / done_pairs:.1f}"
                      f": {est_job_s:.0f} s",
            "measured_units": done, "total_units": len(specs), "measured_s": round(wall, 2),
            "extrapolation_factor": round(total_pairs / done_pairs, 3), "est_job_s": round(est_job_s, 1)}


def device_inputs(shape, seed: int, device):
    """Seeded inputs drawn on the GPU (torch's Philox generator): the same
    distributions as the host recipe (Q, K, V ~ N(0,1)/sqrt(d), dO ~ N(0,1),
    rounded to bf16), used for the per-config rows so that the large
    workloads need no host-side generation."""
    import torch
    g = torch.Generator(device=device)
    g.manual_seed(seed)
    d = shape.head_dim
    inv = 1.0 / math.sqrt(d)
    tp, tr, hq, hkv = shape.total_prompt, shape.total_resp, shape.num_q_heads, shape.num_kv_heads
    x = {}
    for name, rows, heads, scale in (("q_p", tp, hq, inv), ("k_p", tp, hkv, inv), ("v_p", tp, hkv, inv),
                                     ("q_r", tr, hq, inv), ("k_r", tr, hkv, inv), ("v_r", tr, hkv, inv),
                                     ("do_p", tp, hq, None), ("do_r", tr, hq, None)):
        t = torch.randn((rows, heads, d), generator=g, device=device, dtype=torch.float32)
        if scale is not None:
            t.mul_(scale)
        x[name] = t.to(torch.bfloat16)
        del t
    return x


# per-config rows: (steps, warmup) of the shared and the flattened step
PER_CONFIG_STEPS = {"tiny": (200, 20), "balanced": (10, 3), "prompt": (10, 3), "response": (5, 2), "ragged": (2, 1)}


def measure_config(name: str, mode: int, path: str, steps=None, warmup=None, flattened=True):
    """ms per step of the shared step and of the flattened baseline on a named
    workload (device inputs), and the derived rates."""
    import torch

    from paper_2609_33133_amd import inputs as I
    from paper_2609_33133_amd.api import GroupBatch
    from paper_2609_33133_amd.group_attention import FlattenedStep, SharedStep
    s = I.config_shape(name)
    st, wu = PER_CONFIG_STEPS.get(name, (5, 2))
    st, wu = steps or st, warmup or wu
    b = GroupBatch.from_shape(s)
    x = device_inputs(s, 1000 + I.CONFIG_SEEDS[name], "cuda:0")
    step = SharedStep(b, "cuda:0", mode=mode, path=path)
    ms, wall_ms, per = time_steps(lambda: step.run(x), st, wu)
    del step
    torch.cuda.empty_cache()
    flat_ms = None
    if flattened:
        fstep = FlattenedStep(b, "cuda:0")
        fstep.materialize(x)
        flat_ms, _, _ = time_steps(fstep.run, st, wu)
        del fstep
    del x
    torch.cuda.empty_cache()
    vp = s.valid_pairs()
    counted = 14.0 * s.head_dim * s.num_q_heads * vp["shared"]
    tf = counted / (ms * 1e-3) / 1e12
    return {"workload": WORKLOAD_TEXT[name], "steps": st, "warmup": wu, "ms_per_step": round(ms, 4),
            "median_ms": round(float(np.median(per)), 4), "host_wall_ms_per_step": round(wall_ms, 4),
            "TFLOP/s": round(tf, 2), "pct_peak": round(100 * tf / PEAK_BF16_TFLOPS, 2),
            "flattened_ms_per_step": None if flat_ms is None else round(flat_ms, 4),
            "speedup_vs_flattened": None if flat_ms is None else round(flat_ms / ms, 3),
            "work_ratio": round(vp["flattened"] / vp["shared"], 3)}


def device_peak():
    """bf16 dense MFMA peak from the device properties: CUs x peak engine
    clock x 4096 flop per clock per CU (CDNA4: 4 SIMDs x 1024 flop/clk)."""
    import torch
    pr = torch.cuda.get_device_properties(0)
    clock_khz = None
    try:
        from paper_2609_33133_amd import _lib  # noqa: F401
        import ctypes.util  # noqa: F401
        hip = ctypes.CDLL("libamdhip64.so")
        v = ctypes.c_int(0)
        # hipDeviceAttributeClockRate = 5 (kHz)
        if hip.hipDeviceGetAttribute(ctypes.byref(v), 5, 0) == 0:
            clock_khz = v.value
    except OSError:
        pass
    cus = pr.multi_processor_count
    peak = None if clock_khz is None else cus * clock_khz * 1e3 * 4096 / 1e12
    return {"compute_units": cus, "peak_clock_mhz": None if clock_khz is None else clock_khz / 1e3,
            "bf16_dense_tflops_from_device": None if peak is None else round(peak, 1)}


class RoleLog:
    """Logs the role of every library launch (launch hook), tagged with the
    step that made it, for attributing counter dispatches to roles."""

    def __init__(self, lib):
        from paper_2609_33133_amd._lib import LAUNCH_HOOK
        self.lib = lib
        self.tag = "shared"
        self.launches = []
        self._cb = LAUNCH_HOOK(self._hook)

    def _hook(self, role, phase, stream, user):
        if phase == 0:
            self.launches.append(f"{self.tag}:{role.decode()}")

    def __enter__(self):
        self.lib.augtree_set_launch_hook(self._cb, None)
        return self

    def __exit__(self, *a):
        self.lib.augtree_set_launch_hook(ctypes.cast(None, type(self._cb)), None)


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--workload", default="prompt", choices=sorted(WORKLOAD_TEXT))
    ap.add_argument("--mode", default="fused", choices=("fused", "split", "auto"),
                    help="replay forward: fused, split, or per group by the library's cost rule")
    ap.add_argument("--path", default="tree", choices=("tree", "calls"),
                    help="tree: augtree_tree_fwd + augtree_tree_bwd; calls: the six separate entry points")
    ap.add_argument("--n-seed", type=int, default=None, help="prompt-key chunks of the six-call path")
    ap.add_argument("--chunk-blocks", type=int, default=0,
                    help="tree backward: query blocks per prompt-key sweep before it is chunked (0: the default)")
    ap.add_argument("--no-flattened", action="store_true")
    ap.add_argument("--no-cpu", action="store_true")
    ap.add_argument("--no-per-config", action="store_true")
    ap.add_argument("--no-breakdown", action="store_true")
    ap.add_argument("--cpu-budget", type=float, default=20.0, help="seconds of oracle units to start")
    ap.add_argument("--profile-roles", default=None, metavar="FILE",
                    help="only run W + K steps of the shared step and of the flattened baseline with the launch "
                         "roles logged to FILE (JSON), for attributing rocprofv3 counter dispatches; then exit")
    ap.add_argument("--summarize-pmc", default=None, metavar="DIR",
                    help="print the HBM traffic summary of rocprofv3 counter passes in DIR/{fetch,write,cfetch,cwrite} "
                         "(no GPU needed) and exit")
    ap.add_argument("--roles", default=None, metavar="FILE",
                    help="with --summarize-pmc / --summarize-counters: the --profile-roles log")
    ap.add_argument("--summarize-counters", default=None, metavar="DIR",
                    help="print MFMA busy %% and achieved HBM GB/s per kernel from rocprofv3 counter passes in "
                         "DIR/{sq,fetch,write,cfetch,cwrite} (no GPU needed) and exit")
    ap.add_argument("--summarize-trace", default=None, metavar="CSV",
                    help="print a table of a rocprofv3 kernel_stats.csv (no GPU needed) and exit")
    ap.add_argument("--copy-calibration", action="store_true",
                    help="only run a 1 GiB device-to-device copy 3 times (HBM counter calibration) and exit")
    args = ap.parse_args()
    if args.summarize_pmc:
        print(summarize_pmc(args.summarize_pmc, args.workload, args.roles))
        return
    if args.summarize_counters:
        print(summarize_counters(args.summarize_counters, args.roles))
        return
    if args.summarize_trace:
        print(summarize_trace(args.summarize_trace))
        return
    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) > 1:
        print("bench.py measures one GPU: the library has no multi-GPU path (the hot path shards by whole "
              "groups or KV heads with no exchange inside the op); run with --gpus 1", file=sys.stderr)
        sys.exit(2)

    import torch

    from paper_2609_33133_amd import _lib
    from paper_2609_33133_amd import inputs as I
    from paper_2609_33133_amd import api
    from paper_2609_33133_amd.api import REPLAY_AUTO, REPLAY_FUSED, REPLAY_SPLIT, GroupBatch
    from paper_2609_33133_amd.group_attention import FlattenedStep, SharedStep, upload

    lib = _lib.load()
    if not torch.cuda.is_available() or lib.augtree_check_device() != 0:
        print("bench.py needs an MI355X (gfx950): " + lib.augtree_last_error().decode(), file=sys.stderr)
        sys.exit(3)
    torch.cuda.set_device(0)
    api.set_tree_chunk_blocks(args.chunk_blocks)
    if args.copy_calibration:
        src = torch.ones(1 << 28, dtype=torch.float32, device="cuda:0")
        dst = torch.empty_like(src)
        for _ in range(3):
            dst.copy_(src)
        torch.cuda.synchronize()
        print(json.dumps({"copy_bytes_read": src.numel() * 4, "copy_bytes_written": dst.numel() * 4}))
        return
    mode = {"fused": REPLAY_FUSED, "split": REPLAY_SPLIT, "auto": REPLAY_AUTO}[args.mode]
    print(f"[bench] building inputs: {args.workload}", file=sys.stderr, flush=True)
    gi = I.make_config(args.workload)
    s = gi.shape
    b = GroupBatch.from_shape(s)
    x = upload(gi, "cuda:0")
    step = SharedStep(b, "cuda:0", mode=mode, n_seed=args.n_seed, path=args.path)

    if args.profile_roles:
        with RoleLog(lib) as log:
            for _ in range(args.warmup + args.steps):
                step.run(x)
            torch.cuda.synchronize()
            del step
            torch.cuda.empty_cache()
            log.tag = "flattened"
            fstep = FlattenedStep(b, "cuda:0")
            fstep.materialize(x)
            for _ in range(args.warmup + args.steps):
                fstep.run()
            torch.cuda.synchronize()
        os.makedirs(os.path.dirname(os.path.abspath(args.profile_roles)), exist_ok=True)
        with open(args.profile_roles, "w") as f:
            json.dump({"workload": args.workload, "path": args.path, "launches": log.launches,
                       "flattened_rows": int(fstep.tf)}, f)
        print(f"[bench] {len(log.launches)} launches logged to {args.profile_roles}", file=sys.stderr, flush=True)
        return

    vp = s.valid_pairs()
    counted = 14.0 * s.head_dim * s.num_q_heads * vp["shared"]

    print(f"[bench] shared path ({args.path})", file=sys.stderr, flush=True)
    ms, wall_ms, per_step = time_steps(lambda: step.run(x), args.steps, args.warmup)
    tflops = counted / (ms * 1e-3) / 1e12

    split = None
    if mode == REPLAY_SPLIT:
        split = [1] * s.num_groups
    elif mode == REPLAY_AUTO:
        split = [int(v) for v in api.replay_split_groups(b)]

    def kernel_pass(st, n_seed):
        """Per-kernel HIP-event durations over args.steps steps of `st`."""
        with KernelTimer(lib) as kt:
            for _ in range(args.steps):
                st.run(x)
            torch.cuda.synchronize()
        kernels, breakdown = {}, {}
        for role, times in kt.summary().items():
            k = ROLE_KERNEL[role]
            kind, work = role_work(role, s, n_seed, split, lib.augtree_tree_chunk_blocks())
            e = kernels.setdefault(k, {"ms": 0.0, "launches": 0, "work": 0.0, "kind": kind})
            e["ms"] += float(np.sum(times))
            e["launches"] += len(times)
            e["work"] += work * args.steps
            breakdown[ROLE_STEP[role]] = breakdown.get(ROLE_STEP[role], 0.0) + float(np.sum(times)) / args.steps
        return kernels, breakdown

    kernels, breakdown = kernel_pass(step, step.n_seed)
    dom_name, dom = max(kernels.items(), key=lambda kv: kv[1]["ms"])
    avg_ms = dom["ms"] / dom["launches"]
    per_launch = dom["work"] / dom["launches"]
    if dom["kind"] == "flop":
        achieved = per_launch / (avg_ms * 1e-3) / 1e12
        roof = {"bound": "mfma", "achieved": round(achieved, 2), "peak": PEAK_BF16_TFLOPS, "unit": "TFLOP/s",
                "frac": round(achieved / PEAK_BF16_TFLOPS, 4)}
    else:
        achieved = per_launch / (avg_ms * 1e-3) / 1e9
        roof = {"bound": "hbm", "achieved": round(achieved, 1), "peak": PEAK_HBM_GBS, "unit": "GB/s",
                "frac": round(achieved / PEAK_HBM_GBS, 4)}
    roof["kernel"] = dom_name
    roof["avg_launch_ms"] = round(avg_ms, 4)
    roof["launches_per_step"] = dom["launches"] // args.steps
    roof["work_per_launch"] = per_launch
    # HBM bytes per launch measured by the FETCH_SIZE / WRITE_SIZE counter
    # passes (copy-calibrated) on these exact sources, else null
    roof["traffic"] = recorded_traffic(args.workload, dom_name, args.path)
    roof["traffic_unit"] = "bytes per launch"
    kernel_table = {k: {"ms_per_step": round(v["ms"] / args.steps, 4),
                        ("TFLOP/s" if v["kind"] == "flop" else "GB/s"):
                            round(v["work"] / (v["ms"] * 1e-3) / (1e12 if v["kind"] == "flop" else 1e9), 2)}
                    for k, v in sorted(kernels.items(), key=lambda kv: -kv[1]["ms"])}
    n_seed = int(step.n_seed)
    del step
    torch.cuda.empty_cache()

    # prefill / replay breakdown: the six-call path puts each step of the
    # method in launches of its own
    calls_ms = None
    if not args.no_breakdown and args.path == "tree":
        print("[bench] six-call path (breakdown)", file=sys.stderr, flush=True)
        cstep = SharedStep(b, "cuda:0", mode=mode, n_seed=args.n_seed, path="calls")
        calls_ms, _, _ = time_steps(lambda: cstep.run(x), args.steps, args.warmup)
        _, breakdown_calls = kernel_pass(cstep, cstep.n_seed)
        breakdown.update(breakdown_calls)
        del cstep
        torch.cuda.empty_cache()

    flat_ms = None
    if not args.no_flattened:
        print("[bench] flattened baseline", file=sys.stderr, flush=True)
        fstep = FlattenedStep(b, "cuda:0")
        fstep.materialize(x)
        flat_ms, _, _ = time_steps(fstep.run, args.steps, args.warmup)
        del fstep
        torch.cuda.empty_cache()
    del x
    torch.cuda.empty_cache()

    per_config = None
    if not args.no_per_config:
        per_config = {}
        for name in I.CONFIG_NAMES:
            if name == args.workload:
                per_config[name] = {"workload": WORKLOAD_TEXT[name], "steps": args.steps, "warmup": args.warmup,
                                    "ms_per_step": round(ms, 4), "TFLOP/s": round(tflops, 2),
                                    "pct_peak": round(100 * tflops / PEAK_BF16_TFLOPS, 2),
                                    "flattened_ms_per_step": None if flat_ms is None else round(flat_ms, 4),
                                    "speedup_vs_flattened": None if flat_ms is None else round(flat_ms / ms, 3),
                                    "work_ratio": round(vp["flattened"] / vp["shared"], 3),
                                    "inputs": "host PCG64 recipe (the headline run)"}
                continue
            print(f"[bench] per-config row: {name}", file=sys.stderr, flush=True)
            per_config[name] = measure_config(name, mode, args.path, flattened=not args.no_flattened)
            per_config[name]["inputs"] = "device Philox draws, same distributions"

    cpu = None
    if not args.no_cpu:
        print("[bench] cpu oracle sample", file=sys.stderr, flush=True)
        cpu = cpu_baseline(gi, counted, budget_s=args.cpu_budget)

    line = {
        "metric": METRIC, "value": round(tflops, 2), "unit": "TFLOP/s", "n_gpus": 1, "steps": args.steps,
        "warmup": args.warmup, "ms_per_step": round(ms, 4), "higher_is_better": True, "scaling": "weak",
        "vs_baseline": None, "dtype": "bf16", "data": "synthetic",
        "config": {"workload": WORKLOAD_TEXT[args.workload], "replay_mode": args.mode, "path": args.path,
                   "n_seed": n_seed if args.path == "calls" else None,
                   "tree_chunk_blocks": api.tree_chunk_blocks() if args.path == "tree" else None,
                   "counted_tflop_per_step": round(counted / 1e12, 4), "flop_convention": "14*d*Hq*valid_pairs"},
        "pct_peak": round(100 * tflops / PEAK_BF16_TFLOPS, 2),
        "peak": {"bf16_dense_tflops_used": PEAK_BF16_TFLOPS, "source": "MI355X published dense bf16 MFMA peak",
                 **device_peak()},
        "speedup_vs_flattened": None if flat_ms is None else round(flat_ms / ms, 3),
        "flattened_ms_per_step": None if flat_ms is None else round(flat_ms, 4),
        "six_call_ms_per_step": None if calls_ms is None else round(calls_ms, 4),
        "host_wall_ms_per_step": round(wall_ms, 4),
        "step_ms": {"median": round(float(np.median(per_step)), 4), "min": round(float(np.min(per_step)), 4),
                    "max": round(float(np.max(per_step)), 4)},
        # the same time with the no-recompute convention 12 * d * Hq * valid_pairs
        "tflops_12d": round(tflops * 12.0 / 14.0, 2),
        "roofline": roof,
        "kernels": kernel_table,
        # time per step of each step of the method, from the per-launch events
        "breakdown_ms": {k: round(v, 4) for k, v in breakdown.items()},
        "replay_split_groups": None if split is None else int(sum(split)),
        "per_config": per_config,
        "cpu_baseline": cpu,
    }
    print(json.dumps(line), flush=True)


if __name__ == "__main__":
    main()
