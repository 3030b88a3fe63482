#!/usr/bin/env python3
"""Benchmark of the PQ matmul hot path on one MI355X.

One step = one Llama-3-8B decoder layer of decode GEMVs at effective 4 bits
(q, k, v, o, gate, up, down; M = 1, d = 2, C = 256, 8-bit ids), every matrix
read cold from HBM: the inputs are rotated over enough distinct copies
(>= 1 GiB) that the 256 MB Infinity Cache cannot serve them.

The timed region runs one launch list of `steps` consecutive layers
(fasq_launch_list_*: the launches are recorded once through the library
calls, then queued by the library with one hipLaunchKernel each, as a
serving loop would replay a decode step); each layer is four launches, as
deployed, since matrices that read the same activations go out as one
grouped call (q + k + v and gate + up through fasq_pq_gemv_batched; o and
down alone).  The same layers replayed from HIP graphs (several consecutive
layers per graph) are timed beside it and reported as us_per_layer_graph.  Separately, per-launch durations come from HIP events on the
launch stream around back-to-back launches of one group on distinct cold
copies (behind a spin kernel, so that host launch latency does not enter the
measurement): the difference between a 10-launch and a 2-launch batch,
divided by 8, which cancels the cost of the event pair.  These give the
roofline figures and the kernel-sum microseconds per layer.  --per-matrix
adds the same layer with one launch per matrix.

Also reported: the effective 3-bit layer plus lm_head (d = 4, C = 4096,
12-bit ids), the prefill GEMM (M = 128 / 512 / 2048 tokens, d = 4,
C = 256, 8-bit ids) in TFLOP/s, and the Qwen3-8B decode layer at M = 1, 4
and 16 tokens (C = 65536, 16-bit ids, a codebook larger than LDS), with the
L2 request counts of its launches when profiles/counters.json matches the
kernel sources.

Algorithmic bytes of one GEMV: N*R (packed ids) + C*d*2 (codebook) +
M*K*2 (x) + M*N*2 (y), with x counted once per grouped launch; flops of one
GEMM: 2*M*N*K.

Prints ONE JSON line on stdout; progress goes to stderr.
"""

from __future__ import annotations

import argparse
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

HBM_PEAK_GBS = 8000.0          # MI355X HBM3E
FP16_MFMA_PEAK_TFLOPS = 2500.0  # MI355X dense fp16 matrix peak
METRIC = "PQ GEMV HBM GB/s (% of peak) + us per Llama-3-8B layer; prefill PQ GEMM TFLOP/s"
ROTATION_BYTES = 1 << 30
SPACER_CYCLES = 2_000_000      # spin kernel queued ahead of event-timed launches
TIMING_COPIES = 12             # distinct copies one timing sample walks through
MODEL_LAYERS = 32              # decoder layers of Llama-3-8B: the most layers one graph replays


def log(*a):
    print(*a, file=sys.stderr, flush=True)


def gemv_bytes(M, K, N, d, C, bits):
    R = (K // d * bits + 7) // 8
    return N * R + C * d * 2 + M * K * 2 + M * N * 2


# ---------------------------------------------------------------------------
# Launch groups: matrices of a decoder layer that read the same activations go
# out as one grouped call (q, k, v; gate, up), the others alone.
# ---------------------------------------------------------------------------

SHARED_INPUT = (("q_proj", "k_proj", "v_proj"), ("gate_proj", "up_proj"))


def launch_groups(names):
    """Partition matrix indices into launch groups, in layer order."""
    groups, seen = [], set()
    for i, n in enumerate(names):
        if i in seen:
            continue
        g = [i]
        for members in SHARED_INPUT:
            if n in members:
                g = [j for j, m in enumerate(names) if m in members]
        seen.update(g)
        groups.append(g)
    return groups


# ---------------------------------------------------------------------------
# A set of matrices with rotating device copies
# ---------------------------------------------------------------------------

class MatrixSet:
    """Device copies of a list of PQ problems, rotated to defeat the MALL.

    ``groups`` lists the launch groups (lists of matrix indices); a group of
    several matrices is one fasq_pq_gemv_batched call on the x of its first
    matrix, a group of one is one fasq_pq_gemv call (fasq_pq_gemv_ex with a
    workspace when the call can use one).
    """

    def __init__(self, torch, fasq, problems, names, groups=None, min_copies=1, rotation_bytes=ROTATION_BYTES,
                 regime="gemv"):
        self.torch, self.fasq = torch, fasq
        self.regime = regime
        self.problems, self.names = problems, names
        self.groups = groups if groups is not None else [[i] for i in range(len(problems))]
        self.bytes = [gemv_bytes(p.M, p.K, p.N, p.d, p.C, p.idx_bits) for p in problems]
        self.bytes_per_set = sum(self.bytes)
        self.copies = max(min_copies, math.ceil(rotation_bytes / self.bytes_per_set) + 1)
        dev = torch.device("cuda:0")
        base = []
        for p in problems:
            base.append(dict(
                x=torch.from_numpy(p.x).to(dev), idx=torch.from_numpy(p.idx).to(dev),
                cb=torch.from_numpy(p.codebook).to(dev)))
        self.sets = []
        for c in range(self.copies):
            s = []
            for p, b in zip(problems, base):
                t = dict(x=b["x"].clone(), idx=b["idx"].clone(), cb=b["cb"].clone(),
                         y=torch.empty((p.M, p.N), dtype=torch.float16, device=dev))
                s.append(t)
            self.sets.append(s)
        del base
        # one workspace per matrix (launches run in order on one stream), for
        # the decode calls that use one
        self.ws = []
        for p in problems:
            need = (fasq.gemv_ex_workspace_bytes(p.M, p.K, p.N, p.idx_bits, p.d, p.C, 0) if regime == "gemv" else
                    fasq.gemm_ex_workspace_bytes(p.M, p.K, p.N, p.idx_bits, p.d, p.C) if regime == "gemm_ex" else 0)
            self.ws.append(torch.empty(need, dtype=torch.uint8, device=dev) if need > 0 else None)
        torch.cuda.synchronize()

    def group_bytes(self, g):
        """Algorithmic bytes of one launch of group g (x is read once)."""
        ps = [self.problems[i] for i in self.groups[g]]
        x_extra = sum(p.M * p.K * 2 for p in ps[1:])
        return sum(self.bytes[i] for i in self.groups[g]) - x_extra

    def group_name(self, g):
        return "+".join(self.names[i] for i in self.groups[g])

    def group_kernel(self, g):
        p = self.problems[self.groups[g][0]]
        if self.regime == "lut":
            return "k_gemm_lut"
        regime = "gemv_batched" if self.regime == "gemv" and len(self.groups[g]) > 1 else self.regime
        regime = "gemm" if regime == "gemm_ex" else regime
        return self.fasq.plan(regime, p.M, p.K, p.N, p.idx_bits, p.d, p.C)

    def launch(self, c, g, stream):
        members = self.groups[g]
        s = self.sets[c]
        p0, x = self.problems[members[0]], s[members[0]]["x"].data_ptr()
        if len(members) == 1:
            t = s[members[0]]
            ws = self.ws[members[0]]
            if self.regime == "gemm_ex":
                st = self.fasq.gemm_ex_raw(x, p0.M, p0.K, p0.N, t["idx"].data_ptr(), p0.idx_bits, p0.d,
                                           t["cb"].data_ptr(), p0.C, t["y"].data_ptr(),
                                           ws.data_ptr() if ws is not None else 0, ws.numel() if ws is not None else 0,
                                           stream)
            elif self.regime == "gemv" and ws is not None:
                # the decode call hands this matrix to the GEMM, which may split
                # K with a workspace (fasq_pq_gemv_ex with one shared codebook)
                st = self.fasq.gemv_ex_raw(x, p0.M, p0.K, p0.N, t["idx"].data_ptr(), p0.idx_bits, p0.d,
                                           t["cb"].data_ptr(), p0.C, 0, t["y"].data_ptr(), ws.data_ptr(),
                                           ws.numel(), stream)
            else:
                fn = dict(gemm=self.fasq.gemm_raw, lut=self.fasq.gemm_lut_raw).get(self.regime, self.fasq.gemv_raw)
                st = fn(x, p0.M, p0.K, p0.N, t["idx"].data_ptr(), p0.idx_bits, p0.d,
                        t["cb"].data_ptr(), p0.C, t["y"].data_ptr(), stream)
        else:
            st = self.fasq.gemv_batched_raw(
                x, p0.M, p0.K, [s[i]["idx"].data_ptr() for i in members], [self.problems[i].N for i in members],
                [s[i]["cb"].data_ptr() for i in members], [self.problems[i].C for i in members],
                [s[i]["y"].data_ptr() for i in members], p0.idx_bits, p0.d, stream)
        if st != 0:
            raise RuntimeError(f"launch failed: {self.fasq.status_string(st)}: {self.fasq.last_error()}")

    def launch_all(self, c, stream):
        for g in range(len(self.groups)):
            self.launch(c, g, stream)

    def capture_graphs(self, layers_per_graph=1):
        """Graph c replays the layer on copies c, c + 1, ... (layers_per_graph
        of them, modulo the number of copies)."""
        torch = self.torch
        s = torch.cuda.Stream()
        # eager warm-up first: one-time host-side set-up happens outside capture
        for c in range(self.copies):
            self.launch_all(c, torch.cuda.current_stream().cuda_stream)
        torch.cuda.synchronize()
        graphs = []
        for c in range(self.copies):
            g = torch.cuda.CUDAGraph()
            with torch.cuda.graph(g, stream=s):
                for k in range(layers_per_graph):
                    self.launch_all((c + k) % self.copies, torch.cuda.current_stream().cuda_stream)
            graphs.append(g)
        torch.cuda.synchronize()
        return graphs

    def time_kernels(self, steps, short=2, long=10):
        """Per-launch duration (seconds) of each launch group, from HIP events
        on the launch stream around back-to-back launches on distinct cold
        copies.

        Each sample is (t(long launches) - t(short launches)) / (long - short),
        which cancels the fixed cost of the event pair.  A spin kernel is queued
        ahead of every batch so that the launches reach the GPU back to back,
        whatever the host launch latency.
        """
        assert self.copies >= short + long
        torch = self.torch
        n = len(self.groups)
        per = [[] for _ in range(n)]
        stream = torch.cuda.current_stream()
        handle = stream.cuda_stream

        def batch(g, first, count):
            e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            torch.cuda._sleep(SPACER_CYCLES)
            e0.record(stream)
            for j in range(count):
                self.launch(first + j, g, handle)
            e1.record(stream)
            e1.synchronize()
            return e0.elapsed_time(e1) * 1e-3

        for _ in range(steps):
            for g in range(n):
                t_short = batch(g, long, short)
                t_long = batch(g, 0, long)
                per[g].append((t_long - t_short) / (long - short))
        return per


CALIBRATION_BYTES = 256 << 20


def calibration_kernel(torch, nbytes=CALIBRATION_BYTES, reps=3):
    """A plain elementwise kernel of known traffic (fp16 negation: reads and
    writes nbytes each), for scaling the HBM traffic counters (FETCH_SIZE,
    WRITE_SIZE) of the profiled kernels."""
    a = torch.ones(nbytes // 2, dtype=torch.float16, device="cuda:0")
    b = torch.empty_like(a)
    torch.cuda.synchronize()
    for _ in range(reps):
        torch.neg(a, out=b)
    torch.cuda.synchronize()
    del a, b


def source_hash():
    h = hashlib.sha256()
    csrc = os.path.join(ROOT, "paper_2605_04084_amd", "csrc")
    for f in sorted(os.listdir(csrc)):
        with open(os.path.join(csrc, f), "rb") as fh:
            h.update(f.encode())
            h.update(fh.read())
    return h.hexdigest()[:16]


# ---------------------------------------------------------------------------
# Counter passes.  `--pmc-pass MANIFEST` runs a short fixed launch sequence
# (a calibration kernel of known traffic, then PMC_REPS cold launches of every
# launch of the counter workloads below) under one `rocprofv3 --pmc` run per
# counter group; `--pmc-report MANIFEST OUT_DIR PASS_DIR...` maps the
# dispatches of all passes back onto the manifest and writes
# profiles/counters.json (keyed to the kernel sources) and one Markdown
# summary per kernel family.
# ---------------------------------------------------------------------------

PMC_REPS = 4
COUNTERS_PATH = os.path.join(ROOT, "profiles", "counters.json")
# variant builds (python -m paper_2605_04084_amd._build -D ... --out LIB) by library file name
VARIANT_DEFINES = {"libfasq_decode_mfma.so": ["FASQ_DECODE_DOT=0"]}

# rocprofv3 --pmc groups, one run each (within the per-block limits: at most
# 8 SQ, 4 TCC, 4 TCP, 2 GRBM counters per run).
PMC_GROUPS = {
    "fetch": ["FETCH_SIZE"],
    "write": ["WRITE_SIZE"],
    "lds": ["SQ_INSTS_LDS", "SQ_LDS_BANK_CONFLICT", "SQ_LDS_ADDR_CONFLICT", "SQ_ACTIVE_INST_LDS",
            "SQ_WAIT_INST_LDS", "SQ_LDS_IDX_ACTIVE", "SQ_BUSY_CU_CYCLES", "SQ_WAVES", "GRBM_GUI_ACTIVE"],
    "alu": ["SQ_INSTS_VALU", "SQ_INSTS_MFMA", "SQ_VALU_MFMA_BUSY_CYCLES", "SQ_ACTIVE_INST_VALU",
            "SQ_INSTS_SALU", "SQ_INSTS_VMEM_RD", "SQ_INSTS_SMEM", "SQ_WAVE_CYCLES", "GRBM_GUI_ACTIVE"],
    "util": ["MfmaUtil", "LDSBankConflict", "VALUBusy"],
    "l2": ["TCC_HIT_sum", "TCC_MISS_sum", "TCC_REQ_sum", "TCC_TAG_STALL_sum",
           "TCP_TOTAL_CACHE_ACCESSES_sum", "TCP_TCC_READ_REQ_sum", "TCP_PENDING_STALL_CYCLES_sum",
           "TCP_TCR_TCP_STALL_CYCLES_sum"],
}

# Counter workloads: (set, workload, M, launch grouping).  Every launch of a
# set goes out PMC_REPS times on distinct copies.
PMC_SETS = (
    ("llama3_8b_4bit", "llama3_8b_4bit", 1),
    ("llama3_8b_3bit", "llama3_8b_3bit", 1),
    ("qwen3_8b_M1", "qwen3_8b_sweep", 1),
    ("qwen3_8b_M4", "qwen3_8b_sweep", 4),
    ("qwen3_8b_M16", "qwen3_8b_sweep", 16),
)
PMC_PREFILL = ((0, 128), (0, 2048), (1, 2048), (2, 512))  # (prefill matrix, M)


def _ids_of(p):
    return p.N * (p.K // p.d)


def pmc_pass(torch, fasq, pi, manifest_path):
    """The calibration kernel, then PMC_REPS cold launches of every launch of
    the counter workloads, in order.  Writes the launch manifest."""
    calibration_kernel(torch)
    stream = torch.cuda.current_stream().cuda_stream
    seq = []
    for set_name, wl_name, M in PMC_SETS:
        wl = pi.workload(wl_name)
        problems = [wl.problem(i, M=M) for i in range(len(wl.matrices))]
        names = [m.name for m in wl.matrices]
        ms = MatrixSet(torch, fasq, problems, names, launch_groups(names), min_copies=PMC_REPS)
        torch.cuda.synchronize()
        for g in range(len(ms.groups)):
            for r in range(PMC_REPS):
                ms.launch(r % ms.copies, g, stream)
            torch.cuda.synchronize()
            ps = [problems[i] for i in ms.groups[g]]
            seq.append(dict(set=set_name, name=ms.group_name(g), reps=PMC_REPS, bytes=ms.group_bytes(g),
                            kernel=ms.group_kernel(g), M=M, K=ps[0].K, N=[p.N for p in ps],
                            ids=sum(_ids_of(p) for p in ps), flops=sum(2 * p.M * p.N * p.K for p in ps)))
        del ms
        torch.cuda.empty_cache()
    wl = pi.workload("prefill")
    dev = torch.device("cuda:0")
    for i, M in PMC_PREFILL:
        p = wl.problem(i, M=M)
        x, idx, cb = (torch.from_numpy(a).to(dev) for a in (p.x, p.idx, p.codebook))
        y = torch.empty((M, p.N), dtype=torch.float16, device=dev)
        need = fasq.gemm_ex_workspace_bytes(M, p.K, p.N, p.idx_bits, p.d, p.C)
        ws = torch.empty(max(need, 4), dtype=torch.uint8, device=dev)
        torch.cuda.synchronize()
        for r in range(PMC_REPS):
            st = fasq.gemm_ex_raw(x.data_ptr(), M, p.K, p.N, idx.data_ptr(), p.idx_bits, p.d, cb.data_ptr(), p.C,
                                  y.data_ptr(), ws.data_ptr(), need, stream)
            assert st == 0, fasq.last_error()
        torch.cuda.synchronize()
        seq.append(dict(set="prefill", name=f"{wl.matrices[i].name} M={M}", reps=PMC_REPS,
                        bytes=gemv_bytes(M, p.K, p.N, p.d, p.C, p.idx_bits),
                        kernel=fasq.plan("gemm", M, p.K, p.N, p.idx_bits, p.d, p.C), M=M, K=p.K, N=[p.N],
                        ids=_ids_of(p), flops=2 * M * p.N * p.K, k_split=need // (M * p.N * 4) if need else 1))
        del x, idx, cb, y, ws
    torch.cuda.empty_cache()
    with open(manifest_path, "w") as f:
        json.dump(dict(source_hash=source_hash(), calibration_bytes=CALIBRATION_BYTES, launches=seq,
                       lib=os.path.relpath(fasq.LIB_PATH, ROOT)), f, indent=1)
    log(f"[bench] pmc pass: {len(seq)} launches x {PMC_REPS}, manifest {manifest_path}")


def _read_counter_rows(pass_dir):
    """{dispatch id: (kernel name, start, end, {counter: value})} of one pass."""
    import csv
    import glob

    files = [pass_dir] if os.path.isfile(pass_dir) else sorted(
        glob.glob(os.path.join(pass_dir, "**", "*counter_collection.csv"), recursive=True))
    if not files:
        raise SystemExit(f"no counter_collection.csv under {pass_dir}")
    out = {}
    for fn in files:
        with open(fn) as f:
            for r in csv.DictReader(f):
                d = out.setdefault(int(r["Dispatch_Id"]), [r["Kernel_Name"], int(r["Start_Timestamp"]),
                                                           int(r["End_Timestamp"]), {}])
                d[3][r["Counter_Name"]] = d[3].get(r["Counter_Name"], 0.0) + float(r["Counter_Value"])
    return out


def _short_kernel(name):
    """'k_gemv_m1' from 'void fasq::k_gemv_m1<8, 2, 2, 0, false>(fasq::GemvM1Args)'."""
    i = name.find("fasq::")
    rest = name[i + 6:] if i >= 0 else name
    return rest.split("<")[0].split("(")[0]


def _pass_launches(rows, man):
    """Counter sums of every manifest launch (all its dispatches, averaged over
    its reps), the calibration counters, and the main kernel's mean duration."""
    disp = sorted(rows.items())
    cal = [v for _, v in disp if "neg" in v[0]]
    ours = [v for _, v in disp if "fasq::" in v[0]]
    pos = 0
    res = []
    for e in man["launches"]:
        base = e["kernel"].split("<")[0]
        sums, durs = {}, []
        for _ in range(e["reps"]):
            if pos >= len(ours) or _short_kernel(ours[pos][0]) != base:
                got = _short_kernel(ours[pos][0]) if pos < len(ours) else "nothing"
                raise SystemExit(f"dispatch {pos}: expected {base} for {e['set']}/{e['name']}, found {got}")
            durs.append(ours[pos][2] - ours[pos][1])
            while True:  # the main kernel and any helper kernels it queues (e.g. a split-K sum)
                for c, v in ours[pos][3].items():
                    sums[c] = sums.get(c, 0.0) + v
                pos += 1
                if pos >= len(ours) or _short_kernel(ours[pos][0]) == base or \
                        not _short_kernel(ours[pos][0]).startswith(("k_gemm_split_reduce", "k_sub_reduce")):
                    break
        res.append(({c: v / e["reps"] for c, v in sums.items()}, float(np.median(durs)) * 1e-3))
    if pos != len(ours):
        raise SystemExit(f"{len(ours) - pos} library dispatches left over after the manifest")
    calc = {}
    for v in cal:
        for c, x in v[3].items():
            calc.setdefault(c, []).append(x)
    return res, {c: float(np.median(x)) for c, x in calc.items()}


def pmc_report(manifest_path, out_dir, pass_dirs):
    with open(manifest_path) as f:
        man = json.load(f)
    launches = [dict(e, counters={}, counter_us={}) for e in man["launches"]]
    factors = {}
    for d in pass_dirs:
        res, cal = _pass_launches(_read_counter_rows(d), man)
        for (cnt, us), L in zip(res, launches):
            L["counters"].update(cnt)
            for c in cnt:
                L["counter_us"][c] = us
        for c in ("FETCH_SIZE", "WRITE_SIZE"):
            if c in cal:  # KiB the counter reads per byte the calibration kernel moves
                factors[c] = cal[c] * 1024.0 / man["calibration_bytes"]
    for L in launches:
        c = L["counters"]
        der = {}
        if "FETCH_SIZE" in c and "WRITE_SIZE" in c and factors:
            hbm = c["FETCH_SIZE"] * 1024.0 / factors["FETCH_SIZE"] + c["WRITE_SIZE"] * 1024.0 / factors["WRITE_SIZE"]
            der["hbm_bytes"] = hbm
            der["traffic_over_algorithmic"] = hbm / L["bytes"]
        if c.get("SQ_INSTS_LDS"):
            der["lds_bank_conflict_cycles_per_lds_inst"] = c.get("SQ_LDS_BANK_CONFLICT", 0.0) / c["SQ_INSTS_LDS"]
        for k, name in (("SQ_INSTS_VALU", "valu"), ("SQ_INSTS_MFMA", "mfma"), ("SQ_INSTS_LDS", "lds"),
                        ("SQ_INSTS_VMEM_RD", "vmem_rd"), ("SQ_INSTS_SALU", "salu")):
            if k in c:  # wave instructions x 64 lanes, per id
                der[f"{name}_lane_insts_per_id"] = c[k] * 64.0 / L["ids"]
        for k in ("MfmaUtil", "LDSBankConflict", "VALUBusy"):
            if k in c:
                der[k] = c[k]
        if "TCC_HIT_sum" in c and "TCC_MISS_sum" in c and c["TCC_HIT_sum"] + c["TCC_MISS_sum"] > 0:
            der["l2_hit_pct"] = 100.0 * c["TCC_HIT_sum"] / (c["TCC_HIT_sum"] + c["TCC_MISS_sum"])
        for k, name in (("TCC_REQ_sum", "l2_requests"), ("TCP_TOTAL_CACHE_ACCESSES_sum", "l1_tag_accesses"),
                        ("TCP_TCC_READ_REQ_sum", "l1_to_l2_reads")):
            if k in c:
                der[f"{name}_per_id"] = c[k] / L["ids"]
        L["derived"] = der
    lib = man.get("lib", "paper_2605_04084_amd/libfasq.so")
    defines = [] if lib == "paper_2605_04084_amd/libfasq.so" else VARIANT_DEFINES.get(os.path.basename(lib), [])
    groups = [g for g, cs in PMC_GROUPS.items() if any(c in L["counters"] for L in launches for c in cs)]
    out = dict(source_hash=man["source_hash"], calibration_factors=factors, reps=PMC_REPS, lib=lib,
               defines=defines, groups=groups, launches={f"{L['set']}/{L['name']}": L for L in launches})
    os.makedirs(out_dir, exist_ok=True)
    with open(os.path.join(out_dir, "counters.json"), "w") as f:
        json.dump(out, f, indent=1)
        f.write("\n")
    for L in launches:
        d = L["derived"]
        log(f"{L['set'] + '/' + L['name']:40s} {L['kernel']:36s} " +
            " ".join(f"{k}={v:.3g}" for k, v in d.items()))


# Markdown summaries of counters.json, one per counter set family.
PMC_MD_FILES = (
    ("k_gemv_m1_llama3_8b_4bit_counters.md", ("llama3_8b_4bit",),
     "k_gemv_m1: Llama-3-8B decode layer at effective 4 bits (d = 2, C = 256, 8-bit ids, M = 1)"),
    ("k_gemv_m1_llama3_8b_3bit_counters.md", ("llama3_8b_3bit",),
     "k_gemv_m1: Llama-3-8B decode layer at effective 3 bits, lm_head included (d = 4, C = 4096, 12-bit ids, M = 1)"),
    ("decode_qwen3_8b_counters.md", ("qwen3_8b_M1", "qwen3_8b_M4", "qwen3_8b_M16"),
     "Qwen3-8B decode layer, 65536-entry codebooks larger than LDS (d = 4, 16-bit ids), M = 1, 4, 16"),
    ("k_gemm_mfma_prefill_counters.md", ("prefill",),
     "k_gemm_mfma: prefill GEMM (d = 4, C = 256, 8-bit ids) on Llama-3-8B shapes"),
)

PMC_MD_DERIVED = (
    ("traffic_over_algorithmic", "HBM / algorithmic bytes", "{:.2f}"),
    ("lds_bank_conflict_cycles_per_lds_inst", "LDS conflict cycles / LDS inst", "{:.2f}"),
    ("LDSBankConflict", "LDS conflict % of time", "{:.1f}"),
    ("valu_lane_insts_per_id", "VALU / id", "{:.2f}"),
    ("mfma_lane_insts_per_id", "MFMA / id", "{:.3f}"),
    ("lds_lane_insts_per_id", "LDS / id", "{:.2f}"),
    ("VALUBusy", "VALU busy %", "{:.1f}"),
    ("MfmaUtil", "MFMA busy %", "{:.1f}"),
    ("l2_hit_pct", "L2 hit %", "{:.1f}"),
    ("l2_requests_per_id", "L2 requests / id", "{:.3f}"),
    ("l1_tag_accesses_per_id", "L1 tag accesses / id", "{:.3f}"),
)


def pmc_markdown(counters_path, out_dir, variant=None):
    """One Markdown summary per counter family.  `variant` names a variant
    build (bench.py --lib) whose counters these are: its summaries go to
    files tagged with it."""
    with open(counters_path) as f:
        data = json.load(f)
    groups_run = PMC_GROUPS if variant is None else {g: PMC_GROUPS[g] for g in data.get("groups", PMC_GROUPS)}
    lib = "" if variant is None else f" --lib {data.get('lib', 'LIB')}"
    build = "" if variant is None else (f"python3 -m paper_2605_04084_amd._build {' '.join('-D ' + d for d in data.get('defines', []))} "
                                        f"--out {data.get('lib', 'LIB')}\n")
    groups = "\n".join(f"timeout -s KILL 300 rocprofv3 --pmc {' '.join(cs)} --output-format csv -d gpurun_out/pmc_{g} "
                       f"-o run -- \\\n    python3 bench.py{lib} --pmc-pass gpurun_out/pmc_manifest.json"
                       for g, cs in groups_run.items())
    groups = build + groups
    report = ("python3 bench.py --pmc-report gpurun_out/pmc_manifest.json gpurun_out/counters " +
              " ".join(f"gpurun_out/pmc_{g}" for g in groups_run) +
              f"\npython3 bench.py --pmc-markdown gpurun_out/counters/counters.json profiles" +
              ("" if variant is None else f" {variant}"))
    fac = data.get("calibration_factors", {})
    for fname, sets, title in PMC_MD_FILES:
        rows = [(k, e) for k, e in data["launches"].items() if e["set"] in sets]
        if not rows:
            continue
        if variant is not None:
            fname = fname.replace("_counters.md", f"_{variant}_counters.md")
            title = f"{title}, variant build {variant} ({', '.join(data.get('defines', []))})"
        lines = [f"# {title}: rocprofv3 counters", "",
                 "Commands (from the repository root on one MI355X; one `rocprofv3 --pmc` run per counter group, "
                 "each over the same fixed launch sequence):", "", "```", "export TMPDIR=/tmp", groups, report, "```",
                 "",
                 f"Every launch below ran {data.get('reps', PMC_REPS)} times on distinct cold copies of its "
                 "operands; values are means per launch.  SQ instruction counters count wave instructions; "
                 "\"per id\" columns are wave instructions x 64 lanes / codeword ids of the launch (lane "
                 "instructions per id), or L2 / L1 requests per id.  HBM bytes are FETCH_SIZE and WRITE_SIZE "
                 "scaled by what they read for a 256 MiB fp16 negation (factors "
                 + ", ".join(f"{k} {v:.4f}" for k, v in fac.items()) + "); FETCH_SIZE counts every L2 miss, "
                 "so a line served by the Infinity Cache counts as HBM traffic here.  MfmaUtil, LDSBankConflict "
                 "and VALUBusy are rocprofv3's derived percentages of GPU time.",
                 "", f"Kernel sources hash: `{data['source_hash']}` (bench.py uses these counters only while the "
                 "sources match).", ""]
        hdr = "| Launch | Kernel | µs (counter run) | " + " | ".join(h for _, h, _ in PMC_MD_DERIVED) + " |"
        lines += [hdr, "|" + "---|" * 3 + "---:|" * len(PMC_MD_DERIVED)]
        for k, e in rows:
            d = e["derived"]
            us = next(iter(e.get("counter_us", {}).values()), float("nan"))
            cells = [fmt.format(d[key]) if key in d else "—" for key, _, fmt in PMC_MD_DERIVED]
            lines.append(f"| {k} | `{e['kernel']}` | {us:.1f} | " + " | ".join(cells) + " |")
        lines += ["", "Raw counters (mean per launch):", ""]
        names = sorted({c for _, e in rows for c in e["counters"]})
        lines += ["| Launch | " + " | ".join(names) + " |", "|---|" + "---:|" * len(names)]
        for k, e in rows:
            lines.append(f"| {k} | " + " | ".join(f"{e['counters'][c]:.4g}" if c in e["counters"] else "—"
                                                     for c in names) + " |")
        lines += ["", "Algorithmic bytes, ids and flops per launch:", "",
                  "| Launch | Algorithmic bytes | HBM bytes (counters) | ids | flops |", "|---|---:|---:|---:|---:|"]
        for k, e in rows:
            hb = e["derived"].get("hbm_bytes")
            lines.append(f"| {k} | {e['bytes']} | {hb:.0f} | {e['ids']} | {e['flops']} |" if hb is not None else
                         f"| {k} | {e['bytes']} | — | {e['ids']} | {e['flops']} |")
        with open(os.path.join(out_dir, fname), "w") as f:
            f.write("\n".join(lines) + "\n")
        log(f"[bench] wrote {os.path.join(out_dir, fname)}")


def trace_markdown(trace_dir, bench_json, out_path):
    """The kernel-statistics summary of a `rocprofv3 --kernel-trace --stats`
    run of the default bench (without the CPU leg), with the agreement between
    the profiler's durations and bench.py's HIP-event figures."""
    import csv
    import glob

    def one(pattern):
        files = sorted(glob.glob(os.path.join(trace_dir, "**", pattern), recursive=True))
        if not files:
            raise SystemExit(f"no {pattern} under {trace_dir}")
        with open(files[0]) as f:
            return list(csv.DictReader(f))

    stats = one("*kernel_stats.csv")
    trace = sorted(one("*kernel_trace.csv"), key=lambda r: int(r["Dispatch_Id"]))
    with open(bench_json) as f:
        bt = json.load(f)

    def short(name):
        """Kernel name without namespaces and arguments; plain (mangled)
        names of non-template kernels are cut down to their identifier."""
        m = re.match(r"_ZN4fasq(?:12_GLOBAL__N_1)?(\d+)", name)
        if m:
            n = int(m.group(1))
            return name[m.end():m.end() + n]
        name = name.replace("void ", "").replace("fasq::", "").replace("(anonymous namespace)::", "")
        return name.split("(")[0].replace("false", "0").replace("true", "1")

    lines = ["# libfasq kernels: rocprofv3 kernel statistics of the default bench.py run", "",
             "Command (from the repository root, on one MI355X):", "", "```", "export TMPDIR=/tmp",
             "rocprofv3 --kernel-trace --stats --output-format csv -d gpurun_out/prof -o run -- \\",
             "    python3 bench.py --no-cpu --out gpurun_out/bench_under_trace.json",
             f"python3 bench.py --trace-markdown gpurun_out/prof gpurun_out/bench_under_trace.json {out_path}",
             "```", "",
             "The profiled run is the default bench without the CPU oracle leg: the Llama-3-8B decode layers at "
             "effective 4 bits (M = 1 and 2) and 3 bits (lm_head included), the prefill GEMM, the Qwen3-8B decode "
             "layer at M = 1, 4, 16, the batch-size crossover and the sensitivity points.  Only library kernels "
             "are listed.", "",
             "| Kernel | Calls | Average µs | Min µs | Max µs |", "|---|---:|---:|---:|---:|"]
    avg = {}
    for r in stats:
        if "fasq::" not in r["Name"] and not r["Name"].startswith("_ZN4fasq"):
            continue
        avg[short(r["Name"])] = float(r["AverageNs"]) / 1e3
        lines.append(f"| `{short(r['Name'])}` | {r['Calls']} | {float(r['AverageNs']) / 1e3:.3f} | "
                     f"{float(r['MinNs']) / 1e3:.3f} | {float(r['MaxNs']) / 1e3:.3f} |")
    rl = bt["roofline"]
    dom, on = rl["kernel"].split(" on ")
    lines += ["", f"Dominant kernel of the decode layer: `{dom}` ({on}).", "",
              f"- bench.py, HIP events in the same profiled run: {rl['us_per_launch']:.3f} µs per launch "
              "(mean over its launches)",
              f"- rocprofv3 average over every launch of that kernel in the run: {avg.get(dom, float('nan')):.3f} µs "
              "(this average also takes in the eager warm-up launches and every other workload that maps to the "
              "same instantiation)", ""]
    tab = bt["launch_table"]
    nl = len(tab)
    lpg = int(bt["layers_per_graph"])
    kern = {r["kernel"] for r in tab}
    g = [r for r in trace if short(r["Kernel_Name"]) in kern]
    dur = np.array([(int(r["End_Timestamp"]) - int(r["Start_Timestamp"])) / 1e3 for r in g])
    # the layer's launches come first, in this order: the eager warm-up (one
    # layer per copy), the warm-up list (max(warmup, 1) layers), the timed
    # list (steps layers), the warm-up graph replays (at least warmup layers,
    # whole graphs of lpg layers) and the timed graph replays (steps layers)
    W, K = bt["warmup"], bt["steps"]
    lw, gw = max(W, 1), max(1, -(-W // lpg)) * lpg
    seg = {"list": bt["config"]["rotation_copies"] + lw}
    seg["graph"] = seg["list"] + K + gw
    nlay = seg["graph"] + K
    if dur.size >= nlay * nl:
        D = dur[:nlay * nl].reshape(nlay, nl)
        lines += ["Per launch of the effective-4-bit layer (M = 1): rocprofv3 median duration over the eager "
                  "warm-up, the launch lists and the graph replays, against bench.py's HIP events:", "",
                  "| Launch | rows (N) × K | rocprofv3 median µs | bench.py µs (events) |", "|---|---|---:|---:|"]
        for j, m in enumerate(tab):
            lines.append(f"| {m['name']} | {'+'.join(str(n) for n in m['N'])} × {m['K']} | "
                         f"{np.median(D[:, j]):.2f} | {m['us_median']:.2f} |")
        dj = [j for j, m in enumerate(tab) if m["kernel"] == dom]
        if dj:
            lines += ["", f"The dominant kernel over its launches in this layer ({', '.join(tab[j]['name'] for j in dj)}): "
                      f"rocprofv3 {np.mean([np.median(D[:, j]) for j in dj]):.3f} µs per launch (mean of the "
                      f"per-launch medians) against bench.py's {rl['us_per_launch']:.3f} µs."]
        starts = np.array([int(r["Start_Timestamp"]) for r in g[:nlay * nl]], dtype=np.float64)
        ends = np.array([int(r["End_Timestamp"]) for r in g[:nlay * nl]], dtype=np.float64)

        def gaps_of(first_layer, layers, per):
            """Gaps between consecutive kernels of `layers` layers from
            `first_layer`, within runs of `per` layers (one graph or list)."""
            out = []
            for k in range(layers // per):
                a = (first_layer + k * per) * nl
                out.extend((starts[a + 1:a + per * nl] - ends[a:a + per * nl - 1]) / 1e3)
            return np.array(out)

        lg = gaps_of(seg["list"], K, K)
        a, b = seg["list"] * nl, (seg["list"] + K) * nl
        lines += ["", f"Gap between consecutive kernels inside the timed launch-list run ({lg.size} gaps): "
                  f"median {np.median(lg):.2f} µs, mean {lg.mean():.2f} µs, max {lg.max():.2f} µs; the run "
                  f"spans {(ends[b - 1] - starts[a]) / 1e3 / K:.2f} µs per layer from the first kernel's start "
                  f"to the last kernel's end.  Kernel tracing intercepts every hipLaunchKernel, which slows the "
                  f"host's issue of the list's launches below the GPU's pace (bench.py under the profiler: "
                  f"{bt['us_per_layer']:.2f} µs per layer from the list, {bt['us_per_layer_graph']:.2f} from the "
                  f"graphs); the graph's launches go out in one call.  The untraced figures are in the bench "
                  f"record."]
        gg = gaps_of(seg["graph"], K, lpg)
        if gg.size:
            lines += ["", f"Gap between the end of one kernel and the start of the next inside the timed graph "
                      f"replays ({gg.size} gaps): median {np.median(gg):.2f} µs, mean {gg.mean():.2f} µs, "
                      f"max {gg.max():.2f} µs."]
    with open(out_path, "w") as f:
        f.write("\n".join(lines) + "\n")
    log(f"[bench] wrote {out_path}")


def load_counters():
    """counters.json if it was taken on the current kernel sources, else None."""
    if not os.path.exists(COUNTERS_PATH):
        return None
    try:
        with open(COUNTERS_PATH) as f:
            data = json.load(f)
    except (OSError, ValueError):
        return None
    return data if data.get("source_hash") == source_hash() else None


def load_traffic(kernel, set_name, names):
    """Mean HBM bytes per launch of `kernel` over the launches `names` of
    counter set `set_name`; None unless the counters were taken on the
    current kernel sources."""
    data = load_counters()
    if data is None:
        return None
    vals = []
    for n in names:
        e = data["launches"].get(f"{set_name}/{n}")
        if e is None or e.get("kernel") != kernel or "hbm_bytes" not in e.get("derived", {}):
            return None
        vals.append(e["derived"]["hbm_bytes"])
    return float(np.mean(vals))


def decode_roofline(res, set_name):
    """The HBM roofline of a decode layer's dominant kernel: the
    instantiation with the largest share of the layer's kernel time
    (launches that map to the same instantiation are pooled), algorithmic
    bytes per launch over its mean launch time, and the counter traffic of
    the same launches (counter set `set_name`) when the counters match the
    sources."""
    pools = {}
    for r in res["launch_table"]:
        g = pools.setdefault(r["kernel"], dict(us=0.0, bytes=0, n=0, names=[]))
        g["us"] += r["us_median"]
        g["bytes"] += r["bytes"]
        g["n"] += 1
        g["names"].append(r["name"])
    dom_kernel, dom = max(pools.items(), key=lambda kv: kv[1]["us"])
    achieved = (dom["bytes"] / dom["n"]) / (dom["us"] / dom["n"] * 1e-6) / 1e9
    return dict(bound="hbm", achieved=achieved, peak=HBM_PEAK_GBS, unit="GB/s", frac=achieved / HBM_PEAK_GBS,
                traffic=None if set_name is None else load_traffic(dom_kernel, set_name, dom["names"]),
                kernel=f"{dom_kernel} on {', '.join(dom['names'])}",
                bytes_per_launch=dom["bytes"] / dom["n"], us_per_launch=dom["us"] / dom["n"])


# ---------------------------------------------------------------------------
# Workload runners
# ---------------------------------------------------------------------------

def decode_layer(torch, fasq, pi, wl_name, steps, warmup, M=1, include=None, grouped=True):
    wl = pi.workload(wl_name)
    mats = list(range(len(wl.matrices))) if include is None else include
    log(f"[bench] {wl_name} M={M}: generating {len(mats)} matrices")
    problems = [wl.problem(i, M=M) for i in mats]
    names = [wl.matrices[i].name for i in mats]
    groups = launch_groups(names) if grouped else None
    # Consecutive layers go into one graph, as a decode step replays every
    # layer of the model from one graph: the graph launch boundary is paid
    # once per lpg layers, lpg the largest divisor of the step count that is
    # at most MODEL_LAYERS.  Each layer of a graph reads its own copy.
    lpg = max(k for k in range(1, min(steps, MODEL_LAYERS) + 1) if steps % k == 0)
    ms = MatrixSet(torch, fasq, problems, names, groups, min_copies=max(TIMING_COPIES, lpg))
    log(f"[bench] {wl_name}: {ms.bytes_per_set / 1e6:.1f} MB per layer, {ms.copies} copies, "
        f"{len(ms.groups)} launches, {lpg} layers per graph")
    graphs = ms.capture_graphs(lpg)  # launches every copy once, in order, before capturing
    stream = torch.cuda.current_stream()
    C = ms.copies
    # Copies are read in order, cyclically, by everything below: each read of
    # a copy comes C layers (at least 1 GiB) after its previous read, far more
    # than the 256 MB MALL holds.  `nxt` is the next copy to read.
    nxt = 0

    def record(first, count):
        lst = fasq.LaunchList()
        with lst:
            for k in range(count):
                ms.launch_all((first + k) % C, stream.cuda_stream)
        return lst

    # The timed region: launch lists (fasq_launch_list_*), the launches
    # recorded once through the same calls, then queued by the library with
    # one hipLaunchKernel each.  `warmup` layers from a warm-up list, then the
    # timed list of `steps` layers.  Events on the stream beside the wall
    # clock show how much of the wall time is the host's start of the run;
    # the first is recorded just before the clock starts (it queues no work
    # and its host call is not part of a step).
    lwarm = max(warmup, 1)
    warm_list, timed_list = record(nxt, lwarm), record(nxt + lwarm, steps)
    nxt = (nxt + lwarm + steps) % C
    warm_list.run(stream)
    torch.cuda.synchronize()
    ev4, ev5 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    ev4.record(stream)
    t0 = time.perf_counter()
    timed_list.run(stream)
    ev5.record(stream)
    torch.cuda.synchronize()
    wall_list = time.perf_counter() - t0
    gpu_list = ev4.elapsed_time(ev5) * 1e-3
    warm_list.close()
    timed_list.close()
    # The same layers from HIP graphs, reported beside it: graph c replays
    # copies c .. c + lpg - 1; warm-up replays covering at least `warmup`
    # layers, then steps / lpg timed replays.
    gwarm = max(1, -(-warmup // lpg))
    for r in range(gwarm):
        graphs[(nxt + r * lpg) % C].replay()
    nxt = (nxt + gwarm * lpg) % C
    torch.cuda.synchronize()
    ev0, ev1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    ev0.record(stream)
    t0 = time.perf_counter()
    for r in range(steps // lpg):
        graphs[(nxt + r * lpg) % C].replay()
    ev1.record(stream)
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    gpu_graph = ev0.elapsed_time(ev1) * 1e-3
    nxt = (nxt + steps) % C
    del graphs
    # The same layers launched eagerly, back to back behind a spin kernel
    # (the host's launches run ahead of the GPU): the GPU time without the
    # graph, from events on the stream.  Reported beside the graph figure.
    ev2, ev3 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    eager_layers = min(steps, C)
    torch.cuda._sleep(SPACER_CYCLES * 4)
    ev2.record(stream)
    for k in range(eager_layers):
        ms.launch_all((nxt + k) % C, stream.cuda_stream)
    ev3.record(stream)
    torch.cuda.synchronize()
    eager = ev2.elapsed_time(ev3) * 1e-3 / eager_layers
    per = ms.time_kernels(max(steps // 2, 10))
    med = [max(float(np.median(v)), 1e-7) for v in per]
    mean = [max(float(np.mean(v)), 1e-7) for v in per]
    rows = []
    for g, (tm, ta) in enumerate(zip(med, mean)):
        b = ms.group_bytes(g)
        ps = [problems[i] for i in ms.groups[g]]
        rows.append(dict(name=ms.group_name(g), N=[p.N for p in ps], K=ps[0].K, kernel=ms.group_kernel(g),
                         bytes=b, us_median=tm * 1e6, us_mean=ta * 1e6,
                         gbs=b / tm / 1e9, pct_hbm=100.0 * b / tm / 1e9 / HBM_PEAK_GBS))
    step_bytes = sum(r["bytes"] for r in rows)
    res = dict(workload=wl_name, M=M, bytes_per_layer=step_bytes, copies=ms.copies, launches=len(rows),
               layers_per_graph=lpg,
               wall_s=wall_list, steps=steps, us_per_layer_list=wall_list / steps * 1e6,
               us_per_layer_list_events=gpu_list / steps * 1e6,
               wall_graph_s=wall, us_per_layer_graph=wall / steps * 1e6,
               us_per_layer_graph_events=gpu_graph / steps * 1e6, us_per_layer_eager_events=eager * 1e6,
               us_per_layer_kernel_sum=sum(med) * 1e6, launch_table=rows)
    res["gbs_list"] = step_bytes * steps / wall_list / 1e9
    res["gbs_graph"] = step_bytes * steps / wall / 1e9
    res["gbs_kernel_sum"] = step_bytes / sum(med) / 1e9
    del ms
    torch.cuda.empty_cache()
    return res


# ---------------------------------------------------------------------------
# Sensitivity sweeps on one 4096 x 4096 layer (the paper's Fig. sensitivity):
# codebook size, sub-vector length, batch size (GEMV against GEMM: the
# dispatch crossover of fasq_pq_linear) and prefill length.  Every launch
# reads cold copies, as in the decode timing.
# ---------------------------------------------------------------------------

SENS_N = SENS_K = 4096


def time_single(torch, fasq, p, regime, steps=10):
    """Median per-launch seconds of one PQ problem (cold rotated copies)."""
    ms = MatrixSet(torch, fasq, [p], ["m"], min_copies=TIMING_COPIES, regime=regime)
    for c in range(ms.copies):
        ms.launch_all(c, torch.cuda.current_stream().cuda_stream)
    torch.cuda.synchronize()
    t = max(float(np.median(ms.time_kernels(steps)[0])), 1e-7)
    kernel = ms.group_kernel(0)
    del ms
    return t, kernel


def time_per_subspace(torch, fasq, pi, rng, d=2, C=256, bits=8, M=1, steps=10, short=2, long=10):
    """fasq_pq_gemv_ex with one codebook per subspace (the paper's general
    form; its sensitivity layer is 4096 x 4096 at d = 2, K_s = 256) at M
    tokens, over rotated cold copies; the call is two kernels (the K-split
    partials and their sum)."""
    S = SENS_K // d
    books = pi.draw_codebook(rng, S * C, d).reshape(S, C, d)
    ids = pi.draw_ids(rng, SENS_N, S, C)
    idx = pi.pack_indices(ids, bits)
    x = pi.draw_x(rng, M, SENS_K)
    dev = torch.device("cuda:0")
    nbytes = idx.nbytes + books.nbytes + x.nbytes + M * SENS_N * 2
    copies = max(short + long, math.ceil(ROTATION_BYTES / nbytes) + 1)
    ws_bytes = fasq.gemv_ex_workspace_bytes(M, SENS_K, SENS_N, bits, d, C, C * d)
    base = [torch.from_numpy(a).to(dev) for a in (x, idx, books)]
    sets = [[t.clone() for t in base] + [torch.empty((M, SENS_N), dtype=torch.float16, device=dev),
                                         torch.zeros(max(ws_bytes, 4), dtype=torch.uint8, device=dev)]
            for _ in range(copies)]
    stream = torch.cuda.current_stream()

    def launch(c):
        xs, ids_d, bk, y, ws = sets[c]
        st = fasq.gemv_ex_raw(xs.data_ptr(), M, SENS_K, SENS_N, ids_d.data_ptr(), bits, d, bk.data_ptr(), C, C * d,
                              y.data_ptr(), ws.data_ptr(), ws_bytes, stream.cuda_stream)
        assert st == 0, fasq.last_error()

    for c in range(copies):
        launch(c)
    torch.cuda.synchronize()

    def batch(first, count):
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        torch.cuda._sleep(SPACER_CYCLES)
        e0.record(stream)
        for j in range(count):
            launch(first + j)
        e1.record(stream)
        e1.synchronize()
        return e0.elapsed_time(e1) * 1e-3

    t = max(float(np.median([(batch(0, long) - batch(long, short)) / (long - short) for _ in range(steps)])), 1e-7)
    del sets, base
    torch.cuda.empty_cache()
    log(f"[bench] sensitivity per-subspace codebooks (4096 x 4096, d={d}, C={C}, M={M}): {t * 1e6:.2f} us, "
        f"{nbytes / t / 1e9:.0f} GB/s (ids + books)")
    r = dict(d=d, C=C, idx_bits=bits, M=M, us=t * 1e6, bytes=nbytes, gbs=nbytes / t / 1e9, workspace_bytes=ws_bytes)
    if M == 1:
        r["paper_rtx3090_us"] = 32.0
    return r


def time_dense(torch, M, K, N, steps=10, short=2, long=10):
    """Median per-call seconds of torch.matmul on fp16 x [M x K] and W [K x N]
    (uncompressed weights), over rotated cold copies of W."""
    dev = torch.device("cuda:0")
    copies = max(short + long, math.ceil(ROTATION_BYTES / (K * N * 2)) + 1)
    ws = [(torch.randn((K, N), device=dev) * 0.02).to(torch.float16) for _ in range(copies)]
    x = torch.randn((M, K), device=dev).to(torch.float16)
    y = torch.empty((M, N), dtype=torch.float16, device=dev)
    stream = torch.cuda.current_stream()
    for w in ws:
        torch.matmul(x, w, out=y)

    def batch(first, count):
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        torch.cuda._sleep(SPACER_CYCLES)
        e0.record(stream)
        for j in range(count):
            torch.matmul(x, ws[first + j], out=y)
        e1.record(stream)
        e1.synchronize()
        return e0.elapsed_time(e1) * 1e-3

    per = [(batch(0, long) - batch(long, short)) / (long - short) for _ in range(steps)]
    del ws
    torch.cuda.empty_cache()
    return max(float(np.median(per)), 1e-7)


def sensitivity(torch, fasq, pi, core=False):
    """The paper's sensitivity sweeps (Sec. 4.4, Fig. sensitivity) on one
    4096 x 4096 layer.  core: the points the default run reports (codebook
    size 16 / 64 / 256, every sub-vector length, the L = 32 prefill, the
    per-subspace layer); the batch-size sweep is the crossover measurement."""
    out = dict(shape=f"{SENS_N}x{SENS_K}", codebook_size=[], subvector=[], batch=[], prefill=[])
    rng = np.random.default_rng(2026)

    def gemv_row(M, d, C, bits, regime="gemv"):
        p = pi.draw_problem(rng, M, SENS_K, SENS_N, d, C, bits)
        t, kern = time_single(torch, fasq, p, regime)
        b = gemv_bytes(M, SENS_K, SENS_N, d, C, bits)
        return dict(M=M, d=d, C=C, idx_bits=bits, regime=regime, us=t * 1e6, gbs=b / t / 1e9,
                    tflops=2.0 * M * SENS_N * SENS_K / t / 1e12, kernel=kern)

    out["per_subspace"] = time_per_subspace(torch, fasq, pi, rng)
    out["per_subspace_tokens"] = [time_per_subspace(torch, fasq, pi, rng, M=M) for M in (4, 16)]
    dense1 = time_dense(torch, 1, SENS_K, SENS_N)
    out["dense_fp16_gemv_us"] = dense1 * 1e6
    log(f"[bench] sensitivity: dense fp16 GEMV (torch.matmul, M=1) {dense1 * 1e6:.2f} us")
    for C in ((16, 64, 256) if core else (16, 32, 64, 128, 256)):
        r = gemv_row(1, 2, C, 8)
        out["codebook_size"].append(r)
        log(f"[bench] sensitivity C={C:4d} d=2: {r['us']:.2f} us ({r['gbs']:.0f} GB/s) {r['kernel']}")
    for d in (1, 2, 4, 8):
        r = gemv_row(1, d, 256, 8)
        out["subvector"].append(r)
        log(f"[bench] sensitivity d={d} C=256: {r['us']:.2f} us ({r['gbs']:.0f} GB/s) {r['kernel']}")
    for M in (() if core else (1, 2, 4, 8, 16, 32, 64, 128)):
        row = dict(M=M, dense_us=time_dense(torch, M, SENS_K, SENS_N) * 1e6)
        if M <= 16:
            row["gemv_us"] = gemv_row(M, 2, 256, 8)["us"]
        row["gemm_us"] = gemv_row(M, 2, 256, 8, regime="gemm")["us"]
        out["batch"].append(row)
        log(f"[bench] sensitivity batch M={M:3d}: gemv {row.get('gemv_us', float('nan')):8.2f} us, "
            f"gemm {row['gemm_us']:8.2f} us, dense fp16 {row['dense_us']:8.2f} us")
    for L in ((32,) if core else (32, 64, 128, 256, 512, 1024, 2048)):
        r = gemv_row(L, 2, 256, 8, regime="gemm")
        r["k_split_us"] = gemv_row(L, 2, 256, 8, regime="gemm_ex")["us"]
        r["dense_us"] = time_dense(torch, L, SENS_K, SENS_N) * 1e6
        if L in (32, 128, 512, 2048):  # the paper's lookup-table GEMM design (Alg. 3), for comparison
            r["lut_us"] = gemv_row(L, 2, 256, 8, regime="lut")["us"]
        out["prefill"].append(r)
        log(f"[bench] sensitivity prefill L={L:5d}: {r['us']:8.2f} us ({r['tflops']:.0f} TFLOP/s), "
            f"with K split {r['k_split_us']:8.2f} us, "
            f"dense fp16 {r['dense_us']:8.2f} us" + (f", lookup-table GEMM {r['lut_us']:9.2f} us" if "lut_us" in r else ""))
    torch.cuda.empty_cache()
    return out


CROSSOVER_M = (1, 2, 4, 8, 12, 16, 20, 24, 32, 48, 64)
CROSSOVER_MATS = (0, 1, 4, 6)  # q_proj, k_proj, gate_proj, down_proj of the Llama-3-8B layer


def crossover(torch, fasq, pi, Ms=CROSSOVER_M, steps=5, short=2, long=10):
    """Batch-size dispatch of the decode entry point (the paper leaves an
    adaptive GEMV/GEMM switch to future work, Sec. 4.4 "Batch size").

    On the four distinct Llama-3-8B layer shapes at effective 4 bits (d = 2,
    C = 256, 8-bit ids), per-call time of fasq_pq_gemv (the kernel its
    dispatch picks for M tokens) and of the prefill GEMM with its K split
    (fasq_pq_gemm_ex, workspace allocated outside the timed region), at every
    M in Ms.  The id table is read cold (rotated copies); x and y stay hot."""
    wl = pi.workload("llama3_8b_4bit")
    dev = torch.device("cuda:0")
    stream = torch.cuda.current_stream()
    out = []
    for i in CROSSOVER_MATS:
        spec = wl.matrices[i]
        p = wl.problem(i, M=max(Ms))
        copies = max(short + long, math.ceil(ROTATION_BYTES / p.idx.nbytes) + 1)
        base = torch.from_numpy(p.idx).to(dev)
        idxs = [base.clone() for _ in range(copies)]
        del base
        cb = torch.from_numpy(p.codebook).to(dev)
        x_all = torch.from_numpy(p.x).to(dev)
        y = torch.empty((max(Ms), p.N), dtype=torch.float16, device=dev)
        need_max = max(max(fasq.gemm_ex_workspace_bytes(M, p.K, p.N, p.idx_bits, p.d, p.C),
                           fasq.gemv_ex_workspace_bytes(M, p.K, p.N, p.idx_bits, p.d, p.C, 0)) for M in Ms)
        ws = torch.empty(max(need_max, 4), dtype=torch.uint8, device=dev)
        torch.cuda.synchronize()
        for M in Ms:
            x = x_all[:M]
            need = fasq.gemm_ex_workspace_bytes(M, p.K, p.N, p.idx_bits, p.d, p.C)

            need_ex = fasq.gemv_ex_workspace_bytes(M, p.K, p.N, p.idx_bits, p.d, p.C, 0)
            assert need_ex <= ws.numel()

            def call(regime, c):
                if regime == "gemv":
                    st = fasq.gemv_raw(x.data_ptr(), M, p.K, p.N, idxs[c].data_ptr(), p.idx_bits, p.d, cb.data_ptr(),
                                       p.C, y.data_ptr(), stream.cuda_stream)
                elif regime == "gemv_ex":
                    st = fasq.gemv_ex_raw(x.data_ptr(), M, p.K, p.N, idxs[c].data_ptr(), p.idx_bits, p.d,
                                          cb.data_ptr(), p.C, 0, y.data_ptr(), ws.data_ptr(), need_ex,
                                          stream.cuda_stream)
                else:
                    st = fasq.gemm_ex_raw(x.data_ptr(), M, p.K, p.N, idxs[c].data_ptr(), p.idx_bits, p.d,
                                          cb.data_ptr(), p.C, y.data_ptr(), ws.data_ptr(), need, stream.cuda_stream)
                assert st == 0, fasq.last_error()

            row = dict(name=spec.name, N=p.N, K=p.K, M=M)
            for regime in ("gemv", "gemv_ex", "gemm_ex"):
                for c in range(copies):
                    call(regime, c)

                def batch(first, count):
                    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
                    torch.cuda._sleep(SPACER_CYCLES)
                    e0.record(stream)
                    for j in range(count):
                        call(regime, (first + j) % copies)
                    e1.record(stream)
                    e1.synchronize()
                    return e0.elapsed_time(e1) * 1e-3

                t = [(batch(0, long) - batch(long, short)) / (long - short) for _ in range(steps)]
                row[f"{regime}_us"] = max(float(np.median(t)), 1e-7) * 1e6
            row["gemv_kernel"] = fasq.plan("gemv", M, p.K, p.N, p.idx_bits, p.d, p.C)
            row["gemm_kernel"] = fasq.plan("gemm", M, p.K, p.N, p.idx_bits, p.d, p.C)
            row["gemm_k_split"] = need // (M * p.N * 4) if need else 1
            row["gemv_ex_kernel"] = row["gemm_kernel"] if need_ex > 0 else row["gemv_kernel"]
            row["faster"] = "gemv" if row["gemv_us"] <= row["gemm_ex_us"] else "gemm_ex"
            out.append(row)
            log(f"[bench] crossover {spec.name:9s} M={M:3d}: fasq_pq_gemv {row['gemv_us']:7.2f} us "
                f"({row['gemv_kernel']}), fasq_pq_gemv_ex {row['gemv_ex_us']:7.2f} us "
                f"({row['gemv_ex_kernel']}), GEMM with K split {row['gemm_ex_us']:7.2f} us "
                f"(split {row['gemm_k_split']})")
        del idxs, cb, x_all, y, ws
        torch.cuda.empty_cache()
    return out


def tiny_latency(torch, fasq, pi, reps=200):
    """The tiny workload (M = 1, 128 x 256, d = 4, C = 256): a latency case.
    GPU: per-call time of back-to-back launches on the same (hot) operands;
    CPU: the fp64 oracle, median of 5."""
    from oracle import pq_oracle as orc

    p = pi.workload("tiny").problem(0)
    dev = torch.device("cuda:0")
    x, idx, cb = (torch.from_numpy(a).to(dev) for a in (p.x, p.idx, p.codebook))
    y = torch.empty((p.M, p.N), dtype=torch.float16, device=dev)
    stream = torch.cuda.current_stream()
    args = (x.data_ptr(), p.M, p.K, p.N, idx.data_ptr(), p.idx_bits, p.d, cb.data_ptr(), p.C, y.data_ptr(),
            stream.cuda_stream)
    assert fasq.gemv_raw(*args) == 0, fasq.last_error()

    def batch(count):
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        torch.cuda._sleep(SPACER_CYCLES)
        e0.record(stream)
        for _ in range(count):
            fasq.gemv_raw(*args)
        e1.record(stream)
        e1.synchronize()
        return e0.elapsed_time(e1) * 1e-3

    t = float(np.median([(batch(20) - batch(4)) / 16 for _ in range(reps // 20)]))
    cpu = []
    for _ in range(5):
        t0 = time.perf_counter()
        orc.pq_linear(p.x, p.idx, p.idx_bits, p.d, p.codebook)
        cpu.append(time.perf_counter() - t0)
    out = dict(shape="128x256", M=1, d=4, C=256, idx_bits=8, us=t * 1e6,
               kernel=fasq.plan("gemv", p.M, p.K, p.N, p.idx_bits, p.d, p.C), cpu_oracle_ms=float(np.median(cpu)) * 1e3)
    log(f"[bench] tiny 128x256 d=4: {t * 1e6:.2f} us per call on the GPU ({out['kernel']}); "
        f"CPU oracle {out['cpu_oracle_ms']:.3f} ms")
    return out


def encode_timing(torch, fasq, pi, N=4096, K=4096, d=2, C=256, bits=8):
    """The k-means encoder (fasq_pq_encode) on one dense 4096 x 4096 fp16
    matrix: seconds per Lloyd iteration, from the difference between 10 and 2
    iterations; and the CPU oracle's rate on a 256-row sample."""
    from oracle import pq_encode as enc

    rng = np.random.default_rng(2027)
    w_h = pi.draw_weights(rng, N, K)
    init_h = pi.subvectors_at(w_h, d, pi.init_point_ids(rng, N * K // d, C))
    dev = torch.device("cuda:0")
    w, init = torch.from_numpy(w_h).to(dev), torch.from_numpy(init_h).to(dev)
    ws = torch.empty(fasq.encode_workspace_bytes(N, K, d, C), dtype=torch.uint8, device=dev)
    fasq.pq_encode(w, d, bits, init, 1, workspace=ws)
    torch.cuda.synchronize()

    def run(iters):
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record()
        fasq.pq_encode(w, d, bits, init, iters, workspace=ws)
        e1.record()
        e1.synchronize()
        return e0.elapsed_time(e1) * 1e-3

    per = float(np.median([(run(10) - run(2)) / 8 for _ in range(3)]))
    total = run(10)
    P = N * K // d
    rows = 256
    t0 = time.perf_counter()
    enc.kmeans_encode(w_h[:rows], d, init_h, 2)
    cpu = time.perf_counter() - t0
    out = dict(shape=f"{N}x{K}", d=d, C=C, idx_bits=bits, points=P, s_per_iteration=per, s_10_iterations=total,
               distance_evals_per_s=P * C / per,
               cpu_oracle=dict(rows=rows, iterations=2, seconds=cpu,
                               points_iterations_per_s=rows * (K // d) * 3 / cpu))
    log(f"[bench] encode {N}x{K} d={d} C={C}: {per * 1e3:.3f} ms per Lloyd iteration, {total * 1e3:.2f} ms for 10 "
        f"({P * C / per / 1e12:.2f} T distance evaluations/s); CPU oracle {rows} rows x 2 iterations: {cpu:.2f} s")
    del w, init, ws
    torch.cuda.empty_cache()
    return out


def dense_gemm_seconds(torch, x, w, reps, short, long):
    """Per-call time of torch.matmul(x, w) (fp16, rocBLAS/hipBLASLt), timed
    like the PQ GEMM: differential over back-to-back calls."""
    y = torch.empty((x.shape[0], w.shape[1]), dtype=torch.float16, device=x.device)
    stream = torch.cuda.current_stream()
    torch.matmul(x, w, out=y)

    def batch(count):
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        torch.cuda._sleep(SPACER_CYCLES)
        e0.record(stream)
        for _ in range(count):
            torch.matmul(x, w, out=y)
        e1.record(stream)
        e1.synchronize()
        return e0.elapsed_time(e1) * 1e-3

    times = [(batch(long) - batch(short)) / (long - short) for _ in range(reps)]
    return max(float(np.median(times)), 1e-7)


def prefill(torch, fasq, pi, Ms, reps, short=1, long=4):
    """Prefill GEMM per-launch time, from back-to-back launches (the same
    operands each time: at these sizes the GEMM is bound by the matrix cores,
    not by reading its inputs)."""
    wl = pi.workload("prefill")
    out = []
    dev = torch.device("cuda:0")
    stream = torch.cuda.current_stream()
    for i, spec in enumerate(wl.matrices):
        base = wl.problem(i, M=max(Ms))
        x_all = torch.from_numpy(base.x).to(dev)
        idx = torch.from_numpy(base.idx).to(dev)
        cb = torch.from_numpy(base.codebook).to(dev)
        gen = torch.Generator(device=dev).manual_seed(i)
        w_dense = (torch.randn((spec.K, spec.N), generator=gen, device=dev) * 0.02).to(torch.float16)
        for M in Ms:
            x = x_all[:M].contiguous()
            y = torch.empty((M, spec.N), dtype=torch.float16, device=dev)
            # fasq_pq_gemm_ex: small grids also split K, with a workspace
            # allocated here, outside the timed region
            need = fasq.gemm_ex_workspace_bytes(M, spec.K, spec.N, base.idx_bits, base.d, base.C)
            ws = torch.empty(max(need, 4), dtype=torch.uint8, device=dev)
            args = (x.data_ptr(), M, spec.K, spec.N, idx.data_ptr(), base.idx_bits, base.d, cb.data_ptr(),
                    base.C, y.data_ptr(), ws.data_ptr(), need, stream.cuda_stream)
            assert fasq.gemm_ex_raw(*args) == 0, fasq.last_error()

            def batch(count):
                e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
                torch.cuda._sleep(SPACER_CYCLES)
                e0.record(stream)
                for _ in range(count):
                    assert fasq.gemm_ex_raw(*args) == 0
                e1.record(stream)
                e1.synchronize()
                return e0.elapsed_time(e1) * 1e-3

            times = []
            for _ in range(reps):
                times.append((batch(long) - batch(short)) / (long - short))
            t = max(float(np.median(times)), 1e-7)
            fl = 2.0 * M * spec.N * spec.K
            # Context, not the product: the vendor library's dense fp16 GEMM on
            # the same shape, with the weights stored uncompressed (K x N).
            td = dense_gemm_seconds(torch, x, w_dense, reps, short, long)
            out.append(dict(name=spec.name, M=M, N=spec.N, K=spec.K, us=t * 1e6, tflops=fl / t / 1e12,
                            pct_mfma=100.0 * fl / t / 1e12 / FP16_MFMA_PEAK_TFLOPS,
                            dense_fp16_tflops=fl / td / 1e12, vs_dense_fp16=td / t,
                            kernel=fasq.plan("gemm", M, spec.K, spec.N, base.idx_bits, base.d, base.C),
                            k_split=max(1, need // (M * spec.N * 4))))
            log(f"[bench] prefill {spec.name} M={M}: {t * 1e6:.1f} us, {fl / t / 1e12:.1f} TFLOP/s "
                f"(dense fp16 library GEMM: {fl / td / 1e12:.1f}){' K split ' + str(need // (M * spec.N * 4)) if need else ''}")
        del x_all, idx, cb, w_dense
    torch.cuda.empty_cache()
    return out


def cpu_baseline(pi, frac=1.0):
    """The CPU oracle (fp64 NumPy) on a bounded sample of the decode layer:
    the first `frac` of the output rows of each of the seven matrices."""
    from oracle import pq_oracle as orc

    try:
        from threadpoolctl import threadpool_info

        blas = max([i.get("num_threads", 1) for i in threadpool_info()] or [1])
    except Exception:  # threadpoolctl missing or failing: report the affinity mask
        blas = len(os.sched_getaffinity(0))
    wl = pi.workload("llama3_8b_4bit")
    total_bytes = 0
    elapsed = 0.0
    for i, spec in enumerate(wl.matrices):
        p = wl.problem(i)
        rows = np.arange(int(spec.N * frac))
        t0 = time.perf_counter()
        orc.pq_linear(p.x, p.idx, p.idx_bits, p.d, p.codebook, rows=rows)
        elapsed += time.perf_counter() - t0
        total_bytes += gemv_bytes(1, spec.K, rows.size, p.d, p.C, p.idx_bits)
    return dict(value=total_bytes / elapsed / 1e9, unit="GB/s", cores=int(blas), kind="oracle",
                seconds=elapsed,
                sample=f"first {int(frac * 100)}% of the output rows of each of the 7 matrices of one "
                       f"effective-4-bit Llama-3-8B layer (M=1), {total_bytes / 1e6:.1f} MB of algorithmic "
                       f"bytes; id decoding and gather single-threaded NumPy, fp64 matmul on "
                       f"{blas} BLAS threads; {len(os.sched_getaffinity(0))} cores in the affinity mask")


# L2 (TCC) requests per second that random 8-byte gathers from a 512 KB
# table (L2-resident) reach on MI355X: 278 G gathers/s measured at 0.94
# TCC_REQ per gather.  (8 XCDs x 16 channels x one tag lookup per clock would
# be 307 G/s at 2.4 GHz; the measured rate corresponds to about 2.04 GHz.)
L2_REQ_PER_S = 261e9


def qwen_l2_summary(counters, M, res):
    """L2 requests per layer of the Qwen3-8B launches at M tokens (counters
    taken on the current sources), and the time the L2 request rate alone
    would need for them; None without such counters."""
    if counters is None:
        return None
    reqs, hits, misses = 0.0, 0.0, 0.0
    for r in res["launch_table"]:
        e = counters["launches"].get(f"qwen3_8b_M{M}/{r['name']}")
        if e is None or "TCC_REQ_sum" not in e["counters"]:
            return None
        c = e["counters"]
        reqs += c["TCC_REQ_sum"]
        hits += c.get("TCC_HIT_sum", 0.0)
        misses += c.get("TCC_MISS_sum", 0.0)
    return dict(requests_per_layer=reqs, l2_hit_pct=100.0 * hits / max(hits + misses, 1.0),
                request_floor_us=reqs / L2_REQ_PER_S * 1e6, request_rate_measured_per_s=L2_REQ_PER_S,
                source="profiles/counters.json (rocprofv3 --pmc TCC_REQ_sum, TCC_HIT_sum, TCC_MISS_sum)")


def report_layer(tag, res):
    for r in res["launch_table"]:
        log(f"[bench] {tag} {r['name']:26s} K={r['K']:6d}: {r['us_median']:7.2f} us "
            f"{r['gbs']:7.1f} GB/s ({r['pct_hbm']:.1f}% of HBM peak) {r['kernel']}")
    log(f"[bench] {tag} layer: launch list {res['us_per_layer_list']:.2f} us/layer ({res['gbs_list']:.1f} GB/s; "
        f"{res['us_per_layer_list_events']:.2f} us between events), "
        f"graph {res['us_per_layer_graph']:.2f} us/layer "
        f"({res['gbs_graph']:.1f} GB/s; {res['us_per_layer_graph_events']:.2f} us between events on the stream), "
        f"eager {res['us_per_layer_eager_events']:.2f} us/layer, "
        f"kernel sum {res['us_per_layer_kernel_sum']:.2f} us ({res['gbs_kernel_sum']:.1f} GB/s)")


def main():
    ap = argparse.ArgumentParser(description=__doc__.split("\n")[0])
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=50)
    ap.add_argument("--warmup", type=int, default=10)
    ap.add_argument("--sweep", action="store_true",
                    help="the Qwen3-8B M=1/4/16 decode sweep even with --no-extra (it is part of the default run)")
    ap.add_argument("--no-cpu", action="store_true", help="skip the CPU oracle baseline")
    ap.add_argument("--no-extra", action="store_true", help="only the effective-4-bit decode layer")
    ap.add_argument("--per-matrix", action="store_true", help="add the 4-bit layer with one launch per matrix")
    ap.add_argument("--encode", action="store_true", help="add the k-means encoder timing on one 4096x4096 matrix")
    ap.add_argument("--sensitivity", action="store_true",
                    help="add the codebook-size, sub-vector, batch and prefill-length sweeps on one 4096x4096 layer")
    ap.add_argument("--out", default=None, help="also write the JSON record to this file")
    ap.add_argument("--lib", default=None,
                    help="load this libfasq.so instead of the in-tree one (a variant build, for A/B runs)")
    ap.add_argument("--pmc-pass", metavar="MANIFEST", default=None,
                    help="run the short launch sequence for a rocprofv3 --pmc pass and write its manifest")
    ap.add_argument("--pmc-groups", action="store_true",
                    help="print the rocprofv3 --pmc counter groups, one line each (name: counters)")
    ap.add_argument("--pmc-report", nargs="+", metavar="ARG", default=None,
                    help="MANIFEST OUT_DIR PASS_DIR...: turn --pmc passes into counters.json")
    ap.add_argument("--trace-markdown", nargs=3, metavar=("TRACE_DIR", "BENCH_JSON", "OUT_MD"), default=None,
                    help="write the kernel-statistics summary of a rocprofv3 --kernel-trace --stats run")
    ap.add_argument("--pmc-markdown", nargs="+", metavar="ARG", default=None,
                    help="COUNTERS_JSON OUT_DIR [VARIANT]: write the Markdown counter summaries of a counters.json")
    args = ap.parse_args()

    if args.pmc_groups:
        for g, cs in PMC_GROUPS.items():
            print(f"{g}: {' '.join(cs)}")
        return
    if args.trace_markdown:
        trace_markdown(*args.trace_markdown)
        return
    if args.pmc_markdown:
        if len(args.pmc_markdown) not in (2, 3):
            ap.error("--pmc-markdown needs COUNTERS_JSON OUT_DIR [VARIANT]")
        pmc_markdown(*args.pmc_markdown)
        return
    if args.pmc_report:
        if len(args.pmc_report) < 3:
            ap.error("--pmc-report needs MANIFEST OUT_DIR PASS_DIR...")
        pmc_report(args.pmc_report[0], args.pmc_report[1], args.pmc_report[2:])
        return

    if args.gpus != 1:
        print(f"bench.py runs on one GPU only (asked for --gpus {args.gpus}); the library has no "
              f"multi-GPU path", file=sys.stderr)
        sys.exit(2)

    import torch

    import paper_2605_04084_amd as fasq
    import pq_inputs as pi

    if args.lib:
        fasq.LIB_PATH = os.path.abspath(args.lib)
    elif not os.path.exists(fasq.LIB_PATH):
        import __graft_entry__

        __graft_entry__.build()
    fasq.lib()
    if not torch.cuda.is_available():
        print("bench.py needs a GPU", file=sys.stderr)
        sys.exit(1)

    if args.pmc_pass:
        pmc_pass(torch, fasq, pi, args.pmc_pass)
        return

    main_res = decode_layer(torch, fasq, pi, "llama3_8b_4bit", args.steps, args.warmup)
    report_layer("4bit", main_res)
    roofline = decode_roofline(main_res, "llama3_8b_4bit")

    extra = {}
    if not args.no_extra:
        r3 = decode_layer(torch, fasq, pi, "llama3_8b_3bit", max(10, args.steps // 2), 3)
        report_layer("3bit", r3)
        r3["roofline"] = decode_roofline(r3, "llama3_8b_3bit")
        extra["llama3_8b_3bit"] = r3
        extra["prefill"] = prefill(torch, fasq, pi, (128, 512, 2048), 10)
        extra["tiny"] = tiny_latency(torch, fasq, pi)
        r2 = decode_layer(torch, fasq, pi, "llama3_8b_4bit", max(10, args.steps // 2), 3, M=2)
        report_layer("4bit, M=2", r2)
        r2["roofline"] = decode_roofline(r2, None)
        extra["llama3_8b_4bit_M2"] = r2
    if args.per_matrix:
        r1 = decode_layer(torch, fasq, pi, "llama3_8b_4bit", max(10, args.steps // 2), 3, grouped=False)
        report_layer("4bit, one launch per matrix", r1)
        extra["llama3_8b_4bit_per_matrix"] = r1
    if not args.no_extra or args.sweep:
        # The Qwen3-8B decode layer (65536-entry codebooks, larger than LDS)
        # at 1, 4 and 16 tokens, with what the L2 counters of the same
        # launches say about the gather path.
        counters = load_counters()
        for M in (1, 4, 16):
            r5 = decode_layer(torch, fasq, pi, "qwen3_8b_sweep", max(10, args.steps // 2), 3, M=M)
            report_layer(f"qwen3 M={M}", r5)
            r5["l2"] = qwen_l2_summary(counters, M, r5)
            r5["roofline"] = decode_roofline(r5, f"qwen3_8b_M{M}")
            log(f"[bench] qwen3 M={M}: kernel sum {r5['us_per_layer_kernel_sum']:.2f} us/layer "
                f"({r5['gbs_kernel_sum']:.1f} GB/s); x36 layers {36 * r5['us_per_layer_kernel_sum'] / 1e3:.3f} ms"
                + (f"; L2 requests {r5['l2']['requests_per_layer'] / 1e6:.1f} M per layer, request-rate floor "
                   f"{r5['l2']['request_floor_us']:.1f} us" if r5["l2"] else ""))
            extra[f"qwen3_8b_M{M}"] = r5

    if not args.no_extra:
        extra["crossover"] = crossover(torch, fasq, pi)
    if args.sensitivity:
        extra["sensitivity"] = sensitivity(torch, fasq, pi)
    elif not args.no_extra:
        extra["sensitivity"] = sensitivity(torch, fasq, pi, core=True)
    if args.encode:
        extra["encode"] = encode_timing(torch, fasq, pi)

    cpu = None
    if not args.no_cpu:
        log("[bench] timing the CPU oracle")
        cpu = cpu_baseline(pi)
        log(f"[bench] oracle: {cpu['value'] * 1e3:.2f} MB/s over {cpu['seconds']:.1f} s")

    ms_per_step = main_res["wall_s"] / args.steps * 1e3
    value = main_res["gbs_list"]
    record = {
        "metric": METRIC,
        "value": value,
        "unit": "GB/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": ms_per_step,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "f16",
        "data": "synthetic",
        "config": {
            "workload": "Llama-3-8B decoder layer, decode GEMV at effective 4 bits: q,k,v,o,gate,up,down; "
                        "M=1, d=2, C=256, 8-bit ids, one fp16 codebook per matrix, uniform ids, seed 0",
            "bytes_per_step": main_res["bytes_per_layer"],
            "rotation_copies": main_res["copies"],
            "timed_region": f"one launch-list run of {args.steps} consecutive layers (fasq_launch_list_run: the "
                            "launches recorded once through the library calls, queued with one hipLaunchKernel "
                            "each), 4 launches per layer (q+k+v and gate+up grouped, o, down), inputs cold in HBM",
        },
        "layers_per_graph": main_res["layers_per_graph"],
        "pct_of_hbm_peak": 100.0 * value / HBM_PEAK_GBS,
        "us_per_layer": main_res["us_per_layer_list"],
        "us_per_layer_list_events": main_res["us_per_layer_list_events"],
        "us_per_layer_graph": main_res["us_per_layer_graph"],
        "gbs_graph": main_res["gbs_graph"],
        "us_per_layer_graph_events": main_res["us_per_layer_graph_events"],
        "us_per_layer_eager_events": main_res["us_per_layer_eager_events"],
        "us_per_layer_kernel_sum": main_res["us_per_layer_kernel_sum"],
        "gbs_kernel_sum": main_res["gbs_kernel_sum"],
        "launch_table": main_res["launch_table"],
        "roofline": roofline,
        "cpu_baseline": cpu,
        "extra": extra,
    }
    if "prefill" in extra:
        best = max(extra["prefill"], key=lambda r: r["tflops"])
        record["prefill_tflops_best"] = best["tflops"]
        record["prefill_best_config"] = f"{best['name']} M={best['M']}"
    line = json.dumps(record)
    print(line, flush=True)
    if args.out:
        with open(args.out, "w") as f:
            f.write(line + "\n")


if __name__ == "__main__":
    main()
