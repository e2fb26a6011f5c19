"""Benchmark of the mixed-state denoising step on one MI355X.

One step = dual-cache block attention (every layer) -> parallel decode with the
token/mask gather and scatter fused in, enqueued by one bs_mixed_state_step
call on one stream. Inputs are synthetic and resident in HBM before timing.
Between steps (outside the per-step events) the decoded token/mask state is
restored from pristine copies and a 512 MiB buffer is read, so the 256 MB
Infinity Cache holds none of the step's data (cold numbers). The sweep reads
rather than writes: a written sweep would leave the cache full of dirty lines
whose write-back would then be charged to the timed step.

The headline (`ms_per_step`, `value`) times K plain steps, each bracketed by
HIP events on the step's stream: the start event without a system-scope fence
(the cache maintenance it would do belongs to the untimed restore), the end
event with it (the step's own dirty lines are written back inside the
region). A second region of K steps arms the library's
event ring, which records the phase times (attention over all layers, decode
row reductions, selection) on the same stream; the roofline's launch duration
comes from it. A third region repeats the steps without the sweep (the warm
number, reported alongside), and a plain device copy of the step's byte count
is timed the same way as a reference. A fourth region enqueues the K steps
back to back between one pair of events (each step on its own token/mask copy,
rotating over four copies of the layer inputs and logits so the data stays
cold), with a back-to-back copy reference beside it. `--config 5` times the 32-layer churn
step (compaction, then the fused step) with device-drawn inputs; `--layers N`
gives the one-layer workloads N attention layers (layers past the first
drawn on the device) before their one decode. The ring's events cost a few microseconds each, so they are
kept out of the headline region. Prints ONE JSON line: positions/s, ms per step, phase times,
algorithmic HBM traffic, the roofline of the dominant kernel and the CPU oracle
timed on a bounded sample of the same workload.
"""
from __future__ import annotations

import argparse
import json
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

HBM_PEAK_GBS = 8000.0
MFMA_BF16_PEAK_TFLOPS = 2500.0


def algorithmic_bytes(w):
    """Bytes the step must move (padding and unmasked rows never counted)."""
    eb = w.elem
    lens = (w.reqs["p"] + w.reqs["g"]).astype(np.int64)
    spans = w.spans()
    B = np.array([s[1] for s in spans], np.int64)
    kv = int(lens.sum()) * w.Hkv * w.D * 2 * eb
    qo = 2 * int(B.sum()) * w.Hq * w.D * eb
    wt = int(B.sum()) * w.Hkv * w.D * 2 * eb
    attn = (kv + qo + wt) * w.layers
    flops = int((4 * B * lens).sum()) * w.Hq * w.D * w.layers
    return dict(attn=attn, attn_per_layer=attn // w.layers, kv=kv * w.layers, qo=qo * w.layers,
                write_through=wt * w.layers, attn_flops=flops, positions=int(B.sum()))


def build_state(w, dev_logits_fill=True):
    import torch
    import synth
    from paper_2607_08930_amd import step as bstep
    tok, msk, blk = synth.gen_state(w)
    layers, host = [], []
    for l in range(w.layers):
        q = synth.gen_q(w, l)
        kn, vn = synth.gen_kv_new(w, l)
        kc, vc = synth.gen_cache(w, l)
        out = torch.empty(q.shape, dtype=bstep.torch_dtype(w.dtype), device="cuda")
        layers.append(bstep.Layer(bstep.to_device(q, w.dtype), bstep.to_device(kn, w.dtype),
                                  bstep.to_device(vn, w.dtype), bstep.to_device(kc, w.dtype),
                                  bstep.to_device(vc, w.dtype), out))
        host.append(dict(q=q, k_new=kn, v_new=vn, k_cache=kc, v_cache=vc))
    logits = synth.gen_logits(w, blk)
    st = bstep.StepState(w.L, w.Hq, w.Hkv, w.D, w.V, w.dtype, w.R, w.W, bstep.to_device(tok),
                         bstep.to_device(msk), layers, bstep.to_device(logits, w.dtype), w.n, tau=w.tau,
                         q_min=w.q_min, eos_id=w.eos_id).alloc()
    return st, dict(tokens=tok, mask=msk, blk=blk, layers=host, logits=logits)


def deeper_state(w, st, layers):
    """Adds layers 1 .. layers-1 to a one-layer step: each gets its own device
    tensors of layer 0's shapes and value distributions (queries and fresh
    block K/V ~ N(0, 1), cached K/V ~ N(0, 1/D)), drawn on the device. The
    whole-depth step then runs attention once per layer, then one decode."""
    import torch
    from paper_2607_08930_amd import step as bstep
    g = torch.Generator(device="cuda").manual_seed(1000 + w.cfg)
    l0 = st.layers[0]

    def draw(like, sigma):
        x = torch.empty(like.shape, dtype=torch.float32, device="cuda").normal_(0.0, sigma, generator=g)
        return x.to(like.dtype)

    for _ in range(1, layers):
        st.layers.append(bstep.Layer(draw(l0.q, 1.0), draw(l0.k_new, 1.0), draw(l0.v_new, 1.0),
                                     draw(l0.k_cache, w.D ** -0.5), draw(l0.v_cache, w.D ** -0.5),
                                     torch.empty_like(l0.out)))
    torch.cuda.synchronize()
    w.layers = layers
    w.name += f"-depth{layers}"


B2B_SETS = 4      # input sets the back-to-back region rotates through


def back_to_back(w, st, ctx, tok0, msk0, flush, stream, steps, reps=3):
    """Median over `reps` regions of `steps` fused steps enqueued back to back
    between one pair of HIP events (ms per step), and the host's enqueue time
    per step. Returns (ms, host ms)."""
    import dataclasses
    import torch
    from paper_2607_08930_amd import step as bstep
    sets = [st]
    for _ in range(B2B_SETS - 1):
        lay = [bstep.Layer(x.q.clone(), x.k_new.clone(), x.v_new.clone(), x.k_cache.clone(), x.v_cache.clone(),
                           torch.empty_like(x.out)) for x in st.layers]
        sets.append(dataclasses.replace(st, layers=lay, logits=st.logits.clone()))
    toks = [tok0.clone() for _ in range(steps)]
    msks = [msk0.clone() for _ in range(steps)]
    out, host = [], []
    for rep in range(reps + 1):                       # the first region warms the enqueue path
        for k in range(steps):
            toks[k].copy_(tok0)
            msks[k].copy_(msk0)
        flush.sum()
        torch.cuda.synchronize()
        e0, e1 = region_events()
        e0.record(stream)
        t0 = time.perf_counter()
        for k in range(steps):
            s_ = sets[k % B2B_SETS]
            s_.tokens, s_.mask = toks[k], msks[k]
            bstep.run_step(ctx, s_, w.reqs, stream=stream)
        t1 = time.perf_counter()
        e1.record(stream)
        torch.cuda.synchronize()
        if rep:
            out.append(e0.elapsed_time(e1) / steps)
            host.append((t1 - t0) / steps * 1e3)
    st.tokens, st.mask = sets[0].tokens, sets[0].mask
    del sets, toks, msks
    torch.cuda.synchronize()
    return float(np.median(out)), float(np.median(host))


def copy_back_to_back(nbytes, flush, stream, steps, reps=3):
    """A plain device copy of nbytes (half read, half written) enqueued
    `steps` times back to back over B2B_SETS buffer pairs: ms per copy."""
    import torch
    half = (nbytes // 2 + 255) // 256 * 256
    pairs = [(torch.ones(half // 4, dtype=torch.float32, device="cuda"),
              torch.empty(half // 4, dtype=torch.float32, device="cuda")) for _ in range(B2B_SETS)]
    out = []
    for rep in range(reps + 1):
        flush.sum()
        torch.cuda.synchronize()
        e0, e1 = region_events()
        e0.record(stream)
        for k in range(steps):
            src, dst = pairs[k % B2B_SETS]
            dst.copy_(src)
        e1.record(stream)
        torch.cuda.synchronize()
        if rep:
            out.append(e0.elapsed_time(e1) / steps)
    del pairs
    return float(np.median(out))


def masked_rows(blk):
    return int(blk.sum())


def blas_threads():
    try:
        from threadpoolctl import threadpool_info
        return int(max([i.get("num_threads", 1) for i in threadpool_info()] or [1]))
    except Exception:
        return 1


def host_description():
    """The host the CPU baseline ran on: logical CPUs, the cores this process
    may use, BLAS threads, NumPy version and CPU model."""
    model = ""
    try:
        with open("/proc/cpuinfo") as f:
            model = next((ln.split(":", 1)[1].strip() for ln in f if ln.startswith("model name")), "")
    except OSError:
        pass
    return {"os_cpu_count": os.cpu_count(), "affinity_cores": len(os.sched_getaffinity(0)),
            "blas_threads": blas_threads(), "numpy": np.__version__, "cpu_model": model}


def cpu_baseline(w, host, budget_s=12.0, max_reps=200):
    """The oracle as it stands, timed on this host on the same inputs: whole
    oracle steps are repeated until about budget_s seconds have passed.
    Returns (record, the first step's result)."""
    import oracle
    threads = blas_threads()
    positions = sum(s[1] for s in w.spans())
    t0 = time.perf_counter()
    reps = 0
    first = None
    while True:
        r = oracle.mixed_state_step(w.reqs, w.L, host["tokens"], host["mask"], host["layers"], host["logits"],
                                    tau=w.tau, q_min=w.q_min, eos_id=w.eos_id, dtype=w.dtype)
        first = r if first is None else first
        reps += 1
        el = time.perf_counter() - t0
        if el >= budget_s or reps >= max_reps:
            break
    rec = {"value": round(positions * reps / el, 1), "unit": "positions/s", "cores": threads, "kind": "oracle",
           "sample": f"{reps} whole oracle steps of the same workload ({positions} positions, "
                     f"{w.layers} layer(s) each), fp64 NumPy, {el:.1f} s"}
    rec.update(host=host_description())
    return rec, first


def step_parity(w, host, got, ref):
    """The GPU step (one step from the pristine state) against the oracle's
    step on the same inputs: attention error per layer, cache cells that
    differ, and the decode compared per position (a confidence within 1e-3 of
    the threshold or of a tie at the selection boundary exempts that
    position; every other decision must match bit for bit)."""
    sys.path.insert(0, os.path.join(ROOT, "tests"))
    from gpu_util import check_step_decode
    import oracle
    out = {"what": "one GPU step against the oracle's step on the same inputs"}
    err = rel = 0.0
    cells = 0
    for g, r in zip(got["layers"], ref["layers"]):
        o = oracle.widen(g["out"], w.dtype)
        for i, (s0, B, _) in enumerate(w.spans()):
            d = np.abs(o[i, :B] - r["out"][i, :B])
            err = max(err, float(d.max()))
            rel = max(rel, float(d.max() / max(np.abs(r["out"][i, :B]).max(), 1e-30)))
        cells += int((g["k_cache"] != r["k_cache"]).sum() + (g["v_cache"] != r["v_cache"]).sum())
    out.update(attention_max_abs_err=float(f"{err:.3g}"), attention_max_rel_err=float(f"{rel:.3g}"),
               cache_cells_differing=cells)
    try:
        st = check_step_decode(w, w.reqs, got, ref["decode"], host["tokens"], host["mask"], "bench")
        out.update(masked_positions=st.positions, exempt_positions=st.band, requests_with_open_count=st.open_requests,
                   decision_mismatches=0)
    except AssertionError as e:
        out.update(decision_mismatches=1, first_mismatch=str(e)[:300])
    return out


KERNEL_SOURCES = {   # kernel name prefix -> sources whose change voids its counter-derived traffic
    "k_attn_bf16": ["k_attention.hip", "bs_internal.h", "bs_lds.h"],
    "k_attn_f32": ["k_attention.hip", "bs_internal.h"],
    "k_lm_head": ["k_lm_head.hip", "bs_internal.h", "bs_lds.h"],
    "k_refresh_attn": ["k_refresh.hip", "bs_refresh.h", "bs_internal.h", "bs_lds.h"],
    "k_refresh_kv": ["k_refresh.hip", "bs_refresh.h", "bs_internal.h"],
    "k_decode_parts": ["k_decode.hip", "bs_internal.h"],
    "k_decode_select": ["k_decode.hip", "bs_internal.h"],
}
CALIB_BYTES = 256 << 20          # the --pmc-calibration copy reads and writes this many bytes


def source_hash(kernel):
    import hashlib
    h = hashlib.sha256()
    for f in KERNEL_SOURCES[next(k for k in KERNEL_SOURCES if kernel.startswith(k))] + ["../build.py"]:
        h.update(open(os.path.join(ROOT, "paper_2607_08930_amd", "csrc", f), "rb").read())
    return h.hexdigest()[:16]


def measured_hashes(dirs):
    """Source hashes a --pmc-calibration bench run printed into the log kept
    beside its profiler output directory (<dir>.log), or None when no log
    holds them; every directory given must agree."""
    found = None
    for d in dirs:
        fn = d.rstrip("/") + ".log"
        if not os.path.exists(fn):
            return None
        got = None
        for line in open(fn, errors="replace"):
            if line.startswith("[bench] source hashes "):
                got = json.loads(line[len("[bench] source hashes "):])
        if got is None or (found is not None and got != found):
            return None
        found = got
    return found


def hash_note(measured):
    return ("hash of the kernel's sources in the measured run" if measured is not None else
            "hash of the kernel's sources when this summary was written (the run's log did not record it)")


def traffic_file(workload):
    return os.path.join(ROOT, "profiles", f"traffic_{workload}.md")


class HipEvent:
    """A HIP timing event on the process's HIP runtime (the one torch loaded).
    The start event of a timed region is created with
    hipEventDisableSystemFence: recording it performs no system-scope cache
    write-back and invalidation, which would otherwise charge the previous
    (untimed) work's cache maintenance to the region. The end event keeps the
    default fence, so the region's own dirty lines are written back inside
    it."""
    _lib = None
    DISABLE_SYSTEM_FENCE = 0x20000000

    def __init__(self, fence: bool):
        import ctypes
        if HipEvent._lib is None:
            paths = set()
            with open("/proc/self/maps") as f:
                for line in f:
                    p_ = line.split()[-1] if line.strip() else ""
                    if "libamdhip64" in p_:
                        paths.add(os.path.realpath(p_))
            assert len(paths) == 1, f"expected one HIP runtime, found {sorted(paths)}"
            lib = ctypes.CDLL(paths.pop())
            lib.hipEventCreateWithFlags.argtypes = [ctypes.POINTER(ctypes.c_void_p), ctypes.c_uint]
            lib.hipEventRecord.argtypes = [ctypes.c_void_p, ctypes.c_void_p]
            lib.hipEventElapsedTime.argtypes = [ctypes.POINTER(ctypes.c_float), ctypes.c_void_p, ctypes.c_void_p]
            lib.hipEventDestroy.argtypes = [ctypes.c_void_p]
            HipEvent._lib = lib
        self._ct = __import__("ctypes")
        self.h = self._ct.c_void_p()
        st = HipEvent._lib.hipEventCreateWithFlags(self._ct.byref(self.h), 0 if fence else self.DISABLE_SYSTEM_FENCE)
        assert st == 0, f"hipEventCreateWithFlags failed ({st})"

    def record(self, stream):
        st = HipEvent._lib.hipEventRecord(self.h, self._ct.c_void_p(stream.cuda_stream))
        assert st == 0, f"hipEventRecord failed ({st})"

    def elapsed_time(self, end) -> float:
        ms = self._ct.c_float()
        st = HipEvent._lib.hipEventElapsedTime(self._ct.byref(ms), self.h, end.h)
        assert st == 0, f"hipEventElapsedTime failed ({st})"
        return float(ms.value)

    def __del__(self):
        if self._lib is not None and self.h:
            self._lib.hipEventDestroy(self.h)


def region_events():
    """(start, end) events of one timed region (see HipEvent)."""
    return HipEvent(fence=False), HipEvent(fence=True)


def read_traffic(workload, kernel):
    """Measured HBM bytes per launch of `kernel` from the committed counter
    summary, or None when there is none or the kernel's sources changed since."""
    path = traffic_file(workload)
    if not os.path.exists(path):
        return None
    for line in open(path):
        f = line.strip().strip("`").split()
        if len(f) == 4 and f[0] == "traffic" and kernel.startswith(f[1]) and f[3] == source_hash(f[1]):
            return int(f[2])
    return None


def traffic_summary(args, workload):
    """Counter CSVs of a FETCH_SIZE run and a WRITE_SIZE run -> profiles/traffic_<workload>.md.
    Both counters are KiB per dispatch; each is scaled by what it reads for the
    calibration copy of CALIB_BYTES."""
    import csv
    import glob

    def load(d, counter):
        per, copies = {}, []
        for fn in glob.glob(os.path.join(d, "**", "*counter_collection.csv"), recursive=True):
            for r in csv.DictReader(open(fn)):
                if r["Counter_Name"] == counter:
                    per.setdefault(r["Kernel_Name"], []).append(float(r["Counter_Value"]))
                    if "copyBuffer" in r["Kernel_Name"]:
                        copies.append((int(r["Dispatch_Id"]), float(r["Counter_Value"])))
        return per, sorted(copies)

    (fetch, fcop), (write, wcop) = load(args.traffic_summary[0], "FETCH_SIZE"), load(args.traffic_summary[1], "WRITE_SIZE")
    # the calibration copy is the first runtime copy of more than 32 MiB (it
    # runs before any timed region; later copies, such as the bench's copy
    # reference, can be larger), the same dispatch in both runs
    cal_id = next(i for i, v in fcop if v * 1024 > (32 << 20))
    cal_f = next(v for i, v in fcop if i == cal_id)
    cal_w = next(v for i, v in wcop if i == cal_id)
    kf, kw = CALIB_BYTES / (cal_f * 1024), CALIB_BYTES / (cal_w * 1024)
    lines = [f"# Measured HBM traffic per launch: {workload}", "",
             "Commands (repo root as `$R`, one MI355X; the bench adds one 256 MiB device copy as the",
             "calibration kernel):", "", "```", "cd /tmp && export TMPDIR=/tmp"]
    mode = " --lm-head" if args.lm_head else (" --refresh" if args.refresh else "")
    for c, d in (("FETCH_SIZE", "<fetch dir>"), ("WRITE_SIZE", "<write dir>")):
        lines.append(f"rocprofv3 --pmc {c} -d {d} -o run --output-format csv -- "
                     f"python3 $R/bench.py{mode} --config {args.config} --steps 5 --warmup 1 --no-cpu-baseline --pmc-calibration")
    lines += [f"python3 $R/bench.py{mode} --config {args.config} --traffic-summary <fetch dir> <write dir>", "```", "",
              f"Calibration (256 MiB copy): FETCH_SIZE reads {cal_f:.0f} KiB (scale x{kf:.3f}), "
              f"WRITE_SIZE reads {cal_w:.0f} KiB (scale x{kw:.3f}).", "",
              "| kernel | dispatches | FETCH_SIZE KiB | WRITE_SIZE KiB | read bytes | written bytes | total bytes |",
              "|---|---:|---:|---:|---:|---:|---:|"]
    keep = []
    hashes = measured_hashes(args.traffic_summary)
    for name in sorted(set(fetch) & set(write)):
        short = name.replace("void ", "").replace("bs::(anonymous namespace)::", "").split("(")[0]
        pref = next((k for k in KERNEL_SOURCES if short.startswith(k)), None)
        if pref is None:
            continue
        f_ = float(np.mean(fetch[name])); w_ = float(np.mean(write[name]))
        rd, wr = f_ * 1024 * kf, w_ * 1024 * kw
        lines.append(f"| `{short}` | {len(fetch[name])} | {f_:.0f} | {w_:.0f} | {rd:.0f} | {wr:.0f} | {rd + wr:.0f} |")
        hsh = hashes[pref] if hashes is not None else source_hash(pref)
        keep.append(f"`traffic {pref} {int(round(rd + wr))} {hsh}`")
    lines += ["", f"Machine-readable (kernel, bytes per launch, {hash_note(hashes)};",
              "bench.py reports `traffic` only while the hash matches):", ""] + [k + "  " for k in keep] + [""]
    open(traffic_file(workload), "w").write("\n".join(lines))
    print("\n".join(lines))


COUNTER_PASSES = (
    ("SQ_VALU_MFMA_BUSY_CYCLES", "SQ_BUSY_CYCLES", "SQ_WAVE_CYCLES", "SQ_INSTS_VALU", "SQ_INSTS_MFMA",
     "SQ_ACTIVE_INST_VALU", "SQ_INSTS_LDS", "GRBM_GUI_ACTIVE"),
    ("SQ_WAIT_INST_ANY", "SQ_WAIT_ANY", "SQ_LDS_BANK_CONFLICT", "SQ_LDS_IDX_ACTIVE", "SQ_ACTIVE_INST_LDS",
     "SQ_VALU_MFMA_COEXEC_CYCLES", "SQ_INSTS_VALU_TRANS_F32", "SQ_ACTIVE_INST_ANY", "GRBM_GUI_ACTIVE"),
)
CU_NUM, SIMD_NUM = 256, 1024


def counter_summary(args, workload):
    """Counter CSVs of the two COUNTER_PASSES runs -> profiles/counters_<workload>.md:
    per library kernel, the mean per dispatch of each counter and the derived
    shares (the vendor's MfmaUtil, VALUBusy, LdsUtil and LdsBankConflict
    expressions; wait and co-execution shares of wave and MFMA cycles)."""
    import csv
    import glob
    vals, dur = {}, {}
    n_xcc = 8
    for fn in glob.glob(os.path.join(args.counter_summary[0], "**", "*agent_info.csv"), recursive=True):
        for r in csv.DictReader(open(fn)):
            if r.get("Agent_Type") == "GPU":
                n_xcc = int(r["Num_Xcc"])
    for d in args.counter_summary:
        for fn in glob.glob(os.path.join(d, "**", "*counter_collection.csv"), recursive=True):
            for r in csv.DictReader(open(fn)):
                name = r["Kernel_Name"].replace("void ", "").replace("bs::(anonymous namespace)::", "").split("(")[0]
                if "Cijk_" in name:                  # the library GEMM of the unfused output-head comparison
                    name = "hipBLASLt GEMM " + next((t for t in name.split("_") if t.startswith("MT")), "")
                elif not any(name.startswith(k) for k in KERNEL_SOURCES):
                    continue
                vals.setdefault(name, {}).setdefault(r["Counter_Name"], []).append(float(r["Counter_Value"]))
                key = (d, r["Dispatch_Id"])
                dur.setdefault(name, {})[key] = (int(r["End_Timestamp"]) - int(r["Start_Timestamp"])) / 1e3
    mode = " --lm-head" if args.lm_head else (" --refresh" if args.refresh else "")
    lines = [f"# Hardware counters per launch: {workload}", "",
             "Commands (repo root as `$R`, one MI355X; counters sampled per dispatch, values summed over the",
             "chip by rocprofv3, then averaged over the dispatches of each kernel):", "", "```",
             "cd /tmp && export TMPDIR=/tmp"]
    for k, pas in enumerate(COUNTER_PASSES):
        lines.append(f"rocprofv3 --pmc {' '.join(pas)} -d <dir{k}> -o run --output-format csv -- "
                     f"python3 $R/bench.py{mode} --config {args.config} --only --steps 5 --warmup 1 "
                     f"--no-cpu-baseline --pmc-calibration")
    lines += [f"python3 $R/bench.py{mode} --config {args.config} --counter-summary <dir0> <dir1>", "```", "",
              "Derived (GRBM_GUI_ACTIVE = active cycles of the dispatch, per XCC: rocprofv3 sums the 8 XCCs;",
              "it also counts a fixed sampling window of about 10 us, so short kernels read a low clock;",
              "256 CUs, 1024 SIMDs):",
              "* MFMA busy = SQ_VALU_MFMA_BUSY_CYCLES / (GRBM_GUI_ACTIVE x 1024) (vendor MfmaUtil);",
              "* VALU busy = SQ_ACTIVE_INST_VALU / (GRBM_GUI_ACTIVE x 256) (vendor VALUBusy);",
              "* LDS busy = SQ_LDS_IDX_ACTIVE / (GRBM_GUI_ACTIVE x 256) (vendor LdsUtil); bank conflicts =",
              "  SQ_LDS_BANK_CONFLICT / (SQ_LDS_IDX_ACTIVE - SQ_LDS_BANK_CONFLICT) (vendor LdsBankConflict);",
              "* waits = SQ_WAIT_ANY / SQ_WAVE_CYCLES and SQ_WAIT_INST_ANY / SQ_WAVE_CYCLES (shares of wave",
              "  time; the two passes are separate runs of the same launches);",
              "* co-issue = SQ_VALU_MFMA_COEXEC_CYCLES / SQ_VALU_MFMA_BUSY_CYCLES (MFMA-busy cycles in which a",
              "  VALU instruction also issued); clock = GRBM_GUI_ACTIVE / duration.", "",
              "| kernel | launches | us | clock GHz | MFMA busy | VALU busy | LDS busy | bank confl. | waits any | "
              "waits issue | co-issue | MFMA insts | VALU insts | trans. insts | LDS insts |",
              "|---|---:|---:|---:|---:|---:|---:|---:|---:|---:|---:|---:|---:|---:|---:|"]
    keep = []
    hashes = measured_hashes(args.counter_summary)
    for name in sorted(vals):
        v = {c: float(np.mean(x)) for c, x in vals[name].items()}
        us = float(np.mean(list(dur[name].values())))
        g = v.get("GRBM_GUI_ACTIVE", float("nan")) / n_xcc      # rocprofv3 sums the XCCs' (equal) counts

        def pct(x):
            return f"{100 * x:.1f}%" if x == x else "-"

        get = lambda c: v.get(c, float("nan"))
        mfma = get("SQ_VALU_MFMA_BUSY_CYCLES") / (g * SIMD_NUM)
        valu = get("SQ_ACTIVE_INST_VALU") / (g * CU_NUM)
        lds = get("SQ_LDS_IDX_ACTIVE") / (g * CU_NUM)
        bc = get("SQ_LDS_BANK_CONFLICT") / max(get("SQ_LDS_IDX_ACTIVE") - get("SQ_LDS_BANK_CONFLICT"), 1.0)
        wa = get("SQ_WAIT_ANY") / get("SQ_WAVE_CYCLES")
        wi = get("SQ_WAIT_INST_ANY") / get("SQ_WAVE_CYCLES")
        co = get("SQ_VALU_MFMA_COEXEC_CYCLES") / max(get("SQ_VALU_MFMA_BUSY_CYCLES"), 1.0)
        n_disp = len(dur[name])
        lines.append(f"| `{name}` | {n_disp} | {us:.2f} | {g / us / 1e3:.2f} | {pct(mfma)} | {pct(valu)} | "
                     f"{pct(lds)} | {pct(bc)} | {pct(wa)} | {pct(wi)} | {pct(co)} | {get('SQ_INSTS_MFMA'):.0f} | "
                     f"{get('SQ_INSTS_VALU'):.0f} | {get('SQ_INSTS_VALU_TRANS_F32'):.0f} | {get('SQ_INSTS_LDS'):.0f} |")
        pref = next((k for k in KERNEL_SOURCES if name.startswith(k)), None)
        if pref is not None:
            keep.append(f"`counters {pref} {hashes[pref] if hashes is not None else source_hash(pref)}`")
    lines += ["", f"Sources of each library kernel ({hash_note(hashes)}; a changed kernel makes the row",
              "stale):", ""] + [k + "  " for k in sorted(set(keep))] + [""]
    if any(r.startswith("| `hipBLASLt") for r in lines):
        lines += ["The `hipBLASLt GEMM` row is the library GEMM (torch.matmul) that the bench's unfused",
                  "comparison runs in the same process on the same rows (no source hash: not this library's code).",
                  ""]
    open(os.path.join(ROOT, "profiles", f"counters_{workload}.md"), "w").write("\n".join(lines))
    print("\n".join(lines))


def kernel_summary(args):
    """A rocprofv3 --kernel-trace CSV of a bench run -> profiles/<name>_kernel_stats.md:
    per kernel, launches and mean / min / max duration; per step (one attention
    launch followed by the decode row reductions and the selection), the median
    of each kernel and of the gaps between them, by attention kernel."""
    import csv
    import glob
    d, name = args.kernel_summary
    if os.sep in name or name.startswith("."):
        sys.exit(f"--kernel-summary: NAME must be a plain file stem under profiles/, not {name!r}")
    cmd = args.bench_args
    rows = []
    for fn in glob.glob(os.path.join(d, "**", "*kernel_trace.csv"), recursive=True):
        rows += list(csv.DictReader(open(fn)))
    ks = sorted((int(r["Start_Timestamp"]), int(r["End_Timestamp"]), r["Kernel_Name"]) for r in rows)

    def short(n):
        n = n.replace("void ", "").replace("bs::(anonymous namespace)::", "")
        if "reduce_kernel" in n:
            return "torch reduce_kernel (cache sweep / state restore, outside timing)"
        if "elementwise" in n or "FillFunctor" in n or n.startswith("__amd_rocclr"):
            return "torch / runtime copy or fill (outside timing)"
        return n.split("(")[0]

    # step triples (attention, decode rows, selection), by attention kernel
    steps = {}
    tag = {}
    for a, b, c in zip(ks, ks[1:], ks[2:]):
        if "k_attn" in a[2] and "k_decode_parts" in b[2] and "k_decode_select" in c[2]:
            ka = short(a[2])
            steps.setdefault(ka, []).append(((a[1] - a[0]) / 1e3, (b[0] - a[1]) / 1e3, (b[1] - b[0]) / 1e3,
                                             (c[0] - b[1]) / 1e3, (c[1] - c[0]) / 1e3, (c[1] - a[0]) / 1e3))
            tag[b] = tag[c] = f" (step of {ka})"
            tag[a] = ""
    if steps:
        # attention launches of the same run that belong to no step (the
        # straggler batches of the default run) are listed apart
        for k in ks:
            if "k_attn" in k[2] and k not in tag:
                tag[k] = " (outside a step)"
    per = {}
    for k in ks:
        per.setdefault(short(k[2]) + tag.get(k, ""), []).append((k[1] - k[0]) / 1e3)
    lines = [f"# Kernel durations: {name}", "", "Commands (repo root as `$R`, one MI355X):", "", "```",
             "cd /tmp && export TMPDIR=/tmp",
             f"rocprofv3 --kernel-trace --stats -d <dir> -o run --output-format csv -- python3 $R/bench.py {cmd}",
             f"python3 $R/bench.py --kernel-summary <dir> {name} --bench-args='{cmd}' --steps {args.steps} "
             f"--warmup {args.warmup}", "```", "",
             "| kernel | launches | mean us | min us | max us |", "|---|---:|---:|---:|---:|"]
    for k in sorted(per, key=lambda k: -sum(per[k])):
        v = per[k]
        lines.append(f"| `{k}` | {len(v)} | {np.mean(v):.2f} | {np.min(v):.2f} | {np.max(v):.2f} |")
    if steps:
        lines += ["", "Per step (attention launch, then the decode row reductions and the selection): median over the",
                  "steps of every timed region of the run (isolated, phase ring, warm, back to back):", "",
                  "| attention kernel | steps | attention us | gap us | decode rows us | gap us | selection us | "
                  "first start to last end us |", "|---|---:|---:|---:|---:|---:|---:|---:|"]
    for k, v in steps.items():
        m = np.median(np.array(v), axis=0)
        lines.append(f"| `{k}` | {len(v)} | " + " | ".join(f"{x:.2f}" for x in m) + " |")
    # regions in the order the step bench runs them (W warm-up steps, then K
    # plain, K with the phase ring, K warm, and the back-to-back region)
    W, K = args.warmup, args.steps
    regions = [("warm-up", W), ("plain (headline)", K), ("phase ring (roofline)", K), ("warm", K),
               ("back to back", None)]
    region_lines = []
    for k, v in steps.items():
        v = np.array(v)
        if len(v) != W + 3 * K + 4 * K:      # not the one-layer bench's region layout
            continue
        at = 0
        for rn, cnt in regions:
            cnt = len(v) - at if cnt is None else cnt
            seg = v[at:at + cnt]
            at += cnt
            if len(seg):
                region_lines.append(f"| `{k}` | {rn} | {len(seg)} | {seg[:, 0].mean():.2f} | "
                                    f"{seg[:, 2].mean():.2f} | {seg[:, 4].mean():.2f} |")
    if region_lines:
        lines += ["", f"Per region (mean us per launch; regions by launch order for --warmup {W} --steps {K}):", "",
                  "| attention kernel | region | steps | attention | decode rows | selection |",
                  "|---|---|---:|---:|---:|---:|"] + region_lines
    if "--stragglers" in cmd:
        # launch order of the straggler bench: per batch, W + K whole-row
        # launches, then W + K split-KV launches each followed by its merge
        att = [k for k in ks if "k_attn" in k[2] and "merge" not in k[2]]
        mrg = [k for k in ks if "k_attn_merge" in k[2]]
        W, K = args.warmup, args.steps
        lines += ["", f"Per batch and mode (mean over the {K} timed launches after {W} warm-up ones; the split-KV "
                  "span runs from the attention's start to the merge's end):", "",
                  "| batch | mode | attention us | merge us | span us |", "|---|---|---:|---:|---:|"]
        mi = 0
        for case in range(len(att) // (2 * (W + K))):
            base = case * 2 * (W + K)
            whole = att[base + W:base + W + K]
            lines.append(f"| {case} | whole rows | {np.mean([(b - a) / 1e3 for a, b, _ in whole]):.2f} | - | - |")
            split = att[base + 2 * W + K:base + 2 * (W + K)]
            ms = mrg[mi + W:mi + W + K]
            mi += W + K
            if len(ms) == len(split):
                lines.append(f"| {case} | split-KV | {np.mean([(b - a) / 1e3 for a, b, _ in split]):.2f} | "
                             f"{np.mean([(b - a) / 1e3 for a, b, _ in ms]):.2f} | "
                             f"{np.mean([(m[1] - a[0]) / 1e3 for a, m in zip(split, ms)]):.2f} |")
    lines.append("")
    fn = os.path.join(ROOT, "profiles", f"{name}_kernel_stats.md")
    open(fn, "w").write("\n".join(lines))
    print("\n".join(lines))


class DeviceProvider:
    """Model stand-in for the serving bench: inputs of the right shapes and
    distributions made once on the device (queries, fresh block KV, spiked
    logits whose max probability spreads around the threshold) and reused by
    every step; prefilled KV drawn per admission. Seeded torch generator."""

    def __init__(self, cfg, seed=11):
        import torch
        self.torch, self.cfg = torch, cfg
        g = self.gen = torch.Generator(device="cuda")
        g.manual_seed(seed)
        R, L, td = cfg.rows, cfg.L, torch.bfloat16
        s = 1.0 / np.sqrt(cfg.D)
        self.layers = [(torch.randn((R, L, cfg.Hq, cfg.D), generator=g, device="cuda").to(td),
                        (torch.randn((R, L, cfg.Hkv, cfg.D), generator=g, device="cuda") * s).to(td),
                        (torch.randn((R, L, cfg.Hkv, cfg.D), generator=g, device="cuda") * s).to(td))
                       for _ in range(cfg.layers)]
        x = torch.randn((R * L, cfg.V), generator=g, device="cuda")
        sid = torch.randint(2, cfg.V, (R * L,), generator=g, device="cuda")
        m = torch.rand((R * L,), generator=g, device="cuda") * 8.0
        x.scatter_(1, sid[:, None], (torch.logsumexp(x, dim=1) + m)[:, None])
        self.logits = x.view(R, L, cfg.V).to(td)
        self.prompt_rng = np.random.default_rng(seed)

    def prefill(self, ids, p, g, W):
        torch, cfg = self.torch, self.cfg
        n, ws = len(ids), int((p + g).max())
        s = 1.0 / np.sqrt(cfg.D)
        sk = (torch.randn((cfg.layers, n, cfg.Hkv, ws, cfg.D), generator=self.gen, device="cuda") * s).to(torch.bfloat16)
        sv = (torch.randn((cfg.layers, n, cfg.Hkv, ws, cfg.D), generator=self.gen, device="cuda") * s).to(torch.bfloat16)
        tok = np.zeros((n, W), np.int32)
        msk = np.zeros((n, W), np.uint8)
        for a in range(n):
            off = W - int(p[a] + g[a])
            tok[a, off:off + int(p[a])] = self.prompt_rng.integers(2, cfg.V, int(p[a]))
            msk[a, off + int(p[a]):] = 1
        return sk, sv, tok, msk

    def step(self, ids, descs, cycle, step):
        n = len(ids)
        return [(q[:n], kn[:n], vn[:n]) for q, kn, vn in self.layers], self.logits[:n]

    def refresh(self, ids, descs, cycle):
        """Projections of the whole box at a block start, made once and reused."""
        torch, cfg = self.torch, self.cfg
        if not hasattr(self, "box"):
            g, td, s = self.gen, torch.bfloat16, 1.0 / np.sqrt(cfg.D)
            R, W = cfg.rows, cfg.width
            self.box = [(torch.randn((R, W, cfg.Hq, cfg.D), generator=g, device="cuda").to(td),
                         (torch.randn((R, W, cfg.Hkv, cfg.D), generator=g, device="cuda") * s).to(td),
                         (torch.randn((R, W, cfg.Hkv, cfg.D), generator=g, device="cuda") * s).to(td))
                        for _ in range(cfg.layers)]
        return self.box


def lm_head_bench(args):
    """The output head fused with the decoding step (bs_lm_head_decode) against
    the same step unfused: a hipBLASLt GEMM over the masked rows
    (torch.matmul), its bf16 logits copied into the [n][L] row layout, then
    bs_parallel_decode. Prints one JSON line."""
    import torch
    import synth
    import paper_2607_08930_amd as bs
    from paper_2607_08930_amd import step as bstep

    torch.cuda.set_device(0)
    w = synth.workload(args.config)
    d = synth.LM_HEAD_DIM[args.config]
    print(f"[bench] output head {w.name} d={d} V={w.V}: generating inputs", file=sys.stderr, flush=True)
    wv = synth.gen_lm_weight(w, d)
    hidden = synth.gen_lm_hidden(w, wv)
    tok, msk, blk = synth.gen_state(w)
    # compact block state (host copy of the active blocks; padding rows zero)
    tok_c = np.zeros((w.n, w.L), np.int32)
    msk_c = np.zeros((w.n, w.L), np.uint8)
    for i, (r, (s0, B, _)) in enumerate(zip(w.reqs, w.spans())):
        c0 = int(r["off"]) + s0
        tok_c[i, :B] = tok[int(r["row"]), c0:c0 + B]
        msk_c[i, :B] = msk[int(r["row"]), c0:c0 + B]
    R = int(blk.sum())
    dW = bstep.to_device(wv, "bf16")
    dH = bstep.to_device(hidden, "bf16")
    pb = bs.bs_lm_head_pack_bytes(w.V, d)
    dP = torch.empty(pb // 2, dtype=torch.bfloat16, device="cuda")
    t0, m0 = bstep.to_device(tok_c), bstep.to_device(msk_c)
    dt, dm = t0.clone(), m0.clone()
    nun = torch.empty(w.n, dtype=torch.int32, device="cuda")
    done = torch.empty(w.n, dtype=torch.uint8, device="cuda")
    eos = torch.empty(w.n, dtype=torch.uint8, device="cuda")
    conf = torch.empty((w.n, w.L), dtype=torch.float32, device="cuda")
    wsb = bs.bs_lm_head_workspace_bytes(w.n, w.L, w.V)
    ws = torch.empty(max(wsb, 16), dtype=torch.uint8, device="cuda")
    idx = torch.as_tensor(np.nonzero(blk.reshape(-1))[0], device="cuda")
    vpad = (w.V + 7) // 8 * 8
    logits = torch.empty((w.n * w.L, vpad), dtype=torch.bfloat16, device="cuda")
    dws = bs.bs_decode_workspace_bytes(w.n, w.L, w.V, bs.BS_BF16)
    dwsb = torch.empty(max(dws, 16), dtype=torch.uint8, device="cuda")
    flush = torch.ones(128 << 20, dtype=torch.float32, device="cuda")
    ctx = bs.Context(0)
    stream = torch.cuda.current_stream()
    if args.pmc_calibration:
        src_ = torch.ones(CALIB_BYTES // 4, dtype=torch.float32, device="cuda")
        dst_ = torch.empty_like(src_)
        dst_.copy_(src_)
        torch.cuda.synchronize()
        del src_, dst_
    bs.bs_lm_head_pack(ctx, dW, d, w.V, d, bs.BS_BF16, dP, pb, stream=stream)    # once per model
    H2 = dH.view(w.n * w.L, d)

    def fused():
        bs.bs_lm_head_decode(ctx, w.reqs, w.L, d, w.V, bs.BS_BF16, dH, dP, dt, dm, w.tau, w.q_min, w.eos_id,
                             nun, done, eos, conf, ws, wsb, stream=stream)

    def gemm():
        return torch.matmul(H2.index_select(0, idx), dW.t())

    def unfused():
        logits[idx, :w.V] = gemm()
        bs.bs_parallel_decode(ctx, w.reqs, w.L, w.V, bs.BS_BF16, logits, vpad, dt, dm, w.tau, w.q_min, w.eos_id,
                              nun, done, eos, conf, dwsb, dws, stream=stream)

    def timed(fn, k):
        out = []
        for _ in range(k):
            dt.copy_(t0)
            dm.copy_(m0)
            flush.sum()
            e0, e1 = region_events()
            e0.record(stream)
            fn()
            e1.record(stream)
            torch.cuda.synchronize()
            out.append(e0.elapsed_time(e1))
        return float(np.median(out))

    for fn in (fused, unfused, gemm):
        timed(fn, args.warmup)
    bs.bs_profile_begin(ctx, args.steps)          # phases of every fused call: row list | GEMM | merge + select
    ms = timed(fused, args.steps)
    ph = bs.bs_profile_end(ctx, args.steps)
    gemm_ms = float(np.median(ph[:, 1]))
    ms_unf = timed(unfused, args.steps)
    ms_gemm = timed(gemm, args.steps)
    flops = 2.0 * R * d * w.V
    positions = int(sum(s[1] for s in w.spans()))
    tflops = flops / (gemm_ms / 1e3) / 1e12
    ctx.close()
    res = {
        "metric": "denoised block positions/s per decoding step with the output head",
        "value": round(positions / (ms / 1e3), 1), "unit": "positions/s", "n_gpus": 1, "steps": args.steps,
        "warmup": args.warmup, "ms_per_step": round(ms, 5), "higher_is_better": True, "scaling": "weak",
        "vs_baseline": None, "dtype": "bf16", "data": "synthetic",
        "config": {"workload": w.name + f"-lm-head-d{d}", "n_requests": w.n, "masked_rows": R, "d": d, "V": w.V,
                   "cache": "cold (512 MiB read sweep between steps)"},
        "unfused_ms": round(ms_unf, 5), "unfused_gemm_ms": round(ms_gemm, 5),
        "speedup_vs_unfused": round(ms_unf / ms, 3),
        "phases_ms": {"rows": round(float(np.median(ph[:, 0])), 5), "gemm": round(gemm_ms, 5),
                      "merge_select": round(float(np.median(ph[:, 2])), 5)},
        "roofline": {"kernel": "k_lm_head", "bound": "mfma", "achieved": round(tflops, 1),
                     "peak": MFMA_BF16_PEAK_TFLOPS, "unit": "TFLOP/s", "frac": round(tflops / MFMA_BF16_PEAK_TFLOPS, 4),
                     "algorithmic_flops_per_launch": flops, "avg_launch_ms": round(gemm_ms, 5),
                     "traffic": read_traffic(w.name + f"-lm-head-d{d}", "k_lm_head")},
    }
    if not args.no_cpu_baseline:
        import oracle
        print("[bench] timing the CPU oracle on a sample of the same inputs", file=sys.stderr, flush=True)
        threads = blas_threads()
        tic, reps, pos = time.perf_counter(), 0, 0
        while time.perf_counter() - tic < 12.0 and reps < w.n:
            oracle.lm_head_decode(w.reqs, w.L, hidden, wv, tok_c, msk_c, tau=w.tau, q_min=w.q_min,
                                  eos_id=w.eos_id, dtype="bf16", only=[reps])
            pos += w.spans()[reps][1]
            reps += 1
        el = time.perf_counter() - tic
        res["cpu_baseline"] = {"value": round(pos / el, 1), "unit": "positions/s", "cores": int(threads), "host": host_description(),
                               "kind": "oracle",
                               "sample": f"{reps} requests' decoding steps with the output head (fp64), {el:.1f} s"}
    print(json.dumps(res), flush=True)


def straggler_case(ctx, case, steps, warmup):
    """Whole rows against the split-KV plan for one straggler batch
    (synth.straggler(case)): the attention launch bracketed by HIP events on
    its stream, enqueued behind a 512 MiB read sweep (so the host call
    overlaps the sweep and the region holds the launch alone, with a cold
    Infinity Cache). Inputs are drawn on the device (queries and fresh K/V ~
    N(0, 1), cache ~ N(0, 1/D)). Returns the batch's record."""
    import torch
    import synth
    import paper_2607_08930_amd as bs

    stream = torch.cuda.current_stream()
    flush = torch.ones(128 << 20, dtype=torch.float32, device="cuda")
    gen = torch.Generator(device="cuda").manual_seed(7 + case)

    def draw(shape, sigma):
        x = torch.empty(shape, dtype=torch.float32, device="cuda").normal_(0.0, sigma, generator=gen)
        return x.to(torch.bfloat16)

    w = synth.straggler(case)
    print(f"[bench] stragglers: {w.name}", file=sys.stderr, flush=True)
    q = draw((w.n, w.L, w.Hq, w.D), 1.0)
    kn, vn = draw((w.n, w.L, w.Hkv, w.D), 1.0), draw((w.n, w.L, w.Hkv, w.D), 1.0)
    kc, vc = draw((w.R, w.Hkv, w.W, w.D), w.D ** -0.5), draw((w.R, w.Hkv, w.W, w.D), w.D ** -0.5)
    out = torch.empty_like(q)
    torch.cuda.synchronize()
    ab = algorithmic_bytes(w)
    lens = w.reqs["p"] + w.reqs["g"]
    entry = {"workload": w.name, "n_requests": int(w.n), "max_len": int(lens.max()), "sum_len": int(lens.sum()),
             "algorithmic_bytes": int(ab["attn"])}
    for split in (False, True):
        nws = bs.bs_attention_workspace_bytes(w.reqs, w.L, w.Hq, w.Hkv, w.D, bs.BS_BF16) if split else 0
        ws = torch.empty(max(nws, 16), dtype=torch.uint8, device="cuda")

        def call():
            bs.bs_dual_cache_block_attention(ctx, w.reqs, w.L, w.Hq, w.Hkv, w.D, bs.BS_BF16, 0.0, q, kn, vn,
                                             kc, vc, w.R, w.W, 1, out, ws if nws else None, nws, stream=stream)

        for _ in range(warmup):
            call()
        ts = []
        for _ in range(steps):
            flush.sum()
            e0, e1 = region_events()
            e0.record(stream)
            call()
            e1.record(stream)
            torch.cuda.synchronize()
            ts.append(e0.elapsed_time(e1))
        items, parts = bs.bs_attention_work_list(w.reqs, w.L, w.Hq, w.Hkv, w.D, bs.BS_BF16, int(split))
        ms = float(np.median(ts))
        entry["split_kv" if split else "whole_rows"] = {
            "ms": round(ms, 5), "workgroups": int(len(items)), "partial_slots": int(parts),
            "longest_workgroup_tiles": int((items[:, 4] - items[:, 3]).max()),
            "achieved_GBps": round(ab["attn"] / (ms * 1e-3) / 1e9, 1)}
    entry["speedup"] = round(entry["whole_rows"]["ms"] / entry["split_kv"]["ms"], 3)
    del q, kn, vn, kc, vc, out, flush
    torch.cuda.empty_cache()
    return entry


def stragglers_bench(args):
    """Attention of one layer on straggler batches (synth.straggler: a few rows
    far longer than the rest of a Dream-7B- or LLaDA-8B-shaped batch), whole
    rows against the split-KV plan (straggler_case). Prints one JSON line."""
    import torch
    import paper_2607_08930_amd as bs

    torch.cuda.set_device(0)
    ctx = bs.Context(0)
    results = [straggler_case(ctx, case, args.steps, args.warmup) for case in (0, 1, 2)]
    print(json.dumps({"metric": "attention launch time on straggler batches, whole rows vs split-KV", "unit": "ms",
                      "higher_is_better": False, "steps": args.steps, "warmup": args.warmup, "dtype": "bf16",
                      "data": "synthetic", "cache": "cold (512 MiB read sweep before each launch)",
                      "results": results}))


def refresh_bench(args):
    """The dual-cache refresh of one layer (bs_dual_cache_refresh: rotated keys
    and values into the cache, then full-row attention) over the whole box of
    a workload, beside one batched call of torch's SDPA on the same inputs
    padded to the longest row. Prints one JSON line."""
    import torch
    import synth
    import paper_2607_08930_amd as bs
    from paper_2607_08930_amd import step as bstep
    from torch.nn.attention import SDPBackend, sdpa_kernel

    torch.cuda.set_device(0)
    w = synth.workload(args.config)
    base = synth.ROPE_BASE[args.config]
    print(f"[bench] refresh {w.name}: generating the box projections", file=sys.stderr, flush=True)
    q, k, v = synth.gen_refresh(w)
    dq, dk, dv = (bstep.to_device(x, "bf16") for x in (q, k, v))
    dkc = torch.zeros((w.R, w.Hkv, w.W, w.D), dtype=torch.bfloat16, device="cuda")
    dvc = torch.zeros_like(dkc)
    out = torch.zeros_like(dq)
    lens = [int(r["p"] + r["g"]) for r in w.reqs]
    flops = float(sum(4.0 * ln * ln * w.D * w.Hq for ln in lens))     # Q K^T and P V, 2 flops per MAC
    positions = int(sum(lens))
    flush = torch.ones(128 << 20, dtype=torch.float32, device="cuda")
    ctx = bs.Context(0)
    stream = torch.cuda.current_stream()
    if args.pmc_calibration:
        src_ = torch.ones(CALIB_BYTES // 4, dtype=torch.float32, device="cuda")
        dst_ = torch.empty_like(src_)
        dst_.copy_(src_)
        torch.cuda.synchronize()
        del src_, dst_

    def fused():
        bs.bs_dual_cache_refresh(ctx, w.reqs, w.L, w.Hq, w.Hkv, w.D, bs.BS_BF16, 0.0, base, dq, dk, dv, w.R, w.W,
                                 dkc, dvc, out, stream=stream)

    # library comparison: one batched call of torch's SDPA (memory-efficient
    # backend, the one that takes a mask; the math backend is never used)
    # over every request padded to the longest row, with a key-padding mask:
    # queries [n][Hq][Lmax][D] and the cached (rotated) K/V expanded to the
    # query heads. The rotation of the queries changes no work, so the
    # unrotated ones stand in for them. The padded call does n Lmax^2 of work
    # per head against the sum of len^2 of the refresh.
    G = w.Hq // w.Hkv
    lib_in = []

    def prep_library():
        fused()
        torch.cuda.synchronize()
        lmax = max(lens)
        qq = torch.zeros((w.n, w.Hq, lmax, w.D), dtype=torch.bfloat16, device="cuda")
        kk = torch.zeros_like(qq)
        vv = torch.zeros_like(qq)
        mask = torch.zeros((w.n, 1, 1, lmax), dtype=torch.bool, device="cuda")
        for i, (r, ln) in enumerate(zip(w.reqs, lens)):
            row, off = int(r["row"]), int(r["off"])
            kk[i, :, :ln] = dkc[row, :, off:off + ln].repeat_interleave(G, 0)
            vv[i, :, :ln] = dvc[row, :, off:off + ln].repeat_interleave(G, 0)
            qq[i, :, :ln] = dq[row, off:off + ln].transpose(0, 1)
            mask[i, :, :, :ln] = True
        lib_in.append((qq, kk, vv, mask))

    def library():
        qq, kk, vv, mask = lib_in[0]
        with sdpa_kernel([SDPBackend.EFFICIENT_ATTENTION]):
            torch.nn.functional.scaled_dot_product_attention(qq, kk, vv, attn_mask=mask)

    def timed(fn, kreps):
        res = []
        for _ in range(kreps):
            flush.sum()
            e0, e1 = region_events()
            e0.record(stream)
            fn()
            e1.record(stream)
            torch.cuda.synchronize()
            res.append(e0.elapsed_time(e1))
        return float(np.median(res))

    timed(fused, args.warmup)
    bs.bs_profile_begin(ctx, args.steps)          # phases of every call: rotated K/V scatter | attention
    ms = timed(fused, args.steps)
    ph = bs.bs_profile_end(ctx, args.steps)
    kv_ms, att_ms = float(np.median(ph[:, 0])), float(np.median(ph[:, 1]))
    lib_ms = None
    if not args.no_library:
        try:
            prep_library()
            timed(library, max(1, args.warmup))
            lib_ms = timed(library, args.steps)
        except RuntimeError as e:                 # no such kernel for this shape in this PyTorch
            print(f"[bench] library attention unavailable: {e}", file=sys.stderr, flush=True)
    ctx.close()
    tflops = flops / (att_ms / 1e3) / 1e12
    kv_bytes = float(sum(ln * w.Hkv * w.D * 2 * 4 for ln in lens))   # K and V read once, written once
    res = {
        "metric": "refreshed positions/s per layer (dual-cache refresh)",
        "value": round(positions / (ms / 1e3), 1), "unit": "positions/s", "n_gpus": 1, "steps": args.steps,
        "warmup": args.warmup, "ms_per_step": round(ms, 5), "higher_is_better": True, "scaling": "weak",
        "vs_baseline": None, "dtype": "bf16", "data": "synthetic",
        "config": {"workload": w.name + "-refresh", "n_requests": w.n, "positions": positions, "rope_base": base,
                   "cache": "cold (512 MiB read sweep between steps)"},
        "phases_ms": {"rope_kv": round(kv_ms, 5), "attention": round(att_ms, 5)},
        "rope_kv_GBps": round(kv_bytes / (kv_ms / 1e3) / 1e9, 1),
        "library_attention_ms": None if lib_ms is None else round(lib_ms, 5),
        "library_attention": "torch SDPA (memory-efficient backend), one call over the padded batch with a key mask",
        "library_padded_flops": float(4.0 * w.n * max(lens) ** 2 * w.D * w.Hq),
        "attention_speedup_vs_library": None if lib_ms is None else round(lib_ms / att_ms, 3),
        "roofline": {"kernel": "k_refresh_attn", "bound": "mfma", "achieved": round(tflops, 1),
                     "peak": MFMA_BF16_PEAK_TFLOPS, "unit": "TFLOP/s", "frac": round(tflops / MFMA_BF16_PEAK_TFLOPS, 4),
                     "algorithmic_flops_per_launch": flops, "avg_launch_ms": round(att_ms, 5),
                     "traffic": read_traffic(w.name + "-refresh", "k_refresh_attn")},
    }
    if not args.no_cpu_baseline:
        import oracle
        print("[bench] timing the CPU oracle on a sample of the same inputs", file=sys.stderr, flush=True)
        threads = blas_threads()
        order = np.argsort(lens)                  # shortest rows first: several requests fit the budget
        tic, reps, pos = time.perf_counter(), 0, 0
        while time.perf_counter() - tic < 12.0 and reps < w.n:
            i = int(order[reps])
            r = w.reqs[i]
            row = int(r["row"])
            oracle.refresh_row(r, q[row], k[row], v[row], dtype="bf16", rope_base=base)
            pos += lens[i]
            reps += 1
        el = time.perf_counter() - tic
        res["cpu_baseline"] = {"value": round(pos / el, 1), "unit": "positions/s", "cores": int(threads), "host": host_description(),
                               "kind": "oracle",
                               "sample": f"the {reps} shortest requests' full-row refresh, all heads (fp64), "
                                         f"{el:.1f} s"}
    print(json.dumps(res), flush=True)


def churn_bench(args):
    """Workload 5, the LLaDA-8B-shaped 32-layer batch at a block boundary: one
    step is K4 (the admitted requests' staged KV copied into the freed rows of
    every layer, stable slots) followed by the fused step (attention in all 32
    layers, then the decode) on the post-churn descriptors. The churn plan,
    token and mask state come from the seeded generators; the 52 GB of KV,
    the per-layer queries and fresh KV and the logits are drawn on the device
    from a seeded torch generator with the same distributions (host
    generation at this size would take longer than the run). Repeating the
    step is idempotent for the KV (the same rows are copied and written
    through again); the token/mask state is restored between steps. Prints
    one JSON line."""
    import torch
    import synth
    import paper_2607_08930_amd as bs
    from paper_2607_08930_amd import step as bstep

    torch.cuda.set_device(0)
    if args.pmc_calibration:
        # the calibration copy, before any other device copy of the run
        src_ = torch.ones(CALIB_BYTES // 4, dtype=torch.float32, device="cuda")
        dst_ = torch.empty_like(src_)
        dst_.copy_(src_)
        torch.cuda.synchronize()
        del src_, dst_
    w = synth.workload(5)
    tok, msk, _ = synth.gen_state(w)
    plan = synth.churn_plan(w, w.reqs, tok, msk, step=1)          # rewrites tok/msk rows in place
    w.reqs = plan.reqs
    n, R, W, NL, L = w.n, w.R, w.W, w.layers, w.L
    print(f"[bench] {w.name}: {n} requests, {NL} layers, {len(plan.segs)} copy segments; drawing inputs",
          file=sys.stderr, flush=True)
    g = torch.Generator(device="cuda")
    g.manual_seed(260708930)
    td, s = torch.bfloat16, 1.0 / np.sqrt(w.D)

    def normal(shape, sigma):
        return (torch.randn(shape, generator=g, device="cuda") * sigma).to(td)

    kbox = torch.empty((NL, R, w.Hkv, W, w.D), dtype=td, device="cuda")
    vbox = torch.empty_like(kbox)
    for l in range(NL):
        kbox[l] = normal((R, w.Hkv, W, w.D), s)
        vbox[l] = normal((R, w.Hkv, W, w.D), s)
    n_adm = len(plan.stage_reqs)
    wst = int((plan.stage_reqs["p"] + plan.stage_reqs["g"]).max()) if n_adm else 1
    stg_k = normal((NL, max(n_adm, 1), w.Hkv, wst, w.D), s)
    stg_v = normal((NL, max(n_adm, 1), w.Hkv, wst, w.D), s)
    layers = [bstep.Layer(normal((n, L, w.Hq, w.D), 1.0), normal((n, L, w.Hkv, w.D), s),
                          normal((n, L, w.Hkv, w.D), s), kbox[l], vbox[l],
                          torch.empty((n, L, w.Hq, w.D), dtype=td, device="cuda")) for l in range(NL)]
    x = torch.randn((n * L, w.V), generator=g, device="cuda")     # spiked logits (max probability around tau)
    sid = torch.randint(1, w.V, (n * L,), generator=g, device="cuda")
    m = torch.rand((n * L,), generator=g, device="cuda") * 8.0
    x.scatter_(1, sid[:, None], (torch.logsumexp(x, dim=1) + m)[:, None])
    logits = x.view(n, L, w.V).to(td)
    del x
    st = bstep.StepState(L, w.Hq, w.Hkv, w.D, w.V, w.dtype, R, W, bstep.to_device(tok), bstep.to_device(msk),
                         layers, logits, n, tau=w.tau, q_min=w.q_min, eos_id=w.eos_id).alloc()
    tok0, msk0 = st.tokens.clone(), st.mask.clone()
    flush = torch.ones(128 << 20, dtype=torch.float32, device="cuda")
    stream = torch.cuda.current_stream()
    ctx = bs.Context(0)

    def one_step():
        bstep.compact(ctx, plan.segs, NL, w.Hkv, w.D, w.dtype, kbox, vbox, stg_k, stg_v, kbox, vbox, stream=stream)
        bstep.run_step(ctx, st, w.reqs, stream=stream)

    def reset():
        st.tokens.copy_(tok0)
        st.mask.copy_(msk0)
        flush.sum()

    for _ in range(args.warmup):
        reset()
        one_step()
    torch.cuda.synchronize()
    times = []
    for _ in range(args.steps):
        reset()
        e0, e1 = region_events()
        e0.record(stream)
        one_step()
        e1.record(stream)
        torch.cuda.synchronize()
        times.append(e0.elapsed_time(e1))
    # phase durations, live, over a second region of the same steps (the
    # library's event ring brackets the 32 attention launches and the decode)
    bs.bs_profile_begin(ctx, args.steps)
    for _ in range(args.steps):
        reset()
        one_step()
    torch.cuda.synchronize()
    phases = bs.bs_profile_end(ctx, args.steps)
    ctx.close()
    ms = float(np.median(times))
    ab = algorithmic_bytes(w)
    attn_ms = float(np.median(phases[:, 0])) / NL           # per launch, gaps between launches included
    attn_gbs = ab["attn_per_layer"] / (attn_ms / 1e3) / 1e9
    nmask = 0
    for r, (s0, B, _) in zip(w.reqs, w.spans()):
        nmask += int(np.count_nonzero(msk[int(r["row"]), int(r["off"]) + s0:int(r["off"]) + s0 + B]))
    copied = int(plan.segs["len"].sum()) if len(plan.segs) else 0
    copy_bytes = 2 * copied * w.Hkv * w.D * 2 * w.elem * NL
    small = ab["positions"] * (4 + 4 + 1 + 1 + 4)
    step_bytes = ab["attn"] + nmask * w.V * w.elem + copy_bytes + small
    gbs = step_bytes / (ms / 1e3) / 1e9
    res = {
        "metric": "denoised block positions/s per mixed-state step", "value": round(ab["positions"] / (ms / 1e3), 1),
        "unit": "positions/s", "n_gpus": 1, "steps": args.steps, "warmup": args.warmup, "ms_per_step": round(ms, 5),
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None, "dtype": w.dtype,
        "data": "synthetic (KV, queries and logits drawn on the device)",
        "config": {"workload": w.name, "n_requests": n, "layers": NL, "positions_per_step": ab["positions"],
                   "masked_rows": nmask, "copied_tokens": copied, "admitted": n_adm, "finished": plan.n_finish,
                   "cache": "cold (52 GB of KV; 512 MiB read sweep between steps)"},
        "hbm": {"algorithmic_bytes_per_step": step_bytes, "achieved_GBps": round(gbs, 1),
                "frac_of_peak": round(gbs / HBM_PEAK_GBS, 4),
                "parts": {"attention_all_layers": ab["attn"], "logits": nmask * w.V * w.elem,
                          "compaction": copy_bytes, "token_mask_pos": small}},
        "step_ms_p10_p90": [round(float(np.percentile(times, 10)), 5), round(float(np.percentile(times, 90)), 5)],
        "phases_ms": {n_: round(float(np.median(phases[:, i])), 5) for i, n_ in enumerate(bs.PROFILE_PHASES)},
        "roofline": {"kernel": "k_attn_bf16_wave", "bound": "hbm", "achieved": round(attn_gbs, 1),
                     "peak": HBM_PEAK_GBS, "unit": "GB/s", "frac": round(attn_gbs / HBM_PEAK_GBS, 4),
                     "algorithmic_bytes_per_launch": ab["attn_per_layer"], "avg_launch_ms": round(attn_ms, 5),
                     "traffic": read_traffic(w.name, "k_attn_bf16_wave")},
    }
    if not args.no_cpu_baseline:
        import oracle
        print("[bench] timing the CPU oracle on a sample of the same workload", file=sys.stderr, flush=True)
        threads = blas_threads()
        sample = list(range(8))
        q = synth.gen_q(w, 0)
        kn, vn = synth.gen_kv_new(w, 0)
        kc = np.zeros((R, w.Hkv, W, w.D), np.uint16)
        vc = np.zeros_like(kc)
        for i in sample:
            kc[int(w.reqs[i]["row"])], vc[int(w.reqs[i]["row"])] = synth.gen_cache_row(w, 0, int(w.reqs[i]["row"]))
        blk = np.zeros((n, L), bool)
        tok_c = np.zeros((n, L), np.int32)
        msk_c = np.zeros((n, L), np.uint8)
        lg = np.zeros((n, L, w.V), np.uint16)
        for i in sample:
            r = w.reqs[i]
            s0, B, _ = w.spans()[i]
            c0 = int(r["off"]) + s0
            msk_c[i, :B] = msk[int(r["row"]), c0:c0 + B]
            tok_c[i, :B] = tok[int(r["row"]), c0:c0 + B]
            for j in range(B):
                if msk_c[i, j]:
                    lg[i, j] = synth.gen_logits_row(w, i, j)
        t0 = time.perf_counter()
        oracle.dual_cache_block_attention(w.reqs, L, q, kn, vn, kc, vc, dtype="bf16", only=sample)
        t_att = time.perf_counter() - t0
        t0 = time.perf_counter()
        oracle.parallel_decode(w.reqs, L, lg, tok_c, msk_c, tau=w.tau, q_min=w.q_min, eos_id=w.eos_id,
                               dtype="bf16", only=sample)
        t_dec = time.perf_counter() - t0
        pos = sum(w.spans()[i][1] for i in sample)
        t_step = t_att * NL + t_dec
        res["cpu_baseline"] = {"value": round(pos / t_step, 1), "unit": "positions/s", "cores": int(threads), "host": host_description(),
                               "kind": "oracle",
                               "sample": f"{len(sample)} requests: one layer's attention ({t_att:.2f} s) scaled to "
                                         f"{NL} layers, plus their decode ({t_dec:.2f} s); compaction not counted"}
    print(json.dumps(res), flush=True)


def serve_bench(args):
    """Closed-loop serving of a stream shaped like one row of the benchmark
    statistics table; prints one JSON line."""
    import torch
    import synth
    import paper_2607_08930_amd as bs
    from paper_2607_08930_amd import serve

    torch.cuda.set_device(0)
    stream = synth.table_stream(args.serve, args.serve_requests)
    pa, pm, limit, ga, gm = synth.TABLE_STREAMS[args.serve]
    W = max(p + g for _, p, g in stream)
    B = args.batch
    budget = args.budget if args.budget else B * (pa + limit)
    policy = bs.SCHED_FIXED if args.policy == "fixed" else bs.SCHED_BUDGET
    rows = B if policy == bs.SCHED_FIXED else args.rows
    cfg = serve.ServeConfig(L=32, layers=args.layers, Hq=32, Hkv=32, D=128, V=126464, dtype="bf16", rows=rows,
                            width=W, policy=policy, budget=budget, fixed_batch=B, tau=0.9, q_min=1, eos_id=-1,
                            refresh=args.refresh, rope_base=synth.ROPE_BASE[2] if args.refresh else 0.0)
    print(f"[bench] serving {args.serve} x{len(stream)} ({args.policy}, B={B}, budget={budget}, rows={rows}, W={W})",
          file=sys.stderr, flush=True)
    prov = DeviceProvider(cfg)
    with bs.Context(0) as ctx:
        serve.Server(ctx, cfg, prov).run(stream[:8])            # warm-up on a few requests
        torch.cuda.synchronize()
        srv = serve.Server(ctx, cfg, prov)
        t0 = time.perf_counter()
        res = srv.run(stream)
        torch.cuda.synchronize()
        wall = time.perf_counter() - t0
    gen = sum(g for _, _, g in stream)
    R = sum(res.active_counts) / (res.cycles * B)
    print(json.dumps({
        "metric": "closed-loop generated tokens/s", "value": round(gen / wall, 1), "unit": "tokens/s",
        "n_gpus": 1, "higher_is_better": True, "dtype": "bf16", "data": "synthetic",
        "config": {"workload": f"serve-{args.serve}-llada8b-layer", "requests": len(stream), "policy": args.policy,
                   "baseline_batch": B, "budget_tokens": budget, "rows": rows, "W": W, "layers": args.layers,
                   "stream": "prompt/generated lengths shaped like the benchmark statistics table row",
                   "dual_cache_refresh": bool(args.refresh)},
        "wall_s": round(wall, 3), "block_cycles": res.cycles, "denoising_steps": res.steps,
        "generated_tokens": gen, "steps_per_cycle": round(res.steps / res.cycles, 2),
        "mean_active": round(sum(res.active_counts) / res.cycles, 2), "R_eq2": round(R, 3),
        "ms_per_step": round(wall * 1e3 / res.steps, 4), "refresh_calls": res.refreshes}), flush=True)


def step_bench(args, cfg):
    """Times the fused step on workload `cfg` (the regions described at the
    top of this file) and returns its result record."""
    import torch
    import synth
    import paper_2607_08930_amd as bs
    from paper_2607_08930_amd import step as bstep

    assert torch.cuda.is_available()
    torch.cuda.set_device(0)
    w = synth.workload(cfg, block_length=args.block_length)
    if args.prefix_only:
        w.reqs = bstep.prefix_only(w.reqs, w.L)
        w.name += "-prefix-only"
    print(f"[bench] building inputs for {w.name}", file=sys.stderr, flush=True)
    st, host = build_state(w)
    if args.layers > 1:
        deeper_state(w, st, args.layers)
    ab = algorithmic_bytes(w)
    nmask = masked_rows(host["blk"])
    logits_bytes = nmask * w.V * w.elem
    small_bytes = ab["positions"] * (4 + 4 + 1 + 1 + 4)        # token r/w, mask r/w, position id
    step_bytes = ab["attn"] + logits_bytes + small_bytes
    tok0, msk0 = st.tokens.clone(), st.mask.clone()
    flush = torch.ones(128 << 20, dtype=torch.float32, device="cuda")    # 512 MiB, swept by reading
    stream = torch.cuda.current_stream()
    ctx = bs.Context(0)
    if args.pmc_calibration:
        src_ = torch.ones(CALIB_BYTES // 4, dtype=torch.float32, device="cuda")
        dst_ = torch.empty_like(src_)
        dst_.copy_(src_)
        torch.cuda.synchronize()
        del src_, dst_

    def one_step():
        bstep.run_step(ctx, st, w.reqs, stream=stream)

    sweep = [not args.warm]

    def reset():
        st.tokens.copy_(tok0)
        st.mask.copy_(msk0)
        if sweep[0]:
            flush.sum()

    for _ in range(args.warmup):
        reset()
        one_step()
    torch.cuda.synchronize()
    print(f"[bench] warmup done ({args.warmup} steps); timing {args.steps}", file=sys.stderr, flush=True)
    flags_host = [torch.empty(t.shape, dtype=t.dtype, pin_memory=True) for t in (st.n_unmasked, st.done, st.eos_seen)]

    def timed(ring, flags=False):
        """K steps, each bracketed by HIP events on the step's stream; with
        ring, the library's phase events are recorded inside every step; with
        flags, each step ends with the copy of its completion flags to pinned
        host memory (what a serving loop reads before its next step)."""
        evs = [region_events() for _ in range(args.steps)]
        if ring:
            bs.bs_profile_begin(ctx, args.steps)
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        for k in range(args.steps):
            reset()
            evs[k][0].record(stream)
            one_step()
            if flags:
                with torch.cuda.stream(stream):
                    for h, d in zip(flags_host, (st.n_unmasked, st.done, st.eos_seen)):
                        h.copy_(d, non_blocking=True)
            evs[k][1].record(stream)
        torch.cuda.synchronize()
        wall = (time.perf_counter() - t0) / args.steps * 1e3
        ph = bs.bs_profile_end(ctx, args.steps) if ring else None
        return np.array([a.elapsed_time(b) for a, b in evs]), wall, ph

    # headline: plain steps (the phase events cost about 5 us each, so they
    # are kept out of the step that `value` is quoted on)
    step_ms, wall, _ = timed(False)
    # phase durations, live, over a second timed region of the same steps
    ring_ms, _, phases = timed(True)                  # [steps][attention, decode_rows, decode_select]
    # the warm number alongside: the same steps without the cache sweep
    sweep[0] = False
    warm_ms, _, _ = timed(False)
    sweep[0] = not args.warm
    # the same steps, each ending with its completion flags copied to the host
    flag_ms, _, _ = timed(False, flags=True)
    # back to back: K steps between one pair of events, as a serving loop
    # runs them. Step k reads input set k % NB (copies of the layer inputs
    # and logits at other addresses, so a set was last read NB - 1 steps and
    # more than 1 GB of traffic before, cold in the Infinity Cache) and its
    # own copy of the token/mask state, so every step does the same work.
    # (left out of counter runs: its input copies would outsize the calibration copy)
    b2b = None if args.pmc_calibration else back_to_back(w, st, ctx, tok0, msk0, flush, stream, args.steps)
    ms = float(np.median(step_ms))
    attn_ms = float(np.median(phases[:, 0])) / w.layers       # one attention launch
    rows_ms = float(np.median(phases[:, 1]))
    value = ab["positions"] / (ms / 1e3)
    attn_gbs = ab["attn_per_layer"] / (attn_ms / 1e3) / 1e9
    dec_gbs = logits_bytes / (rows_ms / 1e3) / 1e9
    attn_dominant = ab["attn"] >= logits_bytes
    if attn_dominant:
        gw = (w.Hq // w.Hkv) * ((w.L + 31) // 32)
        roof = {"kernel": ("k_attn_bf16_wave" if gw == 1 else "k_attn_bf16_group") if w.dtype == "bf16" else "k_attn_f32",
                "bound": "hbm",
                "achieved": round(attn_gbs, 1), "peak": HBM_PEAK_GBS, "unit": "GB/s",
                "frac": round(attn_gbs / HBM_PEAK_GBS, 4),
                "algorithmic_bytes_per_launch": ab["attn_per_layer"], "avg_launch_ms": round(attn_ms, 5)}
    else:
        roof = {"kernel": "k_decode_parts", "bound": "hbm", "achieved": round(dec_gbs, 1), "peak": HBM_PEAK_GBS,
                "unit": "GB/s", "frac": round(dec_gbs / HBM_PEAK_GBS, 4),
                "algorithmic_bytes_per_launch": logits_bytes, "avg_launch_ms": round(rows_ms, 5)}
    roof["traffic"] = read_traffic(w.name, roof["kernel"])
    ctx.close()
    # reference: a plain device copy that moves the step's algorithmic bytes
    # (half read, half written), cold, timed like a step
    half = (step_bytes // 2 + 255) // 256 * 256
    csrc = torch.ones(half // 4, dtype=torch.float32, device="cuda")
    cdst = torch.empty_like(csrc)
    copy_ms = []
    for k in range(args.steps):
        flush.sum()
        e0, e1 = region_events()
        e0.record(stream)
        cdst.copy_(csrc)
        e1.record(stream)
        torch.cuda.synchronize()
        copy_ms.append(e0.elapsed_time(e1))
    copy_ms = float(np.median(copy_ms))
    del csrc, cdst
    copy_b2b_ms = None if b2b is None else copy_back_to_back(step_bytes, flush, stream, args.steps)
    res = {
        "metric": "denoised block positions/s per mixed-state step",
        "value": round(value, 1), "unit": "positions/s", "n_gpus": 1, "steps": args.steps,
        "warmup": args.warmup, "ms_per_step": round(ms, 5), "higher_is_better": True, "scaling": "weak",
        "vs_baseline": None, "dtype": w.dtype, "data": "synthetic",
        "config": {"workload": w.name, "n_requests": w.n, "positions_per_step": ab["positions"],
                   "masked_rows": nmask, "L": w.L, "Hq": w.Hq, "Hkv": w.Hkv, "D": w.D, "V": w.V,
                   "layers": w.layers, "sum_len": int((w.reqs["p"] + w.reqs["g"]).sum()),
                   "cache": "warm" if args.warm else "cold (512 MiB read sweep between steps)"},
        "hbm": {"algorithmic_bytes_per_step": step_bytes, "achieved_GBps": round(step_bytes / (ms / 1e3) / 1e9, 1),
                "frac_of_peak": round(step_bytes / (ms / 1e3) / 1e9 / HBM_PEAK_GBS, 4),
                "frac_of_copy_reference": round(copy_ms / ms, 4)},
        "ms_per_step_warm": round(float(np.median(warm_ms)), 5),
        "ms_per_step_with_flag_readback": round(float(np.median(flag_ms)), 5),
        "back_to_back": None if b2b is None else {
            "ms_per_step": round(b2b[0], 5), "positions_per_s": round(ab["positions"] / (b2b[0] / 1e3), 1),
            "achieved_GBps": round(step_bytes / (b2b[0] / 1e3) / 1e9, 1),
            "frac_of_peak": round(step_bytes / (b2b[0] / 1e3) / 1e9 / HBM_PEAK_GBS, 4),
            "host_enqueue_ms_per_step": round(b2b[1], 5), "copy_reference_ms": round(copy_b2b_ms, 5),
            "frac_of_copy_reference": round(copy_b2b_ms / b2b[0], 4)},
        "phases_ms": {n_: round(float(np.median(phases[:, i])), 5) for i, n_ in enumerate(bs.PROFILE_PHASES)},
        "kernel_GBps": {"attention": round(attn_gbs, 1), "decode_rows": round(dec_gbs, 1)},
        "attention_tflops": round(ab["attn_flops"] / w.layers / (attn_ms / 1e3) / 1e12, 2),
        "attention_mfma_frac": round(ab["attn_flops"] / w.layers / (attn_ms / 1e3) / 1e12 / MFMA_BF16_PEAK_TFLOPS, 4),
        "wall_ms_per_step_incl_restore": round(wall, 5),
        "step_ms_p10_p90": [round(float(np.percentile(step_ms, 10)), 5), round(float(np.percentile(step_ms, 90)), 5)],
        "ms_per_step_with_phase_events": round(float(np.median(ring_ms)), 5),
        "copy_reference": {"bytes": 2 * half, "ms": round(copy_ms, 5),
                           "GBps": round(2 * half / (copy_ms / 1e3) / 1e9, 1),
                           "what": "device copy of the step's byte count (half read, half written), cold"},
        "roofline": roof,
    }
    if not args.no_cpu_baseline and args.layers == 1:
        # one step from the pristine state, kept for the parity check
        ctx = bs.Context(0)
        st.tokens.copy_(tok0)
        st.mask.copy_(msk0)
        bstep.run_step(ctx, st, w.reqs, stream=stream, want_conf=True)
        torch.cuda.synchronize()
        got = dict(tokens=st.tokens.cpu().numpy(), mask=st.mask.cpu().numpy(), conf=st.conf.cpu().numpy(),
                   n_unmasked=st.n_unmasked.cpu().numpy(), done=st.done.cpu().numpy(),
                   eos_seen=st.eos_seen.cpu().numpy(),
                   layers=[dict(out=bstep.to_host(x.out), k_cache=bstep.to_host(x.k_cache),
                                v_cache=bstep.to_host(x.v_cache)) for x in st.layers])
        ctx.close()
        print("[bench] timing the CPU oracle on the same inputs", file=sys.stderr, flush=True)
        res["cpu_baseline"], ref = cpu_baseline(w, host)
        res["parity"] = step_parity(w, host, got, ref)
    del st, flush
    torch.cuda.synchronize()
    torch.cuda.empty_cache()
    return res


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=50)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--config", type=int, default=2, help="workload 1-5 (2 = LLaDA-8B-shaped layer, 3 = Dream-7B-shaped, 4 = skewed Dream batch, "
                         "5 = 32-layer LLaDA churn step with compaction)")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--only", action="store_true",
                    help="time only the chosen workload (the default run of workload 2 also times workload 3)")
    ap.add_argument("--warm", action="store_true", help="skip the Infinity Cache flush between steps")
    ap.add_argument("--pmc-calibration", action="store_true",
                    help="run one 256 MiB device copy first (the reference kernel for FETCH_SIZE / WRITE_SIZE)")
    ap.add_argument("--traffic-summary", nargs=2, metavar=("FETCH_DIR", "WRITE_DIR"),
                    help="turn two rocprofv3 --pmc runs into profiles/traffic_<workload>.md (no GPU needed)")
    ap.add_argument("--kernel-summary", nargs=2, metavar=("DIR", "NAME"),
                    help="turn a rocprofv3 --kernel-trace run of `bench.py <--bench-args>` into "
                         "profiles/NAME_kernel_stats.md (no GPU needed)")
    ap.add_argument("--bench-args", default="", help="--kernel-summary: the arguments the profiled bench run had "
                                                      "(give as --bench-args=...)")
    ap.add_argument("--counter-summary", nargs="+", metavar="DIR",
                    help="turn the rocprofv3 --pmc runs of COUNTER_PASSES into profiles/counters_<workload>.md "
                         "(no GPU needed)")
    ap.add_argument("--serve", choices=["humaneval-256", "gsm8k-256", "mbpp-512", "truthfulqa-512"],
                    help="closed-loop serving of a table-shaped request stream instead of the step bench")
    ap.add_argument("--serve-requests", type=int, default=256)
    ap.add_argument("--policy", choices=["budget", "fixed"], default="budget")
    ap.add_argument("--batch", type=int, default=16, help="fixed cap, and B of Eq. 2")
    ap.add_argument("--budget", type=int, default=0, help="Eq. 1 budget in tokens (default B * (avg prompt + limit))")
    ap.add_argument("--rows", type=int, default=128, help="rows of the dense box under the budget policy")
    ap.add_argument("--layers", type=int, default=1,
                    help="attention layers per step (step mode: layers past the first are drawn on the device; "
                         "--serve: model depth)")
    ap.add_argument("--block-length", type=int, default=None,
                    help="re-block the workload's requests at L = 16 or 64 (block-length sweep)")
    ap.add_argument("--lm-head", action="store_true",
                    help="time the output head fused with the decoding step against the unfused GEMM + decode")
    ap.add_argument("--refresh", action="store_true",
                    help="time the dual-cache refresh (rotated K/V scatter + full-row attention) of one layer; "
                         "with --serve, rebuild the dual cache at every block start of the serving loop")
    ap.add_argument("--no-library", action="store_true", help="--refresh: skip the library attention comparison")
    ap.add_argument("--stragglers", action="store_true",
                    help="attention on straggler batches (a few very long rows): whole rows vs split-KV")
    ap.add_argument("--prefix-only", action="store_true",
                    help="prefix-cache layout: keys end at the active block (no masked suffix)")
    args = ap.parse_args()
    if args.pmc_calibration:
        # the summaries tie each counter row to the sources that were measured
        print("[bench] source hashes " + json.dumps({k: source_hash(k) for k in KERNEL_SOURCES}),
              file=sys.stderr, flush=True)
    if args.kernel_summary:
        kernel_summary(args)
        return
    if args.lm_head and not (args.traffic_summary or args.counter_summary):
        if args.gpus != 1:
            print("bench.py measures one GPU: the step runs on a single device (run with --gpus 1)",
                  file=sys.stderr, flush=True)
            sys.exit(2)
        lm_head_bench(args)
        return
    if args.config == 5 and not (args.traffic_summary or args.counter_summary) and not args.serve:
        if args.gpus != 1:
            print("bench.py measures one GPU: the step runs on a single device (run with --gpus 1)",
                  file=sys.stderr, flush=True)
            sys.exit(2)
        churn_bench(args)
        return
    if args.stragglers:
        if args.gpus != 1:
            print("bench.py measures one GPU: the attention runs on a single device (run with --gpus 1)",
                  file=sys.stderr, flush=True)
            sys.exit(2)
        stragglers_bench(args)
        return
    if args.refresh and not (args.traffic_summary or args.counter_summary) and not args.serve:
        if args.gpus != 1:
            print("bench.py measures one GPU: the step runs on a single device (run with --gpus 1)",
                  file=sys.stderr, flush=True)
            sys.exit(2)
        refresh_bench(args)
        return
    if args.serve:
        if args.gpus != 1:
            print("bench.py measures one GPU: the step runs on a single device (run with --gpus 1)",
                  file=sys.stderr, flush=True)
            sys.exit(2)
        serve_bench(args)
        return
    if args.traffic_summary or args.counter_summary:
        import synth
        name = synth.workload(args.config, block_length=args.block_length).name
        if args.lm_head:
            name += f"-lm-head-d{synth.LM_HEAD_DIM[args.config]}"
        if args.refresh:
            name += "-refresh"
        name += "-prefix-only" if args.prefix_only else ""
        if args.traffic_summary:
            traffic_summary(args, name)
        else:
            counter_summary(args, name)
        return
    if args.gpus != 1:
        print("bench.py measures one GPU: the step runs on a single device (run with --gpus 1)",
              file=sys.stderr, flush=True)
        sys.exit(2)

    res = step_bench(args, args.config)
    # the Dream-7B-shaped layer is the other binding shape: the default run
    # reports it in the same line, nested
    if (args.config == 2 and not args.only and args.layers == 1 and args.block_length is None
            and not args.prefix_only and not args.pmc_calibration):
        second = step_bench(args, 3)
        res["second_config"] = {k: second[k] for k in ("value", "unit", "ms_per_step", "config", "hbm", "roofline",
                                                       "phases_ms", "kernel_GBps", "attention_tflops",
                                                       "attention_mfma_frac", "step_ms_p10_p90", "back_to_back",
                                                       "ms_per_step_warm", "ms_per_step_with_flag_readback", "copy_reference",
                                                       "parity", "cpu_baseline")
                                if k in second}
        # straggler handling (split-KV) on the LLaDA-8B-shaped batch with one
        # 16000-token prompt: whole rows against the plan, attention only
        import paper_2607_08930_amd as bs
        res["straggler_split_kv"] = straggler_case(bs.Context(0), 2, 10, 2)
    print(json.dumps(res), flush=True)


if __name__ == "__main__":
    main()
