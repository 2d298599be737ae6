"""Benchmark: DP-SGD gradient steps per second on one MI355X.

    python bench.py [--steps K] [--warmup W] [--workload NAME]

A step is one pass of the whole hot path over one batch whose inputs are
already resident in HBM: per-sample gradients of every layer, per-sample
norms, clip factors, clipped sums, noise and division.  W untimed steps, then
K timed steps between two device synchronizations; value = samples / second.

Alongside: the dominant call's roofline (algorithmic bytes or flops per
launch over its average duration, timed with HIP events on the step's stream
around K back-to-back launches of that call after the timed steps), HBM
traffic from committed rocprofv3 counter runs when they still match the
kernel source, and the fp64 oracle timed on the host's cores on a bounded
sample of the same workload.

Counter runs (two passes, one counter each) and their reduction:

    rocprofv3 --pmc FETCH_SIZE -f csv -d DIR_F -o c -- python bench.py --copy-calibration-mib 512 ...
    rocprofv3 --pmc WRITE_SIZE -f csv -d DIR_W -o c -- python bench.py --copy-calibration-mib 512 ...
    python bench.py --record-traffic META DIR_F/c_counter_collection.csv DIR_W/c_counter_collection.csv

(META: the file the counter runs wrote with --meta-out.)

The launches of the dominant call and the calibration copy are bracketed by a
one-byte-element fill kernel that nothing else launches, so the reduction can
find them in the dispatch list; each counter is scaled by the ratio of the
copy's true bytes to what the counter reads for it.
"""
from __future__ import annotations

import argparse
import hashlib
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

HBM_PEAK_GBS = 8000.0
PEAK_TFLOPS = {"f32": 157.3, "bf16": 2500.0}     # dense MFMA peaks
# fp32 vector ALU: 256 CUs x 4 SIMDs x 16 lanes x 2 flops (FMA) x 2 (packed FP32) x 2.4 GHz
ALU_PEAK_TFLOPS = 157.3
METRIC = "DP-SGD grad step samples/sec at 1 MI355X; achieved HBM GB/s / MFMA util"


def log(*a):
    print(*a, file=sys.stderr, flush=True)


# ---------------------------------------------------------------------------
# algorithmic cost of each call of the step
# ---------------------------------------------------------------------------

def call_costs(st, nnz=None):
    """name -> (algorithmic bytes, flops, kernel name, MFMA peak key or None) per call of one step.

    nnz: layer name -> the number of (sample, distinct id) rows an Embedding
    layer's per-sample gradient holds (row_ptr[N], read back after a warm-up
    step); without it the CSR is priced at its capacity N*T."""
    from paper_2109_12298_amd import workloads as W
    from paper_2109_12298_amd import binding as dp
    N = st.N
    bf = st.wl.dtype == W.BF16
    e = 2 if bf else 4
    out = {}
    col_bytes = 0
    for lb in st.layers:
        L = lb.layer
        if isinstance(L, W.Linear):
            bias = L.d_out if L.bias else 0
            grads = N * (L.d_out * L.d_in + bias) * 4
            bf_mfma = bf and L.T > 1 and L.d_in % 8 == 0 and L.d_out % 8 == 0
            if lb.ghost:
                # the two T x T Grams per sample; reads A and B, writes one norm
                # (all ghost layers share one grouped call)
                b0, f0, _, _ = out.get("grad:ghost", (0, 0, None, None))
                out["grad:ghost"] = (b0 + N * L.T * (L.d_in + L.d_out) * e + N * 4,
                                     f0 + 2 * N * L.T * L.T * (L.d_in + L.d_out), "ghost_gram_kernel",
                                     "bf16" if bf else "f32")
            elif L.T == 1:
                out["grad:" + L.name] = (N * (L.d_in + L.d_out) * e + grads + N * 4, N * L.d_out * L.d_in,
                                         "outer_kernel", None)
            else:
                staged = bf_mfma and L.T % 32 == 0
                # fp32 operands whose rows are 16-byte multiples over T % 16 == 0 are staged straight into LDS
                staged32 = not bf and L.T % 16 == 0 and L.d_in % 4 == 0 and L.d_out % 4 == 0
                out["grad:" + L.name] = (N * L.T * (L.d_in + L.d_out) * e + grads + N * 4,
                                         2 * N * L.T * L.d_in * L.d_out,
                                         "bf16_grad_sample_kernel" if staged else
                                         "bf16_per_sample_kernel" if bf_mfma else
                                         "ps_gemm_dma_kernel" if staged32 else "ps_gemm_kernel",
                                         "bf16" if bf_mfma else "f32")
            if lb.clip_mode == "fused":
                # all fused Linear layers' weight sums share one grouped call; their
                # bias sums are column reductions of the stored bias gradients
                grouped = bf and L.T % 32 == 0 and L.d_in % 8 == 0 and L.d_out % 8 == 0
                b0, f0, _, _ = out.get("clip:linears", (0, 0, None, None))
                out["clip:linears"] = (b0 + N * L.T * (L.d_in + L.d_out) * e + L.d_out * L.d_in * 4
                                       + (bias * 4 if lb.ghost else 0),
                                       f0 + 2 * N * L.T * L.d_in * L.d_out,
                                       "bf16_clipsum_many_kernel" if grouped else "clipsum_gemm_kernel",
                                       "bf16" if grouped else "f32")
                col_bytes += 0 if lb.ghost else N * bias * 4
            else:
                col_bytes += grads
        elif isinstance(L, W.Conv2d):
            ho, wo = L.out_hw
            kk = L.c_in * L.k[0] * L.k[1]
            grads = N * L.n_params * 4
            choice = dp.dp_conv2d_kernel_choice(N, L.c_in, L.h, L.w, L.c_out, L.k[0], L.k[1], L.stride[0],
                                                L.stride[1], L.pad[0], L.pad[1])
            kname = {dp.DP_CONV_KERNEL_SMALL: "conv_small_kernel",
                     dp.DP_CONV_KERNEL_ROWS: "conv_rows_kernel"}.get(choice, "conv_per_sample_kernel")
            out["grad:" + L.name] = (N * (L.c_in * L.h * L.w + L.c_out * ho * wo) * e + grads + N * 4,
                                     2 * N * L.c_out * kk * ho * wo, kname, "f32")
            col_bytes += grads
        elif isinstance(L, W.Embedding):
            u = (nnz or {}).get(L.name, N * L.T)
            # reads ids and backprops; writes row_ptr, the distinct ids, their rows and the squared norms
            out["grad:" + L.name] = (N * L.T * (8 + L.D * e) + (N + 1) * 8 + u * (L.D * 4 + 8) + N * 4,
                                     N * L.T * L.D, "emb_fused_kernel" if L.T <= 512 else "emb_csr_kernel", None)
            # reads row_ptr, the ids, the rows and the norms; writes the dense [V][D] sum
            out["clip:" + L.name] = ((N + 1) * 8 + u * (L.D * 4 + 8) + N * 4 + L.V * L.D * 4, 2 * u * L.D,
                                     "emb_clipsum_kernel", None)
        elif isinstance(L, W.LSTMRecurrence):
            # reads the stored gates and cell states, W_hh and dh_last; writes the gate backprop
            G = 4 * L.H
            # (its dot products are vector-ALU FMAs on a chain of T dependent steps: priced as "alu")
            out["grad:" + L.name] = (N * L.T * (2 * G + L.H) * 4 + G * L.H * 4 + N * L.H * 4,
                                     2 * N * L.T * G * L.H, "lstm_bptt_kernel", "alu")
        elif isinstance(L, W.LayerNorm):
            # all LayerNorm layers share one grouped call
            b0, f0, _, _ = out.get("grad:lns", (0, 0, None, None))
            out["grad:lns"] = (b0 + 2 * N * L.T * L.D * e + 2 * N * L.D * 4 + N * 4, f0 + 3 * N * L.T * L.D,
                               "ln_rows_kernel", None)
            col_bytes += 2 * N * L.D * 4
        elif isinstance(L, W.GroupNorm):
            out["grad:" + L.name] = (2 * N * L.C * L.P * e + 2 * N * L.C * 4 + N * 4, 3 * N * L.C * L.P,
                                     "gn_affine_kernel", None)
            col_bytes += 2 * N * L.C * 4
    if st.grad_group:
        # the grouped layers' per-sample gradients: the small layers' launch,
        # the bf16 sequence layers' launch and the fp32 sequence layers' launch
        gb_, gf_, kinds = 0, 0, set()
        for i in st.grad_group:
            b0, f0, kn, _ = out.pop("grad:" + st.layers[i].layer.name)
            gb_ += b0
            gf_ += f0
            kinds.add({"bf16_grad_sample_kernel": "bf16_grad_group_kernel",
                       "ps_gemm_dma_kernel": "ps_dma_group_kernel"}.get(kn, "grad_many_kernel"))
        kname = "+".join(sorted(kinds))
        mt = "bf16" if "bf16_grad_group_kernel" in kinds else "f32" if "ps_dma_group_kernel" in kinds else None
        out["grad:group"] = (gb_, gf_, kname, mt)
    if not st.fold_norms:
        out["norms"] = (len(st.layers) * N * 4 + N * 4, len(st.layers) * N, "norms_kernel", None)
    P = st.wl.n_params
    # one launch: (norms,) read the column-reduced grads once, write S and out, read fused S
    norms_bytes = (len(st.layers) * N * 4 + N * 4) if st.fold_norms else 0
    # virtual steps: the running sums are read and written as well
    acc_bytes = 8 * P if st.virtual_batches > 1 else 0
    out["clip+noise"] = (col_bytes + 12 * P + norms_bytes + acc_bytes, 0, "norms_clip_noise_kernel", None)
    return out


def src_hash(paths):
    h = hashlib.sha256()
    for p in paths:
        with open(os.path.join(ROOT, p), "rb") as f:
            h.update(f.read())
    return h.hexdigest()[:16]


KERNEL_SOURCES = {
    "outer_kernel": ["paper_2109_12298_amd/csrc/linear.hip", "paper_2109_12298_amd/csrc/linear_outer.hpp"],
    "ghost_gram_kernel": ["paper_2109_12298_amd/csrc/ghost.hip", "paper_2109_12298_amd/csrc/bf16_stage.hpp"],
    "gn_affine_kernel": ["paper_2109_12298_amd/csrc/groupnorm.hip"],
    "conv_rows_kernel": ["paper_2109_12298_amd/csrc/conv2d_rows.hip"],
    "conv_small_kernel": ["paper_2109_12298_amd/csrc/conv2d_small.hip",
                          "paper_2109_12298_amd/csrc/conv2d_small_dev.hpp"],
    "grad_many_kernel": ["paper_2109_12298_amd/csrc/grad_many.hip", "paper_2109_12298_amd/csrc/conv2d_small_dev.hpp",
                         "paper_2109_12298_amd/csrc/linear_outer.hpp"],
    "bf16_per_sample_kernel": ["paper_2109_12298_amd/csrc/linear_bf16.hip"],
    "bf16_clipsum_kernel": ["paper_2109_12298_amd/csrc/linear_bf16.hip"],
    "bf16_clipsum_many_kernel": ["paper_2109_12298_amd/csrc/clipsum_many.hip",
                                 "paper_2109_12298_amd/csrc/bf16_stage.hpp"],
    "bf16_grad_sample_kernel": ["paper_2109_12298_amd/csrc/grad_sample_bf16.hip",
                                "paper_2109_12298_amd/csrc/bf16_stage.hpp"],
    "bf16_grad_group_kernel": ["paper_2109_12298_amd/csrc/grad_sample_bf16.hip",
                               "paper_2109_12298_amd/csrc/bf16_stage.hpp", "paper_2109_12298_amd/csrc/grad_many.hip"],
    "ps_gemm_kernel": ["paper_2109_12298_amd/csrc/linear.hip"],
    "ps_gemm_dma_kernel": ["paper_2109_12298_amd/csrc/linear.hip", "paper_2109_12298_amd/csrc/bf16_stage.hpp"],
    "ps_dma_group_kernel": ["paper_2109_12298_amd/csrc/linear.hip", "paper_2109_12298_amd/csrc/bf16_stage.hpp",
                            "paper_2109_12298_amd/csrc/linear_staged.hpp", "paper_2109_12298_amd/csrc/grad_many.hip"],
    "clipsum_gemm_kernel": ["paper_2109_12298_amd/csrc/linear.hip", "paper_2109_12298_amd/csrc/mfma_tile.hpp"],
    "conv_per_sample_kernel": ["paper_2109_12298_amd/csrc/conv2d.hip", "paper_2109_12298_amd/csrc/mfma_tile.hpp"],
    "colsum_kernel": ["paper_2109_12298_amd/csrc/clip.hip"],
    "emb_csr_kernel": ["paper_2109_12298_amd/csrc/embedding.hip"],
    "emb_fused_kernel": ["paper_2109_12298_amd/csrc/embedding.hip"],
    "emb_clipsum_kernel": ["paper_2109_12298_amd/csrc/clip.hip"],
    "ln_partial_kernel": ["paper_2109_12298_amd/csrc/layernorm.hip"],
    "ln_rows_kernel": ["paper_2109_12298_amd/csrc/layernorm.hip"],
    "lstm_bptt_kernel": ["paper_2109_12298_amd/csrc/lstm.hip"],
    "add_noise_kernel": ["paper_2109_12298_amd/csrc/noise.hip"],
    "colsum_many_kernel+finish_many_kernel": ["paper_2109_12298_amd/csrc/group.hip",
                                              "paper_2109_12298_amd/csrc/philox.hpp"],
    "norms_kernel": ["paper_2109_12298_amd/csrc/clip.hip"],
    "norms_clip_noise_kernel": ["paper_2109_12298_amd/csrc/group.hip", "paper_2109_12298_amd/csrc/philox.hpp"],
}


def kernel_sources(kernel):
    """The sources of a kernel, or of every kernel of a "+"-joined group of them."""
    out = []
    for k in kernel.split("+"):
        out += [f for f in KERNEL_SOURCES.get(k, []) if f not in out]
    return out


def traffic_for(kernel, workload, call):
    """HBM bytes per launch from committed counter runs, if the kernel source is unchanged."""
    path = os.path.join(ROOT, "profiles", "traffic.json")
    if not os.path.exists(path):
        return None
    with open(path) as f:
        table = json.load(f)
    rec = table.get("%s/%s" % (workload, call))
    if not rec or rec.get("kernel") != kernel:
        return None
    if rec.get("source_sha") != src_hash(kernel_sources(kernel)):
        return None
    return rec.get("bytes_per_launch")


def counters_for(kernel, workload, call):
    """The counter record of a call from a committed counter run, if the kernel source is unchanged."""
    path = os.path.join(ROOT, "profiles", "counters.json")
    if not os.path.exists(path):
        return None
    with open(path) as f:
        rec = json.load(f).get("%s/%s" % (workload, call))
    if not rec or rec.get("kernel") != kernel or rec.get("source_sha") != src_hash(kernel_sources(kernel)):
        return None
    return rec


# ---------------------------------------------------------------------------
# CPU baseline: the oracle on a bounded sample
# ---------------------------------------------------------------------------

SENTINEL = "FillFunctor<signed char>"


def record_traffic(meta_path, fetch_csv, write_csv):
    """Reduce two counter runs to HBM bytes per launch of the dominant call; update profiles/traffic.json."""
    import csv

    def load(path, counter):
        rows = {}
        for r in csv.DictReader(open(path)):
            if r["Counter_Name"] != counter:
                continue
            d = int(r["Dispatch_Id"])
            rows[d] = (r["Kernel_Name"], rows.get(d, ("", 0.0))[1] + float(r["Counter_Value"]))
        return [rows[d] for d in sorted(rows)]

    def regions(seq):
        # every measured block is bracketed by a pair of sentinel dispatches
        cut = [i for i, (k, _) in enumerate(seq) if SENTINEL in k]
        return [seq[a + 1:b] for a, b in zip(cut[0::2], cut[1::2])]

    with open(meta_path) as f:
        meta = json.load(f)
    calls = meta["calls"]
    per = {}
    for name, path in (("FETCH_SIZE", fetch_csv), ("WRITE_SIZE", write_csv)):
        reg = regions(load(path, name))
        if len(reg) != len(calls) + 1:
            raise SystemExit("record-traffic: %d sentinel regions in %s, expected %d"
                             % (len(reg), path, len(calls) + 1))
        copy = reg[-1]                       # [call 0] ... [call n-1] [copy]
        counted = sum(v for _, v in copy) * 1024.0      # a copy reads and writes copy_bytes
        factor = meta["copy_bytes"] / counted
        for n, r in zip(calls, reg):
            kernels = sorted({k.replace("(anonymous namespace)::", "").replace("void ", "").split("(")[0]
                              for k, _ in r})
            per.setdefault(n, {})[name] = (sum(v for _, v in r) * 1024.0 * factor / meta["launches"], factor,
                                           kernels)
    path = os.path.join(ROOT, "profiles", "traffic.json")
    table = json.load(open(path)) if os.path.exists(path) else {}
    for n in calls:
        kern = meta["kernels"][n]
        f, w = per[n]["FETCH_SIZE"], per[n]["WRITE_SIZE"]
        table["%s/%s" % (meta["workload"], n)] = {
            "kernel": kern, "source_sha": src_hash(kernel_sources(kern)),
            "bytes_per_launch": round(f[0] + w[0]), "fetch_bytes_per_launch": round(f[0]),
            "write_bytes_per_launch": round(w[0]), "fetch_scale": round(f[1], 4), "write_scale": round(w[1], 4),
            "algorithmic_bytes": meta["algorithmic_bytes"][n], "dispatched": f[2]}
    with open(path, "w") as fh:
        json.dump(table, fh, indent=1, sort_keys=True)
        fh.write("\n")
    for n in calls:
        k = "%s/%s" % (meta["workload"], n)
        print(k, table[k]["bytes_per_launch"], "algorithmic", table[k]["algorithmic_bytes"])


def record_counters(meta_path, csv_path):
    """Reduce one rocprofv3 --pmc pass of this benchmark (any counters, e.g.
    MfmaUtil SQ_INSTS_VALU_MFMA_MOPS_BF16 SQ_INSTS_VALU_MFMA_MOPS_F32) to per-launch
    figures of each event-timed call block; update profiles/counters.json.

    MfmaUtil (rocprofv3's derived counter: MFMA-busy cycles over the active
    cycles of all 1024 SIMDs, in percent) is averaged over the block's
    dispatches weighted by their duration; every other counter is summed over
    the block and divided by the number of launches.  The MOPS counters count
    MFMA multiply-adds in units of 256 (512 flops), so they give the MFMA
    flops a launch actually issued, next to its algorithmic flops."""
    import csv

    with open(meta_path) as f:
        meta = json.load(f)
    calls = meta["calls"]
    rows = {}
    for r in csv.DictReader(open(csv_path)):
        d = int(r["Dispatch_Id"])
        e = rows.setdefault(d, {"kernel": r["Kernel_Name"], "ns": 0.0, "c": {}})
        if "End_Timestamp" in r and "Start_Timestamp" in r:
            e["ns"] = float(r["End_Timestamp"]) - float(r["Start_Timestamp"])
        e["c"][r["Counter_Name"]] = e["c"].get(r["Counter_Name"], 0.0) + float(r["Counter_Value"])
    seq = [rows[d] for d in sorted(rows)]
    cut = [i for i, e in enumerate(seq) if SENTINEL in e["kernel"]]
    regs = [seq[a + 1:b] for a, b in zip(cut[0::2], cut[1::2])]
    if len(regs) < len(calls):
        raise SystemExit("record-counters: %d sentinel regions in %s, expected %d" % (len(regs), csv_path,
                                                                                     len(calls)))
    path = os.path.join(ROOT, "profiles", "counters.json")
    table = json.load(open(path)) if os.path.exists(path) else {}
    for n, reg in zip(calls, regs):
        kern = meta["kernels"][n]
        names = sorted({k for e in reg for k in e["c"]})
        rec = {"kernel": kern, "source_sha": src_hash(kernel_sources(kern)), "launches": meta["launches"],
               "algorithmic_flops": meta.get("algorithmic_flops", {}).get(n)}
        for k in names:
            if k == "MfmaUtil":
                w = [max(e["ns"], 1.0) for e in reg if k in e["c"]]
                v = [e["c"][k] for e in reg if k in e["c"]]
                rec[k] = round(sum(a * b for a, b in zip(v, w)) / sum(w), 3)
            else:
                rec[k] = sum(e["c"].get(k, 0.0) for e in reg) / meta["launches"]
        for k in names:
            if k.startswith("SQ_INSTS_VALU_MFMA_MOPS_"):
                rec[k.replace("SQ_INSTS_VALU_MFMA_MOPS_", "mfma_flops_")] = rec[k] * 512
        table["%s/%s" % (meta["workload"], n)] = rec
    with open(path, "w") as fh:
        json.dump(table, fh, indent=1, sort_keys=True)
        fh.write("\n")
    for n in calls:
        print("%s/%s" % (meta["workload"], n), {k: v for k, v in table["%s/%s" % (meta["workload"], n)].items()
                                                 if k not in ("source_sha",)})


def cpu_model() -> str:
    try:
        for line in open("/proc/cpuinfo"):
            if line.startswith("model name"):
                return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return "unknown"


def cpu_baseline(wl, inputs, budget_s: float):
    """The oracle's whole step on a bounded sample of the batch: the median of
    three runs on all of the host's cores, and of three single-threaded runs
    on a smaller sample."""
    import numpy as np
    import oracle
    from paper_2109_12298_amd import workloads as W
    N = wl.N

    def sub(n):
        return [W.LayerInputs(li.layer, A=None if li.A is None else li.A[:n], B=li.B[:n],
                              ids=None if li.ids is None else li.ids[:n]) for li in inputs]

    def timed(n, step):
        s_ = sub(n)
        t0 = time.perf_counter()
        oracle.dp_step(wl, s_, step=step, denom=float(N))
        return time.perf_counter() - t0

    cores = oracle.num_threads()
    # a sample of n samples, grown until one multi-threaded step takes about a
    # sixth of the budget (three of them here, three single-threaded below)
    n = max(1, min(N, 8))
    while True:
        dt = timed(n, 0)
        if dt > budget_s / 6 or n >= N:
            break
        n = min(N, n * 4 if dt < budget_s / 60 else n * 2)
    mt = sorted(timed(n, k + 1) for k in range(3))[1]
    n1 = max(1, n // cores)
    oracle.set_num_threads(1)
    try:
        st1 = sorted(timed(n1, k + 4) for k in range(3))[1]
    finally:
        oracle.set_num_threads(cores)
    return {"value": round(n / mt, 3), "unit": "samples/s", "cores": cores, "kind": "oracle",
            "cpu_model": cpu_model(), "nproc": len(os.sched_getaffinity(0)),
            "median_of": 3, "step_s": round(mt, 3),
            "sample": "%d of the %d samples of one batch, whole step (grads, norms, clip, sum, noise over all "
                      "parameters), median of 3 runs on %d threads" % (n, N, cores),
            "single_thread": {"value": round(n1 / st1, 3), "unit": "samples/s", "cores": 1, "step_s": round(st1, 3),
                              "sample": "%d of the %d samples, median of 3 runs" % (n1, N)}}


def percentiles(ms):
    import numpy as np
    a = np.asarray(ms, dtype=np.float64)
    return {"median": round(float(np.median(a)), 4), "p10": round(float(np.percentile(a, 10)), 4),
            "p90": round(float(np.percentile(a, 90)), 4)}


# ---------------------------------------------------------------------------

def main():
    ap = argparse.ArgumentParser(description=__doc__, formatter_class=argparse.RawDescriptionHelpFormatter)
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=200)
    ap.add_argument("--warmup", type=int, default=20)
    ap.add_argument("--workload", default="transformer_block",
                    help="default: the transformer encoder block (N=32, T=128, d_model 768, bf16), the largest "
                         "workload; the others are parity cases")
    ap.add_argument("--cpu-seconds", type=float, default=20.0)
    ap.add_argument("--cold-reps", type=int, default=20,
                    help="cold-cache steps: one step per replay after a write of --flush-mib of scratch")
    ap.add_argument("--flush-mib", type=int, default=512)
    ap.add_argument("--clip-mode", default="auto", choices=["auto", "fused", "colreduce"],
                    help="clipped-sum route of Linear layers (default: per layer by modelled cost)")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--breakdown", action="store_true", help="print per-call event times to stderr")
    ap.add_argument("--eager", action="store_true", help="time eager launches instead of graph replays")
    ap.add_argument("--virtual-batches", type=int, default=1,
                    help="K > 1: virtual steps, K physical batches (the resident inputs each time) per logical "
                         "step, noised once; a step of the timed region is a logical step of K*N samples")
    ap.add_argument("--norm-mode", default="materialize", choices=["materialize", "ghost"],
                    help="ghost: Linear layers with a fused clipped sum and 2T^2 < d_in*d_out take their "
                         "per-sample norms from the Gram matrices and never form per-sample gradients")
    ap.add_argument("--steps-per-replay", type=int, default=0,
                    help="steps recorded in the replayed graph (default: the largest of 10, 8, 5, 4, 2, 1 "
                         "dividing --steps)")
    ap.add_argument("--copy-calibration-mib", type=int, default=0,
                    help="also run a plain device copy of this size (for counter calibration)")
    ap.add_argument("--meta-out", default="", help="write the dominant call's name and launch count here")
    ap.add_argument("--record-traffic", nargs=3, metavar=("META", "FETCH_CSV", "WRITE_CSV"),
                    help="reduce two rocprofv3 counter runs of this benchmark into profiles/traffic.json")
    ap.add_argument("--record-counters", nargs=2, metavar=("META", "CSV"),
                    help="reduce one rocprofv3 --pmc run of this benchmark into profiles/counters.json")
    args = ap.parse_args()
    if args.record_traffic:
        record_traffic(*args.record_traffic)
        return
    if args.record_counters:
        record_counters(*args.record_counters)
        return
    world = int(os.environ.get("WORLD_SIZE", "1"))
    if args.gpus != 1 or world != 1:
        print("bench.py: the DP-SGD step runs on one GPU only; --gpus %d is not supported "
              "(across GPUs the step would shard by samples, with one all-reduce of the clipped sums)"
              % max(args.gpus, world), file=sys.stderr)
        sys.exit(2)

    import torch
    from paper_2109_12298_amd import workloads as W
    from paper_2109_12298_amd.step import DPStep

    wl = W.get(args.workload)
    log("[bench] workload %s: drawing inputs" % wl.name)
    inputs = W.make_inputs(wl)
    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    st = DPStep(wl, inputs, dev, clip_mode=args.clip_mode, norm_mode=args.norm_mode,
                virtual_batches=args.virtual_batches)
    K = args.virtual_batches

    def eager_step(i):
        for k in range(K):
            st.run(step=i, clear_status=(k == 0), reset=(k == 0), emit=(k == K - 1))
    stream = torch.cuda.current_stream(dev)

    for i in range(3):
        eager_step(i)
    torch.cuda.synchronize()
    # an Embedding layer's CSR holds row_ptr[N] rows: priced at that count
    nnz = {lb.layer.name: int(lb.row_ptr[-1].item()) for lb in st.layers if isinstance(lb.layer, W.Embedding)}
    costs = call_costs(st, nnz)

    # the timed region: K whole steps, replayed from a captured HIP graph that
    # holds r steps back to back (r the largest of 10, 8, 5, 4, 2, 1 that
    # divides K, so that a replay's launch overhead is shared by r steps);
    # eager launches with --eager
    r = args.steps_per_replay or next(d for d in (10, 8, 5, 4, 2, 1) if args.steps % d == 0)
    if args.steps % r:
        raise SystemExit("--steps must be a multiple of --steps-per-replay")
    if not args.eager:
        st.capture(first_step=0, steps_per_replay=r)
        r = st.steps_per_replay          # one when graph branches were the faster
    for i in range(max(args.warmup // r, 1) if not args.eager else args.warmup):
        st.replay() if not args.eager else eager_step(i)
    torch.cuda.synchronize()
    # HIP events on the replay stream around every replay (or eager step)
    # give the spread of step times; the wall clock around the whole region
    # gives the value
    n_rep = args.steps if args.eager else args.steps // r
    ev = [torch.cuda.Event(enable_timing=True) for _ in range(n_rep + 1)]
    t0 = time.perf_counter()
    ev[0].record(stream)
    if args.eager:
        for i in range(args.steps):
            eager_step(args.warmup + i)
            ev[i + 1].record(stream)
    else:
        for i in range(n_rep):
            st.replay()
            ev[i + 1].record(stream)
    torch.cuda.synchronize()
    elapsed = time.perf_counter() - t0
    per_step = [ev[i].elapsed_time(ev[i + 1]) / (1 if args.eager else r) for i in range(n_rep)]
    warm = percentiles(per_step)
    status = int(st.status.item())
    if status != 0:
        log("[bench] device status flags %d" % status)

    # cold cache: one step per replay, each after a write of flush-mib of
    # scratch that evicts the inputs from the 256 MB Infinity Cache and the L2s
    cold = None
    if args.cold_reps > 0 and not args.eager:
        flush = torch.empty((args.flush_mib << 20) // 4, dtype=torch.float32, device=dev)
        st.capture(first_step=args.steps, parallel=st.graph_parallel, steps_per_replay=1)
        st.replay()
        ce = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))
              for _ in range(args.cold_reps)]
        for j in range(args.cold_reps):
            flush.fill_(float(j))
            ce[j][0].record(stream)
            st.replay()
            ce[j][1].record(stream)
        torch.cuda.synchronize()
        cold_ms = [a.elapsed_time(b) for a, b in ce]
        cold = percentiles(cold_ms)
        cold.update({"samples_per_s": round(K * wl.N / (cold["median"] * 1e-3), 1), "reps": args.cold_reps,
                     "flush_mib": args.flush_mib, "steps_per_replay": 1})
        del flush
        status |= int(st.status.item())

    # eager launches of the same steps, for comparison
    torch.cuda.synchronize()
    t1 = time.perf_counter()
    for i in range(args.steps):
        eager_step(i)
    torch.cuda.synchronize()
    eager_ms = (time.perf_counter() - t1) * 1e3 / args.steps

    # each call's kernel time: HIP events on the step's stream around one
    # replay of a HIP graph holding K back-to-back launches of that call
    # alone (so the GPU, not the host's launch rate, sets the pace);
    # consecutive blocks are bracketed by a sentinel kernel so that counter
    # runs can attribute every dispatch
    names = list(costs)
    sentinel = torch.empty(64, dtype=torch.int8, device=dev)
    avg = {}
    for n in names:
        side = torch.cuda.Stream(dev)
        side.wait_stream(stream)
        with torch.cuda.stream(side):
            st.call(n, step=0)                  # warm up outside the capture
        stream.wait_stream(side)
        torch.cuda.synchronize()
        g = torch.cuda.CUDAGraph()
        with torch.cuda.graph(g):
            for i in range(args.steps):
                st.call(n, step=i)
        g.replay()                              # first replay uploads the graph
        torch.cuda.synchronize()
        sentinel.fill_(1)
        e0 = torch.cuda.Event(enable_timing=True)
        e1 = torch.cuda.Event(enable_timing=True)
        e0.record(stream)
        g.replay()
        e1.record(stream)
        sentinel.fill_(1)
        torch.cuda.synchronize()
        avg[n] = e0.elapsed_time(e1) / args.steps
        del g
    if args.copy_calibration_mib > 0:
        nb = args.copy_calibration_mib << 20
        a = torch.empty(nb // 4, dtype=torch.float32, device=dev).fill_(1.0)
        b = torch.empty_like(a)
        torch.cuda.synchronize()
        sentinel.fill_(1)
        b.copy_(a)
        sentinel.fill_(1)
        torch.cuda.synchronize()
    dominant = max(avg, key=avg.get)
    dom_ms = avg[dominant]
    if args.breakdown:
        for n in names:
            b, f, k, _ = costs[n]
            log("[breakdown] %-18s %9.2f us  %10.3f MB  %9.3f GFLOP  %s" % (n, avg[n] * 1e3, b / 1e6, f / 1e9, k))

    ms = elapsed * 1e3 / args.steps
    nbytes, flops, kname, mfma_dtype = costs[dominant]
    dt_s = dom_ms * 1e-3
    hbm_s = nbytes / (HBM_PEAK_GBS * 1e9)
    dtype = "bf16" if wl.dtype == W.BF16 else "f32"
    # MFMA kernels are priced at their own input type's matrix peak; noise and
    # the column reductions are VALU/HBM work and are compared against HBM
    mfma_s = flops / (PEAK_TFLOPS[mfma_dtype] * 1e12) if mfma_dtype in PEAK_TFLOPS else 0.0
    if mfma_dtype == "alu":
        roof = {"bound": "alu", "achieved": round(flops / dt_s / 1e12, 3), "peak": ALU_PEAK_TFLOPS,
                "unit": "TFLOP/s"}
    elif mfma_s > hbm_s:
        roof = {"bound": "mfma", "achieved": round(flops / dt_s / 1e12, 3), "peak": PEAK_TFLOPS[mfma_dtype],
                "unit": "TFLOP/s"}
    else:
        roof = {"bound": "hbm", "achieved": round(nbytes / dt_s / 1e9, 1), "peak": HBM_PEAK_GBS, "unit": "GB/s"}
    roof["frac"] = round(roof["achieved"] / roof["peak"], 4)
    # counter records are kept per workload and norm mode (the ghost step's calls differ)
    pkey = wl.name + ("+ghost" if args.norm_mode == "ghost" else "")
    roof["traffic"] = traffic_for(kname, pkey, dominant)
    crec = counters_for(kname, pkey, dominant)
    # MFMA-busy fraction from a committed counter run of the same kernel source (null otherwise)
    roof["mfma_busy_counter"] = None if crec is None or "MfmaUtil" not in crec else round(crec["MfmaUtil"] / 100, 4)
    roof.update({"kernel": kname, "call": dominant, "avg_us": round(dom_ms * 1e3, 2),
                 "algorithmic_bytes": nbytes, "algorithmic_flops": flops})

    line = {"metric": METRIC, "value": round(K * wl.N * args.steps / elapsed, 1), "unit": "samples/s",
            "n_gpus": 1, "steps": args.steps, "warmup": args.warmup, "ms_per_step": round(ms, 4),
            "launch": "eager" if args.eager else
            ("hip_graph_branches" if st.graph_parallel else "hip_graph_chain"),
            "steps_per_replay": 1 if args.eager else r,
            "ms_per_step_warm": warm,
            "cold_cache": cold,
            "eager_ms_per_step": round(eager_ms, 4),
            "higher_is_better": True, "scaling": "weak", "vs_baseline": None, "dtype": dtype,
            "data": "synthetic",
            "config": {"workload": wl.name, "batch": wl.N, "params": wl.n_params,
                       "layers": [l.name for l in wl.layers], "C": wl.C, "sigma": wl.sigma,
                       "norms": args.norm_mode, "virtual_batches": K},
            "roofline": roof}
    if args.meta_out:
        with open(args.meta_out, "w") as f:
            json.dump({"workload": pkey, "calls": names, "launches": args.steps,
                       "kernels": {n: costs[n][2] for n in names},
                       "algorithmic_bytes": {n: costs[n][0] for n in names},
                       "algorithmic_flops": {n: costs[n][1] for n in names},
                       "avg_us": {n: round(avg[n] * 1e3, 2) for n in names},
                       "copy_bytes": args.copy_calibration_mib << 20}, f)
    if not args.no_cpu_baseline:
        log("[bench] timing the oracle on the host")
        line["cpu_baseline"] = cpu_baseline(wl, inputs, args.cpu_seconds)
    print(json.dumps(line), flush=True)


if __name__ == "__main__":
    main()
