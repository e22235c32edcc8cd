#!/usr/bin/env python
"""Benchmark of the Forward-Forward hot path on one MI355X.

One step = one pipelined training epoch of the 784->2000x4 FF net over the
60 000-vector MNIST-shaped set in 1024+1024-row chunks (one HIP stream per
layer; label embedding, normalisation, fused forward+goodness, loss, dW+Adam,
activity handoff), followed by goodness label scoring of the 10 000-vector
MNIST-shaped set under all 10 labels through a 784->2000x4 net.  Inputs are
seeded synthetic data resident in HBM before the timed region.

Prints one JSON line.  ``value`` is the step's pos+neg layer-step samples
per second over the whole train+score step (training rows x layers /
ms_per_step); the training and scoring parts are also reported on their own
(HIP-event timed: ``train_samples_per_s``, ``images_per_s``).  ``roofline`` is
the dominant kernel's one-stream figure: the step replayed with every layer on
one HIP stream, HIP events around each launch, algorithmic flops over the
summed durations of all its launches in the step (every shape it runs at,
weighted by its launches); ``roofline_overlapped`` is the same kernel inside
the timed, stream-overlapped steps.  ``cpu_baseline`` is the CPU oracle timed
on a bounded sample.

Profiling modes (for rocprofv3 runs): ``--replay K`` (K one-stream steps),
``--focus`` (layer steps of one shape) and ``--hbm`` (the row kernels at their
bench shapes) record every launch and write the list to ``--launch-list``;
``--rocprof-shapes`` matches a rocprofv3 kernel trace of such a run to that
list, launch by launch, and prints per-kernel, per-shape durations and
roofline fractions.
"""
import argparse
import hashlib
import itertools
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

METRIC = ("FF train pos+neg samples/sec per layer-step and label-scored images/sec; "
          "% MFMA peak")
PEAK = {"f32": ("mfma", 157.3, "TFLOP/s"), "bf16": ("mfma", 2500.0, "TFLOP/s")}
HBM_PEAK_GBS = 8000.0


def log(msg):
    print(msg, file=sys.stderr, flush=True)


def kernel_source_hash():
    h = hashlib.sha256()
    with open(os.path.join(ROOT, "paper_2404_08573_amd", "csrc", "ff_kernels.hip"), "rb") as f:
        h.update(f.read())
    return h.hexdigest()[:16]


def load_traffic(kernel, workload):
    """HBM bytes per launch from committed rocprofv3 counter runs, if the kernel is unchanged."""
    p = os.path.join(ROOT, "profiles", "traffic.json")
    if not os.path.exists(p):
        return None
    try:
        d = json.load(open(p))
        e = d.get(workload, {}).get(kernel)
        if not e or e.get("kernel_source_sha256_16") != kernel_source_hash():
            return None
        return e["bytes_per_launch"]
    except Exception:
        return None


KIND_OF = [("k_fwd", "forward"), ("k_dw_adam", "dw_adam"), ("k_dw4", "dw_adam"),
           ("k_embed_norm", "embed_norm"), ("k_loss_rows", "loss"), ("k_loss_t", "loss"),
           ("k_goodness", "goodness"), ("k_argmax", "argmax"), ("k_bf16_shadow", "bf16_shadow"),
           ("k_head_", "head"), ("k_po_dz", "head"),
           ("k_adam_dense", "adam")]
MFMA_KINDS = ("forward", "dw_adam")
ROW_MODES = ["rows", "pairs", "expand", "masked", "neutral"]
HEAD_PARTS = ["", "logits", "layer dZ", "grad partials", "Adam"]


def kind_of(kernel_name):
    return next((k for pat, k in KIND_OF if pat in kernel_name), None)


def shape_label(r):
    """Shape of a recorded launch (sizes by kind as ff_launch_record documents)."""
    kind, m, n, k, aux = r["kind"], r["m"], r["n"], r["k"], r["aux"]
    if kind == "forward":
        return f"{m}x{k}->{n}" + (f" (x{aux} labels)" if aux else "")
    if kind == "dw_adam":
        return f"{n}->{m} over {k} rows" + (" (gradient out)" if aux else "")
    if kind == "adam":
        return f"{m}x{n}"
    if kind == "head":
        return f"{m}x{k}->{n} classes ({HEAD_PARTS[aux]})"
    if kind == "loss":
        return f"{m}x{n}" + (" (+bf16 dZ^T)" if aux & 1 else "") + \
            (" (+next layer operand)" if aux & 2 else "") + \
            (" (+input transpose)" if aux & 4 else "")
    if kind == "goodness":
        return f"{m} rows x {n} partials"
    if kind == "embed_norm":
        return f"{m}x{n} ({ROW_MODES[aux & 15]}, {'bf16' if aux & 16 else 'fp32'} out)"
    return f"{m}x{n}"


def by_shape(recs, dname, durations=None):
    """Per (kernel kind, shape) of the launches: count, average duration,
    algorithmic work per launch and the rate against its roofline (MFMA peak of
    the dtype for the two products, 8 TB/s HBM for the rest).  durations (us,
    one per record) replaces the records' event times."""
    import collections
    groups = collections.OrderedDict()
    for i, r in enumerate(recs):
        us = durations[i] if durations is not None else r["ms"] * 1e3
        groups.setdefault((r["kind"], shape_label(r)), []).append((r, us))
    out = []
    for (kind, lab), rs in groups.items():
        n = len(rs)
        tot_s = sum(us for _, us in rs) * 1e-6
        fl = sum(r["flops"] for r, _ in rs)
        by = sum(r["bytes"] for r, _ in rs)
        e = {"kernel": kind, "shape": lab, "launches": n, "avg_us": tot_s * 1e6 / n,
             "flops_per_launch": fl / n, "bytes_per_launch": by / n}
        if kind in MFMA_KINDS:
            e["TFLOP/s"] = fl / tot_s / 1e12
            e["frac"] = e["TFLOP/s"] / PEAK[dname][1]
        else:
            e["GB/s"] = by / tot_s / 1e9
            e["frac"] = e["GB/s"] / HBM_PEAK_GBS
        out.append(e)
    return out


def kind_totals(recs, dname, durations=None):
    """Per kernel kind over all its launches: summed duration and the rate of
    its summed algorithmic work over it (the shape-weighted fraction)."""
    import collections
    acc = collections.OrderedDict()
    for i, r in enumerate(recs):
        us = durations[i] if durations is not None else r["ms"] * 1e3
        a = acc.setdefault(r["kind"], [0, 0.0, 0.0, 0.0])
        a[0] += 1
        a[1] += us
        a[2] += r["flops"]
        a[3] += r["bytes"]
    out = {}
    for kind, (n, us, fl, by) in acc.items():
        e = {"launches": n, "total_us": us, "avg_us": us / n}
        if kind in MFMA_KINDS:
            e["TFLOP/s"] = fl / (us * 1e-6) / 1e12
            e["frac"] = e["TFLOP/s"] / PEAK[dname][1]
        else:
            e["GB/s"] = by / (us * 1e-6) / 1e9
            e["frac"] = e["GB/s"] / HBM_PEAK_GBS
        out[kind] = e
    return out


def write_launch_list(path, recs, timed, dname, about, **extra):
    """The recorded launches, each marked timed (counted in the summaries) or not."""
    if path:
        for r, t in zip(recs, timed):
            r["timed"] = bool(t)
        with open(path, "w") as f:
            json.dump(dict({"about": about, "dtype": dname,
                            "kernel_source_sha256_16": kernel_source_hash(), "launches": recs},
                           **extra), f)


def rocprof_shapes(trace_csv, list_json):
    """Match the dispatches of this library's kernels in a rocprofv3 kernel
    trace (Dispatch_Id order) one to one with a recorded launch list (enqueue
    order, one stream), then print per-kernel, per-shape rocprof durations and
    fractions over the launches marked timed (markdown)."""
    import csv
    L = json.load(open(list_json))
    recs, dname = L["launches"], L["dtype"]
    ours = []
    for r in csv.DictReader(open(trace_csv)):
        kind = kind_of(r["Kernel_Name"])
        if kind is None:
            continue
        ours.append((int(r["Dispatch_Id"]), kind,
                     (int(r["End_Timestamp"]) - int(r["Start_Timestamp"])) * 1e-3))
    ours.sort()
    # the recorded launches are the trace's last ones (the runs launch nothing of
    # the library's after their profile stops; set-up, such as a bf16 layer's
    # first weight shadow, may come before it starts)
    skip = len(ours) - len(recs)
    if skip < 0:
        raise SystemExit(f"{len(ours)} dispatches of the library's kernels in the trace, "
                         f"{len(recs)} recorded launches")
    ours = ours[skip:]
    for i, ((_, kind, _), r) in enumerate(zip(ours, recs)):
        if kind != r["kind"]:
            raise SystemExit(f"launch {i}: trace has {kind}, list has {r['kind']}")
    sel = [i for i, r in enumerate(recs) if r["timed"]]
    n_all = len(recs)
    recs, us = [recs[i] for i in sel], [ours[i][2] for i in sel]
    print(f"Launch list: {L['about']} ({len(recs)} timed launches of {n_all}, matched to the "
          f"trace's last {n_all} dispatches of the library's kernels after {skip} earlier ones; "
          f"kernel source {L['kernel_source_sha256_16']}).  Durations: rocprofv3 kernel trace "
          f"(End - Start); `event avg` is the library's HIP-event time of the same launches.\n")
    print("| kernel | shape | launches | rocprof avg us | event avg us | work per launch "
          "| rate | fraction of peak |")
    print("|---|---|---|---|---|---|---|---|")
    rows_ev = {(e["kernel"], e["shape"]): e for e in by_shape(recs, dname)}
    for e in by_shape(recs, dname, us):
        evr = rows_ev[(e["kernel"], e["shape"])]
        work = (f"{e['flops_per_launch'] / 1e9:.3f} GFLOP" if e["kernel"] in MFMA_KINDS
                else f"{e['bytes_per_launch'] / 1e6:.2f} MB")
        rate = (f"{e['TFLOP/s']:.1f} TFLOP/s" if e["kernel"] in MFMA_KINDS
                else f"{e['GB/s']:.0f} GB/s")
        print(f"| {e['kernel']} | {e['shape']} | {e['launches']} | {e['avg_us']:.1f} | "
              f"{evr['avg_us']:.1f} | {work} | {rate} | {e['frac'] * 100:.1f} % |")
    print("\nShape-weighted per kernel kind (summed work / summed rocprof duration):\n")
    print("| kernel | launches | total us | rate | fraction of peak |")
    print("|---|---|---|---|---|")
    tot = 0.0
    for kind, e in kind_totals(recs, dname, us).items():
        tot += e["total_us"]
        rate = (f"{e['TFLOP/s']:.1f} TFLOP/s" if kind in MFMA_KINDS else f"{e['GB/s']:.0f} GB/s")
        print(f"| {kind} | {e['launches']} | {e['total_us']:.1f} | {rate} | "
              f"{e['frac'] * 100:.1f} % |")
    print(f"\nSum of the listed kernel durations: {tot / 1e3:.3f} ms"
          + (f" over {L['steps']} step(s), {tot / 1e3 / L['steps']:.3f} ms per step; "
             f"event-timed wall time of a step: {L['step_ms']:.3f} ms" if "steps" in L else ""))


def focus_steps(rows, d_in, d_out, bf16, steps=3, launch_list=None):
    """One untimed and `steps` recorded training steps of one layer shape on one
    stream: the workload of the per-shape rocprofv3 runs."""
    import torch
    import paper_2404_08573_amd as P
    from ffinputs import random_matrix, make_weights
    dev = torch.device("cuda:0")
    dt = P.FF_BF16 if bf16 else P.FF_F32
    x = torch.from_numpy(random_matrix(1, rows, d_in, 0, 1, 0.5)).to(dev)
    (W, b), = make_weights(2, (d_in, d_out))
    L = P.Layer(torch.from_numpy(W).to(dev), torch.from_numpy(b).to(dev), bool(bf16))
    hp = P.HParams(dtype=dt, lr=0.01)
    ws = P.workspace(P.ff_step_workspace_size(rows, d_in, d_out, dt), dev)
    torch.cuda.synchronize()
    P.ff_profile_start(1 << 14)
    a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    for i in range(1 + steps):
        if i == 1:
            a.record()
        P.ff_layer_step(L, hp, x, rows // 2, rows - rows // 2, ws=ws)
    b.record()
    torch.cuda.synchronize()
    _, recs = P.ff_profile_stop(launches=True)
    t0 = len(recs) // (1 + steps)
    dname = "bf16" if bf16 else "f32"
    write_launch_list(launch_list, recs, [i >= t0 for i in range(len(recs))], dname,
                      f"one untimed and {steps} timed layer steps {rows}x{d_in}->{d_out} "
                      f"{dname}, one stream", steps=steps, step_ms=a.elapsed_time(b) / steps)
    print(json.dumps({"focus": [rows, d_in, d_out, bf16], "steps": steps,
                      "step_ms": a.elapsed_time(b) / steps,
                      "shapes": by_shape(recs[t0:], dname)}))


def focus_epoch(rows, d_in, d_out, bf16, chunks=4, launch_list=None):
    """One untimed and one recorded pipelined epoch of a one-layer net over
    `chunks` chunks of rows/2 positive + rows/2 negative rows (label-embedded
    input rows of d_in features): the launch configuration of the pipelined
    epochs' layer steps (in bf16 the weight-gradient product and Adam run as
    separate launches), on one stream, for the per-shape rocprofv3 runs."""
    import torch
    import paper_2404_08573_amd as P
    from ffinputs import make_data, make_weights
    dev = torch.device("cuda:0")
    dt = P.FF_BF16 if bf16 else P.FF_F32
    b = rows // 2
    n = b * chunks
    x_base, y, y_neg = make_data(3, n, d_in, 0.0)
    (W, bias), = make_weights(4, (d_in, d_out))
    xd, yd, ynd = (torch.from_numpy(a).to(dev) for a in (x_base, y, y_neg))
    P.ff_profile_start(1 << 14)
    L = P.Layer(torch.from_numpy(W).to(dev), torch.from_numpy(bias).to(dev), bool(bf16))
    hp = P.HParams(dtype=dt, lr=0.01)
    ws = P.workspace(P.ff_pipeline_workspace_size([L], n, b, P.FF_PIPELINED, dt), dev)
    cur = torch.cuda.current_stream(dev)
    ev = [torch.cuda.Event(enable_timing=True) for _ in range(3)]
    for e in range(2):
        ev[e].record(cur)
        P.ff_pipeline_epoch([L], hp, xd, yd, ynd, 10, b, 1, P.FF_PIPELINED, streams=[cur],
                            ws=ws)
    ev[2].record(cur)
    torch.cuda.synchronize()
    _, recs = P.ff_profile_stop(launches=True)
    half = len(recs) // 2  # the second epoch's launches (the layer's shadow comes first)
    timed = [i >= len(recs) - half for i in range(len(recs))]
    dname = "bf16" if bf16 else "f32"
    step_ms = ev[1].elapsed_time(ev[2]) / chunks
    write_launch_list(launch_list, recs, timed, dname,
                      f"one untimed and one timed pipelined epoch of one {d_in}->{d_out} "
                      f"{dname} layer, {chunks} chunks of {b}+{b} rows, one stream",
                      steps=chunks, step_ms=step_ms)
    print(json.dumps({"focus_epoch": [rows, d_in, d_out, bf16], "chunks": chunks,
                      "step_ms": step_ms,
                      "shapes": by_shape([r for r, t in zip(recs, timed) if t], dname)}))


def copy_calibration(nbytes):
    """One plain device copy of nbytes (read nbytes, write nbytes): the reference
    that scales the FETCH_SIZE / WRITE_SIZE counters to bytes."""
    import torch
    src = torch.ones(nbytes // 4, device="cuda")
    dst = torch.empty_like(src)
    torch.cuda.synchronize()
    dst.copy_(src)
    torch.cuda.synchronize()
    print(json.dumps({"copy_bytes": nbytes}))


COPY_SWEEP_MB = (8, 25, 50, 100, 400, 1024)
COPY_SWEEP_REPS = 24


def _copy_rotation(mb):
    """Buffers per size: enough distinct ones to cover 600 MB (more than the
    256 MB last-level cache), at most 12."""
    return max(1, min(12, 600 // mb))


def copy_sweep():
    """Plain device copies (tensor copy_, which the HIP runtime runs as its own
    copy kernel) of each size in COPY_SWEEP_MB, COPY_SWEEP_REPS timed launches
    after one untimed pass over the buffers, each launch on a buffer pair the
    previous launches did not touch: the HBM rate a copy of that size reaches
    on this GPU, the calibration for the row kernels' fractions.  Prints the
    event-timed rate (launch gaps included); --copy-sweep-summary gives each
    copy's own duration from a rocprofv3 kernel trace of this run."""
    import torch
    dev = torch.device("cuda:0")
    out = {}
    for mb in COPY_SWEEP_MB:
        n = mb * (1 << 20) // 4
        nrot = _copy_rotation(mb)
        src = [torch.rand(n, device=dev) for _ in range(nrot)]
        dst = [torch.empty(n, device=dev) for _ in range(nrot)]
        for i in range(nrot):
            dst[i].copy_(src[i])
        torch.cuda.synchronize()
        a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        a.record()
        for k in range(COPY_SWEEP_REPS):
            dst[k % nrot].copy_(src[k % nrot])
        b.record()
        torch.cuda.synchronize()
        ms = a.elapsed_time(b) / COPY_SWEEP_REPS
        out[f"{mb}MB"] = {"us_per_copy": ms * 1e3, "GB/s": 2 * mb * (1 << 20) / (ms * 1e-3) / 1e9}
        del src, dst
        torch.cuda.empty_cache()
    print(json.dumps(out))


def copy_sweep_summary(trace_csv):
    """Per size of a --copy-sweep run's rocprofv3 kernel trace: the average
    duration of its timed copies (the runtime's copy-kernel dispatches, in
    order) and the rate of the bytes read and written against 8 TB/s."""
    import csv
    cps = sorted((int(r["Dispatch_Id"]), (int(r["End_Timestamp"]) - int(r["Start_Timestamp"])) * 1e-3)
                 for r in csv.DictReader(open(trace_csv)) if "copyBuffer" in r["Kernel_Name"])
    need = sum(_copy_rotation(mb) + COPY_SWEEP_REPS for mb in COPY_SWEEP_MB)
    if len(cps) != need:
        raise SystemExit(f"{len(cps)} copy dispatches in the trace, {need} expected")
    print("| copy size | bytes moved (read + write) | rocprof avg us | rate | fraction of 8 TB/s |")
    print("|---|---|---|---|---|")
    i = 0
    for mb in COPY_SWEEP_MB:
        i += _copy_rotation(mb)
        us = sum(u for _, u in cps[i:i + COPY_SWEEP_REPS]) / COPY_SWEEP_REPS
        i += COPY_SWEEP_REPS
        gbs = 2 * mb * (1 << 20) / (us * 1e-6) / 1e9
        print(f"| {mb} MiB | {2 * mb} MiB | {us:.1f} | {gbs:.0f} GB/s | "
              f"{gbs / HBM_PEAK_GBS * 100:.1f} % |")


def _counter_per_dispatch(csv_path, counter):
    """Mean value per dispatch of `counter`, by kernel kind and for the copy kernel."""
    import csv
    import collections
    tot = collections.defaultdict(float)
    n = collections.defaultdict(set)
    for r in csv.DictReader(open(csv_path)):
        if r["Counter_Name"] != counter:
            continue
        name = r["Kernel_Name"]
        kind = next((k for pat, k in KIND_OF if pat in name), None)
        if kind is None and ("copy" in name.lower() or "elementwise" in name):
            kind = "copy"
        if kind is None:
            continue
        tot[kind] += float(r["Counter_Value"])
        n[kind].add(r["Dispatch_Id"])
    return {k: tot[k] / len(n[k]) for k in tot}, {k: len(n[k]) for k in n}


def _largest_dispatch(csv_path, counter):
    """The copy run's largest single dispatch of `counter` (KiB): the calibration copy."""
    import csv
    return max(float(r["Counter_Value"]) for r in csv.DictReader(open(csv_path))
               if r["Counter_Name"] == counter)


def traffic_summary(fetch_csv, write_csv, cfetch_csv, cwrite_csv, workload, copy_bytes):
    """HBM bytes per launch for each kernel kind, scaled by the copy calibration."""
    f, nf = _counter_per_dispatch(fetch_csv, "FETCH_SIZE")
    w, _ = _counter_per_dispatch(write_csv, "WRITE_SIZE")
    kf = copy_bytes / (_largest_dispatch(cfetch_csv, "FETCH_SIZE") * 1024.0)
    kw = copy_bytes / (_largest_dispatch(cwrite_csv, "WRITE_SIZE") * 1024.0)
    out = {"_about": "HBM bytes per launch from rocprofv3 --pmc FETCH_SIZE and --pmc WRITE_SIZE "
                     "(KiB per dispatch) scaled by the factor each counter reads for a plain "
                     f"device copy of {copy_bytes} bytes; valid only for the kernel source hash",
           "fetch_factor": kf, "write_factor": kw}
    out[workload] = {k: {"bytes_per_launch": f[k] * 1024.0 * kf + w.get(k, 0.0) * 1024.0 * kw,
                         "fetch_bytes_per_launch": f[k] * 1024.0 * kf,
                         "write_bytes_per_launch": w.get(k, 0.0) * 1024.0 * kw,
                         "dispatches": nf[k], "kernel_source_sha256_16": kernel_source_hash()}
                     for k in f if k != "copy"}
    path = os.path.join(ROOT, "profiles", "traffic.json")
    old = json.load(open(path)) if os.path.exists(path) else {}
    old.update(out)
    json.dump(old, open(path, "w"), indent=1)
    print(json.dumps(out, indent=1))


def _per_dispatch(csv_path, counter):
    """[(dispatch id, kind, value)] of the library's kernels for one counter, in dispatch order."""
    import csv
    vals = {}
    for r in csv.DictReader(open(csv_path)):
        if r["Counter_Name"] != counter:
            continue
        kind = kind_of(r["Kernel_Name"])
        if kind is None:
            continue
        d = int(r["Dispatch_Id"])
        k, v = vals.get(d, (kind, 0.0))
        vals[d] = (kind, v + float(r["Counter_Value"]))
    return [(d, k, v) for d, (k, v) in sorted(vals.items())]


def traffic_by_shape(fetch_csv, write_csv, cfetch_csv, cwrite_csv, list_json, workload,
                     copy_bytes):
    """HBM bytes per launch by kernel and shape: the FETCH_SIZE / WRITE_SIZE runs of a
    --replay/--focus/--hbm command matched launch by launch to its recorded list (as
    rocprof_shapes does), each counter scaled by what it reads for a plain device copy
    of copy_bytes.  Prints a markdown table against the algorithmic bytes and stores
    the per-kind averages over the timed launches in profiles/traffic.json under
    `workload`, with the kernel source hash."""
    L = json.load(open(list_json))
    recs = L["launches"]
    kf = copy_bytes / (_largest_dispatch(cfetch_csv, "FETCH_SIZE") * 1024.0)
    kw = copy_bytes / (_largest_dispatch(cwrite_csv, "WRITE_SIZE") * 1024.0)
    cols = []
    for path, counter in ((fetch_csv, "FETCH_SIZE"), (write_csv, "WRITE_SIZE")):
        d = _per_dispatch(path, counter)
        skip = len(d) - len(recs)
        if skip < 0:
            raise SystemExit(f"{counter}: {len(d)} dispatches, {len(recs)} recorded launches")
        d = d[skip:]
        for i, ((_, kind, _), r) in enumerate(zip(d, recs)):
            if kind != r["kind"]:
                raise SystemExit(f"{counter} launch {i}: trace has {kind}, list has {r['kind']}")
        cols.append([v * 1024.0 for _, _, v in d])
    import collections
    groups = collections.OrderedDict()
    kinds = collections.OrderedDict()
    for i, r in enumerate(recs):
        if not r["timed"]:
            continue
        f, w = cols[0][i] * kf, cols[1][i] * kw
        for key, acc in (((r["kind"], shape_label(r)), groups), (r["kind"], kinds)):
            a = acc.setdefault(key, [0, 0.0, 0.0, 0.0])
            a[0] += 1
            a[1] += f
            a[2] += w
            a[3] += r["bytes"]
    print(f"Launch list: {L['about']} (kernel source {L['kernel_source_sha256_16']}).  "
          f"FETCH_SIZE x {kf:.3f}, WRITE_SIZE x {kw:.3f} (the factors a plain device copy of "
          f"{copy_bytes} bytes reads).\n")
    print("| kernel | shape | launches | fetched MB / launch | written MB / launch | "
          "algorithmic MB / launch | measured / algorithmic |")
    print("|---|---|---|---|---|---|---|")
    for (kind, lab), (n, f, w, a) in groups.items():
        print(f"| {kind} | {lab} | {n} | {f / n / 1e6:.1f} | {w / n / 1e6:.1f} | {a / n / 1e6:.1f} | "
              f"{(f + w) / a:.2f} |")
    out = {"_about": "HBM bytes per launch from rocprofv3 --pmc FETCH_SIZE and --pmc WRITE_SIZE "
                     "(KiB per dispatch) scaled by the factor each counter reads for a plain "
                     f"device copy of {copy_bytes} bytes, averaged over the timed launches of "
                     "each kernel kind; valid only for the kernel source hash",
           "fetch_factor": kf, "write_factor": kw}
    out[workload] = {k: {"bytes_per_launch": (f + w) / n, "fetch_bytes_per_launch": f / n,
                         "write_bytes_per_launch": w / n, "algorithmic_bytes_per_launch": a / n,
                         "dispatches": n, "kernel_source_sha256_16": L["kernel_source_sha256_16"]}
                     for k, (n, f, w, a) in kinds.items()}
    path = os.path.join(ROOT, "profiles", "traffic.json")
    old = json.load(open(path)) if os.path.exists(path) else {}
    old.update(out)
    json.dump(old, open(path, "w"), indent=1)


def counter_summary(csv_paths, n_simd=1024, n_xcd=8):
    """Per kernel kind, from rocprofv3 --pmc runs over `--focus` steps: MFMA
    busy fraction = SQ_VALU_MFMA_BUSY_CYCLES / (SIMDs x GPU-active cycles per
    XCD), with GRBM_GUI_ACTIVE summed over the XCDs; wait and LDS figures per
    wave cycle.  Prints a markdown table."""
    import csv
    import collections
    print("| run | kernel kind | dispatches | MFMA busy | wave cycles waiting | waiting on LDS "
          "| LDS bank conflicts / LDS instruction |")
    print("|---|---|---|---|---|---|---|")
    for path in csv_paths:
        agg = collections.defaultdict(lambda: collections.defaultdict(float))
        ids = collections.defaultdict(set)
        for r in csv.DictReader(open(path)):
            kind = next((k for pat, k in KIND_OF if pat in r["Kernel_Name"]), None)
            if kind is None:
                continue
            agg[kind][r["Counter_Name"]] += float(r["Counter_Value"])
            ids[kind].add(r["Dispatch_Id"])
        run = os.path.basename(os.path.dirname(path))
        for kind, c in agg.items():
            n = len(ids[kind])
            gui = c.get("GRBM_GUI_ACTIVE", 0.0) / n_xcd
            busy = c.get("SQ_VALU_MFMA_BUSY_CYCLES", 0.0) / n_simd / gui if gui else float("nan")
            wc = max(c.get("SQ_WAVE_CYCLES", 0.0), 1.0)
            lds = max(c.get("SQ_INSTS_LDS", 0.0), 1.0)
            print(f"| {run} | {kind} | {n} | {busy * 100:.1f} % | "
                  f"{c.get('SQ_WAIT_ANY', 0.0) / wc * 100:.1f} % | "
                  f"{c.get('SQ_WAIT_INST_LDS', 0.0) / wc * 100:.1f} % | "
                  f"{c.get('SQ_LDS_BANK_CONFLICT', 0.0) / lds:.3f} |")


def hbm_kernels(P, torch, reps=20, recorded=False):
    """The row / elementwise kernels alone on one stream at bandwidth-sized
    launches, each timed by the per-launch HIP events of the library's kernel
    timing: algorithmic bytes per launch / average launch duration, against
    the 8 TB/s HBM peak.  Inputs are seeded uniform(0, 1) rows drawn on the
    device; launches rotate over distinct buffers whose total exceeds the
    256 MB last-level cache, so each reads its inputs from HBM.  (Event pairs
    add a few microseconds to each launch: the rocprofv3 durations of the
    same launches, from --hbm, are the kernels' own.)
      embed_norm: normalisation of CIFAR-shaped rows (3072 features): one
        training chunk (4096 rows, bf16 out) and the 49 152-row prefix of the
        set (bf16 and fp32 out);
      bf16_shadow: the bf16 weight copy of a 3072 x 3072 layer.
    recorded: a profile that records every launch is already active (--hbm):
    the launches run without a profile of their own and nothing is returned."""
    from ffinputs import make_weights
    dev = torch.device("cuda:0")
    gen = torch.Generator(device=dev)
    gen.manual_seed(11)
    out = {}

    def timed(kind, fn):
        fn()
        torch.cuda.synchronize()
        if recorded:
            for _ in range(reps):
                fn()
            return None
        P.ff_profile_start(reps * 4, kinds=[kind])
        for _ in range(reps):
            fn()
        st = P.ff_profile_stop()[kind]
        gbs = st["bytes"] / (st["total_ms"] * 1e-3) / 1e9
        return {"avg_us": st["total_ms"] * 1e3 / st["launches"],
                "bytes_per_launch": st["bytes"] / st["launches"], "GB/s": gbs,
                "frac": gbs / HBM_PEAK_GBS, "launches": st["launches"]}

    d, d_out = 3072, 16
    (W, b), = make_weights(12, (d, d_out))
    x = torch.rand(49152, d, generator=gen, device=dev)
    # every launch reads rows the previous ones did not: consecutive row blocks
    # of the 604 MB set (more than the 256 MB last-level cache), round robin
    for rows, bf16 in ((4096, True), (49152, True), (49152, False)):
        dt = P.FF_BF16 if bf16 else P.FF_F32
        L = P.Layer(torch.from_numpy(W).to(dev), torch.from_numpy(b).to(dev), bf16)
        hp = P.HParams(dtype=dt)
        nrot = min(49152 // rows, 12)
        wss = [P.workspace(P.ff_step_workspace_size(rows, d, d_out, dt), dev) for _ in range(nrot)]
        turn = itertools.count()

        def fwd_next():
            i = next(turn) % nrot
            P.ff_layer_forward(L, hp, x[i * rows:(i + 1) * rows], ws=wss[i])
        r = timed("embed_norm", fwd_next)
        if r is not None:
            out[f"embed_norm_{rows}x{d}_{'bf16' if bf16 else 'f32'}_out"] = r
        del wss
    del x
    # 3072 x 3072 layers (37.7 MB of fp32 weights each), round robin over 12
    shadow = [P.Layer(torch.rand(3072, 3072, generator=gen, device=dev) - 0.5,
                      torch.zeros(3072, device=dev), True) for _ in range(12)]
    turn = itertools.count()
    r = timed("bf16_shadow", lambda: P.ff_refresh_bf16_shadow(shadow[next(turn) % 12]))
    if r is not None:
        out["bf16_shadow_3072x3072"] = r
    return out


def trace_epoch(name):
    """One untimed and one timed training epoch of workload `name`, launched as
    other_workloads launches them (fresh streams, one per layer), for a
    rocprofv3 kernel trace of how the layers' kernels share the GPU
    (--overlap-summary takes the second epoch's dispatches).  Prints one JSON
    line with the timed epoch's HIP-event time."""
    import torch
    import paper_2404_08573_amd as P
    from ffinputs import WORKLOADS, make_workload
    dev = torch.device("cuda:0")
    w = WORKLOADS[name]
    x_base, y, y_neg, params = make_workload(w)
    bf16 = w.dtype == "bf16"
    dtype = P.FF_BF16 if bf16 else P.FF_F32
    sched = P.FF_PIPELINED if w.schedule == "pipelined" else P.FF_SEQUENTIAL
    xd, yd, ynd = (torch.from_numpy(a).to(dev) for a in (x_base, y, y_neg))
    layers = [P.Layer(torch.from_numpy(W).to(dev), torch.from_numpy(b).to(dev), bf16)
              for W, b in params]
    hp = P.HParams(theta=w.theta, lr=w.lr, beta1=w.beta1, beta2=w.beta2, adam_eps=w.adam_eps,
                   norm_eps=w.norm_eps, dtype=dtype)
    ws = P.workspace(P.ff_pipeline_workspace_size(layers, w.n, w.chunk_pairs, sched, dtype), dev)
    cur = torch.cuda.current_stream(dev)
    streams = [cur] + [torch.cuda.Stream(dev) for _ in range(w.n_layers - 1)]

    def epoch():
        for s in streams[1:]:
            s.wait_stream(cur)
        P.ff_pipeline_epoch(layers, hp, xd, yd, ynd, w.n_classes, w.chunk_pairs, 1, sched,
                            streams=streams, ws=ws)
        for s in streams[1:]:
            cur.wait_stream(s)

    epoch()
    torch.cuda.synchronize()
    a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    a.record(cur)
    epoch()
    b.record(cur)
    torch.cuda.synchronize()
    print(json.dumps({"workload": name, "schedule": w.schedule, "dtype": w.dtype,
                      "epoch_ms": a.elapsed_time(b)}), flush=True)


def overlap_summary(trace_csv):
    """From a rocprofv3 kernel trace of a --trace-epoch run, the second epoch
    (the later half of the library's dispatches; both epochs launch the same
    kernels): its span, the time any kernel runs, the summed kernel time, each
    kernel kind's launches and durations, and the time each set of kinds runs
    together (markdown)."""
    import csv
    import collections
    ev = []
    for r in csv.DictReader(open(trace_csv)):
        kind = kind_of(r["Kernel_Name"])
        if kind is not None:
            ev.append((int(r["Dispatch_Id"]), int(r["Start_Timestamp"]),
                       int(r["End_Timestamp"]), kind))
    ev.sort()
    if len(ev) % 2:
        raise SystemExit(f"{len(ev)} dispatches of the library's kernels: not two equal epochs")
    ev = ev[len(ev) // 2:]
    t0, t1 = min(e[1] for e in ev), max(e[2] for e in ev)
    span = (t1 - t0) * 1e-3
    marks = sorted([(s, 1, k) for _, s, _, k in ev] + [(e, -1, k) for _, _, e, k in ev])
    active, last, by_mix = collections.Counter(), t0, collections.Counter()
    for t, d, k in marks:
        if t > last:
            mix = " + ".join(sorted(active.elements())) or "(none)"
            by_mix[mix] += (t - last) * 1e-3
        active[k] += d
        last = t
    busy = span - by_mix.get("(none)", 0.0)
    per = collections.defaultdict(lambda: [0, 0.0])
    for _, s, e, k in ev:
        per[k][0] += 1
        per[k][1] += (e - s) * 1e-3
    total = sum(v[1] for v in per.values())
    print(f"Second epoch: {len(ev)} dispatches of the library's kernels over {span / 1e3:.2f} ms; "
          f"some kernel runs {busy / span * 100:.1f} % of that time; summed kernel durations "
          f"{total / 1e3:.2f} ms ({total / span:.2f} kernels at once on average).\n")
    print("| kernel | launches | summed us | average us (beside the others) |")
    print("|---|---|---|---|")
    for k, (n, t) in sorted(per.items(), key=lambda x: -x[1][1]):
        print(f"| {k} | {n} | {t:.1f} | {t / n:.1f} |")
    print("\nTime by the set of kernel kinds running together (the 12 largest):\n")
    print("| kinds running | us | share of the epoch |")
    print("|---|---|---|")
    for mix, t in by_mix.most_common(12):
        print(f"| {mix} | {t:.1f} | {t / span * 100:.1f} % |")


def other_workloads(P, torch, names, reps=2, trials=3):
    """Training epochs of the other training workloads (the sequential fp32
    schedule of the same MNIST-shaped net, its bf16 form, and the CIFAR-shaped
    bf16 pipeline), each on its own, timed with HIP events around whole epochs
    after one untimed epoch.  Each of `trials` runs takes fresh streams: how
    the HIP runtime places a process's streams on its hardware queues varies,
    and a pipeline whose layer streams share a queue runs serialised in part
    (the CIFAR-shaped pipeline measured 23.5 to 29 ms that way).  epoch_ms is
    the median over the trials; all of them are reported."""
    from ffinputs import WORKLOADS, make_workload
    dev = torch.device("cuda:0")
    out = {}
    for name in names:
        w = WORKLOADS[name]
        log(f"bench: workload {name}")
        x_base, y, y_neg, params = make_workload(w)
        bf16 = w.dtype == "bf16"
        dtype = P.FF_BF16 if bf16 else P.FF_F32
        sched = P.FF_PIPELINED if w.schedule == "pipelined" else P.FF_SEQUENTIAL
        xd, yd, ynd = (torch.from_numpy(a).to(dev) for a in (x_base, y, y_neg))
        del x_base
        layers = [P.Layer(torch.from_numpy(W).to(dev), torch.from_numpy(b).to(dev), bf16)
                  for W, b in params]
        hp = P.HParams(theta=w.theta, lr=w.lr, beta1=w.beta1, beta2=w.beta2,
                       adam_eps=w.adam_eps, norm_eps=w.norm_eps, dtype=dtype)
        ws = P.workspace(P.ff_pipeline_workspace_size(layers, w.n, w.chunk_pairs, sched, dtype),
                         dev)
        cur = torch.cuda.current_stream(dev)
        trial_ms = []
        for _ in range(trials):
            streams = [cur] + [torch.cuda.Stream(dev) for _ in range(w.n_layers - 1)]

            def epoch():
                for s in streams[1:]:
                    s.wait_stream(cur)
                P.ff_pipeline_epoch(layers, hp, xd, yd, ynd, w.n_classes, w.chunk_pairs, 1,
                                    sched, streams=streams, ws=ws)
                for s in streams[1:]:
                    cur.wait_stream(s)

            epoch()
            torch.cuda.synchronize()
            a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            a.record(cur)
            for _ in range(reps):
                epoch()
            b.record(cur)
            torch.cuda.synchronize()
            trial_ms.append(a.elapsed_time(b) / reps)
        ms = sorted(trial_ms)[len(trial_ms) // 2]
        flops = sum(8.0 * bb * di * do for (_, bb) in w.chunks()
                    for di, do in zip(w.dims[:-1], w.dims[1:]))
        peak = PEAK["bf16" if bf16 else "f32"][1]
        out[name] = {"epoch_ms": ms, "epoch_ms_trials": trial_ms, "schedule": w.schedule,
                     "dtype": w.dtype,
                     "layers": list(w.dims), "samples": w.n,
                     "rows_per_layer_step": 2 * w.chunk_pairs,
                     "samples_per_s": 2 * w.n * w.n_layers / (ms * 1e-3),
                     "mfma_frac": flops / (ms * 1e-3) / 1e12 / peak}
        del xd, yd, ynd, layers, ws
        torch.cuda.empty_cache()
    return out


def softmax_head(P, torch, sw, sxd, slayers, reps=5, recorded=False):
    """Softmax prediction (one neutral-label pass + the softmax layer over the
    normalised activities of layers 1..) of the scoring set, and one training
    step of the softmax layer on it, each HIP-event timed on its own."""
    from ffinputs import make_data, random_matrix
    dev = torch.device("cuda:0")
    D = sum(sw.dims[2:])
    Wh = torch.from_numpy(random_matrix(96, sw.n_classes, D, -0.05, 0.05)).to(dev)
    head = P.Head(Wh, torch.zeros(sw.n_classes, device=dev))
    _, y, _ = make_data(sw.seed_data, sw.n, sw.dims[0], sw.p_zero, sw.n_classes)
    yd = torch.from_numpy(y).to(dev)
    hp = P.HParams(norm_eps=sw.norm_eps)
    hhp = P.HParams(lr=1e-4)
    ws = P.workspace(P.ff_head_workspace_size(slayers, 1, sw.n, sw.n_classes), dev)
    pred = torch.empty(sw.n, dtype=torch.int32, device=dev)
    loss = torch.empty(1, device=dev)
    if recorded:  # an outer profile records every launch (--hbm): the predictions only
        for _ in range(1 + reps):
            P.ff_head_predict(slayers, hp, head, sxd, 1, pred=pred, ws=ws)
        return None
    out = {}
    for name, fn in (("predict", lambda: P.ff_head_predict(slayers, hp, head, sxd, 1, pred=pred,
                                                           ws=ws)),
                     ("step", lambda: P.ff_head_step(slayers, hp, head, hhp, sxd, yd, 1,
                                                     loss=loss, ws=ws))):
        fn()
        torch.cuda.synchronize()
        a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        a.record()
        for _ in range(reps):
            fn()
        b.record()
        torch.cuda.synchronize()
        out[name + "_ms"] = a.elapsed_time(b) / reps
    out["images_per_s"] = sw.n / (out["predict_ms"] * 1e-3)
    out["features"] = D
    # the softmax layer's logits kernel alone: it reads every feature row once
    P.ff_profile_start(64, kinds=["head"])
    P.ff_head_predict(slayers, hp, head, sxd, 1, pred=pred, ws=ws)
    st = P.ff_profile_stop()["head"]
    gbs = st["bytes"] / (st["total_ms"] * 1e-3) / 1e9
    out["head_logits"] = {"avg_us": st["total_ms"] * 1e3 / max(st["launches"], 1),
                          "bytes_per_launch": st["bytes"] / max(st["launches"], 1),
                          "GB/s": gbs, "frac": gbs / HBM_PEAK_GBS}
    return out


def po_and_adaptive(P, torch, w, xd, yd, layers, reps=2):
    """Performance-Optimised PFF: pipelined epochs of the training workload's
    net and data (no negatives, a classifier per layer, classifier lr 1e-4).
    AdaptiveNEG: the hardest wrong label of every training sample under the
    trained net.  Each HIP-event timed on its own after one untimed call."""
    from ffinputs import random_matrix
    dev = torch.device("cuda:0")
    bf16 = w.dtype == "bf16"
    dtype = P.FF_BF16 if bf16 else P.FF_F32
    hp = P.HParams(theta=w.theta, lr=w.lr, norm_eps=w.norm_eps, dtype=dtype)
    hhp = P.HParams(lr=1e-4)
    heads = [P.Head(torch.from_numpy(random_matrix(97 + l, w.n_classes, d, -0.05, 0.05)).to(dev),
                    torch.zeros(w.n_classes, device=dev)) for l, d in enumerate(w.dims[1:])]
    ws = P.workspace(P.LIB.ff_po_epoch_workspace_size(P._lib._layers_c(layers), len(layers), w.n,
                                                      w.n_classes, w.chunk_pairs, P.FF_PIPELINED,
                                                      dtype), dev)
    cur = torch.cuda.current_stream(dev)
    streams = [cur] + [torch.cuda.Stream(dev) for _ in range(len(layers) - 1)]

    def po():
        for s in streams[1:]:
            s.wait_stream(cur)
        P.ff_po_epoch(layers, heads, hp, hhp, xd, yd, w.n_classes, w.chunk_pairs, 1,
                      P.FF_PIPELINED, streams=streams, ws=ws)
        for s in streams[1:]:
            cur.wait_stream(s)

    sws = P.workspace(P.ff_score_workspace_size(layers, w.n, w.n_classes, dtype), dev)
    yneg = torch.empty_like(yd)

    def adaptive():
        P.ff_adaptive_negatives(layers, hp, xd, yd, w.n_classes, 0, y_neg=yneg, ws=sws)

    out = {}
    for name, fn in (("po_epoch", po), ("adaptive_negatives", adaptive)):
        fn()
        torch.cuda.synchronize()
        a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        a.record(cur)
        for _ in range(reps):
            fn()
        b.record(cur)
        torch.cuda.synchronize()
        out[name + "_ms"] = a.elapsed_time(b) / reps
    flops = sum(4.0 * b * di * do for (_, b) in w.chunks()
                for di, do in zip(w.dims[:-1], w.dims[1:]))
    out["po_samples_per_s"] = w.n * w.n_layers / (out["po_epoch_ms"] * 1e-3)
    out["po_mfma_frac"] = flops / (out["po_epoch_ms"] * 1e-3) / 1e12 / PEAK["bf16" if bf16 else "f32"][1]
    out["adaptive_images_per_s"] = w.n / (out["adaptive_negatives_ms"] * 1e-3)
    return out


def chapters(P, torch, w, xd, yd, ynd, params, epochs=2, splits=2):
    """Chapter schedules (Alg. 1 Single-Layer on one stream per layer, Alg. 2
    All-Layers on two worker streams) of the training workload: `epochs` epochs
    in `splits` chapters, RandomNEG negatives redrawn per chapter, the rate
    cooled down from the second chapter.  Each run starts from fresh weights."""
    from ffinputs import random_labels
    dev = torch.device("cuda:0")
    bf16 = w.dtype == "bf16"
    dtype = P.FF_BF16 if bf16 else P.FF_F32
    hp = P.HParams(theta=w.theta, lr=w.lr, norm_eps=w.norm_eps, dtype=dtype)
    negs = torch.stack([ynd] + [torch.from_numpy(random_labels(200 + c, w.n)[1]).to(dev)
                                for c in range(1, splits)]).contiguous()
    out = {}
    for name, assignment, ns in (("single_layer", P.FF_SINGLE_LAYER, w.n_layers),
                                 ("all_layers", P.FF_ALL_LAYERS, 2)):
        layers = [P.Layer(torch.from_numpy(W).to(dev), torch.from_numpy(b).to(dev), bf16)
                  for W, b in params]
        ws = P.workspace(P.LIB.ff_chapter_workspace_size(P._lib._layers_c(layers), len(layers),
                                                         w.n, w.chunk_pairs, ns, dtype), dev)
        cur = torch.cuda.current_stream(dev)
        streams = [torch.cuda.Stream(dev) for _ in range(ns)]
        torch.cuda.synchronize()
        a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        a.record(cur)
        for s in streams:
            s.wait_stream(cur)
        P.ff_chapter_train(layers, hp, xd, yd, negs, w.n_classes, w.chunk_pairs, epochs, splits,
                           epochs // splits, assignment, streams=streams, ws=ws)
        for s in streams:
            cur.wait_stream(s)
        b.record(cur)
        torch.cuda.synchronize()
        ms = a.elapsed_time(b)
        out[name] = {"ms": ms, "streams": ns,
                     "samples_per_s": 2 * w.n * w.n_layers * epochs / (ms * 1e-3)}
        del layers, ws
    # AdaptiveNEG: chapter c's wrong labels are the hardest ones under the network
    # as chapter c starts, scored on the device (chapter 0 takes the scoring of the
    # fresh weights too)
    for name, assignment, ns in (("single_layer_adaptive", P.FF_SINGLE_LAYER, w.n_layers),
                                 ("all_layers_adaptive", P.FF_ALL_LAYERS, 2)):
        layers = [P.Layer(torch.from_numpy(W).to(dev), torch.from_numpy(b).to(dev), bf16)
                  for W, b in params]
        ws = P.workspace(P.LIB.ff_chapter_adaptive_workspace_size(
            P._lib._layers_c(layers), len(layers), w.n, w.n_classes, w.chunk_pairs, ns, dtype), dev)
        yneg = torch.empty(splits, w.n, dtype=torch.int32, device=dev)
        cur = torch.cuda.current_stream(dev)
        streams = [torch.cuda.Stream(dev) for _ in range(ns)]
        torch.cuda.synchronize()
        a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        a.record(cur)
        for s in streams:
            s.wait_stream(cur)
        P.ff_chapter_train_adaptive(layers, hp, xd, yd, w.n_classes, w.chunk_pairs, epochs,
                                    splits, epochs // splits, assignment, 0,
                                    y_neg_chapters=yneg, streams=streams, ws=ws)
        for s in streams:
            cur.wait_stream(s)
        b.record(cur)
        torch.cuda.synchronize()
        ms = a.elapsed_time(b)
        out[name] = {"ms": ms, "streams": ns,
                     "samples_per_s": 2 * w.n * w.n_layers * epochs / (ms * 1e-3),
                     "note": "includes scoring the 60 000 inputs under every label at each "
                             "chapter start"}
        del layers, ws
    out["epochs"], out["splits"] = epochs, splits
    return out


def cpu_baseline(w, x_base, y, y_neg, params, sw, sx, sparams, budget_s=12.0):
    """The oracle as it stands, on a bounded sample of the same workload."""
    import numpy as np
    import oracle as O
    try:
        from threadpoolctl import threadpool_info
        threads = max([i.get("num_threads", 1) for i in threadpool_info()] or [1])
    except Exception:
        threads = os.cpu_count()
    hp = O.HParams(theta=w.theta, lr=w.lr)
    layers = [O.Layer.from_params(W, b) for W, b in params]
    b = w.chunk_pairs
    t0 = time.perf_counter()
    steps = 0
    rows = 0
    # one chunk through every layer (each layer trains on the previous layer's
    # activities, as in the pipeline), repeated while the time budget lasts
    for c in range(len(w.chunks()) - 1):
        s = c * b
        x = O.chunk_input(x_base, y, y_neg, s, b, w.n_classes)
        for L in layers:
            r = O.layer_step(L, x, b, hp)
            x = r.h
            steps += 1
            rows += 2 * b
        if time.perf_counter() - t0 > budget_s * 0.6:
            break
    t_train = time.perf_counter() - t0
    train_rate = rows / t_train  # layer-step samples per second
    slayers = [O.Layer.from_params(W, b) for W, b in sparams]
    n_img = 0
    t1 = time.perf_counter()
    while n_img < sw.n and time.perf_counter() - t1 < budget_s * 0.4:
        O.score_labels(slayers, sx[n_img:n_img + 10], sw.n_classes, hp, 0)
        n_img += 10
    t_score = time.perf_counter() - t1
    img_rate = n_img / t_score
    # whole-step rate in the bench's unit: the same step on the CPU at these rates
    step_rows = 2 * w.n * w.n_layers
    step_time = step_rows / train_rate + sw.n / img_rate
    return {"value": step_rows / step_time, "unit": "pos+neg samples/s per layer-step",
            "cores": int(threads), "kind": "oracle",
            "sample": f"{steps} layer-steps of {2 * b} rows (chunks 0..{steps // w.n_layers - 1} "
                      f"through all {w.n_layers} layers, {t_train:.1f} s) and label scoring of "
                      f"{n_img} inputs ({t_score:.1f} s); fp64 NumPy, extrapolated to the step",
            "train_samples_per_s": train_rate, "images_per_s": img_rate,
            "tiny_config_one_thread_s": tiny_config_one_thread(),
            "host": host_info()}


def tiny_config_one_thread():
    """The oracle on the tiny configuration (784->500->500, 512 pairs, 5
    full-batch steps per layer, layer by layer, then scoring all 512 inputs
    under 10 labels) with one BLAS thread: seconds."""
    import oracle as O
    from ffinputs import WORKLOADS, make_workload
    try:
        from threadpoolctl import threadpool_limits
    except Exception:
        return None
    w = WORKLOADS["mnist_tiny_784_500x2"]
    x, y, yn, params = make_workload(w)
    hp = O.HParams(theta=w.theta, lr=w.lr)
    with threadpool_limits(limits=1):
        t0 = time.perf_counter()
        layers = [O.Layer.from_params(W, b) for W, b in params]
        O.train_sequential(layers, x, y, yn, w.n_classes, w.chunk_pairs, w.epochs, hp)
        O.score_labels(layers, x, w.n_classes, hp, 0)
        return time.perf_counter() - t0


def host_info():
    """CPU model and the BLAS NumPy uses, for the oracle baseline."""
    import numpy as np
    model = None
    try:
        for line in open("/proc/cpuinfo"):
            if line.startswith("model name"):
                model = line.split(":", 1)[1].strip()
                break
    except OSError:
        pass
    blas = None
    try:
        from threadpoolctl import threadpool_info
        blas = ", ".join(sorted({f"{i.get('internal_api')} {i.get('version')}"
                                 for i in threadpool_info() if i.get("user_api") == "blas"}))
    except Exception:
        pass
    return {"cpu_model": model, "logical_cpus": os.cpu_count(), "blas": blas,
            "numpy": np.__version__}


def main():
    ap = argparse.ArgumentParser(description=__doc__.split("\n")[0])
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=5)
    ap.add_argument("--warmup", type=int, default=2)
    ap.add_argument("--workload", default="mnist_784_2000x4_pipelined")
    ap.add_argument("--score-workload", default="mnist_score_784_2000x4")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-other-workloads", action="store_true",
                    help="skip the epochs of the other training workloads")
    ap.add_argument("--copy-calibration", type=int, metavar="BYTES", default=0,
                    help="run one plain device copy of BYTES (counter calibration) and exit")
    ap.add_argument("--traffic-summary", nargs=4, metavar="CSV",
                    help="FETCH, WRITE, copy FETCH, copy WRITE counter_collection.csv files: "
                         "write profiles/traffic.json for --workload and exit")
    ap.add_argument("--copy-bytes", type=int, default=1 << 30)
    ap.add_argument("--counter-summary", nargs="+", metavar="CSV",
                    help="counter_collection.csv files of rocprofv3 --pmc runs over --focus "
                         "steps: print MFMA-busy and wait fractions per kernel kind and exit")
    ap.add_argument("--focus", nargs=4, type=int, metavar=("ROWS", "D_IN", "D_OUT", "BF16"),
                    help="run a few layer steps of one shape on one stream (for counter runs)")
    ap.add_argument("--focus-epoch", nargs=4, type=int, metavar=("ROWS", "D_IN", "D_OUT", "BF16"),
                    help="run a one-layer pipelined epoch of that shape on one stream (the "
                         "pipelined epochs' launch configuration) and exit")
    ap.add_argument("--replay", type=int, metavar="K", default=0,
                    help="run one untimed and K recorded one-stream replays of the step "
                         "(every layer on one HIP stream, then the scoring) and exit")
    ap.add_argument("--hbm", action="store_true",
                    help="run the row kernels at their bench shapes (embedding + "
                         "normalisation, bf16 weight shadow, softmax-layer logits) with every "
                         "launch recorded and exit")
    ap.add_argument("--copy-sweep", action="store_true",
                    help="time plain device copies of 8 MiB to 1 GiB on cold buffers and exit "
                         "(the HBM calibration of the row kernels)")
    ap.add_argument("--copy-sweep-summary", metavar="KERNEL_TRACE_CSV",
                    help="per-size copy durations from a rocprofv3 kernel trace of --copy-sweep")
    ap.add_argument("--launch-list", metavar="JSON",
                    help="with --replay, --focus or --hbm: write the recorded launches here")
    ap.add_argument("--trace-epoch", metavar="WORKLOAD",
                    help="run one untimed and one timed training epoch of that workload (as "
                         "the other workloads run) for a kernel trace, and exit")
    ap.add_argument("--overlap-summary", metavar="KERNEL_TRACE_CSV",
                    help="busy time and kernel mixes of a --trace-epoch run's second epoch")
    ap.add_argument("--rocprof-shapes", nargs=2, metavar=("KERNEL_TRACE_CSV", "LAUNCH_LIST"),
                    help="match a rocprofv3 kernel trace of a --replay/--focus/--hbm run to its "
                         "launch list and print per-kernel, per-shape durations; exit")
    args = ap.parse_args()
    if args.copy_sweep:
        copy_sweep()
        return
    if args.copy_sweep_summary:
        copy_sweep_summary(args.copy_sweep_summary)
        return
    if args.rocprof_shapes:
        rocprof_shapes(*args.rocprof_shapes)
        return
    if args.overlap_summary:
        overlap_summary(args.overlap_summary)
        return
    if args.trace_epoch:
        trace_epoch(args.trace_epoch)
        return
    if args.focus:
        focus_steps(*args.focus, launch_list=args.launch_list)
        return
    if args.focus_epoch:
        focus_epoch(*args.focus_epoch, launch_list=args.launch_list)
        return
    if args.copy_calibration:
        copy_calibration(args.copy_calibration)
        return
    if args.counter_summary:
        counter_summary(args.counter_summary)
        return
    if args.traffic_summary:
        if args.launch_list:
            traffic_by_shape(*args.traffic_summary, args.launch_list, args.workload,
                             args.copy_bytes)
        else:
            traffic_summary(*args.traffic_summary, args.workload, args.copy_bytes)
        return
    if args.gpus != 1:
        print(f"bench.py measures one GPU only: this build has no multi-GPU path "
              f"(--gpus {args.gpus} requested)", file=sys.stderr)
        sys.exit(2)

    import numpy as np
    import torch

    import paper_2404_08573_amd as P
    from ffinputs import WORKLOADS, make_workload

    w = WORKLOADS[args.workload]
    sw = WORKLOADS[args.score_workload]
    dtype = P.FF_BF16 if w.dtype == "bf16" else P.FF_F32
    sched = P.FF_PIPELINED if w.schedule == "pipelined" else P.FF_SEQUENTIAL
    dev = torch.device("cuda:0")
    log(f"bench: generating {w.name} ({w.n} x {w.dims[0]}) and {sw.name} ({sw.n} x {sw.dims[0]})")
    x_base, y, y_neg, params = make_workload(w)
    sx, _, _, sparams = make_workload(sw)

    xd = torch.from_numpy(x_base).to(dev)
    yd = torch.from_numpy(y).to(dev)
    ynd = torch.from_numpy(y_neg).to(dev)
    sxd = torch.from_numpy(sx).to(dev)
    bf16 = dtype == P.FF_BF16
    layers = [P.Layer(torch.from_numpy(W).to(dev), torch.from_numpy(b).to(dev), bf16)
              for W, b in params]
    slayers = [P.Layer(torch.from_numpy(W).to(dev), torch.from_numpy(b).to(dev), bf16)
               for W, b in sparams]
    hp = P.HParams(theta=w.theta, lr=w.lr, beta1=w.beta1, beta2=w.beta2, adam_eps=w.adam_eps,
                   norm_eps=w.norm_eps, dtype=dtype)
    shp = P.HParams(theta=sw.theta, norm_eps=sw.norm_eps, dtype=dtype)
    nc = len(w.chunks())
    ws = P.workspace(P.ff_pipeline_workspace_size(layers, w.n, w.chunk_pairs, sched, dtype), dev)
    sws = P.workspace(P.ff_score_workspace_size(slayers, sw.n, sw.n_classes, dtype), dev)
    trace = torch.zeros(w.n_layers, nc, device=dev)
    scores = torch.empty(sw.n, sw.n_classes, device=dev)
    pred = torch.empty(sw.n, dtype=torch.int32, device=dev)
    cur = torch.cuda.current_stream(dev)
    side = [torch.cuda.Stream(dev) for _ in range(w.n_layers - 1)]
    streams = [cur] + side

    def step(ev=None, one_stream=False):
        for s in side:
            s.wait_stream(cur)
        if ev:
            ev[0].record(cur)
        P.ff_pipeline_epoch(layers, hp, xd, yd, ynd, w.n_classes, w.chunk_pairs, 1, sched,
                            streams=[cur] * w.n_layers if one_stream else streams,
                            loss_trace=trace, ws=ws)
        for s in side:
            cur.wait_stream(s)
        if ev:
            ev[1].record(cur)
        P.ff_score_labels(slayers, shp, sxd, sw.n_classes, 0, scores=scores, pred=pred, ws=sws)
        if ev:
            ev[2].record(cur)

    launches_per_step = 4 * (w.n_layers * nc * 5 + 4 * (sw.n // 1024 + 1) * 4 + 64)
    dname = "bf16" if bf16 else "f32"

    def replay(k):
        """k one-stream replays of the step, every launch recorded: (launches, ms per step)."""
        ev = [torch.cuda.Event(enable_timing=True) for _ in range(3)]
        P.ff_profile_start(launches_per_step * k)
        ev[0].record(cur)
        for _ in range(k):
            step(one_stream=True)
        ev[1].record(cur)
        torch.cuda.synchronize()
        _, recs = P.ff_profile_stop(launches=True)
        return recs, ev[0].elapsed_time(ev[1]) / k

    if args.replay:
        if args.hbm:
            raise SystemExit("--replay and --hbm are separate runs")
        log(f"bench: one untimed and {args.replay} recorded one-stream replay(s)")
        P.ff_profile_start(launches_per_step)
        step(one_stream=True)
        torch.cuda.synchronize()
        _, warm = P.ff_profile_stop(launches=True)
        recs, rms = replay(args.replay)
        about = (f"one untimed and {args.replay} recorded one-stream replays of the step: the "
                 f"{w.name} epoch with every layer on one HIP stream, then scoring {sw.name}")
        write_launch_list(args.launch_list, warm + recs,
                          [False] * len(warm) + [True] * len(recs), dname, about,
                          steps=args.replay, step_ms=rms)
        print(json.dumps({"replay_steps": args.replay, "step_ms": rms,
                          "kernels": kind_totals(recs, dname)}))
        return
    if args.hbm:
        P.ff_profile_start(1 << 14)
        hbm_kernels(P, torch, recorded=True)
        softmax_head(P, torch, sw, sxd, slayers, recorded=True)
        torch.cuda.synchronize()
        _, recs = P.ff_profile_stop(launches=True)
        # each kernel's first launch at a shape is untimed, its repeats are timed
        seen, timed = set(), []
        for r in recs:
            key = (r["kind"], shape_label(r))
            timed.append(key in seen)
            seen.add(key)
        write_launch_list(args.launch_list, recs, timed, dname,
                          "the row kernels at their bench shapes on one stream (with the "
                          "products that feed them): each kernel's first launch at a shape "
                          "untimed, its repeats timed")
        print(json.dumps({"shapes": by_shape([r for r, t in zip(recs, timed) if t], dname)}))
        return

    log(f"bench: warmup {args.warmup} step(s)")
    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()

    # One-stream replay: each launch runs alone, so its event time is the
    # kernel's own; the dominant product and its roofline come from here.
    log("bench: one-stream replay")
    step(one_stream=True)
    torch.cuda.synchronize()
    orecs, replay_ms = replay(1)
    otot = kind_totals(orecs, dname)
    dom = max((k for k in MFMA_KINDS if k in otot), key=lambda k: otot[k]["total_us"])

    # One untimed overlapped step with every launch bracketed by events: the
    # per-kernel table of the pipelined step.
    pev = [torch.cuda.Event(enable_timing=True) for _ in range(3)]
    P.ff_profile_start(launches_per_step)
    step(pev)
    torch.cuda.synchronize()
    kstats = P.ff_profile_stop()
    profiled_ms = pev[0].elapsed_time(pev[2])

    # Timed region: events around the dominant kernel's launches only (events
    # at every launch boundary cost the pipelined step about 1 %).
    evs = [[torch.cuda.Event(enable_timing=True) for _ in range(3)] for _ in range(args.steps)]
    P.ff_profile_start(launches_per_step * args.steps + 64, kinds=[dom])
    log(f"bench: timing {args.steps} step(s)")
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for k in range(args.steps):
        step(evs[k])
    torch.cuda.synchronize()
    t1 = time.perf_counter()
    ds = P.ff_profile_stop()[dom]
    ms_per_step = (t1 - t0) * 1e3 / args.steps
    train_ms = sum(e[0].elapsed_time(e[1]) for e in evs) / args.steps
    score_ms = sum(e[1].elapsed_time(e[2]) for e in evs) / args.steps
    step_rows = 2 * w.n * w.n_layers
    assert torch.isfinite(trace).all().item(), "non-finite loss in the timed steps"

    # whole-step algorithmic flops of the training epoch (both products of every layer step)
    train_flops = sum(4.0 * 2 * b * di * do for (_, b) in w.chunks()
                      for di, do in zip(w.dims[:-1], w.dims[1:]))
    # the algorithmic minimum: layer 0's positive and negative rows share their
    # base row, so an exact rewrite halves layer 0's products (the scoring pass
    # already runs that rewrite; training launches the full products)
    train_min_flops = train_flops - sum(4.0 * b * w.dims[0] * w.dims[1] for (_, b) in w.chunks())
    kernel_ms = sum(v["total_ms"] for v in kstats.values())
    bound, peak, punit = PEAK[dname]
    dom_recs = [r for r in orecs if r["kind"] == dom]
    one = otot[dom]
    achieved_ov = ds["flops"] / (ds["total_ms"] * 1e-3) / 1e12
    traffic = load_traffic(dom, w.name)  # HBM bytes per launch (counter runs)
    kernels = {}
    for k, v in kstats.items():
        if not v["launches"]:
            continue
        t = v["total_ms"] * 1e-3
        kernels[k] = {"launches": v["launches"], "avg_us": v["total_ms"] * 1e3 / v["launches"],
                      "share": v["total_ms"] / sum(x["total_ms"] for x in kstats.values()),
                      "TFLOP/s": v["flops"] / t / 1e12 if v["flops"] else None,
                      "GB/s": v["bytes"] / t / 1e9}
    out = {
        "metric": METRIC,
        "value": step_rows / (ms_per_step * 1e-3),
        "unit": "pos+neg samples/s per layer-step over the train+score step",
        "value_definition": "training rows x layers per step / ms_per_step, where the timed "
                            "step is one training epoch plus scoring the score set; the "
                            "training part alone is train_samples_per_s, the scoring part "
                            "images_per_s",
        "n_gpus": 1, "steps": args.steps, "warmup": args.warmup,
        "ms_per_step": ms_per_step, "higher_is_better": True, "scaling": "weak",
        "vs_baseline": None, "dtype": dname, "data": "synthetic",
        "config": {"workload": w.name, "rows_per_layer_step": 2 * w.chunk_pairs,
                   "layers": list(w.dims), "samples": w.n, "chunks": nc,
                   "schedule": w.schedule, "score_workload": sw.name, "score_images": sw.n,
                   "score_layers": list(sw.dims)},
        "train_ms_per_step": train_ms,
        "train_samples_per_s": step_rows / (train_ms * 1e-3),
        "score_ms_per_step": score_ms,
        "images_per_s": sw.n / (score_ms * 1e-3),
        "roofline": {"bound": bound, "kernel": dom, "achieved": one["TFLOP/s"], "peak": peak,
                     "unit": punit, "frac": one["frac"], "traffic": traffic,
                     "avg_launch_us": one["avg_us"], "launches": one["launches"],
                     "algorithmic_flops_per_launch": sum(r["flops"] for r in dom_recs)
                     / len(dom_recs),
                     "algorithmic_bytes_per_launch": sum(r["bytes"] for r in dom_recs)
                     / len(dom_recs),
                     "shapes": by_shape(dom_recs, dname),
                     "replay_ms_per_step": replay_ms,
                     "method": "one-stream replay of the step (every layer on one HIP stream, "
                               "then the scoring): HIP events around each launch; achieved = "
                               "the kernel's algorithmic flops summed over all its launches in "
                               "the step / their summed durations (`shapes`: per shape)"},
        "roofline_overlapped": {
            "kernel": dom, "achieved": achieved_ov, "peak": peak, "unit": punit,
            "frac": achieved_ov / peak, "avg_launch_us": ds["total_ms"] * 1e3 / ds["launches"],
            "launches": ds["launches"],
            "note": "events around this kernel's launches in the timed steps; per-launch "
                    "durations include time shared with the other layers' streams: kernel time "
                    "summed over launches is `concurrency` times the step's wall time"},
        "replay_kernels": otot,
        "concurrency": kernel_ms / profiled_ms,
        "train_mfma_frac": train_flops / (train_ms * 1e-3) / 1e12 / peak,
        "train_effective_frac": train_min_flops / (train_ms * 1e-3) / 1e12 / peak,
        "kernels": kernels,
    }
    if not args.no_other_workloads:
        out["hbm_kernels_isolated"] = hbm_kernels(P, torch)
        out["softmax_head"] = softmax_head(P, torch, sw, sxd, slayers)
        out["performance_optimised_and_adaptive_neg"] = po_and_adaptive(P, torch, w, xd, yd,
                                                                        layers)
        out["chapter_schedules"] = chapters(P, torch, w, xd, yd, ynd, params)
        others = other_workloads(P, torch, ["mnist_784_2000x4", "mnist_784_2000x4_bf16",
                                            "cifar_3072x4_bf16_pipelined"])
        out["other_workloads"] = others
        seq = others.get("mnist_784_2000x4")
        if seq and w.name == "mnist_784_2000x4_pipelined":
            out["pipelined_vs_sequential"] = {
                "sequential_epoch_ms": seq["epoch_ms"], "pipelined_epoch_ms": train_ms,
                "speedup": seq["epoch_ms"] / train_ms,
                "note": "one GPU: the layer streams share its CUs (the paper's 3.75x is "
                        "four nodes, Table 1)"}
    if not args.no_cpu_baseline:
        log("bench: timing the CPU oracle on a bounded sample")
        out["cpu_baseline"] = cpu_baseline(w, x_base, y, y_neg, params, sw, sx, sparams)
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
