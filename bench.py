"""Throughput of the fused turn-KL forward + backward on one MI355X.

Workload: the long-horizon agent batch, 65,536 packed tokens x vocabulary
151,936 (bf16 logits), 30 trajectories with 20-50 turns of lognormal length,
40% observation-masked, teacher noise decaying with turn depth, alpha = 0.5
(synth/configs.py).  One step = one turnkl_fwd_bwd call: segments, weights,
per-token reverse KL, the student-logit gradient for every row, the loss and
the per-turn statistics.  Inputs are generated in HBM before timing.

Prints one JSON line: tokens/s for the whole step, plus the row kernel's
roofline (algorithmic bytes / measured duration against 8 TB/s) and the CPU
oracle's throughput on a bounded sample of the same batch.
"""
import argparse
import hashlib
import json
import os
import re
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

HBM_PEAK_GBS = 8000.0
ROW_KERNEL_SOURCES = ["paper_2607_05804_amd/csrc/rowkl.hip",
                      "paper_2607_05804_amd/csrc/turnkl_internal.h",
                      "paper_2607_05804_amd/csrc/block_ops.h"]
COUNTER_FILE = os.path.join(ROOT, "profiles", "rowkl_long_horizon_counters.md")


def row_kernel_digest() -> str:
    """Digest of the row kernel's sources with comments and blank space
    removed, so that it changes with the code and not with its comments."""
    h = hashlib.sha256()
    for p in ROW_KERNEL_SOURCES:
        with open(os.path.join(ROOT, p)) as f:
            src = f.read()
        src = re.sub(r"/\*.*?\*/", " ", src, flags=re.S)
        src = re.sub(r"//[^\n]*", " ", src)
        h.update(" ".join(src.split()).encode())
    return h.hexdigest()[:16]


WORKLOAD_NAMES = {"long_horizon": "long-horizon agent batch", "peaked": "peaked-teacher batch",
                  "stress": "stress batch", "agent": "agent batch"}


def committed_traffic():
    """HBM bytes per row-kernel launch from the committed counter summary,
    or None when it is missing or was taken on a different kernel source."""
    if not os.path.exists(COUNTER_FILE):
        return None
    txt = open(COUNTER_FILE).read()
    m = re.search(r"kernel_source_digest:\s*([0-9a-f]+)", txt)
    t = re.search(r"hbm_bytes_per_launch:\s*([0-9.eE+]+)", txt)
    if not m or not t or m.group(1) != row_kernel_digest():
        return None
    return float(t.group(1))


def cpu_model() -> str | None:
    """The host CPU's model name (first processor in /proc/cpuinfo)."""
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return None


def host_rows_of(zs, zt, rows, batch: int = 2048):
    """Host copies (bit patterns) of the listed rows of the device logits, the
    CPU oracle's input: the same bits the host generator would write."""
    import numpy as np
    import torch
    rows = np.asarray(rows, np.int64)
    bits = np.uint16 if zs.dtype == torch.bfloat16 else np.float32
    view = torch.int16 if zs.dtype == torch.bfloat16 else torch.float32
    hs = np.empty((rows.size, zs.shape[1]), dtype=bits)
    ht = np.empty((rows.size, zs.shape[1]), dtype=bits)
    for k0 in range(0, rows.size, batch):
        idx = torch.from_numpy(rows[k0:k0 + batch]).to(zs.device)
        hs[k0:k0 + idx.numel()] = zs.index_select(0, idx).view(view).cpu().numpy().view(bits)
        ht[k0:k0 + idx.numel()] = zt.index_select(0, idx).view(view).cpu().numpy().view(bits)
    return hs, ht


def cpu_baseline(w, sample_tokens: int, host_rows):
    """The float64 oracle, timed on a prefix of the batch (all its rows,
    loss, gradient of every supervised row and per-turn stats).  host_rows:
    the supervised rows of that prefix, copied from the device before the
    clock starts, with row_at[i] their position."""
    import numpy as np
    from oracle import turnkl_oracle as O

    n = min(sample_tokens, w.n_tokens)
    traj, turn, mask = w.traj_id[:n], w.turn_id[:n], w.loss_mask[:n]
    sup = np.nonzero(mask)[0]
    (hs, ht), row_at = host_rows
    src = lambda rows: (hs[row_at[rows]], ht[row_at[rows]])
    t0 = time.perf_counter()
    ref = O.fwd_bwd(traj, turn, mask, w.alphas[0], w.max_turns, src, O.DTYPE_BF16, 1.0,
                    grad_rows=sup)
    dt = time.perf_counter() - t0
    assert ref.status == O.OK
    return {"value": n / dt, "unit": "tokens/s", "cores": O.max_threads(), "kind": "oracle",
            "cpu_model": cpu_model(), "host_cpus": os.cpu_count(),
            "sample": (f"the whole batch" if n == w.n_tokens else f"first {n} tokens of the batch")
                      + f" ({sup.size} supervised rows, full vocabulary {w.vocab}, logits copied "
                        f"to the host before the clock starts), {dt:.1f} s"}


def success_stand_in(w):
    """Turn counts of the even-numbered trajectories, standing in for the
    successful completions of a probe batch (the synthetic batch has none)."""
    import numpy as np
    return [int(np.unique(w.turn_id[w.traj_id == b]).size)
            for b in np.unique(w.traj_id[w.traj_id >= 0]) if b % 2 == 0]


def depth_controller_timing(T, stats, w, reps: int = 2000):
    """Host time of one rollout-depth controller update (turnkl_depth_update,
    Sec. 5.1) on this batch's per-turn statistics, ctypes call included."""
    st = T.read_turn_stats(stats)
    succ = success_stand_in(w)
    ctl = T.DepthController()
    t0 = time.perf_counter()
    for _ in range(reps):
        ctl.update(st, succ)
    lib_us = (time.perf_counter() - t0) / reps * 1e6
    return {"update_us": lib_us, "turns": int(st.shape[0]), "successes": len(succ),
            "h_eff": ctl.state.h_eff, "h_cov": ctl.state.h_cov,
            "cap_after_probe": ctl.plan(4)[0]}


def oracle_controller_timing(stats_np, w, reps: int = 200):
    """The oracle's controller update on the same statistics (CPU baseline)."""
    from oracle import depth_controller as D
    succ = success_stand_in(w)
    cfg = D.Config()
    st = D.init(cfg)
    k, n = list(stats_np["kl_mean"]), list(stats_np["n_traj"])
    t0 = time.perf_counter()
    for _ in range(reps):
        st = D.update(cfg, st, k, n, succ)
    return (time.perf_counter() - t0) / reps * 1e6


def topk_timing(T, zs, zt, turn, traj, mask, w, steps: int, warmup: int, k: int = 50):
    """The top-K variant (App. D's top-K reverse KL, teacher support K = 50)
    on the same batch: teacher support from the device teacher logits, dense
    bf16 gradient out of place.  Its traffic is the dense gradient write plus
    the support reads, so it is bound by HBM writes."""
    import numpy as np
    import torch
    top_v, top_i = torch.topk(zt, k, dim=1)
    ids = top_i.to(torch.int32).contiguous()
    vals = top_v.float().contiguous()
    del top_v, top_i
    n, V = zs.shape
    grad = torch.empty_like(zs)
    stats = T.new_turn_stats(w.max_turns)
    ws = T.TopkWorkspace(n, k, w.max_turns)

    def step():
        return T.fwd_bwd_topk(zs, ids, vals, turn, traj, mask, w.alphas[0], grad=grad,
                              max_turns=w.max_turns, turn_stats=stats, workspace=ws, check=False)

    for _ in range(warmup):
        step()
    torch.cuda.synchronize()
    ev = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))
          for _ in range(steps)]
    for a, b in ev:
        a.record()
        b.record()
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for a, b in ev:
        T.profile_row_kernel(a, b)
        step()
    T.profile_row_kernel(None, None)
    torch.cuda.synchronize()
    elapsed = time.perf_counter() - t0
    if ws.status() != T.OK:
        raise RuntimeError(T.status_string(ws.status()))
    kern_ms = float(np.mean([a.elapsed_time(b) for a, b in ev]))
    n_sup = int(w.n_supervised)
    by = n * V * 2 + n_sup * k * (4 + 4 + 2)
    out = {"k": k, "tokens_per_s": n * steps / elapsed, "ms_per_step": elapsed * 1e3 / steps,
           "kernels_ms": kern_ms, "algorithmic_bytes_per_call": by,
           "roofline": {"bound": "hbm", "achieved": by / (kern_ms * 1e-3) / 1e9,
                        "peak": HBM_PEAK_GBS, "unit": "GB/s",
                        "frac": by / (kern_ms * 1e-3) / 1e9 / HBM_PEAK_GBS},
           "gradient": "dense bf16, out of place (zero off the support)"}
    host = (ids.cpu().numpy(), vals.cpu().numpy())
    idx = ids.long()
    zs_at = torch.gather(zs, 1, idx).view(torch.int16).cpu().numpy().view(np.uint16)
    del grad, idx, ws
    torch.cuda.empty_cache()
    return out, host + (zs_at,)


def all_supervised_timing(T, zs, zt, turn, traj, w, grad, steps: int, warmup: int):
    """The same logits with every token supervised (loss mask all ones): every
    row reads both logit rows and writes its gradient, 3 V s bytes per token,
    the row kernel's clean roofline case."""
    import numpy as np
    import torch
    dev = zs.device
    n, V = zs.shape
    mask = (traj >= 0).to(torch.uint8)  # every token but padding
    n_sup = int(mask.sum().item())
    stats = T.new_turn_stats(w.max_turns, device=dev)
    ws = T.Workspace(n, V, T.BF16, w.max_turns, device=dev)

    def step():
        return T.fwd_bwd(zs, zt, turn, traj, mask, w.alphas[0], grad=grad, max_turns=w.max_turns,
                         turn_stats=stats, workspace=ws, check=False)

    for _ in range(warmup):
        step()
    torch.cuda.synchronize()
    ev = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))
          for _ in range(steps)]
    for a, b in ev:
        a.record()
        b.record()
    torch.cuda.synchronize()
    for a, b in ev:
        T.profile_row_kernel(a, b)
        step()
    T.profile_row_kernel(None, None)
    torch.cuda.synchronize()
    if ws.status() != T.OK:
        raise RuntimeError(T.status_string(ws.status()))
    ms = np.array([a.elapsed_time(b) for a, b in ev])
    by = n_sup * 3 * V * 2 + (n - n_sup) * V * 2
    del ws
    return {"tokens": n, "supervised_tokens": n_sup, "algorithmic_bytes_per_launch": by,
            "kernel_ms_mean": float(ms.mean()), "kernel_ms_median": float(np.median(ms)),
            "achieved_gbs": by / (ms.mean() * 1e-3) / 1e9,
            "frac": by / (ms.mean() * 1e-3) / 1e9 / HBM_PEAK_GBS,
            "note": "same logits with every non-padding token supervised (3 V s bytes per token)"}


def options_timing(T, zs, zt, turn, traj, mask, w, grad, steps: int, warmup: int):
    """The fused call with App. D's turn-support floor (8, 0.15) and the
    per-outcome statistics (success flags: the even-numbered trajectories
    stand in for the successful ones), timed against the plain call in the
    same process, alternating.  Both variants add only work outside the row
    kernel (one segment kernel, 2 * max_turns statistics workgroups), so the
    comparison is of everything around the row kernel."""
    import numpy as np
    import torch
    dev = zs.device
    succ = torch.from_numpy((w.traj_id % 2 == 0).astype(np.uint8)).to(dev)
    stats = T.new_turn_stats(w.max_turns, device=dev)
    ostats = T.new_turn_stats(2 * w.max_turns, device=dev)
    ws = T.Workspace(zs.shape[0], zs.shape[1], T.BF16, w.max_turns, device=dev)

    def step(opt):
        kw = dict(support_floor=8, support_frac=0.15, success=succ, outcome_stats=ostats) \
            if opt else {}
        return T.fwd_bwd(zs, zt, turn, traj, mask, w.alphas[0], grad=grad, max_turns=w.max_turns,
                         turn_stats=stats, workspace=ws, check=False, **kw)

    for _ in range(warmup):
        step(False)
        step(True)
    torch.cuda.synchronize()
    mk = lambda: torch.cuda.Event(enable_timing=True)
    rec = {opt: [tuple(mk() for _ in range(4)) for _ in range(steps)] for opt in (False, True)}
    for evs in rec.values():  # materialise the events before they are handed to the library
        for e in evs:
            for x in e:
                x.record()
    torch.cuda.synchronize()
    for k in range(steps):
        for opt in (False, True):
            a, ra, rb, b = rec[opt][k]
            a.record()
            T.profile_row_kernel(ra, rb)
            step(opt)
            T.profile_row_kernel(None, None)
            b.record()
    torch.cuda.synchronize()
    if ws.status() != T.OK:
        raise RuntimeError(T.status_string(ws.status()))

    def summary(evs):
        call = [a.elapsed_time(b) for a, _, _, b in evs]
        row = [ra.elapsed_time(rb) for _, ra, rb, _ in evs]
        return float(np.median(call)), float(np.median(call) - np.median(row))

    plain_ms, plain_other = summary(rec[False])
    opt_ms, opt_other = summary(rec[True])
    st = T.read_turn_stats(stats)
    n_b = int(np.unique(w.traj_id[(w.traj_id >= 0) & (w.loss_mask > 0)]).size)
    n_min = max(8, int(np.ceil(0.15 * n_b)))
    budget = T.budget_report(st, n_b, 8, 0.15)
    gap = T.outcome_gap(ostats)
    del ws
    return {"support_floor": 8, "support_frac": 0.15, "n_min": n_min,
            "valid_turns": int(np.sum(st["n_traj"] >= n_min)),
            "supervised_turns": int(np.sum(st["n_traj"] > 0)),
            "budget": {k: budget[k] for k in ("prefix", "third", "shallow_budget", "deep_budget",
                                              "deep_support", "deep_shallow_kl")},
            "outcome_gap_turns_0_to_4": [None if np.isnan(x) else float(x) for x in gap[:5]],
            "call_ms_median": opt_ms, "plain_call_ms_median": plain_ms,
            "outside_row_kernel_ms": opt_other, "plain_outside_row_kernel_ms": plain_other,
            "note": "floor and outcome split on vs off, alternating in one process; the "
                    "difference is the cost of the two options"}


def graph_timing(T, step, ws, steps: int):
    """The same call captured once in a HIP graph and replayed: the per-step
    time without per-launch host overhead (the library's calls enqueue only
    kernels and never synchronise, so they can be captured)."""
    import torch
    s = torch.cuda.Stream()
    s.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(s):
        step()
        g = torch.cuda.CUDAGraph()
        with torch.cuda.graph(g, stream=s):
            step()
        g.replay()
        s.synchronize()
        t0 = time.perf_counter()
        for _ in range(steps):
            g.replay()
        s.synchronize()
        el = time.perf_counter() - t0
    torch.cuda.current_stream().wait_stream(s)
    if ws.status() != T.OK:
        raise RuntimeError(T.status_string(ws.status()))
    del g
    return {"ms_per_step": el * 1e3 / steps,
            "note": "the timed call captured in a HIP graph and replayed; value uses the eager call"}


def oracle_topk_timing(w, host):
    """The top-K oracle on the whole batch (CPU baseline of the top-K path)."""
    from oracle import topk_oracle as K
    from oracle import turnkl_oracle as O
    ids, vals, zs_at = host
    t0 = time.perf_counter()
    ref = K.fwd_bwd_topk(w.traj_id, w.turn_id, w.loss_mask, w.alphas[0], w.max_turns,
                         lambda r, i: zs_at[r], ids, vals, O.DTYPE_BF16)
    dt = time.perf_counter() - t0
    assert ref.status == O.OK
    return w.n_tokens / dt


def copy_probe(gib: float, steps: int) -> int:
    """torch's device-to-device copy of a buffer of known size."""
    import torch
    n = int(gib * (1 << 30))
    src = torch.empty(n, dtype=torch.uint8, device="cuda")
    src.fill_(1)
    dst = torch.empty_like(src)
    dst.copy_(src)
    torch.cuda.synchronize()
    a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    a.record()
    for _ in range(steps):
        dst.copy_(src)
    b.record()
    torch.cuda.synchronize()
    ms = a.elapsed_time(b) / steps
    print(json.dumps({"copy_bytes": n, "read_plus_write_bytes": 2 * n, "ms": ms,
                      "gbs": 2 * n / (ms * 1e-3) / 1e9}), flush=True)
    return 0


def sustain(T, step, ws, n_tokens: int, seconds: float) -> int:
    """The timed call back to back for `seconds` (synchronising every 50
    calls), with one progress line per second: the steady load under which
    clocks and power are read."""
    import torch
    t0 = time.perf_counter()
    last = t0
    calls = 0
    while time.perf_counter() - t0 < seconds:
        for _ in range(50):
            step()
        torch.cuda.synchronize()
        calls += 50
        now = time.perf_counter()
        if now - last >= 1.0:
            print(f"sustain: {calls} calls, {now - t0:.1f} s, {(now - t0) * 1e3 / calls:.3f} ms per call",
                  flush=True)
            last = now
    el = time.perf_counter() - t0
    if ws.status() != T.OK:
        raise RuntimeError(T.status_string(ws.status()))
    print(json.dumps({"sustained_s": el, "calls": calls, "ms_per_call": el * 1e3 / calls,
                      "tokens_per_s": n_tokens * calls / el, "start_unix": time.time() - el,
                      "end_unix": time.time()}), flush=True)
    return 0


def main() -> int:
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--cpu-sample-tokens", type=int, default=65536,
                    help="tokens of the batch (a prefix) the CPU oracle is timed on")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--copy-probe", type=float, default=0.0, metavar="GIB",
                    help="instead of the step, time a plain device copy of this many GiB "
                         "(bandwidth context and counter calibration)")
    ap.add_argument("--workload", default="long_horizon", choices=sorted(WORKLOAD_NAMES),
                    help="the batch to time (the default is the headline batch; the others "
                         "are the parity batches: peaked 16,534 tokens, stress 131,072 tokens "
                         "with the gradient in place, agent 4,480 tokens at V = 32,000)")
    ap.add_argument("--out-of-place", action="store_true",
                    help="write the stress batch's gradient to a separate buffer instead of "
                         "over the student logits")
    ap.add_argument("--sustain", type=float, default=0.0, metavar="SECONDS",
                    help="instead of the measurements, run the timed call back to back for "
                         "this long and report its rate (for clock and power readings under "
                         "a steady load)")
    args = ap.parse_args()
    if args.gpus != 1:
        print(f"bench.py runs on one GPU only (asked for --gpus {args.gpus}); the multi-GPU "
              "layout is data-parallel by trajectory and is not built here.", file=sys.stderr)
        return 2

    import numpy as np
    import torch

    if args.copy_probe > 0:
        return copy_probe(args.copy_probe, args.steps)

    import synth
    from paper_2607_05804_amd import turnkl as T

    T.lib()  # fails loudly when the HIP library is missing
    dev = torch.device("cuda:0")
    w = synth.make(args.workload)
    alpha = w.alphas[0]
    n, V = w.n_tokens, w.vocab
    n_sup = w.n_supervised
    zs, zt = w.device_logits(device=dev)
    turn = torch.from_numpy(w.turn_id).to(dev)
    traj = torch.from_numpy(w.traj_id).to(dev)
    mask = torch.from_numpy(w.loss_mask).to(dev)
    # The stress batch writes its gradient over the student logits.  Every
    # timed call then needs the original logits back: a device-to-device copy
    # from a pristine copy, made before the call's events are recorded.
    in_place = w.in_place and not args.out_of_place
    pristine = zs.clone() if in_place else None
    # the CPU oracle's input: the supervised rows of its sample, copied now
    # (an in-place call overwrites the student logits)
    cpu_rows = None
    if not args.no_cpu_baseline:
        sup_rows = np.nonzero(w.loss_mask[:min(args.cpu_sample_tokens, n)])[0]
        row_at = np.full(n, -1, np.int64)
        row_at[sup_rows] = np.arange(sup_rows.size)
        cpu_rows = (host_rows_of(zs, zt, sup_rows), row_at)
    grad = zs if in_place else torch.empty_like(zs)
    stats = T.new_turn_stats(w.max_turns, device=dev)
    kl = torch.empty(n, dtype=torch.float32, device=dev)
    ws = T.Workspace(n, V, T.BF16, w.max_turns, device=dev)

    def step():
        return T.fwd_bwd(zs, zt, turn, traj, mask, alpha, grad=grad, max_turns=w.max_turns,
                         turn_stats=stats, token_kl=kl, workspace=ws, check=False)

    def restore():
        if in_place:
            zs.copy_(pristine)

    for _ in range(args.warmup):
        restore()
        step()
    torch.cuda.synchronize()
    if ws.status() != T.OK:
        raise RuntimeError(T.status_string(ws.status()))
    if args.sustain > 0:
        if in_place:
            raise SystemExit("--sustain times the out-of-place call (add --out-of-place)")
        return sustain(T, step, ws, n, args.sustain)

    mk = lambda: torch.cuda.Event(enable_timing=True)
    ev = [(mk(), mk()) for _ in range(args.steps)]     # around the row kernel
    # around the whole call, in place only: there the wall clock also holds
    # the restoring copies, so the step time comes from these events; out of
    # place the wall clock is the step time and no event sits between calls
    call = [(mk(), mk()) for _ in range(args.steps)] if in_place else []
    for e in ev + call:  # materialise the events before the timed region
        e[0].record()
        e[1].record()
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for k, (a, b) in enumerate(ev):
        restore()
        if in_place:
            call[k][0].record()
        T.profile_row_kernel(a, b)
        step()
        if in_place:
            call[k][1].record()
    T.profile_row_kernel(None, None)
    torch.cuda.synchronize()
    elapsed = time.perf_counter() - t0
    if ws.status() != T.OK:
        raise RuntimeError(T.status_string(ws.status()))

    row_all = np.array([a.elapsed_time(b) for a, b in ev])
    call_all = np.array([a.elapsed_time(b) for a, b in call])
    row_ms = float(row_all.mean())
    ms_per_step = float(call_all.mean()) if in_place else elapsed * 1e3 / args.steps
    es = 2
    row_bytes = n_sup * 3 * V * es + (n - n_sup) * V * es
    achieved = row_bytes / (row_ms * 1e-3) / 1e9
    # the committed counters are those of the headline batch
    traffic = committed_traffic() if args.workload == "long_horizon" else None
    out = {
        "metric": "fused turn-KL fwd+bwd tokens/sec and achieved HBM GB/s (% of peak), V=151936",
        "value": n / (ms_per_step * 1e-3),
        "unit": "tokens/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": ms_per_step,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "f32",
        "data": "synthetic",
        "config": {
            "workload": f"{WORKLOAD_NAMES[args.workload]}: {n} tokens x V={V} bf16 logits, "
                        f"{int(w.traj_id.max()) + 1} trajectories, "
                        f"{round(100 * (1 - n_sup / n))}% of tokens masked, alpha={alpha}",
            "n_tokens": n, "vocab": V, "supervised_tokens": n_sup, "logits": "bf16",
            "gradient": ("bf16, in place over the student logits (restored from a pristine "
                         "device copy before each call, outside the call's events)"
                         if in_place else "bf16, out of place"),
            "parallelism": "single GPU", "workspace_bytes": ws.nbytes,
        },
        "roofline": {
            "bound": "hbm",
            "achieved": achieved,
            "peak": HBM_PEAK_GBS,
            "unit": "GB/s",
            "frac": achieved / HBM_PEAK_GBS,
            "traffic": traffic,
            "kernel": "rowkl_kernel",
            "kernel_ms": row_ms,
            "kernel_ms_median": float(np.median(row_all)),
            "kernel_ms_p10": float(np.percentile(row_all, 10)),
            "kernel_ms_p90": float(np.percentile(row_all, 90)),
            "algorithmic_bytes_per_launch": row_bytes,
        },
        "step_hbm_gbs": row_bytes / (ms_per_step * 1e-3) / 1e9,
        "supervised_tokens_per_s": n_sup / (ms_per_step * 1e-3),
        "call_ms_median": float(np.median(call_all)) if in_place else None,
        "wall_ms_per_step": elapsed * 1e3 / args.steps,
    }
    stats_np = T.read_turn_stats(stats)
    topk_host = None
    if not in_place:
        # further measurements on the same batch (the in-place batch's student
        # logits now hold its gradient; those measurements exist out of place)
        out["graph_replay"] = graph_timing(T, step, ws, args.steps)
        out["depth_controller"] = depth_controller_timing(T, stats, w)
        out["floor_and_outcome"] = options_timing(T, zs, zt, turn, traj, mask, w, grad,
                                                  args.steps, args.warmup)
        out["all_supervised"] = all_supervised_timing(T, zs, zt, turn, traj, w, grad, args.steps,
                                                      args.warmup)
        del grad
        torch.cuda.empty_cache()
        out["topk"], topk_host = topk_timing(T, zs, zt, turn, traj, mask, w, args.steps,
                                             args.warmup)
    del zs, zt
    torch.cuda.empty_cache()
    if not args.no_cpu_baseline:
        out["cpu_baseline"] = cpu_baseline(w, args.cpu_sample_tokens, cpu_rows)
        del cpu_rows
        out["cpu_baseline"]["depth_controller_update_us"] = oracle_controller_timing(stats_np, w)
        if topk_host is not None:
            out["cpu_baseline"]["topk_tokens_per_s"] = oracle_topk_timing(w, topk_host)
    print(json.dumps(out), flush=True)
    return 0


if __name__ == "__main__":
    sys.exit(main())
