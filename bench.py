"""Benchmark of the xHC sublayer connection on one MI355X.

    python bench.py [--gpus 1] [--steps K] [--warmup W] [--no-cpu-baseline]

One step = the forward connection of one xHC block at the large-MoE width
(T = 16384 tokens in 2 sequences of 8192, N = 16 streams, k = 4 active, m = 2
fixed, C = 4096, bf16 state): an attention-type sublayer (xhc_pre + xhc_post,
one write-back component) followed by an MLP-type sublayer (xhc_pre +
xhc_post with the 4/8/12 causal convolutions and Gram-Schmidt).  The
sublayer output F is a given tensor (the attention / MLP themselves are
outside the connection).  `value` is sublayer-tokens per second, 2T / step
time, i.e. tokens/s per xHC sublayer averaged over the block as the paper
averages its traffic.

Prints ONE JSON line.  Inputs are synthetic (seeded) and resident in HBM
before the timed region.  The roofline object is for the dominant kernel;
its achieved bandwidth is the algorithmic bytes per launch divided by the
launch's average duration, both measured here with HIP events on the stream
the kernel runs on.  cpu_baseline times the CPU fp64 oracle on a bounded
sample of the same workload.
"""

from __future__ import annotations

import argparse
import json
import os
import sys
import time

import torch

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

from paper_2607_14530_amd import accounting as A  # noqa: E402
from paper_2607_14530_amd import synth  # noqa: E402
from paper_2607_14530_amd import xhc as X  # noqa: E402

HBM_PEAK_GBPS = 8000.0
METRIC = "tokens/s and achieved HBM GB/s per xHC sublayer (fwd) at N=16,k=4,C=4096"
TRAFFIC_SUMMARY = os.path.join(ROOT, "profiles", "traffic_xhc_pre_T16384_N16_C4096.md")


# the sources whose device code one xhc_pre call runs (k_zero2, k_pre_fused,
# k_pre_coef_sum and the helpers they inline)
PRE_SOURCES = ("xhc_device.h", "xhc_pre.hip", "xhc_pre_fused.hip")


def sources_digest():
    """sha256 over the pre kernels' sources (name + bytes, sorted): a traffic
    figure measured on other sources no longer describes the kernels."""
    import hashlib
    h = hashlib.sha256()
    csrc = os.path.join(ROOT, "paper_2607_14530_amd", "csrc")
    for name in sorted(PRE_SOURCES):
        with open(os.path.join(csrc, name), "rb") as f:
            h.update(name.encode())
            h.update(f.read())
    return h.hexdigest()


def measured_traffic():
    """HBM bytes per xhc_pre call from the committed rocprofv3 counter summary,
    or None when it is missing or was taken on different kernel sources."""
    try:
        with open(TRAFFIC_SUMMARY) as f:
            kv = dict(line.split(":", 1) for line in f if line.startswith(("traffic_bytes_per_call:",
                                                                             "sources_sha256:")))
    except OSError:
        return None
    if kv.get("sources_sha256", "").strip() != sources_digest():
        return None
    return float(kv["traffic_bytes_per_call"])


def calibrate_copy(gib=1):
    """A plain device copy of known size, for scaling the HBM byte counters."""
    n = gib << 29   # bf16 elements
    src = torch.randn(n, device="cuda", dtype=torch.bfloat16)
    dst = torch.empty_like(src)
    for _ in range(3):
        dst.copy_(src)
    torch.cuda.synchronize()
    print(json.dumps({"copy_bytes_read": 2 * n, "copy_bytes_written": 2 * n, "launches": 3}), flush=True)


def host_cpu():
    """CPU model and physical core count of this host (lscpu; /proc/cpuinfo)."""
    import subprocess
    model, sockets, per_socket = None, None, None
    try:
        out = subprocess.run(["lscpu"], capture_output=True, text=True, timeout=10).stdout
        for line in out.splitlines():
            key, _, val = line.partition(":")
            key, val = key.strip(), val.strip()
            if key == "Model name":
                model = val
            elif key == "Socket(s)":
                sockets = int(val)
            elif key == "Core(s) per socket":
                per_socket = int(val)
    except (OSError, ValueError, subprocess.SubprocessError):
        pass
    physical = sockets * per_socket if sockets and per_socket else None
    return model, physical


def _oracle_tokens_per_s(n, seconds, label):
    """Oracle pre + post of both sublayer kinds on n tokens, n grown until the
    run takes about `seconds`; returns (sublayer-tokens/s, n, elapsed)."""
    from oracle import xhc_oracle as O
    F64 = torch.float64
    while True:
        elapsed = 0.0
        for Kr in (1, 4):
            w = synth.sparse_c4096(Kr)
            ws = synth.Workload(T=n, S=n, N=w.N, k=w.k, m=w.m, C=w.C, Kr=Kr)
            inp = synth.sublayer_inputs(ws, 7)
            Xd = inp["X"].to(F64)
            t0 = time.perf_counter()
            r = O.xhc_pre(Xd, inp["W_r"], inp["W_pre"], inp["W_res"], inp["W_post"],
                          tuple(inp["alpha"].tolist()), inp["b_pre"], inp["b_res"], inp["b_post"],
                          m=ws.m, k=ws.k, Kr=Kr)
            O.xhc_post(Xd, inp["F"], inp["conv_w"], r["idx"], r["p"], r["Hres"], r["Hpost"],
                       S=ws.S, kappa=ws.kappa)
            elapsed += time.perf_counter() - t0
        print(f"[cpu_baseline] {label}: {n} tokens: {elapsed:.2f} s", file=sys.stderr, flush=True)
        if elapsed >= seconds or n >= 16384:
            return 2 * n / elapsed, n, elapsed
        n = min(16384, max(n * 2, int(n * seconds / max(elapsed, 1e-3) * 1.1)))


def cpu_baseline(seconds=12.0, seconds_single=8.0):
    """Time the fp64 oracle (pre + post of both sublayer kinds) on a sample of
    tokens of the same workload, on all of torch's threads and on one thread."""
    threads = torch.get_num_threads()
    value, n, elapsed = _oracle_tokens_per_s(16, seconds, f"{threads} threads")
    torch.set_num_threads(1)
    try:
        single, n1, e1 = _oracle_tokens_per_s(4, seconds_single, "1 thread")
    finally:
        torch.set_num_threads(threads)
    model, physical = host_cpu()
    return {"value": value, "unit": "tokens/s", "cores": threads, "kind": "oracle",
            "sample": f"{n} tokens x (attention-type + MLP-type sublayer), N=16 k=4 m=2 C=4096, fp64, "
                      f"{elapsed:.1f} s on {threads} threads; single thread: {n1} tokens, {e1:.1f} s",
            "single_thread_value": single, "cpu_model": model, "physical_cores": physical,
            "logical_cpus": os.cpu_count()}


def pctl(xs, q):
    """q-th percentile (0..100) of xs, linear interpolation."""
    v = sorted(xs)
    if not v:
        return None
    pos = (len(v) - 1) * q / 100.0
    lo = int(pos)
    hi = min(lo + 1, len(v) - 1)
    return v[lo] + (v[hi] - v[lo]) * (pos - lo)


def _time(fn, iters, stream):
    """Average milliseconds of fn() over iters calls, HIP events on `stream`."""
    fn()
    torch.cuda.synchronize()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record(stream)
    for _ in range(iters):
        fn()
    e1.record(stream)
    torch.cuda.synchronize()
    return e0.elapsed_time(e1) / iters


SECTIONS = ("flash_q4", "flash_q2", "mhc_n4", "config2_c1024", "prefill_t2048", "bwd_mlp_sweep", "bwd_mlp_n16",
            "flash_bwd_q4")


def extra_sections(dev, stream, iters=5, only=None):
    """xHC-Flash groups, the dense mHC N=4 comparator and the backward, each
    timed on its own (outside the timed steps of the main workload); only:
    names of the sections to run (all when None)."""
    out = {}
    unit = lambda C: 2 * C   # bytes of one "C" (bf16 elements of width C)
    want = lambda name: only is None or name in only
    # xHC-Flash, Q = 4 and Q = 2, at T = 16384 (2 x 8192), N = 16, k = 4, C = 4096
    for Q in (4, 2):
        if not want(f"flash_q{Q}"):
            continue
        w = synth.sparse_c4096(4)
        d = synth.flash_inputs(w, Q, 40 + Q, device=dev)
        g = X.FlashGroup(X.dims_for(w), Q, d, dev)
        state = d["X"]
        ms = _time(lambda: g.run(state, d["F_list"], stream), iters, stream)
        Kq = [1 if q % 2 == 1 else w.Kr for q in range(1, Q + 1)]
        b = A.algorithmic_bytes_flash_pre(w.N, w.k, w.C, Q)
        for q in range(1, Q + 1):
            b += A.algorithmic_bytes_flash_post(w.N, w.k, w.C, Kq[q - 1], q == Q, Kq[q] if q < Q else 0)
        out[f"flash_q{Q}"] = {
            "workload": f"xHC-Flash group of {Q} sublayers, T=16384 (2 x 8192), N=16, k=4, m=2, C=4096",
            "ms_per_group": ms, "tokens_per_s_per_sublayer": Q * w.T / (ms * 1e-3),
            "achieved_GBps": b * w.T / (ms * 1e-3) / 1e9,
            "bytes_per_token_C": b / Q / unit(w.C), "paper_bytes_per_token_C": 40.0 if Q == 4 else 51.0}
        del g, d, state
        torch.cuda.empty_cache()
    if want("mhc_n4"):
        # dense mHC N = 4 (k = m = N, one write-back component) at the same T and C
        w = synth.Workload(T=16384, S=8192, N=4, k=4, m=4, C=4096, Kr=1, name="mhc-n4")
        inp = synth.sublayer_inputs(w, 9, device=dev)
        sub = X.Sublayer(X.dims_for(w), inp, dev)
        st = inp["X"]
        ms = _time(lambda: (sub.pre(st, stream), sub.post(st, inp["F"], stream)), iters, stream)
        b = A.algorithmic_bytes_sublayer(4, 4, w.C, 1)
        out["mhc_n4"] = {"workload": "dense mHC N=4 (k=m=4, one write-back component), T=16384, C=4096",
                         "ms_per_sublayer": ms, "tokens_per_s": w.T / (ms * 1e-3),
                         "achieved_GBps": b * w.T / (ms * 1e-3) / 1e9, "bytes_per_token_C": b / unit(w.C),
                         "paper_bytes_per_token_C": 34.0}
        del sub, inp, st
        torch.cuda.empty_cache()
    if want("config2_c1024"):
        # xHC sparse at C = 1024: T = 4096 (one sequence), N = 16, k = 4, an
        # attention-type and an MLP-type sublayer (forward), single-pass pre
        # with teams of 8 workgroups
        wa, wm = synth.sparse_c1024(1), synth.sparse_c1024(4)
        ia, im = synth.sublayer_inputs(wa, 21, device=dev), synth.sublayer_inputs(wm, 22, device=dev)
        sa = X.Sublayer(X.dims_for(wa), ia, dev)
        sm = X.Sublayer(X.dims_for(wm), im, dev)
        st = ia["X"]
        ms = _time(lambda: (sa.pre(st, stream), sa.post(st, ia["F"], stream),
                            sm.pre(st, stream), sm.post(st, im["F"], stream)), 20, stream)
        pre_ms = _time(lambda: sa.pre(st, stream), 20, stream)
        b = A.algorithmic_bytes_sublayer(wa.N, wa.k, wa.C, 1) + A.algorithmic_bytes_sublayer(wm.N, wm.k, wm.C, 4)
        out["config2_c1024"] = {"workload": "xHC forward block (attention-type + MLP-type sublayer), T=4096, N=16, "
                                            "k=4, m=2, C=1024",
                                "ms_per_block": ms, "tokens_per_s": 2 * wa.T / (ms * 1e-3),
                                "achieved_GBps": b * wa.T / (ms * 1e-3) / 1e9,
                                "bytes_per_token_C": b / 2 / unit(wa.C), "ms_xhc_pre": pre_ms}
        del sa, sm, ia, im, st
        torch.cuda.empty_cache()
    if want("prefill_t2048"):
        # prefill-latency regime: one 2048-token sequence through an attention-type
        # and an MLP-type sublayer (forward), for each pre implementation
        pre_ms = {}
        for name, impl in (("auto", X.XHC_IMPL_AUTO), ("multi", X.XHC_IMPL_MULTI), ("fused", X.XHC_IMPL_FUSED)):
            wa = synth.Workload(T=2048, S=2048, N=16, k=4, m=2, C=4096, Kr=1, name="prefill-attn")
            wm = synth.Workload(T=2048, S=2048, N=16, k=4, m=2, C=4096, Kr=4, name="prefill-mlp")
            ia, im = synth.sublayer_inputs(wa, 11, device=dev), synth.sublayer_inputs(wm, 12, device=dev)
            sa = X.Sublayer(X.dims_for(wa, impl=impl), ia, dev)
            sm = X.Sublayer(X.dims_for(wm, impl=impl), im, dev)
            st = ia["X"]
            pre_ms[name] = _time(lambda: (sa.pre(st, stream), sa.post(st, ia["F"], stream),
                                          sm.pre(st, stream), sm.post(st, im["F"], stream)), 20, stream)
            del sa, sm, ia, im, st
            torch.cuda.empty_cache()
        out["prefill_t2048"] = {"workload": "xHC forward block (attention-type + MLP-type sublayer), one 2048-token "
                                            "sequence, N=16, k=4, m=2, C=4096",
                                "ms_per_block": pre_ms["auto"], "ms_per_block_multi": pre_ms["multi"],
                                "ms_per_block_fused": pre_ms["fused"],
                                "tokens_per_s": 2048 / (pre_ms["auto"] * 1e-3)}
    for sec_name, Ns in (("bwd_mlp_sweep", (4, 8, 16, 32)), ("bwd_mlp_n16", (16,))):
        if not want(sec_name) or (sec_name == "bwd_mlp_n16" and only is None):
            continue   # (the N = 16 case alone, for profiling; part of the sweep otherwise)
        # backward of an MLP-type sublayer, T = 8192, k = 4, C = 4096, N = 4, 8, 16, 32
        res = {}
        for N in Ns:
            w = synth.bwd_sweep(N, 4)
            inp = synth.sublayer_inputs(w, 10, device=dev, grads=True)
            sub = X.TrainableSublayer(X.dims_for(w), inp, dev)
            st = inp["X"]
            fwd_ms = _time(lambda: sub.forward(st, inp["F"], stream), 2, stream)
            sub.forward(st, inp["F"], stream)

            def fb():   # dL/dX is formed in place in the upstream gradient's buffer
                sub.backward(st, inp["G_X"], inp["G_in"], inp["F"], stream, in_place=True)
                sub.forward(st, inp["F"], stream)
            ms = _time(fb, 3, stream)
            res[f"N{N}"] = {"ms_forward_with_saves": fwd_ms, "ms_backward": ms - fwd_ms,
                            "tokens_per_s_backward": w.T / ((ms - fwd_ms) * 1e-3)}
            del sub, inp, st
            torch.cuda.empty_cache()
        out[sec_name] = {"workload": "xHC MLP-type sublayer backward, T=8192, k=4, m=2, C=4096, "
                                     f"N in {{{', '.join(str(n) for n in Ns)}}}", **res}
    if want("flash_bwd_q4"):
        # xHC-Flash group backward, Q = 4, T = 8192, N = 16, k = 4, C = 4096
        w = synth.bwd_sweep(16, 4)
        Q = 4
        fd = synth.flash_inputs(w, Q, 13, device=dev, grads=True)
        grp = X.TrainableFlashGroup(X.dims_for(w), Q, fd, dev)
        X0 = fd["X"]
        st = X0.clone()
        ffwd = _time(lambda: (st.copy_(X0), grp.forward(st, fd["F_list"], stream)), 2, stream)
        cp = _time(lambda: st.copy_(X0), 2, stream)
        G_in = torch.stack(fd["G_in_list"])   # [Q, T, C], as the backward takes it
        # dL/dX is formed in place in the upstream gradient's buffer
        fbwd = _time(lambda: grp.backward(X0, fd["G_X"], G_in, fd["F_list"], stream, in_place=True), 2, stream)
        out["flash_bwd_q4"] = {"workload": "xHC-Flash group backward, Q=4, T=8192, N=16, k=4, m=2, C=4096",
                               "ms_forward_with_saves": ffwd - cp, "ms_backward": fbwd,
                               "tokens_per_s_per_sublayer_backward": Q * w.T / (fbwd * 1e-3)}
    return out


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-extra", action="store_true",
                    help="skip the Flash / mHC / prefill / backward sections")
    ap.add_argument("--section", action="append", default=None, choices=SECTIONS,
                    help="run only this extra section (repeatable) and print its figures")
    ap.add_argument("--calibrate-copy", action="store_true",
                    help="only run a 1 GiB device copy (counter calibration under rocprofv3 --pmc)")
    args = ap.parse_args()
    if args.calibrate_copy:
        calibrate_copy()
        return
    if args.gpus != 1:
        print(f"bench.py measures one GPU: this build runs the connection on a single MI355X "
              f"(--gpus {args.gpus} requested)", file=sys.stderr)
        sys.exit(2)

    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    if args.section:
        stream = torch.cuda.current_stream()
        print(json.dumps({"sections": extra_sections(dev, stream, only=set(args.section))}), flush=True)
        return
    w_attn, w_mlp = synth.sparse_c4096(1), synth.sparse_c4096(4)
    T, N, k, C = w_attn.T, w_attn.N, w_attn.k, w_attn.C
    inp_a = synth.sublayer_inputs(w_attn, 1, device=dev)
    inp_m = synth.sublayer_inputs(w_mlp, 2, device=dev)
    sub_a = X.Sublayer(X.dims_for(w_attn), inp_a, dev)
    sub_m = X.Sublayer(X.dims_for(w_mlp), inp_m, dev)
    state = inp_a["X"]                       # [T, N, C] bf16, updated in place
    F_a, F_m = inp_a["F"], inp_m["F"]
    stream = torch.cuda.current_stream()

    def step(ev=None):
        if ev is not None:
            ev[0].record(stream)
        sub_a.pre(state, stream)
        if ev is not None:
            ev[1].record(stream)
        sub_a.post(state, F_a, stream)
        if ev is not None:
            ev[2].record(stream)
        sub_m.pre(state, stream)
        if ev is not None:
            ev[3].record(stream)
        sub_m.post(state, F_m, stream)
        if ev is not None:
            ev[4].record(stream)

    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()

    evs = [[torch.cuda.Event(enable_timing=True) for _ in range(5)] for _ in range(args.steps)]
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for i in range(args.steps):
        step(evs[i])
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0

    seg = [[e[j].elapsed_time(e[j + 1]) for e in evs] for j in range(4)]   # ms
    mean = [sum(s) / len(s) for s in seg]
    step_ms = sum(mean)
    per_step = [sum(seg[j][i] for j in range(4)) for i in range(args.steps)]
    value = 2 * T / (step_ms * 1e-3)

    b_pre = A.algorithmic_bytes_pre(N, k, C, 1) * T
    b_post_a = A.algorithmic_bytes_post(N, k, C, 1) * T
    b_pre_m = A.algorithmic_bytes_pre(N, k, C, 4) * T
    b_post_m = A.algorithmic_bytes_post(N, k, C, 4) * T
    total_bytes = b_pre + b_post_a + b_pre_m + b_post_m
    gbps = total_bytes / (step_ms * 1e-3) / 1e9
    pre_ms = (mean[0] + mean[2]) / 2
    pre_bytes = (b_pre + b_pre_m) / 2
    achieved = pre_bytes / (pre_ms * 1e-3) / 1e9

    out = {
        "metric": METRIC, "value": value, "unit": "tokens/s", "n_gpus": 1, "steps": args.steps,
        "warmup": args.warmup, "ms_per_step": step_ms, "higher_is_better": True, "scaling": "weak",
        "vs_baseline": None, "dtype": "bf16", "data": "synthetic",
        "config": {"workload": "xHC forward block (attention-type + MLP-type sublayer), T=16384 (2 x 8192), "
                               "N=16, k=4, m=2, C=4096, kappa=4/8/12, bf16 state, fp32 coefficients",
                   "T": T, "S": w_attn.S, "N": N, "k": k, "m": w_attn.m, "C": C},
        "achieved_GBps": gbps, "hbm_frac": gbps / HBM_PEAK_GBPS,
        "bytes_per_token_C": total_bytes / (2 * T) / (2 * C),
        "paper_bytes_per_token_C": 73.5,
        "ms_per_step_p10_p50_p90": [pctl(per_step, 10), pctl(per_step, 50), pctl(per_step, 90)],
        "segments_ms": {"attn_pre": mean[0], "attn_post": mean[1], "mlp_pre": mean[2], "mlp_post": mean[3]},
        "segments_ms_p10_p50_p90": {n: [pctl(seg[j], 10), pctl(seg[j], 50), pctl(seg[j], 90)]
                                    for j, n in enumerate(("attn_pre", "attn_post", "mlp_pre", "mlp_post"))},
        "wall_s": wall,
        "roofline": {"kernel": "xhc_pre entry point (single-pass cooperative kernel k_pre_fused: projection, "
                               "routing, dense read, gathered projection; then the per-token coefficient pass), "
                               "mean of the two sublayer kinds",
                     "bound": "hbm", "achieved": achieved, "peak": HBM_PEAK_GBPS, "unit": "GB/s",
                     "frac": achieved / HBM_PEAK_GBPS, "traffic": measured_traffic(),
                     "algorithmic_bytes_per_call": pre_bytes},
    }
    if not args.no_extra:
        del sub_a, sub_m, inp_a, inp_m, state
        torch.cuda.empty_cache()
        out["sections"] = extra_sections(dev, stream)
    if not args.no_cpu_baseline:
        out["cpu_baseline"] = cpu_baseline()
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
