#!/usr/bin/env python3
"""FPO hot-path throughput on one MI355X.

One step = one pass of the whole hot path over one batch of T tokens:
fpo_output_error (final-norm recompute, vocabulary-chunked logits + online
softmax + error, projection through W_U, clamped RMSNorm VJP) followed by
fpo_pseudograd with the fused update (per-layer outer products for every
target layer staged in bf16 as the paper's bf16 einsum produces them,
relative 1% clip, SGD-momentum on fp32 masters, bf16 copy). The default
workload is the Qwen3-8B-shaped training batch (config 2); config 4 is the
layer-viability diagnostic (every layer's pseudogradient reduced against a
reference gradient in the GEMM epilogue); --full-mlp also updates W1 and W2.
Inputs are seeded synthetic tensors of the workload's shapes, resident in HBM
before timing starts. Prints one JSON line on stdout; progress goes to stderr.

  python bench.py [--gpus 1] [--steps K] [--warmup W] [--config 2] [--full-mlp]
"""
from __future__ import annotations

import argparse
import ctypes as C
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

METRIC = "FPO update tokens/sec at 8B shapes; % bf16 MFMA peak; HBM GB/s on VJP/update"
PEAK_BF16_TFLOPS = 2500.0   # MI355X dense bf16 MFMA
PEAK_F32_TFLOPS = 157.3     # MI355X fp32 matrix
PEAK_HBM_GBS = 8000.0       # MI355X HBM3E
# optimizer HBM bytes per parameter at step > 1: dW read 4, master r/w 8, bf16 copy
# write 2, plus state r/w (momentum 8; AdamW moments 16; plain SGD none)
OPT_BYTES = {"sgd-momentum": 22.0, "sgd": 14.0, "adamw": 30.0}
OPT_NAME = {"sgd-momentum": "SGD-momentum", "sgd": "plain SGD (no state)", "adamw": "AdamW"}


def log(*a):
    print(*a, file=sys.stderr, flush=True)


def parse():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--config", type=int, default=2,
                    help="workload id (paper_2608_14563_amd.inputs.CONFIGS): 1-3 training steps, 4 the diagnostic")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--vocab-chunk", type=int, default=0,
                    help="vocabulary chunk width (0: the library's planner)")
    ap.add_argument("--cpu-tokens", type=int, default=0,
                    help="tokens in the oracle's timed sample (0: about 10 TFLOP of float64 work, at most the "
                         "whole batch)")
    ap.add_argument("--full-mlp", action="store_true",
                    help="update W1 and W2 too, through the fixed feedback W3_init (eq. errh)")
    ap.add_argument("--post-ffn", action="store_true",
                    help="compose each target layer's post-FFN RMSNorm VJP (OLMo-2 / Gemma 3 layout)")
    ap.add_argument("--grad-f32", action="store_true",
                    help="hand the fused update an fp32 pseudogradient instead of the bf16-staged one "
                         "(FPO_MODE_GRAD_BF16, the precision of the paper's bf16 einsum)")
    ap.add_argument("--clip-target", choices=["gradient", "update"], default="gradient",
                    help="what the 1%% clip bounds: the gradient before the step (App. A pseudocode) or the "
                         "step applied to W (two passes, no overlap with the outer products)")
    ap.add_argument("--optimizer", choices=sorted(OPT_BYTES), default="sgd-momentum",
                    help="optimizer on the fp32 masters (HBM bytes per parameter: " +
                         ", ".join(f"{k} {v}" for k, v in sorted(OPT_BYTES.items())) + ")")
    ap.add_argument("--e2e-diagnostic", default=None, metavar="MODEL",
                    help="instead of the training step, time the end-to-end layer-viability diagnostic on a "
                         "random-init transformer (paper_2608_14563_amd.inputs.MODELS, e.g. qwen3-8b)")
    ap.add_argument("--calibrate-copy", type=int, default=0, metavar="MIB",
                    help="only run a plain device-to-device copy of MIB MiB (HBM counter calibration)")
    return ap.parse_args()


def calibrate_copy(mib: int) -> None:
    """A plain copy of known size: the HBM read/write counters of this
    dispatch calibrate the FETCH_SIZE / WRITE_SIZE readings of the kernels."""
    import torch
    n = mib * (1 << 20)
    src = torch.ones(n, dtype=torch.uint8, device="cuda:0")
    dst = torch.empty_like(src)
    torch.cuda.synchronize()
    dst.copy_(src)
    torch.cuda.synchronize()
    print(json.dumps({"calibrate_copy_bytes": n}), flush=True)


def prof_lib():
    from paper_2608_14563_amd import _lib
    lib = _lib.load()
    lib.fpo_prof_enable.argtypes = [C.c_char_p]
    lib.fpo_prof_read.argtypes = [C.c_int, C.c_char_p, C.POINTER(C.c_double), C.POINTER(C.c_int64)]
    return lib


def prof_read(lib):
    n = 64
    names = C.create_string_buffer(32 * n)
    ms = (C.c_double * n)()
    cnt = (C.c_int64 * n)()
    k = lib.fpo_prof_read(n, names, ms, cnt)
    if k < 0:
        raise RuntimeError("fpo_prof_read failed")
    return {names.raw[32 * i:32 * i + 32].split(b"\0")[0].decode(): (ms[i], cnt[i]) for i in range(k)}


def max_engine_clock_mhz():
    """The GPU's highest engine-clock level (MHz) from the amdgpu driver's
    sysfs table (pp_dpm_sclk), or None when it is not readable. Read from
    files only: no child process is started from this (GPU-using) process."""
    import glob
    import re
    best = None
    for f in sorted(glob.glob("/sys/class/drm/card*/device/pp_dpm_sclk")):
        try:
            txt = open(f).read()
        except OSError:
            continue
        for m in re.finditer(r"(\d+)\s*[Mm][Hh]z", txt):
            v = int(m.group(1))
            best = v if best is None else max(best, v)
    return best


def source_hash() -> str:
    """Hash of the library sources with comments and blank lines removed; a
    profile's traffic figure applies only while the code it was measured on
    is unchanged (comment edits do not invalidate it)."""
    import hashlib
    import re
    h = hashlib.sha256()
    d = os.path.join(ROOT, "paper_2608_14563_amd", "csrc")
    for f in sorted(os.listdir(d)):
        if f.endswith((".hip", ".hpp")):
            txt = open(os.path.join(d, f), encoding="utf-8").read()
            txt = re.sub(r"/\*.*?\*/", "", txt, flags=re.S)
            txt = re.sub(r"//[^\n]*", "", txt)
            code = "\n".join(ln.rstrip() for ln in txt.splitlines() if ln.strip())
            h.update(f.encode())
            h.update(code.encode())
    return h.hexdigest()[:16]


def profiled_traffic(workload: str, kernel: str):
    """HBM bytes per dispatch of `kernel` from the committed rocprofv3 counter
    summary (profiles/*.md, FETCH_SIZE and WRITE_SIZE scaled by the plain-copy
    calibration), or None when absent or taken on different kernel sources."""
    pdir = os.path.join(ROOT, "profiles")
    if not os.path.isdir(pdir):
        return None
    want = source_hash()
    for f in sorted(os.listdir(pdir)):
        if not f.endswith(".md"):
            continue
        for line in open(os.path.join(pdir, f)):
            p = line.split()
            if len(p) == 5 and p[0] == "traffic" and p[1] == workload and p[2] == kernel and p[3] == want:
                return float(p[4])
    return None


def kernel_work(name, c, steps, nchunk, opt="sgd-momentum", pffn=False, grad_bf16=False, clip_update=False,
                full=False):
    """Algorithmic work of one kernel over `steps` steps: (amount, unit, bound).
    Flops count only the method's contractions; bytes count each operand once."""
    T, d, V, dff, L = c.T, c.d, c.V, c.d_ff, c.L
    if name in ("logits_chunk", "proj_chunk"):
        return 2.0 * T * V * d * steps, "flop", "mfma"
    if name == "outer":  # W3 (and, full-MLP, W1 and W2) outer products of every layer
        return 2.0 * T * d * dff * L * (3 if full else 1) * steps, "flop", "mfma"
    if name == "errh":  # E = g~ W3_init per layer
        return 2.0 * T * d * dff * L * steps, "flop", "mfma"
    nm = 3 * L if full else L
    gb = 2.0 if grad_bf16 else 4.0  # a staged bf16 pseudogradient reads 2 bytes instead of 4
    if name == "update" and clip_update:  # pass 2: W r/w, bf16 copy, the new state (or dW) read
        per = {"sgd-momentum": 14.0, "sgd": 10.0 + gb, "adamw": 18.0}[opt]
        return per * nm * d * dff * steps, "byte", "hbm"
    if name == "update_delta":  # pass 1: dW (and state, W for AdamW) read, new state written
        per = {"sgd-momentum": gb + 8.0, "sgd": gb, "adamw": gb + 20.0}[opt]
        return per * nm * d * dff * steps, "byte", "hbm"
    if name == "update":
        return (OPT_BYTES[opt] - (4.0 - gb)) * nm * d * dff * steps, "byte", "hbm"
    if name == "chunk_stats":
        # per-(token, 128-entry block) max / sum / argmax read; per-token state read and written
        return (12.0 * T * ((V + 127) // 128) + 36.0 * T) * steps, "byte", "hbm"
    if name == "rms_forward":
        return (6.0 * T * d) * steps, "byte", "hbm"  # x read, y written, the target's W_U row read (bf16)
    if name == "pffn_stats":  # per layer: g~ fp32 and MLP output read
        return (6.0 * T * d * L) * steps, "byte", "hbm"
    if name == "signal_transpose":
        # shared signal: read + token-contiguous copy written (bf16); post-FFN, per layer:
        # g~ fp32 and MLP output read, composed signal written
        return ((8.0 * T * d * L) if pffn else (4.0 * T * d)) * steps, "byte", "hbm"
    if name == "finalize_vjp":
        return (T * d * (4 + 2 + 2 + 4 + 2)) * steps, "byte", "hbm"
    return None


def _cpu_info():
    blas = None
    try:
        from threadpoolctl import threadpool_info
        info = threadpool_info()
        thr = max([i.get("num_threads", 1) for i in info] or [1])
        blas = ", ".join(sorted({f"{i.get('internal_api')} ({i.get('num_threads')} threads)" for i in info}))
    except Exception:  # pragma: no cover
        thr = len(os.sched_getaffinity(0))
    cpu_model = None
    try:
        for line in open("/proc/cpuinfo"):
            if line.startswith("model name"):
                cpu_model = line.split(":", 1)[1].strip()
                break
    except OSError:  # pragma: no cover
        pass
    return thr, blas, cpu_model


def auto_cpu_tokens(c, per_token_flop, budget=1.0e13):
    """Token sample for the oracle: about 10 TFLOP of float64 work (10-20 s
    on 16 host cores), at most the whole batch."""
    return max(1, min(c.T, int(budget // per_token_flop)))


def cpu_baseline(c, tokens, x, gam, W_U, y, acts, Wm, full=None):
    """The oracle, timed on the host cores: the first `tokens` tokens through
    the output error and every layer's outer product (full-MLP: also the W1/W2
    signals through W3_init), then every matrix's clipped SGD-momentum step.
    With fewer than T tokens the full step is estimated as per-token time x T
    + the measured updates."""
    import numpy as np

    import oracle as O
    thr, blas, cpu_model = _cpu_info()
    per_tok = 8.0 * c.V * c.d + 2.0 * c.d * c.d_ff * c.L * (4 if full else 1)
    ts = auto_cpu_tokens(c, per_tok) if tokens <= 0 else min(tokens, c.T)
    t0 = time.perf_counter()
    out = O.output_error(x[:ts], gam, W_U, y[:ts], eps=c.eps, min_rms=c.min_rms, vocab_chunk=8192)
    Ds = [O.pseudograd(out["g_tilde"], a[:ts], scale=1.0 / c.T) for a in acts]
    if full:
        D1s, D2s = [], []
        for l in range(c.L):
            D1, D2 = O.full_mlp_grads(out["g_tilde"], full["W3i"][l], full["q"][l][:ts], full["u"][l][:ts],
                                      full["x_in"][l][:ts], scale=1.0 / c.T)
            D1s.append(D1)
            D2s.append(D2)
        Ds = Ds + D1s + D2s
    t1 = time.perf_counter()
    for D, W in zip(Ds, Wm):
        s = O.clip_scale(float((D * D).sum()), float((W.astype(np.float64) ** 2).sum()), c.clip_frac)
        O.sgd_momentum(W, np.zeros_like(D), s * D, c.lr, 0.9, step=2)
    t2 = time.perf_counter()
    est = (t1 - t0) / ts * c.T + (t2 - t1)
    what = f"all {c.L} layers' {'W1, W2 and W3 pseudogradients' if full else 'outer products'}"
    nm = len(Ds)
    if ts == c.T:
        sample = (f"the whole step: {c.T} tokens through output error (full V={c.V}) and {what} "
                  f"({t1 - t0:.1f} s), then all {nm} clipped SGD-momentum steps ({t2 - t1:.1f} s)")
    else:
        sample = (f"first {ts} of {c.T} tokens through output error (full V={c.V}) and {what} ({t1 - t0:.1f} s), "
                  f"then all {nm} clipped SGD-momentum steps ({t2 - t1:.1f} s); full step estimated as "
                  f"per-token time x T + updates = {est:.1f} s")
    return {"value": c.T / est, "unit": "tokens/s", "cores": int(thr), "kind": "oracle", "sample": sample,
            "seconds": round(t2 - t0, 2), "affinity_cpus": len(os.sched_getaffinity(0)),
            "cpu_model": cpu_model, "blas": blas}


def cpu_baseline_diag(c, tokens, x, gam, W_U, y, tacts, refs):
    """The oracle on a sample of the diagnostic workload: the first `tokens`
    tokens through the output error and all layers' outer products (scaled to
    T per token), and every layer's cosine against its full-size reference
    (whose cost does not depend on T)."""
    import numpy as np

    import oracle as O
    thr, blas, cpu_model = _cpu_info()
    ts = min(tokens, c.T)
    acts = [a[:ts].view(__import__("torch").int16).cpu().numpy().view(np.uint16) for a in tacts]
    t0 = time.perf_counter()
    out = O.output_error(x[:ts], gam, W_U, y[:ts], eps=c.eps, min_rms=c.min_rms, vocab_chunk=8192)
    Ds = [O.pseudograd(out["g_tilde"], a, scale=1.0 / c.T) for a in acts]
    t1 = time.perf_counter()
    tc = 0.0
    for D, R in zip(Ds, refs):
        Rh = R.cpu().numpy()
        tr = time.perf_counter()
        O.cosine(D, Rh)
        tc += time.perf_counter() - tr
    est = (t1 - t0) / ts * c.T + tc
    return {"value": c.T / est, "unit": "tokens/s", "cores": int(thr), "kind": "oracle",
            "sample": (f"first {ts} of {c.T} tokens through output error (full V={c.V}) and all {c.L} layers' outer "
                       f"products ({t1 - t0:.1f} s), then all {c.L} cosines against the full-size references "
                       f"({tc:.1f} s); full job estimated as per-token time x T + cosines = {est:.1f} s"),
            "seconds": round(t1 - t0 + tc, 2), "affinity_cpus": len(os.sched_getaffinity(0)),
            "cpu_model": cpu_model, "blas": blas}


def cpu_baseline_e2e(m, model, ids, tokens=512):
    """The oracle's end-to-end diagnostic (float64 model, autograd, FPO
    oracle) timed on the host cores on a bounded sample: the first `tokens`
    tokens of one sequence through the full-vocabulary head and one, then two,
    of the model's blocks (its last ones, weights copied from the device).
    The difference prices one block; the full job is estimated as
    (head + L blocks) x T / tokens (per-token cost; attention's length-dependent
    share is about 2% of a block at 512 tokens)."""
    import numpy as np
    import torch

    from oracle import transformer as OT
    h = lambda t: t.detach().float().cpu().numpy()  # noqa: E731
    head = {k: h(v) for k, v in model.head.items()}
    L = m.n_layers
    lay = [{k: h(v) for k, v in model.layers[l].items()} for l in (L - 2, L - 1)]
    sid = ids[:1, :tokens + 1].cpu().numpy()
    OT.diagnostic(m.shrink(n_layers=1, batch=1, seq=8), head, lay[1:], sid[:, :9])  # warm-up, untimed
    times = []
    for k in (1, 2):
        mk = m.shrink(n_layers=k, batch=1, seq=tokens)
        t0 = time.perf_counter()
        OT.diagnostic(mk, head, lay[2 - k:], sid)
        times.append(time.perf_counter() - t0)
    per_block = max(times[1] - times[0], 0.0)
    head_s = max(times[0] - per_block, 0.0)
    est = (head_s + L * per_block) * m.T / tokens
    return {"value": m.T / est, "unit": "tokens/s", "cores": torch.get_num_threads(), "kind": "oracle",
            "sample": (f"first {tokens} tokens of one sequence through the head (V={m.V}) and 1, then 2, of the "
                       f"{L} blocks: {times[0]:.1f} s and {times[1]:.1f} s, so head {head_s:.1f} s + "
                       f"{per_block:.1f} s per block; full job estimated as (head + {L} blocks) x {m.T}/{tokens} "
                       f"= {est:.0f} s"),
            "seconds": round(sum(times), 2)}


def bench_e2e(args):
    """End-to-end layer-viability diagnostic (Sec. 2.2): one step = the
    model's float32 forward with cache, its autograd gradient, and the FPO
    side in libfpo (output error, every layer's W3 pseudogradient reduced
    against the true gradient, output cosines) over one calibration batch."""
    import numpy as np
    import torch

    from paper_2608_14563_amd import diagnostic as D
    from paper_2608_14563_amd import inputs as I
    if not torch.cuda.is_available():
        print("bench.py needs a GPU", file=sys.stderr)
        sys.exit(1)
    torch.backends.cuda.matmul.allow_tf32 = False
    dev = torch.device("cuda:0")
    m = I.MODELS[args.e2e_diagnostic]
    op = torch.bfloat16
    log(f"[bench] e2e diagnostic {m.name}: V={m.V} d={m.d} d_ff={m.d_ff} layers={m.n_layers} heads={m.n_heads}/"
        f"{m.n_kv_heads} T={m.batch}x{m.seq}={m.T} layout={m.layout}")
    model = D.Transformer.seeded_on_device(m, dev)
    ids = torch.from_numpy(I.model_tokens(m).astype(np.int64)).to(dev)
    lib = prof_lib()

    def once(ev=None):
        if ev:
            ev[0].record()
        c = D.forward_with_cache(model, ids, op)
        if ev:
            ev[1].record()
        tg = D.true_gradients(c)
        if ev:
            ev[2].record()
        out = D.fpo_launch(model, c, tg, op)
        if ev:
            ev[3].record()
        return out

    for _ in range(args.warmup):
        D.fpo_finish(once())
    torch.cuda.synchronize()
    lib.fpo_prof_reset()
    lib.fpo_prof_enable(b"")
    res = D.fpo_finish(once())
    torch.cuda.synchronize()
    lib.fpo_prof_disable()
    per_kernel = prof_read(lib)
    lib.fpo_prof_reset()
    dom = max(per_kernel, key=lambda k: per_kernel[k][0])
    log("[bench] libfpo ms per diagnostic: " + ", ".join(f"{k}={v[0]:.3f}/{v[1]}" for k, v in sorted(per_kernel.items(), key=lambda kv: -kv[1][0])))
    lib.fpo_prof_enable(dom.encode())
    evs = [[torch.cuda.Event(enable_timing=True) for _ in range(4)] for _ in range(args.steps)]
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    e0.record()
    for k in range(args.steps):
        out = once(evs[k])
        del out
    e1.record()
    torch.cuda.synchronize()
    lib.fpo_prof_disable()
    dom_stats = prof_read(lib)[dom]
    lib.fpo_prof_reset()
    ms_step = e0.elapsed_time(e1) / args.steps
    med = lambda v: sorted(v)[len(v) // 2]  # noqa: E731
    fwd = med([e[0].elapsed_time(e[1]) for e in evs])
    bwd = med([e[1].elapsed_time(e[2]) for e in evs])
    fpo = med([e[2].elapsed_time(e[3]) for e in evs])
    c = I.Config(-1, m.name, "bf16", m.d, m.d_ff, m.V, m.T, m.n_layers, zipf=True, outliers=False, diag=True)
    roof = None
    w = kernel_work(dom, c, args.steps, None)
    if w is not None:
        amount, unit, bound = w
        secs = dom_stats[0] / 1000.0
        ach = amount / secs / (1e12 if unit == "flop" else 1e9)
        peak = PEAK_BF16_TFLOPS if unit == "flop" else PEAK_HBM_GBS
        roof = {"bound": bound, "achieved": round(ach, 2), "peak": peak, "unit": "TFLOP/s" if unit == "flop" else "GB/s",
                "frac": round(ach / peak, 4), "traffic": profiled_traffic(m.name + "-e2e", dom), "kernel": dom,
                "avg_launch_ms": round(dom_stats[0] / dom_stats[1], 4), "launches": dom_stats[1]}
    flops_fpo = 4.0 * m.T * m.V * m.d + 2.0 * m.T * m.d * m.d_ff * m.n_layers
    tok_s = m.T / (ms_step / 1e3)
    log(f"[bench] {args.steps} diagnostics: {ms_step:.1f} ms each ({tok_s:.0f} tokens/s); forward {fwd:.1f} ms, "
        f"autograd {bwd:.1f} ms, libfpo {fpo:.2f} ms; W3 cos last quarter {D.summary(res['cos_w3']):.3f}")
    out = {
        "metric": "end-to-end layer-viability diagnostic tokens/sec (forward with cache + autograd true gradient + "
                  "FPO pseudogradient cosines, every layer)",
        "value": round(tok_s, 1), "unit": "tokens/s", "n_gpus": 1, "steps": args.steps, "warmup": args.warmup,
        "ms_per_step": round(ms_step, 3), "higher_is_better": True, "scaling": "weak", "vs_baseline": None,
        "dtype": "f32 model / bf16 FPO operands", "data": "synthetic (random-init weights, Zipf tokens)",
        "config": {"workload": f"{m.name}-shaped random-init transformer, diagnostic over {m.batch} sequences x "
                               f"{m.seq} tokens, all {m.n_layers} layers scored", "V": m.V, "d": m.d, "d_ff": m.d_ff,
                   "layers": m.n_layers, "heads": m.n_heads, "kv_heads": m.n_kv_heads, "T": m.T, "layout": m.layout},
        "substeps": {"forward_ms_median": round(fwd, 2), "autograd_ms_median": round(bwd, 2),
                     "libfpo_ms_median": round(fpo, 3),
                     "libfpo_mfma_frac": round(flops_fpo / (fpo / 1e3) / 1e12 / PEAK_BF16_TFLOPS, 4)},
        "roofline": roof,
        "kernels": {k: {"ms": round(v[0], 4), "launches": v[1]} for k, v in per_kernel.items()},
        "cos_w3": [round(float(x), 4) for x in res["cos_w3"]],
        "cos_out": [round(float(x), 4) for x in res["cos_out"]],
    }
    if not args.no_cpu_baseline:
        log("[bench] timing the CPU oracle on a sample")
        out["cpu_baseline"] = cpu_baseline_e2e(m, model, ids)
    else:
        out["cpu_baseline"] = None
    print(json.dumps(out), flush=True)


def _to_dev(dev):
    import numpy as np
    import torch

    def t(a):
        a = np.ascontiguousarray(a)
        if a.dtype == np.uint16:
            return torch.from_numpy(a.view(np.int16)).view(torch.bfloat16).to(dev)
        return torch.from_numpy(a).to(dev)
    return t


def roofline_entry(dom, dom_stats, work, traffic):
    """The line's roofline object for kernel `dom`: its algorithmic work over
    the timed region divided by its summed event time."""
    if work is None:
        return None
    amount, unit, bound = work
    secs = dom_stats[0] / 1000.0
    flop = unit == "flop"
    ach = amount / secs / (1e12 if flop else 1e9)
    peak = PEAK_BF16_TFLOPS if flop else PEAK_HBM_GBS
    return {"bound": bound, "achieved": round(ach, 2 if flop else 1), "peak": peak,
            "unit": "TFLOP/s" if flop else "GB/s", "frac": round(ach / peak, 4), "traffic": traffic,
            "kernel": dom, "avg_launch_ms": round(dom_stats[0] / dom_stats[1], 4), "launches": dom_stats[1]}


KERNEL_TIMING_NOTE = ("per-kernel figures from hipEvent pairs around every launch of one untimed step, on the "
                      "stream each kernel runs on; microsecond-scale kernels include the launch gap, so their "
                      "rates are lower bounds (the rocprofv3 durations are in profiles/)")


def bench_diag(args, clk_mhz):
    """Diagnostic workload hot path (eq. cosine; Sec. 2.2-2.3): one step is
    fpo_output_error over the 16 x 512 calibration tokens and fpo_pseudograd
    reducing every one of the 36 layers' outer products against a supplied
    reference gradient R = D + sigma N (sigma so that E[cos] = 1/2) in the
    GEMM epilogue: dot products, norms and cosines, no dW stored. The
    activations and the noise are drawn on the device (seeded Philox); D for
    the reference comes from one untimed fpo_pseudograd call."""
    import numpy as np
    import torch

    from paper_2608_14563_amd import api
    from paper_2608_14563_amd import inputs as I
    dev = torch.device("cuda:0")
    c = I.CONFIGS[4]
    T, d, L = c.T, c.d, c.L
    log(f"[bench] diagnostic workload {c.name}: T={T} d={d} d_ff={c.d_ff} V={c.V}, all {L} layers; generating inputs")
    t = _to_dev(dev)
    x, gam, W_U, y = I.hidden(c), I.gain(c), I.unembedding(c), I.targets(c)
    tx, tgam, tW, ty = t(x), t(gam), t(W_U), t(y)
    tacts = [I.device_activation(c, l, dev) for l in range(L)]
    g_t = torch.empty(T, d, dtype=torch.float32, device=dev)
    g_lp = torch.empty(T, d, dtype=torch.bfloat16, device=dev)
    loss = torch.empty(T, dtype=torch.float32, device=dev)
    ws_oe = api.workspace(api.fpo_output_error_workspace(T, d, c.V, torch.bfloat16), dev)
    ws_pg = api.workspace(api.fpo_pseudograd_workspace(T, d, c.d_ff, L, torch.bfloat16), dev)
    ss = torch.empty(L, dtype=torch.float64, device=dev)
    dot = torch.empty(L, dtype=torch.float64, device=dev)
    rsq = torch.empty(L, dtype=torch.float64, device=dev)
    cos = torch.empty(L, dtype=torch.float32, device=dev)
    # reference gradients: the pseudogradient plus noise (expected cosine 1/2)
    api.fpo_output_error(tx, tgam, tW, ty, g_t, g_tilde_lp=g_lp, ws=ws_oe, eps=c.eps, min_rms=c.min_rms)
    refs = [torch.empty(d, c.d_ff, dtype=torch.float32, device=dev) for _ in range(L)]
    api.fpo_pseudograd(g_lp, tacts, dW3=refs, sumsq=ss, ws=ws_pg)
    torch.cuda.synchronize()
    for l in range(L):
        sigma = float(np.sqrt(3.0) * np.sqrt(float(ss[l])) / np.sqrt(d * c.d_ff))
        refs[l].add_(I.device_noise(c, l, (d, c.d_ff), dev), alpha=sigma)
    torch.cuda.synchronize()
    log("[bench] inputs ready on the device")

    def step(mid=None):
        api.fpo_output_error(tx, tgam, tW, ty, g_t, g_tilde_lp=g_lp, loss=loss, ws=ws_oe, eps=c.eps,
                             min_rms=c.min_rms)
        if mid is not None:
            mid.record()
        api.fpo_pseudograd(g_lp, tacts, dW3=None, sumsq=ss, ref=refs, ref_dot=dot, ref_sumsq=rsq, ref_cos=cos,
                           ws=ws_pg)

    res = timed_run(args, step, lambda k: k not in ("update",), c, clk_mhz, T,
                    flops_oe=4.0 * T * c.V * d, flops_pg=2.0 * T * d * c.d_ff * L,
                    work=lambda k, n: kernel_work(k, c, n, None))
    cos_h = cos.cpu().numpy().astype(np.float64)
    k = int(round(L / 4))
    res.update({
        "metric": "FPO layer-viability diagnostic tokens/sec at 8B shapes (output error + every layer's "
                  "pseudogradient reduced against a reference gradient); % bf16 MFMA peak",
        "config": {"workload": f"{c.name}-shaped diagnostic hot path: T={T} tokens (16 x 512), d={d}, "
                               f"d_ff={c.d_ff}, V={c.V}, all {L} layers scored against R = D + sigma N "
                               f"(E[cos] = 1/2), bf16 operands / fp32 accumulate, cosines from float64 sums",
                   "T": T, "d": d, "d_ff": c.d_ff, "V": c.V, "L": L},
        "cos_per_layer": [round(float(v), 4) for v in cos_h],
        "cos_summary_last_quarter": round(float(np.mean(cos_h[-k:])), 4),
    })
    if not args.no_cpu_baseline:
        log("[bench] timing the CPU oracle on a sample")
        res["cpu_baseline"] = cpu_baseline_diag(c, args.cpu_tokens or 96, x, gam, W_U, y, tacts, refs)
    else:
        res["cpu_baseline"] = None
    print(json.dumps(res), flush=True)


def timed_run(args, step, on_step_stream, c, clk_mhz, T, flops_oe, flops_pg, work, traffic_name=None):
    """Warm-up steps, one untimed fully instrumented step (per-kernel times;
    the dominant kernel on the step's own stream), then args.steps timed steps
    with the dominant kernel bracketed by events on its launch stream. Returns
    the bench line's common fields."""
    lib = prof_lib()
    for _ in range(args.warmup):
        step()
    import torch
    torch.cuda.synchronize()
    lib.fpo_prof_reset()
    lib.fpo_prof_enable(b"")
    step()
    torch.cuda.synchronize()
    lib.fpo_prof_disable()
    per_kernel = prof_read(lib)
    lib.fpo_prof_reset()
    dom = max((k for k in per_kernel if on_step_stream(k)), key=lambda k: per_kernel[k][0])
    log("[bench] per-kernel ms in one step: " + ", ".join(f"{k}={v[0]:.3f}/{v[1]}" for k, v in sorted(per_kernel.items(), key=lambda kv: -kv[1][0])))
    lib.fpo_prof_enable(dom.encode())
    torch.cuda.synchronize()
    e0 = torch.cuda.Event(enable_timing=True)
    e1 = torch.cuda.Event(enable_timing=True)
    # per-step events: [start, output error done, pseudograd (+ update) done]
    marks = [[torch.cuda.Event(enable_timing=True) for _ in range(3)] for _ in range(args.steps)]
    e0.record()
    for k in range(args.steps):
        marks[k][0].record()
        step(marks[k][1])
        marks[k][2].record()
    e1.record()
    torch.cuda.synchronize()
    lib.fpo_prof_disable()
    ms_total = e0.elapsed_time(e1)
    per_step = sorted(m[0].elapsed_time(m[2]) for m in marks)
    per_oe = sorted(m[0].elapsed_time(m[1]) for m in marks)
    per_pg = sorted(m[1].elapsed_time(m[2]) for m in marks)
    dom_stats = prof_read(lib)[dom]
    lib.fpo_prof_reset()
    ms_step = ms_total / args.steps
    tok_s = T / (ms_step / 1000.0)
    log(f"[bench] {args.steps} steps: {ms_step:.3f} ms/step, {tok_s:.0f} tokens/s; dominant kernel {dom}: "
        f"{dom_stats[0] / dom_stats[1]:.3f} ms avg over {dom_stats[1]} launches")
    roof = roofline_entry(dom, dom_stats, work(dom, args.steps), profiled_traffic(traffic_name or c.name, dom))
    kernels = {}
    for k, (ms, n) in per_kernel.items():
        wk = work(k, 1)
        e = {"ms_per_step": round(ms, 4), "launches": n}
        if wk is not None:
            amount, unit, bound = wk
            if unit == "flop":
                e["tflops"] = round(amount / (ms / 1e3) / 1e12, 1)
                e["mfma_frac"] = round(amount / (ms / 1e3) / 1e12 / PEAK_BF16_TFLOPS, 4)
            else:
                e["gbs"] = round(amount / (ms / 1e3) / 1e9, 1)
                e["hbm_frac"] = round(amount / (ms / 1e3) / 1e9 / PEAK_HBM_GBS, 4)
        kernels[k] = e
    med = lambda v: v[len(v) // 2]  # noqa: E731
    props = torch.cuda.get_device_properties(0)
    peak_clk = (props.multi_processor_count * clk_mhz * 1e6 * 4096 / 1e12) if clk_mhz else None
    substeps = {
        "step_ms_median": round(med(per_step), 4), "step_ms_min": round(per_step[0], 4),
        "output_error_ms_median": round(med(per_oe), 4),
        "pseudograd_update_ms_median": round(med(per_pg), 4),
        "output_error_mfma_frac": round(flops_oe / (med(per_oe) / 1e3) / 1e12 / PEAK_BF16_TFLOPS, 4),
        "pseudograd_update_mfma_frac": round(flops_pg / (med(per_pg) / 1e3) / 1e12 / PEAK_BF16_TFLOPS, 4),
        "mfma_peak_tflops_nominal": PEAK_BF16_TFLOPS,
        "mfma_peak_tflops_at_max_clock": round(peak_clk, 1) if peak_clk else None,
        "max_engine_clock_mhz": clk_mhz,
    }
    log(f"[bench] median step {substeps['step_ms_median']:.3f} ms (min {substeps['step_ms_min']:.3f}): output error "
        f"{substeps['output_error_ms_median']:.3f} ms, pseudograd {substeps['pseudograd_update_ms_median']:.3f} ms")
    return {
        "metric": METRIC, "value": round(tok_s, 1), "unit": "tokens/s", "n_gpus": 1, "steps": args.steps,
        "warmup": args.warmup, "ms_per_step": round(ms_step, 4), "higher_is_better": True, "scaling": "weak",
        "vs_baseline": None, "dtype": "bf16", "data": "synthetic",
        "step_mfma_frac": round((flops_oe + flops_pg) / (ms_step / 1e3) / 1e12 / PEAK_BF16_TFLOPS, 4),
        "substeps": substeps, "roofline": roof, "kernels": kernels, "kernels_timing": KERNEL_TIMING_NOTE,
    }


def main():
    args = parse()
    if args.calibrate_copy:
        calibrate_copy(args.calibrate_copy)
        return
    if args.gpus != 1:
        print(f"bench.py measures one GPU only (asked for --gpus {args.gpus}): the library has no "
              "multi-GPU path (the sharding design is documented, not built); run with --gpus 1",
              file=sys.stderr)
        sys.exit(2)
    clk_mhz = max_engine_clock_mhz()
    if args.e2e_diagnostic:
        bench_e2e(args)
        return
    import numpy as np
    import torch

    from paper_2608_14563_amd import api
    from paper_2608_14563_amd import inputs as I

    if not torch.cuda.is_available():
        print("bench.py needs a GPU", file=sys.stderr)
        sys.exit(1)
    dev = torch.device("cuda:0")
    c = I.CONFIGS[args.config]
    if c.diag:
        bench_diag(args, clk_mhz)
        return
    if c.dtype != "bf16":
        print("bench workloads are the bf16 configurations 1-4", file=sys.stderr)
        sys.exit(2)
    full = args.full_mlp
    if full and (args.post_ffn or args.clip_target == "update"):
        print("--full-mlp is timed with the final-norm signal and the gradient clip", file=sys.stderr)
        sys.exit(2)
    log(f"[bench] workload {c.name}: T={c.T} d={c.d} d_ff={c.d_ff} V={c.V} L={c.L}"
        f"{' full-MLP' if full else ''}; generating inputs")
    tg0 = time.perf_counter()
    x, gam, W_U, y = I.hidden(c), I.gain(c), I.unembedding(c), I.targets(c)
    if full:
        caches = [I.mlp_cache(c, l) for l in range(c.L)]
        acts = [cc[2] for cc in caches]
        extras = [I.full_mlp_extra(c, l) for l in range(c.L)]
    else:
        acts = [I.activation(c, l) for l in range(c.L)]
    Wm_host = [I.master_weight(c, l) for l in range(c.L)]
    if full:  # masters in the order of the pseudogradient's norms: W3(0..L-1), W1(..), W2(..)
        Wm_host += [e[1] for e in extras] + [e[2] for e in extras]
    log(f"[bench] inputs generated in {time.perf_counter() - tg0:.1f} s; uploading")
    t = _to_dev(dev)
    tx, tgam, tW, ty = t(x), t(gam), t(W_U), t(y)
    tacts = [t(a) for a in acts]
    Wm = [t(w) for w in Wm_host]
    fkw = {}
    if full:
        fkw = dict(W3_init=[w.to(torch.bfloat16) for w in Wm[:c.L]], gate=[t(cc[0]) for cc in caches],
                   up=[t(cc[1]) for cc in caches], x_in=[t(e[0]) for e in extras],
                   dW1=[torch.empty(c.d_ff, c.d, dtype=torch.float32, device=dev) for _ in range(c.L)],
                   dW2=[torch.empty(c.d_ff, c.d, dtype=torch.float32, device=dev) for _ in range(c.L)])
        host_q, host_u = [cc[0] for cc in caches], [cc[1] for cc in caches]
        del caches
    pffn = None
    if args.post_ffn:
        pf_host = [I.post_ffn(c, l) for l in range(c.L)]
        pffn_mo = [t(m) for m, _ in pf_host]
        pffn_g = [t(g) for _, g in pf_host]
        del pf_host
    plain = args.optimizer == "sgd"
    adam = args.optimizer == "adamw"
    s1 = None if plain else [torch.zeros_like(w) for w in Wm]
    s2 = [torch.zeros_like(w) for w in Wm] if adam else None
    Wlp = [w.to(torch.bfloat16) for w in Wm]
    Wsq = torch.tensor([float((w.astype(np.float64) ** 2).sum()) for w in Wm_host], dtype=torch.float64, device=dev)
    T, d = c.T, c.d
    g_t = torch.empty(T, d, dtype=torch.float32, device=dev)
    g_lp = torch.empty(T, d, dtype=torch.bfloat16, device=dev)
    lse = torch.empty(T, dtype=torch.float32, device=dev)
    loss = torch.empty(T, dtype=torch.float32, device=dev)
    amax = torch.empty(T, dtype=torch.int32, device=dev)
    bad = torch.empty(1, dtype=torch.int32, device=dev)
    dW = [torch.empty(d, c.d_ff, dtype=torch.float32, device=dev) for _ in range(c.L)]
    ss = torch.empty(3 * c.L if full else c.L, dtype=torch.float64, device=dev)
    ws_oe = api.workspace(api.fpo_output_error_workspace(T, d, c.V, torch.bfloat16, args.vocab_chunk), dev)
    stage_default = not args.grad_f32 and not full
    ws_pg = api.workspace(max(api.fpo_pseudograd_workspace(T, d, c.d_ff, c.L, torch.bfloat16, full_mlp=full,
                                                           post_ffn=args.post_ffn, grad_bf16=stg)
                              for stg in ((False, True) if not full else (False,))), dev)
    if args.post_ffn:
        pffn = api.PostFfn(g_t, pffn_mo, pffn_g, c.eps, c.min_rms)
    torch.cuda.synchronize()
    step_no = [0]
    stage = [stage_default]

    def step(mid=None):
        step_no[0] += 1
        api.fpo_output_error(tx, tgam, tW, ty, g_t, g_tilde_lp=g_lp, lse=lse, loss=loss, argmax=amax,
                             bad_targets=bad, ws=ws_oe, eps=c.eps, min_rms=c.min_rms,
                             vocab_chunk=args.vocab_chunk)
        if mid is not None:
            mid.record()
        api.fpo_pseudograd(g_lp, tacts, dW3=None if stage[0] else dW, sumsq=ss, grad_bf16=stage[0],
                           opt=api.OptConfig(kind=1 if adam else 0, lr=c.lr, momentum=0.0 if plain else 0.9,
                                             clip_frac=c.clip_frac, step=step_no[0],
                                             clip_target=1 if args.clip_target == "update" else 0),
                           W_master=Wm, W_lp=Wlp, state1=s1, state2=s2, W_sumsq=Wsq, ws=ws_pg, post_ffn=pffn,
                           **fkw)

    # On the overlapped path (bf16 pseudogradient, gradient clip; W3 only or
    # the full MLP) every optimizer launch runs on a side stream beside the
    # GEMM launches that follow, and the two summed times are close (OLMo-2
    # shapes: within a few percent), so the dominant kernel is taken among the
    # step stream's own.
    overlapped = args.clip_target != "update"
    cu = args.clip_target == "update"

    def work(k, n):
        return kernel_work(k, c, n, None, args.optimizer, args.post_ffn, stage[0], cu, full)

    flops_oe = 4.0 * c.T * c.V * c.d
    flops_pg = 2.0 * c.T * c.d * c.d_ff * c.L * (4 if full else 1)
    # the committed counter profiles cover the default step and the full-MLP step; other variants (post-FFN,
    # optimizer, clip target, fp32 staging, chunk width) change the dominant kernel's traffic: none is looked up
    variant = (args.post_ffn or args.optimizer != "sgd-momentum" or args.clip_target != "gradient" or args.grad_f32
               or args.vocab_chunk)
    tname = c.name + ("-full-mlp" if full else "") + ("-variant" if variant else "")
    res = timed_run(args, step, lambda k: not (overlapped and k == "update"), c, clk_mhz, T, flops_oe, flops_pg,
                    work, traffic_name=tname)
    res["config"] = {"workload": f"{c.name}-shaped FPO step: T={c.T} tokens, d={c.d}, d_ff={c.d_ff}, V={c.V}, "
                                 f"{c.L} target layers ({'W1, W2 and W3 (full-MLP)' if full else 'W3'}"
                                 f"{', post-FFN norm VJP per layer' if args.post_ffn else ''}), bf16 operands / fp32 "
                                 f"accumulate, pseudogradient handed to the update in "
                                 f"{'bf16' if stage_default else 'fp32'}, {OPT_NAME[args.optimizer]} "
                                 f"on fp32 masters, 1% relative clip", "T": c.T, "d": c.d, "d_ff": c.d_ff,
                     "V": c.V, "L": c.L, "optimizer": args.optimizer, "post_ffn_norm": bool(args.post_ffn),
                     "full_mlp": bool(full), "pseudogradient_staging": "bf16" if stage_default else "f32",
                     "clip_target": args.clip_target}
    if stage_default and overlapped:
        # the same step with the pseudogradient handed to the optimizer in fp32
        stage[0] = False
        for _ in range(2):
            step()
        torch.cuda.synchronize()
        ev = [torch.cuda.Event(enable_timing=True) for _ in range(2)]
        ev[0].record()
        for _ in range(args.steps):
            step()
        ev[1].record()
        torch.cuda.synchronize()
        ms32 = ev[0].elapsed_time(ev[1]) / args.steps
        res["substeps"]["grad_f32_ms_per_step"] = round(ms32, 4)
        res["substeps"]["grad_f32_tokens_per_s"] = round(c.T / (ms32 / 1e3), 1)
        log(f"[bench] with the pseudogradient handed over in fp32: {ms32:.3f} ms/step")
    if not args.no_cpu_baseline:
        log("[bench] timing the CPU oracle")
        fb = None
        if full:
            fb = {"W3i": [I.to_storage(w, "bf16") for w in Wm_host[:c.L]], "q": host_q, "u": host_u,
                  "x_in": [e[0] for e in extras]}
        res["cpu_baseline"] = cpu_baseline(c, args.cpu_tokens, x, gam, W_U, y, acts, Wm_host, fb)
    else:
        res["cpu_baseline"] = None
    print(json.dumps(res), flush=True)


if __name__ == "__main__":
    main()
