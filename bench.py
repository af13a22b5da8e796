#!/usr/bin/env python3
"""Batched paged decode throughput on one MI355X.

    python bench.py [--gpus 1] [--steps K] [--warmup W] [--workload NAME]

One step = decode_step + sample over the whole active batch: embedding, per
layer RMSNorm + QKV projection, RoPE + KV page write, paged split-K attention,
O projection + residual, RMSNorm + gate/up + SwiGLU, down projection +
residual, then final norm, LM head and greedy argmax.  Greedy tokens feed the
next step on the device.

Inputs are synthetic and seeded: random-init weights of the named shape,
context lengths drawn from the named distribution, and KV pages filled with
N(0,1) bf16 values (the contexts are staged with kv_extend_uninit rather than
prefilled: decode cost does not depend on KV values).  Prints one JSON line.
"""

from __future__ import annotations

import argparse
import dataclasses
import hashlib
import json
import os
import platform
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

METRIC = "decode tokens/sec at batch B + achieved HBM GB/s (% of peak), 1 MI355X"
HBM_PEAK_GBS = 8000.0

# name -> (batch, length distribution)
WORKLOADS = {
    # 8B-shaped decoder, throughput regime: lognormal contexts, median 4096.
    "decode-8b-b256-lognormal": (256, ("lognormal", 4096, 0.8, 256, 32768)),
    # 8B-shaped decoder, long-context tail: B=8, contexts U[65536, 131072].
    "decode-8b-b8-long": (8, ("uniform", 65536, 131072)),
    # multi-turn batch sweep points (capped Pareto contexts), decode only.
    "decode-8b-b16-pareto": (16, ("pareto", 1.5, 1024, 65536)),
    "decode-8b-b64-pareto": (64, ("pareto", 1.5, 1024, 65536)),
    "decode-8b-b256-pareto": (256, ("pareto", 1.5, 1024, 65536)),
    "decode-8b-b512-pareto": (512, ("pareto", 1.5, 1024, 65536)),
    # The same lognormal contexts at the 14B and 32B Qwen3 dimensions (batches
    # sized so that weights and KV fit in one GPU's 288 GB).
    "decode-14b-b128-lognormal": (128, ("lognormal", 4096, 0.8, 256, 32768)),
    "decode-32b-b64-lognormal": (64, ("lognormal", 4096, 0.8, 256, 32768)),
}
# Decoder shape by the model tag in a workload name (decode-<tag>-...).
SHAPE_TAGS = ("8b", "14b", "32b")
# The same workloads with KV pages stored as fp8 (E4M3) codes, scales 1.
FP8_KV = {f"{name}-fp8kv": name for name in ("decode-8b-b256-lognormal", "decode-8b-b8-long",
                                               "decode-8b-b16-pareto", "decode-8b-b64-pareto")}
# The same workloads with the Qwen3-style per-head q/k RMSNorm (gains 1 + 0.1 N(0, 1)).
QK_NORM = {f"{name}-qknorm": name for name in ("decode-8b-b256-lognormal", "decode-8b-b16-pareto")}
DEFAULT_WORKLOAD = "decode-8b-b256-lognormal"
# Multi-turn rollouts: decode segments of 128 steps separated by tool-output
# appends of U[512, 2048] tokens per trajectory through kv_append_prefix.
MULTITURN = {f"multiturn-8b-b{b}": b for b in (16, 64, 256, 512)}


def describe_shape(shape):
    """One line naming a decoder shape, for the JSON config."""
    tag = {4096: "8B", 5120: "14B" if shape.n_layers == 40 else "32B"}.get(shape.d_model, "")
    extra = ", q/k norm" if shape.qk_norm else ""
    return (f"{tag}-shaped decoder ({shape.n_layers}x{shape.d_model}, {shape.n_q_heads}/"
            f"{shape.n_kv_heads} heads, Dh {shape.head_dim}, FFN {shape.ffn_dim}, vocab "
            f"{shape.vocab}{extra}, RoPE base {shape.rope_base:g}), random init")


def log(msg):
    sys.stderr.write(f"[bench] {msg}\n")
    sys.stderr.flush()


def draw_lengths(batch, spec, seed=1):
    from workload import lengths_lognormal, lengths_pareto, lengths_uniform
    kind = spec[0]
    if kind == "lognormal":
        return lengths_lognormal(batch, spec[1], spec[2], spec[3], spec[4], seed)
    if kind == "uniform":
        return lengths_uniform(batch, spec[1], spec[2], seed)
    if kind == "pareto":
        return lengths_pareto(batch, spec[1], spec[2], spec[3], seed)
    raise ValueError(kind)


def gpu_weights(shape, seed=0, std=0.02):
    """Random-init bf16 weights of the given shape, drawn on the GPU."""
    import torch
    g = torch.Generator(device="cuda")
    g.manual_seed(seed)

    import paper_2609_36899_amd as P

    def mat(rows, cols):
        w = torch.empty((rows, cols), dtype=torch.bfloat16, device="cuda")
        w.normal_(0.0, std, generator=g)
        return w

    def proj(rows, cols):  # projections are stored packed
        return P.pack_weight(mat(rows, cols))

    ones = lambda: torch.ones(shape.d_model, dtype=torch.float32, device="cuda")
    out = {"embed": mat(shape.vocab, shape.d_model), "layers": []}
    for _ in range(shape.n_layers):
        out["layers"].append({
            "wq": proj(shape.q_dim, shape.d_model), "wk": proj(shape.kv_dim, shape.d_model),
            "wv": proj(shape.kv_dim, shape.d_model), "wo": proj(shape.d_model, shape.q_dim),
            "w_gate": proj(shape.ffn_dim, shape.d_model),
            "w_up": proj(shape.ffn_dim, shape.d_model),
            "w_down": proj(shape.d_model, shape.ffn_dim), "attn_norm": ones(), "ffn_norm": ones()})
    if getattr(shape, "qk_norm", False):
        for lay in out["layers"]:
            for k in ("q_norm", "k_norm"):
                gain = torch.empty(shape.head_dim, dtype=torch.float32, device="cuda")
                lay[k] = gain.normal_(0.0, 0.1, generator=g).add_(1.0)
    out["lm_head"] = proj(shape.vocab, shape.d_model)
    out["final_norm"] = ones()
    return out


def weight_bytes_per_step(shape, batch, elem=2):
    """Weights read once per step: every matrix except the embedding table,
    of which only the batch's rows are gathered."""
    per_layer = (shape.q_dim + 2 * shape.kv_dim) * shape.d_model + shape.d_model * shape.q_dim \
        + 3 * shape.ffn_dim * shape.d_model
    return elem * (shape.n_layers * per_layer + shape.vocab * shape.d_model
                   + batch * shape.d_model)


class ClockSampler:
    """Samples the GPU's current graphics and memory clocks (MHz) through
    amd-smi while a timed region runs; clocks are not pinned, so they are
    reported beside the timings.  Sampling failures leave the record empty
    with the reason."""

    def __init__(self, device=0, period_s=0.2):
        import threading
        self.device, self.period_s = device, period_s
        self.gfx, self.mem, self.error = [], [], None
        self._stop = threading.Event()
        self._thread = threading.Thread(target=self._run, daemon=True)
        self.bdf = None
        try:
            import amdsmi
            import torch
            props = torch.cuda.get_device_properties(device)
            amdsmi.amdsmi_init()
            # The processor whose PCI domain:bus:device matches this device's.
            for h in amdsmi.amdsmi_get_processor_handles():
                bdf = amdsmi.amdsmi_get_gpu_device_bdf(h)
                dom, bus, dev = bdf.split(".")[0].split(":")
                if (int(dom, 16), int(bus, 16), int(dev, 16)) == (
                        props.pci_domain_id, props.pci_bus_id, props.pci_device_id):
                    self._handle, self.bdf = h, bdf
                    break
            else:
                raise RuntimeError("no amd-smi processor has this device's PCI address")
            self._smi = amdsmi
        except Exception as e:  # no amd-smi on this host: report why
            self._smi, self.error = None, f"{type(e).__name__}: {e}"

    def _read(self):
        t = self._smi.AmdSmiClkType
        for kind, dst in ((t.GFX, self.gfx), (t.MEM, self.mem)):
            info = self._smi.amdsmi_get_clock_info(self._handle, kind)
            v = info.get("clk", info.get("cur_clk"))
            if isinstance(v, (int, float)):
                dst.append(float(v))

    def _run(self):
        while not self._stop.is_set():
            try:
                self._read()
            except Exception as e:
                self.error = f"{type(e).__name__}: {e}"
                return
            self._stop.wait(self.period_s)

    def __enter__(self):
        if self._smi is not None:
            self._thread.start()
        return self

    def __exit__(self, *exc):
        self._stop.set()
        if self._smi is not None:
            self._thread.join()

    def summary(self):
        def stats(v):
            return ({"min": min(v), "median": float(np.median(v)), "max": max(v)}
                    if v else None)
        return {"pinned": False, "source": "amd-smi current clock, sampled every "
                f"{self.period_s:g} s over the timed steps", "pci": self.bdf,
                "samples": len(self.gfx),
                "gfx_mhz": stats(self.gfx), "mem_mhz": stats(self.mem), "error": self.error}


def stream_copy_gbs(n=1 << 30, iters=10):
    """Practical HBM ceiling: a device-to-device copy of n bytes (torch copy_),
    counted as n read + n written per copy, averaged over iters copies."""
    import torch
    a = torch.empty(n, dtype=torch.uint8, device="cuda")
    a.fill_(1)
    b = torch.empty_like(a)
    b.copy_(a)
    ev0, ev1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    ev0.record()
    for _ in range(iters):
        b.copy_(a)
    ev1.record()
    torch.cuda.synchronize()
    ms = ev0.elapsed_time(ev1) / iters
    del a, b
    return {"bytes_per_copy": 2 * n, "avg_ms": round(ms, 4),
            "gbps": round(2 * n / (ms / 1e3) / 1e9, 1), "kernel": "torch copy_ (uint8, 1 GiB)"}


# The decode attention kernel's sources: its counters are reused only while
# all of these are unchanged.
ATTENTION_SOURCES = tuple(os.path.join(ROOT, "paper_2609_36899_amd", "csrc", f)
                          for f in ("attention.hip", "hip_common.h", "fp8_e4m3.h"))


def file_hash(*paths):
    """First 16 hex digits of the SHA-256 of the files' contents, in order."""
    h = hashlib.sha256()
    for path in paths:
        with open(path, "rb") as f:
            h.update(f.read())
    return h.hexdigest()[:16]


def load_traffic(workload, kernel_srcs=ATTENTION_SOURCES):
    """Counter-based HBM bytes per attention launch, if measured for this
    exact kernel source and workload (profiles/attention_traffic.json)."""
    path = os.path.join(ROOT, "profiles", "attention_traffic.json")
    if not os.path.exists(path):
        return None
    try:
        rec = json.load(open(path)).get(workload)
    except (OSError, ValueError):
        return None
    if not rec or rec.get("kernel_sha256_16") != file_hash(*kernel_srcs):
        return None
    return rec.get("bytes_per_launch")


# ---------------------------------------------------------------------------
# CPU baseline: the oracle as it stands, on a bounded sample.
# ---------------------------------------------------------------------------

def cpu_baseline(shape, lens, budget_s=15.0, seed=7):
    """Time the float32 oracle decoder for single trajectories of the batch.

    The sample is a one-layer slice of the model (full layer width) plus the
    LM head, stepped once for a seeded random subset of the batch's
    trajectories at their real context lengths.  Per-token time is
    extrapolated as layers x (step - LM head) + LM head; the oracle handles
    one trajectory at a time, so its throughput is 1 / per-token time.
    """
    import torch

    from oracle import decoder as od
    try:
        from threadpoolctl import threadpool_info
        cores = max((i.get("num_threads", 0) for i in threadpool_info()), default=os.cpu_count())
    except Exception:  # pragma: no cover
        cores = os.cpu_count()
    gen = torch.Generator().manual_seed(seed)

    def mat(r, c):
        return (torch.randn((r, c), generator=gen, dtype=torch.float32) * 0.02).numpy()

    lm = mat(shape.vocab, shape.d_model)
    layer = {"wq": mat(shape.q_dim, shape.d_model), "wk": mat(shape.kv_dim, shape.d_model),
             "wv": mat(shape.kv_dim, shape.d_model), "wo": mat(shape.d_model, shape.q_dim),
             "w_gate": mat(shape.ffn_dim, shape.d_model), "w_up": mat(shape.ffn_dim, shape.d_model),
             "w_down": mat(shape.d_model, shape.ffn_dim),
             "attn_norm": np.ones(shape.d_model, np.float32),
             "ffn_norm": np.ones(shape.d_model, np.float32)}
    w = od.ModelWeights(n_layers=1, n_q_heads=shape.n_q_heads, n_kv_heads=shape.n_kv_heads,
                        head_dim=shape.head_dim, rms_eps=shape.rms_eps, rope_base=shape.rope_base,
                        embed=lm, lm_head=lm, final_norm=np.ones(shape.d_model, np.float32),
                        layers=[layer])
    dec = od.Decoder(w)
    x = np.ones(shape.d_model, np.float32)
    t0 = time.perf_counter()
    for _ in range(3):
        w.lm_head @ od.rmsnorm(x, w.final_norm, w.rms_eps)
    t_lm = (time.perf_counter() - t0) / 3
    order = np.random.default_rng(seed).permutation(len(lens))
    rng = np.random.default_rng(seed + 1)
    per_token, used, spent = [], [], 0.0
    for b in order:
        n = int(lens[b])
        st = dec.new_state()
        st["k"][0] = rng.standard_normal((n, shape.n_kv_heads, shape.head_dim), dtype=np.float32)
        st["v"][0] = rng.standard_normal((n, shape.n_kv_heads, shape.head_dim), dtype=np.float32)
        st["len"] = n
        t0 = time.perf_counter()
        dec.step(st, int(b) % shape.vocab)
        t_step = time.perf_counter() - t0
        spent += t_step
        per_token.append(shape.n_layers * max(t_step - t_lm, 0.0) + t_lm)
        used.append(n)
        if spent >= budget_s:
            break
    t_tok = float(np.mean(per_token))
    return {"value": 1.0 / t_tok, "unit": "tokens/s", "cores": int(cores), "kind": "oracle",
            "sample": (f"float32 oracle, one layer at full width plus the LM head, one decode "
                       f"step for {len(used)} of the batch's {len(lens)} trajectories at their "
                       f"context lengths (mean {np.mean(used):.0f}); per-token time = "
                       f"{shape.n_layers} x (step - LM head {t_lm * 1e3:.1f} ms) + LM head; "
                       f"{spent:.1f} s of stepping"),
            "ms_per_token": t_tok * 1e3}


# ---------------------------------------------------------------------------
# GPU decode run.
# ---------------------------------------------------------------------------

def cpu_model():
    """The host CPU's model name (from /proc/cpuinfo), else the machine type."""
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return platform.processor() or platform.machine()


def run_decode(workload, steps, warmup, with_cpu, seed=1):
    """One decode workload; names in FP8_KV run the same batch with fp8 KV pages,
    names in QK_NORM with per-head q/k RMSNorm."""
    import torch

    import paper_2609_36899_amd as P
    from paper_2609_36899_amd import _native as N
    from workload import EIGHT_B, QWEN3_14B_SHAPED, QWEN3_32B_SHAPED

    base = {"8b": EIGHT_B, "14b": QWEN3_14B_SHAPED, "32b": QWEN3_32B_SHAPED}[workload.split("-")[1]]
    qk = workload in QK_NORM or base.qk_norm
    shape = dataclasses.replace(base, qk_norm=True) if qk else base
    kv_fp8 = (1.0, 1.0) if workload in FP8_KV else None
    batch, spec = WORKLOADS[FP8_KV.get(workload, QK_NORM.get(workload, workload))]
    lens = draw_lengths(batch, spec, seed=seed)
    grow = warmup + steps + min(steps, 8) + 1  # warmup, timed and breakdown steps
    pages = int(np.sum((lens + grow + 15) // 16)) + 64
    per_tok = P.kv_bytes_per_token(shape, P.BF16, kv_fp8)
    pool_bytes = pages * 16 * per_tok
    log(f"{workload}: B={batch}, mean context {lens.mean():.0f}, pool {pool_bytes / 2**30:.1f} GiB")

    torch.cuda.set_device(0)
    weights = gpu_weights(shape)
    E = P.Engine(shape, weights, P.BF16, pool_bytes, max_seqs=batch,
                 max_seq_len=int(lens.max()) + grow + 16, max_batch=batch, max_chunk=16,
                 kv_fp8=kv_fp8)
    g = torch.Generator(device="cuda")
    g.manual_seed(3)
    chunk = 1 << 30
    if kv_fp8 is None:
        pool = E.kv_pool.view(torch.bfloat16)
        for i in range(0, pool.numel(), chunk):
            pool[i:i + chunk].normal_(0.0, 1.0, generator=g)
    else:  # finite E4M3 codes sign | e << 3 | m with e in 4..9 (|x| in 2^-3 .. 2^2.9)
        pool = E.kv_pool
        for i in range(0, pool.numel(), chunk):
            n = min(chunk, pool.numel() - i)
            sign = torch.randint(0, 2, (n,), dtype=torch.uint8, device="cuda", generator=g)
            e = torch.randint(4, 10, (n,), dtype=torch.uint8, device="cuda", generator=g)
            m = torch.randint(0, 8, (n,), dtype=torch.uint8, device="cuda", generator=g)
            pool[i:i + n] = (sign << 7) | (e << 3) | m
            del sign, e, m
    ids = np.array([E.kv_alloc(0) for _ in range(batch)], dtype=np.int32)
    for sid, n in zip(ids, lens):
        E.kv_extend_uninit(int(sid), int(n))
    tok = torch.randint(0, shape.vocab, (batch,), dtype=torch.int32, device="cuda", generator=g)
    logits = torch.empty((batch, shape.vocab), dtype=torch.float32, device="cuda")
    torch.cuda.synchronize()

    def step():
        E.decode_step(ids, tok, logits)
        E.sample(logits, tok)

    for _ in range(warmup):
        step()
    torch.cuda.synchronize()
    log(f"warmup done ({warmup} steps); timing {steps} steps")
    # One event after every step: per-step times for the median and P95.
    marks = [torch.cuda.Event(enable_timing=True) for _ in range(steps + 1)]
    # Only attention launches (the roofline kernel) are timed in the timed
    # region, and only one in every n_layers + 1 of them: a timed launch
    # leaves the GPU idle for a few microseconds around it, and all layers of
    # a step have the same shapes, so one per step (the layer rotating from
    # step to step) measures the kernel without lengthening the step.
    attn_every = shape.n_layers + 1
    E.profile([N.TIMER_ATTENTION], every=attn_every)
    torch.cuda.synchronize()
    with ClockSampler() as clocks:
        w0 = time.perf_counter()
        marks[0].record()
        for i in range(steps):
            step()
            marks[i + 1].record()
        torch.cuda.synchronize()
        wall = time.perf_counter() - w0
    E.profile([])
    gpu_ms = marks[0].elapsed_time(marks[-1])
    step_ms = np.array([marks[i].elapsed_time(marks[i + 1]) for i in range(steps)])
    attn_ms, attn_n = E.profile_read(N.TIMER_ATTENTION)
    # Projection / LM-head breakdown from a few further steps, outside the
    # timed region (their event pairs would lengthen the timed steps).
    bsteps = min(steps, 8)
    E.profile([N.TIMER_GEMM, N.TIMER_LM_HEAD])
    for _ in range(bsteps):
        step()
    torch.cuda.synchronize()
    E.profile([])
    gemm_ms, gemm_n = E.profile_read(N.TIMER_GEMM)
    lm_ms, lm_n = E.profile_read(N.TIMER_LM_HEAD)
    assert np.isfinite(logits[:4].cpu().numpy()).all()

    ms_step = gpu_ms / steps
    tok_s = batch * steps / (gpu_ms / 1e3)
    # Algorithmic bytes, averaged over the timed steps: context at timed step
    # t is lens + warmup + t, and each step reads its new token's KV too.
    mean_keys = float(np.mean([np.sum(lens + warmup + t + 1) for t in range(steps)]))
    kv_read = mean_keys * per_tok
    kv_write = batch * per_tok
    w_bytes = weight_bytes_per_step(shape, batch)
    logit_bytes = 2 * batch * shape.vocab * 4  # LM-head write + argmax read
    step_bytes = kv_read + kv_write + w_bytes + logit_bytes
    hbm = step_bytes / (ms_step / 1e3) / 1e9
    # Per-trajectory effective bandwidth (the paper's bandwidth share): each
    # trajectory's own KV bytes plus its 1/B share of the weights, per step.
    traj_keys = lens + warmup + (steps + 1) / 2.0
    share = (traj_keys * per_tok + w_bytes / batch) / (ms_step / 1e3) / 1e9
    kv_elem = 1 if kv_fp8 is not None else 2
    attn_bytes = mean_keys * shape.n_kv_heads * shape.head_dim * 2 * kv_elem  # per layer launch
    attn_avg_ms = attn_ms / max(attn_n, 1)
    attn_gbs = attn_bytes / (attn_avg_ms / 1e3) / 1e9
    traffic = load_traffic(workload)
    out = {
        "metric": METRIC, "value": round(tok_s, 2), "unit": "tokens/s", "n_gpus": 1,
        "steps": steps, "warmup": warmup, "ms_per_step": round(ms_step, 4),
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None, "dtype": "bf16",
        "data": "synthetic",
        "config": {"workload": workload, "decoder_shape": describe_shape(shape),
                   "batch": int(batch), "context_mean": round(float(lens.mean()), 1),
                   "context_min": int(lens.min()), "context_max": int(lens.max()),
                   "length_distribution": list(spec), "length_seed": seed, "page_tokens": 16,
                   "kv_pages": "fp8 e4m3, scales 1" if kv_fp8 is not None else "bf16",
                   "qk_norm": qk},
        "hbm_gbps": round(hbm, 1), "hbm_frac_of_peak": round(hbm / HBM_PEAK_GBS, 4),
        "step_bytes": int(step_bytes), "wall_s": round(wall, 3),
        "per_trajectory_gbps": {"mean": round(float(share.mean()), 2),
                                "min": round(float(share.min()), 2),
                                "max": round(float(share.max()), 2),
                                "definition": "(own KV bytes + weights / B) per step time"},
        "step_ms": {"median": round(float(np.median(step_ms)), 4),
                    "p95": round(float(np.percentile(step_ms, 95)), 4),
                    "min": round(float(step_ms.min()), 4),
                    "max": round(float(step_ms.max()), 4)},
        "clocks": clocks.summary(),
        "breakdown_ms_per_step": {"attention": round(attn_avg_ms * shape.n_layers, 3),
                                  "projections": round(gemm_ms / bsteps, 3),
                                  "lm_head": round(lm_ms / bsteps, 3)},
        "roofline": {"kernel": "attn_split_bf16<128>" + (" (fp8 pages)" if kv_fp8 else ""),
                     "bound": "hbm",
                     "achieved": round(attn_gbs, 1), "peak": HBM_PEAK_GBS, "unit": "GB/s",
                     "frac": round(attn_gbs / HBM_PEAK_GBS, 4),
                     "traffic": traffic, "bytes_per_launch": int(attn_bytes),
                     "avg_launch_ms": round(attn_avg_ms, 5), "launches": int(attn_n),
                     "launch_sample": f"1 in {attn_every} attention launches of the timed "
                                      "steps (one per step, layer rotating)"},
    }
    del E, weights, logits, pool
    torch.cuda.empty_cache()
    out["stream_copy"] = stream_copy_gbs()
    if with_cpu and not qk:
        log("timing the CPU oracle on a bounded sample")
        out["cpu_baseline"] = cpu_baseline(shape, lens)
    else:
        out["cpu_baseline"] = None
    return out


def append_flops(shape, ctx0, n):
    """Algorithmic flops of appending n tokens onto a cached context of ctx0
    tokens: the layer projections for every new token (2 flops per weight)
    plus attention, 4 Dh flops per (new query, visible key) pair and query
    head; no LM head."""
    per_layer_w = (shape.d_model * (shape.q_dim + 2 * shape.kv_dim) + shape.q_dim * shape.d_model
                   + 3 * shape.d_model * shape.ffn_dim)
    gemm = 2.0 * n * shape.n_layers * per_layer_w
    pairs = n * ctx0 + n * (n + 1) / 2
    return gemm + 4.0 * shape.head_dim * pairs * shape.n_q_heads * shape.n_layers


def run_multiturn(workload, segments, seg_steps, warmup, per_sequence_appends=False,
                  append_chunk=4096):
    """Decode segments with tool-output appends in between.

    Capacity: the pool takes what HBM leaves after weights and workspace.
    When an append does not fit, trajectories depart longest first until it
    does (the pacing rule of evicting the longest resident), and the batch
    continues without them.  Decode tokens/s counts decode_step + sample only;
    append time is reported separately.  Each round of appends is one
    kv_append_prefix_batch call over every live trajectory (tokens packed into
    passes of append_chunk rows), or with per_sequence_appends one
    kv_append_prefix call per trajectory.

    Per decode segment: algorithmic HBM bytes per step (weights once, each
    cached KV byte once, the new KV, the logits write and argmax read) at
    that segment's contexts, and the attention pass's bytes per launch over
    its average launch time (one launch in every n_layers + 1 timed, as in
    the decode workloads).
    """
    import torch

    import paper_2609_36899_amd as P
    from paper_2609_36899_amd import _native as N
    from workload import EIGHT_B, lengths_uniform

    shape = EIGHT_B
    batch = MULTITURN[workload]
    lens = draw_lengths(batch, ("pareto", 1.5, 1024, 65536))
    adds = [lengths_uniform(batch, 512, 2048, seed=10 + k) for k in range(segments - 1)]
    per_tok = P.kv_bytes_per_token(shape, P.BF16)
    kv_layer_tok = shape.n_kv_heads * shape.head_dim * 2 * 2  # K + V bytes per token per layer
    torch.cuda.set_device(0)
    weights = gpu_weights(shape)
    free_b, _ = torch.cuda.mem_get_info()
    want = int(np.sum(lens)) + int(sum(a.sum() for a in adds)) + batch * (segments * seg_steps + warmup + 48)
    pool_tokens = min(want, int((free_b - (24 << 30)) // per_tok))
    pool_bytes = (pool_tokens // 16) * 16 * per_tok
    max_len = int(lens.max()) + int(sum(a.max() for a in adds)) + segments * seg_steps + warmup + 32
    log(f"{workload}: B={batch}, mean context {lens.mean():.0f}, pool {pool_bytes / 2**30:.1f} GiB")
    E = P.Engine(shape, weights, P.BF16, pool_bytes, max_seqs=batch, max_seq_len=max_len,
                 max_batch=batch, max_chunk=append_chunk)
    g = torch.Generator(device="cuda")
    g.manual_seed(3)
    pool_bf16 = E.kv_pool.view(torch.bfloat16)
    for i in range(0, pool_bf16.numel(), 1 << 30):
        pool_bf16[i:i + (1 << 30)].normal_(0.0, 1.0, generator=g)
    ids = [E.kv_alloc(0) for _ in range(batch)]
    for sid, n in zip(ids, lens):
        E.kv_extend_uninit(int(sid), int(n))
    live = list(range(batch))
    tok = torch.randint(0, shape.vocab, (batch,), dtype=torch.int32, device="cuda", generator=g)
    logits = torch.empty((batch, shape.vocab), dtype=torch.float32, device="cuda")
    rng = np.random.default_rng(5)
    dec_ms, dec_tokens, app_ms, app_tokens, app_flops, departed = 0.0, 0, 0.0, 0, 0.0, 0
    dec_bytes = 0.0
    seg_rows = []
    attn_every = shape.n_layers + 1
    w_bytes_b = {}
    ev0, ev1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    for seg in range(segments):
        idarr = np.array([ids[i] for i in live], dtype=np.int32)
        B = len(idarr)
        for _ in range(warmup if seg == 0 else 0):
            E.decode_step(idarr, tok, logits)
            E.sample(logits, tok, batch=B)
        ctx = np.array([E.kv_len(int(s)) for s in idarr], dtype=np.int64)
        torch.cuda.synchronize()
        E.profile([N.TIMER_ATTENTION], every=attn_every)
        ev0.record()
        for _ in range(seg_steps):
            E.decode_step(idarr, tok, logits)
            E.sample(logits, tok, batch=B)
        ev1.record()
        torch.cuda.synchronize()
        E.profile([])
        ms = ev0.elapsed_time(ev1)
        attn_ms, attn_n = E.profile_read(N.TIMER_ATTENTION)
        # Keys read at step t: sum(ctx + t + 1); the mean over the segment.
        mean_keys = float(np.sum(ctx)) + B * (seg_steps + 1) / 2.0
        if B not in w_bytes_b:
            w_bytes_b[B] = weight_bytes_per_step(shape, B)
        step_bytes = (mean_keys * per_tok + B * per_tok + w_bytes_b[B]
                      + 2 * B * shape.vocab * 4)
        hbm = step_bytes / (ms / seg_steps / 1e3) / 1e9
        attn_launch_bytes = mean_keys * kv_layer_tok
        attn_avg_ms = attn_ms / max(attn_n, 1)
        seg_rows.append({"segment": seg, "batch": B, "context_mean": round(float(ctx.mean()), 1),
                         "ms_per_step": round(ms / seg_steps, 4),
                         "tokens_per_s": round(B * seg_steps / (ms / 1e3), 1),
                         "hbm_gbps": round(hbm, 1), "hbm_frac_of_peak": round(hbm / HBM_PEAK_GBS, 4),
                         "attention_gbps": round(attn_launch_bytes / (attn_avg_ms / 1e3) / 1e9, 1),
                         "attention_avg_launch_ms": round(attn_avg_ms, 5),
                         "attention_launches": int(attn_n)})
        dec_ms += ms
        dec_bytes += step_bytes * seg_steps
        dec_tokens += B * seg_steps
        log(f"segment {seg}: B={B}, {ms / seg_steps:.2f} ms/step, {hbm:.0f} GB/s")
        if seg == segments - 1:
            break
        need = int(sum(adds[seg][i] for i in live)) + len(live) * (seg_steps + 32)
        while E.kv_headroom() < need and live:
            longest = max(live, key=lambda i: E.kv_len(ids[i]))
            E.kv_free(ids[longest])
            live.remove(longest)
            departed += 1
            need = int(sum(adds[seg][i] for i in live)) + len(live) * (seg_steps + 32)
        toks = [rng.integers(0, shape.vocab, size=int(adds[seg][i]), dtype=np.int32) for i in live]
        app_flops += sum(append_flops(shape, E.kv_len(ids[i]), len(t)) for i, t in zip(live, toks))
        torch.cuda.synchronize()
        ev0.record()
        if per_sequence_appends:
            for i, t in zip(live, toks):
                E.kv_append_prefix(ids[i], t, chunk_tokens=append_chunk)
        else:
            E.kv_append_prefix_batch([ids[i] for i in live], toks, chunk_tokens=append_chunk)
        ev1.record()
        torch.cuda.synchronize()
        app_tokens += int(sum(len(t) for t in toks))
        app_ms += ev0.elapsed_time(ev1)
        log(f"append {seg}: {app_tokens} tokens so far, {ev0.elapsed_time(ev1):.0f} ms")
    hbm_all = dec_bytes / (dec_ms / 1e3) / 1e9
    # Attention roofline over all segments: bytes-weighted over the segments' launches.
    a_bytes = sum(r["attention_gbps"] * r["attention_avg_launch_ms"] for r in seg_rows)
    a_ms = sum(r["attention_avg_launch_ms"] for r in seg_rows)
    attn_gbs = a_bytes / a_ms if a_ms else None
    out = {
        "metric": METRIC, "value": round(dec_tokens / (dec_ms / 1e3), 2), "unit": "tokens/s",
        "n_gpus": 1, "steps": segments * seg_steps, "warmup": warmup,
        "ms_per_step": round(dec_ms / (segments * seg_steps), 4), "higher_is_better": True,
        "scaling": "weak", "vs_baseline": None, "dtype": "bf16", "data": "synthetic",
        "config": {"workload": workload, "batch": batch, "segments": segments,
                   "steps_per_segment": seg_steps, "append_tokens": "U[512, 2048] per trajectory",
                   "append_call": ("kv_append_prefix per trajectory" if per_sequence_appends
                                   else "kv_append_prefix_batch over the live trajectories"),
                   "append_chunk_tokens": append_chunk,
                   "context_mean_initial": round(float(lens.mean()), 1),
                   "pool_tokens": int(pool_bytes // per_tok)},
        "hbm_gbps": round(hbm_all, 1), "hbm_frac_of_peak": round(hbm_all / HBM_PEAK_GBS, 4),
        "segments_detail": seg_rows,
        "roofline": {"kernel": "attn_split_bf16<128>", "bound": "hbm",
                     "achieved": round(attn_gbs, 1) if attn_gbs else None,
                     "peak": HBM_PEAK_GBS, "unit": "GB/s",
                     "frac": round(attn_gbs / HBM_PEAK_GBS, 4) if attn_gbs else None,
                     "traffic": None,
                     "launch_sample": f"1 in {attn_every} attention launches of the decode "
                                      "segments (layer rotating), bytes-weighted over segments"},
        "departed": departed, "final_batch": len(live),
        "append": {"tokens": int(app_tokens), "ms": round(app_ms, 1),
                   "prefill_tokens_per_s": round(app_tokens / (app_ms / 1e3), 1) if app_ms else None,
                   "tflops_per_s": round(app_flops / (app_ms / 1e3) / 1e12, 1) if app_ms else None,
                   "mfma_frac": round(app_flops / (app_ms / 1e3) / 1e12 / PEAK_BF16_TFLOPS, 4)
                   if app_ms else None},
        # decoded tokens over decode and append time together
        "end_to_end_tokens_per_s": round(dec_tokens / ((dec_ms + app_ms) / 1e3), 2),
        "cpu_baseline": None,
    }
    return out


# Decode landscape: batch x mean context x within-batch skew (lognormal sigma).
LANDSCAPE = {"batches": (1, 4, 16, 64, 256), "means": (1024, 4096, 16384, 65536),
             "sigmas": (0.0, 1.0)}


def run_landscape(steps=8, warmup=2):
    """Decode throughput over batch x mean context x skew (one engine per cell).

    Per cell: tokens/s, step time, achieved HBM GB/s over the algorithmic
    bytes (weights once + every cached KV byte once + new KV + logits) and
    the mean per-trajectory bandwidth share (KV_b + W / B) / step time.
    Cells whose KV does not fit in free HBM are reported as skipped.
    """
    import torch

    import paper_2609_36899_amd as P
    from workload import EIGHT_B, lengths_skewed

    shape = EIGHT_B
    torch.cuda.set_device(0)
    weights = gpu_weights(shape)
    per_tok = P.kv_bytes_per_token(shape, P.BF16)
    w_bytes_layerless = weight_bytes_per_step(shape, 0)
    cells = []
    for batch in LANDSCAPE["batches"]:
        for mean in LANDSCAPE["means"]:
            for sigma in LANDSCAPE["sigmas"]:
                if batch == 1 and sigma > 0:
                    continue
                lens = lengths_skewed(batch, mean, sigma, seed=batch * 7919 + mean)
                grow = warmup + steps + 1
                pages = int(np.sum((lens + grow + 15) // 16)) + 64
                pool_bytes = pages * 16 * per_tok
                free, _ = torch.cuda.mem_get_info()
                cell = {"batch": batch, "mean_context": mean, "sigma": sigma,
                        "max_context": int(lens.max()), "kv_gib": round(pool_bytes / 2**30, 1)}
                if pool_bytes > free - (8 << 30):
                    cell["skipped"] = "KV exceeds free HBM"
                    cells.append(cell)
                    continue
                E = P.Engine(shape, weights, P.BF16, pool_bytes, max_seqs=batch,
                             max_seq_len=int(lens.max()) + grow + 16, max_batch=batch,
                             max_chunk=16)
                g = torch.Generator(device="cuda")
                g.manual_seed(batch + mean)
                pool = E.kv_pool.view(torch.bfloat16)
                for i in range(0, pool.numel(), 1 << 30):
                    pool[i:i + (1 << 30)].normal_(0.0, 1.0, generator=g)
                ids = np.array([E.kv_alloc(0) for _ in range(batch)], dtype=np.int32)
                for sid, n in zip(ids, lens):
                    E.kv_extend_uninit(int(sid), int(n))
                tok = torch.randint(0, shape.vocab, (batch,), dtype=torch.int32, device="cuda",
                                    generator=g)
                logits = torch.empty((batch, shape.vocab), dtype=torch.float32, device="cuda")
                for _ in range(warmup):
                    E.decode_step(ids, tok, logits)
                    E.sample(logits, tok)
                torch.cuda.synchronize()
                a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
                a.record()
                for _ in range(steps):
                    E.decode_step(ids, tok, logits)
                    E.sample(logits, tok)
                b.record()
                torch.cuda.synchronize()
                ms = a.elapsed_time(b) / steps
                keys = float(np.mean([np.sum(lens + warmup + t + 1) for t in range(steps)]))
                w_bytes = w_bytes_layerless + 2 * batch * shape.d_model
                step_bytes = keys * per_tok + batch * per_tok + w_bytes + 2 * batch * shape.vocab * 4
                share = (float(np.mean(lens)) * per_tok + w_bytes / batch) / (ms / 1e3) / 1e9
                cell.update({"tokens_per_s": round(batch / (ms / 1e3), 1), "ms_per_step": round(ms, 3),
                             "hbm_gbps": round(step_bytes / (ms / 1e3) / 1e9, 1),
                             "hbm_frac": round(step_bytes / (ms / 1e3) / 1e9 / HBM_PEAK_GBS, 3),
                             "share_gbps_per_traj": round(share, 1)})
                cells.append(cell)
                log(f"landscape B={batch} mean={mean} sigma={sigma}: {cell['tokens_per_s']} tok/s, "
                    f"{cell['hbm_gbps']} GB/s")
                del E, pool, logits
                torch.cuda.empty_cache()
    return {"metric": "decode tokens/s over batch x mean context x skew, 1 MI355X",
            "value": None, "unit": "tokens/s", "n_gpus": 1, "steps": steps, "warmup": warmup,
            "higher_is_better": True, "data": "synthetic", "dtype": "bf16",
            "config": {"workload": "landscape-8b", **{k: list(v) for k, v in LANDSCAPE.items()}},
            "cells": cells, "cpu_baseline": None}


def run_sampling(batches=(1, 4, 16, 32, 64, 256, 512), vocab=128256, iters=20):
    """Greedy argmax and temperature/top-p sampling over 8B-sized logit rows:
    time per call (HIP events) at each batch size; top-p both in the form the
    library picks for the batch (split over several groups per row for small
    batches) and with one work group per row."""
    import torch

    import paper_2609_36899_amd as P
    from workload import TINY

    torch.cuda.set_device(0)
    g = torch.Generator(device="cuda")
    g.manual_seed(0)
    # greedy sampling goes through an engine's `sample`; a tiny engine with
    # the full vocabulary supplies it (only its vocab size matters here).
    shape = dataclasses.replace(TINY, vocab=vocab)
    w = gpu_weights_f32_tiny(shape)
    E = P.Engine(shape, w, P.F32, 4 * 16 * P.kv_bytes_per_token(shape, P.F32), max_seqs=1,
                 max_seq_len=16, max_batch=max(batches), max_chunk=16)
    ev0, ev1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    rows = []
    for b in batches:
        logits = (torch.randn((b, vocab), device="cuda", generator=g) * 3.0).contiguous()
        u = torch.rand(b, device="cuda", generator=g)
        out = torch.empty(b, dtype=torch.int32, device="cuda")
        res = {"batch": b}
        need = P.sample_top_p_workspace_bytes(b)
        ws = torch.empty(max(need, 1), dtype=torch.uint8, device="cuda")
        for name, fn in (("greedy_us", lambda: E.sample(logits, out, batch=b)),
                         ("top_p_us", lambda: P.sample_top_p(logits, out, 0.8, 0.95, u,
                                                             workspace=ws)),
                         ("top_p_one_group_us", lambda: P.sample_top_p(logits, out, 0.8, 0.95,
                                                                       u, split=False))):
            for _ in range(3):
                fn()
            torch.cuda.synchronize()
            ev0.record()
            for _ in range(iters):
                fn()
            ev1.record()
            torch.cuda.synchronize()
            res[name] = round(ev0.elapsed_time(ev1) / iters * 1e3, 2)
        rows.append(res)
        log(f"sampling B={b}: {res}")
    return {"metric": "sampling time per call over 128256-token logit rows, 1 MI355X",
            "value": None, "unit": "us", "n_gpus": 1, "higher_is_better": False,
            "data": "synthetic", "dtype": "f32",
            "config": {"workload": "sampling-8b", "vocab": vocab, "temperature": 0.8,
                       "top_p": 0.95},
            "rows": rows, "cpu_baseline": None}


def gpu_weights_f32_tiny(shape):
    """fp32 weights of a small shape, drawn on the GPU and packed."""
    import torch

    import paper_2609_36899_amd as P
    g = torch.Generator(device="cuda")
    g.manual_seed(1)

    def mat(r, c):
        return torch.empty((r, c), device="cuda").normal_(0.0, 0.02, generator=g)

    ones = lambda: torch.ones(shape.d_model, device="cuda")
    layers = [{"wq": P.pack_weight(mat(shape.q_dim, shape.d_model)),
               "wk": P.pack_weight(mat(shape.kv_dim, shape.d_model)),
               "wv": P.pack_weight(mat(shape.kv_dim, shape.d_model)),
               "wo": P.pack_weight(mat(shape.d_model, shape.q_dim)),
               "w_gate": P.pack_weight(mat(shape.ffn_dim, shape.d_model)),
               "w_up": P.pack_weight(mat(shape.ffn_dim, shape.d_model)),
               "w_down": P.pack_weight(mat(shape.d_model, shape.ffn_dim)),
               "attn_norm": ones(), "ffn_norm": ones()} for _ in range(shape.n_layers)]
    return {"embed": mat(shape.vocab, shape.d_model),
            "lm_head": P.pack_weight(mat(shape.vocab, shape.d_model)),
            "final_norm": ones(), "layers": layers}


def run_attention_isolated(calls=50):
    """The attention pass alone (paged_decode_attention) on the isolated
    workload: B=64, 32/8 heads, Dh 128, contexts U[1024, 8192], block tables
    from one random permutation of a 200k-page pool; K/V pages N(0,1) bf16.
    Per call: host planning, one metadata upload, the split pass and the
    merge, timed with HIP events over back-to-back calls."""
    import torch

    import paper_2609_36899_amd as P
    from workload import lazy_paged_attention_case, lengths_uniform

    B, HQ, HKV, DH, POOL = 64, 32, 8, 128, 200000
    lens = lengths_uniform(B, 1024, 8192, seed=21)
    case = lazy_paged_attention_case(B, HQ, HKV, DH, lens, POOL, seed=22)
    torch.cuda.set_device(0)
    g = torch.Generator(device="cuda")
    g.manual_seed(5)
    k = torch.empty((POOL, HKV, 16, DH), dtype=torch.bfloat16, device="cuda").normal_(generator=g)
    v = torch.empty((POOL, HKV, DH, 16), dtype=torch.bfloat16, device="cuda").normal_(generator=g)
    q = torch.empty((B, HQ, DH), dtype=torch.bfloat16, device="cuda").normal_(generator=g)
    bt = torch.from_numpy(case.block_table).cuda()
    out = torch.empty((B, HQ, DH), dtype=torch.float32, device="cuda")
    ws = torch.empty(P.paged_attention_workspace_bytes(B, HQ, HKV, DH), dtype=torch.uint8,
                     device="cuda")
    P.paged_decode_attention(q, k, v, bt, lens, out, ws)  # checks the page ids once
    for _ in range(3):
        P.paged_decode_attention(q, k, v, bt, lens, out, ws, check_pages=False)
    torch.cuda.synchronize()
    ev0, ev1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    ev0.record()
    for _ in range(calls):
        P.paged_decode_attention(q, k, v, bt, lens, out, ws, check_pages=False)
    ev1.record()
    torch.cuda.synchronize()
    us = ev0.elapsed_time(ev1) / calls * 1e3
    kv_bytes = int(np.sum(lens)) * HKV * DH * 2 * 2
    assert np.isfinite(out[:2].cpu().numpy()).all()
    gbs = kv_bytes / (us * 1e-6) / 1e9
    return {"metric": "isolated paged decode attention, 1 MI355X", "value": round(gbs, 1),
            "unit": "GB/s (K+V bytes read once / call time)", "n_gpus": 1,
            "higher_is_better": True, "data": "synthetic", "dtype": "bf16",
            "config": {"workload": "attention-b64", "batch": B, "heads": [HQ, HKV], "head_dim": DH,
                       "context": "U[1024, 8192]", "pool_pages": POOL,
                       "context_mean": round(float(lens.mean()), 1)},
            "us_per_call": round(us, 2), "kv_bytes": kv_bytes,
            "frac_of_peak": round(gbs / HBM_PEAK_GBS, 4), "calls": calls, "cpu_baseline": None}


def run_tiny(steps=32, warmup=3):
    """Decode-step latency of the tiny fp32 decoder (2 layers, d 256, 4/2
    heads, Dh 64, FFN 688, vocab 1024) at B=4 after prefixes {17, 40, 96,
    128}: a launch-bound shape, reported as time per step."""
    import torch

    import paper_2609_36899_amd as P
    from workload import TINY, random_tokens

    torch.cuda.set_device(0)
    w = gpu_weights_f32_tiny(TINY)
    prefixes = (17, 40, 96, 128)
    per_tok = P.kv_bytes_per_token(TINY, P.F32)
    E = P.Engine(TINY, w, P.F32, 4096 * per_tok, max_seqs=4, max_seq_len=512, max_batch=4,
                 max_chunk=128)
    ids = []
    for i, n in enumerate(prefixes):
        s_id = E.kv_alloc(0)
        E.kv_append_prefix(s_id, random_tokens(n, TINY.vocab, seed=100 + i), chunk_tokens=128)
        ids.append(s_id)
    ids = np.array(ids, dtype=np.int32)
    tok = torch.zeros(4, dtype=torch.int32, device="cuda")
    logits = torch.empty((4, TINY.vocab), dtype=torch.float32, device="cuda")
    for _ in range(warmup):
        E.decode_step(ids, tok, logits)
        E.sample(logits, tok)
    torch.cuda.synchronize()
    marks = [torch.cuda.Event(enable_timing=True) for _ in range(steps + 1)]
    w0 = time.perf_counter()
    marks[0].record()
    for i in range(steps):
        E.decode_step(ids, tok, logits)
        E.sample(logits, tok)
        marks[i + 1].record()
    torch.cuda.synchronize()
    wall = time.perf_counter() - w0
    step_ms = np.array([marks[i].elapsed_time(marks[i + 1]) for i in range(steps)])
    return {"metric": "decode step latency, tiny fp32 decoder, 1 MI355X",
            "value": round(float(np.median(step_ms)), 4), "unit": "ms per step (median)",
            "n_gpus": 1, "higher_is_better": False, "data": "synthetic", "dtype": "f32",
            "config": {"workload": "tiny-fp32", "batch": 4, "prefixes": list(prefixes)},
            "steps": steps, "step_ms_p95": round(float(np.percentile(step_ms, 95)), 4),
            "wall_ms_per_step": round(wall / steps * 1e3, 4),
            "tokens_per_s": round(4 / (float(np.mean(step_ms)) / 1e3), 1), "cpu_baseline": None}


def run_copy_calibration(n=1 << 30):
    """One device copy of n bytes (torch copy_): the reference kernel whose
    FETCH_SIZE / WRITE_SIZE counters calibrate the HBM traffic figures."""
    import torch
    torch.cuda.set_device(0)
    a = torch.empty(n, dtype=torch.uint8, device="cuda")
    a.fill_(1)
    b = torch.empty_like(a)
    torch.cuda.synchronize()
    b.copy_(a)
    torch.cuda.synchronize()
    return {"metric": "device copy for counter calibration", "value": n, "unit": "bytes",
            "n_gpus": 1, "config": {"workload": "copy-1gib"}, "cpu_baseline": None}


def run_paced_rollout(n_traj=160, decode=256, max_batch=160, pool_frac=0.5, delta=16):
    """Headroom-paced rollout (pacing_plan + PacedRollout) on the 8B shape.

    n_traj trajectories with lognormal prompts (median 1024, clamped to
    [256, 4096]) each decode ``decode`` teacher-forced tokens; the KV pool
    holds pool_frac of their final KV and at most max_batch reside at once;
    decode growth outruns the per-resident reserve delta, so the rollout
    evicts (longest first below the floor) and places (shortest first above
    the reserve).  New prompts are staged without
    computing KV, as in the decode workloads; evicted trajectories come back
    by KV snapshot restore or by re-prefill, one run each.
    """
    import torch

    import paper_2609_36899_amd as P
    from workload import EIGHT_B, lengths_lognormal, random_tokens

    shape = EIGHT_B
    torch.cuda.set_device(0)
    weights = gpu_weights(shape)
    prompts = lengths_lognormal(n_traj, 1024, 0.8, 256, 4096, seed=21)
    per_tok = P.kv_bytes_per_token(shape, P.BF16)
    final_tokens = int(np.sum((prompts + decode + 15) // 16 * 16))
    pool_bytes = int(final_tokens * pool_frac) // 16 * 16 * per_tok
    runs = {}
    for restore in ("snapshot", "reprefill"):
        E = P.Engine(shape, weights, P.BF16, pool_bytes, max_seqs=n_traj + 8,
                     max_seq_len=int(prompts.max()) + decode + 32, max_batch=max_batch,
                     max_chunk=2048)
        drv = P.PacedRollout(E, h_min=max_batch * 16, delta=delta, restore=restore,
                             chunk_tokens=2048)
        for i, n in enumerate(prompts):
            drv.add(i, random_tokens(int(n) + decode, shape.vocab, seed=500 + i), int(n),
                    staged=True)
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        steps = decoded = 0
        while not drv.finished and steps < 50 * decode:
            decoded += len(drv.step())
            steps += 1
        torch.cuda.synchronize()
        wall = time.perf_counter() - t0
        assert drv.finished
        runs[restore] = {"decode_tokens_per_s": round(decoded / wall, 1), "wall_s": round(wall, 3),
                         "steps": steps, "decoded_tokens": decoded, **drv.stats}
        log(f"paced rollout ({restore}): {runs[restore]}")
        E.close()
        del E, drv
        torch.cuda.empty_cache()
    return {"metric": "decode tokens/s of a headroom-paced rollout, 1 MI355X",
            "value": runs["snapshot"]["decode_tokens_per_s"], "unit": "tokens/s", "n_gpus": 1,
            "higher_is_better": True, "data": "synthetic", "dtype": "bf16",
            "config": {"workload": "paced-rollout-8b", "trajectories": n_traj,
                       "decode_tokens": decode, "max_batch": max_batch, "pool_fraction": pool_frac,
                       "prompt_lengths": ["lognormal", 1024, 0.8, 256, 4096],
                       "h_min_tokens": max_batch * 16, "delta_tokens": delta},
            "runs": runs, "cpu_baseline": None}


PROJ_SHAPES = [("qkv", 6144, 4096), ("o", 4096, 4096), ("gate_up", 28672, 4096),
               ("down", 4096, 14336), ("lm_head", 128256, 4096)]


def run_projections(batches=(1, 2, 4, 8, 16, 32, 64, 128, 256, 512), iters=24,
                    workload="projections-8b", value_batch=256):
    """The 8B projection shapes through weight_projection, swept over the batch,
    and the gate/up pair through swiglu_projection (the decode step's path).

    Per shape and batch: time per call (HIP events), weight-stream GB/s,
    TFLOP/s, and the roofline time max(weights / 8 TB/s, flops / 2.5 PF/s).
    Calls rotate over copies of the weight totalling >= 768 MB, so every call
    streams its weight from HBM rather than from the 256 MB last-level cache
    (as in a decode step, where 32 layers' weights pass through).  The time
    includes the split-K reduction kernel, which inside a decode step is fused
    into the consumer.  For context, torch.matmul (hipBLASLt) on row-major
    copies of the same weights, rotated the same way, bf16 output.
    """
    import torch

    import paper_2609_36899_amd as P

    torch.cuda.set_device(0)
    g = torch.Generator(device="cuda")
    g.manual_seed(0)
    ev0, ev1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)

    def timed(fn, n_copies):
        for i in range(3):
            fn(i % n_copies)
        torch.cuda.synchronize()
        n = max(iters, 2 * n_copies)
        ev0.record()
        for i in range(n):
            fn(i % n_copies)
        ev1.record()
        torch.cuda.synchronize()
        return ev0.elapsed_time(ev1) / n * 1e3

    rows = []
    for name, n, k in PROJ_SHAPES:
        copies = max(1, -(-(768 << 20) // (2 * n * k)))
        raw = [torch.empty((n, k), dtype=torch.bfloat16, device="cuda").normal_(
            0, 0.02, generator=g) for _ in range(copies)]
        packed = [P.pack_weight(w) for w in raw]
        for m in batches:
            x = torch.empty((m, k), dtype=torch.bfloat16, device="cuda").normal_(generator=g)
            out = torch.empty((m, n), dtype=torch.float32, device="cuda")
            ws = torch.empty(max(1, P.weight_projection_workspace_bytes(P.BF16, m, n, k)),
                             dtype=torch.uint8, device="cuda")
            us = timed(lambda i: P.weight_projection(x, packed[i], out, ws), copies)
            ref_us = timed(lambda i: torch.matmul(x, raw[i].t()), copies)
            wbytes, flops = 2 * n * k, 2 * m * n * k
            roof_us = max(wbytes / HBM_PEAK_GBS / 1e3, flops / 2.5e15 * 1e6)
            rows.append({"shape": name, "N": n, "K": k, "M": m, "us": round(us, 2),
                         "weight_GBps": round(wbytes / us / 1e3, 1),
                         "TFLOPs": round(flops / us / 1e6, 1),
                         "roofline_us": round(roof_us, 2), "frac_of_roofline": round(roof_us / us, 3),
                         "torch_matmul_us": round(ref_us, 2)})
        del raw, packed
        torch.cuda.empty_cache()
        log(f"projections {name} done")
    # The decode step's own gate/up path: both matrices in one call with the
    # SwiGLU applied in the GEMM epilogue where the plan has no K split.
    from workload import EIGHT_B
    F, d = EIGHT_B.ffn_dim, EIGHT_B.d_model
    copies = max(1, -(-(768 << 20) // (4 * F * d)))
    pairs = [[P.pack_weight(torch.empty((F, d), dtype=torch.bfloat16, device="cuda").normal_(
        0, 0.02, generator=g)) for _ in range(2)] for _ in range(copies)]
    for m in batches:
        x = torch.empty((m, d), dtype=torch.bfloat16, device="cuda").normal_(generator=g)
        u = torch.empty((m, F), dtype=torch.bfloat16, device="cuda")
        ws = torch.empty(max(1, P.swiglu_projection_workspace_bytes(P.BF16, m, F, d)),
                         dtype=torch.uint8, device="cuda")
        us = timed(lambda i: P.swiglu_projection(x, pairs[i][0], pairs[i][1], u, ws), copies)
        wbytes, flops = 4 * F * d, 4 * m * F * d
        roof_us = max(wbytes / HBM_PEAK_GBS / 1e3, flops / 2.5e15 * 1e6)
        rows.append({"shape": "gate_up_swiglu", "N": 2 * F, "K": d, "M": m, "us": round(us, 2),
                     "weight_GBps": round(wbytes / us / 1e3, 1),
                     "TFLOPs": round(flops / us / 1e6, 1),
                     "roofline_us": round(roof_us, 2), "frac_of_roofline": round(roof_us / us, 3),
                     "torch_matmul_us": None})
    del pairs
    torch.cuda.empty_cache()
    log("projections gate_up_swiglu done")
    layer, layer_ref = {}, {}
    # Per layer as the decode step runs it: qkv + o + fused gate/up + down.
    for r in rows:
        if r["shape"] in ("qkv", "o", "gate_up_swiglu", "down"):
            layer[r["M"]] = layer.get(r["M"], 0.0) + r["us"]
        if r["shape"] in ("qkv", "o", "gate_up", "down"):
            layer_ref[r["M"]] = layer_ref.get(r["M"], 0.0) + r["torch_matmul_us"]
    return {"metric": "weight projection time per 8B layer, 1 MI355X",
            "value": layer.get(value_batch), "unit": f"us at batch {value_batch}", "n_gpus": 1,
            "higher_is_better": False, "data": "synthetic", "dtype": "bf16",
            "config": {"workload": workload, "batches": list(batches)},
            "layer_us": {str(m): round(v, 1) for m, v in layer.items()},
            "layer_us_torch_matmul": {str(m): round(v, 1) for m, v in layer_ref.items()},
            "rows": rows, "cpu_baseline": None}


PEAK_BF16_TFLOPS = 2500.0  # MI355X dense bf16 MFMA


def prefill_flops(shape, n):
    """Algorithmic flops of prefilling n tokens from an empty context: the
    layer projections for every token (2 flops per weight) plus causal
    attention, 4 Dh flops per (query, visible key) pair and query head.
    No LM head (the append computes no logits here)."""
    per_layer_w = (shape.d_model * (shape.q_dim + 2 * shape.kv_dim) + shape.q_dim * shape.d_model
                   + 3 * shape.d_model * shape.ffn_dim)
    gemm = 2.0 * n * shape.n_layers * per_layer_w
    attn = 4.0 * shape.head_dim * (n * (n + 1) / 2) * shape.n_q_heads * shape.n_layers
    return gemm + attn


def run_kv_transfer(lengths=(4096, 16384, 65536), chunk=4096, kv_fp8=None):
    """Prepared KV versus re-prefill for one departing trajectory.

    For each context length: kv_export of the trajectory's KV into pinned
    host memory (device to host), kv_import into a fresh sequence (host to
    device), and kv_append_prefix re-prefilling the same tokens in passes of
    `chunk` rows.  This is the prepared-transfer versus re-prefill trade-off
    of late-bound KV preparation, on one GPU.  One untimed pass first loads
    the kernels.  kv_fp8 = (k_scale, v_scale) stores the pages as E4M3 codes.
    """
    import torch

    import paper_2609_36899_amd as P
    from workload import EIGHT_B, random_tokens

    shape = EIGHT_B
    per_tok = P.kv_bytes_per_token(shape, P.BF16, kv_fp8)
    torch.cuda.set_device(0)
    weights = gpu_weights(shape)
    pool_tokens = 3 * max(lengths) + 4096
    E = P.Engine(shape, weights, P.BF16, pool_tokens * per_tok, max_seqs=8,
                 max_seq_len=max(lengths) + 64, max_batch=8, max_chunk=chunk, kv_fp8=kv_fp8)
    ev0, ev1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    warm = E.kv_alloc(0)
    E.kv_append_prefix(warm, random_tokens(chunk, shape.vocab, seed=1), chunk_tokens=chunk)
    torch.cuda.synchronize()
    E.kv_free(warm)
    rows = []
    for n in lengths:
        toks = random_tokens(n, shape.vocab, seed=n)
        a = E.kv_alloc(0)
        torch.cuda.synchronize()
        ev0.record()
        E.kv_append_prefix(a, toks, chunk_tokens=chunk)
        ev1.record()
        torch.cuda.synchronize()
        prefill_ms = ev0.elapsed_time(ev1)
        snap = torch.empty(E.kv_snapshot_bytes(n), dtype=torch.uint8).pin_memory()
        ev0.record()
        E.kv_export(a, snap)
        ev1.record()
        torch.cuda.synchronize()
        export_ms = ev0.elapsed_time(ev1)
        E.kv_free(a)
        b = E.kv_alloc(0)
        ev0.record()
        E.kv_import(b, snap, n)
        ev1.record()
        torch.cuda.synchronize()
        import_ms = ev0.elapsed_time(ev1)
        E.kv_free(b)
        nbytes = snap.numel()
        rows.append({"tokens": n, "snapshot_bytes": nbytes, "export_ms": round(export_ms, 2),
                     "export_GBps": round(nbytes / export_ms / 1e6, 1),
                     "import_ms": round(import_ms, 2),
                     "import_GBps": round(nbytes / import_ms / 1e6, 1),
                     "reprefill_ms": round(prefill_ms, 1),
                     "reprefill_tokens_per_s": round(n / prefill_ms * 1e3, 1),
                     "reprefill_tflops_per_s": round(prefill_flops(shape, n) / prefill_ms / 1e9, 1),
                     "reprefill_mfma_frac": round(prefill_flops(shape, n) / prefill_ms / 1e9
                                                  / PEAK_BF16_TFLOPS, 3)})
        log(f"kv transfer {n}: export {export_ms:.1f} ms, import {import_ms:.1f} ms, "
            f"re-prefill {prefill_ms:.0f} ms")
        del snap
    return {"metric": "KV snapshot/restore vs re-prefill, 8B-shaped, 1 MI355X",
            "value": rows[-1]["reprefill_ms"] / rows[-1]["import_ms"], "unit": "x (re-prefill / import)",
            "n_gpus": 1, "higher_is_better": True, "data": "synthetic", "dtype": "bf16",
            "config": {"workload": "kv-transfer-8b" + ("-fp8kv" if kv_fp8 else ""),
                       "lengths": list(lengths), "chunk_tokens": chunk,
                       "kv_pages": "fp8 e4m3, scales 1" if kv_fp8 else "bf16"}, "rows": rows,
            "cpu_baseline": None}


def main():
    ap = argparse.ArgumentParser(description=__doc__, formatter_class=argparse.RawTextHelpFormatter)
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=64)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--workload", default=DEFAULT_WORKLOAD,
                    choices=sorted(WORKLOADS) + sorted(FP8_KV) + sorted(QK_NORM)
                    + sorted(MULTITURN)
                    + ["kv-transfer-8b", "kv-transfer-8b-fp8kv", "projections-8b", "landscape-8b", "sampling-8b",
                       "copy-1gib", "paced-rollout-8b", "attention-b64", "tiny-fp32",
                       "projections-8b-prefill"])
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--seed", type=int, default=1,
                    help="seed of the context-length draw of the decode workloads")
    ap.add_argument("--append-per-sequence", action="store_true",
                    help="multi-turn: one kv_append_prefix call per trajectory")
    ap.add_argument("--append-chunk", type=int, default=4096,
                    help="rows per prefill pass: multi-turn appends and the kv-transfer re-prefill")
    args = ap.parse_args()
    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) != 1:
        print("bench.py runs on exactly one GPU: the decode engine is one worker's backend "
              "and trajectories shard across GPUs as independent engines (data parallel, no "
              "exchange).  Run with --gpus 1.", file=sys.stderr)
        sys.exit(2)
    if args.workload == "kv-transfer-8b":
        out = run_kv_transfer(chunk=args.append_chunk)
    elif args.workload == "kv-transfer-8b-fp8kv":
        out = run_kv_transfer(chunk=args.append_chunk, kv_fp8=(1.0, 1.0))
    elif args.workload == "projections-8b-prefill":
        out = run_projections(batches=(1024, 2048, 4096), workload="projections-8b-prefill",
                              value_batch=4096)
    elif args.workload == "projections-8b":
        out = run_projections()
    elif args.workload == "landscape-8b":
        out = run_landscape()
    elif args.workload == "sampling-8b":
        out = run_sampling()
    elif args.workload == "copy-1gib":
        out = run_copy_calibration()
    elif args.workload == "attention-b64":
        out = run_attention_isolated()
    elif args.workload == "tiny-fp32":
        out = run_tiny()
    elif args.workload == "paced-rollout-8b":
        out = run_paced_rollout()
    elif args.workload in MULTITURN:
        out = run_multiturn(args.workload, segments=3, seg_steps=args.steps, warmup=args.warmup,
                            per_sequence_appends=args.append_per_sequence,
                            append_chunk=args.append_chunk)
    else:
        out = run_decode(args.workload, args.steps, args.warmup, not args.no_cpu_baseline,
                         seed=args.seed)
    out["host"] = {"cpu": cpu_model(), "cpu_count": os.cpu_count()}
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
