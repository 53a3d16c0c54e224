"""Benchmark of the ELAS low-rank 2:4 FFN (forward + backward) on one MI355X.

One step = elas_lowrank_ffn_fwd + elas_lowrank_ffn_bwd over one batch of the
LLaMA-1B-shape FFN layer (T = 65536 tokens, d = 2048, d_ff = 5464 (5461 padded),
r = 512), seeded synthetic bf16 inputs resident in HBM.  Prints one JSON line.

Three passes of K steps each: a per-kernel pass with HIP events recorded by
the library on the launch stream around every launch (the kernel table and
the choice of the dominant kernel), the timed region, in which the library
records events around the dominant kernel's launches only (tokens/s and that
kernel's live average duration), and a reference pass without events.
Besides tokens/s it reports:
  roofline  -- the kernel with the largest share of the step, under
               algorithmic accounting: intensity = algorithmic FLOP /
               algorithmic bytes per launch; bound = the lower of the bf16
               MFMA peak and intensity x the HBM peak; achieved and peak in
               that bound's unit, from its average launch time in the timed
               region;
  spgemm    -- the 2:4 sparse x dense down projection (v_smfmac) against the
               sparse bf16 peak (dense-equivalent), and the same for dP;
  kernels   -- every kernel's launches, average time, rates, bound and
               roofline fraction (per-kernel pass);
  cold      -- the step and the sparsify kernel with the caches flushed
               before every call (a 512 MB write);
  configs   -- forward + backward tokens/s of the 60M, 130M and 350M shapes,
               and of the 1B shape with the straight-through backward;
and, timed separately, the standalone sparsify kernel on h [65536 x 2736]
(the 350M-shape activation) against the HBM peak, the 2:4-compressed vs dense
activation run at T = 262144 (large_batch), the forward-only comparison with
the full-rank ReLU^2 FFN at the shapes of the paper's Table 3 (table3), plus
the CPU oracle on a bounded sample of the same workload and on the whole
60M-shape workload with one thread (cpu_baseline).
"""
from __future__ import annotations

import argparse
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

METRIC = "low-rank FFN fwd+bwd tokens/s at 1B shape; 2:4 SpGEMM TFLOP/s vs MFMA peak"
PEAK_BF16_TFLOPS = 2500.0      # MI355X dense bf16 MFMA
PEAK_HBM_GBS = 8000.0          # MI355X HBM3E


def algorithmic_flops(tag: str, T: int, d: int, F: int, r: int) -> float | None:
    """Algorithmic FLOP of one launch of a kernel tag (T tokens per launch).

    Dense products count 2 FLOP per multiply-add.  Products whose one side is
    the 2:4 activation count only the kept half (T r F instead of 2 T r F),
    including the masked dH product whose discarded half is still computed.
    """
    table = {
        "k1_up_gemm": 2 * T * d * r, "k2_up_relu2_sparsify": 2 * T * r * F, "k3_spmm_down": T * r * F,
        "k4_down_gemm": 2 * T * r * d, "b1_dZ": 2 * T * d * r, "b2_dV_down": 2 * T * d * r,
        "b3_dH_masked": T * r * F, "b4_dU_down": T * r * F, "b5_spmm_dP": T * r * F, "b6_dV_up": T * r * F,
        "b7_dU_up": 2 * T * d * r, "b8_dx": 2 * T * d * r,
        # straight-through backward (Eq. 4): dH, dP and dV_up at every position
        "b3_dH_ste": 2 * T * r * F, "b5_dP_dense": 2 * T * r * F, "b6_dV_up_dense": 2 * T * r * F,
    }
    v = table.get(tag)
    return None if v is None else float(v)


def executed_flops(tag: str, T: int, d: int, F: int, r: int) -> float | None:
    """FLOP the kernel actually issues (dense-equivalent for smfmac)."""
    a = algorithmic_flops(tag, T, d, F, r)
    if a is None:
        return None
    Fp = 64 * ((F + 63) // 64)
    if tag in ("k2_up_relu2_sparsify",):
        return 2.0 * T * r * Fp
    if tag in ("k3_spmm_down", "b3_dH_masked", "b4_dU_down", "b5_spmm_dP", "b6_dV_up"):
        return 2.0 * T * r * Fp
    if tag == "b3_dH_ste":   # relu(h) recomputed in the same tile: h and dS, both dense
        return 4.0 * T * r * Fp
    return a


def algorithmic_bytes(tag: str, T: int, d: int, F: int, r: int) -> float | None:
    """HBM bytes one launch must move if every operand is read once and every
    output written once: bf16 tensors 2 B per element, the compressed 2:4
    activation 1.125 B per feature (kept values plus 2-bit codes, Table 2's
    storage), its metadata 0.125 B per feature when read with dH's values,
    fp32 weight gradients 4 B per element."""
    S = T * F * 1.125                 # compressed S: F/2 bf16 values + F/8 code bytes per token
    dH = T * F * 1.0                  # compressed dH values (its codes are S's)
    meta = T * F * 0.125
    table = {
        "k1_up_gemm": 2 * (T * d + d * r + T * r), "k2_up_relu2_sparsify": 2 * (T * r + r * F) + S,
        "k3_spmm_down": S + 2 * (F * r + T * r), "k4_down_gemm": 2 * (T * r + r * d + T * d),
        "b1_dZ": 2 * (T * d + r * d + T * r), "b2_dV_down": 2 * (T * r + T * d) + 4 * r * d,
        "b3_dH_masked": 2 * (T * r + F * r) + S + dH, "b4_dU_down": S + 2 * T * r + 4 * F * r,
        "b5_spmm_dP": dH + meta + 2 * (r * F + T * r), "b6_dV_up": dH + meta + 2 * T * r + 4 * r * F,
        "b7_dU_up": 2 * (T * d + T * r) + 4 * d * r, "b8_dx": 2 * (T * r + d * r + T * d),
        "b3_dH_ste": 2 * (2 * T * r + 2 * F * r) + 2 * T * F, "b5_dP_dense": 2 * (T * F + r * F + T * r),
        "b6_dV_up_dense": 2 * (T * F + T * r) + 4 * r * F,
    }
    v = table.get(tag)
    return None if v is None else float(v)


def roofline_of(tag: str, T: int, d: int, F: int, r: int, avg_s: float) -> dict | None:
    """Roofline of one launch under algorithmic accounting: intensity =
    algorithmic FLOP / algorithmic bytes; the attainable rate is the lower of
    the MFMA peak (2.5 PFLOP/s bf16; also the useful-FLOP peak of the 2:4
    smfmac, which does twice the dense-equivalent work at the dense rate) and
    intensity x 8 TB/s.  The bound is whichever is lower; achieved and peak
    are reported in that bound's unit (TFLOP/s or GB/s)."""
    fl, by = algorithmic_flops(tag, T, d, F, r), algorithmic_bytes(tag, T, d, F, r)
    if fl is None or by is None:
        return None
    ai = fl / by
    hbm_limited = ai * PEAK_HBM_GBS * 1e9 < PEAK_BF16_TFLOPS * 1e12
    if hbm_limited:
        achieved, peak, unit = by / avg_s / 1e9, PEAK_HBM_GBS, "GB/s"
    else:
        achieved, peak, unit = fl / avg_s / 1e12, PEAK_BF16_TFLOPS, "TFLOP/s"
    return {"bound": "hbm" if hbm_limited else "mfma", "achieved": round(achieved, 1), "peak": peak, "unit": unit,
            "frac": round(achieved / peak, 4), "intensity_flop_per_byte": round(ai, 1),
            "alg_flop_per_launch": fl, "alg_bytes_per_launch": by}


TRAFFIC_FILE = os.path.join(ROOT, "profiles", "hbm_traffic_llama1b_fwd_bwd.txt")


def kernel_sources_sha256() -> str:
    """sha256 over the HIP sources (file name then content, sorted by name)."""
    import glob
    import hashlib
    h = hashlib.sha256()
    for f in sorted(glob.glob(os.path.join(ROOT, "paper_2605_03667_amd", "csrc", "*"))):
        h.update(os.path.basename(f).encode())
        with open(f, "rb") as fh:
            h.update(fh.read())
    return h.hexdigest()


def measured_traffic(tag: str):
    """(read bytes, write bytes) per launch of a kernel tag from the committed
    rocprofv3 FETCH_SIZE / WRITE_SIZE summary (copy-calibrated), or None when
    the kernel sources changed since the counters were taken."""
    if not os.path.exists(TRAFFIC_FILE):
        return None
    sha, rows = None, {}
    with open(TRAFFIC_FILE) as f:
        for line in f:
            if line.startswith("kernel_sources_sha256:"):
                sha = line.split(":", 1)[1].strip()
            parts = [x.strip() for x in line.split("|")]
            if len(parts) >= 5 and parts[3].isdigit() and parts[4].isdigit():
                for t in parts[0].split(","):
                    rows[t.strip()] = (int(parts[3]), int(parts[4]))
    if sha != kernel_sources_sha256():
        return None
    return rows.get(tag)


def large_batch_compare(steps: int, warmup: int) -> dict:
    """The 1B shape at T = 262144 tokens, 2:4-compressed vs dense activations:
    tokens/s of forward + backward and activation memory.  `stored_bytes` are
    the tensors the forward keeps for the backward (P, Z and S, compressed or
    dense); `peak_bytes` is torch's allocator high-water mark above the inputs,
    weights and gradients over one forward + backward, each call allocating
    its workspace and freeing it afterwards."""
    import numpy as np
    import torch

    import paper_2605_03667_amd as elas
    from synthetic import CONFIGS, config_inputs

    name = "llama1b_t262144"
    cfg = CONFIGS[name]
    T, d, F, r = cfg["T"], cfg["d"], cfg["d_ff"], cfg["r"]
    dev = torch.device("cuda:0")
    bits = config_inputs(name)
    t = {k: torch.from_numpy(v.view(np.int16)).view(torch.bfloat16).to(dev) for k, v in bits.items()}
    del bits
    f32 = torch.float32
    grads = {"dx": torch.empty((T, d), dtype=torch.bfloat16, device=dev),
             "dU_up": torch.empty((d, r), dtype=f32, device=dev), "dV_up": torch.empty((r, F), dtype=f32, device=dev),
             "dU_down": torch.empty((F, r), dtype=f32, device=dev),
             "dV_down": torch.empty((r, d), dtype=f32, device=dev)}
    out = {}
    for mode, fflags, bflags in (("sparse_2to4", 0, 0), ("dense", elas.ELAS_MODE_DENSE, elas.ELAS_MODE_DENSE)):
        torch.cuda.synchronize()
        base = torch.cuda.memory_allocated(dev)
        torch.cuda.reset_peak_memory_stats(dev)
        ws = torch.empty(elas.elas_lowrank_ffn_fwd_workspace_bytes(T, d, F, r, fflags), dtype=torch.uint8, device=dev)
        saved = elas.elas_lowrank_ffn_fwd(t["x"], t["U_up"], t["V_up"], t["U_down"], t["V_down"], flags=fflags,
                                          workspace=ws)
        del ws
        ws = torch.empty(elas.elas_lowrank_ffn_bwd_workspace_bytes(T, d, F, r, bflags), dtype=torch.uint8, device=dev)
        elas.elas_lowrank_ffn_bwd(t["dY"], t["x"], t["U_up"], t["V_up"], t["U_down"], t["V_down"], saved,
                                  flags=bflags, grads=grads, workspace=ws)
        del ws
        torch.cuda.synchronize()
        peak = torch.cuda.max_memory_allocated(dev) - base
        stored = {k: v.numel() * v.element_size() for k, v in saved.items() if k != "y" and v is not None}
        ws_f = torch.empty(elas.elas_lowrank_ffn_fwd_workspace_bytes(T, d, F, r, fflags), dtype=torch.uint8,
                           device=dev)
        ws_b = torch.empty(elas.elas_lowrank_ffn_bwd_workspace_bytes(T, d, F, r, bflags), dtype=torch.uint8,
                           device=dev)

        def step():
            elas.elas_lowrank_ffn_fwd(t["x"], t["U_up"], t["V_up"], t["U_down"], t["V_down"], flags=fflags,
                                      out=saved, workspace=ws_f)
            elas.elas_lowrank_ffn_bwd(t["dY"], t["x"], t["U_up"], t["V_up"], t["U_down"], t["V_down"], saved,
                                      flags=bflags, grads=grads, workspace=ws_b)

        for _ in range(warmup):
            step()
        a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        torch.cuda.synchronize()
        a.record()
        for _ in range(steps):
            step()
        b.record()
        torch.cuda.synchronize()
        ms = a.elapsed_time(b) / steps
        out[mode] = {"tokens_per_s": round(T / (ms / 1e3), 1), "ms_per_step": round(ms, 3),
                     "stored_bytes": sum(stored.values()), "stored_breakdown": stored, "peak_bytes": int(peak)}
        del saved, ws_f, ws_b
        torch.cuda.empty_cache()
    sp, de = out["sparse_2to4"], out["dense"]
    out["stored_ratio_sparse_over_dense"] = round(sp["stored_bytes"] / de["stored_bytes"], 4)
    s_sp = sp["stored_breakdown"]["s_vals"] + sp["stored_breakdown"]["s_meta"]
    out["activation_ratio_sparse_over_dense"] = round(s_sp / de["stored_breakdown"]["s_vals"], 4)
    out["peak_ratio_sparse_over_dense"] = round(sp["peak_bytes"] / de["peak_bytes"], 4)
    out["config"] = {"workload": name, "T": T, "d": d, "d_ff": F, "r": r}
    return out


# Table 3 (Sec. 4.2.3): FFN speed-up of ELAS over the full-rank FFN, printed
# there as full-rank time / ELAS time for the four model sizes; kept as context.
TABLE3_SEQ = [512, 2048, 4096, 8192, 16384, 32768, 65536]
TABLE3_PAPER = {
    "llama60m": [0.50, 1.57, 1.75, 1.50, 1.55, 1.59, 1.55],
    "llama130m": [0.75, 1.56, 1.80, 1.52, 1.51, 1.53, 1.52],
    "llama350m": [1.29, 1.87, 1.86, 1.82, 1.85, 1.88, 1.88],
    "llama1b": [2.05, 2.47, 2.48, 2.55, 2.63, 2.73, 2.75],
}


def table3_compare(iters: int = 20, warmup: int = 3) -> dict:
    """Forward-only ELAS FFN (2:4 activations) vs the full-rank ReLU^2 FFN
    (elas_fullrank_ffn_fwd, dense MFMA) at the four model shapes and the token
    counts of Table 3, as device time per call (see device_us).  Both blocks
    take their weights as a linear layer stores them (ELAS with
    ELAS_FACTORS_AB: the A, B factors of Eq. 1), which is the kernels'
    operand layout.  `elas_with_relayout_us` times the default ELAS call,
    which re-lays out the four factors on every call (one launch;
    `elas_weight_relayout_us` is that launch).  `fullrank_hipblaslt_us` times
    the same full-rank block built from torch.matmul (hipBLASLt) and torch
    elementwise kernels, as a reference for the baseline's quality.
    `elas_fused_us` times the one-launch fused forward (ELAS_FWD_FUSED) where
    the shape allows it (d <= 1024, r = 128 or 256), else null."""
    import numpy as np
    import torch

    import paper_2605_03667_amd as elas
    from synthetic import CONFIGS, config_inputs, fullrank_inputs

    dev = torch.device("cuda:0")
    Tmax = max(TABLE3_SEQ)

    def to_dev(b):
        return torch.from_numpy(np.ascontiguousarray(b).view(np.int16)).view(torch.bfloat16).to(dev)

    # Device time per call: the calls are queued behind a spin kernel, so the
    # events bracket back-to-back GPU work rather than the host's launch rate.
    a0, b0 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    a0.record()
    torch.cuda._sleep(1 << 22)
    b0.record()
    torch.cuda.synchronize()
    cycles_per_ms = (1 << 22) / max(a0.elapsed_time(b0), 1e-3)
    host_bound = []

    def device_us(fn, queue_ms=30.0):
        for _ in range(warmup):
            fn()
        torch.cuda.synchronize()
        a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        best = float("inf")
        for _ in range(3):
            torch.cuda._sleep(int(cycles_per_ms * queue_ms))
            h0 = time.perf_counter()
            a.record()
            for _ in range(iters):
                fn()
            b.record()
            host_ms = (time.perf_counter() - h0) * 1e3
            torch.cuda.synchronize()
            if host_ms > 0.8 * queue_ms:
                host_bound.append(host_ms)
            best = min(best, a.elapsed_time(b) / iters)
        return best * 1e3

    models = {}
    for k, name in enumerate(TABLE3_PAPER):
        c = CONFIGS[name]
        d, F, r = c["d"], c["d_ff"], c["r"]
        lo = config_inputs(name, T=Tmax, seed_base=40 + k)
        lo.pop("dY")
        fr = fullrank_inputs(0, d, F, c["d_ff_true"], seed_base=40 + k)
        t = {n: to_dev(v) for n, v in lo.items()}
        W_up, W_down = to_dev(fr["W_up"]), to_dev(fr["W_down"])
        del lo, fr
        bf = torch.bfloat16
        o_lo = {"y": torch.empty((Tmax, d), dtype=bf, device=dev), "P": torch.empty((Tmax, r), dtype=bf, device=dev),
                "s_vals": torch.empty((Tmax, elas.elas_vals_ld(F)), dtype=bf, device=dev),
                "s_meta": torch.empty((Tmax, elas.elas_meta_ld(F)), dtype=torch.uint8, device=dev),
                "Z": torch.empty((Tmax, r), dtype=bf, device=dev)}
        o_fr = {"y": torch.empty((Tmax, d), dtype=bf, device=dev), "S": torch.empty((Tmax, F), dtype=bf, device=dev)}
        # the workspace need is not monotonic in T (split-K partials at small T)
        AB = elas.ELAS_FACTORS_AB
        ws = torch.empty(max(1, *(elas.elas_lowrank_ffn_fwd_workspace_bytes(T, d, F, r, fl)
                                  for T in TABLE3_SEQ for fl in (0, AB))), dtype=torch.uint8, device=dev)
        fab = {n: t[n].t().contiguous() for n in ("U_up", "V_up", "U_down", "V_down")}
        row = {"elas_us": [], "elas_with_relayout_us": [], "elas_fused_us": [], "fullrank_us": [],
               "fullrank_hipblaslt_us": [], "speedup": [], "speedup_vs_best": []}
        fused_ok = d % 64 == 0 and d <= 1024 and r in (128, 256)
        Wu_t, Wd_t = W_up.t(), W_down.t()
        for T in TABLE3_SEQ:
            x = t["x"][:T]
            ol = {n: v[:T] for n, v in o_lo.items()}
            of = {n: v[:T] for n, v in o_fr.items()}
            e = device_us(lambda: elas.elas_lowrank_ffn_fwd(x, fab["U_up"], fab["V_up"], fab["U_down"], fab["V_down"],
                                                            flags=AB, out=ol, workspace=ws))
            e_rl = device_us(lambda: elas.elas_lowrank_ffn_fwd(x, t["U_up"], t["V_up"], t["U_down"], t["V_down"],
                                                               out=ol, workspace=ws))
            if fused_ok:
                ef = device_us(lambda: elas.elas_lowrank_ffn_fwd(
                    x, fab["U_up"], fab["V_up"], fab["U_down"], fab["V_down"], flags=AB | elas.ELAS_FWD_FUSED,
                    out=ol, workspace=ws))
                row["elas_fused_us"].append(round(ef, 2))
            f = device_us(lambda: elas.elas_fullrank_ffn_fwd(x, W_up, W_down, out=of))
            # the same block from the vendor GEMM library (torch.matmul -> hipBLASLt) and
            # torch elementwise kernels, as a reference for the full-rank time
            v = device_us(lambda: torch.matmul(torch.relu(torch.matmul(x, Wu_t)).square_(), Wd_t))
            row["elas_us"].append(round(e, 2))
            row["elas_with_relayout_us"].append(round(e_rl, 2))
            row["fullrank_us"].append(round(f, 2))
            row["fullrank_hipblaslt_us"].append(round(v, 2))
            row["speedup"].append(round(f / e, 3))
            row["speedup_vs_best"].append(round(min(f, v) / e, 3))
        # the per-call weight re-layout of the ELAS entry point
        elas.elas_timing_enable(True)
        for _ in range(iters):
            elas.elas_lowrank_ffn_fwd(t["x"][:512], t["U_up"], t["V_up"], t["U_down"], t["V_down"],
                                      out={n: v[:512] for n, v in o_lo.items()}, workspace=ws)
        torch.cuda.synchronize()
        elas.elas_timing_enable(False)
        n_tr, ms_tr = elas.elas_timing_collect().get("weight_transpose", (0, 0.0))
        row["elas_weight_relayout_us"] = round(ms_tr / iters * 1e3, 2)
        T = Tmax
        row["fullrank_tflops_at_max_T"] = round(4.0 * T * d * F / (row["fullrank_us"][-1] * 1e-6) / 1e12, 1)
        row["elas_alg_tflops_at_max_T"] = round(T * (4.0 * d * r + 3.0 * r * F) / (row["elas_us"][-1] * 1e-6) / 1e12, 1)
        if not fused_ok:
            row["elas_fused_us"] = None
        row["shape"] = {"d": d, "d_ff": F, "d_ff_true": c["d_ff_true"], "r": r}
        row["paper_speedup"] = TABLE3_PAPER[name]
        models[name] = row
        del t, fab, W_up, W_down, Wu_t, Wd_t, o_lo, o_fr, ws
        torch.cuda.empty_cache()
    return {"seq": TABLE3_SEQ, "speedup_is": "fullrank_us / elas_us (forward only); speedup_vs_best uses the "
                                              "faster of fullrank_us and fullrank_hipblaslt_us",
            "timing": f"device time per call, best of 3 runs of {iters} calls queued behind a spin kernel",
            "host_bound_runs": len(host_bound), "models": models}


def cpu_model() -> str:
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return "unknown"


def cpu_baseline(cfg: dict, sample_tokens: int) -> dict:
    """The oracle as it stands on the host cores: forward + backward on a
    bounded sample of the 1B-shape workload with every BLAS thread, and the
    whole 60M-shape workload (2048 tokens) on one thread."""
    from threadpoolctl import threadpool_info, threadpool_limits

    from oracle import ffn as offn
    from synthetic import config_inputs

    bits = config_inputs("llama1b", T=sample_tokens)
    t0 = time.perf_counter()
    offn.run(bits)
    dt = time.perf_counter() - t0
    threads = max([p.get("num_threads", 1) for p in threadpool_info() if p.get("user_api") == "blas"] or [1])
    small = config_inputs("llama60m")
    with threadpool_limits(limits=1, user_api="blas"):
        t1 = time.perf_counter()
        offn.run(small)
        dt1 = time.perf_counter() - t1
    return {"value": sample_tokens / dt, "unit": "tokens/s", "cores": int(threads), "kind": "oracle",
            "seconds": dt, "cpu_model": cpu_model(),
            "sample": f"{sample_tokens} tokens of the 1B-shape FFN workload (d={cfg['d']}, d_ff={cfg['d_ff']}, "
                      f"r={cfg['r']}), float64 numpy oracle, forward + backward with bf16 rounding points",
            "llama60m_one_thread": {"tokens_per_s": round(small["x"].shape[0] / dt1, 1), "seconds": round(dt1, 3),
                                    "tokens": int(small["x"].shape[0]), "threads": 1}}


def cold_us(fn, iters: int, flush) -> dict:
    """Device time of fn per call with the caches cold: before every call a
    write of `flush` (512 MB, twice the 256 MB Infinity Cache and far more
    than the L2s) evicts the inputs; each call is bracketed by its own
    events on the current stream."""
    import torch
    out = []
    for i in range(iters):
        flush.fill_(i & 0xFF)
        a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        a.record()
        fn()
        b.record()
        torch.cuda.synchronize()
        out.append(a.elapsed_time(b) * 1e3)
    out.sort()
    return {"median_us": round(out[len(out) // 2], 2), "min_us": round(out[0], 2), "iters": iters}


def config_steps(name: str, steps: int, warmup: int, bwd_flags: int = 0) -> dict:
    """Forward + backward tokens/s of one named workload (warm caches);
    bwd_flags selects the backward (e.g. ELAS_BWD_STE after the 2:4
    forward)."""
    import numpy as np
    import torch

    import paper_2605_03667_amd as elas
    from synthetic import CONFIGS, config_inputs

    c = CONFIGS[name]
    T, d, F, r = c["T"], c["d"], c["d_ff"], c["r"]
    dev = torch.device("cuda:0")
    t = {k: torch.from_numpy(v.view(np.int16)).view(torch.bfloat16).to(dev) for k, v in config_inputs(name).items()}
    ws_f = torch.empty(max(1, elas.elas_lowrank_ffn_fwd_workspace_bytes(T, d, F, r)), dtype=torch.uint8, device=dev)
    ws_b = torch.empty(max(1, elas.elas_lowrank_ffn_bwd_workspace_bytes(T, d, F, r, bwd_flags)), dtype=torch.uint8,
                       device=dev)
    saved = elas.elas_lowrank_ffn_fwd(t["x"], t["U_up"], t["V_up"], t["U_down"], t["V_down"], workspace=ws_f)
    grads = elas.elas_lowrank_ffn_bwd(t["dY"], t["x"], t["U_up"], t["V_up"], t["U_down"], t["V_down"], saved,
                                      flags=bwd_flags, workspace=ws_b)

    def step():
        elas.elas_lowrank_ffn_fwd(t["x"], t["U_up"], t["V_up"], t["U_down"], t["V_down"], out=saved, workspace=ws_f)
        elas.elas_lowrank_ffn_bwd(t["dY"], t["x"], t["U_up"], t["V_up"], t["U_down"], t["V_down"], saved,
                                  flags=bwd_flags, grads=grads, workspace=ws_b)

    for _ in range(warmup):
        step()
    a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    a.record()
    for _ in range(steps):
        step()
    b.record()
    torch.cuda.synchronize()
    ms = a.elapsed_time(b) / steps
    out = {"tokens_per_s": round(T / (ms / 1e3), 1), "ms_per_step": round(ms, 4), "steps": steps,
           "T": T, "d": d, "d_ff": F, "r": r}
    if bwd_flags:
        # per-kernel table of this line: a separate pass with events around every launch
        elas.elas_timing_only(None)
        elas.elas_timing_enable(True)
        torch.cuda.synchronize()
        for _ in range(steps):
            step()
        torch.cuda.synchronize()
        elas.elas_timing_enable(False)
        ks = {}
        for tag, (n, kms) in sorted(elas.elas_timing_collect().items(), key=lambda kv: -kv[1][1]):
            us = kms / n * 1e3
            row = {"launches": n, "avg_us": round(us, 2)}
            fl = algorithmic_flops(tag, T, d, F, r)
            if fl is not None:
                row["alg_tflops"] = round(fl / (us * 1e-6) / 1e12, 1)
                ex = executed_flops(tag, T, d, F, r)
                row["exec_tflops"] = round(ex / (us * 1e-6) / 1e12, 1)
            ks[tag] = row
        out["kernels"] = ks
    del t, ws_f, ws_b, saved, grads
    torch.cuda.empty_cache()
    return out


def main() -> int:
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--workload", default="llama1b")
    ap.add_argument("--cpu-sample", type=int, default=24576, help="tokens for the CPU oracle baseline (0: skip)")
    ap.add_argument("--no-sparsify", action="store_true", help="skip the standalone sparsify measurement")
    ap.add_argument("--no-large-batch", action="store_true",
                    help="skip the T = 262144 compressed-vs-dense activation comparison")
    ap.add_argument("--no-configs", action="store_true",
                    help="skip the forward + backward lines of the 60M, 130M and 350M shapes")
    ap.add_argument("--no-table3", action="store_true",
                    help="skip the forward-only ELAS vs full-rank FFN comparison (Table 3 shapes)")
    ap.add_argument("--copy-calibration", action="store_true",
                    help="also run a plain 1 GiB device copy (known traffic) for HBM counter calibration")
    args = ap.parse_args()
    if args.gpus != 1:
        print(f"bench.py measures one GPU only (--gpus {args.gpus} requested): the ELAS FFN path here is "
              f"single-GPU (data parallelism over tokens would add one all-reduce of the four weight "
              f"gradients per step, not built).", file=sys.stderr)
        return 2

    import numpy as np
    import torch

    import paper_2605_03667_amd as elas
    from synthetic import CONFIGS, SPARSIFY_SHAPE, config_inputs, h_input

    cfg = CONFIGS[args.workload]
    T, d, F, r = cfg["T"], cfg["d"], cfg["d_ff"], cfg["r"]
    dev = torch.device("cuda:0")
    bits = config_inputs(args.workload)

    def to_dev(b):
        return torch.from_numpy(b.view(np.int16)).view(torch.bfloat16).to(dev)

    t = {k: to_dev(v) for k, v in bits.items()}
    del bits
    bf, f32 = torch.bfloat16, torch.float32
    out = {"y": torch.empty((T, d), dtype=bf, device=dev), "P": torch.empty((T, r), dtype=bf, device=dev),
           "s_vals": torch.empty((T, elas.elas_vals_ld(F)), dtype=bf, device=dev),
           "s_meta": torch.empty((T, elas.elas_meta_ld(F)), dtype=torch.uint8, device=dev),
           "Z": torch.empty((T, r), dtype=bf, device=dev)}
    grads = {"dx": torch.empty((T, d), dtype=bf, device=dev), "dU_up": torch.empty((d, r), dtype=f32, device=dev),
             "dV_up": torch.empty((r, F), dtype=f32, device=dev), "dU_down": torch.empty((F, r), dtype=f32, device=dev),
             "dV_down": torch.empty((r, d), dtype=f32, device=dev)}
    ws_f = torch.empty(max(1, elas.elas_lowrank_ffn_fwd_workspace_bytes(T, d, F, r)), dtype=torch.uint8, device=dev)
    ws_b = torch.empty(max(1, elas.elas_lowrank_ffn_bwd_workspace_bytes(T, d, F, r)), dtype=torch.uint8, device=dev)

    def step():
        elas.elas_lowrank_ffn_fwd(t["x"], t["U_up"], t["V_up"], t["U_down"], t["V_down"], out=out, workspace=ws_f)
        elas.elas_lowrank_ffn_bwd(t["dY"], t["x"], t["U_up"], t["V_up"], t["U_down"], t["V_down"], out,
                                  grads=grads, workspace=ws_b)

    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()
    print(f"[bench] warmup done ({args.warmup} steps)", file=sys.stderr, flush=True)

    start, stop = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)

    # ---- per-kernel pass: K steps with events around every launch (the kernel
    # table and the choice of the dominant kernel) ----
    elas.elas_timing_only(None)
    elas.elas_timing_enable(True)
    torch.cuda.synchronize()
    start.record()
    for _ in range(args.steps):
        step()
    stop.record()
    torch.cuda.synchronize()
    elas.elas_timing_enable(False)
    all_ms = start.elapsed_time(stop)
    kernels = elas.elas_timing_collect()
    gemm_tags = [k for k in kernels if algorithmic_flops(k, T, d, F, r) is not None]
    dom = max(gemm_tags, key=lambda k: kernels[k][1])

    # ---- timed region: K steps; the library records events around the
    # dominant kernel's launches only (its live duration for the roofline) ----
    elas.elas_timing_only(dom)
    elas.elas_timing_enable(True)
    torch.cuda.synchronize()
    start.record()
    for _ in range(args.steps):
        step()
    stop.record()
    torch.cuda.synchronize()
    elas.elas_timing_enable(False)
    elas.elas_timing_only(None)
    total_ms = start.elapsed_time(stop)
    dom_timed = elas.elas_timing_collect()[dom]
    ms_per_step = total_ms / args.steps
    tokens_per_s = T / (ms_per_step / 1e3)
    print(f"[bench] timed {args.steps} steps: {ms_per_step:.3f} ms/step", file=sys.stderr, flush=True)

    # same steps without per-kernel events, for reference
    torch.cuda.synchronize()
    start.record()
    for _ in range(args.steps):
        step()
    stop.record()
    torch.cuda.synchronize()
    ms_plain = start.elapsed_time(stop) / args.steps

    ktab = {}
    for tag, (n, ms) in sorted(kernels.items(), key=lambda kv: -kv[1][1]):
        avg_us = ms / n * 1e3
        row = {"launches": n, "avg_us": round(avg_us, 2), "share": round(ms / all_ms, 4)}
        a = algorithmic_flops(tag, T, d, F, r)
        if a is not None:
            row["alg_tflops"] = round(a / (avg_us * 1e-6) / 1e12, 1)
            row["exec_tflops"] = round(executed_flops(tag, T, d, F, r) / (avg_us * 1e-6) / 1e12, 1)
            rf = roofline_of(tag, T, d, F, r, avg_us * 1e-6)
            row.update({"bound": rf["bound"], "frac": rf["frac"], "intensity": rf["intensity_flop_per_byte"]})
        ktab[tag] = row
    dom_avg_s = dom_timed[1] / dom_timed[0] / 1e3
    tr = measured_traffic(dom) if args.workload == "llama1b" else None
    roofline = dict({"kernel": dom}, **roofline_of(dom, T, d, F, r, dom_avg_s))
    roofline.update({"traffic": None if tr is None else tr[0] + tr[1], "avg_us": round(dom_avg_s * 1e6, 2),
                     "alg_tflops": round(algorithmic_flops(dom, T, d, F, r) / dom_avg_s / 1e12, 1),
                     "frac_of_bf16_mfma_peak": round(algorithmic_flops(dom, T, d, F, r) / dom_avg_s / 1e12
                                                     / PEAK_BF16_TFLOPS, 4)})
    if tr is not None:
        roofline["traffic_read_bytes"], roofline["traffic_write_bytes"] = tr
        roofline["traffic_source"] = os.path.relpath(TRAFFIC_FILE, ROOT)

    sp_tag = "k3_spmm_down"
    sp_avg_s = kernels[sp_tag][1] / kernels[sp_tag][0] / 1e3
    sp_alg = algorithmic_flops(sp_tag, T, d, F, r) / sp_avg_s / 1e12
    # The smfmac products: useful (algorithmic) FLOP T r d_ff; the instruction
    # does the 2:4 operand's dense-equivalent work, twice that, at the dense
    # bf16 rate, so its dense-equivalent peak is 5.0 PFLOP/s.
    sp_b5 = kernels["b5_spmm_dP"][1] / kernels["b5_spmm_dP"][0] / 1e3
    spgemm = {"kernel": sp_tag, "avg_us": round(sp_avg_s * 1e6, 2), "alg_tflops": round(sp_alg, 1),
              "dense_equiv_tflops": round(2 * sp_alg, 1),
              "frac_of_sparse_bf16_peak": round(2 * sp_alg / (2 * PEAK_BF16_TFLOPS), 4),
              "sparse_bf16_peak_tflops": 2 * PEAK_BF16_TFLOPS,
              "hbm_gbs": round(algorithmic_bytes(sp_tag, T, d, F, r) / sp_avg_s / 1e9, 1),
              "roofline": roofline_of(sp_tag, T, d, F, r, sp_avg_s),
              "b5_spmm_dP": {"avg_us": round(sp_b5 * 1e6, 2),
                             "frac_of_sparse_bf16_peak": round(algorithmic_flops("b5_spmm_dP", T, d, F, r) / sp_b5
                                                               / 1e12 / PEAK_BF16_TFLOPS, 4)}}

    result = {
        "metric": METRIC, "value": round(tokens_per_s, 1), "unit": "tokens/s", "n_gpus": 1,
        "steps": args.steps, "warmup": args.warmup, "ms_per_step": round(ms_per_step, 4),
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None, "dtype": "bf16",
        "data": "synthetic (seeded Gaussian bf16 inputs, fan-in scaled weights)",
        "config": {"workload": f"{args.workload}_ffn_fwd_bwd", "T": T, "d": d, "d_ff": F,
                   "d_ff_true": cfg["d_ff_true"], "r": r},
        "roofline": roofline, "spgemm": spgemm, "ms_per_step_no_kernel_events": round(ms_plain, 4),
        "ms_per_step_all_kernel_events": round(all_ms / args.steps, 4),
        "kernels": ktab,
    }

    # ---- cold caches: the same step with the Infinity Cache and L2 flushed
    # before every step (a 512 MB write) ----
    flush = torch.empty(512 << 20, dtype=torch.uint8, device=dev)
    cold = cold_us(step, 5, flush)
    result["cold"] = {"step": dict(cold, tokens_per_s=round(T / (cold["median_us"] * 1e-6), 1),
                                   flush_bytes=flush.numel())}

    # ---- the other model shapes, forward + backward (warm) ----
    if not args.no_configs and args.workload == "llama1b":
        del out, grads, ws_f, ws_b, t
        torch.cuda.empty_cache()
        result["configs"] = {n: config_steps(n, args.steps, args.warmup)
                             for n in ("llama60m", "llama130m", "llama350m")}
        # the straight-through backward of Eq. 4 after the 2:4 forward, same workload
        result["configs"]["llama1b_ste_backward"] = config_steps("llama1b", args.steps, args.warmup,
                                                                  elas.ELAS_BWD_STE)
        t = None

    # ---- standalone sparsify on h [65536 x 2736] -----------------------------
    if not args.no_sparsify:
        M, N = SPARSIFY_SHAPE
        if t is not None:
            del out, grads, ws_f, ws_b, t
        torch.cuda.empty_cache()
        h = to_dev(h_input(M, N, seed=2))
        vals = torch.empty((M, elas.elas_vals_ld(N)), dtype=bf, device=dev)
        meta = torch.empty((M, elas.elas_meta_ld(N)), dtype=torch.uint8, device=dev)
        for _ in range(3):
            elas.elas_sparsify_24(h, vals=vals, meta=meta)
        torch.cuda.synchronize()
        elas.elas_timing_enable(True)
        for _ in range(20):
            elas.elas_sparsify_24(h, vals=vals, meta=meta)
        torch.cuda.synchronize()
        elas.elas_timing_enable(False)
        n, ms = elas.elas_timing_collect()["sparsify24"]
        avg_s = ms / n / 1e3
        alg_bytes = M * N * (2 + 1.125)      # read bf16 h, write half the values + 2 bits each
        gbs = alg_bytes / avg_s / 1e9
        # achievable-bandwidth context: a plain device copy of h's size (torch's copy kernel)
        hc = torch.empty_like(h)
        for _ in range(3):
            hc.copy_(h)
        c0, c1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        torch.cuda.synchronize()
        c0.record()
        for _ in range(20):
            hc.copy_(h)
        c1.record()
        torch.cuda.synchronize()
        copy_gbs = 2 * h.numel() * 2 / (c0.elapsed_time(c1) / 20 / 1e3) / 1e9
        del hc
        sp_cold = cold_us(lambda: elas.elas_sparsify_24(h, vals=vals, meta=meta), 10, flush)
        sp_cold["gbs"] = round(alg_bytes / (sp_cold["median_us"] * 1e-6) / 1e9, 1)
        sp_cold["frac"] = round(sp_cold["gbs"] / PEAK_HBM_GBS, 4)
        result["cold"]["sparsify"] = sp_cold
        del flush
        result["sparsify"] = {"shape": [M, N], "avg_us": round(avg_s * 1e6, 2), "alg_bytes": alg_bytes,
                              "copy_gbs_same_size": round(copy_gbs, 1),
                              "frac_of_copy": round(gbs / copy_gbs, 4),
                              "achieved": round(gbs, 1), "peak": PEAK_HBM_GBS, "unit": "GB/s",
                              "frac": round(gbs / PEAK_HBM_GBS, 4)}

    # achievable-MFMA context: a large square bf16 GEMM through torch (hipBLASLt)
    if not args.no_sparsify:
        n_sq = 8192
        a_sq = torch.randn(n_sq, n_sq, device=dev).to(bf)
        b_sq = torch.randn(n_sq, n_sq, device=dev).to(bf)
        c_sq = torch.empty(n_sq, n_sq, device=dev, dtype=bf)
        for _ in range(3):
            torch.matmul(a_sq, b_sq, out=c_sq)
        g0, g1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        torch.cuda.synchronize()
        g0.record()
        for _ in range(10):
            torch.matmul(a_sq, b_sq, out=c_sq)
        g1.record()
        torch.cuda.synchronize()
        sq_tflops = 2.0 * n_sq ** 3 / (g0.elapsed_time(g1) / 10 / 1e3) / 1e12
        result["mfma_achievable"] = {"gemm": f"bf16 {n_sq}^3, torch.matmul (hipBLASLt)",
                                     "tflops": round(sq_tflops, 1), "frac_of_peak": round(sq_tflops / PEAK_BF16_TFLOPS, 4),
                                     "dominant_kernel_alg_tflops_over_achievable": round(roofline["alg_tflops"] / sq_tflops, 4)}
        del a_sq, b_sq, c_sq
        torch.cuda.empty_cache()

    if not args.no_large_batch and args.workload == "llama1b":
        print("[bench] large batch (T = 262144): compressed vs dense activations", file=sys.stderr, flush=True)
        torch.cuda.empty_cache()
        result["large_batch"] = large_batch_compare(steps=5, warmup=2)

    if not args.no_table3 and args.workload == "llama1b":
        print("[bench] forward-only ELAS vs full-rank FFN (Table 3 shapes)", file=sys.stderr, flush=True)
        torch.cuda.empty_cache()
        result["table3"] = table3_compare()

    if args.copy_calibration:
        # a plain copy of known size: reads 1 GiB and writes 1 GiB per launch
        src = torch.empty(1 << 29, dtype=torch.int16, device=dev).fill_(1)
        dst = torch.empty_like(src)
        for _ in range(5):
            dst.copy_(src)
        torch.cuda.synchronize()
        result["copy_calibration"] = {"bytes_read": src.numel() * 2, "bytes_written": dst.numel() * 2,
                                      "launches": 5}
        del src, dst

    if args.cpu_sample > 0:
        print(f"[bench] cpu oracle on {args.cpu_sample} tokens", file=sys.stderr, flush=True)
        result["cpu_baseline"] = cpu_baseline(cfg, args.cpu_sample)

    print(json.dumps(result), flush=True)
    return 0


if __name__ == "__main__":
    sys.exit(main())
