"""Time-to-first-token from an evicted state on one MI355X.

One step = evict (idle phase, untimed) -> [restore_and_prefill -> first_token]
(timed).  The timed part is the whole hot path: restore planning, swap-in on
the side stream, recompute of dropped chunks layer by layer, output head and
argmax.  Inputs (model, context KV, host swap space) are resident before the
timed region starts.

    python bench.py [--gpus 1] [--steps K] [--warmup W] [--workload 8b]

Prints one JSON line: recompute tokens/s (positions pushed through the model
per second of TTFT) as `value`, TTFT in ms, the dominant kernel's roofline
(HIP-event timing of its launches inside the timed steps) and the CPU
oracle's rate on a bounded sample of the same workload.
"""

import argparse
import json
import os
import statistics
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

METRIC = "KV-recompute prefill tokens/s + TTFT ms from evicted state, 1 MI355X"
# HBM bytes per launch of the dominant kernel, from rocprofv3 FETCH_SIZE and
# WRITE_SIZE passes scaled by a 1 GiB copy (profiles/attn_8b_32k_hbm_traffic.md),
# valid only for the kernel source they were taken on and the 8B workload.
MEASURED_TRAFFIC = {"kernel": "attn_kernel", "workload": "8b",
                    "source": "paper_2609_01338_amd/csrc/attention.hip",
                    "sha256": "e379ff2aaacd1b9dd9310f20c3a615f36248714731ee685123cbb4cc4c9eb928",
                    "bytes_per_launch": 1.662e9}
PEAK_MFMA_TFLOPS = 2500.0      # MI355X dense bf16 / fp16 MFMA
PEAK_HBM_GBPS = 8000.0


# Child process that samples the board through amdsmi (read-only metrics):
# one line "time power clk0 clk1 ..." every period, appended to a file.
_SAMPLER = r"""
import sys, time
out, period = sys.argv[1], float(sys.argv[2])
try:
    import amdsmi
    amdsmi.amdsmi_init()
    h = amdsmi.amdsmi_get_processor_handles()[0]
    cap = amdsmi.amdsmi_get_power_cap_info(h)["power_cap"] / 1e6
except Exception as e:
    open(out, "w").write("error %s: %s\n" % (type(e).__name__, e))
    sys.exit(0)
with open(out, "w", buffering=1) as f:
    f.write("cap %r\n" % cap)
    while True:
        try:
            m = amdsmi.amdsmi_get_gpu_metrics_info(h)
            clk = [c for c in (m.get("current_gfxclks") or []) if isinstance(c, (int, float)) and c < 10000]
            pw = m.get("current_socket_power")
            if isinstance(pw, (int, float)) and clk:
                f.write("%.6f %r %s\n" % (time.time(), float(pw), " ".join(str(c) for c in clk)))
        except Exception as e:
            f.write("error %s: %s\n" % (type(e).__name__, e))
        time.sleep(period)
"""


class BoardMonitor:
    """Socket power and per-XCD shader clocks, sampled every `period_s` by a
    child process (started before this process touches the GPU, so the
    sampling takes no time of the measured process) and kept for the time
    windows passed to `window`; the summary is None where amdsmi is
    unavailable."""

    def __init__(self, period_s=0.02):
        import subprocess
        import tempfile
        self.period, self.windows = period_s, []
        fd, self.path = tempfile.mkstemp(prefix="board_", suffix=".txt")
        os.close(fd)
        self.proc = subprocess.Popen([sys.executable, "-c", _SAMPLER, self.path, str(period_s)],
                                     stdin=subprocess.DEVNULL, stdout=subprocess.DEVNULL,
                                     stderr=subprocess.DEVNULL)
        import atexit
        atexit.register(self._stop)   # every exit path ends the sampler

    def _stop(self):
        if self.proc.poll() is None:
            self.proc.terminate()
            try:
                self.proc.wait(timeout=10)
            except Exception:
                self.proc.kill()
                self.proc.wait()

    def window(self, t0, t1):
        self.windows.append((t0, t1))

    def summary(self):
        self._stop()
        try:
            lines = open(self.path).read().splitlines()
        finally:
            os.unlink(self.path)
        cap, samples, err = None, [], None
        for ln in lines:
            f = ln.split()
            if not f:
                continue
            if f[0] == "cap":
                cap = float(f[1])
            elif f[0] == "error":
                err = ln
            else:
                t = float(f[0])
                if any(a <= t <= b for a, b in self.windows):
                    samples.append((float(f[1]), [float(c) for c in f[2:]]))
        if not samples:
            return {"error": err} if err else None
        pw = np.array([x[0] for x in samples])
        n = min(len(x[1]) for x in samples)
        clk = np.array([x[1][:n] for x in samples], dtype=np.float64)
        return {"socket_power_w_mean": round(float(pw.mean()), 1), "socket_power_w_max": round(float(pw.max()), 1),
                "power_cap_w": round(cap, 1) if cap else None, "gfxclk_mhz_mean": round(float(clk.mean()), 1),
                "gfxclk_mhz_per_xcd": [round(float(c), 1) for c in clk.mean(axis=0)],
                "samples": len(samples),
                "source": f"amdsmi current_socket_power / current_gfxclks every {self.period * 1e3:.0f} ms from a "
                          "child process, samples inside the timed steps (GPU busy and idle parts alike)"}


def measured_traffic(kernel, workload):
    """The recorded counter traffic if it still describes this kernel's source, else None."""
    import hashlib
    t = MEASURED_TRAFFIC
    if kernel != t["kernel"] or workload != t["workload"]:
        return None
    try:
        with open(os.path.join(ROOT, t["source"]), "rb") as f:
            if hashlib.sha256(f.read()).hexdigest() != t["sha256"]:
                return None
    except OSError:
        return None
    return t["bytes_per_launch"]


def log(*a):
    print(*a, file=sys.stderr, flush=True)


def host_info():
    """Host the oracle runs on: cores this process may use, CPU model, BLAS."""
    model = ""
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    model = line.split(":", 1)[1].strip()
                    break
    except OSError:
        pass
    blas, threads = "unknown", None
    try:
        from threadpoolctl import threadpool_info
        for i in threadpool_info():
            if i.get("user_api") == "blas":
                blas = f"{i.get('internal_api')} {i.get('version')}"
                threads = int(i.get("num_threads", 1))
                break
    except Exception:
        pass
    cores = len(os.sched_getaffinity(0))
    return {"cores_available": cores, "cpu_model": model, "blas": blas,
            "blas_threads": threads if threads else cores}


def cpu_baseline(w, blob, plan_nR, sample_rows=64):
    """The oracle as it stands, on a bounded sample of the workload's restore:
    one layer's weight decode plus `sample_rows` evenly spaced positions
    through that layer (attention over a synthetic KV cache of the full
    context), extrapolated to the whole restore (L decodes and sum_l nR(l)
    row-layers): an estimate, labelled as one.  The oracle's full restore is
    timed by --cpu-full."""
    import oracle as O
    info = host_info()
    m = w.model
    hp = O.Hyper(m)
    wts = O.Weights(hp, blob)
    S = w.n_ctx + w.n_prompt
    t0 = time.perf_counter()
    lw = wts.layer(0)
    t_decode = time.perf_counter() - t0
    pos = np.linspace(0, S - 1, sample_rows).astype(np.int64)
    rng = np.random.default_rng(0)
    K = rng.standard_normal((S, m.dkv)).astype(np.float16)
    V = rng.standard_normal((S, m.dkv)).astype(np.float16)
    h = wts.rows("emb", rng.integers(0, m.vocab, sample_rows))
    t1 = time.perf_counter()
    O.layer_forward(hp, lw, h, pos, lambda k, v: None,
                    lambda last: (K[:last].astype(np.float64), V[:last].astype(np.float64)))
    t_rows = time.perf_counter() - t1
    total = m.n_layers * t_decode + t_rows * float(np.sum(plan_nR)) / sample_rows
    return {"value": round(plan_nR[0] / total, 3), "unit": "tokens/s", "cores": info["blas_threads"],
            "kind": "oracle", "estimate": True, **info,
            "sample": (f"layer-0 weight decode ({t_decode:.2f} s) + {sample_rows} evenly spaced positions "
                       f"through layer 0 with attention over all {S} keys ({t_rows:.2f} s), extrapolated "
                       f"to {m.n_layers} layers and sum nR = {int(np.sum(plan_nR))} row-layers "
                       f"(est. {total:.1f} s per restore); fp64 numpy, BLAS on {info['blas_threads']} threads")}


def cpu_full_restore(W, key):
    """The oracle's complete evict -> restore -> first token on workload
    `key` (its own plan, context and prompt), timed on this host: the
    never-evicted prefill that builds the cached KV (untimed when nothing is
    kept), then the eviction and the timed restore and first token."""
    import oracle as O
    w = W.WORKLOADS[key]
    m = w.model
    blob = W.make_blob(w)
    ctx, prompt = W.make_tokens(w)
    plan = W.make_plan(w)
    threads = host_info()["blas_threads"]
    ox = O.OracleContext(m, blob, threads=threads)
    t0 = time.perf_counter()
    if (plan.kv_state == W.DROP).all():
        ox.set_context(ctx)           # every chunk is recomputed: no cached KV is read
    else:
        ox.prefill_context(ctx)
    t_pre = time.perf_counter() - t0
    ox.evict(plan.kv_state, plan.w_state)
    t1 = time.perf_counter()
    st = ox.restore_and_prefill(prompt)
    tok, _ = ox.first_token()
    t_restore = time.perf_counter() - t1
    return {"workload": key, "ttft_s": round(t_restore, 3), "tokens_per_s": round(st["nR"][0] / t_restore, 3),
            "nR0": int(st["nR"][0]), "sum_nR": int(sum(st["nR"])), "token": int(tok),
            "context_build_s": round(t_pre, 3)}


def tp_shard_kernels(w, tp):
    """Row GEMMs and attention at the per-GPU shapes of a tp-way split by KV
    head (n_q/tp query heads, n_kv/tp KV heads, d_ffn/tp FFN columns; O and
    down row-split), all S rows, timed through the kernel-level C ABI with HIP
    events on one stream.  Random Q4_0 weights and activations."""
    import torch
    from paper_2609_01338_amd import mz
    from paper_2609_01338_amd import workloads as W
    m = w.model
    S = w.n_ctx + w.n_prompt
    nq, nkv, ff = m.n_q_heads // tp, m.n_kv_heads // tp, m.d_ffn // tp
    hd, d, C = m.head_dim, m.d_model, m.chunk_tokens
    rng = np.random.default_rng(0)
    st = torch.cuda.current_stream()
    sp = st.cuda_stream
    out = {"tp": tp, "rows": S, "n_q_heads": nq, "n_kv_heads": nkv, "ffn_cols": ff}

    def timed(fn, reps=3):
        fn()
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record(st)
        for _ in range(reps):
            fn()
        e1.record(st)
        torch.cuda.synchronize()
        return e0.elapsed_time(e1) / reps

    x = (torch.randn(S, max(d, ff, nq * hd), device="cuda") * 0.5).to(torch.float16)
    for name, n, k, epi in [("q", nq * hd, d, 0), ("kv", 2 * nkv * hd, d, 0), ("o", d, nq * hd, 1),
                            ("gateup", ff, d, 2), ("down", d, ff, 1)]:
        if epi == 2:
            g = W.encode_q4_0((rng.standard_normal((n, k)) * 0.02).astype(np.float32))
            u = W.encode_q4_0((rng.standard_normal((n, k)) * 0.02).astype(np.float32))
            packed = mz.mz_q4_gemm_pack(g, n, k, w_up=u)
            n_pad = 2 * ((n + 127) // 128 * 128)
            y = torch.zeros(S, n_pad // 2, device="cuda", dtype=torch.float16)
        else:
            packed = mz.mz_q4_gemm_pack(W.encode_q4_0((rng.standard_normal((n, k)) * 0.02).astype(np.float32)), n, k)
            n_pad = (n + 255) // 256 * 256
            y = torch.zeros(S, n_pad, device="cuda")
        wt = torch.from_numpy(packed).cuda()
        xa = x[:, :k].contiguous()
        ms = timed(lambda: mz.mz_q4_gemm(xa.data_ptr(), S, n_pad, k, wt.data_ptr(), epi, y.data_ptr(), sp))
        flops = 2.0 * S * (2 * n if epi == 2 else n) * k
        out[f"gemm_{name}"] = {"N": int(2 * n if epi == 2 else n), "K": int(k), "ms": round(ms, 4),
                               "TFLOPs": round(flops / ms / 1e9, 1)}
        del wt, y, xa
    nch = (S + C - 1) // C
    slab = (torch.randn(nch, 2 * C * nkv * hd, device="cuda") * 1.0).to(torch.float16)
    table = torch.arange(nch, device="cuda", dtype=torch.int32)
    q = torch.randn(S, nq * hd, device="cuda").to(torch.float16)
    pos = torch.arange(S, device="cuda", dtype=torch.int32)
    o = torch.empty(S, nq * hd, device="cuda", dtype=torch.float16)
    ms = timed(lambda: mz.mz_attention(q.data_ptr(), pos.data_ptr(), S, slab.data_ptr(), table.data_ptr(), nch, C,
                                       nq, nkv, hd, o.data_ptr(), sp))
    flops = 4.0 * nq * hd * S * (S + 1) / 2
    out["attention"] = {"ms": round(ms, 4), "TFLOPs": round(flops / ms / 1e9, 1)}
    return out


def run_ablation(mz, W, eng, w, prompt, clean_logits, recompute_tflops, link_gbps, steps=3,
                 parts=("plans", "codec", "overlap", "size")):
    """TTFT of every eviction order x placement at the workload's evicted amount
    (as many KV chunks and weight units as its own plan evicts), with the
    planner's estimate beside each, then overlap on/off for two plans."""
    m = w.model
    e = eng.ctx
    base = W.make_plan(w)
    n_kv = int((base.kv_state != W.RES).sum())
    n_w = int((base.w_state != W.RES).sum())
    cfg = mz.make_cfg(m, w.n_ctx + w.n_prompt)

    def ttft_of(kv, ws):
        ts, err = [], 0.0
        for step in range(steps + 1):
            mz.mz_evict(e, kv, ws)
            t0 = time.perf_counter()
            mz.mz_restore_and_prefill(e, prompt)
            tok, logits = mz.mz_first_token(e, m.vocab)
            dt = time.perf_counter() - t0
            mz.mz_truncate_context(e, w.n_ctx)
            if step:
                ts.append(dt * 1e3)
            err = max(err, float(np.abs(logits - clean_logits).max()))
        return statistics.median(ts), err

    rows = []
    for order in (mz.ORDERS if "plans" in parts else ()):
        for placement in mz.PLACEMENTS:
            kv, ws, est = mz.mz_plan_evict(cfg, w.n_ctx, w.n_prompt, n_kv, n_w, order, placement, 1,
                                           link_gbps * 1e9, recompute_tflops * 1e12)
            t, err = ttft_of(kv, ws)
            rows.append({"order": order, "placement": placement, "swap_chunks": int((kv == W.SWAP).sum()),
                         "drop_chunks": int((kv == W.DROP).sum()), "ttft_ms": round(t, 2),
                         "est_link_ms": round(est["link_s"] * 1e3, 2),
                         "est_recompute_ms": round(est["recompute_s"] * 1e3, 2), "max_logit_err_vs_clean": err})
            log(f"[ablation] {order:14s} {placement:15s} TTFT {t:8.2f} ms (est link {est['link_s'] * 1e3:7.1f}, "
                f"recompute {est['recompute_s'] * 1e3:7.1f}) swap/drop {rows[-1]['swap_chunks']}/{rows[-1]['drop_chunks']}")
    codec_rows = []
    mz.mz_set_option(e, "kv_codec", 1)
    for placement in (("balanced", "all-swap", "interleave-2-1") if "codec" in parts else ()):
        kv, ws, est = mz.mz_plan_evict(cfg, w.n_ctx, w.n_prompt, n_kv, n_w, "backward-out", placement, 1,
                                       link_gbps * 1e9, recompute_tflops * 1e12, kv_codec=True)
        t, err = ttft_of(kv, ws)
        codec_rows.append({"order": "backward-out", "placement": placement, "kv_codec": True,
                           "swap_chunks": int((kv == W.SWAP).sum()), "drop_chunks": int((kv == W.DROP).sum()),
                           "ttft_ms": round(t, 2), "est_link_ms": round(est["link_s"] * 1e3, 2),
                           "est_recompute_ms": round(est["recompute_s"] * 1e3, 2),
                           "max_logit_err_vs_clean": err})
        log(f"[ablation] codec backward-out {placement:15s} TTFT {t:8.2f} ms (est link {est['link_s'] * 1e3:7.1f}, "
            f"recompute {est['recompute_s'] * 1e3:7.1f}) swap/drop {codec_rows[-1]['swap_chunks']}/"
            f"{codec_rows[-1]['drop_chunks']} max|logit - clean| {err:.3e}")
    mz.mz_set_option(e, "kv_codec", 0)
    overlap = []
    for placement in (("interleave-2-1", "balanced") if "overlap" in parts else ()):
        kv, ws, _ = mz.mz_plan_evict(cfg, w.n_ctx, w.n_prompt, n_kv, n_w, "backward-out", placement, 1,
                                     link_gbps * 1e9, recompute_tflops * 1e12)
        res = {"placement": placement}
        for ov in (1, 0):
            mz.mz_set_option(e, "overlap", ov)
            res["ttft_ms_overlap" if ov else "ttft_ms_serialized"] = round(ttft_of(kv, ws)[0], 2)
        mz.mz_set_option(e, "overlap", 1)
        overlap.append(res)
        log(f"[ablation] overlap {res}")
    # short requests: all units resident, a 128-token prompt and a single
    # token, then the size-driven 25 % restore, each with the split paths
    # (split-key attention, split-K GEMMs) on and off, per-kind kernel time
    short_rows = []
    if "short" in parts:
        mz.mz_set_option(e, "kv_codec", 1)
        slot_ = m.chunk_tokens * m.dkv * 4
        _, _, eu = mz.mz_plan_evict(cfg, w.n_ctx, w.n_prompt, 0, 1, "backward-out", "all-swap")
        quarter = (m.n_layers * w.n_chunks * slot_ + m.n_layers * int(eu["swap_bytes"])) // 4
        cases = [("resident, 128-token prompt", None, prompt), ("resident, one token", None, prompt[:1]),
                 ("size-driven 25 %, codec",
                  lambda: mz.mz_evict_size(e, quarter, link_gbps * 1e9, recompute_tflops * 1e12, m.n_layers,
                                           w.n_prompt), prompt)]
        for name, evict, prm in cases:
            for split in (1, 0):
                mz.mz_set_option(e, "attn_split", split)
                mz.mz_set_option(e, "gemm_split", split)
                ts = []
                for step in range(steps + 1):
                    if evict:
                        evict()
                    if step == 1:
                        mz.mz_set_option(e, "kernel_timing", 1)
                    t0 = time.perf_counter()
                    mz.mz_restore_and_prefill(e, prm)
                    mz.mz_first_token(e)
                    dt = time.perf_counter() - t0
                    mz.mz_truncate_context(e, w.n_ctx)
                    if step:
                        ts.append(dt * 1e3)
                st = mz.mz_stats(e)
                mz.mz_set_option(e, "kernel_timing", 0)
                kms = {k: round(v["ms"] / steps, 3) for k, v in st["kernels"].items() if v["ms"] > 0}
                t = statistics.median(ts)
                host = {"plan_and_stage_ms": round(st["host_plan_ms"], 3),
                        "enqueue_ms": round(st["host_enqueue_ms"], 3)}
                short_rows.append({"request": name, "split": bool(split), "ttft_ms": round(t, 2),
                                   "kernel_ms": kms, "kernel_sum_ms": round(sum(kms.values()), 3), "host": host})
                log(f"[ablation] short {name:28s} split={split} TTFT {t:8.2f} ms kernel sum "
                    f"{sum(kms.values()):7.2f} ms host {host} kernels {kms}")
        mz.mz_set_option(e, "attn_split", 1)
        mz.mz_set_option(e, "gemm_split", 1)
        mz.mz_set_option(e, "kv_codec", 0)

    # size-driven eviction (hybrid-swap state machine) at fractions of the
    # context's device bytes (every KV slot and weight unit), codec on, with
    # the balanced plan for the same numbers of units beside it
    size_rows = []
    nc = w.n_chunks
    slot = m.chunk_tokens * m.dkv * 4
    _, _, e1 = mz.mz_plan_evict(cfg, w.n_ctx, w.n_prompt, 0, 1, "backward-out", "all-swap")
    total = m.n_layers * nc * slot + m.n_layers * int(e1["swap_bytes"])
    mz.mz_set_option(e, "kv_codec", 1)
    cases = [(r, f) for r in ("paper", "total") for f in (0.25, 0.5, 0.75, 1.0)] if "size" in parts else []
    for rule, frac in cases:
        want = int(total * frac)
        kv0 = np.zeros((m.n_layers, nc), np.uint8)
        ws0 = np.zeros(m.n_layers, np.uint8)
        kv, ws, _, stg, info = mz.mz_plan_evict_size(cfg, w.n_ctx, kv0, ws0, want, link_gbps * 1e9,
                                                     recompute_tflops * 1e12, m.n_layers, w.n_prompt, True, rule)
        ts, err = [], 0.0
        for step in range(steps + 1):
            got = mz.mz_evict_size(e, want, link_gbps * 1e9, recompute_tflops * 1e12, m.n_layers, w.n_prompt,
                                   rule)
            assert got["released"] == info["released"]
            t0 = time.perf_counter()
            mz.mz_restore_and_prefill(e, prompt)
            tok, logits = mz.mz_first_token(e, m.vocab)
            dt = time.perf_counter() - t0
            mz.mz_truncate_context(e, w.n_ctx)
            if step:
                ts.append(dt * 1e3)
            err = max(err, float(np.abs(logits - clean_logits).max()))
        t = statistics.median(ts)
        n_kv_s, n_w_s = int((kv != W.RES).sum()), int((ws != W.RES).sum())
        kvb, wsb, _ = mz.mz_plan_evict(cfg, w.n_ctx, w.n_prompt, n_kv_s, n_w_s, "backward-out", "balanced", 1,
                                       link_gbps * 1e9, recompute_tflops * 1e12, kv_codec=True)
        tb, _ = ttft_of(kvb, wsb)
        counts = np.bincount(stg, minlength=4)
        size_rows.append({"rule": rule, "fraction": frac, "released_bytes": info["released"], "T": info["T"],
                          "stage_units": {"kv_only": int(counts[0]), "kv_and_w": int(counts[1]),
                                          "w_only": int(counts[2])},
                          "swap_chunks": int((kv == W.SWAP).sum()), "drop_chunks": int((kv == W.DROP).sum()),
                          "weight_layers": n_w_s, "ttft_ms": round(t, 2), "max_logit_err_vs_clean": err,
                          "balanced_plan_same_units_ttft_ms": round(tb, 2)})
        log(f"[ablation] evict_size ({rule}) {frac:4.2f} of {total / 1e9:.2f} GB: T {info['T']} stages {counts[:3].tolist()} "
            f"swap/drop {size_rows[-1]['swap_chunks']}/{size_rows[-1]['drop_chunks']} weights {n_w_s} "
            f"TTFT {t:8.2f} ms (balanced plan, same units: {tb:8.2f} ms) max|logit - clean| {err:.3e}")
    mz.mz_set_option(e, "kv_codec", 0)
    return {"n_kv_evicted": n_kv, "n_w_evicted": n_w, "link_gbps": link_gbps,
            "recompute_tflops": recompute_tflops, "plans": rows, "codec_plans": codec_rows, "overlap": overlap,
            "evict_size": size_rows, "short": short_rows}


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=5)
    ap.add_argument("--warmup", type=int, default=2)
    ap.add_argument("--workload", default="8b")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-overlap", action="store_true")
    ap.add_argument("--no-shard", action="store_true", help="skip the per-GPU shard kernel timings")
    ap.add_argument("--decode-only", type=int, default=0, metavar="N",
                    help="after the clean prefill, one restore by the plan, then N timed greedy decode steps "
                         "(no timed restores, CPU baseline or shard timings); prints one JSON line")
    ap.add_argument("--no-decode", action="store_true",
                    help="skip the decode steps after the timed restores (profiler runs of the restore alone)")
    ap.add_argument("--ablation", action="store_true",
                    help="instead of the timed steps: TTFT per eviction order x placement (one JSON line)")
    ap.add_argument("--ablation-parts", default="plans,codec,overlap,size,short",
                    help="comma list of ablation parts: plans, codec, overlap, size, short")
    ap.add_argument("--recompute-tflops", type=float, default=400.0,
                    help="recompute rate the balanced placement assumes (partial-layer recompute of a "
                         "balanced plan runs at about 400 TFLOP/s on MI355X: few rows per GEMM)")
    ap.add_argument("--cpu-full", default=None,
                    help="comma list of workloads: instead of the GPU steps, time the oracle's full evict -> "
                         "restore -> first token on this host (one JSON line)")
    ap.add_argument("--calibrate-copy", action="store_true",
                    help="run one plain 1 GiB device copy first (reference for profiler byte counters)")
    args = ap.parse_args()
    if args.gpus != 1:
        print(f"bench.py measures one GPU: the engine has no multi-GPU path (asked for --gpus {args.gpus})",
              file=sys.stderr)
        sys.exit(2)
    if args.cpu_full:
        from paper_2609_01338_amd import workloads as W
        runs = []
        for key in args.cpu_full.split(","):
            runs.append(cpu_full_restore(W, key))
            log(f"[bench] oracle full restore: {runs[-1]}")
        print(json.dumps({"cpu_full_restore": runs, "kind": "oracle", **host_info()}), flush=True)
        return
    board = BoardMonitor()   # before anything touches the GPU

    # torch (device buffers of the calibration copy and the shard-kernel
    # timings) brings its own HIP runtime; initialising it before libmz is
    # first used makes libmz bind to that same runtime, so one runtime serves
    # the whole process.
    import torch
    torch.cuda.init()
    from paper_2609_01338_amd import mz
    from paper_2609_01338_amd import workloads as W

    if args.calibrate_copy:
        src = torch.ones(1 << 28, device="cuda", dtype=torch.float32)
        dst = torch.empty_like(src)
        dst.copy_(src)
        torch.cuda.synchronize()
        log("[bench] calibration copy: 1 GiB read + 1 GiB written")
        del src, dst

    w = W.WORKLOADS[args.workload]
    m = w.model
    S = w.n_ctx + w.n_prompt
    ceilings = mz.mz_probe_ceilings(0)
    log(f"[bench] measured ceilings: {ceilings}")
    t = time.perf_counter()
    blob = W.make_blob(w)
    log(f"[bench] {w.key}: blob {blob.nbytes / 1e9:.2f} GB in {time.perf_counter() - t:.1f} s")
    ctx_tok, prompt = W.make_tokens(w)
    plan = W.make_plan(w)

    t = time.perf_counter()
    eng = mz.Engine(m, blob, max_ctx=S + 64 + args.decode_only)   # room for the decode steps after the restore
    e = eng.ctx
    log(f"[bench] model loaded in {time.perf_counter() - t:.1f} s")
    if args.no_overlap:
        mz.mz_set_option(e, "overlap", 0)

    # never-evicted reference: clean prefill of context + prompt
    t = time.perf_counter()
    mz.mz_prefill_context(e, np.concatenate([ctx_tok, prompt]))
    clean_tok, clean_logits = mz.mz_first_token(e, m.vocab)
    mz.mz_truncate_context(e, w.n_ctx)
    log(f"[bench] clean prefill of {S} tokens in {time.perf_counter() - t:.2f} s, token {clean_tok}")

    if args.decode_only:
        mz.mz_evict(e, plan.kv_state, plan.w_state)
        mz.mz_restore_and_prefill(e, prompt)
        tok = mz.mz_first_token(e)
        toks = mz.mz_generate(e, tok, 4)                      # warm
        w0 = time.time()
        t = time.perf_counter()
        mz.mz_generate(e, int(toks[-1]), args.decode_only)
        dt = time.perf_counter() - t
        board.window(w0, time.time())
        eng.close()
        res = {"tokens": args.decode_only, "ms_per_token": round(dt * 1e3 / args.decode_only, 3),
               "tokens_per_s": round(args.decode_only / dt, 1), "context": S + 5}
        log(f"[bench] decode after restore: {res['ms_per_token']} ms/token over {args.decode_only} tokens")
        print(json.dumps({"decode_after_restore": res, "workload": w.key, "board": board.summary()}), flush=True)
        return

    if args.ablation:
        res = run_ablation(mz, W, eng, w, prompt, clean_logits, args.recompute_tflops,
                           ceilings["h2d_pinned_gbps"], parts=tuple(args.ablation_parts.split(",")))
        eng.close()
        print(json.dumps({"ablation": res, "workload": w.key, "ceilings_measured": ceilings}), flush=True)
        return

    ttft, toks, logit_err = [], [], []
    stats = None
    for step in range(args.warmup + args.steps):
        timed = step >= args.warmup
        if step == args.warmup:
            mz.mz_set_option(e, "kernel_timing", 1)
        mz.mz_evict(e, plan.kv_state, plan.w_state)
        w0 = time.time()
        t0 = time.perf_counter()
        mz.mz_restore_and_prefill(e, prompt)
        tok, logits = mz.mz_first_token(e, m.vocab)
        dt = time.perf_counter() - t0
        if timed:
            board.window(w0, time.time())
        if timed:
            ttft.append(dt)
        toks.append(tok)
        logit_err.append(float(np.abs(logits - clean_logits).max()))
        stats = mz.mz_stats(e)
        mz.mz_truncate_context(e, w.n_ctx)
        log(f"[bench] step {step} {'timed' if timed else 'warmup'}: TTFT {dt * 1e3:.2f} ms, token {tok}, "
            f"max |logit - clean| {logit_err[-1]:.2e}")

    nR = stats["nR"]
    n_tok = nR[0]
    total_s = sum(ttft)
    ttft_med = statistics.median(ttft)
    value = n_tok * len(ttft) / total_s
    # per-kernel aggregates over the timed steps, grouped by HIP kernel symbol
    by_kernel = {}
    for kind, k in stats["kernels"].items():
        g = by_kernel.setdefault(k["kernel"], {"launches": 0, "ms": 0.0, "flops": 0.0, "bytes": 0.0,
                                               "roles": []})
        for f in ("launches", "ms", "flops", "bytes"):
            g[f] += k[f]
        g["roles"].append(kind)
    dom_name, dom = max(by_kernel.items(), key=lambda kv: kv[1]["ms"])
    if dom["flops"] > 0:
        achieved = dom["flops"] / (dom["ms"] * 1e-3) / 1e12
        roof = {"bound": "mfma", "achieved": round(achieved, 2), "peak": PEAK_MFMA_TFLOPS,
                "unit": "TFLOP/s", "frac": round(achieved / PEAK_MFMA_TFLOPS, 4),
                "traffic": measured_traffic(dom_name, w.key),
                "kernel": dom_name, "roles": dom["roles"],
                "measured_peak": ceilings["mfma_f16_tflops"],
                "frac_of_measured_peak": round(achieved / ceilings["mfma_f16_tflops"], 4),
                "avg_launch_ms": round(dom["ms"] / dom["launches"], 5),
                "flops_per_launch": dom["flops"] / dom["launches"]}
    else:
        achieved = dom["bytes"] / (dom["ms"] * 1e-3) / 1e9
        roof = {"bound": "hbm", "achieved": round(achieved, 2), "peak": PEAK_HBM_GBPS, "unit": "GB/s",
                "frac": round(achieved / PEAK_HBM_GBPS, 4), "traffic": None, "kernel": dom_name,
                "measured_peak": ceilings["hbm_copy_gbps"],
                "frac_of_measured_peak": round(achieved / ceilings["hbm_copy_gbps"], 4),
                "avg_launch_ms": round(dom["ms"] / dom["launches"], 5)}
    steps = len(ttft)
    kernels_ms_per_step = {k: round(v["ms"] / steps, 3) for k, v in stats["kernels"].items()}
    # the recompute projections together (Q, K/V, O, gate/up, down; their
    # split-K forms included): total FLOPs over total kernel time
    proj = [v for k, v in stats["kernels"].items() if k.startswith("gemm_q4")]
    proj_ms, proj_flops = sum(v["ms"] for v in proj), sum(v["flops"] for v in proj)
    proj_tflops = proj_flops / (proj_ms * 1e-3) / 1e12 if proj_ms > 0 else 0.0
    projections = {"ms_per_step": round(proj_ms / steps, 3), "tflops": round(proj_tflops, 1),
                   "frac": round(proj_tflops / PEAK_MFMA_TFLOPS, 4),
                   "frac_of_measured_peak": round(proj_tflops / ceilings["mfma_f16_tflops"], 4)}
    kernel_tflops = {k: round(v["flops"] / (v["ms"] * 1e-3) / 1e12, 1)
                     for k, v in stats["kernels"].items() if v["flops"] > 0}
    algo = stats["algo_flops"]
    out = {
        "metric": METRIC, "value": round(value, 1), "unit": "tokens/s", "n_gpus": 1, "steps": steps,
        "warmup": args.warmup, "ms_per_step": round(total_s / steps * 1e3, 3), "higher_is_better": True,
        "scaling": "weak", "vs_baseline": None, "dtype": "f16", "data": "synthetic",
        "config": {"workload": f"{w.key}: {w.description}", "model": m.name, "n_ctx": w.n_ctx,
                   "n_prompt": w.n_prompt, "chunk_tokens": m.chunk_tokens, "plan": plan.counts(),
                   "weight_units_swapped": int((plan.w_state == W.SWAP).sum()),
                   "nR0": n_tok, "sum_nR": int(sum(nR)), "sum_nD": int(sum(stats["nD"])),
                   "overlap": not args.no_overlap},
        "ttft_ms": round(ttft_med * 1e3, 3),
        "ttft_ms_steps": [round(x * 1e3, 3) for x in ttft],
        "algo_tflop": round(algo / 1e12, 3),
        "host_ms": {"plan_and_stage": round(stats["host_plan_ms"], 3),
                    "enqueue_restore": round(stats["host_enqueue_ms"], 3)},
        "ttft_mfma_frac": round(algo / ttft_med / 1e12 / PEAK_MFMA_TFLOPS, 4),
        "swap_in": {"kv_bytes": stats["swap_kv_bytes"], "w_bytes": stats["swap_w_bytes"],
                    "copies": stats["copies"], "ms": stats["swap_ms"],
                    "GBps": (round((stats["swap_kv_bytes"] + stats["swap_w_bytes"]) / stats["swap_ms"] / 1e6, 2)
                             if stats["swap_ms"] and stats["swap_ms"] > 0 else None)},
        "ceilings_measured": ceilings,
        "board_during_timed_steps": board.summary(),
        "kernel_ms_per_step": kernels_ms_per_step,
        "kernel_tflops": kernel_tflops,
        "projections": projections,
        "invariant": {"clean_token": clean_tok, "tokens": toks,
                      "max_logit_err_vs_clean": max(logit_err)},
        "roofline": roof,
    }
    # past the first token: after the same restore, greedy decode steps
    # (one row each: split-key attention over the whole context and split-K
    # projections), timed as a whole
    mz.mz_set_option(e, "kernel_timing", 0)
    n_dec = 0 if args.no_decode else 32
    if n_dec:
        mz.mz_evict(e, plan.kv_state, plan.w_state)
        mz.mz_restore_and_prefill(e, prompt)
        tok = mz.mz_first_token(e)
        mz.mz_generate(e, tok, 4)                      # warm
        t = time.perf_counter()
        mz.mz_generate(e, int(tok), n_dec)
        dt = time.perf_counter() - t
        out["decode_after_restore"] = {"tokens": n_dec, "ms_per_token": round(dt * 1e3 / n_dec, 3),
                                       "tokens_per_s": round(n_dec / dt, 1), "context": S + 4}
        log(f"[bench] decode after restore: {dt * 1e3 / n_dec:.2f} ms/token over {n_dec} tokens")
        mz.mz_truncate_context(e, w.n_ctx)
    eng.close()
    if w.model.n_kv_heads % 8 == 0 and not args.no_shard:
        t = time.perf_counter()
        out["tp8_shard_kernels"] = tp_shard_kernels(w, 8)
        log(f"[bench] tp8 shard kernels in {time.perf_counter() - t:.1f} s: {out['tp8_shard_kernels']}")
    if not args.no_cpu_baseline:
        t = time.perf_counter()
        out["cpu_baseline"] = cpu_baseline(w, blob, nR)
        log(f"[bench] cpu baseline in {time.perf_counter() - t:.1f} s")
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
