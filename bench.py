#!/usr/bin/env python3
"""MomentKV hot-path benchmark on one MI355X.

Workload (default): the Qwen3-4B-shaped 36-layer stack with 32K-token prefill contexts
(32 query heads, 8 KV heads, head_dim 128, bf16), at budgets 128, 256, 512, 1024 and 2048
retained tokens per KV head.  Seeded synthetic post-RoPE inputs are generated on the
GPU and stay resident in HBM.  One timed step is one pass of the whole hot path:

  for every budget: momentkv_compress of each of the 36 layers (per-layer calls), writing
                    that layer's retained cache and moments into a 36-layer stack, then
                    momentkv_prepare_summary over the stack (the summaries' decode form);
  then 128 decode tokens: for each token and each budget one momentkv_decode_attn launch
                    over the flattened (layer x sequence) batch of 36 caches, appending the
                    token's key/value (budgets interleaved, so consecutive launches touch
                    different caches and the 256 MB last-level cache cannot hold them).

The decode phase of a step (all 128 x 5 launches) is captured once as a HIP graph and
replayed, as a serving loop would run it: the host does not pace the GPU; so is each
budget's compress phase (the 36 calls and the summaries' decode form).  Every replay is
checked bit for bit against the same phase run eagerly.

Reported (one JSON line): decode attention+correction GB/s (algorithmic bytes / replay
time, the `value`), decode tokens/s, compress ms/layer per budget, per-budget decode
times (replay of the whole phase minus replay of the phase without that budget, so the
other budgets still keep the last-level cache cold), a roofline object for the decode call
and the fp64 oracle timed on the host as a CPU baseline; `compress_roofline` sets the
compress call and its context-streaming kernels against HBM and the bf16 MFMA peak (kernel
times, traffic and MFMA activity from the committed rocprofv3 summary of the workload), and
`compress_stacked` times one compress call over the whole stack per budget.  Further phases are measured
the same way on the same compressed stacks and reported beside the headline, which they do
not change: the decode with the summary in half precision (`decode_half_summary`), the
compress with head-adaptive budgets (`compress_adaptive`) and the decode step with
moment-informed eviction at every token (`evict_decode`).  Events are
recorded on the stream the library launches on.
"""
from __future__ import annotations

import argparse
import json
import math
import os
import sys
import time

import torch

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

from paper_2606_01563_amd import synth  # noqa: E402
from paper_2606_01563_amd import momentkv as mk  # noqa: E402

HBM_PEAK_GBS = 8000.0
MFMA_BF16_PEAK_TFLOPS = 2500.0   # dense bf16 matrix peak of the MI355X


# max_len from which momentkv_decode_evict (n_split = 0) takes the one-read shape: a scoring
# launch with the attention, then a finishing launch (shorter caches: one launch)
EVICT_ONE_READ_MIN_LEN = 320

def decode_bytes(n_heads: int, G: int, d: int, lens_after: int, elem: int = 2) -> int:
    """Algorithmic HBM bytes of one decode launch (per KV head, summed over heads):
    retained K and V rows read, the d x d summary and its two vectors and count read,
    the G queries read and G outputs written, the appended key/value read and written,
    and lens read and written."""
    per_head = (2 * lens_after * d * elem + 4 * d * d + 8 * d + 4 + 2 * G * d * elem
                + 4 * d * elem + 8)
    return n_heads * per_head


def compress_bytes(n_kv_heads: int, N: int, d: int, L: int, elem: int = 2) -> int:
    """Algorithmic bytes of one layer's compress: K and V read once, retained rows written,
    the summary written."""
    return n_kv_heads * (2 * N * d * elem + 2 * L * d * elem + 4 * d * d + 8 * d + 4 + 4 * L)


def compress_kernel_work(n_heads: int, G: int, w: int, N: int, d: int, n_sink: int = 1,
                         elem: int = 2) -> dict:
    """Algorithmic HBM bytes and flops per launch of the compress passes that stream the
    context, for one call over `n_heads` KV heads (C = N - w - n_sink candidates):
      k_rows_cov   K and V read once; window logits 2 G w N d (MFMA) and the candidate
                   covariance V_C^T K_C, 2 |C| d^2 (MFMA);
      k_mass       K read once; the window logits again, 2 G w N d (MFMA);
      k_residual   K and V of the candidates read once; S_tilde0 k_j for every candidate on
                   two bf16 planes, 2 x 2 |C| d^2 (MFMA)."""
    C = N - w - n_sink
    logits = 2 * G * w * N * d * n_heads
    cov = 2 * C * d * d * n_heads
    return {"k_rows_cov": {"bytes": 2 * N * d * elem * n_heads, "flops": logits + cov,
                           "covariance_flops": cov},
            "k_mass": {"bytes": N * d * elem * n_heads, "flops": logits},
            "k_residual": {"bytes": 2 * C * d * elem * n_heads, "flops": 2 * cov}}


def _profile_json(path: str, sha_key: str):
    """The machine-readable block of a committed rocprofv3 summary, or None when the file is
    missing or the sources it lists have changed since the counters were taken."""
    import hashlib
    import re
    if not os.path.exists(path):
        return None
    m = re.search(r"```json\n(\{.*?\})\n```", open(path).read(), re.S)
    if not m:
        return None
    data = json.loads(m.group(1))
    h = hashlib.sha256()
    for src in data["sources"]:
        with open(os.path.join(ROOT, src), "rb") as f:
            h.update(f.read())
    return data if h.hexdigest() == data[sha_key] else None


def compress_roofline(wl, budgets, ms_per_layer: dict) -> dict:
    """Compress against its roofs.  The whole call: algorithmic bytes per layer (K and V read
    once, retained rows and summary written) over the measured ms per layer (HBM roof).  The
    passes that stream the context, from the committed rocprofv3 summary of this workload
    (profiles/compress_<workload>.md, only while the compress sources are unchanged): kernel
    time per launch, algorithmic bytes over it against HBM, MFMA flops over it against the
    bf16 peak, MFMA-busy share of the kernel's time (SQ_VALU_MFMA_BUSY_CYCLES), measured HBM
    traffic per call (FETCH_SIZE + WRITE_SIZE, calibrated on a plain copy) over the
    algorithmic bytes; and the covariance's own MFMA utilisation: its flops over the
    kernel's time, against the bf16 peak."""
    H, N, d = wl.batch * wl.n_kv_heads, wl.ctx_len, wl.head_dim
    per_budget = {}
    for L in budgets:
        by = compress_bytes(H, N, d, min(L, N))
        ms = ms_per_layer[str(L)]
        per_budget[str(L)] = {"bytes": by, "ms": ms, "GBps": by / (ms * 1e-3) / 1e9,
                              "frac": by / (ms * 1e-3) / 1e9 / HBM_PEAK_GBS}
    avg_by = sum(v["bytes"] for v in per_budget.values()) / len(per_budget)
    avg_ms = sum(v["ms"] for v in per_budget.values()) / len(per_budget)
    res = {"kernel": "momentkv_compress call (one layer)", "bound": "hbm",
           "achieved": avg_by / (avg_ms * 1e-3) / 1e9, "peak": HBM_PEAK_GBS, "unit": "GB/s",
           "frac": avg_by / (avg_ms * 1e-3) / 1e9 / HBM_PEAK_GBS, "bytes_per_layer": avg_by,
           "ms_per_layer": avg_ms, "per_budget": per_budget, "traffic": None, "kernels": None,
           "covariance_mfma": None}
    prof = _profile_json(os.path.join(ROOT, "profiles", f"compress_{wl.name}.md"),
                         "compress_sources_sha256")
    if prof is None:
        return res
    work = compress_kernel_work(H, wl.group, wl.window, N, d, wl.n_sink)
    kernels = {}
    for name, k in prof["kernels"].items():
        short = name.split("<")[0].split("::")[-1]
        ent = {"avg_us": k["avg_us"], "mfma_busy_pct": k.get("mfma_busy_pct")}
        if short in work:
            wk = work[short]
            t = k["avg_us"] * 1e-6
            ent.update({"bytes": wk["bytes"], "GBps": wk["bytes"] / t / 1e9,
                        "frac_hbm": wk["bytes"] / t / 1e9 / HBM_PEAK_GBS,
                        "mfma_TFLOPs": wk["flops"] / t / 1e12,
                        "frac_mfma_bf16": wk["flops"] / t / 1e12 / MFMA_BF16_PEAK_TFLOPS})
        kernels[name] = ent
    res["kernels"] = kernels
    ratio = prof.get("traffic_over_algorithmic")
    res["traffic"] = None if ratio is None else ratio * avg_by
    rc = [(n, k) for n, k in prof["kernels"].items() if "k_rows_cov" in n]
    if rc:
        name, k = rc[0]
        t = k["avg_us"] * 1e-6
        cov = work["k_rows_cov"]["covariance_flops"]
        share = cov / work["k_rows_cov"]["flops"]
        res["covariance_mfma"] = {
            "what": "V_C^T K_C on v_mfma_f32_16x16x32_bf16 inside k_rows_cov (which also runs "
                    "the window logits on the same instruction)",
            "flops_per_layer": cov, "kernel": name, "kernel_us": k["avg_us"],
            "achieved_TFLOPs": cov / t / 1e12,
            "util_of_bf16_peak": cov / t / 1e12 / MFMA_BF16_PEAK_TFLOPS,
            "kernel_mfma_busy_pct": k.get("mfma_busy_pct"),
            "covariance_share_of_kernel_mfma": share,
            "covariance_mfma_busy_pct": None if k.get("mfma_busy_pct") is None
            else k["mfma_busy_pct"] * share}
    return res


def measured_traffic(workload: str, alg_per_call: dict) -> float | None:
    """HBM bytes per decode call from the committed rocprofv3 FETCH_SIZE / WRITE_SIZE summary
    (profiles/traffic_decode_<workload>.md): its measured traffic / algorithmic ratio per
    budget applied to this run's algorithmic bytes per call, averaged over the budgets.
    None when there is no summary for the workload or budgets, or when the decode sources
    differ from the ones the counters were taken with."""
    import hashlib
    import re
    path = os.path.join(ROOT, "profiles", f"traffic_decode_{workload}.md")
    if not os.path.exists(path):
        return None
    m = re.search(r"```json\n(\{.*?\})\n```", open(path).read(), re.S)
    if not m:
        return None
    data = json.loads(m.group(1))
    h = hashlib.sha256()
    for src in data["sources"]:
        with open(os.path.join(ROOT, src), "rb") as f:
            h.update(f.read())
    ratios = data["traffic_over_algorithmic"]
    if h.hexdigest() != data["decode_sources_sha256"] or any(str(L) not in ratios for L in alg_per_call):
        return None
    return sum(ratios[str(L)] * b for L, b in alg_per_call.items()) / len(alg_per_call)


def build_stack(wl, layers, device):
    t0 = time.time()
    data = [synth.make_layer(wl, l, device=device) for l in range(layers)]
    torch.cuda.synchronize()
    return data, time.time() - t0


def percentiles(xs) -> dict:
    """p10 / p50 / p90 (linear interpolation) and the sample count of a list of times."""
    import numpy as np
    q = np.percentile(np.asarray(xs, dtype=np.float64), [10, 50, 90])
    return {"p10": float(q[0]), "p50": float(q[1]), "p90": float(q[2]), "n": len(xs)}


def cpu_baseline(wl, layers_data, budgets, steps: int) -> dict:
    """The fp64 oracle on the host over a bounded sample of the same workload: every KV head
    of the given layers, at every budget, compressed, then `steps` decode steps with appends
    of each (layer, budget) cache, the sequence the GPU decode phase runs.  `value` is the
    decode phase's algorithmic bytes over its host time (GB/s like the GPU's `value`);
    compress is reported in ms per layer, measured on whole layers."""
    import numpy as np
    import oracle as O
    try:
        from threadpoolctl import threadpool_info
        blas_threads = max((i.get("num_threads", 1) for i in threadpool_info()), default=1)
    except Exception:  # noqa: BLE001
        blas_threads = 1
    f64 = lambda t: t.float().cpu().double().numpy()  # noqa: E731
    d, G, Hkv, N = wl.head_dim, wl.group, wl.n_kv_heads, wl.ctx_len
    t_comp = t_dec = 0.0
    nbytes = 0
    for data in layers_data:
        q = f64(data["q_win"])[0]
        K = f64(data["k"])[0]
        V = f64(data["v"])[0]
        qd = f64(data["q_dec"][:steps])[:, 0]
        kn = f64(data["k_new"][:steps])[:, 0]
        vn = f64(data["v_new"][:steps])[:, 0]
        for L in budgets:
            t0 = time.perf_counter()
            comp = [O.compress_head(q[h * G:(h + 1) * G], K[h], V[h], L) for h in range(Hkv)]
            t_comp += time.perf_counter() - t0
            n0 = min(L, N)
            cap = n0 + steps
            kcap = np.zeros((1, Hkv, cap, d))
            vcap = np.zeros((1, Hkv, cap, d))
            kcap[0, :, :n0] = np.stack([c.k_out for c in comp])
            vcap[0, :, :n0] = np.stack([c.v_out for c in comp])
            ln = np.full((1, Hkv), n0)
            moms = [[c.moments for c in comp]]
            t0 = time.perf_counter()
            for t in range(steps):
                _, _, _, (kcap, vcap, ln) = O.decode(qd[t][None], kcap, vcap, ln, moms,
                                                     k_new=kn[t][None], v_new=vn[t][None])
            t_dec += time.perf_counter() - t0
            nbytes += sum(decode_bytes(Hkv, G, d, n0 + t + 1) for t in range(steps))
    n_lay = len(layers_data)
    return {"value": nbytes / t_dec / 1e9, "unit": "GB/s", "cores": int(blas_threads),
            "host_cpus": len(os.sched_getaffinity(0)), "kind": "oracle",
            "sample": f"layers 0-{n_lay - 1} of {wl.layers} (sequence 0 of {wl.batch}), all {Hkv} "
                      f"KV heads, budgets "
                      f"{list(budgets)}: compress each (layer, budget), then {steps} decode "
                      f"steps with appends (fp64 NumPy)",
            "compress_ms_per_layer": t_comp / (n_lay * len(budgets)) * 1e3,
            "decode_s": t_dec, "compress_s": t_comp}


def half_summary_measurement(args, wl, budgets, stacks, q_steps, kn_steps, vn_steps, out, dws,
                             compress_phase, capture, timed_replay) -> dict:
    """The decode phase again with the summary in half precision (one bf16 plane of the
    centred covariance, momentkv_prepare_summary(half=True), summary = 2): the moments'
    storage precision of the paper's App. C.2.  Same graph replay and per-budget
    subtraction as the headline decode; bytes count the summary at 2 bytes per entry."""
    N, Hkv, d = wl.ctx_len, wl.n_kv_heads, wl.head_dim
    G = wl.group
    T, LB = q_steps.shape[0], q_steps.shape[1]
    compress_phase(None)
    torch.cuda.synchronize()
    # the summaries do not change while decoding, and every compress rewrites them bit for bit
    halfs = {L: mk.momentkv_prepare_summary(stacks[L].n_e, stacks[L].s_k, stacks[L].s_v,
                                            stacks[L].S, dtype=wl.dtype, half=True)
             for L in budgets}

    def call(t, L):
        st = stacks[L]
        mk.momentkv_decode_attn(q_steps[t], st.k_out, st.v_out, st.lens, st.n_e, st.s_k, st.s_v,
                                halfs[L], k_new=kn_steps[t], v_new=vn_steps[t],
                                max_len=min(L, N) + T, out=out, workspace=dws[L], summary=2)

    def phase(skip=None):
        for t in range(T):
            for L in budgets:
                if L != skip:
                    call(t, L)

    print("[bench] decode with the half-precision summary: capture", file=sys.stderr, flush=True)
    graph = capture(phase=phase)
    without = {L: capture(skip=L, phase=phase) for L in budgets}
    ev = []
    for _ in range(args.steps):
        compress_phase(None)
        ev.append(timed_replay(graph))
    torch.cuda.synchronize()
    if any(int(dws[L][:4].view(torch.int32)[0]) for L in budgets):
        return {"error": "append overflow in the half-precision summary phase"}
    total = sum(a.elapsed_time(b) for a, b in ev) / len(ev)
    per_budget = {}
    all_bytes = 0
    for L in budgets:
        tl = []
        for _ in range(args.steps):
            compress_phase(None)
            tl.append(timed_replay(without[L]))
        torch.cuda.synchronize()
        budget_ms = total - sum(a.elapsed_time(b) for a, b in tl) / len(tl)
        by = sum(decode_bytes(LB * Hkv, G, d, min(L, N) + t + 1) - LB * Hkv * 2 * d * d
                 for t in range(T))
        all_bytes += by
        per_budget[str(L)] = {"us_per_call": budget_ms / T * 1e3,
                              "GBps": by / (budget_ms * 1e-3) / 1e9,
                              "tokens_per_s": wl.batch * T / (budget_ms * 1e-3)}
    return {"what": "the decode phase with momentkv_prepare_summary(half=True) (summary = 2)",
            "ms_per_step": total, "tokens_per_s": wl.batch * T * len(budgets) / (total * 1e-3),
            "GBps": all_bytes / (total * 1e-3) / 1e9, "per_budget": per_budget}


def adaptive_measurement(args, wl, data, layers, L, dev) -> dict:
    """Compress of every layer with head-adaptive budgets at budget L (the layer's
    candidate budget split over its heads by pooled mass): ms per layer from HIP events
    around the layers' calls, and the spread of the per-head retained lengths."""
    N, Hkv, d, w = wl.ctx_len, wl.n_kv_heads, wl.head_dim, wl.window
    cap = mk.compress_rows(N, Hkv, L, w, adaptive=True)
    B = wl.batch
    f32 = dict(dtype=torch.float32, device=dev)
    i32 = dict(dtype=torch.int32, device=dev)
    outs = [mk.CompressOutput(
        k_out=torch.empty(B, Hkv, cap, d, dtype=wl.dtype, device=dev),
        v_out=torch.empty(B, Hkv, cap, d, dtype=wl.dtype, device=dev),
        idx=torch.empty(B, Hkv, cap, **i32), lens=torch.empty(B, Hkv, **i32),
        n_e=torch.empty(B, Hkv, **i32), s_k=torch.empty(B, Hkv, d, **f32),
        s_v=torch.empty(B, Hkv, d, **f32), S=torch.empty(B, Hkv, d, d, **f32))
        for _ in range(layers)]
    ws = torch.empty(mk.momentkv_compress_workspace_bytes(
        mk.compress_params(data[0]["q_win"], data[0]["k"], L, cap=cap, adaptive=True)),
        dtype=torch.uint8, device=dev)

    def run():
        for l in range(layers):
            x = data[l]
            mk.momentkv_compress(x["q_win"], x["k"], x["v"], L, cap=cap, adaptive=True,
                                 out=outs[l], workspace=ws)

    run()
    torch.cuda.synchronize()
    ev = []
    for _ in range(args.steps):
        e0 = torch.cuda.Event(enable_timing=True)
        e1 = torch.cuda.Event(enable_timing=True)
        e0.record()
        run()
        e1.record()
        ev.append((e0, e1))
    torch.cuda.synchronize()
    ms = sum(a.elapsed_time(b) for a, b in ev) / len(ev) / layers
    lens = torch.stack([o.lens for o in outs]).float()
    return {"what": f"momentkv_compress(adaptive=True) of each layer at budget {L}",
            "budget": L, "compress_ms_per_layer": ms,
            "retained_rows_per_head": {"min": int(lens.min()), "mean": float(lens.mean()),
                                       "max": int(lens.max())}}


def evict_bytes(n_heads: int, G: int, d: int, L: int, elem: int = 2) -> int:
    """Algorithmic HBM bytes of one decode call with eviction at budget L (per KV head,
    summed): the decode bytes over the L + 1 rows seen by Phase 1 (retained rows read once,
    the new row read and written, the summary, queries and outputs), plus the summary
    written back by the rank-one update (S, s_k, s_v, n_e) and the row moved into the
    freed slot (read and written)."""
    per_head = 4 * d * d + 8 * d + 4 + 2 * 2 * d * elem
    return decode_bytes(n_heads, G, d, L + 1) + n_heads * per_head


def evict_measurement(args, wl, budgets, stacks, q_steps, kn_steps, vn_steps, out,
                      compress_phase, capture, timed_replay) -> dict:
    """Decode with moment-informed eviction (Algorithm 1 Phase 1 then Phase 2) on the same
    compressed stacks: for each of the decode tokens and each budget one
    momentkv_decode_evict call over the 36 caches (cache held at the budget, summary
    updated by each eviction).  Captured as a graph like the decode phase; per-budget
    times by subtraction."""
    dev = out.device
    N, Hkv, d = wl.ctx_len, wl.n_kv_heads, wl.head_dim
    G = wl.group
    T = q_steps.shape[0]
    LB = q_steps.shape[1]
    ews = {}
    for L in budgets:
        Lr = min(L, N)
        p = mk.decode_params(q_steps[0], stacks[L].k_out, max_len=Lr + 1)
        ews[L] = torch.zeros(mk.momentkv_decode_evict_workspace_bytes(p), dtype=torch.uint8,
                             device=dev)

    def evict_call(t, L):
        st = stacks[L]
        Lr = min(L, N)
        mk.momentkv_decode_evict(q_steps[t], st.k_out, st.v_out, st.lens, st.n_e, st.s_k,
                                 st.s_v, st.S, kn_steps[t], vn_steps[t], Lr, max_len=Lr + 1,
                                 out=out, workspace=ews[L])

    def evict_phase(skip=None):
        for t in range(T):
            for L in budgets:
                if L != skip:
                    evict_call(t, L)

    print("[bench] decode with eviction: warm-up and capture", file=sys.stderr, flush=True)
    compress_phase(None)
    evict_phase()
    torch.cuda.synchronize()
    graph = capture(phase=evict_phase)
    without = {L: capture(skip=L, phase=evict_phase) for L in budgets}
    ev = []
    for i in range(args.steps):
        compress_phase(None)
        ev.append(timed_replay(graph))
    torch.cuda.synchronize()
    flags = [int(ews[L][:4].view(torch.int32)[0]) for L in budgets]
    if any(flags):
        return {"error": f"eviction flags {flags}"}
    # replay against the eager phase, bit for bit (output, lengths, counts, summary, cache)
    compress_phase(None)
    graph.replay()
    torch.cuda.synchronize()
    got = [out.clone()] + [x.clone() for L in budgets for x in
                           (stacks[L].lens, stacks[L].n_e, stacks[L].S, stacks[L].k_out)]
    compress_phase(None)
    evict_phase()
    torch.cuda.synchronize()
    now = [out] + [x for L in budgets for x in
                   (stacks[L].lens, stacks[L].n_e, stacks[L].S, stacks[L].k_out)]
    if not all(torch.equal(a, b) for a, b in zip(got, now)):
        return {"error": "eviction graph replay differs from the eager phase"}
    del got
    ms = [a.elapsed_time(b) for a, b in ev]
    total = sum(ms) / len(ms)
    per_budget = {}
    all_bytes = 0
    for L in budgets:
        tl = []
        for _ in range(args.steps):
            compress_phase(None)
            tl.append(timed_replay(without[L]))
        torch.cuda.synchronize()
        budget_ms = total - sum(a.elapsed_time(b) for a, b in tl) / len(tl)
        by = evict_bytes(LB * Hkv, G, d, min(L, N)) * T
        all_bytes += by
        per_budget[str(L)] = {"us_per_call": budget_ms / T * 1e3,
                              "GBps": by / (budget_ms * 1e-3) / 1e9,
                              "tokens_per_s": wl.batch * T / (budget_ms * 1e-3)}
    achieved = all_bytes / (total * 1e-3) / 1e9
    # measured HBM traffic per call: the committed FETCH_SIZE / WRITE_SIZE summary's ratio
    # per budget applied to this run's algorithmic bytes (None once the sources differ)
    prof = _profile_json(os.path.join(ROOT, "profiles", f"traffic_evict_{wl.name}.md"),
                         "evict_sources_sha256")
    traffic = None
    if prof is not None and all(str(L) in prof["traffic_over_algorithmic"] for L in budgets):
        traffic = sum(prof["traffic_over_algorithmic"][str(L)] * evict_bytes(LB * Hkv, G, d, min(L, N))
                      for L in budgets) / len(budgets)
    return {"what": "per token and budget one momentkv_decode_evict call over the 36 "
                    "caches: append, Phase 1 eviction, Phase 2 corrected attention; cache "
                    "kept at the budget.  Caches under 320 rows: one k_evict_attn launch that "
                    "scores, selects, updates and attends to the new cache; above: "
                    "k_evict_attn scoring and attention in one read of the cache, then "
                    "k_evict_finish",
            "ms_per_step": total, "tokens_per_s": wl.batch * T * len(budgets) / (total * 1e-3),
            "per_budget": per_budget,
            "roofline": {"kernel": "momentkv_decode_evict call (1-2 launches)", "bound": "hbm",
                         "achieved": achieved, "peak": HBM_PEAK_GBS, "unit": "GB/s",
                         "frac": achieved / HBM_PEAK_GBS, "traffic": traffic,
                         "bytes_per_call": all_bytes / (T * len(budgets)),
                         "avg_call_us": total / (T * len(budgets)) * 1e3}}


def stacked_measurement(args, wl, data, layers, budgets, dev) -> dict:
    """momentkv_compress once per budget over the whole stack (batch = layers x sequences,
    every layer's KV heads in one call): the same per-head work as the per-layer calls, with
    the fixed cost of each launch shared by the stack's heads.  ms per layer = HIP-event time
    of the call over the layers; the inputs are the per-layer tensors concatenated (outside
    the timing)."""
    N, Hkv, d, w = wl.ctx_len, wl.n_kv_heads, wl.head_dim, wl.window
    q = torch.cat([x["q_win"] for x in data]).contiguous()
    k = torch.cat([x["k"] for x in data]).contiguous()
    v = torch.cat([x["v"] for x in data]).contiguous()
    res = {}
    for L in budgets:
        cap = min(L, N)
        p = mk.compress_params(q, k, L, cap=cap)
        ws = torch.empty(mk.momentkv_compress_workspace_bytes(p), dtype=torch.uint8, device=dev)
        out = mk.momentkv_compress(q, k, v, L, cap=cap, workspace=ws)  # warm-up, allocates out
        torch.cuda.synchronize()
        ev = []
        for _ in range(args.steps):
            e0 = torch.cuda.Event(enable_timing=True)
            e1 = torch.cuda.Event(enable_timing=True)
            e0.record()
            mk.momentkv_compress(q, k, v, L, cap=cap, out=out, workspace=ws)
            e1.record()
            ev.append((e0, e1))
        torch.cuda.synchronize()
        ms = sum(a.elapsed_time(b) for a, b in ev) / len(ev)
        by = compress_bytes(Hkv * wl.batch, N, d, cap)
        res[str(L)] = {"ms_per_layer": ms / layers, "GBps": by / (ms / layers * 1e-3) / 1e9,
                       "ms_per_call": ms}
        del out, ws
    del q, k, v
    return {"what": f"one momentkv_compress call per budget over all {layers} layers "
                    f"(batch {layers * wl.batch}); the per-layer calls are the headline",
            "per_budget": res,
            "ms_per_layer": sum(x["ms_per_layer"] for x in res.values()) / len(res)}


def main() -> int:
    ap = argparse.ArgumentParser(description=__doc__.split("\n")[0])
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=5)
    ap.add_argument("--warmup", type=int, default=2)
    ap.add_argument("--workload", default="qwen3_4b_stack_n32768", choices=sorted(synth.WORKLOADS))
    ap.add_argument("--layers", type=int, default=None)
    ap.add_argument("--budgets", default=None, help="comma list overriding the workload's")
    ap.add_argument("--decode-steps", type=int, default=None)
    ap.add_argument("--cpu-layers", type=int, default=2,
                    help="layers in the oracle's host sample (all heads, budgets and steps)")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-evict", action="store_true",
                    help="skip the decode-with-eviction measurement")
    ap.add_argument("--no-half", action="store_true",
                    help="skip the half-precision summary measurement")
    ap.add_argument("--no-adaptive", action="store_true",
                    help="skip the head-adaptive compress measurement")
    ap.add_argument("--no-stacked", action="store_true",
                    help="skip the one-call-per-stack compress measurement")
    ap.add_argument("--compress-probe", action="store_true",
                    help="for rocprofv3 runs: one plain copy of known size, then one compress "
                         "of every layer per budget (eager); prints the plan as JSON and exits")
    ap.add_argument("--evict-probe", action="store_true",
                    help="for rocprofv3 runs: one plain copy of known size, then 4 tokens x "
                         "budgets of eager decode calls with eviction; prints the plan as JSON "
                         "and exits")
    ap.add_argument("--traffic-probe", action="store_true",
                    help="for rocprofv3 --pmc FETCH_SIZE / WRITE_SIZE runs: one plain copy of "
                         "known size, then 4 tokens x budgets of eager decode calls; prints "
                         "the dispatch plan as JSON and exits")
    args = ap.parse_args()
    world = int(os.environ.get("WORLD_SIZE", "1"))
    if args.gpus != 1 or world != 1:
        print("bench.py measures one GPU: the MomentKV hot path shards over (sequence, KV head) "
              "with no exchange, and this build runs on a single MI355X; use --gpus 1.",
              file=sys.stderr)
        return 2
    if not torch.cuda.is_available():
        print("bench.py needs a GPU", file=sys.stderr)
        return 2
    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    wl = synth.WORKLOADS[args.workload]
    layers = args.layers or wl.layers
    budgets = tuple(int(x) for x in args.budgets.split(",")) if args.budgets else wl.budgets
    T = args.decode_steps if args.decode_steps is not None else wl.decode_steps
    wl = synth.shrink(wl, decode_steps=T)
    B, Hq, Hkv, d, N, w = wl.batch, wl.n_q_heads, wl.n_kv_heads, wl.head_dim, wl.ctx_len, wl.window
    G = wl.group
    print(f"[bench] generating {layers} layers of {wl.name} on {torch.cuda.get_device_name(0)}",
          file=sys.stderr, flush=True)
    data, gen_s = build_stack(wl, layers, dev)
    print(f"[bench] inputs ready in {gen_s:.1f}s", file=sys.stderr, flush=True)

    # decode inputs stacked over layers: [T, layers*B, ...]
    q_steps = torch.stack([x["q_dec"] for x in data], dim=1).reshape(T, layers * B, Hq, d).contiguous()
    kn_steps = torch.stack([x["k_new"] for x in data], dim=1).reshape(T, layers * B, Hkv, d).contiguous()
    vn_steps = torch.stack([x["v_new"] for x in data], dim=1).reshape(T, layers * B, Hkv, d).contiguous()

    LB = layers * B
    f32 = dict(dtype=torch.float32, device=dev)
    i32 = dict(dtype=torch.int32, device=dev)
    stacks = {}
    for L in budgets:
        cap = min(L, N) + T
        stacks[L] = mk.CompressOutput(
            k_out=torch.empty(LB, Hkv, cap, d, dtype=wl.dtype, device=dev),
            v_out=torch.empty(LB, Hkv, cap, d, dtype=wl.dtype, device=dev),
            idx=torch.empty(LB, Hkv, min(L, N), **i32), lens=torch.empty(LB, Hkv, **i32),
            n_e=torch.empty(LB, Hkv, **i32), s_k=torch.empty(LB, Hkv, d, **f32),
            s_v=torch.empty(LB, Hkv, d, **f32), S=torch.empty(LB, Hkv, d, d, **f32))
    cws_bytes = max(mk.momentkv_compress_workspace_bytes(
        mk.compress_params(data[0]["q_win"], data[0]["k"], L, cap=min(L, N) + T)) for L in budgets)
    cws = torch.empty(cws_bytes, dtype=torch.uint8, device=dev)
    dws = {}
    out = torch.empty(LB, Hq, d, dtype=wl.dtype, device=dev)
    for L in budgets:
        p = mk.decode_params(q_steps[0], stacks[L].k_out, max_len=min(L, N) + T)
        dws[L] = torch.zeros(mk.momentkv_decode_workspace_bytes(p), dtype=torch.uint8, device=dev)

    def layer_view(st, l):
        sl = slice(l * B, (l + 1) * B)
        return mk.CompressOutput(st.k_out[sl], st.v_out[sl], st.idx[sl], st.lens[sl], st.n_e[sl],
                                 st.s_k[sl], st.s_v[sl], st.S[sl])

    views = {L: [layer_view(stacks[L], l) for l in range(layers)] for L in budgets}
    pshape = (LB, Hkv, 2, d, d) if wl.dtype == torch.bfloat16 else (LB, Hkv, d, d)
    prepared = {L: torch.empty(pshape, dtype=wl.dtype, device=dev) for L in budgets}

    def compress_phase(timing):
        for L in budgets:
            e0 = torch.cuda.Event(enable_timing=True)
            e1 = torch.cuda.Event(enable_timing=True)
            e0.record()
            marks = []
            for l in range(layers):
                if timing is not None and l > 0:   # per-call spread: an event between calls
                    marks.append(torch.cuda.Event(enable_timing=True))
                    marks[-1].record()
                x = data[l]
                mk.momentkv_compress(x["q_win"], x["k"], x["v"], L, cap=min(L, N) + T,
                                     out=views[L][l], workspace=cws)
            if timing is not None:
                marks.append(torch.cuda.Event(enable_timing=True))
                marks[-1].record()
                timing["calls"][L].append([e0] + marks)
            st = stacks[L]   # the decode form of the 36 summaries, once per compression
            mk.momentkv_prepare_summary(st.n_e, st.s_k, st.s_v, st.S, dtype=wl.dtype,
                                        out=prepared[L])
            e1.record()
            if timing is not None:
                timing["compress"][L].append((e0, e1))

    def compress_budget(L):
        """One budget's compress of every layer and the summaries' decode form (no events)."""
        for l in range(layers):
            x = data[l]
            mk.momentkv_compress(x["q_win"], x["k"], x["v"], L, cap=min(L, N) + T,
                                 out=views[L][l], workspace=cws)
        st = stacks[L]
        mk.momentkv_prepare_summary(st.n_e, st.s_k, st.s_v, st.S, dtype=wl.dtype,
                                    out=prepared[L])

    def capture_fn(fn):
        """fn captured as a HIP graph (run once eagerly first on the capture stream)."""
        g = torch.cuda.CUDAGraph()
        cs = torch.cuda.Stream()
        cs.wait_stream(torch.cuda.current_stream())
        with torch.cuda.stream(cs):
            fn()
            torch.cuda.synchronize()
            with torch.cuda.graph(g, stream=cs):
                fn()
        torch.cuda.current_stream().wait_stream(cs)
        torch.cuda.synchronize()
        return g

    def compress_replay(cgraphs, timing):
        """The compress phase as graph replays, one per budget, timed by HIP events."""
        for L in budgets:
            e0 = torch.cuda.Event(enable_timing=True)
            e1 = torch.cuda.Event(enable_timing=True)
            e0.record()
            cgraphs[L].replay()
            e1.record()
            timing["compress"][L].append((e0, e1))

    def decode_call(t, L):
        st = stacks[L]
        mk.momentkv_decode_attn(q_steps[t], st.k_out, st.v_out, st.lens, st.n_e, st.s_k,
                                st.s_v, prepared[L], k_new=kn_steps[t], v_new=vn_steps[t],
                                max_len=min(L, N) + T, out=out, workspace=dws[L], summary=1)

    def decode_phase(skip=None):
        for t in range(T):
            for L in budgets:
                if L != skip:
                    decode_call(t, L)

    def new_timing():
        return {"compress": {L: [] for L in budgets}, "calls": {L: [] for L in budgets}}

    def capture(skip=None, phase=None):
        g = torch.cuda.CUDAGraph()
        cap_stream = torch.cuda.Stream()
        cap_stream.wait_stream(torch.cuda.current_stream())
        with torch.cuda.stream(cap_stream):
            compress_phase(None)
            torch.cuda.synchronize()
            with torch.cuda.graph(g, stream=cap_stream):
                (phase or decode_phase)(skip)
        torch.cuda.current_stream().wait_stream(cap_stream)
        torch.cuda.synchronize()
        return g

    def timed_replay(g):
        d0 = torch.cuda.Event(enable_timing=True)
        d1 = torch.cuda.Event(enable_timing=True)
        d0.record()
        g.replay()
        d1.record()
        return d0, d1

    if args.compress_probe:
        copy_bytes = 256 << 20
        src = torch.empty(copy_bytes, dtype=torch.uint8, device=dev)
        dst = torch.empty_like(src)
        dst.copy_(src)                 # calibration: copy_bytes read, copy_bytes written
        torch.cuda.synchronize()
        compress_phase(None)
        torch.cuda.synchronize()
        print(json.dumps({"copy_bytes": copy_bytes, "budgets": list(budgets), "layers": layers,
                          "bytes_per_call": {str(L): compress_bytes(Hkv * B, N, d, min(L, N))
                                             for L in budgets},
                          "work": compress_kernel_work(Hkv * B, G, w, N, d, wl.n_sink)}))
        return 0

    if args.evict_probe:
        compress_phase(None)
        torch.cuda.synchronize()
        copy_bytes = 256 << 20
        src = torch.empty(copy_bytes, dtype=torch.uint8, device=dev)
        dst = torch.empty_like(src)
        dst.copy_(src)                 # calibration: copy_bytes read, copy_bytes written
        ews = {}
        for L in budgets:
            p = mk.decode_params(q_steps[0], stacks[L].k_out, max_len=min(L, N) + 1)
            ews[L] = torch.zeros(mk.momentkv_decode_evict_workspace_bytes(p), dtype=torch.uint8,
                                 device=dev)
        calls = []
        for t in range(4):
            for L in budgets:
                st = stacks[L]
                Lr = min(L, N)
                mk.momentkv_decode_evict(q_steps[t], st.k_out, st.v_out, st.lens, st.n_e,
                                         st.s_k, st.s_v, st.S, kn_steps[t], vn_steps[t], Lr,
                                         max_len=Lr + 1, out=out, workspace=ews[L])
                calls.append({"token": t, "budget": L, "fused": Lr + 1 >= EVICT_ONE_READ_MIN_LEN,
                              "bytes": evict_bytes(LB * Hkv, G, d, Lr)})
        torch.cuda.synchronize()
        print(json.dumps({"copy_bytes": copy_bytes, "calls": calls}))
        return 0

    if args.traffic_probe:
        compress_phase(None)
        torch.cuda.synchronize()
        copy_bytes = 256 << 20
        src = torch.empty(copy_bytes, dtype=torch.uint8, device=dev)
        dst = torch.empty_like(src)
        dst.copy_(src)                 # calibration: copy_bytes read, copy_bytes written
        calls = []
        for t in range(4):
            for L in budgets:
                decode_call(t, L)
                n = min(L, N) + t + 1
                calls.append({"token": t, "budget": L, "lens_after": n,
                              "fused": min(L, N) + T <= 384,
                              "bytes": decode_bytes(LB * Hkv, G, d, n)})
        torch.cuda.synchronize()
        print(json.dumps({"copy_bytes": copy_bytes, "calls": calls}))
        return 0

    # warm-up, eagerly
    for _ in range(args.warmup):
        compress_phase(None)
        decode_phase()
    torch.cuda.synchronize()
    # capture the decode phase (the library allocates nothing and records no memset), and
    # the phase without each budget in turn: a budget's decode time is the difference
    graph = capture()
    graph_without = {L: capture(skip=L) for L in budgets}
    # the compress phase as graphs too (per budget: the layers' calls and the summaries'
    # decode form), checked bit for bit against the eager phase
    cgraphs = {L: capture_fn(lambda L=L: compress_budget(L)) for L in budgets}
    compress_phase(None)
    torch.cuda.synchronize()
    eager = [(stacks[L].idx.clone(), stacks[L].S.clone(), prepared[L].clone()) for L in budgets]
    for L in budgets:
        stacks[L].S.zero_()
        cgraphs[L].replay()
    torch.cuda.synchronize()
    if not all(torch.equal(i, stacks[L].idx) and torch.equal(S, stacks[L].S) and
               torch.equal(pr, prepared[L]) for (i, S, pr), L in zip(eager, budgets)):
        print("[bench] compress graph replay differs from the eager compress", file=sys.stderr)
        return 7
    del eager

    timing = new_timing()
    dec_events = []
    s0 = torch.cuda.Event(enable_timing=True)
    s1 = torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    wall0 = time.perf_counter()
    s0.record()
    for i in range(args.steps):
        compress_replay(cgraphs, timing)
        dec_events.append(timed_replay(graph))
        print(f"[bench] step {i + 1}/{args.steps} enqueued", file=sys.stderr, flush=True)
    s1.record()
    torch.cuda.synchronize()
    wall = time.perf_counter() - wall0
    total_ms = s0.elapsed_time(s1)
    flags = [int(dws[L][:4].view(torch.int32)[0]) for L in budgets]
    if any(flags):
        print(f"[bench] append overflow flags {flags}", file=sys.stderr)
        return 3

    # the replayed graph against the same phase run eagerly, bit for bit
    compress_phase(None)
    graph.replay()
    torch.cuda.synchronize()
    got = (out.clone(), [stacks[L].lens.clone() for L in budgets],
           [stacks[L].k_out.clone() for L in budgets])
    compress_phase(None)
    decode_phase()
    torch.cuda.synchronize()
    same = torch.equal(got[0], out) and all(
        torch.equal(a, stacks[L].lens) and torch.equal(k, stacks[L].k_out)
        for a, k, L in zip(got[1], got[2], budgets))
    del got
    if not same:
        print("[bench] graph replay differs from the eager decode phase", file=sys.stderr)
        return 4
    without_ms = {}
    for L in budgets:
        ev = []
        for _ in range(args.steps):
            compress_phase(None)
            ev.append(timed_replay(graph_without[L]))
        torch.cuda.synchronize()
        without_ms[L] = sum(a.elapsed_time(b) for a, b in ev) / len(ev)
    # per-call spread of the compress: eager calls with an event between consecutive calls
    spread_timing = new_timing()
    for _ in range(args.steps):
        compress_phase(spread_timing)
    torch.cuda.synchronize()

    per_budget = {}
    alg_per_call = {}
    phase_bytes = 0.0
    dec_ms = [a.elapsed_time(b) for a, b in dec_events]      # one graph replay per step
    dec_s = sum(dec_ms) * 1e-3
    for L in budgets:
        cms = [a.elapsed_time(b) for a, b in timing["compress"][L]]
        dby = sum(decode_bytes(LB * Hkv, G, d, min(L, N) + t + 1) for t in range(T))
        phase_bytes += dby
        alg_per_call[L] = dby / T
        budget_ms = sum(dec_ms) / len(dec_ms) - without_ms[L]
        per_budget[str(L)] = {
            "compress_ms_per_layer": sum(cms) / len(cms) / layers,
            "compress_GBps": compress_bytes(Hkv * B, N, d, min(L, N)) / (sum(cms) / len(cms) / layers * 1e-3) / 1e9,
            "decode_us_per_call": budget_ms / T * 1e3,
            "decode_GBps": dby / (budget_ms * 1e-3) / 1e9,
            "decode_tokens_per_s": B * T / (budget_ms * 1e-3),
        }
    value = phase_bytes * len(dec_ms) / dec_s / 1e9
    spread = {"decode_step_ms": percentiles(dec_ms),
              "compress_call_ms": {str(L): percentiles(
                  [a.elapsed_time(b) for ev in spread_timing["calls"][L] for a, b in zip(ev, ev[1:])])
                  for L in budgets}}
    half = None
    if wl.dtype == torch.bfloat16 and not args.no_half:
        half = half_summary_measurement(args, wl, budgets, stacks, q_steps, kn_steps, vn_steps, out,
                                        dws, compress_phase, capture, timed_replay)
        if half.get("error"):
            print(f"[bench] {half['error']}", file=sys.stderr)
            return 6
    ada = None if args.no_adaptive else adaptive_measurement(args, wl, data, layers,
                                                              budgets[0], dev)
    stacked = None if args.no_stacked else stacked_measurement(args, wl, data, layers, budgets,
                                                               dev)
    evict = None if args.no_evict else evict_measurement(
        args, wl, budgets, stacks, q_steps, kn_steps, vn_steps, out, compress_phase, capture,
        timed_replay)
    if evict is not None and evict.get("error"):
        print(f"[bench] {evict['error']}", file=sys.stderr)
        return 5
    n_launch = T * len(budgets)
    avg_launch_s = dec_s / len(dec_ms) / n_launch
    avg_bytes = phase_bytes / n_launch
    res = {
        "metric": "decode attn+correction GB/s & tokens/s; compress ms/layer @32K ctx",
        "value": value,
        "unit": "GB/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": total_ms / args.steps,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16" if wl.dtype == torch.bfloat16 else "f32",
        "data": "synthetic",
        "config": {"workload": wl.name, "layers": layers, "batch": B, "ctx_len": N,
                   "budgets": list(budgets), "window": w, "decode_steps": T, "n_q_heads": Hq,
                   "n_kv_heads": Hkv, "head_dim": d},
        "decode_tokens_per_s": B * T * len(budgets) * len(dec_ms) / dec_s,
        "decode_ms_per_step": sum(dec_ms) / len(dec_ms),
        "compress_ms_per_layer": {k: v["compress_ms_per_layer"] for k, v in per_budget.items()},
        "per_budget": per_budget,
        "roofline": {"kernel": "momentkv_decode_attn call over the stack: one launch, "
                               "k_decode_fused (max_len <= 384) or k_decode_slice (the last "
                               "wave of each head merges it); time per call from the graph "
                               "replays",
                     "bound": "hbm", "achieved": avg_bytes / avg_launch_s / 1e9,
                     "peak": HBM_PEAK_GBS, "unit": "GB/s",
                     "frac": avg_bytes / avg_launch_s / 1e9 / HBM_PEAK_GBS,
                     "traffic": measured_traffic(wl.name, alg_per_call),
                     "bytes_per_launch": avg_bytes,
                     "avg_launch_us": avg_launch_s * 1e6},
        "compress_roofline": compress_roofline(
            wl, budgets, {k: v["compress_ms_per_layer"] for k, v in per_budget.items()}),
        "wall_s_timed": wall,
        "spread": spread,
    }
    if stacked is not None:
        res["compress_stacked"] = stacked
    if half is not None:
        res["decode_half_summary"] = half
    if ada is not None:
        res["compress_adaptive"] = ada
    if evict is not None:
        res["evict_decode"] = evict
    if not args.no_cpu_baseline:
        print("[bench] timing the oracle on the host", file=sys.stderr, flush=True)
        res["cpu_baseline"] = cpu_baseline(wl, data[:max(1, args.cpu_layers)], budgets, T)
    print(json.dumps(res))
    return 0


if __name__ == "__main__":
    sys.exit(main())
