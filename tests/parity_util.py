"""Helpers shared by the GPU parity tests: run the HIP path, run the oracle on the same
bits, and compare with the tolerances of the parity protocol.

Tolerances (relative L2 / Frobenius, per KV head or per query head):
  fp32 inputs: 1e-5;  bf16 inputs: 2e-2 (outputs are bf16; arithmetic is fp32).
Selection: the GPU's kept sets must equal the top-k of the GPU's own scores exactly
(ties: lower position), and differ from the oracle's only by swaps inside a near-tie
band around the k-th score (1e-5 relative for fp32, 1e-4 for bf16).
"""
from __future__ import annotations

import math

import numpy as np
import torch

import oracle as O
from paper_2606_01563_amd import momentkv as mk

TOL = {torch.float32: 1e-5, torch.bfloat16: 2e-2}
SEL_BAND = {torch.float32: 1e-5, torch.bfloat16: 1e-4}


def rel_l2(got, ref) -> float:
    got = np.asarray(got, np.float64)
    ref = np.asarray(ref, np.float64)
    den = np.linalg.norm(ref)
    return float(np.linalg.norm(got - ref) / (den if den > 0 else 1.0))


def h64(t: torch.Tensor) -> np.ndarray:
    return t.detach().float().cpu().double().numpy() if t.dtype == torch.bfloat16 \
        else t.detach().cpu().double().numpy()


def top_by_score(score: np.ndarray, k: int, offset: int) -> np.ndarray:
    """Kept positions (ascending) = top-k by (-score, position)."""
    return np.sort(O.select_top(score, k) + offset)


def check_selection_against_own_scores(score_gpu: np.ndarray, kept_gpu: np.ndarray, k: int,
                                       offset: int):
    expect = top_by_score(score_gpu, k, offset)
    np.testing.assert_array_equal(np.sort(kept_gpu), expect)


def check_set_near_ties(kept_gpu, score_ref, k, offset, band) -> int:
    """kept_gpu vs oracle top-k of score_ref: every swap must sit in the near-tie band.
    Returns the number of swapped positions."""
    ref = top_by_score(score_ref, k, offset)
    diff = np.setxor1d(np.asarray(kept_gpu), ref)
    if diff.size == 0:
        return 0
    kth = np.sort(score_ref)[::-1][k - 1]
    gaps = np.abs(score_ref[diff - offset] - kth)
    assert np.all(gaps <= band * max(kth, 1e-30)), (
        f"{diff.size} swaps, max gap {gaps.max():.3e} vs band {band * kth:.3e}")
    return int(diff.size)


def run_compress(inp: dict, budget: int, **kw) -> mk.CompressOutput:
    out = mk.momentkv_compress(inp["q_win"], inp["k"], inp["v"], budget, debug=True, **kw)
    torch.cuda.synchronize()
    return out


def check_compress_head(inp_cpu: dict, out: mk.CompressOutput, b: int, h: int, budget: int, *,
                        n_sink=1, chunk=4, mi_rounds=1, tau=1e-6, check_oracle_scores=True):
    """Full protocol for one (sequence, KV head).  Returns a dict of measured errors."""
    dt = inp_cpu["k"].dtype
    tol, band = TOL[dt], SEL_BAND[dt]
    q = h64(inp_cpu["q_win"][b:b + 1])   # one sequence, converted after slicing
    K = h64(inp_cpu["k"][b, h])
    V = h64(inp_cpu["v"][b, h])
    Hkv = inp_cpu["k"].shape[1]
    G = q.shape[1] // Hkv
    N, d = K.shape
    w = q.shape[2]
    scale = 1.0 / math.sqrt(d)
    n_out = min(budget, N)
    idx = out.idx[b, h, :n_out].cpu().numpy().astype(np.int64)
    errs = {}
    # retained rows are copies of the input rows (bit-exact)
    tidx = torch.from_numpy(idx)
    assert torch.equal(out.k_out[b, h, :n_out].cpu(), inp_cpu["k"][b, h][tidx])
    assert torch.equal(out.v_out[b, h, :n_out].cpu(), inp_cpu["v"][b, h][tidx])
    assert int(out.lens[b, h]) == n_out
    if budget >= N:
        np.testing.assert_array_equal(idx, np.arange(N))
        assert int(out.n_e[b, h]) == 0
        assert not out.S[b, h].any() and not out.s_k[b, h].any() and not out.s_v[b, h].any()
        return errs
    k_keep = budget - n_sink - w
    cand = np.arange(n_sink, N - w)
    kept = idx[n_sink: n_sink + k_keep]
    # structure: sinks + ascending kept candidates + window
    np.testing.assert_array_equal(idx[:n_sink], np.arange(n_sink))
    np.testing.assert_array_equal(idx[n_sink + k_keep:], np.arange(N - w, N))
    assert np.all(np.diff(idx) > 0)
    evicted = np.setdiff1d(cand, kept)
    assert int(out.n_e[b, h]) == len(evicted) == len(cand) - k_keep

    abar_g = out.abar[b, h].cpu().double().numpy()
    s0_g = out.score0[b, h].cpu().double().numpy()
    s1_g = out.score[b, h].cpu().double().numpy()
    kept0 = (out.kept0[b, h, :k_keep].cpu().numpy().astype(np.int64) if k_keep > 0
             else np.zeros(0, np.int64))
    # 1. selection logic is exact on the GPU's own scores
    if k_keep > 0:
        first = abar_g if mi_rounds < 0 else s0_g
        check_selection_against_own_scores(first, kept0 if mi_rounds >= 1 else kept, k_keep, n_sink)
        if mi_rounds >= 1:
            check_selection_against_own_scores(s1_g, kept, k_keep, n_sink)
    # 2. scores against the oracle (moment round fed the GPU's provisional set)
    ref = O.compress_head(q[0, h * G:(h + 1) * G], K, V, budget, n_sink=n_sink, chunk=chunk,
                          mi_rounds=mi_rounds, tau=tau,
                          r0_override=kept0 if (mi_rounds >= 1 and k_keep > 0) else None)
    if check_oracle_scores:
        errs["abar"] = rel_l2(abar_g, ref.abar)
        assert errs["abar"] <= tol, errs
        if mi_rounds >= 0:
            errs["score0"] = rel_l2(s0_g, ref.sigma0)
            assert errs["score0"] <= tol, errs
        if mi_rounds >= 1:
            errs["score"] = rel_l2(s1_g, ref.sigma)
            assert errs["score"] <= tol, errs
        # 3. sets equal the oracle's up to near-ties
        if k_keep > 0:
            if mi_rounds >= 1:
                ref_own = O.compress_head(q[0, h * G:(h + 1) * G], K, V, budget, n_sink=n_sink,
                                          chunk=chunk, mi_rounds=0, tau=tau)
                errs["swaps0"] = check_set_near_ties(kept0, ref_own.sigma0, k_keep, n_sink, band)
                errs["swaps"] = check_set_near_ties(kept, ref.sigma, k_keep, n_sink, band)
            else:
                first_ref = ref.abar if mi_rounds < 0 else ref.sigma0
                errs["swaps"] = check_set_near_ties(kept, first_ref, k_keep, n_sink, band)
    # 4./5. moments equal the oracle's sums over the GPU's evicted set
    m = O.evicted_moments(K, V, evicted)
    errs["S"] = rel_l2(out.S[b, h].cpu().double().numpy(), m.S)
    errs["s_k"] = rel_l2(out.s_k[b, h].cpu().double().numpy(), m.s_k)
    errs["s_v"] = rel_l2(out.s_v[b, h].cpu().double().numpy(), m.s_v)
    mtol = 1e-5 if dt == torch.float32 else 1e-5   # inputs exact; fp32 accumulation only
    assert errs["S"] <= mtol and errs["s_k"] <= mtol and errs["s_v"] <= mtol, errs
    return errs


def oracle_moments(out: mk.CompressOutput, b: int, h: int) -> O.Moments:
    return O.Moments(int(out.n_e[b, h]), out.s_k[b, h].cpu().double().numpy(),
                     out.s_v[b, h].cpu().double().numpy(), out.S[b, h].cpu().double().numpy())


def run_decode_steps(inp: dict, comp: mk.CompressOutput, steps: int, *, order=1, tau=1e-6,
                     append=True, n_split=0, lens0=None, summary=0):
    """Run `steps` decode calls on the GPU, each checked against the oracle fed the GPU's
    retained cache and fp32 moments.  `lens0` ([B, Hkv], each at most the compressed
    length) replaces the retained lengths before the first step.  Returns the list of max
    relative errors.  summary=1 (2) passes the prepared (half-precision) summary (the oracle reads the raw
    moments)."""
    dt = inp["k"].dtype
    tol = TOL[dt]
    B, Hkv, cap, d = comp.k_out.shape
    Hq = inp["q_win"].shape[1]
    G = Hq // Hkv
    S_arg = comp.S if summary == 0 else mk.momentkv_prepare_summary(
        comp.n_e, comp.s_k, comp.s_v, comp.S, dtype=dt, tau=tau, half=summary == 2)
    lens = comp.lens.clone()
    if lens0 is not None:
        lens0 = torch.as_tensor(lens0, dtype=torch.int32)
        assert bool((lens0 <= comp.lens.cpu()).all())
        lens.copy_(lens0)
    moments = [[oracle_moments(comp, b, h) for h in range(Hkv)] for b in range(B)]
    kc_ref = h64(comp.k_out)
    vc_ref = h64(comp.v_out)
    ln_ref = lens.cpu().numpy().astype(np.int64)
    lse = torch.empty(B, Hq, dtype=torch.float32, device=comp.k_out.device)
    w_r = torch.empty_like(lse)
    ws = None
    worst = []
    for t in range(steps):
        q = inp["q_dec"][t]
        kn = inp["k_new"][t] if append else None
        vn = inp["v_new"][t] if append else None
        out, _, _, ws = mk.momentkv_decode_attn(
            q, comp.k_out, comp.v_out, lens, comp.n_e, comp.s_k, comp.s_v, S_arg, k_new=kn,
            v_new=vn, max_len=cap, order=order, tau=tau, lse=lse, w_r=w_r, workspace=ws,
            n_split=n_split, summary=summary)
        torch.cuda.synchronize()
        ref_out, ref_lz, ref_wr, (kc_ref, vc_ref, ln_ref) = O.decode(
            h64(q), kc_ref, vc_ref, ln_ref, moments,
            k_new=None if kn is None else h64(kn), v_new=None if vn is None else h64(vn),
            tau=tau, order=order)
        got = h64(out)
        e = max(rel_l2(got[b, hq], ref_out[b, hq]) for b in range(B) for hq in range(Hq))
        e_w = float(np.max(np.abs(w_r.cpu().double().numpy() - ref_wr)))
        got_lz = lse.cpu().double().numpy()
        same = got_lz == ref_lz                     # equal infinities (empty retained set)
        e_l = float(np.max(np.where(same, 0.0, np.abs(got_lz - ref_lz) /
                                    np.maximum(1.0, np.abs(np.where(same, 0.0, ref_lz))))))
        assert e <= tol, (t, e)
        assert e_w <= max(tol, 1e-5), (t, e_w)
        assert e_l <= max(tol, 1e-5), (t, e_l)
        np.testing.assert_array_equal(lens.cpu().numpy(), ln_ref)
        worst.append(e)
    # appended rows landed in the cache
    if append:
        np.testing.assert_array_equal(h64(comp.k_out), kc_ref)
        np.testing.assert_array_equal(h64(comp.v_out), vc_ref)
    assert int(ws[:4].view(torch.int32)[0]) == 0
    return worst


EVICT_BAND = 1e-4   # relative band of the oracle's lowest score within which rows may swap


def run_evict_steps(inp: dict, comp: mk.CompressOutput, steps: int, budget: int, *, order=1,
                    tau=1e-6, n_split=0, flag=0, start=None):
    """Run `steps` decode calls with eviction on the GPU against the oracle's own
    trajectory.  The oracle starts from the GPU's compressed state (cache rows, lens and
    fp32 moments, all checked by the compress parity) and then evolves on its own.  At
    every step, per head:
      * the evicted row is the oracle's argmin, or a row whose oracle score lies within
        EVICT_BAND of the lowest (then the oracle follows that row, and it is counted);
      * lens, n_e and every cache row are exact; s_k, s_v, S within 1e-5 (relative L2);
      * out, w_R and log Z_R are within the dtype's tolerance.
    The GPU buffers are copies, so `comp` is left as it was; `start` = (lens, n_e) replaces
    the compressed lengths and counts first.  The workspace flag must end equal to `flag`.
    Returns (worst rel err of out, band swaps, evictions)."""
    dt = inp["k"].dtype
    tol = TOL[dt]
    B, Hkv, cap, d = comp.k_out.shape
    Hq = inp["q_win"].shape[1]
    G = Hq // Hkv
    kc, vc, lens = comp.k_out.clone(), comp.v_out.clone(), comp.lens.clone()
    n_e, s_k, s_v, S = comp.n_e.clone(), comp.s_k.clone(), comp.s_v.clone(), comp.S.clone()
    if start is not None:
        lens.copy_(torch.as_tensor(start[0], dtype=torch.int32))
        n_e.copy_(torch.as_tensor(start[1], dtype=torch.int32))
    moments = [[O.Moments(int(n_e[b, h]), h64(s_k[b, h]), h64(s_v[b, h]), h64(S[b, h]))
                for h in range(Hkv)] for b in range(B)]
    kc_ref, vc_ref = h64(comp.k_out), h64(comp.v_out)
    ln_ref = lens.cpu().numpy().astype(np.int64)
    lse = torch.empty(B, Hq, dtype=torch.float32, device=kc.device)
    w_r = torch.empty_like(lse)
    ev = torch.empty(B, Hkv, dtype=torch.int32, device=kc.device)
    ws = None
    worst, swaps, evictions = 0.0, 0, 0
    for t in range(steps):
        q, kn, vn = inp["q_dec"][t], inp["k_new"][t], inp["v_new"][t]
        out, _, _, _, ws = mk.momentkv_decode_evict(
            q, kc, vc, lens, n_e, s_k, s_v, S, kn, vn, budget, max_len=cap, order=order,
            tau=tau, n_split=n_split, lse=lse, w_r=w_r, evicted=ev, workspace=ws)
        torch.cuda.synchronize()
        ev_gpu = ev.cpu().numpy().astype(np.int64)
        args = (h64(q), kc_ref, vc_ref, ln_ref, moments, h64(kn), h64(vn), budget)
        ref = O.decode_evict(*args, tau=tau, order=order)
        ev_ref, heads = ref[4], ref[5]
        if not np.array_equal(ev_gpu, ev_ref):
            for b in range(B):
                for h in range(Hkv):
                    if ev_gpu[b, h] == ev_ref[b, h]:
                        continue
                    assert ev_gpu[b, h] >= 0 and ev_ref[b, h] >= 0, (t, b, h)
                    sc = heads[b][h]["score"]
                    lo = sc.min()
                    assert sc[ev_gpu[b, h]] <= lo * (1 + EVICT_BAND) + 1e-300, \
                        (t, b, h, sc[ev_gpu[b, h]], lo)
                    swaps += 1
            ref = O.decode_evict(*args, tau=tau, order=order, forced=ev_gpu)
        ref_out, ref_lz, ref_wr, (kc_ref, vc_ref, ln_ref, moments), ev_ref, _ = ref
        np.testing.assert_array_equal(ev_gpu, ev_ref)
        evictions += int((ev_gpu >= 0).sum())
        np.testing.assert_array_equal(lens.cpu().numpy(), ln_ref)
        np.testing.assert_array_equal(h64(kc), kc_ref)
        np.testing.assert_array_equal(h64(vc), vc_ref)
        ne_g = n_e.cpu().numpy()
        for b in range(B):
            for h in range(Hkv):
                m = moments[b][h]
                assert int(ne_g[b, h]) == m.n_e, (t, b, h)
                assert rel_l2(h64(s_k[b, h]), m.s_k) <= 1e-5
                assert rel_l2(h64(s_v[b, h]), m.s_v) <= 1e-5
                assert rel_l2(h64(S[b, h]), m.S) <= 1e-5
        got = h64(out)
        e = max(rel_l2(got[b, hq], ref_out[b, hq]) for b in range(B) for hq in range(Hq))
        e_w = float(np.max(np.abs(w_r.cpu().double().numpy() - ref_wr)))
        e_l = float(np.max(np.abs(lse.cpu().double().numpy() - ref_lz) /
                           np.maximum(1.0, np.abs(ref_lz))))
        assert e <= tol, (t, e)
        assert e_w <= max(tol, 1e-5), (t, e_w)
        assert e_l <= max(tol, 1e-5), (t, e_l)
        worst = max(worst, e)
    assert int(ws[:4].view(torch.int32)[0]) == flag
    return worst, swaps, evictions


def check_head_budgets(inp_cpu: dict, out: mk.CompressOutput, b: int, budget: int, *,
                       n_sink=1, chunk=4) -> tuple[np.ndarray, int]:
    """Head-adaptive split of sequence b: the GPU's per-head counts (lens - n_sink - w) are
    exactly the split of the GPU's own pooled masses (layer-wide order by (-mass, head,
    position)); against the oracle's masses, the layer-wide kept sets may differ only by
    swaps inside the selection band of the boundary mass.  Returns (k_h, swaps)."""
    dt = inp_cpu["k"].dtype
    Hkv = inp_cpu["k"].shape[1]
    w = inp_cpu["q_win"].shape[2]
    N, d = inp_cpu["k"].shape[2], inp_cpu["k"].shape[3]
    G = inp_cpu["q_win"].shape[1] // Hkv
    k_keep = budget - n_sink - w
    kh = out.lens[b].cpu().numpy().astype(np.int64) - n_sink - w
    ab_g = out.abar[b].cpu().double().numpy()                      # [Hkv, n_c]
    np.testing.assert_array_equal(O.head_budgets(ab_g, k_keep), kh)
    q = h64(inp_cpu["q_win"][b:b + 1])
    ab_o = np.stack([O.chunk_pool(O.window_attention_mass(q[0, h * G:(h + 1) * G],
                                                          h64(inp_cpu["k"][b, h]), 1 / math.sqrt(d)),
                                  n_sink, chunk) for h in range(Hkv)])
    assert rel_l2(ab_g, ab_o) <= TOL[dt]
    n = ab_o.shape[1]
    def kept_set(ab, counts):
        sel = set()
        for h in range(Hkv):
            order = np.lexsort((np.arange(n), -ab[h]))[:counts[h]]
            sel.update(int(h * n + j) for j in order)
        return sel
    got = kept_set(ab_g, kh)
    ref = kept_set(ab_o, O.head_budgets(ab_o, k_keep))
    flat = ab_o.reshape(-1)
    T = np.sort(flat)[::-1][Hkv * k_keep - 1]
    band = SEL_BAND[dt]
    for x in got ^ ref:
        assert abs(flat[x] - T) <= band * T, (x, flat[x], T)
    return kh, len(got ^ ref) // 2
