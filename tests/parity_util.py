"""Helpers shared by the GPU parity tests: run the HIP path, run the oracle on the same
bits, and compare with the tolerances of the parity protocol.

Tolerances.
  * Outputs rounded to the element type (the decode's `out`): relative L2 per query head
    1e-5 for fp32, 2e-2 for bf16 (one bf16 rounding is 2^-8 relative).
  * Moments (n_e exact; s_k, s_v, S): relative L2 1e-5 (exact inputs, fp32 sums).
  * fp32 intermediates that are never rounded to bf16 (abar, the provisional and
    moment-round scores, log Z_R, w_R): element by element, within an error bound derived
    from the fp32 arithmetic that produces them (see `compress_score_bounds` and
    `decode_bounds`): every input is exact in fp32 (bf16 values, or fp32 values), dot
    products of length n carry gamma(n) = n u / (1 - n u) of the sum of absolute terms
    (u = 2^-23, one fp32 rounding taken at twice the round-to-nearest unit so that
    truncating adds inside a matrix instruction are covered), long reductions (softmax
    normalisers over the context, covariance sums over the candidates) carry the
    probabilistic bound lambda sqrt(n) u with lambda = 8 (Higham and Mary, SIAM J. Sci.
    Comput. 2019: exceeded with probability below 2 exp(-lambda^2 / 2) per sum, whatever
    the order of the additions), and the bf16 hi/lo split of the provisional summary adds
    2^-16 of each entry.
Selection: the GPU's kept sets must equal the top-k of the GPU's own scores exactly
(ties: lower position), and differ from the oracle's only by swaps inside a near-tie
band around the k-th score (1e-5 relative for fp32, 1e-4 for bf16).

Setting MKV_PARITY_LOG to a file name appends each checked quantity's measured maximum
(relative error and fraction of its bound) as one JSON line.
"""
from __future__ import annotations

import json
import math
import os

import numpy as np
import torch

import oracle as O
from paper_2606_01563_amd import momentkv as mk

TOL = {torch.float32: 1e-5, torch.bfloat16: 2e-2}
SEL_BAND = {torch.float32: 1e-5, torch.bfloat16: 1e-4}

U32 = 2.0 ** -23          # one fp32 rounding (twice the round-to-nearest unit)
LAMBDA = 8.0              # probabilistic bound of long sums: lambda sqrt(n) u
TINY = 2.0 ** -100        # absolute floor: probabilities below it may flush to zero
BF16_SPLIT = 2.0 ** -16   # |x - (hi + lo)| of the bf16 hi/lo split, relative to |x|


def gamma(n: int) -> float:
    """Worst-case relative error of an n-term fp32 sum of exact terms (n u / (1 - n u))."""
    return n * U32 / (1.0 - n * U32)


def gamma_long(n: int) -> float:
    """Probabilistic relative error bound of a long fp32 sum of n terms (lambda sqrt(n) u)."""
    return LAMBDA * math.sqrt(max(n, 1)) * U32


def _log(entry: dict):
    path = os.environ.get("MKV_PARITY_LOG")
    if path:
        entry = dict(test=os.environ.get("PYTEST_CURRENT_TEST", "").split(" ")[0], **entry)
        with open(path, "a") as f:
            f.write(json.dumps(entry) + "\n")


def check_within(got, ref, bound, what: str) -> dict:
    """Element-wise |got - ref| <= bound.  Returns the measured maxima: relative error
    (|got - ref| / |ref| over entries with ref != 0) and the fraction of the bound."""
    got = np.asarray(got, np.float64)
    ref = np.asarray(ref, np.float64)
    bound = np.broadcast_to(np.asarray(bound, np.float64), ref.shape)
    same = got == ref                    # equal infinities (an empty retained set)
    with np.errstate(invalid="ignore"):  # inf - inf where `same` holds
        err = np.where(same, 0.0, np.abs(got - ref))
    bad = ~(err <= bound)
    if bad.any():
        i = int(np.flatnonzero(bad.reshape(-1))[0])
        raise AssertionError(
            f"{what}: {int(bad.sum())} of {bad.size} entries beyond the bound; first at flat "
            f"index {i}: got {got.reshape(-1)[i]!r}, ref {ref.reshape(-1)[i]!r}, "
            f"bound {bound.reshape(-1)[i]:.3e}")
    nz = (np.abs(ref) > 0) & ~same
    rel = float(np.max(err[nz] / np.abs(ref[nz]))) if nz.any() else 0.0
    frac = float(np.max(np.where(bound > 0, err / np.where(bound > 0, bound, 1.0), 0.0)))
    out = dict(max_rel=rel, max_frac_of_bound=frac)
    _log(dict(quantity=what, n=int(ref.size), **out))
    return out


def abar_eps(qg, K, chunk: int) -> float:
    """Relative error bound of the GPU's pooled window mass for one KV head (qg [G, w, d],
    K [N, d], exact inputs): logit errors gamma(d+1) kappa + 3u |s| (kappa the scaled sum
    of |q_ti k_ji|; the products, the scale and the base-2 conversion), twice (the
    probability's own logit and its row's normaliser), the normaliser's long sum
    gamma_long(N), the exp and the products 6u, the mean over the G w rows and the chunk
    gamma(G w + c + 2)."""
    G, w, d = qg.shape
    scale = 1.0 / math.sqrt(d)
    Q = qg.reshape(G * w, d)
    s = scale * (Q @ K.T)
    kappa = scale * (np.abs(Q) @ np.abs(K).T)
    ds = gamma(d + 1) * kappa + 3 * U32 * np.abs(s)
    return 2.0 * float(ds.max()) + gamma_long(K.shape[0]) + gamma(G * w + chunk + 2) + 6 * U32


def compress_score_bounds(qg, K, V, ref, kept0, *, n_sink: int, chunk: int, mi_rounds: int,
                          tau: float, split: bool) -> dict:
    """Per-candidate absolute error bounds of the GPU's abar, score0 and score for one KV
    head, from exact fp32 inputs and fp32 arithmetic.

    qg [G, w, d], K, V [N, d] (fp64 copies of the inputs); ref: the oracle's result with
    the GPU's provisional kept set (kept0, absolute positions) as round 0; split: the
    provisional summary is a bf16 hi/lo pair (bf16 inputs).
      logits   s_tj = scale q_t.k_j: |ds| <= gamma(d+1) kappa_tj + 3u |s_tj|, kappa the
               scaled sum of |q_ti k_ji| (products, the scale and the base-2 conversion);
      abar     each softmax probability: its logit, the row's normaliser (its logits and a
               long sum over the context) and the exp: eps_a = 2 max|ds| + gamma_long(N) +
               6u; then the mean over the G w rows and the chunk: + gamma(G w + c + 2);
      score0   abar ||v||: + gamma(d+1)/2 (sum of squares, halved by the root) + 3u;
      score    abar ||v - v_bar0 - (scale/n0) S_tilde0 k||: the provisional sums carry
               gamma_long(n_c) + gamma(64) of the sums of absolute terms they add (the
               candidates' and the kept rows'); the centring 4u; the hi/lo split 2^-16;
               the MFMA product gamma(2d+2); the residual's own roundings; the norm
               gamma(d+1)/2.  Second-order terms are covered by a factor 1.05."""
    G, w, d = qg.shape
    N = K.shape[0]
    scale = 1.0 / math.sqrt(d)
    eps_a = abar_eps(qg, K, chunk)
    out = dict(eps_abar=eps_a, abar=1.05 * eps_a * ref.abar + TINY)
    if mi_rounds < 0:
        return out
    cand = np.arange(n_sink, N - w)
    vn = np.sqrt((V[cand] ** 2).sum(axis=1))
    eps0 = eps_a + gamma(d + 1) / 2 + 3 * U32
    out["score0"] = 1.05 * eps0 * ref.sigma0 + TINY * (1.0 + vn)
    if mi_rounds < 1:
        return out
    Kc, Vc = K[cand], V[cand]
    # the summary of the last round is the round before's evicted set: the GPU's provisional
    # one for mi_rounds = 1, else the oracle's (the GPU's unless an intermediate cut fell on
    # a near-tie, which the final comparison would then report)
    R0 = np.asarray(kept0 if mi_rounds < 2 else ref.rounds[-2], dtype=np.int64)
    n0 = len(cand) - len(R0)
    m0 = O.evicted_moments(K, V, np.setdiff1d(cand, R0))
    if n0 == 0:
        rn = vn
        out["score"] = 1.05 * (ref.abar * rn * (eps_a + gamma(d + 1) / 2 + 3 * U32)) + TINY * (1 + rn)
        return out
    eps_acc = gamma_long(len(cand)) + gamma(64)
    A = np.abs(Vc).T @ np.abs(Kc) + np.abs(V[R0]).T @ np.abs(K[R0])
    av = np.abs(Vc).sum(axis=0) + np.abs(V[R0]).sum(axis=0)
    ak = np.abs(Kc).sum(axis=0) + np.abs(K[R0]).sum(axis=0)
    dS0, dsv, dsk = eps_acc * A, eps_acc * av, eps_acc * ak
    outer = np.outer(m0.s_v, m0.s_k) / n0
    St = m0.S - outer
    dSt = (dS0 + (np.outer(dsv, np.abs(m0.s_k)) + np.outer(np.abs(m0.s_v), dsk)) / n0
           + 4 * U32 * (np.abs(m0.S) + np.abs(outer)) + tau)
    E = dSt + (BF16_SPLIT if split else 0.0) * np.abs(St) + gamma(2 * d + 2) * np.abs(St)
    coef = scale / n0
    acc = (m0.s_v / scale)[:, None] + St @ Kc.T                    # [d, n_c]
    dacc = (E @ np.abs(Kc).T + (gamma(2 * d + 2) * np.abs(m0.s_v) + U32 * np.abs(m0.s_v)
                                + dsv)[:, None] / scale)
    r = Vc.T - coef * acc
    dr = coef * dacc + U32 * np.abs(Vc.T) + 3 * U32 * coef * np.abs(acc)
    rn = np.sqrt((r * r).sum(axis=0))
    drn = np.sqrt((dr * dr).sum(axis=0)) + (gamma(d + 1) / 2 + 2 * U32) * rn
    out["score"] = 1.05 * (ref.abar * drn + ref.abar * rn * (eps_a + U32)) + TINY * (1 + rn)
    return out


def decode_bounds(q, K, lz_ref, w_ref, m: "O.Moments", *, amplify: float = 1.0,
                  sk_err: float = 0.0) -> tuple[float, float]:
    """Absolute error bounds of the GPU's log Z_R and w_R for one query against one KV
    head's retained rows K [n, d] (fp64 copies of the exact inputs):
      log Z_R   max over rows of the logit error (gamma(d+1) kappa + 3u |s|), the long
                sum of exps (gamma_long(n)), the split-K merge and the final log and base
                conversion (gamma(16) + 3u |log Z_R|); `amplify` multiplies the sum's part
                where a term is taken out of an accumulated sum afterwards;
      log Z_E   log n_e + scale q.s_k / n_e: gamma(d+1) of the absolute terms, 3u of the
                terms themselves, plus `sk_err` (relative) for a key sum that was itself
                accumulated on the GPU in fp32;
      w_R       w_R = exp(log Z_R - lse) with lse = logsumexp(log Z_R, log Z_E): the errors
                of the two logs move it by w_R (1 - w_R) (|d log Z_R| + |d log Z_E|) (1.05 for
                second order); lse's own roundings (the max, the log, the add) move it by
                w_R 4u (|log Z_R| + |log Z_E| + 2); the exp 4u."""
    d = q.shape[0]
    scale = 1.0 / math.sqrt(d)
    if K.shape[0] > 0:
        s = scale * (K @ q)
        kappa = scale * (np.abs(K) @ np.abs(q))
        dlz = float(np.max(gamma(d + 1) * kappa + 3 * U32 * np.abs(s))) + \
            amplify * (gamma_long(K.shape[0] + 1) + gamma(16)) + 3 * U32 * abs(lz_ref)
    else:
        dlz = 0.0
    if m.n_e == 0:
        return dlz, 4 * U32
    sbar = scale * float(q @ m.s_k) / m.n_e
    dlze = (gamma(d + 1) + sk_err) * scale * float(np.abs(q) @ np.abs(m.s_k)) / m.n_e + \
        3 * U32 * (abs(math.log(m.n_e)) + abs(sbar))
    if not math.isfinite(lz_ref):
        return dlz, 4 * U32
    lze = math.log(m.n_e) + sbar
    dw = 1.05 * w_ref * (1.0 - w_ref) * (dlz + dlze) + \
        w_ref * 4 * U32 * (abs(lz_ref) + abs(lze) + 2.0) + 4 * U32
    return dlz, dw


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
        bnd = compress_score_bounds(q[0, h * G:(h + 1) * G], K, V, ref, kept0, n_sink=n_sink,
                                    chunk=chunk, mi_rounds=mi_rounds, tau=tau,
                                    split=dt == torch.bfloat16)
        errs["abar"] = check_within(abar_g, ref.abar, bnd["abar"], "abar")
        if mi_rounds >= 0:
            errs["score0"] = check_within(s0_g, ref.sigma0, bnd["score0"], "score0")
        if mi_rounds >= 1:
            errs["score"] = check_within(s1_g, ref.sigma, bnd["score"], "score")
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
    mtol = 1e-5                                     # inputs exact; fp32 accumulation only
    assert errs["S"] <= mtol and errs["s_k"] <= mtol and errs["s_v"] <= mtol, errs
    _log(dict(quantity="moments", n_e=int(out.n_e[b, h]), k_keep=int(k_keep),
              S=errs["S"], s_k=errs["s_k"], s_v=errs["s_v"]))
    return errs


def _decode_bound_arrays(q, kc, vc, lens, moments, lz_ref, w_ref, **kw):
    """decode_bounds for every (sequence, query head): arrays [B, Hq] for log Z_R and w_R.
    Query head hq reads KV head hq // G (the layout pinned in the oracle's tests)."""
    B, Hq, _ = q.shape
    Hkv = kc.shape[1]
    G = Hq // Hkv
    blz = np.zeros((B, Hq))
    bw = np.zeros((B, Hq))
    for b in range(B):
        for hq in range(Hq):
            h = hq // G
            blz[b, hq], bw[b, hq] = decode_bounds(q[b, hq], kc[b, h, :lens[b, h]],
                                                  float(lz_ref[b, hq]), float(w_ref[b, hq]),
                                                  moments[b][h], **kw)
    return blz, bw


def oracle_moments(out: mk.CompressOutput, b: int, h: int) -> O.Moments:
    return O.Moments(int(out.n_e[b, h]), out.s_k[b, h].cpu().double().numpy(),
                     out.s_v[b, h].cpu().double().numpy(), out.S[b, h].cpu().double().numpy())


def run_decode_steps(inp: dict, comp: mk.CompressOutput, steps: int, *, order=1, tau=1e-6,
                     append=True, n_split=0, lens0=None, summary=0):
    """Run `steps` decode calls on the GPU, each checked against the oracle fed the GPU's
    retained cache and fp32 moments.  `lens0` ([B, Hkv], each at most the compressed
    length) replaces the retained lengths before the first step.  Returns the list of max
    relative errors.  summary=1 (2) passes the prepared (half-precision) summary (the oracle reads the raw
    moments); summary=3 passes a raw S stored in bf16 (compress with moment_dtype bf16), which
    the oracle reads as it is."""
    dt = inp["k"].dtype
    tol = TOL[dt]
    B, Hkv, cap, d = comp.k_out.shape
    Hq = inp["q_win"].shape[1]
    G = Hq // Hkv
    # summary 3: comp.S is the raw sum stored in bf16, and the oracle reads the same values
    S_arg = comp.S if summary in (0, 3) else mk.momentkv_prepare_summary(
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
        assert e <= tol, (t, e)
        _log(dict(quantity="out", rel_l2=e))
        blz, bw = _decode_bound_arrays(h64(q), kc_ref, vc_ref, ln_ref, moments, ref_lz, ref_wr)
        check_within(lse.cpu().double().numpy(), ref_lz, blz, f"log Z_R (step {t})")
        check_within(w_r.cpu().double().numpy(), ref_wr, bw, f"w_R (step {t})")
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
        assert e <= tol, (t, e)
        _log(dict(quantity="out (eviction)", rel_l2=e))
        # the long-cache shape takes the evicted row's term out of an accumulated sum and
        # recomputes where more than 1/17 of the sum would be left: up to 17x its error;
        # the key sum has gone through t + 1 fp32 rank-one additions since the compression
        blz, bw = _decode_bound_arrays(h64(q), kc_ref, vc_ref, ln_ref, moments, ref_lz, ref_wr,
                                       amplify=17.0, sk_err=gamma(t + 2))
        check_within(lse.cpu().double().numpy(), ref_lz, blz, f"log Z_R (eviction step {t})")
        check_within(w_r.cpu().double().numpy(), ref_wr, bw, f"w_R (eviction step {t})")
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
    for h in range(Hkv):
        eps = abar_eps(q[0, h * G:(h + 1) * G], h64(inp_cpu["k"][b, h]), chunk)
        check_within(ab_g[h], ab_o[h], 1.05 * eps * ab_o[h] + TINY, "abar (layer-wide split)")
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
