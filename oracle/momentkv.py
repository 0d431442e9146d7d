"""Plain fp64 CPU oracle for the MomentKV hot path (compress + corrected decode).

TEST INFRASTRUCTURE ONLY.  This module is the independent reference that the HIP
path is checked against.  Only the test suite, the smoke check and the CPU-baseline
leg of the benchmark may import it; the product path never does, and this module
imports nothing from the product package.  Inputs arrive as NumPy arrays (any
float dtype; they are upcast exactly to float64) and every result is float64
(indices and counts are int64).

Paper: "MomentKV: Closing the Directional Gap in KV Cache Eviction for
Long-Context Inference" (arXiv 2606.01563).  Each function names the passage it
follows.  Where the paper is silent the adopted reading is stated in the function
and listed in the design doc's reading table.

Pinning status (what fixes each function other than itself; see tests/):
  window_attention_mass   pinned: torch SDPA with one-hot values, brute-force loops
  chunk_pool              pinned: chunk-sum invariants, chunk=1 identity
  select_top              pinned: Python's stable sorted() on planted ties
  evicted_moments         pinned: sequential rank-one updates, numpy cov identity
  centered_moments        pinned: n_e=1 and zero-spread closed forms, cov identity
  residual_scores         pinned: second-order convergence to v_j - f_E(k_j) (SDPA)
  compress                pinned: structure, full-budget case, permutation equivariance,
                          SnapKV-mode reduction; the batched selection rule itself
                          (one provisional round + moment rounds) is a reading of
                          Algorithm 1 and is *parity unpinned* beyond its definition.
  head_budgets            pinned: brute-force sort of (-mass, head, position) on tiny
                          layers, one head = the uniform budget, identical heads split evenly
  decode                  pinned: no-eviction == SDPA, zero key spread == full
                          attention, second-order error, Jensen bound, weight bias
  greedy_evict            quality reference only (parity unpinned; no printed example)
  eviction_diagnostics    built from attention_parts and decode_head (pinned above); the
                          order = -1 ablation pinned to SDPA over the retained rows
  evict_scores_head       pinned: planted zero-residual token, alpha ordering at equal
                          residual norms, n_e = 0 reduction to alpha ||v||
  decode_evict            pinned: zero key spread (evicts the value nearest the mean and
                          still equals full attention over every token seen), moments
                          equal brute-force sums over everything evicted, token
                          conservation, Phase 2 on the post-eviction state
  batched wrappers        the query-head -> KV-head grouping of compress, decode and
  (GQA mapping)           decode_evict pinned to torch SDPA with enable_gqa (which KV head
                          each query head reads is read off SDPA's own output)
"""
from __future__ import annotations

import math
from dataclasses import dataclass, field

import numpy as np

F64 = np.float64

__all__ = [
    "Moments", "CompressResult", "DecodeResult",
    "window_attention_mass", "chunk_pool", "select_top", "evicted_moments",
    "centered_moments", "moment_residuals", "residual_scores", "select_candidates",
    "compress", "compress_head", "head_budgets",
    "decode", "decode_head", "append_tokens", "attention_parts", "greedy_evict",
    "evict_scores_head", "decode_evict_head", "decode_evict", "eviction_diagnostics",
    "moment_storage_bytes",
]


def _f64(x) -> np.ndarray:
    return np.asarray(x, dtype=F64)


# --------------------------------------------------------------------------------------
# Moment statistics (Sec. 4.1; App. A.1 Eqs. app_sufficient, app_S_tilde, app_update)
# --------------------------------------------------------------------------------------
@dataclass
class Moments:
    """Raw sufficient statistics of one KV head's evicted set E.

    n_e = |E|, s_k = sum_E k_i, s_v = sum_E v_i, S = sum_E v_i k_i^T
    (row index = value dimension, column index = key dimension).
    Stored raw, centred at query time (Sec. 4.1, covariance identity).
    """
    n_e: int
    s_k: np.ndarray  # [d]
    s_v: np.ndarray  # [d]
    S: np.ndarray    # [d, d]

    @staticmethod
    def zeros(d: int) -> "Moments":
        """Zero initial state at the start of a generation (Sec. 5.1 setup)."""
        return Moments(0, np.zeros(d, F64), np.zeros(d, F64), np.zeros((d, d), F64))


def evicted_moments(k: np.ndarray, v: np.ndarray, evicted: np.ndarray) -> Moments:
    """Sufficient statistics over the evicted rows (App. A.1 Eq. app_sufficient).

    k, v: [N, d]; evicted: integer positions of E.  S = V_E^T K_E is the sum of the
    rank-one terms v_i k_i^T that Eq. app_update adds one eviction at a time.
    """
    k = _f64(k)
    v = _f64(v)
    e = np.asarray(evicted, dtype=np.int64)
    d = k.shape[1]
    if e.size == 0:
        return Moments.zeros(d)
    ke, ve = k[e], v[e]
    return Moments(int(e.size), ke.sum(axis=0), ve.sum(axis=0), ve.T @ ke)


def centered_moments(m: Moments, tau: float):
    """Recover k_bar, v_bar and the clamped covariance S_tilde.

    k_bar = s_k/n_e, v_bar = s_v/n_e, S_tilde = S - s_v s_k^T / n_e
    (App. A.1 Eq. app_S_tilde), then every entry of S_tilde with magnitude below tau
    is set to zero (App. C.2 numerical safeguard; reading: strict '<', absolute,
    applied to S_tilde itself).  With n_e = 0 Algorithm 1 sets v_bar and S_tilde to
    zero (its Phase 1 else-branch); k_bar is then undefined and returned as zeros.
    """
    d = m.s_k.shape[0]
    if m.n_e == 0:
        z = np.zeros(d, F64)
        return z.copy(), z.copy(), np.zeros((d, d), F64)
    n = F64(m.n_e)
    k_bar = m.s_k / n
    v_bar = m.s_v / n
    S_t = m.S - np.outer(m.s_v, m.s_k) / n
    if tau > 0:
        S_t = np.where(np.abs(S_t) < tau, 0.0, S_t)
    return k_bar, v_bar, S_t


# --------------------------------------------------------------------------------------
# Prefill scoring: observation-window attention mass (Sec. 5.1 prefill protocol)
# --------------------------------------------------------------------------------------
def window_attention_mass(q_win: np.ndarray, k: np.ndarray, scale: float) -> np.ndarray:
    """Attention mass each prefix token receives from the observation window.

    q_win: [G, w, d] window queries of the G query heads sharing this KV head;
    k: [N, d].  Logits s = scale * q^T k (Sec. 2, full-attention definition).  Each
    window row t (absolute position N-w+t) attends causally to keys j <= N-w+t and is
    softmax-normalised over them.  a_j is the mean over the G*w rows of the
    probability on key j, for j < N-w (readings: GQA rows averaged; causal window).
    Returns a: [N-w].
    """
    q = _f64(q_win)
    kk = _f64(k)
    G, w, d = q.shape
    N = kk.shape[0]
    rows = q.reshape(G * w, d)
    logits = scale * (rows @ kk.T)                               # [G*w, N]
    t = np.tile(np.arange(w), G)                                 # window offset of each row
    visible = np.arange(N)[None, :] <= (N - w + t)[:, None]
    logits = np.where(visible, logits, -np.inf)
    shifted = logits - logits.max(axis=1, keepdims=True)
    p = np.exp(shifted)
    p /= p.sum(axis=1, keepdims=True)
    return p[:, : N - w].sum(axis=0) / F64(G * w)


def chunk_pool(a: np.ndarray, n_sink: int, chunk: int) -> np.ndarray:
    """Merge adjacent candidates into chunks before scoring (Sec. 5.1 prefill protocol).

    Reading: aligned, non-overlapping chunks of absolute positions [c*m, c*m+c); each
    candidate j in C = [n_sink, len(a)) gets the mean of a over the candidates of its
    chunk.  Returns abar over C (length len(a) - n_sink).  chunk = 1 is the identity.
    """
    a = _f64(a)
    n_cand_end = a.shape[0]
    pos = np.arange(n_sink, n_cand_end)
    out = np.empty(pos.shape[0], F64)
    if chunk <= 1:
        return a[n_sink:].copy()
    for c0 in range((n_sink // chunk) * chunk, n_cand_end, chunk):
        lo, hi = max(c0, n_sink), min(c0 + chunk, n_cand_end)
        if lo >= hi:
            continue
        out[lo - n_sink: hi - n_sink] = a[lo:hi].mean()
    return out


def select_top(score: np.ndarray, k: int) -> np.ndarray:
    """Indices (into score) of the k largest scores; equal scores keep the lower index.

    This is the batched form of "evict the lowest score first" (Algorithm 1, argmin
    step; Sec. 4.2): the k retained are the first k of the order (-score, index).
    Returned in that order (best first).
    """
    s = _f64(score)
    order = np.lexsort((np.arange(s.shape[0]), -s))
    return order[:k].astype(np.int64)


def moment_residuals(k: np.ndarray, v: np.ndarray, m: Moments, scale: float,
                     tau: float) -> np.ndarray:
    """Moment residual vectors r_j = v_j - v_bar - S_tilde k_j / (n_e sqrt(d)).

    Sec. 4.2 Eq. residual, for every row of k, v ([n, d]); 1/sqrt(d) is `scale`.  With
    n_e = 0 the summary is empty, v_bar = S_tilde = 0 and r_j = v_j (Algorithm 1
    Phase 1 else-branch).
    """
    kk = _f64(k)
    vv = _f64(v)
    if m.n_e == 0:
        return vv.copy()
    _, v_bar, S_t = centered_moments(m, tau)
    return vv - v_bar[None, :] - (scale / F64(m.n_e)) * (kk @ S_t.T)


def residual_scores(k: np.ndarray, v: np.ndarray, abar: np.ndarray, cand: np.ndarray,
                    m: Moments, scale: float, tau: float) -> tuple[np.ndarray, np.ndarray]:
    """Moment-residual eviction score of every candidate (Sec. 4.2).

    score_j = alpha_j * ||r_j|| with r_j from Eq. residual and alpha_j the pooled
    window mass abar_j (low score = safe to evict).  Returns (score, ||r||) over the
    candidate positions `cand`.
    """
    r = moment_residuals(_f64(k)[cand], _f64(v)[cand], m, scale, tau)
    rn = np.sqrt((r * r).sum(axis=1))
    return _f64(abar) * rn, rn


# --------------------------------------------------------------------------------------
# Compress: one-shot prefill eviction with moment-informed selection
# --------------------------------------------------------------------------------------
@dataclass
class CompressResult:
    idx: np.ndarray            # [L'] ascending retained positions
    k_out: np.ndarray          # [L', d]
    v_out: np.ndarray          # [L', d]
    moments: Moments           # raw sums over E
    retained: np.ndarray       # candidate positions kept by selection (ascending)
    evicted: np.ndarray        # E (ascending)
    a: np.ndarray | None = None        # window mass [N-w]
    abar: np.ndarray | None = None     # pooled mass over C
    sigma0: np.ndarray | None = None   # provisional score over C
    sigma: np.ndarray | None = None    # last moment-round score over C
    rounds: list = field(default_factory=list)  # per-round retained sets (ascending)


def select_candidates(abar: np.ndarray, k_c: np.ndarray, v_c: np.ndarray, k_keep: int, *,
                      mi_rounds: int = 1, scale: float, tau: float = 1e-6,
                      r0_override: np.ndarray | None = None) -> dict:
    """Batched reading of Algorithm 1 Phase 1 over the candidate rows (reading R1).

    abar: [n] pooled window mass of the candidates (their alpha_j); k_c, v_c: [n, d].
      round 0: the summary is empty, so r_j = v_j and score0 = abar_j ||v_j||; keep the
               top k_keep, the rest form E0;
      rounds 1..mi_rounds: the summary is the moments of the previous round's evicted
               set; score = abar_j ||r_j|| (Eq. residual); keep the top k_keep.
    mi_rounds = -1 keeps the top abar (attention-only, the SnapKV rule).  Keeping the top
    k_keep by (-score, index) is evicting lowest-score first (Sec. 4.2).
    Returns dict(rounds=[ascending kept candidate offsets per round], sigma0, sigma).
    r0_override replaces round 0's kept set (offsets), e.g. by the GPU's own.
    """
    n = abar.shape[0]
    everyone = np.arange(n, dtype=np.int64)
    sigma0 = sigma = None
    if mi_rounds < 0:
        return dict(rounds=[np.sort(select_top(abar, k_keep))], sigma0=None, sigma=None)
    vnorm = np.sqrt((_f64(v_c) ** 2).sum(axis=1))
    sigma0 = _f64(abar) * vnorm
    kept = np.sort(select_top(sigma0, k_keep))
    if r0_override is not None:
        kept = np.sort(np.asarray(r0_override, dtype=np.int64))
    rounds = [kept]
    for _ in range(mi_rounds):
        evicted = np.setdiff1d(everyone, kept)
        m_prev = evicted_moments(k_c, v_c, evicted)
        sigma, _ = residual_scores(k_c, v_c, abar, everyone, m_prev, scale, tau)
        kept = np.sort(select_top(sigma, k_keep))
        rounds.append(kept)
    return dict(rounds=rounds, sigma0=sigma0, sigma=sigma)


def compress_head(q_win, k, v, budget: int, *, n_sink: int = 1, chunk: int = 4,
                  mi_rounds: int = 1, scale: float | None = None, tau: float = 1e-6,
                  r0_override: np.ndarray | None = None) -> CompressResult:
    """Compress one KV head's prefill cache to `budget` tokens.

    Prefill protocol (Sec. 5.1): window attention mass over the last w prompt tokens,
    first n_sink tokens kept as attention sinks, the w window tokens kept, chunk
    pooling of the mass.  Candidates C = [n_sink, N-w); k_keep = budget - n_sink - w of
    them survive.

    Selection is `select_candidates` (the batched reading of Algorithm 1 Phase 1);
    mi_rounds = -1 is attention-only, 0 stops after the provisional round.  The output
    moments are the raw sums over the final evicted set (Eq. app_sufficient).
    budget >= N keeps everything with zero moments.

    r0_override: use this retained candidate set for round 0 instead of the oracle's
    own (parity tests feed the GPU's provisional set so that the moment round is
    compared on equal footing).
    """
    q = _f64(q_win)
    kk = _f64(k)
    vv = _f64(v)
    G, w, d = q.shape
    N = kk.shape[0]
    if scale is None:
        scale = 1.0 / math.sqrt(d)
    if budget >= N:
        idx = np.arange(N, dtype=np.int64)
        return CompressResult(idx, kk.copy(), vv.copy(), Moments.zeros(d),
                              np.arange(n_sink, N - w, dtype=np.int64),
                              np.zeros(0, np.int64))
    if w < 1 or w >= N:
        raise ValueError("window must satisfy 1 <= w < N")
    if budget < n_sink + w:
        raise ValueError("budget must cover the sink and window tokens")
    k_keep = budget - n_sink - w
    cand = np.arange(n_sink, N - w, dtype=np.int64)

    a = window_attention_mass(q, kk, scale)
    abar = chunk_pool(a, n_sink, chunk)

    sel = select_candidates(abar, kk[cand], vv[cand], k_keep, mi_rounds=mi_rounds,
                            scale=scale, tau=tau,
                            r0_override=None if r0_override is None
                            else np.asarray(r0_override, dtype=np.int64) - n_sink)
    rounds = [cand[r] for r in sel["rounds"]]
    kept = rounds[-1]
    sigma0, sigma = sel["sigma0"], sel["sigma"]

    evicted = np.setdiff1d(cand, kept)
    mom = evicted_moments(kk, vv, evicted)
    idx = np.sort(np.concatenate([np.arange(n_sink, dtype=np.int64), kept,
                                  np.arange(N - w, N, dtype=np.int64)]))
    return CompressResult(idx, kk[idx], vv[idx], mom, kept, evicted, a, abar,
                          sigma0, sigma, rounds)


def head_budgets(abar_heads, k_keep: int) -> np.ndarray:
    """Head-adaptive split of a layer's candidate budget (Sec. 5.1: the budget is allocated
    across the heads of a layer by their attention mass, as in Ada-KV).

    abar_heads: [Hkv, n_c] pooled window mass of every head's candidates.  Reading: the
    Hkv * k_keep candidates with the largest mass over the whole layer are kept, equal
    masses in (head, position) order; head h keeps as many candidates as it has among
    them.  Returns k_h per head (they sum to Hkv * k_keep, or to every candidate)."""
    a = _f64(abar_heads)
    H, n = a.shape
    flat = a.reshape(-1)
    keep = min(H * k_keep, flat.size)
    order = np.lexsort((np.arange(flat.size), -flat))[:keep]
    return np.bincount(order // n, minlength=H).astype(np.int64)


def compress(q_win, k, v, budget: int, *, adaptive: bool = False, **kw):
    """Batched compress over [B, Hq, w, d] window queries and [B, Hkv, N, d] K/V.

    Query head hq uses KV head hq // G with G = Hq / Hkv (GQA).  Returns a nested list
    [B][Hkv] of CompressResult.  adaptive: the per-head candidate counts come from
    head_budgets over the layer (each head then selects its k_h moment-informed), so head h
    keeps n_sink + w + k_h tokens.
    """
    q = np.asarray(q_win)
    B, Hq, w, d = q.shape
    K, V = np.asarray(k), np.asarray(v)
    Hkv, N = K.shape[1], K.shape[2]
    if Hq % Hkv:
        raise ValueError("Hq must be a multiple of Hkv")
    G = Hq // Hkv
    if not adaptive or budget >= N:
        return [[compress_head(q[b, h * G:(h + 1) * G], K[b, h], V[b, h], budget, **kw)
                 for h in range(Hkv)] for b in range(B)]
    n_sink, chunk = kw.get("n_sink", 1), kw.get("chunk", 4)
    scale = kw.get("scale") or 1.0 / math.sqrt(d)
    if budget < n_sink + w:
        raise ValueError("budget must cover the sink and window tokens")
    out = []
    for b in range(B):
        abar = np.stack([chunk_pool(window_attention_mass(q[b, h * G:(h + 1) * G], K[b, h], scale),
                                    n_sink, chunk) for h in range(Hkv)])
        kh = head_budgets(abar, budget - n_sink - w)
        out.append([compress_head(q[b, h * G:(h + 1) * G], K[b, h], V[b, h],
                                  n_sink + w + int(kh[h]), **kw) for h in range(Hkv)])
    return out


# --------------------------------------------------------------------------------------
# Decode: normalisation-corrected attention (Algorithm 1 Phase 2; Eqs. fhat, jensen,
# fused; log-domain mixing weight of App. C.2)
# --------------------------------------------------------------------------------------
@dataclass
class DecodeResult:
    out: np.ndarray        # [d] corrected output f_hat(q)
    f_R: np.ndarray        # [d] retained-set attention output
    log_Z_R: float         # log of the retained partition function
    w_R: float             # mixing weight on f_R (1 when nothing is evicted)
    f_E_hat: np.ndarray | None
    log_Z_E_hat: float | None


def decode_head(q, k_ret, v_ret, m: Moments, *, scale: float | None = None,
                tau: float = 1e-6, order: int = 1) -> DecodeResult:
    """Corrected attention output for one query against one KV head.

    f_R, Z_R: softmax attention over the retained rows (Sec. 2 Eq. sub-outputs),
    with log Z_R from a max-shifted sum.  If n_e = 0 the output is f_R.  Otherwise
      s_bar      = q^T k_bar / sqrt(d),        log Z_E_hat = log n_e + s_bar  (Eq. jensen)
      f_E_hat    = v_bar + S_tilde q / (n_e sqrt(d))                          (Eq. fhat)
      log w_R    = log Z_R - logsumexp(log Z_R, log Z_E_hat)                 (App. C.2)
      out        = w_R f_R + (1 - w_R) f_E_hat                               (Eq. fused)
    order = 0 drops the covariance term (zeroth-order variant, f_E_hat = v_bar);
    order = -1 drops the correction altogether (out = f_R, the ablation without it).
    """
    q = _f64(q)
    K = _f64(k_ret)
    V = _f64(v_ret)
    d = q.shape[0]
    if scale is None:
        scale = 1.0 / math.sqrt(d)
    if K.shape[0] == 0 and m.n_e == 0:
        raise ValueError("empty cache and empty summary")
    if K.shape[0] > 0:
        s = scale * (K @ q)
        mx = s.max()
        e = np.exp(s - mx)
        l_sum = e.sum()
        f_R = (e @ V) / l_sum
        log_Z_R = float(mx + math.log(l_sum))
    else:
        f_R = np.zeros(d, F64)
        log_Z_R = -math.inf
    if m.n_e == 0 or order < 0:
        return DecodeResult(f_R, f_R, log_Z_R, 1.0, None, None)
    k_bar, v_bar, S_t = centered_moments(m, tau)
    s_bar = float(scale * (q @ k_bar))
    log_Z_E = math.log(m.n_e) + s_bar
    f_E_hat = v_bar.copy()
    if order >= 1:
        f_E_hat = f_E_hat + (scale / F64(m.n_e)) * (S_t @ q)
    hi = max(log_Z_R, log_Z_E)
    lse = hi + math.log(math.exp(log_Z_R - hi) + math.exp(log_Z_E - hi))
    w_R = math.exp(log_Z_R - lse)
    out = w_R * f_R + (1.0 - w_R) * f_E_hat
    return DecodeResult(out, f_R, log_Z_R, w_R, f_E_hat, log_Z_E)


def append_tokens(k_cache, v_cache, lens, k_new, v_new):
    """Append the new key/value to R (Algorithm 1, before Phase 1), batched, on copies.

    k_cache, v_cache: [B, Hkv, cap, d]; lens: [B, Hkv]; k_new, v_new: [B, Hkv, d].
    Returns (k_cache', v_cache', lens').  Reading: appended tokens join R and no
    eviction runs in the hot path (the summary is frozen after compress).
    """
    kc = _f64(k_cache).copy()
    vc = _f64(v_cache).copy()
    ln = np.asarray(lens, dtype=np.int64).copy()
    B, H = ln.shape
    for b in range(B):
        for h in range(H):
            if ln[b, h] >= kc.shape[2]:
                raise ValueError("cache full")
            kc[b, h, ln[b, h]] = _f64(k_new)[b, h]
            vc[b, h, ln[b, h]] = _f64(v_new)[b, h]
            ln[b, h] += 1
    return kc, vc, ln


def decode(q, k_cache, v_cache, lens, moments, *, k_new=None, v_new=None,
           scale: float | None = None, tau: float = 1e-6, order: int = 1):
    """Batched corrected decode.

    q: [B, Hq, d]; k_cache, v_cache: [B, Hkv, cap, d]; lens: [B, Hkv]; moments: nested
    [B][Hkv] of Moments.  Optional k_new/v_new [B, Hkv, d] are appended first.
    Returns (out [B,Hq,d], log_Z_R [B,Hq], w_R [B,Hq], (k_cache', v_cache', lens')).
    """
    q = _f64(q)
    B, Hq, d = q.shape
    kc, vc, ln = _f64(k_cache), _f64(v_cache), np.asarray(lens, dtype=np.int64)
    if k_new is not None:
        kc, vc, ln = append_tokens(kc, vc, ln, k_new, v_new)
    Hkv = kc.shape[1]
    G = Hq // Hkv
    out = np.zeros((B, Hq, d), F64)
    lz = np.zeros((B, Hq), F64)
    wr = np.zeros((B, Hq), F64)
    for b in range(B):
        for hq in range(Hq):
            h = hq // G
            r = decode_head(q[b, hq], kc[b, h, : ln[b, h]], vc[b, h, : ln[b, h]],
                            moments[b][h], scale=scale, tau=tau, order=order)
            out[b, hq], lz[b, hq], wr[b, hq] = r.out, r.log_Z_R, r.w_R
    return out, lz, wr, (kc, vc, ln)


# --------------------------------------------------------------------------------------
# Diagnostics (Sec. 2 Eqs. sub-outputs/decomposition; Sec. 3 Eqs. eviction_error,
# relative_error).  Exact, using every token; tests only.
# --------------------------------------------------------------------------------------
def attention_parts(q, k, v, retained, scale: float | None = None) -> dict:
    """Exact full output f, sub-outputs f_R, f_E, partition functions and weights."""
    q = _f64(q)
    K = _f64(k)
    V = _f64(v)
    d = q.shape[0]
    if scale is None:
        scale = 1.0 / math.sqrt(d)
    N = K.shape[0]
    R = np.zeros(N, bool)
    R[np.asarray(retained, dtype=np.int64)] = True
    s = scale * (K @ q)
    mx = s.max()
    e = np.exp(s - mx)
    Z, Z_R, Z_E = e.sum(), e[R].sum(), e[~R].sum()
    f = (e @ V) / Z
    f_R = (e[R] @ V[R]) / Z_R if Z_R > 0 else np.zeros(d, F64)
    f_E = (e[~R] @ V[~R]) / Z_E if Z_E > 0 else np.zeros(d, F64)
    nr, ne_ = np.linalg.norm(f_R), np.linalg.norm(f_E)
    cos = float(f_R @ f_E / (nr * ne_)) if nr > 0 and ne_ > 0 else float("nan")
    gamma = float(np.linalg.norm(f_E - f_R) / np.linalg.norm(f))  # since f - f_R = w_E (f_E - f_R)
    return dict(f=f, f_R=f_R, f_E=f_E, w_R=float(Z_R / Z), w_E=float(Z_E / Z),
                log_Z=float(mx + math.log(Z)),
                log_Z_R=float(mx + math.log(Z_R)) if Z_R > 0 else -math.inf,
                log_Z_E=float(mx + math.log(Z_E)) if Z_E > 0 else -math.inf,
                cos_theta=cos, gamma=gamma)


def eviction_diagnostics(q, k, v, retained, *, scale: float | None = None, tau: float = 1e-6,
                         order: int = 1) -> dict:
    """Exact quantities of Sec. 3 and Sec. 4 for one query against one head's full context:
    the evicted weight w_E, cos(theta) between f_E and f_R (Fig. 2), the relative errors
    of f_R and of the corrected output against full attention f (Eq. relative_error), and
    how close the moment estimate is to the evicted output: cos(f_E, f_E_hat) and
    ||f_E_hat - f_E|| / ||f_E|| (Fig. 3).  E is everything not retained; the summary is its
    exact moments.  Diagnostics only (tests)."""
    K = _f64(k)
    V = _f64(v)
    qq = _f64(q)
    d = qq.shape[0]
    if scale is None:
        scale = 1.0 / math.sqrt(d)
    parts = attention_parts(qq, K, V, retained, scale)
    R = np.asarray(retained, dtype=np.int64)
    E = np.setdiff1d(np.arange(K.shape[0]), R)
    m = evicted_moments(K, V, E)
    r = decode_head(qq, K[R], V[R], m, scale=scale, tau=tau, order=order)
    f, f_E = parts["f"], parts["f_E"]
    nf = np.linalg.norm(f)
    out = dict(w_E=parts["w_E"], cos_theta=parts["cos_theta"],
               rel_err_retained=float(np.linalg.norm(parts["f_R"] - f) / nf),
               rel_err_corrected=float(np.linalg.norm(r.out - f) / nf))
    if r.f_E_hat is not None:
        nE, nH = np.linalg.norm(f_E), np.linalg.norm(r.f_E_hat)
        out["cos_fE_fEhat"] = float(f_E @ r.f_E_hat / (nE * nH)) if nE > 0 and nH > 0 else float("nan")
        out["rel_err_fEhat"] = float(np.linalg.norm(r.f_E_hat - f_E) / nE) if nE > 0 else float("nan")
    return out


def greedy_evict(alpha, k, v, protected, budget: int, scale: float | None = None,
                 tau: float = 1e-6):
    """Algorithm 1 Phase 1 applied literally: one eviction at a time (quality reference).

    alpha: [N] fixed per-token attention weights (window mass); protected: positions
    never evicted (sink, window).  While more than `budget` tokens remain, score every
    unprotected retained token by alpha_j ||r_j|| under the current summary, evict the
    argmin (lower index on ties) and add it to the moments by the rank-one update of
    Eq. app_update.  O(N^2 d^2): tiny inputs only.  Returns (retained, Moments).
    """
    K = _f64(k)
    V = _f64(v)
    N, d = K.shape
    if scale is None:
        scale = 1.0 / math.sqrt(d)
    alive = np.ones(N, bool)
    prot = np.zeros(N, bool)
    prot[np.asarray(protected, dtype=np.int64)] = True
    m = Moments.zeros(d)
    while alive.sum() > budget:
        cand = np.nonzero(alive & ~prot)[0]
        score, _ = residual_scores(K, V, _f64(alpha)[cand], cand, m, scale, tau)
        j = int(cand[select_top(-score, 1)[0]])      # lowest score, lower index on ties
        alive[j] = False
        m = Moments(m.n_e + 1, m.s_k + K[j], m.s_v + V[j], m.S + np.outer(V[j], K[j]))
    return np.nonzero(alive)[0], m


# --------------------------------------------------------------------------------------
# Decode-time eviction: Algorithm 1 Phase 1 run at every generated token, then Phase 2
# --------------------------------------------------------------------------------------
def evict_scores_head(q, k, v, m: Moments, *, scale: float, tau: float = 1e-6):
    """Phase 1 scores of every retained row for the current decode query group.

    q: [G, d] queries of the G query heads sharing the KV head; k, v: [n, d] the
    retained rows (the appended token included).  alpha_g = softmax_j(scale q_g^T k_j)
    over the n rows (Algorithm 1, the softmax before the residual loop); with grouped
    queries alpha_j is the mean of the G heads' weights (reading: the same group mean
    as the window mass).  r_j is the moment residual of Sec. 4.2 Eq. residual under the
    current summary, score_j = alpha_j ||r_j|| (low = safe to evict).
    Returns (score, alpha, ||r||), each [n].
    """
    Q = np.atleast_2d(_f64(q))
    K = _f64(k)
    s = scale * (K @ Q.T)                       # [n, G]
    e = np.exp(s - s.max(axis=0, keepdims=True))
    alpha = (e / e.sum(axis=0, keepdims=True)).mean(axis=1)
    r = moment_residuals(K, v, m, scale, tau)
    rn = np.sqrt((r * r).sum(axis=1))
    return alpha * rn, alpha, rn


def decode_evict_head(q, k_cache, v_cache, length: int, k_new, v_new, m: Moments,
                      budget: int, *, scale: float | None = None, tau: float = 1e-6,
                      order: int = 1, forced: int | None = None) -> dict:
    """One decoding step of Algorithm 1 for one KV head and its G query heads.

    1. The new key/value joins R in slot `length` (Algorithm 1, before Phase 1).
    2. Phase 1 (reading: one eviction per call, the loop's single pass when R held at
       most `budget` rows before the append; a cache above `budget` keeps its length):
       if more than `budget` rows are retained,
       score them (evict_scores_head), evict the argmin (the lowest slot among equal
       scores) or the slot `forced`, and fold it into the summary by the rank-one update
       of App. A.1 Eq. app_update.  The last retained row moves into the freed slot
       (R is a set; this fixes the slot layout that a cache in memory keeps).
    3. Phase 2: corrected attention of every query over the new R and summary
       (decode_head).
    k_cache, v_cache: [cap, d] (copied, not modified).  Returns a dict with out [G, d],
    log_Z_R [G], w_R [G], k_cache, v_cache, length, moments (after the step), evicted
    (the slot, or -1) and score / alpha / rnorm over the slots scored (or None).
    """
    Q = np.atleast_2d(_f64(q))
    G, d = Q.shape
    if scale is None:
        scale = 1.0 / math.sqrt(d)
    kc = _f64(k_cache).copy()
    vc = _f64(v_cache).copy()
    if length >= kc.shape[0]:
        raise ValueError("cache full")
    kc[length] = _f64(k_new)
    vc[length] = _f64(v_new)
    n = length + 1
    evicted, score, alpha, rn = -1, None, None, None
    if n > budget:
        score, alpha, rn = evict_scores_head(Q, kc[:n], vc[:n], m, scale=scale, tau=tau)
        evicted = int(np.argmin(score)) if forced is None else int(forced)
        kj, vj = kc[evicted].copy(), vc[evicted].copy()
        m = Moments(m.n_e + 1, m.s_k + kj, m.s_v + vj, m.S + np.outer(vj, kj))
        kc[evicted] = kc[n - 1]
        vc[evicted] = vc[n - 1]
        n -= 1
    out = np.zeros((G, d), F64)
    lz = np.zeros(G, F64)
    wr = np.zeros(G, F64)
    for g in range(G):
        r = decode_head(Q[g], kc[:n], vc[:n], m, scale=scale, tau=tau, order=order)
        out[g], lz[g], wr[g] = r.out, r.log_Z_R, r.w_R
    return dict(out=out, log_Z_R=lz, w_R=wr, k_cache=kc, v_cache=vc, length=n, moments=m,
                evicted=evicted, score=score, alpha=alpha, rnorm=rn)


def decode_evict(q, k_cache, v_cache, lens, moments, k_new, v_new, budget: int, *,
                 scale: float | None = None, tau: float = 1e-6, order: int = 1,
                 forced=None):
    """Batched decode_evict_head over every (sequence, KV head).

    q: [B, Hq, d]; k_cache, v_cache: [B, Hkv, cap, d]; lens: [B, Hkv]; moments: nested
    [B][Hkv] Moments; k_new, v_new: [B, Hkv, d]; forced: optional [B, Hkv] slots to
    evict in place of the argmin (-1 or None entries: the argmin).
    Returns (out [B,Hq,d], log_Z_R [B,Hq], w_R [B,Hq],
             (k_cache', v_cache', lens', moments'), evicted [B,Hkv], per-head dicts).
    """
    Q = _f64(q)
    B, Hq, d = Q.shape
    kc = _f64(k_cache).copy()
    vc = _f64(v_cache).copy()
    ln = np.asarray(lens, dtype=np.int64).copy()
    Hkv = kc.shape[1]
    G = Hq // Hkv
    out = np.zeros((B, Hq, d), F64)
    lz = np.zeros((B, Hq), F64)
    wr = np.zeros((B, Hq), F64)
    ev = np.full((B, Hkv), -1, np.int64)
    mom = [[None] * Hkv for _ in range(B)]
    heads = [[None] * Hkv for _ in range(B)]
    for b in range(B):
        for h in range(Hkv):
            f = None if forced is None or forced[b][h] < 0 else int(forced[b][h])
            r = decode_evict_head(Q[b, h * G:(h + 1) * G], kc[b, h], vc[b, h], int(ln[b, h]),
                                  _f64(k_new)[b, h], _f64(v_new)[b, h], moments[b][h], budget,
                                  scale=scale, tau=tau, order=order, forced=f)
            out[b, h * G:(h + 1) * G] = r["out"]
            lz[b, h * G:(h + 1) * G] = r["log_Z_R"]
            wr[b, h * G:(h + 1) * G] = r["w_R"]
            kc[b, h], vc[b, h], ln[b, h] = r["k_cache"], r["v_cache"], r["length"]
            mom[b][h] = r["moments"]
            ev[b, h] = r["evicted"]
            heads[b][h] = r
    return out, lz, wr, (kc, vc, ln, mom), ev, heads


def moment_storage_bytes(n_layers: int, n_kv_heads: int, head_dim: int,
                         bytes_per_value: int = 2) -> int:
    """Auxiliary storage of the summary: layers x heads x (d^2 + 2d) values (App. A.1)."""
    return n_layers * n_kv_heads * (head_dim * head_dim + 2 * head_dim) * bytes_per_value
