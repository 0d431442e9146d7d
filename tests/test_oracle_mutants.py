"""Planted-mistake check of the oracle's pins (CPU only).

Each case copies the oracle's source, plants one plausible slip (transposed operand,
wrong sign, dropped term, wrong scale, off-by-one mask, wrong tie rule ...), loads the
copy as a separate module and runs the pins of tests/test_oracle_pins.py against it.
At least one pin must fail for every slip; the real oracle is never modified.
"""
import os
import sys
import types

import pytest

import tests.test_oracle_pins as pins

SRC_PATH = os.path.join(os.path.dirname(os.path.dirname(os.path.abspath(__file__))),
                        "oracle", "momentkv.py")
with open(SRC_PATH) as _f:
    SRC = _f.read()

MUTANTS = {
    "S_transposed": ("return Moments(int(e.size), ke.sum(axis=0), ve.sum(axis=0), ve.T @ ke)",
                     "return Moments(int(e.size), ke.sum(axis=0), ve.sum(axis=0), ke.T @ ve)"),
    "centering_outer_transposed": ("S_t = m.S - np.outer(m.s_v, m.s_k) / n",
                                   "S_t = m.S - np.outer(m.s_k, m.s_v) / n"),
    "centering_sign": ("S_t = m.S - np.outer(m.s_v, m.s_k) / n",
                       "S_t = m.S + np.outer(m.s_v, m.s_k) / n"),
    "clamp_relative": ("S_t = np.where(np.abs(S_t) < tau, 0.0, S_t)",
                       "S_t = np.where(np.abs(S_t) <= tau, 0.0, S_t)"),
    "mask_off_by_one": ("visible = np.arange(N)[None, :] <= (N - w + t)[:, None]",
                        "visible = np.arange(N)[None, :] < (N - w + t)[:, None]"),
    "no_causal_mask": ("logits = np.where(visible, logits, -np.inf)", "pass"),
    "mass_not_row_normalised": ("p /= p.sum(axis=1, keepdims=True)", "pass"),
    "chunk_alignment_shift": ("for c0 in range((n_sink // chunk) * chunk, n_cand_end, chunk):",
                              "for c0 in range(n_sink, n_cand_end, chunk):"),
    "ties_keep_higher_index": ("order = np.lexsort((np.arange(s.shape[0]), -s))",
                               "order = np.lexsort((-np.arange(s.shape[0]), -s))"),
    "residual_drops_mean": ("return vv - v_bar[None, :] - (scale / F64(m.n_e)) * (kk @ S_t.T)",
                            "return vv - (scale / F64(m.n_e)) * (kk @ S_t.T)"),
    "residual_transposed_cov": ("return vv - v_bar[None, :] - (scale / F64(m.n_e)) * (kk @ S_t.T)",
                                "return vv - v_bar[None, :] - (scale / F64(m.n_e)) * (kk @ S_t)"),
    "residual_wrong_scale": ("return vv - v_bar[None, :] - (scale / F64(m.n_e)) * (kk @ S_t.T)",
                             "return vv - v_bar[None, :] - (1.0 / F64(m.n_e)) * (kk @ S_t.T)"),
    "decode_cov_sign": ("f_E_hat = f_E_hat + (scale / F64(m.n_e)) * (S_t @ q)",
                        "f_E_hat = f_E_hat - (scale / F64(m.n_e)) * (S_t @ q)"),
    "decode_cov_transposed": ("f_E_hat = f_E_hat + (scale / F64(m.n_e)) * (S_t @ q)",
                              "f_E_hat = f_E_hat + (scale / F64(m.n_e)) * (S_t.T @ q)"),
    "decode_missing_scale": ("f_E_hat = f_E_hat + (scale / F64(m.n_e)) * (S_t @ q)",
                             "f_E_hat = f_E_hat + (1.0 / F64(m.n_e)) * (S_t @ q)"),
    "jensen_missing_count": ("log_Z_E = math.log(m.n_e) + s_bar", "log_Z_E = s_bar"),
    "jensen_unscaled_mean_logit": ("s_bar = float(scale * (q @ k_bar))", "s_bar = float(q @ k_bar)"),
    "mix_weights_swapped": ("out = w_R * f_R + (1.0 - w_R) * f_E_hat",
                            "out = (1.0 - w_R) * f_R + w_R * f_E_hat"),
    "provisional_score_unweighted": ("sigma0 = _f64(abar) * vnorm", "sigma0 = vnorm"),
    "moment_round_uses_retained": ("evicted = np.setdiff1d(everyone, kept)",
                                   "evicted = kept"),
    "moment_round_skipped": ("kept = np.sort(select_top(sigma, k_keep))", "pass"),
    "evict_softmax_over_queries": ("alpha = (e / e.sum(axis=0, keepdims=True)).mean(axis=1)",
                                   "alpha = (e / e.sum(axis=1, keepdims=True)).mean(axis=1)"),
    "evict_alpha_max_not_mean": ("alpha = (e / e.sum(axis=0, keepdims=True)).mean(axis=1)",
                                 "alpha = (e / e.sum(axis=0, keepdims=True)).max(axis=1)"),
    "evict_score_unweighted": ("return alpha * rn, alpha, rn", "return rn, alpha, rn"),
    "evict_argmax": ("evicted = int(np.argmin(score)) if forced is None else int(forced)",
                     "evicted = int(np.argmax(score)) if forced is None else int(forced)"),
    "evict_update_outer_swapped": ("m = Moments(m.n_e + 1, m.s_k + kj, m.s_v + vj, m.S + np.outer(vj, kj))",
                                   "m = Moments(m.n_e + 1, m.s_k + kj, m.s_v + vj, m.S + np.outer(kj, vj))"),
    "evict_update_no_count": ("m = Moments(m.n_e + 1, m.s_k + kj, m.s_v + vj, m.S + np.outer(vj, kj))",
                              "m = Moments(m.n_e, m.s_k + kj, m.s_v + vj, m.S + np.outer(vj, kj))"),
    "evict_no_slot_move": ("        kc[evicted] = kc[n - 1]\n", "\n"),
    "evict_at_budget": ("    if n > budget:\n", "    if n >= budget:\n"),
    "no_correction_ignored": ("    if m.n_e == 0 or order < 0:", "    if m.n_e == 0:"),
    "head_budget_ties_reversed": ("    order = np.lexsort((np.arange(flat.size), -flat))[:keep]",
                                  "    order = np.lexsort((-np.arange(flat.size), -flat))[:keep]"),
    "decode_head_modulo": ("            h = hq // G\n", "            h = hq % Hkv\n"),
    "compress_strided_group": (
        "return [[compress_head(q[b, h * G:(h + 1) * G], K[b, h], V[b, h], budget, **kw)",
        "return [[compress_head(q[b, h::Hkv], K[b, h], V[b, h], budget, **kw)"),
    "decode_evict_strided_group": (
        "r = decode_evict_head(Q[b, h * G:(h + 1) * G], kc[b, h], vc[b, h], int(ln[b, h]),",
        "r = decode_evict_head(Q[b, h::Hkv], kc[b, h], vc[b, h], int(ln[b, h]),"),
    "head_budget_lowest_mass": ("    order = np.lexsort((np.arange(flat.size), -flat))[:keep]",
                                "    order = np.lexsort((np.arange(flat.size), flat))[:keep]"),
}

PIN_TESTS = [name for name in dir(pins) if name.startswith("test_")]


def _load(old, new):
    assert SRC.count(old) == 1, f"mutation anchor not unique: {old!r}"
    name = "oracle_mutant"
    mod = types.ModuleType(name)
    mod.__file__ = SRC_PATH
    sys.modules[name] = mod
    try:
        exec(compile(SRC.replace(old, new), SRC_PATH, "exec"), mod.__dict__)
    finally:
        del sys.modules[name]
    return mod


def _run_pins(monkeypatch):
    """Run every pin (all parametrisations); return the names that failed."""
    failed = []
    for name in PIN_TESTS:
        fn = getattr(pins, name)
        marks = getattr(fn, "pytestmark", [])
        cases = [()]
        for m in marks:
            if m.name == "parametrize":
                cases = list(m.args[1])
        for case in cases:
            args = case if isinstance(case, tuple) else (case,)
            try:
                fn(*args)
            except Exception:          # noqa: BLE001 - any failure counts as caught
                failed.append(name)
                break
    return failed


def test_real_oracle_passes_all_pins(monkeypatch):
    assert _run_pins(monkeypatch) == []


@pytest.mark.parametrize("mutant", sorted(MUTANTS))
def test_planted_mistake_is_caught(monkeypatch, mutant):
    old, new = MUTANTS[mutant]
    monkeypatch.setattr(pins, "O", _load(old, new))
    assert _run_pins(monkeypatch), f"no pin caught the planted mistake {mutant}"
