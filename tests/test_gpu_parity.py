"""GPU parity of the HIP path against the fp64 oracle (through the C ABI).

Inputs are the seeded synthetic workloads; the oracle consumes host copies of exactly
the bits the GPU consumed.  Sizes are small enough for the oracle to finish in seconds
while spanning many 64-token tiles and a ragged tail; the full-size cases check sampled
heads.  See tests/parity_util.py for the protocol and tolerances.
"""
import math
import types

import numpy as np
import pytest
import torch

import oracle as O
from paper_2606_01563_amd import synth
from paper_2606_01563_amd import momentkv as mk
from tests import parity_util as P

pytestmark = pytest.mark.gpu


def layer(name, layer_idx=0, steps=None, **over):
    wl = synth.WORKLOADS[name]
    if over:
        wl = synth.shrink(wl, **over)
    cpu = synth.make_layer(wl, layer_idx, device="cpu", decode_steps=steps)
    gpu = {k: v.cuda() for k, v in cpu.items()}
    return wl, cpu, gpu


def announce(msg):
    print(f"[parity] {msg}", flush=True)


# ---------------------------------------------------------------- tiny fp32 workload
def test_tiny_fp32_compress_and_decode():
    wl, cpu, gpu = layer("tiny_fp32_n2048", steps=16)
    L = wl.budgets[0]
    announce(f"{wl.name} compress L={L}")
    out = P.run_compress(gpu, L, cap=L + 16)
    errs = P.check_compress_head(cpu, out, 0, 0, L)
    announce(f"errors {errs}")
    assert errs["swaps"] == 0 and errs["swaps0"] == 0
    worst = P.run_decode_steps(gpu, out, 16)
    announce(f"decode worst rel err {max(worst):.2e}")


def test_llama_layer_bf16_compress_and_decode():
    wl, cpu, gpu = layer("llama31_8b_layer_n8192", steps=24)
    L = wl.budgets[0]
    announce(f"{wl.name} compress L={L}")
    out = P.run_compress(gpu, L, cap=L + 24)
    for h in range(wl.n_kv_heads):
        errs = P.check_compress_head(cpu, out, 0, h, L)
        announce(f"head {h} errors {errs}")
    worst = P.run_decode_steps(gpu, out, 24)
    announce(f"decode worst rel err {max(worst):.2e}")


@pytest.mark.parametrize("n_split", [1, 2, 5, 0])
def test_decode_slice_counts(n_split):
    """The single-launch path (one workgroup per KV head), explicit slice counts and the
    automatic choice give the same results as the oracle."""
    wl, cpu, gpu = layer("llama31_8b_layer_n8192", steps=3, ctx_len=3000, batch=2)
    out = P.run_compress(gpu, 400, cap=403)
    P.run_decode_steps(gpu, out, 3, n_split=n_split)


@pytest.mark.parametrize("n_split", [1, 3])
@pytest.mark.parametrize("G", [8, 16])
def test_decode_large_query_groups(G, n_split):
    """G = 8 and 16 query heads per KV head, more queries than the four waves of a
    workgroup: the single launch and three slices, with appends over several steps (each
    query of a head must see the length from before the step's append)."""
    wl, cpu, gpu = layer("tiny_fp32_n2048", steps=3, dtype=torch.bfloat16, head_dim=128,
                         ctx_len=1000, batch=2, n_q_heads=2 * G, n_kv_heads=2, window=16,
                         budgets=(97,))
    out = P.run_compress(gpu, 97, cap=100)
    announce(f"G={G} n_split={n_split}")
    P.run_decode_steps(gpu, out, 3, n_split=n_split, summary=1)


@pytest.mark.parametrize("n_split", [1, 3])
@pytest.mark.parametrize("dtype", [torch.float32, torch.bfloat16])
def test_bf16_moment_storage(dtype, n_split):
    """Moments stored in 16 bits (App. C.2): compress with moment_dtype bf16 writes the
    fp32 sum rounded once to bf16 (bit for bit torch's round-to-nearest-even cast of the
    fp32 output of the same call, every other output unchanged; against the oracle's
    brute-force sum over the evicted set, within the bf16 unit roundoff 2^-8 of each entry
    plus the probabilistic fp32 summation bound 8 sqrt(n) 2^-24 sum |v_a k_b|),
    and the decode reading that raw bf16 S (summary 3, centred in fp32) matches the oracle
    fed the same bf16 values, through appends."""
    wl, cpu, gpu = layer("tiny_fp32_n2048", steps=3, dtype=dtype, head_dim=128, ctx_len=1500,
                         batch=2, n_q_heads=8, n_kv_heads=2, window=16, budgets=(97,))
    ref = P.run_compress(gpu, 97, cap=100)
    out = P.run_compress(gpu, 97, cap=100, moment_dtype=torch.bfloat16)
    assert out.S.dtype == torch.bfloat16
    assert torch.equal(out.S, ref.S.to(torch.bfloat16))
    for f in ("idx", "lens", "n_e", "s_k", "s_v"):
        assert torch.equal(getattr(out, f), getattr(ref, f)), f
    # rows past lens are unwritten (the outputs were allocated uninitialised)
    assert torch.equal(out.k_out[:, :, :97], ref.k_out[:, :, :97])
    assert torch.equal(out.v_out[:, :, :97], ref.v_out[:, :, :97])
    for b in range(2):
        for h in range(2):
            n_out = int(out.lens[b, h])
            idx = out.idx[b, h, :n_out].cpu().numpy()
            K, V = P.h64(cpu["k"][b, h]), P.h64(cpu["v"][b, h])
            ev = np.setdiff1d(np.arange(K.shape[0]), idx)
            exact = O.evicted_moments(K, V, ev).S
            got = P.h64(out.S[b, h])
            sum_abs = np.abs(V[ev]).T @ np.abs(K[ev])
            delta = 8.0 * math.sqrt(len(ev)) * 2.0 ** -24 * sum_abs
            bound = 2.0 ** -8 * np.abs(exact) + (1 + 2.0 ** -8) * delta
            assert bool(np.all(np.abs(got - exact) <= bound)), (b, h, float(np.max(np.abs(got - exact) / bound)))
    announce(f"{dtype} n_split={n_split}: bf16 S within its rounding bound")
    worst = P.run_decode_steps(gpu, out, 3, n_split=n_split, summary=3)
    announce(f"decode from bf16 raw moments, worst rel err {max(worst):.2e}")


def test_split_decode_repeats_bit_exact_and_leaves_counters_at_zero():
    """The split shape merges each head in the launch (the last slice to finish): 24
    repeated calls on the same inputs give the same bits whichever wave merged, the
    per-head arrival counters are back at zero after every call, the result agrees with
    the single-workgroup shape, and a workspace first used by a call with fewer heads
    serves a call with more (its extra counter bytes are zeroed by the binding)."""
    g = torch.Generator(device="cuda").manual_seed(7)
    B, Hkv, G, d, cap = 36, 8, 4, 128, 700
    kc = torch.randn(B, Hkv, cap, d, device="cuda", generator=g).to(torch.bfloat16)
    vc = torch.randn(B, Hkv, cap, d, device="cuda", generator=g).to(torch.bfloat16)
    q = torch.randn(B, Hkv * G, d, device="cuda", generator=g).to(torch.bfloat16)
    lens = torch.randint(0, cap + 1, (B, Hkv), device="cuda", generator=g, dtype=torch.int32)
    n_e = torch.randint(0, 5000, (B, Hkv), device="cuda", generator=g, dtype=torch.int32)
    s_k = torch.randn(B, Hkv, d, device="cuda", generator=g) * 30
    s_v = torch.randn(B, Hkv, d, device="cuda", generator=g) * 30
    S = torch.randn(B, Hkv, d, d, device="cuda", generator=g) * 50
    args = (q, kc, vc, lens, n_e, s_k, s_v, S)
    small = tuple(t[:2] for t in args)
    for n_split in (3, 0):
        ws = mk.momentkv_decode_attn(*small, max_len=cap, n_split=n_split)[3]
        ref = None
        for rep in range(24):
            o, lse, w, ws = mk.momentkv_decode_attn(*args, max_len=cap, n_split=n_split,
                                                    lse=torch.empty(B, Hkv * G, device="cuda"),
                                                    w_r=torch.empty(B, Hkv * G, device="cuda"),
                                                    workspace=ws)
            if ref is None:
                ref = (o.clone(), lse.clone(), w.clone())
            else:
                assert torch.equal(o, ref[0]) and torch.equal(lse, ref[1]) and torch.equal(w, ref[2]), rep
            cnt = ws[256:256 + 4 * B * Hkv].view(torch.int32)
            assert int(cnt.abs().sum()) == 0, rep
        one, lse1, w1, _ = mk.momentkv_decode_attn(*args, max_len=cap, n_split=1,
                                                   lse=torch.empty(B, Hkv * G, device="cuda"),
                                                   w_r=torch.empty(B, Hkv * G, device="cuda"))
        rel = (one.float() - ref[0].float()).norm(dim=-1) / one.float().norm(dim=-1).clamp_min(1e-30)
        announce(f"n_split={n_split}: split vs single workgroup, max rel {float(rel.max()):.2e}")
        assert float(rel.max()) < 2e-2
        finite = torch.isfinite(lse1)
        assert torch.equal(finite, torch.isfinite(ref[1]))
        assert float((lse1[finite] - ref[1][finite]).abs().max()) < 1e-4
        assert float((w1 - ref[2]).abs().max()) < 1e-4


@pytest.mark.parametrize("append", [True, False])
@pytest.mark.parametrize("n_split", [0, 3, 4])
@pytest.mark.parametrize("dtype", [torch.float32, torch.bfloat16])
def test_decode_varied_lengths_and_slice_boundaries(dtype, n_split, append):
    """Per-head retained lengths 0, 31, 32, 33, 64 and 65: an empty retained set, a ragged
    first block, and appends landing on the first row of a block (single launch, n_split
    0 here) or of a 64- or 32-row slice (n_split 3, 4: that slice writes the row and
    attends to nothing; the next step reads the row back)."""
    wl, cpu, gpu = layer("tiny_fp32_n2048", steps=3, dtype=dtype, head_dim=128, ctx_len=1000,
                         batch=3, n_q_heads=4, n_kv_heads=2, window=16, budgets=(97,))
    out = P.run_compress(gpu, 97, cap=100)
    lens0 = [[0, 31], [32, 33], [64, 65]]
    announce(f"lengths {lens0} {dtype} n_split={n_split} append={append}")
    P.run_decode_steps(gpu, out, 3, n_split=n_split, append=append, lens0=lens0,
                       summary=int(append))


@pytest.mark.parametrize("cap", [128, 300])
@pytest.mark.parametrize("dtype", [torch.float32, torch.bfloat16])
@pytest.mark.parametrize("d", [64, 128])
def test_decode_single_launch_block_rounds(d, dtype, cap):
    """The single launch (one 4-wave workgroup per KV head) at per-head lengths on both
    sides of the 4- and 8-block boundaries (one, two or three 32-row blocks per wave), an
    empty head, appends, prepared summary."""
    L = cap - 3
    wl, cpu, gpu = layer("tiny_fp32_n2048", steps=3, dtype=dtype, head_dim=d, ctx_len=1000,
                         batch=3, n_q_heads=4, n_kv_heads=2, window=16, budgets=(L,))
    out = P.run_compress(gpu, L, cap=cap)
    lens0 = ([[0, 31], [95, 96], [124, 125]] if cap == 128
             else [[0, 127], [128, 160], [255, 297]])
    announce(f"single launch d={d} {dtype} cap={cap} lengths {lens0}")
    P.run_decode_steps(gpu, out, 3, n_split=1, lens0=lens0, summary=1)


# ---------------------------------------------------------------- edge cases
@pytest.mark.parametrize("summary", [0, 1])
@pytest.mark.parametrize("dtype", [torch.float32, torch.bfloat16])
@pytest.mark.parametrize("d", [64, 128])
def test_ragged_shapes_and_both_head_dims(dtype, d, summary):
    """N not a multiple of 64, batch 2, GQA 2, both head dims and dtypes, raw and prepared
    summary."""
    wl, cpu, gpu = layer("tiny_fp32_n2048", steps=3, dtype=dtype, head_dim=d, ctx_len=1000,
                         batch=2, n_q_heads=4, n_kv_heads=2, window=16, budgets=(97,))
    announce(f"ragged d={d} {dtype} summary={summary}")
    out = P.run_compress(gpu, 97, cap=100)
    for b in range(2):
        for h in range(2):
            P.check_compress_head(cpu, out, b, h, 97)
    P.run_decode_steps(gpu, out, 3, summary=summary)
    P.run_decode_steps(gpu, out, 2, summary=summary, n_split=2)


@pytest.mark.parametrize("q_scale", [1.0, 12.0])
def test_window_rows_not_a_multiple_of_16(q_scale):
    """G = 3 and a window of 7 give 21 window rows per KV head: the second 16-row tile is
    mostly padding.  With the queries scaled up, the window logits reach hundreds, so a
    padded row that repeated the last real row could overflow exp in the window mass; the
    masses, selections and moments must still follow the oracle."""
    wl, cpu, gpu = layer("tiny_fp32_n2048", steps=1, ctx_len=900, n_q_heads=6, n_kv_heads=2,
                         window=7, budgets=(60,))
    cpu["q_win"] = cpu["q_win"] * q_scale
    gpu["q_win"] = cpu["q_win"].cuda()
    out = P.run_compress(gpu, 60, cap=60)
    assert torch.isfinite(out.abar).all() and torch.isfinite(out.score0).all()
    for h in range(2):
        P.check_compress_head(cpu, out, 0, h, 60)


@pytest.mark.parametrize("mi_rounds", [-1, 0, 1])
@pytest.mark.parametrize("chunk", [1, 4, 8])
def test_selection_modes_and_chunks(mi_rounds, chunk):
    wl, cpu, gpu = layer("tiny_fp32_n2048", steps=1, ctx_len=700, budgets=(80,))
    out = P.run_compress(gpu, 80, chunk=chunk, mi_rounds=mi_rounds)
    P.check_compress_head(cpu, out, 0, 0, 80, chunk=chunk, mi_rounds=mi_rounds)


@pytest.mark.parametrize("mi_rounds,budget", [(2, 97), (3, 97), (8, 97), (2, 950)])
@pytest.mark.parametrize("dtype", [torch.float32, torch.bfloat16])
def test_several_moment_rounds(dtype, mi_rounds, budget):
    """mi_rounds > 1: each round scores with the moments of the round before's evicted set
    (k_reduce, k_residual and the selection repeated); the final scores, kept set and
    moments against the oracle's rounds.  Budget 950 of 1000 evicts fewer candidates than
    it keeps, so every round sums the evicted rows directly."""
    wl, cpu, gpu = layer("tiny_fp32_n2048", steps=1, dtype=dtype, head_dim=128, ctx_len=1000,
                         batch=1, n_q_heads=4, n_kv_heads=2, window=16, budgets=(budget,))
    announce(f"mi_rounds={mi_rounds} budget={budget} {dtype}")
    out = P.run_compress(gpu, budget, cap=budget, mi_rounds=mi_rounds)
    for h in range(2):
        errs = P.check_compress_head(cpu, out, 0, h, budget, mi_rounds=mi_rounds)
        announce(f"head {h} {errs}")
    if mi_rounds == 2 and budget == 97:
        # on this input the first moment round changes the kept set of both heads, so the
        # second round scores with other moments than the first did
        one = P.run_compress(gpu, budget, cap=budget, mi_rounds=1)
        assert not torch.equal(one.score, out.score)


def test_budget_equal_to_protected_tokens_evicts_every_candidate():
    wl, cpu, gpu = layer("tiny_fp32_n2048", steps=2, ctx_len=300)
    L = 1 + wl.window
    out = P.run_compress(gpu, L, cap=L + 2)
    P.check_compress_head(cpu, out, 0, 0, L)
    assert int(out.n_e[0, 0]) == 300 - L
    P.run_decode_steps(gpu, out, 2)


@pytest.mark.parametrize("budget", [300, 5000])
def test_budget_at_least_context_keeps_everything(budget):
    wl, cpu, gpu = layer("tiny_fp32_n2048", steps=2, ctx_len=300)
    out = P.run_compress(gpu, budget, cap=302)
    P.check_compress_head(cpu, out, 0, 0, budget)
    P.run_decode_steps(gpu, out, 2)  # n_e = 0: plain softmax attention


def test_long_window_group_rows_256():
    """G * w = 256 window rows (the 128K workload's window of 64)."""
    wl, cpu, gpu = layer("ruler_n131072", steps=2, ctx_len=3000, budgets=(200,),
                         n_q_heads=8, n_kv_heads=2)
    out = P.run_compress(gpu, 200, cap=202)
    for h in range(2):
        P.check_compress_head(cpu, out, 0, h, 200)
    P.run_decode_steps(gpu, out, 2)


@pytest.mark.parametrize("dtype", [torch.float32, torch.bfloat16])
@pytest.mark.parametrize("budget", [8100, 33 + 4080, 33 + 4079])
def test_budget_close_to_context_sums_the_evicted_rows(dtype, budget):
    """A budget close to the context evicts few candidates (92 of 8159 at 8100): the
    moments are then summed over the evicted rows themselves, which are fewer than the kept
    ones, so they stay within 1e-5 however small n_e is (the candidates' sums minus the
    kept rows' would lose about n_c / n_e times more).  Both sides of the switch: 4079
    evicted against 4080 kept (direct) and 4080 against 4079 (subtracted)."""
    wl, cpu, gpu = layer("llama31_8b_layer_n8192", steps=2, n_q_heads=8, n_kv_heads=2,
                         dtype=dtype)
    announce(f"budget {budget} of {wl.ctx_len} {dtype}")
    out = P.run_compress(gpu, budget, cap=budget + 2)
    for h in range(2):
        errs = P.check_compress_head(cpu, out, 0, h, budget)
        announce(f"head {h}: n_e {int(out.n_e[0, h])} S rel err {errs['S']:.2e}")
    P.run_decode_steps(gpu, out, 2)


@pytest.mark.parametrize("order", [0, -1])
def test_zeroth_order_or_no_correction_decode_and_no_append(order):
    wl, cpu, gpu = layer("tiny_fp32_n2048", steps=3, ctx_len=600, budgets=(64,))
    out = P.run_compress(gpu, 64, cap=64)
    P.run_decode_steps(gpu, out, 3, order=order, append=False)


def test_ablations_correction_lowers_error_against_full_attention():
    """Synthetic analog of the component ablation (Sec. 5.3): for the SnapKV-style selection
    (mi_rounds = -1) and the moment-informed one (mi_rounds = 1), the corrected decode
    (order 1) is closer to exact attention over the whole context than the uncorrected one
    (order -1), averaged over the queries; the errors of all four are reported."""
    wl, cpu, gpu = layer("llama31_8b_layer_n8192", steps=4)
    L = 128
    N, d = wl.ctx_len, wl.head_dim
    G = wl.group
    errs = {}
    for mi in (-1, 1):
        out = P.run_compress(gpu, L, cap=L, mi_rounds=mi)
        for order in (-1, 1):
            e = []
            for t in range(4):
                q = gpu["q_dec"][t]
                res, _, _, _ = mk.momentkv_decode_attn(q, out.k_out, out.v_out, out.lens, out.n_e,
                                                       out.s_k, out.s_v, out.S, order=order,
                                                       max_len=L)
                # exact attention over all N prefill rows (fp32; the group's KV head)
                kf = gpu["k"][0].float()
                vf = gpu["v"][0].float()
                qf = q[0].float().view(wl.n_kv_heads, G, d)
                s = torch.matmul(qf, kf.transpose(1, 2).contiguous()) / math.sqrt(d)
                full = torch.matmul(torch.softmax(s, -1), vf).reshape(-1, d)
                e.append(float(((res[0].float() - full).norm(dim=-1) / full.norm(dim=-1)).mean()))
            errs[(mi, order)] = sum(e) / len(e)
    announce("mean rel err vs full attention " +
             ", ".join(f"mi={k[0]} order={k[1]}: {v:.4f}" for k, v in sorted(errs.items())))
    for mi in (-1, 1):
        assert errs[(mi, 1)] < errs[(mi, -1)]


def test_append_into_full_cache_sets_flag_and_skips():
    wl, cpu, gpu = layer("tiny_fp32_n2048", steps=1, ctx_len=400, budgets=(64,))
    out = P.run_compress(gpu, 64, cap=64)
    lens_before = out.lens.clone()
    res, _, _, ws = mk.momentkv_decode_attn(
        gpu["q_dec"][0], out.k_out, out.v_out, out.lens, out.n_e, out.s_k, out.s_v, out.S,
        k_new=gpu["k_new"][0], v_new=gpu["v_new"][0], max_len=64)
    torch.cuda.synchronize()
    assert int(ws[:4].view(torch.int32)[0]) == 1
    assert torch.equal(out.lens, lens_before)
    m = [[P.oracle_moments(out, 0, 0)]]
    ref, _, _, _ = O.decode(P.h64(gpu["q_dec"][0]), P.h64(out.k_out), P.h64(out.v_out),
                            out.lens.cpu().numpy(), m)
    assert P.rel_l2(P.h64(res)[0, 0], ref[0, 0]) <= 1e-5


def test_compress_and_decode_are_bit_deterministic():
    wl, cpu, gpu = layer("llama31_8b_layer_n8192", steps=1, ctx_len=4000)
    a = P.run_compress(gpu, 300, cap=301)
    b = P.run_compress(gpu, 300, cap=301)
    for f in ("idx", "lens", "n_e", "s_k", "s_v", "S", "abar", "score0", "score", "kept0"):
        assert torch.equal(getattr(a, f), getattr(b, f)), f
    # rows past lens are unwritten (the outputs were allocated uninitialised)
    assert torch.equal(a.k_out[:, :, :300], b.k_out[:, :, :300])
    assert torch.equal(a.v_out[:, :, :300], b.v_out[:, :, :300])
    outs = []
    for c in (a, b):
        o, _, _, _ = mk.momentkv_decode_attn(gpu["q_dec"][0], c.k_out, c.v_out, c.lens, c.n_e,
                                             c.s_k, c.s_v, c.S, k_new=gpu["k_new"][0],
                                             v_new=gpu["v_new"][0], max_len=301)
        outs.append(o)
    torch.cuda.synchronize()
    assert torch.equal(outs[0], outs[1])


@pytest.mark.parametrize("ctx_len", [12000, 33000])
@pytest.mark.parametrize("mi_rounds", [-1, 0])
def test_selection_with_all_scores_equal_keeps_the_lowest_positions(ctx_len, mi_rounds):
    """Every candidate score equal (identical candidate keys give equal window masses;
    zero values give zero scores): the kept set is the k lowest candidate positions, the
    tie rule of the selection.  Both sizes put more keys in the k-th key's bin than the
    refinement stages in LDS (it then reads them from global memory), over 6 and 17
    slices of 2048 positions."""
    wl, cpu, gpu = layer("tiny_fp32_n2048", steps=1, ctx_len=ctx_len, budgets=(200,))
    n_s, budget = 4, 200  # candidates start and end on chunk boundaries: no short chunk
    c_hi = ctx_len - wl.window
    k = cpu["k"].clone()
    k[0, 0, n_s:c_hi] = k[0, 0, 5]
    v = cpu["v"].clone()
    if mi_rounds == 0:
        v[0, 0, n_s:c_hi] = 0.0  # ||v_j|| = 0: every provisional score is 0
    gpu["k"], gpu["v"] = k.cuda(), v.cuda()
    out = P.run_compress(gpu, budget, cap=budget, mi_rounds=mi_rounds, n_sink=n_s)
    k_keep = budget - n_s - wl.window
    first = (out.abar if mi_rounds < 0 else out.score0)[0, 0].cpu().numpy()
    assert np.all(first == first[0])
    expect = np.arange(n_s, n_s + k_keep)
    idx = out.idx[0, 0].cpu().numpy()
    np.testing.assert_array_equal(idx[n_s:n_s + k_keep], expect)
    np.testing.assert_array_equal(out.kept0[0, 0, :k_keep].cpu().numpy(), expect)
    assert int(out.n_e[0, 0]) == c_hi - n_s - k_keep


def test_zero_key_spread_decode_equals_full_attention_on_gpu():
    """Paper invariant end to end: with every candidate key equal, the corrected decode
    output equals full attention over all N tokens (Sec. 4.2, App. B.2)."""
    wl, cpu, gpu = layer("tiny_fp32_n2048", steps=1, ctx_len=500, budgets=(100,))
    k = cpu["k"].clone()
    k[0, 0, 1:500 - wl.window] = k[0, 0, 7]
    cpu["k"] = k
    gpu["k"] = k.cuda()
    out = P.run_compress(gpu, 100, cap=100)
    res, _, _, _ = mk.momentkv_decode_attn(gpu["q_dec"][0], out.k_out, out.v_out, out.lens,
                                           out.n_e, out.s_k, out.s_v, out.S, max_len=100)
    torch.cuda.synchronize()
    q = P.h64(cpu["q_dec"][0])[0]
    K, V = P.h64(k)[0, 0], P.h64(cpu["v"])[0, 0]
    full = np.stack([O.attention_parts(q[g], K, V, np.arange(500))["f"] for g in range(4)])
    assert P.rel_l2(P.h64(res)[0], full) <= 1e-5


@pytest.mark.parametrize("dtype", [torch.float32, torch.bfloat16])
@pytest.mark.parametrize("d", [64, 128])
def test_prepared_summary_matches_centred_clamped_covariance(dtype, d):
    """momentkv_prepare_summary against the oracle's S_tilde from the same fp32 moments: the
    fp32 centring error (a few ulp of |S| + |s_v s_k^T| / n_e), the bf16 hi + lo split
    (2^-16 of |S_tilde|) and, for entries within that of tau, the clamp decision."""
    wl, cpu, gpu = layer("tiny_fp32_n2048", steps=1, dtype=dtype, head_dim=d, ctx_len=1500,
                         batch=2, n_q_heads=4, n_kv_heads=2, window=16, budgets=(97,))
    out = P.run_compress(gpu, 97, cap=97)
    prep = mk.momentkv_prepare_summary(out.n_e, out.s_k, out.s_v, out.S, dtype=dtype)
    torch.cuda.synchronize()
    if dtype == torch.bfloat16:
        got = P.h64(prep[:, :, 0]) + P.h64(prep[:, :, 1])
    else:
        got = P.h64(prep)
    tau = 1e-6
    for b in range(2):
        for h in range(2):
            m = P.oracle_moments(out, b, h)
            _, _, ref = O.centered_moments(m, tau)
            S, sv, sk = P.h64(out.S[b, h]), P.h64(out.s_v[b, h]), P.h64(out.s_k[b, h])
            bound = (2.0 ** -16 * np.abs(ref) + 2.0 ** -21 * (np.abs(S) + np.abs(np.outer(sv, sk)) / m.n_e)
                     + 2 * tau)
            err = np.abs(got[b, h] - ref)
            assert np.all(err <= bound), float(np.max(err / bound))
            assert np.any(ref != 0)


def test_half_precision_summary_is_rounded_covariance():
    """The one-plane form is RNE_bf16 of the fp32-centred S_tilde: within half a bf16 ulp
    (8 significant bits: 2^-8 of |S_tilde|) plus the centring error and the clamp band."""
    wl, cpu, gpu = layer("tiny_fp32_n2048", steps=1, dtype=torch.bfloat16, head_dim=128,
                         ctx_len=1500, batch=2, n_q_heads=4, n_kv_heads=2, window=16,
                         budgets=(97,))
    out = P.run_compress(gpu, 97, cap=97)
    half = mk.momentkv_prepare_summary(out.n_e, out.s_k, out.s_v, out.S, dtype=torch.bfloat16,
                                       half=True)
    full = mk.momentkv_prepare_summary(out.n_e, out.s_k, out.s_v, out.S, dtype=torch.bfloat16)
    torch.cuda.synchronize()
    assert half.shape == (2, 2, 128, 128)
    assert torch.equal(half, full[:, :, 0])           # the hi plane of the two-plane form
    got = P.h64(half)
    for b in range(2):
        for h in range(2):
            m = P.oracle_moments(out, b, h)
            _, _, ref = O.centered_moments(m, 1e-6)
            S, sv, sk = P.h64(out.S[b, h]), P.h64(out.s_v[b, h]), P.h64(out.s_k[b, h])
            bound = (2.0 ** -8 * np.abs(ref) + 2.0 ** -21 * (np.abs(S) + np.abs(np.outer(sv, sk)) / m.n_e)
                     + 2e-6)
            assert np.all(np.abs(got[b, h] - ref) <= bound)


@pytest.mark.parametrize("n_split", [1, 0])
def test_decode_with_half_precision_summary(n_split):
    wl, cpu, gpu = layer("llama31_8b_layer_n8192", steps=3, ctx_len=3000, batch=2)
    out = P.run_compress(gpu, 400, cap=403)
    P.run_decode_steps(gpu, out, 3, n_split=n_split, summary=2)


def test_half_precision_summary_error_against_fp32_summary():
    """Synthetic analog of the paper's FP16-vs-FP32 moment comparison (App. C.2): one 32K
    layer at budget 128, where the summary is the largest share of the decode.  Against the
    oracle and against exact full attention, the half-precision summary's extra error is
    small next to the approximation error itself."""
    wl, cpu, gpu = layer("qwen3_4b_stack_n32768", steps=2)
    L = 128
    out = P.run_compress(gpu, L, cap=L)
    d, G = wl.head_dim, wl.group
    moments = [[P.oracle_moments(out, 0, h) for h in range(wl.n_kv_heads)]]
    kf, vf = gpu["k"][0].float(), gpu["v"][0].float()
    res = {}
    for summ in (1, 2):
        S_arg = mk.momentkv_prepare_summary(out.n_e, out.s_k, out.s_v, out.S, dtype=torch.bfloat16,
                                            half=summ == 2)
        e_orc, e_full = [], []
        for t in range(2):
            q = gpu["q_dec"][t]
            got, _, _, _ = mk.momentkv_decode_attn(q, out.k_out, out.v_out, out.lens, out.n_e, out.s_k,
                                                   out.s_v, S_arg, max_len=L, summary=summ)
            ref, _, _, _ = O.decode(P.h64(q), P.h64(out.k_out), P.h64(out.v_out),
                                    out.lens.cpu().numpy(), moments)
            g64 = P.h64(got)
            e_orc.append(max(P.rel_l2(g64[0, i], ref[0, i]) for i in range(wl.n_q_heads)))
            qf = q[0].float().view(wl.n_kv_heads, G, d)
            s = torch.matmul(qf, kf.transpose(1, 2).contiguous()) / math.sqrt(d)
            full = torch.matmul(torch.softmax(s, -1), vf).reshape(-1, d)
            e_full.append(float(((got[0].float() - full).norm(dim=-1) / full.norm(dim=-1)).mean()))
        res[summ] = (max(e_orc), sum(e_full) / len(e_full))
    announce(f"two-plane summary: max rel err vs oracle {res[1][0]:.2e}, vs full attention "
             f"{res[1][1]:.4f}; half precision: {res[2][0]:.2e}, {res[2][1]:.4f}")
    assert res[2][0] <= 2e-2
    assert abs(res[2][1] - res[1][1]) <= 0.05 * res[1][1]


# ---------------------------------------------------------------- full-size sampled heads
@pytest.mark.parametrize("budget", [128, 256, 512, 1024, 2048])
def test_qwen_stack_layer_full_size_sampled_heads(budget):
    """One 32K-context layer of the Qwen3-4B-shaped stack at every budget of the stack
    workload, checked on two sampled KV heads; then decode in the benchmark's launch shape
    (capacity budget + 128, so the single launch up to budget 256 and the split launch from
    512): 8 steps at 256 and 512 with the prepared summary, 2 steps otherwise."""
    steps = 8 if budget in (256, 512) else 2
    wl, cpu, gpu = layer("qwen3_4b_stack_n32768", layer_idx=3, steps=steps)
    announce(f"{wl.name} L={budget}")
    out = P.run_compress(gpu, budget, cap=budget + 128)
    for h in (0, 5):
        errs = P.check_compress_head(cpu, out, 0, h, budget)
        announce(f"head {h} {errs}")
    if steps == 8:
        P.run_decode_steps(gpu, out, 8, summary=1)
    else:
        P.run_decode_steps(gpu, out, 1)
        P.run_decode_steps(gpu, out, 1, summary=1)


def test_llama_stack_batch8_needles_full_size_sampled_heads():
    """One 32K-context layer of the LLaMA-3.1-8B-shaped stack with 8 sequences and
    planted-needle queries at budget 256: 64 KV heads compressed in one call, sampled
    (sequence, head) pairs checked, then decode with the prepared summary."""
    wl, cpu, gpu = layer("llama31_8b_stack_b8_n32768", layer_idx=5, steps=2)
    announce(f"{wl.name} B={wl.batch}")
    out = P.run_compress(gpu, 256, cap=258)
    for b, h in ((0, 0), (3, 5), (7, 7)):
        errs = P.check_compress_head(cpu, out, b, h, 256)
        announce(f"seq {b} head {h} {errs}")
    P.run_decode_steps(gpu, out, 2, summary=1)


def test_ruler_128k_full_size_sampled_heads():
    """The 128K-context stress layer (window 64, planted needles) at budget 1024: two
    sampled KV heads through the full compress protocol, then two decode steps over all
    heads."""
    wl, cpu, gpu = layer("ruler_n131072", layer_idx=0, steps=2)
    announce(f"{wl.name}")
    out = P.run_compress(gpu, 1024, cap=1026)
    for h in (2, 6):
        errs = P.check_compress_head(cpu, out, 0, h, 1024)
        announce(f"head {h} {errs}")
    P.run_decode_steps(gpu, out, 2)


def test_adaptive_budgets_ruler_128k_sampled_head():
    """Head-adaptive budgets on the 128K layer: the layer-wide selection runs over
    8 x 131007 candidates (512 slices); the per-head counts are checked against the GPU's
    masses and the oracle's, one sampled head follows the full compress protocol with its
    own count, and the decode runs over the per-head lengths."""
    wl, cpu, gpu = layer("ruler_n131072", layer_idx=1, steps=1)
    L = 1024
    cap = mk.compress_rows(wl.ctx_len, 8, L, wl.window, adaptive=True)
    out = P.run_compress(gpu, L, cap=cap, adaptive=True)
    kh, swaps = P.check_head_budgets(cpu, out, 0, L)
    announce(f"128K per-head counts {list(kh)}, swaps {swaps}")
    h = int(np.argmax(kh))
    P.check_compress_head(cpu, out, 0, h, int(1 + wl.window + kh[h]))
    P.run_decode_steps(gpu, out, 1)


# ---------------------------------------------------------------- decode-time eviction
def test_evict_tiny_fp32_follows_oracle_trajectory():
    wl, cpu, gpu = layer("tiny_fp32_n2048", steps=16)
    L = wl.budgets[0]
    out = P.run_compress(gpu, L, cap=L + 1)
    announce(f"{wl.name} evict L={L}")
    worst, swaps, n = P.run_evict_steps(gpu, out, 16, L)
    announce(f"worst rel err {worst:.2e}, swaps {swaps} of {n}")
    assert n == 16 and swaps == 0


@pytest.mark.parametrize("n_split", [0, 1, 3])
def test_evict_llama_layer_bf16_launch_shapes(n_split):
    """Two sequences x 8 KV heads; the attention after the eviction on the automatic, the
    single-launch and a 3-slice split shape."""
    wl, cpu, gpu = layer("llama31_8b_layer_n8192", steps=10, ctx_len=3000, batch=2)
    L = 300
    out = P.run_compress(gpu, L, cap=L + 1)
    announce(f"{wl.name} evict L={L} n_split={n_split}")
    worst, swaps, n = P.run_evict_steps(gpu, out, 10, L, n_split=n_split)
    announce(f"worst rel err {worst:.2e}, swaps {swaps} of {n}")
    assert n == 10 * 16 and swaps <= n // 50


@pytest.mark.parametrize("n_split", [0, 2])
@pytest.mark.parametrize("dtype", [torch.float32, torch.bfloat16])
@pytest.mark.parametrize("d", [64, 128])
def test_evict_budgets_and_lengths_around_the_bound(dtype, d, n_split):
    """Rows over several 32-row blocks with a ragged tail, G = 4; per-head lengths below
    the budget (no eviction: the step is the decode with the append), at it (steady state)
    and one row over it (flag bit 3, length kept).  n_split 0: one launch that scores,
    selects, updates and attends to the new cache; 2: one read of the cache over two scoring workgroups per head."""
    wl, cpu, gpu = layer("tiny_fp32_n2048", steps=3, dtype=dtype, head_dim=d, ctx_len=1200,
                         batch=2, n_q_heads=8, n_kv_heads=2, window=16, budgets=(290,))
    out = P.run_compress(gpu, 290, cap=293)
    announce(f"evict dtype={dtype} d={d} n_split={n_split}")
    P.run_evict_steps(gpu, out, 3, 290, n_split=n_split)                  # steady state
    P.run_evict_steps(gpu, out, 3, 292, start=([[290, 289], [260, 1]], out.n_e.cpu()),
                      n_split=n_split)
    P.run_evict_steps(gpu, out, 2, 289, flag=8, n_split=n_split)         # above budget


@pytest.mark.parametrize("budget", [318, 319])
def test_evict_at_the_launch_shape_bound(budget):
    """Caches of 319 and 320 rows (max_len = budget + 1), the two sides of the automatic
    choice between the short-cache launch and the one-read shape (G = 4, bf16, d = 128):
    both follow the oracle's trajectory."""
    wl, cpu, gpu = layer("tiny_fp32_n2048", steps=3, dtype=torch.bfloat16, head_dim=128,
                         ctx_len=1200, batch=1, n_q_heads=8, n_kv_heads=2, window=16,
                         budgets=(budget,))
    out = P.run_compress(gpu, budget, cap=budget + 1)
    announce(f"evict at the shape bound: budget {budget}, max_len {budget + 1}")
    worst, swaps, n = P.run_evict_steps(gpu, out, 3, budget)
    announce(f"worst rel err {worst:.2e}, swaps {swaps} of {n}")
    assert n == 3 * 2


@pytest.mark.parametrize("n_split,ctx", [(0, 300), (0, 700), (1, 700)])
def test_evict_with_empty_summary_scores_alpha_times_value_norm(n_split, ctx):
    """Budget above the context keeps every token, so n_e = 0: the first evictions use
    v_bar = S_tilde = 0 and later ones the summary they build (the short-cache launch at
    300 rows, the one-read shape at 700 rows over all CUs and one workgroup per head)."""
    wl, cpu, gpu = layer("tiny_fp32_n2048", steps=6, dtype=torch.bfloat16, head_dim=128,
                         ctx_len=ctx, batch=1, n_q_heads=4, n_kv_heads=2, window=16,
                         budgets=(900,))
    out = P.run_compress(gpu, 900, cap=ctx + 1)
    assert int(out.n_e.max()) == 0 and int(out.lens.min()) == ctx
    worst, swaps, n = P.run_evict_steps(gpu, out, 6, ctx, n_split=n_split)
    assert n == 12


@pytest.mark.parametrize("n_split", [0, 1])
def test_evict_full_cache_sets_flag_and_keeps_state(n_split):
    wl, cpu, gpu = layer("tiny_fp32_n2048", steps=1, dtype=torch.bfloat16, head_dim=64,
                         ctx_len=600, batch=1, n_q_heads=4, n_kv_heads=1, window=16,
                         budgets=(100,))
    out = P.run_compress(gpu, 100, cap=100)
    kc, vc, lens = out.k_out.clone(), out.v_out.clone(), out.lens.clone()
    n_e, s_k, s_v, S = out.n_e.clone(), out.s_k.clone(), out.s_v.clone(), out.S.clone()
    ev = torch.empty_like(lens)
    res, _, _, _, ws = mk.momentkv_decode_evict(gpu["q_dec"][0], kc, vc, lens, n_e, s_k, s_v, S,
                                                gpu["k_new"][0], gpu["v_new"][0], 99,
                                                n_split=n_split)
    torch.cuda.synchronize()
    assert int(ws[:4].view(torch.int32)[0]) & 1
    assert torch.equal(lens, out.lens) and torch.equal(n_e, out.n_e) and torch.equal(S, out.S)
    assert torch.equal(kc, out.k_out)
    # the output is the corrected attention over the full cache, without the new token
    moments = [[O.Moments(int(out.n_e[0, 0]), P.h64(out.s_k[0, 0]), P.h64(out.s_v[0, 0]),
                          P.h64(out.S[0, 0]))]]
    ref = O.decode(P.h64(gpu["q_dec"][0]), P.h64(out.k_out), P.h64(out.v_out),
                   out.lens.cpu().numpy(), moments)[0]
    got = P.h64(res)
    assert max(P.rel_l2(got[0, g], ref[0, g]) for g in range(4)) <= P.TOL[torch.bfloat16]


def test_evict_qwen_stack_layer_full_size_budget_2048():
    """One layer of the 32K-context stack at budget 2048 (rows over 17 scoring slices of
    128), two steps, every head checked."""
    wl, cpu, gpu = layer("qwen3_4b_stack_n32768", steps=2)
    out = P.run_compress(gpu, 2048, cap=2049)
    announce(f"{wl.name} evict L=2048")
    worst, swaps, n = P.run_evict_steps(gpu, out, 2, 2048)
    announce(f"worst rel err {worst:.2e}, swaps {swaps} of {n}")
    assert n == 2 * 8 and swaps <= 1


@pytest.mark.parametrize("G,budget", [(1, 300), (8, 1100), (16, 1100), (4, 4200)])
def test_evict_group_sizes_and_long_caches(G, budget):
    """Group sizes 1, 8 and 16 (the selection's register layouts for G <= 4, <= 8 and
    <= 16), and rows past one selection batch (more than 4096 rows at G = 4, 1024 at
    G = 16)."""
    wl, cpu, gpu = layer("tiny_fp32_n2048", steps=2, dtype=torch.bfloat16, head_dim=128,
                         ctx_len=max(2000, budget + 900), batch=1, n_q_heads=2 * G,
                         n_kv_heads=2, window=32, budgets=(budget,))
    out = P.run_compress(gpu, budget, cap=budget + 1)
    announce(f"evict G={G} budget={budget}")
    worst, swaps, n = P.run_evict_steps(gpu, out, 2, budget)
    announce(f"worst rel err {worst:.2e}, swaps {swaps} of {n}")
    assert n == 4


@pytest.mark.parametrize("n_split", [1, 3])
@pytest.mark.parametrize("gap,exact", [(5.0, False), (7.5, False), (12.0, True), (40.0, True)])
def test_evict_row_that_holds_most_of_the_attention(gap, exact, n_split):
    """The evicted row is one the summary predicts, and its key sits `gap` logits above the
    rest for every query (G = 4, fp32 caches, one workgroup per head or three slices).
    Predicted: v_j = v_bar + scale / n_e S_tilde k_j up to fp32 rounding; or exactly, with
    a summary of zero values (S_tilde = v_bar = 0) and v_j = 0.  At gap 5 the row holds
    about half of each query's mass and at 7.5 about 92%: its term leaves the accumulated
    attention in place.  At 12 (99.9%) and 40 (all but ~1e-17) too little would remain,
    and the attention over the new cache is computed again."""
    d, G, n, n_ev, js = 128, 4, 100, 50, 37
    rng = np.random.default_rng(11)
    K = rng.standard_normal((n + 1, d))
    V = rng.standard_normal((n + 1, d))
    ke, ve = rng.standard_normal((n_ev, d)), rng.standard_normal((n_ev, d))
    if exact:
        ve[:] = 0.0
    s_k, s_v, S = ke.sum(0), ve.sum(0), ve.T @ ke
    q0 = rng.standard_normal(d)
    Q = q0 + 0.1 * rng.standard_normal((G, d))
    scale = 1.0 / math.sqrt(d)
    K[js] = (gap * math.sqrt(d) * q0 / (q0 @ q0)).astype(np.float32)
    st = S - np.outer(s_v, s_k) / n_ev
    V[js] = (s_v / n_ev + scale / n_ev * st @ K[js]).astype(np.float32)
    f32 = lambda a: torch.tensor(np.asarray(a, np.float32)).cuda()
    comp = types.SimpleNamespace(k_out=f32(K)[None, None], v_out=f32(V)[None, None],
                                 lens=torch.tensor([[n]], dtype=torch.int32).cuda(),
                                 n_e=torch.tensor([[n_ev]], dtype=torch.int32).cuda(),
                                 s_k=f32(s_k)[None, None], s_v=f32(s_v)[None, None],
                                 S=f32(S)[None, None])
    inp = {"k": comp.k_out, "q_win": torch.zeros(1, G, 1, d).cuda(),
           "q_dec": f32(Q)[None, None], "k_new": f32(rng.standard_normal(d))[None, None, None],
           "v_new": f32(rng.standard_normal(d))[None, None, None]}
    announce(f"evict dominant row gap={gap} exact={exact} n_split={n_split}")
    worst, swaps, nev = P.run_evict_steps(inp, comp, 1, n, n_split=n_split)
    announce(f"worst rel err {worst:.2e}")
    assert nev == 1 and swaps == 0


# ---------------------------------------------------------------- head-adaptive budgets
@pytest.mark.parametrize("mi_rounds", [1, 0, -1])
def test_adaptive_budgets_llama_layer(mi_rounds):
    """Two sequences x 8 KV heads at budget 160 with the layer's candidate budget split by
    pooled mass; head 0 made sharper and head 1 flatter so the counts spread widely.  The
    split, every head's selection with its own count, the moments and the retained rows
    follow the full protocol; then decode runs over the per-head lengths."""
    wl, cpu, gpu = layer("llama31_8b_layer_n8192", steps=2, ctx_len=3000, batch=2)
    for x in (cpu, gpu):
        x["k"][:, 0] *= 3.0
        x["k"][:, 1] *= 0.05
    L = 160
    cap = mk.compress_rows(3000, 8, L, wl.window, adaptive=True)
    out = P.run_compress(gpu, L, cap=cap, adaptive=True, mi_rounds=mi_rounds)
    for b in range(2):
        kh, swaps = P.check_head_budgets(cpu, out, b, L)
        announce(f"mi_rounds={mi_rounds} seq {b} per-head counts {list(kh)}, swaps {swaps}")
        assert kh.sum() == 8 * (L - 1 - wl.window) and len(set(kh)) > 2
        for h in range(8):
            P.check_compress_head(cpu, out, b, h, int(1 + wl.window + kh[h]), mi_rounds=mi_rounds)
    if mi_rounds == 1:
        P.run_decode_steps(gpu, out, 2)


def test_adaptive_budgets_with_one_head_equal_uniform():
    wl, cpu, gpu = layer("tiny_fp32_n2048", steps=1)
    L = wl.budgets[0]
    uni = P.run_compress(gpu, L, cap=L)
    ada = P.run_compress(gpu, L, cap=L, adaptive=True)
    for name in ("k_out", "v_out", "idx", "lens", "n_e", "s_k", "s_v", "S"):
        assert torch.equal(getattr(uni, name), getattr(ada, name)), name


def test_adaptive_budgets_qwen_layer_full_size():
    """One 32K layer at budget 128: the layer-wide selection runs over 8 x 32735
    candidates (128 slices); counts checked against the GPU's masses and the oracle's."""
    wl, cpu, gpu = layer("qwen3_4b_stack_n32768", steps=1)
    L = 128
    cap = mk.compress_rows(wl.ctx_len, 8, L, wl.window, adaptive=True)
    out = P.run_compress(gpu, L, cap=cap, adaptive=True)
    kh, swaps = P.check_head_budgets(cpu, out, 0, L)
    announce(f"qwen 32K per-head counts {list(kh)}, swaps {swaps}")
    for h in (0, 5):
        P.check_compress_head(cpu, out, 0, h, int(1 + wl.window + kh[h]))
