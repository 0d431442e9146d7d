"""C ABI checks that need no GPU: the library loads, exports every declared entry point,
sizes workspaces, and rejects invalid arguments before launching anything.

Every call below fails host-side validation (or is a pure size query), so no HIP work
is ever enqueued.
"""
import ctypes
import os

import pytest

from paper_2606_01563_amd import momentkv as mk

OK, NULL, SHAPE, BUDGET, DTYPE, WORKSPACE, CAPACITY, ALIAS, HIP, UNSUP = range(10)


@pytest.fixture(scope="module")
def L():
    if not os.path.exists(mk.LIB_PATH):
        pytest.fail("libmomentkv.so is not built (run __graft_entry__.build())")
    return mk.lib()


def test_exports_every_declared_symbol(L):
    syms = mk.declared_symbols()
    assert {"momentkv_compress", "momentkv_decode_attn"} <= set(syms)
    for s in syms:
        assert hasattr(L, s), s


def test_abi_version_and_status_strings(L):
    assert mk.momentkv_abi_version() == 7
    for code in range(10):
        assert mk.momentkv_status_string(code) not in ("", "unknown status")
    assert mk.momentkv_status_string(99) == "unknown status"


def cparams(**kw):
    base = dict(batch=1, n_q_heads=32, n_kv_heads=8, head_dim=128, ctx_len=32768, budget=512,
                window=32, n_sink=1, chunk=4, mi_rounds=1, cap=512, dtype=1, scale=0.0, tau=1e-6,
                adaptive=0, moment_dtype=0)
    base.update(kw)
    return mk.CompressParams(**base)


def dparams(**kw):
    base = dict(batch=36, n_q_heads=32, n_kv_heads=8, head_dim=128, cap=640, max_len=640,
                order=1, dtype=1, scale=0.0, tau=1e-6, n_split=0, summary=0)
    base.update(kw)
    return mk.DecodeParams(**base)


def compress_status(p, ptr=1 << 20, ws_bytes=None, ws=1 << 40):
    """Call momentkv_compress with fake, non-overlapping device addresses; validation must
    reject the call before any of them is touched."""
    size = mk.momentkv_compress_workspace_bytes(p)
    if ws_bytes is None:
        ws_bytes = size
    step = 1 << 36
    ptrs = [ptr + i * step if ptr else None for i in range(11)]
    return mk.lib().momentkv_compress(ctypes.byref(p), *ptrs, None, ws, ws_bytes, None)


def decode_status(p, ptr=1 << 20, ws=1 << 40, ws_bytes=None, k_new=True):
    size = mk.momentkv_decode_workspace_bytes(p)
    if ws_bytes is None:
        ws_bytes = size
    step = 1 << 36
    ptrs = [ptr + i * step if ptr else None for i in range(13)]
    if not k_new:
        ptrs[4] = None
    return mk.lib().momentkv_decode_attn(ctypes.byref(p), *ptrs, ws, ws_bytes, None)


def test_workspace_bytes_and_earlier_size_names_agree(L):
    """The *_workspace_bytes queries and the earlier *_workspace_size names are one
    function each."""
    for p in (cparams(), cparams(budget=2048, ctx_len=131072, window=64), cparams(head_dim=96)):
        assert L.momentkv_compress_workspace_bytes(ctypes.byref(p)) == \
            L.momentkv_compress_workspace_size(ctypes.byref(p))
    for p in (dparams(), dparams(max_len=2048, cap=2048), dparams(max_len=641)):
        assert L.momentkv_decode_workspace_bytes(ctypes.byref(p)) == \
            L.momentkv_decode_workspace_size(ctypes.byref(p))
        assert L.momentkv_decode_evict_workspace_bytes(ctypes.byref(p)) == \
            L.momentkv_decode_evict_workspace_size(ctypes.byref(p))


def test_workspace_sizes(L):
    assert mk.momentkv_compress_workspace_bytes(cparams()) > 0
    assert mk.momentkv_decode_workspace_bytes(dparams()) > 0
    assert mk.momentkv_compress_workspace_bytes(cparams(head_dim=96)) == 0
    assert mk.momentkv_decode_workspace_bytes(dparams(max_len=641)) == 0
    # size grows with context and with budget
    assert mk.momentkv_compress_workspace_bytes(cparams(ctx_len=131072, window=64, budget=1024, cap=1024)) > \
        mk.momentkv_compress_workspace_bytes(cparams())


def test_decode_zero_prefix_covers_the_flag_and_one_counter_per_head(L):
    """The leading bytes to zero: the flag's 256-byte slot, then one int32 arrival counter
    per KV head (rounded up to 256 bytes), inside the workspace; 0 on invalid parameters."""
    for batch in (1, 36, 65):
        p = dparams(batch=batch)
        heads = batch * p.n_kv_heads
        zb = mk.momentkv_decode_workspace_zero_bytes(p)
        assert zb == 256 + (4 * heads + 255) // 256 * 256
        assert zb < mk.momentkv_decode_workspace_bytes(p)
    assert mk.momentkv_decode_workspace_zero_bytes(dparams(max_len=641)) == 0


@pytest.mark.parametrize("kw,code", [
    (dict(n_q_heads=30), SHAPE),            # Hq % Hkv != 0
    (dict(batch=0), SHAPE),
    (dict(window=0), SHAPE),
    (dict(window=32768), SHAPE),            # w >= N
    (dict(chunk=0), SHAPE),
    (dict(tau=-1.0), SHAPE),
    (dict(scale=float("nan")), SHAPE),
    (dict(head_dim=96), UNSUP),
    (dict(chunk=3), UNSUP),                 # chunk must divide 64
    (dict(mi_rounds=9), UNSUP),             # at most 8 moment rounds
    (dict(n_q_heads=8 * 17), UNSUP),        # G > 16
    (dict(window=200), UNSUP),              # G * w > 512
    (dict(budget=20), BUDGET),              # < n_sink + window
    (dict(cap=100), CAPACITY),
    (dict(dtype=7), DTYPE),
    (dict(adaptive=2), SHAPE),
    (dict(adaptive=1), CAPACITY),          # a head may take up to 8 x 479 candidates
    (dict(adaptive=1, ctx_len=140000, cap=9000), UNSUP),  # 8 x n_c candidates > 1048576
    (dict(moment_dtype=2), DTYPE),           # output S: fp32 or bf16
    (dict(moment_dtype=-1), DTYPE),
])
def test_compress_rejects_invalid_parameters(L, kw, code):
    assert compress_status(cparams(**kw)) == code


def test_compress_rejects_null_alias_and_small_workspace(L):
    p = cparams()
    assert compress_status(p, ptr=0) == NULL
    assert mk.lib().momentkv_compress(None, *([None] * 11), None, None, 0, None) == NULL
    assert compress_status(p, ws_bytes=16) == WORKSPACE
    assert compress_status(p, ws=0) == WORKSPACE
    assert compress_status(p, ws=(1 << 40) + 8) == WORKSPACE       # misaligned
    # k_out aliasing k
    ptrs = [(1 << 20) + i * (1 << 36) for i in range(11)]
    ptrs[3] = ptrs[1]
    size = mk.momentkv_compress_workspace_bytes(p)
    assert mk.lib().momentkv_compress(ctypes.byref(p), *ptrs, None, 1 << 40, size, None) == ALIAS
    # workspace overlapping v
    ptrs = [(1 << 20) + i * (1 << 36) for i in range(11)]
    assert mk.lib().momentkv_compress(ctypes.byref(p), *ptrs, None, ptrs[2], size, None) == ALIAS


def test_adaptive_workspace_and_capacity(L):
    rows = 1 + 32 + 8 * 479
    p = cparams(adaptive=1, cap=rows)
    assert mk.momentkv_compress_workspace_bytes(p) > mk.momentkv_compress_workspace_bytes(cparams())
    assert mk.compress_rows(32768, 8, 512, 32, 1, adaptive=True) == rows
    assert compress_status(cparams(adaptive=1, cap=rows - 1)) == CAPACITY


def test_budget_at_least_context_is_valid(L):
    p = cparams(ctx_len=300, budget=5000, cap=300)
    assert mk.momentkv_compress_workspace_bytes(p) > 0


@pytest.mark.parametrize("kw,code", [
    (dict(n_q_heads=30), SHAPE),
    (dict(cap=0), SHAPE),
    (dict(order=2), SHAPE),
    (dict(n_split=-1), SHAPE),
    (dict(summary=4), SHAPE),
    (dict(summary=2, dtype=0), SHAPE),      # the half-precision summary needs bf16 caches
    (dict(batch=500000), UNSUP),            # decode grid limit: 4M heads x 5 waves
    (dict(head_dim=80), UNSUP),
    (dict(max_len=0), CAPACITY),
    (dict(max_len=641), CAPACITY),
    (dict(dtype=3), DTYPE),
])
def test_decode_rejects_invalid_parameters(L, kw, code):
    assert decode_status(dparams(**kw)) == code


def test_decode_rejects_null_alias_and_small_workspace(L):
    p = dparams()
    assert decode_status(p, ptr=0) == NULL
    assert decode_status(p, k_new=False) == NULL        # k_new without v_new
    assert decode_status(p, ws_bytes=8) == WORKSPACE
    ptrs = [(1 << 20) + i * (1 << 36) for i in range(13)]
    ptrs[10] = ptrs[1]                                   # out aliases the key cache
    size = mk.momentkv_decode_workspace_bytes(p)
    assert mk.lib().momentkv_decode_attn(ctypes.byref(p), *ptrs, 1 << 40, size, None) == ALIAS


def test_prepared_summary_size_and_validation(L):
    p = dparams()
    assert mk.momentkv_prepared_summary_size(p) == 36 * 8 * 128 * 128 * 4
    assert mk.momentkv_prepared_summary_size(dparams(summary=2)) == 36 * 8 * 128 * 128 * 2
    assert mk.momentkv_prepared_summary_size(dparams(head_dim=80)) == 0
    ptrs = [(1 << 20) + i * (1 << 36) for i in range(5)]
    f = mk.lib().momentkv_prepare_summary
    assert f(ctypes.byref(p), None, *ptrs[1:], None) == NULL
    assert f(ctypes.byref(p), *ptrs[:4], None, None) == NULL
    assert f(ctypes.byref(p), *ptrs[:4], ptrs[4] + 8, None) == SHAPE      # misaligned
    assert f(ctypes.byref(p), *ptrs[:4], ptrs[3] + 64, None) == ALIAS     # overlaps S
    assert f(ctypes.byref(dparams(dtype=5)), *ptrs, None) == DTYPE
    # the raw sum stored in bf16 (summary = 3) is read by the decode as it is: nothing to
    # prepare
    assert mk.momentkv_prepared_summary_size(dparams(summary=3)) == 0
    assert f(ctypes.byref(dparams(summary=3)), *ptrs, None) == SHAPE
    assert mk.momentkv_decode_workspace_bytes(dparams(summary=3)) > 0  # a valid decode form


def evict_status(p, budget, ptr=1 << 20, ws=1 << 40, ws_bytes=None, drop=None):
    size = mk.momentkv_decode_evict_workspace_bytes(p)
    if ws_bytes is None:
        ws_bytes = size
    ptrs = [ptr + i * (1 << 36) if ptr else None for i in range(14)]
    if drop is not None:
        ptrs[drop] = None
    return mk.lib().momentkv_decode_evict(ctypes.byref(p), budget, *ptrs, ws, ws_bytes, None)


def test_decode_evict_sizes_and_validation(L):
    p = dparams()
    size = mk.momentkv_decode_evict_workspace_bytes(p)
    # per head: (G + 2) fp32 record planes of max_len rows and (G + 1) running maxima per
    # 32-row block, after the 256-byte flag
    assert size >= 256 + 36 * 8 * (6 * 640 + 5 * 20) * 4
    assert mk.momentkv_decode_evict_workspace_bytes(dparams(summary=1)) == 0
    assert evict_status(p, 0) == BUDGET
    assert evict_status(dparams(summary=1), 512) == SHAPE
    assert evict_status(dparams(head_dim=80), 512) == UNSUP
    assert evict_status(dparams(max_len=641), 512) == CAPACITY
    assert evict_status(p, 512, ptr=0) == NULL
    for i in (4, 5, 10):                      # k_new, v_new and out are required
        assert evict_status(p, 512, drop=i) == NULL
    assert evict_status(p, 512, ws_bytes=size - 1) == WORKSPACE
    assert evict_status(p, 512, ws=(1 << 40) + 64) == WORKSPACE
    ptrs = [(1 << 20) + i * (1 << 36) for i in range(14)]
    ptrs[10] = ptrs[9]                        # out overlaps S
    assert mk.lib().momentkv_decode_evict(ctypes.byref(p), 512, *ptrs, 1 << 40, size, None) == ALIAS
    ptrs = [(1 << 20) + i * (1 << 36) for i in range(14)]
    ptrs[9] = ptrs[1]                         # S overlaps the key cache
    assert mk.lib().momentkv_decode_evict(ctypes.byref(p), 512, *ptrs, 1 << 40, size, None) == ALIAS


# ------------------------------------------------ binding-side tensor validation (CPU)
def _decode_tensors(B=2, Hq=8, Hkv=2, d=64, cap=16, dt=None):
    import torch
    dt = dt or torch.bfloat16
    f32, i32 = torch.float32, torch.int32
    return dict(q=torch.zeros(B, Hq, d, dtype=dt), k_cache=torch.zeros(B, Hkv, cap, d, dtype=dt),
                v_cache=torch.zeros(B, Hkv, cap, d, dtype=dt), lens=torch.zeros(B, Hkv, dtype=i32),
                n_e=torch.zeros(B, Hkv, dtype=i32), s_k=torch.zeros(B, Hkv, d, dtype=f32),
                s_v=torch.zeros(B, Hkv, d, dtype=f32), S=torch.zeros(B, Hkv, d, d, dtype=f32))


@pytest.mark.parametrize("name,bad", [
    ("lens", lambda t: t.long()),
    ("n_e", lambda t: t[:, :1]),
    ("s_k", lambda t: t.bfloat16()),
    ("S", lambda t: t[..., :32]),
    ("v_cache", lambda t: t.float()),
])
def test_decode_binding_rejects_wrong_tensors_before_the_library(name, bad):
    """A wrong dtype or shape is a ValueError naming the tensor, raised before any pointer
    reaches the library (an int64 lens or a short summary would be read out of bounds)."""
    t = _decode_tensors()
    t[name] = bad(t[name])
    with pytest.raises(ValueError, match=name):
        mk.momentkv_decode_attn(**t)
    with pytest.raises(ValueError, match=name):
        mk.momentkv_decode_evict(**t, k_new=t["q"][:, :2].clone(), v_new=t["q"][:, :2].clone(),
                                 budget=4)


def test_decode_binding_checks_summary_form_new_rows_and_device():
    import torch
    t = _decode_tensors()
    with pytest.raises(ValueError, match="prepared"):      # summary=1 wants the bf16 planes
        mk.momentkv_decode_attn(**t, summary=1)
    with pytest.raises(ValueError, match="raw, bf16"):     # summary=3 wants a bf16 raw S
        mk.momentkv_decode_attn(**t, summary=3)
    with pytest.raises(ValueError, match="summary must be"):
        mk.momentkv_decode_attn(**t, summary=4)
    with pytest.raises(ValueError, match="together"):
        mk.momentkv_decode_attn(**t, k_new=torch.zeros(2, 2, 64, dtype=torch.bfloat16))
    with pytest.raises(ValueError, match="required"):
        mk.momentkv_decode_evict(**t, k_new=None, v_new=None, budget=4)
    with pytest.raises(ValueError, match="k_new"):
        mk.momentkv_decode_attn(**t, k_new=torch.zeros(2, 2, 64), v_new=torch.zeros(2, 2, 64))
    with pytest.raises(ValueError, match="lse"):
        mk.momentkv_decode_attn(**t, lse=torch.zeros(2, 8, dtype=torch.float64))
    with pytest.raises(ValueError, match="on the GPU"):    # right shapes, host memory
        mk.momentkv_decode_attn(**t)


def test_compress_and_prepare_binding_reject_wrong_tensors():
    import torch
    q = torch.zeros(1, 8, 4, 64, dtype=torch.bfloat16)
    k = torch.zeros(1, 2, 100, 64, dtype=torch.bfloat16)
    with pytest.raises(ValueError, match="v"):
        mk.momentkv_compress(q, k, k.float(), 20)
    with pytest.raises(ValueError, match="q_win"):
        mk.momentkv_compress(q[:, :, :, :32], k, k, 20)
    with pytest.raises(ValueError, match="on the GPU"):
        mk.momentkv_compress(q, k, k, 20)
    with pytest.raises(ValueError, match="moment_dtype"):
        mk.momentkv_compress(q, k, k, 20, moment_dtype=torch.float16)
    t = _decode_tensors()
    with pytest.raises(ValueError, match="n_e"):
        mk.momentkv_prepare_summary(t["n_e"].long(), t["s_k"], t["s_v"], t["S"],
                                    dtype=torch.bfloat16)
    with pytest.raises(ValueError, match="out"):
        mk.momentkv_prepare_summary(t["n_e"], t["s_k"], t["s_v"], t["S"], dtype=torch.bfloat16,
                                    out=torch.zeros(2, 2, 64, 64, dtype=torch.bfloat16))


def test_noalloc_decode_rejects_requests_beyond_its_scratch_before_any_device_call(L):
    """The decode that allocates nothing refuses work whose workspace would exceed its
    16 MiB device array, and missing pointers, before touching the GPU."""
    big = dparams(batch=4096, cap=4096, max_len=4096)
    assert mk.momentkv_decode_workspace_bytes(big) > mk.NOALLOC_SCRATCH_BYTES
    small = dparams()
    assert mk.momentkv_decode_workspace_bytes(small) <= mk.NOALLOC_SCRATCH_BYTES
    step = 1 << 36
    ptrs = [(1 << 20) + i * step for i in range(13)]
    assert L.momentkv_decode_attn_noalloc(ctypes.byref(big), *ptrs, None, None) == WORKSPACE
    nulls = list(ptrs)
    nulls[0] = None
    assert L.momentkv_decode_attn_noalloc(ctypes.byref(small), *nulls, None, None) == NULL
    assert L.momentkv_decode_attn_noalloc(ctypes.byref(dparams(head_dim=96)), *ptrs, None,
                                          None) == UNSUP
    assert L.momentkv_decode_attn_noalloc(None, *ptrs, None, None) == NULL
