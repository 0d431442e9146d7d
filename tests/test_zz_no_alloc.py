"""momentkv_decode_attn_noalloc (the decode that allocates nothing: its partial results
live in a library-owned device array) against momentkv_decode_attn through the C ABI:
two calls in a row, the second on a smaller input, each bit-identical to the workspace
entry point on copies of the same buffers, and the smaller one also against the oracle."""
import numpy as np
import pytest
import torch

import oracle as O
from paper_2606_01563_amd import momentkv as mk
from tests import parity_util as P

pytestmark = pytest.mark.gpu


def _inputs(B, Hq, Hkv, d, cap, dtype, seed, n_e_max=5000):
    g = torch.Generator().manual_seed(seed)
    t = lambda *s: torch.randn(*s, generator=g)
    lens = torch.randint(cap // 2, cap - 1, (B, Hkv), generator=g, dtype=torch.int32)
    n_e = torch.randint(0, n_e_max, (B, Hkv), generator=g, dtype=torch.int32)
    n_e[0, 0] = 0                                             # one head with an empty summary
    kk = t(B, Hkv, 64, d)
    vv = t(B, Hkv, 64, d) + 0.5
    S = torch.einsum("bhna,bhnc->bhac", vv, kk) * (n_e[..., None, None].float() / 64)
    cpu = dict(q=t(B, Hq, d).to(dtype), k_cache=t(B, Hkv, cap, d).to(dtype),
               v_cache=t(B, Hkv, cap, d).to(dtype), lens=lens, n_e=n_e,
               s_k=kk.sum(2) * (n_e[..., None].float() / 64),
               s_v=vv.sum(2) * (n_e[..., None].float() / 64), S=S.contiguous(),
               k_new=t(B, Hkv, d).to(dtype), v_new=t(B, Hkv, d).to(dtype))
    return cpu, {k: v.cuda() for k, v in cpu.items()}


def _both(gpu, dtype, max_len):
    """The workspace entry point and the one that allocates nothing, each on its own copy
    of the caches and lengths (the append writes them)."""
    B, Hq, d = gpu["q"].shape
    res = {}
    for name in ("workspace", "noalloc"):
        kc, vc, ln = gpu["k_cache"].clone(), gpu["v_cache"].clone(), gpu["lens"].clone()
        out = torch.empty_like(gpu["q"])
        lse = torch.empty(B, Hq, device="cuda")
        w_r = torch.empty(B, Hq, device="cuda")
        args = (gpu["q"], kc, vc, ln, gpu["n_e"], gpu["s_k"], gpu["s_v"], gpu["S"])
        kw = dict(k_new=gpu["k_new"], v_new=gpu["v_new"], max_len=max_len, out=out, lse=lse,
                  w_r=w_r)
        if name == "workspace":
            mk.momentkv_decode_attn(*args, **kw)
            flag = None
        else:
            flag = torch.zeros(1, dtype=torch.int32, device="cuda")
            mk.momentkv_decode_attn_noalloc(*args, **kw, flag=flag)
        torch.cuda.synchronize()
        res[name] = dict(out=out, lse=lse, w_r=w_r, kc=kc, vc=vc, lens=ln, flag=flag)
    a, b = res["workspace"], res["noalloc"]
    for key in ("out", "lse", "w_r", "kc", "vc", "lens"):
        assert torch.equal(a[key], b[key]), key
    assert int(b["flag"][0]) == 0
    return b


def test_noalloc_decode_equals_workspace_decode_on_two_calls():
    # 1: 16 caches x 8 KV heads, 1100 rows, bf16: the split-K shape (about 1.6 MB of scratch)
    print("[noalloc] call 1: B=16 Hkv=8 d=128 cap=1100 bf16 (split shape)", flush=True)
    cpu, gpu = _inputs(16, 32, 8, 128, 1100, torch.bfloat16, seed=1)
    _both(gpu, torch.bfloat16, 1100)
    # 2: a smaller input right after: 2 caches x 2 KV heads, 200 rows, fp32 (single launch)
    print("[noalloc] call 2: B=2 Hkv=2 d=64 cap=200 fp32 (single launch)", flush=True)
    cpu, gpu = _inputs(2, 8, 2, 64, 200, torch.float32, seed=2)
    got = _both(gpu, torch.float32, 200)
    mom = [[O.Moments(int(cpu["n_e"][b, h]), cpu["s_k"][b, h].double().numpy(),
                      cpu["s_v"][b, h].double().numpy(), cpu["S"][b, h].double().numpy())
            for h in range(2)] for b in range(2)]
    ref, _, _, _ = O.decode(P.h64(cpu["q"]), P.h64(cpu["k_cache"]), P.h64(cpu["v_cache"]),
                            cpu["lens"].numpy(), mom, k_new=P.h64(cpu["k_new"]),
                            v_new=P.h64(cpu["v_new"]))
    o = P.h64(got["out"])
    err = max(P.rel_l2(o[b, hq], ref[b, hq]) for b in range(2) for hq in range(8))
    assert err <= P.TOL[torch.float32], err
    np.testing.assert_array_equal(got["lens"].cpu().numpy(), cpu["lens"].numpy() + 1)


def test_noalloc_decode_reports_a_full_cache_in_the_callers_flag():
    cpu, gpu = _inputs(1, 4, 1, 64, 40, torch.float32, seed=3)
    gpu["lens"].fill_(40)                                     # full: the append is skipped
    flag = torch.zeros(1, dtype=torch.int32, device="cuda")
    out = torch.empty_like(gpu["q"])
    mk.momentkv_decode_attn_noalloc(gpu["q"], gpu["k_cache"], gpu["v_cache"], gpu["lens"],
                                    gpu["n_e"], gpu["s_k"], gpu["s_v"], gpu["S"],
                                    k_new=gpu["k_new"], v_new=gpu["v_new"], max_len=40, out=out,
                                    flag=flag)
    torch.cuda.synchronize()
    assert int(flag[0]) == 1 and int(gpu["lens"][0, 0]) == 40
