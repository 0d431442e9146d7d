"""Thin ctypes binding of libmomentkv.so (C ABI in include/momentkv.h).

Functions carry the C names.  `momentkv_compress` and `momentkv_decode_attn` take torch
tensors that already live on the GPU, allocate the outputs and the workspace when the
caller does not pass them, and forward device pointers plus the current HIP stream to
the library.  No arithmetic of the method happens here: every step runs in the HIP
kernels.  The library is loaded on first use; a missing library raises.
"""
from __future__ import annotations

import ctypes
import os
import re
from dataclasses import dataclass

import torch

_HERE = os.path.dirname(os.path.abspath(__file__))
# MKV_LIB selects another build of the same library (the host-sanitized copy used by the
# CPU-only checks of the C ABI); the default is the in-tree product library.
LIB_PATH = os.environ.get("MKV_LIB") or os.path.join(_HERE, "libmomentkv.so")
HEADER_PATH = os.path.join(os.path.dirname(_HERE), "include", "momentkv.h")

MKV_F32, MKV_BF16 = 0, 1
NOALLOC_SCRATCH_BYTES = 16 << 20   # MOMENTKV_NOALLOC_SCRATCH_BYTES
STATUS = {0: "MKV_OK", 1: "MKV_ERR_NULL", 2: "MKV_ERR_SHAPE", 3: "MKV_ERR_BUDGET",
          4: "MKV_ERR_DTYPE", 5: "MKV_ERR_WORKSPACE", 6: "MKV_ERR_CAPACITY",
          7: "MKV_ERR_ALIAS", 8: "MKV_ERR_HIP", 9: "MKV_ERR_UNSUPPORTED"}


class MomentKVError(RuntimeError):
    def __init__(self, code: int, what: str):
        super().__init__(f"{what}: {STATUS.get(code, code)} ({momentkv_status_string(code)})")
        self.code = code


class CompressParams(ctypes.Structure):
    _fields_ = [("batch", ctypes.c_int32), ("n_q_heads", ctypes.c_int32),
                ("n_kv_heads", ctypes.c_int32), ("head_dim", ctypes.c_int32),
                ("ctx_len", ctypes.c_int32), ("budget", ctypes.c_int32),
                ("window", ctypes.c_int32), ("n_sink", ctypes.c_int32),
                ("chunk", ctypes.c_int32), ("mi_rounds", ctypes.c_int32),
                ("cap", ctypes.c_int32), ("dtype", ctypes.c_int32),
                ("scale", ctypes.c_float), ("tau", ctypes.c_float),
                ("adaptive", ctypes.c_int32), ("moment_dtype", ctypes.c_int32)]


class CompressDebug(ctypes.Structure):
    _fields_ = [("abar", ctypes.c_void_p), ("score0", ctypes.c_void_p),
                ("score", ctypes.c_void_p), ("kept0", ctypes.c_void_p)]


class DecodeParams(ctypes.Structure):
    _fields_ = [("batch", ctypes.c_int32), ("n_q_heads", ctypes.c_int32),
                ("n_kv_heads", ctypes.c_int32), ("head_dim", ctypes.c_int32),
                ("cap", ctypes.c_int32), ("max_len", ctypes.c_int32),
                ("order", ctypes.c_int32), ("dtype", ctypes.c_int32),
                ("scale", ctypes.c_float), ("tau", ctypes.c_float),
                ("n_split", ctypes.c_int32), ("summary", ctypes.c_int32)]


_lib = None
_VP = ctypes.c_void_p


def lib() -> ctypes.CDLL:
    """Load libmomentkv.so (once).  Raises if it has not been built."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise RuntimeError(f"{LIB_PATH} is missing: build it with __graft_entry__.build()")
        L = ctypes.CDLL(LIB_PATH)
        for name in ("momentkv_compress_workspace_bytes", "momentkv_compress_workspace_size"):
            getattr(L, name).argtypes = [ctypes.POINTER(CompressParams)]
            getattr(L, name).restype = ctypes.c_size_t
        for name in ("momentkv_decode_workspace_bytes", "momentkv_decode_workspace_size",
                     "momentkv_decode_workspace_zero_bytes",
                     "momentkv_decode_evict_workspace_bytes",
                     "momentkv_decode_evict_workspace_size"):
            getattr(L, name).argtypes = [ctypes.POINTER(DecodeParams)]
            getattr(L, name).restype = ctypes.c_size_t
        L.momentkv_compress.argtypes = [ctypes.POINTER(CompressParams)] + [_VP] * 11 + \
            [ctypes.POINTER(CompressDebug), _VP, ctypes.c_size_t, _VP]
        L.momentkv_compress.restype = ctypes.c_int
        L.momentkv_decode_attn.argtypes = [ctypes.POINTER(DecodeParams)] + [_VP] * 13 + \
            [_VP, ctypes.c_size_t, _VP]
        L.momentkv_decode_attn.restype = ctypes.c_int
        L.momentkv_decode_attn_noalloc.argtypes = [ctypes.POINTER(DecodeParams)] + [_VP] * 15
        L.momentkv_decode_attn_noalloc.restype = ctypes.c_int
        L.momentkv_status_string.argtypes = [ctypes.c_int32]
        L.momentkv_prepared_summary_size.argtypes = [ctypes.POINTER(DecodeParams)]
        L.momentkv_prepared_summary_size.restype = ctypes.c_size_t
        L.momentkv_prepare_summary.argtypes = [ctypes.POINTER(DecodeParams)] + [_VP] * 6
        L.momentkv_prepare_summary.restype = ctypes.c_int
        L.momentkv_decode_evict.argtypes = [ctypes.POINTER(DecodeParams), ctypes.c_int32] + \
            [_VP] * 14 + [_VP, ctypes.c_size_t, _VP]
        L.momentkv_decode_evict.restype = ctypes.c_int
        L.momentkv_status_string.restype = ctypes.c_char_p
        L.momentkv_abi_version.argtypes = []
        L.momentkv_abi_version.restype = ctypes.c_int32
        _lib = L
    return _lib


def declared_symbols() -> list[str]:
    """Entry points declared in include/momentkv.h."""
    with open(HEADER_PATH) as f:
        text = f.read()
    return sorted(set(re.findall(r"\b(momentkv_[a-z_]+)\s*\(", text)))


def momentkv_status_string(code: int) -> str:
    return lib().momentkv_status_string(int(code)).decode()


def momentkv_abi_version() -> int:
    return int(lib().momentkv_abi_version())


def momentkv_compress_workspace_bytes(p: CompressParams) -> int:
    return int(lib().momentkv_compress_workspace_bytes(ctypes.byref(p)))


def momentkv_decode_workspace_bytes(p: DecodeParams) -> int:
    return int(lib().momentkv_decode_workspace_bytes(ctypes.byref(p)))


def momentkv_decode_evict_workspace_bytes(p: DecodeParams) -> int:
    return int(lib().momentkv_decode_evict_workspace_bytes(ctypes.byref(p)))


# the same functions under their earlier names
momentkv_compress_workspace_size = momentkv_compress_workspace_bytes
momentkv_decode_workspace_size = momentkv_decode_workspace_bytes
momentkv_decode_evict_workspace_size = momentkv_decode_evict_workspace_bytes


def momentkv_prepared_summary_size(p: DecodeParams) -> int:
    return int(lib().momentkv_prepared_summary_size(ctypes.byref(p)))


# ------------------------------------------------------------------------ marshalling
def _dtype_code(t: torch.Tensor) -> int:
    if t.dtype == torch.float32:
        return MKV_F32
    if t.dtype == torch.bfloat16:
        return MKV_BF16
    raise TypeError(f"unsupported dtype {t.dtype}")


def _ptr(t: torch.Tensor | None) -> int | None:
    if t is None:
        return None
    if not t.is_cuda:
        raise ValueError("tensor must be on the GPU")
    if not t.is_contiguous():
        raise ValueError("tensor must be contiguous")
    return t.data_ptr()


def _expect(t, name: str, shape: tuple, dtype: torch.dtype, optional: bool = False):
    """Raise ValueError unless `t` is a tensor of exactly this shape and dtype (None is
    allowed when optional).  Runs before any pointer reaches the library: a tensor with
    the wrong element size or too few elements would be read out of bounds on the GPU."""
    if t is None:
        if optional:
            return
        raise ValueError(f"{name} is required")
    if not isinstance(t, torch.Tensor):
        raise ValueError(f"{name} must be a torch.Tensor")
    if t.dtype != dtype:
        raise ValueError(f"{name} must be {dtype}, got {t.dtype}")
    if tuple(t.shape) != tuple(shape):
        raise ValueError(f"{name} must have shape {tuple(shape)}, got {tuple(t.shape)}")


def _same_device(named: dict):
    """Every given tensor on the GPU, contiguous, and on one device."""
    devs = set()
    for name, t in named.items():
        if t is None:
            continue
        if not t.is_cuda:
            raise ValueError(f"{name} must be on the GPU")
        if not t.is_contiguous():
            raise ValueError(f"{name} must be contiguous")
        devs.add(t.device)
    if len(devs) > 1:
        raise ValueError(f"tensors are on several devices: {sorted(map(str, devs))}")


def _check_workspace(ws, name: str = "workspace"):
    if ws is not None and (not isinstance(ws, torch.Tensor) or ws.dtype != torch.uint8
                           or ws.dim() != 1):
        raise ValueError(f"{name} must be a 1-D torch.uint8 tensor")


def _stream() -> int:
    return torch.cuda.current_stream().cuda_stream


def _workspace(nbytes: int, device, ws: torch.Tensor | None) -> torch.Tensor:
    if ws is None or ws.numel() < nbytes:
        ws = torch.empty(max(nbytes, 256), dtype=torch.uint8, device=device)
    if ws.data_ptr() % 256:
        raise ValueError("workspace must be 256-byte aligned")
    return ws


@dataclass
class CompressOutput:
    k_out: torch.Tensor       # [B, Hkv, cap, d]
    v_out: torch.Tensor
    idx: torch.Tensor         # [B, Hkv, min(L, N)] int32
    lens: torch.Tensor        # [B, Hkv] int32
    n_e: torch.Tensor         # [B, Hkv] int32
    s_k: torch.Tensor         # [B, Hkv, d] fp32
    s_v: torch.Tensor
    S: torch.Tensor           # [B, Hkv, d, d] fp32, or bf16 (moment_dtype=torch.bfloat16)
    abar: torch.Tensor | None = None
    score0: torch.Tensor | None = None
    score: torch.Tensor | None = None
    kept0: torch.Tensor | None = None


def compress_rows(N: int, Hkv: int, budget: int, window: int, n_sink: int = 1,
                  adaptive: bool = False) -> int:
    """Most rows any head keeps: min(budget, N), or with head-adaptive budgets
    n_sink + window + min(n_c, Hkv * k_keep)."""
    if not adaptive or budget >= N:
        return min(budget, N)
    n_c = N - window - n_sink
    return n_sink + window + min(n_c, Hkv * (budget - n_sink - window))


def compress_params(q_win, k, budget, *, n_sink=1, chunk=4, mi_rounds=1, cap=None,
                    scale=0.0, tau=1e-6, adaptive=False,
                    moment_dtype=torch.float32) -> CompressParams:
    B, Hq, w, d = q_win.shape
    _, Hkv, N, _ = k.shape
    n_out = compress_rows(N, Hkv, budget, w, n_sink, adaptive)
    if moment_dtype not in (torch.float32, torch.bfloat16):
        raise ValueError(f"moment_dtype must be float32 or bfloat16, got {moment_dtype}")
    return CompressParams(B, Hq, Hkv, d, N, budget, w, n_sink, chunk, mi_rounds,
                          n_out if cap is None else cap, _dtype_code(k), scale, tau,
                          1 if adaptive else 0,
                          MKV_BF16 if moment_dtype == torch.bfloat16 else MKV_F32)


def momentkv_compress(q_win: torch.Tensor, k: torch.Tensor, v: torch.Tensor, budget: int, *,
                      n_sink: int = 1, chunk: int = 4, mi_rounds: int = 1, cap: int | None = None,
                      scale: float = 0.0, tau: float = 1e-6, adaptive: bool = False,
                      moment_dtype: torch.dtype = torch.float32,
                      debug: bool = False, out: CompressOutput | None = None,
                      workspace: torch.Tensor | None = None) -> CompressOutput:
    """Compress [B, Hkv, N, d] prefill K/V to `budget` rows per KV head (see the header);
    adaptive=True splits the layer's candidate budget across heads (idx then has `cap`
    entries per head, the first `lens` of them valid); moment_dtype=torch.bfloat16 stores
    the output S in bf16 (pass it to the decode with summary=3)."""
    if not isinstance(q_win, torch.Tensor) or q_win.dim() != 4:
        raise ValueError("q_win must be a [B, Hq, w, d] tensor")
    if not isinstance(k, torch.Tensor) or k.dim() != 4:
        raise ValueError("k must be a [B, Hkv, N, d] tensor")
    p = compress_params(q_win, k, budget, n_sink=n_sink, chunk=chunk, mi_rounds=mi_rounds,
                        cap=cap, scale=scale, tau=tau, adaptive=adaptive,
                        moment_dtype=moment_dtype)
    B, Hq, w, d = q_win.shape
    _, Hkv, N, _ = k.shape
    dev = k.device
    ada = adaptive and budget < N
    n_out = p.cap if ada else min(budget, N)
    _expect(q_win, "q_win", (B, Hq, w, d), k.dtype)
    _expect(v, "v", tuple(k.shape), k.dtype)
    _check_workspace(workspace)
    if out is not None:
        f32, i32 = torch.float32, torch.int32
        for name, shape, dt in (("k_out", (B, Hkv, p.cap, d), k.dtype),
                                ("v_out", (B, Hkv, p.cap, d), k.dtype),
                                ("idx", (B, Hkv, n_out), i32), ("lens", (B, Hkv), i32),
                                ("n_e", (B, Hkv), i32), ("s_k", (B, Hkv, d), f32),
                                ("s_v", (B, Hkv, d), f32), ("S", (B, Hkv, d, d), moment_dtype)):
            _expect(getattr(out, name), f"out.{name}", shape, dt)
    _same_device({"q_win": q_win, "k": k, "v": v, "workspace": workspace,
                  **({} if out is None else {f"out.{n}": getattr(out, n) for n in
                                             ("k_out", "v_out", "idx", "lens", "n_e", "s_k",
                                              "s_v", "S")})})
    if out is None:
        f32 = dict(dtype=torch.float32, device=dev)
        i32 = dict(dtype=torch.int32, device=dev)
        out = CompressOutput(
            k_out=torch.empty(B, Hkv, p.cap, d, dtype=k.dtype, device=dev),
            v_out=torch.empty(B, Hkv, p.cap, d, dtype=k.dtype, device=dev),
            idx=torch.empty(B, Hkv, n_out, **i32), lens=torch.empty(B, Hkv, **i32),
            n_e=torch.empty(B, Hkv, **i32), s_k=torch.empty(B, Hkv, d, **f32),
            s_v=torch.empty(B, Hkv, d, **f32),
            S=torch.empty(B, Hkv, d, d, dtype=moment_dtype, device=dev))
    dbg = None
    if debug and budget < N:
        n_c = N - w - n_sink
        k_keep = budget - n_sink - w
        f32 = dict(dtype=torch.float32, device=dev)
        out.abar = torch.zeros(B, Hkv, n_c, **f32)
        out.score0 = torch.zeros(B, Hkv, n_c, **f32)
        out.score = torch.zeros(B, Hkv, n_c, **f32)
        k_rows = min(n_c, Hkv * k_keep) if ada else k_keep
        out.kept0 = torch.zeros(B, Hkv, max(k_rows, 0), dtype=torch.int32, device=dev)
        dbg = CompressDebug(_ptr(out.abar), _ptr(out.score0), _ptr(out.score),
                            _ptr(out.kept0) if k_keep > 0 else None)
    nbytes = momentkv_compress_workspace_bytes(p)
    if nbytes == 0:
        code = lib().momentkv_compress(ctypes.byref(p), *([None] * 11), None, None, 0, None)
        raise MomentKVError(code, "momentkv_compress")
    ws = _workspace(nbytes, dev, workspace)
    code = lib().momentkv_compress(
        ctypes.byref(p), _ptr(q_win), _ptr(k), _ptr(v), _ptr(out.k_out), _ptr(out.v_out),
        _ptr(out.idx), _ptr(out.lens), _ptr(out.n_e), _ptr(out.s_k), _ptr(out.s_v), _ptr(out.S),
        ctypes.byref(dbg) if dbg is not None else None, ws.data_ptr(), ws.numel(), _stream())
    if code != 0:
        raise MomentKVError(code, "momentkv_compress")
    return out


def momentkv_decode_workspace_zero_bytes(p: DecodeParams) -> int:
    """Leading decode-workspace bytes that must be zero before a call (the append-overflow
    flag and the per-head arrival counters, which every call leaves at zero)."""
    return int(lib().momentkv_decode_workspace_zero_bytes(ctypes.byref(p)))


def _zero_prefix(ws: torch.Tensor, nbytes: int) -> None:
    """Zeroes the leading nbytes of a decode workspace unless this tensor object is known
    to have them at zero already (zeroed here before; calls leave them at zero)."""
    if getattr(ws, "_mkv_zeroed", 0) < nbytes:
        ws[:nbytes].zero_()
        ws._mkv_zeroed = nbytes


def decode_params(q, k_cache, *, max_len, order=1, scale=0.0, tau=1e-6,
                  n_split=0, summary=0) -> DecodeParams:
    B, Hq, d = q.shape
    _, Hkv, cap, _ = k_cache.shape
    return DecodeParams(B, Hq, Hkv, d, cap, max_len, order, _dtype_code(q), scale, tau, n_split,
                        summary)


def momentkv_prepare_summary(n_e: torch.Tensor, s_k: torch.Tensor, s_v: torch.Tensor,
                             S: torch.Tensor, *, dtype: torch.dtype, tau: float = 1e-6,
                             half: bool = False, out: torch.Tensor | None = None) -> torch.Tensor:
    """Decode form of the summary (see the header): bf16 hi/lo planes [B, Hkv, 2, d, d] for
    dtype bf16, fp32 [B, Hkv, d, d] for fp32; half=True (bf16 only) the one-plane
    half-precision form [B, Hkv, d, d].  Pass it as `S` with summary=1 (summary=2 if half)."""
    if not isinstance(S, torch.Tensor) or S.dim() != 4:
        raise ValueError("S must be a [B, Hkv, d, d] tensor")
    if dtype not in (torch.float32, torch.bfloat16):
        raise ValueError(f"unsupported dtype {dtype}")
    B, Hkv, d, _ = S.shape
    _expect(S, "S", (B, Hkv, d, d), torch.float32)
    _expect(n_e, "n_e", (B, Hkv), torch.int32)
    _expect(s_k, "s_k", (B, Hkv, d), torch.float32)
    _expect(s_v, "s_v", (B, Hkv, d), torch.float32)
    code = MKV_BF16 if dtype == torch.bfloat16 else MKV_F32
    p = DecodeParams(B, Hkv, Hkv, d, 1, 1, 1, code, 0.0, tau, 0, 2 if half else 0)
    shape = (B, Hkv, 2, d, d) if dtype == torch.bfloat16 and not half else (B, Hkv, d, d)
    if out is None:
        out = torch.empty(shape, dtype=dtype, device=S.device)
    _expect(out, "out", shape, dtype)
    _same_device({"n_e": n_e, "s_k": s_k, "s_v": s_v, "S": S, "out": out})
    if out.numel() * out.element_size() < momentkv_prepared_summary_size(p):
        raise ValueError("prepared summary buffer too small")
    code = lib().momentkv_prepare_summary(ctypes.byref(p), _ptr(n_e), _ptr(s_k), _ptr(s_v),
                                          _ptr(S), _ptr(out), _stream())
    if code != 0:
        raise MomentKVError(code, "momentkv_prepare_summary")
    return out


def _check_decode_args(q, k_cache, v_cache, lens, n_e, s_k, s_v, S, k_new, v_new, out, lse,
                       w_r, workspace, summary: int, evicted=None, need_new: bool = False):
    if not isinstance(q, torch.Tensor) or q.dim() != 3:
        raise ValueError("q must be a [B, Hq, d] tensor")
    if not isinstance(k_cache, torch.Tensor) or k_cache.dim() != 4:
        raise ValueError("k_cache must be a [B, Hkv, cap, d] tensor")
    if q.dtype not in (torch.float32, torch.bfloat16):
        raise ValueError(f"q must be float32 or bfloat16, got {q.dtype}")
    B, Hq, d = q.shape
    _, Hkv, cap, _ = k_cache.shape
    f32, i32 = torch.float32, torch.int32
    _expect(k_cache, "k_cache", (B, Hkv, cap, d), q.dtype)
    _expect(v_cache, "v_cache", (B, Hkv, cap, d), q.dtype)
    _expect(lens, "lens", (B, Hkv), i32)
    _expect(n_e, "n_e", (B, Hkv), i32)
    _expect(s_k, "s_k", (B, Hkv, d), f32)
    _expect(s_v, "s_v", (B, Hkv, d), f32)
    if summary == 0:
        _expect(S, "S", (B, Hkv, d, d), f32)
    elif summary == 1:
        if q.dtype == torch.bfloat16:
            _expect(S, "S (prepared)", (B, Hkv, 2, d, d), torch.bfloat16)
        else:
            _expect(S, "S (prepared)", (B, Hkv, d, d), f32)
    elif summary == 2:
        _expect(S, "S (half-precision prepared)", (B, Hkv, d, d), torch.bfloat16)
    elif summary == 3:
        _expect(S, "S (raw, bf16)", (B, Hkv, d, d), torch.bfloat16)
    else:
        raise ValueError(f"summary must be 0, 1, 2 or 3, got {summary}")
    if (k_new is None) != (v_new is None) or (need_new and k_new is None):
        raise ValueError("k_new and v_new must be given together" +
                         (" (required here)" if need_new else ""))
    _expect(k_new, "k_new", (B, Hkv, d), q.dtype, optional=True)
    _expect(v_new, "v_new", (B, Hkv, d), q.dtype, optional=True)
    _expect(out, "out", (B, Hq, d), q.dtype, optional=True)
    _expect(lse, "lse", (B, Hq), f32, optional=True)
    _expect(w_r, "w_r", (B, Hq), f32, optional=True)
    _expect(evicted, "evicted", (B, Hkv), i32, optional=True)
    _check_workspace(workspace)
    _same_device(dict(q=q, k_cache=k_cache, v_cache=v_cache, lens=lens, n_e=n_e, s_k=s_k,
                      s_v=s_v, S=S, k_new=k_new, v_new=v_new, out=out, lse=lse, w_r=w_r,
                      evicted=evicted, workspace=workspace))


def momentkv_decode_attn(q: torch.Tensor, k_cache: torch.Tensor, v_cache: torch.Tensor,
                         lens: torch.Tensor, n_e: torch.Tensor, s_k: torch.Tensor,
                         s_v: torch.Tensor, S: torch.Tensor, *, k_new: torch.Tensor | None = None,
                         v_new: torch.Tensor | None = None, max_len: int | None = None,
                         order: int = 1, scale: float = 0.0, tau: float = 1e-6,
                         n_split: int = 0, summary: int = 0,
                         out: torch.Tensor | None = None, lse: torch.Tensor | None = None,
                         w_r: torch.Tensor | None = None,
                         workspace: torch.Tensor | None = None):
    """Corrected decode attention (see the header).  Returns (out, lse, w_r, workspace).

    `S` is the raw sum (summary=0), the output of momentkv_prepare_summary (summary=1, or 2
    for its half-precision form), or the raw sum stored in bf16 (summary=3).

    `max_len` bounds lens after the append (defaults to the cache capacity).  The first
    int32 of the workspace is the sticky append-overflow flag.  The leading
    momentkv_decode_workspace_zero_bytes(p) bytes (the flag and the per-head arrival
    counters) are zeroed here the first time a workspace tensor is used with this prefix
    length (the flag included); calls leave the counters at zero.
    """
    _check_decode_args(q, k_cache, v_cache, lens, n_e, s_k, s_v, S, k_new, v_new, out, lse, w_r,
                       workspace, summary)
    cap = k_cache.shape[2]
    p = decode_params(q, k_cache, max_len=cap if max_len is None else max_len, order=order,
                      scale=scale, tau=tau, n_split=n_split, summary=summary)
    dev = q.device
    if out is None:
        out = torch.empty_like(q)
    nbytes = momentkv_decode_workspace_bytes(p)
    if nbytes == 0:
        code = lib().momentkv_decode_attn(ctypes.byref(p), *([None] * 13), None, 0, None)
        raise MomentKVError(code, "momentkv_decode_attn")
    ws = _workspace(nbytes, dev, workspace)
    _zero_prefix(ws, momentkv_decode_workspace_zero_bytes(p))
    code = lib().momentkv_decode_attn(
        ctypes.byref(p), _ptr(q), _ptr(k_cache), _ptr(v_cache), _ptr(lens), _ptr(k_new),
        _ptr(v_new), _ptr(n_e), _ptr(s_k), _ptr(s_v), _ptr(S), _ptr(out), _ptr(lse), _ptr(w_r),
        ws.data_ptr(), ws.numel(), _stream())
    if code != 0:
        raise MomentKVError(code, "momentkv_decode_attn")
    return out, lse, w_r, ws


def momentkv_decode_attn_noalloc(q: torch.Tensor, k_cache: torch.Tensor, v_cache: torch.Tensor,
                                 lens: torch.Tensor, n_e: torch.Tensor, s_k: torch.Tensor,
                                 s_v: torch.Tensor, S: torch.Tensor, *,
                                 k_new: torch.Tensor | None = None,
                                 v_new: torch.Tensor | None = None, max_len: int | None = None,
                                 order: int = 1, scale: float = 0.0, tau: float = 1e-6,
                                 n_split: int = 0, summary: int = 0, out: torch.Tensor,
                                 lse: torch.Tensor | None = None, w_r: torch.Tensor | None = None,
                                 flag: torch.Tensor | None = None):
    """The corrected decode with no workspace argument (see the header): the library keeps
    the partial results in its own per-GPU device array.  Every buffer, `out` included, is
    the caller's, so nothing is allocated here either.  `flag`: None or a one-element int32
    tensor that the call sets to 1 when an append finds a full cache.  Returns out."""
    _check_decode_args(q, k_cache, v_cache, lens, n_e, s_k, s_v, S, k_new, v_new, out, lse, w_r,
                       None, summary)
    _expect(flag, "flag", (1,), torch.int32, optional=True)
    _same_device(dict(q=q, flag=flag))
    cap = k_cache.shape[2]
    p = decode_params(q, k_cache, max_len=cap if max_len is None else max_len, order=order,
                      scale=scale, tau=tau, n_split=n_split, summary=summary)
    code = lib().momentkv_decode_attn_noalloc(
        ctypes.byref(p), _ptr(q), _ptr(k_cache), _ptr(v_cache), _ptr(lens), _ptr(k_new),
        _ptr(v_new), _ptr(n_e), _ptr(s_k), _ptr(s_v), _ptr(S), _ptr(out), _ptr(lse), _ptr(w_r),
        _ptr(flag), _stream())
    if code != 0:
        raise MomentKVError(code, "momentkv_decode_attn_noalloc")
    return out


def momentkv_decode_evict(q: torch.Tensor, k_cache: torch.Tensor, v_cache: torch.Tensor,
                          lens: torch.Tensor, n_e: torch.Tensor, s_k: torch.Tensor,
                          s_v: torch.Tensor, S: torch.Tensor, k_new: torch.Tensor,
                          v_new: torch.Tensor, budget: int, *, max_len: int | None = None,
                          order: int = 1, scale: float = 0.0, tau: float = 1e-6,
                          n_split: int = 0, out: torch.Tensor | None = None,
                          lse: torch.Tensor | None = None, w_r: torch.Tensor | None = None,
                          evicted: torch.Tensor | None = None,
                          workspace: torch.Tensor | None = None):
    """Decode step with moment-informed eviction (see the header).  The caches, lens and
    the raw summary (n_e, s_k, s_v, S) are updated in place.
    Returns (out, lse, w_r, evicted, workspace)."""
    _check_decode_args(q, k_cache, v_cache, lens, n_e, s_k, s_v, S, k_new, v_new, out, lse, w_r,
                       workspace, 0, evicted=evicted, need_new=True)
    cap = k_cache.shape[2]
    p = decode_params(q, k_cache, max_len=cap if max_len is None else max_len, order=order,
                      scale=scale, tau=tau, n_split=n_split, summary=0)
    dev = q.device
    if out is None:
        out = torch.empty_like(q)
    nbytes = momentkv_decode_evict_workspace_bytes(p)
    if nbytes == 0:
        code = lib().momentkv_decode_evict(ctypes.byref(p), int(budget), *([None] * 14), None,
                                           0, None)
        raise MomentKVError(code, "momentkv_decode_evict")
    fresh = workspace is None or workspace.numel() < nbytes
    ws = _workspace(nbytes, dev, workspace)
    if fresh:
        ws[:256].zero_()  # the sticky flag
    code = lib().momentkv_decode_evict(
        ctypes.byref(p), int(budget), _ptr(q), _ptr(k_cache), _ptr(v_cache), _ptr(lens),
        _ptr(k_new), _ptr(v_new), _ptr(n_e), _ptr(s_k), _ptr(s_v), _ptr(S), _ptr(out),
        _ptr(lse), _ptr(w_r), _ptr(evicted), ws.data_ptr(), ws.numel(), _stream())
    if code != 0:
        raise MomentKVError(code, "momentkv_decode_evict")
    return out, lse, w_r, evicted, ws
