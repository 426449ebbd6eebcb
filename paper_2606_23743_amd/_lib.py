"""ctypes binding of libsva.so (include/sva.h).  Argument marshalling only:
every step of the path runs in the library's HIP kernels.  torch supplies device
memory and the current stream; nothing here computes on the host, and there is
no fallback -- a missing or unloadable library raises.
"""
from __future__ import annotations

import ctypes
import os
import re
from typing import Optional, Tuple

HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(HERE, "libsva.so")
HEADER = os.path.join(os.path.dirname(HERE), "include", "sva.h")

SVA_OK, SVA_ERR_INVALID_ARG, SVA_ERR_SHAPE, SVA_ERR_ALIGNMENT, SVA_ERR_UNSUPPORTED, SVA_ERR_HIP = range(6)
SVA_BF16, SVA_F32 = 0, 1
SVA_SELECT_TOPK, SVA_SELECT_CUMMASS = 0, 1
SVA_SELECT_MAX_BLOCKS = 2048


class SvaError(RuntimeError):
    def __init__(self, status: int, what: str):
        self.status = status
        super().__init__(f"{what}: status {status} ({status_string(status)})")


class Problem(ctypes.Structure):
    _fields_ = [("batch", ctypes.c_int32), ("heads", ctypes.c_int32), ("seq_len", ctypes.c_int32),
                ("head_dim", ctypes.c_int32), ("grid_t", ctypes.c_int32), ("grid_h", ctypes.c_int32),
                ("grid_w", ctypes.c_int32), ("block_size", ctypes.c_int32),
                ("softmax_scale", ctypes.c_double), ("out_dtype", ctypes.c_int32)]


class RopeParams(ctypes.Structure):
    _fields_ = [("eps", ctypes.c_double), ("rope_base", ctypes.c_double)]


class Tokens(ctypes.Structure):
    _fields_ = [("batch", ctypes.c_int32), ("tokens", ctypes.c_int32), ("channels", ctypes.c_int32)]


class Fp8Tensors(ctypes.Structure):
    _fields_ = [("q8", ctypes.c_void_p), ("k8", ctypes.c_void_p), ("v8", ctypes.c_void_p),
                ("q_exp", ctypes.c_void_p), ("k_exp", ctypes.c_void_p), ("v_exp", ctypes.c_void_p),
                ("k_mean", ctypes.c_void_p)]


class SelectParams(ctypes.Structure):
    _fields_ = [("mode", ctypes.c_int32), ("keep_ratio", ctypes.c_double), ("topk", ctypes.c_int32),
                ("mass_threshold", ctypes.c_double), ("max_keep_ratio", ctypes.c_double),
                ("force_first_frame", ctypes.c_int32)]


_lib = None


def load(path: str = LIB_PATH) -> ctypes.CDLL:
    """Load libsva.so once; raise if it is missing (build it with
    `python -m paper_2606_23743_amd.build`)."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(path):
        raise RuntimeError(f"{path} not found: build the HIP library first "
                           "(python -m paper_2606_23743_amd.build)")
    lib = ctypes.CDLL(path)
    P, S = ctypes.POINTER(Problem), ctypes.POINTER(SelectParams)
    vp, i32p = ctypes.c_void_p, ctypes.POINTER(ctypes.c_int32)
    sig = {
        "sva_num_blocks": [P, i32p],
        "sva_max_keep": [P, S, i32p],
        "sva_pool_blocks": [P, vp, vp, vp, vp, vp],
        "sva_qknorm_rope_pool": [P, ctypes.POINTER(RopeParams), vp, vp, vp, vp, vp, vp, vp, vp, vp],
        "sva_select_blocks": [P, S, vp, vp, ctypes.c_int32, vp, vp, vp, vp],
        "sva_sparse_attention": [P, vp, vp, vp, vp, vp, ctypes.c_int32, vp, vp, vp],
        "sva_dense_attention": [P, vp, vp, vp, vp, vp, vp],
        "sva_remainder_workspace": [P, ctypes.POINTER(ctypes.c_size_t)],
        "sva_remainder_workspace_heads": [P, ctypes.c_int32, ctypes.POINTER(ctypes.c_size_t)],
        "sva_block_moments": [P, vp, vp, vp, vp, vp, vp],
        "sva_sparse_attention_remainder": [P, vp, vp, vp, vp, vp, vp, vp, ctypes.c_int32, vp,
                                           ctypes.c_size_t, vp, vp, vp],
        "sva_token_keep_count": [ctypes.POINTER(Tokens), ctypes.c_double, i32p],
        "sva_token_select_workspace": [ctypes.POINTER(Tokens), ctypes.POINTER(ctypes.c_size_t)],
        "sva_token_select": [ctypes.POINTER(Tokens), ctypes.c_double, vp, vp, vp, vp, vp,
                             ctypes.c_size_t, vp],
        "sva_token_select_noalloc": [ctypes.POINTER(Tokens), ctypes.c_double, vp, vp, vp, vp, vp],
        "sva_token_gather": [ctypes.POINTER(Tokens), ctypes.c_int32, vp, vp, vp, vp],
        "sva_token_scatter": [ctypes.POINTER(Tokens), ctypes.c_int32, vp, vp, vp, vp, vp],
        "sva_fp8_padded_len": [P, i32p],
        "sva_fp8_code_dim": [P, i32p],
        "sva_quantize_fp8": [P, vp, vp, vp, ctypes.POINTER(Fp8Tensors), vp],
        "sva_sparse_attention_fp8": [P, ctypes.POINTER(Fp8Tensors), vp, vp, ctypes.c_int32, vp, vp, vp],
        "sva_dense_attention_fp8": [P, ctypes.POINTER(Fp8Tensors), vp, vp, vp],
        "sva_status_string": [ctypes.c_int],
        "sva_version": [],
    }
    for name, args in sig.items():
        fn = getattr(lib, name)
        fn.argtypes = args
        fn.restype = ctypes.c_char_p if name == "sva_status_string" else ctypes.c_int
    _lib = lib
    return lib


def header_functions(header: str = HEADER):
    """Names of the functions include/sva.h declares."""
    text = open(header).read()
    return sorted(set(re.findall(r"^\s*(?:const\s+char\*|int)\s+(sva_\w+)\s*\(", text, re.M)))


def status_string(status: int) -> str:
    try:
        return load().sva_status_string(int(status)).decode()
    except Exception:  # pragma: no cover - only while reporting another error
        return "?"


def _check(status: int, what: str):
    if status != SVA_OK:
        raise SvaError(status, what)


# ----------------------------------------------------------------- parameters

def problem(batch, heads, seq_len, head_dim, grid, block_size, softmax_scale=0.0,
            out_dtype="bf16") -> Problem:
    t, h, w = grid
    return Problem(batch, heads, seq_len, head_dim, t, h, w, block_size, float(softmax_scale),
                   SVA_F32 if out_dtype in ("f32", "float32", SVA_F32) else SVA_BF16)


def problem_for(wl, out_dtype="bf16", softmax_scale=0.0) -> Problem:
    return problem(wl.batch, wl.heads, wl.seq_len, wl.head_dim, (wl.grid_t, wl.grid_h, wl.grid_w),
                   wl.block, softmax_scale, out_dtype)


def select_topk(keep_ratio: float = 0.0, topk: int = 0) -> SelectParams:
    return SelectParams(SVA_SELECT_TOPK, float(keep_ratio), int(topk), 0.0, 0.0, 0)


def select_mass(tau: float, max_keep_ratio: float, force_first_frame: bool) -> SelectParams:
    return SelectParams(SVA_SELECT_CUMMASS, 0.0, 0, float(tau), float(max_keep_ratio),
                        1 if force_first_frame else 0)


def select_for(wl, keep_ratio: Optional[float] = None) -> SelectParams:
    if wl.mode == "mass":
        return select_mass(wl.mass_threshold, wl.max_keep_ratio, wl.force_first_frame)
    if keep_ratio is not None:
        return select_topk(keep_ratio, 0)
    return select_topk(wl.keep_ratio, wl.topk)


def num_blocks(prob: Problem) -> int:
    out = ctypes.c_int32()
    _check(load().sva_num_blocks(ctypes.byref(prob), ctypes.byref(out)), "sva_num_blocks")
    return out.value


def max_keep(prob: Problem, sel: SelectParams) -> int:
    out = ctypes.c_int32()
    _check(load().sva_max_keep(ctypes.byref(prob), ctypes.byref(sel), ctypes.byref(out)), "sva_max_keep")
    return out.value


# ------------------------------------------------------------- device calls

def _torch():
    import torch
    return torch


def _ptr(t) -> Optional[int]:
    return None if t is None else t.data_ptr()


def _stream(stream) -> Optional[int]:
    torch = _torch()
    if stream is None:
        stream = torch.cuda.current_stream()
    return stream.cuda_stream if hasattr(stream, "cuda_stream") else int(stream)


def _side_stream(stream):
    """The stream a call was given, as a torch stream object, when it is not
    the current stream (None otherwise)."""
    torch = _torch()
    if stream is None:
        return None
    cur = torch.cuda.current_stream().cuda_stream
    if isinstance(stream, torch.cuda.Stream):
        return None if stream.cuda_stream == cur else stream
    h = int(stream.cuda_stream if hasattr(stream, "cuda_stream") else stream)
    return None if h == cur else torch.cuda.ExternalStream(h)


def _record(stream, *tensors):
    """Mark every tensor a call reads or writes as in use on the call's stream
    when that is not the current stream: the caching allocator then keeps the
    memory of a tensor freed meanwhile (a workspace or output allocated here
    on the current stream, or an input the caller drops) from being handed to
    another allocation until the work enqueued on that stream has finished."""
    s = _side_stream(stream)
    if s is None:
        return
    for x in tensors:
        if isinstance(x, dict):
            _record(stream, *x.values())
        elif x is not None:
            x.record_stream(s)


def _need(t, dtype, shape, name):
    torch = _torch()
    if not isinstance(t, torch.Tensor):
        raise TypeError(f"{name} must be a torch tensor")
    if not t.is_cuda:
        raise ValueError(f"{name} must be a device tensor")
    if t.dtype != dtype:
        raise TypeError(f"{name} must be {dtype}, got {t.dtype}")
    if tuple(t.shape) != tuple(shape):
        raise ValueError(f"{name} must have shape {tuple(shape)}, got {tuple(t.shape)}")
    if not t.is_contiguous():
        raise ValueError(f"{name} must be contiguous")


def _qkv_shape(prob):
    return (prob.batch, prob.heads, prob.seq_len, prob.head_dim)


def pool_blocks(prob: Problem, q, k, q_pool=None, k_pool=None, stream=None) -> Tuple:
    torch = _torch()
    nb = num_blocks(prob)
    shp = _qkv_shape(prob)
    _need(q, torch.bfloat16, shp, "q")
    _need(k, torch.bfloat16, shp, "k")
    pshape = (prob.batch, prob.heads, nb, prob.head_dim)
    if q_pool is None:
        q_pool = torch.empty(pshape, dtype=torch.float32, device=q.device)
    if k_pool is None:
        k_pool = torch.empty(pshape, dtype=torch.float32, device=q.device)
    _need(q_pool, torch.float32, pshape, "q_pool")
    _need(k_pool, torch.float32, pshape, "k_pool")
    _check(load().sva_pool_blocks(ctypes.byref(prob), _ptr(q), _ptr(k), _ptr(q_pool), _ptr(k_pool),
                                  _stream(stream)), "sva_pool_blocks")
    _record(stream, q, k, q_pool, k_pool)
    return q_pool, k_pool


def qknorm_rope_pool(prob: Problem, q_in, k_in, gamma_q, gamma_k, eps: float = 1e-6,
                     rope_base: float = 10000.0, q_out=None, k_out=None, q_pool=None, k_pool=None,
                     stream=None) -> Tuple:
    """RMSNorm + 3-D RoPE of Q and K with the block summaries of the written
    values (sva_qknorm_rope_pool).  q_out / k_out may be q_in / k_in (in place)."""
    torch = _torch()
    nb = num_blocks(prob)
    shp = _qkv_shape(prob)
    _need(q_in, torch.bfloat16, shp, "q_in")
    _need(k_in, torch.bfloat16, shp, "k_in")
    _need(gamma_q, torch.float32, (prob.head_dim,), "gamma_q")
    _need(gamma_k, torch.float32, (prob.head_dim,), "gamma_k")
    if q_out is None:
        q_out = torch.empty_like(q_in)
    if k_out is None:
        k_out = torch.empty_like(k_in)
    _need(q_out, torch.bfloat16, shp, "q_out")
    _need(k_out, torch.bfloat16, shp, "k_out")
    pshape = (prob.batch, prob.heads, nb, prob.head_dim)
    if q_pool is None:
        q_pool = torch.empty(pshape, dtype=torch.float32, device=q_in.device)
    if k_pool is None:
        k_pool = torch.empty(pshape, dtype=torch.float32, device=q_in.device)
    _need(q_pool, torch.float32, pshape, "q_pool")
    _need(k_pool, torch.float32, pshape, "k_pool")
    rp = RopeParams(float(eps), float(rope_base))
    _check(load().sva_qknorm_rope_pool(ctypes.byref(prob), ctypes.byref(rp), _ptr(q_in), _ptr(k_in),
                                       _ptr(gamma_q), _ptr(gamma_k), _ptr(q_out), _ptr(k_out),
                                       _ptr(q_pool), _ptr(k_pool), _stream(stream)),
           "sva_qknorm_rope_pool")
    _record(stream, q_in, k_in, gamma_q, gamma_k, q_out, k_out, q_pool, k_pool)
    return q_out, k_out, q_pool, k_pool


def select_blocks(prob: Problem, sel: SelectParams, q_pool, k_pool, kmax: Optional[int] = None,
                  kv_idx=None, kv_count=None, want_mask: bool = False, mask=None, stream=None) -> Tuple:
    torch = _torch()
    nb = num_blocks(prob)
    pshape = (prob.batch, prob.heads, nb, prob.head_dim)
    _need(q_pool, torch.float32, pshape, "q_pool")
    _need(k_pool, torch.float32, pshape, "k_pool")
    if kmax is None:
        kmax = max_keep(prob, sel)
    dev = q_pool.device
    if kv_idx is None:
        kv_idx = torch.empty((prob.batch, prob.heads, nb, kmax), dtype=torch.int32, device=dev)
    if kv_count is None:
        kv_count = torch.empty((prob.batch, prob.heads, nb), dtype=torch.int32, device=dev)
    _need(kv_idx, torch.int32, (prob.batch, prob.heads, nb, kmax), "kv_idx")
    _need(kv_count, torch.int32, (prob.batch, prob.heads, nb), "kv_count")
    if want_mask and mask is None:
        mask = torch.empty((prob.batch, prob.heads, nb, nb), dtype=torch.uint8, device=dev)
    if mask is not None:
        _need(mask, torch.uint8, (prob.batch, prob.heads, nb, nb), "mask")
    _check(load().sva_select_blocks(ctypes.byref(prob), ctypes.byref(sel), _ptr(q_pool), _ptr(k_pool),
                                    int(kmax), _ptr(kv_idx), _ptr(kv_count), _ptr(mask), _stream(stream)),
           "sva_select_blocks")
    _record(stream, q_pool, k_pool, kv_idx, kv_count, mask)
    return kv_idx, kv_count, mask


def _out_tensor(prob, like, out):
    torch = _torch()
    dt = torch.float32 if prob.out_dtype == SVA_F32 else torch.bfloat16
    if out is None:
        out = torch.empty(_qkv_shape(prob), dtype=dt, device=like.device)
    _need(out, dt, _qkv_shape(prob), "out")
    return out


def sparse_attention(prob: Problem, q, k, v, kv_idx, kv_count, out=None, want_lse: bool = False,
                     lse=None, stream=None) -> Tuple:
    torch = _torch()
    nb = num_blocks(prob)
    shp = _qkv_shape(prob)
    for t, n in ((q, "q"), (k, "k"), (v, "v")):
        _need(t, torch.bfloat16, shp, n)
    kmax = kv_idx.shape[-1]
    _need(kv_idx, torch.int32, (prob.batch, prob.heads, nb, kmax), "kv_idx")
    _need(kv_count, torch.int32, (prob.batch, prob.heads, nb), "kv_count")
    out = _out_tensor(prob, q, out)
    if want_lse and lse is None:
        lse = torch.empty(shp[:3], dtype=torch.float32, device=q.device)
    if lse is not None:
        _need(lse, torch.float32, shp[:3], "lse")
    _check(load().sva_sparse_attention(ctypes.byref(prob), _ptr(q), _ptr(k), _ptr(v), _ptr(kv_idx),
                                       _ptr(kv_count), int(kmax), _ptr(out), _ptr(lse), _stream(stream)),
           "sva_sparse_attention")
    _record(stream, q, k, v, kv_idx, kv_count, out, lse)
    return out, lse


def remainder_workspace(prob: Problem, heads: Optional[int] = None) -> int:
    """Workspace bytes of sparse_attention_remainder: for all (batch, head)
    pairs in one pass (sva_remainder_workspace), or for passes of `heads`
    pairs (sva_remainder_workspace_heads)."""
    out = ctypes.c_size_t(0)
    if heads is None:
        _check(load().sva_remainder_workspace(ctypes.byref(prob), ctypes.byref(out)), "sva_remainder_workspace")
    else:
        _check(load().sva_remainder_workspace_heads(ctypes.byref(prob), int(heads), ctypes.byref(out)),
               "sva_remainder_workspace_heads")
    return out.value


def block_moments(prob: Problem, k, v, kbar=None, vbar=None, moments=None, stream=None) -> Tuple:
    """sva_block_moments: (kbar bf16 [B, H, nB, D], vbar bf16 [B, H, nB, D],
    moments bf16 [B, H, nB, D, D] with M[e][d] = sum_t V[t][e] (K[t][d] - kbar[d]))."""
    torch = _torch()
    nb = num_blocks(prob)
    shp = _qkv_shape(prob)
    B, H, _, D = shp
    for t, n in ((k, "k"), (v, "v")):
        _need(t, torch.bfloat16, shp, n)
    if kbar is None:
        kbar = torch.empty((B, H, nb, D), dtype=torch.bfloat16, device=k.device)
    if vbar is None:
        vbar = torch.empty((B, H, nb, D), dtype=torch.bfloat16, device=k.device)
    if moments is None:
        moments = torch.empty((B, H, nb, D, D), dtype=torch.bfloat16, device=k.device)
    _need(kbar, torch.bfloat16, (B, H, nb, D), "kbar")
    _need(vbar, torch.bfloat16, (B, H, nb, D), "vbar")
    _need(moments, torch.bfloat16, (B, H, nb, D, D), "moments")
    _check(load().sva_block_moments(ctypes.byref(prob), _ptr(k), _ptr(v), _ptr(kbar), _ptr(vbar), _ptr(moments),
                                    _stream(stream)), "sva_block_moments")
    _record(stream, k, v, kbar, vbar, moments)
    return kbar, vbar, moments


def sparse_attention_remainder(prob: Problem, q, k, v, q_pool, k_pool, kv_idx, kv_count, out=None,
                               want_lse: bool = False, lse=None, workspace=None, stream=None) -> Tuple:
    """sva_sparse_attention_remainder: the kept blocks exactly plus the
    first-order remainder of the dropped ones.  workspace: a uint8 device
    tensor of remainder_workspace bytes (allocated when None), or of at least
    remainder_workspace(prob, 1), with which the (batch, head) pairs are done
    in groups of as many as fit."""
    torch = _torch()
    nb = num_blocks(prob)
    shp = _qkv_shape(prob)
    for t, n in ((q, "q"), (k, "k"), (v, "v")):
        _need(t, torch.bfloat16, shp, n)
    _need(q_pool, torch.float32, (prob.batch, prob.heads, nb, prob.head_dim), "q_pool")
    _need(k_pool, torch.float32, (prob.batch, prob.heads, nb, prob.head_dim), "k_pool")
    kmax = kv_idx.shape[-1]
    _need(kv_idx, torch.int32, (prob.batch, prob.heads, nb, kmax), "kv_idx")
    _need(kv_count, torch.int32, (prob.batch, prob.heads, nb), "kv_count")
    out = _out_tensor(prob, q, out)
    if want_lse and lse is None:
        lse = torch.empty(shp[:3], dtype=torch.float32, device=q.device)
    if lse is not None:
        _need(lse, torch.float32, shp[:3], "lse")
    if workspace is None:
        workspace = torch.empty(remainder_workspace(prob), dtype=torch.uint8, device=q.device)
    ws_min = remainder_workspace(prob, 1)
    if workspace.dtype != torch.uint8 or not workspace.is_cuda or workspace.numel() < ws_min:
        raise ValueError(f"workspace must be a uint8 device tensor of at least {ws_min} bytes")
    _check(load().sva_sparse_attention_remainder(
        ctypes.byref(prob), _ptr(q), _ptr(k), _ptr(v), _ptr(q_pool), _ptr(k_pool), _ptr(kv_idx), _ptr(kv_count),
        int(kmax), _ptr(workspace), int(workspace.numel()), _ptr(out), _ptr(lse), _stream(stream)),
        "sva_sparse_attention_remainder")
    _record(stream, q, k, v, q_pool, k_pool, kv_idx, kv_count, workspace, out, lse)
    return out, lse


def dense_attention(prob: Problem, q, k, v, out=None, want_lse: bool = False, lse=None,
                    stream=None) -> Tuple:
    torch = _torch()
    shp = _qkv_shape(prob)
    for t, n in ((q, "q"), (k, "k"), (v, "v")):
        _need(t, torch.bfloat16, shp, n)
    out = _out_tensor(prob, q, out)
    if want_lse and lse is None:
        lse = torch.empty(shp[:3], dtype=torch.float32, device=q.device)
    if lse is not None:
        _need(lse, torch.float32, shp[:3], "lse")
    _check(load().sva_dense_attention(ctypes.byref(prob), _ptr(q), _ptr(k), _ptr(v), _ptr(out),
                                      _ptr(lse), _stream(stream)), "sva_dense_attention")
    _record(stream, q, k, v, out, lse)
    return out, lse


# --------------------------------------------------------- fp8 (e4m3) attention

def fp8_padded_len(prob: Problem) -> int:
    out = ctypes.c_int32(0)
    _check(load().sva_fp8_padded_len(ctypes.byref(prob), ctypes.byref(out)), "sva_fp8_padded_len")
    return out.value


def fp8_code_dim(prob: Problem) -> int:
    out = ctypes.c_int32(0)
    _check(load().sva_fp8_code_dim(ctypes.byref(prob), ctypes.byref(out)), "sva_fp8_code_dim")
    return out.value


def _fp8_struct(t: dict) -> Fp8Tensors:
    return Fp8Tensors(*(_ptr(t.get(n)) for n in ("q8", "k8", "v8", "q_exp", "k_exp", "v_exp", "k_mean")))


def _need_fp8(prob: Problem, t: dict, need_mean: bool):
    torch = _torch()
    nb, npad, dp = num_blocks(prob), fp8_padded_len(prob), fp8_code_dim(prob)
    B, H, D = prob.batch, prob.heads, prob.head_dim
    _need(t["q8"], torch.uint8, (B, H, npad, dp), "q8")
    _need(t["k8"], torch.uint8, (B, H, npad, dp), "k8")
    _need(t["v8"], torch.uint8, (B, H, npad // 64, dp, 64), "v8")
    _need(t["q_exp"], torch.int32, (B, H, nb), "q_exp")
    _need(t["k_exp"], torch.int32, (B, H, nb), "k_exp")
    _need(t["v_exp"], torch.int32, (B, H, dp), "v_exp")
    if need_mean:
        _need(t["k_mean"], torch.bfloat16, (B, H, D), "k_mean")


def quantize_fp8(prob: Problem, q, k, v, out: Optional[dict] = None, stream=None) -> dict:
    """e4m3 codes and power-of-two exponents of Q, K (smoothed) and V
    (sva_quantize_fp8).  Returns {q8, k8, v8, q_exp, k_exp, v_exp, k_mean}."""
    torch = _torch()
    shp = _qkv_shape(prob)
    for t, n in ((q, "q"), (k, "k"), (v, "v")):
        _need(t, torch.bfloat16, shp, n)
    if out is None:
        nb, npad, dp = num_blocks(prob), fp8_padded_len(prob), fp8_code_dim(prob)
        B, H, D = prob.batch, prob.heads, prob.head_dim
        dev = q.device
        out = {"q8": torch.empty((B, H, npad, dp), dtype=torch.uint8, device=dev),
               "k8": torch.empty((B, H, npad, dp), dtype=torch.uint8, device=dev),
               "v8": torch.empty((B, H, npad // 64, dp, 64), dtype=torch.uint8, device=dev),
               "q_exp": torch.empty((B, H, nb), dtype=torch.int32, device=dev),
               "k_exp": torch.empty((B, H, nb), dtype=torch.int32, device=dev),
               "v_exp": torch.empty((B, H, dp), dtype=torch.int32, device=dev),
               "k_mean": torch.empty((B, H, D), dtype=torch.bfloat16, device=dev)}
    _need_fp8(prob, out, True)
    st = _fp8_struct(out)
    _check(load().sva_quantize_fp8(ctypes.byref(prob), _ptr(q), _ptr(k), _ptr(v), ctypes.byref(st),
                                   _stream(stream)), "sva_quantize_fp8")
    _record(stream, q, k, v, out)
    return out


def sparse_attention_fp8(prob: Problem, quant: dict, kv_idx, kv_count, out=None,
                         want_lse: bool = False, lse=None, stream=None) -> Tuple:
    """Block-sparse attention on the codes of quantize_fp8 (sva_sparse_attention_fp8)."""
    torch = _torch()
    nb = num_blocks(prob)
    shp = _qkv_shape(prob)
    _need_fp8(prob, quant, False)
    kmax = kv_idx.shape[-1]
    _need(kv_idx, torch.int32, (prob.batch, prob.heads, nb, kmax), "kv_idx")
    _need(kv_count, torch.int32, (prob.batch, prob.heads, nb), "kv_count")
    ref = quant["q8"]
    if out is None:
        dt = torch.float32 if prob.out_dtype == SVA_F32 else torch.bfloat16
        out = torch.empty(shp, dtype=dt, device=ref.device)
    _need(out, torch.float32 if prob.out_dtype == SVA_F32 else torch.bfloat16, shp, "out")
    if want_lse and lse is None:
        lse = torch.empty(shp[:3], dtype=torch.float32, device=ref.device)
    if lse is not None:
        _need(lse, torch.float32, shp[:3], "lse")
    st = _fp8_struct(quant)
    _check(load().sva_sparse_attention_fp8(ctypes.byref(prob), ctypes.byref(st), _ptr(kv_idx),
                                           _ptr(kv_count), int(kmax), _ptr(out), _ptr(lse),
                                           _stream(stream)), "sva_sparse_attention_fp8")
    _record(stream, quant, kv_idx, kv_count, out, lse)
    return out, lse


def dense_attention_fp8(prob: Problem, quant: dict, out=None, want_lse: bool = False, lse=None,
                        stream=None) -> Tuple:
    """Every block kept, on the codes of quantize_fp8 (sva_dense_attention_fp8)."""
    torch = _torch()
    shp = _qkv_shape(prob)
    _need_fp8(prob, quant, False)
    ref = quant["q8"]
    dt = torch.float32 if prob.out_dtype == SVA_F32 else torch.bfloat16
    if out is None:
        out = torch.empty(shp, dtype=dt, device=ref.device)
    _need(out, dt, shp, "out")
    if want_lse and lse is None:
        lse = torch.empty(shp[:3], dtype=torch.float32, device=ref.device)
    if lse is not None:
        _need(lse, torch.float32, shp[:3], "lse")
    st = _fp8_struct(quant)
    _check(load().sva_dense_attention_fp8(ctypes.byref(prob), ctypes.byref(st), _ptr(out), _ptr(lse),
                                          _stream(stream)), "sva_dense_attention_fp8")
    _record(stream, quant, out, lse)
    return out, lse


# ------------------------------------------------------------- token pruning

def tokens(batch: int, n_tokens: int, channels: int) -> Tokens:
    return Tokens(int(batch), int(n_tokens), int(channels))


def token_keep_count(t: Tokens, keep_ratio: float) -> int:
    out = ctypes.c_int32(0)
    _check(load().sva_token_keep_count(ctypes.byref(t), float(keep_ratio), ctypes.byref(out)),
           "sva_token_keep_count")
    return out.value


def token_select_workspace(t: Tokens) -> int:
    out = ctypes.c_size_t(0)
    _check(load().sva_token_select_workspace(ctypes.byref(t), ctypes.byref(out)),
           "sva_token_select_workspace")
    return out.value


def token_select(x, keep_ratio: float, scores=None, kept_idx=None, kept_pos=None,
                 workspace=None, stream=None) -> Tuple:
    """feat_norm scores and kept tokens of hidden states x (bf16 [B, N, C]),
    sva_token_select: returns (scores float64 [B, N], kept_idx int32 [B, k]
    ascending, kept_pos int32 [B, N] with -1 for dropped tokens).  workspace:
    a uint8 device tensor of token_select_workspace bytes (allocated when
    None; pass one to reuse it)."""
    torch = _torch()
    if x.dim() != 3:
        raise ValueError("x must be [B, N, C]")
    B, N, C = x.shape
    t = tokens(B, N, C)
    k = token_keep_count(t, keep_ratio)
    _need(x, torch.bfloat16, (B, N, C), "x")
    if scores is None:
        scores = torch.empty((B, N), dtype=torch.float64, device=x.device)
    if kept_idx is None:
        kept_idx = torch.empty((B, k), dtype=torch.int32, device=x.device)
    if kept_pos is None:
        kept_pos = torch.empty((B, N), dtype=torch.int32, device=x.device)
    _need(scores, torch.float64, (B, N), "scores")
    _need(kept_idx, torch.int32, (B, k), "kept_idx")
    _need(kept_pos, torch.int32, (B, N), "kept_pos")
    ws_bytes = token_select_workspace(t)
    if workspace is None:
        workspace = torch.empty(ws_bytes, dtype=torch.uint8, device=x.device)
    if not (isinstance(workspace, torch.Tensor) and workspace.is_cuda and workspace.is_contiguous()
            and workspace.numel() * workspace.element_size() >= ws_bytes):
        raise ValueError(f"workspace must be a contiguous device tensor of >= {ws_bytes} bytes")
    _check(load().sva_token_select(ctypes.byref(t), float(keep_ratio), _ptr(x), _ptr(scores),
                                   _ptr(kept_idx), _ptr(kept_pos), _ptr(workspace),
                                   workspace.numel() * workspace.element_size(), _stream(stream)),
           "sva_token_select")
    _record(stream, x, scores, kept_idx, kept_pos, workspace)
    return scores, kept_idx, kept_pos


def token_select_noalloc(x, keep_ratio: float, scores=None, kept_idx=None, kept_pos=None, stream=None) -> Tuple:
    """sva_token_select_noalloc: token_select with the library's static
    workspace (at most 16 batch entries; calls on one GPU must not overlap).
    Outputs are allocated here when not given; the library call itself
    allocates nothing."""
    torch = _torch()
    if x.dim() != 3:
        raise ValueError("x must be [B, N, C]")
    B, N, C = x.shape
    t = tokens(B, N, C)
    k = token_keep_count(t, keep_ratio)
    _need(x, torch.bfloat16, (B, N, C), "x")
    if scores is None:
        scores = torch.empty((B, N), dtype=torch.float64, device=x.device)
    if kept_idx is None:
        kept_idx = torch.empty((B, k), dtype=torch.int32, device=x.device)
    if kept_pos is None:
        kept_pos = torch.empty((B, N), dtype=torch.int32, device=x.device)
    _need(scores, torch.float64, (B, N), "scores")
    _need(kept_idx, torch.int32, (B, k), "kept_idx")
    _need(kept_pos, torch.int32, (B, N), "kept_pos")
    _check(load().sva_token_select_noalloc(ctypes.byref(t), float(keep_ratio), _ptr(x), _ptr(scores),
                                           _ptr(kept_idx), _ptr(kept_pos), _stream(stream)),
           "sva_token_select_noalloc")
    _record(stream, x, scores, kept_idx, kept_pos)
    return scores, kept_idx, kept_pos


def token_gather(x, kept_idx, x_kept=None, stream=None):
    """x_kept[b, j] = x[b, kept_idx[b, j]] (sva_token_gather)."""
    torch = _torch()
    B, N, C = x.shape
    k = kept_idx.shape[1]
    _need(x, torch.bfloat16, (B, N, C), "x")
    _need(kept_idx, torch.int32, (B, k), "kept_idx")
    if x_kept is None:
        x_kept = torch.empty((B, k, C), dtype=torch.bfloat16, device=x.device)
    _need(x_kept, torch.bfloat16, (B, k, C), "x_kept")
    _check(load().sva_token_gather(ctypes.byref(tokens(B, N, C)), k, _ptr(x), _ptr(kept_idx),
                                   _ptr(x_kept), _stream(stream)), "sva_token_gather")
    _record(stream, x, kept_idx, x_kept)
    return x_kept


def token_scatter(y_kept, kept_pos, base, out=None, stream=None):
    """out[b, n] = y_kept[b, kept_pos[b, n]] for kept tokens, base[b, n] for the
    others (sva_token_scatter); out may be base (in place)."""
    torch = _torch()
    B, N, C = base.shape
    k = y_kept.shape[1]
    _need(y_kept, torch.bfloat16, (B, k, C), "y_kept")
    _need(kept_pos, torch.int32, (B, N), "kept_pos")
    _need(base, torch.bfloat16, (B, N, C), "base")
    if out is None:
        out = torch.empty_like(base)
    _need(out, torch.bfloat16, (B, N, C), "out")
    _check(load().sva_token_scatter(ctypes.byref(tokens(B, N, C)), k, _ptr(y_kept), _ptr(kept_pos),
                                    _ptr(base), _ptr(out), _stream(stream)), "sva_token_scatter")
    _record(stream, y_kept, kept_pos, base, out)
    return out
