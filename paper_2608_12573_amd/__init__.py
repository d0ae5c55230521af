"""Prof-K top-k selection on MI355X: Python binding of libprofk.so.

This module only marshals arguments: every step of the selection runs in the
HIP kernels of libprofk.so (built by paper_2608_12573_amd.build).  PyTorch
provides device memory and the current stream.  If the library has not been
built, every call raises instead of computing anything on the CPU.

    vals, idx, info = topk(x, k)                  # x: 1-D fp32/bf16 CUDA tensor
    vals, idx, info = topk_rows(x, k)             # x: [B, D]
    vals, idx, info = batchtopk(x, k_row)         # global top-(B*k_row) of [B, D]
"""

import ctypes
import os
import re

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libprofk.so")
HEADER_PATH = os.path.join(os.path.dirname(_HERE), "include", "profk.h")

F32 = 0
BF16 = 1
MODE_FILTER, MODE_DIRECT = 0, 1
FORCE_AUTO, FORCE_FILTER, FORCE_DIRECT = 0, 1, 2
STATUS_FILTERED, STATUS_UNDERFLOW, STATUS_OVERFLOW, STATUS_DIRECT = 0, 1, 2, 3
OK, EINVAL, EDTYPE, EWORKSPACE, ENULL, EHIP = 0, -1, -2, -3, -4, -5
NOALLOC_SCRATCH_BYTES = 16 << 20   # PROFK_NOALLOC_SCRATCH_BYTES of include/profk.h


class PlanOpts(ctypes.Structure):
    _fields_ = [("S_min", ctypes.c_int32), ("S_max", ctypes.c_int32),
                ("cost_ratio", ctypes.c_double), ("eps_split", ctypes.c_double),
                ("paper_literal", ctypes.c_int32), ("force_mode", ctypes.c_int32),
                ("lexicographic", ctypes.c_int32)]


class Plan(ctypes.Structure):
    _fields_ = [("N", ctypes.c_int64), ("k", ctypes.c_int64),
                ("eps", ctypes.c_double), ("recall", ctypes.c_double),
                ("k_req", ctypes.c_int64), ("S", ctypes.c_int64), ("t", ctypes.c_int64),
                ("M", ctypes.c_int64), ("mode", ctypes.c_int32), ("lexicographic", ctypes.c_int32),
                ("p_underflow", ctypes.c_double), ("p_overflow", ctypes.c_double)]

    def as_dict(self):
        return {name: getattr(self, name) for name, _ in self._fields_}


INFO_DTYPE = np.dtype([("count", "<u8"), ("tau_key", "<u4"), ("status", "<i4"), ("n_valid", "<i8")])
INFO_BYTES = INFO_DTYPE.itemsize


class ProfkError(RuntimeError):
    pass


_lib = None


def lib():
    """The loaded libprofk.so; raises when it has not been built.

    PyTorch-ROCm ships its own HIP runtime.  Importing torch first makes the
    library's libamdhip64.so.7 dependency resolve to that same runtime (by
    soname), so tensors, streams and our kernels share one HIP instance;
    loading the library first would bring in a second runtime whose launches
    cannot use torch's streams."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise ProfkError(f"{LIB_PATH} is missing: run paper_2608_12573_amd.build.build() first")
        try:
            import torch  # noqa: F401  (see the docstring)
        except ImportError:
            pass
        L = ctypes.CDLL(LIB_PATH)
        vp, i32, i64, u32, u64, dbl = (ctypes.c_void_p, ctypes.c_int32, ctypes.c_int64,
                                       ctypes.c_uint32, ctypes.c_uint64, ctypes.c_double)
        P = ctypes.POINTER
        L.profk_default_opts.argtypes = [P(PlanOpts)]
        L.profk_default_row_opts.argtypes = [P(PlanOpts)]
        L.profk_default_sae_opts.argtypes = [P(PlanOpts)]
        L.profk_plan.argtypes = [i64, i64, dbl, dbl, P(PlanOpts), P(Plan)]
        L.profk_plan_rows.argtypes = [i64, i64, dbl, dbl, P(PlanOpts), P(Plan)]
        L.profk_workspace_size.argtypes = [P(Plan), i32, i64]
        L.profk_workspace_size.restype = ctypes.c_size_t
        L.profk_topk.argtypes = [P(Plan), i32, vp, i64, i64, u64, vp, vp, vp, ctypes.c_size_t, vp, vp]
        L.profk_topk_tau.argtypes = [P(Plan), i32, vp, i64, i64, u32, vp, vp, vp, ctypes.c_size_t, vp, vp]
        L.profk_topk_simple.argtypes = [vp, i64, i64, u64, vp, vp]
        L.profk_topk_noalloc.argtypes = [P(Plan), i32, vp, i64, i64, u64, vp, vp, vp, vp]
        L.profk_topk_rows.argtypes = [P(Plan), i32, vp, i64, i64, i64, i64, u64, vp, vp, vp,
                                      ctypes.c_size_t, vp, vp]
        L.profk_batchtopk.argtypes = [P(Plan), i32, vp, i64, i64, i64, u64, vp, vp, vp,
                                      ctypes.c_size_t, vp, vp]
        L.profk_debug_sample_indices.argtypes = [u64, i64, i64, i64, vp, vp]
        L.profk_debug_filter.argtypes = [P(Plan), i32, vp, i64, u32, vp, vp, vp, vp, ctypes.c_size_t, vp]
        L.profk_debug_read_probe.argtypes = [vp, u64, i32, i32, vp, P(u32), vp]
        L.profk_status_string.argtypes = [ctypes.c_int]
        L.profk_status_string.restype = ctypes.c_char_p
        L.profk_last_hip_error.restype = ctypes.c_int
        L.profk_set_trace_events.argtypes = [vp, vp]
        sz = ctypes.c_size_t
        L.profk_sae_workspace_size.argtypes = [P(Plan), i64, i64]
        L.profk_sae_workspace_size.restype = sz
        L.profk_sae_encode_topk.argtypes = [P(Plan), vp, vp, vp, i64, i64, i64, i64, u64, vp, vp, vp, sz, vp, vp]
        L.profk_sae_encode_dense.argtypes = [vp, vp, vp, i64, i64, i64, vp, vp]
        L.profk_sae_decode_workspace_size.argtypes = [i64, i64]
        L.profk_sae_decode_workspace_size.restype = sz
        L.profk_sae_decode.argtypes = [vp, vp, i64, vp, vp, i64, i64, i64, vp, vp, sz, vp]
        L.profk_debug_sae_sample.argtypes = [P(Plan), vp, vp, vp, i64, i64, i64, u64, vp, vp, sz, vp]
        _lib = L
    return _lib


def header_functions():
    """Names of the functions include/profk.h declares."""
    with open(HEADER_PATH) as f:
        text = f.read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(profk_\w+)\s*\(", text)))


def _check(rc):
    if rc != OK:
        msg = lib().profk_status_string(rc).decode()
        if rc == EHIP:
            msg += f" (hipError {lib().profk_last_hip_error()})"
        raise ProfkError(msg)


def opts(flat=True, sae=False, **kw):
    o = PlanOpts()
    if sae:
        lib().profk_default_sae_opts(ctypes.byref(o))
    else:
        (lib().profk_default_opts if flat else lib().profk_default_row_opts)(ctypes.byref(o))
    for key, val in kw.items():
        setattr(o, key, val)
    return o


def plan(N, k, eps=1e-6, recall=1.0, **kw):
    """profk_plan: (S, t, M) for N values and top-k."""
    p = Plan()
    _check(lib().profk_plan(N, k, eps, recall, ctypes.byref(opts(True, **kw)), ctypes.byref(p)))
    return p


def plan_sae(B, d_dict, k_row, eps=1e-6, recall=1.0, **kw):
    """profk_plan for the fused SAE path (N = B*d_dict, K = B*k_row) with
    profk_default_sae_opts."""
    p = Plan()
    _check(lib().profk_plan(B * d_dict, B * k_row, eps, recall, ctypes.byref(opts(True, sae=True, **kw)),
                            ctypes.byref(p)))
    return p


def plan_rows(D, k, eps=1e-6, recall=1.0, **kw):
    """profk_plan_rows: the per-row plan for rows of D values."""
    p = Plan()
    _check(lib().profk_plan_rows(D, k, eps, recall, ctypes.byref(opts(False, **kw)), ctypes.byref(p)))
    return p


def workspace_size(p, dtype, batch=1):
    return int(lib().profk_workspace_size(ctypes.byref(p), dtype, batch))


# ----------------------------------------------------------- torch side ---

def _torch():
    import torch
    return torch


def _dtype_code(t):
    torch = _torch()
    if t.dtype == torch.float32:
        return F32
    if t.dtype == torch.bfloat16:
        return BF16
    raise ProfkError(f"unsupported dtype {t.dtype}")


def _stream():
    torch = _torch()
    return ctypes.c_void_p(torch.cuda.current_stream().cuda_stream)


def _ptr(t):
    return ctypes.c_void_p(t.data_ptr()) if t is not None else None


def workspace(p, dtype, batch=1, device="cuda"):
    torch = _torch()
    return torch.empty(max(workspace_size(p, dtype, batch), 1), dtype=torch.uint8, device=device)


def read_info(info_tensor):
    """Host copy of profk_info_t records (synchronises the tensor's stream)."""
    raw = info_tensor.cpu().numpy().tobytes()
    return np.frombuffer(raw, dtype=INFO_DTYPE)


def _on_device(t, name, device):
    """t must be a CUDA tensor on `device` (checked after its layout, so that
    every layout rule is reported the same way with or without a GPU)."""
    if not t.is_cuda:
        raise ProfkError(f"{name} must be a CUDA tensor (got device {t.device})")
    if device is not None and t.device != device:
        raise ProfkError(f"{name} is on {t.device}, the input on {device}")


def _input(x, name, dims, dtypes=(F32, BF16), layout="contiguous"):
    """Checks an input tensor: rank, dtype, memory layout, then device.
    layout: "contiguous", or "rows" (unit column stride, rows at any
    stride at least D apart)."""
    torch = _torch()
    if not isinstance(x, torch.Tensor):
        raise ProfkError(f"{name} must be a torch tensor")
    if x.dim() != dims:
        raise ProfkError(f"{name} must have {dims} dimension(s), got shape {tuple(x.shape)}")
    dt = _dtype_code(x)
    if dt not in dtypes:
        raise ProfkError(f"{name} must be {' or '.join('float32' if d == F32 else 'bfloat16' for d in dtypes)}")
    if layout == "contiguous" and not x.is_contiguous():
        raise ProfkError(f"{name} must be contiguous (strides {tuple(x.stride())})")
    if layout == "rows" and (x.stride(1) != 1 or (x.shape[0] > 1 and x.stride(0) < x.shape[1])):
        raise ProfkError(f"{name} must be [B, D] with unit column stride and rows at least D apart "
                         f"(strides {tuple(x.stride())})")
    _on_device(x, name, None)
    return dt


def _buffer(t, name, dtype, numel, device):
    """A caller-given output: the dtype, at least `numel` contiguous
    elements, on the input's device."""
    torch = _torch()
    if not isinstance(t, torch.Tensor):
        raise ProfkError(f"{name} must be a torch tensor")
    if dtype is not None and t.dtype != dtype:
        raise ProfkError(f"{name} must be {dtype}, got {t.dtype}")
    if not t.is_contiguous() or t.numel() < numel:
        raise ProfkError(f"{name} must be contiguous with at least {numel} elements")
    _on_device(t, name, device)


def _bytes_buffer(t, name, nbytes, device):
    """A caller-given workspace or report buffer of at least nbytes bytes."""
    torch = _torch()
    if not isinstance(t, torch.Tensor) or not t.is_contiguous():
        raise ProfkError(f"{name} must be a contiguous torch tensor")
    if t.numel() * t.element_size() < nbytes:
        raise ProfkError(f"{name} holds {t.numel() * t.element_size()} bytes, {nbytes} needed")
    _on_device(t, name, device)


def _nbytes(t):
    return t.numel() * t.element_size()


def _outputs(x, n, out, info, n_info):
    """Preallocated or new (values, int64 indices) and info for n results."""
    torch = _torch()
    if out is None:
        out = (torch.empty(n, dtype=x.dtype, device=x.device),
               torch.empty(n, dtype=torch.int64, device=x.device))
    else:
        _buffer(out[0], "out[0]", x.dtype, n, x.device)
        _buffer(out[1], "out[1]", torch.int64, n, x.device)
    if info is None:
        info = torch.empty(n_info * INFO_BYTES, dtype=torch.uint8, device=x.device)
    else:
        _bytes_buffer(info, "info", n_info * INFO_BYTES, x.device)
    return out, info


def _workspace_for(p, dt, batch, ws, device):
    need = workspace_size(p, dt, batch)
    if need == 0:
        raise ProfkError("the plan does not fit this call (N, k or dtype)")
    if ws is None:
        return workspace(p, dt, batch, device)
    _bytes_buffer(ws, "ws", need, device)
    return ws


def topk(x, k, eps=1e-6, recall=1.0, seed=0, p=None, ws=None, out=None, info=None):
    """Top-k of a 1-D fp32/bf16 CUDA tensor: (values, int64 indices, info)."""
    dt = _input(x, "x", 1)
    N = x.numel()
    p = p if p is not None else plan(N, k, eps, recall)
    ws = _workspace_for(p, dt, 1, ws, x.device)
    out, info = _outputs(x, k, out, info, 1)
    _check(lib().profk_topk(ctypes.byref(p), dt, _ptr(x), N, k, seed, _ptr(out[0]), _ptr(out[1]),
                            _ptr(ws), _nbytes(ws), _stream(), _ptr(info)))
    return out[0], out[1], info


def topk_noalloc(x, k, eps=1e-6, recall=1.0, seed=0, p=None, out=None, info=None):
    """profk_topk_noalloc: topk with the library's fixed per-GPU scratch as
    the workspace (no device allocation by the library)."""
    dt = _input(x, "x", 1)
    N = x.numel()
    p = p if p is not None else plan(N, k, eps, recall)
    out, info = _outputs(x, k, out, info, 1)
    _check(lib().profk_topk_noalloc(ctypes.byref(p), dt, _ptr(x), N, k, seed, _ptr(out[0]), _ptr(out[1]),
                                    _stream(), _ptr(info)))
    return out[0], out[1], info


def topk_tau(x, k, tau_key, p, ws=None, eps=1e-6):
    """profk_topk_tau: the pipeline with the threshold given (forces the
    fallback paths on purpose)."""
    dt = _input(x, "x", 1)
    N = x.numel()
    ws = _workspace_for(p, dt, 1, ws, x.device)
    (vals, idx), info = _outputs(x, k, None, None, 1)
    _check(lib().profk_topk_tau(ctypes.byref(p), dt, _ptr(x), N, k, tau_key, _ptr(vals), _ptr(idx),
                                _ptr(ws), _nbytes(ws), _stream(), _ptr(info)))
    return vals, idx, info


def topk_simple(x, k, seed=0):
    """profk_topk_simple: fp32 only, synchronous, library-held workspace."""
    _input(x, "x", 1, dtypes=(F32,))
    (vals, idx), _ = _outputs(x, k, None, None, 1)
    _check(lib().profk_topk_simple(_ptr(x), x.numel(), k, seed, _ptr(vals), _ptr(idx)))
    return vals, idx


def topk_rows(x, k, eps=1e-6, recall=1.0, seed=0, p=None, ws=None, out=None, info=None):
    """Per-row top-k of a [B, D] CUDA tensor (rows may be strided)."""
    dt = _input(x, "x", 2, layout="rows")
    B, D = x.shape
    p = p if p is not None else plan_rows(D, k, eps, recall)
    ws = _workspace_for(p, dt, B, ws, x.device)
    out, info = _outputs(x, B * k, out, info, B)
    _check(lib().profk_topk_rows(ctypes.byref(p), dt, _ptr(x), B, D, x.stride(0), k, seed,
                                 _ptr(out[0]), _ptr(out[1]), _ptr(ws), _nbytes(ws), _stream(),
                                 _ptr(info)))
    return out[0].view(B, k), out[1].view(B, k), info


def batchtopk(x, k_row, eps=1e-6, recall=1.0, seed=0, p=None, ws=None, out=None, info=None):
    """BatchTopK: the B*k_row largest entries of a contiguous [B, D] tensor,
    with flat indices row*D + col."""
    dt = _input(x, "x", 2)
    B, D = x.shape
    K = B * k_row
    p = p if p is not None else plan(B * D, K, eps, recall)
    ws = _workspace_for(p, dt, 1, ws, x.device)
    out, info = _outputs(x, K, out, info, 1)
    _check(lib().profk_batchtopk(ctypes.byref(p), dt, _ptr(x), B, D, k_row, seed, _ptr(out[0]),
                                 _ptr(out[1]), _ptr(ws), _nbytes(ws), _stream(), _ptr(info)))
    return out[0], out[1], info


def debug_sample_indices(seed, row, S, N, device="cuda"):
    torch = _torch()
    out = torch.empty(S, dtype=torch.int64, device=device)
    _on_device(out, "out", None)
    _check(lib().profk_debug_sample_indices(seed, row, S, N, _ptr(out), _stream()))
    return out


def debug_filter(x, tau_key, p, ws=None):
    """Stage 3 alone: (buffer keys, buffer indices, count) for a given tau."""
    torch = _torch()
    dt = _input(x, "x", 1)
    ws = _workspace_for(p, dt, 1, ws, x.device)
    bk = torch.empty(p.M, dtype=torch.int32, device=x.device)
    bi = torch.empty(p.M, dtype=torch.int32, device=x.device)
    cnt = torch.empty(1, dtype=torch.int32, device=x.device)
    _check(lib().profk_debug_filter(ctypes.byref(p), dt, _ptr(x), x.numel(), tau_key, _ptr(bk), _ptr(bi),
                                    _ptr(cnt), _ptr(ws), _nbytes(ws), _stream()))
    return bk, bi, cnt


def debug_read_probe(x, blocks_per_cu=2, loads_per_lane=4, out=None):
    """profk_debug_read_probe over the bytes of a contiguous CUDA tensor whose
    size is a multiple of 16 bytes: (per-workgroup XOR words, workgroups)."""
    torch = _torch()
    if not isinstance(x, torch.Tensor) or not x.is_contiguous():
        raise ProfkError("x must be a contiguous tensor")
    _on_device(x, "x", None)
    if out is None:
        out = torch.empty(1024, dtype=torch.int32, device=x.device)
    else:
        _buffer(out, "out", torch.int32, 1024, x.device)
    grid = ctypes.c_uint32(0)
    _check(lib().profk_debug_read_probe(_ptr(x), _nbytes(x), blocks_per_cu, loads_per_lane, _ptr(out),
                                        ctypes.byref(grid), _stream()))
    return out, int(grid.value)


# ------------------------------------------------------ BatchTopK SAE layer ---

def _sae_shape(x, w_enc, b_enc):
    torch = _torch()
    if x.dim() != 2 or w_enc.dim() != 2 or x.shape[1] != w_enc.shape[1] or b_enc.shape != (w_enc.shape[0],):
        raise ProfkError("x [B, d_model], w_enc [d_dict, d_model] and b_enc [d_dict] required")
    if x.dtype != torch.bfloat16 or w_enc.dtype != torch.bfloat16 or b_enc.dtype != torch.float32:
        raise ProfkError("x and w_enc must be bfloat16, b_enc float32")
    if not (x.is_contiguous() and w_enc.is_contiguous() and b_enc.is_contiguous()):
        raise ProfkError("x, w_enc and b_enc must be contiguous")
    _on_device(x, "x", None)
    _on_device(w_enc, "w_enc", x.device)
    _on_device(b_enc, "b_enc", x.device)
    return x.shape[0], x.shape[1], w_enc.shape[0]


def sae_workspace(p, B, d_dict, device="cuda"):
    torch = _torch()
    n = int(lib().profk_sae_workspace_size(ctypes.byref(p), B, d_dict))
    if n == 0:
        raise ProfkError("plan does not match the latent shape")
    return torch.empty(n, dtype=torch.uint8, device=device)


def sae_encode_topk(x, w_enc, b_enc, k_row, eps=1e-6, recall=1.0, seed=0, p=None, ws=None, out=None,
                    info=None):
    """BatchTopK over the SAE latents relu(x w_enc^T + b_enc), with Prof-K
    fused into the encoder GEMM: (values fp32 [K], flat indices [K], info)."""
    torch = _torch()
    B, d_model, d_dict = _sae_shape(x, w_enc, b_enc)
    K = B * k_row
    p = p if p is not None else plan_sae(B, d_dict, k_row, eps, recall)
    if ws is None:
        ws = sae_workspace(p, B, d_dict, x.device)
    else:
        _bytes_buffer(ws, "ws", int(lib().profk_sae_workspace_size(ctypes.byref(p), B, d_dict)), x.device)
    if out is None:
        out = (torch.empty(K, dtype=torch.float32, device=x.device),
               torch.empty(K, dtype=torch.int64, device=x.device))
    else:
        _buffer(out[0], "out[0]", torch.float32, K, x.device)
        _buffer(out[1], "out[1]", torch.int64, K, x.device)
    if info is None:
        info = torch.empty(INFO_BYTES, dtype=torch.uint8, device=x.device)
    else:
        _bytes_buffer(info, "info", INFO_BYTES, x.device)
    _check(lib().profk_sae_encode_topk(ctypes.byref(p), _ptr(x), _ptr(w_enc), _ptr(b_enc), B, d_model, d_dict,
                                       k_row, seed, _ptr(out[0]), _ptr(out[1]), _ptr(ws), _nbytes(ws),
                                       _stream(), _ptr(info)))
    return out[0], out[1], info


def sae_encode_dense(x, w_enc, b_enc, out=None):
    """The latent matrix relu(x w_enc^T + b_enc), fp32 [B, d_dict]."""
    torch = _torch()
    B, d_model, d_dict = _sae_shape(x, w_enc, b_enc)
    if out is None:
        out = torch.empty((B, d_dict), dtype=torch.float32, device=x.device)
    else:
        _buffer(out, "out", torch.float32, B * d_dict, x.device)
    _check(lib().profk_sae_encode_dense(_ptr(x), _ptr(w_enc), _ptr(b_enc), B, d_model, d_dict, _ptr(out),
                                        _stream()))
    return out


def sae_decode(vals, flat_idx, w_dec, b_dec, B, out=None, ws=None):
    """x_hat fp32 [B, d_model] from selected latents (flat indices b*d_dict + j)."""
    torch = _torch()
    d_dict, d_model = w_dec.shape
    K = vals.numel()
    if w_dec.dtype != torch.bfloat16 or b_dec.dtype != torch.float32 or vals.dtype != torch.float32 or \
            flat_idx.dtype != torch.int64 or flat_idx.numel() != K:
        raise ProfkError("vals fp32 [K], flat_idx int64 [K], w_dec bf16 [d_dict, d_model], b_dec fp32 [d_model]")
    if not (vals.is_contiguous() and flat_idx.is_contiguous() and w_dec.is_contiguous() and b_dec.is_contiguous()):
        raise ProfkError("vals, flat_idx, w_dec and b_dec must be contiguous")
    if b_dec.numel() != d_model:
        raise ProfkError("b_dec must hold d_model values")
    for t, name in ((vals, "vals"), (flat_idx, "flat_idx"), (w_dec, "w_dec"), (b_dec, "b_dec")):
        _on_device(t, name, None if name == "vals" else vals.device)
    if out is None:
        out = torch.empty((B, d_model), dtype=torch.float32, device=vals.device)
    else:
        _buffer(out, "out", torch.float32, B * d_model, vals.device)
    n = int(lib().profk_sae_decode_workspace_size(B, K))
    if ws is None:
        ws = torch.empty(max(n, 1), dtype=torch.uint8, device=vals.device)
    else:
        _bytes_buffer(ws, "ws", n, vals.device)
    _check(lib().profk_sae_decode(_ptr(vals), _ptr(flat_idx), K, _ptr(w_dec), _ptr(b_dec), B, d_model, d_dict,
                                  _ptr(out), _ptr(ws), _nbytes(ws), _stream()))
    return out


def debug_sae_sample(x, w_enc, b_enc, p, seed=0, ws=None):
    """The keys of the S latents the fused path samples (uint32 as int64)."""
    torch = _torch()
    B, d_model, d_dict = _sae_shape(x, w_enc, b_enc)
    if ws is None:
        ws = sae_workspace(p, B, d_dict, x.device)
    else:
        _bytes_buffer(ws, "ws", int(lib().profk_sae_workspace_size(ctypes.byref(p), B, d_dict)), x.device)
    keys = torch.empty(p.S, dtype=torch.int32, device=x.device)
    _check(lib().profk_debug_sae_sample(ctypes.byref(p), _ptr(x), _ptr(w_enc), _ptr(b_enc), B, d_model, d_dict,
                                        seed, _ptr(keys), _ptr(ws), _nbytes(ws), _stream()))
    return keys.to(torch.int64) & 0xFFFFFFFF

