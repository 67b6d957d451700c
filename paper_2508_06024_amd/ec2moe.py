"""Python binding of libec2moe.so (ctypes): argument marshalling only.

Every function here checks tensor placement, dtype and shape, passes raw device
pointers and the current HIP stream to the C entry point of the same name, and raises
Ec2moeError on a non-OK status. All computation happens in the library's HIP kernels;
PyTorch only provides device memory and the stream. Importing this module fails
loudly if the library has not been built.
"""
from __future__ import annotations

import ctypes
import os
from typing import Optional, Sequence

import torch

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libec2moe.so")

F32, BF16 = 0, 1
GATE_RENORMALIZE = 1
EXPERT_RELU = 2
ACTIVATIONS = ("swiglu", "relu")

STATUS = {0: "ok", 1: "invalid argument", 2: "unsupported", 3: "too few candidates",
          4: "workspace too small", 5: "HIP error"}


class Ec2moeError(RuntimeError):
    def __init__(self, status: int, detail: str):
        super().__init__(f"{STATUS.get(status, status)}: {detail}")
        self.status = status
        self.detail = detail


class MoeDesc(ctypes.Structure):
    # field order of ec2moe_moe_desc: T, d, M, K, k, H, dtype (an int-sized enum), flags
    _fields_ = [("n_tokens", ctypes.c_int32), ("d_model", ctypes.c_int32), ("n_experts", ctypes.c_int32),
                ("n_groups", ctypes.c_int32), ("top_k", ctypes.c_int32), ("ffn_hidden", ctypes.c_int32),
                ("dtype", ctypes.c_int), ("flags", ctypes.c_uint32)]


class CodecDesc(ctypes.Structure):
    _fields_ = [("n_slices", ctypes.c_int32), ("h", ctypes.c_int32), ("w", ctypes.c_int32),
                ("r_h", ctypes.c_int32), ("r_w", ctypes.c_int32), ("dtype", ctypes.c_int)]


class GateOpts(ctypes.Structure):
    _fields_ = [("top_groups", ctypes.c_int32), ("group_sizes", ctypes.POINTER(ctypes.c_int32)),
                ("workspace", ctypes.c_void_p), ("workspace_bytes", ctypes.c_size_t)]


class DeviceState(ctypes.Structure):
    _fields_ = [("cpu", ctypes.c_double), ("mem", ctypes.c_double), ("power", ctypes.c_double),
                ("bandwidth", ctypes.c_double)]


class SelectionParams(ctypes.Structure):
    _fields_ = [("w_cpu", ctypes.c_double), ("w_mem", ctypes.c_double), ("w_power", ctypes.c_double),
                ("w_bandwidth", ctypes.c_double), ("epsilon", ctypes.c_double), ("max_fraction", ctypes.c_double)]


class ScheduleParams(ctypes.Structure):
    _fields_ = [(n, ctypes.c_double) for n in ("alpha", "beta", "epsilon", "t_end", "load_end", "load_cloud",
                                                "speed_end", "speed_cloud")]


class KernelStat(ctypes.Structure):
    _fields_ = [("name", ctypes.c_char * 48), ("launches", ctypes.c_int64), ("total_ms", ctypes.c_double)]


def _load():
    if not os.path.exists(LIB_PATH):
        raise ImportError(f"{LIB_PATH} is not built: run `python -m paper_2508_06024_amd.build` "
                          "(the HIP library is required; there is no fallback)")
    return ctypes.CDLL(LIB_PATH)


_lib = _load()

_P = ctypes.c_void_p
_SIGS = {
    "ec2moe_group_gate": [ctypes.POINTER(MoeDesc), ctypes.POINTER(ctypes.c_uint64), _P, _P, _P, _P, _P, _P, _P, _P, _P],
    "ec2moe_group_gate_ex": [ctypes.POINTER(MoeDesc), ctypes.POINTER(GateOpts), ctypes.POINTER(ctypes.c_uint64),
                             _P, _P, _P, _P, _P, _P, _P, _P, _P],
    "ec2moe_gate_workspace_size": [ctypes.POINTER(MoeDesc), ctypes.POINTER(ctypes.c_size_t)],
    "ec2moe_moe_workspace_size": [ctypes.POINTER(MoeDesc), ctypes.POINTER(ctypes.c_size_t)],
    "ec2moe_permute": [ctypes.POINTER(MoeDesc), _P, _P, _P, _P, _P, _P, _P, ctypes.c_size_t, _P],
    "ec2moe_permute_noalloc": [ctypes.POINTER(MoeDesc), _P, _P, _P, _P, _P, _P, _P],
    "ec2moe_expert_ffn": [ctypes.POINTER(MoeDesc), _P, _P, _P, _P, _P, _P, _P, _P, ctypes.c_size_t, _P],
    "ec2moe_combine": [ctypes.POINTER(MoeDesc), _P, _P, _P, _P, _P],
    "ec2moe_moe_forward": [ctypes.POINTER(MoeDesc), _P, _P, _P, _P, _P, _P, _P, ctypes.c_size_t, _P],
    "ec2moe_lowrank_workspace_size": [ctypes.POINTER(CodecDesc), ctypes.POINTER(ctypes.c_size_t)],
    "ec2moe_lowrank_encode": [ctypes.POINTER(CodecDesc), _P, _P, _P, _P, _P, ctypes.c_size_t, _P],
    "ec2moe_lowrank_decode": [ctypes.POINTER(CodecDesc), _P, _P, _P, _P, _P, ctypes.c_size_t, _P],
    "ec2moe_lowrank_fit_workspace_size": [ctypes.POINTER(CodecDesc), ctypes.POINTER(ctypes.c_size_t)],
    "ec2moe_lowrank_fit": [ctypes.POINTER(CodecDesc), _P, _P, _P, ctypes.c_int32, _P, _P, _P, _P, ctypes.c_size_t, _P],
    "ec2moe_status_string": [ctypes.c_int],
    "ec2moe_last_error": [],
    "ec2moe_profile_enable": [ctypes.c_int32],
    "ec2moe_profile_collect": [ctypes.POINTER(KernelStat), ctypes.c_int32, ctypes.POINTER(ctypes.c_int32)],
    "ec2moe_profile_select": [ctypes.c_char_p],
    "ec2moe_select_candidates": [ctypes.POINTER(DeviceState), ctypes.POINTER(SelectionParams), _P, ctypes.c_int32,
                                 ctypes.POINTER(ctypes.c_uint64), ctypes.POINTER(ctypes.c_int32)],
    "ec2moe_schedule_tasks": [ctypes.POINTER(ScheduleParams), _P, _P, ctypes.c_int32, _P, _P, _P],
}
for _name, _args in _SIGS.items():
    _fn = getattr(_lib, _name)
    _fn.argtypes = _args
    _fn.restype = ctypes.c_char_p if _name in ("ec2moe_status_string", "ec2moe_last_error") else ctypes.c_int

EXPORTS = tuple(_SIGS)


def _check(status: int):
    if status != 0:
        raise Ec2moeError(status, _lib.ec2moe_last_error().decode())


def _ptr(t: Optional[torch.Tensor]):
    return None if t is None else ctypes.c_void_p(t.data_ptr())


def _stream():
    return ctypes.c_void_p(torch.cuda.current_stream().cuda_stream)


def dtype_code(dt: torch.dtype) -> int:
    if dt == torch.bfloat16:
        return BF16
    if dt == torch.float32:
        return F32
    raise TypeError(f"unsupported dtype {dt}")


def _dev(t: torch.Tensor, name: str, dtype=None, shape=None):
    if not t.is_cuda:
        raise ValueError(f"{name} must be a device tensor")
    if not t.is_contiguous():
        raise ValueError(f"{name} must be contiguous")
    if dtype is not None and t.dtype != dtype:
        raise TypeError(f"{name} has dtype {t.dtype}, expected {dtype}")
    if shape is not None and tuple(t.shape) != tuple(shape):
        raise ValueError(f"{name} has shape {tuple(t.shape)}, expected {tuple(shape)}")
    return t


def moe_desc(n_tokens, n_experts, n_groups, d_model, ffn_hidden, top_k, dtype, renormalize=True,
             activation="swiglu") -> MoeDesc:
    if activation not in ACTIVATIONS:
        raise ValueError(f"activation must be one of {ACTIVATIONS}, got {activation!r}")
    flags = (GATE_RENORMALIZE if renormalize else 0) | (EXPERT_RELU if activation == "relu" else 0)
    return MoeDesc(n_tokens=n_tokens, d_model=d_model, n_experts=n_experts, n_groups=n_groups, top_k=top_k,
                   ffn_hidden=ffn_hidden, dtype=dtype if isinstance(dtype, int) else dtype_code(dtype), flags=flags)


def w_in_rows(ffn_hidden: int, activation: str) -> int:
    """Rows of one expert's input-layer weight: gate and up branches (SwiGLU) or W_in (ReLU)."""
    return ffn_hidden if activation == "relu" else 2 * ffn_hidden


def mask_array(words: Sequence[int]):
    return (ctypes.c_uint64 * len(words))(*[int(w) for w in words])


# ----------------------------------------------------------------------------- gate

def group_gate(desc: MoeDesc, mask_words, x, w_global, b_global, w_local, b_local, topk_idx, topk_w,
               probs=None):
    """Raw call: writes topk_idx [T][k] int32, topk_w [T][k] float32 (and probs [T][M])."""
    _check(_lib.ec2moe_group_gate(ctypes.byref(desc), mask_array(mask_words), _ptr(x), _ptr(w_global),
                                  _ptr(b_global), _ptr(w_local), _ptr(b_local), _ptr(topk_idx),
                                  _ptr(topk_w), _ptr(probs), _stream()))


def gate_opts(top_groups: int = 0, group_sizes: Optional[Sequence[int]] = None, workspace=None) -> GateOpts:
    """Options of group_gate_ex; workspace: a device tensor of gate_workspace_size bytes
    (small batches split d over more workgroups) or None."""
    sizes = None if group_sizes is None else (ctypes.c_int32 * len(group_sizes))(*[int(m) for m in group_sizes])
    opts = GateOpts(int(top_groups), ctypes.cast(sizes, ctypes.POINTER(ctypes.c_int32)) if sizes is not None else None,
                    None if workspace is None else workspace.data_ptr(),
                    0 if workspace is None else workspace.numel() * workspace.element_size())
    opts._sizes = sizes  # keeps the array and the workspace alive with the options
    opts._ws = workspace
    return opts


def gate_workspace_size(desc: MoeDesc) -> int:
    n = ctypes.c_size_t(0)
    _check(_lib.ec2moe_gate_workspace_size(ctypes.byref(desc), ctypes.byref(n)))
    return n.value


def group_gate_ex(desc: MoeDesc, opts: Optional[GateOpts], mask_words, x, w_global, b_global, w_local, b_local,
                  topk_idx, topk_w, probs=None):
    """Raw call with options (top-G groups, unequal group sizes)."""
    _check(_lib.ec2moe_group_gate_ex(ctypes.byref(desc), ctypes.byref(opts) if opts is not None else None,
                                     mask_array(mask_words), _ptr(x), _ptr(w_global), _ptr(b_global),
                                     _ptr(w_local), _ptr(b_local), _ptr(topk_idx), _ptr(topk_w), _ptr(probs),
                                     _stream()))


def gate(x, mask_words, w_global, b_global, w_local, b_local, n_groups, top_k, renormalize=True,
         with_probs=False, top_groups=0, group_sizes=None, split=False):
    """Group gate of x [T][d]; split: pass a gate workspace (small batches then split d)."""
    T, d = x.shape
    M = w_local.shape[0]
    dt = x.dtype
    _dev(x, "x", dt)
    _dev(w_global, "w_global", dt, (n_groups, d))
    _dev(w_local, "w_local", dt, (M, d))
    for b, n, name in ((b_global, n_groups, "b_global"), (b_local, M, "b_local")):
        if b is not None:
            _dev(b, name, torch.float32, (n,))
    desc = moe_desc(T, M, n_groups, d, 128, top_k, dt, renormalize)
    idx = torch.empty((T, top_k), dtype=torch.int32, device=x.device)
    w = torch.empty((T, top_k), dtype=torch.float32, device=x.device)
    probs = torch.empty((T, M), dtype=torch.float32, device=x.device) if with_probs else None
    if top_groups or group_sizes is not None or split:
        ws = None
        if split:
            ws = workspace(gate_workspace_size(desc), x.device)
        group_gate_ex(desc, gate_opts(top_groups, group_sizes, ws), mask_words, x, w_global, b_global, w_local,
                      b_local, idx, w, probs)
    else:
        group_gate(desc, mask_words, x, w_global, b_global, w_local, b_local, idx, w, probs)
    return (idx, w, probs) if with_probs else (idx, w)


# ----------------------------------------------------------------------------- MoE

def moe_workspace_size(desc: MoeDesc) -> int:
    n = ctypes.c_size_t(0)
    _check(_lib.ec2moe_moe_workspace_size(ctypes.byref(desc), ctypes.byref(n)))
    return n.value


def workspace(nbytes: int, device) -> torch.Tensor:
    return torch.empty(max(nbytes, 1), dtype=torch.uint8, device=device)


def _desc_for(x, top_k, n_experts, ffn_hidden, renormalize=True, n_groups=1):
    T, d = x.shape
    return moe_desc(T, n_experts, n_groups, d, ffn_hidden, top_k, x.dtype, renormalize)


def permute(topk_idx, n_experts, x=None, d_model=None, dtype=None, ws=None):
    T, k = topk_idx.shape
    _dev(topk_idx, "topk_idx", torch.int32)
    dev = topk_idx.device
    if x is not None:
        _dev(x, "x")
        d_model, dtype = x.shape[1], x.dtype
    d_model = d_model or 128
    dtype = dtype or torch.bfloat16
    desc = moe_desc(T, n_experts, 1, d_model, 128, k, dtype)
    ws = ws if ws is not None else workspace(moe_workspace_size(desc), dev)
    seg = torch.empty(n_experts + 1, dtype=torch.int32, device=dev)
    perm_src = torch.empty(T * k, dtype=torch.int32, device=dev)
    inv_perm = torch.empty(T * k, dtype=torch.int32, device=dev)
    x_perm = torch.empty((T * k, d_model), dtype=dtype, device=dev) if x is not None else None
    _check(_lib.ec2moe_permute(ctypes.byref(desc), _ptr(topk_idx), _ptr(x), _ptr(seg), _ptr(perm_src),
                               _ptr(inv_perm), _ptr(x_perm), _ptr(ws), ws.numel(), _stream()))
    return seg, perm_src, inv_perm, x_perm


def expert_ffn(x, seg_offsets, perm_src, w_gate_up, w_down, top_k, with_act=False, ws=None,
               activation="swiglu"):
    T, d = x.shape
    M, _, H = w_down.shape
    dt = x.dtype
    _dev(x, "x", dt)
    _dev(w_gate_up, "w_gate_up", dt, (M, w_in_rows(H, activation), d))
    _dev(w_down, "w_down", dt, (M, d, H))
    _dev(seg_offsets, "seg_offsets", torch.int32, (M + 1,))
    _dev(perm_src, "perm_src", torch.int32, (T * top_k,))
    desc = moe_desc(T, M, 1, d, H, top_k, dt, activation=activation)
    ws = ws if ws is not None else workspace(moe_workspace_size(desc), x.device)
    act = torch.empty((T * top_k, H), dtype=dt, device=x.device) if with_act else None
    y_perm = torch.empty((T * top_k, d), dtype=dt, device=x.device)
    _check(_lib.ec2moe_expert_ffn(ctypes.byref(desc), _ptr(x), _ptr(seg_offsets), _ptr(perm_src),
                                  _ptr(w_gate_up), _ptr(w_down), _ptr(act), _ptr(y_perm), _ptr(ws),
                                  ws.numel(), _stream()))
    return (y_perm, act) if with_act else y_perm


def combine(y_perm, inv_perm, topk_w):
    T, k = topk_w.shape
    d = y_perm.shape[1]
    _dev(y_perm, "y_perm", None, (T * k, d))
    _dev(inv_perm, "inv_perm", torch.int32, (T * k,))
    _dev(topk_w, "topk_w", torch.float32)
    desc = moe_desc(T, max(k, 1), 1, d, 128, k, y_perm.dtype)
    y = torch.empty((T, d), dtype=y_perm.dtype, device=y_perm.device)
    _check(_lib.ec2moe_combine(ctypes.byref(desc), _ptr(y_perm), _ptr(inv_perm), _ptr(topk_w), _ptr(y),
                               _stream()))
    return y


def permute_noalloc_into(desc: MoeDesc, topk_idx, seg_offsets, perm_src, inv_perm, x=None, x_perm=None):
    """Raw call of the workspace-free permutation (caller-owned outputs; the library allocates
    nothing)."""
    _check(_lib.ec2moe_permute_noalloc(ctypes.byref(desc), _ptr(topk_idx), _ptr(x), _ptr(seg_offsets),
                                       _ptr(perm_src), _ptr(inv_perm), _ptr(x_perm), _stream()))


def permute_into(desc: MoeDesc, topk_idx, seg_offsets, perm_src, inv_perm, ws, x=None, x_perm=None):
    """Raw call with caller-owned outputs and workspace (no allocation)."""
    _check(_lib.ec2moe_permute(ctypes.byref(desc), _ptr(topk_idx), _ptr(x), _ptr(seg_offsets), _ptr(perm_src),
                               _ptr(inv_perm), _ptr(x_perm), _ptr(ws), ws.numel(), _stream()))


def expert_ffn_into(desc: MoeDesc, x, seg_offsets, perm_src, w_gate_up, w_down, y_perm, ws, act=None):
    """Raw call with caller-owned outputs and workspace (no allocation)."""
    _check(_lib.ec2moe_expert_ffn(ctypes.byref(desc), _ptr(x), _ptr(seg_offsets), _ptr(perm_src),
                                  _ptr(w_gate_up), _ptr(w_down), _ptr(act), _ptr(y_perm), _ptr(ws),
                                  ws.numel(), _stream()))


def combine_into(desc: MoeDesc, y_perm, inv_perm, topk_w, y):
    """Raw call with a caller-owned output."""
    _check(_lib.ec2moe_combine(ctypes.byref(desc), _ptr(y_perm), _ptr(inv_perm), _ptr(topk_w), _ptr(y),
                               _stream()))


def moe_forward_into(desc: MoeDesc, x, topk_idx, topk_w, w_gate_up, w_down, y, ws):
    """Raw call with caller-owned output and workspace (no allocation)."""
    _check(_lib.ec2moe_moe_forward(ctypes.byref(desc), _ptr(x), _ptr(topk_idx), _ptr(topk_w),
                                   _ptr(w_gate_up), _ptr(w_down), _ptr(y), _ptr(ws), ws.numel(), _stream()))


def moe_forward(x, topk_idx, topk_w, w_gate_up, w_down, ws=None, activation="swiglu"):
    T, d = x.shape
    M, _, H = w_down.shape
    k = topk_idx.shape[1]
    dt = x.dtype
    _dev(x, "x", dt)
    _dev(topk_idx, "topk_idx", torch.int32, (T, k))
    _dev(topk_w, "topk_w", torch.float32, (T, k))
    _dev(w_gate_up, "w_gate_up", dt, (M, w_in_rows(H, activation), d))
    _dev(w_down, "w_down", dt, (M, d, H))
    desc = moe_desc(T, M, 1, d, H, k, dt, activation=activation)
    ws = ws if ws is not None else workspace(moe_workspace_size(desc), x.device)
    y = torch.empty((T, d), dtype=dt, device=x.device)
    moe_forward_into(desc, x, topk_idx, topk_w, w_gate_up, w_down, y, ws)
    return y


# ----------------------------------------------------------------------------- codec

def codec_desc(h, w, r_h, r_w, dtype, n_slices=1) -> CodecDesc:
    return CodecDesc(n_slices, h, w, r_h, r_w, dtype if isinstance(dtype, int) else dtype_code(dtype))


def lowrank_workspace_size(desc: CodecDesc) -> int:
    n = ctypes.c_size_t(0)
    _check(_lib.ec2moe_lowrank_workspace_size(ctypes.byref(desc), ctypes.byref(n)))
    return n.value


def lowrank_encode_into(desc: CodecDesc, x, u, v, z, ws):
    _check(_lib.ec2moe_lowrank_encode(ctypes.byref(desc), _ptr(x), _ptr(u), _ptr(v), _ptr(z), _ptr(ws),
                                      ws.numel(), _stream()))


def lowrank_decode_into(desc: CodecDesc, z, u_hat, v_hat, x_hat, ws):
    _check(_lib.ec2moe_lowrank_decode(ctypes.byref(desc), _ptr(z), _ptr(u_hat), _ptr(v_hat), _ptr(x_hat),
                                      _ptr(ws), ws.numel(), _stream()))


def lowrank_encode(x, u, v, ws=None):
    """Z = U^T X V; x [h][w] or [c][h][w]; returns float32 Z [r_h][r_w] (or [c][r_h][r_w])."""
    squeeze = x.dim() == 2
    xs = x.unsqueeze(0) if squeeze else x
    c, h, w = xs.shape
    r_h, r_w = u.shape[1], v.shape[1]
    dt = x.dtype
    _dev(xs, "x", dt)
    _dev(u, "u", dt, (h, r_h))
    _dev(v, "v", dt, (w, r_w))
    desc = codec_desc(h, w, r_h, r_w, dt, c)
    ws = ws if ws is not None else workspace(lowrank_workspace_size(desc), x.device)
    z = torch.empty((c, r_h, r_w), dtype=torch.float32, device=x.device)
    lowrank_encode_into(desc, xs, u, v, z, ws)
    return z[0] if squeeze else z


def lowrank_decode(z, u_hat, v_hat, ws=None):
    """X_hat = U_hat Z V_hat^T; returns [h][w] (or [c][h][w]) in the projections' dtype."""
    squeeze = z.dim() == 2
    zs = z.unsqueeze(0) if squeeze else z
    c, r_h, r_w = zs.shape
    h, w = u_hat.shape[0], v_hat.shape[0]
    dt = u_hat.dtype
    _dev(zs, "z", torch.float32)
    _dev(u_hat, "u_hat", dt, (h, r_h))
    _dev(v_hat, "v_hat", dt, (w, r_w))
    desc = codec_desc(h, w, r_h, r_w, dt, c)
    ws = ws if ws is not None else workspace(lowrank_workspace_size(desc), z.device)
    x_hat = torch.empty((c, h, w), dtype=dt, device=z.device)
    lowrank_decode_into(desc, zs, u_hat, v_hat, x_hat, ws)
    return x_hat[0] if squeeze else x_hat


def lowrank_fit(x, omega_u, omega_v, iters, ws=None):
    """Fit U [h][r_h], V [w][r_w] to calibration slices x [h][w] or [c][h][w] (layer dtype) from
    float32 start blocks; returns (u, v, status) with status a device int32 (0 = ok)."""
    xs = x if x.dim() == 3 else x.unsqueeze(0)
    c, h, w = xs.shape
    rh, rw = omega_u.shape[1], omega_v.shape[1]
    _dev(xs, "x")
    _dev(omega_u, "omega_u", torch.float32, (h, rh))
    _dev(omega_v, "omega_v", torch.float32, (w, rw))
    desc = codec_desc(h, w, rh, rw, xs.dtype, c)
    n = ctypes.c_size_t(0)
    _check(_lib.ec2moe_lowrank_fit_workspace_size(ctypes.byref(desc), ctypes.byref(n)))
    ws = ws if ws is not None else workspace(n.value, xs.device)
    u = torch.empty((h, rh), dtype=xs.dtype, device=xs.device)
    v = torch.empty((w, rw), dtype=xs.dtype, device=xs.device)
    status = torch.empty((1,), dtype=torch.int32, device=xs.device)
    _check(_lib.ec2moe_lowrank_fit(ctypes.byref(desc), _ptr(xs), _ptr(omega_u), _ptr(omega_v), int(iters), _ptr(u),
                                   _ptr(v), _ptr(status), _ptr(ws), ws.numel(), _stream()))
    return u, v, status


# ----------------------------------------------------------------------------- kernel timing

def profile_enable(on: bool = True):
    _check(_lib.ec2moe_profile_enable(1 if on else 0))


def profile_select(name=None):
    """Time only the kernels called `name` (None: all)."""
    _check(_lib.ec2moe_profile_select(name.encode() if name else None))


def profile_collect(max_entries: int = 64):
    """{kernel name: (launches, total ms)} of the kernels launched while profiling was on."""
    arr = (KernelStat * max_entries)()
    n = ctypes.c_int32(0)
    _check(_lib.ec2moe_profile_collect(arr, max_entries, ctypes.byref(n)))
    return {arr[i].name.decode(): (int(arr[i].launches), float(arr[i].total_ms)) for i in range(n.value)}


def last_error() -> str:
    return _lib.ec2moe_last_error().decode()


def status_string(code: int) -> str:
    return _lib.ec2moe_status_string(code).decode()


# ----------------------------------------------------------------------------- host planner

def _f64(a):
    import numpy as np
    return np.ascontiguousarray(a, dtype=np.float64)


def select_candidates(state: DeviceState, params: SelectionParams, complexity):
    """Candidate mask words of the experts the end device may run (host call; no GPU)."""
    v = _f64(complexity)
    M = int(v.size)
    words = (ctypes.c_uint64 * max(1, (M + 63) // 64))()
    n = ctypes.c_int32(0)
    _check(_lib.ec2moe_select_candidates(ctypes.byref(state), ctypes.byref(params), v.ctypes.data_as(_P), M, words,
                                         ctypes.byref(n)))
    return [int(w) for w in words][: (M + 63) // 64], n.value


def schedule_tasks(params: ScheduleParams, complexity, comm):
    """(location int32 [N]: 0 end, 1 cloud; order int32 [N]; (objective, load_end, load_cloud))."""
    import numpy as np
    c, m = _f64(complexity), _f64(comm)
    n = int(c.size)
    loc = np.zeros(n, np.int32)
    order = np.zeros(n, np.int32)
    summary = np.zeros(3, np.float64)
    _check(_lib.ec2moe_schedule_tasks(ctypes.byref(params), c.ctypes.data_as(_P), m.ctypes.data_as(_P), n,
                                      loc.ctypes.data_as(_P), order.ctypes.data_as(_P), summary.ctypes.data_as(_P)))
    return loc, order, tuple(float(x) for x in summary)
